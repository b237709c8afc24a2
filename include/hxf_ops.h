/*
 * hxf_ops.h -- the individual gfx950 kernels of one decoder iteration, exposed
 * for kernel-level parity tests, benchmarks and callers that drive their own
 * forward pass.
 *
 * All pointers are DEVICE pointers unless marked "host".  bf16 tensors are
 * uint16 bit patterns.  Every call enqueues work on `stream` (hipStream_t, may
 * be 0) and returns HXF_OK (0) or a negative hxf error code; errors are not
 * sticky and leave nothing enqueued.  The caller owns every buffer.  Calls
 * that build a work list on the host (attention) copy it into the caller's
 * `workspace` with an asynchronous host-to-device copy and synchronise the
 * stream before returning, so their host arguments may be freed afterwards.
 *
 * Physical KV layout (one layer), kv-head major: K pool [Hkv][n_blocks][dh/8][16][8]
 * (element (token t, dim d) of a page at ((d/8)*16 + t)*8 + d%8), then a separate
 * V pool [Hkv][n_blocks][dh][16] (V transposed inside a page: element (t, d) at
 * d*16 + v_pos(t), v_pos swapping bits 2 and 3 of t, i.e. the page's tokens in
 * groups of four in the order 0-3, 8-11, 4-7, 12-15); the token at
 * position p of a sequence with block table bt lives in slot bt[p/16]*16 + p%16.
 * `n_blocks` is the number of pages of the pool (its kv-head stride).
 */
#ifndef HXF_OPS_H
#define HXF_OPS_H

#include <stdint.h>

#include "hxf.h"

#ifdef __cplusplus
extern "C" {
#endif

/* GEMM epilogues, and layout flags that may be or-ed into the epilogue argument */
enum { HXF_EPI_BF16 = 0, HXF_EPI_RESID = 1, HXF_EPI_SWIGLU = 2, HXF_EPI_F32 = 3 };
enum { HXF_GEMM_A_PACKED = 0x100, HXF_GEMM_C_PACKED = 0x200 };

/* C = A[M,K] . B[N,K]^T, bf16 inputs, fp32 accumulation.  A is row-major with row
 * stride lda; B (and B2) are PACKED weights (hxf_op_pack_weight of the row-major
 * [N,K] matrix, or [F,K] for SwiGLU).
 *   HXF_EPI_BF16:   C bf16 [M, ldc]            C = bf16(acc)
 *   HXF_EPI_RESID:  C fp32 [M, ldc]            C += acc          (residual stream)
 *   HXF_EPI_SWIGLU: B = W_gate [F,K], B2 = W_up [F,K], N = 2F; C bf16 [M, ldc],
 *                   C[:, f] = bf16(silu(gate_f) * up_f), silu(z) = z / (1 + e^-z)
 *   HXF_EPI_F32:    C fp32 [M, ldc]            C = acc
 * K % 8 == 0, lda >= K.  workspace: hxf_op_gemm_workspace_bytes(M, N, K) bytes
 * (split-K partials for M <= 512, enough for every epilogue; may be 0 bytes).
 * HXF_GEMM_A_PACKED: A is in the packed layout of the weights (hxf_op_pack_weight of the
 * row-major [M,K] activations, ceil(M/16)*16 rows; lda unused), so that a 16 x 32 block of
 * it is one contiguous kilobyte; K % 32 == 0 (and F % 32 == 0 for SwiGLU).
 * HXF_GEMM_C_PACKED (SwiGLU, F % 32 == 0): C is written in that packed layout ([M,F] with
 * F/32 tiles per row tile; ldc unused), the form in which the down projection reads it.
 * Either flag on another shape: HXF_EINVAL. */
int64_t hxf_op_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K);
int hxf_op_gemm(const void* A, int32_t lda, const void* B, const void* B2, void* C, int32_t ldc, int32_t M, int32_t N,
                int32_t K, int32_t epilogue, void* workspace, int64_t workspace_bytes, void* stream);

/* hxf_op_gemm without a workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid it).
 * Same arguments and result as hxf_op_gemm (the layout flags are refused: HXF_EINVAL);
 * the split-K partials go to a device
 * array of HXF_GEMM_NOALLOC_MAX_BYTES that the library holds on each GPU it runs on
 * until the process ends (its address is looked up on the first call on a device,
 * which must be the current device).  Nothing is allocated.  HXF_ENOMEM (nothing
 * enqueued) when the plan's partials, splits * M * N * 4 bytes, exceed that size:
 * every plan with M <= 128 fits.  Calls on one GPU share the array: calls that
 * overlap on one GPU (several streams, several threads) race and must be serialised
 * by the caller. */
#define HXF_GEMM_NOALLOC_MAX_BYTES (16LL << 20)
int hxf_op_gemm_noalloc(const void* A, int32_t lda, const void* B, const void* B2, void* C, int32_t ldc, int32_t M,
                        int32_t N, int32_t K, int32_t epilogue, void* stream);

/* Packed weight layout, used for every GEMM weight: W [N,K] bf16 row-major becomes
 * tiles of 16 rows x 32 columns (1 KB), row-tiles outermost, zero padded to
 * ceil(N/16)*16 rows and ceil(K/32)*32 columns; inside a tile the 8-element chunks
 * are in the order [k%32 / 8][n%16], i.e. element (n, k) is at
 *   ((n/16) * ceil(K/32) + k/32) * 512 + ((k%32)/8) * 128 + (n%16) * 8 + k%8.
 * This is the operand order of the 16x16x32 bf16 MFMA, so a wavefront reads a tile
 * as one contiguous kilobyte.  hxf_op_pack_weight converts W (device, K % 8 == 0)
 * into out (device, hxf_packed_weight_bytes(N, K) bytes); W and out must not overlap. */
int64_t hxf_packed_weight_bytes(int32_t N, int32_t K);
int hxf_op_pack_weight(const void* W, int32_t N, int32_t K, void* out, void* stream);

/* out[r] = bf16(x[rows[r]] / sqrt(mean(x[rows[r]]^2) + eps) * g); rows may be NULL (identity).
 * x fp32 [*, d], g bf16 [d], out bf16 [n_rows, d]; d % 4 == 0. */
int hxf_op_rmsnorm(const float* x, const int32_t* rows, const void* g, void* out, int32_t n_rows, int32_t d,
                   float eps, void* stream);

/* resid[t] = float(E[ids[t]]); out[t] = rmsnorm(resid[t]) * g.  E bf16 [V, d]. */
int hxf_op_embed_rmsnorm(const int32_t* ids, const void* E, const void* g, float* resid, void* out, int32_t T,
                         int32_t d, float eps, void* stream);

/* RoPE table for positions [0, max_pos): float pairs (cos, sin) of p * base^(-2i/dh), i < dh/2,
 * computed in double on the host and copied to dst (max_pos * dh/2 * 8 bytes). */
int hxf_op_rope_table(void* dst, int32_t max_pos, int32_t head_dim, float base, void* stream);

/* qkv bf16 [T, (Hq+2Hkv)*dh] rows (q heads, k heads, v heads): rotate-half RoPE of q (in place)
 * and k at pos[t]; write rotated k and v to slot[t] of the K and V pools. */
int hxf_op_rope_kv_write(void* qkv, const int32_t* pos, const int32_t* slot, const void* rope_table, void* k_pool,
                         void* v_pool, int64_t n_blocks, int32_t T, int32_t Hq, int32_t Hkv, int32_t head_dim,
                         void* stream);

/* Write k, v bf16 [T, Hkv, dh] to slot[t] of the pools (no rotation). */
int hxf_op_kv_scatter(const void* k, const void* v, const int32_t* slot, void* k_pool, void* v_pool, int64_t n_blocks,
                      int32_t T, int32_t Hkv, int32_t head_dim, void* stream);

/* Decode attention, one query token per sequence: q bf16 [B, Hq, dh] (rotated), attends to positions
 * [0, ctx_host[b]) of sequence b through block table bt [B, bt_stride] (device); out bf16 [B, Hq, dh].
 * bt_host (may be NULL): the same block table on the host.  When given, sequences whose tables start
 * with the same physical pages (forks of one retained parent, e.g. the parallel candidate requests
 * of one query, Section 2.1) are grouped and their common full pages are read once for up to
 * min(8, 32 / (Hq/Hkv)) of them (a second 16-column MFMA tile reuses every K/V read when more
 * than 16 / (Hq/Hkv) rows share an item); the result is the same attention.  Each (sequence, kv-head) stream is
 * split into equal page-aligned partitions (at least 256 tokens, sized so that the work items fill
 * the wavefronts the chip holds at once, or, with more streams than those, no longer than an even
 * share of all the tokens over them), merged by log-sum-exp.
 * workspace: hxf_op_decode_attention_workspace_bytes(...) bytes (same ctx_host, bt_host, bt_stride). */
int64_t hxf_op_decode_attention_workspace_bytes(int32_t B, int32_t Hq, int32_t Hkv, int32_t head_dim,
                                                const int32_t* ctx_host, const int32_t* bt_host, int32_t bt_stride);
/* Introspection (host only, no device work): the decode-attention work list the two calls above
 * build.  items: n_items records of 24 int32 {kvh, t0, t1, n_rows, entry[8], part[8], pad[4]}
 * (tokens [t0, t1) of kv-head kvh through the pages of entry[0], attended by the first n_rows
 * entries, partial of row r in slot part[r]); the one-tile items (n_rows <= max(1, 16 / G)) come
 * first, then the two-tile items, each longest first; merges: n_merges records of 4 int32
 * {entry, kvh, part0, n_part}.  Returns HXF_ENOMEM (with the counts set) when a capacity is short. */
int hxf_op_decode_plan(int32_t B, int32_t Hq, int32_t Hkv, const int32_t* ctx_host, const int32_t* bt_host,
                       int32_t bt_stride, int32_t* items, int32_t items_cap, int32_t* n_items, int32_t* merges,
                       int32_t merges_cap, int32_t* n_merges);
int hxf_op_decode_attention(const void* q, const void* k_pool, const void* v_pool, int64_t n_blocks, const int32_t* bt,
                            int32_t bt_stride, const int32_t* ctx_host, const int32_t* bt_host, void* out, int32_t B,
                            int32_t Hq, int32_t Hkv, int32_t head_dim, void* workspace, int64_t workspace_bytes,
                            void* stream);

/* Causal prefill attention over chunks: chunk s has n_host[s] queries at positions
 * pos0_host[s] .. pos0_host[s]+n-1, stored at rows row0_host[s].. of q bf16 [*, Hq, dh];
 * it attends to positions [0, pos0+i] of its block table row bt[s] (device).  out rows as q. */
int64_t hxf_op_prefill_attention_workspace_bytes(int32_t S, int32_t Hq, int32_t Hkv, const int32_t* n_host);
/* Introspection (host only, no device work): the prefill-attention work list the call below
 * builds for the same chunks.  items: n_items records of 8 int32 {entry, kvh, q0, nq, t0, t1, part,
 * pad} (queries [q0, q0 + nq) of chunk `entry` on kv-head kvh over key tiles [t0, t1) of 32
 * positions; part = -1 for an item that writes its output, else the partial slot of a cut item),
 * in launch order; merges: n_merges records of 8 int32 {entry, kvh, q0, nq, part0, n_part, pad,
 * pad} (the partial slots [part0, part0 + n_part) of one cut item, combined by log-sum-exp).
 * Items are cut into key ranges only when there are fewer of them than CUs: those longer than an
 * even share of all key tiles over the resident workgroups (two per CU), at least 8 tiles.
 * HXF_ENOMEM (with the counts set) when a capacity is short. */
int hxf_op_prefill_plan(int32_t S, int32_t Hq, int32_t Hkv, const int32_t* pos0_host, const int32_t* n_host,
                        int32_t* items, int32_t items_cap, int32_t* n_items, int32_t* merges, int32_t merges_cap,
                        int32_t* n_merges);
int hxf_op_prefill_attention(const void* q, const void* k_pool, const void* v_pool, int64_t n_blocks, const int32_t* bt,
                             int32_t bt_stride, const int32_t* row0_host, const int32_t* pos0_host,
                             const int32_t* n_host, void* out, int32_t S, int32_t Hq, int32_t Hkv, int32_t head_dim,
                             void* workspace, int64_t workspace_bytes, void* stream);

/* out[r] = argmax over v of logits fp32 [R, V]; the lowest index wins ties. */
int hxf_op_argmax(const float* logits, int32_t* out, int32_t R, int32_t V, void* stream);

/* dst = src, bytes % 16 == 0 (HBM bandwidth probe). */
int hxf_op_copy(const void* src, void* dst, int64_t bytes, void* stream);

/* HBM read-bandwidth probe: reads src (bytes % 16 == 0) once with 16-byte loads and
 * writes to sink (device, HXF_READ_SINK_WORDS uint32 words, caller-owned) one word per
 * thread of the launch, the XOR of the 32-bit words that thread read; words of sink
 * past the launch's threads are left as they are, so the XOR of the whole sink, zeroed
 * first, is the XOR of every 32-bit word of src. */
#define HXF_READ_SINK_WORDS (4096 * 256)
int hxf_op_read(const void* src, int64_t bytes, uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* HXF_OPS_H */
