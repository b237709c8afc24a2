// Host-side launchers of the gfx950 kernels (one translation unit each).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace hxf {

// Physical KV layout (per layer; K pool then V pool), kv-head major:
//   K: [Hkv][n_blocks][dh/8][16 tokens][8]  (8-dimension chunks of the 16 tokens
//      side by side: the order in which a wavefront feeds them to the MFMA)
//   V: [Hkv][n_blocks][dh][16 positions]    (a dimension's 16 tokens contiguous, token t
//      at position v_pos(t): groups of four tokens in the order 0-3, 8-11, 4-7, 12-15,
//      the key order of the 32x32x16 MFMA's P operand in the prefill kernel)
// so one (page, kv-head) is one contiguous 16*dh*2-byte tile in each pool, and
// the pages of one kv-head of a sequence allocated together are contiguous.
constexpr int kPage = 16;
__host__ __device__ inline size_t kv_tile(int kvh, int64_t n_blocks, int blk, int dh) {
  return ((size_t)kvh * n_blocks + blk) * kPage * dh;
}
// Position of token t (0..15) inside a V page row: bits 2 and 3 swapped.
__host__ __device__ inline int v_pos(int t) { return (t & 3) | ((t >> 1) & 4) | ((t << 1) & 8); }

// ------------------------------------------------------------------ GEMM
enum { EPI_BF16 = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_F32 = 3 };

// Packed tile layout of a bf16 [rows, K] matrix (the weights', also used for the
// activations the prefill GEMMs read): 16-row x 32-column tiles of 1 KB, row tiles
// outermost, kt = ceil(K / 32) tiles per row tile, inside a tile [k%32 / 8][r%16][k%8].
// A DMA of one 16 x 32 block is then one contiguous kilobyte instead of 16 row pieces.
__host__ __device__ inline size_t packed_elem(int r, int k, int kt) {
  return ((size_t)(r >> 4) * kt + (k >> 5)) * 512 + ((k >> 3) & 3) * 128 + (r & 15) * 8 + (k & 7);
}

struct GemmArgs {
  const uint16_t* A;   // bf16 [M, lda]
  const uint16_t* B;   // bf16 [N, K] (SwiGLU: gate rows [F, K])
  const uint16_t* B2;  // SwiGLU: up rows [F, K]
  void* C;             // bf16 / fp32 output or fp32 residual, row stride ldc
  float* partial;      // split-K partials [splits][M][N] fp32
  int M, N, K;         // N is logical (2F for SwiGLU); K % 8 == 0
  int lda, ldc;
  int k_chunk;
  int kt;              // K tiles of the packed weights, ceil(K / 32)
  int a_packed;        // A is in the packed tile layout (lda unused); streaming and big-tile kernels
  int c_kt;            // SwiGLU: > 0 writes C in the packed tile layout with c_kt tiles per row tile
};

struct GemmPlan {
  bool stream = false;  // decode-sized M: LDS-DMA weight-streaming kernel
  bool big = false;     // prefill-sized M: LDS-DMA 32x32x16 MFMA kernel
  int cfg = 0;          // big kernel: macro-tile configuration
  int bm = 128;
  int bn = 128;
  int splits = 1;
  int k_chunk = 0;
};

// swiglu: the plan is for the SwiGLU epilogue (N = 2F logical columns)
GemmPlan gemm_plan(int M, int N, int K, int max_splits, bool swiglu = false);
// With reduce == false a split-K plan leaves its fp32 partials [splits][M][N] in
// a.partial for the consumer to sum (no reduction launch).  e0 / e1 (may be null):
// events recorded at the first kernel's start and the last kernel's end.
hipError_t gemm_launch(const GemmArgs& a, int epi, const GemmPlan& p, hipStream_t st, bool reduce = true,
                       hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// Weight packing: W bf16 [N, K] row-major -> tiles of 16 rows x 32 columns in MFMA
// operand order, zero padded to ceil(N/16)*16 rows and ceil(K/32)*32 columns.
size_t packed_weight_elems(int N, int K);
hipError_t pack_weight_launch(const uint16_t* W, int N, int K, uint16_t* out, hipStream_t st);

// ------------------------------------------------------------------ norms / embedding
// out[r] = bf16(rmsnorm(x[rows ? rows[r] : r]) * g); x fp32 [*, d]
hipError_t rmsnorm_launch(const float* x, const int32_t* rows, const uint16_t* g, uint16_t* out,
                          int n_rows, int d, float eps, hipStream_t st);
// x[rows[r]] += sum over z < S of part[z][rows[r]] (split-K partials [S][part_rows][d] of a
// residual GEMM, in split order), then out[r] = bf16(rmsnorm(x[rows[r]]) * g); out_kt > 0
// writes out in the packed tile layout (d / 32 tiles per row tile, d % 32 == 0)
hipError_t resid_rmsnorm_launch(float* x, const float* part, int S, int part_rows, const int32_t* rows,
                                const uint16_t* g, uint16_t* out, int n_rows, int d, float eps, hipStream_t st,
                                int out_kt = 0);
// resid[t] = E[ids[t]] (fp32); out[t] = bf16(rmsnorm(resid[t]) * g) (packed as above with out_kt)
hipError_t embed_rmsnorm_launch(const int32_t* ids, const uint16_t* E, const uint16_t* g, float* resid,
                                uint16_t* out, int T, int d, float eps, hipStream_t st, int out_kt = 0);

// ------------------------------------------------------------------ RoPE + KV write
// qkv bf16 [T, (Hq+2Hkv)*dh]: rotates q (in place) and k at pos[t] with the
// table cs[pos][i] = (cos, sin) of pos * base^(-2i/dh); writes k and v to slot[t].
hipError_t rope_kv_launch(uint16_t* qkv, const int32_t* pos, const int32_t* slot, const float2* cs,
                          uint16_t* k_pool, uint16_t* v_pool, int64_t n_blocks, int T, int Hq, int Hkv, int dh,
                          hipStream_t st);
// The same with the projection given as S split-K partials part [S][T][(Hq+2Hkv)*dh]
// (each value = bf16 of their sum in split order); rotated q goes to qkv.
hipError_t rope_kv_partials_launch(uint16_t* qkv, const float* part, int S, const int32_t* pos, const int32_t* slot,
                                   const float2* cs, uint16_t* k_pool, uint16_t* v_pool, int64_t n_blocks, int T,
                                   int Hq, int Hkv, int dh, hipStream_t st);
// Write k, v bf16 [T, Hkv, dh] to slot[t] (no rotation).
hipError_t kv_scatter_launch(const uint16_t* k, const uint16_t* v, const int32_t* slot, uint16_t* k_pool,
                             uint16_t* v_pool, int64_t n_blocks, int T, int Hkv, int dh, hipStream_t st);

// ------------------------------------------------------------------ attention
// One decode work item: tokens [t0, t1) of kv-head `kvh`, read through the block
// table of entry[0], attended by the queries of entries entry[0 .. n_rows) (more
// than one when they share those pages: forks of one parent); row r's partial
// result goes to slot part[r].  The query columns of a wavefront are (row, head)
// pairs: one tile of 16 (at most 16 / G rows) or, for a wide item, two tiles of 16
// (at most min(kDecodeRows, 32 / G) rows) that share every K/V read.
constexpr int kDecodeRows = 8;
struct DecodeItem {
  int32_t kvh, t0, t1, n_rows;
  int32_t entry[kDecodeRows];
  int32_t part[kDecodeRows];
  int32_t pad[4];
};
// Rows one 16-column tile holds, and the rows a wide (two-tile) item holds, for GQA group G.
inline int decode_rows_narrow(int G) { return std::max(1, std::min(kDecodeRows, 16 / G)); }
inline int decode_rows_wide(int G) { return std::max(1, std::min(kDecodeRows, 32 / G)); }
// Launch order of the decode items: longest first (equal lengths keep their
// order), so that the wavefronts that start last, when the chip drains, are the
// short tail partitions.  Partial slots are unchanged, so the merge is unaffected.
inline void order_decode_items(DecodeItem* it, size_t n) {
  std::stable_sort(it, it + n, [](const DecodeItem& x, const DecodeItem& y) { return x.t1 - x.t0 > y.t1 - y.t0; });
}
// Decode work split.  Each (sequence, kv-head) context is cut into equal, page-aligned
// partitions no longer than a per-launch target.  With fewer (stream, kv-head) pairs than
// the wavefronts the chip holds at once (two per SIMD at the one-tile kernel's register
// count, 2 x 4 x 256), the target makes the items just fill them.  With more pairs each
// already has an item, and the target is an even share of all the tokens over the
// resident wavefronts: a stream much longer than the others (the shared prefix of a fork
// group next to the forks' short own tails) is cut instead of running alone after the
// rest have drained.  A partition is never shorter than kDecodeMinPartition tokens
// unless its whole context is.
constexpr int kDecodeResident = 2048;
constexpr int kDecodeMinPartition = 256;
inline int64_t decode_target_tokens(int64_t sum_ctx, int64_t n_seqs, int64_t hkv) {
  const int64_t pairs = n_seqs * hkv;
  const int64_t slots = pairs < kDecodeResident ? kDecodeResident - pairs : kDecodeResident;
  return std::max<int64_t>((sum_ctx * hkv + slots - 1) / slots, kDecodeMinPartition);
}
// Partition length (a whole number of pages) for a context of ctx tokens; its
// ceil(ctx / length) parts number at most ceil(ctx / target).
inline int decode_part_len(int ctx, int64_t target) {
  const int64_t n = ((int64_t)ctx + target - 1) / target;
  const int64_t len = ((int64_t)ctx + n - 1) / n;
  return (int)((len + kPage - 1) / kPage * kPage);
}
// One merge job per (entry, kv-head): partials [part0, part0 + n_part).
struct MergeItem {
  int32_t entry, kvh, part0, n_part;
};
struct DecodeAttnArgs {
  const uint16_t* q;       // bf16, q of entry e at q + q_row[e]*q_stride (+ head*dh)
  const int32_t* q_row;    // [entries]
  int q_stride;
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  int64_t n_blocks;
  const int32_t* bt;       // [entries][bt_stride]
  int bt_stride;
  const DecodeItem* items;     // n_items one-tile items, then n_wide two-tile items
  int n_items;                 // one-tile items, or that launch's capacity when n_items_dev is set
  int n_wide;                  // two-tile items, or that launch's capacity when n_items_dev is set
  const int32_t* n_items_dev;  // may be null: both counts in device memory (captured launches)
  const MergeItem* merges;
  int n_merges;
  float* part_o;           // [parts][G][dh]
  float* part_ml;          // [parts][G][2]  (max in log2 units, sum)
  uint16_t* out;           // bf16, row q_row[e]*out_stride + head*dh
  int out_stride;
  int out_kt;              // > 0: out in the packed tile layout with out_kt tiles per row tile
  int Hq, Hkv, dh;
  float scale_log2;        // log2(e) / sqrt(dh)
};
// Split-K partials of every work item, then the log-sum-exp merge into `out`.
// ev_start / ev_stop (may be null): events that record the kernel's own start and end.
hipError_t decode_attn_launch(const DecodeAttnArgs& a, hipStream_t st, hipEvent_t ev_start = nullptr,
                              hipEvent_t ev_stop = nullptr);
hipError_t decode_merge_launch(const DecodeAttnArgs& a, hipStream_t st, hipEvent_t ev_start = nullptr,
                               hipEvent_t ev_stop = nullptr);

// One prefill work item: queries [q0, q0 + nq) (chunk-local) of entry `entry`, kv-head
// `kvh`, attending keys of the 32-key tiles [t0, t1).  part < 0: the item covers every
// key its queries see and writes the normalized output; otherwise it writes its
// unnormalized partial (output, running max, sum) to slot `part`, and a merge job
// combines the slots of its query block by log-sum-exp.
struct PrefillItem {
  int32_t entry, kvh, q0, nq;
  int32_t t0, t1, part, pad;
};
// Merge job: partial slots [part0, part0 + n_part) of (entry, kvh, queries [q0, q0 + nq)).
struct PrefillMerge {
  int32_t entry, kvh, q0, nq;
  int32_t part0, n_part, pad0, pad1;
};
// Launch order of the prefill items: most key tiles first (equal counts keep their
// order), so that the short items fill the chip's tail instead of the long ones.
inline void order_prefill_items(PrefillItem* it, size_t n) {
  std::stable_sort(it, it + n, [](const PrefillItem& x, const PrefillItem& y) { return x.t1 - x.t0 > y.t1 - y.t0; });
}
// Workgroups of the prefill kernel resident at once (two per CU: 80 KB of LDS each),
// and the shortest key range an item is split into.
constexpr int kPrefillResident = 512;
// (query, head) pairs of one prefill item (its workgroup's columns), and of a partial slot
constexpr int kPrefillPairs = 128;
constexpr int kPrefillMinTiles = 8;
struct PrefillAttnArgs {
  const uint16_t* q;       // bf16 rows; entry e's query i at row row0[e] + i
  int q_stride;
  const int32_t* row0;     // [entries]
  const int32_t* pos0;     // [entries] position of the entry's first query
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  int64_t n_blocks;
  const int32_t* bt;       // [entries][bt_stride]
  int bt_stride;
  const PrefillItem* items;
  int n_items;
  const PrefillMerge* merges;   // merge jobs of the split items
  int n_merges;
  float* part_o;                // [slots][128 pairs][dh]: unnormalized partial outputs
  float* part_ml;               // [slots][128 pairs][2]: (max in log2 units, sum)
  uint16_t* out;
  int out_stride;
  int out_kt;                   // > 0: out in the packed tile layout with out_kt tiles per row tile
  int Hq, Hkv, dh;
  float scale_log2;
};
// The items, then (when some are split) the merge of their partials.
hipError_t prefill_attn_launch(const PrefillAttnArgs& a, hipStream_t st, hipEvent_t ev_start = nullptr,
                               hipEvent_t ev_stop = nullptr);
// Queries covered by one prefill work item for a given GQA group size.
int prefill_queries_per_item(int group);

// ------------------------------------------------------------------ sampling / misc
// out[r] = argmax_v logits[r][v], the lowest index among equal maxima.
hipError_t argmax_launch(const float* logits, int32_t* out, int R, int V, hipStream_t st);
// dst = src (bytes % 16 == 0); HBM bandwidth probe.
hipError_t copy_launch(const void* src, void* dst, size_t bytes, hipStream_t st);
// Read-bandwidth probe: at most kReadProbeBlocks workgroups of 256 threads; thread t of
// the launch writes sink[t] (the XOR of the words it read), the rest of sink is untouched.
constexpr int kReadProbeBlocks = 4096;
hipError_t read_launch(const void* src, size_t bytes, uint32_t* sink, hipStream_t st);

}  // namespace hxf
