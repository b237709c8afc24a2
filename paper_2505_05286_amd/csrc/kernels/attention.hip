// Paged attention on CDNA4 matrix cores: flash-decoding split-K decode
// (+ log-sum-exp merge) and chunked-prefill causal attention.
//
// Both run the same per-wavefront inner loop over pairs of 16-token pages,
// in a transposed formulation so that every lane owns one query column:
//
//   S^T[32 tok x 16 cols] = K_pages[32 x dh] . Q^T[dh x 16]     (v_mfma_f32_16x16x32_bf16)
//   O^T[dh x 16 cols]    += V^T[dh x 32 tok] . P^T[32 x 16]
//
// A column is one (query, head) pair: the G heads of a GQA group for decode
// (one K/V read serves the whole group), or QPW queries x G heads for
// prefill.  With the MFMA output layout (lane l holds rows 4*(l/16)+e of
// column l%16), the score tile that QK^T leaves in a lane is exactly the P^T
// operand the PV product needs from that lane, so softmax runs in registers
// with only two cross-lane exchanges per page pair (xor 16, xor 32).
// K pages are stored in MFMA operand order (see kernels.hpp), so each K load
// instruction of a wavefront reads 1 KiB of contiguous memory; V pages are
// stored transposed ([dh][token]) and read as 8-byte vectors, 512 contiguous
// bytes per instruction.
#include <hip/hip_ext.h>

#include "common.hpp"
#include "kernels.hpp"

namespace hxf {

namespace {

constexpr float kNegInf = -__builtin_huge_valf();

template <int DH>
struct PairRegs {
  uint4 ka[DH / 32], kb[DH / 32];
  uint2 va[DH / 16], vb[DH / 16];
};

template <int DH>
struct AttnState {
  f32x4 acc[DH / 16];
  float m;   // running max of this lane's column (log2 units); identical across the 4 lane rows
  float l;   // lane-local partial softmax denominator
};

template <int DH>
__device__ __forceinline__ void load_page(uint4* k, uint2* v, const uint16_t* k_pool, const uint16_t* v_pool,
                                          size_t tile, int lane) {
  const uint16_t* kp = k_pool + tile + lane * 8;
  const uint16_t* vp = v_pool + tile + (lane & 15) * kPage + v_pos((lane >> 4) * 4);   // tokens 4g..4g+3
#pragma unroll
  for (int s = 0; s < DH / 32; ++s) k[s] = load_stream16(kp + s * 512);
#pragma unroll
  for (int n = 0; n < DH / 16; ++n) v[n] = load_stream8(vp + n * 16 * kPage);
}

template <int DH>
__device__ __forceinline__ void load_pair(PairRegs<DH>& R, const uint16_t* k_pool, const uint16_t* v_pool,
                                          const int32_t* bt, int64_t nb, int kvh, int page, int t_end, int lane) {
  load_page<DH>(R.ka, R.va, k_pool, v_pool, kv_tile(kvh, nb, bt[page], DH), lane);
  if ((page + 1) * kPage < t_end) {
    load_page<DH>(R.kb, R.vb, k_pool, v_pool, kv_tile(kvh, nb, bt[page + 1], DH), lane);
  } else {
#pragma unroll
    for (int s = 0; s < DH / 32; ++s) R.kb[s] = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int n = 0; n < DH / 16; ++n) R.vb[n] = make_uint2(0, 0);
  }
}

// Mask keeping the first n (0..4) of the 4 bf16 V entries a lane holds for one
// page: tokens at or beyond the context end may hold anything, and a zero
// probability times a NaN would still be NaN.
__device__ __forceinline__ uint2 keep_mask(int n) {
  const uint64_t m = n >= 4 ? ~0ull : (n <= 0 ? 0ull : ((1ull << (16 * n)) - 1));
  return make_uint2((uint32_t)m, (uint32_t)(m >> 32));
}

// Scores, online softmax and PV product of one page pair for NT column tiles of 16
// (query, head) pairs each; the K/V registers are shared by the tiles.
template <int DH, bool CAUSAL, int NT>
__device__ __forceinline__ void compute_pair(AttnState<DH> (&S)[NT], const PairRegs<DH>& R,
                                             const bf16x8 (&qf)[NT][DH / 32], int page, int t_end, int lim,
                                             float scale_log2, int lane) {
  const int rq = lane >> 4;
  const int ta = page * kPage + rq * 4;   // first token of this lane's rows in page a
  const int tb = ta + kPage;
  const bool full = (page + 2) * kPage <= t_end;   // wavefront-uniform
  uint2 ma = make_uint2(~0u, ~0u), mb = make_uint2(~0u, ~0u);
  if (!full) {
    ma = keep_mask(t_end - ta);
    mb = keep_mask(t_end - tb);
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < DH / 32; ++s) {
      sa = mfma16x16x32(as_bf16x8(R.ka[s]), qf[t][s], sa);
      sb = mfma16x16x32(as_bf16x8(R.kb[s]), qf[t][s], sb);
    }
    float x[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = sa[e] * scale_log2;
      x[4 + e] = sb[e] * scale_log2;
    }
    if (!full) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (ta + e >= t_end) x[e] = kNegInf;
        if (tb + e >= t_end) x[4 + e] = kNegInf;
      }
    }
    if (CAUSAL) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (ta + e > lim) x[e] = kNegInf;
        if (tb + e > lim) x[4 + e] = kNegInf;
      }
    }
    float mx = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
    mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float m_new = fmaxf(S[t].m, mx);
    const float alpha = exp2f(S[t].m - m_new);
    float p[8];
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      p[e] = exp2f(x[e] - m_new);
      psum += p[e];
    }
    S[t].l = S[t].l * alpha + psum;
    S[t].m = m_new;
    const bf16x8 pf = as_bf16x8(make_uint4(pack_bf2(p[0], p[1]), pack_bf2(p[2], p[3]), pack_bf2(p[4], p[5]),
                                           pack_bf2(p[6], p[7])));
#pragma unroll
    for (int n = 0; n < DH / 16; ++n) {
      S[t].acc[n] *= alpha;
      const uint4 v = make_uint4(R.va[n].x & ma.x, R.va[n].y & ma.y, R.vb[n].x & mb.x, R.vb[n].y & mb.y);
      S[t].acc[n] = mfma16x16x32(as_bf16x8(v), pf, S[t].acc[n]);
    }
  }
}

// Attend the lanes' columns (NT tiles) to tokens [t_begin, t_end) (t_begin page
// aligned); tokens beyond `lim` are masked.
template <int DH, bool CAUSAL, int NT>
__device__ __forceinline__ void attn_range(AttnState<DH> (&S)[NT], const bf16x8 (&qf)[NT][DH / 32],
                                           const uint16_t* k_pool, const uint16_t* v_pool, const int32_t* bt,
                                           int64_t nb, int kvh, int t_begin, int t_end, int lim, float scale_log2,
                                           int lane) {
#pragma unroll
  for (int t = 0; t < NT; ++t) {
#pragma unroll
    for (int n = 0; n < DH / 16; ++n) S[t].acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
    S[t].m = kNegInf;
    S[t].l = 0.f;
  }
  const int p0 = t_begin / kPage, p_end = (t_end + kPage - 1) / kPage;
  // two register buffers used in turn: the loads of the next page pair are in
  // flight while the current one is multiplied
  PairRegs<DH> ra, rb;
  load_pair<DH>(ra, k_pool, v_pool, bt, nb, kvh, p0, t_end, lane);
  for (int p = p0; p < p_end; p += 4) {
    if (p + 2 < p_end) load_pair<DH>(rb, k_pool, v_pool, bt, nb, kvh, p + 2, t_end, lane);
    compute_pair<DH, CAUSAL, NT>(S, ra, qf, p, t_end, lim, scale_log2, lane);
    if (p + 2 >= p_end) break;
    if (p + 4 < p_end) load_pair<DH>(ra, k_pool, v_pool, bt, nb, kvh, p + 4, t_end, lane);
    compute_pair<DH, CAUSAL, NT>(S, rb, qf, p + 2, t_end, lim, scale_log2, lane);
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    S[t].l += __shfl_xor(S[t].l, 16, kWave);
    S[t].l += __shfl_xor(S[t].l, 32, kWave);
  }
}

template <int DH>
__device__ __forceinline__ void load_q(bf16x8* qf, const uint16_t* qrow, bool ok, int lane) {
  const int rq = lane >> 4;
#pragma unroll
  for (int s = 0; s < DH / 32; ++s)
    qf[s] = ok ? as_bf16x8(*reinterpret_cast<const uint4*>(qrow + s * 32 + rq * 8)) : as_bf16x8(make_uint4(0, 0, 0, 0));
}

// One wavefront per work item.  NT = 1: the 16 query columns are (row, head of the
// group) pairs of up to 16/G rows; NT = 2 (wide items of a shared prefix): 32 columns,
// up to 32/G rows, the second tile reusing every K/V page read for the first.  The
// NT = 1 kernel takes the items [0, n_items), the NT = 2 kernel the n_wide items
// that follow them (counts from device memory in captured launches).
template <int DH, int NT>
__global__ __launch_bounds__(64) void decode_attn_kernel(DecodeAttnArgs a) {
  const int lane = threadIdx.x;
  int w = blockIdx.x;
  if (NT == 1) {
    if (w >= (a.n_items_dev ? a.n_items_dev[0] : a.n_items)) return;
  } else {
    if (w >= (a.n_items_dev ? a.n_items_dev[1] : a.n_wide)) return;
    w += a.n_items_dev ? a.n_items_dev[0] : a.n_items;
  }
  // the item's scalar fields are wavefront-uniform loads; a lane reads its own row's
  // entry and partial slot with one vector load each (no private copy of the record)
  const DecodeItem* it = a.items + w;
  const int kvh = it->kvh, t0 = it->t0, t1 = it->t1, n_rows = it->n_rows, entry0 = it->entry[0];
  const int G = a.Hq / a.Hkv;
  bf16x8 qf[NT][DH / 32];
  bool ok[NT];
  int part[NT], g[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    // column (tile t, lane % 16) = (row, head of the group); rows past n_rows are idle columns
    const int col = t * 16 + (lane & 15);
    const int row = col / G;
    g[t] = col - row * G;
    ok[t] = row < n_rows && row < kDecodeRows;
    const int r = ok[t] ? row : 0;
    const int entry = it->entry[r];
    part[t] = it->part[r];
    const int head = kvh * G + (ok[t] ? g[t] : 0);
    load_q<DH>(qf[t], a.q + (size_t)a.q_row[entry] * a.q_stride + head * DH, ok[t], lane);
  }
  AttnState<DH> S[NT];
  attn_range<DH, false, NT>(S, qf, a.k_pool, a.v_pool, a.bt + (size_t)entry0 * a.bt_stride, a.n_blocks, kvh, t0, t1,
                            0x7FFFFFFF, a.scale_log2, lane);
  const int rq = lane >> 4;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (!ok[t]) continue;
    float* o = a.part_o + ((size_t)part[t] * G + g[t]) * DH;
#pragma unroll
    for (int n = 0; n < DH / 16; ++n)
      *reinterpret_cast<float4*>(o + n * 16 + rq * 4) =
          make_float4(S[t].acc[n][0], S[t].acc[n][1], S[t].acc[n][2], S[t].acc[n][3]);
    if (rq == 0) *reinterpret_cast<float2*>(a.part_ml + ((size_t)part[t] * G + g[t]) * 2) = make_float2(S[t].m, S[t].l);
  }
}

// Log-sum-exp merge of the split-K partials; one wavefront per (entry, q-head).
// Lane j holds (max, sum) of partial j, so the common maximum, the weights and
// their sum take one load and two cross-lane reductions; the partial outputs of
// the first kMergeChunk partials are loaded before that, so a merge of up to
// kMergeChunk partials is one memory round trip.  Partials beyond 64 (contexts
// over 64 partitions) are weighted from broadcast loads.
constexpr int kMergeChunk = 8;

template <int DH>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeAttnArgs a) {
  const int G = a.Hq / a.Hkv;
  // wavefront-uniform job: the item and the output row come through scalar loads
  const int job = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (job >= a.n_merges * G) return;
  const int lane = threadIdx.x & 63;
  const MergeItem mi = a.merges[job / G];
  const int g = job % G;
  const int n = mi.n_part;
  const int orow = a.q_row[mi.entry];
  constexpr int PER = DH / 64;   // dims per lane
  const float2* ml = reinterpret_cast<const float2*>(a.part_ml) + (size_t)mi.part0 * G + g;
  const float* po = a.part_o + ((size_t)mi.part0 * G + g) * DH + lane * PER;
  const size_t ostride = (size_t)G * DH;
  float x[kMergeChunk][PER];
#pragma unroll
  for (int j = 0; j < kMergeChunk; ++j) {
    if (j < n) {
      if constexpr (PER == 2) {
        const float2 v = *reinterpret_cast<const float2*>(po + j * ostride);
        x[j][0] = v.x;
        x[j][PER - 1] = v.y;
      } else {
        x[j][0] = po[j * ostride];
      }
    }
  }
  const float2 mine = lane < n ? ml[(size_t)lane * G] : make_float2(kNegInf, 0.f);
  float M = mine.x;
  for (int p = lane + kWave; p < n; p += kWave) M = fmaxf(M, ml[(size_t)p * G].x);
  M = wave_max(M);
  const float wl = lane < n ? exp2f(mine.x - M) : 0.f;
  float L = wave_sum(wl * mine.y);
  float acc[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) acc[k] = 0.f;
#pragma unroll
  for (int j = 0; j < kMergeChunk; ++j) {
    if (j < n) {
      const float w = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wl), j));
#pragma unroll
      for (int k = 0; k < PER; ++k) acc[k] += w * x[j][k];
    }
  }
  for (int p = kMergeChunk; p < n; ++p) {
    float w;
    if (p < kWave) {
      w = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wl), p));
    } else {
      const float2 v = ml[(size_t)p * G];
      w = exp2f(v.x - M);
      L += w * v.y;
    }
    const float* o = po + p * ostride;
    if constexpr (PER == 2) {
      const float2 v = *reinterpret_cast<const float2*>(o);
      acc[0] += w * v.x;
      acc[PER - 1] += w * v.y;
    } else {
      acc[0] += w * o[0];
    }
  }
  const float inv = 1.f / L;
  const int col = (mi.kvh * G + g) * DH + lane * PER;   // (PER columns in one 8-column group)
  uint16_t* out = a.out + (a.out_kt ? packed_elem(orow, col, a.out_kt) : (size_t)orow * a.out_stride + col);
  if constexpr (PER == 2) *reinterpret_cast<uint32_t*>(out) = pack_bf2(acc[0] * inv, acc[PER - 1] * inv);
  else out[0] = f2bf(acc[0] * inv);
}

// Chunked-prefill causal attention, one workgroup per (chunk, kv-head, block of
// 128·PT/G queries): the 128·PT (query, head) pairs of the block are the columns of
//   S^T[32 keys x 32 pairs] = K[32 x dh] . Q^T[dh x 32]       (v_mfma_f32_32x32x16_bf16)
//   O^T[32 dims x 32 pairs] += V^T[32 x 32 keys] . P^T[32 x 32]
// (PT tiles of 32 pairs per wavefront; the library launches PT = 1, 128 pairs per
// workgroup).  Tiles of 32 keys (two pages) of K and V are moved into LDS by the DMA
// path, five tiles in flight, and shared by the four wavefronts.  A lane of the S^T
// accumulator holds keys 8m + 4h + i (h = lane / 32) of its pair; taken in the order
// m = 2s, 2s + 1 these are the 8 keys of the P^T operand for the 16-key step s (page s
// of the tile); the V pool stores each page row with its tokens in that order (see
// v_pos), so the V^T operand of a lane is one contiguous 16-byte LDS read.  Softmax is
// online in log2 units, one exchange of the wavefront halves per tile for the max.
template <int DH, int PT>
__global__ __launch_bounds__(256) void prefill_flash_kernel(PrefillAttnArgs a) {
  constexpr int KS = DH / 16;                  // 16-dim steps of QK^T
  constexpr int DT = DH / 32;                  // 32-dim tiles of O^T
  constexpr int KT = 32 * DH;                  // elements of a K (or V) tile of 32 keys
  constexpr int STAGE = 2 * KT;                // K tile then V tile
  constexpr int K_W = KT / 512 / 4;            // 16-byte DMA instructions per wavefront for K
  constexpr int V_W = KT / 512 / 4;            // and for V
  constexpr int PER_W = K_W + V_W;
  constexpr int NS = 5;                        // key tiles in flight: NS - 1 ahead of the one computed
  __shared__ __attribute__((aligned(1024))) bf16_t L0[STAGE], L1[STAGE], L2[STAGE], L3[STAGE], L4[STAGE];
  auto slot = [&](auto ic) -> bf16_t* {
    constexpr int I = decltype(ic)::value % NS;
    if constexpr (I == 0) return L0; else if constexpr (I == 1) return L1; else if constexpr (I == 2) return L2;
    else if constexpr (I == 3) return L3; else return L4;
  };
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const PrefillItem it = a.items[blockIdx.x];
  const int G = a.Hq / a.Hkv;
  const int npairs = it.nq * G;
  const int pos0 = a.pos0[it.entry];
  const int kend = pos0 + it.q0 + it.nq;       // keys [0, kend) are visible to some pair
  const int tbase = it.t0;                     // this item's key tiles: [t0, t1)
  const int ntiles = it.t1 - it.t0;
  const int last_page = (kend - 1) / kPage;
  // the block table does not change during the kernel: read it through the constant
  // address space, so that its (wavefront-uniform) entries come by scalar loads, which
  // are counted apart from the vector loads and do not wait for the DMAs in flight
  const __attribute__((address_space(4))) int32_t* bt =
      (const __attribute__((address_space(4))) int32_t*)(a.bt + (size_t)it.entry * a.bt_stride);
  const int h = lane >> 5;

  // this lane's pairs (column lane % 32 of each of the wavefront's PT pair tiles)
  int qpos[PT];
  bf16x8 qf[PT][KS];
#pragma unroll
  for (int pt = 0; pt < PT; ++pt) {
    const int p = (w * PT + pt) * 32 + (lane & 31);
    const bool ok = p < npairs;
    const int qi = ok ? p / G : 0, hj = ok ? p % G : 0;
    qpos[pt] = ok ? pos0 + it.q0 + qi : -1;     // -1: every key masked
    const uint16_t* qrow = a.q + (size_t)(a.row0[it.entry] + it.q0 + qi) * a.q_stride + (it.kvh * G + hj) * DH;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint4 v = ok ? *reinterpret_cast<const uint4*>(qrow + ks * 16 + h * 8) : make_uint4(0, 0, 0, 0);
      qf[pt][ks] = as_bf16x8(v);
    }
  }

  // DMA of key tile t into a stage: the two K pages, then the two V pages, as stored.  A
  // wavefront's blocks all lie in one page of the tile (pg), whose block-table entry the
  // caller passes in (read one step ahead, see below).
  static_assert(K_W == V_W && (KT / 1024) % K_W == 0, "a wavefront's blocks in one page");
  const int pg = (w * K_W) / (KT / 1024);
  auto entry_of = [&](int t) __attribute__((always_inline)) {
    const int tt = tbase + min(t, ntiles - 1);
    return bt[min(tt * 2 + pg, last_page)];
  };
  auto issue = [&](int entry, bf16_t* base) __attribute__((always_inline)) {
    const size_t tile = kv_tile(it.kvh, a.n_blocks, entry, DH);
#pragma unroll
    for (int u = 0; u < K_W; ++u) {
      const int blk = w * K_W + u;               // 1 KB block of the K tile
      dma16(a.k_pool + tile + (blk % (KT / 1024)) * 512 + lane * 8, base + blk * 512);
    }
#pragma unroll
    for (int u = 0; u < V_W; ++u) {
      const int blk = w * V_W + u;               // 1 KB block of the V tile
      // the two 16-byte halves of dims 8..15 (mod 16) of a block swap places in LDS, so that
      // the 16 lanes of one V^T read pass hit distinct banks
      dma16(a.v_pool + tile + (blk % (KT / 1024)) * 512 + (lane ^ ((lane >> 4) & 1)) * 8, base + KT + blk * 512);
    }
  };

  f32x16 o[PT][DT];
#pragma unroll
  for (int pt = 0; pt < PT; ++pt)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[pt][dt][e] = 0.f;
  // running maxima start finite, so that fully masked pairs keep zero weights, never NaN
  float m[PT], l[PT];
#pragma unroll
  for (int pt = 0; pt < PT; ++pt) {
    m[pt] = -1e30f;
    l[pt] = 0.f;
  }
  // operand offsets inside a stage: K for key lane%32 (page (lane%32)/16), dims chunk ks*2 + h;
  // V^T for dim dt*32 + lane%32, page s, positions 8h..8h+7
  const int k_off = ((lane & 31) >> 4) * (KT / 2) + (lane & 15) * 8 + h * 128;
  const int v_off = KT + (lane & 31) * 16 + (h ^ ((lane >> 3) & 1)) * 8;

  // One key tile.  Every LDS operand of the tile is requested first: the K fragments feed
  // the QK^T chain as they arrive, and the V^T fragments are in registers by the time the
  // softmax is done, so a wavefront alone on its SIMD does not wait on LDS between MFMAs.
  auto compute = [&](const bf16_t* base, int t) __attribute__((always_inline)) {
    bf16x8 kf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kf[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(base + k_off + ks * 256));
    uint4 vv[2][DT];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) vv[st][dt] = *reinterpret_cast<const uint4*>(base + v_off + (st * DH + dt * 32) * 16);
    f32x16 s[PT];
#pragma unroll
    for (int pt = 0; pt < PT; ++pt)
#pragma unroll
      for (int e = 0; e < 16; ++e) s[pt][e] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int pt = 0; pt < PT; ++pt) s[pt] = mfma32x32x16(kf[ks], qf[pt][ks], s[pt]);
    const int k0 = (tbase + t) * 32;
    const bool edge = (k0 + 32 > kend) || (k0 + 31 > pos0 + it.q0);   // wavefront-uniform: a mask is needed
    if (edge) {
#pragma unroll
      for (int pt = 0; pt < PT; ++pt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + (r >> 2) * 8 + h * 4 + (r & 3);
          if (key > qpos[pt] || key >= kend) s[pt][r] = kNegInf;
        }
    }
    // raw-score maxima (the scale is positive), then one wavefront-wide decision for
    // all pair tiles: the reference max only moves when a score exceeds it by more
    // than 2^8 (the exponentials then stay below 256, harmless in fp32 and bf16)
    float mx[PT];
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
      float v = s[pt][0];
#pragma unroll
      for (int r = 1; r < 16; ++r) v = fmaxf(v, s[pt][r]);
      mx[pt] = half_swap_max(v) * a.scale_log2;
    }
    bool grow = false;
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) grow = grow || mx[pt] > m[pt] + 8.f;
    if (__any(grow)) {
#pragma unroll
      for (int pt = 0; pt < PT; ++pt) {
        const float m_new = fmaxf(m[pt], mx[pt]);
        const float alpha = __builtin_amdgcn_exp2f(m[pt] - m_new);
        m[pt] = m_new;
        l[pt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int e = 0; e < 16; ++e) o[pt][dt][e] *= alpha;
      }
    }
    bf16x8 pf[PT][2];
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
      float ps = 0.f;
      float pv[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        pv[r] = __builtin_amdgcn_exp2f(fmaf(s[pt][r], a.scale_log2, -m[pt]));   // masked: exp2(-inf) = 0
        ps += pv[r];
      }
      l[pt] += ps;
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        bf16x8 v;
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (__bf16)pv[st * 8 + j];
        pf[pt][st] = v;
      }
    }
    // V^T . P^T; past the end of the context the V entries are zeroed (garbage may be NaN)
    if (k0 + 32 > kend) {
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const int tok0 = k0 + st * 16 + h * 4;    // keys of this lane's k slots: tok0 + 0..3, tok0 + 8..11
        const uint2 lo = keep_mask(kend - tok0), hi = keep_mask(kend - tok0 - 8);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          vv[st][dt].x &= lo.x;
          vv[st][dt].y &= lo.y;
          vv[st][dt].z &= hi.x;
          vv[st][dt].w &= hi.y;
        }
      }
    }
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) o[pt][dt] = mfma32x32x16(as_bf16x8(vv[st][dt]), pf[pt][st], o[pt][dt]);
  };

  // The block-table entry of the DMA issued at a step is loaded at the end of the step
  // before (a scalar load that the wait at the loop head drains together with the DMA
  // wait), so that no LDS read waits on it.
  static_for<NS - 1>([&](auto ic) { issue(entry_of(decltype(ic)::value), slot(ic)); });
  int next_entry = entry_of(NS - 1);
  int t0 = 0;
  for (; t0 + NS <= ntiles; t0 += NS) {
    static_for<NS>([&](auto ic) {
      constexpr int J = decltype(ic)::value;
      wait_vmcnt_lgkm0<(NS - 2) * PER_W>();
      __builtin_amdgcn_s_barrier();
      issue(next_entry, slot(std::integral_constant<int, J + NS - 1>{}));
      __builtin_amdgcn_sched_barrier(0);   // the DMAs go out before this tile's LDS reads
      compute(slot(ic), t0 + J);
      __builtin_amdgcn_sched_barrier(0);
      next_entry = entry_of(t0 + J + NS);
    });
  }
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  static_for<NS - 1>([&](auto ic) {
    constexpr int J = decltype(ic)::value;
    if (t0 + J < ntiles) compute(slot(ic), t0 + J);
  });

  // O^T lane holds pair lane % 32 and dims dt*32 + 8*(r/4) + 4h + r%4
  float lt[PT];
#pragma unroll
  for (int pt = 0; pt < PT; ++pt) lt[pt] = l[pt] + __shfl_xor(l[pt], 32, kWave);
  if (it.part >= 0) {
    // a part of a split item: unnormalized output, max and sum for the merge
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
      const int p = (w * PT + pt) * 32 + (lane & 31);
      if (p >= npairs) continue;
      float* po = a.part_o + ((size_t)it.part * kPrefillPairs + p) * DH;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4)
          *reinterpret_cast<float4*>(po + dt * 32 + g4 * 8 + h * 4) =
              make_float4(o[pt][dt][g4 * 4], o[pt][dt][g4 * 4 + 1], o[pt][dt][g4 * 4 + 2], o[pt][dt][g4 * 4 + 3]);
      if (h == 0)
        *reinterpret_cast<float2*>(a.part_ml + ((size_t)it.part * kPrefillPairs + p) * 2) = make_float2(m[pt], lt[pt]);
    }
    return;
  }
#pragma unroll
  for (int pt = 0; pt < PT; ++pt) {
    const int p = (w * PT + pt) * 32 + (lane & 31);
    if (p >= npairs) continue;
    const float inv = 1.f / lt[pt];
    const int qi = p / G, hj = p % G;
    const int orow = a.row0[it.entry] + it.q0 + qi, col0 = (it.kvh * G + hj) * DH;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d = dt * 32 + g4 * 8 + h * 4;   // 4 columns inside one 8-column group
        const size_t at = a.out_kt ? packed_elem(orow, col0 + d, a.out_kt) : (size_t)orow * a.out_stride + col0 + d;
        *reinterpret_cast<uint2*>(a.out + at) =
            make_uint2(pack_bf2(o[pt][dt][g4 * 4] * inv, o[pt][dt][g4 * 4 + 1] * inv),
                       pack_bf2(o[pt][dt][g4 * 4 + 2] * inv, o[pt][dt][g4 * 4 + 3] * inv));
      }
  }
}

// Log-sum-exp merge of the key-range parts of split prefill items: DH/8 lanes per
// (query, head) pair, each lane 8 dims, a job's 128 pairs over DH/16 workgroups.
template <int DH>
__global__ __launch_bounds__(256) void prefill_merge_kernel(PrefillAttnArgs a) {
  // TPP threads per (query, head) pair, 8 output dimensions each; the pairs of one job
  // span BPJ workgroups
  constexpr int TPP = DH / 8, PPB = 256 / TPP, BPJ = kPrefillPairs / PPB;
  const int job = blockIdx.x / BPJ;
  const PrefillMerge mg = a.merges[job];
  const int G = a.Hq / a.Hkv;
  const int p = (blockIdx.x % BPJ) * PPB + threadIdx.x / TPP;
  if (p >= mg.nq * G) return;
  const int d0 = (threadIdx.x % TPP) * 8;
  // one pass in groups of four partials whose loads are issued together; the running
  // maximum is finite from the first group on (partial 0 starts at key 0, which every
  // query sees), and a partial whose keys are all masked has weight zero
  float M = -__builtin_huge_valf(), L = 0.f;
  float acc[8];
#pragma unroll
  for (int d = 0; d < 8; ++d) acc[d] = 0.f;
  for (int j0 = 0; j0 < mg.n_part; j0 += 4) {
    float2 ml[4];
    float4 v[4][2];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const size_t slot = (size_t)(mg.part0 + min(j0 + u, mg.n_part - 1)) * kPrefillPairs + p;
      ml[u] = *reinterpret_cast<const float2*>(a.part_ml + slot * 2);
      const float4* po = reinterpret_cast<const float4*>(a.part_o + slot * DH + d0);
      v[u][0] = po[0];
      v[u][1] = po[1];
    }
    float mx = M;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (j0 + u < mg.n_part) mx = fmaxf(mx, ml[u].x);
    const float sc = __builtin_amdgcn_exp2f(M - mx);
    M = mx;
    L *= sc;
#pragma unroll
    for (int d = 0; d < 8; ++d) acc[d] *= sc;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float w = j0 + u < mg.n_part ? __builtin_amdgcn_exp2f(ml[u].x - M) : 0.f;
      L += w * ml[u].y;
      acc[0] += w * v[u][0].x;
      acc[1] += w * v[u][0].y;
      acc[2] += w * v[u][0].z;
      acc[3] += w * v[u][0].w;
      acc[4] += w * v[u][1].x;
      acc[5] += w * v[u][1].y;
      acc[6] += w * v[u][1].z;
      acc[7] += w * v[u][1].w;
    }
  }
  const float inv = 1.f / L;
  const int qi = p / G, hj = p % G;
  const int orow = a.row0[mg.entry] + mg.q0 + qi, col = (mg.kvh * G + hj) * DH + d0;   // one 8-column group
  uint16_t* out = a.out + (a.out_kt ? packed_elem(orow, col, a.out_kt) : (size_t)orow * a.out_stride + col);
  *reinterpret_cast<uint4*>(out) = make_uint4(pack_bf2(acc[0] * inv, acc[1] * inv), pack_bf2(acc[2] * inv, acc[3] * inv),
                                              pack_bf2(acc[4] * inv, acc[5] * inv), pack_bf2(acc[6] * inv, acc[7] * inv));
}

}  // namespace

// pair tiles of 32 (query, head) pairs per wavefront in the prefill kernel
constexpr int kPrefillPT = 1;

static_assert(4 * 32 * kPrefillPT == kPrefillPairs, "pairs of a prefill item");
int prefill_queries_per_item(int group) { return kPrefillPairs / group; }

// With events, they take the kernel's own start and end timestamps; without, a plain
// launch (the form a stream capture records).
template <typename K>
static hipError_t launch_stamped(K kernel, dim3 grid, dim3 block, hipStream_t st, hipEvent_t e0, hipEvent_t e1,
                                 const DecodeAttnArgs& a) {
  if (e0 || e1) hipExtLaunchKernelGGL(kernel, grid, block, 0, st, e0, e1, 0, a);
  else hipLaunchKernelGGL(kernel, grid, block, 0, st, a);
  return hipGetLastError();
}

hipError_t decode_attn_launch(const DecodeAttnArgs& a, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (a.dh != 128 && a.dh != 64) return hipErrorInvalidValue;
  const bool narrow = a.n_items > 0, wide = a.n_wide > 0;
  if (narrow) {
    hipEvent_t e1 = wide ? nullptr : ev_stop;
    hipError_t e = a.dh == 128 ? launch_stamped(decode_attn_kernel<128, 1>, dim3(a.n_items), dim3(64), st, ev_start, e1, a)
                               : launch_stamped(decode_attn_kernel<64, 1>, dim3(a.n_items), dim3(64), st, ev_start, e1, a);
    if (e != hipSuccess) return e;
  }
  if (wide) {
    hipEvent_t e0 = narrow ? nullptr : ev_start;
    return a.dh == 128 ? launch_stamped(decode_attn_kernel<128, 2>, dim3(a.n_wide), dim3(64), st, e0, ev_stop, a)
                       : launch_stamped(decode_attn_kernel<64, 2>, dim3(a.n_wide), dim3(64), st, e0, ev_stop, a);
  }
  return hipSuccess;
}

hipError_t decode_merge_launch(const DecodeAttnArgs& a, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (a.n_merges <= 0) return hipSuccess;
  const int jobs = a.n_merges * (a.Hq / a.Hkv);
  const dim3 grid((jobs + 3) / 4);
  if (a.dh == 128) return launch_stamped(decode_merge_kernel<128>, grid, dim3(256), st, ev_start, ev_stop, a);
  if (a.dh == 64) return launch_stamped(decode_merge_kernel<64>, grid, dim3(256), st, ev_start, ev_stop, a);
  return hipErrorInvalidValue;
}

hipError_t prefill_attn_launch(const PrefillAttnArgs& a, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (a.n_items <= 0) return hipSuccess;
  if (a.dh != 128 && a.dh != 64) return hipErrorInvalidValue;
  // with merges, the start event goes on the item kernel and the end event on the merge
  hipEvent_t e1 = a.n_merges > 0 ? nullptr : ev_stop;
  auto go = [&](auto kernel, dim3 grid, hipEvent_t s0, hipEvent_t s1) {
    if (s0 || s1) hipExtLaunchKernelGGL(kernel, grid, dim3(256), 0, st, s0, s1, 0, a);
    else hipLaunchKernelGGL(kernel, grid, dim3(256), 0, st, a);
    return hipGetLastError();
  };
  hipError_t e = a.dh == 128 ? go(prefill_flash_kernel<128, kPrefillPT>, dim3(a.n_items), ev_start, e1)
                             : go(prefill_flash_kernel<64, kPrefillPT>, dim3(a.n_items), ev_start, e1);
  if (e != hipSuccess || a.n_merges <= 0) return e;
  // workgroups per merge job: 128 pairs x dh / 8 threads over 256-thread workgroups
  const unsigned grid = (unsigned)a.n_merges * (kPrefillPairs * (a.dh / 8) / 256);
  return a.dh == 128 ? go(prefill_merge_kernel<128>, dim3(grid), nullptr, ev_stop)
                     : go(prefill_merge_kernel<64>, dim3(grid), nullptr, ev_stop);
}

}  // namespace hxf
