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

template <int DH, bool CAUSAL>
__device__ __forceinline__ void compute_pair(AttnState<DH>& S, const PairRegs<DH>& R, const bf16x8* qf, int page,
                                             int t_end, int lim, float scale_log2, int lane) {
  const int rq = lane >> 4;
  f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < DH / 32; ++s) {
    sa = mfma16x16x32(as_bf16x8(R.ka[s]), qf[s], sa);
    sb = mfma16x16x32(as_bf16x8(R.kb[s]), qf[s], sb);
  }
  const int ta = page * kPage + rq * 4;   // first token of this lane's rows in page a
  const int tb = ta + kPage;
  const bool full = (page + 2) * kPage <= t_end;   // wavefront-uniform
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
  const float m_new = fmaxf(S.m, mx);
  const float alpha = exp2f(S.m - m_new);
  float p[8];
  float psum = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    p[e] = exp2f(x[e] - m_new);
    psum += p[e];
  }
  S.l = S.l * alpha + psum;
  S.m = m_new;
  const bf16x8 pf = as_bf16x8(make_uint4(pack_bf2(p[0], p[1]), pack_bf2(p[2], p[3]), pack_bf2(p[4], p[5]),
                                         pack_bf2(p[6], p[7])));
  uint2 ma = make_uint2(~0u, ~0u), mb = make_uint2(~0u, ~0u);
  if (!full) {
    ma = keep_mask(t_end - ta);
    mb = keep_mask(t_end - tb);
  }
#pragma unroll
  for (int n = 0; n < DH / 16; ++n) {
    S.acc[n] *= alpha;
    const uint4 v = make_uint4(R.va[n].x & ma.x, R.va[n].y & ma.y, R.vb[n].x & mb.x, R.vb[n].y & mb.y);
    S.acc[n] = mfma16x16x32(as_bf16x8(v), pf, S.acc[n]);
  }
}

// Attend the lane's column to tokens [t_begin, t_end) (t_begin page aligned);
// tokens beyond `lim` are masked for this column.
template <int DH, bool CAUSAL>
__device__ __forceinline__ void attn_range(AttnState<DH>& S, const bf16x8* qf, const uint16_t* k_pool,
                                           const uint16_t* v_pool, const int32_t* bt, int64_t nb, int kvh, int t_begin,
                                           int t_end, int lim, float scale_log2, int lane) {
#pragma unroll
  for (int n = 0; n < DH / 16; ++n) S.acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  S.m = kNegInf;
  S.l = 0.f;
  const int p0 = t_begin / kPage, p_end = (t_end + kPage - 1) / kPage;
  // two register buffers used in turn: the loads of the next page pair are in
  // flight while the current one is multiplied
  PairRegs<DH> ra, rb;
  load_pair<DH>(ra, k_pool, v_pool, bt, nb, kvh, p0, t_end, lane);
  for (int p = p0; p < p_end; p += 4) {
    if (p + 2 < p_end) load_pair<DH>(rb, k_pool, v_pool, bt, nb, kvh, p + 2, t_end, lane);
    compute_pair<DH, CAUSAL>(S, ra, qf, p, t_end, lim, scale_log2, lane);
    if (p + 2 >= p_end) break;
    if (p + 4 < p_end) load_pair<DH>(ra, k_pool, v_pool, bt, nb, kvh, p + 4, t_end, lane);
    compute_pair<DH, CAUSAL>(S, rb, qf, p + 2, t_end, lim, scale_log2, lane);
  }
  S.l += __shfl_xor(S.l, 16, kWave);
  S.l += __shfl_xor(S.l, 32, kWave);
}

template <int DH>
__device__ __forceinline__ void load_q(bf16x8* qf, const uint16_t* qrow, bool ok, int lane) {
  const int rq = lane >> 4;
#pragma unroll
  for (int s = 0; s < DH / 32; ++s)
    qf[s] = ok ? as_bf16x8(*reinterpret_cast<const uint4*>(qrow + s * 32 + rq * 8)) : as_bf16x8(make_uint4(0, 0, 0, 0));
}

static_assert(kDecodeRows == 4, "the row selects below assume four rows");

template <int DH>
__global__ __launch_bounds__(64) void decode_attn_kernel(DecodeAttnArgs a) {
  const int lane = threadIdx.x;
  const int w = blockIdx.x;
  if (w >= (a.n_items_dev ? *a.n_items_dev : a.n_items)) return;
  const DecodeItem it = a.items[w];
  const int G = a.Hq / a.Hkv;
  // column (lane % 16) = (row, head of the group); rows past n_rows are idle columns
  const int col = lane & 15;
  const int row = col / G, g = col - row * G;
  const bool ok = row < it.n_rows && row < kDecodeRows;
  const int r = ok ? row : 0;
  const int entry = r == 0 ? it.entry[0] : r == 1 ? it.entry[1] : r == 2 ? it.entry[2] : it.entry[3];
  const int part = r == 0 ? it.part[0] : r == 1 ? it.part[1] : r == 2 ? it.part[2] : it.part[3];
  const int head = it.kvh * G + (ok ? g : 0);
  bf16x8 qf[DH / 32];
  load_q<DH>(qf, a.q + (size_t)a.q_row[entry] * a.q_stride + head * DH, ok, lane);
  AttnState<DH> S;
  attn_range<DH, false>(S, qf, a.k_pool, a.v_pool, a.bt + (size_t)it.entry[0] * a.bt_stride, a.n_blocks, it.kvh,
                        it.t0, it.t1, 0x7FFFFFFF, a.scale_log2, lane);
  if (!ok) return;
  const int rq = lane >> 4;
  float* o = a.part_o + ((size_t)part * G + g) * DH;
#pragma unroll
  for (int n = 0; n < DH / 16; ++n)
    *reinterpret_cast<float4*>(o + n * 16 + rq * 4) = make_float4(S.acc[n][0], S.acc[n][1], S.acc[n][2], S.acc[n][3]);
  if (rq == 0) *reinterpret_cast<float2*>(a.part_ml + ((size_t)part * G + g) * 2) = make_float2(S.m, S.l);
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
  uint16_t* out = a.out + (size_t)orow * a.out_stride + (mi.kvh * G + g) * DH + lane * PER;
  if constexpr (PER == 2) *reinterpret_cast<uint32_t*>(out) = pack_bf2(acc[0] * inv, acc[PER - 1] * inv);
  else out[0] = f2bf(acc[0] * inv);
}

// Chunked-prefill causal attention, one workgroup per (chunk, kv-head, block of
// 256/G queries): the 256 (query, head) pairs of the block are the columns of
//   S^T[32 keys x 32 pairs] = K[32 x dh] . Q^T[dh x 32]       (v_mfma_f32_32x32x16_bf16)
//   O^T[32 dims x 32 pairs] += V^T[32 x 32 keys] . P^T[32 x 32]
// (64 pairs per wavefront, two 32-pair tiles).  Tiles of 32 keys (two pages)
// of K and V are moved into LDS by the DMA path, five tiles in flight, and
// shared by the four wavefronts.  A lane of the S^T accumulator holds keys
// 8m + 4h + i (h = lane / 32) of its pair; taken in the order m = 2s, 2s + 1
// these are the 8 keys of the P^T operand for the 16-key step s (page s of the
// tile); the V pool stores each page row with its tokens in that order (see
// v_pos), so the V^T operand of a lane is one contiguous 16-byte LDS read.  Softmax is
// online in log2 units, one cross-lane exchange (xor 32) per tile for the max.
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
  const int ntiles = (kend + 31) / 32;
  const int last_page = (kend - 1) / kPage;
  // the block table does not change during the kernel: read it through the constant
  // address space, so that its (wavefront-uniform) entries come by scalar loads, which
  // are counted apart from the vector loads and do not wait for the DMAs in flight
  const __attribute__((address_space(4))) int32_t* bt =
      (const __attribute__((address_space(4))) int32_t*)(a.bt + (size_t)it.entry * a.bt_stride);
  const int h = lane >> 5;

  // this lane's two pairs (columns lane % 32 of the wavefront's two pair tiles)
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

  // DMA of key tile t into a stage: the two K pages, then the two V pages, as stored
  auto issue = [&](int t, bf16_t* base) __attribute__((always_inline)) {
    const int tt = min(t, ntiles - 1);
#pragma unroll
    for (int u = 0; u < K_W; ++u) {
      const int blk = w * K_W + u;               // 1 KB block of the K tile
      const int pg = blk / (KT / 1024);          // page of the tile (each page is KT / 2 elements)
      const int page = min(tt * 2 + pg, last_page);
      const size_t tile = kv_tile(it.kvh, a.n_blocks, bt[page], DH);
      dma16(a.k_pool + tile + (blk % (KT / 1024)) * 512 + lane * 8, base + blk * 512);
    }
#pragma unroll
    for (int u = 0; u < V_W; ++u) {
      const int blk = w * V_W + u;               // 1 KB block of the V tile
      const int pg = blk / (KT / 1024);
      const int page = min(tt * 2 + pg, last_page);
      const size_t tile = kv_tile(it.kvh, a.n_blocks, bt[page], DH);
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

  auto compute = [&](const bf16_t* base, int t) __attribute__((always_inline)) {
    f32x16 s[PT];
#pragma unroll
    for (int pt = 0; pt < PT; ++pt)
#pragma unroll
      for (int e = 0; e < 16; ++e) s[pt][e] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 kf = as_bf16x8(*reinterpret_cast<const uint4*>(base + k_off + ks * 256));
#pragma unroll
      for (int pt = 0; pt < PT; ++pt) s[pt] = mfma32x32x16(kf, qf[pt][ks], s[pt]);
    }
    const int k0 = t * 32;
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
    // both pair tiles: the reference max only moves when a score exceeds it by more
    // than 2^8 (the exponentials then stay below 256, harmless in fp32 and bf16)
    float mx[PT];
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
      float v = s[pt][0];
#pragma unroll
      for (int r = 1; r < 16; ++r) v = fmaxf(v, s[pt][r]);
      v = fmaxf(v, __shfl_xor(v, 32, kWave));
      mx[pt] = v * a.scale_log2;
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
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int tok0 = k0 + st * 16 + h * 4;      // keys of this lane's k slots: tok0 + 0..3, tok0 + 8..11
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        uint4 vv = *reinterpret_cast<const uint4*>(base + v_off + (st * DH + dt * 32) * 16);
        if (k0 + 32 > kend) {
          const uint2 lo = keep_mask(kend - tok0), hi = keep_mask(kend - tok0 - 8);
          vv.x &= lo.x; vv.y &= lo.y; vv.z &= hi.x; vv.w &= hi.y;
        }
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) o[pt][dt] = mfma32x32x16(as_bf16x8(vv), pf[pt][st], o[pt][dt]);
      }
    }
  };

  static_for<NS - 1>([&](auto ic) { issue(decltype(ic)::value, slot(ic)); });
  int t0 = 0;
  for (; t0 + NS <= ntiles; t0 += NS) {
    static_for<NS>([&](auto ic) {
      constexpr int J = decltype(ic)::value;
      wait_vmcnt<(NS - 2) * PER_W>();
      __builtin_amdgcn_s_barrier();
      issue(t0 + J + NS - 1, slot(std::integral_constant<int, J + NS - 1>{}));
      compute(slot(ic), t0 + J);
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
#pragma unroll
  for (int pt = 0; pt < PT; ++pt) {
    const int p = (w * PT + pt) * 32 + (lane & 31);
    if (p >= npairs) continue;
    const float inv = 1.f / lt[pt];
    const int qi = p / G, hj = p % G;
    uint16_t* out = a.out + (size_t)(a.row0[it.entry] + it.q0 + qi) * a.out_stride + (it.kvh * G + hj) * DH;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d = dt * 32 + g4 * 8 + h * 4;
        *reinterpret_cast<uint2*>(out + d) =
            make_uint2(pack_bf2(o[pt][dt][g4 * 4] * inv, o[pt][dt][g4 * 4 + 1] * inv),
                       pack_bf2(o[pt][dt][g4 * 4 + 2] * inv, o[pt][dt][g4 * 4 + 3] * inv));
      }
  }
}

}  // namespace

// pair tiles of 32 (query, head) pairs per wavefront in the prefill kernel
constexpr int kPrefillPT = 1;

int prefill_queries_per_item(int group) { return 4 * 32 * kPrefillPT / group; }

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
  if (a.n_items <= 0) return hipSuccess;
  if (a.dh == 128) return launch_stamped(decode_attn_kernel<128>, dim3(a.n_items), dim3(64), st, ev_start, ev_stop, a);
  if (a.dh == 64) return launch_stamped(decode_attn_kernel<64>, dim3(a.n_items), dim3(64), st, ev_start, ev_stop, a);
  return hipErrorInvalidValue;
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
  auto go = [&](auto kernel) {
    if (ev_start || ev_stop) hipExtLaunchKernelGGL(kernel, dim3(a.n_items), dim3(256), 0, st, ev_start, ev_stop, 0, a);
    else hipLaunchKernelGGL(kernel, dim3(a.n_items), dim3(256), 0, st, a);
    return hipGetLastError();
  };
  if (a.dh == 128) return go(prefill_flash_kernel<128, kPrefillPT>);
  if (a.dh == 64) return go(prefill_flash_kernel<64, kPrefillPT>);
  return hipErrorInvalidValue;
}

}  // namespace hxf
