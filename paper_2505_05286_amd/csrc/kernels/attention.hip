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
// K pages are read as [token][dh] rows, V pages as [dh][token] rows (the pool
// stores V transposed within a page), both as 16-byte / 8-byte vector loads.
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
__device__ __forceinline__ void load_pair(PairRegs<DH>& R, const uint16_t* k_pool, const uint16_t* v_pool,
                                          const int32_t* bt, int Hkv, int kvh, int page, int t_end, int lane) {
  const int tok = lane & 15, rq = lane >> 4;
  {
    const size_t tile = ((size_t)bt[page] * Hkv + kvh) * kPage * DH;
    const uint16_t* kp = k_pool + tile + tok * DH + rq * 8;
    const uint16_t* vp = v_pool + tile + (lane & 15) * kPage + rq * 4;
#pragma unroll
    for (int s = 0; s < DH / 32; ++s) R.ka[s] = *reinterpret_cast<const uint4*>(kp + s * 32);
#pragma unroll
    for (int n = 0; n < DH / 16; ++n) R.va[n] = *reinterpret_cast<const uint2*>(vp + n * 16 * kPage);
  }
  if ((page + 1) * kPage < t_end) {
    const size_t tile = ((size_t)bt[page + 1] * Hkv + kvh) * kPage * DH;
    const uint16_t* kp = k_pool + tile + tok * DH + rq * 8;
    const uint16_t* vp = v_pool + tile + (lane & 15) * kPage + rq * 4;
#pragma unroll
    for (int s = 0; s < DH / 32; ++s) R.kb[s] = *reinterpret_cast<const uint4*>(kp + s * 32);
#pragma unroll
    for (int n = 0; n < DH / 16; ++n) R.vb[n] = *reinterpret_cast<const uint2*>(vp + n * 16 * kPage);
  } else {
#pragma unroll
    for (int s = 0; s < DH / 32; ++s) R.kb[s] = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int n = 0; n < DH / 16; ++n) R.vb[n] = make_uint2(0, 0);
  }
}

// Zero the bf16 V entries of tokens at or beyond t_end (their memory may hold
// anything; a zero probability times a NaN would still be NaN).
__device__ __forceinline__ uint2 mask_v(uint2 v, int first_tok, int t_end) {
  const int n_ok = t_end - first_tok;   // valid tokens among the 4 held
  if (n_ok >= 4) return v;
  if (n_ok <= 0) return make_uint2(0, 0);
  if (n_ok == 1) return make_uint2(v.x & 0xFFFFu, 0);
  if (n_ok == 2) return make_uint2(v.x, 0);
  return make_uint2(v.x, v.y & 0xFFFFu);
}

template <int DH>
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
  float x[8];
  float mx = kNegInf;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bool oka = (ta + e) < t_end && (ta + e) <= lim;
    const bool okb = (tb + e) < t_end && (tb + e) <= lim;
    x[e] = oka ? sa[e] * scale_log2 : kNegInf;
    x[4 + e] = okb ? sb[e] * scale_log2 : kNegInf;
    mx = fmaxf(mx, fmaxf(x[e], x[4 + e]));
  }
  mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
  mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
  const float m_new = fmaxf(S.m, mx);
  const float alpha = exp2f(S.m - m_new);
  float psum = 0.f;
  float p[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    p[e] = exp2f(x[e] - m_new);
    psum += p[e];
  }
  S.l = S.l * alpha + psum;
  S.m = m_new;
  const uint4 pw = make_uint4(pack_bf2(p[0], p[1]), pack_bf2(p[2], p[3]), pack_bf2(p[4], p[5]), pack_bf2(p[6], p[7]));
  const bf16x8 pf = as_bf16x8(pw);
#pragma unroll
  for (int n = 0; n < DH / 16; ++n) {
    S.acc[n] *= alpha;
    const uint2 a = mask_v(R.va[n], ta, t_end);
    const uint2 b = mask_v(R.vb[n], tb, t_end);
    S.acc[n] = mfma16x16x32(as_bf16x8(make_uint4(a.x, a.y, b.x, b.y)), pf, S.acc[n]);
  }
}

// Attend the lane's column to tokens [t_begin, t_end) (t_begin page aligned);
// tokens beyond `lim` are masked for this column.
template <int DH>
__device__ __forceinline__ void attn_range(AttnState<DH>& S, const bf16x8* qf, const uint16_t* k_pool,
                                           const uint16_t* v_pool, const int32_t* bt, int Hkv, int kvh, int t_begin,
                                           int t_end, int lim, float scale_log2, int lane) {
#pragma unroll
  for (int n = 0; n < DH / 16; ++n) S.acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  S.m = kNegInf;
  S.l = 0.f;
  const int p0 = t_begin / kPage, p_end = (t_end + kPage - 1) / kPage;
  PairRegs<DH> cur, nxt;
  load_pair<DH>(cur, k_pool, v_pool, bt, Hkv, kvh, p0, t_end, lane);
  for (int p = p0; p < p_end; p += 2) {
    if (p + 2 < p_end) load_pair<DH>(nxt, k_pool, v_pool, bt, Hkv, kvh, p + 2, t_end, lane);
    compute_pair<DH>(S, cur, qf, p, t_end, lim, scale_log2, lane);
    cur = nxt;
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

template <int DH>
__global__ __launch_bounds__(256) void decode_attn_kernel(DecodeAttnArgs a) {
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= a.n_items) return;
  const DecodeItem it = a.items[w];
  const int G = a.Hq / a.Hkv;
  const int col = lane & 15;
  const bool ok = col < G;
  const int head = it.kvh * G + (ok ? col : 0);
  bf16x8 qf[DH / 32];
  load_q<DH>(qf, a.q + (size_t)a.q_row[it.entry] * a.q_stride + head * DH, ok, lane);
  AttnState<DH> S;
  attn_range<DH>(S, qf, a.k_pool, a.v_pool, a.bt + (size_t)it.entry * a.bt_stride, a.Hkv, it.kvh, it.t0, it.t1,
                 0x7FFFFFFF, a.scale_log2, lane);
  if (!ok) return;
  const int rq = lane >> 4;
  float* o = a.part_o + ((size_t)it.part * G + col) * DH;
#pragma unroll
  for (int n = 0; n < DH / 16; ++n)
    *reinterpret_cast<float4*>(o + n * 16 + rq * 4) = make_float4(S.acc[n][0], S.acc[n][1], S.acc[n][2], S.acc[n][3]);
  if (rq == 0) *reinterpret_cast<float2*>(a.part_ml + ((size_t)it.part * G + col) * 2) = make_float2(S.m, S.l);
}

// Log-sum-exp merge of the split-K partials; one wavefront per (entry, q-head).
template <int DH>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeAttnArgs a) {
  const int G = a.Hq / a.Hkv;
  const int job = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (job >= a.n_merges * G) return;
  const int lane = threadIdx.x & 63;
  const MergeItem mi = a.merges[job / G];
  const int g = job % G;
  float M = kNegInf;
  for (int p = 0; p < mi.n_part; ++p) M = fmaxf(M, a.part_ml[((size_t)(mi.part0 + p) * G + g) * 2]);
  float L = 0.f;
  float acc[DH / 64];
#pragma unroll
  for (int k = 0; k < DH / 64; ++k) acc[k] = 0.f;
  for (int p = 0; p < mi.n_part; ++p) {
    const size_t b = (size_t)(mi.part0 + p) * G + g;
    const float2 ml = *reinterpret_cast<const float2*>(a.part_ml + b * 2);
    const float wgt = exp2f(ml.x - M);
    L += wgt * ml.y;
#pragma unroll
    for (int k = 0; k < DH / 64; ++k) acc[k] += wgt * a.part_o[b * DH + lane + 64 * k];
  }
  const float inv = 1.f / L;
  uint16_t* out = a.out + (size_t)a.q_row[mi.entry] * a.out_stride + (mi.kvh * G + g) * DH;
#pragma unroll
  for (int k = 0; k < DH / 64; ++k) out[lane + 64 * k] = f2bf(acc[k] * inv);
}

template <int DH>
__global__ __launch_bounds__(256) void prefill_attn_kernel(PrefillAttnArgs a) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const PrefillItem it = a.items[blockIdx.x];
  const int G = a.Hq / a.Hkv;
  const int qpw = 16 / G;                       // queries per wavefront
  const int col = lane & 15;
  const int qi = col / G, j = col % G;
  const int wq0 = it.q0 + wid * qpw;            // first query of this wave
  const int wq_end = min(it.q0 + it.nq, wq0 + qpw);
  if (wq0 >= wq_end) return;
  const int qloc = wq0 + qi;
  const bool ok = (col < qpw * G) && (qloc < wq_end);
  const int pos0 = a.pos0[it.entry];
  const int row = a.row0[it.entry] + (ok ? qloc : wq0);
  const int head = it.kvh * G + j;
  bf16x8 qf[DH / 32];
  load_q<DH>(qf, a.q + (size_t)row * a.q_stride + head * DH, ok, lane);
  const int lim = pos0 + (ok ? qloc : wq0);
  const int t_end = pos0 + wq_end;              // last query position + 1
  AttnState<DH> S;
  attn_range<DH>(S, qf, a.k_pool, a.v_pool, a.bt + (size_t)it.entry * a.bt_stride, a.Hkv, it.kvh, 0, t_end, lim,
                 a.scale_log2, lane);
  if (!ok) return;
  const float inv = 1.f / S.l;
  const int rq = lane >> 4;
  uint16_t* out = a.out + (size_t)row * a.out_stride + head * DH;
#pragma unroll
  for (int n = 0; n < DH / 16; ++n) {
    const uint2 v = make_uint2(pack_bf2(S.acc[n][0] * inv, S.acc[n][1] * inv),
                               pack_bf2(S.acc[n][2] * inv, S.acc[n][3] * inv));
    *reinterpret_cast<uint2*>(out + n * 16 + rq * 4) = v;
  }
}

}  // namespace

int prefill_queries_per_item(int group) { return 4 * (16 / group); }

hipError_t decode_attn_launch(const DecodeAttnArgs& a, hipStream_t st) {
  if (a.n_items <= 0) return hipSuccess;
  if (a.dh == 128) hipLaunchKernelGGL(decode_attn_kernel<128>, dim3((a.n_items + 3) / 4), dim3(256), 0, st, a);
  else if (a.dh == 64) hipLaunchKernelGGL(decode_attn_kernel<64>, dim3((a.n_items + 3) / 4), dim3(256), 0, st, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t decode_merge_launch(const DecodeAttnArgs& a, hipStream_t st) {
  if (a.n_merges <= 0) return hipSuccess;
  const int jobs = a.n_merges * (a.Hq / a.Hkv);
  if (a.dh == 128) hipLaunchKernelGGL(decode_merge_kernel<128>, dim3((jobs + 3) / 4), dim3(256), 0, st, a);
  else if (a.dh == 64) hipLaunchKernelGGL(decode_merge_kernel<64>, dim3((jobs + 3) / 4), dim3(256), 0, st, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t prefill_attn_launch(const PrefillAttnArgs& a, hipStream_t st) {
  if (a.n_items <= 0) return hipSuccess;
  if (a.dh == 128) hipLaunchKernelGGL(prefill_attn_kernel<128>, dim3(a.n_items), dim3(256), 0, st, a);
  else if (a.dh == 64) hipLaunchKernelGGL(prefill_attn_kernel<64>, dim3(a.n_items), dim3(256), 0, st, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace hxf
