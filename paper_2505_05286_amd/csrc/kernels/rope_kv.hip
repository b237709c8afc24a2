// Rotate-half RoPE on q and k (fp32 math from a float64-built cos/sin table)
// fused with the paged KV write, optionally also with the split-K reduction of
// the QKV projection.
#include "common.hpp"
#include "kernels.hpp"

namespace hxf {

namespace {

// Offset of (dimension d, token tok) inside one K (page, kv-head) tile.
__device__ __forceinline__ int k_offset(int d, int tok) { return ((d >> 3) * kPage + tok) * 8 + (d & 7); }

// Four consecutive values (col .. col+3) of token t's projection row: the bf16 row
// itself (S == 0), or the bf16 rounding of its S split-K partial sums (part
// [S][T][width]) added in split order, exactly as the GEMM's own reduction would
// have stored them.  The loads are 8 bytes (bf16) or 16 bytes (each partial), all
// issued together.
template <int S>
__device__ __forceinline__ void proj_values4(const uint16_t* row, const float* prow, size_t zs, int col, float v[4],
                                            uint16_t raw[4]) {
  if constexpr (S == 0) {
    const uint2 u = *reinterpret_cast<const uint2*>(row + col);
    raw[0] = u.x & 0xFFFF; raw[1] = u.x >> 16; raw[2] = u.y & 0xFFFF; raw[3] = u.y >> 16;
  } else {
    float4 p[S];
#pragma unroll
    for (int z = 0; z < S; ++z) p[z] = *reinterpret_cast<const float4*>(prow + z * zs + col);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int z = 0; z < S; ++z) {
      acc.x += p[z].x; acc.y += p[z].y; acc.z += p[z].z; acc.w += p[z].w;
    }
    raw[0] = f2bf(acc.x); raw[1] = f2bf(acc.y); raw[2] = f2bf(acc.z); raw[3] = f2bf(acc.w);
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = bf2f(raw[e]);
}

// One workgroup of 64 threads per (token, four heads of the q|k|v row); 16 threads per
// head at dh = 128 (8 at dh = 64, the rest idle), a thread owning dimensions i..i+3 and
// their rotation partners i+dh/2..i+dh/2+3.  Rotated q is written back to the qkv row.
template <int S>
__global__ __launch_bounds__(64) void rope_kv_kernel(uint16_t* qkv, const float* part, int T, const int32_t* pos,
                                                     const int32_t* slot, const float2* cs, uint16_t* k_pool,
                                                     uint16_t* v_pool, int64_t n_blocks, int Hq, int Hkv, int dh,
                                                     int write_v) {
  const int t = blockIdx.x;
  const int h = blockIdx.y * 4 + (threadIdx.x >> 4);
  const int half = dh >> 1;
  const int i = (threadIdx.x & 15) * 4;
  if (h >= Hq + 2 * Hkv || i >= half || (!write_v && h >= Hq + Hkv)) return;
  const int width = (Hq + 2 * Hkv) * dh;
  uint16_t* row = qkv + (size_t)t * width;
  const float* prow = part + (size_t)t * width;
  const size_t zs = (size_t)T * width;
  float a[4], b[4];
  uint16_t ra[4], rb[4];
  proj_values4<S>(row, prow, zs, h * dh + i, a, ra);
  proj_values4<S>(row, prow, zs, h * dh + i + half, b, rb);
  const int s = slot[t];
  const int blk = s / kPage, off = s % kPage;
  if (h >= Hq + Hkv) {                                     // v: no rotation (write_v == 1 only)
    uint16_t* vp = v_pool + kv_tile(h - Hq - Hkv, n_blocks, blk, dh);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      vp[(i + e) * kPage + v_pos(off)] = ra[e];
      vp[(i + e + half) * kPage + v_pos(off)] = rb[e];
    }
    return;
  }
  const float4* c4 = reinterpret_cast<const float4*>(cs + (size_t)pos[t] * half + i);
  const float4 c01 = c4[0], c23 = c4[1];                   // (cos, sin) of dims i..i+3
  const float cc[4] = {c01.x, c01.z, c23.x, c23.z}, sn[4] = {c01.y, c01.w, c23.y, c23.w};
  uint16_t o1[4], o2[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    o1[e] = f2bf(a[e] * cc[e] - b[e] * sn[e]);
    o2[e] = f2bf(b[e] * cc[e] + a[e] * sn[e]);
  }
  const uint2 w1 = make_uint2(o1[0] | ((uint32_t)o1[1] << 16), o1[2] | ((uint32_t)o1[3] << 16));
  const uint2 w2 = make_uint2(o2[0] | ((uint32_t)o2[1] << 16), o2[2] | ((uint32_t)o2[3] << 16));
  if (h < Hq) {
    *reinterpret_cast<uint2*>(row + h * dh + i) = w1;
    *reinterpret_cast<uint2*>(row + h * dh + i + half) = w2;
  } else {
    // K page layout [dh/8][16 tokens][8]: dims i..i+3 are contiguous (i % 4 == 0)
    uint16_t* kp = k_pool + kv_tile(h - Hq, n_blocks, blk, dh);
    *reinterpret_cast<uint2*>(kp + k_offset(i, off)) = w1;
    *reinterpret_cast<uint2*>(kp + k_offset(i + half, off)) = w2;
  }
}

// The V rows of prefill-sized batches: one workgroup per (16 consecutive tokens, kv-head).
// A page row of V holds one dimension of 16 tokens (32 bytes), so a token's V row lands
// as dh scattered 2-byte stores; here the 16 x dh block is staged in LDS and, when the 16
// tokens fill one page in order (a prefill chunk's whole pages), written as dh page rows
// of 16 contiguous bytes per lane.  Otherwise each value goes to its own slot.
template <int DH>
__global__ __launch_bounds__(256) void v_page_kernel(const uint16_t* qkv, int T, const int32_t* slot,
                                                     uint16_t* v_pool, int64_t n_blocks, int Hq, int Hkv) {
  __shared__ uint16_t tile[16][DH + 8];   // [token][dimension]; the pad spreads the column reads over banks
  const int t0 = blockIdx.x * 16, kvh = blockIdx.y;
  const int tok = threadIdx.x / 16, ch = threadIdx.x % 16;   // load: 8 dimensions of one token
  const int width = (Hq + 2 * Hkv) * DH;
  const uint16_t* vrow = qkv + (size_t)(Hq + Hkv + kvh) * DH;
  const bool have = ch < DH / 8 && t0 + tok < T;
  if (have) {
    const uint4 v = *reinterpret_cast<const uint4*>(vrow + (size_t)(t0 + tok) * width + ch * 8);
    *reinterpret_cast<uint4*>(&tile[tok][ch * 8]) = v;
  }
  const int s0 = t0 < T ? slot[t0] : 0;
  const bool in_order = threadIdx.x >= 16 || (t0 + (int)threadIdx.x < T && slot[t0 + threadIdx.x] == s0 + (int)threadIdx.x);
  const bool whole_page = __syncthreads_and(in_order) && s0 % kPage == 0;   // also orders the LDS writes
  if (whole_page) {
    // thread (d, half): stored positions 8 half .. 8 half + 7 of page row d, i.e. the tokens
    // v_pos(position) (v_pos swaps bits 2 and 3, so it is its own inverse)
    const int d = threadIdx.x / 2, half = threadIdx.x % 2;
    if (d < DH) {
      uint16_t e[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) e[j] = tile[v_pos(half * 8 + j)][d];
      uint16_t* vp = v_pool + kv_tile(kvh, n_blocks, s0 / kPage, DH) + d * kPage + half * 8;
      *reinterpret_cast<uint4*>(vp) = make_uint4(e[0] | ((uint32_t)e[1] << 16), e[2] | ((uint32_t)e[3] << 16),
                                                 e[4] | ((uint32_t)e[5] << 16), e[6] | ((uint32_t)e[7] << 16));
    }
    return;
  }
  if (!have) return;
  const int sl = slot[t0 + tok];
  uint16_t* vp = v_pool + kv_tile(kvh, n_blocks, sl / kPage, DH) + v_pos(sl % kPage);
#pragma unroll
  for (int j = 0; j < 8; ++j) vp[(ch * 8 + j) * kPage] = tile[tok][ch * 8 + j];
}

__global__ __launch_bounds__(256) void kv_scatter_kernel(const uint16_t* k, const uint16_t* v, const int32_t* slot,
                                                         uint16_t* k_pool, uint16_t* v_pool, int64_t n_blocks, int Hkv,
                                                         int dh) {
  const int t = blockIdx.x;
  const int s = slot[t];
  const int blk = s / kPage, off = s % kPage;
  for (int j = threadIdx.x; j < Hkv * dh; j += 256) {
    const int kh = j / dh, d = j % dh;
    k_pool[kv_tile(kh, n_blocks, blk, dh) + k_offset(d, off)] = k[(size_t)t * Hkv * dh + j];
    v_pool[kv_tile(kh, n_blocks, blk, dh) + d * kPage + v_pos(off)] = v[(size_t)t * Hkv * dh + j];
  }
}

}  // namespace

hipError_t rope_kv_launch(uint16_t* qkv, const int32_t* pos, const int32_t* slot, const float2* cs,
                          uint16_t* k_pool, uint16_t* v_pool, int64_t n_blocks, int T, int Hq, int Hkv, int dh,
                          hipStream_t st) {
  return rope_kv_partials_launch(qkv, nullptr, 0, pos, slot, cs, k_pool, v_pool, n_blocks, T, Hq, Hkv, dh, st);
}

hipError_t rope_kv_partials_launch(uint16_t* qkv, const float* part, int S, const int32_t* pos, const int32_t* slot,
                                   const float2* cs, uint16_t* k_pool, uint16_t* v_pool, int64_t n_blocks, int T,
                                   int Hq, int Hkv, int dh, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  if (dh > 128 || dh % 8) return hipErrorInvalidValue;
  // prefill-sized batches without split partials write V through v_page_kernel
  const bool v_pages = S == 0 && T >= 64 && (dh == 128 || dh == 64);
  const dim3 grid(T, ((v_pages ? Hq + Hkv : Hq + 2 * Hkv) + 3) / 4);
#define HXF_ROPE(SS)                                                                                            \
  case SS:                                                                                                      \
    hipLaunchKernelGGL(rope_kv_kernel<SS>, grid, dim3(64), 0, st, qkv, part, T, pos, slot, cs, k_pool, v_pool, \
                       n_blocks, Hq, Hkv, dh, v_pages ? 0 : 1);                                                \
    break;
  switch (S) {
    HXF_ROPE(0) HXF_ROPE(1) HXF_ROPE(2) HXF_ROPE(3) HXF_ROPE(4) HXF_ROPE(5) HXF_ROPE(6) HXF_ROPE(7) HXF_ROPE(8)
    default: return hipErrorInvalidValue;
  }
#undef HXF_ROPE
  if (hipError_t e = hipGetLastError(); e != hipSuccess || !v_pages) return e;
  const dim3 vgrid((T + 15) / 16, Hkv);
  if (dh == 128)
    hipLaunchKernelGGL(v_page_kernel<128>, vgrid, dim3(256), 0, st, qkv, T, slot, v_pool, n_blocks, Hq, Hkv);
  else
    hipLaunchKernelGGL(v_page_kernel<64>, vgrid, dim3(256), 0, st, qkv, T, slot, v_pool, n_blocks, Hq, Hkv);
  return hipGetLastError();
}

hipError_t kv_scatter_launch(const uint16_t* k, const uint16_t* v, const int32_t* slot, uint16_t* k_pool,
                             uint16_t* v_pool, int64_t n_blocks, int T, int Hkv, int dh, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(kv_scatter_kernel, dim3(T), dim3(256), 0, st, k, v, slot, k_pool, v_pool, n_blocks, Hkv, dh);
  return hipGetLastError();
}

}  // namespace hxf
