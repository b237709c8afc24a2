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
                                                     uint16_t* v_pool, int64_t n_blocks, int Hq, int Hkv, int dh) {
  const int t = blockIdx.x;
  const int h = blockIdx.y * 4 + (threadIdx.x >> 4);
  const int half = dh >> 1;
  const int i = (threadIdx.x & 15) * 4;
  if (h >= Hq + 2 * Hkv || i >= half) return;
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
  if (h >= Hq + Hkv) {                                     // v: no rotation
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
  const dim3 grid(T, (Hq + 2 * Hkv + 3) / 4);
#define HXF_ROPE(SS)                                                                                            \
  case SS:                                                                                                      \
    hipLaunchKernelGGL(rope_kv_kernel<SS>, grid, dim3(64), 0, st, qkv, part, T, pos, slot, cs, k_pool, v_pool, \
                       n_blocks, Hq, Hkv, dh);                                                                 \
    break;
  switch (S) {
    HXF_ROPE(0) HXF_ROPE(1) HXF_ROPE(2) HXF_ROPE(3) HXF_ROPE(4) HXF_ROPE(5) HXF_ROPE(6) HXF_ROPE(7) HXF_ROPE(8)
    default: return hipErrorInvalidValue;
  }
#undef HXF_ROPE
  return hipGetLastError();
}

hipError_t kv_scatter_launch(const uint16_t* k, const uint16_t* v, const int32_t* slot, uint16_t* k_pool,
                             uint16_t* v_pool, int64_t n_blocks, int T, int Hkv, int dh, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(kv_scatter_kernel, dim3(T), dim3(256), 0, st, k, v, slot, k_pool, v_pool, n_blocks, Hkv, dh);
  return hipGetLastError();
}

}  // namespace hxf
