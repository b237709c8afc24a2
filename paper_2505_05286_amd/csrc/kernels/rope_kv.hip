// Rotate-half RoPE on q and k (fp32 math from a float64-built cos/sin table)
// fused with the paged KV write, optionally also with the split-K reduction of
// the QKV projection.
#include "common.hpp"
#include "kernels.hpp"

namespace hxf {

namespace {

// Offset of (dimension d, token tok) inside one K (page, kv-head) tile.
__device__ __forceinline__ int k_offset(int d, int tok) { return ((d >> 3) * kPage + tok) * 8 + (d & 7); }

// Value `col` of token t's projection row: the bf16 row itself (S == 0), or the
// bf16 rounding of its S split-K partial sums (part [S][T][width]) added in split
// order, exactly as the GEMM's own reduction would have stored it.  The S loads
// are independent and issued together.
template <int S>
__device__ __forceinline__ uint16_t proj_value(const uint16_t* row, const float* prow, size_t zs, int col) {
  if constexpr (S == 0) {
    return row[col];
  } else {
    float p[S];
#pragma unroll
    for (int z = 0; z < S; ++z) p[z] = prow[z * zs + col];
    float acc = 0.f;
#pragma unroll
    for (int z = 0; z < S; ++z) acc += p[z];
    return f2bf(acc);
  }
}

// One workgroup of 64 threads per (token, head of the q|k|v row); a thread owns the
// dimension pair (i, i + dh/2).  Rotated q is written back to the qkv row.
template <int S>
__global__ __launch_bounds__(64) void rope_kv_kernel(uint16_t* qkv, const float* part, int T, const int32_t* pos,
                                                     const int32_t* slot, const float2* cs, uint16_t* k_pool,
                                                     uint16_t* v_pool, int64_t n_blocks, int Hq, int Hkv, int dh) {
  const int t = blockIdx.x, h = blockIdx.y, i = threadIdx.x;
  const int half = dh >> 1;
  if (i >= half) return;
  const int width = (Hq + 2 * Hkv) * dh;
  uint16_t* row = qkv + (size_t)t * width;
  const float* prow = part + (size_t)t * width;
  const size_t zs = (size_t)T * width;
  const uint16_t a = proj_value<S>(row, prow, zs, h * dh + i), b = proj_value<S>(row, prow, zs, h * dh + i + half);
  const int s = slot[t];
  const int blk = s / kPage, off = s % kPage;
  if (h >= Hq + Hkv) {                                     // v: no rotation
    uint16_t* vp = v_pool + kv_tile(h - Hq - Hkv, n_blocks, blk, dh);
    vp[i * kPage + v_pos(off)] = a;
    vp[(i + half) * kPage + v_pos(off)] = b;
    return;
  }
  const float x1 = bf2f(a), x2 = bf2f(b);
  const float2 cc = cs[(size_t)pos[t] * half + i];
  const uint16_t o1 = f2bf(x1 * cc.x - x2 * cc.y);
  const uint16_t o2 = f2bf(x2 * cc.x + x1 * cc.y);
  if (h < Hq) {
    row[h * dh + i] = o1;
    row[h * dh + i + half] = o2;
  } else {
    uint16_t* kp = k_pool + kv_tile(h - Hq, n_blocks, blk, dh);
    kp[k_offset(i, off)] = o1;
    kp[k_offset(i + half, off)] = o2;
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
  if (dh > 128 || dh % 2) return hipErrorInvalidValue;
  const dim3 grid(T, Hq + 2 * Hkv);
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
