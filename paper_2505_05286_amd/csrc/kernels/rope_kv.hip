// Rotate-half RoPE on q and k (fp32 math from a float64-built cos/sin table)
// fused with the paged KV write.  One workgroup per token.
#include "common.hpp"
#include "kernels.hpp"

namespace hxf {

namespace {

// Offset of (dimension d, token tok) inside one K (page, kv-head) tile.
__device__ __forceinline__ int k_offset(int d, int tok) { return ((d >> 3) * kPage + tok) * 8 + (d & 7); }

__global__ __launch_bounds__(256) void rope_kv_kernel(uint16_t* qkv, const int32_t* pos, const int32_t* slot,
                                                      const float2* cs, uint16_t* k_pool, uint16_t* v_pool,
                                                      int64_t n_blocks, int Hq, int Hkv, int dh) {
  const int t = blockIdx.x;
  const int half = dh >> 1;
  const int width = (Hq + 2 * Hkv) * dh;
  uint16_t* row = qkv + (size_t)t * width;
  const float2* c = cs + (size_t)pos[t] * half;
  const int s = slot[t];
  const int blk = s / kPage, off = s % kPage;
  const int n_rot = (Hq + Hkv) * half;
  for (int j = threadIdx.x; j < n_rot; j += 256) {
    const int h = j / half, i = j % half;
    uint16_t* x = row + h * dh;
    const float x1 = bf2f(x[i]), x2 = bf2f(x[i + half]);
    const float2 cc = c[i];
    const uint16_t o1 = f2bf(x1 * cc.x - x2 * cc.y);
    const uint16_t o2 = f2bf(x2 * cc.x + x1 * cc.y);
    if (h < Hq) {
      x[i] = o1;
      x[i + half] = o2;
    } else {
      const int kh = h - Hq;
      uint16_t* kp = k_pool + kv_tile(kh, n_blocks, blk, dh);
      kp[k_offset(i, off)] = o1;
      kp[k_offset(i + half, off)] = o2;
    }
  }
  const uint16_t* v = row + (Hq + Hkv) * dh;
  for (int j = threadIdx.x; j < Hkv * dh; j += 256) {
    const int kh = j / dh, d = j % dh;
    v_pool[kv_tile(kh, n_blocks, blk, dh) + d * kPage + off] = v[j];
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
    v_pool[kv_tile(kh, n_blocks, blk, dh) + d * kPage + off] = v[(size_t)t * Hkv * dh + j];
  }
}

}  // namespace

hipError_t rope_kv_launch(uint16_t* qkv, const int32_t* pos, const int32_t* slot, const float2* cs,
                          uint16_t* k_pool, uint16_t* v_pool, int64_t n_blocks, int T, int Hq, int Hkv, int dh,
                          hipStream_t st) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_kv_kernel, dim3(T), dim3(256), 0, st, qkv, pos, slot, cs, k_pool, v_pool, n_blocks, Hq, Hkv,
                     dh);
  return hipGetLastError();
}

hipError_t kv_scatter_launch(const uint16_t* k, const uint16_t* v, const int32_t* slot, uint16_t* k_pool,
                             uint16_t* v_pool, int64_t n_blocks, int T, int Hkv, int dh, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(kv_scatter_kernel, dim3(T), dim3(256), 0, st, k, v, slot, k_pool, v_pool, n_blocks, Hkv, dh);
  return hipGetLastError();
}

}  // namespace hxf
