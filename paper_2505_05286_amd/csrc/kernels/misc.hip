// Greedy sampling (row argmax, lowest index on ties) and a streaming copy used
// as the HBM bandwidth probe.
#include "common.hpp"
#include "kernels.hpp"

namespace hxf {

namespace {

__device__ __forceinline__ void better(float& bv, int& bi, float v, int i) {
  // v beats (bv, bi) if larger, or equal with a lower index; NaN never wins
  if (v > bv || (v == bv && i < bi)) {
    bv = v;
    bi = i;
  }
}

__global__ __launch_bounds__(1024) void argmax_kernel(const float* logits, int32_t* out, int V) {
  __shared__ float sv[16];
  __shared__ int si[16];
  const float* row = logits + (size_t)blockIdx.x * V;
  float bv = -__builtin_huge_valf();
  int bi = 0x7FFFFFFF;
  const int n4 = V >> 2;
  const float4* r4 = reinterpret_cast<const float4*>(row);
  // four loads in flight per thread, then the comparisons (their order does not matter:
  // better() breaks ties by index)
  int i = threadIdx.x;
  for (; i + 3 * 1024 < n4; i += 4 * 1024) {
    float4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = r4[i + u * 1024];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = 4 * (i + u * 1024);
      better(bv, bi, v[u].x, j);
      better(bv, bi, v[u].y, j + 1);
      better(bv, bi, v[u].z, j + 2);
      better(bv, bi, v[u].w, j + 3);
    }
  }
  for (; i < n4; i += 1024) {
    const float4 v = r4[i];
    better(bv, bi, v.x, 4 * i);
    better(bv, bi, v.y, 4 * i + 1);
    better(bv, bi, v.z, 4 * i + 2);
    better(bv, bi, v.w, 4 * i + 3);
  }
  for (int i = 4 * n4 + threadIdx.x; i < V; i += 1024) better(bv, bi, row[i], i);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o, kWave);
    const int oi = __shfl_xor(bi, o, kWave);
    better(bv, bi, ov, oi);
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sv[w] = bv;
    si[w] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < 16; ++k) better(bv, bi, sv[k], si[k]);
    out[blockIdx.x] = (bi == 0x7FFFFFFF) ? 0 : bi;
  }
}

__global__ __launch_bounds__(256) void copy_kernel(const uint4* src, uint4* dst, size_t n) {
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * 256;
  for (; i < n; i += stride) dst[i] = src[i];
}

// Streaming read: thread t XORs the 16-byte words it reads (grid-stride, four loads in
// flight per step) into sink[t], so that no load is dead.
__global__ __launch_bounds__(256) void read_kernel(const uint4* src, size_t n, uint32_t* sink) {
  uint32_t acc = 0;
  const size_t stride = (size_t)gridDim.x * 1024;
  for (size_t i = (size_t)blockIdx.x * 1024 + threadIdx.x; i < n; i += stride) {
    uint4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = i + u * 256 < n ? src[i + u * 256] : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < 4; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  sink[(size_t)blockIdx.x * 256 + threadIdx.x] = acc;
}

}  // namespace

hipError_t argmax_launch(const float* logits, int32_t* out, int R, int V, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  hipLaunchKernelGGL(argmax_kernel, dim3(R), dim3(1024), 0, st, logits, out, V);
  return hipGetLastError();
}

hipError_t copy_launch(const void* src, void* dst, size_t bytes, hipStream_t st) {
  const size_t n = bytes / 16;
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 256 * 64) blocks = 256 * 64;
  hipLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(256), 0, st, reinterpret_cast<const uint4*>(src),
                     reinterpret_cast<uint4*>(dst), n);
  return hipGetLastError();
}

hipError_t read_launch(const void* src, size_t bytes, uint32_t* sink, hipStream_t st) {
  const size_t n = bytes / 16;
  size_t blocks = (n + 1023) / 1024;
  if (blocks > kReadProbeBlocks) blocks = kReadProbeBlocks;
  if (blocks == 0) blocks = 1;   // no words: every sink word is written as 0
  hipLaunchKernelGGL(read_kernel, dim3((unsigned)blocks), dim3(256), 0, st, reinterpret_cast<const uint4*>(src), n,
                     sink);
  return hipGetLastError();
}

}  // namespace hxf
