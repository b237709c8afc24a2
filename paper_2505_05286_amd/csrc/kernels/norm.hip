// RMSNorm over the fp32 residual stream (one workgroup per row, fp32 math,
// bf16 output), optionally fused with the token-embedding gather.
#include "common.hpp"
#include "kernels.hpp"

namespace hxf {

namespace {

// Sum over the NT threads of a workgroup (NT / 64 wavefronts), in wavefront order.
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float s = red[0];
#pragma unroll
  for (int k = 1; k < NT / 64; ++k) s += red[k];
  __syncthreads();
  return s;
}

// out: the output matrix; row `row` of it is written, row-major with stride d, or in the
// packed tile layout with out_kt tiles per row tile (each thread's 4 columns stay
// contiguous there: they lie in one 8-column group)
template <int NT = 256>
__device__ __forceinline__ void norm_store(const float4* x4, const uint16_t* g, uint16_t* out, int row, int out_kt,
                                           int d, float eps, float* red) {
  const int n4 = d >> 2;
  float ss = 0.f;
  for (int i = threadIdx.x; i < n4; i += NT) {
    const float4 v = x4[i];
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  const float r = rsqrtf(block_sum<NT>(ss, red) / (float)d + eps);
  const uint2* g2 = reinterpret_cast<const uint2*>(g);
  for (int i = threadIdx.x; i < n4; i += NT) {
    const float4 v = x4[i];
    const uint2 gg = g2[i];
    const float g0 = bf2f(gg.x & 0xFFFF), g1 = bf2f(gg.x >> 16), g2v = bf2f(gg.y & 0xFFFF), g3 = bf2f(gg.y >> 16);
    const size_t o = out_kt ? packed_elem(row, 4 * i, out_kt) : (size_t)row * d + 4 * i;
    *reinterpret_cast<uint2*>(out + o) =
        make_uint2(pack_bf2(v.x * r * g0, v.y * r * g1), pack_bf2(v.z * r * g2v, v.w * r * g3));
  }
}

// With S > 0 the row first takes the S split-K partial sums of a residual GEMM
// (part [S][part_rows][d], summed in split order, then added), exactly as the
// GEMM's own reduction would have, and the updated row is stored back.  The S
// partial loads of an element are independent and issued together.  NT threads per
// row: 1024 for the few rows of a decode batch (one round of loads per row instead of
// four), 256 otherwise.
template <int S, int NT>
__global__ __launch_bounds__(NT) void rmsnorm_kernel(float* x, const int32_t* rows, const float* part, int part_rows,
                                                     const uint16_t* g, uint16_t* out, int d, float eps, int out_kt) {
  __shared__ float red[NT / 64];
  const int r = blockIdx.x;
  const int src = rows ? rows[r] : r;
  float4* x4 = reinterpret_cast<float4*>(x + (size_t)src * d);
  if constexpr (S > 0) {
    const float4* p4 = reinterpret_cast<const float4*>(part + (size_t)src * d);
    const size_t zs = (size_t)part_rows * d / 4;
    for (int i = threadIdx.x; i < (d >> 2); i += NT) {
      float4 q[S];
#pragma unroll
      for (int z = 0; z < S; ++z) q[z] = p4[z * zs + i];
      float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int z = 0; z < S; ++z) {
        s.x += q[z].x; s.y += q[z].y; s.z += q[z].z; s.w += q[z].w;
      }
      float4 v = x4[i];
      v.x += s.x; v.y += s.y; v.z += s.z; v.w += s.w;
      x4[i] = v;
    }
  }
  norm_store<NT>(x4, g, out, r, out_kt, d, eps, red);
}

__global__ __launch_bounds__(256) void embed_rmsnorm_kernel(const int32_t* ids, const uint16_t* E, const uint16_t* g,
                                                            float* resid, uint16_t* out, int d, float eps, int out_kt) {
  __shared__ float red[4];
  const int t = blockIdx.x;
  const uint2* e2 = reinterpret_cast<const uint2*>(E + (size_t)ids[t] * d);
  float4* r4 = reinterpret_cast<float4*>(resid + (size_t)t * d);
  for (int i = threadIdx.x; i < (d >> 2); i += 256) {
    const uint2 e = e2[i];
    r4[i] = make_float4(bf2f(e.x & 0xFFFF), bf2f(e.x >> 16), bf2f(e.y & 0xFFFF), bf2f(e.y >> 16));
  }
  __syncthreads();
  norm_store<256>(r4, g, out, t, out_kt, d, eps, red);
}

}  // namespace

hipError_t rmsnorm_launch(const float* x, const int32_t* rows, const uint16_t* g, uint16_t* out, int n_rows, int d,
                          float eps, hipStream_t st) {
  return resid_rmsnorm_launch(const_cast<float*>(x), nullptr, 0, 0, rows, g, out, n_rows, d, eps, st);
}

hipError_t resid_rmsnorm_launch(float* x, const float* part, int S, int part_rows, const int32_t* rows,
                                const uint16_t* g, uint16_t* out, int n_rows, int d, float eps, hipStream_t st,
                                int out_kt) {
  if (n_rows <= 0) return hipSuccess;
  if (out_kt && (d % 32 || out_kt != d / 32)) return hipErrorInvalidValue;
#define HXF_NORM(SS)                                                                                        \
  case SS:                                                                                                  \
    if (n_rows <= 256)                                                                                      \
      hipLaunchKernelGGL((rmsnorm_kernel<SS, 1024>), dim3(n_rows), dim3(1024), 0, st, x, rows, part, part_rows, g, \
                         out, d, eps, out_kt);                                                              \
    else                                                                                                    \
      hipLaunchKernelGGL((rmsnorm_kernel<SS, 256>), dim3(n_rows), dim3(256), 0, st, x, rows, part, part_rows, g, \
                         out, d, eps, out_kt);                                                              \
    break;
  switch (S) {
    HXF_NORM(0) HXF_NORM(1) HXF_NORM(2) HXF_NORM(3) HXF_NORM(4) HXF_NORM(5) HXF_NORM(6) HXF_NORM(7) HXF_NORM(8)
    default: return hipErrorInvalidValue;
  }
#undef HXF_NORM
  return hipGetLastError();
}

hipError_t embed_rmsnorm_launch(const int32_t* ids, const uint16_t* E, const uint16_t* g, float* resid,
                                uint16_t* out, int T, int d, float eps, hipStream_t st, int out_kt) {
  if (T <= 0) return hipSuccess;
  if (out_kt && (d % 32 || out_kt != d / 32)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(embed_rmsnorm_kernel, dim3(T), dim3(256), 0, st, ids, E, g, resid, out, d, eps, out_kt);
  return hipGetLastError();
}

}  // namespace hxf
