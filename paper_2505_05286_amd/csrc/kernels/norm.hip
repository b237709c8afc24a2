// RMSNorm over the fp32 residual stream (one workgroup per row up to 256 rows, one
// wavefront per row beyond; fp32 math, bf16 output), optionally fused with the
// token-embedding gather.
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
// four), 256 for more rows whose width or split count the one-wavefront kernel below
// is not built for.
template <int S, int NT>
__global__ __launch_bounds__(NT) void rmsnorm_kernel(float* x, const int32_t* rows, const float* part, int part_rows,
                                                     const uint16_t* g, uint16_t* out, int d, float eps, int out_kt) {
  __shared__ float red[NT / 64];
  const int r = blockIdx.x;
  const int src = rows ? rows[r] : r;
  float4* x4 = reinterpret_cast<float4*>(x + (size_t)src * d);
  const int n4 = d >> 2;
  if (n4 <= 2 * NT) {
    // at most two float4 per thread (d <= 8 NT): kept in registers between the two passes,
    // the same arithmetic in the same order as the loop below
    float4 v[2];
    float ss = 0.f;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int i = threadIdx.x + u * NT;
      if (i >= n4) continue;
      if constexpr (S > 0) {
        const float4* p4 = reinterpret_cast<const float4*>(part + (size_t)src * d);
        const size_t zs = (size_t)part_rows * d / 4;
        float4 q[S];
#pragma unroll
        for (int z = 0; z < S; ++z) q[z] = p4[z * zs + i];
        float4 sm = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int z = 0; z < S; ++z) {
          sm.x += q[z].x; sm.y += q[z].y; sm.z += q[z].z; sm.w += q[z].w;
        }
        v[u] = x4[i];
        v[u].x += sm.x; v[u].y += sm.y; v[u].z += sm.z; v[u].w += sm.w;
        x4[i] = v[u];
      } else {
        v[u] = x4[i];
      }
      ss += v[u].x * v[u].x + v[u].y * v[u].y + v[u].z * v[u].z + v[u].w * v[u].w;
    }
    const float rs = rsqrtf(block_sum<NT>(ss, red) / (float)d + eps);
    const uint2* g2 = reinterpret_cast<const uint2*>(g);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int i = threadIdx.x + u * NT;
      if (i >= n4) continue;
      const uint2 gg = g2[i];
      const float g0 = bf2f(gg.x & 0xFFFF), g1 = bf2f(gg.x >> 16), g2v = bf2f(gg.y & 0xFFFF), g3 = bf2f(gg.y >> 16);
      const size_t o = out_kt ? packed_elem(r, 4 * i, out_kt) : (size_t)r * d + 4 * i;
      *reinterpret_cast<uint2*>(out + o) =
          make_uint2(pack_bf2(v[u].x * rs * g0, v[u].y * rs * g1), pack_bf2(v[u].z * rs * g2v, v[u].w * rs * g3));
    }
    return;
  }
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

// Many rows (prefill-sized iterations): one wavefront per row, four rows per workgroup.
// The row's V float4 per lane are loaded together and kept in registers, so the second
// pass (scale and store) reads no memory and every wavefront has its whole row in flight.
// The residual update sums the S partials of an element in split order, as above; the
// sum of squares is the lane's own V elements, then a wavefront sum.
template <int S, int V>
__global__ __launch_bounds__(256) void rmsnorm_rows_kernel(float* x, const int32_t* rows, const float* part,
                                                          int part_rows, const uint16_t* g, uint16_t* out, int n_rows,
                                                          int d, float eps, int out_kt) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= n_rows) return;
  const int lane = threadIdx.x & 63;
  const int src = rows ? rows[r] : r;
  float4* x4 = reinterpret_cast<float4*>(x + (size_t)src * d);
  float4 v[V];
#pragma unroll
  for (int j = 0; j < V; ++j) v[j] = x4[j * 64 + lane];
  if constexpr (S > 0) {
    const float4* p4 = reinterpret_cast<const float4*>(part + (size_t)src * d);
    const size_t zs = (size_t)part_rows * d / 4;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      float4 q[S];
#pragma unroll
      for (int z = 0; z < S; ++z) q[z] = p4[z * zs + j * 64 + lane];
      float4 sm = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int z = 0; z < S; ++z) {
        sm.x += q[z].x; sm.y += q[z].y; sm.z += q[z].z; sm.w += q[z].w;
      }
      v[j].x += sm.x; v[j].y += sm.y; v[j].z += sm.z; v[j].w += sm.w;
      x4[j * 64 + lane] = v[j];
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < V; ++j) ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
  const float rs = rsqrtf(wave_sum(ss) / (float)d + eps);
  const uint2* g2 = reinterpret_cast<const uint2*>(g);
#pragma unroll
  for (int j = 0; j < V; ++j) {
    const int i = j * 64 + lane;
    const uint2 gg = g2[i];
    const float g0 = bf2f(gg.x & 0xFFFF), g1 = bf2f(gg.x >> 16), g2v = bf2f(gg.y & 0xFFFF), g3 = bf2f(gg.y >> 16);
    const size_t o = out_kt ? packed_elem(r, 4 * i, out_kt) : (size_t)r * d + 4 * i;
    *reinterpret_cast<uint2*>(out + o) =
        make_uint2(pack_bf2(v[j].x * rs * g0, v[j].y * rs * g1), pack_bf2(v[j].z * rs * g2v, v[j].w * rs * g3));
  }
}

template <int S>
hipError_t rmsnorm_rows_launch(float* x, const float* part, int part_rows, const int32_t* rows, const uint16_t* g,
                               uint16_t* out, int n_rows, int d, float eps, hipStream_t st, int out_kt) {
  const dim3 grid((n_rows + 3) / 4);
#define HXF_ROWS(VV)                                                                                          \
  case VV:                                                                                                    \
    hipLaunchKernelGGL((rmsnorm_rows_kernel<S, VV>), grid, dim3(256), 0, st, x, rows, part, part_rows, g, out, \
                       n_rows, d, eps, out_kt);                                                               \
    return hipGetLastError();
  switch (d / 256) {
    HXF_ROWS(4) HXF_ROWS(8) HXF_ROWS(16) HXF_ROWS(20) HXF_ROWS(24) HXF_ROWS(32)
  }
#undef HXF_ROWS
  return hipErrorNotSupported;
}

// d / 256 float4 per lane for which the one-wavefront-per-row kernel is built
inline bool rows_kernel_fits(int d, int S) {
  if (d % 256 || S > 4) return false;
  const int v = d / 256;
  return v == 4 || v == 8 || v == 16 || v == 20 || v == 24 || v == 32;
}

// The embedding gather + first RMSNorm for many rows: one wavefront per row, as
// rmsnorm_rows_kernel (the gathered row stays in registers for the norm).
template <int V>
__global__ __launch_bounds__(256) void embed_rmsnorm_rows_kernel(const int32_t* ids, const uint16_t* E,
                                                                const uint16_t* g, float* resid, uint16_t* out,
                                                                int n_rows, int d, float eps, int out_kt) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= n_rows) return;
  const int lane = threadIdx.x & 63;
  const uint2* e2 = reinterpret_cast<const uint2*>(E + (size_t)ids[r] * d);
  float4* r4 = reinterpret_cast<float4*>(resid + (size_t)r * d);
  uint2 e[V];
#pragma unroll
  for (int j = 0; j < V; ++j) e[j] = e2[j * 64 + lane];
  float4 v[V];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < V; ++j) {
    v[j] = make_float4(bf2f(e[j].x & 0xFFFF), bf2f(e[j].x >> 16), bf2f(e[j].y & 0xFFFF), bf2f(e[j].y >> 16));
    r4[j * 64 + lane] = v[j];
    ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
  }
  const float rs = rsqrtf(wave_sum(ss) / (float)d + eps);
  const uint2* g2 = reinterpret_cast<const uint2*>(g);
#pragma unroll
  for (int j = 0; j < V; ++j) {
    const int i = j * 64 + lane;
    const uint2 gg = g2[i];
    const float g0 = bf2f(gg.x & 0xFFFF), g1 = bf2f(gg.x >> 16), g2v = bf2f(gg.y & 0xFFFF), g3 = bf2f(gg.y >> 16);
    const size_t o = out_kt ? packed_elem(r, 4 * i, out_kt) : (size_t)r * d + 4 * i;
    *reinterpret_cast<uint2*>(out + o) =
        make_uint2(pack_bf2(v[j].x * rs * g0, v[j].y * rs * g1), pack_bf2(v[j].z * rs * g2v, v[j].w * rs * g3));
  }
}

__global__ __launch_bounds__(256) void embed_rmsnorm_kernel(const int32_t* ids, const uint16_t* E, const uint16_t* g,
                                                            float* resid, uint16_t* out, int d, float eps, int out_kt) {
  __shared__ float red[4];
  const int t = blockIdx.x;
  const uint2* e2 = reinterpret_cast<const uint2*>(E + (size_t)ids[t] * d);
  float4* r4 = reinterpret_cast<float4*>(resid + (size_t)t * d);
  // four gathers in flight per thread
  int i = threadIdx.x;
  for (; i + 3 * 256 < (d >> 2); i += 4 * 256) {
    uint2 e[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) e[u] = e2[i + u * 256];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      r4[i + u * 256] = make_float4(bf2f(e[u].x & 0xFFFF), bf2f(e[u].x >> 16), bf2f(e[u].y & 0xFFFF), bf2f(e[u].y >> 16));
  }
  for (; i < (d >> 2); i += 256) {
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
  if (n_rows > 256 && rows_kernel_fits(d, S)) {
    switch (S) {
      case 0: return rmsnorm_rows_launch<0>(x, part, part_rows, rows, g, out, n_rows, d, eps, st, out_kt);
      case 1: return rmsnorm_rows_launch<1>(x, part, part_rows, rows, g, out, n_rows, d, eps, st, out_kt);
      case 2: return rmsnorm_rows_launch<2>(x, part, part_rows, rows, g, out, n_rows, d, eps, st, out_kt);
      case 3: return rmsnorm_rows_launch<3>(x, part, part_rows, rows, g, out, n_rows, d, eps, st, out_kt);
      case 4: return rmsnorm_rows_launch<4>(x, part, part_rows, rows, g, out, n_rows, d, eps, st, out_kt);
    }
  }
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
  if (T > 256 && rows_kernel_fits(d, 0)) {
    const dim3 grid((T + 3) / 4);
#define HXF_EROWS(VV)                                                                                           \
  case VV:                                                                                                      \
    hipLaunchKernelGGL(embed_rmsnorm_rows_kernel<VV>, grid, dim3(256), 0, st, ids, E, g, resid, out, T, d, eps, \
                       out_kt);                                                                                 \
    return hipGetLastError();
    switch (d / 256) {
      HXF_EROWS(4) HXF_EROWS(8) HXF_EROWS(16) HXF_EROWS(20) HXF_EROWS(24) HXF_EROWS(32)
    }
#undef HXF_EROWS
  }
  hipLaunchKernelGGL(embed_rmsnorm_kernel, dim3(T), dim3(256), 0, st, ids, E, g, resid, out, d, eps, out_kt);
  return hipGetLastError();
}

}  // namespace hxf
