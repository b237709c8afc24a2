// bf16 "NT" GEMM on CDNA4 matrix cores: C[M,N] = A[M,K] * B[N,K]^T with an
// fp32 accumulator and fused epilogues (bf16 store, fp32 residual add,
// SwiGLU gate*up, fp32 store) or fp32 split-K partials.
//
// Tiling: 256 threads = 4 wavefronts in a 2x2 arrangement; each wave owns a
// (BM/2)x(BN/2) sub-tile made of 16x16 v_mfma_f32_16x16x32_bf16 tiles.  K is
// staged through LDS 64 at a time; the next K tile is fetched into registers
// while the current one is multiplied.  Workgroups are renumbered so that
// consecutive output tiles (which share a weight slice) land on the same XCD
// and its L2.
#include "common.hpp"
#include "kernels.hpp"

namespace hxf {

namespace {

constexpr int BK = 64;
constexpr int LDS_ROW = BK + 8;   // bf16 elements per LDS row (16-byte pad)

// Logical column c of a SwiGLU GEMM: groups of 32 = 16 gate rows then 16 up rows.
__device__ __forceinline__ const bf16_t* b_row(const GemmArgs& a, int c, bool swiglu) {
  if (!swiglu) return a.B + (size_t)c * a.K;
  const int g = c >> 5, w = c & 31;
  return ((w < 16) ? a.B : a.B2) + (size_t)(g * 16 + (w & 15)) * a.K;
}

__device__ __forceinline__ int xcd_remap(int i, int nb) {
  const int xcd = i & 7, local = i >> 3;
  const int per = nb >> 3, rem = nb & 7;
  return (xcd < rem) ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

template <int BM, int BN, int EPI, bool SPLIT>
__global__ __launch_bounds__(256) void gemm_nt_kernel(GemmArgs a) {
  constexpr int TM = BM / 32, TN = BN / 32;         // MFMA tiles per wave
  constexpr int A_CH = BM * (BK / 8) / 256;         // 16-byte chunks per thread
  constexpr int B_CH = BN * (BK / 8) / 256;
  constexpr bool SW = (EPI == EPI_SWIGLU);
  __shared__ __attribute__((aligned(16))) bf16_t As[BM * LDS_ROW];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[BN * LDS_ROW];

  const int tiles_m = (a.M + BM - 1) / BM;
  const int tiles_n = (a.N + BN - 1) / BN;
  const int L = xcd_remap(blockIdx.x, tiles_m * tiles_n);
  const int tn = L / tiles_m, tm = L % tiles_m;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kb = SPLIT ? blockIdx.z * a.k_chunk : 0;
  const int ke = SPLIT ? min(a.K, kb + a.k_chunk) : a.K;

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid >> 1, wn = wid & 1;

  // global load bookkeeping: chunk j of this thread = row (tid + j*256) / 8, col16 (tid % 8)
  const int c16 = tid & 7;
  const bf16_t* a_ptr[A_CH];
  const bf16_t* b_ptr[B_CH];
  bool a_ok[A_CH], b_ok[B_CH];
#pragma unroll
  for (int j = 0; j < A_CH; ++j) {
    const int r = (tid + j * 256) >> 3;
    a_ok[j] = (m0 + r) < a.M;
    a_ptr[j] = a.A + (size_t)(a_ok[j] ? m0 + r : 0) * a.lda + c16 * 8;
  }
#pragma unroll
  for (int j = 0; j < B_CH; ++j) {
    const int r = (tid + j * 256) >> 3;
    b_ok[j] = (n0 + r) < a.N;
    b_ptr[j] = b_row(a, b_ok[j] ? n0 + r : 0, SW) + c16 * 8;
  }
  uint4 ra[A_CH], rb[B_CH];
  auto fetch = [&](int k0) {
    const bool kin = (k0 + c16 * 8) < ke;
#pragma unroll
    for (int j = 0; j < A_CH; ++j)
      ra[j] = (a_ok[j] && kin) ? *reinterpret_cast<const uint4*>(a_ptr[j] + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int j = 0; j < B_CH; ++j)
      rb[j] = (b_ok[j] && kin) ? *reinterpret_cast<const uint4*>(b_ptr[j] + k0) : make_uint4(0, 0, 0, 0);
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  fetch(kb);
  for (int k0 = kb; k0 < ke; k0 += BK) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < A_CH; ++j) {
      const int r = (tid + j * 256) >> 3;
      *reinterpret_cast<uint4*>(&As[r * LDS_ROW + c16 * 8]) = ra[j];
    }
#pragma unroll
    for (int j = 0; j < B_CH; ++j) {
      const int r = (tid + j * 256) >> 3;
      *reinterpret_cast<uint4*>(&Bs[r * LDS_ROW + c16 * 8]) = rb[j];
    }
    __syncthreads();
    if (k0 + BK < ke) fetch(k0 + BK);
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      const int kc = ks * 32 + (lane >> 4) * 8;
      bf16x8 fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * (BM / 2) + i * 16 + (lane & 15);
        fa[i] = as_bf16x8(*reinterpret_cast<const uint4*>(&As[r * LDS_ROW + kc]));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * (BN / 2) + j * 16 + (lane & 15);
        fb[j] = as_bf16x8(*reinterpret_cast<const uint4*>(&Bs[r * LDS_ROW + kc]));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma16x16x32(fa[i], fb[j], acc[i][j]);
    }
  }

  // epilogue: lane holds rows (lane/16)*4 + e, column lane%16 of each 16x16 tile
  const int col_in = lane & 15, row_q = (lane >> 4) * 4;
  if (SPLIT) {
    float* P = a.partial + (size_t)blockIdx.z * a.M * a.N;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = n0 + wn * (BN / 2) + j * 16 + col_in;
        if (col >= a.N) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = m0 + wm * (BM / 2) + i * 16 + row_q + e;
          if (row < a.M) P[(size_t)row * a.N + col] = acc[i][j][e];
        }
      }
    return;
  }
  if (EPI == EPI_SWIGLU) {
    bf16_t* C = reinterpret_cast<bf16_t*>(a.C);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; j += 2) {
        const int lc = n0 + wn * (BN / 2) + j * 16;          // first (gate) logical column of the pair
        if (lc >= a.N) continue;
        const int col = (lc >> 5) * 16 + col_in;              // output column
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = m0 + wm * (BM / 2) + i * 16 + row_q + e;
          if (row < a.M) {
            const float g = acc[i][j][e], u = acc[i][j + 1][e];
            C[(size_t)row * a.ldc + col] = f2bf(g / (1.f + __expf(-g)) * u);
          }
        }
      }
    return;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + wn * (BN / 2) + j * 16 + col_in;
      if (col >= a.N) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = m0 + wm * (BM / 2) + i * 16 + row_q + e;
        if (row >= a.M) continue;
        const size_t o = (size_t)row * a.ldc + col;
        if (EPI == EPI_BF16) reinterpret_cast<bf16_t*>(a.C)[o] = f2bf(acc[i][j][e]);
        else if (EPI == EPI_RESID) reinterpret_cast<float*>(a.C)[o] += acc[i][j][e];
        else reinterpret_cast<float*>(a.C)[o] = acc[i][j][e];
      }
    }
}

// Sum split-K partials in a fixed order and apply the epilogue.
template <int EPI>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs a, int S) {
  const int n_out = (EPI == EPI_SWIGLU) ? a.N / 2 : a.N;
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)a.M * n_out) return;
  const int row = idx / n_out, col = idx % n_out;
  const size_t MN = (size_t)a.M * a.N;
  if (EPI == EPI_SWIGLU) {
    const int lg = (col >> 4) * 32 + (col & 15);
    float g = 0.f, u = 0.f;
    for (int z = 0; z < S; ++z) {
      g += a.partial[z * MN + (size_t)row * a.N + lg];
      u += a.partial[z * MN + (size_t)row * a.N + lg + 16];
    }
    reinterpret_cast<bf16_t*>(a.C)[(size_t)row * a.ldc + col] = f2bf(g / (1.f + __expf(-g)) * u);
    return;
  }
  float s = 0.f;
  for (int z = 0; z < S; ++z) s += a.partial[z * MN + (size_t)row * a.N + col];
  const size_t o = (size_t)row * a.ldc + col;
  if (EPI == EPI_BF16) reinterpret_cast<bf16_t*>(a.C)[o] = f2bf(s);
  else if (EPI == EPI_RESID) reinterpret_cast<float*>(a.C)[o] += s;
  else reinterpret_cast<float*>(a.C)[o] = s;
}

template <int BM, int BN, int EPI>
hipError_t launch_tile(const GemmArgs& a, int S, hipStream_t st) {
  const int nb = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  if (S <= 1) {
    hipLaunchKernelGGL((gemm_nt_kernel<BM, BN, EPI, false>), dim3(nb), dim3(256), 0, st, a);
  } else {
    hipLaunchKernelGGL((gemm_nt_kernel<BM, BN, EPI, true>), dim3(nb, 1, S), dim3(256), 0, st, a);
    const int n_out = (EPI == EPI_SWIGLU) ? a.N / 2 : a.N;
    const size_t tot = (size_t)a.M * n_out;
    hipLaunchKernelGGL((splitk_reduce_kernel<EPI>), dim3((tot + 255) / 256), dim3(256), 0, st, a, S);
  }
  return hipGetLastError();
}

template <int EPI>
hipError_t launch_epi(GemmArgs a, const GemmPlan& p, hipStream_t st) {
  a.k_chunk = p.k_chunk;
  if (p.bm == 128) return launch_tile<128, 128, EPI>(a, p.splits, st);
  return launch_tile<64, 64, EPI>(a, p.splits, st);
}

}  // namespace

// Tile and split-K choice.  Large M: 128x128 tiles.  Small M (decode): 64x64
// tiles, split along K until the grid has about 1024 workgroups, keeping at
// least 256 K-elements per split.
GemmPlan gemm_plan(int M, int N, int K, int max_splits) {
  GemmPlan p;
  if (M > 256) {
    p.bm = 128;
    p.splits = 1;
    p.k_chunk = K;
    return p;
  }
  p.bm = 64;
  const int tiles = ((M + 63) / 64) * ((N + 63) / 64);
  int s = 1;
  while (s < max_splits && tiles * s < 1024 && (K / (s * 2)) >= 256) s *= 2;
  const int kc = (((K + s - 1) / s) + BK - 1) / BK * BK;
  p.splits = (K + kc - 1) / kc;
  p.k_chunk = kc;
  return p;
}

hipError_t gemm_launch(const GemmArgs& a, int epi, const GemmPlan& p, hipStream_t st) {
  switch (epi) {
    case EPI_BF16: return launch_epi<EPI_BF16>(a, p, st);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, p, st);
    case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(a, p, st);
    default: return launch_epi<EPI_F32>(a, p, st);
  }
}

}  // namespace hxf
