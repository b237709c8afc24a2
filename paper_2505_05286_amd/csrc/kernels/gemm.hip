// bf16 "NT" GEMMs on CDNA4 matrix cores: C[M,N] = A[M,K] * B[N,K]^T with an
// fp32 accumulator and fused epilogues (bf16 store, fp32 residual add, SwiGLU
// gate*up, fp32 store) or fp32 split-K partials.  A is row-major activations, B
// the packed weights (see below).  Three kernels (gemm_plan picks):
//   gemm_stream_kernel: weight streaming through LDS DMA on 16x16x32 MFMAs, split K;
//     M <= 128;
//   gemm_big_kernel: macro tiles of up to 256 x 256 on 32x32x16 MFMAs fed by LDS DMA,
//     four or eight wavefronts, tile shape chosen per GEMM; M > 512, outputs of
//     N >= 16384 above 64 rows, SwiGLU above 128 rows, and 128 < M <= 512 with split
//     K otherwise;
//   gemm_nt_kernel: 128x128 tiles of 16x16x32 MFMAs, K staged through LDS from
//     registers; SwiGLU whose N is not a multiple of 64 on the big kernel's shapes.
// Workgroups are renumbered so that consecutive output tiles (which share a
// weight slice) land on the same XCD and its L2.
#include <hip/hip_ext.h>

#include <algorithm>
#include <utility>

#include "common.hpp"
#include "kernels.hpp"

namespace hxf {

namespace {

constexpr int BK_MAX = 128;

// B operands are packed weights: 16-row x 32-column tiles of 1 KB, row-tiles
// outermost, and inside a tile the 8-element chunks in MFMA operand order
// [k/8][row][8] (element (n, k) at ((n/16)*kt + k/32)*512 + ((k%32)/8)*128 +
// (n%16)*8 + k%8, kt = ceil(K/32), zero padding).  One wavefront-wide 16-byte
// load of a tile is 1 KB of contiguous memory.
__device__ __forceinline__ size_t b_koff(int k) { return (size_t)(k >> 5) * 512 + ((k >> 3) & 3) * 128; }

// Start of weight row n (k = 0) of a packed matrix.
__device__ __forceinline__ const bf16_t* b_packed_row(const bf16_t* W, int kt, int n) {
  return W + (size_t)(n >> 4) * kt * 512 + (n & 15) * 8;
}

// Logical column c of a GEMM; SwiGLU interleaves groups of 32 = 16 gate rows then 16 up rows.
__device__ __forceinline__ const bf16_t* b_row(const GemmArgs& a, int c, bool swiglu) {
  if (!swiglu) return b_packed_row(a.B, a.kt, c);
  const int g = c >> 5, w = c & 31;
  return b_packed_row((w < 16) ? a.B : a.B2, a.kt, g * 16 + (w & 15));
}

// 16-byte load from a 16-byte aligned address (one global_load_dwordx4).
__device__ __forceinline__ uint4 load16(const bf16_t* p) {
  const u32x4_t v = *reinterpret_cast<const u32x4_t*>(__builtin_assume_aligned(p, 16));
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ int xcd_remap(int i, int nb) {
  const int xcd = i & 7, local = i >> 3;
  const int per = nb >> 3, rem = nb & 7;
  return (xcd < rem) ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// Launch; with events, the kernel itself records its start (e0) and end (e1).
template <typename K, typename... Args>
hipError_t launch_ev(K kernel, dim3 grid, dim3 block, hipStream_t st, hipEvent_t e0, hipEvent_t e1, Args... args) {
  if (e0 || e1) hipExtLaunchKernelGGL(kernel, grid, block, 0, st, e0, e1, 0, args...);
  else hipLaunchKernelGGL(kernel, grid, block, 0, st, args...);
  return hipGetLastError();
}

template <int BM, int BN, int BK, int NS, int EPI, bool SPLIT>
__global__ __launch_bounds__(256) void gemm_nt_kernel(GemmArgs a) {
  constexpr int LDS_ROW = BK + 8;                   // bf16 elements per LDS row (16-byte pad)
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

  // global load bookkeeping: chunk j of this thread = row (tid + j*256) / CPR, col16 (tid % CPR)
  constexpr int CPR = BK / 8;                       // 16-byte chunks per row of a K tile
  const int c16 = tid % CPR;
  const bf16_t* a_ptr[A_CH];
  const bf16_t* b_ptr[B_CH];
  bool a_ok[A_CH], b_ok[B_CH];
#pragma unroll
  for (int j = 0; j < A_CH; ++j) {
    const int r = (tid + j * 256) / CPR;
    a_ok[j] = (m0 + r) < a.M;
    a_ptr[j] = a.A + (size_t)(a_ok[j] ? m0 + r : 0) * a.lda + c16 * 8;
  }
#pragma unroll
  for (int j = 0; j < B_CH; ++j) {
    const int r = (tid + j * 256) / CPR;
    b_ok[j] = (n0 + r) < a.N;
    b_ptr[j] = b_row(a, b_ok[j] ? n0 + r : 0, SW) + b_koff(c16 * 8);
  }
  // NS register stages: the K tiles it+1 .. it+NS-1 are in flight while tile it
  // is multiplied (one stage is the tile being stored to LDS).
  uint4 ra[NS][A_CH], rb[NS][B_CH];
  auto fetch = [&](uint4 (&xa)[A_CH], uint4 (&xb)[B_CH], int k0) {
    const bool kin = (k0 + c16 * 8) < ke;
#pragma unroll
    for (int j = 0; j < A_CH; ++j)
      xa[j] = (a_ok[j] && kin) ? *reinterpret_cast<const uint4*>(a_ptr[j] + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int j = 0; j < B_CH; ++j)
      xb[j] = (b_ok[j] && kin) ? *reinterpret_cast<const uint4*>(b_ptr[j] + (size_t)k0 * 16) : make_uint4(0, 0, 0, 0);
  };
  auto stage_to_lds = [&](const uint4 (&xa)[A_CH], const uint4 (&xb)[B_CH]) {
#pragma unroll
    for (int j = 0; j < A_CH; ++j) {
      const int r = (tid + j * 256) / CPR;
      *reinterpret_cast<uint4*>(&As[r * LDS_ROW + c16 * 8]) = xa[j];
    }
#pragma unroll
    for (int j = 0; j < B_CH; ++j) {
      const int r = (tid + j * 256) / CPR;
      *reinterpret_cast<uint4*>(&Bs[r * LDS_ROW + c16 * 8]) = xb[j];
    }
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&]() {
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
  };

#pragma unroll
  for (int st = 0; st < NS; ++st)
    if (kb + st * BK < ke) fetch(ra[st], rb[st], kb + st * BK);
  for (int k0 = kb; k0 < ke; k0 += NS * BK) {
#pragma unroll
    for (int st = 0; st < NS; ++st) {
      const int kt = k0 + st * BK;
      if (kt < ke) {
        __syncthreads();
        stage_to_lds(ra[st], rb[st]);
        __syncthreads();
        if (kt + NS * BK < ke) fetch(ra[st], rb[st], kt + NS * BK);
        compute();
      }
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
    reinterpret_cast<bf16_t*>(a.C)[a.c_kt ? packed_elem(row, col, a.c_kt) : (size_t)row * a.ldc + col] =
        f2bf(g / (1.f + __expf(-g)) * u);
    return;
  }
  float s = 0.f;
  for (int z = 0; z < S; ++z) s += a.partial[z * MN + (size_t)row * a.N + col];
  const size_t o = (size_t)row * a.ldc + col;
  if (EPI == EPI_BF16) reinterpret_cast<bf16_t*>(a.C)[o] = f2bf(s);
  else if (EPI == EPI_RESID) reinterpret_cast<float*>(a.C)[o] += s;
  else reinterpret_cast<float*>(a.C)[o] = s;
}

// Decode-sized M (at most 16 * MT rows): a weight-streaming kernel fed by the
// LDS DMA path (global_load_lds, 16 bytes per lane, no registers).  Each of
// the WV wavefronts owns NTW 16-column tiles; a stage holds 32*KB K-elements of
// the A rows (MT x KB MFMA blocks, loaded by all wavefronts together) and of
// each wavefront's weight tiles (NTW x KB blocks), each block 1 KB laid out in
// MFMA operand order.  NSTG stages are in flight: a wavefront waits for its
// own DMAs of the oldest stage (vmcnt), one barrier makes everybody's visible
// and frees the slot consumed one step earlier, which is refilled before the
// multiplies.  Stages live in distinct LDS arrays and the loop is unrolled by
// NSTG so the compiler can see that the LDS reads of a stage do not alias the
// DMAs in flight (otherwise it waits for all of them).  The weights, read once per
// step, are fetched with the non-temporal hint (decode step 8.41 -> 8.25 ms; the same
// hint on the prefill kernel's operands, which other workgroups re-read from L2, made
// workload-3 iterations 9% slower).  Split K (grid.y) writes fp32 partials; a
// reduction kernel (or the consumer) finishes them.
constexpr int ST_WV = 4, ST_NTW = 2, ST_KB = 2, ST_NSTG = 3;
constexpr int ST_COLS = ST_WV * ST_NTW * 16;          // output columns per workgroup
constexpr int ST_KS = 32 * ST_KB;                     // K per stage

// Stages of the streaming kernel with MT row tiles: as many as asked for that fit 160 KB
// of LDS (wide row tiles may get fewer; below 2 the kernel is not used).
template <int MT>
constexpr int stream_stages() {
  constexpr int bytes = (MT * ST_KB + ST_WV * ST_NTW * ST_KB) * 1024;
  return ST_NSTG < 160 * 1024 / bytes ? ST_NSTG : 160 * 1024 / bytes;
}

template <int MT, int EPI, bool SPLIT>
__global__ __launch_bounds__(64 * ST_WV) void gemm_stream_kernel(GemmArgs a) {
  constexpr int WV = ST_WV, NTW = ST_NTW, KB = ST_KB, KS = ST_KS;
  constexpr int A_BLK = MT * KB, B_BLK_W = NTW * KB;
  constexpr int STAGE = (A_BLK + WV * B_BLK_W) * 512;       // bf16 elements per stage
  constexpr int NSTG = stream_stages<MT>();
  constexpr int A_PER_W = (A_BLK + WV - 1) / WV;            // A blocks each wavefront moves (last one repeated)
  constexpr int PER_STAGE = A_PER_W + B_BLK_W;              // DMA instructions per wavefront per stage
  constexpr bool SW = (EPI == EPI_SWIGLU);
  static_assert(NSTG >= 2 && NSTG <= 6, "stage layout");
  static_assert((NSTG - 2) * PER_STAGE < 64, "vmcnt range");
  __shared__ __attribute__((aligned(1024))) bf16_t L0[STAGE], L1[STAGE], L2[NSTG > 2 ? STAGE : 8],
      L3[NSTG > 3 ? STAGE : 8], L4[NSTG > 4 ? STAGE : 8], L5[NSTG > 5 ? STAGE : 8];
  auto slot = [&](auto ic) -> bf16_t* {
    constexpr int I = decltype(ic)::value;
    if constexpr (I == 0) return L0; else if constexpr (I == 1) return L1; else if constexpr (I == 2) return L2;
    else if constexpr (I == 3) return L3; else if constexpr (I == 4) return L4; else return L5;
  };
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15, g = lane >> 4;
  const int c0 = (blockIdx.x * WV + w) * NTW * 16;          // first logical column of this wavefront
  const int kb = blockIdx.y * a.k_chunk;
  const int ke = min(a.K, kb + a.k_chunk);
  const int kend = a.kt * 32;                               // packed K (zero padded past K)
  const int nst = (ke - kb + KS - 1) / KS;

  // weight tile sources, lane offset included (tiles past the end repeat the last one; dropped)
  const bf16_t* bsrc[NTW];
#pragma unroll
  for (int j = 0; j < NTW; ++j) bsrc[j] = b_row(a, min(c0 + j * 16, a.N - 1) & ~15, SW) + lane * 8;
  // A block b = (row tile b / KB, 32-column block b % KB): lane reads row 16 (b / KB) + r
  // (rows past M repeat M-1)
  // packed activations: the block's row tile (past M: the last one) with the lane's offset
  const bf16_t* arow[A_PER_W];
  int ablk[A_PER_W];
#pragma unroll
  for (int u = 0; u < A_PER_W; ++u) {
    ablk[u] = min(w * A_PER_W + u, A_BLK - 1);
    arow[u] = a.a_packed ? a.A + (size_t)min(ablk[u] / KB, (a.M - 1) / 16) * a.kt * 512 + lane * 8
                         : a.A + (size_t)min((ablk[u] / KB) * 16 + r, a.M - 1) * a.lda;
  }
  auto issue = [&](int s, bf16_t* base) {
    const int k0 = kb + min(s, nst - 1) * KS;               // past the last stage: reload it (never read)
#pragma unroll
    for (int u = 0; u < A_PER_W; ++u) {
      const int kk = ablk[u] % KB;
      // row-major: stays in the row (the weights are zero past K); packed: a whole tile
      const size_t off = a.a_packed ? (size_t)min(k0 / 32 + kk, a.kt - 1) * 512 : (size_t)min(k0 + kk * 32 + g * 8, a.K - 8);
      dma16(arow[u] + off, base + ablk[u] * 512);
    }
#pragma unroll
    for (int j = 0; j < NTW; ++j)
#pragma unroll
      for (int kk = 0; kk < KB; ++kk) {
        const int t = min(k0 / 32 + kk, a.kt - 1);
        dma16_nt(bsrc[j] + (size_t)t * 512, base + (A_BLK + w * B_BLK_W + j * KB + kk) * 512);
      }
  };
  f32x4 acc[MT][NTW];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NTW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const bf16_t* base, int s) {
    const int k0 = kb + s * KS;
#pragma unroll
    for (int kk = 0; kk < KB; ++kk) {
      if (k0 + kk * 32 >= kend) break;                      // a 32-block wholly past the packed K
      bf16x8 fa[MT], fb[NTW];
#pragma unroll
      for (int i = 0; i < MT; ++i)
        fa[i] = as_bf16x8(*reinterpret_cast<const uint4*>(base + (i * KB + kk) * 512 + lane * 8));
#pragma unroll
      for (int j = 0; j < NTW; ++j)
        fb[j] = as_bf16x8(*reinterpret_cast<const uint4*>(base + (A_BLK + w * B_BLK_W + j * KB + kk) * 512 + lane * 8));
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NTW; ++j) acc[i][j] = mfma16x16x32(fa[i], fb[j], acc[i][j]);
    }
  };

  static_for<NSTG - 1>([&](auto ic) { issue(decltype(ic)::value, slot(ic)); });
  int s0 = 0;
  for (; s0 + NSTG <= nst; s0 += NSTG) {
    static_for<NSTG>([&](auto ic) {
      constexpr int J = decltype(ic)::value;
      wait_vmcnt<(NSTG - 2) * PER_STAGE>();
      __builtin_amdgcn_s_barrier();
      issue(s0 + J + NSTG - 1, slot(std::integral_constant<int, (J + NSTG - 1) % NSTG>{}));
      compute(slot(ic), s0 + J);
    });
  }
  // the remaining nst - s0 < NSTG stages are already in flight, in slots 0, 1, ..
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  static_for<NSTG - 1>([&](auto ic) {
    if (s0 + decltype(ic)::value < nst) compute(slot(ic), s0 + decltype(ic)::value);
  });

  // lane holds rows 16i + 4g + e, column c0 + 16j + r
  if (SPLIT) {
    float* P = a.partial + (size_t)blockIdx.y * a.M * a.N;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = i * 16 + g * 4 + e;
        if (row >= a.M) continue;
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
          const int col = c0 + j * 16 + r;
          if (col < a.N) P[(size_t)row * a.N + col] = acc[i][j][e];
        }
      }
    return;
  }
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = i * 16 + g * 4 + e;
      if (row >= a.M) continue;
      if (SW) {
        // SwiGLU: tile pairs (2q, 2q+1) are the gate and up rows of logical group (c0 + 32q) / 32
#pragma unroll
        for (int q = 0; q < NTW / 2; ++q) {
          const int cq = c0 + q * 32;
          if (cq >= a.N) continue;
          const float gt = acc[i][2 * q][e], up = acc[i][2 * q + 1][e];
          const int oc = (cq >> 5) * 16 + r;
          reinterpret_cast<bf16_t*>(a.C)[a.c_kt ? packed_elem(row, oc, a.c_kt) : (size_t)row * a.ldc + oc] =
              f2bf(gt / (1.f + __expf(-gt)) * up);
        }
      } else {
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
          const int col = c0 + j * 16 + r;
          if (col >= a.N) continue;
          const size_t o = (size_t)row * a.ldc + col;
          if (EPI == EPI_BF16) reinterpret_cast<bf16_t*>(a.C)[o] = f2bf(acc[i][j][e]);
          else if (EPI == EPI_RESID) reinterpret_cast<float*>(a.C)[o] += acc[i][j][e];
          else reinterpret_cast<float*>(a.C)[o] = acc[i][j][e];
        }
      }
    }
}

template <int MT, int EPI>
hipError_t launch_stream(const GemmArgs& a, int S, hipStream_t st, bool reduce, hipEvent_t e0, hipEvent_t e1) {
  const int nb = (a.N + ST_COLS - 1) / ST_COLS;
  if (S > 1) {
    if (hipError_t e = launch_ev(gemm_stream_kernel<MT, EPI, true>, dim3(nb, S), dim3(64 * ST_WV), st, e0,
                                 reduce ? nullptr : e1, a))
      return e;
    if (!reduce) return hipSuccess;
    const int n_out = (EPI == EPI_SWIGLU) ? a.N / 2 : a.N;
    const size_t tot = (size_t)a.M * n_out;
    return launch_ev(splitk_reduce_kernel<EPI>, dim3((tot + 255) / 256), dim3(256), st, nullptr, e1, a, S);
  }
  return launch_ev(gemm_stream_kernel<MT, EPI, false>, dim3(nb, 1), dim3(64 * ST_WV), st, e0, e1, a);
}

// Prefill-sized M: BM x BN macro tiles on the 32x32x16 bf16 MFMA, fed by the
// LDS DMA path.  A stage is 32 of K: the BM/16 A blocks (16 rows x 32 columns
// of the activations, 1 KB each, in the MFMA operand order [k/8][row][8]) and
// the BN/16 packed weight tiles, DMA'd by the WM x WN wavefronts together (each
// moves the same number of blocks; where the blocks do not divide evenly the
// last block is moved again, an identical write); NSTG stages in flight in
// distinct LDS arrays (see the streaming kernel for the wait and barrier
// discipline).  Wavefront (wm, wn) owns rows wm*BM/WM.. and columns wn*BN/WN..
// as tiles of 32 x 32.  With eight wavefronts two share each SIMD, so one issues
// MFMAs while the other waits on LDS.  BM is any multiple of 32 so that the
// row tiles can match the batch (2080 rows = 13 x 160).  SwiGLU groups logical
// columns by 64 (32 gate rows, then the 32 matching up rows) so one lane holds
// both; it needs BN/WN a multiple of 64.  SPLIT: grid.y splits K into chunks of
// k_chunk (a multiple of 32) and each writes its fp32 partial [M][N] to slot
// blockIdx.y of a.partial, summed by the consumer (not with SwiGLU).
template <int BM, int BN, int WM, int WN, int NSTG, int EPI, bool SPLIT>
__global__ __launch_bounds__(64 * WM * WN, 1) void gemm_big_kernel(GemmArgs a) {
  constexpr int W = WM * WN;
  constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
  static_assert(TM * WM * 32 == BM && TN * WN * 32 == BN, "wavefront tiling");
  constexpr int AB = BM / 16, BB = BN / 16, NBLK = AB + BB;   // 1 KB blocks per stage
  constexpr int PER_W = (NBLK + W - 1) / W;                   // DMA instructions per wavefront per stage
  constexpr int STAGE = NBLK * 512;
  constexpr bool SW = (EPI == EPI_SWIGLU);
  static_assert(!SW || TN % 2 == 0, "SwiGLU pairs 32-column tiles");
  static_assert(!(SW && SPLIT), "split partials hold logical columns; SwiGLU needs both halves summed first");
  static_assert(NSTG >= 3 && NSTG <= 5 && NSTG * STAGE * 2 <= 160 * 1024, "stage layout");
  __shared__ __attribute__((aligned(1024))) bf16_t L0[STAGE], L1[STAGE], L2[STAGE], L3[NSTG > 3 ? STAGE : 8],
      L4[NSTG > 4 ? STAGE : 8];
  auto slot = [&](auto ic) -> bf16_t* {
    constexpr int I = decltype(ic)::value;
    if constexpr (I == 0) return L0; else if constexpr (I == 1) return L1; else if constexpr (I == 2) return L2;
    else if constexpr (I == 3) return L3; else return L4;
  };
  const int tiles_m = (a.M + BM - 1) / BM;
  const int tiles_n = (a.N + BN - 1) / BN;
  const int L = xcd_remap(blockIdx.x, tiles_m * tiles_n);
  const int tn = L / tiles_m, tm = L % tiles_m;
  const int m0 = tm * BM, n0 = tn * BN;
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w / WN, wn = w % WN;
  const int kb = SPLIT ? blockIdx.y * a.k_chunk : 0;
  const int ke = SPLIT ? min(a.K, kb + a.k_chunk) : a.K;
  const int nst = (ke - kb + 31) / 32;

  // This wavefront's DMA blocks w*PER_W + u: an A block (16 activation rows, the
  // lane's row and 8-column chunk; with packed activations a 1 KB tile like the
  // weights') or a packed weight tile (1 KB contiguous).  No per-block branches at
  // issue time, so the compiler keeps track of which LDS array each DMA writes.
  const bf16_t* src[PER_W];
  int step[PER_W];   // elements per stage: 32 along an activation row, 512 for a weight tile
  int dst[PER_W];
#pragma unroll
  for (int u = 0; u < PER_W; ++u) {
    const int gb = min(w * PER_W + u, NBLK - 1);
    dst[u] = gb * 512;
    if (gb < AB && a.a_packed) {
      // row tiles past M repeat the last one (its rows past M are never stored)
      src[u] = a.A + (size_t)min(m0 / 16 + gb, (a.M - 1) / 16) * a.kt * 512 + lane * 8;
      step[u] = 512;
    } else if (gb < AB) {
      src[u] = a.A + (size_t)min(m0 + gb * 16 + (lane & 15), a.M - 1) * a.lda + (lane >> 4) * 8;
      step[u] = 32;
    } else {
      const int c = min(n0 + (gb - AB) * 16, a.N - 1) & ~15;   // logical column of the tile (past N: repeat)
      const bf16_t* mat = a.B;
      int row = c;
      if (SW) {
        const int g = c >> 6, w64 = c & 63;
        mat = (w64 < 32) ? a.B : a.B2;
        row = g * 32 + (w64 & 31);
      }
      src[u] = mat + (size_t)(row >> 4) * a.kt * 512 + lane * 8;
      step[u] = 512;
    }
  }
  // A past K: a chunk of the row is read again (its weights are zero): the lane's last
  // in-row chunk, or the row's first when K < 32 (never an address before the row)
  const int a_last = max(a.K - 8 - (lane >> 4) * 8, 0);
  auto issue = [&](int s, bf16_t* base) {
    const int k0 = kb + min(s, nst - 1) * 32;   // past the end: reload the last stage (unused)
#pragma unroll
    for (int u = 0; u < PER_W; ++u) {
      const int off = step[u] == 32 ? min(k0, a_last) : (k0 >> 5) * 512;
      dma16(src[u] + off, base + dst[u]);
    }
  };
  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  // 32x32x16 operand of lane l: row (or column) l % 32 of the tile, k chunk l / 32 of the
  // 16-wide slice.  The offsets are precomputed so that every LDS read is its array plus
  // one offset: the compiler must still see which array a read comes from, or it waits
  // for every DMA in flight.
  const int lo = ((lane & 31) >> 4) * 512 + (lane >> 5) * 128 + (lane & 15) * 8;
  int a_off[TM], b_off[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) a_off[i] = ((wm * TM + i) * 2) * 512 + lo;
#pragma unroll
  for (int j = 0; j < TN; ++j) b_off[j] = (AB + (wn * TN + j) * 2) * 512 + lo;
  // all fragments of a stage are read first (distinct registers), then the MFMAs; the
  // scheduling groups interleave one LDS read with one MFMA so that the reads' latency
  // hides under the matrix pipe instead of stalling it
  auto compute = [&](const bf16_t* base) {
    bf16x8 fa[2][TM], fb[2][TN];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
#pragma unroll
      for (int j = 0; j < TN; ++j) fb[q][j] = as_bf16x8(*reinterpret_cast<const uint4*>(base + b_off[j] + q * 256));
#pragma unroll
      for (int i = 0; i < TM; ++i) fa[q][i] = as_bf16x8(*reinterpret_cast<const uint4*>(base + a_off[i] + q * 256));
    }
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(fa[q][i], fb[q][j], acc[i][j]);
    constexpr int RD = 2 * (TM + TN), MF = 2 * TM * TN, PAIRS = RD < MF ? RD : MF;
    static_for<PAIRS>([&](auto) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
    });
    if constexpr (MF > PAIRS) __builtin_amdgcn_sched_group_barrier(0x008, MF - PAIRS, 0);
    if constexpr (RD > PAIRS) __builtin_amdgcn_sched_group_barrier(0x100, RD - PAIRS, 0);
  };

  static_for<NSTG - 1>([&](auto ic) { issue(decltype(ic)::value, slot(ic)); });
  int s0 = 0;
  for (; s0 + NSTG <= nst; s0 += NSTG) {
    static_for<NSTG>([&](auto ic) {
      constexpr int J = decltype(ic)::value;
      wait_vmcnt<(NSTG - 2) * PER_W>();
      __builtin_amdgcn_s_barrier();
      issue(s0 + J + NSTG - 1, slot(std::integral_constant<int, (J + NSTG - 1) % NSTG>{}));
      compute(slot(ic));
    });
  }
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  static_for<NSTG - 1>([&](auto ic) {
    if (s0 + decltype(ic)::value < nst) compute(slot(ic));
  });

  // lane holds column l % 32 and rows 8*(r/4) + 4*(lane/32) + r%4 of each 32x32 tile
  const int l32 = lane & 31, rq = (lane >> 5) * 4;
  const int wr0 = m0 + wm * (BM / WM), wc0 = n0 + wn * (BN / WN);
  if (SPLIT) {
    float* P = a.partial + (size_t)blockIdx.y * a.M * a.N;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wr0 + i * 32 + (r >> 2) * 8 + rq + (r & 3);
        if (row >= a.M) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int col = wc0 + j * 32 + l32;
          if (col < a.N) P[(size_t)row * a.N + col] = acc[i][j][r];
        }
      }
    return;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    if (EPI == EPI_RESID) {
      // residual loads of RB rows first, then the adds and stores (one wait per RB rows)
      constexpr int RB = TN > 3 ? 4 : TN > 1 ? 8 : 16;
      float* C = reinterpret_cast<float*>(a.C);
#pragma unroll
      for (int r0 = 0; r0 < 16; r0 += RB) {
        float old[RB][TN];
#pragma unroll
        for (int r = 0; r < RB; ++r) {
          const int rr = r0 + r;
          const int row = min(wr0 + i * 32 + (rr >> 2) * 8 + rq + (rr & 3), a.M - 1);
#pragma unroll
          for (int j = 0; j < TN; ++j) old[r][j] = C[(size_t)row * a.ldc + min(wc0 + j * 32 + l32, a.N - 1)];
        }
#pragma unroll
        for (int r = 0; r < RB; ++r) {
          const int rr = r0 + r;
          const int row = wr0 + i * 32 + (rr >> 2) * 8 + rq + (rr & 3);
          if (row >= a.M) continue;
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int col = wc0 + j * 32 + l32;
            if (col < a.N) C[(size_t)row * a.ldc + col] = old[r][j] + acc[i][j][rr];
          }
        }
      }
      continue;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = wr0 + i * 32 + (r >> 2) * 8 + rq + (r & 3);
      if (row >= a.M) continue;
      if (SW) {
#pragma unroll
        for (int j = 0; j < TN; j += 2) {
          const int lc = wc0 + j * 32;   // first (gate) logical column of the 64-group
          if (lc >= a.N) continue;
          const float g = acc[i][j][r], u = acc[i][j + 1][r];
          const int oc = (lc >> 6) * 32 + l32;
          reinterpret_cast<bf16_t*>(a.C)[a.c_kt ? packed_elem(row, oc, a.c_kt) : (size_t)row * a.ldc + oc] =
              f2bf(g / (1.f + __expf(-g)) * u);
        }
      } else {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int col = wc0 + j * 32 + l32;
          if (col >= a.N) continue;
          const size_t o = (size_t)row * a.ldc + col;
          if (EPI == EPI_BF16) reinterpret_cast<bf16_t*>(a.C)[o] = f2bf(acc[i][j][r]);
          else reinterpret_cast<float*>(a.C)[o] = acc[i][j][r];
        }
      }
    }
  }
}

// Macro-tile shapes of the big kernel: (BM, BN, WM x WN wavefronts), a per-flop cost
// factor measured on the projection shapes (smaller tiles move more bytes per flop,
// one-row wavefront grids read more LDS per MFMA), and whether the wavefront column
// span suits SwiGLU.  Stages: as many as fit 160 KB of LDS, at most five.
struct BigCfg {
  int bm, bn, wm, wn;
  double f;
  bool swiglu;
};
constexpr BigCfg kBig[] = {
    {256, 256, 4, 2, 1.02, true}, {224, 256, 1, 8, 1.10, false}, {192, 256, 2, 4, 1.0, true},
    {160, 256, 1, 8, 1.17, false}, {128, 256, 2, 4, 1.3, true},    {128, 128, 2, 2, 1.6, true},
    {256, 128, 2, 2, 1.3, true},
};
constexpr int kNumBig = sizeof(kBig) / sizeof(kBig[0]);
constexpr int kNumPrefillBig = 6;   // the shapes chosen among for M > 512

template <int BM, int BN, int WM, int WN, int EPI>
hipError_t launch_big(const GemmArgs& a, int S, hipStream_t st, bool reduce, hipEvent_t e0, hipEvent_t e1) {
  constexpr int STAGE_BYTES = (BM + BN) * 64;
  constexpr int NSTG = std::min(5, 160 * 1024 / STAGE_BYTES);
  const int nb = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  if constexpr (EPI != EPI_SWIGLU) {
    if (S > 1) {
      if (hipError_t e = launch_ev(gemm_big_kernel<BM, BN, WM, WN, NSTG, EPI, true>, dim3(nb, S), dim3(64 * WM * WN),
                                   st, e0, reduce ? nullptr : e1, a))
        return e;
      if (!reduce) return hipSuccess;
      const size_t tot = (size_t)a.M * a.N;
      return launch_ev(splitk_reduce_kernel<EPI>, dim3((tot + 255) / 256), dim3(256), st, nullptr, e1, a, S);
    }
  } else {
    if (S > 1) return hipErrorInvalidValue;
  }
  return launch_ev(gemm_big_kernel<BM, BN, WM, WN, NSTG, EPI, false>, dim3(nb), dim3(64 * WM * WN), st, e0, e1, a);
}

template <int EPI>
hipError_t launch_big_cfg(const GemmArgs& a, int cfg, int S, hipStream_t st, bool reduce, hipEvent_t e0,
                          hipEvent_t e1) {
  switch (cfg) {
    case 0: return launch_big<256, 256, 4, 2, EPI>(a, S, st, reduce, e0, e1);
    case 2: return launch_big<192, 256, 2, 4, EPI>(a, S, st, reduce, e0, e1);
    case 4: return launch_big<128, 256, 2, 4, EPI>(a, S, st, reduce, e0, e1);
    case 5: return launch_big<128, 128, 2, 2, EPI>(a, S, st, reduce, e0, e1);
    case 6: return launch_big<256, 128, 2, 2, EPI>(a, S, st, reduce, e0, e1);
    default: break;
  }
  if constexpr (EPI != EPI_SWIGLU) {
    if (cfg == 1) return launch_big<224, 256, 1, 8, EPI>(a, S, st, reduce, e0, e1);
    if (cfg == 3) return launch_big<160, 256, 1, 8, EPI>(a, S, st, reduce, e0, e1);
  }
  return hipErrorInvalidValue;
}

template <int BM, int BN, int BK, int NS, int EPI>
hipError_t launch_tile(const GemmArgs& a, int S, hipStream_t st, bool reduce, hipEvent_t e0, hipEvent_t e1) {
  const int nb = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  if (S <= 1) return launch_ev(gemm_nt_kernel<BM, BN, BK, NS, EPI, false>, dim3(nb), dim3(256), st, e0, e1, a);
  if (hipError_t e = launch_ev(gemm_nt_kernel<BM, BN, BK, NS, EPI, true>, dim3(nb, 1, S), dim3(256), st, e0,
                               reduce ? nullptr : e1, a))
    return e;
  if (!reduce) return hipSuccess;
  const int n_out = (EPI == EPI_SWIGLU) ? a.N / 2 : a.N;
  const size_t tot = (size_t)a.M * n_out;
  return launch_ev(splitk_reduce_kernel<EPI>, dim3((tot + 255) / 256), dim3(256), st, nullptr, e1, a, S);
}

template <int EPI>
hipError_t launch_epi(GemmArgs a, const GemmPlan& p, hipStream_t st, bool reduce, hipEvent_t e0, hipEvent_t e1) {
  a.k_chunk = p.k_chunk;
  if (p.stream) {
    if (p.bm <= 32) return launch_stream<2, EPI>(a, p.splits, st, reduce, e0, e1);
    if (p.bm <= 64) return launch_stream<4, EPI>(a, p.splits, st, reduce, e0, e1);
    return launch_stream<8, EPI>(a, p.splits, st, reduce, e0, e1);
  }
  if (p.big) {
    // SwiGLU on the big kernel pairs 32 gate with 32 up columns: needs F % 32 == 0
    if (EPI == EPI_SWIGLU && a.N % 64 != 0) return launch_tile<128, 128, 64, 2, EPI>(a, 1, st, true, e0, e1);
    return launch_big_cfg<EPI>(a, p.cfg, p.splits, st, reduce, e0, e1);
  }
  return launch_tile<128, 128, 64, 2, EPI>(a, p.splits, st, reduce, e0, e1);
}

// One 16-byte chunk of the packed layout per thread: chunk q is tile q / 64 and,
// inside it, [k/8 = (q % 64) / 16][row = q % 16].
__global__ __launch_bounds__(256) void pack_weight_kernel(const bf16_t* __restrict__ W, int N, int K, int kt,
                                                         bf16_t* __restrict__ out, size_t n_chunks) {
  const size_t q = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= n_chunks) return;
  const size_t tile = q >> 6;
  const int c = (int)(q & 63);
  const int n = (int)(tile / kt) * 16 + (c & 15);
  const int k = (int)(tile % kt) * 32 + (c >> 4) * 8;
  uint4 v = make_uint4(0, 0, 0, 0);
  if (n < N && k < K) v = load16(W + (size_t)n * K + k);
  *reinterpret_cast<uint4*>(out + q * 8) = v;
}

}  // namespace

size_t packed_weight_elems(int N, int K) { return (size_t)((N + 15) / 16) * 16 * (size_t)((K + 31) / 32) * 32; }

hipError_t pack_weight_launch(const uint16_t* W, int N, int K, uint16_t* out, hipStream_t st) {
  const size_t n_chunks = packed_weight_elems(N, K) / 8;
  hipLaunchKernelGGL(pack_weight_kernel, dim3((unsigned)((n_chunks + 255) / 256)), dim3(256), 0, st,
                     reinterpret_cast<const bf16_t*>(W), N, K, (K + 31) / 32, reinterpret_cast<bf16_t*>(out), n_chunks);
  return hipGetLastError();
}

// Kernel, tile and split-K choice.  M <= 128: the weight-streaming kernel, except
// for wide outputs (N >= 16384) above 64 rows, which take the big-tile kernel as
// every M > 512 and every SwiGLU above 128 rows do.  The other 128 < M <= 512
// shapes: the big-tile kernel with split K.
GemmPlan gemm_plan(int M, int N, int K, int max_splits, bool swiglu) {
  GemmPlan p;
  // big tiles: the shape minimising whole rounds of one workgroup per CU times tile area
  // times its cost factor (the last round costs as much as a full one)
  auto big = [&]() {
    double best = 0;
    for (int c = 0; c < kNumPrefillBig; ++c) {
      const BigCfg& g = kBig[c];
      if (swiglu && !g.swiglu) continue;
      const int tiles = ((M + g.bm - 1) / g.bm) * ((N + g.bn - 1) / g.bn);
      const double cost = (double)((tiles + 255) / 256) * g.bm * g.bn * g.f;
      if (best == 0 || cost < best - 1e-6) {
        best = cost;
        p.cfg = c;
        p.bm = g.bm;
        p.bn = g.bn;
      }
    }
    p.big = true;
    p.splits = 1;
    p.k_chunk = K;
    return p;
  };
  // 128 < M <= 512, N < 16384, not SwiGLU: big tiles with K split (fp32 partials the
  // consumer sums).  Shape and split minimise a per-launch estimate fitted to measured
  // times on the 8B projections at 128-512 rows: 0.366 us per million tile-area x
  // K-chunk x cost-factor units (every workgroup of a round runs at once), plus 0.24 us
  // per MB of partials written and read back.
  auto mid = [&]() {
    double best = 0;
    for (int c : {4, 5, 0, 6}) {
      const BigCfg& g = kBig[c];
      const int tiles = ((M + g.bm - 1) / g.bm) * ((N + g.bn - 1) / g.bn);
      for (int s = 1; s <= max_splits; ++s) {
        if (s > 1 && (tiles * s > 256 || K / s < 512)) break;
        const int kc = ((K + s - 1) / s + 31) / 32 * 32;
        const int splits = (K + kc - 1) / kc;
        const double rounds = (tiles * splits + 255) / 256;
        const double t = 0.366e-6 * rounds * g.bm * g.bn * (double)kc * g.f +
                         (splits > 1 ? 0.24e-6 * splits * (double)M * N * 4 : 0.0);
        if (best == 0 || t < best - 1e-9) {
          best = t;
          p.cfg = c;
          p.bm = g.bm;
          p.bn = g.bn;
          p.k_chunk = kc;
          p.splits = splits;
        }
      }
    }
    p.big = true;
    return p;
  };
  if (M > 128 && M <= 512 && N < 16384 && !swiglu) return mid();
  if (M > 512 || (M > 64 && N >= 16384) || (M > 128 && swiglu)) return big();
  if (M <= 128) {
    // weight streaming (16 * MT rows): 128 columns per workgroup; K split into the most
    // pieces that keep the grid within one workgroup per CU and >= 512 of K per piece
    p.stream = true;
    p.bm = M <= 32 ? 32 : M <= 64 ? 64 : 128;
    const int tiles = (N + ST_COLS - 1) / ST_COLS;
    int s = 1;
    while (s + 1 <= max_splits && tiles * (s + 1) <= 256 && K / (s + 1) >= 512) ++s;
    p.k_chunk = (((K + s - 1) / s) + ST_KS - 1) / ST_KS * ST_KS;
    p.splits = (K + p.k_chunk - 1) / p.k_chunk;
    return p;
  }
  p.bm = 128;
  p.splits = 1;
  p.k_chunk = K;
  return p;
}

hipError_t gemm_launch(const GemmArgs& a, int epi, const GemmPlan& p, hipStream_t st, bool reduce, hipEvent_t e0,
                       hipEvent_t e1) {
  // packed activations in, or a packed SwiGLU output: the streaming and the big-tile kernels
  // (and the split-K reduction) with K % 32 == 0 and F % 32 == 0
  if ((a.a_packed && (a.K % 32 || !(p.stream || p.big) || (epi == EPI_SWIGLU && a.N % 64 != 0))) ||
      (a.c_kt && (!(p.stream || p.big) || epi != EPI_SWIGLU || a.N % 64 != 0 || a.c_kt * 64 != a.N)))
    return hipErrorInvalidValue;
  switch (epi) {
    case EPI_BF16: return launch_epi<EPI_BF16>(a, p, st, reduce, e0, e1);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, p, st, reduce, e0, e1);
    case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(a, p, st, reduce, e0, e1);
    default: return launch_epi<EPI_F32>(a, p, st, reduce, e0, e1);
  }
}

}  // namespace hxf
