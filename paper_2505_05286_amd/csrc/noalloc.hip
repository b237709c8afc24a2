// hxf_op_gemm_noalloc: the GEMM entry point for callers that cannot allocate
// device memory (code under HIP graph capture, serving loops, harnesses that
// forbid allocation).  Its split-K partials live in a device array owned by the
// library instead of a caller workspace.
#include <hip/hip_runtime.h>

#include <mutex>

#include "hxf_ops.h"
#include "kernels/kernels.hpp"

using namespace hxf;

namespace {

constexpr int64_t kScratchBytes = HXF_GEMM_NOALLOC_MAX_BYTES;

// One copy per GPU, held until the process ends.  In host code `scratch` names a
// host-side stand-in: kernels get the device address from hipGetSymbolAddress.
__device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of this device's `scratch`, looked up once per device (with
// that device current) and kept.
int scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return HXF_EDEVICE;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return HXF_EDEVICE;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return HXF_OK;
}

}  // namespace

extern "C" int hxf_op_gemm_noalloc(const void* A, int32_t lda, const void* B, const void* B2, void* C, int32_t ldc,
                                   int32_t M, int32_t N, int32_t K, int32_t epi, void* stream) {
  if (!A || !B || !C || M < 0 || N <= 0 || K <= 0 || K % 8 || lda < K || epi < 0 || epi > 3) return HXF_EINVAL;
  if (epi == HXF_EPI_SWIGLU && (!B2 || N % 32)) return HXF_EINVAL;
  if (ldc < (epi == HXF_EPI_SWIGLU ? N / 2 : N)) return HXF_EINVAL;
  if (M == 0) return HXF_OK;
  const GemmPlan p = gemm_plan(M, N, K, 8, epi == HXF_EPI_SWIGLU);
  const int64_t need = p.splits > 1 ? (int64_t)p.splits * M * N * 4 : 0;
  if (need > kScratchBytes) return HXF_ENOMEM;
  GemmArgs a{};
  if (need > 0) {
    void* s = nullptr;
    if (int rc = scratch_address(&s)) return rc;
    a.partial = static_cast<float*>(s);
  }
  a.A = (const uint16_t*)A;
  a.B = (const uint16_t*)B;
  a.B2 = (const uint16_t*)B2;
  a.C = C;
  a.M = M;
  a.N = N;
  a.K = K;
  a.lda = lda;
  a.ldc = ldc;
  a.kt = (K + 31) / 32;
  return gemm_launch(a, epi, p, (hipStream_t)stream) == hipSuccess ? HXF_OK : HXF_EDEVICE;
}
