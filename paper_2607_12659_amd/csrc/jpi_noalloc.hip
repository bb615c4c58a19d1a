// The allocation-free variant of the library's GEMM entry point
// (jpi_gemm_noalloc, include/jpi.h).  jpi_debug_gemm allocates the split-K
// partial slices on every call and synchronises its stream; this variant
// runs the same kernels with the slices in a file-scope device array and
// enqueues without synchronising, so that callers that cannot allocate
// (code under HIP graph capture, tight serving loops) can use it.
#include <mutex>
#include <string>

#include "jpi_internal.h"

namespace jpi {
namespace {

constexpr size_t SCRATCH_BYTES = size_t(16) << 20;  // split-K slices: splitk * M * N fp32
constexpr int MAX_DEVICES = 64;

// Each GPU the library runs on holds its own copy until the process ends.
// In host code `scratch` names a host-side stand-in, never the device
// memory: host code uses the per-device address from hipGetSymbolAddress.
__device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];

std::mutex g_mu;
void* g_scratch[MAX_DEVICES] = {};

// Device address of `scratch` on the current device (looked up once per
// device, with that device current).
hipError_t scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

thread_local std::string g_err;

jpi_status fail(jpi_status st, const std::string& msg) {
  g_err = msg;
  return st;
}

}  // namespace
}  // namespace jpi

using namespace jpi;

extern "C" {

size_t jpi_gemm_noalloc_scratch_bytes(void) { return SCRATCH_BYTES; }

const char* jpi_gemm_noalloc_last_error(void) { return g_err.c_str(); }

jpi_status jpi_gemm_noalloc(const void* A, const void* Wt, float* C, int M, int N, int K, jpi_dtype dt, int splitk,
                            void* stream) {
  if (!A || !Wt || !C) return fail(JPI_ERR_ARG, "jpi_gemm_noalloc: NULL pointer");
  if (M < 1 || N < 1 || K < 1 || splitk < 1) return fail(JPI_ERR_ARG, "jpi_gemm_noalloc: sizes must be >= 1");
  if (dt != JPI_F32 && dt != JPI_BF16) return fail(JPI_ERR_ARG, "jpi_gemm_noalloc: bad dtype");
  const int q = gemm_k_quantum(dt, M);
  if (K % (q * splitk) != 0)
    return fail(JPI_ERR_ARG, "jpi_gemm_noalloc: K must be a multiple of " + std::to_string(q) + "*splitk");
  const size_t need = splitk > 1 ? (size_t)splitk * (size_t)M * (size_t)N * sizeof(float) : 0;
  if (need > SCRATCH_BYTES)
    return fail(JPI_ERR_ARG, "jpi_gemm_noalloc: splitk*M*N*4 = " + std::to_string(need) +
                                 " bytes exceeds the static scratch of " + std::to_string(SCRATCH_BYTES) + " bytes");
  hipStream_t s = (hipStream_t)stream;
  GemmLaunch g{};
  g.A = A;
  g.W = Wt;
  g.M = M;
  g.N = N;
  g.K = K;
  g.splitk = splitk;
  g.epi = EPI_STORE_F32;
  g.ep.out_f32 = C;
  hipError_t e = hipSuccess;
  float* part = nullptr;
  if (splitk > 1) {
    // every slice is written whole by the GEMM before the sum reads it, so
    // the scratch needs no clearing between calls
    e = scratch_ptr(reinterpret_cast<void**>(&part));
    g.ep.out_f32 = part;
  }
  if (e == hipSuccess) e = launch_gemm(dt, g, s);
  if (e == hipSuccess && splitk > 1) e = launch_sum_slices(part, C, splitk, (size_t)M * N, s);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(JPI_ERR_HIP, std::string("jpi_gemm_noalloc: ") + hipGetErrorString(e));
  }
  return JPI_OK;
}

}  // extern "C"
