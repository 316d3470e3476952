// nmdlm_qbsm_noalloc: the spike product without a caller workspace, for
// callers that cannot allocate device memory (code under stream capture,
// serving loops, harnesses that forbid allocation).  Its scratch memory is a
// file-scope device array; each GPU the library runs on holds its own copy
// until the process ends.
#include <mutex>

#include "common.h"

namespace nmdlm {
namespace {

// The scratch of every nmdlm_qbsm_noalloc call on one GPU.  In host code the
// name stands for a host-side shadow, not the device memory: the device
// address is taken once per device with hipGetSymbolAddress and used
// everywhere host code needs the array (kernel arguments, the fill below).
__device__ __align__(256) unsigned char scratch[NMDLM_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];  // device address of `scratch`, per device (null: not set up)

// Device address of this device's scratch; the first call on a device takes
// it (with the device current) and clears the array on the caller's stream.
nmdlm_status device_scratch(hipStream_t st, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return NMDLM_ERR_HIP;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return NMDLM_ERR_HIP;
    const nmdlm_status rc = launch_fill_zero(p, NMDLM_NOALLOC_SCRATCH_BYTES, st);
    if (rc != NMDLM_OK) return rc;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return NMDLM_OK;
}

}  // namespace
}  // namespace nmdlm

extern "C" nmdlm_status nmdlm_qbsm_noalloc(const uint64_t* s_in, int T, int M, int K,
                                           const int8_t* W, int N, int64_t ldw,
                                           const int32_t* bias, int32_t* cur_out, int32_t theta,
                                           const int32_t* theta_vec, uint64_t* s_out,
                                           nmdlm_qbsm_stats* stats, unsigned flags, void* stream) {
  // the same argument checks as nmdlm_qbsm, and the size limit, before any HIP call
  if (!s_in || T < 1 || M < 1 || K < 1 || N < 1) return NMDLM_ERR_INVALID_ARG;
  if (T > NMDLM_MAX_T || K > NMDLM_MAX_K) return NMDLM_ERR_UNSUPPORTED;
  if ((int64_t)T * M > (1 << 19)) return NMDLM_ERR_UNSUPPORTED;
  if (!cur_out && !s_out) return NMDLM_ERR_INVALID_ARG;
  if (s_out && !theta_vec && theta <= 0) return NMDLM_ERR_INVALID_ARG;
  const size_t need = nmdlm_qbsm_workspace_size(T, M, K, N);
  if (need == 0 || need > (size_t)NMDLM_NOALLOC_SCRATCH_BYTES) return NMDLM_ERR_UNSUPPORTED;
  if (!W || ldw < N || (ldw % 16) != 0 || reinterpret_cast<uintptr_t>(W) % 16 != 0)
    return NMDLM_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  void* ws = nullptr;
  const nmdlm_status rc = nmdlm::device_scratch(st, &ws);
  if (rc != NMDLM_OK) return rc;
  return nmdlm_qbsm(s_in, T, M, K, W, N, ldw, bias, cur_out, theta, theta_vec, s_out, stats, flags,
                    ws, (size_t)NMDLM_NOALLOC_SCRATCH_BYTES, stream);
}
