// Integrate-and-fire neurons (Sec. II-B, Eqs. (3)-(4)) and the 8-bit table
// non-linearity, as standalone kernels over int32 currents.
#include "common.h"

namespace nmdlm {

// One wave per (token, 64-neuron word); lane = neuron.  Integrate-then-fire
// with soft reset; the membrane is int64 so any int32 currents are exact.
// Timesteps go in rounds of R (4 for T <= 4, else 8) whose current (and
// residual) loads are all issued before the recurrence uses the first of
// them; a round past T repeats the last timestep's address and drops it.
template <int R>
__global__ __launch_bounds__(256) void k_if(const int32_t* __restrict__ cur, int T, int M, int N,
                                            int32_t theta, const int32_t* __restrict__ theta_vec,
                                            const uint64_t* __restrict__ resid,
                                            int32_t* __restrict__ v_inout,
                                            uint64_t* __restrict__ s_out,
                                            uint64_t* __restrict__ u_out) {
  const int Nw = (N + 63) / 64;
  // M * Nw <= 2^19 * 1024 units: 32-bit, wave-uniform (scalar) arithmetic
  const int unit = __builtin_amdgcn_readfirstlane((int)blockIdx.x * 4 + ((int)threadIdx.x >> 6));
  if (unit >= M * Nw) return;  // wave-uniform
  const int lane = threadIdx.x & 63;
  const int m = unit / Nw, w = unit - m * Nw;
  const int n = w * 64 + lane;
  const bool nv = n < N;
  const int nc = nv ? n : N - 1;  // lanes past N read a valid current and drop it
  const long long th = theta_vec ? theta_vec[nc] : theta;
  long long V = (v_inout && nv) ? v_inout[(size_t)m * N + n] : 0;
  uint64_t uor = 0;
  for (int t0 = 0; t0 < T; t0 += R) {
    int32_t cu[R];
    uint64_t rw[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int t = min(t0 + u, T - 1);
      cu[u] = cur[((size_t)t * M + m) * N + nc];
      rw[u] = resid ? resid[((size_t)t * M + m) * Nw + w] : 0ull;
    }
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int t = t0 + u;
      if (t >= T) break;  // wave-uniform
      long long I = nv ? cu[u] : 0;
      if ((rw[u] >> lane) & 1ull) I += th;
      V += I;
      const bool s = nv && V >= th;
      if (s) V -= th;
      const uint64_t word = __builtin_amdgcn_ballot_w64(s);
      uor |= word;
      if (lane == 0) s_out[((size_t)t * M + m) * Nw + w] = word;
    }
  }
  if (v_inout && nv) v_inout[(size_t)m * N + n] = (int32_t)V;
  // partial union over t of this token's word, for a following product
  if (u_out && lane == 0) u_out[(size_t)m * Nw + w] = uor;
}

__global__ __launch_bounds__(256) void k_qnl(const int32_t* __restrict__ x, int64_t n, int shift,
                                             int mode, const uint8_t* __restrict__ lut,
                                             uint8_t* __restrict__ y) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) {
    const int v = x[i];
    int idx;
    if (mode == NMDLM_QNL_S8) {
      int q = v >> shift;  // arithmetic shift: floor(v / 2^shift)
      q = min(127, max(-128, q));
      idx = q & 0xFF;
    } else {
      idx = min(255, max(0, v));
    }
    y[i] = lut[idx];
  }
}

__global__ __launch_bounds__(256) void k_fill_zero(uint4* __restrict__ p, size_t n16) {
  const size_t stride = (size_t)gridDim.x * 256;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += stride)
    p[i] = uint4{0u, 0u, 0u, 0u};
}

nmdlm_status launch_if(const int32_t* cur, int T, int M, int N, int32_t theta,
                       const int32_t* theta_vec, const uint64_t* resid, int32_t* v_inout,
                       uint64_t* s_out, hipStream_t st, uint64_t* u_out) {
  const long long units = (long long)M * ((N + 63) / 64);
  const long long blocks = (units + 3) / 4;
  if (T <= 4)
    hipLaunchKernelGGL(k_if<4>, dim3((unsigned)blocks), dim3(256), 0, st, cur, T, M, N, theta,
                       theta_vec, resid, v_inout, s_out, u_out);
  else
    hipLaunchKernelGGL(k_if<8>, dim3((unsigned)blocks), dim3(256), 0, st, cur, T, M, N, theta,
                       theta_vec, resid, v_inout, s_out, u_out);
  return hip_status();
}

nmdlm_status launch_qnl(const int32_t* x, int64_t n, int shift, int mode, const uint8_t* lut,
                        uint8_t* y, hipStream_t st) {
  if (n == 0) return NMDLM_OK;
  long long blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_qnl, dim3((unsigned)blocks), dim3(256), 0, st, x, n, shift, mode, lut, y);
  return hip_status();
}

nmdlm_status launch_fill_zero(void* p, size_t bytes, hipStream_t st) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return NMDLM_OK;
  size_t blocks = (n16 + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)blocks), dim3(256), 0, st,
                     reinterpret_cast<uint4*>(p), n16);
  return hip_status();
}

}  // namespace nmdlm
