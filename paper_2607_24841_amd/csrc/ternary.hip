// Ternary bitwise coding of integer activations (Sec. III-B, Eqs. (7)-(8)).
//
//   V_th = mean(|a|) / K = S / (D K),   S = sum_i |a_i|
//   q_i  = round(a_i / V_th) = round(a_i D K / S)   (halves away from zero;
//          0 when S = 0; |q| capped at 2^T - 1)
//   s_{i,t} = sign(q_i) * bit t-1 of |q_i|,  t = 1..T
//
// The +1 and -1 spikes go out as two packed planes [T][M][ceil(D/64)] (the
// product reads both; the row-load rule takes their union).  The division is
// exact integer arithmetic, so the planes do not depend on rounding order.
#include "common.h"

namespace nmdlm {

constexpr int kTernThreads = 256;

// One workgroup per token: the magnitude sum, then one wave per 64-channel
// word (lane = channel), one ballot per plane and timestep.
__global__ __launch_bounds__(kTernThreads) void k_ternary_encode(
    const int32_t* __restrict__ a, int M, int D, int K, int T, uint64_t* __restrict__ sp,
    uint64_t* __restrict__ sn, int64_t* __restrict__ s_sum) {
  __shared__ long long sPart[kTernThreads / 64];
  const int m = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t* row = a + (size_t)m * D;
  long long part = 0;
  for (int i = tid; i < D; i += kTernThreads) part += llabs((long long)row[i]);
  for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o);
  if (lane == 0) sPart[wave] = part;
  __syncthreads();
  long long S = 0;
#pragma unroll
  for (int w = 0; w < kTernThreads / 64; ++w) S += sPart[w];
  if (s_sum && tid == 0) s_sum[m] = S;

  const int Dw = (D + 63) / 64;
  const long long lim = (1LL << T) - 1, DK = (long long)D * K;
  for (int w = wave; w < Dw; w += kTernThreads / 64) {  // wave-uniform
    const int i = w * 64 + lane;
    const int v = i < D ? row[i] : 0;
    long long mag = 0;
    if (S > 0 && v != 0) {
      const long long num = llabs((long long)v) * DK;
      mag = min((2 * num + S) / (2 * S), lim);  // floor(|a| D K / S + 1/2)
    }
    for (int t = 0; t < T; ++t) {
      const bool bit = (mag >> t) & 1;
      const uint64_t pw = __builtin_amdgcn_ballot_w64(bit && v > 0);
      const uint64_t nw = __builtin_amdgcn_ballot_w64(bit && v < 0);
      if (lane == 0) {
        sp[((size_t)t * M + m) * Dw + w] = pw;
        sn[((size_t)t * M + m) * Dw + w] = nw;
      }
    }
  }
}

nmdlm_status launch_ternary_encode(const int32_t* a, int M, int D, int K, int T, uint64_t* sp,
                                   uint64_t* sn, int64_t* s_sum, hipStream_t st) {
  hipLaunchKernelGGL(k_ternary_encode, dim3(M), dim3(kTernThreads), 0, st, a, M, D, K, T, sp, sn,
                     s_sum);
  return hip_status();
}

}  // namespace nmdlm
