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
constexpr int kTernWords = kTernThreads / 64;  // 64-channel words per workgroup (one per wave)
constexpr int kTernSumUnroll = 16;  // loads per thread per batch of the magnitude sum

// floor(n / d) for 0 <= n < 2^53, 0 < d < 2^53: a double estimate corrected
// by integer multiplies (the estimate is within one of the quotient).
__device__ __forceinline__ long long div_floor(long long n, long long d) {
  long long q = (long long)((double)n / (double)d);
  if (q * d > n) --q;
  if ((q + 1) * d <= n) ++q;
  return q;
}

// Workgroup (token m, chunk j): the token's magnitude sum S (every chunk
// recomputes it; the row is read from cache), then wave w quantises word
// 4j + w (lane = channel) and writes one ballot per plane and timestep.
__global__ __launch_bounds__(kTernThreads) void k_ternary_encode(
    const int32_t* __restrict__ a, int M, int D, int K, int T, uint64_t* __restrict__ sp,
    uint64_t* __restrict__ sn, int64_t* __restrict__ s_sum) {
  __shared__ long long sPart[kTernWords];
  const int m = blockIdx.x, chunk = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t* row = a + (size_t)m * D;
  const int Dw = (D + 63) / 64;
  const int w = chunk * kTernWords + wave;
  const int i = w * 64 + lane;
  const int v = (w < Dw && i < D) ? row[i] : 0;  // this lane's channel, loaded with the row
  // the magnitude sum: batches of kTernSumUnroll loads per thread, all
  // issued before the first is added (16-byte loads when the row allows)
  long long part = 0;
  if ((D & 3) == 0 && (reinterpret_cast<uintptr_t>(row) & 15) == 0) {
    const int4* r4 = reinterpret_cast<const int4*>(row);
    const int D4 = D >> 2;
    for (int i0 = tid; i0 < D4; i0 += kTernThreads * kTernSumUnroll) {
      int4 x[kTernSumUnroll];
#pragma unroll
      for (int u = 0; u < kTernSumUnroll; ++u) {
        const int j = i0 + u * kTernThreads;
        x[u] = j < D4 ? r4[j] : int4{0, 0, 0, 0};
      }
#pragma unroll
      for (int u = 0; u < kTernSumUnroll; ++u)
        part += llabs((long long)x[u].x) + llabs((long long)x[u].y) + llabs((long long)x[u].z) +
                llabs((long long)x[u].w);
    }
  } else {
    for (int i0 = tid; i0 < D; i0 += kTernThreads * kTernSumUnroll) {
      int32_t x[kTernSumUnroll];
#pragma unroll
      for (int u = 0; u < kTernSumUnroll; ++u) {
        const int j = i0 + u * kTernThreads;
        x[u] = j < D ? row[j] : 0;
      }
#pragma unroll
      for (int u = 0; u < kTernSumUnroll; ++u) part += llabs((long long)x[u]);
    }
  }
  for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o);
  if (lane == 0) sPart[wave] = part;
  __syncthreads();
  long long S = 0;
#pragma unroll
  for (int ww = 0; ww < kTernWords; ++ww) S += sPart[ww];
  if (s_sum && chunk == 0 && tid == 0) s_sum[m] = S;

  if (w >= Dw) return;  // wave-uniform
  const long long lim = (1LL << T) - 1, DK = (long long)D * K;
  long long mag = 0;
  if (S > 0 && v != 0) {
    const long long num = llabs((long long)v) * DK;
    mag = min(div_floor(2 * num + S, 2 * S), lim);  // floor(|a| D K / S + 1/2)
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

nmdlm_status launch_ternary_encode(const int32_t* a, int M, int D, int K, int T, uint64_t* sp,
                                   uint64_t* sn, int64_t* s_sum, hipStream_t st) {
  const int Dw = (D + 63) / 64;
  hipLaunchKernelGGL(k_ternary_encode, dim3(M, (Dw + kTernWords - 1) / kTernWords),
                     dim3(kTernThreads), 0, st, a, M, D, K, T, sp, sn, s_sum);
  return hip_status();
}

}  // namespace nmdlm
