// Attention on spike operands: binary-binary scores (popcount of AND), table
// weights, integer-normalised weighted sum of binary values.
//
//   s = popcount(Q_i AND K_j) per head;  p = lut[s] in [0, 255]
//   num[i,c] = sum_j p_ij V[j,c];  den[i] = sum_j p_ij
//   a[i,c] = floor(256 * num / den)   (0 if den = 0)
//
// The weighted sum runs on v_mfma_i32_16x16x64_i8: the A operand holds
// p - 128 (signed byte), the B operand the value bits expanded to bytes, and
// 128 * (number of ones of V[.,c]) is added back, so the int32 result is exact.
#include "common.h"

namespace nmdlm {

__device__ __forceinline__ uint32_t expand4_a(uint32_t nib) {
  return (nib * 0x00204081u) & 0x01010101u;
}

// grid (H, ceil(M/16), T); 4 waves take 64-key chunks in turn.
template <int DHW>
__global__ __launch_bounds__(256) void k_attn(const uint64_t* __restrict__ q,
                                              const uint64_t* __restrict__ kc,
                                              const uint64_t* __restrict__ vt, int64_t cap, int T,
                                              int M, int C, int H,
                                              const uint8_t* __restrict__ lut,
                                              int32_t* __restrict__ a_out) {
  constexpr int DH = DHW * 64;
  constexpr int NT = DH / 16;
  __shared__ int sLut[256];
  __shared__ int sNum[4][16][DH];
  __shared__ int sDen[16];
  __shared__ int sCnt[DH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int h = blockIdx.x, qb = blockIdx.y, t = blockIdx.z;
  const int d = H * DH, dw = d / 64;
  const int capw = (int)(cap / 64);
  const int J = C + M;
  const int nch = (J + 63) / 64;

  sLut[tid] = lut[tid];
  if (tid < 16) sDen[tid] = 0;
  for (int i = tid; i < DH; i += 256) sCnt[i] = 0;

  const int iq = qb * 16 + c;
  const bool qv = iq < M;
  uint64_t qw[DHW];
#pragma unroll
  for (int w = 0; w < DHW; ++w) qw[w] = qv ? q[((size_t)t * M + iq) * dw + h * DHW + w] : 0ull;
  __syncthreads();

  v4i acc[NT];
  int cnt[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    acc[i] = v4i{0, 0, 0, 0};
    cnt[i] = 0;
  }
  int den = 0;

  for (int jc = wave; jc < nch; jc += 4) {
    const int j0 = jc * 64 + 16 * g;
    uint32_t pk[4] = {0u, 0u, 0u, 0u};
    // keys past C+M read a valid row (clamped) and are masked, so that all
    // sixteen key loads are issued back to back
    uint64_t kw[16][DHW];
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      const int jj = min(j0 + s, J - 1);
      const uint64_t* kr = kc + ((size_t)t * cap + jj) * dw + h * DHW;
#pragma unroll
      for (int w = 0; w < DHW; ++w) kw[s][w] = kr[w];
    }
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      int sc = 0;
#pragma unroll
      for (int w = 0; w < DHW; ++w) sc += __popcll(qw[w] & kw[s][w]);
      const bool jv = j0 + s < J;
      const int p = jv ? sLut[sc] : 0;
      den += p;
      pk[s >> 2] |= jv ? (uint32_t)((p - 128) & 0xFF) << ((s & 3) * 8) : 0u;
    }
    const v4i af = v4i{(int)pk[0], (int)pk[1], (int)pk[2], (int)pk[3]};
    const int nvalid = J - j0;
    const uint32_t vmask = nvalid >= 16 ? 0xFFFFu : (nvalid <= 0 ? 0u : ((1u << nvalid) - 1u));
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int ch = h * DH + nt * 16 + c;
      const uint64_t wv = vt[((size_t)t * d + ch) * capw + jc];
      const uint32_t bits = (uint32_t)(wv >> (16 * g)) & vmask;
      cnt[nt] += __popc(bits);
      const v4i bf = v4i{(int)expand4_a(bits & 0xFu), (int)expand4_a((bits >> 4) & 0xFu),
                         (int)expand4_a((bits >> 8) & 0xFu), (int)expand4_a(bits >> 12)};
      acc[nt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, bf, acc[nt], 0, 0, 0);
    }
  }

#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int e = 0; e < 4; ++e) sNum[wave][g * 4 + e][nt * 16 + c] = acc[nt][e];
  atomicAdd(&sDen[c], den);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) atomicAdd(&sCnt[nt * 16 + c], cnt[nt]);
  __syncthreads();

  for (int i = tid; i < 16 * DH; i += 256) {
    const int qi = i / DH, ch = i - qi * DH;
    const int iq2 = qb * 16 + qi;
    if (iq2 < M) {
      const long long num = (long long)sNum[0][qi][ch] + sNum[1][qi][ch] + sNum[2][qi][ch] +
                            sNum[3][qi][ch] + 128LL * sCnt[ch];
      const long long dn = sDen[qi];
      a_out[((size_t)t * M + iq2) * d + h * DH + ch] = dn > 0 ? (int32_t)((256LL * num) / dn) : 0;
    }
  }
}

nmdlm_status launch_attn(const uint64_t* q, const uint64_t* k_cache, const uint64_t* vt_cache,
                         int64_t cap, int T, int M, int C, int H, int dh, const uint8_t* lut,
                         int32_t* a_out, hipStream_t st) {
  const dim3 grid(H, (M + 15) / 16, T);
  switch (dh / 64) {
    case 1:
      hipLaunchKernelGGL(k_attn<1>, grid, dim3(256), 0, st, q, k_cache, vt_cache, cap, T, M, C, H,
                         lut, a_out);
      break;
    case 2:
      hipLaunchKernelGGL(k_attn<2>, grid, dim3(256), 0, st, q, k_cache, vt_cache, cap, T, M, C, H,
                         lut, a_out);
      break;
    default:
      return NMDLM_ERR_UNSUPPORTED;
  }
  return hip_status();
}

}  // namespace nmdlm
