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

// Table bytes 4*lane .. 4*lane+3 as one dword (byte loads: any alignment).
__device__ __forceinline__ int lut_dword(const uint8_t* __restrict__ lut, int lane) {
  const uint8_t* b = lut + 4 * lane;
  return (int)((uint32_t)b[0] | ((uint32_t)b[1] << 8) | ((uint32_t)b[2] << 16) |
               ((uint32_t)b[3] << 24));
}

// floor(256 * num / den) for 0 <= num <= den (0 when den = 0).  For fewer
// than 65536 keys, a = 256 num < 2^32 and den < 2^24: the quotient (at most
// 256) is estimated as a float product with the hardware reciprocal, whose
// relative error (a few units of 2^-24) keeps the estimate within one of
// the exact floor, and one remainder test corrects it (the remainder
// a - q den lies in (-2 den, 2 den), exact in wrapped 32-bit arithmetic).
// Larger key counts divide in 64 bits.
__device__ __forceinline__ int32_t attn_norm(long long num, long long den, bool small) {
  if (den <= 0) return 0;
  if (small) {
    const uint32_t a = 256u * (uint32_t)num, b = (uint32_t)den;
    uint32_t q = (uint32_t)((float)a * __builtin_amdgcn_rcpf((float)b));
    const int32_t r = (int32_t)(a - q * b);
    if (r < 0) --q;
    else if ((uint32_t)r >= b) ++q;
    return (int32_t)q;
  }
  return (int32_t)((256LL * num) / den);
}

// grid (H, n_seq * ceil(M/16), T), M queries per sequence, rows of q and
// a_out sequence-major (n_seq * M per timestep), the caches of sequence s at
// s * seq_words words past kc / vt; wave i takes 64-key chunks i, i+NW, ...  Every
// load of a chunk (16 keys per lane, NT value words) is issued before it is
// scored; with up to 64*NW keys each wave has one chunk, so all the key and
// value loads of the workgroup are in flight together.  The table is read
// with ds_bpermute from lut_dw (entry s sits in byte s%4 of lane s/4).
template <int DHW, int NW>
__global__ __launch_bounds__(NW * 64) void k_attn(const uint64_t* __restrict__ q,
                                                  const uint64_t* __restrict__ kc,
                                                  const uint64_t* __restrict__ vt, int64_t cap,
                                                  int T, int M, int C, int H,
                                                  const uint8_t* __restrict__ lut,
                                                  int32_t* __restrict__ a_out, int n_seq,
                                                  int64_t seq_words) {
  constexpr int DH = DHW * 64;
  constexpr int NT = DH / 16;
  constexpr int NTH = NW * 64;
  __shared__ int sNum[16][DH];
  __shared__ int sDen[16];
  __shared__ int sCnt[DH];
  __shared__ uint64_t sKey[NW][64 * DHW];  // each wave's chunk of key rows
  __shared__ uint64_t sVal[NW][DH];        // and its value words, one per channel

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  // neighbouring heads share key lines: consecutive logical ids, head fastest
  const int nwg = gridDim.x * gridDim.y * gridDim.z;
  const int lid = xcd_order(blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z), nwg);
  const int h = lid % gridDim.x, qbg = (lid / gridDim.x) % gridDim.y,
            t = lid / (gridDim.x * gridDim.y);
  const int qbps = gridDim.y / n_seq;               // query blocks per sequence
  const int sq = qbg / qbps, qb = qbg - sq * qbps;  // sequence, block within it
  const int Mt = n_seq * M, r0 = sq * M;            // rows per timestep, first row of sq
  kc += sq * seq_words;
  vt += sq * seq_words;
  const int d = H * DH, dw = d / 64;
  const int capw = (int)(cap / 64);
  const int J = C + M;
  const int nch = (J + 63) / 64;

  const int lut_dw = lut_dword(lut, lane);
  const int iq = qb * 16 + c;
  uint64_t qw[DHW];
#pragma unroll
  for (int w = 0; w < DHW; ++w)
    qw[w] = q[((size_t)t * Mt + r0 + min(iq, M - 1)) * dw + h * DHW + w];
  for (int i = tid; i < 16 * DH; i += NTH) (&sNum[0][0])[i] = 0;
  if (tid < 16) sDen[tid] = 0;
  for (int i = tid; i < DH; i += NTH) sCnt[i] = 0;

  v4i acc[NT];
  int cnt[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    acc[i] = v4i{0, 0, 0, 0};
    cnt[i] = 0;
  }
  int den = 0;
  // rows of queries past M (clamped loads) are scored too; they are never read

  uint64_t* const sK = sKey[wave];
  uint64_t* const sV = sVal[wave];
  for (int jc = wave; jc < nch; jc += NW) {  // wave-uniform
    const int j0 = jc * 64 + 16 * g;
    // lane l loads key row jc*64 + l (rows past C+M read a valid row, masked
    // when scored) and the chunk's rows meet in the wave's LDS buffer
    const uint64_t* kr = kc + ((size_t)t * cap + min(jc * 64 + lane, J - 1)) * dw + h * DHW;
    uint64_t kl[DHW];
#pragma unroll
    for (int w = 0; w < DHW; ++w) kl[w] = kr[w];
    // lane l loads the chunk's value words of channels l, l + 64, ...
    uint64_t vl[DHW];
#pragma unroll
    for (int w = 0; w < DHW; ++w) vl[w] = vt[((size_t)t * capw + jc) * d + h * DH + w * 64 + lane];
    __builtin_amdgcn_sched_barrier(0);  // every load above is issued before the first use
#pragma unroll
    for (int w = 0; w < DHW; ++w) {
      sK[lane * DHW + w] = kl[w];
      sV[w * 64 + lane] = vl[w];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    uint32_t pk[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      int sc = 0;
#pragma unroll
      for (int w = 0; w < DHW; ++w) sc += __popcll(qw[w] & sK[(16 * g + s) * DHW + w]);
      const bool jv = j0 + s < J;
      const int pw = __builtin_amdgcn_ds_bpermute((sc >> 2) << 2, lut_dw);
      const int p = jv ? (pw >> ((sc & 3) * 8)) & 0xFF : 0;
      den += p;
      pk[s >> 2] |= jv ? (uint32_t)((p - 128) & 0xFF) << ((s & 3) * 8) : 0u;
    }
    const v4i af = v4i{(int)pk[0], (int)pk[1], (int)pk[2], (int)pk[3]};
    const int nvalid = J - j0;
    const uint32_t vmask = nvalid >= 16 ? 0xFFFFu : (nvalid <= 0 ? 0u : ((1u << nvalid) - 1u));
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const uint32_t bits = (uint32_t)(sV[nt * 16 + c] >> (16 * g)) & vmask;
      cnt[nt] += __popc(bits);
      const v4i bf = v4i{(int)expand4_a(bits & 0xFu), (int)expand4_a((bits >> 4) & 0xFu),
                         (int)expand4_a((bits >> 8) & 0xFu), (int)expand4_a(bits >> 12)};
      acc[nt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, bf, acc[nt], 0, 0, 0);
    }
    __builtin_amdgcn_wave_barrier();  // the buffers' reads precede the next chunk's stores
  }
  __syncthreads();  // the partial sums are cleared
  if (wave < nch) {  // wave-uniform
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int e = 0; e < 4; ++e) atomicAdd(&sNum[g * 4 + e][nt * 16 + c], acc[nt][e]);
    atomicAdd(&sDen[c], den);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) atomicAdd(&sCnt[nt * 16 + c], cnt[nt]);
  }
  __syncthreads();

  const bool small = J < 65536;
  for (int i = tid; i < 16 * DH; i += NTH) {
    const int qi = i / DH, ch = i - qi * DH;
    const int iq2 = qb * 16 + qi;
    if (iq2 < M) {
      const long long num = (long long)sNum[qi][ch] + 128LL * sCnt[ch];
      a_out[((size_t)t * Mt + r0 + iq2) * d + h * DH + ch] = attn_norm(num, sDen[qi], small);
    }
  }
}

// waves per workgroup: 16 for dh = 64; 8 or 12 for dh = 128 (its 16 keys of
// two words per lane need more than the 128 registers of a 1024-thread group);
// halved while the grid would not fit the chip in one round (many sequences:
// fewer waves per workgroup take more key chunks each, the workgroups of all
// sequences run at once)
constexpr int kAttnWaves64 = 16, kAttnWaves128 = 8;
// waves resident at once: 256 CUs x 16 (the kernels' registers allow 4-5
// waves per SIMD)
constexpr long long kAttnResidentWaves = 256LL * 16;
constexpr long long kAttnCus = 256;

struct AttnLaunch {
  const uint64_t* q;
  const uint64_t* kc;
  const uint64_t* vt;
  int64_t cap;
  int T, M, C, H;
  const uint8_t* lut;
  int32_t* a_out;
  int n_seq;
  int64_t seq_words;
};

template <int DHW, int NW>
static void attn_launch(const dim3& grid, const AttnLaunch& l, hipStream_t st) {
  hipLaunchKernelGGL((k_attn<DHW, NW>), grid, dim3(NW * 64), 0, st, l.q, l.kc, l.vt, l.cap, l.T, l.M,
                     l.C, l.H, l.lut, l.a_out, l.n_seq, l.seq_words);
}

nmdlm_status launch_attn(const uint64_t* q, const uint64_t* k_cache, const uint64_t* vt_cache,
                         int64_t cap, int T, int M, int C, int H, int dh, const uint8_t* lut,
                         int32_t* a_out, hipStream_t st, int n_seq, int64_t seq_words) {
  if (n_seq < 1) return NMDLM_ERR_INVALID_ARG;
  const dim3 grid(H, n_seq * ((M + 15) / 16), T);
  const long long wgs = (long long)grid.x * grid.y * grid.z;
  int nw = (dh == 64) ? kAttnWaves64 : kAttnWaves128;
  // dh = 128: 12 waves (168 registers: three waves per SIMD, one workgroup
  // per CU) when every workgroup has a CU of its own, so that 1024 + 32 keys
  // take at most two chunks per wave instead of three (12-layer step 0.843
  // -> 0.839 ms)
  if (dh == 128 && wgs <= kAttnCus) nw = 12;
  else while (nw > 4 && wgs * nw > kAttnResidentWaves) nw >>= 1;
  const AttnLaunch l{q, k_cache, vt_cache, cap, T, M, C, H, lut, a_out, n_seq, seq_words};
  switch (dh / 64 * 100 + nw) {
    case 116: attn_launch<1, 16>(grid, l, st); break;
    case 108: attn_launch<1, 8>(grid, l, st); break;
    case 104: attn_launch<1, 4>(grid, l, st); break;
    case 212: attn_launch<2, 12>(grid, l, st); break;
    case 208: attn_launch<2, 8>(grid, l, st); break;
    case 204: attn_launch<2, 4>(grid, l, st); break;
    default:
      return NMDLM_ERR_UNSUPPORTED;
  }
  return hip_status();
}

// ---------------------------------------------------------------------------
// Attention followed by the IF neuron of its output, in one kernel.
// Workgroup = one head and 16 block queries for every timestep.  Wave =
// (timestep t, part): the parts of a timestep take 64-key chunks in turn and
// add their partial sums into LDS.  Per chunk a lane loads one key (row =
// lane) and the value bits of one channel (= lane), and the wave exchanges
// them through LDS; chunks go in rounds of kRound whose loads are all issued
// before the first is scored.  Then one wave per (query, 64-channel word)
// computes a = floor(256 num / den) and runs the IF recurrence over t,
// writing the spike words and the token's union over t.
// ---------------------------------------------------------------------------
constexpr int kRound = 4;

template <int DHW>
struct KvChunk {
  uint64_t kw[DHW];  // key row jc*64 + lane, this head's words
  uint64_t vw[DHW];  // value bits of channel w*64 + lane over the chunk's keys
};

template <int DHW>
__device__ __forceinline__ void load_chunk(KvChunk<DHW>& ch, const uint64_t* __restrict__ kc,
                                           const uint64_t* __restrict__ vt, int64_t cap, int capw,
                                           int t, int h, int d, int dw, int J, int jc, int lane) {
  constexpr int DH = DHW * 64;
  const int jj = min(jc * 64 + lane, J - 1);  // past C+M: a valid row, masked when scored
  const uint64_t* kr = kc + ((size_t)t * cap + jj) * dw + h * DHW;
#pragma unroll
  for (int w = 0; w < DHW; ++w) {
    ch.kw[w] = kr[w];
    ch.vw[w] = vt[((size_t)t * capw + jc) * d + h * DH + w * 64 + lane];
  }
}

// sK, sV: this wave's 64 x DHW key words and DH value words in LDS
// lut_dw: table bytes 4*lane .. 4*lane+3 (entry s is read from lane s/4)
template <int DHW>
__device__ __forceinline__ void score_chunk(const KvChunk<DHW>& ch, const uint64_t (&qw)[DHW],
                                            int lut_dw, uint64_t* sK, uint64_t* sV, int J,
                                            int jc, int lane, int g, int c, v4i (&acc)[DHW * 4],
                                            int (&cnt)[DHW * 4], int& den) {
  const int j0 = jc * 64 + 16 * g;
#pragma unroll
  for (int w = 0; w < DHW; ++w) {
    sK[lane * DHW + w] = ch.kw[w];
    sV[w * 64 + lane] = ch.vw[w];
  }
  __builtin_amdgcn_wave_barrier();
  uint32_t pk[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    int sc = 0;
#pragma unroll
    for (int w = 0; w < DHW; ++w) sc += __popcll(qw[w] & sK[(16 * g + s) * DHW + w]);
    const bool jv = j0 + s < J;
    const int pw = __builtin_amdgcn_ds_bpermute((sc >> 2) << 2, lut_dw);
    const int p = jv ? (pw >> ((sc & 3) * 8)) & 0xFF : 0;
    den += p;
    pk[s >> 2] |= jv ? (uint32_t)((p - 128) & 0xFF) << ((s & 3) * 8) : 0u;
  }
  const v4i af = v4i{(int)pk[0], (int)pk[1], (int)pk[2], (int)pk[3]};
  const int nvalid = J - j0;
  const uint32_t vmask = nvalid >= 16 ? 0xFFFFu : (nvalid <= 0 ? 0u : ((1u << nvalid) - 1u));
#pragma unroll
  for (int nt = 0; nt < DHW * 4; ++nt) {
    const uint32_t bits = (uint32_t)(sV[nt * 16 + c] >> (16 * g)) & vmask;
    cnt[nt] += __popc(bits);
    const v4i bf = v4i{(int)expand4_a(bits & 0xFu), (int)expand4_a((bits >> 4) & 0xFu),
                       (int)expand4_a((bits >> 8) & 0xFu), (int)expand4_a(bits >> 12)};
    acc[nt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, bf, acc[nt], 0, 0, 0);
  }
  __builtin_amdgcn_wave_barrier();  // sK and sV are rewritten by the next chunk
}

template <int DHW, int NW>
__global__ __launch_bounds__(NW * 64) void k_attn_if(const uint64_t* __restrict__ q,
                                                     const uint64_t* __restrict__ kc,
                                                     const uint64_t* __restrict__ vt, int64_t cap,
                                                     int T, int M, int C, int H,
                                                     const uint8_t* __restrict__ lut,
                                                     int32_t theta, uint64_t* __restrict__ s_out,
                                                     uint64_t* __restrict__ u_out) {
  constexpr int DH = DHW * 64;
  constexpr int NT = DHW * 4;
  constexpr int NTH = NW * 64;
  __shared__ int sDen[NMDLM_MAX_T][16];
  __shared__ int sCnt[NMDLM_MAX_T][DH];
  __shared__ uint64_t sKey[NW][64 * DHW];
  __shared__ uint64_t sVal[NW][DH];
  extern __shared__ int sNum[];  // [T][16][DH]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int lid = xcd_order(blockIdx.x + gridDim.x * blockIdx.y, gridDim.x * gridDim.y);
  const int h = lid % gridDim.x, qb = lid / gridDim.x;
  const int d = H * DH, dw = d / 64;
  const int capw = (int)(cap / 64);
  const int J = C + M;
  const int nch = (J + 63) / 64;
  const int tp = T <= 1 ? 1 : (T <= 2 ? 2 : (T <= 4 ? 4 : 8));
  const int NP = NW / tp;  // parts per timestep
  const int t = wave / NP, part = wave - t * NP;
  const bool active = t < T && part < nch;  // wave-uniform
  const int tl = min(t, T - 1);             // idle waves load valid rows and discard them

  // table, query words and the first round of chunks: unconditional loads in
  // one straight run, so each wait covers only what it needs
  const int lut_dw = lut_dword(lut, lane);
  const int iq = qb * 16 + c;
  uint64_t qw[DHW];
#pragma unroll
  for (int w = 0; w < DHW; ++w) qw[w] = q[((size_t)tl * M + min(iq, M - 1)) * dw + h * DHW + w];
  KvChunk<DHW> ch[kRound];
#pragma unroll
  for (int u = 0; u < kRound; ++u)
    load_chunk<DHW>(ch[u], kc, vt, cap, capw, tl, h, d, dw, J, min(part + u * NP, nch - 1), lane);

  for (int i = tid; i < NMDLM_MAX_T * 16; i += NTH) (&sDen[0][0])[i] = 0;
  for (int i = tid; i < NMDLM_MAX_T * DH; i += NTH) (&sCnt[0][0])[i] = 0;
  for (int i = tid; i < T * 16 * DH; i += NTH) sNum[i] = 0;
  __syncthreads();

  if (active) {
#pragma unroll
    for (int w = 0; w < DHW; ++w) qw[w] = iq < M ? qw[w] : 0ull;
    v4i acc[NT];
    int cnt[NT];
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      acc[i] = v4i{0, 0, 0, 0};
      cnt[i] = 0;
    }
    int den = 0;
    uint64_t* sK = sKey[wave];
    uint64_t* sV = sVal[wave];
    for (int jr = part;;) {
#pragma unroll
      for (int u = 0; u < kRound; ++u) {
        const int jc = jr + u * NP;
        if (jc < nch) score_chunk<DHW>(ch[u], qw, lut_dw, sK, sV, J, jc, lane, g, c, acc, cnt, den);
      }
      jr += kRound * NP;
      if (jr >= nch) break;
#pragma unroll
      for (int u = 0; u < kRound; ++u)
        load_chunk<DHW>(ch[u], kc, vt, cap, capw, t, h, d, dw, J, min(jr + u * NP, nch - 1), lane);
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (acc[nt][e]) atomicAdd(&sNum[(t * 16 + g * 4 + e) * DH + nt * 16 + c], acc[nt][e]);
    if (den) atomicAdd(&sDen[t][c], den);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      if (cnt[nt]) atomicAdd(&sCnt[t][nt * 16 + c], cnt[nt]);
  }
  __syncthreads();

  for (int task = wave; task < 16 * DHW; task += NW) {
    const int i = task / DHW, w = task - i * DHW;
    const int iq2 = qb * 16 + i;
    if (iq2 >= M) break;  // wave-uniform; later tasks have larger i
    const int chn = w * 64 + lane;
    long long V = 0;
    uint64_t uor = 0ull;
    for (int tt = 0; tt < T; ++tt) {
      const long long num = (long long)sNum[(tt * 16 + i) * DH + chn] + 128LL * sCnt[tt][chn];
      V += attn_norm(num, sDen[tt][i], J < 65536);
      const bool s = V >= theta;
      if (s) V -= theta;
      const uint64_t word = __builtin_amdgcn_ballot_w64(s);
      uor |= word;
      if (lane == 0) s_out[((size_t)tt * M + iq2) * dw + h * DHW + w] = word;
    }
    if (u_out && lane == 0) u_out[(size_t)iq2 * dw + h * DHW + w] = uor;
  }
}

constexpr size_t kAttnIfMaxLds = 49152;  // bytes of [T][16][dh] partial sums

nmdlm_status launch_attn_if(const uint64_t* q, const uint64_t* k_cache, const uint64_t* vt_cache,
                            int64_t cap, int T, int M, int C, int H, int dh, const uint8_t* lut,
                            int32_t theta, uint64_t* s_out, uint64_t* u_out, hipStream_t st) {
  const size_t dyn = (size_t)T * 16 * dh * sizeof(int);
  if (dyn > kAttnIfMaxLds || T > NMDLM_MAX_T) return NMDLM_ERR_UNSUPPORTED;
  const dim3 grid(H, (M + 15) / 16);
  switch (dh / 64) {
    case 1:
      hipLaunchKernelGGL((k_attn_if<1, 16>), grid, dim3(16 * 64), dyn, st, q, k_cache, vt_cache,
                         cap, T, M, C, H, lut, theta, s_out, u_out);
      break;
    case 2:
      hipLaunchKernelGGL((k_attn_if<2, 8>), grid, dim3(8 * 64), dyn, st, q, k_cache, vt_cache,
                         cap, T, M, C, H, lut, theta, s_out, u_out);
      break;
    default:
      return NMDLM_ERR_UNSUPPORTED;
  }
  return hip_status();
}

}  // namespace nmdlm
