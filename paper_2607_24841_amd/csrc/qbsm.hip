// Quantised-weight x binary-spike product with block-union row skipping.
//
// Sec. IV-A: Y = X W over the B*T spike rows of a block; by assumption (ii) a
// weight row is read only if its input neuron spikes somewhere in the block.
// Three kernels per product:
//   k_union_scan  OR of all T*M spike rows -> ascending active-row list
//   k_compact     spike bits gathered onto the active rows, k-step major
//   k_qbsm        int8 MFMA over (T*M) x K_active x N with a fused epilogue
//                 (currents, integrate-and-fire, table + IF, or head logits)
#include "common.h"

namespace nmdlm {

constexpr int kPrepThreads = 1024;
constexpr int kMaxWords = NMDLM_MAX_K / 64;
constexpr int kCompactRows = 64;

// ---------------------------------------------------------------------------
// Block union and the active-row list.  One workgroup: the inputs of a block
// step are at most a few hundred rows of <= 1024 words.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kPrepThreads) void k_union_scan(
    const uint64_t* __restrict__ S, int R, int Kw, int K, int dense, uint32_t ldw, int N,
    uint32_t* __restrict__ act_off, int32_t* __restrict__ act_idx, int32_t* __restrict__ kact,
    nmdlm_qbsm_stats* __restrict__ stats, int32_t* __restrict__ counters, int n_counters) {
  __shared__ unsigned long long sU[kMaxWords];
  __shared__ int sWaveSum[kPrepThreads / kWave];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;

  for (int i = tid; i < n_counters; i += kPrepThreads) counters[i] = 0;
  for (int w = tid; w < Kw; w += kPrepThreads) sU[w] = dense ? ~0ull : 0ull;
  __syncthreads();
  if (!dense) {
    const int rg = kPrepThreads / Kw;  // row groups (Kw <= 1024)
    const int w = tid % Kw, r0 = tid / Kw;
    if (r0 < rg) {
      unsigned long long acc = 0;
      for (int r = r0; r < R; r += rg) acc |= S[(size_t)r * Kw + w];
      if (acc) atomicOr(&sU[w], acc);
    }
  }
  __syncthreads();
  if (tid == 0 && (K & 63)) sU[Kw - 1] &= (1ull << (K & 63)) - 1ull;
  __syncthreads();

  // exclusive prefix sum of the per-word popcounts (one word per thread)
  const int cnt = tid < Kw ? __popcll(sU[tid]) : 0;
  int incl = cnt;
  for (int o = 1; o < kWave; o <<= 1) {
    const int v = __shfl_up(incl, o);
    if (lane >= o) incl += v;
  }
  if (lane == kWave - 1) sWaveSum[wave] = incl;
  __syncthreads();
  int before = 0, total = 0;
  for (int i = 0; i < kPrepThreads / kWave; ++i) {
    if (i < wave) before += sWaveSum[i];
    total += sWaveSum[i];
  }
  if (tid < Kw) {
    unsigned long long u = sU[tid];
    int o = before + incl - cnt;
    while (u) {
      const int b = __ffsll((unsigned long long)u) - 1;
      const int k = tid * 64 + b;
      act_off[o] = (uint32_t)k * ldw;
      act_idx[o] = k;
      ++o;
      u &= u - 1ull;
    }
  }
  // pad the list to whole k-steps with row 0 (its spike bits are zero)
  const int padded = (total + 63) & ~63;
  for (int i = total + tid; i < padded; i += kPrepThreads) {
    act_off[i] = 0u;
    act_idx[i] = -1;
  }
  if (tid == 0) {
    *kact = total;
    if (stats) {
      stats->k_total = K;
      stats->k_active = total;
      stats->n = N;
      stats->weight_bytes = (int64_t)total * (int64_t)N;
    }
  }
}

// ---------------------------------------------------------------------------
// Compaction: sc[j][r] bit i = S[r][act[64 j + i]].  Block (j, row range).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_compact(const uint64_t* __restrict__ S, int R, int Kw,
                                                 const int32_t* __restrict__ act_idx,
                                                 const int32_t* __restrict__ kact,
                                                 uint64_t* __restrict__ sc) {
  const int j = blockIdx.x;
  const int ka = *kact;
  if (j * 64 >= ka) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = j * 64 + lane;
  const int idx = i < ka ? act_idx[i] : -1;
  const int wi = idx >= 0 ? (idx >> 6) : 0;
  const int bi = idx & 63;
  const int r0 = blockIdx.y * kCompactRows;
  const int r1 = min(R, r0 + kCompactRows);
  for (int r = r0 + wave; r < r1; r += 4) {
    const uint64_t word = S[(size_t)r * Kw + wi];
    const bool bit = idx >= 0 && ((word >> bi) & 1ull);
    const uint64_t m = __builtin_amdgcn_ballot_w64(bit);
    if (lane == 0) sc[(size_t)j * R + r] = m;
  }
}

// ---------------------------------------------------------------------------
// The product.
//
// Workgroup = 4 waves, tile = (16*RT rows of the block) x (64 columns).  The
// waves take k-steps (64 active rows each) in turn and reduce in LDS.
// Per k-step a lane (g = lane/16, c = lane%16) loads, for the 16 active rows
// k_{g,0..15}, the dword W[k][n0+4c .. n0+4c+3]; an in-register 4x4 byte
// transpose turns these into four MFMA B operands whose column c stands for
// weight column n0 + 4c + v (v = 0..3).  The A operand (16 spike rows x 64
// active rows) is expanded from the compacted bits.  v_mfma_i32_16x16x64_i8
// accumulates exactly in int32; output element (lane, e) is row 4g + e.
// Block rows are ordered t-major: local row r -> (t = r / Mb, token r % Mb).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t expand4(uint32_t nib) {
  // 4 bits -> 4 bytes of 0/1 (bit i -> byte i); the shifted copies of the
  // nibble do not overlap, so the multiply adds no carries.
  return (nib * 0x00204081u) & 0x01010101u;
}

__device__ __forceinline__ int phys_col(int col) { return (col & 3) * 16 + (col >> 2); }

template <int RT>
__global__ __launch_bounds__(256) void k_qbsm(QbsmArgs a) {
  constexpr int ROWS = RT * 16;
  __shared__ int sTile[ROWS * kTileLd];
  __shared__ uint32_t sOff[kChunkSteps * 64];
  __shared__ int sLast;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  const int x = blockIdx.x, y = blockIdx.y, z = blockIdx.z;
  const int n0 = x * 64;
  const int R = a.T * a.M;

  for (int i = tid; i < ROWS * kTileLd; i += 256) sTile[i] = 0;

  const int ka = *a.kact;
  const int KS = (ka + 63) >> 6;
  const int ks0 = (int)(((long long)KS * z) / a.P);
  const int ks1 = (int)(((long long)KS * (z + 1)) / a.P);

  int rowq[RT];
#pragma unroll
  for (int q = 0; q < RT; ++q) {
    const int jr = q * 16 + c;
    const int t = jr / a.Mb, ml = jr - t * a.Mb, m = y * a.Mb + ml;
    rowq[q] = (t < a.T && m < a.M) ? t * a.M + m : -1;
  }
  const uint32_t colb = (n0 + 4 * c < a.N) ? (uint32_t)(n0 + 4 * c) : (uint32_t)n0;
  const char* Wb = reinterpret_cast<const char*>(a.W) + colb;
  const uint32_t* sc32 = reinterpret_cast<const uint32_t*>(a.sc);

  v4i acc[RT][4];
#pragma unroll
  for (int q = 0; q < RT; ++q)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[q][v] = v4i{0, 0, 0, 0};

  for (int cs = ks0; cs < ks1; cs += kChunkSteps) {
    const int ce = min(cs + kChunkSteps, ks1);
    __syncthreads();
    for (int i = tid; i < (ce - cs) * 64; i += 256) sOff[i] = a.act_off[(size_t)cs * 64 + i];
    __syncthreads();
    for (int j = cs + wave; j < ce; j += 4) {
      const uint4* po = reinterpret_cast<const uint4*>(sOff + (j - cs) * 64 + 16 * g);
      uint32_t off[16];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint4 o = po[u];
        off[4 * u + 0] = o.x;
        off[4 * u + 1] = o.y;
        off[4 * u + 2] = o.z;
        off[4 * u + 3] = o.w;
      }
      uint32_t xw[16];
#pragma unroll
      for (int s = 0; s < 16; ++s) xw[s] = *reinterpret_cast<const uint32_t*>(Wb + off[s]);

      uint32_t bits[RT];
#pragma unroll
      for (int q = 0; q < RT; ++q)
        bits[q] = rowq[q] >= 0
                      ? (sc32[((size_t)j * R + rowq[q]) * 2 + (g >> 1)] >> ((g & 1) * 16)) & 0xFFFFu
                      : 0u;

      v4i b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t x0 = xw[4 * u], x1 = xw[4 * u + 1], x2 = xw[4 * u + 2], x3 = xw[4 * u + 3];
        const uint32_t t0 = __builtin_amdgcn_perm(x1, x0, 0x05010400u);  // x0[0] x1[0] x0[1] x1[1]
        const uint32_t t1 = __builtin_amdgcn_perm(x1, x0, 0x07030602u);  // x0[2] x1[2] x0[3] x1[3]
        const uint32_t t2 = __builtin_amdgcn_perm(x3, x2, 0x05010400u);
        const uint32_t t3 = __builtin_amdgcn_perm(x3, x2, 0x07030602u);
        b[0][u] = (int)__builtin_amdgcn_perm(t2, t0, 0x05040100u);     // column 4c+0 of rows 4u..4u+3
        b[1][u] = (int)__builtin_amdgcn_perm(t2, t0, 0x07060302u);
        b[2][u] = (int)__builtin_amdgcn_perm(t3, t1, 0x05040100u);
        b[3][u] = (int)__builtin_amdgcn_perm(t3, t1, 0x07060302u);
      }
#pragma unroll
      for (int q = 0; q < RT; ++q) {
        const uint32_t bq = bits[q];
        const v4i af = v4i{(int)expand4(bq & 0xFu), (int)expand4((bq >> 4) & 0xFu),
                           (int)expand4((bq >> 8) & 0xFu), (int)expand4(bq >> 12)};
#pragma unroll
        for (int v = 0; v < 4; ++v)
          acc[q][v] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, b[v], acc[q][v], 0, 0, 0);
      }
    }
  }

  __syncthreads();
#pragma unroll
  for (int q = 0; q < RT; ++q)
#pragma unroll
    for (int v = 0; v < 4; ++v)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int val = acc[q][v][e];
        if (val) atomicAdd(&sTile[(q * 16 + g * 4 + e) * kTileLd + v * 16 + c], val);
      }
  __syncthreads();

  if (a.P > 1) {
    // K split across workgroups: every split stores its whole tile (zeros
    // included) into its own slot; the last workgroup to arrive sums the
    // slots in split order.  No slot has to be zero beforehand.
    const size_t tile_id = (size_t)y * gridDim.x + x;
    const size_t slot_elems = (size_t)ROWS * 64;
    const size_t n_tiles = (size_t)gridDim.x * gridDim.y;
    int* mine = a.part + ((size_t)z * n_tiles + tile_id) * slot_elems;
    for (int i = tid; i < ROWS * 64; i += 256)
      __hip_atomic_store(&mine[i], sTile[(i >> 6) * kTileLd + phys_col(i & 63)], __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    __threadfence();
    __syncthreads();
    if (tid == 0) sLast = (atomicAdd(&a.counters[tile_id], 1) == a.P - 1) ? 1 : 0;
    __syncthreads();
    if (!sLast) return;
    __threadfence();
    for (int i = tid; i < ROWS * 64; i += 256) {
      int v = 0;
      for (int p = 0; p < a.P; ++p)
        v += __hip_atomic_load(a.part + ((size_t)p * n_tiles + tile_id) * slot_elems + i,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      sTile[(i >> 6) * kTileLd + phys_col(i & 63)] = v;
    }
    __syncthreads();
  }

  // ------------------------------------------------------------------ epilogue
  const int col = lane, n = n0 + col;
  const bool nv = n < a.N;
  const int pc = phys_col(col);
  if (a.mode == EPI_HEAD) {
    const float sc = nv ? a.scale[n] : 0.f;
    for (int ml = wave; ml < a.Mb; ml += 4) {
      const int m = y * a.Mb + ml;
      if (m >= a.M) break;
      int s = 0;
      for (int t = 0; t < a.T; ++t) s += sTile[(t * a.Mb + ml) * kTileLd + pc];
      if (nv) a.logits[(size_t)m * a.N + n] = (float)s * sc;
    }
    return;
  }

  const int segi = (a.mode == EPI_CUR) ? 0 : n0 / a.seg_w;
  const SpikeSeg seg = a.seg[segi];
  const int wseg = (n0 - segi * a.seg_w) >> 6;
  const int bias_n = (a.bias && nv) ? a.bias[n] : 0;
  const int theta = a.theta_vec ? (nv ? a.theta_vec[n] : 1) : seg.theta;
  const bool spikes = a.mode != EPI_CUR;
  const bool tr = spikes && seg.transposed;
  const int wbase = tr ? ((seg.pos0 + y * a.Mb) >> 6) : 0;
  uint64_t tb0[NMDLM_MAX_T], tb1[NMDLM_MAX_T];
#pragma unroll
  for (int t = 0; t < NMDLM_MAX_T; ++t) tb0[t] = tb1[t] = 0ull;
  uint64_t tm0 = 0ull, tm1 = 0ull;

  for (int ml = wave; ml < a.Mb; ml += 4) {
    const int m = y * a.Mb + ml;
    if (m >= a.M) break;
    int V = 0;
    const int pos = seg.pos0 + m;
    const int rel = (pos >> 6) - wbase;
    const uint64_t pbit = 1ull << (pos & 63);
    if (tr) {
      if (rel == 0) tm0 |= pbit;
      else tm1 |= pbit;
    }
#pragma unroll
    for (int t = 0; t < NMDLM_MAX_T; ++t) {
      if (t < a.T) {
        int I = sTile[(t * a.Mb + ml) * kTileLd + pc] + bias_n;
        if (a.cur_out && nv) a.cur_out[((size_t)t * a.M + m) * a.N + n] = I;
        if (spikes) {
          if (a.mode == EPI_QNL_IF) {
            int qv = I >> a.lut_shift;
            qv = min(127, max(-128, qv));
            I = (int)(int8_t)a.lut[qv & 0xFF];
          }
          if (a.resid && ((a.resid[t * a.rld_t + (int64_t)m * a.rld_m + x] >> col) & 1ull)) I += theta;
          V += I;
          const bool s = nv && V >= theta;
          if (s) V -= theta;
          if (!tr) {
            const uint64_t word = __builtin_amdgcn_ballot_w64(s);
            if (lane == 0) seg.ptr[t * seg.ld_t + (int64_t)m * seg.ld_m + wseg] = word;
          } else if (s) {
            if (rel == 0) tb0[t] |= pbit;
            else tb1[t] |= pbit;
          }
        }
      }
    }
  }
  if (tr && nv) {
    // channel-major cache: clear this wave's token bits, then set the spikes
    const int ch = n - segi * a.seg_w;
#pragma unroll
    for (int t = 0; t < NMDLM_MAX_T; ++t) {
      if (t < a.T) {
        unsigned long long* row = reinterpret_cast<unsigned long long*>(
            seg.ptr + t * seg.ld_t + (int64_t)ch * seg.ld_m + wbase);
        if (tm0) {
          atomicAnd(row, ~tm0);
          if (tb0[t]) atomicOr(row, tb0[t]);
        }
        if (tm1) {
          atomicAnd(row + 1, ~tm1);
          if (tb1[t]) atomicOr(row + 1, tb1[t]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
static int pick_rt(int R) {
  if (R <= 16) return 1;
  if (R <= 32) return 2;
  if (R <= 64) return 4;
  return 8;
}

QbsmLimits qbsm_limits_single(int T, int M, int K, int N) {
  QbsmLimits L;
  L.Kmax = K;
  L.Rmax = T * M;
  L.Nmax = N;
  L.tiles_max = ((N + 63) / 64) * M;
  L.split_rows = (T * M <= kSplitMaxRows) ? T * M : 0;
  L.split_N = N;
  return L;
}

void carve_qbsm_scratch(Carver& cv, const QbsmLimits& L, QbsmScratch* s) {
  const size_t kpad = align_up((size_t)L.Kmax, 64);
  s->act_off = cv.take<uint32_t>(kpad);
  s->act_idx = cv.take<int32_t>(kpad);
  s->kact = cv.take<int32_t>(1);
  s->sc = cv.take<uint64_t>((size_t)((L.Kmax + 63) / 64) * (size_t)L.Rmax);
  // split slots: up to kSplitSlots tiles of (row tiles x 64 columns) per column
  size_t rows_cap = 0;
  if (L.split_rows > 0) rows_cap = L.split_rows <= 128 ? 16 * (size_t)pick_rt(L.split_rows) : 256;
  s->part_elems = (size_t)kSplitSlots * rows_cap * align_up((size_t)L.split_N, 64);
  s->part = s->part_elems ? cv.take<int32_t>(s->part_elems) : nullptr;
  s->n_counters = (size_t)L.tiles_max;
  s->counters = cv.take<int32_t>(s->n_counters);
}

nmdlm_status launch_qbsm(const QbsmCall& c, const QbsmScratch& scr, hipStream_t st) {
  const int R = c.T * c.M;
  const int Kw = (c.K + 63) / 64;
  const int dense = (c.flags & NMDLM_FORCE_DENSE) ? 1 : 0;
  bool has_tr = false;
  if (c.mode == EPI_IF || c.mode == EPI_QNL_IF)
    for (int i = 0; i < c.nseg; ++i) has_tr = has_tr || c.seg[i].transposed;

  int RT = (int)((c.flags >> NMDLM_ROWTILE_SHIFT) & 0xFu);
  if (RT != 1 && RT != 2 && RT != 4 && RT != 8) RT = pick_rt(R);
  while (RT > 1 && 16 * RT / 2 >= R && 16 * RT / 2 >= c.T) RT >>= 1;  // no empty tiles
  while (has_tr && RT > 1 && (16 * RT) / c.T > 64) RT >>= 1;
  if (16 * RT < c.T) return NMDLM_ERR_UNSUPPORTED;
  const int Mb = (16 * RT) / c.T;
  const int gx = (c.N + 63) / 64, gy = (c.M + Mb - 1) / Mb;
  const int tiles = gx * gy;
  if ((size_t)tiles > scr.n_counters) return NMDLM_ERR_WORKSPACE;

  int P = (int)((c.flags >> NMDLM_SPLIT_SHIFT) & 0xFFu);
  if (P == 0) {
    P = 1;
    if (tiles < 240) P = (480 + tiles - 1) / tiles;
    P = std::min(P, std::max(1, Kw / 4));
  }
  P = std::max(1, std::min(P, Kw));
  const size_t slot_elems = (size_t)16 * RT * 64 * (size_t)tiles;  // one tile slot per split
  if (P > 1) {
    const size_t cap = scr.part ? scr.part_elems / slot_elems : 0;
    P = (int)std::min<size_t>((size_t)P, cap);
    if (P < 2) P = 1;
  }

  hipLaunchKernelGGL(k_union_scan, dim3(1), dim3(kPrepThreads), 0, st, c.s_in, R, Kw, c.K, dense,
                     (uint32_t)c.ldw, c.N, scr.act_off, scr.act_idx, scr.kact, c.stats,
                     scr.counters, tiles);
  hipLaunchKernelGGL(k_compact, dim3(Kw, (R + kCompactRows - 1) / kCompactRows), dim3(256), 0, st,
                     c.s_in, R, Kw, scr.act_idx, scr.kact, scr.sc);

  QbsmArgs a;
  a.sc = scr.sc;
  a.act_off = scr.act_off;
  a.kact = scr.kact;
  a.W = c.W;
  a.ldw = c.ldw;
  a.K = c.K;
  a.N = c.N;
  a.T = c.T;
  a.M = c.M;
  a.Mb = Mb;
  a.P = P;
  a.mode = c.mode;
  a.bias = c.bias;
  a.cur_out = c.cur_out;
  a.theta_vec = c.theta_vec;
  a.nseg = c.nseg;
  a.seg_w = c.seg_w;
  for (int i = 0; i < kMaxSeg; ++i) a.seg[i] = c.seg[i];
  a.resid = c.resid;
  a.rld_t = c.rld_t;
  a.rld_m = c.rld_m;
  a.lut = c.lut;
  a.lut_shift = c.lut_shift;
  a.logits = c.logits;
  a.scale = c.scale;
  a.part = scr.part;
  a.counters = scr.counters;

  const dim3 grid(gx, gy, P);
  switch (RT) {
    case 1: hipLaunchKernelGGL(k_qbsm<1>, grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL(k_qbsm<2>, grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL(k_qbsm<4>, grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL(k_qbsm<8>, grid, dim3(256), 0, st, a); break;
  }
  return hip_status();
}

}  // namespace nmdlm
