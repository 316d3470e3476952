// Quantised-weight x binary-spike product with block-union row skipping.
//
// Sec. IV-A: Y = X W over the B*T spike rows of a block; by assumption (ii) a
// weight row is read only if its input neuron spikes somewhere in the block.
// One kernel per product (k_qbsm_fused): block union from the producer's
// partial unions (or the spikes), active-row list and spike compaction in
// LDS, then int8 MFMA over (T*M) x K_active x N with a fused epilogue
// (currents, integrate-and-fire, table + IF, or head logits) that also emits
// the partial union of its output spikes.  Blocks too large for LDS (long
// prefills) take a prep pass (k_union, k_prep) and k_qbsm_list.
#include <hip/hip_ext.h>

#include "common.h"

namespace nmdlm {

constexpr int kMaxWords = NMDLM_MAX_K / 64;
constexpr int kPrepRows = 64;      // rows compacted per prep workgroup
constexpr int kUnionDirect = 8192; // words of S a prep workgroup ORs itself

// ---------------------------------------------------------------------------
// Column OR of a large spike block (used when R*Kw is too large for every
// prep workgroup to recompute it): U[w] = OR_r S[r][w].  Block w.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_union(const uint64_t* __restrict__ S, int R, int Kw,
                                               uint64_t* __restrict__ U) {
  __shared__ unsigned long long sAcc[256];
  const int w = blockIdx.x, tid = threadIdx.x;
  unsigned long long acc = 0;
  for (int r = tid; r < R; r += 256) acc |= S[(size_t)r * Kw + w];
  sAcc[tid] = acc;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) sAcc[tid] |= sAcc[tid + s];
    __syncthreads();
  }
  if (tid == 0) U[w] = sAcc[0];
}

// Position of the r-th (0-based) set bit of u (r < popcount(u)).
__device__ __forceinline__ int select_bit(unsigned long long u, int r) {
  int pos = 0;
  uint32_t v = (uint32_t)u;
  int c = __popc(v);
  if (r >= c) {
    r -= c;
    pos = 32;
    v = (uint32_t)(u >> 32);
  }
  c = __popc(v & 0xFFFFu);
  if (r >= c) { r -= c; pos += 16; v >>= 16; }
  c = __popc(v & 0xFFu);
  if (r >= c) { r -= c; pos += 8; v >>= 8; }
  c = __popc(v & 0xFu);
  if (r >= c) { r -= c; pos += 4; v >>= 4; }
  c = __popc(v & 0x3u);
  if (r >= c) { r -= c; pos += 2; v >>= 2; }
  if (r >= (int)(v & 1u)) pos += 1;
  return pos;
}

struct PrepArgs {
  const uint64_t* S;       // [R][Kw] spikes
  int R, Kw, K;
  const uint64_t* upart;   // [nparts][Kw] partial unions, or null (OR S directly)
  int nparts;
  int dense;               // every row active
  uint32_t ldw;
  int N;
  uint32_t* act_off;       // [round_up(K,64)]
  int32_t* act_idx;
  int32_t* kact;
  nmdlm_qbsm_stats* stats;
  int32_t* counters;
  int n_counters;
  uint64_t* sc;            // [Kw][R]
};

// ---------------------------------------------------------------------------
// Block union, active-row list and compaction in one pass.  Block (j, y):
// every workgroup forms the union (from producer partial unions when given)
// and its prefix popcounts, locates active rows 64j..64j+63 by binary search
// over the prefix sums, and gathers the spike bits of rows [64y, 64y+64) onto
// them: sc[j][r] bit i = S[r][act[64j + i]].
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_prep(PrepArgs p) {
  __shared__ unsigned long long sU[kMaxWords];
  __shared__ int sP[kMaxWords + 1];
  __shared__ int sWave[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Kw = p.Kw;

  if (p.dense) {
    for (int w = tid; w < Kw; w += 256) sU[w] = ~0ull;
  } else if (p.upart) {
    for (int w = tid; w < Kw; w += 256) {
      unsigned long long acc = 0;
      for (int q = 0; q < p.nparts; ++q) acc |= p.upart[(size_t)q * Kw + w];
      sU[w] = acc;
    }
  } else {
    for (int w = tid; w < Kw; w += 256) sU[w] = 0ull;
    __syncthreads();
    if (Kw <= 256) {
      const int rg = 256 / Kw, w = tid % Kw, r0 = tid / Kw;
      if (r0 < rg) {
        unsigned long long acc = 0;
        for (int r = r0; r < p.R; r += rg) acc |= p.S[(size_t)r * Kw + w];
        if (acc) atomicOr(&sU[w], acc);
      }
    } else {
      for (int w = tid; w < Kw; w += 256) {
        unsigned long long acc = 0;
        for (int r = 0; r < p.R; ++r) acc |= p.S[(size_t)r * Kw + w];
        sU[w] = acc;
      }
    }
  }
  __syncthreads();
  if (tid == 0 && (p.K & 63)) sU[Kw - 1] &= (1ull << (p.K & 63)) - 1ull;
  __syncthreads();

  // exclusive prefix sums of popcounts: thread t owns words 4t..4t+3
  int cw[4], s = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int w = 4 * tid + i;
    cw[i] = w < Kw ? __popcll(sU[w]) : 0;
    s += cw[i];
  }
  int incl = s;
  for (int o = 1; o < kWave; o <<= 1) {
    const int v = __shfl_up(incl, o);
    if (lane >= o) incl += v;
  }
  if (lane == kWave - 1) sWave[wave] = incl;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (i < wave) before += sWave[i];
    total += sWave[i];
  }
  int run = before + incl - s;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int w = 4 * tid + i;
    if (w < Kw) sP[w] = run;
    run += cw[i];
  }
  if (tid == 0) sP[Kw] = total;
  __syncthreads();

  const int j = blockIdx.x, y = blockIdx.y;
  if (j == 0 && y == 0) {
    for (int i = tid; i < p.n_counters; i += 256) p.counters[i] = 0;
    if (tid == 0) {
      *p.kact = total;
      if (p.stats) {
        p.stats->k_total = p.K;
        p.stats->k_active = total;
        p.stats->n = p.N;
        p.stats->weight_bytes = (int64_t)total * (int64_t)p.N;
      }
    }
  }
  if (j * 64 >= total) return;

  const int i = j * 64 + lane;
  const bool valid = i < total;
  int k = 0;
  if (valid) {
    int lo = 0, hi = Kw - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (sP[mid] <= i) lo = mid;
      else hi = mid - 1;
    }
    k = lo * 64 + select_bit(sU[lo], i - sP[lo]);
  }
  if (y == 0 && wave == 0) {
    p.act_off[i] = valid ? (uint32_t)k * p.ldw : 0u;
    p.act_idx[i] = valid ? k : -1;
  }
  const int wi = k >> 6, bi = k & 63;
  const int r1 = min(p.R, (y + 1) * kPrepRows);
  for (int r = y * kPrepRows + wave; r < r1; r += 4) {
    const uint64_t word = p.S[(size_t)r * Kw + wi];
    const bool bit = valid && ((word >> bi) & 1ull);
    const uint64_t m = __builtin_amdgcn_ballot_w64(bit);
    if (lane == 0) p.sc[(size_t)j * p.R + r] = m;
  }
}

// ---------------------------------------------------------------------------
// The product.
//
// Workgroup = NW waves, tile = (16*RT rows of the block) x (64 columns).
// Block rows are ordered t-major inside a row block: local row r ->
// (t = r / Mb, token r % Mb), so a token's T currents land in one tile.
// The waves take groups of kGroup k-steps (64 active rows each) and reduce in
// LDS.  Per k-step a lane (g = lane/16, c = lane%16) loads, for the 16 active
// rows k_{g,0..15}, the dword W[k][n0+4c .. n0+4c+3]; an in-register 4x4 byte
// transpose turns them into four MFMA B operands whose column c stands for
// weight column n0 + 4c + v (v = 0..3).  The A operand (16 rows x 64 active
// rows of 0/1 bytes) is expanded from 16 compacted spike bits per lane.
// v_mfma_i32_16x16x64_i8 accumulates exactly in int32; output element
// (lane, e) is tile row 4g + e.
//
// k_qbsm_fused builds the union, the active-row list and the compacted
// spike bits in LDS itself; k_qbsm_list reads them from the prep pass.
// ---------------------------------------------------------------------------
constexpr int kGroup = 2;
constexpr int kFusedMaxWords = 256;     // K <= 16384 for the single-kernel product
constexpr size_t kLdsBudget = 65536;    // LDS per workgroup used by the product kernel
constexpr int kMaxEpiTokens = 128;      // row-block tokens whose residual words are staged
constexpr int kUpLoads = 2;             // partial-union loads per thread staged in registers
constexpr int kRowLoads = 2;            // spike-row words per thread staged in registers
constexpr int kStageBatch = 8;
// a wave reads the blocked weight copy when its active words have at least
// this many active rows of 64 on average (at most twice the row bytes)
constexpr int kBlockedMinRows = NMDLM_BLOCKED_MIN_ROWS;          // further spike-row words per thread per staging batch
static_assert(kMaxEpiTokens >= 8 * 16, "every tile's residual words are staged (RT <= 8)");

__device__ __forceinline__ uint32_t expand4(uint32_t nib) {
  // 4 bits -> 4 bytes of 0/1 (bit i -> byte i); the shifted copies of the
  // nibble do not overlap, so the multiply adds no carries.
  return (nib * 0x00204081u) & 0x01010101u;
}

__device__ __forceinline__ v4i a_operand(uint32_t b16) {
  return v4i{(int)expand4(b16 & 0xFu), (int)expand4((b16 >> 4) & 0xFu),
             (int)expand4((b16 >> 8) & 0xFu), (int)expand4(b16 >> 12)};
}

// Signed A operand of ternary spikes: byte 1 where the +1 bit is set, 0xFF
// (-1) where the -1 bit is set (the two never coincide), else 0.
__device__ __forceinline__ v4i a_operand_tern(uint32_t p16, uint32_t n16) {
  return v4i{(int)(expand4(p16 & 0xFu) | expand4(n16 & 0xFu) * 0xFFu),
             (int)(expand4((p16 >> 4) & 0xFu) | expand4((n16 >> 4) & 0xFu) * 0xFFu),
             (int)(expand4((p16 >> 8) & 0xFu) | expand4((n16 >> 8) & 0xFu) * 0xFFu),
             (int)(expand4(p16 >> 12) | expand4(n16 >> 12) * 0xFFu)};
}

// Four B operands (columns 4c+v) from 16 row dwords (rows 0..15, 4 columns each).
__device__ __forceinline__ void b_operands(const uint32_t* xw, v4i (&b)[4]) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const uint32_t x0 = xw[4 * u], x1 = xw[4 * u + 1], x2 = xw[4 * u + 2], x3 = xw[4 * u + 3];
    const uint32_t t0 = __builtin_amdgcn_perm(x1, x0, 0x05010400u);  // x0[0] x1[0] x0[1] x1[1]
    const uint32_t t1 = __builtin_amdgcn_perm(x1, x0, 0x07030602u);  // x0[2] x1[2] x0[3] x1[3]
    const uint32_t t2 = __builtin_amdgcn_perm(x3, x2, 0x05010400u);
    const uint32_t t3 = __builtin_amdgcn_perm(x3, x2, 0x07030602u);
    b[0][u] = (int)__builtin_amdgcn_perm(t2, t0, 0x05040100u);  // column 4c+0, rows 4u..4u+3
    b[1][u] = (int)__builtin_amdgcn_perm(t2, t0, 0x07060302u);
    b[2][u] = (int)__builtin_amdgcn_perm(t3, t1, 0x05040100u);
    b[3][u] = (int)__builtin_amdgcn_perm(t3, t1, 0x07060302u);
  }
}

__device__ __forceinline__ int phys_col(int col) { return (col & 3) * 16 + (col >> 2); }

// Epilogue operands staged in LDS at kernel entry, so that the epilogue
// issues no dependent global load.
struct EpiStage {
  int bias[64];
  int theta[64];
  unsigned long long resid[kMaxEpiTokens];  // [t * Mb + token]
  signed char lut[256];                     // activation table (EPI_QNL_IF)
  uint32_t vbits[NMDLM_MAX_T * 64];         // channel-major output: token bits per (t, column)
};

// The epilogue operands one thread stages (at most one of each kind per
// thread: 64 columns, T * Mb <= kMaxEpiTokens residual words, 256 table
// bytes), loaded into registers first so that the staging loads of a kernel
// are all in flight together.  The loads take clamped (valid) addresses and
// no per-lane condition; the conditions are applied when the values are
// stored, so that no load is waited for before the last one is issued.
struct EpiRegs {
  int bias, theta_ch, theta_seg;
  unsigned long long resid;
  int lut;
};

template <int NT>
__device__ __forceinline__ EpiRegs epi_load(const QbsmArgs& a, int tid, int x, int y) {
  static_assert(NT >= 256 && NT >= kMaxEpiTokens, "one staged item of each kind per thread");
  EpiRegs r{0, 0, 0, 0ull, 0};
  // each kind is loaded by the waves that hold one of its items (a
  // wave-uniform test), every lane of such a wave at a valid address
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nc = min(x * 64 + (tid & 63), a.N - 1);
  if (wv == 0) {
    if (a.bias) r.bias = a.bias[nc];
    if (a.theta_vec) r.theta_ch = a.theta_vec[nc];
  }
  if (a.mode == EPI_IF || a.mode == EPI_QNL_IF)
    r.theta_seg = a.seg[a.nseg > 1 ? div_small(x * 64, a.inv_segw) : 0].theta;
  if (a.resid && wv * 64 < a.T * a.Mb) {  // T * Mb <= 16 * RT <= kMaxEpiTokens
    const int i = min(tid, a.T * a.Mb - 1);
    const int t = div_small(i, a.inv_mb), m = min(y * a.Mb + (i - t * a.Mb), a.M - 1);
    r.resid = a.resid[t * a.rld_t + (int64_t)m * a.rld_m + x];
  }
  if (a.mode == EPI_QNL_IF && wv < 4) r.lut = (int)(signed char)a.lut[tid & 255];
  return r;
}

template <int NT>
__device__ __forceinline__ void epi_store(const QbsmArgs& a, EpiStage& ep, const EpiRegs& r, int tid,
                                          int x, int y) {
  if (tid < 64) {
    const bool nv = x * 64 + tid < a.N;
    ep.bias[tid] = nv ? r.bias : 0;
    // firing threshold of each column: per channel, else the segment's
    ep.theta[tid] = a.theta_vec ? (nv ? r.theta_ch : 1) : r.theta_seg;
  }
  if (a.resid && tid < a.T * a.Mb) {
    const int t = div_small(tid, a.inv_mb), m = y * a.Mb + (tid - t * a.Mb);
    ep.resid[tid] = m < a.M ? r.resid : 0ull;
  }
  if (a.mode == EPI_QNL_IF && tid < 256) ep.lut[tid] = (signed char)r.lut;
  for (int i = tid; i < NMDLM_MAX_T * 64; i += NT) ep.vbits[i] = 0u;
}

template <int NT>
__device__ __forceinline__ void stage_epilogue(const QbsmArgs& a, EpiStage& ep, int tid, int x, int y) {
  epi_store<NT>(a, ep, epi_load<NT>(a, tid, x, y), tid, x, y);
}

// Sum the waves' accumulators into the LDS tile (physical column order).
template <int RT>
__device__ __forceinline__ void reduce_tile(const v4i (&acc)[RT][4], int* sTile, int g, int c) {
#pragma unroll
  for (int q = 0; q < RT; ++q)
#pragma unroll
    for (int v = 0; v < 4; ++v)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        atomicAdd(&sTile[(q * 16 + g * 4 + e) * kTileLd + v * 16 + c], acc[q][v][e]);
      }
}

// One wave's accumulators stored into the LDS tile (every entry of it).
template <int RT>
__device__ __forceinline__ void store_tile(const v4i (&acc)[RT][4], int* sTile, int g, int c) {
#pragma unroll
  for (int q = 0; q < RT; ++q)
#pragma unroll
    for (int v = 0; v < 4; ++v)
#pragma unroll
      for (int e = 0; e < 4; ++e) sTile[(q * 16 + g * 4 + e) * kTileLd + v * 16 + c] = acc[q][v][e];
}

// K split across workgroups: every split adds its tile into the tile's
// accumulator (int32, zero between products) with device-scope atomic adds
// whose returned values are waited for, so that each add has been performed
// at the device's point of coherence before the barrier after them; one
// thread then counts the arrival.  The split that arrives last (it sees P - 1
// earlier arrivals, each counted after that split's adds were performed)
// takes the sums with atomic exchanges that leave the accumulator zero, and
// resets the counter.  Every access to the accumulator and the counter is a
// device-scope atomic, so no cache has to be written back or invalidated.
// Integer addition makes the sums independent of the order of arrival.
// Returns false for the workgroups that are not last.
template <int ROWS, int NT>
__device__ bool split_fixup(const QbsmArgs& a, int* sTile, int* sLast, int tid, int x, int y, int z) {
  (void)z;
  const size_t tile_id = (size_t)y * gridDim.x + x;
  int* acc = a.part + tile_id * (size_t)(ROWS * 64);
  int sink = 0;
  for (int i = tid; i < ROWS * 64; i += NT) {
    const int v = sTile[(i >> 6) * kTileLd + phys_col(i & 63)];
    if (v != 0) sink |= __hip_atomic_fetch_add(&acc[i], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  asm volatile("" ::"v"(sink));  // every returned value (so every add) is waited for
  __syncthreads();
  if (tid == 0)
    *sLast = (__hip_atomic_fetch_add(&a.counters[tile_id], 1, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT) == a.P - 1) ? 1 : 0;
  __syncthreads();
  if (!*sLast) return false;
  for (int i = tid; i < ROWS * 64; i += NT)
    sTile[(i >> 6) * kTileLd + phys_col(i & 63)] =
        __hip_atomic_exchange(&acc[i], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (tid == 0) __hip_atomic_store(&a.counters[tile_id], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  return true;
}

// Channel-major output of a row block (the value cache): the tokens' bits of
// every (step, column) have met in ep.vbits; wave 0 writes them, in plain byte
// stores when the block's tokens fill whole bytes of the position words (this
// workgroup owns them), else by clearing and setting its bits with one pair
// of atomics per word.
__device__ __forceinline__ void write_channel_major(const QbsmArgs& a, const EpiStage& ep,
                                                    SpikeSeg seg, int segi, int wave, int col,
                                                    int n, bool nv, int y) {
  const bool tr_bytes = (a.Mb & 7) == 0 && (seg.pos0 & 7) == 0;
  if (wave == 0 && nv) {
    const int ch = n - segi * a.seg_w;
    // several sequences: the row block lies within sequence (y Mb) / seq_len
    const int yb = y * a.Mb;
    const int sq = seg.seq_len > 0 ? yb / seg.seq_len : 0;
    const int p0 = seg.pos0 + (seg.seq_len > 0 ? yb - sq * seg.seq_len : yb);
    seg.ptr += (int64_t)sq * seg.ld_s;
    const int nvalid = min(a.Mb, a.M - y * a.Mb);  // tokens of the block, <= 32
    if (tr_bytes) {
      // p0 is a multiple of 8: store the (up to 4) bytes holding a token of
      // the block; they may straddle two position words
      const int nb = (nvalid + 7) >> 3;
      for (int t = 0; t < a.T; ++t) {
        const uint32_t bits = ep.vbits[t * 64 + col];
        uint64_t* base = seg.ptr + t * seg.ld_t + (int64_t)ch * seg.ld_m;
        for (int b = 0; b < nb; ++b) {
          const int pb = (p0 >> 3) + b;  // byte index along the positions
          uint8_t* wb = reinterpret_cast<uint8_t*>(base + (int64_t)(pb >> 3) * seg.ld_p);
          wb[pb & 7] = (uint8_t)(bits >> (8 * b));
        }
      }
    } else {
      // the block's bits start at bit off of word p0/64 and may run into
      // the next word
      const int off = p0 & 63;
      const uint64_t full = (nvalid >= 32) ? 0xFFFFFFFFull : ((1ull << nvalid) - 1ull);
      const uint64_t m0 = full << off;
      const uint64_t m1 = off ? (full >> (64 - off)) : 0ull;
      for (int t = 0; t < a.T; ++t) {
        unsigned long long* row = reinterpret_cast<unsigned long long*>(
            seg.ptr + t * seg.ld_t + (int64_t)ch * seg.ld_m + (int64_t)(p0 >> 6) * seg.ld_p);
        const uint64_t bits = ep.vbits[t * 64 + col];
        const uint64_t b0 = bits << off;
        const uint64_t b1 = off ? (bits >> (64 - off)) : 0ull;
        atomicAnd(row, ~m0);
        if (b0) atomicOr(row, b0);
        if (m1) {
          atomicAnd(row + seg.ld_p, ~m1);
          if (b1) atomicOr(row + seg.ld_p, b1);
        }
      }
    }
  }
}

// Integrate-and-fire of the tokens ml = wave, wave + NW, ... of a row block
// (one sequence; no currents written), specialised at compile time for the
// table non-linearity (QNL), a residual input (RES) and a channel-major output
// (TR): a token's T currents (and residual words) are read, unconditionally,
// before its membrane steps, so that the reads overlap, and each step is a
// handful of instructions.  Natural outputs: word (t, m) of the column
// segment at rowbase[t*ld_t + m*ld_m].
template <int NW, bool QNL, bool RES, bool TR>
__device__ __forceinline__ void if_tokens(const QbsmArgs& a, const int* sTile, const EpiStage& ep,
                                          int lane, int wave, int y, int pc, bool nv, int bias_n,
                                          int theta, uint64_t* rowbase, int64_t ld_t, int64_t ld_m,
                                          uint32_t (&vb)[NMDLM_MAX_T], uint64_t& uor) {
  const int T = a.T, Mb = a.Mb;
  const int mlim = min(Mb, a.M - y * Mb);
  for (int ml = wave; ml < mlim; ml += NW) {
    int I[NMDLM_MAX_T];
    unsigned long long rw[NMDLM_MAX_T];
#pragma unroll
    for (int t = 0; t < NMDLM_MAX_T; ++t) {  // steps past T re-read step T - 1 (unused)
      const int tc = min(t, T - 1);
      I[t] = sTile[(tc * Mb + ml) * kTileLd + pc] + bias_n;
      rw[t] = RES ? ep.resid[tc * Mb + ml] : 0ull;
    }
    if constexpr (QNL) {
#pragma unroll
      for (int t = 0; t < NMDLM_MAX_T; ++t) {
        const int q = min(127, max(-128, I[t] >> a.lut_shift));
        I[t] = (int)ep.lut[q & 0xFF];
      }
    }
    // the membrane is int64: T steps of currents up to 2^31 in magnitude
    // plus theta stay exact
    long long V = 0;
    uint64_t* rp = TR ? nullptr : rowbase + (int64_t)(y * Mb + ml) * ld_m;
#pragma unroll
    for (int t = 0; t < NMDLM_MAX_T; ++t) {
      if (t < T) {
        long long Iv = I[t];
        if (RES && ((rw[t] >> lane) & 1ull)) Iv += theta;
        V += Iv;
        const bool s = nv && V >= theta;
        if (s) V -= theta;
        if constexpr (TR) {
          vb[t] |= (uint32_t)s << ml;
        } else {
          const uint64_t word = __builtin_amdgcn_ballot_w64(s);
          uor |= word;
          if (lane == 0) rp[t * ld_t] = word;
        }
      }
    }
  }
}

// Epilogue: currents, IF (optionally after the activation table), or head
// logits, from the reduced tile; emits the partial union of the output.
template <int NW>
__device__ void epilogue(const QbsmArgs& a, const int* sTile, EpiStage& ep,
                         unsigned long long* sUn, int tid, int lane, int wave, int x, int y) {
  const int n0 = x * 64;
  const int col = lane, n = n0 + col;
  const bool nv = n < a.N;
  const int pc = phys_col(col);
  if (a.mode == EPI_BITWISE) {
    // Eq. (11): sum_t 2^(t-1) I_t, t = 1..T (row t-1 of the tile); exact in
    // int32 within the bound the launcher checks
    for (int ml = wave; ml < a.Mb; ml += NW) {
      const int m = y * a.Mb + ml;
      if (m >= a.M) break;
      int s = 0;
      for (int t = 0; t < a.T; ++t) s += sTile[(t * a.Mb + ml) * kTileLd + pc] << t;
      if (nv) a.cur_out[(size_t)m * a.N + n] = s;
    }
    return;
  }
  if (a.mode == EPI_MODIF) {
    // Eqs. (9)-(10): the modified IF neuron over the bit-timesteps t = 0..T-1
    // of this row block's tokens (input weight 2^t, thresholds +-2^t Vth,
    // Vth = thr_num[m] / thr_den; the membrane is kept times thr_den, in
    // int64: integer arithmetic, exact), emitting ternary spike planes
    const SpikeSeg& so = a.seg[0];
    for (int ml = wave; ml < a.Mb; ml += NW) {
      const int m = y * a.Mb + ml;
      if (m >= a.M) break;
      const long long num = a.thr_num[m];
      const bool live = nv && num > 0;  // a zero threshold is silent
      long long V = 0;
      for (int t = 0; t < a.T; ++t) {
        V += (a.thr_den << t) * (long long)sTile[(t * a.Mb + ml) * kTileLd + pc];
        const long long thr = num << t;
        const bool up = live && V >= thr;
        const bool dn = live && !up && V <= -thr;
        if (up) V -= thr;
        if (dn) V += thr;
        const uint64_t wp = __builtin_amdgcn_ballot_w64(up);
        const uint64_t wn = __builtin_amdgcn_ballot_w64(dn);
        if (lane == 0) {
          const int64_t o = t * so.ld_t + (int64_t)m * so.ld_m + x;
          so.ptr[o] = wp;
          a.s_neg_out[o] = wn;
        }
      }
      if (a.v_out && nv) a.v_out[(size_t)m * a.N + n] = V;
    }
    return;
  }
  if (a.mode == EPI_HEAD) {
    const float sc = nv ? a.scale[n] : 0.f;
    for (int ml = wave; ml < a.Mb; ml += NW) {
      const int m = y * a.Mb + ml;
      if (m >= a.M) break;
      int s = 0;
      for (int t = 0; t < a.T; ++t) s += sTile[(t * a.Mb + ml) * kTileLd + pc];
      if (nv) a.logits[(size_t)m * a.N + n] = (float)s * sc;
    }
    return;
  }
  const int segi = (a.mode == EPI_CUR || a.nseg == 1) ? 0 : div_small(n0, a.inv_segw);
  SpikeSeg seg = a.seg[segi];
  const int wseg = (n0 - segi * a.seg_w) >> 6;
  const int bias_n = ep.bias[col];
  const int theta = ep.theta[col];
  const bool spikes = a.mode != EPI_CUR;
  const bool tr = spikes && seg.transposed;
  // channel-major output (row blocks of at most 32 tokens): the waves' token
  // bits meet in LDS and one wave writes them (write_channel_major)
  uint32_t vb[NMDLM_MAX_T];
#pragma unroll
  for (int t = 0; t < NMDLM_MAX_T; ++t) vb[t] = 0u;
  uint64_t uor = 0ull;  // union of this wave's output words (wave-uniform)

  // the common case (spikes only, one sequence) takes the specialised loop
  const bool lean = spikes && !a.cur_out && seg.seq_len == 0;  // workgroup-uniform
  if (lean) {
    uint64_t* rb = seg.ptr + wseg;
    const bool qnl = a.mode == EPI_QNL_IF, res = a.resid != nullptr;
#define NMDLM_IF_TOKENS(Q, R, X)                                                                   \
  if_tokens<NW, Q, R, X>(a, sTile, ep, lane, wave, y, pc, nv, bias_n, theta, rb, seg.ld_t, seg.ld_m, \
                         vb, uor)
    if (qnl) {
      if (res) { if (tr) NMDLM_IF_TOKENS(true, true, true); else NMDLM_IF_TOKENS(true, true, false); }
      else { if (tr) NMDLM_IF_TOKENS(true, false, true); else NMDLM_IF_TOKENS(true, false, false); }
    } else {
      if (res) { if (tr) NMDLM_IF_TOKENS(false, true, true); else NMDLM_IF_TOKENS(false, true, false); }
      else { if (tr) NMDLM_IF_TOKENS(false, false, true); else NMDLM_IF_TOKENS(false, false, false); }
    }
#undef NMDLM_IF_TOKENS
  }
  for (int ml = wave; ml < a.Mb && !lean; ml += NW) {
    const int m = y * a.Mb + ml;
    if (m >= a.M) break;
    // the membrane (and a current with its residual) is int64: T steps of
    // currents up to 2^31 in magnitude plus theta stay exact
    long long V = 0;
#pragma unroll
    for (int t = 0; t < NMDLM_MAX_T; ++t) {
      if (t < a.T) {
        int I = sTile[(t * a.Mb + ml) * kTileLd + pc] + bias_n;
        if (a.cur_out && nv) a.cur_out[((size_t)t * a.M + m) * a.N + n] = I;
        if (spikes) {
          if (a.mode == EPI_QNL_IF) {
            int qv = I >> a.lut_shift;
            qv = min(127, max(-128, qv));
            I = (int)ep.lut[qv & 0xFF];
          }
          long long Iv = I;
          if (a.resid) {
            // staged at entry: T * Mb <= 16 * RT <= kMaxEpiTokens rows
            const unsigned long long rw = ep.resid[t * a.Mb + ml];
            if ((rw >> col) & 1ull) Iv += theta;
          }
          V += Iv;
          const bool s = nv && V >= theta;
          if (s) V -= theta;
          if (!tr) {
            const uint64_t word = __builtin_amdgcn_ballot_w64(s);
            uor |= word;
            const int64_t mo = seg.seq_len > 0
                                   ? (int64_t)(m / seg.seq_len) * seg.ld_s + (int64_t)(m % seg.seq_len) * seg.ld_m
                                   : (int64_t)m * seg.ld_m;
            if (lane == 0) seg.ptr[t * seg.ld_t + mo + wseg] = word;
          } else if (s) {
            vb[t] |= 1u << ml;
          }
        }
      }
    }
  }
  if (tr) {
    // the waves' token bits meet in LDS; wave 0 then writes each column's
    // bits of the row block's tokens
#pragma unroll
    for (int t = 0; t < NMDLM_MAX_T; ++t)
      if (t < a.T && vb[t]) atomicOr(&ep.vbits[t * 64 + col], vb[t]);
    __syncthreads();
    write_channel_major(a, ep, seg, segi, wave, col, n, nv, y);
  }
  if (a.u_out && spikes && !tr) {
    // partial union of this row block's output word, for the next product
    if (lane == 0) sUn[wave] = uor;
    __syncthreads();
    if (tid == 0) {
      unsigned long long u = 0;
      for (int w = 0; w < NW; ++w) u |= sUn[w];
      a.u_out[(size_t)y * a.u_ld + x] = u;
    }
  }
}

// Epilogue of a wide tile (one wave, one 64-column tile, 64 rows), from the
// wave's accumulators: acc[q][v][e] of lane (g, c) is tile row 16q + 4g + e,
// column 4c + v.  With row blocks of Mb = 64 / T tokens (T = 1, 2, 4), row
// t Mb + m lies in q = t Mb / 16 + m / 16 with 4g + e = m % 16, so a lane
// holds all T currents of its 16 neurons (tokens 16k + 4g + e, k < Mb / 16;
// columns 4c + v) and integrates them in registers.  Spike words (t, m) of
// the tile's 64 columns are assembled in the wave's 256 LDS dwords: each
// lane writes the nibble of its four columns as a byte, lane i then packs
// the 16 nibbles of word i.  Channel-major output meets in ep.vbits as in
// the workgroup epilogue.  Modes: currents, IF, table + IF, head logits.
template <int T>
__device__ __forceinline__ void wide_epilogue(const QbsmArgs& a, const v4i (&acc)[4][4], EpiStage& ep,
                                              uint32_t* nib, int lane, int x, int y) {
  constexpr int KB = 4 / T;       // 16-token groups of a row block
  constexpr int Mb = 16 * KB;     // tokens of the row block
  const int g = lane >> 4, c = lane & 15;
  const int n0 = x * 64;
  if (a.mode == EPI_HEAD) {
    // logits: the sum over the steps, dequantised per column
    float sc[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) sc[v] = n0 + 4 * c + v < a.N ? a.scale[n0 + 4 * c + v] : 0.f;
#pragma unroll
    for (int k = 0; k < KB; ++k)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = y * Mb + 16 * k + 4 * g + e;
        if (m >= a.M) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          int sum = 0;
#pragma unroll
          for (int t = 0; t < T; ++t) sum += acc[t * KB + k][v][e];
          const int n = n0 + 4 * c + v;
          if (n < a.N) a.logits[(size_t)m * a.N + n] = (float)sum * sc[v];
        }
      }
    return;
  }
  const bool spikes = a.mode != EPI_CUR;
  const int segi = (a.mode == EPI_CUR || a.nseg == 1) ? 0 : div_small(n0, a.inv_segw);
  SpikeSeg seg = a.seg[segi];
  const int wseg = (n0 - segi * a.seg_w) >> 6;
  const bool tr = spikes && seg.transposed;
  const bool qnl = a.mode == EPI_QNL_IF, res = a.resid != nullptr;
  // spike bits: byte (t, k, e) of this lane holds columns 4c..4c+3
  uint32_t sb[T * KB];
#pragma unroll
  for (int i = 0; i < T * KB; ++i) sb[i] = 0u;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int col = 4 * c + v, n = n0 + col;
    const bool nv = n < a.N;
    const int bias_n = ep.bias[col], theta = ep.theta[col];
#pragma unroll
    for (int k = 0; k < KB; ++k)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int ml = 16 * k + 4 * g + e, m = y * Mb + ml;
        long long V = 0;  // int64: T currents up to 2^31 in magnitude plus theta
#pragma unroll
        for (int t = 0; t < T; ++t) {
          int I = acc[t * KB + k][v][e] + bias_n;
          if (a.cur_out && nv && m < a.M) a.cur_out[((size_t)t * a.M + m) * a.N + n] = I;
          if (!spikes) continue;
          if (qnl) I = (int)ep.lut[min(127, max(-128, I >> a.lut_shift)) & 0xFF];
          long long Iv = I;
          if (res && ((ep.resid[t * Mb + ml] >> col) & 1ull)) Iv += theta;
          V += Iv;
          const bool s = nv && V >= theta;
          if (s) V -= theta;
          sb[t * KB + k] |= (uint32_t)s << (8 * e + v);
        }
      }
  }
  if (!spikes) return;
  if (tr) {
    // channel-major: the row block's token bits of each (step, column)
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        uint32_t bits = 0u;
#pragma unroll
        for (int k = 0; k < KB; ++k)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            bits |= ((sb[t * KB + k] >> (8 * e + v)) & 1u) << (16 * k + 4 * g + e);
        if (bits) atomicOr(&ep.vbits[t * 64 + 4 * c + v], bits);
      }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    write_channel_major(a, ep, seg, segi, 0, lane, n0 + lane, n0 + lane < a.N, y);
    return;
  }
  // natural words: byte c of word (t, ml) at nib[(t Mb + ml) * 4 + c / 4]
  uint8_t* nb = reinterpret_cast<uint8_t*>(nib);
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int k = 0; k < KB; ++k)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        nb[(t * Mb + 16 * k + 4 * g + e) * 16 + c] = (uint8_t)((sb[t * KB + k] >> (8 * e)) & 0xFu);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // lane i: word i = (t, ml) (64 = T * Mb words), the low nibbles of its 16 bytes
  const int t = lane / Mb, ml = lane - t * Mb, m = y * Mb + ml;
  uint32_t h[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    uint32_t w = nib[lane * 4 + d] & 0x0F0F0F0Fu;
    w = (w | (w >> 4)) & 0x00FF00FFu;
    h[d] = (w | (w >> 8)) & 0x0000FFFFu;
  }
  const uint64_t word = (uint64_t)(h[0] | (h[1] << 16)) | ((uint64_t)(h[2] | (h[3] << 16)) << 32);
  const bool mv = m < a.M;
  if (mv) {
    const int64_t mo = seg.seq_len > 0
                           ? (int64_t)(m / seg.seq_len) * seg.ld_s + (int64_t)(m % seg.seq_len) * seg.ld_m
                           : (int64_t)m * seg.ld_m;
    seg.ptr[t * seg.ld_t + mo + wseg] = word;
  }
  if (a.u_out) {
    // partial union of the tile's output word over the row block
    uint64_t u = mv ? word : 0ull;
    for (int o = kWave / 2; o > 0; o >>= 1) u |= __shfl_xor(u, o);
    if (lane == 0) a.u_out[(size_t)y * a.u_ld + x] = u;
  }
}

// ------------------------------------------------- weight-skip statistics
// The statistics of a product are those of the whole block: the number of
// input rows (channels) active in the union of all its spike rows.  Workgroup
// (0,0,0) computes them between the barriers the product already has, so they
// add no round trip at the end of the kernel:
//   stats_slice  (with the staging loads) this thread's OR over a slice of
//                the union sources: the producer's partial unions when given,
//                else the spike rows (a product whose own union already is
//                the block union counts that instead)
//   stats_merge  (after the first barrier) ORs the slices into sStat
//   stats_count  (after a later barrier) adds the popcounts into sCnt
//   stats_write  (after a later barrier) thread 0 stores the record
// OR of src[r][w] (r < nsrc, row stride Kw) over a slice of the rows: with
// NT >= Kw, thread tid takes word tid % Kw and rows tid / Kw, + NT / Kw, ...,
// so that few loads per thread are all in flight together.
template <int NT>
__device__ __forceinline__ unsigned long long or_slice(const uint64_t* src, int nsrc, int Kw,
                                                       int tid) {
  unsigned long long u = 0ull;
  if (NT < Kw) return u;
  const float inv_kw = 1.0f / (float)Kw;
  const int slices = div_small(NT, inv_kw), s0 = div_small(tid, inv_kw), w = tid - s0 * Kw;
  if (s0 >= slices) return u;
  int r = s0;
  for (; r + 3 * slices < nsrc; r += 4 * slices)
    u |= src[(size_t)r * Kw + w] | src[(size_t)(r + slices) * Kw + w] |
         src[(size_t)(r + 2 * slices) * Kw + w] | src[(size_t)(r + 3 * slices) * Kw + w];
  for (; r < nsrc; r += slices) u |= src[(size_t)r * Kw + w];
  return u;
}

// dst[w] = OR of the slices (dst cleared before the barrier that precedes
// this call); bits of the last word past K are dropped with last_mask.
template <int NT>
__device__ __forceinline__ void or_merge(unsigned long long* dst, const uint64_t* src, int nsrc,
                                         int Kw, int tid, unsigned long long u,
                                         unsigned long long last_mask) {
  if (NT >= Kw) {
    const float inv_kw = 1.0f / (float)Kw;
    const int slices = div_small(NT, inv_kw), s0 = div_small(tid, inv_kw), w = tid - s0 * Kw;
    if (w == Kw - 1) u &= last_mask;
    if (s0 < slices && u) atomicOr(&dst[w], u);
  } else {
    // more words than threads: each thread ORs every source of its words
    for (int w = tid; w < Kw; w += NT) {
      unsigned long long v = 0ull;
      for (int r = 0; r < nsrc; ++r) v |= src[(size_t)r * Kw + w];
      dst[w] = (w == Kw - 1) ? (v & last_mask) : v;  // the only writer of word w
    }
  }
}

template <int NT>
__device__ __forceinline__ unsigned long long stats_slice(const QbsmArgs& a, int Kw, int tid) {
  if (a.dense) return 0ull;
  return a.upart ? or_slice<NT>(a.upart, a.nparts, Kw, tid) : or_slice<NT>(a.S, a.T * a.M, Kw, tid);
}

template <int NT>
__device__ __forceinline__ void stats_merge(const QbsmArgs& a, unsigned long long* sStat, int Kw,
                                            int tid, unsigned long long u) {
  if (a.dense) return;
  if (a.upart) or_merge<NT>(sStat, a.upart, a.nparts, Kw, tid, u, ~0ull);
  else or_merge<NT>(sStat, a.S, a.T * a.M, Kw, tid, u, ~0ull);
}

template <int NT>
__device__ __forceinline__ void stats_count(const QbsmArgs& a, const unsigned long long* sStat,
                                            int* sCnt, int Kw, int tid, int lane) {
  const unsigned long long last_mask = (a.K & 63) ? (1ull << (a.K & 63)) - 1ull : ~0ull;
  int cnt = 0;
  if (a.dense) {
    cnt = tid == 0 ? a.K : 0;
  } else {
    for (int w = tid; w < Kw; w += NT) {
      const unsigned long long u = sStat[w];
      cnt += __popcll((w == Kw - 1) ? (u & last_mask) : u);
    }
  }
  for (int o = kWave / 2; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o);
  if (lane == 0 && cnt) atomicAdd(sCnt, cnt);
}

__device__ __forceinline__ void stats_write(const QbsmArgs& a, int total) {
  a.stats->k_total = a.K;
  a.stats->k_active = total;
  a.stats->n = a.N;
  a.stats->weight_bytes = (int64_t)total * (int64_t)a.N;
}

// ------------------------------------------------- scalar accumulation
// The gather-accumulate product (path 5; on MI355X it measured no faster than
// MFMA at any point of the FFN sweep d=4096 -> 14336 -> 4096, density 0.02 to
// 0.30, so the automatic choice keeps MFMA): each thread takes a
// task (block row lr, column quad j) and a slice of the words of K (w0 + s,
// w0 + s + S, ...); for every spike k of the row in its words it loads the
// four weights W[k][4j .. 4j+3] (one dword) and adds them, sign-extended, to
// four int32 sums, which meet in the tile (LDS atomics, physical column
// order).  A row's spikes are taken eight at a time, each group's loads all
// in flight (lanes past the last spike re-load the group's first row and add
// nothing).  Integer addition: the sums equal the MFMA path's exactly.  Only
// the rows of the block's tokens get tasks, and the slices spread the spikes
// of a row over the threads left.
constexpr int kScalarGroup = 8;

template <int ROWS, int NT>
__device__ void scalar_accumulate(const QbsmArgs& a, const uint32_t* sS, int lds_row, int* sTile,
                                  int tid, int x, int y, int w0, int w1) {
  const int mvalid = min(a.Mb, a.M - y * a.Mb);  // tokens of the row block
  const int rows = a.T * mvalid;                 // rows with spikes: t * Mb + ml, ml < mvalid
  const int tasks = rows * 16;
  if (tasks <= 0) return;
  const int S = NT >= tasks ? NT / tasks : 1;    // word slices per task
  const int nwork = NT >= tasks ? tasks * S : NT;
  if (tid >= nwork) return;
  const float inv_mv = 1.0f / (float)mvalid;
  const char* Wb = reinterpret_cast<const char*>(a.W);
  const uint32_t ldw = (uint32_t)a.ldw;
  for (int task = NT >= tasks ? tid % tasks : tid; task < tasks; task += NT >= tasks ? tasks : NT) {
    const int slice = NT >= tasks ? tid / tasks : 0;
    const int r = task >> 4, j = task & 15;
    const int t = div_small(r, inv_mv), ml = r - t * mvalid;
    const int lr = t * a.Mb + ml;
    const int col = x * 64 + 4 * j;
    if (col >= a.N) continue;  // ldw is a multiple of 16 >= N: the dword of a valid quad is in the row
    int s4[4] = {0, 0, 0, 0};
    for (int w = w0 + slice; w < w1; w += S) {
      unsigned long long word = (unsigned long long)sS[lr * lds_row + 2 * w] |
                                ((unsigned long long)sS[lr * lds_row + 2 * w + 1] << 32);
      while (word) {
        const int kfirst = w * 64 + (int)__builtin_ctzll(word);
        uint32_t wv[kScalarGroup];
        uint32_t valid = 0u;
#pragma unroll
        for (int i = 0; i < kScalarGroup; ++i) {
          const bool v = word != 0ull;
          const int k = v ? w * 64 + (int)__builtin_ctzll(word) : kfirst;
          valid |= (uint32_t)v << i;
          word &= word - 1ull;  // 0 stays 0
          wv[i] = *reinterpret_cast<const uint32_t*>(Wb + (uint32_t)k * ldw + (uint32_t)col);
        }
#pragma unroll
        for (int i = 0; i < kScalarGroup; ++i) {
          const int m = -(int)((valid >> i) & 1u);  // all ones for a spike of the group
          const int q = (int)wv[i] & m;
#pragma unroll
          for (int b = 0; b < 4; ++b) s4[b] += (int)(signed char)(q >> (8 * b));
        }
      }
    }
#pragma unroll
    for (int b = 0; b < 4; ++b)
      if (s4[b]) atomicAdd(&sTile[lr * kTileLd + phys_col(4 * j + b)], s4[b]);
  }
}

// ------------------------------------------------- word-granular product
// k-steps are the original 64-channel words.  The A operand comes straight
// from the staged spike rows (no list, no compaction).  Within a word, a lane
// loads only the rows active in this tile's rows (its local union): a row
// absent from the local union has a zero spike in every tile row, so its B
// slot (left stale) is multiplied by zero.  Across row blocks the rows read
// are the block union; repeated reads hit the cache.  Words with no active
// row are skipped.
// BLK: a blocked copy of the weights (a.Wb, operand order) is also given: a
// word is then four 16-byte loads per lane, already B operands, with every
// row of an active word read (rows outside the local union meet zero spikes)
// and a word with no active row skipped.  Each wave takes the copy or the
// row-major rows by the density of its words' union (a.blk_min).
// SCA: the variant with the scalar gather-accumulate product (a.accum == 1);
// kept out of the others, whose registers it would raise.
// The 64-row blocked variant is held to four waves per SIMD (the head's
// 1000 workgroups then run in one round instead of two: 29.7 -> 22.5 us at
// the 12-layer shape); the compiler then keeps a dozen values that live
// across the word loop in scratch, stored once before it and reloaded once
// after it.
// WIDE: a workgroup takes NW adjacent 64-column tiles of one row block, wave
// j the tile NW x + j over every word of K (blocked copy only): the spike
// staging, the union and the epilogue operands are shared by NW tiles, and
// each wave finishes its own tile from its accumulators (wide_epilogue).
// Entry points aligned to 1 KB: with the default 256-byte placement the
// twelve-layer step measured 0.8-1.5% slower, depending on where the code
// object's other contents happened to put the kernels.
template <int RT, int NW, bool TERN = false, bool BLK = false, bool SCA = false, bool WIDE = false>
__global__ __launch_bounds__(NW * 64, (BLK && RT == 4 && NW == 4) ? 4 : 1) __attribute__((aligned(1024)))
void k_qbsm_words(QbsmArgs a) {
  static_assert(!WIDE || (BLK && !TERN && !SCA && RT == 4 && NW == 4), "wide tiles: blocked, 64 rows");
  constexpr int ROWS = RT * 16;
  constexpr int NT = NW * 64;
  constexpr int NE = WIDE ? NW : 1;  // column tiles (epilogue stages) per workgroup
  // ALIAS (64-row tiles): the reduction tile takes the place of the spike
  // rows, which are dead once the word loop is done, so that long-K tiles
  // keep four workgroups per CU (the host sizes the dynamic LDS for both)
  constexpr bool ALIAS = RT == 4 && !WIDE && !SCA;
  // WIDE: the waves' 1 KB spike-word exchanges in place of the LDS tile
  __shared__ int sTileS[WIDE ? NW * 256 : (ALIAS ? 1 : ROWS * kTileLd)];
  __shared__ unsigned long long sUn[NW];
  __shared__ EpiStage ep[NE];
  __shared__ int sLast;
  __shared__ int sStatCnt;
  // dynamic: local union [Kw] (u64), the block union of the statistics [Kw]
  // (u64), then the tile's spike rows as dwords with row stride 2*Kw+1 (odd:
  // the 16 rows a wave reads fall in different banks)
  extern __shared__ unsigned long long sDyn[];

  touch_kernargs<sizeof(QbsmArgs)>();
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  int x, y, z;
  tile_coords_inv(x, y, z, a.inv_gy, a.inv_gxy);
  const int Kw = (a.K + 63) >> 6;
  const int lds_row = 2 * Kw + 1;
  unsigned long long* sLU = sDyn;
  unsigned long long* sStat = sDyn + Kw;
  uint32_t* sS = reinterpret_cast<uint32_t*>(sDyn + 2 * Kw);
  int* const sTile = ALIAS ? reinterpret_cast<int*>(sDyn + 2 * Kw) : sTileS;
  // ternary input: the -1 spike rows follow the +1 rows, same layout
  uint32_t* sSn = sS + ROWS * lds_row;
  const bool stats_wg = a.stats && x == 0 && y == 0 && z == 0;  // workgroup-uniform
  const int gx = WIDE ? (a.N + 63) >> 6 : 0;  // column tiles (WIDE)
  // this wave's column tile (WIDE), else the workgroup's
  const int xs = WIDE ? x * NW + wave : x;

  const unsigned long long last_mask = (a.K & 63) ? (1ull << (a.K & 63)) - 1ull : ~0ull;
  // With the producer's partial unions, the union is their OR over the whole
  // block (a superset of this row block's own union: the extra rows meet zero
  // spikes): each thread ORs a slice of them with the staging loads, and the
  // slices meet in LDS after the first barrier.  Otherwise it is the OR of
  // the staged rows.  Either way a second barrier publishes it.
  const bool from_parts = a.upart && !a.dense;
  const bool stats_rows = stats_wg && !from_parts && !a.dense;  // block union from the rows

  // ---- staging, load phase: every load goes out before the first is used
  const EpiRegs er = epi_load<NT>(a, tid, WIDE ? min(x * NW, gx - 1) : x, y);
  EpiRegs erw[NE > 1 ? NE - 1 : 1];  // WIDE: the other column tiles' operands
  if constexpr (WIDE) {
#pragma unroll
    for (int j = 1; j < NE; ++j) erw[j - 1] = epi_load<NT>(a, tid, min(x * NW + j, gx - 1), y);
  }
  // thread tid takes word wq = tid % Kw and rows r0 = tid / Kw, + rpp, ...
  // (rpp = NT / Kw rows per pass; none when the words outnumber the threads)
  const float inv_kw = a.inv_kw, inv_mb = a.inv_mb;
  const int r0 = div_small(tid, inv_kw), wq = tid - r0 * Kw;
  const int rpp = div_small(NT, inv_kw);
  const int wr0 = __builtin_amdgcn_readfirstlane(r0);  // first row of this wave's lanes
  // partial unions: part s = r0 + k * rpp of word wq
  const int slices = rpp;
  const int s0 = r0;
  const bool up_regs = from_parts && slices > 0 && a.nparts > 0 && a.nparts <= kUpLoads * slices;
  unsigned long long upv[kUpLoads];
#pragma unroll
  for (int k = 0; k < kUpLoads; ++k) {
    upv[k] = 0ull;
    // waves with a part to load (uniform); other lanes load a valid word
    if (up_regs && wr0 + k * slices < a.nparts)
      upv[k] = a.upart[(uint32_t)(min(s0 + k * slices, a.nparts - 1) * Kw + wq)];
  }
  // this row block's spike rows: tile row lr = r0 + k * rpp, word wq; rows
  // past the tile or the block load a valid word and drop it
  unsigned long long rv[kRowLoads], rvn[kRowLoads];
  int rdst[kRowLoads];  // dword offset of the item in sS, or -1
  uint32_t keep = 0u;   // bit k: item k lies in the block (else it is stored as zero)
#pragma unroll
  for (int k = 0; k < kRowLoads; ++k) {
    const int lr = r0 + k * rpp;
    rdst[k] = -1;
    rv[k] = 0ull;
    rvn[k] = 0ull;
    if (wr0 < rpp && wr0 + k * rpp < ROWS) {  // wave-uniform
      const int lc = min(lr, ROWS - 1);
      const int t = div_small(lc, inv_mb), m = y * a.Mb + (lc - t * a.Mb);
      // T*M <= 2^19 rows of at most 1024 words: 32-bit offsets
      const uint32_t src = (uint32_t)(min(t, a.T - 1) * a.M + min(m, a.M - 1)) * (uint32_t)Kw + wq;
      rv[k] = a.S[src];
      if constexpr (TERN) rvn[k] = a.Sn[src];
      rdst[k] = (r0 < rpp && lr < ROWS) ? lr * lds_row + 2 * wq : -1;
      keep |= (uint32_t)(t < a.T && m < a.M) << k;
    }
  }
  // many partial unions (or more words than threads): OR loops
  unsigned long long upart_or = 0ull;
  if (from_parts && !up_regs) upart_or = or_slice<NT>(a.upart, a.nparts, Kw, tid);
  unsigned long long spart = 0ull;
  if (stats_rows) spart = or_slice<NT>(a.S, a.T * a.M, Kw, tid);
  if constexpr (TERN) {
    if (stats_rows) spart |= or_slice<NT>(a.Sn, a.T * a.M, Kw, tid);
  }
  __builtin_amdgcn_sched_barrier(0);

  // ---- staging, store phase
  if constexpr (!WIDE && !ALIAS)
    for (int i = tid; i < ROWS * kTileLd; i += NT) sTile[i] = 0;
  epi_store<NT>(a, ep[0], er, tid, WIDE ? min(x * NW, gx - 1) : x, y);
  if constexpr (WIDE) {
#pragma unroll
    for (int j = 1; j < NE; ++j) epi_store<NT>(a, ep[j], erw[j - 1], tid, min(x * NW + j, gx - 1), y);
  }
  if (from_parts || (ROWS > 32 && !a.dense && NT >= Kw))
    for (int w = tid; w < Kw; w += NT) sLU[w] = 0ull;
  if (stats_wg && tid == 0) sStatCnt = 0;
  if (stats_rows)
    for (int w = tid; w < Kw; w += NT) sStat[w] = 0ull;
#pragma unroll
  for (int k = 0; k < kRowLoads; ++k)
    if (rdst[k] >= 0) {
      const unsigned long long v = ((keep >> k) & 1u) ? rv[k] : 0ull;
      sS[rdst[k]] = (uint32_t)v;
      sS[rdst[k] + 1] = (uint32_t)(v >> 32);
      if constexpr (TERN) {
        const unsigned long long vn = ((keep >> k) & 1u) ? rvn[k] : 0ull;
        sSn[rdst[k]] = (uint32_t)vn;
        sSn[rdst[k] + 1] = (uint32_t)(vn >> 32);
      }
    }
  // rows past kRowLoads passes (all rows when the words outnumber the
  // threads): batches of kStageBatch words per thread, every load of a batch
  // issued (at a clamped address) before the first is stored
  const int items = ROWS * Kw;
  for (int i0 = tid + kRowLoads * rpp * Kw; i0 - tid < items; i0 += kStageBatch * NT) {
    unsigned long long v[kStageBatch], vn[kStageBatch];
    uint32_t kp = 0u;  // bit j: item j lies in the tile and the block
#pragma unroll
    for (int j = 0; j < kStageBatch; ++j) {
      const int i = i0 + j * NT, ic = min(i, items - 1);
      const int lr = div_small(ic, inv_kw), w = ic - lr * Kw;
      const int t = div_small(lr, inv_mb), m = y * a.Mb + (lr - t * a.Mb);
      const uint32_t src = (uint32_t)(min(t, a.T - 1) * a.M + min(m, a.M - 1)) * (uint32_t)Kw + w;
      v[j] = a.S[src];
      if constexpr (TERN) vn[j] = a.Sn[src];
      kp |= (uint32_t)(i < items && t < a.T && m < a.M) << j;
    }
#pragma unroll
    for (int j = 0; j < kStageBatch; ++j) {
      const int i = i0 + j * NT;
      if (i < items) {
        const int lr = div_small(i, inv_kw), w = i - lr * Kw;
        const unsigned long long vv = ((kp >> j) & 1u) ? v[j] : 0ull;
        sS[lr * lds_row + 2 * w] = (uint32_t)vv;
        sS[lr * lds_row + 2 * w + 1] = (uint32_t)(vv >> 32);
        if constexpr (TERN) {
          const unsigned long long vvn = ((kp >> j) & 1u) ? vn[j] : 0ull;
          sSn[lr * lds_row + 2 * w] = (uint32_t)vvn;
          sSn[lr * lds_row + 2 * w + 1] = (uint32_t)(vvn >> 32);
        }
      }
    }
  }
  if (up_regs && s0 < slices) {
#pragma unroll
    for (int k = 0; k < kUpLoads; ++k)
      if (s0 + k * slices < a.nparts) upart_or |= upv[k];
  }
  __syncthreads();
  if (from_parts) {
    or_merge<NT>(sLU, a.upart, a.nparts, Kw, tid, upart_or, last_mask);
  } else if (ROWS > 32 && !a.dense && NT >= Kw) {
    // many rows: thread tid ORs rows r0, r0 + rpp, ... of word wq (the
    // slices were cleared before the first barrier), one LDS OR per thread
    unsigned long long u = 0ull;
    if (r0 < rpp)
      for (int lr = r0; lr < ROWS; lr += rpp) {
        u |= (unsigned long long)sS[lr * lds_row + 2 * wq] |
             ((unsigned long long)sS[lr * lds_row + 2 * wq + 1] << 32);
        if constexpr (TERN)
          u |= (unsigned long long)sSn[lr * lds_row + 2 * wq] |
               ((unsigned long long)sSn[lr * lds_row + 2 * wq + 1] << 32);
      }
    if (wq == Kw - 1) u &= last_mask;
    if (u) atomicOr(&sLU[wq], u);
  } else {
    for (int w = tid; w < Kw; w += NT) {
      unsigned long long u = ~0ull;
      if (!a.dense) {
        u = 0ull;
        for (int lr = 0; lr < ROWS; ++lr) {
          u |= (unsigned long long)sS[lr * lds_row + 2 * w] |
               ((unsigned long long)sS[lr * lds_row + 2 * w + 1] << 32);
          if constexpr (TERN)
            u |= (unsigned long long)sSn[lr * lds_row + 2 * w] |
                 ((unsigned long long)sSn[lr * lds_row + 2 * w + 1] << 32);
        }
      }
      sLU[w] = (w == Kw - 1) ? (u & last_mask) : u;
    }
  }
  if (stats_rows) or_merge<NT>(sStat, a.S, a.T * a.M, Kw, tid, spart, ~0ull);  // ternary: NT >= Kw
  __syncthreads();
  // first active row (the target of the loads of inactive rows), per wave
  int first = 0x7fffffff;
  for (int w = lane; w < Kw; w += kWave) {
    const unsigned long long u = sLU[w];
    if (u) {
      first = w * 64 + (int)__builtin_ctzll(u);
      break;
    }
  }
  for (int o = kWave / 2; o > 0; o >>= 1) first = min(first, __shfl_xor(first, o));

  // the K split's words (Kw <= 1024, z < P <= 255: 32-bit products)
  const int w0 = a.P > 1 ? (Kw * z) / a.P : 0;
  const int w1 = a.P > 1 ? (Kw * (z + 1)) / a.P : Kw;
  const uint32_t colb = (x * 64 + 4 * c < a.N) ? (uint32_t)(x * 64 + 4 * c) : (uint32_t)(x * 64);
  const uint32_t ldw = (uint32_t)a.ldw;
  const uint32_t lane_base = (uint32_t)(16 * g) * ldw + colb;   // row 16g of word 0
  const char* Wb = reinterpret_cast<const char*>(a.W);

  v4i acc[RT][4];
#pragma unroll
  for (int q = 0; q < RT; ++q)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[q][v] = v4i{0, 0, 0, 0};
  // Weight loads are unconditional: a lane whose row is not active in this
  // tile (or a word past the range) loads the tile's first active row, whose
  // line is read anyway.  Every word then issues the same 16 loads, so the
  // next word's loads can be in flight while the current one is multiplied.
  const uint32_t first_off = (uint32_t)first * ldw + colb;
  const int stride = WIDE ? 1 : NW;
  auto load_rows = [&](int w, uint32_t (&xg)[16]) {
    const unsigned long long u = (w < w1) ? sLU[w] : 0ull;
    const uint32_t m16 = (uint32_t)(u >> (16 * g)) & 0xFFFFu;
    const uint32_t wbase = (uint32_t)w * 64u * ldw + lane_base;
#pragma unroll
    for (int s2 = 0; s2 < 16; ++s2) {
      const uint32_t off = ((m16 >> s2) & 1u) ? wbase + (uint32_t)s2 * ldw : first_off;
      xg[s2] = *reinterpret_cast<const uint32_t*>(Wb + off);
    }
  };
  // blocked copy: a word of the tile is four 16-byte operand loads; an
  // inactive word (or one past the range) re-reads the first active word
  const int gxb = (a.N + 63) >> 6;
  const char* Wbb = reinterpret_cast<const char*>(a.Wb) + (size_t)(WIDE ? min(xs, gxb - 1) : x) * 4096 +
                    (size_t)lane * 16;
  auto load_blocked = [&](int w, uint32_t (&xg)[16]) {
    const unsigned long long u = (w < w1) ? sLU[w] : 0ull;
    const int ws = u ? w : (first >> 6);
    const char* p = Wbb + (size_t)ws * gxb * 4096;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const v4i q = *reinterpret_cast<const v4i*>(p + v * 1024);
#pragma unroll
      for (int e = 0; e < 4; ++e) xg[4 * v + e] = (uint32_t)q[e];
    }
  };
  auto mul_b = [&](int w, const v4i (&b)[4]) {
#pragma unroll
    for (int q = 0; q < RT; ++q) {
      const int sidx = (q * 16 + c) * lds_row + 2 * w + (g >> 1);
      const uint32_t b16 = (sS[sidx] >> (16 * (g & 1))) & 0xFFFFu;
      v4i af;
      if constexpr (TERN) af = a_operand_tern(b16, (sSn[sidx] >> (16 * (g & 1))) & 0xFFFFu);
      else af = a_operand(b16);
#pragma unroll
      for (int v = 0; v < 4; ++v)
        acc[q][v] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, b[v], acc[q][v], 0, 0, 0);
    }
  };
  auto mul_rows = [&](int w, const uint32_t (&xg)[16]) {
    const unsigned long long u = (w < w1) ? sLU[w] : 0ull;
    if (u == 0ull) return;  // wave-uniform
    v4i b[4];
    b_operands(xg, b);
    mul_b(w, b);
  };
  auto mul_blocked = [&](int w, const uint32_t (&xg)[16]) {
    const unsigned long long u = (w < w1) ? sLU[w] : 0ull;
    if (u == 0ull) return;  // wave-uniform
    v4i b[4];
#pragma unroll
    for (int v = 0; v < 4; ++v)
      b[v] = v4i{(int)xg[4 * v], (int)xg[4 * v + 1], (int)xg[4 * v + 2], (int)xg[4 * v + 3]};
    mul_b(w, b);
  };
  // the words of this wave, the next one's loads in flight while the
  // current one is multiplied
  auto loop = [&](auto&& load, auto&& mul) {
    int jw = WIDE ? w0 : w0 + wave;
    uint32_t xa[16], xb[16];
    load(jw, xa);
    while (true) {
      load(jw + stride, xb);
      mul(jw, xa);
      jw += stride;
      if (jw >= w1) break;
      load(jw + stride, xa);
      mul(jw, xb);
      jw += stride;
      if (jw >= w1) break;
    }
  };
  // MFMA over the words, or (requested) the scalar gather-accumulate product
  const bool scalar = SCA && !TERN && !BLK && a.accum == 1 && !a.dense;  // workgroup-uniform
  if (!scalar && first != 0x7fffffff && (WIDE ? xs < gx : w0 + wave < w1)) {  // wave-uniform
    // with a blocked copy, each wave reads it when its active words have
    // on average at least a.blk_min active rows of 64 counted over the row
    // blocks that read the same words (whole words, shared in L2 by the row
    // blocks, then cost at most 64 / blk_min times the rows' HBM bytes; the
    // rows cost about 128 vector instructions per word), else the rows
    bool blocked = WIDE;
    if constexpr (BLK && !WIDE) {
      int rows = 0, words = 0;
      for (int w = w0 + wave + lane * stride; w < w1; w += 64 * stride) {
        const unsigned long long u = sLU[w];
        rows += __popcll(u);
        words += u != 0ull;
      }
      for (int o = kWave / 2; o > 0; o >>= 1) {
        rows += __shfl_xor(rows, o);
        words += __shfl_xor(words, o);
      }
      blocked = rows * (int)gridDim.y >= words * a.blk_min;
    }
    if (BLK && blocked) loop(load_blocked, mul_blocked);
    else loop(load_rows, mul_rows);
  }
  if (scalar) scalar_accumulate<ROWS, NT>(a, sS, lds_row, sTile, tid, x, y, w0, w1);

  __syncthreads();
  if constexpr (ALIAS) {
    // the tile over the spike rows: wave 0 stores its sums, the others add
    if (wave == 0) store_tile<RT>(acc, sTile, g, c);
    __syncthreads();
    if (wave != 0) reduce_tile<RT>(acc, sTile, g, c);
  } else if (!scalar && !WIDE) {
    reduce_tile<RT>(acc, sTile, g, c);
  }
  if (stats_wg) stats_count<NT>(a, from_parts ? sLU : sStat, &sStatCnt, Kw, tid, lane);
  __syncthreads();
  if (stats_wg && tid == 0) stats_write(a, sStatCnt);
  if constexpr (WIDE) {
    // each wave finishes its own tile from its accumulators (no barrier)
    if (xs < gx) {
      uint32_t* nib = reinterpret_cast<uint32_t*>(sTile) + wave * 256;
      if (a.T == 4) wide_epilogue<4>(a, acc, ep[wave], nib, lane, xs, y);
      else if (a.T == 2) wide_epilogue<2>(a, acc, ep[wave], nib, lane, xs, y);
      else wide_epilogue<1>(a, acc, ep[wave], nib, lane, xs, y);
    }
    return;
  }
  const bool last = !(a.P > 1) || split_fixup<ROWS, NT>(a, sTile, &sLast, tid, x, y, z);
  if (last) epilogue<NW>(a, sTile, ep[0], sUn, tid, lane, wave, x, y);
}

// ------------------------------------------------- LDS-streamed product
// Same tiles and operands as k_qbsm_words, but the active weight rows are
// gathered straight into LDS (global_load_lds_dwordx4: 16 bytes per lane,
// no registers held while in flight).  A word (64 rows x 64 columns) is four
// such loads, each covering 16 rows: lane l takes row 16q + l/4, bytes
// 16(l%4)..16(l%4)+15 of the tile's columns.  Each wave keeps D words in
// flight in a ring of D slots of its own; before using slot i it waits until
// at most 4(D-1) loads are outstanding.  A lane whose row is inactive (or a
// word past the range) loads the block's first active row instead, so every
// word issues exactly four loads and the count stays exact.
constexpr int kDmaChunk = 1088;         // bytes per 16-row chunk: 16 x 64 + 64 (bank offset)
constexpr int kDmaSlot = 4 * kDmaChunk;  // bytes per word slot

template <int D>
__device__ __forceinline__ void dma_wait() {
  if constexpr (D == 1) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if constexpr (D == 2) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if constexpr (D == 3) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(12)" ::: "memory");
}

template <int RT, int NW, int D>
__global__ __launch_bounds__(NW * 64) void k_qbsm_dma(QbsmArgs a) {
  static_assert(D >= 1 && D <= 4, "ring depth");
  constexpr int ROWS = RT * 16;
  constexpr int NT = NW * 64;
  constexpr int kNoRow = 0x7fffffff;
  __shared__ int sTile[ROWS * kTileLd];
  __shared__ unsigned long long sUn[NW];
  __shared__ EpiStage ep;
  __shared__ int sLast;
  __shared__ int sFirst;
  __shared__ int sStatCnt;
  // dynamic: ring [NW][D][kDmaSlot] bytes, local union [Kw] (u64), the block
  // union of the statistics [Kw] (u64), the block's spike rows as dwords with
  // row stride 2*Kw+1
  extern __shared__ __attribute__((aligned(16))) unsigned char sRaw[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  int x, y, z;
  tile_coords(x, y, z);
  const int Kw = (a.K + 63) >> 6;
  const int lds_row = 2 * Kw + 1;
  unsigned char* ring = sRaw + (size_t)wave * D * kDmaSlot;
  unsigned long long* sLU = reinterpret_cast<unsigned long long*>(sRaw + (size_t)NW * D * kDmaSlot);
  unsigned long long* sStat = sLU + Kw;
  uint32_t* sS = reinterpret_cast<uint32_t*>(sStat + Kw);
  const bool stats_wg = a.stats && x == 0 && y == 0 && z == 0;  // workgroup-uniform

  for (int i = tid; i < ROWS * kTileLd; i += NT) sTile[i] = 0;
  if (tid == 0) sFirst = kNoRow;
  stage_epilogue<NT>(a, ep, tid, x, y);
  unsigned long long spart = 0ull;
  if (stats_wg) {
    for (int w = tid; w < Kw; w += NT) sStat[w] = 0ull;
    if (tid == 0) sStatCnt = 0;
    spart = stats_slice<NT>(a, Kw, tid);
  }
  for (int i = tid; i < ROWS * Kw; i += NT) {
    const int lr = i / Kw, w = i - lr * Kw;
    const int t = lr / a.Mb, m = y * a.Mb + (lr - t * a.Mb);
    const unsigned long long v = (t < a.T && m < a.M) ? a.S[(size_t)(t * a.M + m) * Kw + w] : 0ull;
    sS[lr * lds_row + 2 * w] = (uint32_t)v;
    sS[lr * lds_row + 2 * w + 1] = (uint32_t)(v >> 32);
  }
  __syncthreads();
  if (stats_wg) stats_merge<NT>(a, sStat, Kw, tid, spart);
  const unsigned long long last_mask = (a.K & 63) ? (1ull << (a.K & 63)) - 1ull : ~0ull;
  for (int w = tid; w < Kw; w += NT) {
    unsigned long long u = ~0ull;
    if (!a.dense) {
      u = 0ull;
      for (int lr = 0; lr < ROWS; ++lr)
        u |= (unsigned long long)sS[lr * lds_row + 2 * w] |
             ((unsigned long long)sS[lr * lds_row + 2 * w + 1] << 32);
    }
    u = (w == Kw - 1) ? (u & last_mask) : u;
    sLU[w] = u;
    if (u) atomicMin(&sFirst, w * 64 + (int)__builtin_ctzll(u));
  }
  __syncthreads();

  const int w0 = (int)(((long long)Kw * z) / a.P);
  const int w1 = (int)(((long long)Kw * (z + 1)) / a.P);
  const int first = sFirst;

  v4i acc[RT][4];
#pragma unroll
  for (int q = 0; q < RT; ++q)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[q][v] = v4i{0, 0, 0, 0};

  const int jw0 = w0 + wave;
  if (first != kNoRow && jw0 < w1) {  // wave-uniform
    // this lane's part of a 16-row chunk: row rq, 16 bytes at column cbyte
    const int rq = lane >> 2;
    const int cbyte = x * 64 + (lane & 3) * 16;
    const uint32_t ldw = (uint32_t)a.ldw;  // K * ldw < 2^31: 32-bit row offsets
    // 1 when the lane's 16 bytes lie inside the row (the padded width); the
    // masks and the row choice are arithmetic, so that the compiler keeps
    // exactly one load per chunk instead of splitting lanes into branches
    const uint32_t colmask = (uint32_t)((cbyte + 15 - (int)ldw) >> 31) & 1u;
    const char* Wcol = reinterpret_cast<const char*>(a.W) + x * 64 + colmask * (cbyte - x * 64);
    auto issue = [&](int w, int slot) {
      const unsigned long long u = (w < w1) ? sLU[w] : 0ull;
      unsigned char* dst = ring + slot * kDmaSlot;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t on = (uint32_t)(u >> (16 * q + rq)) & colmask;
        const uint32_t row = (uint32_t)first + on * ((uint32_t)(w * 64 + 16 * q + rq) - (uint32_t)first);
        __builtin_amdgcn_global_load_lds(Wcol + row * ldw, dst + q * kDmaChunk, 16, 0, 0);
      }
      asm volatile("" ::: "memory");
    };
    const int nw = (w1 - jw0 + NW - 1) / NW;
#pragma unroll
    for (int i = 0; i < D; ++i) issue(jw0 + i * NW, i);
    for (int i = 0; i < nw; ++i) {
      const int w = jw0 + i * NW;
      const int slot = i % D;
      dma_wait<D>();
      const unsigned long long u = sLU[w];
      if (u) {  // wave-uniform
        const unsigned char* src = ring + slot * kDmaSlot + g * kDmaChunk + 4 * c;
        uint32_t xg[16];
#pragma unroll
        for (int s2 = 0; s2 < 16; ++s2) xg[s2] = *reinterpret_cast<const uint32_t*>(src + s2 * 64);
        v4i b[4];
        b_operands(xg, b);
#pragma unroll
        for (int q = 0; q < RT; ++q) {
          const uint32_t b16 =
              (sS[(q * 16 + c) * lds_row + 2 * w + (g >> 1)] >> (16 * (g & 1))) & 0xFFFFu;
          const v4i af = a_operand(b16);
#pragma unroll
          for (int v = 0; v < 4; ++v)
            acc[q][v] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, b[v], acc[q][v], 0, 0, 0);
        }
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // slot reads done before it is refilled
      issue(w + D * NW, slot);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // no LDS write in flight past the loop
  }

  __syncthreads();
  reduce_tile<RT>(acc, sTile, g, c);
  if (stats_wg) stats_count<NT>(a, sStat, &sStatCnt, Kw, tid, lane);
  __syncthreads();
  if (stats_wg && tid == 0) stats_write(a, sStatCnt);
  const bool last = !(a.P > 1) || split_fixup<ROWS, NT>(a, sTile, &sLast, tid, x, y, z);
  if (last) epilogue<NW>(a, sTile, ep, sUn, tid, lane, wave, x, y);
}

// -------------------------------------------------------------- single kernel
template <int RT, int NW>
__global__ __launch_bounds__(NW * 64) void k_qbsm_fused(QbsmArgs a) {
  constexpr int ROWS = RT * 16;
  constexpr int NT = NW * 64;
  constexpr int CH = NW * kGroup;  // k-steps per chunk
  __shared__ int sTile[ROWS * kTileLd];
  __shared__ __attribute__((aligned(16))) uint32_t sOff[CH * 64];
  __shared__ __attribute__((aligned(16))) int sIdx[CH * 64];
  __shared__ unsigned long long sU[kFusedMaxWords];
  __shared__ int sP[kFusedMaxWords + 1];
  __shared__ int sWave[NW];
  __shared__ unsigned long long sUn[NW];
  // compacted bits per wave/step/row; before the main loop also the column-OR
  // scratch of up to NT words
  constexpr int kBitsLen = (NW * kGroup * ROWS > NT) ? NW * kGroup * ROWS : NT;
  __shared__ unsigned long long sBits[kBitsLen];
  __shared__ EpiStage ep;
  __shared__ int sLast;
  // this tile's spike rows as dwords, row stride 2*Kw+1 (odd: the rows a
  // wave reads at one active row fall in different banks)
  extern __shared__ uint32_t sS[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  int x, y, z;
  tile_coords(x, y, z);
  const int R = a.T * a.M;
  const int Kw = (a.K + 63) >> 6;
  const int lds_row = 2 * Kw + 1;

  // ---- prologue: every global load here is independent of the others
  for (int i = tid; i < ROWS * kTileLd; i += NT) sTile[i] = 0;
  stage_epilogue<NT>(a, ep, tid, x, y);
  for (int i = tid; i < ROWS * Kw; i += NT) {
    const int lr = i / Kw, w = i - lr * Kw;
    const int t = lr / a.Mb, m = y * a.Mb + (lr - t * a.Mb);
    const unsigned long long v = (t < a.T && m < a.M) ? a.S[(size_t)(t * a.M + m) * Kw + w] : 0ull;
    sS[lr * lds_row + 2 * w] = (uint32_t)v;
    sS[lr * lds_row + 2 * w + 1] = (uint32_t)(v >> 32);
  }
  const unsigned long long last_mask = (a.K & 63) ? (1ull << (a.K & 63)) - 1ull : ~0ull;
  if (a.dense || a.upart) {
    for (int w = tid; w < Kw; w += NT) {
      unsigned long long u = ~0ull;
      if (!a.dense) {
        u = 0ull;
        for (int q = 0; q < a.nparts; ++q) u |= a.upart[(size_t)q * Kw + w];
      }
      sU[w] = (w == Kw - 1) ? (u & last_mask) : u;
    }
  } else {
    // column OR of all R rows (R*Kw is bounded by the host): rg row groups
    // per word into a scratch table, then one pass over the groups
    const int rg = max(1, NT / Kw);
    unsigned long long* sOr = sBits;  // free until the main loop
    if (tid < rg * Kw) {
      const int w = tid % Kw, r0 = tid / Kw;
      unsigned long long u = 0;
      for (int r = r0; r < R; r += rg) u |= a.S[(size_t)r * Kw + w];
      sOr[r0 * Kw + w] = u;
    }
    __syncthreads();
    for (int w = tid; w < Kw; w += NT) {
      unsigned long long u = 0;
      for (int q = 0; q < rg; ++q) u |= sOr[q * Kw + w];
      sU[w] = (w == Kw - 1) ? (u & last_mask) : u;
    }
  }
  __syncthreads();
  // prefix popcounts (Kw <= NT: one word per thread)
  const int cnt = tid < Kw ? __popcll(sU[tid]) : 0;
  int incl = cnt;
  for (int o = 1; o < kWave; o <<= 1) {
    const int v = __shfl_up(incl, o);
    if (lane >= o) incl += v;
  }
  if (lane == kWave - 1) sWave[wave] = incl;
  __syncthreads();
  int before = 0, ka = 0;
  for (int i = 0; i < NW; ++i) {
    if (i < wave) before += sWave[i];
    ka += sWave[i];
  }
  if (tid < Kw) sP[tid] = before + incl - cnt;
  if (tid == 0) sP[Kw] = ka;
  if (a.stats && tid == 0 && x == 0 && y == 0 && z == 0) {
    a.stats->k_total = a.K;
    a.stats->k_active = ka;
    a.stats->n = a.N;
    a.stats->weight_bytes = (int64_t)ka * (int64_t)a.N;
  }
  __syncthreads();

  const int KS = (ka + 63) >> 6;
  const int ks0 = (int)(((long long)KS * z) / a.P);
  const int ks1 = (int)(((long long)KS * (z + 1)) / a.P);
  const uint32_t colb = (x * 64 + 4 * c < a.N) ? (uint32_t)(x * 64 + 4 * c) : (uint32_t)(x * 64);
  const char* Wb = reinterpret_cast<const char*>(a.W) + colb;

  v4i acc[RT][4];
#pragma unroll
  for (int q = 0; q < RT; ++q)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[q][v] = v4i{0, 0, 0, 0};

  for (int cs = ks0; cs < ks1; cs += CH) {
    const int ce = min(cs + CH, ks1);
    const int e0 = cs * 64, e1 = min(ce * 64, ka);
    __syncthreads();  // previous chunk's list and bits are consumed
    // list entries [e0, e1): one union word per wave, one bit per lane, rank
    // by masked popcount; entries past e1 in the chunk point at row 0
    for (int i = (e1 - e0) + tid; i < CH * 64; i += NT) {
      sIdx[i] = -1;
      sOff[i] = 0u;
    }
    for (int w = wave; w < Kw; w += NW) {
      const int p0 = sP[w];
      if (p0 >= e1 || sP[w + 1] <= e0) continue;  // wave-uniform
      const unsigned long long u = sU[w];
      const int e = p0 + __popcll(u & ((1ull << lane) - 1ull));
      if (((u >> lane) & 1ull) && e >= e0 && e < e1) {
        const int k = w * 64 + lane;
        sIdx[e - e0] = k;
        sOff[e - e0] = (uint32_t)k * (uint32_t)a.ldw;
      }
    }
    __syncthreads();
    const int jb = cs + wave * kGroup;
    const int nv = min(kGroup, ce - jb);
    if (nv <= 0) continue;  // wave-uniform

    // weight loads of the whole group first
    uint32_t xw[kGroup][16];
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const uint4* po = reinterpret_cast<const uint4*>(sOff + (wave * kGroup + i) * 64 + 16 * g);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint4 o = po[u];
        xw[i][4 * u + 0] = *reinterpret_cast<const uint32_t*>(Wb + o.x);
        xw[i][4 * u + 1] = *reinterpret_cast<const uint32_t*>(Wb + o.y);
        xw[i][4 * u + 2] = *reinterpret_cast<const uint32_t*>(Wb + o.z);
        xw[i][4 * u + 3] = *reinterpret_cast<const uint32_t*>(Wb + o.w);
      }
    }
    // while they are in flight: compact the spike bits of the tile rows onto
    // this wave's active rows (lane = active row, one ballot per tile row)
    unsigned long long* myBits = sBits + wave * kGroup * ROWS;
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const int k = sIdx[(wave * kGroup + i) * 64 + lane];
      const int kd = max(k, 0) >> 5, kb = k & 31;
#pragma unroll
      for (int lr = 0; lr < ROWS; ++lr) {
        const bool bit = k >= 0 && ((sS[lr * lds_row + kd] >> kb) & 1u);
        const unsigned long long m = __builtin_amdgcn_ballot_w64(bit);
        if (lane == 0) myBits[i * ROWS + lr] = m;
      }
    }
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      v4i b[4];
      b_operands(xw[i], b);
#pragma unroll
      for (int q = 0; q < RT; ++q) {
        const uint32_t b16 = (uint32_t)(myBits[i * ROWS + q * 16 + c] >> (16 * g)) & 0xFFFFu;
        const v4i af = a_operand(b16);
#pragma unroll
        for (int v = 0; v < 4; ++v)
          acc[q][v] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, b[v], acc[q][v], 0, 0, 0);
      }
    }
  }

  __syncthreads();
  reduce_tile<RT>(acc, sTile, g, c);
  __syncthreads();
  if (a.P > 1 && !split_fixup<ROWS, NT>(a, sTile, &sLast, tid, x, y, z)) return;
  epilogue<NW>(a, sTile, ep, sUn, tid, lane, wave, x, y);
}

// ------------------------------------------------- list from the prep pass
template <int RT, int NW>
__global__ __launch_bounds__(NW * 64) void k_qbsm_list(QbsmArgs a) {
  constexpr int ROWS = RT * 16;
  constexpr int NT = NW * 64;
  constexpr int CH = NW * kGroup;
  __shared__ int sTile[ROWS * kTileLd];
  __shared__ __attribute__((aligned(16))) uint32_t sOff[CH * 64];
  __shared__ unsigned long long sUn[NW];
  __shared__ EpiStage ep;
  __shared__ int sLast;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  int x, y, z;
  tile_coords(x, y, z);
  const int R = a.T * a.M;

  for (int i = tid; i < ROWS * kTileLd; i += NT) sTile[i] = 0;
  stage_epilogue<NT>(a, ep, tid, x, y);
  const int ka = *a.kact;
  const int KS = (ka + 63) >> 6;
  const int ks0 = (int)(((long long)KS * z) / a.P);
  const int ks1 = (int)(((long long)KS * (z + 1)) / a.P);

  int rowq[RT];
  bool rowv[RT];
#pragma unroll
  for (int q = 0; q < RT; ++q) {
    const int jr = q * 16 + c;
    const int t = jr / a.Mb, ml = jr - t * a.Mb, m = y * a.Mb + ml;
    rowv[q] = t < a.T && m < a.M;
    rowq[q] = rowv[q] ? t * a.M + m : 0;
  }
  const uint32_t colb = (x * 64 + 4 * c < a.N) ? (uint32_t)(x * 64 + 4 * c) : (uint32_t)(x * 64);
  const char* Wb = reinterpret_cast<const char*>(a.W) + colb;
  const uint32_t* sc32 = reinterpret_cast<const uint32_t*>(a.sc);

  v4i acc[RT][4];
#pragma unroll
  for (int q = 0; q < RT; ++q)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[q][v] = v4i{0, 0, 0, 0};

  for (int cs = ks0; cs < ks1; cs += CH) {
    const int ce = min(cs + CH, ks1);
    __syncthreads();
    for (int i = tid; i < CH * 64; i += NT)
      sOff[i] = (cs * 64 + i < ce * 64) ? a.act_off[(size_t)cs * 64 + i] : 0u;
    __syncthreads();
    const int jb = cs + wave * kGroup;
    const int nv = min(kGroup, ce - jb);
    if (nv <= 0) continue;  // wave-uniform

    uint32_t xw[kGroup][16];
    uint32_t bits[kGroup][RT];
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const uint4* po = reinterpret_cast<const uint4*>(sOff + (wave * kGroup + i) * 64 + 16 * g);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint4 o = po[u];
        xw[i][4 * u + 0] = *reinterpret_cast<const uint32_t*>(Wb + o.x);
        xw[i][4 * u + 1] = *reinterpret_cast<const uint32_t*>(Wb + o.y);
        xw[i][4 * u + 2] = *reinterpret_cast<const uint32_t*>(Wb + o.z);
        xw[i][4 * u + 3] = *reinterpret_cast<const uint32_t*>(Wb + o.w);
      }
    }
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const int j = min(jb + i, ce - 1);
#pragma unroll
      for (int q = 0; q < RT; ++q) {
        const uint32_t raw = sc32[((size_t)j * R + rowq[q]) * 2 + (g >> 1)];
        bits[i][q] = (rowv[q] && i < nv) ? (raw >> ((g & 1) * 16)) & 0xFFFFu : 0u;
      }
    }
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      v4i b[4];
      b_operands(xw[i], b);
#pragma unroll
      for (int q = 0; q < RT; ++q) {
        const v4i af = a_operand(bits[i][q]);
#pragma unroll
        for (int v = 0; v < 4; ++v)
          acc[q][v] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, b[v], acc[q][v], 0, 0, 0);
      }
    }
  }

  __syncthreads();
  reduce_tile<RT>(acc, sTile, g, c);
  __syncthreads();
  if (a.P > 1 && !split_fixup<ROWS, NT>(a, sTile, &sLast, tid, x, y, z)) return;
  epilogue<NW>(a, sTile, ep, sUn, tid, lane, wave, x, y);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
constexpr size_t kWordsLdsBudget = 81920;  // word product: two workgroups per CU fit in LDS
constexpr int kWideMinTiles = 1536;  // output tiles (64 x 64) from which blocked products go wide
constexpr int kCus = 256;            // compute units of the device
// resident threads per compute unit of the word kernel: its variants take
// 74-128 registers, four or five waves per SIMD, 16-20 waves per CU
constexpr int kThreadsPerCu = 1024;

// Waves per workgroup of the word product: 16 for one row group with more
// than 32 words of K, 8 for up to two row groups with 8 or more, else 4.
static int words_waves(int RT, int kwords) {
  return (kwords > 32 && RT == 1) ? 16 : ((kwords >= 4 * kGroup && RT <= 2) ? 8 : 4);
}

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
  s->U = cv.take<uint64_t>((size_t)((L.Kmax + 63) / 64));
  // K-split accumulators: one (row tile x 64 columns) tile per output tile;
  // the row tiles cover at most R + 128 rows
  const size_t rows_cap = L.split_rows > 0 ? (size_t)L.split_rows + 128 : 0;
  s->part_elems = rows_cap * align_up((size_t)L.split_N, 64);
  s->part = s->part_elems ? cv.take<int32_t>(s->part_elems) : nullptr;
  s->n_counters = (size_t)L.tiles_max;
  s->counters = cv.take<int32_t>(s->n_counters);
}

// Product launches: hipExtLaunchKernelGGL stamps the optional start/stop
// events from the kernel's own dispatch (no marker packets around it).
template <int RT, int NW>
static void launch_fused(const dim3& grid, const QbsmArgs& a, size_t dyn, hipStream_t st,
                         hipEvent_t e0, hipEvent_t e1) {
  hipExtLaunchKernelGGL((k_qbsm_fused<RT, NW>), grid, dim3(NW * 64), (uint32_t)dyn, st, e0, e1, 0, a);
}

template <int RT, int NW>
static nmdlm_status launch_words(const dim3& grid, const QbsmArgs& a, size_t dyn, hipStream_t st,
                                 hipEvent_t e0, hipEvent_t e1, bool wide = false) {
  // wide tiles: NW column tiles per workgroup over the blocked weights
  if constexpr (RT == 4 && NW == 4) {
    if (wide) {
      const void* fn = reinterpret_cast<const void*>(&k_qbsm_words<4, 4, false, true, false, true>);
      if (dyn > 65536 &&
          hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn) != hipSuccess)
        return NMDLM_ERR_HIP;
      hipExtLaunchKernelGGL((k_qbsm_words<4, 4, false, true, false, true>), grid, dim3(256),
                            (uint32_t)dyn, st, e0, e1, 0, a);
      return NMDLM_OK;
    }
  }
  // blocked weights: the variant loading operand-order words
  if (a.Wb) {
    if (dyn > 65536 &&
        hipFuncSetAttribute(reinterpret_cast<const void*>(&k_qbsm_words<RT, NW, false, true>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn) != hipSuccess)
      return NMDLM_ERR_HIP;
    hipExtLaunchKernelGGL((k_qbsm_words<RT, NW, false, true>), grid, dim3(NW * 64), (uint32_t)dyn,
                          st, e0, e1, 0, a);
    return NMDLM_OK;
  }
  // ternary input (-1 spikes given): the variant staging both spike planes
  if (a.Sn) {
    if (dyn > 65536 &&
        hipFuncSetAttribute(reinterpret_cast<const void*>(&k_qbsm_words<RT, NW, true>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn) != hipSuccess)
      return NMDLM_ERR_HIP;
    hipExtLaunchKernelGGL((k_qbsm_words<RT, NW, true>), grid, dim3(NW * 64), (uint32_t)dyn, st, e0,
                          e1, 0, a);
    return NMDLM_OK;
  }
  // the scalar gather-accumulate product (requested path 5)
  if (a.accum == 1) {
    if (dyn > 65536 &&
        hipFuncSetAttribute(reinterpret_cast<const void*>(&k_qbsm_words<RT, NW, false, false, true>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn) != hipSuccess)
      return NMDLM_ERR_HIP;
    hipExtLaunchKernelGGL((k_qbsm_words<RT, NW, false, false, true>), grid, dim3(NW * 64),
                          (uint32_t)dyn, st, e0, e1, 0, a);
    return NMDLM_OK;
  }
  if (dyn > 65536 &&
      hipFuncSetAttribute(reinterpret_cast<const void*>(&k_qbsm_words<RT, NW>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn) != hipSuccess)
    return NMDLM_ERR_HIP;
  hipExtLaunchKernelGGL((k_qbsm_words<RT, NW>), grid, dim3(NW * 64), (uint32_t)dyn, st, e0, e1, 0, a);
  return NMDLM_OK;
}

template <int RT, int NW, int D>
static nmdlm_status launch_dma(const dim3& grid, const QbsmArgs& a, size_t dyn, hipStream_t st,
                               hipEvent_t e0, hipEvent_t e1) {
  if (dyn > 65536 &&
      hipFuncSetAttribute(reinterpret_cast<const void*>(&k_qbsm_dma<RT, NW, D>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn) != hipSuccess)
    return NMDLM_ERR_HIP;
  hipExtLaunchKernelGGL((k_qbsm_dma<RT, NW, D>), grid, dim3(NW * 64), (uint32_t)dyn, st, e0, e1, 0, a);
  return NMDLM_OK;
}

// Static LDS of k_qbsm_dma (mirrors its declarations) and its dynamic part.
static size_t dma_lds(int RT, int NW, int D, int Kw) {
  return (size_t)RT * 16 * kTileLd * 4 + (size_t)NW * 12 + sizeof(EpiStage) + 64 +
         (size_t)NW * D * kDmaSlot + (size_t)Kw * 16 + (size_t)RT * 16 * (2 * Kw + 1) * 4;
}
constexpr size_t kDmaLdsMax = 163840;  // LDS per workgroup on the device

template <int RT, int NW>
static void launch_list(const dim3& grid, const QbsmArgs& a, hipStream_t st, hipEvent_t e0,
                        hipEvent_t e1) {
  hipExtLaunchKernelGGL((k_qbsm_list<RT, NW>), grid, dim3(NW * 64), 0u, st, e0, e1, 0, a);
}

// Blocked weight layout (see weight_blocked_bytes): thread i writes the
// 16-byte operand lane i % 64 of operand (i / 64) % 4 of block i / 256, each
// byte read from the row-major weights (zero past K or N).
__global__ __launch_bounds__(256) void k_weight_block(const int8_t* __restrict__ W, int K, int N,
                                                      int64_t ldw, int8_t* __restrict__ Wb,
                                                      long long n_lanes) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_lanes) return;
  const int gx = (N + 63) / 64;
  const int lane = (int)(i & 63), v = (int)((i >> 6) & 3);
  const long long blk = i >> 8;
  const int x = (int)(blk % gx), w = (int)(blk / gx);
  const int g = lane >> 4, c = lane & 15;
  const int col = x * 64 + 4 * c + v;
  uint32_t q[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    uint32_t d = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int row = w * 64 + 16 * g + 4 * e + b;
      const uint32_t byte = (row < K && col < N) ? (uint8_t)W[(int64_t)row * ldw + col] : 0u;
      d |= byte << (8 * b);
    }
    q[e] = d;
  }
  *reinterpret_cast<uint4*>(Wb + i * 16) = uint4{q[0], q[1], q[2], q[3]};
}

nmdlm_status launch_weight_block(const int8_t* W, int K, int N, int64_t ldw, int8_t* Wb,
                                 hipStream_t st) {
  const long long n_lanes = (long long)(weight_blocked_bytes(K, N) / 16);
  if (n_lanes == 0) return NMDLM_OK;
  hipLaunchKernelGGL(k_weight_block, dim3((unsigned)((n_lanes + 255) / 256)), dim3(256), 0, st, W, K,
                     N, ldw, Wb, n_lanes);
  return hip_status();
}

// Static LDS of k_qbsm_words<RT, NW> and its dynamic part (mirror the declarations).
// 64-row tiles of the one-tile kernel (not the scalar variant) keep the
// reduction tile in the dynamic part, over the spike rows.
static bool words_alias(int RT, bool wide, bool sca) { return RT == 4 && !wide && !sca; }
static size_t words_dyn(int RT, int Kw, bool tern = false, bool wide = false, bool sca = false) {
  const size_t rows = (size_t)RT * 16 * (2 * Kw + 1) * 4 * (tern ? 2 : 1);
  const size_t tile = (size_t)RT * 16 * kTileLd * 4;
  return (size_t)Kw * 16 + (words_alias(RT, wide, sca) ? std::max(rows, tile) : rows);
}
static size_t words_lds(int RT, int NW, int Kw, bool tern = false, bool wide = false,
                        bool sca = false) {
  const size_t tile = wide ? (size_t)NW * 1024
                           : (words_alias(RT, wide, sca) ? 4 : (size_t)RT * 16 * kTileLd * 4);
  return tile + (size_t)NW * 12 + sizeof(EpiStage) * (wide ? NW : 1) + 64 +
         words_dyn(RT, Kw, tern, wide, sca);
}

// Static LDS of k_qbsm_fused<RT, NW> (mirrors its declarations).
static size_t fused_static_lds(int RT, int NW) {
  const size_t ch = (size_t)NW * kGroup * 64;
  const size_t bits = std::max((size_t)NW * kGroup * RT * 16, (size_t)NW * 64);
  return (size_t)RT * 16 * kTileLd * 4 + ch * 4 * 2 + kFusedMaxWords * 8 + (kFusedMaxWords + 1) * 4 +
         (size_t)NW * 12 + bits * 8 + sizeof(EpiStage) + 64;
}

nmdlm_status launch_qbsm(const QbsmCall& c, const QbsmScratch& scr, hipStream_t st, int* gy_out) {
  const int R = c.T * c.M;
  const int Kw = (c.K + 63) / 64;
  const int dense = (c.flags & NMDLM_FORCE_DENSE) ? 1 : 0;
  const int gx = (c.N + 63) / 64;
  bool has_tr = false;
  if (c.mode == EPI_IF || c.mode == EPI_QNL_IF)
    for (int i = 0; i < c.nseg; ++i) has_tr = has_tr || c.seg[i].transposed;

  // product path: 1 = prep pass + list kernel, 2 = single kernel with a
  // compacted list, 3 = word-granular single kernel, 0 = automatic
  int path = (int)((c.flags >> NMDLM_PATH_SHIFT) & 0x7u);
  const bool path_auto = path == 0;
  const int rt_full = pick_rt(R);
  int RT = (int)((c.flags >> NMDLM_ROWTILE_SHIFT) & 0xFu);
  const bool rt_forced = (RT == 1 || RT == 2 || RT == 4 || RT == 8);
  if (!rt_forced) {
    // rows per tile group (at most 4): the largest that gives >= 512
    // workgroups all resident at once (256 CUs x 1024 threads), else >= 256
    // resident, else 1 (the most row blocks; they re-read weights from L2)
    RT = 1;
    bool found = false;
    for (int want = 512; want >= 256 && !found; want /= 2) {
      for (int r = std::min(rt_full, 4); r >= 1; r >>= 1) {
        const int mb = (16 * r) / c.T;
        if (mb < 1) continue;
        const long long wgs = (long long)gx * ((c.M + mb - 1) / mb);
        const int nw = words_waves(r, Kw);
        if (wgs >= want && wgs * nw * 64 <= (long long)kCus * kThreadsPerCu) {
          RT = r;
          found = true;
          break;
        }
      }
    }
    if (!found) {
      // no height keeps the grid resident: when even the tallest tiles
      // oversubscribe the chip, they re-read each weight tile the fewest times
      const int r = std::min(rt_full, 4), mb = (16 * r) / c.T;
      if (mb >= 1) {
        const long long wgs = (long long)gx * ((c.M + mb - 1) / mb);
        if (wgs * words_waves(r, Kw) * 64 > (long long)kCus * kThreadsPerCu) RT = r;
      }
    }
    // a channel-major output segment is written in whole bytes when a row
    // block's tokens fill them: take the fewest rows that do, if the grid
    // keeps >= 256 workgroups
    bool pos_ok = true;
    for (int i = 0; i < c.nseg; ++i)
      if (c.seg[i].transposed && (c.seg[i].pos0 & 7)) pos_ok = false;
    if (has_tr && pos_ok) {
      for (int r = RT; r <= 8; r <<= 1) {
        const int mb = (16 * r) / c.T;
        if (mb > 32) break;
        if (mb % 8 == 0) {
          if (r == RT || (long long)gx * ((c.M + mb - 1) / mb) >= 256) RT = r;
          break;
        }
      }
    }
  }
  while (RT > 1 && 16 * RT / 2 >= R && 16 * RT / 2 >= c.T) RT >>= 1;  // no empty tiles
  while (has_tr && RT > 1 && (16 * RT) / c.T > 32) RT >>= 1;  // channel-major: <= 32 tokens
  if (has_tr && c.seq_len > 0) {
    // several sequences: a channel-major segment keeps every row block
    // within one sequence
    while (RT > 1 && c.seq_len % ((16 * RT) / c.T) != 0) RT >>= 1;
    if (16 * RT < c.T || c.seq_len % ((16 * RT) / c.T) != 0) return NMDLM_ERR_UNSUPPORTED;
  }
  const bool tern = c.s_neg != nullptr;
  // wide tiles (a workgroup takes four 64-column tiles of a 64-row block,
  // each wave one tile over all of K, the IF in registers): requested by
  // path 7, or unrequested for blocked products of many output tiles, where
  // the one-tile kernel would repeat the staging, union and reduction of a
  // row block for every column tile.  Decided before the LDS limits of the
  // one-tile kernel: the wide variant holds no LDS tile and may take all of
  // a CU's LDS.
  bool wide = false;
  if (c.Wb && !tern && (path == 0 || path == 7) && RT == 4 &&
      ((c.flags >> NMDLM_SPLIT_SHIFT) & 0xFFu) <= 1u && (c.T == 1 || c.T == 2 || c.T == 4) &&
      (c.mode == EPI_CUR || c.mode == EPI_IF || c.mode == EPI_QNL_IF || c.mode == EPI_HEAD) &&
      words_lds(4, 4, Kw, false, true) <= kDmaLdsMax) {
    const int mb4 = 64 / c.T;
    const long long tiles4 = (long long)gx * ((c.M + mb4 - 1) / mb4);
    wide = path == 7 || tiles4 >= kWideMinTiles;
  }
  if (tern) {
    // ternary input: the word product only (both spike planes staged)
    path = 3;
    while (RT > 1 && words_lds(RT, 4, Kw, true) > kWordsLdsBudget && !rt_forced) RT >>= 1;
    if (words_lds(RT, 4, Kw, true) > kWordsLdsBudget || Kw > 256) return NMDLM_ERR_UNSUPPORTED;
  }
  if (path == 0 && !wide) {
    path = 3;
    while (RT > 1 && words_lds(RT, 4, Kw) > kWordsLdsBudget && !rt_forced) RT >>= 1;
    if (words_lds(RT, 4, Kw) > kWordsLdsBudget) path = 1;
  }
  // 5: the word product with the scalar gather-accumulate product
  int accum = 0;
  if (path == 5) {
    accum = 1;
    path = 3;
  }
  // 6: the word product over blocked weights (requested: every wave reads
  // the copy; unrequested, with a copy: each wave chooses by its union);
  // 7: as 6 with wide tiles where the row tile is 64 rows
  bool blk = false;
  int blk_min = kBlockedMinRows;
  if (wide) {
    blk = true;
    blk_min = 0;
    path = 3;
  } else if (path == 7) {
    path = 6;
  }
  if (path == 6) {
    if (!c.Wb || tern) return NMDLM_ERR_UNSUPPORTED;
    blk = true;
    blk_min = 0;
    path = 3;
    while (RT > 1 && words_lds(RT, 4, Kw) > kWordsLdsBudget && !rt_forced) RT >>= 1;
    if (words_lds(RT, 4, Kw) > kWordsLdsBudget) return NMDLM_ERR_UNSUPPORTED;
  } else if (path_auto && path == 3 && c.Wb && !tern) {
    blk = true;
  }
  if (path == 3 && !wide && words_lds(RT, 4, Kw, tern, false, accum == 1) > kWordsLdsBudget) path = 1;
  if (path == 4 && dma_lds(RT, 4, 4, Kw) > kDmaLdsMax) path = 1;
  if (path > 4) path = 1;
  if (16 * RT < c.T) return NMDLM_ERR_UNSUPPORTED;
  const int Mb = (16 * RT) / c.T;
  // the tile heights lowered for LDS above keep a channel-major segment's
  // row blocks within one sequence, or the call is refused
  if (has_tr && c.seq_len > 0 && c.seq_len % Mb != 0) return NMDLM_ERR_UNSUPPORTED;
  const int gy = (c.M + Mb - 1) / Mb;
  const int tiles = gx * gy;
  if ((size_t)tiles > scr.n_counters) return NMDLM_ERR_WORKSPACE;
  if (gy_out) *gy_out = gy;

  // K splits: requested by the flags, or, unrequested, four ways for a short
  // grid over a long K (at most 64 output tiles, K of 128 words or more:
  // 256 workgroups then share the weight rows instead of 64).  Elsewhere the
  // atomic accumulation costs more round trips than the split saves.
  int P = (int)((c.flags >> NMDLM_SPLIT_SHIFT) & 0xFFu);
  if (P == 0 && path == 3 && !tern && !wide && tiles <= 64 && Kw >= 128) P = 4;
  P = std::max(1, std::min(P, Kw));
  const size_t acc_elems = (size_t)16 * RT * 64 * (size_t)tiles;  // one accumulator tile per output tile
  if (P > 1 && (!scr.part || scr.part_elems < acc_elems)) P = 1;
  // waves per workgroup: many when each workgroup has many k-steps
  const int ks_per_wg = (Kw + P - 1) / P;
  int NW = (ks_per_wg >= 8 * kGroup && RT <= 2) ? 16 : 4;
  size_t dyn = 0;
  bool fused = false, words = false, dma = false;
  int D = 1;
  if (path == 4) {
    // LDS-streamed: 8 waves x 2 words in flight, or 4 waves x 4 words
    dma = true;
    NW = (ks_per_wg >= 16 && RT <= 4) ? 8 : 4;
    D = NW == 8 ? 2 : 4;
    if (dma_lds(RT, NW, D, Kw) > kDmaLdsMax) { NW = 4; D = 4; }
    dyn = dma_lds(RT, NW, D, Kw) - ((size_t)RT * 16 * kTileLd * 4 + (size_t)NW * 12 + sizeof(EpiStage) + 64);
  } else if (path == 3) {
    words = true;
    // 8 waves, not 16: a 1024-thread bound caps registers at 128 and spills
    NW = words_waves(RT, ks_per_wg);
    if (words_lds(RT, NW, Kw) > kWordsLdsBudget) NW = 4;
    if (words_lds(RT, NW, Kw, tern) > kWordsLdsBudget) NW = 4;
    dyn = words_dyn(RT, Kw, tern, wide, accum == 1);
  } else if (path == 2) {
    // one kernel (union, list and spike compaction in LDS) when the tile's
    // spike rows fit; else the prep pass builds them in global memory
    dyn = (size_t)16 * RT * (2 * Kw + 1) * 4;
    fused = Kw <= kFusedMaxWords && RT <= 2;
    if (fused && RT == 2) NW = 4;  // the 16-wave variant of RT=2 would spill registers
    if (fused && fused_static_lds(RT, NW) + dyn > kLdsBudget) NW = 4;
    if (fused && fused_static_lds(RT, NW) + dyn > kLdsBudget) fused = false;
    if (fused && !c.u_in && !dense && (long long)R * Kw > kUnionDirect) fused = false;
  }

  const int gxl = wide ? (gx + 3) / 4 : gx;  // grid columns
  if (wide) NW = 4;

  nmdlm_status rc0 = NMDLM_OK;
  PrepArgs pa;
  pa.S = c.s_in;
  pa.R = R;
  pa.Kw = Kw;
  pa.K = c.K;
  pa.upart = c.u_in;
  pa.nparts = c.u_nparts;
  pa.dense = dense;
  pa.ldw = (uint32_t)c.ldw;
  pa.N = c.N;
  pa.act_off = scr.act_off;
  pa.act_idx = scr.act_idx;
  pa.kact = scr.kact;
  pa.stats = c.stats;
  pa.counters = scr.counters;
  pa.n_counters = tiles;
  pa.sc = scr.sc;
  if (!fused && !words && !dma) {
    if (!dense && !pa.upart && (long long)R * Kw > kUnionDirect) {
      hipLaunchKernelGGL(k_union, dim3(Kw), dim3(256), 0, st, c.s_in, R, Kw, scr.U);
      pa.upart = scr.U;
      pa.nparts = 1;
    }
    hipLaunchKernelGGL(k_prep, dim3(Kw, (R + kPrepRows - 1) / kPrepRows), dim3(256), 0, st, pa);
  }
  // a split product accumulates into the zeroed split region (accumulators
  // and counters), which its last arrivers leave zero again
  if (P > 1 && tiles > 0) {
    int32_t* base = scr.part ? scr.part : scr.counters;
    if ((rc0 = launch_fill_zero(base, (size_t)split_region_elems(scr) * 4, st)) != NMDLM_OK) return rc0;
  }

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
  a.u_out = c.u_out;
  a.u_ld = gx;
  a.inv_gy = 1.0f / (float)gy;
  a.inv_kw = 1.0f / (float)Kw;
  a.inv_mb = 1.0f / (float)Mb;
  a.inv_segw = 1.0f / (float)std::max(1, std::min(c.seg_w, 1 << 22));
  a.inv_gxy = 1.0f / (float)((long long)gxl * gy);
  a.S = c.s_in;
  a.Sn = c.s_neg;
  a.upart = pa.upart;
  a.nparts = pa.nparts;
  a.dense = dense;
  a.stats = c.stats;
  a.thr_num = c.thr_num;
  a.thr_den = c.thr_den;
  a.s_neg_out = c.s_neg_out;
  a.v_out = c.v_out;
  a.accum = accum;
  a.Wb = blk ? c.Wb : nullptr;
  a.blk_min = blk_min;

  const dim3 grid(gxl, gy, P);
  hipEvent_t e0 = c.ev_begin, e1 = c.ev_end;
  if (dma) {
    nmdlm_status rd = NMDLM_OK;
    if (NW == 8) {
      switch (RT) {
        case 1: rd = launch_dma<1, 8, 2>(grid, a, dyn, st, e0, e1); break;
        case 2: rd = launch_dma<2, 8, 2>(grid, a, dyn, st, e0, e1); break;
        default: rd = launch_dma<4, 8, 2>(grid, a, dyn, st, e0, e1); break;
      }
    } else {
      switch (RT) {
        case 1: rd = launch_dma<1, 4, 4>(grid, a, dyn, st, e0, e1); break;
        case 2: rd = launch_dma<2, 4, 4>(grid, a, dyn, st, e0, e1); break;
        case 4: rd = launch_dma<4, 4, 4>(grid, a, dyn, st, e0, e1); break;
        default: rd = launch_dma<8, 4, 4>(grid, a, dyn, st, e0, e1); break;
      }
    }
    if (rd != NMDLM_OK) return rd;
  } else if (words) {
    nmdlm_status rw = NMDLM_OK;
    if (NW == 16) {
      rw = launch_words<1, 16>(grid, a, dyn, st, e0, e1);
    } else if (NW == 8) {
      if (RT == 1) rw = launch_words<1, 8>(grid, a, dyn, st, e0, e1);
      else rw = launch_words<2, 8>(grid, a, dyn, st, e0, e1);
    } else {
      switch (RT) {
        case 1: rw = launch_words<1, 4>(grid, a, dyn, st, e0, e1); break;
        case 2: rw = launch_words<2, 4>(grid, a, dyn, st, e0, e1); break;
        case 4: rw = launch_words<4, 4>(grid, a, dyn, st, e0, e1, wide); break;
        default: rw = launch_words<8, 4>(grid, a, dyn, st, e0, e1); break;
      }
    }
    if (rw != NMDLM_OK) return rw;
  } else if (fused) {
    if (NW == 16) {
      launch_fused<1, 16>(grid, a, dyn, st, e0, e1);
    } else {
      if (RT == 1) launch_fused<1, 4>(grid, a, dyn, st, e0, e1);
      else launch_fused<2, 4>(grid, a, dyn, st, e0, e1);
    }
  } else if (NW == 16) {
    if (RT == 1) launch_list<1, 16>(grid, a, st, e0, e1);
    else launch_list<2, 16>(grid, a, st, e0, e1);
  } else {
    switch (RT) {
      case 1: launch_list<1, 4>(grid, a, st, e0, e1); break;
      case 2: launch_list<2, 4>(grid, a, st, e0, e1); break;
      case 4: launch_list<4, 4>(grid, a, st, e0, e1); break;
      default: launch_list<8, 4>(grid, a, st, e0, e1); break;
    }
  }
  const nmdlm_status rc = hip_status();

  return rc;
}

}  // namespace nmdlm
