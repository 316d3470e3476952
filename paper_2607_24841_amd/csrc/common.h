// Internal declarations shared by the libnmdlm HIP sources (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "nmdlm.h"

namespace nmdlm {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
// floor(i / d) for 0 <= i, 1 <= d and i + d < 2^22, from inv_d = 1.0f / d.
// The quotient of i + 0.5 lies at least 0.5 / d from any integer, and the
// float rounding errors stay below that in this range, so the truncation is
// exact; it costs a conversion and a multiply instead of an integer division.
__device__ __forceinline__ int div_small(int i, float inv_d) {
  return (int)(((float)i + 0.5f) * inv_d);
}

// Kernel arguments are read through the scalar cache, and the compiler
// fetches each field just before its first use, so an argument block that
// spans several 64-byte lines costs one dependent round trip per line.
// Reading one dword of every line at entry (all loads issued, then one
// wait) brings the lines in together; later field reads hit the cache.
template <size_t Bytes>
__device__ __forceinline__ void touch_kernargs() {
  typedef const __attribute__((address_space(4))) uint32_t KargWord;
  KargWord* k = (KargWord*)__builtin_amdgcn_kernarg_segment_ptr();
  constexpr int kLines = (int)((Bytes + 63) / 64);
  uint32_t v[kLines];
#pragma unroll
  for (int i = 0; i < kLines; ++i) v[i] = k[i * 16];
#pragma unroll
  for (int i = 0; i < kLines; ++i) asm volatile("" ::"s"(v[i]));
}

constexpr int kXcds = 8;  // accelerator dies; each has its own L2

// Workgroups are dispatched round-robin over the XCDs (dispatch id d runs on
// XCD d % 8).  xcd_order maps the dispatch id of a grid of n workgroups to a
// logical id such that every XCD holds one contiguous range of logical ids;
// kernels order their tiles so that tiles sharing input lines are
// consecutive.  A bijection of [0, n) for every n.
__device__ __forceinline__ int xcd_order(int d, int n) {
  const int q = n / kXcds, r = n - q * kXcds;
  const int xcd = d % kXcds, slot = d / kXcds;
  return xcd < r ? xcd * (q + 1) + slot : r * (q + 1) + (xcd - r) * q + slot;
}

// Logical (x, y, z) of a workgroup of a 3-D grid, y fastest: the row blocks
// of one column tile, then the neighbouring column tiles, share an XCD.
__device__ __forceinline__ void tile_coords(int& x, int& y, int& z) {
  const int gx = gridDim.x, gy = gridDim.y;
  const int n = gx * gy * gridDim.z;
  const int d = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const int l = xcd_order(d, n);
  y = l % gy;
  x = (l / gy) % gx;
  z = l / (gy * gx);
}
// With inv_gy = 1/gy and inv_gxy = 1/(gx gy) the quotients of grids of
// fewer than 2^21 workgroups are taken in float (exact, see div_small), in
// place of the integer divisions the scalar unit emulates with some forty
// instructions each.
__device__ __forceinline__ void tile_coords_inv(int& x, int& y, int& z, float inv_gy,
                                                float inv_gxy) {
  const int gx = gridDim.x, gy = gridDim.y;
  const int n = gx * gy * gridDim.z;
  if (n >= (1 << 21)) {  // uniform
    tile_coords(x, y, z);
    return;
  }
  const int d = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const int l = xcd_order(d, n);
  const int q = __builtin_amdgcn_readfirstlane(div_small(l, inv_gy));  // l / gy
  z = __builtin_amdgcn_readfirstlane(div_small(l, inv_gxy));           // l / (gx gy)
  y = l - q * gy;
  x = q - z * gx;
}
constexpr int kMaxSeg = 3;
constexpr int kChunkSteps = 16;   // k-steps (of 64 active rows) staged per LDS chunk
constexpr int kTileLd = 68;       // LDS row stride (ints) of the 64-column output tile
constexpr int kSplitMaxRows = 256;  // K splits only for blocks of at most this many rows

enum EpiMode : int {
  EPI_CUR = 0,     // write int32 currents only
  EPI_IF = 1,      // integrate-and-fire -> packed spikes
  EPI_QNL_IF = 2,  // table non-linearity, then integrate-and-fire
  EPI_HEAD = 3,    // sum over t, fp32 dequantisation -> logits
  EPI_BITWISE = 4, // sum over t weighted 2^t (bitwise-coded input) -> int32 [M][N]
  EPI_MODIF = 5    // modified IF over the bit-timesteps -> ternary spike planes
};

// Destination of the spikes of one column segment of a product.
//   natural    : word (t, m, w) at ptr[t*ld_t + m*ld_m + w]
//   transposed : position-packed cache: bit (pos0+m)%64 of the word
//                ptr[t*ld_t + ch*ld_m + ((pos0+m)/64)*ld_p] holds channel ch
//                of token m (word-major caches: ld_m = 1, ld_p = channels)
//   sequences  : with seq_len > 0, token m is token m % seq_len of sequence
//                m / seq_len, whose words start ld_s words further
struct SpikeSeg {
  uint64_t* ptr;
  int64_t ld_t;
  int64_t ld_m;
  int32_t theta;
  int32_t transposed;
  int32_t pos0;
  int32_t ld_p;
  int32_t seq_len;
  int64_t ld_s;
};

struct QbsmArgs {
  // operand prepared by the union/compaction kernels
  const uint64_t* sc;        // compacted spike bits [KSmax][R], R = T*M
  const uint32_t* act_off;   // byte offsets k*ldw of the active rows (padded with 0)
  const int32_t* kact;       // number of active rows
  // weights
  const int8_t* W;
  int64_t ldw;
  int K, N;
  int T, M, Mb;              // Mb tokens per row block
  int P;                     // K splits
  // epilogue
  int mode;
  const int32_t* bias;       // [N] or null
  int32_t* cur_out;          // [T][M][N] or null
  const int32_t* theta_vec;  // [N] or null
  int nseg, seg_w;           // column segments of seg_w columns (multiple of 64)
  SpikeSeg seg[kMaxSeg];
  const uint64_t* resid;     // natural spikes, word (t, m, w) at resid[t*rld_t + m*rld_m + w]
  int64_t rld_t, rld_m;
  const uint8_t* lut;        // activation table (EPI_QNL_IF)
  int lut_shift;
  float* logits;             // EPI_HEAD: [M][N]
  const float* scale;        // EPI_HEAD: [N]
  int32_t* part;             // K-split accumulators [gy*gx][16*RT*64], zero between products
  int32_t* counters;         // [gx*gy] arrival counters, zero between products
  uint64_t* u_out;           // partial unions of the output spikes [gy][u_ld] or null
  int u_ld;
  // single-kernel product: union sources and statistics
  const uint64_t* S;         // input spikes [R][ceil(K/64)]
  const uint64_t* Sn;        // ternary input: the -1 spikes (S holds the +1 spikes), or null
  const uint64_t* upart;     // partial unions [nparts][ceil(K/64)] or null
  int nparts;
  int dense;
  nmdlm_qbsm_stats* stats;
  // EPI_MODIF: threshold thr_num[m] / thr_den per token; the +1 plane goes
  // to seg[0], the -1 plane to s_neg_out (same layout); final membrane
  // (times thr_den) to v_out [M][N] when given
  const int64_t* thr_num;
  int64_t thr_den;
  uint64_t* s_neg_out;
  int64_t* v_out;
  // word product: 0 = MFMA, 1 = scalar gather-accumulate
  int accum;
  // blocked weights (operand order, see launch_weight_block) or null, and
  // the active rows per active word from which a wave reads them
  const int8_t* Wb;
  int blk_min;
  // 1.0f / gridDim.y and 1.0f / (gridDim.x * gridDim.y) (IEEE, from the
  // host): the workgroup's tile coordinates without integer divisions
  float inv_gy, inv_gxy;
  // 1.0f / ceil(K/64), 1.0f / Mb and 1.0f / seg_w (several segments): the
  // in-kernel quotients by div_small
  float inv_kw, inv_mb, inv_segw;
};

// Scratch used by one product (carved from a workspace).
struct QbsmScratch {
  uint32_t* act_off;   // [round_up(K,64)]
  int32_t* act_idx;    // [round_up(K,64)]
  int32_t* kact;       // [1]
  uint64_t* sc;        // [ceil(K/64)][R]
  uint64_t* U;         // [ceil(K/64)] union of a large block
  int32_t* part;       // K-split accumulators (split products only), then
  int32_t* counters;   // [tiles] arrival counters: together the split region
  size_t part_elems;
  size_t n_counters;
};

// The split region [part, counters + n_counters) rounded to whole 16-byte
// units (the carver aligns every region to 256 bytes).
inline int64_t split_region_elems(const QbsmScratch& s) {
  const char* b = s.part ? reinterpret_cast<const char*>(s.part) : reinterpret_cast<const char*>(s.counters);
  const char* e = reinterpret_cast<const char*>(s.counters + s.n_counters);
  return (int64_t)(((size_t)(e - b) + 15) / 16 * 4);
}

// One product request (host side).
struct QbsmCall {
  const uint64_t* s_in;   // [T][M][ceil(K/64)]
  int T, M, K;
  const int8_t* W;
  int64_t ldw;
  int N;
  int mode;
  const int32_t* bias;
  int32_t* cur_out;
  const int32_t* theta_vec;
  int nseg, seg_w;
  SpikeSeg seg[kMaxSeg];
  const uint64_t* resid;
  int64_t rld_t, rld_m;
  const uint8_t* lut;
  int lut_shift;
  float* logits;
  const float* scale;
  nmdlm_qbsm_stats* stats;
  unsigned flags;
  hipEvent_t ev_begin;    // recorded around the product kernel when non-null
  hipEvent_t ev_end;
  const uint64_t* s_neg;  // ternary input: -1 spikes [T][M][ceil(K/64)] (s_in: +1), or null
  int seq_len;            // tokens per sequence when M holds several (0: one sequence); a
                          // channel-major output segment keeps row blocks within a sequence
  const uint64_t* u_in;   // partial unions of s_in [u_nparts][ceil(K/64)] or null
  int u_nparts;
  uint64_t* u_out;        // where to write the partial unions of the output
  const int64_t* thr_num; // EPI_MODIF (see QbsmArgs)
  int64_t thr_den;
  uint64_t* s_neg_out;
  int64_t* v_out;
  const int8_t* Wb;       // the weights in blocked operand order, or null
};

// Blocked weight layout: for word w (rows 64w..64w+63) and column tile x
// (columns 64x..64x+63), 4096 bytes at (w * ceil(N/64) + x) * 4096; within
// them operand v (v = 0..3), lane l = 16g + c, byte j holds
// W[64w + 16g + j][64x + 4c + v] (zero past K or N): the B operand of
// v_mfma_i32_16x16x64_i8 for the tile's columns 4c + v, one 16-byte load.
inline size_t weight_blocked_bytes(int K, int N) {
  return (size_t)((K + 63) / 64) * (size_t)((N + 63) / 64) * 4096;
}
nmdlm_status launch_weight_block(const int8_t* W, int K, int N, int64_t ldw, int8_t* Wb,
                                 hipStream_t st);

// Workspace layout helpers -------------------------------------------------
inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct Carver {
  char* base;
  size_t off;
  size_t cap;
  bool ok;
  template <typename T>
  T* take(size_t n) {
    size_t o = align_up(off, 256);
    size_t bytes = align_up(n * sizeof(T), 256);
    off = o + bytes;
    if (off > cap) ok = false;
    return base ? reinterpret_cast<T*>(base + o) : nullptr;
  }
};

// Sizes of the product scratch for the largest call of a sequence.
struct QbsmLimits {
  int Kmax;       // largest K
  int Rmax;       // largest T*M
  int Nmax;       // largest N
  int tiles_max;  // largest number of (column tile, row block) tiles
  int split_rows; // largest R that may use K splits (0: splits never used)
  int split_N;    // largest N that may use K splits
};

QbsmLimits qbsm_limits_single(int T, int M, int K, int N);
void carve_qbsm_scratch(Carver& cv, const QbsmLimits& L, QbsmScratch* s);

// Launchers (enqueue only; arguments already validated).
// gy_out (optional): row blocks used, i.e. the number of partial unions
// written to call.u_out.
nmdlm_status launch_qbsm(const QbsmCall& call, const QbsmScratch& scr, hipStream_t st,
                         int* gy_out = nullptr);
nmdlm_status launch_if(const int32_t* cur, int T, int M, int N, int32_t theta,
                       const int32_t* theta_vec, const uint64_t* resid,
                       int32_t* v_inout, uint64_t* s_out, hipStream_t st,
                       uint64_t* u_out = nullptr);
nmdlm_status launch_qnl(const int32_t* x, int64_t n, int shift, int mode,
                        const uint8_t* lut, uint8_t* y, hipStream_t st);
// n_seq sequences of M queries each (rows sequence-major); the caches of
// sequence s start s * seq_words words after k_cache / vt_cache
nmdlm_status launch_attn(const uint64_t* q, const uint64_t* k_cache,
                         const uint64_t* vt_cache, int64_t cap, int T, int M, int C,
                         int H, int dh, const uint8_t* lut, int32_t* a_out,
                         hipStream_t st, int n_seq = 1, int64_t seq_words = 0);
// attention with the IF of its output fused in (spikes and per-token union
// over t); NMDLM_ERR_UNSUPPORTED when T*16*dh partial sums exceed its LDS
nmdlm_status launch_attn_if(const uint64_t* q, const uint64_t* k_cache, const uint64_t* vt_cache,
                            int64_t cap, int T, int M, int C, int H, int dh, const uint8_t* lut,
                            int32_t theta, uint64_t* s_out, uint64_t* u_out, hipStream_t st);
nmdlm_status launch_fill_zero(void* p, size_t bytes, hipStream_t st);
nmdlm_status launch_ternary_encode(const int32_t* a, int M, int D, int K, int T, uint64_t* sp,
                                   uint64_t* sn, int64_t* s_sum, hipStream_t st);

inline nmdlm_status hip_status() {
  return hipGetLastError() == hipSuccess ? NMDLM_OK : NMDLM_ERR_HIP;
}

}  // namespace nmdlm
