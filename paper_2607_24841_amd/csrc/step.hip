// One block-denoising step (Sec. III-A, Eq. (6)) through a stack of spiking
// layers: block input assembly, per-layer products/attention/neurons, head,
// confidence and unmasking.  Everything stays on the device; the host only
// enqueues work on the caller's stream.
#include <float.h>

#include <algorithm>

#include "common.h"

namespace nmdlm {

// X[t,m,:] = E[token_m][t] OR the position spike of (pos0 + m % Mseq, t)
// (M rows: sequences of Mseq tokens one after the other); masked positions
// use the mask token (id V).  An id outside [0, V] reads the nearest row and
// sets NMDLM_STATUS_TOKEN_CLAMPED in the caller's status word (if given).
__global__ __launch_bounds__(256) void k_assemble(const uint64_t* __restrict__ emb,
                                                  const int32_t* __restrict__ pos_ch,
                                                  const int32_t* __restrict__ tokens,
                                                  const uint8_t* __restrict__ masked, int V, int T,
                                                  int M, int Mseq, int dw, int pos0,
                                                  uint64_t* __restrict__ X,
                                                  int32_t* __restrict__ status) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long total = (long long)T * M * dw;
  if (i >= total) return;
  const int w = (int)(i % dw);
  const int m = (int)((i / dw) % M);
  const int t = (int)(i / ((long long)dw * M));
  int tok = (masked && masked[m]) ? V : (tokens ? tokens[m] : V);
  if (tok < 0 || tok > V) {
    // an id outside the table is read as the nearest valid row and reported
    if (status && t == 0 && w == 0) atomicOr(status, NMDLM_STATUS_TOKEN_CLAMPED);
    tok = min(max(tok, 0), V);
  }
  uint64_t word = emb[((size_t)tok * T + t) * dw + w];
  const int pc = pos_ch[(size_t)(pos0 + m % Mseq) * T + t];
  if ((pc >> 6) == w) word |= 1ull << (pc & 63);
  X[i] = word;
}

// Per token: argmax of the logits (ties -> smallest id) and the largest
// softmax probability 1 / sum_v exp(l_v - l_max) in float64, in two passes
// spread over the chip.  k_conf_part: workgroup (m, c) takes logits
// [c*kConfChunk, (c+1)*kConfChunk) of token m and records their largest
// value, its id (ties: the smallest) and sum exp(l_v - that) in float64.
// k_conf: l_max is the largest chunk maximum (ties: the first chunk, whose
// ids are the smaller) and sum_v exp(l_v - l_max) = sum_chunks
// sum_chunk * exp(chunk max - l_max).
struct ConfPart {
  float mx;
  int32_t arg;
  double sum;
};
constexpr int kConfThreads = 256;
constexpr int kConfPerThread = 8;
constexpr int kConfChunk = kConfThreads * kConfPerThread;

__device__ __forceinline__ bool conf_better(float a, int ia, float b, int ib) {
  return a > b || (a == b && ia < ib);
}

// Arg-max over the workgroup (ties -> smaller id); every thread gets it.
__device__ __forceinline__ void block_argmax(float& best, int& bi, float* sBest, int* sIdx) {
  constexpr int NW = kConfThreads / 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o);
    const int oi = __shfl_xor(bi, o);
    if (conf_better(ob, oi, best, bi)) {
      best = ob;
      bi = oi;
    }
  }
  if (lane == 0) {
    sBest[wave] = best;
    sIdx[wave] = bi;
  }
  __syncthreads();
  best = sBest[0];
  bi = sIdx[0];
  for (int w = 1; w < NW; ++w)
    if (conf_better(sBest[w], sIdx[w], best, bi)) {
      best = sBest[w];
      bi = sIdx[w];
    }
}

// Sum over the workgroup; thread 0 gets it.
__device__ __forceinline__ double block_sum(double acc, double* sSum) {
  constexpr int NW = kConfThreads / 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) sSum[wave] = acc;
  __syncthreads();
  double sum = 0.0;
  for (int w = 0; w < NW; ++w) sum += sSum[w];
  return sum;
}

__global__ __launch_bounds__(kConfThreads) void k_conf_part(const float* __restrict__ logits, int V,
                                                            ConfPart* __restrict__ part) {
  __shared__ float sBest[kConfThreads / 64];
  __shared__ int sIdx[kConfThreads / 64];
  __shared__ double sSum[kConfThreads / 64];
  const int m = blockIdx.y, ch = blockIdx.x, tid = threadIdx.x;
  const float* row = logits + (size_t)m * V;
  const int v0 = ch * kConfChunk + tid;
  // every load is issued (at a clamped index) before the first is used
  float xs[kConfPerThread];
#pragma unroll
  for (int u = 0; u < kConfPerThread; ++u) xs[u] = row[min(v0 + u * kConfThreads, V - 1)];
  float best = -FLT_MAX;
  int bi = 0x7fffffff;
#pragma unroll
  for (int u = 0; u < kConfPerThread; ++u) {
    const int v = v0 + u * kConfThreads;
    if (v < V && conf_better(xs[u], v, best, bi)) {
      best = xs[u];
      bi = v;
    }
  }
  block_argmax(best, bi, sBest, sIdx);
  const double mx = (double)best;
  double acc = 0.0;
#pragma unroll
  for (int u = 0; u < kConfPerThread; ++u)
    if (v0 + u * kConfThreads < V) acc += exp((double)xs[u] - mx);
  const double sum = block_sum(acc, sSum);
  if (tid == 0) part[(size_t)m * gridDim.x + ch] = ConfPart{best, bi, sum};
}

__global__ __launch_bounds__(kConfThreads) void k_conf(const ConfPart* __restrict__ part, int nch,
                                                       int32_t* __restrict__ pred,
                                                       double* __restrict__ conf) {
  __shared__ float sBest[kConfThreads / 64];
  __shared__ int sIdx[kConfThreads / 64];
  __shared__ double sSum[kConfThreads / 64];
  const int m = blockIdx.x, tid = threadIdx.x;
  const ConfPart* row = part + (size_t)m * nch;
  float best = -FLT_MAX;
  int bi = 0x7fffffff;
  for (int i = tid; i < nch; i += kConfThreads) {
    const ConfPart p = row[i];
    if (conf_better(p.mx, p.arg, best, bi)) {
      best = p.mx;
      bi = p.arg;
    }
  }
  block_argmax(best, bi, sBest, sIdx);
  const double mx = (double)best;
  double acc = 0.0;
  for (int i = tid; i < nch; i += kConfThreads) {
    const ConfPart p = row[i];
    acc += p.sum * exp((double)p.mx - mx);
  }
  const double sum = block_sum(acc, sSum);
  if (tid == 0) {
    pred[m] = bi;
    conf[m] = 1.0 / sum;
  }
}

// Top-k unmasking by one wave: among the positions still masked, take the
// highest confidence (ties -> smaller position) k times.  Lane l owns the
// positions l + 64 j (j < 64, so M <= kUnmaskMaxM) and keeps their masked
// flags in a register mask.  Workgroup s takes sequence s (its M tokens at
// s * M, its k chosen positions at s * k).
constexpr int kUnmaskMaxM = 64 * 64;
static_assert(kUnmaskMaxM >= NMDLM_MAX_HEAD_M, "unmask register mask covers every head step");

__global__ __launch_bounds__(64) void k_unmask(int32_t* __restrict__ tokens,
                                               uint8_t* __restrict__ masked,
                                               const int32_t* __restrict__ pred,
                                               const double* __restrict__ conf, int M, int k,
                                               int32_t* __restrict__ chosen) {
  const int lane = threadIdx.x;
  const size_t so = (size_t)blockIdx.x * M;
  tokens += so;
  masked += so;
  pred += so;
  conf += so;
  if (chosen) chosen += (size_t)blockIdx.x * k;
  if (M <= 64) {
    // one position per lane: its rank among the masked positions (higher
    // confidence first, ties to the lower position) decides it in one pass;
    // the r-th chosen position is the one of rank r (the order the
    // one-at-a-time selection takes them in)
    const bool mv = lane < M && masked[lane];
    const double cm = mv ? conf[lane] : 0.0;
    const uint64_t mm = __builtin_amdgcn_ballot_w64(mv);
    int rank = 0;
    const unsigned long long cbits = __double_as_longlong(cm);
    for (uint64_t rest = mm; rest; rest &= rest - 1) {
      const int j = (int)__builtin_ctzll(rest);  // wave-uniform
      const unsigned long long bj =
          ((unsigned long long)(uint32_t)__builtin_amdgcn_readlane((int)(cbits >> 32), j) << 32) |
          (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)cbits, j);
      const double cj = __longlong_as_double((long long)bj);
      rank += (cj > cm || (cj == cm && j < lane)) ? 1 : 0;
    }
    if (mv && rank < k) {
      tokens[lane] = pred[lane];
      masked[lane] = 0;
      if (chosen) chosen[rank] = lane;
    }
    const int nm = __popcll(mm);
    if (chosen)
      for (int r = lane; r < k; r += 64)
        if (r >= nm) chosen[r] = -1;  // fewer masked positions than k
    return;
  }
  uint64_t mine = 0ull;
  for (int jj = 0, m = lane; m < M; ++jj, m += 64)
    if (masked[m]) mine |= 1ull << jj;
  for (int r = 0; r < k; ++r) {
    double bc = 0.0;
    int bm = -1;
    for (uint64_t rest = mine; rest; rest &= rest - 1) {
      const int m = lane + 64 * (int)__builtin_ctzll(rest);
      const double cm = conf[m];
      if (bm < 0 || cm > bc) {  // ascending m: ties keep the smaller position
        bc = cm;
        bm = m;
      }
    }
    for (int o = 32; o > 0; o >>= 1) {
      const double oc = __shfl_xor(bc, o);
      const int om = __shfl_xor(bm, o);
      if (om >= 0 && (bm < 0 || oc > bc || (oc == bc && om < bm))) {
        bc = oc;
        bm = om;
      }
    }
    if (bm >= 0 && (bm & 63) == lane) mine &= ~(1ull << (bm >> 6));
    if (lane == 0) {
      if (bm >= 0) {
        tokens[bm] = pred[bm];
        masked[bm] = 0;
      }
      if (chosen) chosen[r] = bm;
    }
  }
}

// ---------------------------------------------------------------------------
// workspace layout of a block step
// ---------------------------------------------------------------------------
struct StepBuffers {
  uint64_t* X;      // assembled input [T][M][dw]
  uint64_t* Q;      // [T][M][dw]
  uint64_t* A;
  uint64_t* X1;
  uint64_t* Hs;     // [T][M][Fw]
  uint64_t* Y[2];
  int32_t* a;       // attention output [T][M][d]
  uint64_t* uA;     // partial unions of A  [M][dw]
  uint64_t* uX1;    // partial unions of X1 [M][dw] (at most one per token)
  uint64_t* uH;     // partial unions of H  [M][Fw]
  uint64_t* uY[2];  // partial unions of Y  [M][dw]
  float* logits;    // [M][V] (when the caller gives none)
  ConfPart* cpart;  // [M][ceil(V/kConfChunk)] confidence partials
  int32_t* pred;
  double* conf;
  QbsmScratch qs;
};

static QbsmLimits step_limits(const nmdlm_model* md, int M, unsigned flags) {
  QbsmLimits L;
  const int T = md->T, d = md->d, F = md->F;
  const bool head = !(flags & NMDLM_NO_HEAD);
  L.Kmax = std::max(d, F);
  L.Rmax = T * M;
  int nmax = std::max(3 * d, F);
  if (head) nmax = std::max(nmax, md->V);
  L.Nmax = nmax;
  L.tiles_max = ((nmax + 63) / 64) * M;
  L.split_rows = (T * M <= kSplitMaxRows) ? T * M : 0;
  L.split_N = std::max(3 * d, F);
  return L;
}

static void carve_step(Carver& cv, const nmdlm_model* md, int M, unsigned flags, bool need_x,
                       bool need_logits, bool need_pred, bool need_conf, StepBuffers* b) {
  const int T = md->T, dw = md->d / 64, Fw = (md->F + 63) / 64;
  const size_t sp = (size_t)T * M * dw;
  b->X = need_x ? cv.take<uint64_t>(sp) : nullptr;
  b->Q = cv.take<uint64_t>(sp);
  b->A = cv.take<uint64_t>(sp);
  b->X1 = cv.take<uint64_t>(sp);
  b->Hs = cv.take<uint64_t>((size_t)T * M * Fw);
  b->Y[0] = cv.take<uint64_t>(sp);
  b->Y[1] = cv.take<uint64_t>(sp);
  b->a = cv.take<int32_t>((size_t)T * M * md->d);
  b->uA = cv.take<uint64_t>((size_t)M * dw);
  b->uX1 = cv.take<uint64_t>((size_t)M * dw);
  b->uH = cv.take<uint64_t>((size_t)M * Fw);
  b->uY[0] = cv.take<uint64_t>((size_t)M * dw);
  b->uY[1] = cv.take<uint64_t>((size_t)M * dw);
  const bool head = !(flags & NMDLM_NO_HEAD);
  b->logits = (head && need_logits) ? cv.take<float>((size_t)M * md->V) : nullptr;
  b->cpart = head ? cv.take<ConfPart>((size_t)M * ((md->V + kConfChunk - 1) / kConfChunk)) : nullptr;
  b->pred = (head && need_pred) ? cv.take<int32_t>(M) : nullptr;
  b->conf = (head && need_conf) ? cv.take<double>(M) : nullptr;
  carve_qbsm_scratch(cv, step_limits(md, M, flags), &b->qs);
}

size_t block_step_ws_size(const nmdlm_model* md, int M, unsigned flags) {
  Carver cv{nullptr, 0, (size_t)-1, true};
  StepBuffers b;
  carve_step(cv, md, M, flags, true, true, true, true, &b);
  return align_up(cv.off, 256);
}

static SpikeSeg natural_seg(uint64_t* p, int64_t ld_t, int64_t ld_m, int32_t theta) {
  SpikeSeg s;
  s.ptr = p;
  s.ld_t = ld_t;
  s.ld_m = ld_m;
  s.theta = theta;
  s.transposed = 0;
  s.pos0 = 0;
  s.ld_p = 0;
  s.seq_len = 0;
  s.ld_s = 0;
  return s;
}

static QbsmCall base_call(const uint64_t* s_in, int T, int M, int K, const int8_t* W, int64_t ldw,
                          int N, int mode, unsigned flags, nmdlm_qbsm_stats* stats) {
  QbsmCall c;
  c.s_in = s_in;
  c.T = T;
  c.M = M;
  c.K = K;
  c.W = W;
  c.ldw = ldw;
  c.N = N;
  c.mode = mode;
  c.bias = nullptr;
  c.cur_out = nullptr;
  c.theta_vec = nullptr;
  c.nseg = 1;
  c.seg_w = 1 << 30;
  for (int i = 0; i < kMaxSeg; ++i) c.seg[i] = natural_seg(nullptr, 0, 0, 1);
  c.resid = nullptr;
  c.rld_t = 0;
  c.rld_m = 0;
  c.lut = nullptr;
  c.lut_shift = 0;
  c.logits = nullptr;
  c.scale = nullptr;
  c.stats = stats;
  c.flags = flags & (NMDLM_FORCE_DENSE | (0xFFu << NMDLM_SPLIT_SHIFT) | (0xFu << NMDLM_ROWTILE_SHIFT) |
                     (0x7u << NMDLM_PATH_SHIFT));
  c.ev_begin = nullptr;
  c.ev_end = nullptr;
  c.s_neg = nullptr;
  c.seq_len = 0;
  c.u_in = nullptr;
  c.u_nparts = 0;
  c.u_out = nullptr;
  c.thr_num = nullptr;
  c.thr_den = 1;
  c.s_neg_out = nullptr;
  c.v_out = nullptr;
  c.Wb = nullptr;
  return c;
}

// Attach the caller's timing events of product i (if any).
static void attach_events(QbsmCall& c, const nmdlm_step_io* io, int i) {
  if (io->prof_events && 2 * i + 1 < io->n_prof_events) {
    c.ev_begin = static_cast<hipEvent_t>(io->prof_events[2 * i]);
    c.ev_end = static_cast<hipEvent_t>(io->prof_events[2 * i + 1]);
  }
}

nmdlm_status block_step_impl(const nmdlm_model* md, nmdlm_step_io* io, void* ws, size_t ws_bytes,
                             hipStream_t st) {
  // Ms tokens in each of n_seq sequences; every product takes all M rows
  const int T = md->T, Ms = io->M, n_seq = std::max(io->n_seq, 1), M = n_seq * Ms, C = io->C;
  const int d = md->d, F = md->F, H = md->H;
  const int dh = d / H, dw = d / 64, Fw = (F + 63) / 64;
  const int64_t cap = md->cache_cap, capw = cap / 64;
  const int64_t seq_words = (int64_t)T * cap * dw;  // one sequence's K (and V) cache
  const bool head = !(io->flags & NMDLM_NO_HEAD);

  Carver cv{static_cast<char*>(ws), 0, ws_bytes, true};
  StepBuffers b;
  carve_step(cv, md, M, io->flags, io->x_in == nullptr, io->logits == nullptr,
             io->pred == nullptr, io->conf == nullptr, &b);
  if (!cv.ok) return NMDLM_ERR_WORKSPACE;

  nmdlm_status rc = NMDLM_OK;
  const uint64_t* X = io->x_in;
  if (!X) {
    const long long total = (long long)T * M * dw;
    hipLaunchKernelGGL(k_assemble, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st,
                       md->emb, md->pos_ch, io->tokens, io->masked, md->V, T, M, Ms, dw, io->pos0,
                       b.X, io->status);
    if ((rc = hip_status()) != NMDLM_OK) return rc;
    X = b.X;
  }
  const int64_t sp_t = (int64_t)M * dw;
  // partial unions of the current layer input (null: the prep kernel ORs X)
  const uint64_t* uX = nullptr;
  int uX_parts = 0;
  for (int l = 0; l < md->n_layers; ++l) {
    const nmdlm_layer& ly = md->layers[l];
    nmdlm_qbsm_stats* stl = io->stats ? io->stats + 4 * l : nullptr;
    int gy = 0;

    // Q | K | V, keys and values straight into cache rows [C, C+M)
    QbsmCall qkv = base_call(X, T, M, d, ly.w_qkv, 3 * (int64_t)d, 3 * d, EPI_IF, io->flags,
                             stl ? stl + 0 : nullptr);
    qkv.nseg = 3;
    qkv.seg_w = d;
    qkv.seg[0] = natural_seg(b.Q, sp_t, dw, ly.theta_q);
    qkv.seg[1] = natural_seg(ly.k_cache + (int64_t)C * dw, cap * dw, dw, ly.theta_k);
    // value cache word-major [T][cap/64][d]: position word p of channel ch
    // at (t * capw + p) * d + ch
    qkv.seg[2] = natural_seg(ly.vt_cache, (int64_t)d * capw, 1, ly.theta_v);
    qkv.seg[2].transposed = 1;
    qkv.seg[2].ld_p = d;
    qkv.seg[2].pos0 = C;
    if (n_seq > 1) {
      qkv.seq_len = Ms;
      for (int i = 1; i < 3; ++i) {
        qkv.seg[i].seq_len = Ms;
        qkv.seg[i].ld_s = seq_words;
      }
    }
    qkv.u_in = uX;
    qkv.u_nparts = uX_parts;
    qkv.Wb = ly.w_qkv_b;
    attach_events(qkv, io, 4 * l + 0);
    if ((rc = launch_qbsm(qkv, b.qs, st)) != NMDLM_OK) return rc;

    rc = NMDLM_ERR_UNSUPPORTED;
    if ((io->flags & NMDLM_ATTN_FUSED) && n_seq == 1)
      rc = launch_attn_if(b.Q, ly.k_cache, ly.vt_cache, cap, T, M, C, H, dh, ly.lut_att,
                          ly.theta_a, b.A, b.uA, st);
    if (rc == NMDLM_ERR_UNSUPPORTED) {
      if ((rc = launch_attn(b.Q, ly.k_cache, ly.vt_cache, cap, T, Ms, C, H, dh, ly.lut_att, b.a,
                            st, n_seq, seq_words)) != NMDLM_OK)
        return rc;
      rc = launch_if(b.a, T, M, d, ly.theta_a, nullptr, nullptr, nullptr, b.A, st, b.uA);
    }
    if (rc != NMDLM_OK) return rc;

    QbsmCall o = base_call(b.A, T, M, d, ly.w_o, d, d, EPI_IF, io->flags, stl ? stl + 1 : nullptr);
    o.seg[0] = natural_seg(b.X1, sp_t, dw, ly.theta_o);
    o.resid = X;
    o.rld_t = sp_t;
    o.rld_m = dw;
    o.u_in = b.uA;
    o.u_nparts = M;
    o.u_out = b.uX1;
    o.Wb = ly.w_o_b;
    attach_events(o, io, 4 * l + 1);
    if ((rc = launch_qbsm(o, b.qs, st, &gy)) != NMDLM_OK) return rc;
    const int uX1_parts = gy;

    QbsmCall up = base_call(b.X1, T, M, d, ly.w_up, F, F, EPI_QNL_IF, io->flags,
                            stl ? stl + 2 : nullptr);
    up.seg[0] = natural_seg(b.Hs, (int64_t)M * Fw, Fw, ly.theta_up);
    up.lut = ly.lut_act;
    up.lut_shift = ly.s_up;
    up.u_in = b.uX1;
    up.u_nparts = uX1_parts;
    up.u_out = b.uH;
    up.Wb = ly.w_up_b;
    attach_events(up, io, 4 * l + 2);
    if ((rc = launch_qbsm(up, b.qs, st, &gy)) != NMDLM_OK) return rc;
    const int uH_parts = gy;

    uint64_t* Yl = (l == md->n_layers - 1 && io->y_out) ? io->y_out : b.Y[l & 1];
    QbsmCall dn = base_call(b.Hs, T, M, F, ly.w_dn, d, d, EPI_IF, io->flags,
                            stl ? stl + 3 : nullptr);
    dn.seg[0] = natural_seg(Yl, sp_t, dw, ly.theta_dn);
    dn.resid = b.X1;
    dn.rld_t = sp_t;
    dn.rld_m = dw;
    dn.u_in = b.uH;
    dn.u_nparts = uH_parts;
    dn.u_out = b.uY[l & 1];
    dn.Wb = ly.w_dn_b;
    attach_events(dn, io, 4 * l + 3);
    if ((rc = launch_qbsm(dn, b.qs, st, &gy)) != NMDLM_OK) return rc;
    X = Yl;
    uX = b.uY[l & 1];
    uX_parts = gy;
  }

  if (!head) {
    if (io->y_out && md->n_layers == 0)
      if (hipMemcpyAsync(io->y_out, X, (size_t)T * M * dw * 8, hipMemcpyDeviceToDevice, st) !=
          hipSuccess)
        return NMDLM_ERR_HIP;
    return NMDLM_OK;
  }
  float* logits = io->logits ? io->logits : b.logits;
  int32_t* pred = io->pred ? io->pred : b.pred;
  double* conf = io->conf ? io->conf : b.conf;
  QbsmCall hc = base_call(X, T, M, d, md->w_head, md->V, md->V, EPI_HEAD, io->flags,
                          io->stats ? io->stats + 4 * md->n_layers : nullptr);
  hc.logits = logits;
  hc.scale = md->head_scale;
  hc.u_in = uX;
  hc.u_nparts = uX_parts;
  hc.Wb = md->w_head_b;
  attach_events(hc, io, 4 * md->n_layers);
  if ((rc = launch_qbsm(hc, b.qs, st)) != NMDLM_OK) return rc;
  const int nch = (md->V + kConfChunk - 1) / kConfChunk;
  hipLaunchKernelGGL(k_conf_part, dim3(nch, M), dim3(kConfThreads), 0, st, logits, md->V, b.cpart);
  if ((rc = hip_status()) != NMDLM_OK) return rc;
  hipLaunchKernelGGL(k_conf, dim3(M), dim3(kConfThreads), 0, st, b.cpart, nch, pred, conf);
  if ((rc = hip_status()) != NMDLM_OK) return rc;
  hipLaunchKernelGGL(k_unmask, dim3(n_seq), dim3(64), 0, st, io->tokens, io->masked, pred, conf,
                     Ms, io->k_unmask, io->unmasked_pos);
  return hip_status();
}

}  // namespace nmdlm
