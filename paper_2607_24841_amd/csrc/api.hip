// C ABI of libnmdlm: argument validation (before any HIP call), workspace
// sizing and dispatch to the launchers.
#include <algorithm>
#include <climits>

#include "common.h"

namespace nmdlm {
size_t block_step_ws_size(const nmdlm_model* md, int M, unsigned flags);
nmdlm_status block_step_impl(const nmdlm_model* md, nmdlm_step_io* io, void* ws, size_t ws_bytes,
                             hipStream_t st);
}  // namespace nmdlm

using namespace nmdlm;

namespace {

inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t qbsm_ws(int T, int M, int K, int N) {
  Carver cv{nullptr, 0, (size_t)-1, true};
  QbsmScratch s;
  carve_qbsm_scratch(cv, qbsm_limits_single(T, M, K, N), &s);
  return align_up(cv.off, 256);
}

// an optional blocked copy: NULL, or 16-byte aligned with a size below 2^31
bool blocked_ok(const int8_t* Wb, int K, int N) {
  return !Wb || (((reinterpret_cast<uintptr_t>(Wb) & 15) == 0) &&
                 weight_blocked_bytes(K, N) < ((size_t)1 << 31));
}

bool weights_ok(const int8_t* W, int K, int N, int64_t ldw) {
  if (!W || !aligned(W, 16)) return false;
  if (ldw < N || (ldw % 16) != 0) return false;
  if ((int64_t)K * ldw >= (int64_t)1 << 31) return false;
  return true;
}

}  // namespace

extern "C" {

int nmdlm_abi_version(void) { return NMDLM_ABI_VERSION; }

const char* nmdlm_status_string(nmdlm_status s) {
  switch (s) {
    case NMDLM_OK: return "ok";
    case NMDLM_ERR_INVALID_ARG: return "invalid argument";
    case NMDLM_ERR_UNSUPPORTED: return "unsupported shape or layout";
    case NMDLM_ERR_WORKSPACE: return "workspace missing or too small";
    case NMDLM_ERR_HIP: return "HIP launch error";
  }
  return "unknown status";
}

size_t nmdlm_qbsm_workspace_size(int T, int M, int K, int N) {
  if (T < 1 || T > NMDLM_MAX_T || M < 1 || K < 1 || K > NMDLM_MAX_K || N < 1) return 0;
  return qbsm_ws(T, M, K, N);
}

}  // extern "C"

namespace {

nmdlm_status qbsm_entry(const uint64_t* s_in, int T, int M, int K, const int8_t* W,
                        const int8_t* Wb, int N, int64_t ldw, const int32_t* bias,
                        int32_t* cur_out, int32_t theta, const int32_t* theta_vec,
                        uint64_t* s_out, nmdlm_qbsm_stats* stats, unsigned flags, void* ws,
                        size_t ws_bytes, void* stream) {
  if (!s_in || T < 1 || M < 1 || K < 1 || N < 1) return NMDLM_ERR_INVALID_ARG;
  if (T > NMDLM_MAX_T || K > NMDLM_MAX_K) return NMDLM_ERR_UNSUPPORTED;
  if (!weights_ok(W, K, N, ldw)) return NMDLM_ERR_INVALID_ARG;
  if (!cur_out && !s_out) return NMDLM_ERR_INVALID_ARG;
  if (s_out && !theta_vec && theta <= 0) return NMDLM_ERR_INVALID_ARG;
  if ((int64_t)T * M > (1 << 19)) return NMDLM_ERR_UNSUPPORTED;
  if (!ws || !aligned(ws, 256) || ws_bytes < qbsm_ws(T, M, K, N)) return NMDLM_ERR_WORKSPACE;

  const int Nw = (N + 63) / 64;
  QbsmCall c;
  c.s_in = s_in;
  c.T = T;
  c.M = M;
  c.K = K;
  c.W = W;
  c.ldw = ldw;
  c.N = N;
  c.mode = s_out ? EPI_IF : EPI_CUR;
  c.bias = bias;
  c.cur_out = cur_out;
  c.theta_vec = theta_vec;
  c.nseg = 1;
  c.seg_w = 1 << 30;
  for (int i = 0; i < kMaxSeg; ++i) {
    c.seg[i].ptr = s_out;
    c.seg[i].ld_t = (int64_t)M * Nw;
    c.seg[i].ld_m = Nw;
    c.seg[i].theta = theta;
    c.seg[i].transposed = 0;
    c.seg[i].pos0 = 0;
    c.seg[i].ld_p = 0;
    c.seg[i].seq_len = 0;
    c.seg[i].ld_s = 0;
  }
  c.resid = nullptr;
  c.rld_t = c.rld_m = 0;
  c.lut = nullptr;
  c.lut_shift = 0;
  c.logits = nullptr;
  c.scale = nullptr;
  c.stats = stats;
  c.flags = flags;
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
  c.Wb = Wb;

  Carver cv{static_cast<char*>(ws), 0, ws_bytes, true};
  QbsmScratch scr;
  carve_qbsm_scratch(cv, qbsm_limits_single(T, M, K, N), &scr);
  if (!cv.ok) return NMDLM_ERR_WORKSPACE;
  return launch_qbsm(c, scr, static_cast<hipStream_t>(stream));
}

}  // namespace

extern "C" {

nmdlm_status nmdlm_qbsm(const uint64_t* s_in, int T, int M, int K, const int8_t* W, int N,
                        int64_t ldw, const int32_t* bias, int32_t* cur_out, int32_t theta,
                        const int32_t* theta_vec, uint64_t* s_out, nmdlm_qbsm_stats* stats,
                        unsigned flags, void* ws, size_t ws_bytes, void* stream) {
  return qbsm_entry(s_in, T, M, K, W, nullptr, N, ldw, bias, cur_out, theta, theta_vec, s_out,
                    stats, flags, ws, ws_bytes, stream);
}

size_t nmdlm_weight_blocked_bytes(int K, int N) {
  if (K < 1 || K > NMDLM_MAX_K || N < 1) return 0;
  return weight_blocked_bytes(K, N);
}

nmdlm_status nmdlm_weight_block(const int8_t* W, int K, int N, int64_t ldw, int8_t* Wb,
                                void* stream) {
  if (K < 1 || N < 1) return NMDLM_ERR_INVALID_ARG;
  if (K > NMDLM_MAX_K) return NMDLM_ERR_UNSUPPORTED;
  if (!weights_ok(W, K, N, ldw) || !Wb || !aligned(Wb, 16)) return NMDLM_ERR_INVALID_ARG;
  if (weight_blocked_bytes(K, N) >= ((size_t)1 << 31)) return NMDLM_ERR_UNSUPPORTED;
  return launch_weight_block(W, K, N, ldw, Wb, static_cast<hipStream_t>(stream));
}

nmdlm_status nmdlm_qbsm_blocked(const uint64_t* s_in, int T, int M, int K, const int8_t* W,
                                const int8_t* Wb, int N, int64_t ldw, const int32_t* bias,
                                int32_t* cur_out, int32_t theta, const int32_t* theta_vec,
                                uint64_t* s_out, nmdlm_qbsm_stats* stats, unsigned flags, void* ws,
                                size_t ws_bytes, void* stream) {
  if (!Wb || !aligned(Wb, 16)) return NMDLM_ERR_INVALID_ARG;
  if (weight_blocked_bytes(K, N) >= ((size_t)1 << 31)) return NMDLM_ERR_UNSUPPORTED;
  return qbsm_entry(s_in, T, M, K, W, Wb, N, ldw, bias, cur_out, theta, theta_vec, s_out, stats,
                    flags, ws, ws_bytes, stream);
}

nmdlm_status nmdlm_ternary_encode(const int32_t* a, int M, int D, int K, int T, uint64_t* s_pos,
                                  uint64_t* s_neg, int64_t* s_sum, void* stream) {
  if (!a || !s_pos || !s_neg || M < 1 || D < 1 || K < 1 || T < 1) return NMDLM_ERR_INVALID_ARG;
  if (T > NMDLM_MAX_T || D > NMDLM_MAX_K || (int64_t)D * K >= ((int64_t)1 << 20))
    return NMDLM_ERR_UNSUPPORTED;
  return launch_ternary_encode(a, M, D, K, T, s_pos, s_neg, s_sum, static_cast<hipStream_t>(stream));
}

}  // extern "C"

namespace {

// The product on ternary spike planes, with the 2^(t-1)-weighted sum
// (EPI_BITWISE, acc_out) or the modified IF neuron (EPI_MODIF, spike planes).
nmdlm_status ternary_product(const uint64_t* s_pos, const uint64_t* s_neg, int T, int M, int K,
                             const int8_t* W, int N, int64_t ldw, int mode, int32_t* acc_out,
                             const int64_t* thr_num, int64_t thr_den, uint64_t* out_pos,
                             uint64_t* out_neg, int64_t* v_out, nmdlm_qbsm_stats* stats,
                             unsigned flags, void* ws, size_t ws_bytes, void* stream) {
  const int Nw = (N + 63) / 64;
  QbsmCall c;
  c.s_in = s_pos;
  c.s_neg = s_neg;
  c.seq_len = 0;
  c.T = T;
  c.M = M;
  c.K = K;
  c.W = W;
  c.ldw = ldw;
  c.N = N;
  c.mode = mode;
  c.bias = nullptr;
  c.cur_out = acc_out;
  c.theta_vec = nullptr;
  c.nseg = 1;
  c.seg_w = 1 << 30;
  for (int i = 0; i < kMaxSeg; ++i) {
    c.seg[i].ptr = out_pos;
    c.seg[i].ld_t = (int64_t)M * Nw;
    c.seg[i].ld_m = Nw;
    c.seg[i].theta = 1;
    c.seg[i].transposed = 0;
    c.seg[i].pos0 = 0;
    c.seg[i].ld_p = 0;
    c.seg[i].seq_len = 0;
    c.seg[i].ld_s = 0;
  }
  c.resid = nullptr;
  c.rld_t = c.rld_m = 0;
  c.lut = nullptr;
  c.lut_shift = 0;
  c.logits = nullptr;
  c.scale = nullptr;
  c.stats = stats;
  c.flags = flags;
  c.ev_begin = nullptr;
  c.ev_end = nullptr;
  c.u_in = nullptr;
  c.u_nparts = 0;
  c.u_out = nullptr;
  c.thr_num = thr_num;
  c.thr_den = thr_den;
  c.s_neg_out = out_neg;
  c.v_out = v_out;
  c.Wb = nullptr;

  Carver cv{static_cast<char*>(ws), 0, ws_bytes, true};
  QbsmScratch scr;
  carve_qbsm_scratch(cv, qbsm_limits_single(T, M, K, N), &scr);
  if (!cv.ok) return NMDLM_ERR_WORKSPACE;
  return launch_qbsm(c, scr, static_cast<hipStream_t>(stream));
}

// Checks shared by the two ternary products.
nmdlm_status ternary_args(const uint64_t* s_pos, const uint64_t* s_neg, int T, int M, int K,
                          const int8_t* W, int N, int64_t ldw, void* ws, size_t ws_bytes) {
  if (!s_pos || !s_neg || T < 1 || M < 1 || K < 1 || N < 1) return NMDLM_ERR_INVALID_ARG;
  if (T > NMDLM_MAX_T || K > NMDLM_MAX_TERNARY_K) return NMDLM_ERR_UNSUPPORTED;
  if (!weights_ok(W, K, N, ldw)) return NMDLM_ERR_INVALID_ARG;
  if ((int64_t)T * M > (1 << 19)) return NMDLM_ERR_UNSUPPORTED;
  if (!ws || !aligned(ws, 256) || ws_bytes < qbsm_ws(T, M, K, N)) return NMDLM_ERR_WORKSPACE;
  return NMDLM_OK;
}

}  // namespace

extern "C" {

nmdlm_status nmdlm_qbsm_ternary(const uint64_t* s_pos, const uint64_t* s_neg, int T, int M, int K,
                                const int8_t* W, int N, int64_t ldw, int32_t* acc_out,
                                nmdlm_qbsm_stats* stats, unsigned flags, void* ws, size_t ws_bytes,
                                void* stream) {
  if (!acc_out) return NMDLM_ERR_INVALID_ARG;
  const nmdlm_status rc = ternary_args(s_pos, s_neg, T, M, K, W, N, ldw, ws, ws_bytes);
  if (rc != NMDLM_OK) return rc;
  // |sum_t 2^(t-1) I_t| <= (2^T - 1) K 127 must fit int32
  if ((((int64_t)1 << T) - 1) * K * 127 >= ((int64_t)1 << 31)) return NMDLM_ERR_UNSUPPORTED;
  return ternary_product(s_pos, s_neg, T, M, K, W, N, ldw, EPI_BITWISE, acc_out, nullptr, 1,
                         nullptr, nullptr, nullptr, stats, flags, ws, ws_bytes, stream);
}

nmdlm_status nmdlm_qbsm_ternary_if(const uint64_t* s_pos, const uint64_t* s_neg, int T, int M,
                                   int K, const int8_t* W, int N, int64_t ldw,
                                   const int64_t* thr_num, int64_t thr_den, uint64_t* out_pos,
                                   uint64_t* out_neg, int64_t* v_out, nmdlm_qbsm_stats* stats,
                                   unsigned flags, void* ws, size_t ws_bytes, void* stream) {
  if (!thr_num || !out_pos || !out_neg) return NMDLM_ERR_INVALID_ARG;
  if (thr_den < 1) return NMDLM_ERR_INVALID_ARG;
  if (thr_den > NMDLM_MAX_THR_DEN) return NMDLM_ERR_UNSUPPORTED;
  const nmdlm_status rc = ternary_args(s_pos, s_neg, T, M, K, W, N, ldw, ws, ws_bytes);
  if (rc != NMDLM_OK) return rc;
  return ternary_product(s_pos, s_neg, T, M, K, W, N, ldw, EPI_MODIF, nullptr, thr_num, thr_den,
                         out_pos, out_neg, v_out, stats, flags, ws, ws_bytes, stream);
}

nmdlm_status nmdlm_if_neuron(const int32_t* cur, int T, int M, int N, int32_t theta,
                             const int32_t* theta_vec, const uint64_t* resid, int32_t* v_inout,
                             uint64_t* s_out, void* stream) {
  if (!cur || !s_out || T < 1 || M < 1 || N < 1) return NMDLM_ERR_INVALID_ARG;
  if (!theta_vec && theta <= 0) return NMDLM_ERR_INVALID_ARG;
  // one wave per (token, 64-neuron word): the launch grid stays within 2^32 threads
  if (T > NMDLM_MAX_T * 1024 || (int64_t)M * ((N + 63) / 64) > ((int64_t)1 << 26))
    return NMDLM_ERR_UNSUPPORTED;
  return launch_if(cur, T, M, N, theta, theta_vec, resid, v_inout, s_out,
                   static_cast<hipStream_t>(stream));
}

nmdlm_status nmdlm_qnl_lut(const int32_t* x, int64_t n, int shift, int mode, const uint8_t* lut,
                           uint8_t* y, void* stream) {
  if (n < 0 || !lut || (n > 0 && (!x || !y))) return NMDLM_ERR_INVALID_ARG;
  if (shift < 0 || shift > 31) return NMDLM_ERR_INVALID_ARG;
  if (mode != NMDLM_QNL_S8 && mode != NMDLM_QNL_U8) return NMDLM_ERR_INVALID_ARG;
  return launch_qnl(x, n, shift, mode, lut, y, static_cast<hipStream_t>(stream));
}

size_t nmdlm_bbm_attn_workspace_size(int T, int M, int H, int dh) {
  if (T < 1 || M < 1 || H < 1 || dh < 1) return 0;
  return align_up((size_t)T * M * H * dh * sizeof(int32_t), 256);
}

nmdlm_status nmdlm_bbm_attn(const uint64_t* q, const uint64_t* k_cache, const uint64_t* vt_cache,
                            int64_t cache_cap, int T, int M, int C, int H, int dh,
                            const uint8_t* lut_att, int32_t* a_out, int32_t theta_a,
                            uint64_t* s_out, void* ws, size_t ws_bytes, void* stream) {
  if (!q || !k_cache || !vt_cache || !lut_att) return NMDLM_ERR_INVALID_ARG;
  if (T < 1 || M < 1 || C < 0 || H < 1 || dh < 1) return NMDLM_ERR_INVALID_ARG;
  if (!a_out && !s_out) return NMDLM_ERR_INVALID_ARG;
  if (s_out && theta_a <= 0) return NMDLM_ERR_INVALID_ARG;
  if (T > NMDLM_MAX_T) return NMDLM_ERR_UNSUPPORTED;
  if (dh != 64 && dh != 128) return NMDLM_ERR_UNSUPPORTED;
  if ((int64_t)T * M > (1 << 19) || (int64_t)H * dh > NMDLM_MAX_K) return NMDLM_ERR_UNSUPPORTED;
  if (cache_cap % 64 != 0 || cache_cap < (int64_t)C + M) return NMDLM_ERR_INVALID_ARG;
  if ((int64_t)C + M > NMDLM_MAX_KEYS || cache_cap / 64 > INT_MAX) return NMDLM_ERR_UNSUPPORTED;
  int32_t* a = a_out;
  if (!a) {
    if (!ws || !aligned(ws, 256) || ws_bytes < nmdlm_bbm_attn_workspace_size(T, M, H, dh))
      return NMDLM_ERR_WORKSPACE;
    a = static_cast<int32_t*>(ws);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (!a_out) {
    // spikes only: one kernel with the IF fused in, when its LDS fits
    const nmdlm_status rf = launch_attn_if(q, k_cache, vt_cache, cache_cap, T, M, C, H, dh,
                                           lut_att, theta_a, s_out, nullptr, st);
    if (rf != NMDLM_ERR_UNSUPPORTED) return rf;
  }
  nmdlm_status rc = launch_attn(q, k_cache, vt_cache, cache_cap, T, M, C, H, dh, lut_att, a, st);
  if (rc != NMDLM_OK || !s_out) return rc;
  return launch_if(a, T, M, H * dh, theta_a, nullptr, nullptr, nullptr, s_out, st);
}

size_t nmdlm_block_step_workspace_size(const nmdlm_model* model, int M, unsigned flags) {
  if (!model || M < 1 || model->T < 1 || model->d < 64) return 0;
  return block_step_ws_size(model, M, flags);
}

nmdlm_status nmdlm_block_step(const nmdlm_model* md, nmdlm_step_io* io, void* ws, size_t ws_bytes,
                              void* stream) {
  if (!md || !io) return NMDLM_ERR_INVALID_ARG;
  if (md->n_layers < 0 || md->T < 1 || md->d < 64 || md->H < 1 || md->F < 1 || md->V < 1)
    return NMDLM_ERR_INVALID_ARG;
  if (md->T > NMDLM_MAX_T) return NMDLM_ERR_UNSUPPORTED;
  if (md->d % 64 != 0 || md->d % md->H != 0) return NMDLM_ERR_UNSUPPORTED;
  const int dh = md->d / md->H;
  if (dh != 64 && dh != 128) return NMDLM_ERR_UNSUPPORTED;
  if (md->d > NMDLM_MAX_K || md->F > NMDLM_MAX_K) return NMDLM_ERR_UNSUPPORTED;
  if (io->M < 1 || io->C < 0 || io->pos0 < 0) return NMDLM_ERR_INVALID_ARG;
  if (md->max_seq < 0 || io->n_seq < 0) return NMDLM_ERR_INVALID_ARG;
  const int n_seq = std::max(io->n_seq, 1);
  if (n_seq > std::max(md->max_seq, 1)) return NMDLM_ERR_INVALID_ARG;
  // several sequences: one row block of every product lies within a sequence
  if (n_seq > 1 && io->M % (16 / md->T) != 0) return NMDLM_ERR_UNSUPPORTED;
  const int64_t Mt = (int64_t)n_seq * io->M;
  if ((int64_t)md->T * Mt > (1 << 19)) return NMDLM_ERR_UNSUPPORTED;
  if (md->cache_cap % 64 != 0 || md->cache_cap < (int64_t)io->C + io->M)
    return NMDLM_ERR_INVALID_ARG;
  if ((int64_t)io->C + io->M > NMDLM_MAX_KEYS || md->cache_cap / 64 > INT_MAX)
    return NMDLM_ERR_UNSUPPORTED;
  if (md->n_layers > 0 && !md->layers) return NMDLM_ERR_INVALID_ARG;
  const unsigned path_req = (io->flags >> NMDLM_PATH_SHIFT) & 0x7u;
  const bool forced_blocked = path_req == 6u || path_req == 7u;
  for (int l = 0; l < md->n_layers; ++l) {
    const nmdlm_layer& L = md->layers[l];
    if (!weights_ok(L.w_qkv, md->d, 3 * md->d, 3 * (int64_t)md->d) ||
        !weights_ok(L.w_o, md->d, md->d, md->d) || !weights_ok(L.w_up, md->d, md->F, md->F) ||
        !weights_ok(L.w_dn, md->F, md->d, md->d))
      return NMDLM_ERR_INVALID_ARG;
    if (!L.lut_att || !L.lut_act || !L.k_cache || !L.vt_cache) return NMDLM_ERR_INVALID_ARG;
    if (!blocked_ok(L.w_qkv_b, md->d, 3 * md->d) || !blocked_ok(L.w_o_b, md->d, md->d) ||
        !blocked_ok(L.w_up_b, md->d, md->F) || !blocked_ok(L.w_dn_b, md->F, md->d))
      return NMDLM_ERR_INVALID_ARG;
    // paths 6 and 7 (every word from the blocked copies) need every copy
    if (forced_blocked && (!L.w_qkv_b || !L.w_o_b || !L.w_up_b || !L.w_dn_b))
      return NMDLM_ERR_INVALID_ARG;
    if (L.theta_q <= 0 || L.theta_k <= 0 || L.theta_v <= 0 || L.theta_a <= 0 || L.theta_o <= 0 ||
        L.theta_up <= 0 || L.theta_dn <= 0)
      return NMDLM_ERR_INVALID_ARG;
    if (L.s_up < 0 || L.s_up > 31) return NMDLM_ERR_INVALID_ARG;
  }
  if (!io->x_in) {
    if (!md->emb || !md->pos_ch) return NMDLM_ERR_INVALID_ARG;
    if (!io->tokens && !io->masked) return NMDLM_ERR_INVALID_ARG;
    if ((int64_t)io->pos0 + io->M > md->max_pos) return NMDLM_ERR_INVALID_ARG;
  }
  const bool head = !(io->flags & NMDLM_NO_HEAD);
  if (head) {
    if (!weights_ok(md->w_head, md->d, md->V, md->V) || !md->head_scale ||
        !blocked_ok(md->w_head_b, md->d, md->V) || (forced_blocked && !md->w_head_b))
      return NMDLM_ERR_INVALID_ARG;
    if (!io->tokens || !io->masked || io->k_unmask < 0) return NMDLM_ERR_INVALID_ARG;
    if (io->M > NMDLM_MAX_HEAD_M) return NMDLM_ERR_UNSUPPORTED;
  }
  if (!ws || !aligned(ws, 256) || ws_bytes < block_step_ws_size(md, (int)Mt, io->flags))
    return NMDLM_ERR_WORKSPACE;
  if (io->prof_events && io->n_prof_events > 0) {
    // timing events are plain records: not available inside stream capture
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(static_cast<hipStream_t>(stream), &cs) != hipSuccess) return NMDLM_ERR_HIP;
    if (cs != hipStreamCaptureStatusNone) return NMDLM_ERR_UNSUPPORTED;
  }
  return block_step_impl(md, io, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

nmdlm_status nmdlm_workspace_clear(void* ws, size_t ws_bytes, void* stream) {
  if (!ws || !aligned(ws, 16) || ws_bytes % 16 != 0) return NMDLM_ERR_INVALID_ARG;
  return launch_fill_zero(ws, ws_bytes, static_cast<hipStream_t>(stream));
}

}  // extern "C"
