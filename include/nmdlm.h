/*
 * libnmdlm — the block-denoising step of a neuromorphic masked diffusion
 * language model (N-MDLM), for AMD Instinct MI355X (gfx950).
 *
 * Plain C ABI: device pointers, sizes and a HIP stream (passed as void*,
 * NULL = the default stream).  No call allocates or frees memory; scratch
 * memory is a caller-provided workspace whose size is given by the
 * *_workspace_size functions.  Every call validates its arguments on the
 * host first and, on error, returns a status without enqueueing any work.
 * Calls are asynchronous with respect to the host: outputs (and statistics)
 * are valid once the stream has reached them.  Apart from the static scratch
 * of nmdlm_qbsm_noalloc, the library keeps no global mutable state; two calls
 * may run concurrently on different streams when their workspaces and
 * outputs do not overlap.
 *
 * Spike tensors are {0,1}^{T x M x K} packed little-endian into uint64
 * words: tensor [T][M][ceil(K/64)], bit j of word w is channel 64*w + j.
 * Padding bits must be zero on input and are written as zero on output.
 *
 * Weight matrices are int8 [K][ldw] row-major: row k holds the weights that
 * leave input neuron k (its fan-out), so the products below skip whole rows.
 * ldw is a multiple of 16 and >= N; bytes [N, ldw) of a row may be read and
 * are ignored.  K * ldw must be below 2^31.
 */
#ifndef NMDLM_H
#define NMDLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define NMDLM_ABI_VERSION 5

typedef enum nmdlm_status {
  NMDLM_OK = 0,
  NMDLM_ERR_INVALID_ARG = 1,  /* null pointer, size <= 0, threshold <= 0, ... */
  NMDLM_ERR_UNSUPPORTED = 2,  /* valid but outside the supported envelope     */
  NMDLM_ERR_WORKSPACE = 3,    /* workspace missing or smaller than required   */
  NMDLM_ERR_HIP = 4           /* a HIP launch reported an error               */
} nmdlm_status;

/* flags (bitwise OR) */
#define NMDLM_FORCE_DENSE 0x1u   /* read every weight row: the un-skipped product */
#define NMDLM_NO_HEAD     0x2u   /* block step without head/confidence/unmask    */
#define NMDLM_ATTN_FUSED  0x4u   /* block step: attention and the IF of its output
                                    in one kernel (one workgroup per head and 16
                                    queries, all timesteps); default is two
                                    kernels.  Results do not depend on it.      */
/* bits 8..15 of the flags of nmdlm_qbsm: force the number of K splits
 * (0 = automatic).  Results do not depend on it. */
#define NMDLM_SPLIT_SHIFT 8u
/* bits 16..19: force rows per tile group (0 = automatic; 1,2,4,8 = 16..128
 * rows).  Results do not depend on it. */
#define NMDLM_ROWTILE_SHIFT 16u
/* bits 20..22: product kernel (0 = automatic; 1 = separate pass building the
 * active-row list; 2 = single kernel with an in-kernel list; 3 = single
 * kernel over 64-channel words, loading only active rows into registers;
 * 4 = as 3, gathering the active rows straight into LDS; 5 = as 3 with a
 * scalar gather-accumulate product in place of MFMA: per spike of a row,
 * the active weight row's columns are loaded and added; 6 = as 3 over the
 * blocked copy of the weights, nmdlm_qbsm_blocked only; 7 = as 6 with wide
 * tiles where the row tile is 64 rows: a workgroup takes four 64-column
 * tiles, each wave one of them over all of K).  Results do not depend on
 * it. */
#define NMDLM_PATH_SHIFT 20u
#define NMDLM_NO_FUSE (1u << NMDLM_PATH_SHIFT)

/* Supported envelope (NMDLM_ERR_UNSUPPORTED beyond it). */
#define NMDLM_MAX_TERNARY_K 16384
#define NMDLM_MAX_T 8
#define NMDLM_MAX_K 65536
#define NMDLM_MAX_HEAD_M 4096   /* block tokens of a step that runs the head */
#define NMDLM_MAX_KEYS 8388608  /* attention keys C+M per sequence (2^23): the
                                   sum of the table weights over the keys,
                                   at most 255 per key, stays below 2^31   */

/* bits of the device status word of a block step (nmdlm_step_io.status) */
#define NMDLM_STATUS_TOKEN_CLAMPED 0x1  /* a token id outside [0, V] was read as
                                           the nearest of 0 and V (the mask id) */

/*
 * Statistics of one spike product, written by the device (int64 so the
 * host can sum them).  weight_bytes is the number of weight bytes the
 * product reads: k_active * n (the per-block load of Eq. (13)).
 */
typedef struct nmdlm_qbsm_stats {
  int64_t k_total;       /* K                                             */
  int64_t k_active;      /* input neurons that spike at least once in the
                            block (rows of W that are read)               */
  int64_t n;             /* N                                             */
  int64_t weight_bytes;  /* k_active * n                                  */
} nmdlm_qbsm_stats;

/* ------------------------------------------------------------------------
 * nmdlm_qbsm — quantised-weight x binary-spike product with row skipping
 *
 * Sec. IV-A: the linear operation over the B*T rows of a block,
 *     I[t,m,n] = bias[n] + sum_k S[t,m,k] * W[k,n],
 * where, by assumption (ii), row k of W is read only if input neuron k
 * spikes at least once among all T*M rows.  The result is identical to the
 * dense product (integer arithmetic, no overflow for K*127 + |bias| < 2^31).
 *
 * Optional fused integrate-and-fire epilogue (Sec. II-B, Eqs. (3)-(4),
 * integrate-then-fire with soft reset, membrane starting at 0):
 *     V = 0; for t: V += I[t]; s[t] = (V >= theta); V -= s[t]*theta.
 *
 *   s_in      device, spikes [T][M][ceil(K/64)]
 *   T, M, K   1 <= T <= 8, M >= 1, T*M <= 2^19, 1 <= K <= 65536
 *   W, N, ldw device int8 [K][ldw] (see above), N >= 1
 *   bias      device int32 [N] or NULL (zero)
 *   cur_out   device int32 [T][M][N] or NULL: the currents I
 *   theta     threshold (> 0) used when s_out is given; ignored otherwise
 *   theta_vec device int32 [N] per-neuron thresholds (> 0) or NULL (use theta)
 *   s_out     device spikes [T][M][ceil(N/64)] or NULL; at least one of
 *             cur_out / s_out must be given
 *   stats     device, one nmdlm_qbsm_stats, or NULL
 *   flags     NMDLM_FORCE_DENSE, split/row-tile overrides
 *   ws        device workspace of ws_bytes >= nmdlm_qbsm_workspace_size();
 *             zero-filled before its first use; every call leaves its
 *             counter region zero again
 *   stream    hipStream_t or NULL
 * ------------------------------------------------------------------------ */
nmdlm_status nmdlm_qbsm(const uint64_t* s_in, int T, int M, int K,
                        const int8_t* W, int N, int64_t ldw,
                        const int32_t* bias, int32_t* cur_out,
                        int32_t theta, const int32_t* theta_vec,
                        uint64_t* s_out, nmdlm_qbsm_stats* stats,
                        unsigned flags, void* ws, size_t ws_bytes, void* stream);

size_t nmdlm_qbsm_workspace_size(int T, int M, int K, int N);

/* ------------------------------------------------------------------------
 * Blocked weights — a second layout of a weight matrix for products over
 * many rows (prefills, steps over many sequences), where the block union is
 * dense and the products are plain int8 contractions.
 *
 * Sec. IV-A (Eqs. (12)-(13)): the row-load rule reads row k of W only if
 * input neuron k spikes in the block.  Over the blocked copy the rule is
 * applied per 64-row word: a word with no active row is skipped, every row
 * of an active word is read (rows that do not spike meet zero inputs, so the
 * result is unchanged).  At dense unions the bytes read are those of the
 * row-major path; the copy's bytes sit in MFMA operand order, so a 64-row
 * word of a 64-column tile is four 16-byte loads per lane with no byte
 * transposes.
 *
 * Layout: for word w (rows 64w..64w+63) and column tile x (columns
 * 64x..64x+63), 4096 bytes at offset (w * ceil(N/64) + x) * 4096; within
 * them, operand v (0..3), lane l = 16g + c (0..63), byte j (0..15) at
 * v*1024 + l*16 + j holds W[64w + 16g + j][64x + 4c + v], zero past K or N.
 *
 * nmdlm_weight_blocked_bytes: size of the copy (0 for invalid sizes).
 * nmdlm_weight_block: writes the copy Wb (device, 16-byte aligned, of
 *   nmdlm_weight_blocked_bytes) from W (as for nmdlm_qbsm); asynchronous on
 *   the stream.  The copy must be rebuilt whenever W changes.
 * nmdlm_qbsm_blocked: nmdlm_qbsm (same arguments, results and errors) with
 *   the blocked copy Wb of W also given.  With path 6 in the flags every
 *   word is read from the copy; unforced, each wave of the product reads it
 *   when its words' union is dense: on average at least
 *   NMDLM_BLOCKED_MIN_ROWS active rows of 64 per active word, counted over
 *   the row blocks of the product that read the same words (the whole words
 *   then cost at most twice the active rows' bytes from HBM); else the
 *   row-major rows of W.  Products of 64-row tiles over at least 1536 output
 *   tiles of 64 x 64 (and path 7 in the flags) take wide tiles: four column
 *   tiles per workgroup, each read from the copy over all of K.  Results do
 *   not depend on which is used.
 *   NMDLM_ERR_UNSUPPORTED when the copy would exceed 2^31 bytes.
 * ------------------------------------------------------------------------ */
#define NMDLM_BLOCKED_MIN_ROWS 32
size_t nmdlm_weight_blocked_bytes(int K, int N);
nmdlm_status nmdlm_weight_block(const int8_t* W, int K, int N, int64_t ldw,
                                int8_t* Wb, void* stream);
nmdlm_status nmdlm_qbsm_blocked(const uint64_t* s_in, int T, int M, int K,
                                const int8_t* W, const int8_t* Wb, int N,
                                int64_t ldw, const int32_t* bias,
                                int32_t* cur_out, int32_t theta,
                                const int32_t* theta_vec, uint64_t* s_out,
                                nmdlm_qbsm_stats* stats, unsigned flags,
                                void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * nmdlm_qbsm_noalloc — nmdlm_qbsm without a workspace argument, for callers
 * that cannot allocate device memory (code under stream capture, tight
 * serving loops, harnesses that forbid allocation).  The call allocates
 * nothing: its scratch is a static device array of
 * NMDLM_NOALLOC_SCRATCH_BYTES that each GPU holds from the library's first
 * call on it until the process ends (that first call also clears it with a
 * fill kernel on the stream).  Every call on one GPU shares that GPU's array:
 * calls that overlap on one GPU (other streams, other host threads) race
 * and must not be issued.  Sequential calls on a stream are safe: every call
 * leaves the array's counter region at zero, as nmdlm_qbsm does.
 *
 * Arguments, results and errors are those of nmdlm_qbsm (same computation,
 * same kernels), less ws and ws_bytes; a product whose
 * nmdlm_qbsm_workspace_size() exceeds NMDLM_NOALLOC_SCRATCH_BYTES returns
 * NMDLM_ERR_UNSUPPORTED before any work is enqueued.
 * ------------------------------------------------------------------------ */
#define NMDLM_NOALLOC_SCRATCH_BYTES 16777216  /* 16 MiB per GPU */
nmdlm_status nmdlm_qbsm_noalloc(const uint64_t* s_in, int T, int M, int K,
                                const int8_t* W, int N, int64_t ldw,
                                const int32_t* bias, int32_t* cur_out,
                                int32_t theta, const int32_t* theta_vec,
                                uint64_t* s_out, nmdlm_qbsm_stats* stats,
                                unsigned flags, void* stream);

/* ------------------------------------------------------------------------
 * nmdlm_ternary_encode — adaptive quantisation and ternary bitwise coding of
 * integer activations (Sec. III-B, Eqs. (7)-(8)), per token m:
 *     S = sum_i |a_i|;  V_th = S / (D K)   (mean(|a|) / K, kept exact)
 *     q_i = round(a_i / V_th) = round(a_i D K / S), halves away from zero,
 *           0 when S = 0, |q_i| capped at 2^T - 1;
 *     s_{i,t} = sign(q_i) * bit t-1 of |q_i|,  t = 1..T  (q = sum 2^(t-1) s_t)
 *
 *   a       device int32 [M][D] (a layer's integer output)
 *   K       quantisation levels per mean magnitude (>= 1; D*K < 2^20)
 *   T       bits = timesteps (1..NMDLM_MAX_T)
 *   s_pos   device spikes [T][M][ceil(D/64)]: bit set where s = +1
 *   s_neg   device spikes [T][M][ceil(D/64)]: bit set where s = -1
 *   s_sum   device int64 [M] or NULL: S per token (V_th = S / (D K))
 * Integer arithmetic throughout: the result does not depend on rounding.
 * ------------------------------------------------------------------------ */
nmdlm_status nmdlm_ternary_encode(const int32_t* a, int M, int D, int K, int T,
                                  uint64_t* s_pos, uint64_t* s_neg, int64_t* s_sum,
                                  void* stream);

/* ------------------------------------------------------------------------
 * nmdlm_qbsm_ternary — the spiking product on ternary bitwise-coded spikes
 * and its reconstruction (Sec. III-B, Eqs. (10)-(11); row-load rule of
 * Sec. IV-A on either spike plane):
 *     I_t[m,n] = sum_k (s_pos - s_neg)[t,m,k] * W[k,n]      t = 1..T
 *     acc[m,n] = sum_t 2^(t-1) I_t[m,n]   (= sum_k q[m,k] W[k,n], exact)
 * A weight row k is read only if input k spikes (either sign) somewhere in
 * the block.  The layer output is V_th[m] * acc[m,n] (V_th from
 * nmdlm_ternary_encode); acc can feed nmdlm_ternary_encode of the next
 * layer directly, since the per-token scale cancels in Eq. (7).
 *
 *   s_pos, s_neg  device spikes [T][M][ceil(K/64)] (never both set)
 *   W, ldw, N     as nmdlm_qbsm; K <= NMDLM_MAX_TERNARY_K and
 *                 (2^T - 1) * K * 127 < 2^31 (else NMDLM_ERR_UNSUPPORTED)
 *   acc_out       device int32 [M][N]
 *   stats         as nmdlm_qbsm (active rows of the union of both planes)
 *   flags, ws     as nmdlm_qbsm (ws of nmdlm_qbsm_workspace_size(T, M, K, N))
 * ------------------------------------------------------------------------ */
nmdlm_status nmdlm_qbsm_ternary(const uint64_t* s_pos, const uint64_t* s_neg, int T,
                                int M, int K, const int8_t* W, int N, int64_t ldw,
                                int32_t* acc_out, nmdlm_qbsm_stats* stats,
                                unsigned flags, void* ws, size_t ws_bytes,
                                void* stream);

/* ------------------------------------------------------------------------
 * nmdlm_qbsm_ternary_if — the spiking product on ternary bitwise-coded
 * spikes followed by the modified IF neuron of Sec. III-B (Eqs. (9)-(10)),
 * which turns the per-timestep currents back into ternary spike planes;
 * row-load rule of Sec. IV-A on either input plane.  Per token m and output
 * neuron n, with I_t = sum_k (s_pos - s_neg)[t,m,k] * W[k,n] and the
 * threshold Vth = thr_num[m] / thr_den:
 *     V = 0; for t = 1..T:
 *       V += 2^(t-1) I_t
 *       s_t = +1 if V >= 2^(t-1) Vth, -1 if V <= -2^(t-1) Vth, else 0
 *       V -= 2^(t-1) s_t Vth
 * so that Vth sum_t 2^(t-1) s_t = sum_t 2^(t-1) I_t - V (Eq. (11), the final
 * membrane being its error).  Readings: the 2^t of Eqs. (9)-(10) counts steps
 * from 0 (weight 2^(t-1) for step t = 1..T, as in Eq. (8)); the membrane
 * integrates before it fires, as for Eqs. (3)-(4); a token with
 * thr_num[m] = 0 (Vth = 0, an all-zero activation vector) emits no spike.
 * The paper's threshold is the input's quantisation step: pass s_sum of
 * nmdlm_ternary_encode as thr_num and D*K as thr_den.  All arithmetic is
 * integer (the membrane is kept times thr_den in 64 bits): exact.
 *
 *   s_pos, s_neg  device spikes [T][M][ceil(K/64)] (never both set)
 *   W, ldw, N     as nmdlm_qbsm; K <= NMDLM_MAX_TERNARY_K
 *   thr_num       device int64 [M], each in [0, 2^55) (larger values give
 *                 undefined spikes)
 *   thr_den       1 <= thr_den <= NMDLM_MAX_THR_DEN (else INVALID_ARG /
 *                 UNSUPPORTED)
 *   out_pos       device spikes [T][M][ceil(N/64)]: bit set where s_t = +1
 *   out_neg       device spikes [T][M][ceil(N/64)]: bit set where s_t = -1
 *                 (padding bits written as zero; the planes can feed the next
 *                 nmdlm_qbsm_ternary_if directly)
 *   v_out         device int64 [M][N] or NULL: thr_den * final membrane
 *   stats, flags, ws   as nmdlm_qbsm_ternary
 * ------------------------------------------------------------------------ */
#define NMDLM_MAX_THR_DEN 16777216
nmdlm_status nmdlm_qbsm_ternary_if(const uint64_t* s_pos, const uint64_t* s_neg, int T,
                                   int M, int K, const int8_t* W, int N, int64_t ldw,
                                   const int64_t* thr_num, int64_t thr_den,
                                   uint64_t* out_pos, uint64_t* out_neg, int64_t* v_out,
                                   nmdlm_qbsm_stats* stats, unsigned flags, void* ws,
                                   size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * nmdlm_if_neuron — integrate-and-fire with soft reset (Sec. II-B,
 * Eqs. (3)-(4)), integrate-then-fire order, equality fires, no lower clamp:
 *     V = v_in (or 0); for t: V += cur[t] + theta*resid[t];
 *                             s[t] = (V >= theta); V -= s[t]*theta.
 *
 *   cur       device int32 [T][M][N]
 *   theta     threshold (> 0); theta_vec device int32 [N] or NULL
 *   resid     device spikes [T][M][ceil(N/64)] or NULL: membrane shortcut
 *   v_inout   device int32 [M][N] or NULL: initial membrane in, final out
 *   s_out     device spikes [T][M][ceil(N/64)]
 * Limits: T <= 8192 and M * ceil(N/64) <= 2^26, else NMDLM_ERR_UNSUPPORTED.
 * ------------------------------------------------------------------------ */
nmdlm_status nmdlm_if_neuron(const int32_t* cur, int T, int M, int N,
                             int32_t theta, const int32_t* theta_vec,
                             const uint64_t* resid, int32_t* v_inout,
                             uint64_t* s_out, void* stream);

/* ------------------------------------------------------------------------
 * nmdlm_qnl_lut — 8-bit-in / 8-bit-out table non-linearity.
 * The paper names this operation only in its list of acronyms (QNL: a
 * quantised non-linearity implemented as a look-up table), as one of the
 * operations of the neuromorphic layers of Fig. 1; it gives no formula.
 * This library's reading, also used by the block step on the FFN up
 * current:
 *   NMDLM_QNL_S8: index = byte of clamp(floor(x / 2^shift), -128, 127)
 *   NMDLM_QNL_U8: index = clamp(x, 0, 255)            (shift ignored)
 *   y[i] = lut[index]  (the raw table byte; read it as int8 in S8 mode)
 *
 *   x    device int32 [n];  lut device uint8 [256];  y device uint8 [n]
 *   0 <= shift <= 31; n = 0 enqueues nothing
 * Errors: NMDLM_ERR_INVALID_ARG for n < 0, a missing pointer, a shift out of
 * range or an unknown mode (nothing is enqueued).
 * ------------------------------------------------------------------------ */
#define NMDLM_QNL_S8 0
#define NMDLM_QNL_U8 1
nmdlm_status nmdlm_qnl_lut(const int32_t* x, int64_t n, int shift, int mode,
                           const uint8_t* lut, uint8_t* y, void* stream);

/* ------------------------------------------------------------------------
 * nmdlm_bbm_attn — attention on spike operands.  The paper names the
 * operations involved only in its list of acronyms: binary-binary
 * multiplication (BBM, here the query-key product of two spike vectors),
 * quantised dynamic multiplication (QDM, the table weights times the value
 * spikes), a look-up-table non-linearity (QNL) and fixed-point arithmetic
 * (FixP, the integer normalisation); Fig. 1 places attention in every
 * neuromorphic layer.  The formula below is this library's reading.  For
 * every timestep t, head h, block query i < M and key j < C+M:
 *     s = popcount(Q[t,i,head h] AND K[t,j,head h])       in [0, dh]
 *     p = lut_att[s]                                       (uint8)
 *     a[t,i,c] = floor(256 * sum_j p * V[t,j,c] / sum_j p)   (0 if sum_j p = 0)
 * then optionally A = IF(a, theta_a) over t.  The block's own keys/values
 * must already be in rows [C, C+M) of the caches.
 *
 *   q         device spikes [T][M][d/64], d = H*dh
 *   k_cache   device spikes [T][cache_cap][d/64]  (token-major)
 *   vt_cache  device spikes, word-major: [T][cache_cap/64][d]; bit j%64 of
 *             word (t, j/64, c) is V[t,j,c] (the 64 positions of one word
 *             for every channel lie side by side)
 *   cache_cap multiple of 64, >= C+M
 *   dh        64 or 128 (else NMDLM_ERR_UNSUPPORTED): scores stay within
 *             the 256-entry table
 *   limits    T*M <= 2^19, d <= NMDLM_MAX_K and C+M <= NMDLM_MAX_KEYS, else
 *             NMDLM_ERR_UNSUPPORTED
 *   lut_att   device uint8 [256]
 *   a_out     device int32 [T][M][d] or NULL
 *   theta_a   threshold (> 0) when s_out is given
 *   s_out     device spikes [T][M][d/64] or NULL (at least one output)
 *   ws        workspace of nmdlm_bbm_attn_workspace_size() bytes (used when
 *             a_out is NULL)
 * ------------------------------------------------------------------------ */
nmdlm_status nmdlm_bbm_attn(const uint64_t* q, const uint64_t* k_cache,
                            const uint64_t* vt_cache, int64_t cache_cap,
                            int T, int M, int C, int H, int dh,
                            const uint8_t* lut_att, int32_t* a_out,
                            int32_t theta_a, uint64_t* s_out,
                            void* ws, size_t ws_bytes, void* stream);

size_t nmdlm_bbm_attn_workspace_size(int T, int M, int H, int dh);

/* ------------------------------------------------------------------------
 * nmdlm_block_step — one denoising step z_{s+1} = f_dec(z_s, h) of block
 * diffusion (Sec. III-A, Eq. (6)) through a stack of spiking layers, or a
 * context prefill (Eq. (5): the same stack over the context tokens with
 * C = 0 and NMDLM_NO_HEAD).
 *
 * Per layer (Fig. 1: IF neurons in every layer; the wiring below is this
 * library's reading, the paper gives no layer internals):
 *   Q,K,V = IF(QBSM(X, W_qkv))   (thresholds q, k, v; K,V -> cache rows [C,C+M))
 *   A     = IF(attn(Q, caches), theta_a)
 *   X1    = IF(QBSM(A, W_o), theta_o, residual X)
 *   H     = IF(lut_act[QBSM(X1, W_up) >> s_up], theta_up)
 *   Y     = IF(QBSM(H, W_dn), theta_dn, residual X1)
 * Head (unless NMDLM_NO_HEAD): acc[m,v] = sum_t sum_c Y[t,m,c] W_head[c,v],
 * logit = (float)acc * head_scale[v]; pred = argmax (ties: smallest id);
 * conf = 1 / sum_v exp(logit_v - logit_pred) (fp64); then the k_unmask
 * masked positions of highest confidence (ties: lower position) take their
 * predicted token (B/S tokens per step, Sec. III-A).
 *
 * Several sequences in one step (io->n_seq > 1): n_seq independent
 * sequences at the same block (same M, C, pos0) share every product, so a
 * weight row is read once when it is active for any of their n_seq*M tokens
 * (the row-load rule of Sec. IV over the batch); attention, the caches and
 * the unmasking stay per sequence.  Token-indexed buffers then hold the
 * sequences one after the other: tokens/masked/pred/conf [n_seq][M], spikes
 * [T][n_seq*M][d/64], logits [n_seq*M][V], unmasked_pos [n_seq][k_unmask];
 * the caches of sequence s start s*T*cache_cap*d/64 words into k_cache and
 * vt_cache (both hold model->max_seq sequences).  With n_seq > 1, M must be
 * a multiple of 16/T (integer division) and NMDLM_ATTN_FUSED is ignored.
 *
 * Token ids: the block input reads the token table at row tokens[m] for an
 * unmasked position and at row V (the mask token) for a masked one; ids are
 * expected in [0, V).  An id outside [0, V] is read as the nearest of 0 and V
 * (never out of bounds) and flags NMDLM_STATUS_TOKEN_CLAMPED in io->status.
 * Limits: C+M <= NMDLM_MAX_KEYS and cache_cap/64 <= 2^31-1, else
 * NMDLM_ERR_UNSUPPORTED.
 * ------------------------------------------------------------------------ */
typedef struct nmdlm_layer {
  const int8_t* w_qkv;   /* device [d][3d]: columns Q | K | V */
  const int8_t* w_o;     /* device [d][d]  */
  const int8_t* w_up;    /* device [d][F]  */
  const int8_t* w_dn;    /* device [F][d]  */
  int32_t theta_q, theta_k, theta_v, theta_a, theta_o, theta_up, theta_dn;
  int32_t s_up;          /* right shift before lut_act (0..31) */
  const uint8_t* lut_att;/* device [256] attention score table */
  const uint8_t* lut_act;/* device [256] activation table (int8 bytes) */
  uint64_t* k_cache;     /* device [T][cache_cap][d/64]      */
  uint64_t* vt_cache;    /* device [T][cache_cap/64][d]: bit j%64 of word
                            (t, j/64, c) is value channel c of position j */
  /* Blocked copies (nmdlm_weight_block, ldw = N) of the four weights, or
   * NULL.  With a copy, each wave of a product reads it when its words'
   * union, counted over the row blocks that share the words, is dense
   * (NMDLM_BLOCKED_MIN_ROWS), else the row-major rows.  Path 6 in the flags
   * (every word from the copies) requires every copy, and the head's when
   * the step runs the head (NMDLM_ERR_INVALID_ARG otherwise).  Results do
   * not depend on it. */
  const int8_t* w_qkv_b;
  const int8_t* w_o_b;
  const int8_t* w_up_b;
  const int8_t* w_dn_b;
} nmdlm_layer;

typedef struct nmdlm_model {
  int n_layers, d, H, F, V, T;
  int64_t cache_cap;          /* multiple of 64 */
  int max_pos;                /* rows of pos_ch */
  const nmdlm_layer* layers;  /* HOST array [n_layers] */
  const uint64_t* emb;        /* device [V+1][T][d/64]; row V = mask token */
  const int32_t* pos_ch;      /* device [max_pos][T]: channel of the single
                                 position spike ORed into the token spikes */
  const int8_t* w_head;       /* device [d][V] (NULL allowed with NO_HEAD) */
  const float* head_scale;    /* device [V]                                */
  int max_seq;                /* sequences the caches hold (0 counts as 1):
                                 k_cache [max_seq][T][cache_cap][d/64],
                                 vt_cache [max_seq][T][cache_cap/64][d]     */
  const int8_t* w_head_b;     /* blocked copy of w_head (ldw = V) or NULL   */
} nmdlm_model;

typedef struct nmdlm_step_io {
  int M;                   /* tokens in the block (or context, in prefill)   */
  int C;                   /* cache rows already holding context            */
  int pos0;                /* sequence position of the first block token    */
  unsigned flags;          /* NMDLM_NO_HEAD, NMDLM_FORCE_DENSE              */
  const uint64_t* x_in;    /* device [T][M][d/64] block input spikes, or NULL:
                              assemble from tokens/masked, emb and pos_ch   */
  int32_t* tokens;         /* device [M] in/out (may be NULL with x_in and
                              NO_HEAD)                                       */
  uint8_t* masked;         /* device [M] in/out, 1 = still masked           */
  int k_unmask;            /* tokens revealed by this step                  */
  uint64_t* y_out;         /* device [T][M][d/64] last layer spikes or NULL */
  float* logits;           /* device [M][V] or NULL (workspace is used)     */
  int32_t* pred;           /* device [M] or NULL                            */
  double* conf;            /* device [M] or NULL                            */
  int32_t* unmasked_pos;   /* device [k_unmask] or NULL: chosen positions in
                              selection order, -1 when fewer were masked    */
  nmdlm_qbsm_stats* stats; /* device [4*n_layers + 1] or NULL: per product
                              (QKV, O, up, down per layer, then the head)  */
  void** prof_events;      /* HOST array of hipEvent_t or NULL: when given,
                              events 2i and 2i+1 take the start and end
                              times of the main kernel of product i (same
                              order as stats), stamped by its dispatch;
                              NMDLM_ERR_UNSUPPORTED inside stream capture  */
  int n_prof_events;       /* length of prof_events                         */
  int n_seq;               /* sequences in the step, 1..max(1, max_seq) (0
                              counts as 1); M is per sequence              */
  int32_t* status;         /* device int32 or NULL: the step ORs in
                              NMDLM_STATUS_* bits (the caller clears it);
                              a token id outside [0, V] is read as the
                              nearest of 0 and V and sets
                              NMDLM_STATUS_TOKEN_CLAMPED                   */
} nmdlm_step_io;

nmdlm_status nmdlm_block_step(const nmdlm_model* model, nmdlm_step_io* io,
                              void* ws, size_t ws_bytes, void* stream);

/* Workspace of a step over M block tokens in all (n_seq * M for a step of
 * several sequences). */
size_t nmdlm_block_step_workspace_size(const nmdlm_model* model, int M,
                                       unsigned flags);

/* Clears a workspace region with a fill kernel on the stream (use once on a
 * new workspace). */
nmdlm_status nmdlm_workspace_clear(void* ws, size_t ws_bytes, void* stream);

const char* nmdlm_status_string(nmdlm_status s);
int nmdlm_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* NMDLM_H */
