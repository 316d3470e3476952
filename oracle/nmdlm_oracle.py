"""CPU oracle for the N-MDLM block-denoising step (test infrastructure only).

This module is the checker, not the product.  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  It shares no code with the HIP library: it reads the same seeded
inputs (``workloads.synth``) and nothing else.

Everything here is the plain, dense, un-skipped definition:

* integer products are computed over *all* input channels (multiplying by the
  0/1 spike) with a float64 matrix product.  Every operand is an integer and
  every partial sum is an integer of magnitude < 2**53, so the float64 product
  is exact whatever order the library sums in; the result is checked to fit
  in int32 (the bound the GPU relies on);
* neuron updates, lookup tables, attention normalisation and unmasking are
  written out in the order of the definitions below.

Where the paper is silent, the readings used are listed next to each function
(IF update order, residual path, attention formulation, table placement,
head read-out, unmask rule); they are the binding specification for the GPU
library as well.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

INT32_MAX = 2 ** 31 - 1


def _check_int32(x: np.ndarray, what: str) -> None:
    if x.size and (x.max() > INT32_MAX or x.min() < -INT32_MAX - 1):
        raise OverflowError(f"{what} leaves the int32 range")


def _exact_matmul(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Integer matrix product via float64 (exact: all values are integers whose
    partial sums stay far below 2**53 for the shapes used here)."""
    a64 = np.asarray(a, dtype=np.float64)
    b64 = np.asarray(b, dtype=np.float64)
    bound = np.abs(a64).max(initial=0) * np.abs(b64).max(initial=0) * a64.shape[-1]
    if bound >= 2.0 ** 53:
        raise OverflowError("float64 product would not be exact")
    return np.rint(a64 @ b64).astype(np.int64)


# ----------------------------------------------------------------------------
# QBSM: block linear operation over B*T spike rows (Sec. IV-A)
# ----------------------------------------------------------------------------
def qbsm(S: np.ndarray, W: np.ndarray, bias: np.ndarray | None = None) -> np.ndarray:
    """I[t,m,n] = bias[n] + sum_k S[t,m,k] * W[k,n], over every k.

    Sec. IV-A: Y = X W^T with X the spike trains of the B tokens over T
    steps stacked as B*T rows.  Our W is stored [K][N] (row k = the weights
    leaving input neuron k), so Y = X W here.  The bias is added once per
    timestep (the paper names no bias; zero where none is given).
    S: 0/1 array [T][M][K]; W: int8 [K][N]; returns int64 [T][M][N].
    """
    S = np.asarray(S)
    T, M, K = S.shape
    if W.shape[0] != K:
        raise ValueError("S and W disagree on K")
    I = _exact_matmul(S.reshape(T * M, K), W).reshape(T, M, W.shape[1])
    if bias is not None:
        I = I + np.asarray(bias, dtype=np.int64)[None, None, :]
    _check_int32(I, "QBSM current")
    return I


def block_union(S: np.ndarray) -> np.ndarray:
    """Assumption (ii) of Sec. IV-A: input channel k needs its weight row iff
    it spikes at least once among all B*T rows of the block."""
    S = np.asarray(S, dtype=bool)
    return S.reshape(-1, S.shape[-1]).any(axis=0)


def active_rows(S: np.ndarray) -> np.ndarray:
    """Ascending list of the input channels whose weight row is loaded."""
    return np.flatnonzero(block_union(S)).astype(np.int32)


def touched_weight_bytes(S: np.ndarray, N: int, bytes_per_weight: int = 1) -> int:
    """Weight bytes read by one product: active rows x N (Eq. (13) per block)."""
    return int(block_union(S).sum()) * int(N) * bytes_per_weight


# ----------------------------------------------------------------------------
# IF neuron with soft reset (Sec. II-B, Eqs. (3)-(4))
# ----------------------------------------------------------------------------
def if_neuron(I: np.ndarray, theta, resid: np.ndarray | None = None):
    """Integrate-and-fire with soft reset over the T axis (axis 0).

    Reading of Eqs. (3)-(4): the membrane starts at 0 for every call; at each
    step it first integrates the current, then fires if V >= theta
    (Eq. (3), equality fires) and subtracts theta on a spike (Eq. (4)); there
    is no lower clamp.  ``theta`` is a scalar or one value per neuron (last
    axis).  ``resid`` (0/1, same shape as I) adds theta * resid to the
    current: the membrane shortcut used for the residual path.
    Returns (spikes bool [T,...], final membrane int64 [...]).
    """
    I = np.asarray(I, dtype=np.int64)
    th = np.asarray(theta, dtype=np.int64)
    if np.any(th <= 0):
        raise ValueError("threshold must be positive")
    T = I.shape[0]
    V = np.zeros(I.shape[1:], dtype=np.int64)
    s = np.zeros(I.shape, dtype=bool)
    for t in range(T):
        cur = I[t]
        if resid is not None:
            cur = cur + th * np.asarray(resid[t], dtype=np.int64)
        V = V + cur
        fire = V >= th
        s[t] = fire
        V = V - np.where(fire, th, 0)
    return s, V


# ----------------------------------------------------------------------------
# QNL: 8-bit-in / 8-bit-out lookup table
# ----------------------------------------------------------------------------
QNL_S8 = 0
QNL_U8 = 1


def qnl_lut(x: np.ndarray, shift: int, lut: np.ndarray, mode: int = QNL_S8) -> np.ndarray:
    """Quantised non-linearity by table lookup.

    S8: index = the byte of clamp(floor(x / 2**shift), -128, 127); the table
        entry is read as int8.  U8: index = clamp(x, 0, 255), entry read as
        uint8 (``shift`` is ignored).  Returns int64.
    """
    x = np.asarray(x, dtype=np.int64)
    lut = np.asarray(lut, dtype=np.uint8)
    if mode == QNL_S8:
        q = np.floor_divide(x, 2 ** int(shift))
        q = np.clip(q, -128, 127)
        idx = (q & 0xFF).astype(np.int64)
        return lut.view(np.int8)[idx].astype(np.int64)
    if mode == QNL_U8:
        idx = np.clip(x, 0, 255)
        return lut[idx].astype(np.int64)
    raise ValueError("unknown table mode")


# ----------------------------------------------------------------------------
# BBM attention with table weights and fixed-point normalisation
# ----------------------------------------------------------------------------
def bbm_attention(Q: np.ndarray, Kc: np.ndarray, Vc: np.ndarray, n_keys: int,
                  H: int, lut_att: np.ndarray) -> np.ndarray:
    """Spike attention; the paper names the operations (binary-binary
    products, table non-linearity, fixed-point arithmetic) but not the
    formula, so this is the reading used throughout:

        s[t,i,j] = sum_{c in head h} Q[t,i,c] * K[t,j,c]           (0..dh)
        p[t,i,j] = lut_att[s]                                         (1..255)
        a[t,i,c] = floor(256 * sum_j p * V[t,j,c] / sum_j p)         (0..256)

    Q: 0/1 [T][M][d]; Kc, Vc: 0/1 [T][>=n_keys][d] (keys 0..n_keys-1 used).
    Returns int64 [T][M][d].
    """
    Q = np.asarray(Q)
    T, M, d = Q.shape
    dh = d // H
    lut = np.asarray(lut_att, dtype=np.int64)
    a = np.zeros((T, M, d), dtype=np.int64)
    for t in range(T):
        for h in range(H):
            c0, c1 = h * dh, (h + 1) * dh
            q = Q[t, :, c0:c1]
            k = Kc[t, :n_keys, c0:c1]
            v = Vc[t, :n_keys, c0:c1]
            s = _exact_matmul(q, k.T)                  # [M][n_keys]
            p = lut[s]                                 # [M][n_keys]
            den = p.sum(axis=1)                        # [M]
            num = _exact_matmul(p, v)                  # [M][dh]
            # 256 * num <= 256 * 255 * n_keys: exact in int64 for any number
            # of keys (it leaves int32 from about 32 thousand keys on)
            safe = np.where(den > 0, den, 1)
            a[t, :, c0:c1] = np.where(den[:, None] > 0,
                                      (256 * num) // safe[:, None], 0)
    return a


# ----------------------------------------------------------------------------
# one spiking transformer layer (Fig. 1: IF dynamics in every layer)
# ----------------------------------------------------------------------------
@dataclass
class LayerTrace:
    Q: np.ndarray
    K: np.ndarray
    V: np.ndarray
    A: np.ndarray
    X1: np.ndarray
    H: np.ndarray
    Y: np.ndarray
    unions: dict


def layer_forward(X: np.ndarray, L, k_cache: np.ndarray, v_cache: np.ndarray,
                  c0: int) -> LayerTrace:
    """One layer over a block of M tokens whose keys/values go to cache rows
    [c0, c0+M); attention reads cache rows [0, c0+M).

    Readings (the paper gives only "IF neuron dynamics" per layer and an MLP):
      Q,K,V = IF(QBSM(X, W_q|W_k|W_v))                  thresholds q, k, v
      A     = IF(attention(Q, K_cache, V_cache))         threshold a
      X1    = IF(QBSM(A, W_o), residual X)               threshold o
      H     = IF(table(QBSM(X1, W_up) >> s_up))          threshold up
      Y     = IF(QBSM(H, W_dn), residual X1)             threshold dn
    The residual adds theta * input spike to the membrane (identity when the
    branch current is zero).  No normalisation layer.
    k_cache / v_cache are 0/1 bool arrays [T][cap][d], updated in place.
    """
    X = np.asarray(X, dtype=bool)
    T, M, d = X.shape
    th = L.theta
    qkv = qbsm(X, L.W_qkv)
    Q, _ = if_neuron(qkv[:, :, 0:d], th["q"])
    Kb, _ = if_neuron(qkv[:, :, d:2 * d], th["k"])
    Vb, _ = if_neuron(qkv[:, :, 2 * d:3 * d], th["v"])
    k_cache[:, c0:c0 + M] = Kb
    v_cache[:, c0:c0 + M] = Vb
    a = bbm_attention(Q, k_cache, v_cache, c0 + M, L.H, L.lut_att)
    A, _ = if_neuron(a, th["a"])
    X1, _ = if_neuron(qbsm(A, L.W_o), th["o"], resid=X)
    u = qbsm(X1, L.W_up)
    g = qnl_lut(u, L.s_up, L.lut_act, QNL_S8)
    Hs, _ = if_neuron(g, th["up"])
    Y, _ = if_neuron(qbsm(Hs, L.W_dn), th["dn"], resid=X1)
    unions = {"qkv": block_union(X), "o": block_union(A),
              "up": block_union(X1), "dn": block_union(Hs)}
    return LayerTrace(Q, Kb, Vb, A, X1, Hs, Y, unions)


def stack_forward(X: np.ndarray, layers, k_caches, v_caches, c0: int):
    """X_{l+1} = Y_l over the layer stack; returns (Y_last, traces)."""
    traces = []
    for l, L in enumerate(layers):
        tr = layer_forward(X, L, k_caches[l], v_caches[l], c0)
        traces.append(tr)
        X = tr.Y
    return X, traces


# ----------------------------------------------------------------------------
# block input, head, confidence, unmasking (Sec. III-A, Eq. (6))
# ----------------------------------------------------------------------------
def block_input(tokens: np.ndarray, positions: np.ndarray, emb_bits: np.ndarray,
                pos_ch: np.ndarray) -> np.ndarray:
    """X[t,m,:] = E[token_m][t] OR onehot(pos_ch[pos_m][t]).

    The masked block starts as copies of the mask embedding (Sec. III-A); the
    paper gives no positional signal, so a single seeded position spike per
    (position, step) is ORed in (otherwise all masked rows are identical).
    emb_bits: 0/1 [V+1][T][d]; pos_ch: int [max_pos][T]. Returns bool [T][M][d].
    """
    tokens = np.asarray(tokens)
    positions = np.asarray(positions)
    X = np.asarray(emb_bits[tokens], dtype=bool).transpose(1, 0, 2).copy()  # [T][M][d]
    T, M, d = X.shape
    for m in range(M):
        for t in range(T):
            X[t, m, pos_ch[positions[m], t]] = True
    return X


def head_logits(Y: np.ndarray, W_head: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """Rate read-out: acc[m,v] = sum_t sum_c Y[t,m,c] W_head[c,v] (exact),
    logit = float32(acc) * scale[v] (one IEEE fp32 multiply)."""
    Y = np.asarray(Y)
    T, M, d = Y.shape
    acc = qbsm(Y, W_head).sum(axis=0)                   # int64 [M][V]
    _check_int32(acc, "head accumulator")
    if np.abs(acc).max(initial=0) >= 2 ** 24:
        raise OverflowError("head accumulator not exactly representable in fp32")
    return acc.astype(np.float32) * np.asarray(scale, dtype=np.float32)[None, :]


def confidence(logits: np.ndarray):
    """pred = argmax (ties -> smallest id); conf = max softmax probability in
    float64: 1 / sum_v exp(logit_v - logit_pred)."""
    logits = np.asarray(logits, dtype=np.float32)
    pred = np.argmax(logits, axis=1).astype(np.int32)
    l64 = logits.astype(np.float64)
    mx = l64[np.arange(l64.shape[0]), pred]
    conf = 1.0 / np.exp(l64 - mx[:, None]).sum(axis=1)
    return pred, conf


def unmask(tokens: np.ndarray, masked: np.ndarray, pred: np.ndarray,
           conf: np.ndarray, k: int):
    """Reveal the k most confident masked positions (Sec. III-A: B/S tokens per
    step; the selection rule is not stated, confidence is used).  Order is
    (confidence descending, position ascending); unmasked tokens never change.
    Returns (tokens, masked, chosen positions in selection order)."""
    tokens = np.array(tokens, dtype=np.int32, copy=True)
    masked = np.array(masked, dtype=bool, copy=True)
    cand = [m for m in range(len(tokens)) if masked[m]]
    cand.sort(key=lambda m: (-float(conf[m]), m))
    chosen = cand[:k]
    for m in chosen:
        tokens[m] = pred[m]
        masked[m] = False
    return tokens, masked, np.array(chosen, dtype=np.int32)


# ----------------------------------------------------------------------------
# caches, prefill, block step, generation (Eqs. (2), (5), (6))
# ----------------------------------------------------------------------------
def unpack_model_emb(model) -> np.ndarray:
    """The model stores packed spike tables; the oracle works on 0/1 arrays."""
    from workloads.synth import unpack_bits
    return unpack_bits(model.emb, model.d)


def new_caches(n_layers: int, T: int, cap: int, d: int):
    k = [np.zeros((T, cap, d), dtype=bool) for _ in range(n_layers)]
    v = [np.zeros((T, cap, d), dtype=bool) for _ in range(n_layers)]
    return k, v


def prefill(X_ctx: np.ndarray, layers, k_caches, v_caches):
    """Context encoding (Eq. (5)): run every layer over the C context tokens,
    attending to themselves only (bidirectional), keys/values to cache rows
    [0, C). No head."""
    return stack_forward(X_ctx, layers, k_caches, v_caches, 0)


@dataclass
class StepResult:
    tokens: np.ndarray
    masked: np.ndarray
    chosen: np.ndarray
    pred: np.ndarray
    conf: np.ndarray
    logits: np.ndarray
    Y: np.ndarray
    traces: list


def block_step(model, emb01: np.ndarray, tokens: np.ndarray, masked: np.ndarray,
               pos0: int, C: int, k_caches, v_caches, k_unmask: int) -> StepResult:
    """One denoising step z_{s+1} = f_dec(z_s, h) (Eq. (6)) on the block at
    sequence positions [pos0, pos0+M) whose keys/values occupy cache rows
    [C, C+M): block input -> layer stack -> head -> confidence -> unmask."""
    tokens = np.asarray(tokens, dtype=np.int32)
    masked = np.asarray(masked, dtype=bool)
    M = len(tokens)
    cur = np.where(masked, model.mask_id, tokens)
    X = block_input(cur, np.arange(pos0, pos0 + M), emb01, model.pos_ch)
    Y, traces = stack_forward(X, model.layers, k_caches, v_caches, C)
    logits = head_logits(Y, model.W_head, model.scale)
    pred, conf = confidence(logits)
    new_tokens, new_masked, chosen = unmask(tokens, masked, pred, conf, k_unmask)
    return StepResult(new_tokens, new_masked, chosen, pred, conf, logits, Y, traces)


def generate(model, prompt: np.ndarray, n_blocks: int, B: int, steps: int,
             k_unmask: int, emb01: np.ndarray | None = None):
    """Block-diffusion generation (Eq. (2)): prefill the prompt, then for each
    block start from B mask tokens, run ``steps`` denoising steps revealing
    ``k_unmask`` tokens each, and freeze the keys/values of the block's last
    step as context.  Returns (generated ids, per-step chosen positions)."""
    if emb01 is None:
        emb01 = unpack_model_emb(model)
    P = len(prompt)
    cap = P + n_blocks * B
    kc, vc = new_caches(model.n_layers, model.T, cap, model.d)
    Xp = block_input(prompt, np.arange(P), emb01, model.pos_ch)
    prefill(Xp, model.layers, kc, vc)
    C = P
    out = []
    log = []
    for b in range(n_blocks):
        tokens = np.zeros(B, dtype=np.int32)
        masked = np.ones(B, dtype=bool)
        for s in range(steps):
            r = block_step(model, emb01, tokens, masked, C, C, kc, vc, k_unmask)
            tokens, masked = r.tokens, r.masked
            log.append(r.chosen)
        out.append(tokens)
        C += B
    return np.concatenate(out), log


@dataclass
class E2d2State:
    """Key/value caches of the encoder layers and of the decoder layers."""
    kc_enc: list
    vc_enc: list
    kc_dec: list
    vc_dec: list


def e2d2_new_state(model, n_enc: int, cap: int) -> E2d2State:
    kc_e, vc_e = new_caches(n_enc, model.T, cap, model.d)
    kc_d, vc_d = new_caches(model.n_layers - n_enc, model.T, cap, model.d)
    return E2d2State(kc_e, vc_e, kc_d, vc_d)


def e2d2_encode(model, n_enc: int, tokens: np.ndarray, C: int, state: E2d2State,
                emb01: np.ndarray) -> np.ndarray:
    """The encoder pass of Eq. (5) over the tokens at positions [C, C+M),
    attending to the encoded context [0, C) and to themselves; then every
    decoder layer writes the keys and values of those positions from the
    encoder output h (its own projections of h: the decoder attends to the
    encoder output).  Returns h (bool [T][M][d])."""
    enc, dec = model.layers[:n_enc], model.layers[n_enc:]
    X = block_input(np.asarray(tokens, dtype=np.int32), np.arange(C, C + len(tokens)), emb01,
                    model.pos_ch)
    h, _ = stack_forward(X, enc, state.kc_enc, state.vc_enc, C)
    for l, L in enumerate(dec):
        layer_forward(h, L, state.kc_dec[l], state.vc_dec[l], C)
    return h


def e2d2_generate(model, n_enc: int, prompt: np.ndarray, n_blocks: int, B: int, steps: int,
                  k_unmask: int, emb01: np.ndarray | None = None, return_state: bool = False):
    """Encoder-decoder block diffusion (Sec. III-A, Eqs. (5)-(6)): the first
    n_enc layers are the encoder f_enc, the others the decoder f_dec.

    The encoder gives h^b = f_enc(x^{<b}) (Eq. (5)) block-causally: the prompt
    is encoded once (bidirectional within it), and every finished block is
    encoded over the cached context plus itself, so each token passes the
    encoder once (e2d2_encode).  A block starts as B mask tokens; ``steps``
    denoising steps z_{s+1} = f_dec(z_s, h^b) (Eq. (6)) run the decoder layers
    and the head over it, revealing ``k_unmask`` tokens each.  Returns
    (generated ids, chosen positions per step[, final E2d2State])."""
    import dataclasses
    if emb01 is None:
        emb01 = unpack_model_emb(model)
    dec = model.layers[n_enc:]
    dec_model = dataclasses.replace(model, layers=dec, n_layers=len(dec))
    P = len(prompt)
    state = e2d2_new_state(model, n_enc, P + n_blocks * B)
    e2d2_encode(model, n_enc, prompt, 0, state, emb01)
    C = P
    out, log = [], []
    for b in range(n_blocks):
        tokens = np.zeros(B, dtype=np.int32)
        masked = np.ones(B, dtype=bool)
        for s in range(steps):
            r = block_step(dec_model, emb01, tokens, masked, C, C, state.kc_dec, state.vc_dec,
                           k_unmask)
            tokens, masked = r.tokens, r.masked
            log.append(r.chosen)
        out.append(tokens)
        e2d2_encode(model, n_enc, tokens, C, state, emb01)
        C += B
    if return_state:
        return np.concatenate(out), log, state
    return np.concatenate(out), log


# ----------------------------------------------------------------------------
# Ternary bitwise-coded conversion (Sec. III-B, Eqs. (7)-(11))
# ----------------------------------------------------------------------------
def ternary_quantize(a: np.ndarray, K: int, T: int):
    """Eq. (7): q = round(a / V_th(a)) with V_th(a) = mean(|a|) / K, per token.

    Activations reach the conversion as integers (a layer's int32 output), so
    V_th = S / (D K) with S = sum_i |a_i| is kept as the exact rational and
    q_i = round(a_i D K / S) is computed in integers: rounding half away from
    zero, q = 0 for an all-zero vector, |q| saturating at 2^T - 1 (T bits).
    a: int [M][D].  Returns (q int64 [M][D], S int64 [M])."""
    a = np.asarray(a, dtype=np.int64)
    M, D = a.shape
    S = np.abs(a).sum(axis=1)
    q = np.zeros_like(a)
    lim = (1 << T) - 1
    for m in range(M):
        if S[m] == 0:
            continue
        num = np.abs(a[m]) * (D * K)
        mag = (2 * num + S[m]) // (2 * S[m])        # floor(|a| D K / S + 1/2)
        q[m] = np.sign(a[m]) * np.minimum(mag, lim)
    return q, S


def ternary_planes(q: np.ndarray, T: int) -> np.ndarray:
    """Eq. (8): bitwise coding with ternary spikes, s_{i,t} = sign(q_i) times
    bit t-1 of |q_i| for t = 1..T (q = sum_t 2^(t-1) s_t).  Returns int8
    [T][M][D] in {-1, 0, 1}."""
    q = np.asarray(q, dtype=np.int64)
    mag, sgn = np.abs(q), np.sign(q)
    if mag.max(initial=0) >= (1 << T):
        raise ValueError("value needs more than T bits")
    return np.stack([(sgn * ((mag >> t) & 1)).astype(np.int8) for t in range(T)])


def ternary_union(s: np.ndarray) -> np.ndarray:
    """Assumption (ii) of Sec. IV-A on ternary spikes: input i needs its weight
    row iff s_{i,t} != 0 for some timestep and token of the block."""
    s = np.asarray(s)
    return (s != 0).reshape(-1, s.shape[-1]).any(axis=0)


def qbsm_ternary(s: np.ndarray, W: np.ndarray):
    """The spiking product on ternary spikes: I_t = sum_i w_i s_{i,t} per
    timestep over every input, and the bitwise reconstruction of Eq. (11)
    acc = sum_t 2^(t-1) I_t (the inner product with the decoded q).
    s: int8 [T][M][K]; W: int8 [K][N].  Returns (I int64 [T][M][N], acc int64 [M][N])."""
    s = np.asarray(s)
    T, M, K = s.shape
    I = _exact_matmul(s.reshape(T * M, K), W).reshape(T, M, W.shape[1])
    acc = np.zeros((M, W.shape[1]), dtype=np.int64)
    for t in range(T):
        acc += I[t] << t
    _check_int32(acc, "ternary accumulator")
    return I, acc


def modified_if(I: np.ndarray, thr_num, thr_den: int):
    """The modified IF neuron of Eqs. (9)-(10) over the T bit-timesteps of a
    ternary bitwise-coded input (axis 0 of I), with threshold
    V_th = thr_num / thr_den (one numerator per token: the last-but-one
    axis of I; thr_den > 0).

    Readings: timesteps run t = 1..T and the input at step t carries the
    weight 2^(t-1) of its bit (Eq. (8); the 2^t of Eqs. (9)-(10) counts steps
    from zero); as for the plain IF neuron the membrane integrates before it
    fires.  Per neuron, starting from V = 0:
        V += 2^(t-1) I_t
        s_t = +1 if V >= 2^(t-1) V_th,  -1 if V <= -2^(t-1) V_th,  else 0
        V -= 2^(t-1) s_t V_th
    so that V_th sum_t 2^(t-1) s_t = sum_t 2^(t-1) I_t - V_final (Eq. (11)'s
    reconstruction, with the final membrane as its error).  A token whose
    threshold numerator is 0 (an all-zero activation vector, V_th = 0) emits
    no spike.  The membrane is kept multiplied by thr_den so that every step
    is integer arithmetic.
    I: int [T][M][N]; thr_num: int [M].
    Returns (s int8 [T][M][N] in {-1, 0, 1}, thr_den * V_final int64 [M][N])."""
    I = np.asarray(I, dtype=np.int64)
    num = np.asarray(thr_num, dtype=np.int64)
    den = int(thr_den)
    if den <= 0:
        raise ValueError("threshold denominator must be positive")
    T = I.shape[0]
    silent = (num <= 0)[:, None]
    V = np.zeros(I.shape[1:], dtype=np.int64)          # den * membrane
    s = np.zeros(I.shape, dtype=np.int8)
    for t in range(T):                                  # t here is the paper's t - 1
        w = 1 << t
        V = V + den * w * I[t]
        thr = (w * num)[:, None]
        up = ~silent & (V >= thr)
        dn = ~silent & ~up & (V <= -thr)
        s[t] = up.astype(np.int8) - dn.astype(np.int8)
        V = V - s[t].astype(np.int64) * thr
    return s, V


def bitwise_value(s: np.ndarray) -> np.ndarray:
    """sum_t 2^(t-1) s_t over axis 0 (t = 1..T): the integer a ternary spike
    train codes (Eq. (8)), and the sum Eq. (11) scales by V_th."""
    s = np.asarray(s, dtype=np.int64)
    return sum((1 << t) * s[t] for t in range(s.shape[0]))
