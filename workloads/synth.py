"""Seeded synthetic inputs for the N-MDLM block-denoising step.

This module is the only code shared by the oracle (``oracle/``) and the HIP
path (``paper_2607_24841_amd``).  It draws random numbers and packs bits; it
holds none of the method's arithmetic (no products, no neuron updates, no
attention, no unmasking).

Random streams
--------------
Every array comes from its own PCG64 stream addressed by a spawn key under
the workload's seed: ``np.random.SeedSequence(seed, spawn_key=path)``.
An array therefore never depends on how many other arrays were drawn before
it, and a large model can be generated layer by layer.

Bit layout
----------
Spike tensors are logically ``{0,1}^{T x M x K}`` and physically packed
``uint64 [T][M][ceil(K/64)]``: bit ``j`` of word ``w`` is channel ``64*w + j``
(LSB first); padding bits are zero.

Distributions (the paper's workload model, Sec. IV-A: iid entries with
P(x=0) = sigma; the correlated-activity variant draws a rate per channel)
-------------
* Bernoulli(p): ``u < p`` with ``u`` a float64 uniform on [0, 1).
* Integer uniforms are inclusive on both ends.
* int8 weights: uniform on [-127, 127].
* Per-channel rates ``r ~ Beta(a, b)``; where a target mean density is given,
  ``r`` is scaled by a factor found by bisection so that the mean of
  ``clip(c*r, 0, 1)`` equals the target.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

SEEDS = {"linear": 1001, "block": 1002, "ffn_sweep": 1003, "mdlm12": 1004, "mdlm24": 1005,
         "e2d2": 1006, "ternary": 1007}


# ----------------------------------------------------------------------------
# random streams and bit packing
# ----------------------------------------------------------------------------
def stream(seed: int, *path: int) -> np.random.Generator:
    """Independent PCG64 stream for (seed, path)."""
    ss = np.random.SeedSequence(int(seed), spawn_key=tuple(int(p) for p in path))
    return np.random.Generator(np.random.PCG64(ss))


def pack_bits(bits: np.ndarray) -> np.ndarray:
    """Pack a boolean/0-1 array along its last axis into uint64 words (LSB first)."""
    bits = np.asarray(bits).astype(bool, copy=False)
    k = bits.shape[-1]
    kw = max(1, (k + 63) // 64)
    pad = kw * 64 - k
    if pad:
        bits = np.concatenate(
            [bits, np.zeros(bits.shape[:-1] + (pad,), dtype=bool)], axis=-1)
    by = np.packbits(bits, axis=-1, bitorder="little")
    by = np.ascontiguousarray(by)
    return by.view("<u8").reshape(bits.shape[:-1] + (kw,))


def unpack_bits(words: np.ndarray, k: int) -> np.ndarray:
    """Inverse of :func:`pack_bits`: uint64 words -> bool array with ``k`` channels."""
    words = np.ascontiguousarray(np.asarray(words, dtype="<u8"))
    by = words.view(np.uint8).reshape(words.shape[:-1] + (words.shape[-1] * 8,))
    bits = np.unpackbits(by, axis=-1, bitorder="little")[..., :k]
    return bits.astype(bool)


def bernoulli(rng: np.random.Generator, p, shape) -> np.ndarray:
    return rng.random(shape) < p


def int8_uniform(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.integers(-127, 128, size=shape, dtype=np.int8)


def int_uniform(rng: np.random.Generator, lo: int, hi: int, shape, dtype=np.int32):
    return rng.integers(lo, hi + 1, size=shape, dtype=dtype)


def scale_rates_to_mean(r: np.ndarray, target: float) -> np.ndarray:
    """Scale rates by c (bisection) so that mean(clip(c*r, 0, 1)) == target."""
    r = np.asarray(r, dtype=np.float64)
    if target <= 0:
        return np.zeros_like(r)
    lo, hi = 0.0, 1.0
    while np.clip(hi * r, 0, 1).mean() < target:
        hi *= 2.0
        if hi > 1e12:
            raise ValueError("target density unreachable")
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if np.clip(mid * r, 0, 1).mean() < target:
            lo = mid
        else:
            hi = mid
    return np.clip(hi * r, 0, 1)


def sorted_lut_u8(rng: np.random.Generator) -> np.ndarray:
    """Attention score table: 256 sorted uniform integers on [1, 255] (uint8)."""
    return np.sort(rng.integers(1, 256, size=256)).astype(np.uint8)


def sorted_lut_s8(rng: np.random.Generator) -> np.ndarray:
    """Activation table stored as raw bytes, indexed by the two's-complement byte
    of a signed 8-bit input; values are sorted uniform integers on [-128, 127]
    in the order of the signed input (monotone non-decreasing)."""
    vals = np.sort(rng.integers(-128, 128, size=256)).astype(np.int8)
    lut = np.empty(256, dtype=np.uint8)
    signed_in = np.arange(-128, 128)
    lut[(signed_in & 0xFF)] = vals.view(np.uint8)
    return lut


# ----------------------------------------------------------------------------
# single QBSM + IF (the 4x8x512 -> 512 spiking linear layer and the tiny shapes of the tests)
# ----------------------------------------------------------------------------
@dataclass
class QbsmCase:
    T: int
    M: int
    K: int
    N: int
    S: np.ndarray        # bool [T][M][K]
    W: np.ndarray        # int8 [K][N]
    bias: np.ndarray     # int32 [N]
    theta: int

    @property
    def S_packed(self) -> np.ndarray:
        return pack_bits(self.S)


def make_qbsm_case(seed: int, T: int, M: int, K: int, N: int, density: float,
                   theta: int = 256, bias_range: int = 64) -> QbsmCase:
    S = bernoulli(stream(seed, 0), density, (T, M, K))
    W = int8_uniform(stream(seed, 1), (K, N))
    if bias_range > 0:
        bias = int_uniform(stream(seed, 2), -bias_range, bias_range, (N,))
    else:
        bias = np.zeros(N, dtype=np.int32)
    return QbsmCase(T, M, K, N, S, W, bias, int(theta))


def linear_layer_case(seed: int = SEEDS["linear"]) -> QbsmCase:
    """Single spiking linear layer: T=4, B=8, K=N=512, Bernoulli(0.15) input,
    int8 weights on [-127,127], int32 bias on [-64,64], threshold 256."""
    return make_qbsm_case(seed, T=4, M=8, K=512, N=512, density=0.15, theta=256)


# ----------------------------------------------------------------------------
# transformer layer parameters
# ----------------------------------------------------------------------------
THETA_NAMES = ("q", "k", "v", "a", "o", "up", "dn")


@dataclass
class LayerParams:
    d: int
    F: int
    H: int
    dh: int
    W_qkv: np.ndarray     # int8 [d][3d]: columns [0,d)=Q, [d,2d)=K, [2d,3d)=V
    W_o: np.ndarray       # int8 [d][d]
    W_up: np.ndarray      # int8 [d][F]
    W_dn: np.ndarray      # int8 [F][d]
    theta: dict           # name -> int, names in THETA_NAMES
    lut_att: np.ndarray   # uint8 [256]
    lut_act: np.ndarray   # uint8 [256] (bytes of int8 values)
    s_up: int             # right shift applied before the activation table


def up_shift(d: int) -> int:
    return max(0, int(math.floor(math.log2(d))) - 6)


def make_layer(seed: int, layer: int, d: int, F: int, H: int) -> LayerParams:
    base = 100 + 16 * layer
    W_qkv = int8_uniform(stream(seed, base + 0), (d, 3 * d))
    W_o = int8_uniform(stream(seed, base + 1), (d, d))
    W_up = int8_uniform(stream(seed, base + 2), (d, F))
    W_dn = int8_uniform(stream(seed, base + 3), (F, d))
    th = int_uniform(stream(seed, base + 4), 128, 512, (len(THETA_NAMES),))
    theta = {n: int(v) for n, v in zip(THETA_NAMES, th)}
    lut_att = sorted_lut_u8(stream(seed, base + 5))
    lut_act = sorted_lut_s8(stream(seed, base + 6))
    return LayerParams(d, F, H, d // H, W_qkv, W_o, W_up, W_dn, theta,
                       lut_att, lut_act, up_shift(d))


# ----------------------------------------------------------------------------
# one spiking transformer block (d=1024, 16 heads, FFN 4096), one denoising step
# ----------------------------------------------------------------------------
@dataclass
class BlockCase:
    T: int
    C: int
    M: int
    layer: LayerParams
    X_ctx: np.ndarray     # bool [T][C][d] context inputs (prefill)
    X_blk: np.ndarray     # bool [T][M][d] block inputs


def block_inputs(seed: int, C: int, M: int, d: int, T: int = 4, density: float = 0.10):
    """Context and block input spikes of one sequence (bool [T][C][d], [T][M][d])."""
    return (bernoulli(stream(seed, 0), density, (T, C, d)),
            bernoulli(stream(seed, 1), density, (T, M, d)))


def block_case(seed: int = SEEDS["block"], C: int = 512, M: int = 16, d: int = 1024,
            H: int = 16, F: int = 4096, T: int = 4, density: float = 0.10) -> BlockCase:
    X_ctx, X_blk = block_inputs(seed, C, M, d, T, density)
    layer = make_layer(seed, 0, d, F, H)
    return BlockCase(T, C, M, layer, X_ctx, X_blk)


# ----------------------------------------------------------------------------
# FFN weight-traffic sweep (4096 -> 14336 -> 4096)
# ----------------------------------------------------------------------------
FFN_SWEEP_BLOCKS = (1, 4, 16, 64)
FFN_SWEEP_DENSITIES = (0.02, 0.05, 0.10, 0.30)


@dataclass
class FfnWeights:
    d: int
    F: int
    W_up: np.ndarray      # int8 [d][F]
    W_dn: np.ndarray      # int8 [F][d]
    theta_up: int
    theta_dn: int


@dataclass
class FfnPoint:
    B: int
    density: float
    T: int
    X_up: np.ndarray      # bool [T][B][d]
    X_dn: np.ndarray      # bool [T][B][F]


def ffn_sweep_weights(seed: int = SEEDS["ffn_sweep"], d: int = 4096, F: int = 14336) -> FfnWeights:
    W_up = int8_uniform(stream(seed, 0), (d, F))
    W_dn = int8_uniform(stream(seed, 1), (F, d))
    th = int_uniform(stream(seed, 2), 128, 512, (2,))
    return FfnWeights(d, F, W_up, W_dn, int(th[0]), int(th[1]))


def correlated_spikes(rng: np.random.Generator, T: int, B: int, K: int,
                      density: float, a: float = 0.5, b: float = 8.0) -> np.ndarray:
    """Per-channel rates ~ Beta(a, b) scaled to the target mean, then iid
    Bernoulli(rate_k) over (t, token)."""
    r = scale_rates_to_mean(rng.beta(a, b, size=K), density)
    return rng.random((T, B, K)) < r[None, None, :]


def ffn_sweep_point(iB: int, iR: int, seed: int = SEEDS["ffn_sweep"], d: int = 4096,
                  F: int = 14336, T: int = 4) -> FfnPoint:
    B = FFN_SWEEP_BLOCKS[iB]
    rho = FFN_SWEEP_DENSITIES[iR]
    X_up = correlated_spikes(stream(seed, 10 + 4 * iB + iR, 0), T, B, d, rho)
    X_dn = correlated_spikes(stream(seed, 10 + 4 * iB + iR, 1), T, B, F, rho)
    return FfnPoint(B, rho, T, X_up, X_dn)


# ----------------------------------------------------------------------------
# multi-layer spiking MDLM (12-layer block step, 24-layer generation)
# ----------------------------------------------------------------------------
@dataclass
class MdlmModel:
    n_layers: int
    d: int
    H: int
    F: int
    V: int                # vocabulary size; the mask token id is V
    T: int
    max_pos: int
    emb: np.ndarray       # uint64 [V+1][T][d/64] token spike table (row V = mask)
    pos_ch: np.ndarray    # int32 [max_pos][T] channel of the single position spike
    layers: list = field(default_factory=list)
    W_head: np.ndarray = None   # int8 [d][V]
    scale: np.ndarray = None    # float32 [V]

    @property
    def mask_id(self) -> int:
        return self.V


def make_mdlm(seed: int, n_layers: int, d: int = 2048, H: int = 16, F: int = 8192,
              V: int = 32000, T: int = 4, max_pos: int = 2304,
              emb_beta=(0.5, 6.0), chunk: int = 2048) -> MdlmModel:
    rng_r = stream(seed, 1)
    rates = rng_r.beta(emb_beta[0], emb_beta[1], size=d)
    dw = (d + 63) // 64
    emb = np.empty((V + 1, T, dw), dtype=np.uint64)
    rng_e = stream(seed, 2)
    for v0 in range(0, V + 1, chunk):
        v1 = min(V + 1, v0 + chunk)
        bits = rng_e.random((v1 - v0, T, d)) < rates[None, None, :]
        emb[v0:v1] = pack_bits(bits)
    pos_ch = int_uniform(stream(seed, 3), 0, d - 1, (max_pos, T))
    layers = [make_layer(seed, l, d, F, H) for l in range(n_layers)]
    W_head = int8_uniform(stream(seed, 4), (d, V))
    scale = (stream(seed, 5).uniform(0.5, 1.5, size=V) * 2.0 ** -10).astype(np.float32)
    return MdlmModel(n_layers, d, H, F, V, T, max_pos, emb, pos_ch, layers, W_head, scale)


def random_tokens(seed: int, n: int, V: int, path: int = 6) -> np.ndarray:
    return int_uniform(stream(seed, path), 0, V - 1, (n,))


@dataclass
class MdlmStepCase:
    model: MdlmModel
    ctx_tokens: np.ndarray    # int32 [C]
    C: int
    B: int
    k_unmask: int


def mdlm12_step_case(seed: int = SEEDS["mdlm12"], n_layers: int = 12, C: int = 1024, B: int = 32,
            k_unmask: int = 8, **kw) -> MdlmStepCase:
    model = make_mdlm(seed, n_layers, max_pos=max(C + B, kw.pop("max_pos", 0)), **kw)
    ctx = random_tokens(seed, C, model.V)
    return MdlmStepCase(model, ctx, C, B, k_unmask)


@dataclass
class GenerationCase:
    model: MdlmModel
    prompt: np.ndarray        # int32 [P]
    n_blocks: int
    B: int
    steps: int
    k_unmask: int


def mdlm24_generation_case(seed: int = SEEDS["mdlm24"], n_layers: int = 24, prompt_len: int = 2048,
            n_blocks: int = 8, B: int = 32, steps: int = 8, k_unmask: int = 4,
            **kw) -> GenerationCase:
    model = make_mdlm(seed, n_layers, max_pos=prompt_len + n_blocks * B, **kw)
    prompt = random_tokens(seed, prompt_len, model.V)
    return GenerationCase(model, prompt, n_blocks, B, steps, k_unmask)


@dataclass
class E2d2Case:
    model: MdlmModel          # layers [0, n_enc) encoder, [n_enc, n_layers) decoder
    n_enc: int
    prompt: np.ndarray        # int32 [P]
    n_blocks: int
    B: int
    steps: int
    k_unmask: int


def e2d2_case(seed: int = SEEDS["e2d2"], n_enc: int = 28, n_dec: int = 4, d: int = 512,
              H: int = 8, F: int = 1536, V: int = 32000, T: int = 8, prompt_len: int = 64,
              n_blocks: int = 4, B: int = 4, steps: int = 4, k_unmask: int = 1,
              **kw) -> E2d2Case:
    """The paper's own model shape (Sec. V-A): 28 encoder and 4 decoder
    layers, D = 512, D_hid = 1536, T = 8, one token revealed per step (S = B).
    Synthetic weights and token tables stand in for the converted E2D2 model
    and WMT14 sentences (neither is available); a 64-token prompt stands in
    for a source sentence."""
    model = make_mdlm(seed, n_enc + n_dec, d=d, H=H, F=F, V=V, T=T,
                      max_pos=prompt_len + n_blocks * B, **kw)
    prompt = random_tokens(seed, prompt_len, model.V)
    return E2d2Case(model, n_enc, prompt, n_blocks, B, steps, k_unmask)


@dataclass
class TernaryCase:
    a: np.ndarray             # int32 [M][D] activations (a layer's integer output)
    W: np.ndarray             # int8 [D][N]
    K: int                    # quantisation levels per mean magnitude
    T: int                    # bits (timesteps)


def ternary_activations(rng: np.random.Generator, M: int, D: int, scale: float = 1000.0,
                        beta=(0.5, 6.0)) -> np.ndarray:
    """Integer activations with per-channel magnitudes drawn from Beta(0.5, 6)
    (a few large channels, many small ones, the same for every token) times
    Laplace noise per token: small channels quantise to zero for the whole
    block, which is what the row-load rule skips."""
    c = rng.beta(beta[0], beta[1], size=D)
    x = rng.laplace(0.0, 1.0, size=(M, D)) * c[None, :] * scale
    return np.rint(x).astype(np.int32)


def ternary_case(seed: int = SEEDS["ternary"], M: int = 4, D: int = 4096, N: int = 14336,
                 K: int = 2, T: int = 8) -> TernaryCase:
    a = ternary_activations(stream(seed, 1), M, D)
    W = int8_uniform(stream(seed, 2), (D, N))
    return TernaryCase(a, W, K, T)

