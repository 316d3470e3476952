"""The paper's analytic performance model of a spiking linear layer
(Sec. IV, Eqs. (12)-(16), Table I), evaluated on host.

Per token of a block of B tokens over T timesteps, for a linear layer with
a d_in x d_out weight matrix of b_W-bit weights and input spikes that are
zero with probability sigma (i.i.d.):

* operations, Eq. (12): every spike costs one multiply and one add per
  output, 2 T d_in d_out (1 - sigma);
* weight bits loaded, Eq. (13): a weight row is loaded when its input neuron
  spikes anywhere in the block's B*T rows, d_in d_out (1 - sigma^(B T)) b_W / B;
* token latency, Eq. (14): the larger of the compute time N_ops / L_ops and
  the transfer time N_data / L_data (Eq. (14) as printed; its prose repeats a
  division by B that Eq. (13) already applies, and is not followed);
* end-to-end throughput, Eq. (15): the inverse of the summed latencies of
  the encoder's layers plus the decoder's layers over its S denoising steps;
* energy per token, Eq. (16): N_ops E_ops + N_data E_data summed likewise.

The paper states Eqs. (12)-(13) for square D x D matrices; the products here
are rectangular, so d_in d_out takes the place of D^2.  The measured form of
Eq. (13) replaces 1 - sigma^(B T) by the union fraction a block actually had
(active input rows / d_in), which is what the product kernels read.

Platforms: the two systems of Table I (off-chip and in-chip memory), and
MI355X at its published dense int8 rate and HBM bandwidth.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Iterable, Optional, Sequence


@dataclass(frozen=True)
class Platform:
    name: str
    L_ops: float                   # operations per second
    L_data: float                  # bits per second from weight memory
    E_ops: Optional[float] = None  # joules per operation
    E_data: Optional[float] = None # joules per bit

    @property
    def ridge(self) -> float:
        """Operations per bit at which compute and transfer times are equal."""
        return self.L_ops / self.L_data


# Table I: representative off-chip (HBM) and in-chip memory systems.
OCMS = Platform("OCMS", 300e12, 8e12, 0.05e-12, 10e-12)
ICMS = Platform("ICMS", 20e12, 30e12, 0.05e-12, 0.5e-12)
# MI355X: dense int8 matrix rate 5.0 POP/s, HBM3E 8 TB/s = 64 Tb/s (no energy figures).
MI355X = Platform("MI355X", 5.0e15, 64e12)
PLATFORMS = (MI355X, OCMS, ICMS)


def n_ops(T: int, d_in: int, d_out: int, sigma: float) -> float:
    """Eq. (12): operations per token."""
    return 2.0 * T * d_in * d_out * (1.0 - sigma)


def n_data(B: int, T: int, d_in: int, d_out: int, sigma: float, b_w: int) -> float:
    """Eq. (13): weight bits loaded per token (expected, i.i.d. spikes)."""
    return d_in * d_out * (1.0 - sigma ** (B * T)) * b_w / B


def n_data_measured(B: int, d_in: int, d_out: int, union_frac: float, b_w: int) -> float:
    """Eq. (13) with the block's measured union fraction in place of its
    expectation 1 - sigma^(B T)."""
    return d_in * d_out * union_frac * b_w / B


def sigma_from_union(union_frac: float, B: int, T: int) -> float:
    """The i.i.d. sparsity whose expected union fraction is union_frac
    (inverts 1 - sigma^(B T))."""
    u = min(max(union_frac, 0.0), 1.0)
    if u >= 1.0:
        return 0.0
    return (1.0 - u) ** (1.0 / (B * T))


def token_latency(ops: float, bits: float, plat: Platform) -> tuple[float, str]:
    """Eq. (14): seconds per token and the regime that sets it."""
    tc, tm = ops / plat.L_ops, bits / plat.L_data
    return (tc, "compute") if tc >= tm else (tm, "memory")


def e2e_throughput(enc_latencies: Iterable[float], dec_latencies_per_step: Sequence[Iterable[float]]) -> float:
    """Eq. (15): tokens per second from the encoder layers' latencies and the
    decoder layers' latencies of every denoising step."""
    total = sum(enc_latencies) + sum(sum(step) for step in dec_latencies_per_step)
    return 1.0 / total if total > 0 else math.inf


def energy_per_token(loads: Iterable[tuple[float, float]], plat: Platform) -> float:
    """Eq. (16): joules per token from (N_ops, N_data) of every layer evaluation."""
    if plat.E_ops is None or plat.E_data is None:
        raise ValueError(f"{plat.name} has no energy parameters")
    return sum(o * plat.E_ops + b * plat.E_data for o, b in loads)


def layer_report(name: str, B: int, T: int, d_in: int, d_out: int, union_frac: float,
                 b_w: int = 8, measured_us: Optional[float] = None,
                 sigma: Optional[float] = None) -> dict:
    """Eqs. (12)-(14) for one product of a block step: N_data from its
    measured union fraction, N_ops from the measured input sparsity sigma
    (else from the i.i.d. inversion of the union fraction)."""
    sigma_src = "measured" if sigma is not None else "iid_from_union"
    if sigma is None:
        sigma = sigma_from_union(union_frac, B, T)
    ops = n_ops(T, d_in, d_out, sigma)
    bits = n_data_measured(B, d_in, d_out, union_frac, b_w)
    rep = {"name": name, "d_in": d_in, "d_out": d_out, "union_frac": union_frac,
           "sigma": sigma, "sigma_source": sigma_src,
           "expected_union_iid": 1.0 - sigma ** (B * T),
           "n_ops_per_token": ops, "n_data_bits_per_token": bits}
    for plat in PLATFORMS:
        tl, regime = token_latency(ops, bits, plat)
        rep[plat.name] = {"us_per_block": tl * B * 1e6, "regime": regime}
    if measured_us is not None:
        rep["measured_us_per_block"] = measured_us
    return rep


def block_report(layers: Sequence[dict], measured_step_us: Optional[float] = None) -> dict:
    """Sum of the per-product model latencies (Eq. (15)'s inner sum) per platform."""
    out = {"products": list(layers)}
    for plat in PLATFORMS:
        out[f"{plat.name}_us_per_block"] = sum(l[plat.name]["us_per_block"] for l in layers)
    meas = [l.get("measured_us_per_block") for l in layers]
    if all(m is not None for m in meas):
        out["measured_products_us_per_block"] = sum(meas)
    if measured_step_us is not None:
        out["measured_step_us"] = measured_step_us
    return out


def throughput_curve(D: int, T: int, sigma: float, b_w: int, blocks: Sequence[int],
                     plat: Platform) -> list[tuple[int, float, str]]:
    """Tokens per second of one D x D spiking linear layer against block size
    (Eqs. (12)-(14)): the trend of Sec. V-C (rising with B while memory-bound,
    flat once compute-bound)."""
    out = []
    for B in blocks:
        tl, regime = token_latency(n_ops(T, D, D, sigma), n_data(B, T, D, D, sigma, b_w), plat)
        out.append((B, 1.0 / tl, regime))
    return out


def main() -> None:
    # the paper's setting: D_emb = 512, T = 8, 16-bit weights (Sec. V-A, V-B)
    D, T, b_w = 512, 8, 16
    blocks = (1, 2, 4, 8, 16, 32, 64)
    for plat in (OCMS, ICMS, MI355X):
        print(f"{plat.name}: ridge {plat.ridge:.3g} OP/bit")
        for sigma in (0.0, 0.5, 0.8, 0.95):
            row = throughput_curve(D, T, sigma, b_w, blocks, plat)
            cells = "  ".join(f"B={B}:{tt / 1e6:.3g}M({r[0]})" for B, tt, r in row)
            print(f"  sigma={sigma:<4}  {cells}")


if __name__ == "__main__":
    main()
