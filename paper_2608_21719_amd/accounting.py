"""Algorithmic work of the layer: FLOPs and bytes the method must move.

Follows the paper's per-layer work model (App. B.2, eqs. flops-layer,
bytes-layer, ai-layer and gamma) and its roofline argument (§III-B), written
for a GQA layer with a gated (SwiGLU) FFN. With n_kv = n_q and a non-gated
FFN of width 4d, ``layer_params`` is 12 d^2 and the FLOP/byte counts reduce to
the paper's F = 24 B d^2 + 4 B S d and M = (12 d^2 + 2 B S d) b_w.

These are counts of required work (causal pairs only, no padding), used to
turn measured times into roofline fractions. Pure arithmetic, no device code.
"""
from dataclasses import dataclass

# MI355X public peaks
HBM_PEAK_GBS = 8000.0
BF16_DENSE_PEAK_TFLOPS = 2500.0
FP32_VECTOR_PEAK_TFLOPS = 157.3


# dense bf16 MFMA FLOPs per compute unit per clock on gfx950 (four SIMDs, each
# one 32x32x16 bf16 MFMA = 32768 FLOPs per 32 cycles)
BF16_FLOP_PER_CU_CLOCK = 4096


def bf16_peak_tflops(compute_units: int, clock_mhz: float) -> float:
    """Dense bf16 MFMA peak at a given engine clock (TFLOP/s)."""
    return compute_units * BF16_FLOP_PER_CU_CLOCK * clock_mhz * 1e6 / 1e12


def layer_params(d: int, d_q: int, d_kv: int, ffn: int, gated: bool = True) -> int:
    """Weight count of the four projections (norm gains excluded)."""
    return d * (d_q + 2 * d_kv) + d_q * d + (3 if gated else 2) * d * ffn


def gemm_flops(tokens: int, d: int, d_q: int, d_kv: int, ffn: int, gated: bool = True) -> int:
    """2 FLOPs per multiply-accumulate for every weight and every row."""
    return 2 * tokens * layer_params(d, d_q, d_kv, ffn, gated)


def gemm_flops_by_op(tokens: int, d: int, d_q: int, d_kv: int, ffn: int) -> dict:
    return {
        "qkv": 2 * tokens * d * (d_q + 2 * d_kv),
        "o": 2 * tokens * d_q * d,
        "gate_up": 2 * tokens * d * 2 * ffn,
        "down": 2 * tokens * ffn * d,
    }


def prefill_attention_flops(seq_lens, n_q: int, head_dim: int, prefix_lens=None) -> int:
    """QK^T and PV over causal pairs only: 4 * hd * n_q per visible pair.

    A prompt chunk of n new tokens after a prefix of L cached tokens has
    sum_{i<n} (L + i + 1) visible pairs.
    """
    total = 0
    for i, n in enumerate(seq_lens):
        L = 0 if prefix_lens is None else prefix_lens[i]
        pairs = n * L + n * (n + 1) // 2
        total += 4 * head_dim * n_q * pairs
    return total


def kv_bytes_per_token(n_layers: int, n_kv: int, head_dim: int, elt_bytes: int) -> int:
    """K and V of one token over all layers (the §III-C capacity figure)."""
    return n_layers * 2 * n_kv * head_dim * elt_bytes


def decode_attention_bytes(kv_lens, n_kv: int, head_dim: int, elt_bytes: int) -> int:
    """K and V bytes a decode step must read: kv_len keys per sequence.

    kv_len is the length after the step's append (the new token attends to
    itself). q, o and the split partials are not counted.
    """
    return sum(int(L) * 2 * n_kv * head_dim * elt_bytes for L in kv_lens)


def decode_attention_flops(kv_lens, n_q: int, head_dim: int) -> int:
    return sum(4 * head_dim * n_q * int(L) for L in kv_lens)


def weight_bytes(d: int, d_q: int, d_kv: int, ffn: int, elt_bytes: int) -> int:
    return layer_params(d, d_q, d_kv, ffn) * elt_bytes


# ----------------------------------------------------- the paper's MHA forms
def paper_layer_flops(B: int, d: int, S: int) -> int:
    """App. B.2 eq. flops-layer: 4 B d (6 d + S)."""
    return 4 * B * d * (6 * d + S)


def paper_layer_bytes(B: int, d: int, S: int, b_w: float) -> float:
    """App. B.2 eq. bytes-layer: 2 d (6 d + B S) b_w."""
    return 2 * d * (6 * d + B * S) * b_w


def arithmetic_intensity(flops: float, nbytes: float) -> float:
    return flops / nbytes


def ridge_point(peak_flops: float, peak_bw: float) -> float:
    """FLOP per byte at which compute and bandwidth limits meet (§III-B)."""
    return peak_flops / peak_bw


def gamma(ai: float, ridge: float) -> float:
    """App. B.2 eq. gamma: compute-bound fraction min(1, AI / I*)."""
    return min(1.0, ai / ridge)


@dataclass
class Roofline:
    bound: str
    achieved: float
    peak: float
    unit: str
    traffic: object = None
    extra: dict = None

    def as_dict(self) -> dict:
        d = {"bound": self.bound, "achieved": self.achieved, "peak": self.peak,
             "unit": self.unit, "frac": self.achieved / self.peak, "traffic": self.traffic}
        d.update(self.extra or {})
        return d
