"""A model of the device's bf16 rounding, used to derive end-to-end tolerances.

Test-side only; not the oracle and not the device path. It evaluates the layer
in float32 arithmetic and rounds to bf16 (nearest, ties to even) at exactly
the points where the device stores or feeds bf16: the GEMM inputs (xn, o, hn,
m), the QKV projection's output, the rotated q and k and the stored v, the
softmax weights P that enter the PV product (the normaliser sums the same
rounded P), and the layer output. The residual stream h stays fp32, as on the
device. Compared with the fp64 oracle, its error is the floor that any
pipeline with these rounding points reaches, independent of kernel details.
"""
import numpy as np

from synth import gen


def bf(a) -> np.ndarray:
    """Round to bf16 (RNE) and return the rounded values as float32."""
    return gen.bf16_bits_to_f32(gen.f32_to_bf16_bits(np.asarray(a, np.float32)))


def _rms32(x, g, eps):
    ms = np.mean(x * x, axis=-1, keepdims=True, dtype=np.float32)
    return (x / np.sqrt(ms + np.float32(eps)) * g).astype(np.float32)


def _rope32(x, pos, theta):
    """Rotate-half pairs (j, j + hd/2); angle in float64, rotation in float32."""
    hd = x.shape[-1]
    half = hd // 2
    ang = pos[:, None].astype(np.float64) * theta ** (-2.0 * np.arange(half) / hd)[None, :]
    c = np.cos(ang).astype(np.float32)[:, None, :]
    s = np.sin(ang).astype(np.float32)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def weights_f32(w: dict) -> dict:
    """bf16 storage bits -> float32 values (exact)."""
    return {k: gen.bf16_bits_to_f32(v) for k, v in w.items()}


class WidenedWeights:
    """Read-only mapping name -> weight widened exactly from bf16 bits to
    `dtype`, converted on access into one buffer reused for every matrix.

    Holding a 70B-shaped layer in float64 takes 6.8 GB of fresh memory, and
    faulting it in dominates the run time of a CPU test; the layer
    definitions here and in the oracle read each matrix once, right before
    using it, so one buffer of the largest matrix suffices. An access
    invalidates the array returned by the previous access of a matrix.
    """

    def __init__(self, bits: dict, dtype):
        self.bits = bits
        self.dtype = np.dtype(dtype)
        self.small = {k: gen.bf16_bits_to_f32(v).astype(self.dtype) for k, v in bits.items() if v.ndim == 1}
        big = max((v.size for v in bits.values() if v.ndim > 1), default=0)
        self.buf = np.empty(big, self.dtype)
        self.tmp = np.empty(big, np.uint32)

    def __getitem__(self, k):
        if k in self.small:
            return self.small[k]
        b = self.bits[k]
        t = self.tmp[:b.size].reshape(b.shape)
        np.left_shift(b, 16, out=t, dtype=np.uint32)
        out = self.buf[:b.size].reshape(b.shape)
        out[...] = t.view(np.float32)
        return out

    def keys(self):
        return self.bits.keys()


def layer(w32: dict, shape, x32: np.ndarray, k_hist=None, v_hist=None, return_kv: bool = False):
    """The layer over the new rows of one sequence (rows at positions L..L+n-1,
    L = len(k_hist)); history is bf16-valued float32 [L, n_kv, hd]. With
    return_kv, also the rounded k and v rows the step appends."""
    n = x32.shape[0]
    nq, nkv, hd = shape.n_q, shape.n_kv, shape.head_dim
    G = nq // nkv
    L = 0 if k_hist is None else k_hist.shape[0]
    pos = np.arange(L, L + n)
    xn = bf(_rms32(x32, w32["attn_norm"], shape.eps))
    q = bf(xn @ w32["wq"].T).reshape(n, nq, hd)
    k = bf(xn @ w32["wk"].T).reshape(n, nkv, hd)
    v = bf(xn @ w32["wv"].T).reshape(n, nkv, hd)
    q = bf(_rope32(q, pos, shape.theta))
    k = bf(_rope32(k, pos, shape.theta))
    k_new, v_new = k, v
    if L:
        k = np.concatenate([k_hist, k])
        v = np.concatenate([v_hist, v])
    scale = np.float32(1.0 / np.sqrt(hd))
    visible = np.arange(L + n)[None, :] <= pos[:, None]
    o = np.empty((n, nq, hd), np.float32)
    for h in range(nq):
        s = (q[:, h] @ k[:, h // G].T) * scale
        s = np.where(visible, s, -np.inf)
        p = bf(np.exp(s - s.max(axis=1, keepdims=True)))
        o[:, h] = (p @ v[:, h // G]) / p.sum(axis=1, keepdims=True, dtype=np.float32)
    o = bf(o).reshape(n, nq * hd)
    hres = x32 + o @ w32["wo"].T
    hn = bf(_rms32(hres, w32["ffn_norm"], shape.eps))
    gate = hn @ w32["wg"].T
    up = hn @ w32["wu"].T
    m = bf(gate / (np.float32(1.0) + np.exp(-gate)) * up)
    out = bf(hres + m @ w32["wd"].T)
    return (out, k_new, v_new) if return_kv else out


def lm_logits(h32: np.ndarray, g_final32: np.ndarray, w_lm32: np.ndarray, eps: float) -> np.ndarray:
    """Final RMSNorm rounded to bf16 (the LM head GEMM's input), fp32 logits."""
    return bf(_rms32(h32, g_final32, eps)) @ w_lm32.T
