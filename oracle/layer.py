"""Plain float64 definition of one pre-norm dense GQA decoder layer.

TEST INFRASTRUCTURE ONLY: never imported by the product path.

What is computed. The paper characterises, but never writes out, the forward
pass its serving phases run (§II-B "LLM Serving Phases": prefill computes
attention over every prompt token at once; decode generates one token per
step and is dominated by reading the KV cache; reasoning "think" is a long
decode). Its per-layer work model (App. B.2, eqs. flops-layer and
bytes-layer) counts projections, MLP and attention of a standard layer. The
models it serves are Llama-family (Llama-70B, CodeLlama-34B,
DeepSeek-R1-Llama-70B, Qwen). This module is the plain definition of that
layer in the Llama form:

    xn  = RMSNorm(x) * g_attn
    q, k, v = xn Wq^T, xn Wk^T, xn Wv^T
    q, k = RoPE(q, pos), RoPE(k, pos)          (rotate-half, absolute positions)
    o_h = softmax(q_h K_{h // G}^T / sqrt(hd) + causal) V_{h // G}
    h   = x + concat(o) Wo^T
    hn  = RMSNorm(h) * g_ffn
    out = h + (silu(hn Wg^T) * (hn Wu^T)) Wd^T

Readings of the paper's silences (each also listed in the design notes):
  * pre-norm Llama layer, no biases, W[out, in] with y = x W^T;
  * RMSNorm: eps inside the square root, mean over the hidden dimension,
    gain applied after normalising;
  * RoPE: rotate-half pairs (j, j + hd/2), inverse frequency
    theta^(-2j/hd), angle computed in float64, no frequency scaling,
    applied to q and k only;
  * GQA: query head h reads KV head floor(h / G), contiguous groups;
  * scale 1/sqrt(hd); key j is visible to a query at position i iff j <= i,
    within its own sequence;
  * a decode token at position L (L = cached length) has its k, v appended
    before attention and attends over L + 1 keys, itself included.

No step is blocked, fused or reordered beyond this definition. Inputs arrive
as float64 arrays holding exactly the values the device receives.
"""
import math

import numpy as np


# ------------------------------------------------------------------ stages
def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def linear(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """y = x W^T with W stored [out, in]."""
    return x @ w.T


def rope_inv_freq(head_dim: int, theta: float) -> np.ndarray:
    j = np.arange(head_dim // 2, dtype=np.float64)
    return theta ** (-2.0 * j / head_dim)


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half RoPE. x [T, H, hd], pos [T] absolute 0-based positions.

    Pair (j, j + hd/2) of a head at position p is rotated by angle
    p * theta^(-2j/hd).
    """
    hd = x.shape[-1]
    half = hd // 2
    ang = np.asarray(pos, dtype=np.float64)[:, None] * rope_inv_freq(hd, theta)[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos: np.ndarray,
              return_probs: bool = False):
    """Causal GQA softmax attention for ONE sequence.

    q [T, n_q, hd] at absolute positions q_pos [T]; k, v [L, n_kv, hd] hold
    every key of the sequence, key j at position j. Key j is visible to query
    i iff j <= q_pos[i].
    """
    T, n_q, hd = q.shape
    L, n_kv, _ = k.shape
    G = n_q // n_kv
    scale = 1.0 / math.sqrt(hd)
    visible = np.arange(L)[None, :] <= np.asarray(q_pos)[:, None]
    o = np.empty((T, n_q, hd), dtype=np.float64)
    probs = []
    for h in range(n_q):
        kh = k[:, h // G, :]
        vh = v[:, h // G, :]
        s = (q[:, h, :] @ kh.T) * scale
        s = np.where(visible, s, -np.inf)
        s = s - np.max(s, axis=1, keepdims=True)
        p = np.exp(s)
        p = p / np.sum(p, axis=1, keepdims=True)
        o[:, h, :] = p @ vh
        if return_probs:
            probs.append(p)
    if return_probs:
        return o, np.stack(probs, axis=1)  # [T, n_q, L]
    return o


# ------------------------------------------------------------------ layer
def layer_sequence(w: dict, shape, x: np.ndarray, k_hist: np.ndarray = None,
                   v_hist: np.ndarray = None) -> dict:
    """The layer over the new rows of ONE sequence.

    x [n, d] are the rows at positions L .. L+n-1 where L = len(k_hist)
    (0 without history). k_hist / v_hist [L, n_kv, hd] are what the cache
    holds for positions 0 .. L-1 (keys already rotated). Returns every stage
    so that device stages can be compared one at a time; ``k`` and ``v`` are
    the rotated keys and the values the step appends to the cache.
    """
    n, d = x.shape
    nq, nkv, hd = shape.n_q, shape.n_kv, shape.head_dim
    if k_hist is None:
        k_hist = np.zeros((0, nkv, hd))
        v_hist = np.zeros((0, nkv, hd))
    L = k_hist.shape[0]
    pos = np.arange(L, L + n)

    xn = rmsnorm(x, w["attn_norm"], shape.eps)
    q_raw = linear(xn, w["wq"]).reshape(n, nq, hd)
    k_raw = linear(xn, w["wk"]).reshape(n, nkv, hd)
    v_new = linear(xn, w["wv"]).reshape(n, nkv, hd)
    q = rope(q_raw, pos, shape.theta)
    k_new = rope(k_raw, pos, shape.theta)
    K = np.concatenate([k_hist, k_new], axis=0)
    V = np.concatenate([v_hist, v_new], axis=0)
    o = attention(q, K, V, pos).reshape(n, nq * hd)
    h = x + linear(o, w["wo"])
    hn = rmsnorm(h, w["ffn_norm"], shape.eps)
    gate = linear(hn, w["wg"])
    up = linear(hn, w["wu"])
    m = silu(gate) * up
    out = h + linear(m, w["wd"])
    return {"xn": xn, "q_raw": q_raw, "k_raw": k_raw, "q": q, "k": k_new, "v": v_new,
            "o": o, "h": h, "hn": hn, "gate": gate, "up": up, "m": m, "out": out,
            "pos": pos}


def layer_rows(w: dict, shape, x: np.ndarray, rows, k_hist: np.ndarray = None,
               v_hist: np.ndarray = None) -> np.ndarray:
    """The same layer as layer_sequence, output of the selected new rows only.

    Keys and values come from every row (attention needs them); the query,
    attention, projections and FFN are evaluated for `rows` (indices into x)
    alone. Rows are independent except through attention, so each result
    equals the matching row of layer_sequence. Returns out [len(rows), d].
    """
    n, d = x.shape
    nq, nkv, hd = shape.n_q, shape.n_kv, shape.head_dim
    if k_hist is None:
        k_hist = np.zeros((0, nkv, hd))
        v_hist = np.zeros((0, nkv, hd))
    L = k_hist.shape[0]
    pos = np.arange(L, L + n)
    rows = np.asarray(rows)
    xn = rmsnorm(x, w["attn_norm"], shape.eps)
    k_new = rope(linear(xn, w["wk"]).reshape(n, nkv, hd), pos, shape.theta)
    v_new = linear(xn, w["wv"]).reshape(n, nkv, hd)
    K = np.concatenate([k_hist, k_new], axis=0)
    V = np.concatenate([v_hist, v_new], axis=0)
    q = rope(linear(xn[rows], w["wq"]).reshape(len(rows), nq, hd), pos[rows], shape.theta)
    o = attention(q, K, V, pos[rows]).reshape(len(rows), nq * hd)
    h = x[rows] + linear(o, w["wo"])
    hn = rmsnorm(h, w["ffn_norm"], shape.eps)
    m = silu(linear(hn, w["wg"])) * linear(hn, w["wu"])
    return h + linear(m, w["wd"])


def layer_batch(w: dict, shape, xs, hists=None) -> list:
    """The layer over several independent sequences (no cross-sequence attention)."""
    res = []
    for i, x in enumerate(xs):
        kh, vh = (None, None) if hists is None or hists[i] is None else hists[i]
        res.append(layer_sequence(w, shape, x, kh, vh))
    return res


# ------------------------------------------------------------------ model head
def embed(table: np.ndarray, tokens: np.ndarray) -> np.ndarray:
    return table[np.asarray(tokens)]


def lm_logits(h: np.ndarray, g_final: np.ndarray, w_lm: np.ndarray, eps: float) -> np.ndarray:
    return linear(rmsnorm(h, g_final, eps), w_lm)


def argmax_lowest(logits: np.ndarray) -> np.ndarray:
    """Greedy token: the largest logit, ties broken toward the lowest index."""
    return np.argmax(logits, axis=-1)
