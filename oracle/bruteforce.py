"""Scalar-loop version of the decoder layer for tiny shapes.

TEST INFRASTRUCTURE ONLY. Written independently of ``oracle.layer`` (pure
Python floats and the ``math`` module, explicit loops, no numpy arithmetic)
so that the two agreeing to ~1e-12 pins the vectorised oracle against slips
such as a transposed weight, a wrong GQA head index or an off-by-one causal
mask. Same layer definition and readings as ``oracle.layer``.
"""
import math


def _rms(row, gain, eps):
    ms = 0.0
    for a in row:
        ms += a * a
    ms /= len(row)
    inv = 1.0 / math.sqrt(ms + eps)
    return [row[i] * inv * gain[i] for i in range(len(row))]


def _matvec(W, x):
    # W[out][in], returns W x
    out = []
    for r in W:
        acc = 0.0
        for i in range(len(x)):
            acc += r[i] * x[i]
        out.append(acc)
    return out


def _rotate(vec, pos, theta):
    hd = len(vec)
    half = hd // 2
    res = list(vec)
    for j in range(half):
        ang = pos * math.pow(theta, -2.0 * j / hd)
        c, s = math.cos(ang), math.sin(ang)
        a, b = vec[j], vec[j + half]
        res[j] = a * c - b * s
        res[j + half] = b * c + a * s
    return res


def layer_sequence(w, shape, x, k_hist=None, v_hist=None):
    """Same contract as ``oracle.layer.layer_sequence`` (returns out, k, v)."""
    W = {key: (val.tolist() if hasattr(val, "tolist") else val) for key, val in w.items()}
    X = x.tolist() if hasattr(x, "tolist") else x
    nq, nkv, hd = shape.n_q, shape.n_kv, shape.head_dim
    G = nq // nkv
    K = [] if k_hist is None else (k_hist.tolist() if hasattr(k_hist, "tolist") else k_hist)
    V = [] if v_hist is None else (v_hist.tolist() if hasattr(v_hist, "tolist") else v_hist)
    K = [[list(hrow) for hrow in tok] for tok in K]
    V = [[list(hrow) for hrow in tok] for tok in V]
    L = len(K)
    outs, ks, vs = [], [], []
    # first pass: projections of every new row (keys of later rows must exist
    # before earlier rows are finished only for visibility, which is causal,
    # so rows can be processed in order)
    for t, row in enumerate(X):
        p = L + t
        xn = _rms(row, W["attn_norm"], shape.eps)
        qf = _matvec(W["wq"], xn)
        kf = _matvec(W["wk"], xn)
        vf = _matvec(W["wv"], xn)
        q_heads = [_rotate(qf[h * hd:(h + 1) * hd], p, shape.theta) for h in range(nq)]
        k_heads = [_rotate(kf[g * hd:(g + 1) * hd], p, shape.theta) for g in range(nkv)]
        v_heads = [vf[g * hd:(g + 1) * hd] for g in range(nkv)]
        K.append(k_heads)
        V.append(v_heads)
        ks.append(k_heads)
        vs.append(v_heads)
        o = []
        for h in range(nq):
            g = h // G
            scores = []
            for j in range(p + 1):  # keys 0..p are visible
                dot = 0.0
                for e in range(hd):
                    dot += q_heads[h][e] * K[j][g][e]
                scores.append(dot / math.sqrt(hd))
            z = 0.0
            ex = []
            for sc in scores:
                ex.append(math.exp(sc))
                z += ex[-1]
            for e in range(hd):
                acc = 0.0
                for j in range(p + 1):
                    acc += ex[j] / z * V[j][g][e]
                o.append(acc)
        attn = _matvec(W["wo"], o)
        hres = [row[i] + attn[i] for i in range(len(row))]
        hn = _rms(hres, W["ffn_norm"], shape.eps)
        gate = _matvec(W["wg"], hn)
        up = _matvec(W["wu"], hn)
        m = [gate[i] / (1.0 + math.exp(-gate[i])) * up[i] for i in range(len(gate))]
        down = _matvec(W["wd"], m)
        outs.append([hres[i] + down[i] for i in range(len(hres))])
    return {"out": outs, "k": ks, "v": vs}
