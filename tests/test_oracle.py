"""Pins for the fp64 oracle: what the mathematics and the paper fix.

None of these retype the oracle's formulas; each checks it against something
independent: a scalar-loop implementation, a library routine (torch SDPA in
float64), closed forms, invariants and special cases.
"""
import math

import numpy as np
import pytest
import torch

from oracle import bruteforce
from oracle import layer as O
from synth.configs import LayerShape

TINY_BF = LayerShape(16, 4, 2, 4, 24, 1e-5, 10000.0, "f32")


def _weights(shape, seed, gain_std=0.3):
    r = np.random.default_rng(seed)
    d, dq, dkv, f = shape.hidden, shape.d_q, shape.d_kv, shape.ffn
    s = 0.4
    return {
        "attn_norm": 1.0 + gain_std * r.standard_normal(d),
        "wq": s * r.standard_normal((dq, d)),
        "wk": s * r.standard_normal((dkv, d)),
        "wv": s * r.standard_normal((dkv, d)),
        "wo": s * r.standard_normal((d, dq)),
        "ffn_norm": 1.0 + gain_std * r.standard_normal(d),
        "wg": s * r.standard_normal((f, d)),
        "wu": s * r.standard_normal((f, d)),
        "wd": s * r.standard_normal((d, f)),
    }


def _hist(shape, L, seed):
    r = np.random.default_rng(seed)
    return (r.standard_normal((L, shape.n_kv, shape.head_dim)),
            r.standard_normal((L, shape.n_kv, shape.head_dim)))


# ------------------------------------------------------------ brute force
@pytest.mark.parametrize("L,n", [(0, 5), (3, 5), (7, 1)])
def test_bruteforce_matches_oracle(L, n):
    w = _weights(TINY_BF, 1)
    x = np.random.default_rng(2).standard_normal((n, TINY_BF.hidden))
    kh, vh = _hist(TINY_BF, L, 3) if L else (None, None)
    ref = O.layer_sequence(w, TINY_BF, x, kh, vh)
    bf = bruteforce.layer_sequence(w, TINY_BF, x, kh, vh)
    assert np.max(np.abs(ref["out"] - np.array(bf["out"]))) <= 1e-12
    assert np.max(np.abs(ref["k"] - np.array(bf["k"]))) <= 1e-12
    assert np.max(np.abs(ref["v"] - np.array(bf["v"]))) <= 1e-12


def test_bruteforce_detects_planted_transpose():
    """A plausible slip (Wo applied untransposed) must be caught by the pin."""
    shape = LayerShape(8, 2, 1, 4, 12, 1e-5, 10000.0, "f32")
    w = _weights(shape, 4)
    x = np.random.default_rng(5).standard_normal((3, 8))
    bad = dict(w)
    bad["wo"] = w["wo"].T.copy()
    ref = O.layer_sequence(bad, shape, x)
    bf = bruteforce.layer_sequence(w, shape, x)
    assert np.max(np.abs(ref["out"] - np.array(bf["out"]))) > 1e-3


# ------------------------------------------------------------ attention
def _sdpa(q, k, v, q_pos):
    """torch float64 SDPA with the KV heads repeated over the group."""
    T, nq, hd = q.shape
    L, nkv, _ = k.shape
    G = nq // nkv
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    mask = torch.from_numpy(np.arange(L)[None, :] <= np.asarray(q_pos)[:, None])
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask)
    return o[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("T,L0,nq,nkv,hd", [(9, 0, 4, 2, 8), (5, 11, 8, 1, 16), (1, 40, 6, 3, 4)])
def test_attention_matches_torch_sdpa(T, L0, nq, nkv, hd):
    r = np.random.default_rng(T * 100 + L0)
    q = r.standard_normal((T, nq, hd))
    k = r.standard_normal((L0 + T, nkv, hd))
    v = r.standard_normal((L0 + T, nkv, hd))
    pos = np.arange(L0, L0 + T)
    np.testing.assert_allclose(O.attention(q, k, v, pos), _sdpa(q, k, v, pos), rtol=0, atol=1e-12)


def test_attention_gqa_mapping_matches_sdpa_enable_gqa():
    """torch's own GQA routing (query head h -> kv head h // G) agrees."""
    r = np.random.default_rng(7)
    T, nq, nkv, hd = 6, 8, 2, 8
    q = r.standard_normal((T, nq, hd))
    k = r.standard_normal((T, nkv, hd))
    v = r.standard_normal((T, nkv, hd))
    o = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).permute(1, 0, 2)[None], torch.from_numpy(k).permute(1, 0, 2)[None],
        torch.from_numpy(v).permute(1, 0, 2)[None], is_causal=True, enable_gqa=True)
    np.testing.assert_allclose(O.attention(q, k, v, np.arange(T)), o[0].permute(1, 0, 2).numpy(),
                               rtol=0, atol=1e-12)


def test_softmax_rows_sum_to_one_and_respect_mask():
    r = np.random.default_rng(8)
    q = 3 * r.standard_normal((7, 4, 8))
    k = r.standard_normal((10, 2, 8))
    v = r.standard_normal((10, 2, 8))
    pos = np.arange(3, 10)
    _, p = O.attention(q, k, v, pos, return_probs=True)
    assert np.max(np.abs(p.sum(-1) - 1.0)) <= 1e-12
    for i, pi in enumerate(pos):
        assert np.all(p[i, :, pi + 1:] == 0.0)
        assert np.all(p[i, :, :pi + 1] > 0.0)


def test_attention_single_key_returns_v0():
    """A first token with no history sees only itself: o = v0 for its group."""
    r = np.random.default_rng(9)
    q = r.standard_normal((1, 4, 8))
    k = r.standard_normal((1, 2, 8))
    v = r.standard_normal((1, 2, 8))
    o = O.attention(q, k, v, np.array([0]))
    for h in range(4):
        np.testing.assert_array_equal(o[0, h], v[0, h // 2])


def test_attention_zero_query_is_mean_of_visible_values():
    r = np.random.default_rng(10)
    q = np.zeros((5, 2, 4))
    k = r.standard_normal((8, 1, 4))
    v = r.standard_normal((8, 1, 4))
    pos = np.arange(3, 8)
    o = O.attention(q, k, v, pos)
    for i, p in enumerate(pos):
        np.testing.assert_allclose(o[i, 0], v[:p + 1, 0].mean(0), atol=1e-14)


# ------------------------------------------------------------ RoPE
def test_rope_identity_at_position_zero():
    x = np.random.default_rng(11).standard_normal((1, 3, 16))
    np.testing.assert_array_equal(O.rope(x, np.array([0]), 10000.0), x)


def test_rope_matches_complex_rotation():
    """Pair (j, j+hd/2) as a complex number times exp(i p theta^(-2j/hd))."""
    hd, theta = 16, 500000.0
    x = np.random.default_rng(12).standard_normal((5, 2, hd))
    pos = np.array([0, 1, 7, 1000, 31999])
    z = x[..., :hd // 2] + 1j * x[..., hd // 2:]
    rot = np.array([[cmath_exp(p * theta ** (-2.0 * j / hd)) for j in range(hd // 2)] for p in pos])
    zr = z * rot[:, None, :]
    ref = np.concatenate([zr.real, zr.imag], axis=-1)
    np.testing.assert_allclose(O.rope(x, pos, theta), ref, atol=1e-12)


def cmath_exp(a):
    return complex(math.cos(a), math.sin(a))


def test_rope_preserves_pair_norms_and_relative_dot():
    hd, theta = 32, 10000.0
    r = np.random.default_rng(13)
    q = r.standard_normal((1, 1, hd))
    k = r.standard_normal((1, 1, hd))
    qr = O.rope(q, np.array([17]), theta)
    np.testing.assert_allclose(qr[..., :16] ** 2 + qr[..., 16:] ** 2,
                               q[..., :16] ** 2 + q[..., 16:] ** 2, atol=1e-12)
    d1 = np.sum(O.rope(q, np.array([17]), theta) * O.rope(k, np.array([5]), theta))
    d2 = np.sum(O.rope(q, np.array([117]), theta) * O.rope(k, np.array([105]), theta))
    assert abs(d1 - d2) < 1e-10


def test_rope_two_dims_one_radian():
    x = np.array([[[1.0, 0.0]]])
    y = O.rope(x, np.array([1]), 10000.0)  # hd = 2: inverse frequency 1
    np.testing.assert_allclose(y[0, 0], [math.cos(1.0), math.sin(1.0)], atol=1e-15)


# ------------------------------------------------------------ RMSNorm / SiLU
def test_rmsnorm_unit_gain_output_rms():
    x = np.random.default_rng(14).standard_normal((4, 64)) * 0.01
    eps = 1e-5
    y = O.rmsnorm(x, np.ones(64), eps)
    ms = np.mean(x * x, -1)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, -1)), np.sqrt(ms / (ms + eps)), rtol=1e-12)
    z = O.rmsnorm(x, np.ones(64), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(z * z, -1)), 1.0, rtol=1e-12)


def test_rmsnorm_gain_is_elementwise():
    x = np.random.default_rng(15).standard_normal((3, 8))
    g = np.arange(1, 9, dtype=np.float64)
    np.testing.assert_allclose(O.rmsnorm(x, g, 1e-5), O.rmsnorm(x, np.ones(8), 1e-5) * g, rtol=1e-14)


def test_silu_values():
    assert O.silu(np.array(0.0)) == 0.0
    assert abs(O.silu(np.array(1.0)) - 0.7310585786300049) < 1e-15
    assert abs(O.silu(np.array(40.0)) - 40.0) < 1e-12
    assert abs(O.silu(np.array(-40.0))) < 1e-15


# ------------------------------------------------------------ layer-level
def test_decode_step_equals_last_row_of_prefill():
    shape = LayerShape(32, 4, 2, 8, 48, 1e-5, 10000.0, "f32")
    w = _weights(shape, 16, 0.1)
    x = np.random.default_rng(17).standard_normal((9, 32))
    full = O.layer_sequence(w, shape, x)
    pre = O.layer_sequence(w, shape, x[:8])
    dec = O.layer_sequence(w, shape, x[8:], pre["k"], pre["v"])
    assert np.max(np.abs(dec["out"][0] - full["out"][8])) <= 1e-12
    assert np.max(np.abs(dec["k"][0] - full["k"][8])) <= 1e-12


def test_chunked_prefill_equals_full_prefill():
    shape = LayerShape(32, 4, 1, 8, 48, 1e-5, 500000.0, "f32")
    w = _weights(shape, 18, 0.1)
    x = np.random.default_rng(19).standard_normal((12, 32))
    full = O.layer_sequence(w, shape, x)
    a = O.layer_sequence(w, shape, x[:5])
    b = O.layer_sequence(w, shape, x[5:], a["k"], a["v"])
    assert np.max(np.abs(np.concatenate([a["out"], b["out"]]) - full["out"])) <= 1e-12


def test_zero_projections_give_residual_identity():
    shape = LayerShape(16, 2, 1, 8, 24, 1e-5, 10000.0, "f32")
    w = _weights(shape, 20)
    w["wo"][:] = 0.0
    w["wd"][:] = 0.0
    x = np.random.default_rng(21).standard_normal((4, 16))
    np.testing.assert_array_equal(O.layer_sequence(w, shape, x)["out"], x)


def test_sequences_are_independent():
    shape = LayerShape(16, 2, 1, 8, 24, 1e-5, 10000.0, "f32")
    w = _weights(shape, 22)
    r = np.random.default_rng(23)
    xa, xb = r.standard_normal((3, 16)), r.standard_normal((4, 16))
    both = O.layer_batch(w, shape, [xa, xb])
    np.testing.assert_array_equal(both[1]["out"], O.layer_sequence(w, shape, xb)["out"])


def test_argmax_ties_go_to_lowest_index():
    logits = np.array([[0.0, 3.0, 1.0, 3.0], [5.0, 5.0, 5.0, 5.0]])
    assert list(O.argmax_lowest(logits)) == [1, 0]


# ------------------------------------------------------------ model head
# The model head follows the stack the evaluation serves (§VI: 70B-class
# Llama-family models): h0 = E[token]; logits = RMSNorm(h_L) * g_final . W_lm^T;
# next = argmax. Pinned by scalar loops, one-hot / identity-weight closed forms
# and planted mistakes that the pins must catch.
def _embed_scalar(table, tokens):
    rows = table.tolist()
    return [list(rows[t]) for t in tokens]


def _lm_logits_scalar(h, g, w_lm, eps):
    gl, wl = g.tolist(), w_lm.tolist()
    out = []
    for row in h.tolist():
        ms = 0.0
        for a in row:
            ms += a * a
        inv = 1.0 / math.sqrt(ms / len(row) + eps)
        hn = [row[i] * inv * gl[i] for i in range(len(row))]
        logits = []
        for wr in wl:
            acc = 0.0
            for i in range(len(hn)):
                acc += wr[i] * hn[i]
            logits.append(acc)
        out.append(logits)
    return out


def test_embed_is_a_row_gather():
    r = np.random.default_rng(30)
    table = r.standard_normal((11, 6))
    tokens = np.array([3, 0, 10, 3, 7])
    got = O.embed(table, tokens)
    np.testing.assert_array_equal(got, np.array(_embed_scalar(table, tokens)))
    onehot = np.zeros((len(tokens), 11))
    onehot[np.arange(len(tokens)), tokens] = 1.0
    np.testing.assert_array_equal(got, onehot @ table)  # E^T e_t, exact with one nonzero term
    assert got.shape == (5, 6) and np.array_equal(got[0], got[3])


def _lm_logits_pins_hold():
    """True when oracle.lm_logits passes every pin below (used on planted mutants too)."""
    r = np.random.default_rng(31)
    d, vocab, eps = 12, 17, 1e-5
    h = r.standard_normal((3, d)) * 3.0
    g = 1.0 + 0.3 * r.standard_normal(d)
    w = r.standard_normal((vocab, d))
    ok = np.max(np.abs(O.lm_logits(h, g, w, eps) - np.array(_lm_logits_scalar(h, g, w, eps)))) <= 1e-12
    # identity head, unit gain, eps 0: the logits are the normalised row (RMS exactly 1)
    z = O.lm_logits(h, np.ones(d), np.eye(d), 0.0)
    ok = ok and np.allclose(np.sqrt(np.mean(z * z, -1)), 1.0, rtol=1e-13, atol=0)
    # a final norm makes the head invariant to the scale of h (eps 0)
    ok = ok and np.allclose(O.lm_logits(7.5 * h, g, w, 0.0), O.lm_logits(h, g, w, 0.0), rtol=1e-12, atol=1e-12)
    # the gain multiplies before the head: doubling g doubles every logit
    ok = ok and np.allclose(O.lm_logits(h, 2.0 * g, w, eps), 2.0 * O.lm_logits(h, g, w, eps), rtol=1e-13, atol=0)
    return bool(ok)


def test_lm_logits_pins():
    assert _lm_logits_pins_hold()


@pytest.mark.parametrize("mutant", ["no_final_norm", "no_gain", "eps_outside_sqrt"])
def test_lm_logits_pins_catch_planted_mistakes(monkeypatch, mutant):
    """Plant a plausible slip in the oracle's final norm; the pins must fail."""
    orig = O.rmsnorm
    if mutant == "no_final_norm":
        monkeypatch.setattr(O, "rmsnorm", lambda x, g, eps: x * g)
    elif mutant == "no_gain":
        monkeypatch.setattr(O, "rmsnorm", lambda x, g, eps: orig(x, np.ones_like(g), eps))
    else:
        monkeypatch.setattr(O, "rmsnorm",
                            lambda x, g, eps: x / (np.sqrt(np.mean(x * x, -1, keepdims=True)) + eps) * g)
    assert not _lm_logits_pins_hold()


@pytest.mark.parametrize("L", [0, 6])
def test_layer_rows_equals_the_rows_of_layer_sequence(L):
    shape = LayerShape(32, 4, 2, 8, 48, 1e-5, 10000.0, "f32")
    w = _weights(shape, 24, 0.1)
    x = np.random.default_rng(25).standard_normal((9, 32))
    kh, vh = _hist(shape, L, 26) if L else (None, None)
    full = O.layer_sequence(w, shape, x, kh, vh)["out"]
    rows = [8, 0, 4]
    assert np.max(np.abs(O.layer_rows(w, shape, x, rows, kh, vh) - full[rows])) <= 1e-12
