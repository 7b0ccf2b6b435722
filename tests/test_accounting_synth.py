"""Accounting helpers against the numbers the paper prints; generator checks."""
import json
import os

import numpy as np
import pytest

from paper_2608_21719_amd import accounting as A
from synth import gen
from synth.configs import CONFIGS

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def test_kv_bytes_per_token_llama70b():
    g = GOLD["kv_bytes_per_token_llama70b"]
    s = g["shape"]
    assert A.kv_bytes_per_token(s["n_layers"], s["n_kv"], s["head_dim"], s["elt_bytes"]) == g["value"]
    assert g["value"] == 320 * 1024
    # the 70B-shaped workload has that KV footprint
    sh = CONFIGS["llama70b_model"].shape
    assert A.kv_bytes_per_token(80, sh.n_kv, sh.head_dim, sh.elt_bytes) == g["value"]


def test_kv_chain_and_capacity():
    per_tok = GOLD["kv_bytes_per_token_llama70b"]["value"]
    g = GOLD["kv_bytes_4k_chain_GB"]
    chain = per_tok * g["tokens"] / 1e9
    assert abs(chain - g["value"]) / g["value"] < g["rel_tol"]
    c = GOLD["concurrent_4k_chains_180GB"]
    n = c["capacity_GB"] * 1e9 / (per_tok * c["tokens"])
    assert abs(n - c["value"]) / c["value"] < c["rel_tol"]


def test_a100_ridge_point():
    g = GOLD["a100_ridge_flop_per_byte"]
    assert abs(A.ridge_point(g["peak_tflops"] * 1e12, g["peak_tbs"] * 1e12) - g["value"]) < g["abs_tol"]


def test_decode_ai_is_batch_at_zero_context():
    g = GOLD["decode_ai_equals_batch"]
    d = 8192
    for B in g["batches"]:
        ai = A.arithmetic_intensity(A.paper_layer_flops(B, d, 0), A.paper_layer_bytes(B, d, 0, g["b_w"]))
        assert abs(ai - B) < 1e-12
        # the GQA/SwiGLU accounting gives the same ratio for the weight-streaming GEMMs
        sh = CONFIGS["llama70b_model"].shape
        w = A.weight_bytes(sh.hidden, sh.d_q, sh.d_kv, sh.ffn, g["b_w"])
        assert abs(A.gemm_flops(B, sh.hidden, sh.d_q, sh.d_kv, sh.ffn) / w - B) < 1e-12


def test_gqa_accounting_reduces_to_paper_mha_form():
    d = GOLD["mha_weights_12d2"]["d"]
    assert A.layer_params(d, d, d, 4 * d, gated=False) == 12 * d * d
    B, S = 64, 4096
    ours = A.gemm_flops(B, d, d, d, 4 * d, gated=False) + A.decode_attention_flops([S] * B, d // 128, 128)
    assert ours == A.paper_layer_flops(B, d, S)
    kv = A.decode_attention_bytes([S] * B, d // 128, 128, 2)
    assert A.layer_params(d, d, d, 4 * d, False) * 2 + kv == A.paper_layer_bytes(B, d, S, 2)


def test_gamma_limits():
    assert A.gamma(1e6, 315.0) == 1.0
    assert A.gamma(4.0, 315.0) < 0.02


def test_8b_layer_counts():
    s = CONFIGS["llama8b_prefill"].shape
    assert A.layer_params(s.hidden, s.d_q, s.d_kv, s.ffn) == 218_103_808
    fl = A.gemm_flops(8 * 2048, s.hidden, s.d_q, s.d_kv, s.ffn)
    assert abs(fl / 1e12 - 7.147) < 1e-3
    att = A.prefill_attention_flops([2048] * 8, s.n_q, s.head_dim)
    assert abs(att / 1e9 - 275.0) < 0.1


# ------------------------------------------------------------ generator
def test_bf16_round_to_nearest_even():
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -9, 3.0e38], np.float32)
    bits = gen.f32_to_bf16_bits(vals)
    assert list(bits[:4]) == [0x3F80, 0x3F80, 0x3F82, 0xC020]
    assert bits[4] == 0x3F80
    back = gen.bf16_bits_to_f32(bits)
    assert np.all(np.abs(back - vals) <= np.abs(vals) * 2 ** -8)


def test_generator_is_reproducible_and_keyed():
    wl = CONFIGS["tiny_f32"]
    a = gen.layer_weights(wl, 0)
    b = gen.layer_weights(wl, 0)
    c = gen.layer_weights(wl, 1)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])
    assert not np.array_equal(a["wq"], c["wq"])
    assert abs(np.std(a["wq"]) - 0.02) < 0.002
    assert abs(np.mean(a["attn_norm"]) - 1.0) < 0.01


@pytest.mark.parametrize("name", ["llama8b_decode", "llama8b_think"])
def test_context_length_laws(name):
    wl = CONFIGS[name]
    L = gen.context_lengths(wl)
    assert len(L) == wl.decode_batch
    if wl.ctx_law == "uniform":
        assert L.min() >= 1024 and L.max() <= 4096
    else:
        assert L.min() >= 4096 and L.max() <= 32768
