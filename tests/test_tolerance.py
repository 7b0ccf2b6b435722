"""Where the end-to-end bf16 bounds come from (CPU).

The device rounds to bf16 at fixed points of the layer (GEMM inputs, q/k/v,
P, o, m, the layer output); the oracle rounds nowhere. A float32 model with
bf16 rounding at exactly those points (tests/bf16_emulation.py) gives the
error floor of any such pipeline on the same inputs. Each end-to-end bound in
tests/helpers.py is that floor times a stated margin; these tests recompute
the floor from the oracle's own inputs and check the bound against it.
"""
import numpy as np
import pytest

from oracle import layer as O
from synth import gen
from synth.configs import CONFIGS
from tests import bf16_emulation as E
from tests import helpers as H


def _floor(wl, n_prompt, n_decode=0, ctx=0):
    """Normwise (max, rms) error of the rounding model against the oracle on a
    prompt of n_prompt rows and on n_decode decode rows after ctx history
    tokens; the worst of the cases."""
    sh = wl.shape
    w = gen.layer_weights(wl, 0)
    w32 = E.WidenedWeights(w, np.float32)
    w64 = E.WidenedWeights(w, np.float64)
    worst = [0.0, 0.0]
    x = gen.widen(gen.prefill_input(wl, n_prompt), "bf16").astype(np.float32)
    ref = O.layer_sequence(w64, sh, x.astype(np.float64))["out"]
    for i, e in enumerate(H.normwise(E.layer(w32, sh, x).astype(np.float64), ref)):
        worst[i] = max(worst[i], e)
    xd = gen.widen(gen.decode_input(wl, n_decode, 0), "bf16").astype(np.float32)
    for b in range(n_decode):
        kh, vh = (gen.bf16_bits_to_f32(a) for a in gen.kv_history(wl, 0, b, ctx))
        ref = O.layer_sequence(w64, sh, xd[b:b + 1].astype(np.float64), kh.astype(np.float64),
                               vh.astype(np.float64))["out"]
        got = E.layer(w32, sh, xd[b:b + 1], kh, vh).astype(np.float64)
        for i, e in enumerate(H.normwise(got, ref)):
            worst[i] = max(worst[i], e)
    return tuple(worst)


def test_rounding_model_matches_the_oracle_in_fp32_terms():
    """Sanity of the model itself: with no rounding its result would equal the
    oracle to fp32 accuracy; with rounding, the error is a few bf16 ulps."""
    wl = CONFIGS["llama8b_prefill"]
    sh = wl.shape
    small = type(sh)(256, 4, 2, 64, 512, sh.eps, sh.theta, "bf16")
    wls = type(wl)("t", 40, small)
    w = gen.layer_weights(wls, 0)
    w32 = E.weights_f32(w)
    x = gen.widen(gen.prefill_input(wls, 40), "bf16").astype(np.float32)
    ref = O.layer_sequence({k: v.astype(np.float64) for k, v in w32.items()}, small, x.astype(np.float64))["out"]
    mx, rms = H.normwise(E.layer(w32, small, x).astype(np.float64), ref)
    assert 1e-4 < rms < 1e-2 and mx < 2e-2
    # the lazily widened weights give the same bits as eager widening
    lazy = E.layer(E.WidenedWeights(w, np.float32), small, x)
    np.testing.assert_array_equal(lazy, E.layer(w32, small, x))
    r64 = O.layer_sequence(E.WidenedWeights(w, np.float64), small, x.astype(np.float64))["out"]
    np.testing.assert_array_equal(r64, ref)


def test_8b_bound_has_margin_over_the_rounding_floor():
    mx, rms = _floor(CONFIGS["llama8b_prefill"], 256, n_decode=2, ctx=2048)
    floor = max(mx, rms)
    print(f"8B floor: normwise max {mx:.3e} rms {rms:.3e}")
    assert floor * H.TOL_MARGIN <= H.NORMWISE_TOL, floor


def test_70b_bound_is_the_rounding_floor_times_the_margin():
    """At d = 8192, F = 28672 the FFN branch dominates the output and carries
    the rounding of m, so the floor sits near 1e-2 and the 8B bound cannot
    hold; the 70B bound is this floor times the margin."""
    mx, rms = _floor(CONFIGS["llama70b_model"], 256, n_decode=2, ctx=4096)
    floor = max(mx, rms)
    print(f"70B floor: normwise max {mx:.3e} rms {rms:.3e}")
    assert abs(floor - H.NORMWISE_FLOOR_70B) <= 0.03 * H.NORMWISE_FLOOR_70B, floor
    assert floor * H.TOL_MARGIN <= H.NORMWISE_TOL_70B <= floor * H.TOL_MARGIN * 1.05
