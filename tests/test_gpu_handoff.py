"""Think -> answer handoff between two KV pools on one GPU (ps_kv_transfer).

A reasoning request thinks in one pool and answers in another (the paper's
prefill / think / answer pipeline moves its KV state once, think to answer).
Here both pools sit on one GPU with different sizes and page orders. After
the transfer, every layer's K/V reads back bit-identical from both pools, and
the next decode step run in the answer pool equals, bit for bit, the same
step continued in the think pool: output rows and the K/V rows it writes.
The step is also checked against the fp64 oracle, so the equality is not
between two wrong results.
"""
import numpy as np
import pytest

from oracle import layer as O
from synth import gen
from synth.configs import CONFIGS
from tests import helpers as H

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2608_21719_amd import binding as B  # noqa: E402


def sync():
    torch.cuda.synchronize()


def test_think_to_answer_transfer_then_decode_is_bit_identical():
    wl = CONFIGS["llama8b_think"]
    sh = wl.shape
    L = 2
    w = [gen.layer_weights(wl, l) for l in range(L)]
    wf = [H.weights_f64(x, "bf16") for x in w]
    dev = [H.DeviceLayer(x, "bf16") for x in w]
    think = H.Pool(sh, 96, 6, 16, n_layers=L, seed=101)
    answer = H.Pool(sh, 70, 6, 16, n_layers=L, seed=9999)  # other size, other page order
    layer = B.Layer(think.cfg)
    ws = H.workspace(B.Layer.workspace_bytes(think.cfg, 256, 6, 16))
    lens = [100, 37, 64]
    seqs = [think.kv.open() for _ in lens]
    for s, n in zip(seqs, lens):
        think.kv.alloc(s, n + 8)
    # prefill through both layers (layer l's output feeds layer l + 1), then three think steps
    x = gen.prefill_input(wl, sum(lens))
    xl = H.to_dev(x, "bf16")
    for l in range(L):
        y = H.empty((sum(lens), sh.hidden), "bf16")
        layer.prefill(dev[l].w, think.kv, l, seqs, lens, xl, y, ws)
        xl = y
    think.kv.commit(seqs, lens)
    for step in range(3):
        xd = H.to_dev(gen.decode_input(wl, len(seqs), step), "bf16")
        for l in range(L):
            y = H.empty((len(seqs), sh.hidden), "bf16")
            layer.decode_step(dev[l].w, think.kv, l, B.PS_PHASE_THINK, seqs, xd, y, ws)
            xd = y
        think.kv.commit(seqs, [1] * len(seqs))
    sync()
    moved = seqs[1:]
    new = []
    for s in moved:
        d = answer.kv.open()
        answer.kv.alloc(d, think.kv.seq_len(s) + 4)  # the answer stage's reservation
        B.kv_transfer(think.kv, s, answer.kv, d, ws)
        new.append(d)
    sync()
    assert [answer.kv.seq_len(d) for d in new] == [think.kv.seq_len(s) for s in moved]
    assert think.kv.block_table(moved[0])[:3] != answer.kv.block_table(new[0])[:3]
    for l in range(L):
        for s, d in zip(moved, new):
            n = think.kv.seq_len(s)
            k0, v0 = H.empty((n, sh.n_kv, sh.head_dim), "bf16"), H.empty((n, sh.n_kv, sh.head_dim), "bf16")
            k1, v1 = H.empty((n, sh.n_kv, sh.head_dim), "bf16"), H.empty((n, sh.n_kv, sh.head_dim), "bf16")
            think.kv.gather(l, s, k0, v0, ws)
            answer.kv.gather(l, d, k1, v1, ws)
            sync()
            assert torch.equal(k0.view(torch.int16), k1.view(torch.int16))
            assert torch.equal(v0.view(torch.int16), v1.view(torch.int16))
    # the next step: answer pool vs the think pool continuing (layer 0)
    x = gen.decode_input(wl, len(moved), 7)
    out_t, out_a = H.empty((len(moved), sh.hidden), "bf16"), H.empty((len(moved), sh.hidden), "bf16")
    layer.decode_step(dev[0].w, think.kv, 0, B.PS_PHASE_THINK, moved, H.to_dev(x, "bf16"), out_t, ws)
    layer.decode_step(dev[0].w, answer.kv, 0, B.PS_PHASE_ANSWER, new, H.to_dev(x, "bf16"), out_a, ws)
    think.kv.commit(moved, [1] * len(moved))
    answer.kv.commit(new, [1] * len(new))
    sync()
    assert torch.equal(out_t.view(torch.int16), out_a.view(torch.int16))
    for s, d in zip(moved, new):
        n = think.kv.seq_len(s)
        k0, v0 = H.empty((n, sh.n_kv, sh.head_dim), "bf16"), H.empty((n, sh.n_kv, sh.head_dim), "bf16")
        k1, v1 = H.empty((n, sh.n_kv, sh.head_dim), "bf16"), H.empty((n, sh.n_kv, sh.head_dim), "bf16")
        think.kv.gather(0, s, k0, v0, ws)
        answer.kv.gather(0, d, k1, v1, ws)
        sync()
        assert torch.equal(k0.view(torch.int16), k1.view(torch.int16))
        assert torch.equal(v0.view(torch.int16), v1.view(torch.int16))
        # and the oracle: this step over the sequence's own cached K/V (read back from the pool)
        i = moved.index(s)
        ref = O.layer_sequence(wf[0], sh, gen.widen(x, "bf16")[i:i + 1], H.to_f64(k0)[:n - 1],
                               H.to_f64(v0)[:n - 1])["out"][0]
        mx, rms = H.normwise(H.to_f64(out_a)[i], ref)
        assert mx <= H.NORMWISE_TOL and rms <= H.NORMWISE_TOL, (mx, rms)


def test_transfer_of_an_empty_sequence_and_into_the_same_pool():
    sh = CONFIGS["llama8b_think"].shape
    P = H.Pool(sh, 32, 4, 8, seed=5)
    ws = H.workspace(1 << 16)
    a = P.kv.open()
    b = P.kv.open()
    P.kv.alloc(b, 16)
    B.kv_transfer(P.kv, a, P.kv, b, ws)      # nothing to copy: length 0 stays 0
    assert P.kv.seq_len(b) == 0
    P.kv.alloc(a, 20)
    k = torch.randn((20, sh.n_kv, sh.head_dim), device="cuda").to(torch.bfloat16)
    v = torch.randn((20, sh.n_kv, sh.head_dim), device="cuda").to(torch.bfloat16)
    P.kv.append(0, [a], [20], k, v, ws)
    P.kv.commit([a], [20])
    c = P.kv.open()
    P.kv.alloc(c, 20)
    B.kv_transfer(P.kv, a, P.kv, c, ws)      # a copy inside one pool
    ko, vo = H.empty((20, sh.n_kv, sh.head_dim), "bf16"), H.empty((20, sh.n_kv, sh.head_dim), "bf16")
    P.kv.gather(0, c, ko, vo, ws)
    sync()
    assert torch.equal(ko.view(torch.int16), k.view(torch.int16))
    assert torch.equal(vo.view(torch.int16), v.view(torch.int16))
