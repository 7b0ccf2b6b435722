"""End-to-end layer parity against the fp64 oracle (GPU).

fp32 layer: elementwise |g - r| <= 1e-4 + 1e-4 |r|. bf16 layers: normwise
max|g - r| / max|r| <= 1e-2 and rms(g - r) / rms(r) <= 1e-2 (the oracle
rounds nowhere; bf16 rounding of GEMM inputs alone gives ~5e-3).
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


class Harness:
    def __init__(self, wl, n_pages, max_seqs, max_pages, seed=None, max_rows=1024):
        self.wl = wl
        self.shape = wl.shape
        self.dt = wl.shape.dtype
        self.w = gen.layer_weights(wl, 0)
        self.wf = H.weights_f64(self.w, self.dt)
        self.dev = H.DeviceLayer(self.w, self.dt)
        self.pool = H.Pool(self.shape, n_pages, max_seqs, max_pages,
                           seed=gen.page_order_seed(wl) if seed is None else seed)
        self.kv = self.pool.kv
        self.layer = B.Layer(self.pool.cfg)
        self.ws = H.workspace(B.Layer.workspace_bytes(self.pool.cfg, max_rows, max_seqs, max_pages))
        self.hist = {}  # oracle-side K, V per sequence

    def open(self, reserve):
        s = self.kv.open()
        self.kv.alloc(s, reserve)
        sh = self.shape
        self.hist[s] = (np.zeros((0, sh.n_kv, sh.head_dim)), np.zeros((0, sh.n_kv, sh.head_dim)))
        return s

    def oracle(self, s, x_rows):
        kh, vh = self.hist[s]
        r = O.layer_sequence(self.wf, self.shape, x_rows, kh, vh)
        self.hist[s] = (np.concatenate([kh, r["k"]]), np.concatenate([vh, r["v"]]))
        return r["out"]

    def prefill(self, seqs, n_tok, x):
        out = H.empty((x.shape[0], self.shape.hidden), self.dt)
        self.layer.prefill(self.dev.w, self.kv, 0, seqs, n_tok, H.to_dev(x, self.dt), out, self.ws)
        self.kv.commit(seqs, n_tok)
        sync()
        return H.to_f64(out)

    def decode(self, seqs, x, phase=B.PS_PHASE_ANSWER):
        out = H.empty((x.shape[0], self.shape.hidden), self.dt)
        self.layer.decode_step(self.dev.w, self.kv, 0, phase, seqs, H.to_dev(x, self.dt), out, self.ws)
        self.kv.commit(seqs, [1] * len(seqs))
        sync()
        return H.to_f64(out)


def check(got, ref, dt, what):
    if dt == "f32":
        H.assert_close_elementwise(got, ref, H.F32_TOL_ABS, H.F32_TOL_REL, what)
    else:
        mx, rms = H.normwise(got, ref)
        assert mx <= H.NORMWISE_TOL and rms <= H.NORMWISE_TOL, f"{what}: normwise max {mx:.2e} rms {rms:.2e}"


def test_tiny_fp32_prefill_then_16_decode_steps():
    """The tiny fp32 workload in full: 4 x 128 prefill, 16 decode steps, shuffled pages."""
    wl = CONFIGS["tiny_f32"]
    h = Harness(wl, n_pages=64, max_seqs=4, max_pages=16)
    T, B_ = wl.prefill_tokens, wl.prefill_seqs
    seqs = [h.open(T + wl.decode_steps) for _ in range(B_)]
    x = gen.prefill_input(wl, T * B_)
    got = h.prefill(seqs, [T] * B_, x)
    xf = gen.widen(x, "f32")
    for i, s in enumerate(seqs):
        check(got[i * T:(i + 1) * T], h.oracle(s, xf[i * T:(i + 1) * T]), "f32", f"prefill seq {i}")
    for step in range(wl.decode_steps):
        xd = gen.decode_input(wl, B_, step)
        got = h.decode(seqs, xd)
        xdf = gen.widen(xd, "f32")
        ref = np.concatenate([h.oracle(s, xdf[i:i + 1]) for i, s in enumerate(seqs)])
        check(got, ref, "f32", f"decode step {step}")


@pytest.fixture(scope="module")
def h8():
    return Harness(CONFIGS["llama8b_prefill"], n_pages=512, max_seqs=16, max_pages=64)


def test_8b_layer_prefill_then_decode(h8):
    h = h8
    lens = [100, 37, 64]
    seqs = [h.open(L + 3) for L in lens]
    x = gen.prefill_input(h.wl, sum(lens), step=1)
    got = h.prefill(seqs, lens, x)
    xf = gen.widen(x, "bf16")
    r0 = 0
    for s, L in zip(seqs, lens):
        check(got[r0:r0 + L], h.oracle(s, xf[r0:r0 + L]), "bf16", f"prefill L={L}")
        r0 += L
    for step in range(3):
        xd = gen.decode_input(h.wl, len(seqs), 10 + step)
        got = h.decode(seqs, xd, B.PS_PHASE_THINK)
        xdf = gen.widen(xd, "bf16")
        ref = np.concatenate([h.oracle(s, xdf[i:i + 1]) for i, s in enumerate(seqs)])
        check(got, ref, "bf16", f"decode step {step}")
    for s in seqs:
        h.kv.free(s)


def test_8b_decode_equals_last_row_of_prefill(h8):
    """Two kernels paths, same inputs: prefill of T+1 rows vs prefill T + decode 1."""
    h = h8
    T = 70
    x = gen.prefill_input(h.wl, T + 1, step=2)
    a = h.open(T + 1)
    b = h.open(T + 1)
    full = h.prefill([a], [T + 1], x)
    h.prefill([b], [T], x[:T])
    dec = h.decode([b], x[T:T + 1])
    # end to end, each path is bf16-rounded at several points: normwise bound,
    # against the oracle and against each other
    ref = O.layer_sequence(h.wf, h.shape, gen.widen(x, "bf16"))["out"][T]
    check(dec[0], ref, "bf16", "decode row vs oracle")
    check(full[T], ref, "bf16", "prefill row vs oracle")
    check(dec[0], full[T], "bf16", "decode row vs prefill row")
    # stage level: the K/V both paths wrote at position T (QKV GEMM on the
    # tile vs skinny kernel, same RoPE) agree to one bf16 rounding
    sh = h.shape
    kv_out = {}
    for s in (a, b):
        k = H.empty((T + 1, sh.n_kv, sh.head_dim), "bf16")
        v = H.empty((T + 1, sh.n_kv, sh.head_dim), "bf16")
        h.kv.gather(0, s, k, v, h.ws)
        sync()
        kv_out[s] = (H.to_f64(k)[T], H.to_f64(v)[T])
    for i in range(2):
        H.assert_close_elementwise(kv_out[b][i], kv_out[a][i], H.BF16_TOL_ABS, H.BF16_TOL_REL, "K/V at T")
    for s in (a, b):
        h.kv.free(s)


def test_8b_mixed_step_matches_oracle(h8):
    """Chunked prefill (fresh and with a cached prefix) fused with decodes."""
    h = h8
    c_new = h.open(48)
    c_pre = h.open(20 + 33)
    d1 = h.open(90)
    d2 = h.open(20)
    xp = gen.prefill_input(h.wl, 20 + 80 + 17, step=3)
    xpf = gen.widen(xp, "bf16")
    h.prefill([c_pre, d1, d2], [20, 80, 17], xp)
    for s, (r0, n) in zip([c_pre, d1, d2], [(0, 20), (20, 80), (100, 17)]):
        h.oracle(s, xpf[r0:r0 + n])
    xm = gen.mixed_input(h.wl, 48 + 33 + 2)
    xmf = gen.widen(xm, "bf16")
    out = H.empty((83, h.shape.hidden), "bf16")
    h.layer.mixed_step(h.dev.w, h.kv, 0, [c_new, c_pre], [48, 33], [d1, d2], H.to_dev(xm, "bf16"), out, h.ws)
    h.kv.commit([c_new, c_pre, d1, d2], [48, 33, 1, 1])
    sync()
    got = H.to_f64(out)
    check(got[:48], h.oracle(c_new, xmf[:48]), "bf16", "mixed chunk fresh")
    check(got[48:81], h.oracle(c_pre, xmf[48:81]), "bf16", "mixed chunk with prefix")
    check(got[81:82], h.oracle(d1, xmf[81:82]), "bf16", "mixed decode 1")
    check(got[82:83], h.oracle(d2, xmf[82:83]), "bf16", "mixed decode 2")
    for s in (c_new, c_pre, d1, d2):
        h.kv.free(s)


@pytest.mark.parametrize("n_chunk,n_dec", [(40, 3), (70, 65)])
def test_8b_unforked_mixed_step_matches_oracle(n_chunk, n_dec):
    """Mixed steps that do not fork: 40 chunk rows (every stage on the
    caller's stream over all rows, decode-sized GEMMs), and more than 64
    decode rows beside 70 chunk rows (tile GEMMs over all rows)."""
    h = Harness(CONFIGS["llama8b_prefill"], n_pages=400, max_seqs=80, max_pages=16, max_rows=4096)
    lens = [20 + i for i in range(n_dec)]
    c = h.open(n_chunk)
    decs = [h.open(L + 1) for L in lens]
    xp = gen.prefill_input(h.wl, sum(lens), step=11 + n_dec)
    xpf = gen.widen(xp, "bf16")
    h.prefill(decs, lens, xp)
    checked = (0, n_dec - 1)
    r0 = 0
    for i, (s, L) in enumerate(zip(decs, lens)):
        if i in checked:
            h.oracle(s, xpf[r0:r0 + L])
        r0 += L
    xm = gen.mixed_input(h.wl, n_chunk + n_dec, layer=n_dec)
    xmf = gen.widen(xm, "bf16")
    out = H.empty((n_chunk + n_dec, h.shape.hidden), "bf16")
    h.layer.mixed_step(h.dev.w, h.kv, 0, [c], [n_chunk], decs, H.to_dev(xm, "bf16"), out, h.ws)
    sync()
    got = H.to_f64(out)
    check(got[:n_chunk], h.oracle(c, xmf[:n_chunk]), "bf16", f"unforked chunk ({n_chunk} + {n_dec})")
    for i in checked:
        ref = h.oracle(decs[i], xmf[n_chunk + i:n_chunk + i + 1])
        check(got[n_chunk + i:n_chunk + i + 1], ref, "bf16", f"unforked decode {i} ({n_chunk} + {n_dec})")


def test_8b_forked_mixed_step_chunk_rows_equal_prefill_bit_for_bit(h8):
    """The forked mixed step (more than 64 chunk rows beside decode rows: the
    decode rows' attention, O, SwiGLU and down on the second stream, their
    attention on a capped grid) against ps_prefill of the same chunks on a
    second pool with the same history: the chunk rows take the same kernels
    and plans either way, so their output and written K/V must match bit for
    bit, whatever the decode rows do beside them on the other stream."""
    h = h8
    sh = h.shape
    chunks = [(0, 150), (37, 96)]   # (cached prefix, chunk rows)
    decs = [700, 1500, 90]          # decode rows' history lengths
    hist = [p for p, _ in chunks] + decs
    pools = [H.Pool(sh, sum((L + 160) // 16 for L in hist) + 8, 8, 128, seed=5 + i) for i in range(2)]
    ws = [H.workspace(B.Layer.workspace_bytes(p.cfg, 512, 8, 128)) for p in pools]
    g = torch.Generator(device="cuda").manual_seed(77)
    kvh = [(torch.randn((L, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16),
            torch.randn((L, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)) for L in hist]
    seqs = []
    for p, w in zip(pools, ws):
        ss = []
        for (pre, n), (k, v) in zip(chunks, kvh):
            s = p.kv.open()
            p.kv.alloc(s, pre + n)
            if pre:
                p.kv.append(0, [s], [pre], k, v, w)
                p.kv.commit([s], [pre])
            ss.append(s)
        for L, (k, v) in zip(decs, kvh[len(chunks):]):
            s = p.kv.open()
            p.kv.alloc(s, L + 1)
            p.kv.append(0, [s], [L], k, v, w)
            p.kv.commit([s], [L])
            ss.append(s)
        seqs.append(ss)
    n_chunk = sum(n for _, n in chunks)
    xm = gen.mixed_input(h.wl, n_chunk + len(decs))
    x = H.to_dev(xm, "bf16")
    a, b = pools
    out_m = H.empty((n_chunk + len(decs), sh.hidden), "bf16")
    h.layer.mixed_step(h.dev.w, a.kv, 0, seqs[0][:2], [n for _, n in chunks], seqs[0][2:], x, out_m, ws[0])
    out_p = H.empty((n_chunk, sh.hidden), "bf16")
    h.layer.prefill(h.dev.w, b.kv, 0, seqs[1][:2], [n for _, n in chunks], x[:n_chunk].contiguous(), out_p, ws[1])
    sync()
    assert torch.equal(out_m[:n_chunk].view(torch.int16), out_p.view(torch.int16)), "chunk rows differ"
    for (pre, n), sa, sb in zip(chunks, seqs[0][:2], seqs[1][:2]):
        a.kv.commit([sa], [n])
        b.kv.commit([sb], [n])
        ka = torch.empty((pre + n, sh.n_kv, sh.head_dim), dtype=torch.bfloat16, device="cuda")
        va, kb, vb = torch.empty_like(ka), torch.empty_like(ka), torch.empty_like(ka)
        a.kv.gather(0, sa, ka, va, ws[0])
        b.kv.gather(0, sb, kb, vb, ws[1])
        sync()
        assert torch.equal(ka.view(torch.int16), kb.view(torch.int16)), "written K differs"
        assert torch.equal(va.view(torch.int16), vb.view(torch.int16)), "written V differs"


def test_layer_rejects_capacity_overrun_without_launching(h8):
    h = h8
    s = h.open(16)
    x = gen.prefill_input(h.wl, 17)
    with pytest.raises(B.PsError) as e:
        h.prefill([s], [17], x)
    assert e.value.code == B.PS_E_CAPACITY
    assert h.kv.seq_len(s) == 0
    h.kv.free(s)


@pytest.mark.parametrize("batch", [64, 37])
def test_8b_decode_step_equals_composed_stage_ops_bit_for_bit(h8, batch):
    """ps_decode_step against the same stages called one by one through the
    single-op entry points (norm, QKV GEMM, RoPE + KV write, split-K
    attention, O GEMM + residual, norm, gate_up + SwiGLU, down + residual) on
    a second pool holding the same history: the layer's fused kernels must
    reproduce the composed path exactly, output and written K/V."""
    h = h8
    sh, wl = h.shape, h.wl
    d, dq, dkv, F = sh.hidden, sh.n_q * sh.head_dim, sh.n_kv * sh.head_dim, sh.ffn
    ctx = [40 + (37 * i) % 160 for i in range(batch)]
    pools = [H.Pool(sh, sum((c + 16) // 16 for c in ctx) + 8, batch, 16, seed=11) for _ in range(2)]
    ws = H.workspace(B.Layer.workspace_bytes(pools[0].cfg, 64, batch, 16))
    g = torch.Generator(device="cuda").manual_seed(123)
    seqs = [[], []]
    for c in ctx:
        k = torch.randn((c, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        v = torch.randn((c, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        for p, ss in zip(pools, seqs):
            s = p.kv.open()
            p.kv.alloc(s, c + 1)
            p.kv.append(0, [s], [c], k, v, ws)
            p.kv.commit([s], [c])
            ss.append(s)
    x = H.to_dev(gen.decode_input(wl, batch, 3), "bf16")
    out_layer = H.empty((batch, d), "bf16")
    h.layer.decode_step(h.dev.w, pools[0].kv, 0, B.PS_PHASE_ANSWER, seqs[0], x, out_layer, ws)
    sync()
    t = h.dev.t
    bf, f32 = B.PS_BF16, B.PS_F32
    xn = H.empty((batch, d), "bf16")
    qkv = H.empty((batch, dq + 2 * dkv), "bf16")
    q = H.empty((batch, dq), "bf16")
    o = H.empty((batch, dq), "bf16")
    hh = H.empty((batch, d), "f32")
    hn = H.empty((batch, d), "bf16")
    m = H.empty((batch, F), "bf16")
    out_ops = H.empty((batch, d), "bf16")
    kv2 = pools[1].kv
    B.op_rmsnorm(bf, bf, bf, batch, d, x, t["attn_norm"], sh.eps, xn)
    B.op_gemm(bf, 0, bf, B.PS_EPI_STORE, batch, dq + 2 * dkv, d, xn, t["w_qkv"], None, qkv, ws)
    B.op_rope_kvwrite(kv2, 0, seqs[1], [1] * batch, qkv, q, ws)
    B.op_decode_attention(kv2, 0, seqs[1], q, o, ws)
    B.op_gemm(bf, bf, f32, B.PS_EPI_RESIDUAL, batch, d, dq, o, t["w_o"], x, hh, ws)
    B.op_rmsnorm(f32, bf, bf, batch, d, hh, t["ffn_norm"], sh.eps, hn)
    B.op_gemm(bf, 0, bf, B.PS_EPI_SWIGLU, batch, 2 * F, d, hn, t["w_gate_up"], None, m, ws)
    B.op_gemm(bf, f32, bf, B.PS_EPI_RESIDUAL, batch, d, F, m, t["w_down"], hh, out_ops, ws)
    sync()
    np.testing.assert_array_equal(H.bits(out_layer), H.bits(out_ops))
    for p, ss in zip(pools, seqs):
        p.kv.commit(ss, [1] * batch)
    for i in (0, batch // 2, batch - 1):  # the K/V row each path wrote at position ctx
        got = []
        for p, ss in zip(pools, seqs):
            k = H.empty((ctx[i] + 1, sh.n_kv, sh.head_dim), "bf16")
            v = H.empty((ctx[i] + 1, sh.n_kv, sh.head_dim), "bf16")
            p.kv.gather(0, ss[i], k, v, ws)
            got.append((k[-1], v[-1]))
        sync()
        np.testing.assert_array_equal(H.bits(got[0][0]), H.bits(got[1][0]))
        np.testing.assert_array_equal(H.bits(got[0][1]), H.bits(got[1][1]))


def test_admitted_mixed_batch_matches_oracle():
    """A batch formed by the admission scheduler (per-stage chunk reservation
    by observed lengths): two requests admitted and prefilled earlier decode
    while two newly admitted prompts run as chunk rows of one mixed step,
    after the scheduler reserved the step's growth. The scheduler decides and
    reserves on the host; the layer runs on the GPU against the oracle."""
    wl = CONFIGS["llama8b_think"]
    h = Harness(wl, n_pages=200, max_seqs=8, max_pages=64, seed=4242)
    sched = B.Sched(h.kv, 4, 256, 64, 1024)
    sh = h.shape
    first = [sched.admit(L) for L in (100, 37)]
    assert None not in first and sched.chunk_size() == 256
    for s, L in zip(first, (100, 37)):
        assert h.kv.capacity(s) >= L + 256
        h.hist[s] = (np.zeros((0, sh.n_kv, sh.head_dim)), np.zeros((0, sh.n_kv, sh.head_dim)))
    xp = gen.prefill_input(wl, 137, step=5)
    h.prefill(first, [100, 37], xp)
    xpf = gen.widen(xp, "bf16")
    h.oracle(first[0], xpf[:100])
    h.oracle(first[1], xpf[100:137])
    # a completion elsewhere in the stage moves CS_i before the next admissions
    done = sched.admit(0)
    sched.finish(done, 90)
    assert sched.chunk_size() == 96
    new = [sched.admit(L) for L in (64, 48)]
    assert None not in new
    for s in new:
        h.hist[s] = (np.zeros((0, sh.n_kv, sh.head_dim)), np.zeros((0, sh.n_kv, sh.head_dim)))
    assert sched.reserve_step(first, [1, 1], 8) == []
    xm = gen.mixed_input(wl, 64 + 48 + 2)
    xmf = gen.widen(xm, "bf16")
    out = H.empty((114, sh.hidden), "bf16")
    h.layer.mixed_step(h.dev.w, h.kv, 0, new, [64, 48], first, H.to_dev(xm, "bf16"), out, h.ws)
    h.kv.commit(new + first, [64, 48, 1, 1])
    sync()
    got = H.to_f64(out)
    check(got[:64], h.oracle(new[0], xmf[:64]), "bf16", "admitted chunk 0")
    check(got[64:112], h.oracle(new[1], xmf[64:112]), "bf16", "admitted chunk 1")
    check(got[112:113], h.oracle(first[0], xmf[112:113]), "bf16", "running decode 0")
    check(got[113:114], h.oracle(first[1], xmf[113:114]), "bf16", "running decode 1")
    for s, n in zip(first + new, (1, 1, 64, 48)):
        sched.finish(s, n)
    assert sched.running() == 0 and h.kv.free_pages() == 200
