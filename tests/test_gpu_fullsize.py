"""Parity at the benchmarked sizes, on sampled outputs (GPU).

The layer runs exactly as bench.py times it (8B shape: 8 x 2048 prefill;
decode batch 64 over U{1024..4096} contexts; think decode batch 32 over
log-normal contexts up to 32k plus the fused mixed step. 70B shape, one layer
of the 80-layer model's step: decode batch 64 at context 4096 and the
8 x 1024 prefill). The fp64 oracle then evaluates a sample
of sequences in full (every row of a sampled prefill sequence; the decode row
of sampled decode sequences over their whole history) and the outputs are
compared with the end-to-end normwise bound (the 70B shape's bound is its bf16 rounding floor times the
margin; see tests/test_tolerance.py). Synthetic KV history is drawn by
a seeded torch generator, copied to the host by torch, and written with
ps_kv_append: the oracle's inputs never pass through the library's kernels.
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


@pytest.fixture(scope="module")
def layer8b():
    wl = CONFIGS["llama8b_prefill"]
    w = gen.layer_weights(wl, 0)
    return {"wl": wl, "wf": H.weights_f64(w, "bf16"), "dev": H.DeviceLayer(w, "bf16")}


@pytest.fixture(scope="module")
def layer70b():
    wl = CONFIGS["llama70b_model"]
    w = gen.layer_weights(wl, 0)
    return {"wl": wl, "wf": H.weights_f64(w, "bf16"), "dev": H.DeviceLayer(w, "bf16"), "tol": H.NORMWISE_TOL_70B}


def normwise_ok(got, ref, what, tol=H.NORMWISE_TOL):
    mx, rms = H.normwise(got, ref)
    assert mx <= tol and rms <= tol, f"{what}: normwise max {mx:.2e} rms {rms:.2e} (bound {tol:.2e})"


def test_prefill_8x2048_sampled_sequences(layer8b):
    wl, sh = layer8b["wl"], layer8b["wl"].shape
    n, T = wl.prefill_seqs, wl.prefill_tokens
    pool = H.Pool(sh, n * T // 16 + 8, n, T // 16, seed=gen.page_order_seed(wl))
    layer = B.Layer(pool.cfg)
    seqs = [pool.kv.open() for _ in range(n)]
    for s in seqs:
        pool.kv.alloc(s, T)
    ws = H.workspace(B.Layer.workspace_bytes(pool.cfg, n * T, n, T // 16))
    x = gen.prefill_input(wl, n * T)
    out = H.empty((n * T, sh.hidden), "bf16")
    layer.prefill(layer8b["dev"].w, pool.kv, 0, seqs, [T] * n, H.to_dev(x, "bf16"), out, ws)
    sync()
    got = H.to_f64(out)
    xf = gen.widen(x, "bf16")
    for b in (0, n - 1):
        ref = O.layer_sequence(layer8b["wf"], sh, xf[b * T:(b + 1) * T])["out"]
        normwise_ok(got[b * T:(b + 1) * T], ref, f"prefill seq {b}")
        # and the first and last rows on their own
        normwise_ok(got[b * T], ref[0], f"seq {b} row 0")
        normwise_ok(got[(b + 1) * T - 1], ref[-1], f"seq {b} row {T - 1}")
    # the last row of every prompt (it attends over the whole prompt)
    for b in range(1, n - 1):
        ref = O.layer_rows(layer8b["wf"], sh, xf[b * T:(b + 1) * T], [T - 1])[0]
        normwise_ok(got[(b + 1) * T - 1], ref, f"seq {b} row {T - 1}")


def test_prefill_5x416_three_way_k_split(layer8b):
    """2080 prefill rows: nine 256-row tile rows, so the down GEMM's 144
    tiles are split three ways in K (432 workgroups, two rounds instead of
    one at full K) and summed with the residual by the reduce kernel. The
    last prompt is compared in full, every other prompt on its last row."""
    wl, sh = layer8b["wl"], layer8b["wl"].shape
    n, T = 5, 416
    pool = H.Pool(sh, n * T // 16 + 8, n, T // 16, seed=gen.page_order_seed(wl))
    layer = B.Layer(pool.cfg)
    seqs = [pool.kv.open() for _ in range(n)]
    for s in seqs:
        pool.kv.alloc(s, T)
    ws = H.workspace(B.Layer.workspace_bytes(pool.cfg, n * T, n, T // 16))
    x = gen.prefill_input(wl, n * T)
    out = H.empty((n * T, sh.hidden), "bf16")
    layer.prefill(layer8b["dev"].w, pool.kv, 0, seqs, [T] * n, H.to_dev(x, "bf16"), out, ws)
    sync()
    got = H.to_f64(out)
    xf = gen.widen(x, "bf16")
    ref = O.layer_sequence(layer8b["wf"], sh, xf[(n - 1) * T:])["out"]
    normwise_ok(got[(n - 1) * T:], ref, f"prefill seq {n - 1}")
    for b in range(n - 1):
        r = O.layer_rows(layer8b["wf"], sh, xf[b * T:(b + 1) * T], [T - 1])[0]
        normwise_ok(got[(b + 1) * T - 1], r, f"seq {b} row {T - 1}")


def _decode_fullsize(layer8b, wl, sample, phase, mixed=False):
    sh = wl.shape
    ctx = [int(c) for c in gen.context_lengths(wl)]
    nb = len(ctx)
    chunk, nc = wl.mixed_chunk, wl.mixed_new
    max_pages = (max(max(ctx) + 1, chunk) + 15) // 16
    n_pages = sum((c + 16) // 16 for c in ctx) + nc * ((chunk + 15) // 16) + 8
    pool = H.Pool(sh, n_pages, nb + nc, max_pages, seed=gen.page_order_seed(wl))
    kv = pool.kv
    layer = B.Layer(pool.cfg)
    rows = nb + (nc * chunk if mixed else 0)
    ws = H.workspace(B.Layer.workspace_bytes(pool.cfg, max(rows, 64), nb + nc, max_pages))
    g = torch.Generator(device="cuda").manual_seed(wl.cfg_id * 1000 + 7)
    seqs = [kv.open() for _ in range(nb)]
    hist = {}
    for b, (s, c) in enumerate(zip(seqs, ctx)):
        kv.alloc(s, c + 1)
        k = torch.randn((c, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        v = torch.randn((c, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        kv.append(0, [s], [c], k, v, ws)
        kv.commit([s], [c])
        if b in sample:
            hist[b] = (H.to_f64(k), H.to_f64(v))
        del k, v
    sync()
    xd = gen.decode_input(wl, nb, 0)
    new = []
    if mixed:
        new = [kv.open() for _ in range(nc)]
        for s in new:
            kv.alloc(s, chunk)
        xc = gen.mixed_input(wl, nc * chunk)
        x = np.concatenate([xc, xd])
        out = H.empty((rows, sh.hidden), "bf16")
        layer.mixed_step(layer8b["dev"].w, kv, 0, new, [chunk] * nc, seqs, H.to_dev(x, "bf16"), out, ws)
    else:
        x = xd
        out = H.empty((nb, sh.hidden), "bf16")
        layer.decode_step(layer8b["dev"].w, kv, 0, phase, seqs, H.to_dev(x, "bf16"), out, ws)
    sync()
    got = H.to_f64(out)
    xf = gen.widen(x, "bf16")
    off = nc * chunk if mixed else 0
    tol = layer8b.get("tol", H.NORMWISE_TOL)
    for b in sample:
        ref = O.layer_sequence(layer8b["wf"], sh, xf[off + b:off + b + 1], *hist[b])["out"][0]
        normwise_ok(got[off + b], ref, f"decode seq {b} ctx {ctx[b]}", tol)
    if mixed:
        # every chunk: together they span every tile row of the chunk rows'
        # K-split O and down launches
        for i in range(nc):
            ref = O.layer_sequence(layer8b["wf"], sh, xf[i * chunk:(i + 1) * chunk])["out"]
            normwise_ok(got[i * chunk:(i + 1) * chunk], ref, f"mixed chunk {i}")
    return ctx


def test_decode_batch64_sampled_sequences(layer8b):
    ctx = _decode_fullsize(layer8b, CONFIGS["llama8b_decode"], sample=[0, 17, 63], phase=B.PS_PHASE_ANSWER)
    assert min(ctx) >= 1024 and max(ctx) <= 4096


def test_decode_batch64_four_steps_sampled_sequences(layer8b):
    """Four consecutive decode steps of the B = 64 benchmark batch (fresh
    inputs each step): every step writes its token's K/V and the next step
    reads it back. Sampled sequences include one whose length crosses a
    16-token page boundary during the four steps; each step's rows are
    compared with the oracle's layer over the history plus the steps so far
    (one sequence, causal)."""
    wl = CONFIGS["llama8b_decode"]
    sh = wl.shape
    steps = 4
    ctx = [int(c) for c in gen.context_lengths(wl)]
    nb = len(ctx)
    crossing = next(b for b, c in enumerate(ctx) if c % 16 >= 16 - steps + 1)
    sample = sorted({0, crossing, nb - 1})
    max_pages = (max(ctx) + steps + 15) // 16
    n_pages = sum((c + steps + 15) // 16 for c in ctx) + 8
    pool = H.Pool(sh, n_pages, nb, max_pages, seed=gen.page_order_seed(wl))
    kv = pool.kv
    layer = B.Layer(pool.cfg)
    ws = H.workspace(B.Layer.workspace_bytes(pool.cfg, 64, nb, max_pages))
    g = torch.Generator(device="cuda").manual_seed(wl.cfg_id * 1000 + 11)
    seqs = [kv.open() for _ in range(nb)]
    hist = {}
    for b, (sq, c) in enumerate(zip(seqs, ctx)):
        kv.alloc(sq, c + steps)
        k = torch.randn((c, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        v = torch.randn((c, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        kv.append(0, [sq], [c], k, v, ws)
        kv.commit([sq], [c])
        if b in sample:
            hist[b] = (H.to_f64(k), H.to_f64(v))
        del k, v
    xs, outs = [], []
    for t in range(steps):
        x = gen.decode_input(wl, nb, t)
        out = H.empty((nb, sh.hidden), "bf16")
        layer.decode_step(layer8b["dev"].w, kv, 0, B.PS_PHASE_ANSWER, seqs, H.to_dev(x, "bf16"), out, ws)
        kv.commit(seqs, [1] * nb)
        xs.append(gen.widen(x, "bf16"))
        outs.append(out)
    sync()
    assert [kv.seq_len(sq) for sq in seqs] == [c + steps for c in ctx]
    for b in sample:
        rows = np.stack([xs[t][b] for t in range(steps)])
        ref = O.layer_sequence(layer8b["wf"], sh, rows, *hist[b])["out"]
        for t in range(steps):
            normwise_ok(H.to_f64(outs[t])[b], ref[t], f"decode seq {b} ctx {ctx[b]} step {t}")


def test_think_batch32_long_context_sampled_sequences(layer8b):
    wl = CONFIGS["llama8b_think"]
    ctx = [int(c) for c in gen.context_lengths(wl)]
    longest = int(np.argmax(ctx))
    _decode_fullsize(layer8b, wl, sample=sorted({0, longest}), phase=B.PS_PHASE_THINK)


def test_think_mixed_step_sampled(layer8b):
    _decode_fullsize(layer8b, CONFIGS["llama8b_think"], sample=[1, 31], phase=B.PS_PHASE_THINK, mixed=True)


# ------------------------------------------------------------- 70B shape
def test_70b_decode_batch64_ctx4096_sampled_sequences(layer70b):
    """One 70B-shaped layer of the model's decode step as bench.py runs it:
    64 sequences at context 4096 (four 16-row blocks in the skinny GEMMs,
    G = 8 decode attention)."""
    ctx = _decode_fullsize(layer70b, layer70b["wl"], sample=[0, 31, 63], phase=B.PS_PHASE_ANSWER)
    assert ctx == [4096] * 64


def test_70b_prefill_8x1024_sampled(layer70b):
    """The 70B model's 8 x 1024 prefill through one layer: the last prompt in
    full, and the first rows of the first prompt."""
    wl = layer70b["wl"]
    sh, n, T = wl.shape, wl.prefill_seqs, wl.prefill_tokens
    pool = H.Pool(sh, n * T // 16 + 8, n, T // 16, seed=gen.page_order_seed(wl))
    layer = B.Layer(pool.cfg)
    seqs = [pool.kv.open() for _ in range(n)]
    for s in seqs:
        pool.kv.alloc(s, T)
    ws = H.workspace(B.Layer.workspace_bytes(pool.cfg, n * T, n, T // 16))
    x = gen.prefill_input(wl, n * T)
    out = H.empty((n * T, sh.hidden), "bf16")
    layer.prefill(layer70b["dev"].w, pool.kv, 0, seqs, [T] * n, H.to_dev(x, "bf16"), out, ws)
    sync()
    got = H.to_f64(out)
    xf = gen.widen(x, "bf16")
    tol = layer70b["tol"]
    b = n - 1
    ref = O.layer_sequence(layer70b["wf"], sh, xf[b * T:(b + 1) * T])["out"]
    normwise_ok(got[b * T:(b + 1) * T], ref, f"prefill seq {b}", tol)
    normwise_ok(got[(b + 1) * T - 1], ref[-1], f"seq {b} row {T - 1}", tol)
    ref0 = O.layer_sequence(layer70b["wf"], sh, xf[0:2])["out"]  # causal: a prompt's first rows on their own
    normwise_ok(got[0:2], ref0, "prefill seq 0 rows 0-1", tol)
    for b in range(n - 1):  # the last row of every other prompt
        ref = O.layer_rows(layer70b["wf"], sh, xf[b * T:(b + 1) * T], [T - 1])[0]
        normwise_ok(got[(b + 1) * T - 1], ref, f"seq {b} row {T - 1}", tol)


def test_70b_ragged_decode_and_short_prefill(layer70b):
    """Ragged contexts (4096, 4095, 3000, 17) in one decode step, and a
    256-token prompt, at the 70B shape."""
    wl = layer70b["wl"]
    sh = wl.shape
    ctx = [4096, 4095, 3000, 17]
    pool = H.Pool(sh, sum((c + 16) // 16 for c in ctx) + 32, 8, 260, seed=5)
    kv = pool.kv
    layer = B.Layer(pool.cfg)
    ws = H.workspace(B.Layer.workspace_bytes(pool.cfg, 256, 8, 260))
    g = torch.Generator(device="cuda").manual_seed(99)
    seqs, hist = [], []
    for c in ctx:
        s = kv.open()
        kv.alloc(s, c + 1)
        k = torch.randn((c, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        v = torch.randn((c, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        kv.append(0, [s], [c], k, v, ws)
        kv.commit([s], [c])
        seqs.append(s)
        hist.append((H.to_f64(k), H.to_f64(v)))
    x = gen.decode_input(wl, len(ctx), 0)
    out = H.empty((len(ctx), sh.hidden), "bf16")
    layer.decode_step(layer70b["dev"].w, kv, 0, B.PS_PHASE_ANSWER, seqs, H.to_dev(x, "bf16"), out, ws)
    sync()
    got = H.to_f64(out)
    xf = gen.widen(x, "bf16")
    for b in range(len(ctx)):
        ref = O.layer_sequence(layer70b["wf"], sh, xf[b:b + 1], *hist[b])["out"][0]
        normwise_ok(got[b], ref, f"decode b={b} ctx {ctx[b]}", layer70b["tol"])
    p = kv.open()
    kv.alloc(p, 256)
    xp = gen.prefill_input(wl, 256)
    outp = H.empty((256, sh.hidden), "bf16")
    layer.prefill(layer70b["dev"].w, kv, 0, [p], [256], H.to_dev(xp, "bf16"), outp, ws)
    sync()
    ref = O.layer_sequence(layer70b["wf"], sh, gen.widen(xp, "bf16"))["out"]
    normwise_ok(H.to_f64(outp), ref, "prefill 256", layer70b["tol"])


def test_70b_forked_mixed_step(layer70b):
    """A forked mixed step at the 70B shape (G = 8: two flash workgroups per KV
    head, the capped decode attention over 8 KV heads): a 200-row chunk after
    a 3000-token cached prefix beside four decode rows. The chunk rows and the
    K/V they write equal ps_prefill of the same chunk on a second pool with
    the same history, bit for bit; the decode rows and the chunk's first and
    last rows match the oracle."""
    wl = layer70b["wl"]
    sh = wl.shape
    pre, n = 3000, 200
    decs = [4096, 2000, 17, 900]
    hist_len = [pre] + decs
    pools = [H.Pool(sh, sum((L + 216) // 16 for L in hist_len) + 8, 8, 260, seed=31 + i) for i in range(2)]
    ws = [H.workspace(B.Layer.workspace_bytes(p.cfg, 256, 8, 260)) for p in pools]
    layers = [B.Layer(p.cfg) for p in pools]
    g = torch.Generator(device="cuda").manual_seed(2024)
    kvh = [(torch.randn((L, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16),
            torch.randn((L, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)) for L in hist_len]
    seqs = []
    for p, w in zip(pools, ws):
        ss = []
        for i, (L, (k, v)) in enumerate(zip(hist_len, kvh)):
            s = p.kv.open()
            p.kv.alloc(s, L + (n if i == 0 else 1))
            p.kv.append(0, [s], [L], k, v, w)
            p.kv.commit([s], [L])
            ss.append(s)
        seqs.append(ss)
    xm = gen.mixed_input(wl, n + len(decs))
    x = H.to_dev(xm, "bf16")
    out_m = H.empty((n + len(decs), sh.hidden), "bf16")
    layers[0].mixed_step(layer70b["dev"].w, pools[0].kv, 0, seqs[0][:1], [n], seqs[0][1:], x, out_m, ws[0])
    out_p = H.empty((n, sh.hidden), "bf16")
    layers[1].prefill(layer70b["dev"].w, pools[1].kv, 0, seqs[1][:1], [n], x[:n].contiguous(), out_p, ws[1])
    sync()
    assert torch.equal(out_m[:n].view(torch.int16), out_p.view(torch.int16)), "chunk rows differ from ps_prefill"
    pools[0].kv.commit(seqs[0][:1], [n])
    pools[1].kv.commit(seqs[1][:1], [n])
    ka = torch.empty((pre + n, sh.n_kv, sh.head_dim), dtype=torch.bfloat16, device="cuda")
    va, kb, vb = torch.empty_like(ka), torch.empty_like(ka), torch.empty_like(ka)
    pools[0].kv.gather(0, seqs[0][0], ka, va, ws[0])
    pools[1].kv.gather(0, seqs[1][0], kb, vb, ws[1])
    sync()
    assert torch.equal(ka.view(torch.int16), kb.view(torch.int16)), "written K differs"
    assert torch.equal(va.view(torch.int16), vb.view(torch.int16)), "written V differs"
    got = H.to_f64(out_m)
    xf = gen.widen(xm, "bf16")
    kf, vf = H.to_f64(kvh[0][0]), H.to_f64(kvh[0][1])
    ref = O.layer_rows(layer70b["wf"], sh, xf[:n], [0, n - 1], kf, vf)
    normwise_ok(got[0], ref[0], "chunk row 0", layer70b["tol"])
    normwise_ok(got[n - 1], ref[1], f"chunk row {n - 1}", layer70b["tol"])
    for b, L in enumerate(decs):
        kd, vd = H.to_f64(kvh[1 + b][0]), H.to_f64(kvh[1 + b][1])
        ref = O.layer_sequence(layer70b["wf"], sh, xf[n + b:n + b + 1], kd, vd)["out"][0]
        normwise_ok(got[n + b], ref, f"decode row {b} ctx {L}", layer70b["tol"])
