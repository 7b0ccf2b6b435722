"""Stage-level parity of each libps kernel against the fp64 oracle (GPU).

Each stage is teacher-forced: the oracle evaluates the stage on exactly the
bf16 / fp32 values the device received, so the bound is the stage's own
rounding (|g - r| <= 2e-2 + 1e-2 |r| for bf16 outputs: a few bf16 ulps of the result),
except where a tighter deterministic bound exists (GEMM, bit-exact paging).
"""
import numpy as np
import pytest

from oracle import layer as O
from synth import gen
from synth.configs import CONFIGS, LayerShape
from tests import helpers as H

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2608_21719_amd import binding as B  # noqa: E402

S8 = CONFIGS["llama8b_decode"].shape
S70 = CONFIGS["llama70b_model"].shape
TINY = CONFIGS["tiny_f32"].shape


def rnd(shape, dtype, seed, std=1.0):
    a = np.random.default_rng(seed).standard_normal(shape).astype(np.float32) * np.float32(std)
    return gen.to_storage(a, dtype)


def sync():
    torch.cuda.synchronize()


# ------------------------------------------------------------------ RMSNorm
@pytest.mark.parametrize("xdt,ydt,d,rows", [("bf16", "bf16", 4096, 37), ("f32", "bf16", 4096, 5),
                                             ("f32", "f32", 256, 9), ("bf16", "bf16", 8192, 3),
                                             ("bf16", "bf16", 200, 4)])
def test_rmsnorm(xdt, ydt, d, rows):
    gdt = "f32" if xdt == "f32" and ydt == "f32" else "bf16"
    x = rnd((rows, d), xdt, 1)
    g = gen.to_storage(1 + 0.02 * np.random.default_rng(2).standard_normal(d).astype(np.float32), gdt)
    xd, gd = H.to_dev(x, xdt), H.to_dev(g, gdt)
    y = H.empty((rows, d), ydt)
    code = {"f32": B.PS_F32, "bf16": B.PS_BF16}
    B.op_rmsnorm(code[xdt], code[gdt], code[ydt], rows, d, xd, gd, 1e-5, y)
    sync()
    ref = O.rmsnorm(gen.widen(x, xdt), gen.widen(g, gdt), 1e-5)
    if ydt == "bf16":
        H.assert_close_elementwise(H.to_f64(y), ref, 1e-6, 2 ** -8 + 1e-5, "rmsnorm bf16")
    else:
        H.assert_close_elementwise(H.to_f64(y), ref, 1e-6, 1e-5, "rmsnorm f32")


# ------------------------------------------------------------------ GEMM
def gemm_bound(a, w, K, out_bf16):
    """|g - r| <= 2^-8 |r| (bf16 output) + 2 K 2^-24 sum_k |a_k w_k| + tiny."""
    mag = np.abs(a) @ np.abs(w).T
    return mag * (2 * K * 2.0 ** -24) + 1e-30, (2.0 ** -8 if out_bf16 else 0.0)


@pytest.mark.parametrize("M,N,K", [(300, 512, 448), (256, 256, 64), (520, 768, 1024),   # tile path
                                   (64, 256, 1024), (37, 192, 512), (1, 64, 256), (17, 320, 2048),  # skinny
                                   (64, 32768, 256), (33, 16384, 2048),  # skinny, two blocks per workgroup
                                   # skinny with 3, 5, 6, 7 K splits (one block) and 3 (two blocks); each K is a
                                   # stage count the split count does not divide, so the last split is longer
                                   (24, 4480, 3136), (64, 2880, 5184), (8, 2560, 6208), (50, 2304, 7232),
                                   (40, 10240, 3136)])
def test_gemm_store_bf16(M, N, K):
    a = rnd((M, K), "bf16", 3)
    w = rnd((N, K), "bf16", 4, 0.02)
    A, W = H.to_dev(a, "bf16"), H.to_dev_w(w, "bf16")
    C = H.empty((M, N), "bf16")
    ws = H.workspace(B.op_gemm_workspace_bytes(B.PS_BF16, M, N, K))
    B.op_gemm(B.PS_BF16, 0, B.PS_BF16, B.PS_EPI_STORE, M, N, K, A, W, None, C, ws)
    sync()
    af, wf = gen.widen(a, "bf16"), gen.widen(w, "bf16")
    ref = O.linear(af, wf)
    absb, relb = gemm_bound(af, wf, K, True)
    err = np.abs(H.to_f64(C) - ref)
    assert np.all(err <= absb + relb * np.abs(ref)), f"max err {err.max()}"


@pytest.mark.parametrize("M,N,K", [(300, 512, 448), (64, 256, 1024), (5, 128, 256), (64, 256, 4096), (64, 16384, 2048),
                                   (40, 20480, 128), (64, 2880, 5184)])
@pytest.mark.parametrize("rdt,cdt", [("bf16", "f32"), ("f32", "bf16")])
def test_gemm_residual(M, N, K, rdt, cdt):
    a = rnd((M, K), "bf16", 5)
    w = rnd((N, K), "bf16", 6, 0.02)
    r = rnd((M, N), rdt, 7)
    A, W, R = H.to_dev(a, "bf16"), H.to_dev_w(w, "bf16"), H.to_dev(r, rdt)
    C = H.empty((M, N), cdt)
    ws = H.workspace(B.op_gemm_workspace_bytes(B.PS_BF16, M, N, K))
    code = {"f32": B.PS_F32, "bf16": B.PS_BF16}
    B.op_gemm(B.PS_BF16, code[rdt], code[cdt], B.PS_EPI_RESIDUAL, M, N, K, A, W, R, C, ws)
    sync()
    af, wf = gen.widen(a, "bf16"), gen.widen(w, "bf16")
    ref = gen.widen(r, rdt) + O.linear(af, wf)
    absb, relb = gemm_bound(af, wf, K, cdt == "bf16")
    err = np.abs(H.to_f64(C) - ref)
    assert np.all(err <= absb + relb * np.abs(ref) + 1e-7 * np.abs(ref)), f"max err {err.max()}"


@pytest.mark.parametrize("M,F,K", [(300, 256, 448), (64, 192, 1024), (3, 64, 256), (64, 16384, 256), (20, 8192, 1024),
                                   (20, 8192, 2048), (20, 384, 2048)])
def test_gemm_swiglu(M, F, K):
    a = rnd((M, K), "bf16", 8)
    wg = rnd((F, K), "bf16", 9, 0.05)
    wu = rnd((F, K), "bf16", 10, 0.05)
    A = H.to_dev(a, "bf16")
    W = H.to_dev_w(B.pack_gate_up(wg, wu), "bf16")
    C = H.empty((M, F), "bf16")
    ws = H.workspace(B.op_gemm_workspace_bytes(B.PS_BF16, M, 2 * F, K))
    B.op_gemm(B.PS_BF16, 0, B.PS_BF16, B.PS_EPI_SWIGLU, M, 2 * F, K, A, W, None, C, ws)
    sync()
    af = gen.widen(a, "bf16")
    ref = O.silu(O.linear(af, gen.widen(wg, "bf16"))) * O.linear(af, gen.widen(wu, "bf16"))
    H.assert_close_elementwise(H.to_f64(C), ref, 1e-3, 2 ** -7, "swiglu")


@pytest.mark.parametrize("epi,N,K", [(0, 128, 256), (1, 128, 256), (2, 128, 256), (0, 100, 70), (1, 70, 130)])
@pytest.mark.parametrize("M", [512, 4, 70])
def test_gemm_f32(epi, N, K, M):
    a = rnd((M, K), "f32", 11)
    w = rnd((N, K), "f32", 12, 0.05)
    r = rnd((M, N), "f32", 13)
    wdev = B.pack_gate_up(w[:N // 2], w[N // 2:]) if epi == 2 else w
    A, W, R = H.to_dev(a, "f32"), H.to_dev_w(wdev, "f32"), H.to_dev(r, "f32")
    C = H.empty((M, N // 2 if epi == 2 else N), "f32")
    B.op_gemm(B.PS_F32, B.PS_F32, B.PS_F32, epi, M, N, K, A, W, R if epi == 1 else None, C)
    sync()
    af, wf = a.astype(np.float64), w.astype(np.float64)
    if epi == 2:
        ref = O.silu(O.linear(af, wf[:N // 2])) * O.linear(af, wf[N // 2:])
    else:
        ref = O.linear(af, wf) + (r if epi == 1 else 0)
    H.assert_close_elementwise(H.to_f64(C), ref, 1e-5, 1e-5, "gemm f32")


@pytest.mark.parametrize("dt,N,K", [("bf16", 192, 320), ("bf16", 100, 70), ("f32", 65, 129), ("f32", 1, 1)])
def test_op_tile_weight_matches_host_tiling(dt, N, K):
    """Device tiling is bit-identical to the host helper, padding included."""
    w = rnd((N, K), dt, 14)
    code = B.PS_BF16 if dt == "bf16" else B.PS_F32
    out = H.empty((B.tiled_weight_elems(N, K),), dt)
    out.fill_(1.0)  # padding must be written, not left over
    B.op_tile_weight(code, N, K, H.to_dev(w, dt), out)
    sync()
    np.testing.assert_array_equal(H.bits(out), H.bits(H.to_dev_w(w, dt)))


def test_gemm_rejects_unsupported_shape():
    A = H.empty((300, 100), "bf16")
    with pytest.raises(B.PsError) as e:
        B.op_gemm(B.PS_BF16, 0, B.PS_BF16, 0, 300, 100, 100, A, A, None, A)
    assert e.value.code == B.PS_E_UNSUPPORTED


# ------------------------------------------------------------------ paging
def host_scatter(raw_pool_bits, shape, n_pages, bt, length):
    """Read back K, V [length, n_kv, hd] from raw pool bits via the block table."""
    nkv, hd = shape.n_kv, shape.head_dim
    p = raw_pool_bits.reshape(n_pages, nkv, 2, 16, hd)  # K part [16][hd]; V^T part viewed as [16][hd] raw
    k = np.empty((length, nkv, hd), raw_pool_bits.dtype)
    v = np.empty((length, nkv, hd), raw_pool_bits.dtype)
    for t in range(length):
        page, slot = bt[t // 16], t % 16
        k[t] = p[page, :, 0, slot, :]
        vt = p[page, :, 1].reshape(nkv, hd, 16)   # V^T [hd][16]
        v[t] = vt[:, :, slot]
    return k, v


@pytest.mark.parametrize("dtype,shape", [("bf16", S8), ("f32", TINY)])
def test_kv_append_gather_bit_exact(dtype, shape):
    n_pages = 64
    P = H.Pool(shape, n_pages, 4, 32, seed=99)
    kv = P.kv
    lens = [1, 17, 40]
    seqs = [kv.open() for _ in lens]
    ws = H.workspace(1 << 20)
    ks, vs = [], []
    for i, (s, L) in enumerate(zip(seqs, lens)):
        kv.alloc(s, L)
        k, v = rnd((L, shape.n_kv, shape.head_dim), dtype, 20 + i), rnd((L, shape.n_kv, shape.head_dim), dtype, 30 + i)
        ks.append(k)
        vs.append(v)
    # two appends per sequence: first half, commit, rest
    first = [max(1, L // 2) for L in lens]
    rest = [L - f for L, f in zip(lens, first)]
    kk = np.concatenate([k[:f] for k, f in zip(ks, first)])
    vv = np.concatenate([v[:f] for v, f in zip(vs, first)])
    kv.append(0, seqs, first, H.to_dev(kk, dtype), H.to_dev(vv, dtype), ws)
    kv.commit(seqs, first)
    s2 = [s for s, r in zip(seqs, rest) if r > 0]
    r2 = [r for r in rest if r > 0]
    kk = np.concatenate([k[f:] for k, f, r in zip(ks, first, rest) if r > 0])
    vv = np.concatenate([v[f:] for v, f, r in zip(vs, first, rest) if r > 0])
    kv.append(0, s2, r2, H.to_dev(kk, dtype), H.to_dev(vv, dtype), ws)
    kv.commit(s2, r2)
    sync()
    view_dt = np.int16 if dtype == "bf16" else np.int32
    raw = P.mem.cpu().numpy().view(view_dt)
    for s, L, k, v in zip(seqs, lens, ks, vs):
        ko, vo = H.empty((L, shape.n_kv, shape.head_dim), dtype), H.empty((L, shape.n_kv, shape.head_dim), dtype)
        kv.gather(0, s, ko, vo, ws)
        sync()
        kb, vb = k.view(view_dt), v.view(view_dt)
        np.testing.assert_array_equal(H.bits(ko), kb)
        np.testing.assert_array_equal(H.bits(vo), vb)
        hk, hv = host_scatter(raw, shape, n_pages, kv.block_table(s), L)
        np.testing.assert_array_equal(hk, kb)
        np.testing.assert_array_equal(hv, vb)


def test_metadata_slots_reused_while_the_gpu_lags_on_two_streams():
    """Per-call metadata goes through a 4-slot pinned ring. Here the host runs far ahead of a busy GPU and
    alternates two streams, so every slot is rewritten many times while earlier uploads may still wait in
    a queue; each gather must still see its own sequence (length, block table)."""
    shape = S8
    P = H.Pool(shape, 256, 12, 64, seed=5)
    kv = P.kv
    lens = [1, 15, 16, 17, 33, 64, 100, 161, 250, 333]
    seqs = [kv.open() for _ in lens]
    ws0 = H.workspace(1 << 20)
    ks, vs = [], []
    for i, (s, L) in enumerate(zip(seqs, lens)):
        kv.alloc(s, L)
        k, v = rnd((L, shape.n_kv, shape.head_dim), "bf16", 60 + i), rnd((L, shape.n_kv, shape.head_dim), "bf16", 80 + i)
        kv.append(0, [s], [L], H.to_dev(k, "bf16"), H.to_dev(v, "bf16"), ws0)
        kv.commit([s], [L])
        ks.append(k)
        vs.append(v)
    calls = [(r, i) for r in range(3) for i in range(len(lens))]
    outs = [(H.empty((lens[i], shape.n_kv, shape.head_dim), "bf16"),
             H.empty((lens[i], shape.n_kv, shape.head_dim), "bf16"), H.workspace(1 << 16)) for _, i in calls]
    busy = torch.randn(6144, 6144, device="cuda")
    sync()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for st in streams:
        with torch.cuda.stream(st):
            for _ in range(2):
                busy @ busy  # keeps the queue busy while the host enqueues every gather
    for c, ((_, i), (ko, vo, ws)) in enumerate(zip(calls, outs)):
        kv.gather(0, seqs[i], ko, vo, ws, stream=streams[c % 2])
    sync()
    for (_, i), (ko, vo, _) in zip(calls, outs):
        np.testing.assert_array_equal(H.bits(ko), ks[i].view(np.int16))
        np.testing.assert_array_equal(H.bits(vo), vs[i].view(np.int16))


# ------------------------------------------------------------------ RoPE
@pytest.mark.parametrize("dtype,shape", [("bf16", S8), ("f32", TINY)])
def test_rope_kvwrite(dtype, shape):
    P = H.Pool(shape, 128, 4, 64, seed=5)
    kv = P.kv
    # the last sequence starts at row 64 and position 32: rows 64..95 are two
    # 16-row groups that each fill one page (the bf16 kernel's 16-byte V path);
    # the other groups straddle sequences or pages (its 2-byte V path)
    hist = [0, 5, 300, 32]
    new = [7, 16, 41, 40]
    seqs = [kv.open() for _ in hist]
    ws = H.workspace(1 << 20)
    for s, L, n in zip(seqs, hist, new):
        kv.alloc(s, L + n)
    hs = [s for s, L in zip(seqs, hist) if L]
    hl = [L for L in hist if L]
    kh = rnd((sum(hl), shape.n_kv, shape.head_dim), dtype, 40)
    kv.append(0, hs, hl, H.to_dev(kh, dtype), H.to_dev(kh, dtype), ws)
    kv.commit(hs, hl)
    rows = sum(new)
    dqkv = (shape.n_q + 2 * shape.n_kv) * shape.head_dim
    qkv = rnd((rows, dqkv), dtype, 41)
    q_out = H.empty((rows, shape.d_q), dtype)
    B.op_rope_kvwrite(kv, 0, seqs, new, H.to_dev(qkv, dtype), q_out, ws)
    kv.commit(seqs, new)
    sync()
    qf = gen.widen(qkv, dtype)
    pos = np.concatenate([np.arange(L, L + n) for L, n in zip(hist, new)])
    q_ref = O.rope(qf[:, :shape.d_q].reshape(rows, shape.n_q, shape.head_dim), pos, shape.theta)
    k_ref = O.rope(qf[:, shape.d_q:shape.d_q + shape.d_kv].reshape(rows, shape.n_kv, shape.head_dim), pos,
                   shape.theta)
    v_ref = qkv[:, shape.d_q + shape.d_kv:].reshape(rows, shape.n_kv, shape.head_dim)
    tol = (1e-6, 2 ** -8 + 1e-5) if dtype == "bf16" else (1e-6, 1e-5)
    H.assert_close_elementwise(H.to_f64(q_out).reshape(q_ref.shape), q_ref, *tol, "rope q")
    r0 = 0
    for s, L, n in zip(seqs, hist, new):
        ko = H.empty((L + n, shape.n_kv, shape.head_dim), dtype)
        vo = H.empty((L + n, shape.n_kv, shape.head_dim), dtype)
        kv.gather(0, s, ko, vo, ws)
        sync()
        H.assert_close_elementwise(H.to_f64(ko)[L:], k_ref[r0:r0 + n], *tol, "rope k")
        np.testing.assert_array_equal(H.bits(vo)[L:], v_ref[r0:r0 + n].view(np.int16 if dtype == "bf16" else np.int32))
        r0 += n


# ------------------------------------------------------------------ attention
def fill_kv(P, lens_hist, n_new, dtype, seed, ones_v=False):
    """Open sequences, write history (committed) and new rows (uncommitted)."""
    kv, shape = P.kv, P.shape
    seqs = [kv.open() for _ in lens_hist]
    ws = H.workspace(1 << 22)
    Ks, Vs = [], []
    for i, (s, L, n) in enumerate(zip(seqs, lens_hist, n_new)):
        kv.alloc(s, L + n)
        k = rnd((L + n, shape.n_kv, shape.head_dim), dtype, seed + 2 * i)
        v = rnd((L + n, shape.n_kv, shape.head_dim), dtype, seed + 2 * i + 1)
        if ones_v:
            v = gen.to_storage(np.ones((L + n, shape.n_kv, shape.head_dim), np.float32), dtype)
        Ks.append(k)
        Vs.append(v)
        if L:
            kv.append(0, [s], [L], H.to_dev(k[:L], dtype), H.to_dev(v[:L], dtype), ws)
            kv.commit([s], [L])
        kv.append(0, [s], [n], H.to_dev(k[L:], dtype), H.to_dev(v[L:], dtype), ws)
    return seqs, Ks, Vs


def make_pool(shape, n_pages, max_seqs, max_pages, seed):
    return H.Pool(shape, n_pages, max_seqs, max_pages, seed=seed)


DEC_LENS = [0, 14, 15, 16, 17, 100, 1000, 2500]


@pytest.mark.parametrize("shape", [S8, S70], ids=["G4", "G8"])
@pytest.mark.parametrize("split", [0, 1, 3, 8, 20, 33, 64])
def test_decode_attention(shape, split):
    """split_pages >= 20 puts more than 16 pages in each wave's range of the
    longest sequences (157 pages), so the steady-state page ring runs; 0 is
    the library's choice (at least 8 pages per split)."""
    P = make_pool(shape, 600, 8, 200, seed=77)
    seqs, Ks, Vs = fill_kv(P, DEC_LENS, [1] * len(DEC_LENS), "bf16", 100)
    q = rnd((len(seqs), shape.n_q, shape.head_dim), "bf16", 50)
    o = H.empty((len(seqs), shape.d_q), "bf16")
    ws = H.workspace(1 << 24)
    B.op_decode_attention(P.kv, 0, seqs, H.to_dev(q, "bf16"), o, ws, split_pages=split)
    sync()
    got = H.to_f64(o).reshape(len(seqs), shape.n_q, shape.head_dim)
    qf = gen.widen(q, "bf16")
    for b, L in enumerate(DEC_LENS):
        ref = O.attention(qf[b:b + 1], gen.widen(Ks[b], "bf16"), gen.widen(Vs[b], "bf16"), np.array([L]))
        H.assert_close_elementwise(got[b], ref[0], H.BF16_TOL_ABS, H.BF16_TOL_REL, f"decode b={b} L={L}")


def test_decode_attention_paged_equals_contiguous_and_deterministic():
    shape = S8
    outs = []
    for seed in (0, 4242):
        P = make_pool(shape, 700, 8, 200, seed=seed)
        seqs, _, _ = fill_kv(P, DEC_LENS, [1] * len(DEC_LENS), "bf16", 100)
        q = rnd((len(seqs), shape.n_q, shape.head_dim), "bf16", 50)
        qd = H.to_dev(q, "bf16")
        ws = H.workspace(1 << 24)
        for _ in range(2):
            o = H.empty((len(seqs), shape.d_q), "bf16")
            B.op_decode_attention(P.kv, 0, seqs, qd, o, ws)
            sync()
            outs.append(H.bits(o))
    for x in outs[1:]:
        np.testing.assert_array_equal(x, outs[0])


def test_decode_attention_ones_v_gives_exactly_one():
    P = make_pool(S8, 600, 8, 200, seed=3)
    seqs, _, _ = fill_kv(P, DEC_LENS, [1] * len(DEC_LENS), "bf16", 200, ones_v=True)
    q = rnd((len(seqs), S8.n_q, S8.head_dim), "bf16", 51, 3.0)
    o = H.empty((len(seqs), S8.d_q), "bf16")
    B.op_decode_attention(P.kv, 0, seqs, H.to_dev(q, "bf16"), o, H.workspace(1 << 24))
    sync()
    assert np.all(H.to_f64(o) == 1.0)


def library_split_pages(page_counts, n_kv):
    """The library's documented split choice, restated: the smallest multiple
    of 4 pages, at least 8, whose splits times KV heads stay within 1024
    workgroups (one split per sequence when none does)."""
    target = max(1, 1024 // max(1, n_kv))
    n_items = lambda sp: sum(-(-p // sp) for p in page_counts)
    sp = max(-(-sum(page_counts) // target), 8)
    sp = -(-sp // 4) * 4
    while n_items(sp) > target and sp < max(page_counts):
        sp += 4
    return sp


@pytest.mark.parametrize("n_seqs,hist,expect", [(100, 130, 12), (16, 2000, 16)], ids=["search", "direct"])
def test_decode_library_split_choice(n_seqs, hist, expect):
    """split_pages = 0 gives the same bits as the split the documented rule
    names, and other bits than a split 4 pages smaller (the split fixes the
    merge's rounding order, so the comparison tells splits apart). 100
    sequences of 9 pages: 8 pages per split would make 200 items for 128
    slots, so the rule moves on to 12; 16 sequences of 126 pages: 16 directly."""
    shape = S8
    pages = [-(-(hist + 1) // 16)] * n_seqs
    sp = library_split_pages(pages, shape.n_kv)
    assert sp == expect
    P = make_pool(shape, sum(pages) + 16, n_seqs, max(pages) + 2, seed=31)
    seqs, _, _ = fill_kv(P, [hist] * n_seqs, [1] * n_seqs, "bf16", 300)
    q = H.to_dev(rnd((n_seqs, shape.n_q, shape.head_dim), "bf16", 53), "bf16")
    ws = H.workspace(1 << 26)
    outs = {}
    for split in (0, sp, sp - 4):
        o = H.empty((n_seqs, shape.d_q), "bf16")
        B.op_decode_attention(P.kv, 0, seqs, q, o, ws, split_pages=split)
        sync()
        outs[split] = H.bits(o)
    np.testing.assert_array_equal(outs[0], outs[sp])
    assert np.any(outs[sp - 4] != outs[sp])


def test_decode_plan_run_matches_one_call_and_detects_pool_change():
    """Plan once, run for two layers: bit-identical to the one-call op; a
    commit invalidates the plan."""
    shape = S8
    P = H.Pool(shape, 700, 8, 200, n_layers=2, seed=9)
    seqs, _, _ = fill_kv(P, DEC_LENS, [1] * len(DEC_LENS), "bf16", 100)
    q = H.to_dev(rnd((len(seqs), shape.n_q, shape.head_dim), "bf16", 52), "bf16")
    ws = H.workspace(1 << 24)
    ref = H.empty((len(seqs), shape.d_q), "bf16")
    B.op_decode_attention(P.kv, 0, seqs, q, ref, ws)
    B.op_decode_plan(P.kv, seqs, ws)
    outs = []
    for layer in (0, 1, 0):
        o = H.empty((len(seqs), shape.d_q), "bf16")
        B.op_decode_run(P.kv, layer, q, o, ws)
        outs.append(o)
    sync()
    np.testing.assert_array_equal(H.bits(outs[0]), H.bits(ref))
    np.testing.assert_array_equal(H.bits(outs[2]), H.bits(ref))
    P.kv.commit([seqs[0]], [1])
    with pytest.raises(B.PsError) as e:
        B.op_decode_run(P.kv, 0, q, H.empty((len(seqs), shape.d_q), "bf16"), ws)
    assert e.value.code == B.PS_E_INVALID


PRE_HIST = [0, 0, 16, 31, 100, 0]
PRE_NEW = [1, 63, 64, 65, 200, 130]


@pytest.mark.parametrize("shape", [S8, S70], ids=["G4", "G8"])
def test_prefill_attention(shape):
    P = make_pool(shape, 200, 8, 40, seed=11)
    seqs, Ks, Vs = fill_kv(P, PRE_HIST, PRE_NEW, "bf16", 300)
    rows = sum(PRE_NEW)
    q = rnd((rows, shape.n_q, shape.head_dim), "bf16", 60)
    o = H.empty((rows, shape.d_q), "bf16")
    B.op_attention(P.kv, 0, seqs, PRE_NEW, H.to_dev(q, "bf16"), o, H.workspace(1 << 22))
    sync()
    got = H.to_f64(o).reshape(rows, shape.n_q, shape.head_dim)
    qf = gen.widen(q, "bf16")
    r0 = 0
    for b, (L, n) in enumerate(zip(PRE_HIST, PRE_NEW)):
        ref = O.attention(qf[r0:r0 + n], gen.widen(Ks[b], "bf16"), gen.widen(Vs[b], "bf16"), np.arange(L, L + n))
        H.assert_close_elementwise(got[r0:r0 + n], ref, H.BF16_TOL_ABS, H.BF16_TOL_REL, f"prefill b={b}")
        r0 += n


@pytest.mark.parametrize("shape", [S8, S70], ids=["G4", "G8"])
def test_prefill_attention_late_score_jumps(shape):
    """Keys scaled by 8 to 48 in later key tiles lift some query rows' scores
    tens to hundreds of log2 units above the exponent base the first tile
    set, so P overflows the kernel's 2^32 row-sum check (or fp32 itself) and
    the tile is redone against the new row max, several times per row and
    in tiles that also hold ordinary keys. Random inputs only ever take that
    path on the first tile."""
    hist, new = [0, 300], [200, 65]
    planted = {0: {70: 12.0, 140: 24.0, 199: 48.0}, 1: {200: 16.0, 330: 32.0, 364: 8.0}}
    P = make_pool(shape, 200, 8, 40, seed=13)
    kv = P.kv
    seqs = [kv.open() for _ in hist]
    ws = H.workspace(1 << 22)
    Ks, Vs = [], []
    for i, (sq, L, n) in enumerate(zip(seqs, hist, new)):
        kv.alloc(sq, L + n)
        k = gen.widen(rnd((L + n, shape.n_kv, shape.head_dim), "bf16", 900 + 2 * i), "bf16")
        for key, a in planted[i].items():
            k[key] *= a
        k = gen.to_storage(k.astype(np.float32), "bf16")
        v = rnd((L + n, shape.n_kv, shape.head_dim), "bf16", 901 + 2 * i)
        Ks.append(k)
        Vs.append(v)
        if L:
            kv.append(0, [sq], [L], H.to_dev(k[:L], "bf16"), H.to_dev(v[:L], "bf16"), ws)
            kv.commit([sq], [L])
        kv.append(0, [sq], [n], H.to_dev(k[L:], "bf16"), H.to_dev(v[L:], "bf16"), ws)
    rows = sum(new)
    q = rnd((rows, shape.n_q, shape.head_dim), "bf16", 62)
    o = H.empty((rows, shape.d_q), "bf16")
    B.op_attention(kv, 0, seqs, new, H.to_dev(q, "bf16"), o, ws)
    sync()
    got = H.to_f64(o).reshape(rows, shape.n_q, shape.head_dim)
    assert np.all(np.isfinite(got))
    qf = gen.widen(q, "bf16")
    r0 = 0
    for b, (L, n) in enumerate(zip(hist, new)):
        ref = O.attention(qf[r0:r0 + n], gen.widen(Ks[b], "bf16"), gen.widen(Vs[b], "bf16"), np.arange(L, L + n))
        H.assert_close_elementwise(got[r0:r0 + n], ref, H.BF16_TOL_ABS, H.BF16_TOL_REL, f"score jumps b={b}")
        r0 += n
    # the planted keys do move the base: rows of the first sequence whose max
    # in later tiles exceeds the first tile's by more than 32 log2 units
    G = shape.n_q // shape.n_kv
    s0 = np.einsum("ihd,jhd->hij", qf[:new[0]], np.repeat(gen.widen(Ks[0], "bf16"), G, axis=1))
    s0 = s0 * (np.log2(np.e) / np.sqrt(shape.head_dim))
    causal = np.tril(np.ones((new[0], new[0]), bool))
    s0 = np.where(causal, s0, -np.inf)
    jumps = s0.max(axis=2) - s0[:, :, :32].max(axis=2)
    assert np.count_nonzero(jumps > 32) > 100


def test_prefill_attention_ones_v_and_paging_invariance():
    outs = {}
    for seed, ones in ((0, False), (999, False), (5, True)):
        P = make_pool(S8, 200, 8, 40, seed=seed)
        seqs, _, _ = fill_kv(P, PRE_HIST, PRE_NEW, "bf16", 400, ones_v=ones)
        rows = sum(PRE_NEW)
        q = rnd((rows, S8.n_q, S8.head_dim), "bf16", 61, 3.0)
        o = H.empty((rows, S8.d_q), "bf16")
        B.op_attention(P.kv, 0, seqs, PRE_NEW, H.to_dev(q, "bf16"), o, H.workspace(1 << 22))
        sync()
        outs[(seed, ones)] = o
    np.testing.assert_array_equal(H.bits(outs[(0, False)]), H.bits(outs[(999, False)]))
    assert np.all(H.to_f64(outs[(5, True)]) == 1.0)


def test_prefill_attention_long_prefix_33000_tokens():
    """A 33-row chunk after a 33000-token prefix: a key walk of more than 2000
    pages (1030 key tiles, each page id a scalar load one tile ahead and each
    page's K/V a DMA through its own buffer resource); a short second sequence
    shares the launch."""
    hist, new = [33000, 0], [33, 40]
    P = make_pool(S8, 2100, 2, 2090, seed=21)
    seqs, Ks, Vs = fill_kv(P, hist, new, "bf16", 700)
    rows = sum(new)
    q = rnd((rows, S8.n_q, S8.head_dim), "bf16", 63)
    o = H.empty((rows, S8.d_q), "bf16")
    B.op_attention(P.kv, 0, seqs, new, H.to_dev(q, "bf16"), o, H.workspace(1 << 22))
    sync()
    got = H.to_f64(o).reshape(rows, S8.n_q, S8.head_dim)
    qf = gen.widen(q, "bf16")
    r0 = 0
    for b, (L, n) in enumerate(zip(hist, new)):
        ref = O.attention(qf[r0:r0 + n], gen.widen(Ks[b], "bf16"), gen.widen(Vs[b], "bf16"), np.arange(L, L + n))
        H.assert_close_elementwise(got[r0:r0 + n], ref, H.BF16_TOL_ABS, H.BF16_TOL_REL, f"long prefix b={b}")
        r0 += n


@pytest.mark.parametrize("hist,new", [([0, 3], [5, 1]), ([130, 0], [1, 40])])
def test_attention_f32(hist, new):
    shape = TINY
    P = make_pool(shape, 64, 4, 16, seed=8)
    seqs, Ks, Vs = fill_kv(P, hist, new, "f32", 500)
    rows = sum(new)
    q = rnd((rows, shape.n_q, shape.head_dim), "f32", 62)
    o = H.empty((rows, shape.d_q), "f32")
    B.op_attention(P.kv, 0, seqs, new, H.to_dev(q, "f32"), o, H.workspace(1 << 20))
    sync()
    got = H.to_f64(o).reshape(rows, shape.n_q, shape.head_dim)
    r0 = 0
    for b, (L, n) in enumerate(zip(hist, new)):
        ref = O.attention(q[r0:r0 + n].astype(np.float64), Ks[b].astype(np.float64), Vs[b].astype(np.float64),
                          np.arange(L, L + n))
        H.assert_close_elementwise(got[r0:r0 + n], ref, 1e-5, 1e-5, "attn f32")
        r0 += n
