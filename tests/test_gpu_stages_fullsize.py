"""Stage-level parity at the benchmarked launches (GPU).

Each kernel runs with exactly the launch configuration the benchmark and the
layer use (the library's own decode split plan; the tile GEMM's full grid
with its XCD remap and tile-row grouping; the skinny GEMM's plans at the
decode batch), and is compared element by element with the fp64 oracle
evaluated on the device's own inputs.

Decode attention, per workload (the plan aims at about 1024 workgroups, so
splits hold 44-80 pages at the 8B decode batch, 129-219 in the think phase and
129 at the 70B shape: every wave runs the kernel's steady-state page ring):
  * random K, V ~ N(0, 1) and q ~ N(0, 2^2) (peaked softmax): every head and
    dim of at least 8 sequences (shortest and longest included) against
    oracle.attention at the stage bound |g - r| <= 2e-2 + 1e-2 |r|;
  * a page census over every sequence: q = 0 makes every visible key weigh
    the same, and V marks each key's page (dimension d of KV head h is 1 for
    the keys of pages p with p % (n_kv hd) = h hd + d, else 0), so the
    output is the share of the sequence's keys in those pages. Scores are 0
    and P = 1 exactly, every sum is an exact small integer in fp32, and the
    only rounding is the final bf16 store: |g - r| <= 2^-8 |r|. A page that
    a split drops, repeats or reads from the wrong sequence moves some
    output by 16 keys' share, far outside that bound.
Inputs are drawn by a seeded torch generator on the device and copied to the
host by torch; the library only stores and reads them.
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


# ------------------------------------------------------------ decode attention
DECODE_CASES = {
    "8b_decode_b64": "llama8b_decode",
    "8b_think_b32": "llama8b_think",
    "70b_decode_b64": "llama70b_model",
}


def _contexts(wl):
    if wl.ctx_law == "fixed":
        return [int(wl.ctx_params[0])] * wl.decode_batch
    return [int(c) for c in gen.context_lengths(wl)]


def _sample(ctx, n=8):
    order = np.argsort(ctx, kind="stable")
    picks = {int(order[0]), int(order[-1])}
    for i in np.linspace(0, len(ctx) - 1, n).round().astype(int):
        picks.add(int(order[i]))
    return sorted(picks)


def _census_v(n_tok, n_kv, hd, device="cuda"):
    """V[t, h, d] = 1 if (t // 16) % (n_kv hd) == h hd + d else 0, bf16."""
    slot = (torch.arange(n_tok, device=device) // 16) % (n_kv * hd)
    v = torch.zeros((n_tok, n_kv * hd), dtype=torch.bfloat16, device=device)
    v[torch.arange(n_tok, device=device), slot] = 1.0
    return v.view(n_tok, n_kv, hd)


def _census_ref(n_keys, n_kv, hd, G):
    """Expected census output [n_q, hd] for a query over keys 0..n_keys-1."""
    counts = np.zeros(n_kv * hd)
    pages = np.arange((n_keys + 15) // 16)
    per_page = np.minimum(16, n_keys - 16 * pages)
    np.add.at(counts, pages % (n_kv * hd), per_page)
    return np.repeat((counts / n_keys).reshape(n_kv, 1, hd), G, axis=1).reshape(n_kv * G, hd)


@pytest.mark.parametrize("case", list(DECODE_CASES))
def test_decode_attention_at_the_benchmarked_split_plan(case):
    wl = CONFIGS[DECODE_CASES[case]]
    sh = wl.shape
    ctx = _contexts(wl)
    nb = len(ctx)
    print(f"{case}: batch {nb}, contexts {min(ctx)}..{max(ctx)}", flush=True)
    max_pages = max((c + 16) // 16 for c in ctx)
    n_pages = sum((c + 16) // 16 for c in ctx) + 8
    # layer 0: random K, V; layer 1: random K, census V (same block tables)
    pool = H.Pool(sh, n_pages, nb, max_pages, n_layers=2, seed=gen.page_order_seed(wl))
    kv = pool.kv
    ws = H.workspace(1 << 24)
    g = torch.Generator(device="cuda").manual_seed(1000 + wl.cfg_id)
    sample = _sample(ctx)
    seqs, hist = [], {}
    for b, c in enumerate(ctx):
        s = kv.open()
        kv.alloc(s, c + 1)
        k = torch.randn((c + 1, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        v = torch.randn((c + 1, sh.n_kv, sh.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        vc = _census_v(c + 1, sh.n_kv, sh.head_dim)
        kv.append(0, [s], [c], k[:c], v[:c], ws)
        kv.append(1, [s], [c], k[:c], vc[:c], ws)
        kv.commit([s], [c])
        kv.append(0, [s], [1], k[c:], v[c:], ws)   # the step's own row, not committed
        kv.append(1, [s], [1], k[c:], vc[c:], ws)
        if b in sample:
            hist[b] = (H.to_f64(k), H.to_f64(v))
        seqs.append(s)
        del k, v, vc
    sync()
    q = (torch.randn((nb, sh.n_q, sh.head_dim), generator=g, device="cuda") * 2.0).to(torch.bfloat16)
    q0 = torch.zeros_like(q)
    o = H.empty((nb, sh.d_q), "bf16")
    oc = H.empty((nb, sh.d_q), "bf16")
    aws = H.workspace(64 << 20)
    B.op_decode_plan(kv, seqs, aws)        # the library's own split choice, as the layer and bench use
    B.op_decode_run(kv, 0, q, o, aws)
    B.op_decode_run(kv, 1, q0, oc, aws)
    sync()
    got = H.to_f64(o).reshape(nb, sh.n_q, sh.head_dim)
    qf = H.to_f64(q)
    for b in sample:
        kf, vf = hist[b]
        ref = O.attention(qf[b:b + 1], kf, vf, np.array([ctx[b]]))[0]
        H.assert_close_elementwise(got[b], ref, H.BF16_TOL_ABS, H.BF16_TOL_REL, f"{case} b={b} ctx={ctx[b]}")
    # the capped launch (the mixed step's form: fewer workgroups, each walking
    # several split items) gives the same bits
    for cap in (1, 8 * sh.n_kv, 128):
        ocap = H.empty((nb, sh.d_q), "bf16")
        B.op_decode_run_capped(kv, 0, q, ocap, aws, cap)
        sync()
        assert torch.equal(ocap.view(torch.int16), o.view(torch.int16)), f"{case}: capped at {cap} workgroups differs"
    gc = H.to_f64(oc).reshape(nb, sh.n_q, sh.head_dim)
    for b, c in enumerate(ctx):
        ref = _census_ref(c + 1, sh.n_kv, sh.head_dim, sh.group)
        err = np.abs(gc[b] - ref)
        assert np.all(err <= 2.0 ** -8 * np.abs(ref)), \
            f"{case} census b={b} ctx={c}: max err {err.max():.3e} at {np.unravel_index(err.argmax(), err.shape)}"


# ------------------------------------------------------------------ GEMMs
def _gemm_bound(af, wf, K):
    """2 K 2^-24 sum_k |a_k w_k|: fp32 accumulation of exact bf16 products."""
    return (np.abs(af) @ np.abs(wf).T) * (2 * K * 2.0 ** -24)


def _device_gemm_inputs(M, N, K, seed, swiglu=False):
    g = torch.Generator(device="cuda").manual_seed(seed)
    a = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
    w = (torch.randn((N, K), generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    wt = torch.empty(B.tiled_weight_elems(N, K), dtype=torch.bfloat16, device="cuda")
    B.op_tile_weight(B.PS_BF16, N, K, w, wt)
    return g, a, w, wt


def _check_swiglu(got, af, w_host, K, what):
    """w_host [N, K] in the 32-row gate/up interleave; got [rows, N/2]."""
    N = w_host.shape[0]
    blocks = w_host.reshape(N // 64, 2, 32, K)
    wg = blocks[:, 0].reshape(N // 2, K)
    wu = blocks[:, 1].reshape(N // 2, K)
    gate, up = O.linear(af, wg), O.linear(af, wu)
    eg, eu = _gemm_bound(af, wg, K), _gemm_bound(af, wu, K)
    ref = O.silu(gate) * up
    # |d silu| <= 1.1 |d gate|; then the product, the bf16 store (2^-8) and
    # the hardware exp2/reciprocal in silu (a few fp32 ulp)
    bound = 1.1 * np.abs(up) * eg + (np.abs(O.silu(gate)) + 1.1 * eg) * eu + (2.0 ** -8 + 1e-5) * np.abs(ref)
    err = np.abs(got - ref)
    bad = err > bound
    assert not bad.any(), f"{what}: {int(bad.sum())} outside; max err {err.max():.3e}"


def _tile_rows(M):
    """One row in every 256-row tile row, at a different offset in each."""
    return np.array([256 * t + (37 * t + 11) % 256 for t in range((M + 255) // 256)])


def test_prefill_gate_up_swiglu_16384x28672x4096_every_tile_row():
    """The headline launch: 64 x 112 tiles of 256 (XCD remap, 8-tile-row
    groups); one row of every tile row, every output column."""
    M, N, K = 16384, 28672, 4096
    _, a, w, wt = _device_gemm_inputs(M, N, K, 21)
    m = torch.empty((M, N // 2), dtype=torch.bfloat16, device="cuda")
    B.op_gemm(B.PS_BF16, 0, B.PS_BF16, B.PS_EPI_SWIGLU, M, N, K, a, wt, None, m)
    sync()
    rows = _tile_rows(M)
    ridx = torch.from_numpy(rows).cuda()
    _check_swiglu(H.to_f64(m[ridx]), H.to_f64(a[ridx]), H.to_f64(w), K, "gate_up 16384")


@pytest.mark.parametrize("name,N,K,rdt,cdt", [
    ("qkv", 6144, 4096, None, "bf16"),
    ("o_residual", 4096, 4096, "bf16", "f32"),
    ("down_residual", 4096, 14336, "f32", "bf16"),
])
def test_prefill_gemms_16384_rows_every_tile_row(name, N, K, rdt, cdt):
    """The other three prefill GEMMs of the 8 x 2048 step at M = 16384, with
    the dtypes the layer uses; one row of every tile row, every column."""
    M = 16384
    g, a, w, wt = _device_gemm_inputs(M, N, K, 22 + K)
    code = {"bf16": B.PS_BF16, "f32": B.PS_F32, None: 0}
    tdt = {"bf16": torch.bfloat16, "f32": torch.float32}
    r = torch.randn((M, N), generator=g, device="cuda").to(tdt[rdt]) if rdt else None
    c = torch.empty((M, N), dtype=tdt[cdt], device="cuda")
    epi = B.PS_EPI_RESIDUAL if rdt else B.PS_EPI_STORE
    B.op_gemm(B.PS_BF16, code[rdt], code[cdt], epi, M, N, K, a, wt, r, c)
    sync()
    rows = _tile_rows(M)
    ridx = torch.from_numpy(rows).cuda()
    af, wf = H.to_f64(a[ridx]), H.to_f64(w)
    ref = O.linear(af, wf) + (H.to_f64(r[ridx]) if rdt else 0.0)
    bound = _gemm_bound(af, wf, K) + (2.0 ** -8 if cdt == "bf16" else 2.0 ** -23) * np.abs(ref)
    err = np.abs(H.to_f64(c[ridx]) - ref)
    assert np.all(err <= bound), f"{name}: max err {err.max():.3e}"


DECODE_GEMMS = [
    # (layer shape, name, N, K, epilogue, r dtype, c dtype): the layer's four GEMMs at decode batch 64
    ("8b", "qkv", 6144, 4096, "store", None, "bf16"),
    ("8b", "o", 4096, 4096, "residual", "bf16", "f32"),
    ("8b", "gate_up", 28672, 4096, "swiglu", None, "bf16"),
    ("8b", "down", 4096, 14336, "residual", "f32", "bf16"),
    ("70b", "qkv", 10240, 8192, "store", None, "bf16"),
    ("70b", "o", 8192, 8192, "residual", "bf16", "f32"),
    ("70b", "gate_up", 57344, 8192, "swiglu", None, "bf16"),
    ("70b", "down", 8192, 28672, "residual", "f32", "bf16"),
]


@pytest.mark.parametrize("shape,name,N,K,epi,rdt,cdt", DECODE_GEMMS,
                         ids=[f"{s}_{n}" for s, n, *_ in DECODE_GEMMS])
def test_decode_gemms_at_batch_64_every_element(shape, name, N, K, epi, rdt, cdt):
    """The skinny kernel with the plan the layer takes at M = 64 (K splits and
    the reduce where the plan splits); every row and column."""
    M = 64
    g, a, w, wt = _device_gemm_inputs(M, N, K, 30 + N // 64)
    code = {"bf16": B.PS_BF16, "f32": B.PS_F32, None: 0}
    tdt = {"bf16": torch.bfloat16, "f32": torch.float32}
    r = torch.randn((M, N), generator=g, device="cuda").to(tdt[rdt]) if rdt else None
    cols = N // 2 if epi == "swiglu" else N
    c = torch.empty((M, cols), dtype=tdt[cdt], device="cuda")
    e = {"store": B.PS_EPI_STORE, "residual": B.PS_EPI_RESIDUAL, "swiglu": B.PS_EPI_SWIGLU}[epi]
    ws = H.workspace(B.op_gemm_workspace_bytes(B.PS_BF16, M, N, K))
    B.op_gemm(B.PS_BF16, code[rdt], code[cdt], e, M, N, K, a, wt, r, c, ws)
    sync()
    af, wf = H.to_f64(a), H.to_f64(w)
    if epi == "swiglu":
        _check_swiglu(H.to_f64(c), af, wf, K, f"{shape} {name}")
        return
    ref = O.linear(af, wf) + (H.to_f64(r) if rdt else 0.0)
    bound = _gemm_bound(af, wf, K) + (2.0 ** -8 if cdt == "bf16" else 2.0 ** -23) * np.abs(ref)
    err = np.abs(H.to_f64(c) - ref)
    assert np.all(err <= bound), f"{shape} {name}: max err {err.max():.3e}"
