"""The model path (embedding, layer stack, final norm, LM head, greedy argmax)
against the fp64 oracle (GPU).

Greedy tokens: several answers are correct when logits nearly tie, so a
device token t is accepted iff oracle_logit[t] >= max oracle logit -
(2e-2 + 1e-2 |max|), and logits are compared with the normwise bound. Decode
steps consume predetermined synthetic tokens (not the device's argmax), so
no device output ever becomes an oracle input.
"""
import numpy as np
import pytest

from oracle import layer as O
from synth import gen
from synth.configs import CONFIGS, LayerShape, Workload
from tests import bf16_emulation as E
from tests import helpers as H

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2608_21719_amd import binding as B  # noqa: E402


def sync():
    torch.cuda.synchronize()


def accept_tokens(got_tok, ref_logits, what):
    for i, t in enumerate(got_tok):
        mx = ref_logits[i].max()
        tau = 2e-2 + 1e-2 * abs(mx)
        assert ref_logits[i][t] >= mx - tau, f"{what} row {i}: token {t} logit {ref_logits[i][t]:.4f} < max {mx:.4f} - {tau:.3f}"


@pytest.mark.parametrize("vocab", [128256, 1001])  # 16-byte loads; an odd vocabulary takes 4-byte loads
def test_argmax_full_vocab_with_ties(vocab):
    rows = 64
    r = np.random.default_rng(1)
    lg = r.standard_normal((rows, vocab)).astype(np.float32)
    for i in range(rows):  # plant a tie between two maxima
        a, b = sorted(r.choice(vocab, 2, replace=False))
        lg[i, a] = lg[i, b] = 10.0 + i
    lg[3, :] = 1.0  # all equal: index 0
    d = torch.from_numpy(lg).cuda()
    out = torch.empty(rows, dtype=torch.int32, device="cuda")
    B.op_argmax(rows, vocab, d, out)
    sync()
    np.testing.assert_array_equal(out.cpu().numpy(), O.argmax_lowest(lg.astype(np.float64)))


def test_lm_head_gemm_fullsize_sampled_columns():
    """M=64 decode rows through the 128256 x 8192 LM head (skinny split-K path)."""
    M, N, K = 64, 128256, 8192
    g = torch.Generator(device="cuda").manual_seed(5)
    a = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
    w = (torch.randn((N, K), generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    wt = torch.empty(B.tiled_weight_elems(N, K), dtype=torch.bfloat16, device="cuda")
    B.op_tile_weight(B.PS_BF16, N, K, w, wt)
    c = torch.empty((M, N), dtype=torch.float32, device="cuda")
    ws = H.workspace(B.op_gemm_workspace_bytes(B.PS_BF16, M, N, K))
    B.op_gemm(B.PS_BF16, 0, B.PS_F32, B.PS_EPI_STORE, M, N, K, a, wt, None, c, ws)
    sync()
    cols = np.sort(np.random.default_rng(2).choice(N, 300, replace=False))
    af = H.to_f64(a)
    wf = H.to_f64(w[torch.from_numpy(cols).cuda()])
    ref = O.linear(af, wf)
    got = c.cpu().numpy().astype(np.float64)[:, cols]
    bound = (np.abs(af) @ np.abs(wf).T) * (2 * K * 2.0 ** -24)
    assert np.all(np.abs(got - ref) <= bound + 1e-30), f"max err {np.abs(got - ref).max()}"


SMALL = LayerShape(1024, 8, 1, 128, 2048, 1e-5, 500000.0, "bf16")


def small_model_parts(n_layers=3, vocab=2048):
    wl = Workload("small_model", 12, SMALL, n_layers=n_layers, vocab=vocab)
    layers = [gen.layer_weights(wl, l) for l in range(n_layers)]
    head = gen.model_head_weights(wl)
    return wl, layers, head


def oracle_model_rows(layers_f, head_f, shape, tokens, hists):
    """Run the oracle stack over one sequence's new tokens; returns logits of
    the last row and the per-layer (K, V) it appended."""
    h = O.embed(head_f["embed"], tokens)
    new_hist = []
    for l, wf in enumerate(layers_f):
        kh, vh = hists[l] if hists else (None, None)
        r = O.layer_sequence(wf, shape, h, kh, vh)
        h = r["out"]
        new_hist.append((r["k"], r["v"]))
    logits = O.lm_logits(h[-1:], head_f["final_norm"], head_f["lm_head"], shape.eps)[0]
    return logits, new_hist


def test_small_model_prefill_then_decode():
    wl, layers, head = small_model_parts()
    sh, L, V = wl.shape, wl.n_layers, wl.vocab
    layers_f = [H.weights_f64(w, "bf16") for w in layers]
    head_f = H.weights_f64(head, "bf16")
    dev_layers = [H.DeviceLayer(w, "bf16") for w in layers]
    dev_head = {k: (H.to_dev_w if k == "lm_head" else H.to_dev)(v, "bf16") for k, v in head.items()}
    pool = H.Pool(sh, 64, 4, 8, n_layers=L, seed=21)
    model = B.Model(pool.cfg, [d.w for d in dev_layers], V, dev_head["embed"], dev_head["final_norm"],
                    dev_head["lm_head"])
    lens = [40, 23]
    seqs = [pool.kv.open() for _ in lens]
    for s, n in zip(seqs, lens):
        pool.kv.alloc(s, n + 4)
    ws = H.workspace(B.Model.workspace_bytes(pool.cfg, V, 128, 4, 8))
    toks = gen.token_ids(wl, sum(lens))
    dtok = torch.from_numpy(toks).cuda()
    nxt = torch.empty(len(seqs), dtype=torch.int32, device="cuda")
    logits = torch.empty((len(seqs), V), dtype=torch.float32, device="cuda")
    model.prefill(pool.kv, seqs, lens, dtok, nxt, ws, logits)
    pool.kv.commit(seqs, lens)
    sync()
    hists, r0 = [], 0
    ref_logits = []
    for n in lens:
        lg, hh = oracle_model_rows(layers_f, head_f, sh, toks[r0:r0 + n], None)
        ref_logits.append(lg)
        hists.append(hh)
        r0 += n
    ref_logits = np.stack(ref_logits)
    got_logits = logits.cpu().numpy().astype(np.float64)
    mx, rms = H.normwise(got_logits, ref_logits)
    assert mx <= H.NORMWISE_TOL and rms <= H.NORMWISE_TOL, f"prefill logits normwise {mx:.2e} {rms:.2e}"
    accept_tokens(nxt.cpu().numpy(), ref_logits, "prefill")
    for step in range(3):
        t = gen.token_ids(wl, len(seqs), step=step + 1)
        model.decode_step(pool.kv, B.PS_PHASE_ANSWER, seqs, torch.from_numpy(t).cuda(), nxt, ws, logits)
        pool.kv.commit(seqs, [1] * len(seqs))
        sync()
        ref_logits = []
        for i in range(len(seqs)):
            lg, hh = oracle_model_rows(layers_f, head_f, sh, t[i:i + 1], hists[i])
            hists[i] = [(np.concatenate([kh, k]), np.concatenate([vh, v])) for (kh, vh), (k, v) in zip(hists[i], hh)]
            ref_logits.append(lg)
        ref_logits = np.stack(ref_logits)
        got_logits = logits.cpu().numpy().astype(np.float64)
        mx, rms = H.normwise(got_logits, ref_logits)
        assert mx <= H.NORMWISE_TOL and rms <= H.NORMWISE_TOL, f"decode {step} logits normwise {mx:.2e} {rms:.2e}"
        accept_tokens(nxt.cpu().numpy(), ref_logits, f"decode {step}")


def test_small_model_decode_equals_single_layer_calls_bit_for_bit():
    """The model call (embedding, the layer stack in one call, final norm, LM head, argmax) and the same decode
    step through single-layer calls and the head ops give the same bits: logits, next tokens and every KV byte
    written. The model call shares one metadata upload across its layers; the layer calls each upload their
    own."""
    wl, layers, head = small_model_parts()
    sh, L, V = wl.shape, wl.n_layers, wl.vocab
    dev_layers = [H.DeviceLayer(w, "bf16") for w in layers]
    dev_head = {k: (H.to_dev_w if k == "lm_head" else H.to_dev)(v, "bf16") for k, v in head.items()}
    pools = [H.Pool(sh, 64, 4, 8, n_layers=L, seed=21) for _ in range(2)]
    model = B.Model(pools[0].cfg, [d.w for d in dev_layers], V, dev_head["embed"], dev_head["final_norm"],
                    dev_head["lm_head"])
    lens = [40, 23]
    ws = H.workspace(B.Model.workspace_bytes(pools[0].cfg, V, 128, 4, 8))
    dtok = torch.from_numpy(gen.token_ids(wl, sum(lens))).cuda()
    nxt = torch.empty(len(lens), dtype=torch.int32, device="cuda")
    seqs = []
    for P in pools:
        ss = [P.kv.open() for _ in lens]
        for s, n in zip(ss, lens):
            P.kv.alloc(s, n + 4)
        model.prefill(P.kv, ss, lens, dtok, nxt, ws)
        P.kv.commit(ss, lens)
        seqs.append(ss)
    sync()
    t = torch.from_numpy(gen.token_ids(wl, len(lens), step=1)).cuda()
    logits_m = torch.empty((len(lens), V), dtype=torch.float32, device="cuda")
    nxt_m = torch.empty(len(lens), dtype=torch.int32, device="cuda")
    model.decode_step(pools[0].kv, B.PS_PHASE_ANSWER, seqs[0], t, nxt_m, ws, logits_m)

    layer = B.Layer(pools[1].cfg)
    lws = H.workspace(B.Layer.workspace_bytes(pools[1].cfg, 64, 4, 8))
    x = dev_head["embed"][t.long()].contiguous()
    for l in range(L):
        y = torch.empty_like(x)
        layer.decode_step(dev_layers[l].w, pools[1].kv, l, B.PS_PHASE_ANSWER, seqs[1], x, y, lws)
        x = y
    hn = torch.empty_like(x)
    B.op_rmsnorm(B.PS_BF16, B.PS_BF16, B.PS_BF16, len(lens), sh.hidden, x, dev_head["final_norm"], sh.eps, hn)
    logits_c = torch.empty((len(lens), V), dtype=torch.float32, device="cuda")
    gws = H.workspace(max(16, B.op_gemm_workspace_bytes(B.PS_BF16, len(lens), V, sh.hidden)))
    B.op_gemm(B.PS_BF16, 0, B.PS_F32, B.PS_EPI_STORE, len(lens), V, sh.hidden, hn, dev_head["lm_head"], None,
              logits_c, gws)
    nxt_c = torch.empty(len(lens), dtype=torch.int32, device="cuda")
    B.op_argmax(len(lens), V, logits_c, nxt_c)
    sync()
    assert torch.equal(logits_m.view(torch.int32), logits_c.view(torch.int32))
    assert torch.equal(nxt_m, nxt_c)
    assert torch.equal(pools[0].mem.view(torch.uint8), pools[1].mem.view(torch.uint8))


def test_model_rejects_shallow_pool():
    wl, layers, head = small_model_parts(n_layers=2, vocab=256)
    dev_layers = [H.DeviceLayer(w, "bf16") for w in layers]
    dev_head = {k: (H.to_dev_w if k == "lm_head" else H.to_dev)(v, "bf16") for k, v in head.items()}
    pool = H.Pool(wl.shape, 8, 2, 4, n_layers=1)
    model = B.Model(pool.cfg, [d.w for d in dev_layers], 256, dev_head["embed"], dev_head["final_norm"],
                    dev_head["lm_head"])
    s = pool.kv.open()
    pool.kv.alloc(s, 4)
    ws = H.workspace(B.Model.workspace_bytes(pool.cfg, 256, 16, 2, 4))
    tok = torch.zeros(4, dtype=torch.int32, device="cuda")
    nxt = torch.empty(1, dtype=torch.int32, device="cuda")
    with pytest.raises(B.PsError) as e:
        model.prefill(pool.kv, [s], [4], tok, nxt, ws)
    assert e.value.code == B.PS_E_INVALID


# ------------------------------------------------------------- 70B width
def _lm_chunks(h64, g64, lm_bits, eps, dtype, fn, chunk=16384):
    """Logits over the whole vocabulary, the LM head widened chunk by chunk."""
    out = []
    for v0 in range(0, lm_bits.shape[0], chunk):
        w = gen.bf16_bits_to_f32(lm_bits[v0:v0 + chunk]).astype(dtype)
        out.append(fn(h64, g64, w, eps))
    return np.concatenate(out, axis=-1)


@pytest.mark.timeout(900)
def test_70b_width_two_layer_model_full_vocab():
    """ps_model_prefill and two ps_model_decode_step calls of a 2-layer model
    at the 70B shape (d 8192, 64 / 8 heads, F 28672) with the full 128256
    vocabulary, against the fp64 oracle stack (embedding, both layers, final
    norm, LM head). Weights are drawn on the device by a seeded torch
    generator and copied to the host as bf16 bits; the oracle widens them.

    Bound: the same stack through the bf16 rounding model on the same inputs
    gives the error floor of any pipeline with the device's rounding points;
    the device's logits must be within TOL_MARGIN times that floor (normwise
    max and rms). Tokens: if every logit is within e of the oracle's, the
    device's argmax t has oracle logit >= max - 2e, so a token is accepted
    within 2e with e = the normwise bound times max |logit|."""
    sh = CONFIGS["llama70b_model"].shape
    V, L = CONFIGS["llama70b_model"].vocab, 2
    d, dq, dkv, F = sh.hidden, sh.d_q, sh.d_kv, sh.ffn
    g = torch.Generator(device="cuda").manual_seed(7070)

    def rn(shape, mean=0.0):
        t = torch.randn(shape, generator=g, device="cuda") * 0.02
        return (t + mean).to(torch.bfloat16)

    def host_bits(t):
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)

    def tiled(w):
        out = torch.empty(B.tiled_weight_elems(*w.shape), dtype=torch.bfloat16, device="cuda")
        B.op_tile_weight(B.PS_BF16, w.shape[0], w.shape[1], w, out)
        return out

    keep, dev_layers, bits = [], [], []
    for l in range(L):
        t = {"attn_norm": rn((d,), 1.0), "wq": rn((dq, d)), "wk": rn((dkv, d)), "wv": rn((dkv, d)),
             "wo": rn((d, dq)), "ffn_norm": rn((d,), 1.0), "wg": rn((F, d)), "wu": rn((F, d)), "wd": rn((d, F))}
        gu = torch.stack([t["wg"].view(F // 32, 32, d), t["wu"].view(F // 32, 32, d)], 1).reshape(2 * F, d)
        dev = {"attn_norm": t["attn_norm"], "w_qkv": tiled(torch.cat([t["wq"], t["wk"], t["wv"]])),
               "w_o": tiled(t["wo"]), "ffn_norm": t["ffn_norm"], "w_gate_up": tiled(gu), "w_down": tiled(t["wd"])}
        keep.append(dev)
        dev_layers.append(B.layer_weights(**dev))
        bits.append({k: host_bits(v) for k, v in t.items()})
        del t, gu
    embed, final_norm, lm = rn((V, d)), rn((d,), 1.0), rn((V, d))
    lm_t = tiled(lm)
    embed_bits, gfin_bits, lm_bits = host_bits(embed), host_bits(final_norm), host_bits(lm)
    del lm
    torch.cuda.synchronize()
    print("weights on device and host", flush=True)

    lens = [45, 64]
    pool = H.Pool(sh, 32, 4, 8, n_layers=L, seed=31)
    model = B.Model(pool.cfg, dev_layers, V, embed, final_norm, lm_t)
    seqs = [pool.kv.open() for _ in lens]
    for s, n in zip(seqs, lens):
        pool.kv.alloc(s, n + 2)
    ws = H.workspace(B.Model.workspace_bytes(pool.cfg, V, sum(lens), 4, 8))
    wl = CONFIGS["llama70b_model"]
    toks = gen.token_ids(wl, sum(lens))
    nxt = torch.empty(len(seqs), dtype=torch.int32, device="cuda")
    logits = torch.empty((len(seqs), V), dtype=torch.float32, device="cuda")

    w64 = [E.WidenedWeights(b, np.float64) for b in bits]
    w32 = [E.WidenedWeights(b, np.float32) for b in bits]
    g64 = gen.bf16_bits_to_f32(gfin_bits).astype(np.float64)
    g32 = gen.bf16_bits_to_f32(gfin_bits)
    hist64 = [[None] * L for _ in lens]   # per sequence, per layer (K, V)
    hist32 = [[None] * L for _ in lens]

    def run_oracles(i, tokens):
        h64 = gen.bf16_bits_to_f32(embed_bits[tokens]).astype(np.float64)
        h32 = gen.bf16_bits_to_f32(embed_bits[tokens])
        for l in range(L):
            kh, vh = hist64[i][l] or (None, None)
            r = O.layer_sequence(w64[l], sh, h64, kh, vh)
            hist64[i][l] = (r["k"], r["v"]) if kh is None else (np.concatenate([kh, r["k"]]),
                                                                 np.concatenate([vh, r["v"]]))
            h64 = r["out"]
            kh, vh = hist32[i][l] or (None, None)
            h32, k, v = E.layer(w32[l], sh, h32, kh, vh, return_kv=True)
            hist32[i][l] = (k, v) if kh is None else (np.concatenate([kh, k]), np.concatenate([vh, v]))
        ref = _lm_chunks(h64[-1:], g64, lm_bits, sh.eps, np.float64, O.lm_logits)[0]
        emu = _lm_chunks(h32[-1:], g32, lm_bits, sh.eps, np.float32, E.lm_logits)[0]
        return ref, emu.astype(np.float64)

    def check(step, tokens_per_seq):
        torch.cuda.synchronize()
        got = logits.cpu().numpy().astype(np.float64)
        refs, emus = zip(*[run_oracles(i, t) for i, t in enumerate(tokens_per_seq)])
        ref, emu = np.stack(refs), np.stack(emus)
        floor = max(H.normwise(emu, ref))
        bound = H.TOL_MARGIN * floor
        mx, rms = H.normwise(got, ref)
        print(f"{step}: device normwise max {mx:.3e} rms {rms:.3e}; rounding floor {floor:.3e}", flush=True)
        assert floor < 5e-2, f"{step}: rounding floor {floor:.3e}"
        assert mx <= bound and rms <= bound, f"{step}: normwise {mx:.3e} {rms:.3e} > {bound:.3e}"
        tau = 2 * bound * np.abs(ref).max(axis=1)
        for i, t in enumerate(nxt.cpu().numpy()):
            assert ref[i][t] >= ref[i].max() - tau[i], f"{step} row {i}: token {t}"

    model.prefill(pool.kv, seqs, lens, torch.from_numpy(toks).cuda(), nxt, ws, logits)
    pool.kv.commit(seqs, lens)
    check("prefill", [toks[:lens[0]], toks[lens[0]:]])
    for step in range(2):
        t = gen.token_ids(wl, len(seqs), step=step + 1)
        model.decode_step(pool.kv, B.PS_PHASE_ANSWER, seqs, torch.from_numpy(t).cuda(), nxt, ws, logits)
        pool.kv.commit(seqs, [1] * len(seqs))
        check(f"decode {step}", [t[i:i + 1] for i in range(len(seqs))])
