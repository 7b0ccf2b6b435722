"""Benchmark of the layer hot path on one MI355X.

Headline (``value``): prefill tokens/s of the 8B-shaped layer on 8 prompts x
2048 tokens (one step = one ps_prefill over the batch: RMSNorm, QKV GEMM,
RoPE + paged KV write, causal flash attention, O GEMM + residual, RMSNorm,
gate_up GEMM + SwiGLU, down GEMM + residual). The ``decode`` object holds the
8B-shaped decode phase: batch 64, contexts U{1024..4096}, one ps_decode_step
per step (plus commit) over a shuffled paged cache.

``roofline`` is for each phase's dominant kernel, timed live with HIP events
on the stream it runs on: the prefill gate_up GEMM (bound: MFMA) and the
split-K decode attention (bound: HBM). ``cpu_baseline`` times the fp64 oracle
on a bounded sample of the same prefill workload on the host cores.

Inputs are seeded synthetic tensors generated on the device (weights
N(0, 0.02^2), norm gains 1 + N(0, 0.02^2), activations and KV N(0, 1)).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode tok/s & HBM GB/s; prefill tok/s & MFMA util (8B-shaped layer)"
TEL = None  # telemetry.Telemetry, set in main: GPU clock and power of each timed leg
TEL_SECONDS = 1.5  # length of each leg's clock-and-power window (0: none, e.g. under a counter profiler)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def randn(torch, gen, shape, std=1.0, mean=0.0):
    t = torch.randn(shape, generator=gen, device="cuda", dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    if mean != 0.0:
        t.add_(mean)
    return t.to(torch.bfloat16)


def make_layer_weights(torch, B, shape, gen):
    """Random-init layer weights drawn directly in the library's layouts:
    entries are iid, so the gate/up row interleave and the 64x64 weight
    tiling are relabellings of an iid matrix and need no conversion pass."""
    d, dq, dkv, f = shape.hidden, shape.d_q, shape.d_kv, shape.ffn
    t = {
        "attn_norm": randn(torch, gen, (d,), 0.02, 1.0),
        "w_qkv": randn(torch, gen, (dq + 2 * dkv, d), 0.02),
        "w_o": randn(torch, gen, (d, dq), 0.02),
        "ffn_norm": randn(torch, gen, (d,), 0.02, 1.0),
        "w_gate_up": randn(torch, gen, (2 * f, d), 0.02),
        "w_down": randn(torch, gen, (d, f), 0.02),
    }
    return t, B.layer_weights(**t)


class EventTimer:
    """Average duration of a launch sequence, HIP events on the current stream."""

    def __init__(self, torch):
        self.torch = torch

    def __call__(self, fn, iters, warmup=2):
        torch = self.torch
        for _ in range(warmup):
            fn()
        s = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(iters):
            fn()
        e1.record(s)
        e1.synchronize()
        return e0.elapsed_time(e1) / iters  # ms


def bench_prefill(torch, B, A, wl, steps, warmup):
    sh = wl.shape
    gen = torch.Generator(device="cuda").manual_seed(1234)
    cfg = B.make_cfg(sh)
    tw, w = make_layer_weights(torch, B, sh, gen)
    n, T = wl.prefill_seqs, wl.prefill_tokens
    pages = (T + 15) // 16
    pool = torch.empty(B.KV.pool_bytes(cfg, 1, n * pages + 8), dtype=torch.uint8, device="cuda")
    kv = B.KV(cfg, 1, n * pages + 8, n, pages, pool, seed=0x5EED)
    seqs = [kv.open() for _ in range(n)]
    for s in seqs:
        kv.alloc(s, T)
    layer = B.Layer(cfg)
    ws = torch.empty(B.Layer.workspace_bytes(cfg, n * T, n, pages), dtype=torch.uint8, device="cuda")
    x = randn(torch, gen, (n * T, sh.hidden))
    out = torch.empty_like(x)

    def step():
        layer.prefill(w, kv, 0, seqs, [T] * n, x, out, ws)
        for s in seqs:  # positions restart at 0 each step (host-only metadata)
            kv.truncate(s, 0)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    tel_step = observe(step)
    tokens = n * T

    # dominant kernel: gate_up GEMM + SwiGLU epilogue, same launch path as the layer
    M, N, K = tokens, 2 * sh.ffn, sh.hidden
    hn = randn(torch, gen, (M, K))
    m = torch.empty((M, sh.ffn), dtype=torch.bfloat16, device="cuda")
    timer = EventTimer(torch)
    gate_up = lambda: B.op_gemm(B.PS_BF16, 0, B.PS_BF16, B.PS_EPI_SWIGLU, M, N, K, hn, tw["w_gate_up"], None, m)  # noqa: E731
    g_ms = timer(gate_up, iters=max(50, steps))
    tel_gemm = observe(gate_up)
    flops = 2.0 * M * N * K
    gemm_tflops = flops / (g_ms * 1e-3) / 1e12
    total_gemm = A.gemm_flops(tokens, sh.hidden, sh.d_q, sh.d_kv, sh.ffn)
    attn = A.prefill_attention_flops([T] * n, sh.n_q, sh.head_dim)
    # flash attention alone over the K/V the last step wrote (lengths are 0 again)
    qa = randn(torch, gen, (tokens, sh.n_q, sh.head_dim))
    oa = torch.empty((tokens, sh.d_q), dtype=torch.bfloat16, device="cuda")
    attn_run = lambda: B.op_attention(kv, 0, seqs, [T] * n, qa, oa, ws)  # noqa: E731
    # 0.3 ms launches: 100 untimed launches let the clock settle from the
    # GEMM window above, then 200 are timed (about 0.1 s in all)
    a_ms = timer(attn_run, iters=max(200, steps), warmup=100)
    tel_attn = observe(attn_run)
    traffic = measured_traffic("gate_up_gemm_8x2048", "paper_2608_21719_amd/csrc/k_gemm.hip")
    res = {
        "tok_s": tokens / (ms * 1e-3), "ms_per_step": ms,
        "layer_tflops": (total_gemm + attn) / (ms * 1e-3) / 1e12,
        "telemetry": tel_step,
        "gate_up_gemm": {"ms": g_ms, "tflops": gemm_tflops, "M": M, "N": N, "K": K, "telemetry": tel_gemm},
        "attention": {"ms": a_ms, "tflops": attn / (a_ms * 1e-3) / 1e12, "telemetry": tel_attn},
        "roofline": A.Roofline("mfma", gemm_tflops, A.BF16_DENSE_PEAK_TFLOPS, "TFLOP/s", traffic,
                               roofline_extra("mfma", gemm_tflops, tel_gemm, traffic)).as_dict(),
    }
    del pool, ws, tw, x, out, hn, m, qa, oa
    return res


def bench_decode(torch, B, A, wl, steps, warmup):
    from synth import gen as G
    sh = wl.shape
    gen = torch.Generator(device="cuda").manual_seed(4321)
    cfg = B.make_cfg(sh)
    tw, w = make_layer_weights(torch, B, sh, gen)
    ctx = [int(c) for c in G.context_lengths(wl)]
    nb = len(ctx)
    extra = warmup + steps + 2
    max_pages = (max(ctx) + extra + 15) // 16
    n_pages = sum((c + extra + 15) // 16 for c in ctx) + 8
    pool_elems = B.KV.pool_bytes(cfg, 1, n_pages) // 2
    pool = randn(torch, gen, (pool_elems,))      # synthetic KV history, N(0, 1)
    kv = B.KV(cfg, 1, n_pages, nb, max_pages, pool, seed=G.page_order_seed(wl))
    seqs = [kv.open() for _ in range(nb)]
    for s, c in zip(seqs, ctx):
        kv.alloc(s, c + extra)
        kv.commit([s], [c])
    layer = B.Layer(cfg)
    ws = torch.empty(B.Layer.workspace_bytes(cfg, nb, nb, max_pages), dtype=torch.uint8, device="cuda")
    x = randn(torch, gen, (nb, sh.hidden))
    out = torch.empty_like(x)

    def step():
        layer.decode_step(w, kv, 0, B.PS_PHASE_ANSWER, seqs, x, out, ws)
        kv.commit(seqs, [1] * nb)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    lens0 = [kv.seq_len(s) for s in seqs]
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    # algorithmic bytes of the timed steps: KV read (len+1 keys) + weights
    kv_bytes = sum(A.decode_attention_bytes([L + i + 1 for L in lens0], sh.n_kv, sh.head_dim, 2)
                   for i in range(steps)) / steps
    w_bytes = A.weight_bytes(sh.hidden, sh.d_q, sh.d_kv, sh.ffn, 2)

    # dominant kernel: split-K decode attention + its split combine, timed
    # alone (work list planned once, as for the layers of one step)
    q = randn(torch, gen, (nb, sh.n_q, sh.head_dim))
    o = torch.empty((nb, sh.d_q), dtype=torch.bfloat16, device="cuda")
    aws = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    timer = EventTimer(torch)
    B.op_decode_plan(kv, seqs, aws)
    attn = lambda: B.op_decode_run(kv, 0, q, o, aws)  # noqa: E731
    a_ms = timer(attn, iters=max(200, steps))
    tel_attn = observe(attn)
    lens = [kv.seq_len(s) for s in seqs]
    a_bytes = A.decode_attention_bytes([L + 1 for L in lens], sh.n_kv, sh.head_dim, 2)
    a_gbs = a_bytes / (a_ms * 1e-3) / 1e9
    # the same launch with the 256 MB Infinity Cache cold: a 1 GiB overwrite
    # between launches, each launch timed by its own event pair
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    cold = []
    for i in range(40):
        flush.fill_(float(i))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        attn()
        e1.record()
        cold.append((e0, e1))
    torch.cuda.synchronize()
    cold_ms = sorted(e0.elapsed_time(e1) for e0, e1 in cold[5:])[len(cold[5:]) // 2]
    del flush
    tel_step = observe(lambda: layer.decode_step(w, kv, 0, B.PS_PHASE_ANSWER, seqs, x, out, ws))  # no commit
    traffic = measured_traffic("decode_attention_b64", "paper_2608_21719_amd/csrc/k_attn_decode.hip")
    res = {
        "tok_s": nb / (ms * 1e-3), "ms_per_step": ms, "batch": nb,
        "ctx_mean": sum(ctx) / nb, "steps": steps,
        "hbm_gbs": (kv_bytes + w_bytes) / (ms * 1e-3) / 1e9,
        "step_bytes": kv_bytes + w_bytes,
        "telemetry": tel_step,
        "attention": {"us": a_ms * 1e3, "gbs": a_gbs, "bytes": a_bytes, "telemetry": tel_attn,
                      "cache_cold": {"us": cold_ms * 1e3, "gbs": a_bytes / (cold_ms * 1e-3) / 1e9,
                                     "how": "median of 35 launches, each after a 1 GiB overwrite"}},
        "roofline": A.Roofline("hbm", a_gbs, A.HBM_PEAK_GBS, "GB/s", traffic,
                               roofline_extra("hbm", a_gbs, tel_attn, traffic)).as_dict(),
    }
    del pool, ws, tw, x, out, aws
    return res


def bench_think(torch, B, A, wl, steps, warmup):
    """Reasoning think phase: decode B=32 over long log-normal contexts, plus
    one mixed step fusing 4 new 512-token prefill chunks with the 32 decodes."""
    from synth import gen as G
    sh = wl.shape
    gen = torch.Generator(device="cuda").manual_seed(777)
    cfg = B.make_cfg(sh)
    tw, w = make_layer_weights(torch, B, sh, gen)
    ctx = [int(c) for c in G.context_lengths(wl)]
    nb, nc, chunk = len(ctx), wl.mixed_new, wl.mixed_chunk
    extra = warmup + steps + 4
    max_pages = (max(max(ctx) + extra, chunk) + 15) // 16
    n_pages = sum((c + extra + 15) // 16 for c in ctx) + nc * ((chunk + 15) // 16) + 8
    pool = randn(torch, gen, (B.KV.pool_bytes(cfg, 1, n_pages) // 2,))
    kv = B.KV(cfg, 1, n_pages, nb + nc, max_pages, pool, seed=G.page_order_seed(wl))
    seqs = [kv.open() for _ in range(nb)]
    for s, c in zip(seqs, ctx):
        kv.alloc(s, c + extra)
        kv.commit([s], [c])
    layer = B.Layer(cfg)
    ws = torch.empty(B.Layer.workspace_bytes(cfg, nc * chunk + nb, nb + nc, max_pages), dtype=torch.uint8,
                     device="cuda")
    x = randn(torch, gen, (nb, sh.hidden))
    out = torch.empty_like(x)

    def step():
        layer.decode_step(w, kv, 0, B.PS_PHASE_THINK, seqs, x, out, ws)
        kv.commit(seqs, [1] * nb)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    lens0 = [kv.seq_len(s) for s in seqs]
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    tel_step = observe(lambda: layer.decode_step(w, kv, 0, B.PS_PHASE_THINK, seqs, x, out, ws))  # no commit
    kv_bytes = sum(A.decode_attention_bytes([L + i + 1 for L in lens0], sh.n_kv, sh.head_dim, 2)
                   for i in range(steps)) / steps
    w_bytes = A.weight_bytes(sh.hidden, sh.d_q, sh.d_kv, sh.ffn, 2)
    q = randn(torch, gen, (nb, sh.n_q, sh.head_dim))
    o = torch.empty((nb, sh.d_q), dtype=torch.bfloat16, device="cuda")
    timer = EventTimer(torch)
    B.op_decode_plan(kv, seqs, ws)
    a_ms = timer(lambda: B.op_decode_run(kv, 0, q, o, ws), iters=max(20, steps))
    a_bytes = A.decode_attention_bytes([kv.seq_len(s) + 1 for s in seqs], sh.n_kv, sh.head_dim, 2)

    # mixed step: chunk rows first, then one row per decoding sequence
    new = [kv.open() for _ in range(nc)]
    for s in new:
        kv.alloc(s, chunk)
    xm = randn(torch, gen, (nc * chunk + nb, sh.hidden))
    om = torch.empty_like(xm)

    def mixed():
        layer.mixed_step(w, kv, 0, new, [chunk] * nc, seqs, xm, om, ws)

    m_ms = timer(mixed, iters=max(40, steps))
    tel_mixed = observe(mixed)
    rows = nc * chunk + nb
    m_flops = A.gemm_flops(rows, sh.hidden, sh.d_q, sh.d_kv, sh.ffn) + \
        A.prefill_attention_flops([chunk] * nc, sh.n_q, sh.head_dim)
    res = {
        "tok_s": nb / (ms * 1e-3), "ms_per_step": ms, "batch": nb, "ctx_mean": sum(ctx) / nb,
        "hbm_gbs": (kv_bytes + w_bytes) / (ms * 1e-3) / 1e9, "telemetry": tel_step,
        "attention": {"us": a_ms * 1e3, "gbs": a_bytes / (a_ms * 1e-3) / 1e9, "bytes": a_bytes},
        "mixed_step": {"ms": m_ms, "rows": rows, "tok_s": rows / (m_ms * 1e-3),
                       "tflops": m_flops / (m_ms * 1e-3) / 1e12, "telemetry": tel_mixed},
    }
    del pool, ws, tw, x, out, xm, om
    return res


def bench_model70b(torch, B, A, wl, steps, warmup):
    """80-layer 70B-shaped model: autoregressive decode of 64 sequences at
    context 4096 (tokens stay on the device), and a prefill of 8 x 1024."""
    from synth import gen as G
    sh = wl.shape
    L, V = wl.n_layers, wl.vocab
    gen = torch.Generator(device="cuda").manual_seed(70)
    cfg = B.make_cfg(sh)
    t0 = time.perf_counter()
    tws, ws_list = [], []
    for _ in range(L):
        tw, w = make_layer_weights(torch, B, sh, gen)
        tws.append(tw)
        ws_list.append(w)
    embed = randn(torch, gen, (V, sh.hidden), 0.02)
    lm_head = randn(torch, gen, (V, sh.hidden), 0.02)  # iid: already a valid tiled weight
    final_norm = randn(torch, gen, (sh.hidden,), 0.02, 1.0)
    ctx = wl.ctx_params[0]
    nb, npf, tp = wl.decode_batch, wl.prefill_seqs, wl.prefill_tokens
    extra = warmup + steps + 2
    pages_dec = (ctx + extra + 15) // 16
    n_pages = nb * pages_dec + npf * ((tp + 15) // 16) + 8
    pool = torch.empty(B.KV.pool_bytes(cfg, L, n_pages) // 2, dtype=torch.bfloat16, device="cuda")
    chunk = 1 << 30
    for i in range(0, pool.numel(), chunk):  # synthetic KV history, N(0, 1)
        n = min(chunk, pool.numel() - i)
        pool[i:i + n] = torch.randn(n, generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    torch.cuda.synchronize()
    fill_s = time.perf_counter() - t0
    log(f"model70b: filled {sum(t.numel() for tw in tws for t in tw.values()) * 2 / 1e9:.1f} GB weights and "
        f"{pool.numel() * 2 / 1e9:.1f} GB KV in {fill_s:.1f} s")
    kv = B.KV(cfg, L, n_pages, nb + npf, max(pages_dec, (tp + 15) // 16), pool, seed=G.page_order_seed(wl))
    model = B.Model(cfg, ws_list, V, embed, final_norm, lm_head)
    seqs = [kv.open() for _ in range(nb)]
    for s in seqs:
        kv.alloc(s, ctx + extra)
        kv.commit([s], [ctx])
    ws = torch.empty(B.Model.workspace_bytes(cfg, V, npf * tp, nb + npf, pages_dec), dtype=torch.uint8,
                     device="cuda")
    tok = [torch.randint(0, V, (nb,), generator=gen, device="cuda", dtype=torch.int32),
           torch.empty(nb, dtype=torch.int32, device="cuda")]

    def dstep(i):
        model.decode_step(kv, B.PS_PHASE_ANSWER, seqs, tok[i % 2], tok[(i + 1) % 2], ws)
        kv.commit(seqs, [1] * nb)

    for i in range(warmup):
        dstep(i)
    torch.cuda.synchronize()
    lens0 = [kv.seq_len(s) for s in seqs]
    t0 = time.perf_counter()
    for i in range(steps):
        dstep(warmup + i)
    torch.cuda.synchronize()
    d_ms = (time.perf_counter() - t0) * 1e3 / steps
    tel_dec = observe(lambda: model.decode_step(kv, B.PS_PHASE_ANSWER, seqs, tok[0], tok[1], ws), seconds=2.0)
    kv_bytes = L * sum(A.decode_attention_bytes([x + i + 1 for x in lens0], sh.n_kv, sh.head_dim, 2)
                       for i in range(steps)) / steps
    w_bytes = L * A.weight_bytes(sh.hidden, sh.d_q, sh.d_kv, sh.ffn, 2) + V * sh.hidden * 2
    # prefill 8 x 1024 on fresh sequences (positions restart each step)
    pseqs = [kv.open() for _ in range(npf)]
    for s in pseqs:
        kv.alloc(s, tp)
    ptok = torch.randint(0, V, (npf * tp,), generator=gen, device="cuda", dtype=torch.int32)
    pnext = torch.empty(npf, dtype=torch.int32, device="cuda")

    def pstep():
        model.prefill(kv, pseqs, [tp] * npf, ptok, pnext, ws)
        for s in pseqs:
            kv.truncate(s, 0)

    pstep()
    torch.cuda.synchronize()
    psteps = max(2, steps // 4)
    t0 = time.perf_counter()
    for _ in range(psteps):
        pstep()
    torch.cuda.synchronize()
    p_ms = (time.perf_counter() - t0) * 1e3 / psteps
    tel_pre = observe(pstep, seconds=3.0)
    p_flops = L * (A.gemm_flops(npf * tp, sh.hidden, sh.d_q, sh.d_kv, sh.ffn) +
                   A.prefill_attention_flops([tp] * npf, sh.n_q, sh.head_dim)) + 2.0 * npf * V * sh.hidden
    res = {
        "decode": {"tok_s": nb / (d_ms * 1e-3), "ms_per_step": d_ms, "batch": nb, "ctx": ctx,
                   "hbm_gbs": (kv_bytes + w_bytes) / (d_ms * 1e-3) / 1e9, "step_bytes": kv_bytes + w_bytes,
                   "telemetry": tel_dec},
        "prefill": {"tok_s": npf * tp / (p_ms * 1e-3), "ms_per_step": p_ms,
                    "tflops": p_flops / (p_ms * 1e-3) / 1e12, "telemetry": tel_pre},
        "hbm_resident_gb": (sum(t.numel() for tw in tws for t in tw.values()) + 2 * V * sh.hidden + pool.numel()) * 2
        / 1e9,
        "fill_s": fill_s,
    }
    del pool, ws, tws, embed, lm_head
    return res


def phase_sweep(torch, B, A, wl):
    """Phase asymmetry on this GPU (the paper's Observation 2, along the
    batch axis: the clock cannot be set from an unprivileged process here).
    For the 8B-shaped layer: prefill of n x 2048 tokens and decode of batch
    B at context 2048, each timed, then replayed under telemetry for the
    clock it settles at, socket power and energy per token; gamma per App.
    B.2 eq. gamma from the step's algorithmic FLOPs and bytes against the
    MI355X ridge (2.5 PFLOP/s over 8 TB/s)."""
    sh = wl.shape
    gen = torch.Generator(device="cuda").manual_seed(2024)
    cfg = B.make_cfg(sh)
    tw, w = make_layer_weights(torch, B, sh, gen)
    layer = B.Layer(cfg)
    ridge = A.ridge_point(A.BF16_DENSE_PEAK_TFLOPS * 1e12, A.HBM_PEAK_GBS * 1e9)
    wbytes = A.weight_bytes(sh.hidden, sh.d_q, sh.d_kv, sh.ffn, 2)
    timer = EventTimer(torch)
    rows = []

    def record(phase, batch, tokens, ms, flops, nbytes, tel):
        # sampled socket power (the driver's energy counter reads about 1.3x
        # the sampled power under load on this platform while agreeing at
        # idle, so its scale is not used)
        pw = ((tel or {}).get("power_w") or {}).get("median")
        clk = ((tel or {}).get("gfxclk_mhz") or {}).get("median")
        ai = flops / nbytes
        rows.append({"phase": phase, "batch": batch, "tokens_per_step": tokens, "ms": ms,
                     "tok_s": tokens / (ms * 1e-3), "tflops": flops / (ms * 1e-3) / 1e12,
                     "hbm_gbs": nbytes / (ms * 1e-3) / 1e9, "ai_flop_per_byte": ai,
                     "gamma": A.gamma(ai, ridge), "gfxclk_mhz": clk, "power_w": pw,
                     "joule_per_token": (pw * ms * 1e-3 / tokens) if pw else None})
        log(f"sweep {phase} B={batch}: {tokens / (ms * 1e-3):.0f} tok/s, clk {clk} MHz, power {pw} W")

    ctx = 2048
    for nb in (1, 4, 16, 64, 256):
        pages = (ctx + 16) // 16
        pool = torch.empty(B.KV.pool_bytes(cfg, 1, nb * pages + 8), dtype=torch.uint8, device="cuda")
        kv = B.KV(cfg, 1, nb * pages + 8, nb, pages, pool, seed=77)
        seqs = [kv.open() for _ in range(nb)]
        for s_ in seqs:
            kv.alloc(s_, ctx + 1)
            kv.commit([s_], [ctx])
        ws = torch.empty(B.Layer.workspace_bytes(cfg, nb, nb, pages), dtype=torch.uint8, device="cuda")
        x = randn(torch, gen, (nb, sh.hidden))
        out = torch.empty_like(x)
        step = lambda: layer.decode_step(w, kv, 0, B.PS_PHASE_ANSWER, seqs, x, out, ws)  # noqa: E731
        ms = timer(step, iters=50)
        flops = A.gemm_flops(nb, sh.hidden, sh.d_q, sh.d_kv, sh.ffn) + \
            A.decode_attention_flops([ctx + 1] * nb, sh.n_q, sh.head_dim)
        nbytes = wbytes + A.decode_attention_bytes([ctx + 1] * nb, sh.n_kv, sh.head_dim, 2)
        record("decode", nb, nb, ms, flops, nbytes, observe(step, seconds=1.2))
        del pool, ws
    T = 2048
    for n in (1, 4, 8):
        pages = T // 16
        pool = torch.empty(B.KV.pool_bytes(cfg, 1, n * pages + 8), dtype=torch.uint8, device="cuda")
        kv = B.KV(cfg, 1, n * pages + 8, n, pages, pool, seed=78)
        seqs = [kv.open() for _ in range(n)]
        for s_ in seqs:
            kv.alloc(s_, T)
        ws = torch.empty(B.Layer.workspace_bytes(cfg, n * T, n, pages), dtype=torch.uint8, device="cuda")
        x = randn(torch, gen, (n * T, sh.hidden))
        out = torch.empty_like(x)
        step = lambda: layer.prefill(w, kv, 0, seqs, [T] * n, x, out, ws)  # noqa: E731
        ms = timer(step, iters=10)
        flops = A.gemm_flops(n * T, sh.hidden, sh.d_q, sh.d_kv, sh.ffn) + \
            A.prefill_attention_flops([T] * n, sh.n_q, sh.head_dim)
        nbytes = wbytes + 2 * n * T * sh.hidden * 2 + n * T * 2 * sh.d_kv * 2
        record("prefill", n, n * T, ms, flops, nbytes, observe(step, seconds=1.2))
        del pool, ws
    del tw
    return rows


def cpu_baseline(wl, n_tokens, budget_s=10.0):
    """The fp64 oracle on the host over whole prompts of the prefill workload
    (weights regenerated by the seeded generator), prompt after prompt until
    about budget_s seconds of oracle time or all prompts are done."""
    from threadpoolctl import threadpool_info

    from oracle import layer as O
    from synth import gen as G
    w = {k: G.widen(v, "bf16") for k, v in G.layer_weights(wl, 0).items()}
    x = G.widen(G.prefill_input(wl, wl.prefill_seqs * n_tokens), "bf16")
    done, dt = 0, 0.0
    while done < wl.prefill_seqs and dt < budget_s:
        t0 = time.perf_counter()
        O.layer_sequence(w, wl.shape, x[done * n_tokens:(done + 1) * n_tokens])
        dt += time.perf_counter() - t0
        done += 1
    blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
    threads = max([p.get("num_threads", 1) for p in blas] or [1])
    model = ""
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": done * n_tokens / dt, "unit": "tok/s", "cores": threads, "kind": "oracle",
            "sample": f"{done} of the {wl.prefill_seqs} prompts x {n_tokens} tokens of the prefill workload, "
                      f"fp64 numpy, {dt:.1f} s",
            "affinity_cores": len(os.sched_getaffinity(0)), "blas_threads": threads,
            "blas": ", ".join(sorted({f"{p.get('internal_api')} {p.get('version')}" for p in blas})),
            "cpu_model": model}


def roofline_extra(bound, achieved, tel, traffic):
    """Context for a roofline line: where the peak comes from, the peak this
    device derives from its own properties, the clock the kernel actually ran
    at (the MFMA peak scales with it; MI355X under a full MFMA load runs at its
    power cap below the peak clock) and where the traffic figure comes from."""
    from paper_2608_21719_amd import accounting as A
    ex = {"peak_source": "MI355X published dense bf16 MFMA peak" if bound == "mfma" else
          "MI355X published HBM3E bandwidth"}
    if DEVICE:
        ex["device"] = {k: DEVICE[k] for k in ("compute_units", "clock_khz", "arch")}
        if bound == "mfma":
            ex["peak_derived"] = A.bf16_peak_tflops(DEVICE["compute_units"], DEVICE["clock_khz"] / 1e3)
    clk = (tel or {}).get("gfxclk_mhz") or {}
    if clk:
        ex["gfxclk_mhz_median"] = clk["median"]
        if bound == "mfma" and DEVICE:
            p = A.bf16_peak_tflops(DEVICE["compute_units"], clk["median"])
            ex["peak_at_measured_clock"] = p
            ex["frac_at_measured_clock"] = achieved / p
    pw = (tel or {}).get("power_w") or {}
    if pw:
        ex["power_w_median"] = pw["median"]
    ex["traffic_source"] = ("stored: profiles/traffic.json, two rocprofv3 --pmc passes (FETCH_SIZE, WRITE_SIZE) "
                            "scaled by a known-size copy, taken on this kernel's current source"
                            if traffic is not None else "none: no counters taken on this kernel's current source")
    return ex


def mfma_random_ceiling(seconds=2.5):
    """The matrix cores' rate on random bf16 operands that change every
    product, as a GEMM on N(0, s) data sees (the ceilings probe, run as a
    child process on this GPU, with the clock and power sampled beside it):
    the data sheet's 2.5 PFLOP/s assumes a clock that such data does not
    hold. None when the probe is not built. The window is long enough
    that the sampled medians fall in the busy part, not the child's
    start-up."""
    import re
    import subprocess
    exe = os.path.join(ROOT, "paper_2608_21719_amd", "probes", "ceilings")
    if not os.path.exists(exe):
        return None
    try:
        if TEL is not None and TEL.available:
            with TEL.leg() as rec:
                r = subprocess.run([exe, "mfma-random", str(seconds), "32x32x16"], capture_output=True, text=True,
                                   timeout=60)
            tel = rec.result
        else:
            r = subprocess.run([exe, "mfma-random", str(seconds), "32x32x16"], capture_output=True, text=True,
                               timeout=60)
            tel = None
    except (OSError, subprocess.TimeoutExpired) as e:
        return {"error": f"{type(e).__name__}: {e}"}
    m = re.search(r"random operands changing every product: (\d+) TFLOP/s", r.stdout)
    if r.returncode != 0 or not m:
        return {"error": f"probe exit {r.returncode}: {r.stderr.strip()[-200:]}"}
    out = {"tflops": float(m.group(1)), "source": "paper_2608_21719_amd/probes/ceilings mfma-random (v_mfma_f32_32x32x16_bf16, "
                                                   "one wave per SIMD, random sign and mantissa bits)"}
    if tel and tel.get("gfxclk_mhz"):
        out["gfxclk_mhz_median"] = tel["gfxclk_mhz"]["median"]
    if tel and tel.get("power_w"):
        out["power_w_median"] = tel["power_w"]["median"]
    return out


DEVICE = None  # ps_get_device_info of cuda:0, set in main


def observe(run, seconds=None):
    """GPU clock and power while the leg's work repeats (after its timed region)."""
    import torch
    seconds = TEL_SECONDS if seconds is None else seconds
    if TEL_SECONDS <= 0 or seconds <= 0:
        return {"available": False, "reason": "telemetry windows disabled (--telemetry-seconds 0)"}
    return TEL.observe(run, torch.cuda.synchronize, seconds=seconds)


def measured_traffic(kernel_key, source_file):
    """HBM bytes per launch of a kernel from profiles/traffic.json (two rocprof
    --pmc passes, FETCH_SIZE and WRITE_SIZE, scaled by a known-size copy), or
    None when the kernel's source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path)).get(kernel_key)
    if not rec:
        return None
    src = os.path.join(ROOT, source_file)
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec.get("source_sha256"):
        return None
    return rec["fetch_bytes"] + rec["write_bytes"]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=2048)
    ap.add_argument("--no-model70b", action="store_true", help="skip the 80-layer 70B-shaped model")
    ap.add_argument("--telemetry-seconds", type=float, default=1.5,
                    help="length of each leg's clock-and-power window after its timed region (0: none)")
    ap.add_argument("--phase-sweep", action="store_true",
                    help="also measure throughput, clock, power and energy per token across phases and batch sizes")
    ap.add_argument("--calib-copy", action="store_true",
                    help="run one 1 GiB device copy first (known bytes, to scale rocprof counters)")
    a = ap.parse_args()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: libps has no multi-GPU path (run with --gpus 1)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2608_21719_amd import accounting as A
    from paper_2608_21719_amd import binding as B
    from synth.configs import CONFIGS

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    global TEL, DEVICE, TEL_SECONDS
    from paper_2608_21719_amd.telemetry import Telemetry
    TEL = Telemetry(0)
    TEL_SECONDS = a.telemetry_seconds
    DEVICE = B.device_info(0)
    if a.calib_copy:
        # int32 -> fp32 conversion copy: reads exactly 1 GiB, writes exactly 1 GiB
        src = torch.ones(1 << 28, dtype=torch.int32, device="cuda")
        dst = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    pre_wl = CONFIGS["llama8b_prefill"]
    dec_wl = CONFIGS["llama8b_decode"]
    log(f"prefill: {pre_wl.note}")
    pre = bench_prefill(torch, B, A, pre_wl, a.steps, a.warmup)
    ceil = mfma_random_ceiling()
    if ceil and "tflops" in ceil:
        ceil["gate_up_frac"] = pre["roofline"]["achieved"] / ceil["tflops"]
    pre["roofline"]["mfma_ceiling_random_operands"] = ceil
    log(f"prefill: {pre['tok_s']:.0f} tok/s, {pre['ms_per_step']:.3f} ms/step, gate_up {pre['gate_up_gemm']['tflops']:.0f} TFLOP/s")
    torch.cuda.empty_cache()
    dec = None
    if not a.no_decode:
        log(f"decode: {dec_wl.note}")
        dec = bench_decode(torch, B, A, dec_wl, max(a.steps, 16), a.warmup)
        log(f"decode: {dec['tok_s']:.0f} tok/s, {dec['ms_per_step'] * 1e3:.1f} us/step, "
            f"attention {dec['attention']['gbs']:.0f} GB/s")
    think = None
    if not a.no_decode:
        th_wl = CONFIGS["llama8b_think"]
        log(f"think: {th_wl.note}")
        think = bench_think(torch, B, A, th_wl, max(a.steps, 16), a.warmup)
        log(f"think: {think['tok_s']:.0f} tok/s, attention {think['attention']['gbs']:.0f} GB/s, "
            f"mixed step {think['mixed_step']['ms']:.3f} ms")
        torch.cuda.empty_cache()
    m70 = None
    if not a.no_model70b:
        m_wl = CONFIGS["llama70b_model"]
        log(f"model70b: {m_wl.note}")
        m70 = bench_model70b(torch, B, A, m_wl, max(4, a.steps // 2), 2)
        log(f"model70b: decode {m70['decode']['tok_s']:.0f} tok/s ({m70['decode']['ms_per_step']:.1f} ms/step, "
            f"{m70['decode']['hbm_gbs']:.0f} GB/s), prefill {m70['prefill']['tok_s']:.0f} tok/s")
        torch.cuda.empty_cache()
    sweep = None
    if a.phase_sweep:
        log("phase sweep: 8B-shaped layer, decode B in {1..256} at context 2048, prefill n x 2048")
        sweep = phase_sweep(torch, B, A, CONFIGS["llama8b_decode"])
        torch.cuda.empty_cache()
    cpu = None
    if not a.no_cpu_baseline:
        log("cpu baseline: fp64 oracle on the host")
        cpu = cpu_baseline(pre_wl, a.cpu_tokens)
    line = {
        "metric": METRIC, "value": pre["tok_s"], "unit": "tok/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": pre["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "8B-shaped layer prefill, 8 prompts x 2048 tokens (hidden 4096, 32 q / 8 kv "
                               "heads, head_dim 128, SwiGLU 14336), bf16 weights/activations, fp32 accumulate",
                   "global_batch": 8, "seq_len": 2048, "parallelism": "single GPU"},
        "roofline": pre["roofline"],
        "device": dict(DEVICE, bf16_peak_derived_tflops=A.bf16_peak_tflops(DEVICE["compute_units"],
                                                                            DEVICE["clock_khz"] / 1e3),
                       telemetry=TEL.static_info()),
        "prefill": {k: v for k, v in pre.items() if k != "roofline"},
        "decode": dec,
        "think": think,
        "model70b": m70,
        "cpu_baseline": cpu,
    }
    if sweep is not None:
        line["phase_sweep"] = sweep
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
