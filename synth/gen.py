"""Seeded generators for weights, activations, KV history and context lengths.

Every draw comes from ``numpy.random.Generator(PCG64(SeedSequence(0,
spawn_key=(cfg_id, layer, tensor_code, step))))`` so that any tensor can be
regenerated on its own, on any machine, without generating the others.
Normals are drawn in float32 and, for bf16 workloads, rounded to bf16 with
round-to-nearest-even; the result is kept as raw uint16 bit patterns. Both the
oracle (after widening to float64) and the device path consume exactly these
bits.
"""
import numpy as np

from .configs import PAGE_TOKENS, LayerShape, Workload

# tensor codes for the seed's spawn key
T_ATTN_NORM, T_WQ, T_WK, T_WV, T_WO, T_FFN_NORM, T_WG, T_WU, T_WD = range(1, 10)
T_EMBED, T_FINAL_NORM, T_LM_HEAD = 10, 11, 12
T_X_PREFILL, T_X_DECODE, T_K_HIST, T_V_HIST, T_CTX, T_TOKENS, T_X_MIXED = range(20, 27)
T_PAGE_SEED = 30

WEIGHT_STD = 0.02
BASE_SEED = 0


def rng(cfg_id: int, layer: int, code: int, step: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence(BASE_SEED, spawn_key=(cfg_id, layer, code, step))
    return np.random.Generator(np.random.PCG64(ss))


# ---------------------------------------------------------------- bf16 bits
def f32_to_bf16_bits(a) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bits.

    Inputs are finite draws, so NaN handling is not needed here.
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_storage(a_f32: np.ndarray, dtype: str) -> np.ndarray:
    """float32 draw -> storage array (float32, or uint16 bf16 bits)."""
    if dtype == "f32":
        return np.ascontiguousarray(a_f32, dtype=np.float32)
    if dtype == "bf16":
        return f32_to_bf16_bits(a_f32)
    raise ValueError(dtype)


def widen(a: np.ndarray, dtype: str) -> np.ndarray:
    """Storage array -> float64 (exact)."""
    if dtype == "bf16":
        return bf16_bits_to_f32(a).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def normal(shape, std: float, dtype: str, cfg_id: int, layer: int, code: int, step: int = 0,
           mean: float = 0.0) -> np.ndarray:
    g = rng(cfg_id, layer, code, step)
    a = g.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    if mean != 0.0:
        a += np.float32(mean)
    return to_storage(a, dtype)


# ---------------------------------------------------------------- weights
def _draw(specs: dict) -> dict:
    """normal() for each named spec, the tensors drawn in parallel threads.

    Each tensor has its own generator (its own spawn key), so the bits do not
    depend on the order or the thread that draws them; numpy's bulk draws and
    the bf16 rounding release the GIL.
    """
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=min(8, len(specs))) as ex:
        futs = {k: ex.submit(normal, *args, **kw) for k, (args, kw) in specs.items()}
        return {k: f.result() for k, f in futs.items()}


def layer_weights(wl: Workload, layer: int = 0) -> dict:
    """One layer's parameters, nn.Linear convention W[out, in].

    Projections ~ N(0, 0.02^2); RMSNorm gains ~ 1 + N(0, 0.02^2).
    """
    s: LayerShape = wl.shape
    c, dt = wl.cfg_id, s.dtype
    d, dq, dkv, f = s.hidden, s.d_q, s.d_kv, s.ffn
    return _draw({
        "attn_norm": (((d,), WEIGHT_STD, dt, c, layer, T_ATTN_NORM), {"mean": 1.0}),
        "wq": (((dq, d), WEIGHT_STD, dt, c, layer, T_WQ), {}),
        "wk": (((dkv, d), WEIGHT_STD, dt, c, layer, T_WK), {}),
        "wv": (((dkv, d), WEIGHT_STD, dt, c, layer, T_WV), {}),
        "wo": (((d, dq), WEIGHT_STD, dt, c, layer, T_WO), {}),
        "ffn_norm": (((d,), WEIGHT_STD, dt, c, layer, T_FFN_NORM), {"mean": 1.0}),
        "wg": (((f, d), WEIGHT_STD, dt, c, layer, T_WG), {}),
        "wu": (((f, d), WEIGHT_STD, dt, c, layer, T_WU), {}),
        "wd": (((d, f), WEIGHT_STD, dt, c, layer, T_WD), {}),
    })


def model_head_weights(wl: Workload) -> dict:
    s = wl.shape
    c, dt = wl.cfg_id, s.dtype
    return _draw({
        "embed": (((wl.vocab, s.hidden), WEIGHT_STD, dt, c, 0, T_EMBED), {}),
        "final_norm": (((s.hidden,), WEIGHT_STD, dt, c, 0, T_FINAL_NORM), {"mean": 1.0}),
        "lm_head": (((wl.vocab, s.hidden), WEIGHT_STD, dt, c, 0, T_LM_HEAD), {}),
    })


# ---------------------------------------------------------------- activations
def prefill_input(wl: Workload, n_tokens: int, layer: int = 0, step: int = 0) -> np.ndarray:
    """Layer input rows x ~ N(0, 1) for a prefill of n_tokens rows in total."""
    s = wl.shape
    return normal((n_tokens, s.hidden), 1.0, s.dtype, wl.cfg_id, layer, T_X_PREFILL, step)


def decode_input(wl: Workload, batch: int, step: int, layer: int = 0) -> np.ndarray:
    """Fresh N(0, 1) rows for one decode step of a single layer."""
    s = wl.shape
    return normal((batch, s.hidden), 1.0, s.dtype, wl.cfg_id, layer, T_X_DECODE, step)


def mixed_input(wl: Workload, n_rows: int, layer: int = 0) -> np.ndarray:
    s = wl.shape
    return normal((n_rows, s.hidden), 1.0, s.dtype, wl.cfg_id, layer, T_X_MIXED)


def kv_history(wl: Workload, layer: int, seq: int, length: int):
    """Synthetic cached K and V (treated as already rotated), N(0, 1).

    Shapes [length, n_kv, head_dim] each, storage dtype of the workload.
    """
    s = wl.shape
    shp = (length, s.n_kv, s.head_dim)
    k = normal(shp, 1.0, s.dtype, wl.cfg_id, layer, T_K_HIST, seq)
    v = normal(shp, 1.0, s.dtype, wl.cfg_id, layer, T_V_HIST, seq)
    return k, v


def context_lengths(wl: Workload) -> np.ndarray:
    """Per-sequence KV length before the first decode step."""
    g = rng(wl.cfg_id, 0, T_CTX)
    b = wl.decode_batch
    if wl.ctx_law == "uniform":
        lo, hi = wl.ctx_params
        return g.integers(lo, hi + 1, size=b).astype(np.int64)
    if wl.ctx_law == "lognormal":
        median, sigma, lo, hi = wl.ctx_params
        raw = np.exp(np.log(median) + sigma * g.standard_normal(b))
        return np.clip(np.rint(raw), lo, hi).astype(np.int64)
    if wl.ctx_law == "fixed":
        return np.full(b, wl.ctx_params[0], dtype=np.int64)
    if wl.ctx_law == "after_prefill":
        return np.full(b, wl.prefill_tokens, dtype=np.int64)
    raise ValueError(wl.ctx_law)


def token_ids(wl: Workload, n: int, step: int = 0) -> np.ndarray:
    return rng(wl.cfg_id, 0, T_TOKENS, step).integers(0, wl.vocab, size=n).astype(np.int32)


def pages_needed(tokens: int) -> int:
    return (tokens + PAGE_TOKENS - 1) // PAGE_TOKENS


def page_order_seed(wl: Workload) -> int:
    """Seed for the KV pool's free-page permutation (0 means identity order)."""
    if not wl.shuffled_pages:
        return 0
    return int(rng(wl.cfg_id, 0, T_PAGE_SEED).integers(1, 2**63 - 1))


# ---------------------------------------------------------------- request traces
def request_trace(seed: int, n: int, rate: float, ctx_range=(32, 512), median: float = 300.0,
                  sigma: float = 1.0, len_range=(16, 4000)):
    """Synthetic arrivals for one stage pool: arrival step (Poisson, `rate`
    per step), context tokens already held (uniform integers in ctx_range)
    and the tokens the stage will produce (log-normal, heavy-tailed like the
    reasoning lengths the paper describes, rounded and clipped to len_range).
    Random draws only."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(BASE_SEED, spawn_key=(99, seed))))
    gaps = g.exponential(1.0 / rate, size=n)
    arrival = np.floor(np.cumsum(gaps)).astype(np.int64)
    ctx = g.integers(ctx_range[0], ctx_range[1] + 1, size=n).astype(np.int64)
    raw = np.exp(np.log(median) + sigma * g.standard_normal(n))
    length = np.clip(np.rint(raw), len_range[0], len_range[1]).astype(np.int64)
    return arrival, ctx, length
