"""ctypes binding of libps (include/ps.h): argument marshalling only.

Every computation runs in the HIP kernels of libps.so; this module converts
Python arguments to C types, passes device pointers and the caller's HIP
stream through, and turns non-zero status codes into exceptions. torch is
used for device memory and streams only (``data_ptr()``, ``cuda_stream``).

Importing this module loads the library and raises ``LibraryMissing`` when it
has not been built: there is no fallback path.
"""
import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int32, c_size_t, c_uint64, c_void_p

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libps.so")

PS_OK, PS_E_INVALID, PS_E_NO_PAGES, PS_E_CAPACITY, PS_E_HIP, PS_E_UNSUPPORTED = range(6)
PS_F32, PS_BF16 = 0, 1
PS_PHASE_PREFILL, PS_PHASE_THINK, PS_PHASE_ANSWER = 0, 1, 2
PS_EPI_STORE, PS_EPI_RESIDUAL, PS_EPI_SWIGLU = 0, 1, 2
PAGE_TOKENS = 16
GATE_UP_BLOCK = 32


class LibraryMissing(RuntimeError):
    pass


class PsError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"libps status {code}: {msg}")
        self.code = code


class LayerCfg(ctypes.Structure):
    _fields_ = [("hidden", c_int32), ("n_q_heads", c_int32), ("n_kv_heads", c_int32), ("head_dim", c_int32),
                ("ffn", c_int32), ("rms_eps", c_float), ("rope_theta", c_double), ("dtype", c_int32)]


class DeviceInfo(ctypes.Structure):
    _fields_ = [("compute_units", c_int32), ("clock_khz", c_int32), ("memory_clock_khz", c_int32),
                ("memory_bus_bits", c_int32), ("total_memory", ctypes.c_int64), ("l2_bytes", c_int32),
                ("lds_bytes_per_block", c_int32), ("arch", ctypes.c_char * 64)]


class SchedCfg(ctypes.Structure):
    _fields_ = [("window", c_int32), ("cs_initial", c_int32), ("cs_min", c_int32), ("cs_max", c_int32)]


class PsoptGroup(ctypes.Structure):
    _fields_ = [(n, c_double) for n in ("w", "delta", "k", "nu", "c", "gamma", "lam", "sigma", "c2", "c1", "c0")]


class PsoptResult(ctypes.Structure):
    _fields_ = [("f", c_double), ("eta", c_double), ("impact", c_double), ("rank", c_double), ("f_step", c_int32)]


DVFS_LOCK_FN = ctypes.CFUNCTYPE(c_int32, c_void_p, c_int32)
DVFS_LIMIT_FN = ctypes.CFUNCTYPE(c_int32, c_void_p, c_int32)


class LayerW(ctypes.Structure):
    _fields_ = [("attn_norm", c_void_p), ("w_qkv", c_void_p), ("w_o", c_void_p), ("ffn_norm", c_void_p),
                ("w_gate_up", c_void_p), ("w_down", c_void_p)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise LibraryMissing(f"{LIB_PATH} is not built; run `python -m paper_2608_21719_amd.build`")
    # torch ships its own HIP runtime under the same soname (libamdhip64.so.7).
    # Load it first so that libps binds to the runtime that owns torch's
    # device allocations and streams; a second runtime in the process would
    # not see the device.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    return ctypes.CDLL(LIB_PATH)


lib = _load()

_I = c_int32
_P = c_void_p
_IP = POINTER(c_int32)
_SIGS = {
    "ps_last_error": (c_char_p, []),
    "ps_version": (c_char_p, []),
    "ps_get_device_info": (_I, [_I, POINTER(DeviceInfo)]),
    "ps_pack_gate_up": (_I, [_P, _P, _I, _I, _I, _P]),
    "ps_tiled_weight_elems": (c_size_t, [_I, _I]),
    "ps_tile_weight": (_I, [_P, _I, _I, _I, _P]),
    "ps_op_tile_weight": (_I, [_I, _I, _I, _P, _P, _P]),
    "ps_kv_pool_bytes": (c_size_t, [POINTER(LayerCfg), _I, _I]),
    "ps_kv_create": (_I, [POINTER(LayerCfg), _I, _I, _I, _I, _P, c_uint64, POINTER(c_void_p)]),
    "ps_kv_destroy": (_I, [_P]),
    "ps_kv_seq_open": (_I, [_P, _IP]),
    "ps_kv_alloc": (_I, [_P, _I, _I]),
    "ps_kv_commit": (_I, [_P, _I, _IP, _IP]),
    "ps_kv_truncate": (_I, [_P, _I, _I]),
    "ps_kv_free": (_I, [_P, _I]),
    "ps_kv_seq_len": (_I, [_P, _I, _IP]),
    "ps_kv_capacity": (_I, [_P, _I, _IP]),
    "ps_kv_free_pages": (_I, [_P, _IP]),
    "ps_kv_block_table": (_I, [_P, _I, _IP, _I, _IP]),
    "ps_kv_append": (_I, [_P, _I, _I, _IP, _IP, _P, _P, _P, c_size_t, _P]),
    "ps_kv_gather": (_I, [_P, _I, _I, _P, _P, _P, c_size_t, _P]),
    "ps_kv_transfer": (_I, [_P, _I, _P, _I, _P, c_size_t, _P]),
    "ps_sched_create": (_I, [_P, POINTER(SchedCfg), POINTER(c_void_p)]),
    "ps_sched_destroy": (_I, [_P]),
    "ps_sched_chunk_size": (_I, [_P, _IP]),
    "ps_sched_running": (_I, [_P, _IP]),
    "ps_sched_admit": (_I, [_P, _I, _IP]),
    "ps_sched_reserve_step": (_I, [_P, _I, _IP, _IP, _IP, _I, _IP]),
    "ps_sched_finish": (_I, [_P, _I, _I]),
    "ps_dvfs_create": (_I, [POINTER(c_int32), _I, c_double, c_double, _I, _I, DVFS_LOCK_FN, DVFS_LIMIT_FN, _P,
                            POINTER(c_void_p)]),
    "ps_dvfs_destroy": (_I, [_P]),
    "ps_dvfs_vote": (_I, [_P, ctypes.c_int64, _I, c_double]),
    "ps_dvfs_retract": (_I, [_P, ctypes.c_int64]),
    "ps_dvfs_tick": (_I, [_P, _IP, _IP]),
    "ps_dvfs_start": (_I, [_P, _I]),
    "ps_dvfs_stop": (_I, [_P]),
    "ps_psopt_solve": (_I, [POINTER(PsoptGroup), _I, c_double, c_double, c_double, c_double, POINTER(c_int32), _I,
                            POINTER(PsoptResult), POINTER(c_double), POINTER(c_double), POINTER(c_double)]),
    "ps_layer_create": (_I, [POINTER(LayerCfg), POINTER(c_void_p)]),
    "ps_layer_destroy": (_I, [_P]),
    "ps_workspace_bytes": (c_size_t, [POINTER(LayerCfg), _I, _I, _I]),
    "ps_prefill": (_I, [_P, POINTER(LayerW), _P, _I, _I, _IP, _IP, _P, _P, _P, c_size_t, _P]),
    "ps_decode_step": (_I, [_P, POINTER(LayerW), _P, _I, _I, _I, _IP, _P, _P, _P, c_size_t, _P]),
    "ps_mixed_step": (_I, [_P, POINTER(LayerW), _P, _I, _I, _IP, _IP, _I, _IP, _P, _P, _P, c_size_t, _P]),
    "ps_op_rmsnorm": (_I, [_I, _I, _I, _I, _I, _P, _P, c_float, _P, _P]),
    "ps_op_gemm_workspace_bytes": (c_size_t, [_I, _I, _I, _I]),
    "ps_op_gemm": (_I, [_I, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, c_size_t, _P]),
    "ps_op_gemm_static": (_I, [_I, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P]),
    "ps_op_rope_kvwrite": (_I, [_P, _I, _I, _IP, _IP, _P, _P, _P, c_size_t, _P]),
    "ps_op_gemm_static": (_I, [_I, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P]),
    "ps_op_attention": (_I, [_P, _I, _I, _IP, _IP, _P, _P, _P, c_size_t, _P]),
    "ps_op_decode_attention": (_I, [_P, _I, _I, _IP, _P, _P, _I, _P, c_size_t, _P]),
    "ps_op_decode_plan": (_I, [_P, _I, _IP, _I, _P, c_size_t, _P]),
    "ps_op_decode_run": (_I, [_P, _I, _P, _P, _P, c_size_t, _P]),
    "ps_op_decode_run_capped": (_I, [_P, _I, _P, _P, _P, c_size_t, _I, _P]),
    "ps_op_argmax": (_I, [_I, _I, _P, _P, _P]),
    "ps_model_create": (_I, [POINTER(LayerCfg), _I, _I, _P, POINTER(LayerW), _P, _P, POINTER(c_void_p)]),
    "ps_model_destroy": (_I, [_P]),
    "ps_model_workspace_bytes": (c_size_t, [POINTER(LayerCfg), _I, _I, _I, _I]),
    "ps_model_prefill": (_I, [_P, _P, _I, _IP, _IP, _P, _P, _P, _P, c_size_t, _P]),
    "ps_model_decode_step": (_I, [_P, _P, _I, _I, _IP, _P, _P, _P, _P, c_size_t, _P]),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def last_error() -> str:
    return lib.ps_last_error().decode()


def check(rc: int):
    if rc != PS_OK:
        raise PsError(rc, last_error())


def device_info(device: int = 0) -> dict:
    info = DeviceInfo()
    check(lib.ps_get_device_info(device, ctypes.byref(info)))
    return {f: (getattr(info, f).decode() if f == "arch" else getattr(info, f)) for f, _ in DeviceInfo._fields_}


def ints(seq):
    arr = (c_int32 * len(seq))(*[int(x) for x in seq])
    return arr


def ptr(t):
    """Device (or host) address of a torch tensor / numpy array / int / None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if hasattr(t, "data_ptr"):
        return t.data_ptr()
    if hasattr(t, "ctypes"):
        return t.ctypes.data
    raise TypeError(type(t))


def stream_handle(stream=None):
    """The caller's HIP stream: an explicit handle, a torch stream, or torch's current stream."""
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def make_cfg(shape) -> LayerCfg:
    """LayerCfg from an object with hidden, n_q, n_kv, head_dim, ffn, eps, theta, dtype."""
    return LayerCfg(shape.hidden, shape.n_q, shape.n_kv, shape.head_dim, shape.ffn, shape.eps, shape.theta,
                    PS_BF16 if shape.dtype == "bf16" else PS_F32)


def pack_gate_up(wg, wu):
    """Host numpy interleave of Wg, Wu [F, d] into the w_gate_up row order."""
    import numpy as np
    wg = np.ascontiguousarray(wg)
    wu = np.ascontiguousarray(wu)
    F, d = wg.shape
    out = np.empty((2 * F, d), dtype=wg.dtype)
    check(lib.ps_pack_gate_up(ptr(wg), ptr(wu), F, d, wg.itemsize, ptr(out)))
    return out


def tiled_weight_elems(N: int, K: int) -> int:
    return lib.ps_tiled_weight_elems(N, K)


def tile_weight(w):
    """Host numpy conversion of a row-major [N, K] weight to the tiled layout
    (a flat array of tiled_weight_elems(N, K) elements)."""
    import numpy as np
    w = np.ascontiguousarray(w)
    N, K = w.shape
    out = np.empty(tiled_weight_elems(N, K), dtype=w.dtype)
    check(lib.ps_tile_weight(ptr(w), N, K, w.itemsize, ptr(out)))
    return out


def op_tile_weight(dtype, N, K, w, out, stream=None):
    """Device conversion of a row-major [N, K] weight to the tiled layout."""
    check(lib.ps_op_tile_weight(dtype, N, K, ptr(w), ptr(out), stream_handle(stream)))


# ---------------------------------------------------------------- handles
class KV:
    """Paged KV pool metadata over a caller-owned device pool."""

    def __init__(self, cfg: LayerCfg, n_layers: int, n_pages: int, max_seqs: int, max_pages_per_seq: int,
                 pool, seed: int = 0):
        self.cfg = cfg
        self.n_layers = n_layers
        self.pool = pool  # keep the owner alive
        h = c_void_p()
        check(lib.ps_kv_create(ctypes.byref(cfg), n_layers, n_pages, max_seqs, max_pages_per_seq, ptr(pool),
                               c_uint64(seed), ctypes.byref(h)))
        self.h = h

    @staticmethod
    def pool_bytes(cfg: LayerCfg, n_layers: int, n_pages: int) -> int:
        return lib.ps_kv_pool_bytes(ctypes.byref(cfg), n_layers, n_pages)

    def close(self):
        if self.h:
            check(lib.ps_kv_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def open(self) -> int:
        s = c_int32()
        check(lib.ps_kv_seq_open(self.h, ctypes.byref(s)))
        return s.value

    def alloc(self, seq: int, n_tokens: int):
        check(lib.ps_kv_alloc(self.h, seq, n_tokens))

    def commit(self, seqs, n_tok):
        check(lib.ps_kv_commit(self.h, len(seqs), ints(seqs), ints(n_tok)))

    def truncate(self, seq: int, new_len: int):
        check(lib.ps_kv_truncate(self.h, seq, new_len))

    def free(self, seq: int):
        check(lib.ps_kv_free(self.h, seq))

    def seq_len(self, seq: int) -> int:
        n = c_int32()
        check(lib.ps_kv_seq_len(self.h, seq, ctypes.byref(n)))
        return n.value

    def capacity(self, seq: int) -> int:
        n = c_int32()
        check(lib.ps_kv_capacity(self.h, seq, ctypes.byref(n)))
        return n.value

    def free_pages(self) -> int:
        n = c_int32()
        check(lib.ps_kv_free_pages(self.h, ctypes.byref(n)))
        return n.value

    def block_table(self, seq: int):
        n = c_int32()
        check(lib.ps_kv_block_table(self.h, seq, None, 0, ctypes.byref(n)))
        buf = (c_int32 * max(1, n.value))()
        check(lib.ps_kv_block_table(self.h, seq, buf, n.value, ctypes.byref(n)))
        return list(buf[:n.value])

    def append(self, layer, seqs, n_tok, k, v, ws, stream=None):
        check(lib.ps_kv_append(self.h, layer, len(seqs), ints(seqs), ints(n_tok), ptr(k), ptr(v), ptr(ws),
                               ws.numel() * ws.element_size(), stream_handle(stream)))

    def gather(self, layer, seq, k_out, v_out, ws, stream=None):
        check(lib.ps_kv_gather(self.h, layer, seq, ptr(k_out), ptr(v_out), ptr(ws),
                               ws.numel() * ws.element_size(), stream_handle(stream)))


def kv_transfer(src: KV, src_seq: int, dst: KV, dst_seq: int, ws, stream=None):
    """Copy a sequence's KV state (every layer) from pool src to pool dst (think -> answer handoff)."""
    check(lib.ps_kv_transfer(src.h, src_seq, dst.h, dst_seq, ptr(ws), ws.numel() * ws.element_size(),
                             stream_handle(stream)))


class Sched:
    """Per-stage KV reservation and admission by observed lengths over one pool."""

    def __init__(self, kv: KV, window: int, cs_initial: int, cs_min: int, cs_max: int):
        self.kv = kv
        self.cfg = SchedCfg(window, cs_initial, cs_min, cs_max)
        h = c_void_p()
        check(lib.ps_sched_create(kv.h, ctypes.byref(self.cfg), ctypes.byref(h)))
        self.h = h
        self._cap = 0

    def close(self):
        if self.h:
            check(lib.ps_sched_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def chunk_size(self) -> int:
        v = c_int32()
        check(lib.ps_sched_chunk_size(self.h, ctypes.byref(v)))
        return v.value

    def running(self) -> int:
        v = c_int32()
        check(lib.ps_sched_running(self.h, ctypes.byref(v)))
        return v.value

    def admit(self, ctx_tokens: int):
        """Sequence id, or None when the request does not fit now."""
        v = c_int32()
        check(lib.ps_sched_admit(self.h, ctx_tokens, ctypes.byref(v)))
        return None if v.value < 0 else v.value

    def reserve_step(self, seqs, n_tok, max_seqs: int):
        buf = (c_int32 * max(1, max_seqs))()
        n = c_int32()
        check(lib.ps_sched_reserve_step(self.h, len(seqs), ints(seqs), ints(n_tok), buf, max_seqs, ctypes.byref(n)))
        return list(buf[:n.value])

    def finish(self, seq: int, stage_tokens: int):
        check(lib.ps_sched_finish(self.h, seq, stage_tokens))


class Dvfs:
    """Vote-commit DVFS daemon; lock(mhz) and limit(watts) are Python
    callables (the actuators), called from the ticking thread."""

    def __init__(self, ladder, under_weight, over_weight, power_limit_w, initial_mhz, lock=None, limit=None):
        self._lock = DVFS_LOCK_FN(lambda ctx, mhz: int(lock(mhz) or 0) if lock else 0)
        self._limit = DVFS_LIMIT_FN(lambda ctx, w: int(limit(w) or 0) if limit else 0)
        arr = (c_int32 * len(ladder))(*ladder)
        h = c_void_p()
        check(lib.ps_dvfs_create(arr, len(ladder), under_weight, over_weight, power_limit_w, initial_mhz, self._lock,
                                 self._limit, None, ctypes.byref(h)))
        self.h = h

    def close(self):
        if self.h:
            check(lib.ps_dvfs_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def vote(self, request: int, target_mhz: int, weight: float):
        check(lib.ps_dvfs_vote(self.h, request, target_mhz, weight))

    def retract(self, request: int):
        check(lib.ps_dvfs_retract(self.h, request))

    def tick(self):
        f, ch = c_int32(), c_int32()
        check(lib.ps_dvfs_tick(self.h, ctypes.byref(f), ctypes.byref(ch)))
        return f.value, bool(ch.value)

    def start(self, period_ms: int):
        check(lib.ps_dvfs_start(self.h, period_ms))

    def stop(self):
        check(lib.ps_dvfs_stop(self.h))


def psopt_solve(groups, p_max, f_min, f_max, ladder, dt=0.0):
    """groups: list of dicts with the PsoptGroup fields. Returns (results,
    mu, relaxed power, projected power, status) without raising on PS_E_CAPACITY."""
    n = len(groups)
    g = (PsoptGroup * n)(*[PsoptGroup(*[float(x[f]) for f, _ in PsoptGroup._fields_]) for x in groups])
    out = (PsoptResult * n)()
    lad = (c_int32 * len(ladder))(*ladder)
    mu, pr, pp = c_double(), c_double(), c_double()
    rc = lib.ps_psopt_solve(g, n, p_max, f_min, f_max, dt, lad, len(ladder), out, ctypes.byref(mu), ctypes.byref(pr),
                            ctypes.byref(pp))
    if rc not in (PS_OK, PS_E_CAPACITY):
        check(rc)
    res = [{"f": r.f, "eta": r.eta, "impact": r.impact, "rank": r.rank, "f_step": r.f_step} for r in out]
    return res, mu.value, pr.value, pp.value, rc


class Layer:
    def __init__(self, cfg: LayerCfg):
        self.cfg = cfg
        h = c_void_p()
        check(lib.ps_layer_create(ctypes.byref(cfg), ctypes.byref(h)))
        self.h = h

    def close(self):
        if self.h:
            check(lib.ps_layer_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @staticmethod
    def workspace_bytes(cfg, max_rows, max_seqs, max_pages_per_seq) -> int:
        return lib.ps_workspace_bytes(ctypes.byref(cfg), max_rows, max_seqs, max_pages_per_seq)

    def prefill(self, w: LayerW, kv: KV, layer, seqs, n_tok, x_in, x_out, ws, stream=None):
        check(lib.ps_prefill(self.h, ctypes.byref(w), kv.h, layer, len(seqs), ints(seqs), ints(n_tok), ptr(x_in),
                             ptr(x_out), ptr(ws), ws.numel() * ws.element_size(), stream_handle(stream)))

    def decode_step(self, w: LayerW, kv: KV, layer, phase, seqs, x_in, x_out, ws, stream=None):
        check(lib.ps_decode_step(self.h, ctypes.byref(w), kv.h, layer, phase, len(seqs), ints(seqs), ptr(x_in),
                                 ptr(x_out), ptr(ws), ws.numel() * ws.element_size(), stream_handle(stream)))

    def mixed_step(self, w: LayerW, kv: KV, layer, chunk_seqs, chunk_tok, dec_seqs, x_in, x_out, ws, stream=None):
        check(lib.ps_mixed_step(self.h, ctypes.byref(w), kv.h, layer, len(chunk_seqs), ints(chunk_seqs),
                                ints(chunk_tok), len(dec_seqs), ints(dec_seqs), ptr(x_in), ptr(x_out), ptr(ws),
                                ws.numel() * ws.element_size(), stream_handle(stream)))


class Model:
    """n_layers stacked layers + embedding, final norm, LM head, greedy argmax."""

    def __init__(self, cfg: LayerCfg, layers, vocab: int, embed, final_norm, lm_head):
        self.cfg = cfg
        self.n_layers = len(layers)
        self.keep = (layers, embed, final_norm, lm_head)
        arr = (LayerW * len(layers))(*layers)
        self._arr = arr
        h = c_void_p()
        check(lib.ps_model_create(ctypes.byref(cfg), len(layers), vocab, ptr(embed), arr, ptr(final_norm),
                                  ptr(lm_head), ctypes.byref(h)))
        self.h = h
        self.vocab = vocab

    def close(self):
        if self.h:
            check(lib.ps_model_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @staticmethod
    def workspace_bytes(cfg, vocab, max_rows, max_seqs, max_pages_per_seq) -> int:
        return lib.ps_model_workspace_bytes(ctypes.byref(cfg), vocab, max_rows, max_seqs, max_pages_per_seq)

    def prefill(self, kv: "KV", seqs, n_tok, tokens, next_tok, ws, logits=None, stream=None):
        check(lib.ps_model_prefill(self.h, kv.h, len(seqs), ints(seqs), ints(n_tok), ptr(tokens), ptr(next_tok),
                                   ptr(logits), ptr(ws), ws.numel() * ws.element_size(), stream_handle(stream)))

    def decode_step(self, kv: "KV", phase, seqs, tokens, next_tok, ws, logits=None, stream=None):
        check(lib.ps_model_decode_step(self.h, kv.h, phase, len(seqs), ints(seqs), ptr(tokens), ptr(next_tok),
                                       ptr(logits), ptr(ws), ws.numel() * ws.element_size(), stream_handle(stream)))


def op_argmax(rows, vocab, logits, next_tok, stream=None):
    check(lib.ps_op_argmax(rows, vocab, ptr(logits), ptr(next_tok), stream_handle(stream)))


def layer_weights(attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down) -> LayerW:
    return LayerW(ptr(attn_norm), ptr(w_qkv), ptr(w_o), ptr(ffn_norm), ptr(w_gate_up), ptr(w_down))


# ---------------------------------------------------------------- single ops
def op_rmsnorm(x_dt, g_dt, y_dt, rows, d, x, g, eps, y, stream=None):
    check(lib.ps_op_rmsnorm(x_dt, g_dt, y_dt, rows, d, ptr(x), ptr(g), eps, ptr(y), stream_handle(stream)))


def op_gemm_workspace_bytes(dtype, M, N, K) -> int:
    return lib.ps_op_gemm_workspace_bytes(dtype, M, N, K)


def op_gemm(dtype, r_dt, c_dt, epi, M, N, K, A, W, R, C, ws=None, stream=None):
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    check(lib.ps_op_gemm(dtype, r_dt, c_dt, epi, M, N, K, ptr(A), ptr(W), ptr(R), ptr(C), ptr(ws), wsb,
                         stream_handle(stream)))


def op_gemm_static(dtype, r_dt, c_dt, epi, M, N, K, A, W, R, C, stream=None):
    """ps_op_gemm with split-K partials in the library's static device array (no workspace)."""
    check(lib.ps_op_gemm_static(dtype, r_dt, c_dt, epi, M, N, K, ptr(A), ptr(W), ptr(R), ptr(C),
                                stream_handle(stream)))


def op_rope_kvwrite(kv: KV, layer, seqs, n_tok, qkv, q_out, ws, stream=None):
    check(lib.ps_op_rope_kvwrite(kv.h, layer, len(seqs), ints(seqs), ints(n_tok), ptr(qkv), ptr(q_out), ptr(ws),
                                 ws.numel() * ws.element_size(), stream_handle(stream)))


def op_attention(kv: KV, layer, seqs, n_tok, q, o, ws, stream=None):
    check(lib.ps_op_attention(kv.h, layer, len(seqs), ints(seqs), ints(n_tok), ptr(q), ptr(o), ptr(ws),
                              ws.numel() * ws.element_size(), stream_handle(stream)))


def op_decode_attention(kv: KV, layer, seqs, q, o, ws, split_pages=0, stream=None):
    check(lib.ps_op_decode_attention(kv.h, layer, len(seqs), ints(seqs), ptr(q), ptr(o), split_pages, ptr(ws),
                                     ws.numel() * ws.element_size(), stream_handle(stream)))


def op_decode_plan(kv: KV, seqs, ws, split_pages=0, stream=None):
    check(lib.ps_op_decode_plan(kv.h, len(seqs), ints(seqs), split_pages, ptr(ws), ws.numel() * ws.element_size(),
                                stream_handle(stream)))


def op_decode_run(kv: KV, layer, q, o, ws, stream=None):
    check(lib.ps_op_decode_run(kv.h, layer, ptr(q), ptr(o), ptr(ws), ws.numel() * ws.element_size(),
                               stream_handle(stream)))


def op_decode_run_capped(kv: KV, layer, q, o, ws, max_workgroups, stream=None):
    check(lib.ps_op_decode_run_capped(kv.h, layer, ptr(q), ptr(o), ptr(ws), ws.numel() * ws.element_size(),
                                      max_workgroups, stream_handle(stream)))
