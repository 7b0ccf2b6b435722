"""Test-side plumbing: moving seeded inputs to the device and back.

No arithmetic of the method lives here: the expected values come from
``oracle`` and the computed values from libps through its binding.
"""
import numpy as np

from synth import gen

BF16_TOL_ABS, BF16_TOL_REL = 2e-2, 1e-2      # stage-level bound for bf16 outputs
F32_TOL_ABS, F32_TOL_REL = 1e-4, 1e-4        # fp32 layer bound
# End-to-end bf16 layer bounds (normwise max|g-r|/max|r| and rms(g-r)/rms(r)).
# A float32 model with bf16 rounding at exactly the device's rounding points
# (tests/bf16_emulation.py) sets the floor any such pipeline reaches against
# the fp64 oracle; a bound is that floor times TOL_MARGIN, which covers the
# device's different fp32 summation order and the spread of the max-based
# metric between inputs (tests/test_tolerance.py recomputes the floors).
TOL_MARGIN = 1.3
NORMWISE_TOL = 1e-2                           # d = 4096: floor 5.8e-3, so 1e-2 holds with room
NORMWISE_FLOOR_70B = 1.152e-2                 # d = 8192, F = 28672: the floor on the 256-token prompt
NORMWISE_TOL_70B = 1.5e-2                     # = 1.3 x 1.152e-2, rounded up


def torch_mod():
    import torch
    return torch


def to_dev(a, dtype: str):
    """Storage array (float32, or uint16 bf16 bits) -> device tensor."""
    torch = torch_mod()
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def to_dev_w(w, dtype: str):
    """Row-major [N, K] linear weight (storage array) -> device tensor in the
    library's tiled weight layout (tiling by the library's host helper)."""
    from paper_2608_21719_amd import binding as B
    return to_dev(B.tile_weight(np.ascontiguousarray(w)), dtype)


def to_f64(t) -> np.ndarray:
    """Device tensor (bf16 or fp32) -> float64 numpy, exactly."""
    torch = torch_mod()
    if t.dtype == torch.bfloat16:
        bits = t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        return gen.bf16_bits_to_f32(bits).astype(np.float64)
    return t.detach().float().cpu().numpy().astype(np.float64)


def bits(t) -> np.ndarray:
    torch = torch_mod()
    if t.dtype == torch.bfloat16:
        return t.detach().contiguous().view(torch.int16).cpu().numpy()
    return t.detach().contiguous().view(torch.int32).cpu().numpy()


def empty(shape, dtype: str):
    torch = torch_mod()
    return torch.empty(shape, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32, device="cuda")


def nan_filled_bytes(nbytes: int):
    """Device byte buffer filled with 0xFF (NaN in bf16 and fp32) so that any
    read of unwritten KV memory shows up in the results."""
    torch = torch_mod()
    return torch.full((nbytes,), 255, dtype=torch.uint8, device="cuda")


def workspace(nbytes: int):
    torch = torch_mod()
    return torch.empty((max(nbytes, 256),), dtype=torch.uint8, device="cuda")


def assert_close_elementwise(got: np.ndarray, ref: np.ndarray, atol: float, rtol: float, what: str = ""):
    err = np.abs(got - ref)
    bound = atol + rtol * np.abs(ref)
    bad = err > bound
    if np.any(bad) or not np.all(np.isfinite(got)):
        i = np.unravel_index(np.argmax(err / bound), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} outside |e| <= {atol} + {rtol}|r|; "
                             f"worst at {i}: got {got[i]!r} ref {ref[i]!r}; max|e| {err.max():.3e}")


def normwise(got: np.ndarray, ref: np.ndarray):
    e = got - ref
    return (np.max(np.abs(e)) / np.max(np.abs(ref)), np.sqrt(np.mean(e * e)) / np.sqrt(np.mean(ref * ref)))


def weights_f64(w: dict, dtype: str) -> dict:
    return {k: gen.widen(v, dtype) for k, v in w.items()}


class DeviceLayer:
    """One layer's weights on the device in the libps layout."""

    def __init__(self, w: dict, dtype: str):
        from paper_2608_21719_amd import binding as B
        self.dtype = dtype
        self.t = {
            "attn_norm": to_dev(w["attn_norm"], dtype),
            "w_qkv": to_dev_w(np.concatenate([w["wq"], w["wk"], w["wv"]], axis=0), dtype),
            "w_o": to_dev_w(w["wo"], dtype),
            "ffn_norm": to_dev(w["ffn_norm"], dtype),
            "w_gate_up": to_dev_w(B.pack_gate_up(w["wg"], w["wu"]), dtype),
            "w_down": to_dev_w(w["wd"], dtype),
        }
        self.w = B.layer_weights(**self.t)


class Pool:
    """A KV pool on the device plus its libps metadata handle."""

    def __init__(self, shape, n_pages: int, max_seqs: int, max_pages_per_seq: int, n_layers: int = 1,
                 seed: int = 0, nan_fill: bool = True):
        from paper_2608_21719_amd import binding as B
        self.shape = shape
        self.cfg = B.make_cfg(shape)
        nbytes = B.KV.pool_bytes(self.cfg, n_layers, n_pages)
        self.mem = nan_filled_bytes(nbytes) if nan_fill else workspace(nbytes)
        self.kv = B.KV(self.cfg, n_layers, n_pages, max_seqs, max_pages_per_seq, self.mem, seed)
