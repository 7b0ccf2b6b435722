"""The C ABI without a GPU: exported symbols and the host-side KV pool logic."""
import os
import re

import numpy as np
import pytest

from paper_2608_21719_amd import binding as B
from synth.configs import CONFIGS

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "ps.h")
FAKE_POOL = 0x10000  # never dereferenced by host-only calls


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ps_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_function_is_exported():
    names = declared_functions()
    assert len(names) >= 25
    missing = [n for n in names if not hasattr(B.lib, n)]
    assert not missing, missing


def test_binding_covers_every_declared_function():
    assert set(declared_functions()) == set(B._SIGS)


def _kv(n_pages=64, max_seqs=4, max_pages=16, seed=0):
    cfg = B.make_cfg(CONFIGS["tiny_f32"].shape)
    return B.KV(cfg, 1, n_pages, max_seqs, max_pages, FAKE_POOL, seed)


def test_reserve_commit_truncate_free_cycle():
    kv = _kv()
    s = kv.open()
    assert kv.seq_len(s) == 0 and kv.capacity(s) == 0
    kv.alloc(s, 17)
    assert kv.capacity(s) == 32 and kv.free_pages() == 62
    kv.commit([s], [17])
    assert kv.seq_len(s) == 17
    kv.alloc(s, 15)          # 17 + 15 = 32 fits the 2 pages already held
    assert kv.free_pages() == 62
    kv.alloc(s, 16)
    assert kv.capacity(s) == 48
    kv.truncate(s, 5)
    assert kv.seq_len(s) == 5 and kv.capacity(s) == 48
    kv.free(s)
    assert kv.free_pages() == 64
    with pytest.raises(B.PsError) as e:
        kv.seq_len(s)
    assert e.value.code == B.PS_E_INVALID


def test_identity_and_shuffled_page_order():
    kv = _kv(seed=0)
    s = kv.open()
    kv.alloc(s, 16 * 5)
    assert kv.block_table(s) == [0, 1, 2, 3, 4]
    kv2 = _kv(seed=12345)
    s2 = kv2.open()
    kv2.alloc(s2, 16 * 16)
    bt = kv2.block_table(s2)
    assert sorted(bt) == sorted(set(bt)) and len(bt) == 16 and bt != list(range(16))
    # deterministic for a given seed
    kv3 = _kv(seed=12345)
    s3 = kv3.open()
    kv3.alloc(s3, 16 * 16)
    assert kv3.block_table(s3) == bt


def test_pages_are_recycled_and_never_shared():
    kv = _kv(n_pages=8, max_seqs=4, max_pages=8, seed=7)
    a, b = kv.open(), kv.open()
    kv.alloc(a, 48)
    kv.alloc(b, 64)
    assert not set(kv.block_table(a)) & set(kv.block_table(b))
    assert kv.free_pages() == 1
    kv.free(a)
    c = kv.open()
    kv.alloc(c, 64)
    assert not set(kv.block_table(c)) & set(kv.block_table(b))


def test_exhaustion_fails_without_side_effects():
    kv = _kv(n_pages=4, max_seqs=2, max_pages=16)
    s = kv.open()
    kv.alloc(s, 40)
    before = (kv.block_table(s), kv.free_pages(), kv.capacity(s))
    with pytest.raises(B.PsError) as e:
        kv.alloc(s, 100)
    assert e.value.code == B.PS_E_NO_PAGES
    assert (kv.block_table(s), kv.free_pages(), kv.capacity(s)) == before


def test_per_sequence_page_limit():
    kv = _kv(n_pages=64, max_pages=3)
    s = kv.open()
    with pytest.raises(B.PsError) as e:
        kv.alloc(s, 49)
    assert e.value.code == B.PS_E_CAPACITY
    assert kv.free_pages() == 64


def test_commit_is_all_or_nothing():
    kv = _kv()
    a, b = kv.open(), kv.open()
    kv.alloc(a, 16)
    kv.alloc(b, 16)
    with pytest.raises(B.PsError) as e:
        kv.commit([a, b], [10, 17])
    assert e.value.code == B.PS_E_CAPACITY
    assert kv.seq_len(a) == 0 and kv.seq_len(b) == 0
    with pytest.raises(B.PsError):
        kv.commit([a, a], [1, 1])
    assert kv.seq_len(a) == 0


def test_bad_arguments_are_rejected():
    kv = _kv(max_seqs=1)
    s = kv.open()
    with pytest.raises(B.PsError) as e:
        kv.open()
    assert e.value.code == B.PS_E_CAPACITY
    with pytest.raises(B.PsError):
        kv.truncate(s, 1)
    with pytest.raises(B.PsError):
        kv.alloc(s, -1)
    cfg = B.make_cfg(CONFIGS["tiny_f32"].shape)
    cfg.n_kv_heads = 3
    with pytest.raises(B.PsError):
        B.KV(cfg, 1, 8, 1, 1, FAKE_POOL)


def test_device_calls_validate_before_touching_the_device():
    """Capacity errors surface on the host, before any launch (no GPU here)."""
    kv = _kv()
    s = kv.open()
    kv.alloc(s, 16)
    import ctypes
    ws = np.zeros(1 << 16, np.uint8)
    rc = B.lib.ps_kv_append(kv.h, 0, 1, B.ints([s]), B.ints([17]), ws.ctypes.data, ws.ctypes.data,
                            ws.ctypes.data, ws.nbytes, None)
    assert rc == B.PS_E_CAPACITY
    rc = B.lib.ps_kv_append(kv.h, 3, 1, B.ints([s]), B.ints([1]), ws.ctypes.data, ws.ctypes.data,
                            ws.ctypes.data, ws.nbytes, None)
    assert rc == B.PS_E_INVALID
    assert kv.seq_len(s) == 0
    del ctypes


def test_gemm_shapes_outside_the_kernels_are_rejected_on_the_host():
    """K % 64, N % 256 (M > 64), the 32-bit offset bound K < 2^21 and the
    SwiGLU pairing are checked before any launch (no GPU here)."""
    buf = np.zeros(1 << 12, np.uint8)
    p = buf.ctypes.data
    for M, N, K, epi in [(256, 256, 100, 0), (256, 100, 64, 0), (256, 256, 1 << 21, 0), (32, 96, 64, 2)]:
        rc = B.lib.ps_op_gemm(B.PS_BF16, 0, B.PS_BF16, epi, M, N, K, p, p, None, p, p, buf.nbytes, None)
        assert rc == B.PS_E_UNSUPPORTED, (M, N, K, epi)


def test_pack_gate_up_layout():
    F, d = 64, 3
    wg = np.arange(F * d, dtype=np.float32).reshape(F, d)
    wu = -wg
    out = B.pack_gate_up(wg, wu)
    np.testing.assert_array_equal(out[0:32], wg[0:32])
    np.testing.assert_array_equal(out[32:64], wu[0:32])
    np.testing.assert_array_equal(out[64:96], wg[32:64])
    np.testing.assert_array_equal(out[96:128], wu[32:64])


@pytest.mark.parametrize("N,K,dt", [(128, 192, np.uint16), (100, 70, np.uint16), (65, 129, np.float32),
                                    (1, 1, np.float32), (64, 64, np.uint16)])
def test_tile_weight_layout(N, K, dt):
    """The tiled weight layout: pad W to multiples of 64 with zeros, cut it
    into 64 x 64 tiles, order the tiles row of tiles by row of tiles, each
    tile row-major; also the per-element address formula of the header."""
    r = np.random.default_rng(N * 1000 + K)
    w = r.integers(1, 1 << 15, size=(N, K)).astype(dt)  # nonzero, so padding is visible
    out = B.tile_weight(w)
    nt, kt = -(-N // 64), -(-K // 64)
    assert out.shape == (nt * kt * 4096,) == (B.tiled_weight_elems(N, K),)
    pad = np.zeros((nt * 64, kt * 64), dtype=dt)
    pad[:N, :K] = w
    want = pad.reshape(nt, 64, kt, 64).transpose(0, 2, 1, 3).reshape(-1)
    np.testing.assert_array_equal(out, want)
    n, k = r.integers(0, N, 50), r.integers(0, K, 50)
    np.testing.assert_array_equal(out[((n // 64) * kt + k // 64) * 4096 + (n % 64) * 64 + k % 64], w[n, k])


def test_tile_weight_rejects_bad_arguments():
    assert B.tiled_weight_elems(0, 5) == 0 and B.tiled_weight_elems(5, -1) == 0
    w = np.zeros((4, 4), np.uint8)
    out = np.zeros(4096, np.uint8)
    assert B.lib.ps_tile_weight(B.ptr(w), 4, 4, 1, B.ptr(out)) == B.PS_E_INVALID
    assert B.lib.ps_tile_weight(None, 4, 4, 2, B.ptr(out)) == B.PS_E_INVALID


def test_workspace_and_pool_sizes():
    sh = CONFIGS["llama8b_decode"].shape
    cfg = B.make_cfg(sh)
    assert B.KV.pool_bytes(cfg, 1, 10) == 10 * 8 * 2 * 16 * 128 * 2
    assert B.Layer.workspace_bytes(cfg, 64, 64, 300) > 64 * (4096 + 14336) * 2


def test_decode_run_needs_a_current_plan_and_its_workspace():
    """Host-side checks of plan/run (no sequences, so nothing is launched)."""
    from ctypes import c_void_p
    cfg = B.make_cfg(CONFIGS["llama8b_decode"].shape)
    kv = B.KV(cfg, 1, 64, 4, 16, FAKE_POOL, 0)
    ws, ws2, nbytes = c_void_p(0x20000), c_void_p(0x40000), 1 << 20
    assert B.lib.ps_op_decode_run(kv.h, 0, None, None, ws, nbytes, None) == B.PS_E_INVALID
    assert B.lib.ps_op_decode_plan(kv.h, 0, None, 0, ws, nbytes, None) == B.PS_OK
    assert B.lib.ps_op_decode_run(kv.h, 0, None, None, ws, nbytes, None) == B.PS_OK
    assert B.lib.ps_op_decode_run(kv.h, 0, None, None, ws2, nbytes, None) == B.PS_E_INVALID
    assert B.lib.ps_op_decode_run(kv.h, 1, None, None, ws, nbytes, None) == B.PS_E_INVALID  # layer out of range
    s = kv.open()
    kv.alloc(s, 4)
    assert B.lib.ps_op_decode_run(kv.h, 0, None, None, ws, nbytes, None) == B.PS_OK  # open/alloc keep the plan
    kv.commit([s], [4])
    assert B.lib.ps_op_decode_run(kv.h, 0, None, None, ws, nbytes, None) == B.PS_E_INVALID
    assert "changed" in B.last_error()
    assert B.lib.ps_op_decode_plan(kv.h, 0, None, 0, ws, nbytes, None) == B.PS_OK
    assert B.lib.ps_op_decode_run(kv.h, 0, None, None, ws, nbytes, None) == B.PS_OK
    assert B.lib.ps_op_decode_plan(kv.h, 0, None, -1, ws, nbytes, None) == B.PS_E_INVALID
    assert B.lib.ps_op_decode_run(kv.h, 0, None, None, ws, nbytes, None) == B.PS_E_INVALID  # failed plan leaves none
    assert "no decode attention plan" in B.last_error()
    assert B.lib.ps_op_decode_plan(kv.h, 0, None, 0, ws, nbytes, None) == B.PS_OK
    assert B.lib.ps_op_decode_run_capped(kv.h, 0, None, None, ws, nbytes, 0, None) == B.PS_E_INVALID
    assert "max_workgroups" in B.last_error()
    assert B.lib.ps_op_decode_run_capped(kv.h, 0, None, None, ws, nbytes, 1, None) == B.PS_OK
    assert B.lib.ps_op_decode_run_capped(kv.h, 0, None, None, ws2, nbytes, 1, None) == B.PS_E_INVALID


def test_unaligned_device_pointers_are_rejected_before_launch():
    """Kernels use 16-byte vector accesses: host-side validation refuses
    unaligned buffers (nothing is launched, so fake addresses are safe)."""
    from ctypes import c_void_p
    ok, bad = c_void_p(0x100000), c_void_p(0x100008)
    rc = B.lib.ps_op_gemm(B.PS_BF16, 0, B.PS_BF16, B.PS_EPI_STORE, 256, 256, 256, ok, ok, None, bad, ok, 1 << 20,
                          None)
    assert rc == B.PS_E_INVALID and "aligned" in B.last_error()
    rc = B.lib.ps_op_gemm(B.PS_BF16, 0, B.PS_BF16, B.PS_EPI_STORE, 256, 256, 256, ok, ok, None, ok, bad, 1 << 20,
                          None)
    assert rc == B.PS_E_INVALID and "aligned" in B.last_error()
    cfg = B.make_cfg(CONFIGS["tiny_f32"].shape)
    h = c_void_p()
    from ctypes import byref
    assert B.lib.ps_kv_create(byref(cfg), 1, 8, 2, 4, c_void_p(FAKE_POOL + 4), 0, byref(h)) == B.PS_E_INVALID


def test_config_match_ignores_struct_padding():
    """Layer and pool configurations are compared field by field: garbage in
    the struct's tail padding (a C caller's separately built config) is not a
    difference, a different field is. No launch happens: the call then stops
    at the capacity check."""
    import ctypes
    sh = CONFIGS["llama8b_decode"].shape
    clean = B.make_cfg(sh)
    dirty = B.make_cfg(sh)
    assert ctypes.sizeof(B.LayerCfg) == 40 and B.LayerCfg.dtype.offset == 32
    ctypes.memset(ctypes.addressof(dirty) + 36, 0xAB, 4)
    assert bytes(clean) != bytes(dirty)
    other = B.make_cfg(sh)
    other.ffn = sh.ffn * 2
    kv = B.KV(clean, 1, 64, 4, 16, FAKE_POOL, 0)
    s = kv.open()
    kv.alloc(s, 16)
    fake = 0x100000
    w = B.LayerW(fake, fake, fake, fake, fake, fake)
    for cfg, want in ((dirty, B.PS_E_CAPACITY), (other, B.PS_E_INVALID)):
        layer = B.Layer(cfg)
        rc = B.lib.ps_prefill(layer.h, ctypes.byref(w), kv.h, 0, 1, B.ints([s]), B.ints([17]), fake, fake, fake,
                              1 << 30, None)
        assert rc == want, (rc, B.last_error())
    assert "differ" in B.last_error()


def test_static_gemm_rejects_partials_beyond_its_scratch_on_the_host():
    """ps_op_gemm_static checks the split-K partials against its static array
    before touching the device (no GPU here): a SwiGLU launch on one 64-row
    block per workgroup without a K split writes 4 M N bytes of partials."""
    from ctypes import c_void_p
    p = c_void_p(0x100000)
    M, N, K = 64, 64 * 1025, 64
    assert 4 * M * N > 16 << 20
    rc = B.lib.ps_op_gemm_static(B.PS_BF16, 0, B.PS_BF16, B.PS_EPI_SWIGLU, M, N, K, p, p, None, p, None)
    assert rc == B.PS_E_INVALID and "static scratch" in B.last_error()
    rc = B.lib.ps_op_gemm_static(B.PS_BF16, 0, B.PS_BF16, B.PS_EPI_STORE, 256, 100, 64, p, p, None, p, None)
    assert rc == B.PS_E_UNSUPPORTED


def test_kv_transfer_validates_on_the_host():
    """Every refusal happens before any device work (no GPU here) and leaves
    both pools unchanged."""
    sh = CONFIGS["llama8b_decode"].shape
    src = B.KV(B.make_cfg(sh), 2, 64, 4, 16, FAKE_POOL, 3)
    dst = B.KV(B.make_cfg(sh), 2, 40, 4, 16, FAKE_POOL, 9)
    s = src.open()
    src.alloc(s, 40)
    src.commit([s], [37])
    ws = np.zeros(1 << 12, np.uint8)

    def xfer(a, sa, b, sb):
        return B.lib.ps_kv_transfer(a.h, sa, b.h, sb, ws.ctypes.data, ws.nbytes, None)

    d = dst.open()
    dst.alloc(d, 32)  # 2 pages: too few for 37 tokens
    assert xfer(src, s, dst, d) == B.PS_E_CAPACITY and "destination" in B.last_error()
    assert xfer(src, s, dst, 3) == B.PS_E_INVALID          # destination not open
    assert xfer(src, 2, dst, d) == B.PS_E_INVALID          # source not open
    assert xfer(src, s, src, s) == B.PS_E_INVALID          # same sequence
    other = B.make_cfg(sh)
    other.n_kv_heads = 4
    odd = B.KV(other, 2, 40, 4, 16, FAKE_POOL, 0)
    o = odd.open()
    odd.alloc(o, 64)
    assert xfer(src, s, odd, o) == B.PS_E_INVALID and "configurations differ" in B.last_error()
    shallow = B.KV(B.make_cfg(sh), 1, 40, 4, 16, FAKE_POOL, 0)
    t = shallow.open()
    shallow.alloc(t, 64)
    assert xfer(src, s, shallow, t) == B.PS_E_INVALID and "layer count" in B.last_error()
    dst.alloc(d, 48)
    dst.commit([d], [1])
    assert xfer(src, s, dst, d) == B.PS_E_INVALID and "not empty" in B.last_error()
    assert src.seq_len(s) == 37 and dst.seq_len(d) == 1 and dst.capacity(d) == 48
