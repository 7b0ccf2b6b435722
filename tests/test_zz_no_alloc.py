"""ps_op_gemm_static (split-K partials in the library's static device array,
no workspace argument) against ps_op_gemm with a caller workspace (GPU).

Both run the same kernels with the same launch plan, so the outputs must be
bit-identical. Two calls in a row: the first leaves its partials in the
static array, the second, smaller, must not read any of them. The caller
workspace of the reference call is filled with NaN so that a read of an
unwritten partial would show on either side. The first call is also checked
against the fp64 oracle with the deterministic GEMM bound.
"""
import numpy as np
import pytest

from oracle import layer as O
from tests import helpers as H

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2608_21719_amd import binding as B  # noqa: E402


def _inputs(M, N, K, rdt, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    a = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
    w = (torch.randn((N, K), generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    wt = torch.empty(B.tiled_weight_elems(N, K), dtype=torch.bfloat16, device="cuda")
    B.op_tile_weight(B.PS_BF16, N, K, w, wt)
    r = torch.randn((M, N), generator=g, device="cuda").to(torch.bfloat16 if rdt == B.PS_BF16 else torch.float32)
    return a, w, wt, r


def _pair(M, N, K, epi, rdt, cdt, seed):
    a, w, wt, r = _inputs(M, N, K, rdt, seed)
    cols = N // 2 if epi == B.PS_EPI_SWIGLU else N
    ctype = torch.bfloat16 if cdt == B.PS_BF16 else torch.float32
    ref = torch.empty((M, cols), dtype=ctype, device="cuda")
    got = torch.full((M, cols), float("nan"), dtype=ctype, device="cuda")
    ws = torch.full((max(16, B.op_gemm_workspace_bytes(B.PS_BF16, M, N, K)) // 4,), float("nan"),
                    dtype=torch.float32, device="cuda")
    R = r if epi == B.PS_EPI_RESIDUAL else None
    B.op_gemm(B.PS_BF16, rdt, cdt, epi, M, N, K, a, wt, R, ref, ws)
    B.op_gemm_static(B.PS_BF16, rdt, cdt, epi, M, N, K, a, wt, R, got)
    torch.cuda.synchronize()
    return a, w, r, ref, got


def test_static_scratch_gemm_equals_workspace_gemm_on_two_calls():
    # 1: the 70B down projection at decode batch 64: four K splits, 8 MiB of partials
    M, N, K = 64, 8192, 28672
    print(f"call 1: M={M} N={N} K={K} residual", flush=True)
    a, w, r, ref, got = _pair(M, N, K, B.PS_EPI_RESIDUAL, B.PS_F32, B.PS_BF16, 11)
    assert torch.equal(ref.view(torch.int16), got.view(torch.int16))
    cols = np.sort(np.random.default_rng(3).choice(N, 256, replace=False))
    af = H.to_f64(a)
    wf = H.to_f64(w[torch.from_numpy(cols).cuda()])
    want = O.linear(af, wf) + H.to_f64(r)[:, cols]
    bound = (np.abs(af) @ np.abs(wf).T) * (2 * K * 2.0 ** -24) + 2.0 ** -8 * np.abs(want)
    assert np.all(np.abs(H.to_f64(got)[:, cols] - want) <= bound)
    # 2: smaller, fewer rows and a different split count; must not see call 1's partials
    for M, N, K, epi, rdt, cdt in [(17, 4096, 4096, B.PS_EPI_RESIDUAL, B.PS_BF16, B.PS_F32),
                                   (40, 6144, 4096, B.PS_EPI_STORE, 0, B.PS_BF16)]:
        print(f"call 2: M={M} N={N} K={K} epi={epi}", flush=True)
        _, _, _, ref, got = _pair(M, N, K, epi, rdt, cdt, 12 + M)
        bits = torch.int16 if cdt == B.PS_BF16 else torch.int32
        assert torch.equal(ref.view(bits), got.view(bits))
