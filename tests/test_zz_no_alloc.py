"""surge_op_linear_ln_noalloc, the variant of surge_op_linear_ln for callers
that cannot allocate device memory (its per-row LayerNorm factors live in the
library's static scratch), against surge_op_linear_ln itself: two calls in a
row for each epilogue, the second with fewer rows (the scratch keeps the
first call's rows beyond it), must give bit-identical outputs and row
statistics; a row count beyond the scratch is refused before anything runs.
"""
import numpy as np
import pytest

from gpu_util import torch_cuda
from paper_2605_01060_amd import surge as S
from paper_2605_01060_amd import workload as W

pytestmark = pytest.mark.gpu

SCRATCH_ROWS = 1 << 19


def _inputs(torch, rng, M, N, K, epi):
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    bf = lambda a: torch.from_numpy(W.round_to_bf16(np.asarray(a, np.float32))).to(
        torch.bfloat16).cuda()
    width = 64
    parts_in = (K if epi in (3, 4) else N) // width
    st = np.stack([rng.standard_normal((parts_in, M)) * 0.3,
                   rng.uniform(0.2, 3.0, (parts_in, M))], axis=-1)
    return dict(x=bf(rng.standard_normal((M, K))), w=bf(rng.standard_normal((N, K)) * 0.05),
                bias=f32(rng.standard_normal(N) * 0.1),
                res=bf(rng.standard_normal((M, N))) if epi in (2, 5, 6) else None,
                stats_in=f32(st) if epi in (3, 4, 6) else None, parts_in=parts_in,
                col_s=f32(rng.standard_normal(N)) if epi in (3, 4) else None,
                gamma=f32(1 + 0.1 * rng.standard_normal(N)) if epi == 6 else None,
                beta=f32(0.1 * rng.standard_normal(N)) if epi == 6 else None)


def _run(torch, fn, M, N, K, epi, a):
    y = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    so = torch.full((N // 64, M, 2), float("nan"), device="cuda") if epi >= 5 else None
    fn(M, N, K, a["x"], a["w"], a["bias"], a["res"], epi, a["stats_in"], a["parts_in"],
       a["col_s"], a["gamma"], a["beta"], 1e-12, so, y, torch.cuda.current_stream())
    torch.cuda.synchronize()
    return y, so


@pytest.mark.parametrize("epi,N,K", [(4, 3072, 768), (6, 768, 3072), (3, 2304, 768),
                                     (5, 768, 768), (0, 1152, 384)])
def test_noalloc_matches_the_allocating_entry_point(epi, N, K):
    torch = torch_cuda()
    rng = np.random.default_rng(100 + epi)
    for M in (60001, 4099):  # the second call is smaller
        print(f"[no-alloc] epilogue {epi} M={M} N={N} K={K}", flush=True)
        a = _inputs(torch, rng, M, N, K, epi)
        y0, s0 = _run(torch, S.surge_op_linear_ln, M, N, K, epi, a)
        y1, s1 = _run(torch, S.surge_op_linear_ln_noalloc, M, N, K, epi, a)
        assert not torch.isnan(y1.float()).any().item()
        assert torch.equal(y0, y1)
        if s0 is not None:
            assert torch.equal(s0, s1)


def test_noalloc_refuses_rows_beyond_the_scratch():
    torch = torch_cuda()
    M, N, K = SCRATCH_ROWS + 1, 128, 64
    x = torch.zeros((M, K), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((N, K), dtype=torch.bfloat16, device="cuda")
    b = torch.zeros(N, device="cuda")
    st = torch.ones((1, M, 2), device="cuda")
    cs = torch.zeros(N, device="cuda")
    y = torch.full((M, N), 7.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(S.SurgeError) as ei:
        S.surge_op_linear_ln_noalloc(M, N, K, x, w, b, None, 3, st, 1, cs, None, None, 1e-12,
                                     None, y)
    assert ei.value.status == S.SURGE_ERR_CAPACITY
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())
    # the plain epilogue reads no row factors, so it has no such limit
    S.surge_op_linear_ln_noalloc(M, N, K, x, w, b, None, 0, None, 0, None, None, None, 1e-12,
                                 None, y, torch.cuda.current_stream())
    torch.cuda.synchronize()
    assert bool((y == 0).all())
