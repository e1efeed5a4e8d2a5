"""The allocation-free prompt product (tetra_gemm_noalloc, through the C ABI)
against tetra_gemm with a caller workspace, and both against the oracle.

Two calls in a row on the library's static scratch, the second with a
smaller input: each must give the same bits as tetra_gemm with a full
workspace (same grid, same split, same summation order) and stay within the
parity bar of the float64 oracle.
"""

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import paper_2609_35465_amd as tt  # noqa: E402
from paper_2609_35465_amd import workloads  # noqa: E402
from oracle import gemv as ogemv  # noqa: E402

TOL = 1e-3
TOL_GEMM = 2.0 ** -11     # one fp16 rounding of each scaled weight (the prompt product's bound)


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _case(M, K, N, seed):
    words, sigma, tail = workloads.tetra_matrix(seed, M, K)
    x = workloads.activations(seed + 1, N, K)
    blob = _dev(tt.pack_rows(words, tail, M, K))
    sg = _dev(sigma.astype(np.float16))
    xd = _dev(x.astype(np.float16))
    return words, sigma, tail, x, blob, sg, xd


def test_gemm_noalloc_matches_gemm_twice():
    assert torch.cuda.is_available(), "GPU test"
    ws = tt.gemm_workspace()
    rng = np.random.default_rng(11)
    # the second call is smaller than the first (fewer rows, blocks and tokens)
    for M, K, N in [(1536, 1536 + 8, 203), (200, 24 * 10 + 8, 33)]:
        print(f"[noalloc] M={M} K={K} N={N}", flush=True)
        words, sigma, tail, x, blob, sg, xd = _case(M, K, N, workloads.seed_for(0, 9) + M)
        y_ref = torch.full((N, M), float("nan"), dtype=torch.float32, device="cuda")
        y_na = torch.full((N, M), float("nan"), dtype=torch.float32, device="cuda")
        tt.gemm(blob, sg, xd, y_ref, M, K, N, ws)
        tt.gemm_noalloc(blob, sg, xd, y_na, M, K, N)
        torch.cuda.synchronize()
        a, b = y_ref.cpu().numpy(), y_na.cpu().numpy()
        assert not np.isnan(b).any()
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), "noalloc bits differ from tetra_gemm"
        rows = np.unique(np.concatenate([np.arange(min(M, 64)), rng.integers(0, M, 64), [M - 1]]))
        yr, norm = ogemv.gemv_f64(words, sigma, tail, x, rows=rows)
        worst = float((np.abs(b[:, rows].astype(np.float64) - yr) / np.maximum(norm, 1e-300)).max())
        print(f"[noalloc] worst against the oracle {worst:.3e}", flush=True)
        assert worst <= TOL
        assert worst <= TOL_GEMM
