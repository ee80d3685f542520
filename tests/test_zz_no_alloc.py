"""GPU test of the entry point that allocates nothing
(spear_w4ec_linear_noalloc): through the C ABI, its output equals
spear_w4ec_linear's on a workspace of the caller's bit for bit, on two calls
in a row whose second is smaller, on the decode paths (local EC, producer-
fused GEMV with its tagged region, semi-fused pair) and the prefill GEMM
split over K; and it meets the parity bar against the oracle."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import spear_oracle as O
from paper_2606_11244_amd import synth as S

from gpu_util import assert_parity, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield


# (path, [(M, N, K, rank)] of the two calls in a row, the second smaller)
CASES = [
    (0, [(16, 2048, 4096, 16), (3, 512, 2048, 16)]),     # local EC GEMV
    (1, [(8, 4096, 4096, 32), (1, 1024, 2048, 32)]),     # producer-fused GEMV
    (4, [(16, 2048, 8192, 64), (2, 1024, 4096, 64)]),    # semi-fused pair (GEMV)
    (0, [(200, 1024, 4096, 16), (64, 512, 2048, 16)]),   # fully fused GEMM, split-K
    (4, [(160, 512, 4096, 32), (96, 256, 2048, 32)]),    # semi-fused pair (GEMM), split-K
]


@pytest.mark.parametrize("path,calls", CASES)
def test_noalloc_matches_workspace_call(path, calls):
    from paper_2606_11244_amd import spear as sp
    for i, (M, N, K, r) in enumerate(calls):
        L = S.make_layer(M=M, N=N, K=K, group_size=128, rank=r, seed=31 + i + path)
        dl = sp.DeviceLayer(L)
        prob = dl.problem(force_path=path)
        assert sp.dispatch_plan(prob).workspace_bytes <= sp.SCRATCH_BYTES
        log(f"noalloc path={path} call={i} M={M} N={N} K={K} r={r}")
        ws = sp.allocate_workspace(prob)
        y_ws = torch.empty_like(dl.y)
        dl.run_ec(prob, ws, y=y_ws)
        dl.run_noalloc(prob)
        torch.cuda.synchronize()
        assert torch.equal(dl.y, y_ws), (path, i)
        y = dl.y.float().cpu().numpy().astype(np.float64)
        assert_parity(y, O.w4ec_linear(L), f"noalloc path={path} call={i}")


def test_noalloc_rejects_oversized_problem():
    from paper_2606_11244_amd import spear as sp
    prob = sp.problem(512, 8192, 8192, 128, sp.F16, 64)  # GEMM split-K partials: 34 MB
    assert sp.dispatch_plan(prob).workspace_bytes > sp.SCRATCH_BYTES
    dummy = torch.zeros(16, dtype=torch.float16, device="cuda")
    with pytest.raises(sp.SpearError) as e:
        sp.w4ec_linear_noalloc(prob, dummy, dummy, dummy, dummy, dummy, dummy, dummy, w_g=dummy)
    assert e.value.status == -5  # SPEAR_E_WORKSPACE, before any pointer is used
