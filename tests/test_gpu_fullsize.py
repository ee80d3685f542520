"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (automatic dispatch), checked on sampled output columns that
the oracle computes one by one (all tokens, a seeded subset of rows n,
including the first and last rows of the layer)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import spear_oracle as O
from paper_2606_11244_amd import synth as S

from gpu_util import assert_parity, gpu_y, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield


def _rows(N, k=48, seed=0):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, N - 1], rng.choice(N, size=min(k, N), replace=False)]))


def _check(cid, module, Ms, seed=0, rank=None, paths=(0,), ab_int8=False):
    base = S.config_layer(cid, module, max(Ms), seed=seed, rank=rank, ab_int8=ab_int8)
    rows = _rows(base.N, seed=seed)
    for M in Ms:
        L = (S.config_layer(cid, module, M, seed=seed, rank=rank, ab_int8=ab_int8)
             if M != max(Ms) else base)
        ref = O.w4ec_linear_rows(L, rows)
        for p in paths:
            log(f"full-size config={cid} module={module} M={M} rank={L.rank} path={p} "
                f"int8={ab_int8}")
            y = gpu_y(L, p)
            assert np.all(np.isfinite(y))
            assert_parity(y[:, rows], ref, f"c{cid}/{module}/M={M}/path={p}")


@pytest.mark.parametrize("module", S.MODULES)
def test_llama1b_decode(module):
    _check(1, module, (1, 4, 16), paths=(0, 3, 4))


@pytest.mark.parametrize("module", ["q", "k", "gate", "down"])
def test_llama1b_prefill(module):
    _check(2, module, (512, 2048, 4096))


@pytest.mark.parametrize("module", ["q", "k", "gate", "down"])
def test_llama8b(module):
    _check(3, module, (1, 8, 32, 128, 512, 4096))


@pytest.mark.parametrize("module,Ms", [("k", (1, 16, 512)), ("q", (1, 64, 2048)),
                                       ("down", (1, 16, 512)), ("gate", (1, 256))])
def test_llama70b_modules(module, Ms):
    _check(4, module, Ms)
    if module == "k":  # the modules without an EC run the plain 4-bit kernel
        _check(4, module, (1, 512), rank=0)


@pytest.mark.parametrize("seed", [1, 2])
def test_llama1b_more_seeds(seed):
    _check(1, "o", (1, 16), seed=seed, paths=(0, 3, 4))
    _check(2, "up", (2048,), seed=seed)


@pytest.mark.parametrize("cid,module,Ms", [(1, "q", (1, 16)), (1, "down", (1,)),
                                           (2, "gate", (512, 4096)), (3, "q", (1, 128)),
                                           (4, "down", (1, 64))])
def test_int8_factors_full_size(cid, module, Ms):
    """INT8 per-channel EC factors at the workload sizes, automatic dispatch."""
    _check(cid, module, Ms, ab_int8=True)
