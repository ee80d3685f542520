"""GPU parity on the 70B-shaped whole model the benchmark times: all 80
layers x 7 modules resident (device-random 4-bit weights, the EC on the
seeded quarter of the pairs), every call on its automatic path with one
shared workspace, as in the benchmark's model pass. A seeded sample of 8
(layer, module) pairs, 4 with the EC and 4 without, is checked against the
oracle at every token count of that pass, on sampled tokens (the first, the
last and 6 seeded ones) and sampled output rows (the first, the last and 30
seeded ones), the oracle decoding the device tensors' exact bit patterns."""
from __future__ import annotations

import types

import numpy as np
import pytest
import torch

from oracle import spear_oracle as O
from paper_2606_11244_amd import synth as S

from gpu_util import assert_parity, log

pytestmark = pytest.mark.gpu

MS = (1, 16, 64, 512, 4096, 8192)


@pytest.fixture(scope="module")
def model():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_11244_amd import model70b
    log("70B model: building 80 layers x 7 modules on the device")
    layers, sel = model70b.build("cuda", seed=0)
    torch.cuda.synchronize()
    yield layers, sel
    del layers
    torch.cuda.empty_cache()


def _pick(sel, n_each=4, seed=3):
    rng = np.random.default_rng(seed)
    on = np.argwhere(sel)
    off = np.argwhere(~sel)
    return ([tuple(on[i]) for i in rng.choice(len(on), n_each, replace=False)] +
            [tuple(off[i]) for i in rng.choice(len(off), n_each, replace=False)])


def _sample(n, k, rng):
    return np.unique(np.concatenate([[0, n - 1], rng.choice(n, size=min(k, n), replace=False)]))


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def test_sampled_modules_all_token_counts(model):
    from paper_2606_11244_amd import model70b
    from paper_2606_11244_amd import spear as sp
    layers, sel = model
    r, G = model70b.RANK, model70b.GROUP
    picks = _pick(sel)
    assert sum(bool(sel[l, j]) for l, j in picks) == 4
    rng = np.random.default_rng(11)
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    for l, j in picks:
        m, K, N, q, sc, zr, ec = layers[l][j]
        rows = _sample(N, 30, rng)
        ridx = torch.as_tensor(rows, device="cuda")
        host = types.SimpleNamespace(
            act_dtype=S.F16, group_size=G, rank=r if ec is not None else 0,
            gate_kind=S.GATE_SIGMOID_LINEAR, alpha=1.0, b_g=0.0,
            qweight=q[ridx].cpu().numpy().view(np.uint32),
            scales=sc[ridx].cpu().numpy().view(np.uint16), zeros=zr[ridx].cpu().numpy(),
            A=None if ec is None else _bits(ec[0]), B=None if ec is None else _bits(ec[1][ridx]),
            w_g=None if ec is None else _bits(ec[2]),
            W1=np.zeros((1, 1), np.uint16), b1=np.zeros(1, np.uint16),
            W2=np.zeros((1, 1), np.uint16), b2=np.zeros(1, np.uint16))
        for M in MS:
            pe = sp.problem(M, N, K, G, sp.F16, r, sp.GATE_SIGMOID_LINEAR)
            p4 = sp.problem(M, N, K, G, sp.F16, 0, sp.GATE_SIGMOID_LINEAR)
            ws = torch.zeros(max(256, sp.dispatch_plan(pe).workspace_bytes,
                                 sp.dispatch_plan(p4, with_ec=False).workspace_bytes),
                             dtype=torch.uint8, device="cuda")
            x = torch.randn((M, K), device="cuda", generator=g).half()
            y = torch.empty((M, N), dtype=torch.float16, device="cuda")
            plan = sp.dispatch_plan(pe if ec is not None else p4, with_ec=ec is not None)
            log(f"70B model: layer={l} module={m} K={K} N={N} M={M} ec={ec is not None} "
                f"path={sp.PATH_NAMES[plan.path]}")
            if ec is not None:
                sp.w4ec_linear(pe, x, q, sc, zr, ec[0], ec[1], y, w_g=ec[2], workspace=ws)
            else:
                sp.w4_linear(p4, x, q, sc, zr, y, workspace=ws)
            torch.cuda.synchronize()
            toks = _sample(M, 6, rng)
            host.x = _bits(x[torch.as_tensor(toks, device="cuda")])
            ref = O.w4ec_linear_rows(host, np.arange(len(rows)))
            got = y.float().cpu().numpy().astype(np.float64)[toks][:, rows]
            assert np.all(np.isfinite(got))
            assert_parity(got, ref, f"70B l{l}/{m}/M={M}")
            del ws, x, y
