"""Helpers shared by the GPU tests: run a generated layer through the C ABI
and compare with the CPU oracle under the parity bar."""
from __future__ import annotations

import copy
import sys

import numpy as np
import torch

from oracle import spear_oracle as O
from paper_2606_11244_amd import synth as S

# parity bar: relative Frobenius error and max error relative to max |y_ref|
REL_FROB = 5e-3
MAX_REL = 1e-2


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_y(layer, path: int = 0, with_ec: bool = True, rank=None, gate_kind=None,
          workspace=None, dev=None):
    """Run the layer on the GPU, return y as float64 numpy [M][N]."""
    from paper_2606_11244_amd import spear as sp
    dl = dev if dev is not None else sp.DeviceLayer(layer)
    prob = dl.problem(force_path=path, rank=rank, gate_kind=gate_kind)
    ws = workspace if workspace is not None else sp.allocate_workspace(prob, with_ec)
    if with_ec:
        dl.run_ec(prob, ws)
    else:
        dl.run_w4(prob, ws)
    torch.cuda.synchronize()
    return dl.y.float().cpu().numpy().astype(np.float64)


def assert_parity(y, y_ref, what=""):
    ok, relf, mx, bound = O.tolerance_check(y, y_ref, REL_FROB, MAX_REL)
    assert ok, f"{what}: relF={relf:.3e} (<= {REL_FROB}) max|d|={mx:.3e} (<= {bound:.3e})"
    return relf, mx


def with_fields(layer, **kw):
    out = copy.copy(layer)
    for k, v in kw.items():
        setattr(out, k, v)
    return out


def zero_weight(layer):
    """Codes equal to the zero point everywhere: What == 0, y is the EC term."""
    z = np.full_like(layer.zeros, 7)
    return with_fields(layer, zeros=z,
                       qweight=S.pack_int4(np.full((layer.N, layer.K), 7, dtype=np.int64)))


def scaled_ec(layer, factor):
    """A and B multiplied by `factor` (rounded to the act dtype)."""
    dt = layer.act_dtype
    return with_fields(layer,
                       A=S.to_bits(S.from_bits(layer.A, dt) * factor, dt),
                       B=S.to_bits(S.from_bits(layer.B, dt) * factor, dt))
