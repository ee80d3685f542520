"""Post-EC tail (residual addition + next-layer RMSNorm): host-side
validation of spear_w4ec_linear_tail (CPU only; the GPU parity tests are in
test_gpu_parity.py)."""
from __future__ import annotations

import ctypes
import math

from paper_2606_11244_amd import spear as sp

# fake but distinct, 16-byte aligned addresses: every call below is rejected
# on the host before anything touches them
BASE = 0x7D0000000000
ADDR = {k: BASE + i * (1 << 32) for i, k in enumerate(["x", "y", "q", "s", "z", "A", "B", "w",
                                                        "W", "res", "nw", "yn"])}


def _call(prob, tail, with_ec=True, y="y"):
    w = sp.W4(ADDR["q"], ADDR["s"], ADDR["z"])
    ec = sp.EC(ADDR["A"], ADDR["B"], 1.0, ADDR["w"], 0.0, None, None, None, None, 0, None, None)
    yv = ADDR[y] if isinstance(y, str) else y
    return sp.LIB.spear_w4ec_linear_tail(ctypes.byref(prob), ADDR["x"], ctypes.byref(w),
                                         ctypes.byref(ec) if with_ec else None,
                                         ctypes.byref(tail) if tail is not None else None,
                                         yv, ADDR["W"], 1 << 30, None)


def _tail(res="res", nw="nw", eps=1e-5, yn="yn"):
    def a(k):
        return ADDR[k] if isinstance(k, str) else k
    return sp.Tail(a(res), a(nw), eps, a(yn))


def test_tail_validated_on_host():
    prob = sp.problem(4, 256, 256, 0, sp.F16, 8)
    assert _call(prob, None) == -1                           # no tail
    assert _call(prob, _tail(yn=None)) == -1                 # a norm needs its output
    assert _call(prob, _tail(eps=-1.0)) == -2                # eps must be >= 0
    assert _call(prob, _tail(eps=math.nan)) == -2
    assert _call(prob, _tail(res=ADDR["res"] + 4)) == -4     # alignment
    assert _call(prob, _tail(nw=ADDR["nw"] + 8)) == -4
    assert _call(prob, _tail(yn=ADDR["yn"] + 8)) == -4
    # the residual may be y itself, but may not overlap it otherwise
    assert _call(prob, _tail(res=ADDR["y"] + 16)) == -8
    # y_norm overlaps nothing
    for k in ("y", "x", "res", "nw", "W"):
        assert _call(prob, _tail(yn=ADDR[k] + 16)) == -8, k
    # the same checks without the EC
    assert _call(prob, _tail(yn=None), with_ec=False) == -1
    assert _call(prob, _tail(yn=ADDR["y"] + 16), with_ec=False) == -8


def test_tail_empty_problem_is_noop():
    prob = sp.problem(0, 256, 256, 0, sp.F16, 8)
    assert _call(prob, _tail()) == 0
