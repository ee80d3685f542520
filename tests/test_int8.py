"""INT8 per-channel symmetric EC factors: the seeded generator's quantiser
and the host-side validation of the INT8 format (CPU only; the GPU parity
tests are in test_gpu_parity.py and test_gpu_fullsize.py)."""
from __future__ import annotations

import ctypes

import numpy as np

from paper_2606_11244_amd import spear as sp
from paper_2606_11244_amd import synth as S


def test_quantizer_round_trip_and_range():
    rng = np.random.default_rng(3)
    w = rng.normal(0, 0.05, size=(37, 301)).astype(np.float32)
    w[5] = 0.0
    q, s = S.quantize_int8_rows(w)
    assert q.dtype == np.int8 and s.dtype == np.float32
    assert np.all(np.abs(q.astype(np.int32)) <= 127)
    deq = s[:, None].astype(np.float64) * q.astype(np.float64)
    # round to nearest: at most half a step from the input (fp32 slack)
    assert np.all(np.abs(deq - w) <= 0.5 * s[:, None] * (1 + 1e-6) + 1e-12)
    # the largest magnitude of every nonzero row maps to +-127
    nz = np.abs(w).max(axis=1) > 0
    assert np.all(np.abs(q[nz].astype(np.int32)).max(axis=1) == 127)
    # an all-zero row: scale 1, codes 0
    assert s[5] == 1.0 and not q[5].any()
    # symmetric: negating the input negates the codes and keeps the scales
    q2, s2 = S.quantize_int8_rows(-w)
    assert np.array_equal(q2, -q) and np.array_equal(s2, s)


def test_make_layer_int8_fields():
    L = S.make_layer(M=2, N=24, K=256, group_size=128, rank=8, ab_int8=True)
    assert L.ab_int8 and L.A_q.shape == (8, 256) and L.B_q.shape == (24, 8)
    assert L.a_scale.shape == (8,) and L.b_scale.shape == (24,)
    # the same draw as the activation-dtype factors of the same seed
    L0 = S.make_layer(M=2, N=24, K=256, group_size=128, rank=8)
    A = S.from_bits(L0.A, L0.act_dtype).astype(np.float64)
    deq = L.a_scale[:, None].astype(np.float64) * L.A_q
    assert np.abs(deq - A).max() <= 0.51 * L.a_scale.max() + 1e-3 * np.abs(A).max()


# fake but distinct, 16-byte aligned addresses: every call below is rejected
# on the host before anything touches them
BASE = 0x7E0000000000
ADDR = {k: BASE + i * (1 << 32) for i, k in enumerate("xyqszABwWab")}


def _call(prob, fmt=sp.AB_INT8, a_scale="a", b_scale="b", y="y"):
    w = sp.W4(ADDR["q"], ADDR["s"], ADDR["z"])
    ec = sp.EC(ADDR["A"], ADDR["B"], 1.0, ADDR["w"], 0.0, None, None, None, None, fmt,
               ADDR[a_scale] if isinstance(a_scale, str) else a_scale,
               ADDR[b_scale] if isinstance(b_scale, str) else b_scale)
    yv = ADDR[y] if isinstance(y, str) else y
    return sp.LIB.spear_w4ec_linear(ctypes.byref(prob), ADDR["x"], ctypes.byref(w),
                                    ctypes.byref(ec), yv, ADDR["W"], 1 << 30, None)


def test_int8_format_validated_on_host():
    prob = sp.problem(4, 256, 256, 0, sp.F16, 8)
    assert _call(prob, fmt=7) == -3              # unknown format
    assert _call(prob, a_scale=None) == -1       # INT8 without its scales
    assert _call(prob, b_scale=None) == -1
    assert _call(prob, a_scale=ADDR["a"] + 4) == -4   # misaligned scales
    assert _call(prob, b_scale=ADDR["b"] + 8) == -4
    # the output may not overlap the scales
    assert _call(prob, y=ADDR["a"] + 16) == -8
    assert _call(prob, y=ADDR["b"] + 16) == -8
