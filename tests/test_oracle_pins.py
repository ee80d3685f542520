"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each check_* function takes the oracle module and returns True when the pin
holds, so that the same checks can be run against deliberately broken copies
of the oracle (planted mistakes, bottom of this file) to show that each
plausible mistake is caught by at least one pin.

Pins used:
  * hand-worked golden fixtures of Eq. 3 (tests/golden/ec_worked_examples.json)
  * IEEE rounding fixtures (tests/golden/rounding_fixtures.json)
  * fixed packed words with known nibble contents (the documented layout)
  * the RTN round trip: exact on the 4-bit grid, within s/2 off the grid
  * brute force in exact rational arithmetic on tiny shapes
  * integer-grid inputs, where float64 results must be exact
  * reductions: r = 0, gate == 0, W_hat == 0, A == 0
  * the static low-rank case of the tanh gate (Eq. 2 with W_comp = alpha B A)
  * the factored form (Eq. 4) token by token
  * gate ranges: sigma(0) = 1/2 exactly, gamma in (0, 2), gamma -> 2
"""
from __future__ import annotations

import copy
import json
import math
import os
import types
from fractions import Fraction

import numpy as np
import pytest

from oracle import spear_oracle as O
from paper_2606_11244_amd import synth as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# helpers that build stored layers from plain numbers (no oracle code)
# ---------------------------------------------------------------------------

def _f16_bits(vals):
    return np.asarray(vals, dtype=np.float64).astype(np.float16).view(np.uint16)


def _layer_from_case(c, dtype=S.F16):
    qw = np.array([[int(h, 16) for h in row] for row in c["qweight_hex"]], dtype=np.uint32)
    r = c["rank"]
    K = c["K"]

    def bits(v, shape):
        a = np.asarray(v, dtype=np.float32).reshape(shape)
        return S.to_bits(a, dtype)

    h = len(c.get("b1", [])) or 4 * r
    return S.Layer(
        M=c["M"], N=c["N"], K=K, group_size=c["group_size"], act_dtype=dtype,
        rank=r, gate_kind=c["gate_kind"], qweight=qw,
        scales=_f16_bits(c["scales"]), zeros=np.asarray(c["zeros"], np.uint8),
        x=bits(c["x"], (c["M"], K)), A=bits(c["A"], (r, K)), B=bits(c["B"], (c["N"], r)),
        w_g=bits(c["w_g"], (K,)), b_g=c["b_g"], alpha=c["alpha"],
        W1=bits(c.get("W1", np.zeros((h, r))), (h, r)), b1=bits(c.get("b1", np.zeros(h)), (h,)),
        W2=bits(c.get("W2", np.zeros((r, h))), (r, h)), b2=bits(c.get("b2", np.zeros(r)), (r,)))


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------------------
# pin checks (each returns True when the pin holds for oracle module o)
# ---------------------------------------------------------------------------

def check_unpack_fixed_words(o) -> bool:
    """Layout pin: 0x76543210 holds codes 0..7 lowest nibble first, etc."""
    w = np.array([[0x76543210, 0xFEDCBA98, 0x0000000F, 0xF0000000]], dtype=np.uint32)
    want = list(range(8)) + list(range(8, 16)) + [15] + [0] * 7 + [0] * 7 + [15]
    return o.unpack_int4(w).tolist() == [want]


def check_unpack_exhaustive(o) -> bool:
    """Every code value at every nibble position decodes to itself and leaves
    the other seven positions zero."""
    for v in range(16):
        for i in range(8):
            w = np.array([[v << (4 * i)]], dtype=np.uint32)
            want = [0] * 8
            want[i] = v
            if o.unpack_int4(w).tolist() != [want]:
                return False
    return True


def check_golden_examples(o) -> bool:
    for c in _load("ec_worked_examples.json")["cases"]:
        layer = _layer_from_case(c)
        W_hat = o.dequant(layer.qweight, layer.scales, layer.zeros, layer.group_size)
        if not np.array_equal(W_hat, np.asarray(c["expected_W_hat"], np.float64)):
            return False
        y = o.w4ec_linear(layer)
        if not np.allclose(y, np.asarray(c["expected_y"]), rtol=1e-15, atol=1e-15):
            return False
    return True


def check_rounding_fixtures(o) -> bool:
    for c in _load("rounding_fixtures.json")["cases"]:
        v = np.array([c["value"]])
        if int(o.round_f64_to_bits(v, O.F16)[0]) != int(c["f16"], 16):
            return False
        if int(o.round_f64_to_bits(v, O.BF16)[0]) != int(c["bf16"], 16):
            return False
    return True


def check_rtn_grid_roundtrip(o, seed=0) -> bool:
    """Weights built on the 4-bit grid, with codes 0 and 15 present in every
    group and a dyadic fp16 scale, come back exactly through RTN + dequant."""
    rng = np.random.default_rng(seed)
    N, K = 24, 256
    for G in (K, 128, 64):
        s = 2.0 ** rng.integers(-9, -3, size=(N, K // G))
        z = rng.integers(0, 16, size=(N, K // G))
        q = rng.integers(0, 16, size=(N, K))
        qg = q.reshape(N, K // G, G)
        qg[:, :, 0] = 0
        qg[:, :, 1] = 15
        q = qg.reshape(N, K)
        grp = np.arange(K) // G
        w = ((q - z[:, grp]) * s[:, grp]).astype(np.float32)
        q2, s2, z2 = S.rtn_quantize(w, G)
        W_hat = o.dequant(S.pack_int4(q2), s2, z2, G)
        if not np.array_equal(W_hat, w.astype(np.float64)):
            return False
    return True


def check_rtn_error_bound(o, seed=0) -> bool:
    """Off the grid, round-to-nearest puts every dequantised weight within half
    a step of the original: |w - W_hat| <= s/2, plus at most 16 * 2^-11 * s at
    the top of a group, where the fp16 rounding of s = (hi - lo)/15 can push
    the largest weight just past code 15 before clipping."""
    rng = np.random.default_rng(seed)
    N, K = 32, 512
    for G in (128, K):
        w = rng.normal(0, 0.02, size=(N, K)).astype(np.float32)
        q, s, z = S.rtn_quantize(w, G)
        W_hat = o.dequant(S.pack_int4(q), s, z, G)
        s64 = s.view(np.float16).astype(np.float64)[:, np.arange(K) // G]
        err = np.abs(W_hat - w.astype(np.float64))
        if not np.all(err <= (0.5 + 16 * 2.0 ** -11) * s64 + 1e-15):
            return False
        # and the bound is attained up to a few percent (it is not vacuous)
        if err.max() < 0.4 * s64.min():
            return False
    return True


def _code(layer, n, k):
    """One weight code read from the packed words by the documented layouts,
    scalar by scalar (4-bit: nibble k % 8 of word k // 8; 3-bit: block k // 32,
    position t = 2i + o, low two bits from word 0 (i < 8) or word 1 at bit
    2 (i % 8) + 16 o, high bit from word 2 at bit i + 16 o)."""
    row = layer.qweight[n]
    if getattr(layer, "weight_bits", 4) != 3:
        return (int(row[k // 8]) >> (4 * (k % 8))) & 15
    j, t = divmod(k, 32)
    i, o = divmod(t, 2)
    lo_word = int(row[3 * j + (0 if i < 8 else 1)])
    lo = (lo_word >> (2 * (i % 8) + 16 * o)) & 3
    hi = (int(row[3 * j + 2]) >> (i + 16 * o)) & 1
    return lo | (hi << 2)


def _brute(layer):
    """Scalar exact-rational evaluation of Eq. 3 (gate ONE or SIGMOID with the
    sigmoid taken in float64)."""
    dt = layer.act_dtype
    M, N, K, r = layer.M, layer.N, layer.K, layer.rank
    G = layer.group_size
    xs = S.from_bits(layer.x, dt)
    As = S.from_bits(layer.A, dt)
    Bs = S.from_bits(layer.B, dt)
    wg = S.from_bits(layer.w_g, dt)
    sc = layer.scales.view(np.float16)
    Y = [[None] * N for _ in range(M)]
    for m in range(M):
        u = [sum(Fraction(float(xs[m][k])) * Fraction(float(As[j][k])) for k in range(K))
             for j in range(r)]
        if layer.gate_kind == S.GATE_ONE:
            g = Fraction(1)
        else:
            t = sum(Fraction(float(xs[m][k])) * Fraction(float(wg[k])) for k in range(K))
            t = float(t) + layer.b_g
            g = Fraction(1.0 / (1.0 + math.exp(-t)) if t >= 0 else math.exp(t) / (1 + math.exp(t)))
        for n in range(N):
            acc = Fraction(0)
            for k in range(K):
                code = _code(layer, n, k)
                zz = int(layer.zeros[n][k // G])
                ss = Fraction(float(sc[n][k // G]))
                acc += Fraction(code - zz) * ss * Fraction(float(xs[m][k]))
            ec = sum(Fraction(float(Bs[n][j])) * u[j] for j in range(r))
            Y[m][n] = acc + Fraction(layer.alpha) * g * ec
    return Y


def check_brute_force(o, seed=0) -> bool:
    cases = [dict(M=2, N=5, K=16, group_size=8, rank=3, gate_kind=S.GATE_ONE, alpha=0.75),
             dict(M=3, N=4, K=24, group_size=24, rank=2, gate_kind=S.GATE_SIGMOID_LINEAR, alpha=1.0),
             dict(M=1, N=3, K=32, group_size=16, rank=1, gate_kind=S.GATE_SIGMOID_LINEAR, alpha=2.0),
             dict(M=2, N=3, K=16, group_size=16, rank=0, gate_kind=S.GATE_ONE, alpha=1.0),
             dict(M=2, N=16, K=16, group_size=8, rank=2, gate_kind=S.GATE_ONE, alpha=1.0)]
    for i, c in enumerate(cases):
        for dt in (S.F16, S.BF16):
            layer = S.make_layer(seed=seed + i, act_dtype=dt, ec_std=0.3, wg_std=0.4,
                                 b_g=0.1, **c)
            want = _brute(layer)
            got = o.w4ec_linear(layer)
            for m in range(layer.M):
                for n in range(layer.N):
                    wv = float(want[m][n])
                    if abs(got[m][n] - wv) > 1e-12 * max(1.0, abs(wv)):
                        return False
    return True


def check_integer_grid_exact(o, seed=0) -> bool:
    """Small-integer activations, factors and power-of-two scales: every
    partial sum is an exactly representable float64, so the oracle must equal
    exact rational arithmetic with no tolerance."""
    rng = np.random.default_rng(seed)
    M, N, K, r, G = 3, 7, 64, 4, 16
    q = rng.integers(0, 16, size=(N, K))
    z = rng.integers(0, 16, size=(N, K // G))
    s = 2.0 ** rng.integers(-3, 3, size=(N, K // G))
    x = rng.integers(-4, 5, size=(M, K)).astype(np.float32)
    A = rng.integers(-3, 4, size=(r, K)).astype(np.float32)
    B = rng.integers(-3, 4, size=(N, r)).astype(np.float32)
    layer = S.Layer(M=M, N=N, K=K, group_size=G, act_dtype=S.F16, rank=r,
                    gate_kind=S.GATE_ONE, qweight=S.pack_int4(q),
                    scales=_f16_bits(s), zeros=z.astype(np.uint8),
                    x=S.to_bits(x, S.F16), A=S.to_bits(A, S.F16), B=S.to_bits(B, S.F16),
                    w_g=S.to_bits(np.zeros(K), S.F16), b_g=0.0, alpha=0.5,
                    W1=S.to_bits(np.zeros((4 * r, r)), S.F16), b1=S.to_bits(np.zeros(4 * r), S.F16),
                    W2=S.to_bits(np.zeros((r, 4 * r)), S.F16), b2=S.to_bits(np.zeros(r), S.F16))
    got = o.w4ec_linear(layer)
    grp = np.arange(K) // G
    for m in range(M):
        for n in range(N):
            acc = Fraction(0)
            for k in range(K):
                acc += Fraction(int(q[n, k]) - int(z[n, grp[k]])) * Fraction(float(s[n, grp[k]])) * int(x[m, k])
            for j in range(r):
                uj = sum(int(x[m, k]) * int(A[j, k]) for k in range(K))
                acc += Fraction(1, 2) * int(B[n, j]) * uj
            if Fraction(float(got[m, n])) != acc:
                return False
    return True


def check_reductions(o, seed=0) -> bool:
    """r = 0, gate == 0 (b_g = -1e4), A == 0 and B == 0 all give X W_hat^T;
    q == z (W_hat == 0) leaves exactly the EC term."""
    base = S.make_layer(M=5, N=48, K=256, group_size=128, rank=8, seed=seed,
                        gate_kind=S.GATE_SIGMOID_LINEAR)
    W_hat = o.dequant(base.qweight, base.scales, base.zeros, 128)
    y_plain = S.from_bits(base.x, S.F16).astype(np.float64) @ W_hat.T
    ok = np.allclose(o.w4_linear_layer(base), y_plain, rtol=0, atol=1e-12)
    off = copy.copy(base)
    off.b_g = -1.0e4
    ok &= np.array_equal(o.w4ec_linear(off), o.w4_linear_layer(base))
    r0 = copy.copy(base)
    r0.rank = 0
    r0.A = base.A[:0]
    r0.B = base.B[:, :0]
    ok &= np.array_equal(o.w4ec_linear(r0), o.w4_linear_layer(base))
    a0 = copy.copy(base)
    a0.A = np.zeros_like(base.A)
    ok &= np.array_equal(o.w4ec_linear(a0), o.w4_linear_layer(base))
    # W_hat == 0: codes equal to the zero point everywhere
    wz = copy.copy(base)
    z = np.full_like(base.zeros, 7)
    wz.zeros = z
    wz.qweight = S.pack_int4(np.full((base.N, base.K), 7))
    x = S.from_bits(base.x, S.F16).astype(np.float64)
    A = S.from_bits(base.A, S.F16).astype(np.float64)
    B = S.from_bits(base.B, S.F16).astype(np.float64)
    wgv = S.from_bits(base.w_g, S.F16).astype(np.float64)
    t = x @ wgv + base.b_g
    g = np.where(t >= 0, 1 / (1 + np.exp(-np.abs(t))), np.exp(-np.abs(t)) / (1 + np.exp(-np.abs(t))))
    ec = (g[:, None] * (x @ A.T)) @ B.T * base.alpha
    ok &= np.allclose(o.w4ec_linear(wz), ec, rtol=1e-13, atol=1e-15)
    return bool(ok)


def check_sigmoid_half(o) -> bool:
    """w_g = 0, b_g = 0 gives g = 1/2 exactly: Y = X W^T + (alpha/2) (X A^T) B^T."""
    base = S.make_layer(M=3, N=32, K=128, group_size=128, rank=4, seed=3)
    h = copy.copy(base)
    h.w_g = np.zeros_like(base.w_g)
    h.b_g = 0.0
    g = o.gate_sigmoid_linear(S.from_bits(h.x, S.F16), S.from_bits(h.w_g, S.F16), 0.0)
    if not np.all(g == 0.5):
        return False
    x = S.from_bits(base.x, S.F16).astype(np.float64)
    A = S.from_bits(base.A, S.F16).astype(np.float64)
    B = S.from_bits(base.B, S.F16).astype(np.float64)
    want = o.w4_linear_layer(base) + 0.5 * base.alpha * (x @ A.T) @ B.T
    return bool(np.allclose(o.w4ec_linear(h), want, rtol=1e-13, atol=1e-15))


def check_tanh_static_lora(o, seed=0) -> bool:
    """W2 = 0, b2 = 0 makes gamma == 1, and Eq. 3 becomes the static
    compensator of Eq. 2, y = (W_hat + W_comp) x with W_comp = alpha B A, which
    is checked as one dense product with the explicit matrix."""
    base = S.make_layer(M=4, N=40, K=128, group_size=64, rank=6, seed=seed,
                        gate_kind=S.GATE_TANH_MLP, alpha=0.75)
    st = copy.copy(base)
    st.W2 = np.zeros_like(base.W2)
    st.b2 = np.zeros_like(base.b2)
    W_hat = o.dequant(base.qweight, base.scales, base.zeros, 64)
    A = S.from_bits(base.A, S.F16).astype(np.float64)
    B = S.from_bits(base.B, S.F16).astype(np.float64)
    W_eff = W_hat + 0.75 * (B @ A)
    x = S.from_bits(base.x, S.F16).astype(np.float64)
    return bool(np.allclose(o.w4ec_linear(st), x @ W_eff.T, rtol=1e-12, atol=1e-14))


def check_factored_form(o, seed=0) -> bool:
    """Eq. 4: per token, y_m = (W_hat + alpha B diag(gamma(A x_m)) A) x_m."""
    base = S.make_layer(M=3, N=24, K=128, group_size=128, rank=5, seed=seed,
                        gate_kind=S.GATE_TANH_MLP, alpha=1.25, ec_std=0.2)
    y = o.w4ec_linear(base)
    W_hat = o.dequant(base.qweight, base.scales, base.zeros, 128)
    f = lambda a: S.from_bits(a, S.F16).astype(np.float64)  # noqa: E731
    x, A, B = f(base.x), f(base.A), f(base.B)
    for m in range(base.M):
        u = A @ x[m]
        hid = np.maximum(f(base.W1) @ u + f(base.b1), 0.0)
        gam = 1.0 + np.tanh(f(base.W2) @ hid + f(base.b2))
        W_eff = W_hat + 1.25 * B @ np.diag(gam) @ A
        if not np.allclose(y[m], W_eff @ x[m], rtol=1e-12, atol=1e-14):
            return False
    return True


def check_gate_ranges(o) -> bool:
    """gamma in (0, 2); gamma -> 2 for a large positive b2, -> 0 for a large
    negative b2; sigma is finite and symmetric at +-1e4."""
    rng = np.random.default_rng(0)
    u = rng.normal(0, 3, size=(50, 4))
    W1 = rng.normal(0, 1, size=(16, 4))
    W2 = rng.normal(0, 1, size=(4, 16))
    gam = o.gate_tanh_mlp(u, W1, np.zeros(16), W2, np.zeros(4))
    ok = bool(np.all((gam >= 0) & (gam <= 2)))
    ok &= bool(np.allclose(o.gate_tanh_mlp(u, W1, np.zeros(16), W2 * 0, np.full(4, 40.0)), 2.0))
    ok &= bool(np.allclose(o.gate_tanh_mlp(u, W1, np.zeros(16), W2 * 0, np.full(4, -40.0)), 0.0))
    s = o.sigmoid(np.array([-1e4, 0.0, 1e4, 3.0, -3.0]))
    ok &= bool(s[0] == 0.0 and s[1] == 0.5 and s[2] == 1.0 and abs(s[3] + s[4] - 1) <= 4e-16)
    return ok


def check_dequant_bits_contract(o, seed=0) -> bool:
    """The bit-exact dequantisation reference equals a single nearest-even
    rounding of the exact product: cross-checked against torch's float32 ->
    fp16/bf16 cast (an independent rounding implementation) over every code
    and zero point with random fp16 scales."""
    import torch
    rng = np.random.default_rng(seed)
    N, K = 16 * 16, 128
    z = np.repeat(np.arange(16), 16).reshape(N, 1)
    q = np.tile(np.arange(16), (N, K // 16))
    s = rng.uniform(1e-4, 4.0, size=(N, 1)).astype(np.float16)
    qw = S.pack_int4(q)
    exact = ((q - z) * s.astype(np.float64)).astype(np.float32)
    for dt, tdt in ((O.F16, torch.float16), (O.BF16, torch.bfloat16)):
        want = torch.from_numpy(exact).to(tdt).view(torch.int16).numpy().view(np.uint16)
        got = o.dequant_bits(qw, s.view(np.uint16), z.astype(np.uint8), K, dt)
        if not np.array_equal(got, want):
            return False
    return True


def _brute_int8(layer):
    """Scalar exact-rational evaluation of Eq. 3 with INT8 factors taken from
    the raw codes: A[j][k] = a_scale[j] q_A[j][k], B[n][j] = b_scale[n] q_B[n][j]
    (gate ONE or SIGMOID, the sigmoid in float64)."""
    dt = layer.act_dtype
    M, N, K, r = layer.M, layer.N, layer.K, layer.rank
    G = layer.group_size
    xs = S.from_bits(layer.x, dt)
    wg = S.from_bits(layer.w_g, dt)
    sc = layer.scales.view(np.float16)
    A = [[Fraction(float(layer.a_scale[j])) * int(layer.A_q[j][k]) for k in range(K)]
         for j in range(r)]
    B = [[Fraction(float(layer.b_scale[n])) * int(layer.B_q[n][j]) for j in range(r)]
         for n in range(N)]
    Y = [[None] * N for _ in range(M)]
    for m in range(M):
        u = [sum(Fraction(float(xs[m][k])) * A[j][k] for k in range(K)) for j in range(r)]
        if layer.gate_kind == S.GATE_ONE:
            g = Fraction(1)
        else:
            t = sum(Fraction(float(xs[m][k])) * Fraction(float(wg[k])) for k in range(K))
            t = float(t) + layer.b_g
            g = Fraction(1.0 / (1.0 + math.exp(-t)) if t >= 0 else math.exp(t) / (1 + math.exp(t)))
        for n in range(N):
            acc = Fraction(0)
            for k in range(K):
                word = int(layer.qweight[n][k // 8])
                code = (word >> (4 * (k % 8))) & 15
                acc += (Fraction(code - int(layer.zeros[n][k // G])) *
                        Fraction(float(sc[n][k // G])) * Fraction(float(xs[m][k])))
            Y[m][n] = acc + Fraction(layer.alpha) * g * sum(B[n][j] * u[j] for j in range(r))
    return Y


def check_int8_brute_force(o, seed=0) -> bool:
    """INT8 per-channel factors: the oracle against exact rationals built
    from the codes and scales, on tiny layers of both dtypes."""
    cases = [dict(M=2, N=5, K=16, group_size=8, rank=3, gate_kind=S.GATE_ONE, alpha=0.75),
             dict(M=3, N=4, K=24, group_size=24, rank=2, gate_kind=S.GATE_SIGMOID_LINEAR, alpha=1.0),
             dict(M=1, N=6, K=16, group_size=16, rank=4, gate_kind=S.GATE_SIGMOID_LINEAR, alpha=2.0)]
    for i, c in enumerate(cases):
        for dt in (S.F16, S.BF16):
            layer = S.make_layer(seed=seed + 40 + i, act_dtype=dt, ec_std=0.3, wg_std=0.4,
                                 b_g=0.1, ab_int8=True, **c)
            want = _brute_int8(layer)
            got = o.w4ec_linear(layer)
            rows = np.arange(layer.N)[::2]
            got_rows = o.w4ec_linear_rows(layer, rows)
            for m in range(layer.M):
                for n in range(layer.N):
                    wv = float(want[m][n])
                    if abs(got[m][n] - wv) > 1e-12 * max(1.0, abs(wv)):
                        return False
                for i2, n in enumerate(rows):
                    wv = float(want[m][n])
                    if abs(got_rows[m][i2] - wv) > 1e-12 * max(1.0, abs(wv)):
                        return False
    return True


def check_int8_golden(o) -> bool:
    """Hand-worked INT8 factors (tests/golden/int8_factors.json)."""
    g = _load("int8_factors.json")
    d = g["dequant"]
    if not np.array_equal(o.dequant_int8(np.array(d["q"], np.int8), np.array(d["scale"], np.float32)),
                          np.array(d["want"])):
        return False
    e = g["ec"]
    A = o.dequant_int8(np.array(e["A_q"], np.int8), np.array(e["a_scale"], np.float32))
    B = o.dequant_int8(np.array(e["B_q"], np.int8), np.array(e["b_scale"], np.float32))
    x = np.array(e["x"])
    y = o.w4ec_linear_f64(x, np.zeros((B.shape[0], x.shape[1])), A, B, 1.0, o.GATE_ONE)
    return np.array_equal(y, np.array(e["want"]))


def check_tail_golden(o) -> bool:
    """Hand-worked residual + RMSNorm (tests/golden/post_ec_tail.json)."""
    g = _load("post_ec_tail.json")
    h, yn = o.post_ec_tail(np.array(g["y"]), np.array(g["residual"]), np.array(g["norm_w"]),
                           g["eps"])
    return np.array_equal(h, np.array(g["h"])) and np.array_equal(yn, np.array(g["y_norm"]))


def check_tail_properties(o, seed=0) -> bool:
    """RMSNorm facts: a constant row c gives c w / sqrt(c^2 + eps); at eps = 0
    the normalised row (before the weight) has mean square 1 and the result
    does not change when the row is scaled; residual None equals a zero
    residual; the residual enters once."""
    rng = np.random.default_rng(seed)
    w = rng.normal(1.0, 0.2, size=6)
    for c in (3.0, -0.25):
        _, yn = o.post_ec_tail(np.full((1, 6), c), None, w, 0.5)
        if not np.allclose(yn[0], c * w / math.sqrt(c * c + 0.5), rtol=1e-15, atol=0):
            return False
    y = rng.normal(size=(5, 6))
    r = rng.normal(size=(5, 6))
    _, a = o.post_ec_tail(y, r, np.ones(6), 0.0)
    if not np.allclose(np.mean(a * a, axis=1), 1.0, rtol=1e-14):
        return False
    _, b = o.post_ec_tail(7.5 * y, 7.5 * r, np.ones(6), 0.0)
    if not np.allclose(a, b, rtol=1e-14):
        return False
    h0, n0 = o.post_ec_tail(y, None, w, 1e-3)
    h1, n1 = o.post_ec_tail(y, np.zeros_like(y), w, 1e-3)
    h2, _ = o.post_ec_tail(y, r, w, 1e-3)
    return (np.array_equal(h0, h1) and np.array_equal(n0, n1)
            and np.allclose(h2, y + r, rtol=0, atol=1e-15))


def check_unpack3_fixed_words(o) -> bool:
    """3-bit layout pin: hand-decoded blocks of three words."""
    cases = [((0xFFFFFFFF, 0, 0), [3] * 16 + [0] * 16),
             ((0, 0, 0x0000FFFF), [4, 0] * 16),
             ((0, 0, 0xFFFF0000), [0, 4] * 16),
             ((0x00010000, 0, 0x00010000), [0, 5] + [0] * 30),
             ((0, 0xC0000000, 0x80000000), [0] * 31 + [7]),
             ((0x0000000C, 0, 0x00000002), [0, 0, 7] + [0] * 29),
             ((0, 0x00000003, 0x00000100), [0] * 16 + [7] + [0] * 15)]
    for words, want in cases:
        w = np.array([list(words) * 2], dtype=np.uint32)  # two blocks, same contents
        if o.unpack_int3(w).tolist() != [want * 2]:
            return False
    return True


def check_unpack3_exhaustive(o) -> bool:
    """Every 3-bit code at every one of the 32 positions of a block (second
    block of a row) decodes to itself, through the generator's packer, and
    leaves the other positions zero; the scalar reading of the layout agrees."""
    for v in range(8):
        for t in range(32):
            q = np.zeros((1, 64), dtype=np.int64)
            q[0, 32 + t] = v
            w = S.pack_int3(q)
            if not np.array_equal(o.unpack_int3(w), q):
                return False
            lay = types.SimpleNamespace(qweight=w, weight_bits=3)
            if _code(lay, 0, 32 + t) != v:
                return False
    return True


def check_rtn3_grid_roundtrip(o, seed=0) -> bool:
    """3-bit weights built on the grid (codes 0 and 7 in every group, dyadic
    fp16 scales) come back exactly through the 3-bit RTN and dequant."""
    rng = np.random.default_rng(seed)
    N, K = 24, 256
    for G in (K, 128, 64):
        s = 2.0 ** rng.integers(-9, -3, size=(N, K // G))
        z = rng.integers(0, 8, size=(N, K // G))
        q = rng.integers(0, 8, size=(N, K))
        qg = q.reshape(N, K // G, G)
        qg[:, :, 0] = 0
        qg[:, :, 1] = 7
        q = qg.reshape(N, K)
        grp = np.arange(K) // G
        w = ((q - z[:, grp]) * s[:, grp]).astype(np.float32)
        q2, s2, z2 = S.rtn_quantize(w, G, bits=3)
        if q2.max() > 7 or z2.max() > 7:
            return False
        W_hat = o.dequant(S.pack_int3(q2), s2, z2, G, bits=3)
        if not np.array_equal(W_hat, w.astype(np.float64)):
            return False
    return True


def check_brute_force_w3(o, seed=0) -> bool:
    """Eq. 3 on 3-bit layers against exact rationals (codes read scalar by
    scalar from the documented layout), both dtypes, every output."""
    cases = [dict(M=2, N=5, K=64, group_size=32, rank=3, gate_kind=S.GATE_ONE, alpha=0.75),
             dict(M=3, N=4, K=96, group_size=96, rank=2, gate_kind=S.GATE_SIGMOID_LINEAR, alpha=1.0),
             dict(M=1, N=6, K=32, group_size=32, rank=0, gate_kind=S.GATE_ONE, alpha=1.0)]
    for i, c in enumerate(cases):
        for dt in (S.F16, S.BF16):
            layer = S.make_layer(seed=seed + 80 + i, act_dtype=dt, ec_std=0.3, wg_std=0.4,
                                 b_g=0.1, weight_bits=3, **c)
            want = _brute(layer)
            got = o.w4ec_linear(layer)
            rows = np.array([layer.N - 1, 0])
            got_rows = o.w4ec_linear_rows(layer, rows)
            for m in range(layer.M):
                for n in range(layer.N):
                    wv = float(want[m][n])
                    if abs(got[m][n] - wv) > 1e-12 * max(1.0, abs(wv)):
                        return False
                for i2, n in enumerate(rows):
                    wv = float(want[m][n])
                    if abs(got_rows[m][i2] - wv) > 1e-12 * max(1.0, abs(wv)):
                        return False
    return True


def check_dequant3_bits_contract(o, seed=0) -> bool:
    """3-bit bit-exact dequantisation: one nearest-even rounding of the exact
    product, cross-checked against torch's float32 -> fp16/bf16 cast over every
    code and zero point."""
    import torch
    rng = np.random.default_rng(seed)
    N, K = 8 * 8, 128
    z = np.repeat(np.arange(8), 8).reshape(N, 1)
    q = np.tile(np.arange(8), (N, K // 8))
    s = rng.uniform(1e-4, 4.0, size=(N, 1)).astype(np.float16)
    exact = ((q - z) * s.astype(np.float64)).astype(np.float32)
    for dt, tdt in ((O.F16, torch.float16), (O.BF16, torch.bfloat16)):
        want = torch.from_numpy(exact).to(tdt).view(torch.int16).numpy().view(np.uint16)
        got = o.dequant_bits(S.pack_int3(q), s.view(np.uint16), z.astype(np.uint8), K, dt, bits=3)
        if not np.array_equal(got, want):
            return False
    return True


def check_tolerance_cases(o) -> bool:
    """The parity bar on hand-worked cases (relative Frobenius error
    ||y - y_ref|| / ||y_ref|| and max |y - y_ref| against a fraction of
    max |y_ref|, both inclusive; the reference is always the second
    argument). Values below are chosen so that every quantity is exact in
    float64, or sits well clear of the bound."""
    tc = o.tolerance_check
    cases = []
    # default bar (5e-3, 1e-2): relF just inside and just outside
    yr = np.array([[100.0, 0.0, 0.0, 0.0]])
    cases.append((yr + [[0, 0.49, 0, 0]], yr, {}, True))
    cases.append((yr + [[0, 0.51, 0, 0]], yr, {}, False))
    # a wide reference keeps relF small: the max bound decides
    wide = np.ones((1, 10000))
    d = np.zeros((1, 10000))
    d[0, 17] = 0.0099
    cases.append((wide + d, wide, {}, True))
    d[0, 17] = 0.0101
    cases.append((wide + d, wide, {}, False))
    # a zero reference: only an exact zero passes
    z = np.zeros((2, 3))
    cases.append((z.copy(), z, {}, True))
    tiny = z.copy()
    tiny[1, 2] = 1e-30
    cases.append((tiny, z, {}, False))
    # exact boundaries (dyadic values): both bounds are inclusive
    yr2 = np.array([[4.0, 0.0]])
    y2 = np.array([[4.0, 1.0]])
    cases.append((y2, yr2, dict(rel_frob=0.25, max_rel=0.5), True))
    cases.append((y2, yr2, dict(rel_frob=1.0, max_rel=0.25), True))
    cases.append((y2, yr2, dict(rel_frob=0.2499, max_rel=0.5), False))
    cases.append((y2, yr2, dict(rel_frob=1.0, max_rel=0.2499), False))
    # the reference's norm and max are the denominators, not the result's:
    # y = 2, y_ref = 1 has relF = 1 and max|d| = 1 against max|y_ref| = 1
    one = np.array([[1.0, 0.0]])
    two = np.array([[2.0, 0.0]])
    cases.append((two, one, dict(rel_frob=0.6, max_rel=1.0), False))
    cases.append((one, two, dict(rel_frob=0.6, max_rel=1.0), True))
    cases.append((two, one, dict(rel_frob=10.0, max_rel=0.6), False))
    cases.append((one, two, dict(rel_frob=10.0, max_rel=0.6), True))
    # magnitudes: a negative reference bounds by its absolute value
    cases.append((np.array([[-4.0, 1.0]]), np.array([[-4.0, 0.0]]),
                  dict(rel_frob=1.0, max_rel=0.25), True))
    for y, y_ref, kw, want in cases:
        if bool(tc(y, y_ref, **kw)[0]) != want:
            return False
    # the reported figures themselves
    ok, relf, mx, bound = tc(y2, yr2, rel_frob=0.25, max_rel=0.5)
    return ok and relf == 0.25 and mx == 1.0 and bound == 2.0


def check_rows_brute_force(o, seed=0) -> bool:
    """Eq. 3 on a subset of output columns (activation-dtype factors, both
    dtypes, gates ONE and SIGMOID_LINEAR) against exact rationals, column by
    column; the rows include the first and last and come in a scrambled
    order."""
    cases = [dict(M=2, N=7, K=16, group_size=8, rank=3, gate_kind=S.GATE_ONE, alpha=0.75),
             dict(M=3, N=6, K=24, group_size=24, rank=2, gate_kind=S.GATE_SIGMOID_LINEAR, alpha=1.0),
             dict(M=2, N=5, K=16, group_size=16, rank=0, gate_kind=S.GATE_ONE, alpha=1.0)]
    for i, c in enumerate(cases):
        for dt in (S.F16, S.BF16):
            layer = S.make_layer(seed=seed + 60 + i, act_dtype=dt, ec_std=0.3, wg_std=0.4,
                                 b_g=-0.2, **c)
            want = _brute(layer)
            rows = np.array([layer.N - 1, 0, 3, 1])
            got = o.w4ec_linear_rows(layer, rows)
            if got.shape != (layer.M, len(rows)):
                return False
            for m in range(layer.M):
                for i2, n in enumerate(rows):
                    wv = float(want[m][n])
                    if abs(got[m][i2] - wv) > 1e-12 * max(1.0, abs(wv)):
                        return False
    return True


def check_rows_tanh_factored(o, seed=0) -> bool:
    """Sampled columns under the paper's tanh gate, both dtypes, against the
    factored form (Eq. 4) built per token: y_m[n] = (W_hat[n] + alpha
    B[n] diag(gamma(A x_m)) A) x_m."""
    for dt in (S.F16, S.BF16):
        base = S.make_layer(M=3, N=40, K=128, group_size=64, rank=5, seed=seed + 7, act_dtype=dt,
                            gate_kind=S.GATE_TANH_MLP, alpha=0.5, ec_std=0.2)
        rows = np.array([39, 2, 17, 0])
        got = o.w4ec_linear_rows(base, rows)
        f = lambda a: S.from_bits(a, dt).astype(np.float64)  # noqa: E731
        W_hat = o.dequant(base.qweight, base.scales, base.zeros, 64)
        x, A, B = f(base.x), f(base.A), f(base.B)
        for m in range(base.M):
            u = A @ x[m]
            hid = np.maximum(f(base.W1) @ u + f(base.b1), 0.0)
            gam = 1.0 + np.tanh(f(base.W2) @ hid + f(base.b2))
            for i2, n in enumerate(rows):
                w_eff = W_hat[n] + 0.5 * (B[n] * gam) @ A
                if not np.isclose(got[m, i2], w_eff @ x[m], rtol=1e-12, atol=1e-14):
                    return False
    return True


PINS = [check_unpack_fixed_words, check_unpack_exhaustive, check_golden_examples,
        check_rounding_fixtures, check_rtn_grid_roundtrip, check_rtn_error_bound,
        check_brute_force, check_integer_grid_exact, check_reductions,
        check_sigmoid_half, check_tanh_static_lora, check_factored_form,
        check_gate_ranges, check_dequant_bits_contract, check_int8_brute_force,
        check_int8_golden, check_tail_golden, check_tail_properties,
        check_tolerance_cases, check_rows_brute_force, check_rows_tanh_factored,
        check_unpack3_fixed_words, check_unpack3_exhaustive, check_rtn3_grid_roundtrip,
        check_brute_force_w3, check_dequant3_bits_contract]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    assert pin(O)


# ---------------------------------------------------------------------------
# planted mistakes: each broken copy of the oracle must fail some pin
# ---------------------------------------------------------------------------

def _mutant(**overrides):
    m = types.ModuleType("oracle_mutant")
    m.__dict__.update({k: v for k, v in O.__dict__.items() if not k.startswith("__")})
    m.__dict__.update(overrides)
    # re-bind module-level functions so that internal calls see the overrides
    for name, fn in list(m.__dict__.items()):
        if isinstance(fn, types.FunctionType) and name not in overrides:
            m.__dict__[name] = types.FunctionType(fn.__code__, m.__dict__, name,
                                                  fn.__defaults__, fn.__closure__)
    return m


def _unpack_reversed(qweight):
    w = np.asarray(qweight, dtype=np.uint32)
    n, kw = w.shape
    q = np.empty((n, kw, 8), dtype=np.int64)
    for i in range(8):
        q[:, :, 7 - i] = (w >> np.uint32(4 * i)) & np.uint32(0xF)
    return q.reshape(n, kw * 8)


def _dequant_plus_zero(qweight, scales_bits, zeros, group_size):
    q = O.unpack_int4(qweight)
    n, k = q.shape
    g = k if group_size in (0, k) else group_size
    s = O.bits_to_f64(scales_bits, O.F16)
    grp = np.arange(k) // g
    return (q + np.asarray(zeros, np.int64)[:, grp]) * s[:, grp]


def _dequant_wrong_group(qweight, scales_bits, zeros, group_size):
    q = O.unpack_int4(qweight)
    n, k = q.shape
    g = k if group_size in (0, k) else group_size
    s = O.bits_to_f64(scales_bits, O.F16)
    grp = (np.arange(k) % (k // g))  # interleaved instead of contiguous groups
    return (q - np.asarray(zeros, np.int64)[:, grp]) * s[:, grp]


def _ec_no_alpha(x, W_hat, A, B, alpha, gate_kind, w_g=None, b_g=0.0, W1=None, b1=None,
                 W2=None, b2=None):
    return O.w4ec_linear_f64(x, W_hat, A, B, 1.0, gate_kind, w_g, b_g, W1, b1, W2, b2)


def _ec_minus(x, W_hat, A, B, alpha, gate_kind, w_g=None, b_g=0.0, W1=None, b1=None,
              W2=None, b2=None):
    y0 = O.w4_linear(x, W_hat)
    y1 = O.w4ec_linear_f64(x, W_hat, A, B, alpha, gate_kind, w_g, b_g, W1, b1, W2, b2)
    return y0 - (y1 - y0)


def _gate_no_one(u, W1, b1, W2, b2):
    return O.gate_tanh_mlp(u, W1, b1, W2, b2) - 1.0


def _gate_no_relu(u, W1, b1, W2, b2):
    u = np.asarray(u, np.float64)
    hid = u @ np.asarray(W1, np.float64).T + np.asarray(b1, np.float64)
    return 1.0 + np.tanh(hid @ np.asarray(W2, np.float64).T + np.asarray(b2, np.float64))


def _sigmoid_of_wrong_sign(x, w_g, b_g):
    return O.sigmoid(-(np.asarray(x, np.float64) @ np.asarray(w_g, np.float64) + b_g))


def _round_bf16_truncate(v, dtype):
    if dtype == O.BF16:
        f32 = np.asarray(v, np.float64).astype(np.float32)
        return (f32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    return O.round_f64_to_bits(v, dtype)


def _w4_linear_transposed_b(x, W_hat):
    x = np.asarray(x, np.float64)
    W = np.asarray(W_hat, np.float64)
    if W.shape[0] == W.shape[1]:
        return x @ W  # forgets the transpose on square weights
    return x @ W.T


def _int8_scale_dropped(q, scale):
    return np.asarray(q, np.float64)


def _int8_scale_fp16(q, scale):
    s16 = np.asarray(scale, np.float32).astype(np.float16).astype(np.float64)
    return s16[:, None] * np.asarray(q, np.float64)


def _tail_no_residual(y, residual, norm_w, eps):
    return O.post_ec_tail(y, None, norm_w, eps)


def _tail_sum_not_mean(y, residual, norm_w, eps):
    h = np.asarray(y, np.float64) + (0 if residual is None else np.asarray(residual, np.float64))
    return h, h / np.sqrt(np.sum(h * h, axis=1, keepdims=True) + eps) * np.asarray(norm_w)[None, :]


def _tail_eps_outside(y, residual, norm_w, eps):
    h = np.asarray(y, np.float64) + (0 if residual is None else np.asarray(residual, np.float64))
    return h, h / (np.sqrt(np.mean(h * h, axis=1, keepdims=True)) + eps) * np.asarray(norm_w)[None, :]


def _tol_wrong_denominator(y, y_ref, rel_frob=5e-3, max_rel=1e-2):
    y = np.asarray(y, np.float64)
    y_ref = np.asarray(y_ref, np.float64)
    diff = y - y_ref
    den = np.linalg.norm(y)
    relf = float(np.linalg.norm(diff) / den) if den > 0 else float(np.linalg.norm(diff))
    mx = float(np.abs(diff).max(initial=0.0))
    bound = max_rel * float(np.abs(y_ref).max(initial=0.0))
    return (relf <= rel_frob) and (mx <= bound if bound > 0 else mx == 0.0), relf, mx, bound


def _tol_strict(y, y_ref, rel_frob=5e-3, max_rel=1e-2):
    ok, relf, mx, bound = O.tolerance_check(y, y_ref, rel_frob, max_rel)
    return (relf < rel_frob) and (mx < bound if bound > 0 else mx == 0.0), relf, mx, bound


def _tol_bound_from_result(y, y_ref, rel_frob=5e-3, max_rel=1e-2):
    _, relf, mx, _ = O.tolerance_check(y, y_ref, rel_frob, max_rel)
    bound = max_rel * float(np.abs(np.asarray(y, np.float64)).max(initial=0.0))
    return (relf <= rel_frob) and (mx <= bound if bound > 0 else mx == 0.0), relf, mx, bound


def _tol_zero_reference_passes(y, y_ref, rel_frob=5e-3, max_rel=1e-2):
    ok, relf, mx, bound = O.tolerance_check(y, y_ref, rel_frob, max_rel)
    return (ok or bound == 0.0), relf, mx, bound


def _tol_signed_max(y, y_ref, rel_frob=5e-3, max_rel=1e-2):
    _, relf, mx, _ = O.tolerance_check(y, y_ref, rel_frob, max_rel)
    bound = max_rel * float(np.asarray(y_ref, np.float64).max(initial=0.0))
    return (relf <= rel_frob) and (mx <= bound if bound > 0 else mx == 0.0), relf, mx, bound


def _rows_b_unselected(layer, rows):
    sub = copy.copy(layer)
    sub.B = layer.B[:len(rows)]  # B's first rows instead of the selected ones
    W_hat = O.dequant(layer.qweight[rows], layer.scales[rows], layer.zeros[rows],
                      layer.group_size)
    dt = layer.act_dtype
    x = O.bits_to_f64(layer.x, dt)
    if layer.rank == 0:
        return O.w4_linear(x, W_hat)
    return O.w4ec_linear_f64(x, W_hat, O.bits_to_f64(layer.A, dt), O.bits_to_f64(sub.B, dt),
                             layer.alpha, layer.gate_kind, w_g=O.bits_to_f64(layer.w_g, dt),
                             b_g=layer.b_g, W1=O.bits_to_f64(layer.W1, dt),
                             b1=O.bits_to_f64(layer.b1, dt), W2=O.bits_to_f64(layer.W2, dt),
                             b2=O.bits_to_f64(layer.b2, dt))


def _rows_act_drops_ec(layer, rows):
    if getattr(layer, "ab_int8", False):
        return O.w4ec_linear_rows(layer, rows)
    W_hat = O.dequant(layer.qweight[rows], layer.scales[rows], layer.zeros[rows],
                      layer.group_size)
    return O.w4_linear(O.bits_to_f64(layer.x, layer.act_dtype), W_hat)


def _rows_gate_dropped(layer, rows):
    flat = copy.copy(layer)
    flat.gate_kind = O.GATE_ONE
    return O.w4ec_linear_rows(flat, rows)


def _unpack3_odd_high_from_low_half(qweight):
    q = O.unpack_int3(qweight)
    w = np.asarray(qweight, np.uint32)
    n, nw = w.shape
    hi = w.reshape(n, nw // 3, 3)[:, :, 2]
    qb = q.reshape(n, nw // 3, 32)
    for i in range(16):
        qb[:, :, 2 * i + 1] = (qb[:, :, 2 * i + 1] & 3) | (((hi >> np.uint32(i)) & np.uint32(1)) << np.uint32(2)).astype(np.int64)
    return qb.reshape(n, -1)


def _unpack3_low_words_swapped(qweight):
    w = np.asarray(qweight, np.uint32).copy()
    n, nw = w.shape
    b = w.reshape(n, nw // 3, 3)
    b[:, :, [0, 1]] = b[:, :, [1, 0]]
    return O.unpack_int3(b.reshape(n, nw))


def _dequant_bits_ignored(qweight, scales_bits, zeros, group_size, bits=4):
    return O.dequant(qweight, scales_bits, zeros, group_size, 4)


MUTANTS = {
    "nibble order reversed": dict(unpack_int4=_unpack_reversed),
    "zero point added": dict(dequant=_dequant_plus_zero),
    "groups interleaved": dict(dequant=_dequant_wrong_group),
    "alpha dropped": dict(w4ec_linear_f64=_ec_no_alpha),
    "EC term sign flipped": dict(w4ec_linear_f64=_ec_minus),
    "gate missing the 1 +": dict(gate_tanh_mlp=_gate_no_one),
    "gate missing the ReLU": dict(gate_tanh_mlp=_gate_no_relu),
    "sigmoid argument negated": dict(gate_sigmoid_linear=_sigmoid_of_wrong_sign),
    "bf16 rounding truncates": dict(round_f64_to_bits=_round_bf16_truncate),
    "weight operand not transposed": dict(w4_linear=_w4_linear_transposed_b),
    "INT8 scale dropped": dict(dequant_int8=_int8_scale_dropped),
    "INT8 scale rounded to fp16": dict(dequant_int8=_int8_scale_fp16),
    "tail drops the residual": dict(post_ec_tail=_tail_no_residual),
    "RMSNorm divides by the sum": dict(post_ec_tail=_tail_sum_not_mean),
    "RMSNorm epsilon outside the root": dict(post_ec_tail=_tail_eps_outside),
    "parity bar relative to the result's norm": dict(tolerance_check=_tol_wrong_denominator),
    "parity bar with strict inequalities": dict(tolerance_check=_tol_strict),
    "parity bar's max bound from the result": dict(tolerance_check=_tol_bound_from_result),
    "parity bar passes any zero reference": dict(tolerance_check=_tol_zero_reference_passes),
    "parity bar's max bound from the signed max": dict(tolerance_check=_tol_signed_max),
    "sampled columns take B's first rows": dict(w4ec_linear_rows=_rows_b_unselected),
    "sampled columns drop the EC (act-dtype factors)": dict(w4ec_linear_rows=_rows_act_drops_ec),
    "sampled columns ignore the gate": dict(w4ec_linear_rows=_rows_gate_dropped),
    "3-bit: odd codes' high bit from the low half": dict(unpack_int3=_unpack3_odd_high_from_low_half),
    "3-bit: low-bit words swapped": dict(unpack_int3=_unpack3_low_words_swapped),
    "3-bit codes read as 4-bit": dict(dequant=_dequant_bits_ignored),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistake_is_caught(name):
    mut = _mutant(**MUTANTS[name])
    failed = [p.__name__ for p in PINS if not _safe(p, mut)]
    assert failed, f"planted mistake '{name}' passed every pin"


def _safe(pin, mod):
    try:
        return bool(pin(mod))
    except Exception:
        return False
