"""CPU float64 oracle of the W4+EC linear layer.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute this module: only the tests, the smoke check and the benchmark's CPU
baseline leg use it. It shares no code with the HIP library (no kernels,
headers, helpers, tables or pre/post-processing); its inputs are the stored
tensors produced by the seeded generator, passed in as numpy arrays.

What it computes (SPEAR, section 3.1, Eq. 3, with the quantised backbone of
sections 2.1 and 5.1):

    Y = X . What^T  +  alpha * ( gate(X) (.) (X . A^T) ) . B^T

where What is the dequantised 4-bit (or 3-bit) weight matrix, A [r][K] and B [N][r] are
the EC's low-rank factors and gate() is one of
  * ONE             gamma == 1: the static low-rank compensator (Eq. 2 with
                    W_comp = alpha B A),
  * SIGMOID_LINEAR  a scalar per token g = sigma(w_g . x + b_g),
  * TANH_MLP        the paper's vector gate on the rank-r coordinates u = A x:
                    gamma(u) = 1 + tanh(W2 ReLU(W1 u + b1) + b2) (Eq. 3).

The result has a plain closed-form definition, so each function below is that
definition written out in float64 with numpy; matrix products use numpy's
matmul as a library primitive. All stored inputs (fp16/bf16 bit patterns,
fp16 scales, uint8 zeros) are converted to float64 exactly before use.

Pins (see tests/test_oracle_*.py): brute-force exact rational arithmetic on
tiny shapes, integer-grid exactness, the RTN round trip, reductions to the
plain 4-bit product (r = 0, gate == 0, W_hat == 0), the static-LoRA special
case of the tanh gate, the factored form (Eq. 4), hand-worked golden
fixtures, and planted-mistake checks that each pin catches. The sampled-column
evaluation (w4ec_linear_rows) is pinned column by column against exact
rationals and against the factored form under the tanh gate; the parity bar
itself (tolerance_check) against hand-worked cases at and around both bounds.

INT8 EC factors (the deployed format: A and B stored as int8 codes with one
symmetric scale per output channel) enter as their exact dequantised values
scale[c] * q[c][.]; the rest of the evaluation is unchanged.
"""
from __future__ import annotations

import numpy as np

F16 = 0
BF16 = 1
GATE_ONE = 0
GATE_SIGMOID_LINEAR = 1
GATE_TANH_MLP = 2


# ---------------------------------------------------------------------------
# Stored-format decoding (exact)
# ---------------------------------------------------------------------------

def bits_to_f64(bits, dtype: int) -> np.ndarray:
    """IEEE fp16 or bf16 bit patterns (uint16) -> exact float64 values."""
    b = np.asarray(bits, dtype=np.uint16)
    if dtype == F16:
        return b.view(np.float16).astype(np.float64)
    if dtype == BF16:
        return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    raise ValueError("unknown dtype")


def unpack_int4(qweight) -> np.ndarray:
    """Packed words [N][K/8] -> codes q[N][K] (int64, 0..15).

    Layout: word j of row n holds q[n][8j+i] in bits 4i..4i+3.
    """
    w = np.asarray(qweight, dtype=np.uint32)
    n, kw = w.shape
    q = np.empty((n, kw, 8), dtype=np.int64)
    for i in range(8):
        q[:, :, i] = (w >> np.uint32(4 * i)) & np.uint32(0xF)
    return q.reshape(n, kw * 8)


def unpack_int3(qweight) -> np.ndarray:
    """3-bit codes: packed words [N][3K/32] -> codes q[N][K] (int64, 0..7).

    The paper's 3-bit backbone (Appendix D.1, D.3) does not fix a storage
    layout; this one keeps two-bit fields of neighbouring codes in the two
    16-bit halves of a word. Codes c_t = q[n][32j + t], t = 0..31, of block j
    of row n sit in words 3j, 3j+1, 3j+2 of the row:
      word 3j    bits 2i, 2i+1       : low two bits of c_{2i}       (i = 0..7)
                 bits 16+2i, 17+2i   : low two bits of c_{2i+1}
      word 3j+1  the same for c_{16+2i} and c_{17+2i}
      word 3j+2  bit i               : high bit of c_{2i}          (i = 0..15)
                 bit 16+i            : high bit of c_{2i+1}
    """
    w = np.asarray(qweight, dtype=np.uint32)
    n, nw = w.shape
    if nw % 3:
        raise ValueError("3-bit rows hold a multiple of three words")
    blk = w.reshape(n, nw // 3, 3)
    lo0, lo1, hi = blk[:, :, 0], blk[:, :, 1], blk[:, :, 2]
    q = np.zeros((n, nw // 3, 32), dtype=np.int64)
    for i in range(8):
        q[:, :, 2 * i] = (lo0 >> np.uint32(2 * i)) & np.uint32(3)
        q[:, :, 2 * i + 1] = (lo0 >> np.uint32(16 + 2 * i)) & np.uint32(3)
        q[:, :, 16 + 2 * i] = (lo1 >> np.uint32(2 * i)) & np.uint32(3)
        q[:, :, 17 + 2 * i] = (lo1 >> np.uint32(16 + 2 * i)) & np.uint32(3)
    for i in range(16):
        q[:, :, 2 * i] |= (((hi >> np.uint32(i)) & np.uint32(1)) << np.uint32(2)).astype(np.int64)
        q[:, :, 2 * i + 1] |= (((hi >> np.uint32(16 + i)) & np.uint32(1)) << np.uint32(2)).astype(np.int64)
    return q.reshape(n, (nw // 3) * 32)


def unpack_codes(qweight, bits: int = 4) -> np.ndarray:
    """Codes of a packed weight matrix: 4-bit (unpack_int4) or 3-bit (unpack_int3)."""
    if bits in (0, 4):
        return unpack_int4(qweight)
    if bits == 3:
        return unpack_int3(qweight)
    raise ValueError("weights are 4- or 3-bit")


def dequant(qweight, scales_bits, zeros, group_size: int, bits: int = 4) -> np.ndarray:
    """What[n][k] = (q[n][k] - z[n][k // G]) * s[n][k // G], exact in float64.

    (q - z) is an integer of magnitude <= 15 and s an fp16 value, so the
    product has at most 15 significant bits and is exact (sections 2.1, 5.1:
    asymmetric round-to-nearest per channel or per group of 128; with 3-bit
    codes, Appendix D.1 and D.3, |q - z| <= 7).
    """
    q = unpack_codes(qweight, bits)
    n, k = q.shape
    g = k if group_size in (0, k) else group_size
    s = bits_to_f64(scales_bits, F16)
    z = np.asarray(zeros, dtype=np.int64)
    if s.shape != (n, k // g) or z.shape != (n, k // g):
        raise ValueError("scales/zeros must be [N][K/G]")
    grp = np.arange(k) // g
    return (q - z[:, grp]).astype(np.float64) * s[:, grp]


def round_f64_to_bits(v, dtype: int) -> np.ndarray:
    """Round float64 values to fp16 or bf16, nearest-even, and return bits.

    fp16: numpy's float64 -> float16 cast, which rounds to nearest even.
    bf16: the value is first made float32 (callers pass values exact in
    float32, e.g. dequantised weights), then the low 16 bits of the float32
    pattern are rounded off to nearest even: add 0x7FFF plus the lowest kept
    bit, then truncate. NaN is not expected here.
    """
    v = np.asarray(v, dtype=np.float64)
    if dtype == F16:
        return v.astype(np.float16).view(np.uint16)
    if dtype == BF16:
        f32 = v.astype(np.float32)
        if not np.array_equal(f32.astype(np.float64), v):
            raise ValueError("bf16 rounding here expects float32-exact inputs")
        u = f32.view(np.uint32).astype(np.uint64)
        lsb = (u >> np.uint64(16)) & np.uint64(1)
        r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
        return r.astype(np.uint16)
    raise ValueError("unknown dtype")


def dequant_bits(qweight, scales_bits, zeros, group_size: int, dtype: int,
                 bits: int = 4) -> np.ndarray:
    """The bit-exact dequantisation contract: What rounded once (nearest even)
    to the activation dtype, as uint16 bit patterns [N][K]."""
    return round_f64_to_bits(dequant(qweight, scales_bits, zeros, group_size, bits), dtype)


# ---------------------------------------------------------------------------
# The layer (Eq. 3)
# ---------------------------------------------------------------------------

def sigmoid(t) -> np.ndarray:
    """Numerically stable logistic function in float64."""
    t = np.asarray(t, dtype=np.float64)
    out = np.empty_like(t)
    pos = t >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-t[pos]))
    e = np.exp(t[~pos])
    out[~pos] = e / (1.0 + e)
    return out


def w4_linear(x, W_hat) -> np.ndarray:
    """Y_base = X . W_hat^T  ([M][K] x [N][K] -> [M][N])."""
    return np.asarray(x, np.float64) @ np.asarray(W_hat, np.float64).T


def ec_down(x, A) -> np.ndarray:
    """Rank-r coordinates u = X . A^T ([M][r])."""
    return np.asarray(x, np.float64) @ np.asarray(A, np.float64).T


def gate_sigmoid_linear(x, w_g, b_g: float) -> np.ndarray:
    """Scalar gate per token: g_m = sigma(w_g . x_m + b_g), shape [M]."""
    return sigmoid(np.asarray(x, np.float64) @ np.asarray(w_g, np.float64) + float(b_g))


def gate_tanh_mlp(u, W1, b1, W2, b2) -> np.ndarray:
    """The paper's rank-space gate (Eq. 3): gamma = 1 + tanh(W2 ReLU(W1 u + b1) + b2).

    u [M][r], W1 [h][r], b1 [h], W2 [r][h], b2 [r] -> gamma [M][r] in (0, 2).
    """
    u = np.asarray(u, np.float64)
    hid = np.maximum(u @ np.asarray(W1, np.float64).T + np.asarray(b1, np.float64), 0.0)
    return 1.0 + np.tanh(hid @ np.asarray(W2, np.float64).T + np.asarray(b2, np.float64))


def ec_gate(x, u, gate_kind: int, w_g=None, b_g: float = 0.0,
            W1=None, b1=None, W2=None, b2=None) -> np.ndarray:
    """Gate broadcast to [M][r] for the chosen gate kind."""
    m, r = u.shape
    if gate_kind == GATE_ONE:
        return np.ones((m, r))
    if gate_kind == GATE_SIGMOID_LINEAR:
        return np.repeat(gate_sigmoid_linear(x, w_g, b_g)[:, None], r, axis=1)
    if gate_kind == GATE_TANH_MLP:
        return gate_tanh_mlp(u, W1, b1, W2, b2)
    raise ValueError("unknown gate kind")


def w4ec_linear_f64(x, W_hat, A, B, alpha: float, gate_kind: int, w_g=None,
                    b_g: float = 0.0, W1=None, b1=None, W2=None, b2=None) -> np.ndarray:
    """Eq. 3 on float64 operands: Y = X W_hat^T + alpha * (gate (.) (X A^T)) B^T."""
    y = w4_linear(x, W_hat)
    r = 0 if A is None else np.asarray(A).shape[0]
    if r == 0:
        return y
    u = ec_down(x, A)
    gam = ec_gate(x, u, gate_kind, w_g, b_g, W1, b1, W2, b2)
    v = float(alpha) * gam * u
    return y + v @ np.asarray(B, np.float64).T


def dequant_int8(q, scale) -> np.ndarray:
    """INT8 per-channel symmetric factor (the deployed EC format of section 5.1
    and Appendix B.2: INT8 A and B, one scale per output channel): row c of
    the factor is scale[c] * q[c], evaluated exactly in float64."""
    return np.asarray(scale, np.float64)[:, None] * np.asarray(q, np.float64)


def ec_factors(layer, rows=None):
    """(A, B) of a stored layer as float64: the INT8 codes times their
    per-channel scales when the layer carries them (layer.ab_int8), else the
    activation-dtype bit patterns decoded exactly. `rows` selects rows of B."""
    if getattr(layer, "ab_int8", False):
        A = dequant_int8(layer.A_q, layer.a_scale)
        Bq, bs = layer.B_q, layer.b_scale
        if rows is not None:
            Bq, bs = Bq[rows], bs[rows]
        return A, dequant_int8(Bq, bs)
    dt = layer.act_dtype
    B = layer.B if rows is None else layer.B[rows]
    return bits_to_f64(layer.A, dt), bits_to_f64(B, dt)


def weight_bits(layer) -> int:
    """Code width of a stored layer's weights (4 unless it says 3)."""
    return int(getattr(layer, "weight_bits", 4) or 4)


def w4ec_linear(layer) -> np.ndarray:
    """Eq. 3 on a stored layer (any object with the generator's fields):
    decodes every stored tensor exactly, then evaluates in float64."""
    dt = layer.act_dtype
    W_hat = dequant(layer.qweight, layer.scales, layer.zeros, layer.group_size, weight_bits(layer))
    x = bits_to_f64(layer.x, dt)
    if layer.rank == 0:
        return w4_linear(x, W_hat)
    A, B = ec_factors(layer)
    return w4ec_linear_f64(
        x, W_hat, A, B, layer.alpha,
        layer.gate_kind, w_g=bits_to_f64(layer.w_g, dt), b_g=layer.b_g,
        W1=bits_to_f64(layer.W1, dt), b1=bits_to_f64(layer.b1, dt),
        W2=bits_to_f64(layer.W2, dt), b2=bits_to_f64(layer.b2, dt))


def post_ec_tail(y, residual, norm_w, eps: float):
    """The post-EC tail (section 4.2: residual addition and the next layer's
    RMSNorm after the compensated product), in float64:
        h = y + residual
        y_norm[m][n] = h[m][n] * norm_w[n] / sqrt(mean_n h[m][n]^2 + eps)
    Returns (h, y_norm); residual None adds nothing."""
    h = np.asarray(y, np.float64)
    if residual is not None:
        h = h + np.asarray(residual, np.float64)
    ms = np.mean(h * h, axis=1, keepdims=True)
    return h, h / np.sqrt(ms + float(eps)) * np.asarray(norm_w, np.float64)[None, :]


def w4_linear_layer(layer) -> np.ndarray:
    """The plain 4-bit product X . W_hat^T of a stored layer (EC ignored)."""
    W_hat = dequant(layer.qweight, layer.scales, layer.zeros, layer.group_size, weight_bits(layer))
    return w4_linear(bits_to_f64(layer.x, layer.act_dtype), W_hat)


def w4ec_linear_rows(layer, rows) -> np.ndarray:
    """Eq. 3 for a subset of output columns n in `rows` only (all tokens):
    used to check sampled outputs of full-size layers one by one."""
    rows = np.asarray(rows)
    dt = layer.act_dtype
    W_hat = dequant(layer.qweight[rows], layer.scales[rows], layer.zeros[rows],
                    layer.group_size, weight_bits(layer))
    x = bits_to_f64(layer.x, dt)
    if layer.rank == 0:
        return w4_linear(x, W_hat)
    A, B = ec_factors(layer, rows)
    return w4ec_linear_f64(
        x, W_hat, A, B,
        layer.alpha, layer.gate_kind, w_g=bits_to_f64(layer.w_g, dt), b_g=layer.b_g,
        W1=bits_to_f64(layer.W1, dt), b1=bits_to_f64(layer.b1, dt),
        W2=bits_to_f64(layer.W2, dt), b2=bits_to_f64(layer.b2, dt))


def tolerance_check(y, y_ref, rel_frob: float = 5e-3, max_rel: float = 1e-2):
    """The parity bar: relative Frobenius error <= rel_frob and
    max |y - y_ref| <= max_rel * max |y_ref|. Returns (ok, relF, maxabs, bound)."""
    y = np.asarray(y, np.float64)
    y_ref = np.asarray(y_ref, np.float64)
    diff = y - y_ref
    den = np.linalg.norm(y_ref)
    relf = float(np.linalg.norm(diff) / den) if den > 0 else float(np.linalg.norm(diff))
    mx = float(np.abs(diff).max(initial=0.0))
    bound = max_rel * float(np.abs(y_ref).max(initial=0.0))
    ok = (relf <= rel_frob) and (mx <= bound if bound > 0 else mx == 0.0)
    return ok, relf, mx, bound
