"""Seeded synthetic inputs for the W4+EC linear layer.

This module produces the stored tensors that the layer consumes: packed 4-bit
weight codes with their scales and zero points, activations, the EC factors
A and B, and the gate parameters. It is shared by the tests, the benchmark and
the CPU oracle's callers, and it holds none of the layer's own arithmetic: no
dequantisation, no contraction, no EC projection and no gate. What it does
compute is the offline side that precedes the layer:

* round-to-nearest (RTN) asymmetric 4-bit (or 3-bit) quantisation of a float weight
  matrix, per output channel or per group of input channels (the plain
  linear quantiser the paper compensates: the quantised model of section 2.1,
  evaluated per channel and per group of 128 in section 5.1), and
* packing of the 4-bit codes, eight to a 32-bit word, in the layout the C ABI
  documents: word j of row n holds code q[n][8j+i] in bits 4i..4i+3; and of
  3-bit codes, 32 to three words (pack_int3).

Floating-point values are returned as numpy arrays of IEEE bit patterns
(uint16) in the activation dtype, so that both the GPU path and the oracle see
exactly the same stored numbers. Conversion to bfloat16 uses torch's CPU cast
(round to nearest even).

Distribution readings (the workload configurations give N(0, s) without
saying whether s is a variance): the second argument is the standard
deviation.
"""
from __future__ import annotations

import dataclasses
import numpy as np
import torch

F16 = 0
BF16 = 1

GATE_ONE = 0
GATE_SIGMOID_LINEAR = 1
GATE_TANH_MLP = 2

_DTYPES = {F16: torch.float16, BF16: torch.bfloat16}


def to_bits(a: np.ndarray, dtype: int) -> np.ndarray:
    """Round a float array to fp16/bf16 (nearest even) and return uint16 bits."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(_DTYPES[dtype]).view(torch.int16).numpy().view(np.uint16).copy()


def from_bits(bits: np.ndarray, dtype: int) -> np.ndarray:
    """uint16 bit patterns of fp16/bf16 values -> float32 array (exact)."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(_DTYPES[dtype]).to(torch.float32).numpy()


def pack_int4(q: np.ndarray) -> np.ndarray:
    """Pack codes q[N][K] (values 0..15, K % 8 == 0) into uint32 words [N][K/8].

    Word j of row n holds q[n][8j+i] in bits 4i..4i+3 (lowest nibble first).
    """
    q = np.asarray(q)
    n, k = q.shape
    if k % 8:
        raise ValueError("K must be a multiple of 8 to pack 4-bit codes")
    if q.size and (q.min() < 0 or q.max() > 15):
        raise ValueError("codes must lie in 0..15")
    q8 = q.astype(np.uint8, copy=False)
    # byte j of a row holds codes 2j (low nibble) and 2j+1 (high nibble); four
    # consecutive bytes read as a little-endian uint32 give the word layout
    b = np.ascontiguousarray(q8[:, 0::2] | (q8[:, 1::2] << np.uint8(4)))
    return b.view("<u4").astype(np.uint32, copy=False).reshape(n, k // 8)


def pack_int3(q: np.ndarray) -> np.ndarray:
    """Pack 3-bit codes q[N][K] (values 0..7, K % 32 == 0) into uint32 words
    [N][3K/32]: codes c_t = q[n][32j + t] of block j go to words 3j, 3j+1,
    3j+2 of row n. Word 3j holds the low two bits of c_{2i} in bits 2i..2i+1
    and of c_{2i+1} in bits 16+2i..17+2i (i = 0..7); word 3j+1 the same for
    c_{16+2i}, c_{17+2i}; word 3j+2 holds the high bit of c_{2i} in bit i and
    of c_{2i+1} in bit 16+i (i = 0..15)."""
    q = np.asarray(q)
    n, k = q.shape
    if k % 32:
        raise ValueError("K must be a multiple of 32 to pack 3-bit codes")
    if q.size and (q.min() < 0 or q.max() > 7):
        raise ValueError("codes must lie in 0..7")
    c = q.astype(np.uint32).reshape(n, k // 32, 32)
    even, odd = c[:, :, 0::2], c[:, :, 1::2]  # c_{2i}, c_{2i+1}, i = 0..15
    words = np.zeros((n, k // 32, 3), dtype=np.uint32)
    for i in range(16):
        wi, sh = (0, 2 * i) if i < 8 else (1, 2 * (i - 8))
        words[:, :, wi] |= (even[:, :, i] & 3) << np.uint32(sh)
        words[:, :, wi] |= (odd[:, :, i] & 3) << np.uint32(16 + sh)
        words[:, :, 2] |= (even[:, :, i] >> 2) << np.uint32(i)
        words[:, :, 2] |= (odd[:, :, i] >> 2) << np.uint32(16 + i)
    return words.reshape(n, 3 * k // 32)


def pack_codes(q: np.ndarray, bits: int = 4) -> np.ndarray:
    """pack_int4 or pack_int3 by code width."""
    return pack_int3(q) if bits == 3 else pack_int4(q)


def rtn_quantize(w: np.ndarray, group_size: int, bits: int = 4):
    """Asymmetric min-max round-to-nearest quantisation of w[N][K] to b-bit
    codes (b = 4, or 3 for the paper's 3-bit backbone), L = 2^b - 1.

    For each output row n and each group of `group_size` consecutive input
    columns (group_size == K means one group per row, "per channel"):
      lo, hi = min, max of the group
      s = fp16((hi - lo) / L)             (the stored scale)
      z = clip(rne(-lo / s), 0, L)        (the stored zero point)
      q = clip(rne(w / s) + z, 0, L)      (codes, chosen against the fp16 s)
    A constant group (hi == lo) or a scale that rounds to zero uses s = 1 and
    z = clip(rne(-lo), 0, L).
    Returns (codes uint8 [N][K], scales fp16 bits [N][K/G], zeros uint8 [N][K/G]).
    """
    if bits not in (3, 4):
        raise ValueError("3- or 4-bit codes")
    top = float((1 << bits) - 1)
    w = np.asarray(w, dtype=np.float32)
    n, k = w.shape
    g = k if group_size in (0, k) else group_size
    if k % g:
        raise ValueError("K must be a multiple of the group size")
    q_out = np.empty((n, k), dtype=np.uint8)
    s_out = np.empty((n, k // g), dtype=np.uint16)
    z_out = np.empty((n, k // g), dtype=np.uint8)
    step = max(1, (1 << 23) // k)  # rows per chunk, bounds the temporaries
    for r0 in range(0, n, step):
        r1 = min(n, r0 + step)
        wg = w[r0:r1].reshape(r1 - r0, k // g, g)
        lo = wg.min(axis=2).astype(np.float64)
        hi = wg.max(axis=2).astype(np.float64)
        s = ((hi - lo) / top).astype(np.float16).astype(np.float64)
        degenerate = (hi == lo) | (s == 0)
        s = np.where(degenerate, 1.0, s)
        z = np.clip(np.rint(-lo / s), 0, top)
        # w / s in float32: s is an fp16 value (exact in float32); the quotient's
        # rounding can only matter within 2^-24 of a rounding tie
        qf = np.rint(wg / s.astype(np.float32)[:, :, None])
        qf += z.astype(np.float32)[:, :, None]
        np.clip(qf, 0, top, out=qf)
        q_out[r0:r1] = qf.reshape(r1 - r0, k).astype(np.uint8)
        s_out[r0:r1] = s.astype(np.float16).view(np.uint16)
        z_out[r0:r1] = z.astype(np.uint8)
    return q_out, s_out, z_out


@dataclasses.dataclass
class Layer:
    """Stored tensors of one W4+EC linear layer plus its activations.

    Bit-pattern arrays are uint16 in the activation dtype unless noted.
    """
    M: int
    N: int
    K: int
    group_size: int          # G (== K for per-channel)
    act_dtype: int           # F16 or BF16
    rank: int
    gate_kind: int
    qweight: np.ndarray      # uint32 [N][K/8] (4-bit) or [N][3K/32] (3-bit)
    scales: np.ndarray       # fp16 bits [N][K/G]
    zeros: np.ndarray        # uint8 [N][K/G]
    x: np.ndarray            # [M][K]
    A: np.ndarray            # [r][K]
    B: np.ndarray            # [N][r]
    w_g: np.ndarray          # [K]
    b_g: float
    alpha: float
    W1: np.ndarray           # [h][r]
    b1: np.ndarray           # [h]
    W2: np.ndarray           # [r][h]
    b2: np.ndarray           # [r]
    # INT8 per-channel symmetric copies of A and B (make_layer(ab_int8=True))
    ab_int8: bool = False
    A_q: np.ndarray = None   # int8 [r][K]
    a_scale: np.ndarray = None  # fp32 [r]
    B_q: np.ndarray = None   # int8 [N][r]
    b_scale: np.ndarray = None  # fp32 [N]
    weight_bits: int = 4     # code width of qweight: 4, or 3 (zeros then 0..7)

    @property
    def gate_hidden(self) -> int:
        return int(self.W1.shape[0])


def quantize_int8_rows(w: np.ndarray):
    """Symmetric per-row INT8 quantisation of w[R][C] (the stand-in for the
    post-calibration step that stores the EC factors in INT8):
      s = fp32(max |row| / 127)   (1 for an all-zero row)
      q = clip(rne(row / s), -127, 127)
    Returns (q int8 [R][C], s fp32 [R])."""
    w = np.asarray(w, dtype=np.float32)
    amax = np.abs(w).max(axis=1) if w.shape[1] else np.zeros(w.shape[0], np.float32)
    s = np.where(amax > 0, amax / np.float32(127.0), np.float32(1.0)).astype(np.float32)
    q = np.clip(np.rint(w / s[:, None]), -127, 127).astype(np.int8)
    return q, s


def make_layer(*, M: int, N: int, K: int, group_size: int, rank: int,
               act_dtype: int = F16, gate_kind: int = GATE_SIGMOID_LINEAR,
               seed: int = 0, config_id: int = 0, module_id: int = 0,
               w_std: float = 0.02, x_std: float = 1.0, ec_std: float = 0.01,
               wg_std: float = 0.05, b_g: float = 0.0, alpha: float = 1.0,
               outlier_frac: float = 0.0, outlier_scale: float = 20.0,
               gate_hidden: int = 0, ab_int8: bool = False, weight_bits: int = 4) -> Layer:
    """Draw one layer from the seed tree SeedSequence([seed, config_id, module_id]).

    Draw order: W (fp32) -> RTN -> X (with outlier channels) -> A, B -> w_g ->
    gate-MLP parameters. The gate-MLP weights are drawn N(0, 1/sqrt(r)) for W1
    and N(0, 1/sqrt(h)) for W2 with zero biases, so that the gate differs from
    one across tokens.
    """
    g = K if group_size in (0, K) else group_size
    rng = np.random.default_rng(np.random.SeedSequence([seed, config_id, module_id]))
    w = rng.standard_normal((N, K), dtype=np.float32)
    w *= np.float32(w_std)
    q, s, z = rtn_quantize(w, g, weight_bits)
    del w
    x = rng.standard_normal((M, K), dtype=np.float32)
    x *= np.float32(x_std)
    if outlier_frac > 0.0 and M > 0:
        n_out = int(round(outlier_frac * K))
        idx = rng.choice(K, size=n_out, replace=False)
        x[:, idx] *= outlier_scale
    A = rng.normal(0.0, ec_std, size=(rank, K)).astype(np.float32)
    B = rng.normal(0.0, ec_std, size=(N, rank)).astype(np.float32)
    w_g = rng.normal(0.0, wg_std, size=(K,)).astype(np.float32)
    h = gate_hidden if gate_hidden > 0 else 4 * rank
    W1 = rng.normal(0.0, 1.0 / np.sqrt(max(rank, 1)), size=(h, rank)).astype(np.float32)
    W2 = rng.normal(0.0, 1.0 / np.sqrt(max(h, 1)), size=(rank, h)).astype(np.float32)
    b1 = np.zeros((h,), np.float32)
    b2 = np.zeros((rank,), np.float32)
    i8 = {}
    if ab_int8:
        A_q, a_scale = quantize_int8_rows(A)
        B_q, b_scale = quantize_int8_rows(B)
        i8 = dict(ab_int8=True, A_q=A_q, a_scale=a_scale, B_q=B_q, b_scale=b_scale)
    return Layer(M=M, N=N, K=K, group_size=g, act_dtype=act_dtype, rank=rank,
                 gate_kind=gate_kind, qweight=pack_codes(q, weight_bits), scales=s, zeros=z,
                 x=to_bits(x, act_dtype), A=to_bits(A, act_dtype),
                 B=to_bits(B, act_dtype), w_g=to_bits(w_g, act_dtype),
                 b_g=float(b_g), alpha=float(alpha),
                 W1=to_bits(W1, act_dtype), b1=to_bits(b1, act_dtype),
                 W2=to_bits(W2, act_dtype), b2=to_bits(b2, act_dtype),
                 weight_bits=weight_bits, **i8)


def make_tail(layer: Layer, seed: int = 0, eps: float = 1e-5):
    """Inputs of the post-EC tail for a layer, from a seed stream of their
    own (the layer's draws are unchanged): a residual ~ N(0, 1) [M][N] and
    an RMSNorm weight ~ N(1, 0.1) [N], both as activation-dtype bits."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 77, layer.M, layer.N]))
    res = rng.standard_normal((layer.M, layer.N), dtype=np.float32)
    w = (1.0 + 0.1 * rng.standard_normal(layer.N)).astype(np.float32)
    return dict(residual=to_bits(res, layer.act_dtype), norm_w=to_bits(w, layer.act_dtype),
                eps=float(eps))


# ---------------------------------------------------------------------------
# Workload configurations (synthetic stand-ins for the paper's Llama layers;
# no trained weights are used).
# ---------------------------------------------------------------------------

LLAMA_1B = {  # hidden 2048, 32 q / 8 kv heads x 64, MLP 8192
    "q": (2048, 2048), "k": (2048, 512), "v": (2048, 512), "o": (2048, 2048),
    "gate": (2048, 8192), "up": (2048, 8192), "down": (8192, 2048),
}
LLAMA_8B = {  # hidden 4096, 32 q / 8 kv heads x 128, MLP 14336
    "q": (4096, 4096), "k": (4096, 1024), "v": (4096, 1024), "o": (4096, 4096),
    "gate": (4096, 14336), "up": (4096, 14336), "down": (14336, 4096),
}
LLAMA_70B = {  # hidden 8192, 64 q / 8 kv heads x 128, MLP 28672
    "q": (8192, 8192), "k": (8192, 1024), "v": (8192, 1024), "o": (8192, 8192),
    "gate": (8192, 28672), "up": (8192, 28672), "down": (28672, 8192),
}
MODULES = ("q", "k", "v", "o", "gate", "up", "down")

CONFIGS = {
    # config id: description and per-module (K, N) shapes, token counts, quant.
    0: dict(name="tiny", shapes={"tiny": (256, 256)}, Ms=(4,), group_size=0,
            rank=8, act_dtype=F16, outlier_frac=0.0, layers=1),
    1: dict(name="llama1b-decode", shapes=LLAMA_1B, Ms=(1, 4, 16), group_size=128,
            rank=16, act_dtype=F16, outlier_frac=0.0, layers=16),
    2: dict(name="llama1b-prefill", shapes=LLAMA_1B, Ms=(512, 2048, 4096),
            group_size=128, rank=16, act_dtype=F16, outlier_frac=0.01, layers=16),
    3: dict(name="llama8b", shapes=LLAMA_8B, Ms=(1, 8, 32, 128, 512, 4096),
            group_size=0, rank=32, act_dtype=BF16, outlier_frac=0.0, layers=32),
    4: dict(name="llama70b", shapes=LLAMA_70B,
            Ms=(1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 2048, 4096, 8192),
            group_size=128, rank=64, act_dtype=F16, outlier_frac=0.0, layers=80,
            ec_fraction=0.25),
}


def config_layer(config_id: int, module: str, M: int, seed: int = 0,
                 gate_kind: int = GATE_SIGMOID_LINEAR, rank: int | None = None,
                 ab_int8: bool = False, weight_bits: int = 4) -> Layer:
    """One module of a workload configuration at token count M (ab_int8:
    with INT8 per-channel copies of the EC factors; weight_bits 3: the same
    draws quantised to 3-bit codes)."""
    c = CONFIGS[config_id]
    K, N = c["shapes"][module]
    mod_id = list(c["shapes"]).index(module)
    return make_layer(M=M, N=N, K=K, group_size=c["group_size"],
                      rank=c["rank"] if rank is None else rank,
                      act_dtype=c["act_dtype"], gate_kind=gate_kind, seed=seed,
                      config_id=config_id, module_id=mod_id,
                      outlier_frac=c["outlier_frac"], ab_int8=ab_int8,
                      weight_bits=weight_bits)


def ec_selection_70b(seed: int = 0, layers: int = 80, fraction: float = 0.25) -> np.ndarray:
    """Seeded choice of the (layer, module) pairs of the 70B-shaped model that
    carry an EC: `fraction` of the layers x 7 modules, without replacement.
    Returns a bool array [layers][7]."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 4, 999]))
    total = layers * len(MODULES)
    pick = rng.choice(total, size=int(round(fraction * total)), replace=False)
    sel = np.zeros(total, dtype=bool)
    sel[pick] = True
    return sel.reshape(layers, len(MODULES))
