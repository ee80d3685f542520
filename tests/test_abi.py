"""Host-side tests of the C ABI: the library loads, exports every symbol the
header declares, validates arguments before any launch, and plans paths.
No call here reaches a kernel (every call is rejected on the host or is the
pure planning function), so these run without a GPU."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

from paper_2606_11244_amd import spear as sp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_symbols():
    text = "".join(open(os.path.join(ROOT, "include", h)).read()
                   for h in sorted(os.listdir(os.path.join(ROOT, "include"))) if h.endswith(".h"))
    return sorted(set(re.findall(r"^\S.*?\b(spear_[a-z0-9_]+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported():
    names = _declared_symbols()
    assert set(names) == set(sp.EXPORTED), names
    for n in names:
        assert hasattr(sp.LIB, n), n


def test_version_and_status_strings():
    assert sp.version() == "0.2.0"
    for code in sp.STATUS:
        assert sp.LIB.spear_status_string(code)
    assert sp.LIB.spear_status_string(12345) == b"unknown status"


def _plan(**kw):
    args = dict(M=1, N=2048, K=2048, group_size=128, act_dtype=sp.F16, rank=16,
                gate_kind=sp.GATE_SIGMOID_LINEAR)
    args.update(kw)
    with_ec = args.pop("with_ec", True)
    return sp.dispatch_plan(sp.problem(**args), with_ec)


@pytest.mark.parametrize("kw,code", [
    (dict(K=100), -2), (dict(K=0), -2), (dict(K=192), -2), (dict(M=-1), -2), (dict(N=-3), -2),
    (dict(group_size=64), -2), (dict(group_size=384), -2), (dict(group_size=96), -2),
    (dict(act_dtype=2), -3), (dict(rank=257), -2), (dict(rank=-1), -2),
    (dict(gate_kind=3), -6), (dict(gate_hidden=-1), -2), (dict(gate_hidden=2048), -2),
    (dict(force_path=7), -6),
    (dict(force_path=sp.PATH_FUSED_MFMA, rank=17), -6),
    (dict(force_path=sp.PATH_FUSED_GEMV, M=65), -6),
    (dict(force_path=sp.PATH_FUSED_LOCAL, M=33), -6),
    (dict(force_path=sp.PATH_FUSED_LOCAL, rank=17), -6),
    (dict(M=1 << 20, K=1 << 12), -2),
])
def test_plan_validation(kw, code):
    with pytest.raises(sp.SpearError) as e:
        _plan(**kw)
    assert e.value.status == code


def test_plan_rejects_null():
    out = sp.Plan()
    assert sp.LIB.spear_dispatch_plan(None, 1, ctypes.byref(out)) == -1
    assert sp.LIB.spear_dispatch_plan(ctypes.byref(sp.problem(1, 1, 128)), 1, None) == -1


def test_plan_phase_aware_dispatch():
    """Decode token counts get the single fused kernel, prefill the semi-fused
    pre-kernel + GEMM (section 4.1)."""
    for M in (1, 4, 16, 17, 32):
        # rank 16 + the gate row fit two 16-row tiles: the local fused variant
        p = _plan(M=M)
        assert p.path == sp.PATH_FUSED_LOCAL and p.num_launches == 1, M
        # beyond the local variant: the producer-fused GEMV for one token, the
        # two-kernel path for more on shallow layers (K <= 4096), the fused
        # GEMV again on deeper ones, and the two-kernel path for one token
        # on very deep layers (K >= 16384)
        want = sp.PATH_FUSED_GEMV if M == 1 else sp.PATH_UNFUSED_2K
        p = _plan(M=M, rank=32)
        assert p.path == want and p.num_launches == (1 if M == 1 else 2), M
        # the paper's tanh-MLP gate takes the local variant too (rank 16)
        p = _plan(M=M, gate_kind=sp.GATE_TANH_MLP)
        assert p.path == sp.PATH_FUSED_LOCAL and p.num_launches == 1, M
        p = _plan(M=M, rank=32, K=8192)
        assert p.path == sp.PATH_FUSED_GEMV and p.num_launches == 1, M
        p = _plan(M=M, rank=64, N=8192, K=28672)
        assert p.path == (sp.PATH_UNFUSED_2K if M == 1 else sp.PATH_FUSED_GEMV), M
    # above 32 tokens the GEMM kernels: the fully fused one where it applies,
    # the two-kernel path on the GEMM otherwise
    for M in (33, 64):
        p = _plan(M=M)
        assert p.path == sp.PATH_FUSED_MFMA and p.num_launches == 1, M
        p = _plan(M=M, rank=32)
        assert p.path == sp.PATH_UNFUSED_2K and p.tile_n == 128, M
    # the 4-bit product alone: GEMV up to 32 tokens, GEMM above; force_path
    # picks either kernel
    assert _plan(M=32, with_ec=False).path == sp.PATH_FUSED_GEMV
    assert _plan(M=33, with_ec=False).path == sp.PATH_UNFUSED_2K
    assert _plan(M=4, with_ec=False, force_path=sp.PATH_UNFUSED_2K).tile_n == 128
    assert _plan(M=64, with_ec=False, force_path=sp.PATH_FUSED_GEMV).path == sp.PATH_FUSED_GEMV
    with pytest.raises(sp.SpearError):
        _plan(M=65, with_ec=False, force_path=sp.PATH_FUSED_GEMV)
    assert _plan(M=4, force_path=sp.PATH_FUSED_GEMV).path == sp.PATH_FUSED_GEMV
    for M in (1, 64, 4096):
        p = _plan(M=M, force_path=sp.PATH_FUSED_MFMA)
        assert p.path == sp.PATH_FUSED_MFMA and p.num_launches == 1, M
        assert p.grid == -(-M // 128) * (2048 // 128) * p.split_k, M
        assert p.split_k == (1 if M == 4096 else 8), M
    assert _plan(M=4, force_path=sp.PATH_FUSED_LOCAL).grid == _plan(M=4, with_ec=False).grid
    # prefill: the fully fused GEMM while the grid has at most 256 128 x 128
    # tiles (N = 2048: up to M = 2048), the semi-fused pair above that and
    # for ranks or gates the fused GEMM does not take
    for M in (65, 512, 2048):
        p = _plan(M=M)
        assert p.path == sp.PATH_FUSED_MFMA and p.num_launches == 1, M
    for M in (2049, 4096):
        p = _plan(M=M)
        assert p.path == sp.PATH_UNFUSED_2K and p.num_launches == 2, M
    p = _plan(M=512, rank=32)
    assert p.path == sp.PATH_UNFUSED_2K and p.num_launches == 2
    p = _plan(M=512, gate_kind=sp.GATE_TANH_MLP)
    assert p.path == sp.PATH_FUSED_MFMA and p.num_launches == 1
    assert _plan(M=4, force_path=sp.PATH_UNFUSED_CHAIN).num_launches == 4
    assert _plan(M=4096, force_path=sp.PATH_UNFUSED_CHAIN).num_launches == 4
    assert _plan(M=4, force_path=sp.PATH_UNFUSED_2K).num_launches == 2


def test_gemm_split_k_plan_and_workspace():
    """Small tile grids split K; the workspace holds every slice's fp32 tile
    (the 4-bit-only call included), and a missing workspace is rejected on
    the host."""
    for ec in (True, False):
        p = _plan(M=512, N=1024, K=8192, rank=16, with_ec=ec)
        tiles = 4 * 8
        assert p.split_k == 8 and p.grid == tiles * 8
        assert p.workspace_bytes >= 8 * tiles * 128 * 128 * 4
    assert _plan(M=4096, N=2048, K=2048).split_k == 1   # 256 tiles of 256 tokens: no split
    # 256-token tiles while they alone fill the CUs, else 128
    assert _plan(M=4096, N=2048, K=2048).tile_m == 256
    assert _plan(M=2048, N=2048, K=2048).tile_m == 128
    # deep K counts: 128 tiles of 256 tokens at K = 8192 take the big tile
    assert _plan(M=2048, N=2048, K=8192, with_ec=False).tile_m == 256
    # ... and the EC call then takes the semi-fused pair on that tile
    p = _plan(M=2048, N=2048, K=8192)
    assert p.path == sp.PATH_UNFUSED_2K and p.tile_m == 256
    sp.set_gemm_tile(256)
    try:
        for kw in (dict(with_ec=False), dict(force_path=4)):
            p = _plan(M=512, N=1024, K=8192, rank=16, **kw)
            assert p.tile_m == 256 and p.grid == 2 * 8 * p.split_k, kw
        with pytest.raises(sp.SpearError):
            _plan(M=512, N=1024, K=8192, rank=16, force_path=2)  # fused: 128 only
    finally:
        sp.set_gemm_tile(0)
    # the fully fused GEMM splits alike and adds the slices' EC accumulators
    f = _plan(M=512, N=1024, K=8192, rank=16, force_path=2)
    assert f.path == 2 and f.split_k == 8
    assert f.workspace_bytes >= 8 * tiles * (128 * 128 + 4096) * 4
    prob = sp.problem(512, 1024, 8192, 128, sp.F16, 0)
    w = sp.W4(ADDR["q"], ADDR["s"], ADDR["z"])
    assert sp.LIB.spear_w4_linear(ctypes.byref(prob), ADDR["x"], ctypes.byref(w), ADDR["y"],
                                  None, 0, None) == -5


def test_plan_is_deterministic_and_sized():
    a, b = _plan(M=16).as_dict(), _plan(M=16).as_dict()
    assert a == b
    # rank 0 or no EC -> no EC launches; the 4-bit plan matches
    assert _plan(M=1, rank=0).num_launches == 1
    assert _plan(M=1, with_ec=False).ec_splits == 0
    # empty problems are legal no-ops
    assert _plan(M=0).num_launches == 0 and _plan(N=0).num_launches == 0
    # workspace grows with the token count at fixed shape
    ws = [_plan(M=M).workspace_bytes for M in (1, 8, 16, 64, 128, 1024, 4096)]
    assert all(w > 0 for w in ws)
    # split-K never exceeds the number of 128-wide K iterations
    for K in (128, 256, 2048, 28672):
        p = _plan(M=1, K=K, N=512)
        assert 1 <= p.split_k <= K // 128
        assert 1 <= p.ec_splits <= K // 128


def _call_ec(prob, x=None, y=None, q=None, s=None, z=None, A=None, B=None, w_g=None, ws=None,
             ws_bytes=0):
    w = sp.W4(q, s, z)
    ec = sp.EC(A, B, 1.0, w_g, 0.0, None, None, None, None)
    return sp.LIB.spear_w4ec_linear(ctypes.byref(prob), x, ctypes.byref(w), ctypes.byref(ec), y,
                                    ws, ws_bytes, None)


# fake but distinct, 16-byte aligned addresses: every call below is rejected on
# the host before anything touches them
BASE = 0x7F0000000000
ADDR = {k: BASE + i * (1 << 32) for i, k in enumerate("xyqszABwW")}


def test_null_pointers_rejected():
    prob = sp.problem(4, 256, 256, 0, sp.F16, 8)
    assert _call_ec(prob) == -1
    full = dict(x=ADDR["x"], y=ADDR["y"], q=ADDR["q"], s=ADDR["s"], z=ADDR["z"], A=ADDR["A"],
                B=ADDR["B"], w_g=ADDR["w"], ws=ADDR["W"], ws_bytes=1 << 30)
    for k in ("x", "y", "q", "s", "z", "A", "B", "w_g"):
        args = dict(full)
        args[k] = None
        assert _call_ec(prob, **args) == -1, k


def test_misaligned_pointers_rejected():
    prob = sp.problem(4, 256, 256, 0, sp.F16, 8)
    full = dict(x=ADDR["x"], y=ADDR["y"], q=ADDR["q"], s=ADDR["s"], z=ADDR["z"], A=ADDR["A"],
                B=ADDR["B"], w_g=ADDR["w"], ws=ADDR["W"], ws_bytes=1 << 30)
    for k in ("x", "y", "q", "s", "z", "A", "B", "w_g", "ws"):
        args = dict(full)
        args[k] = args[k] + 8
        assert _call_ec(prob, **args) == -4, k


def test_alias_rejected():
    prob = sp.problem(4, 256, 256, 0, sp.F16, 8)
    full = dict(x=ADDR["x"], y=ADDR["y"], q=ADDR["q"], s=ADDR["s"], z=ADDR["z"], A=ADDR["A"],
                B=ADDR["B"], w_g=ADDR["w"], ws=ADDR["W"], ws_bytes=1 << 30)
    for k in ("x", "q", "s", "z", "A", "B", "w_g", "ws"):
        args = dict(full)
        args["y"] = args[k] + 16
        assert _call_ec(prob, **args) == -8, k


def test_workspace_checked():
    prob = sp.problem(4, 256, 256, 0, sp.F16, 8)
    need = sp.dispatch_plan(prob, True).workspace_bytes
    assert need > 0
    full = dict(x=ADDR["x"], y=ADDR["y"], q=ADDR["q"], s=ADDR["s"], z=ADDR["z"], A=ADDR["A"],
                B=ADDR["B"], w_g=ADDR["w"])
    assert _call_ec(prob, ws=None, ws_bytes=0, **full) == -5
    assert _call_ec(prob, ws=ADDR["W"], ws_bytes=need - 1, **full) == -5


def test_gate_parameters_required():
    prob = sp.problem(4, 256, 256, 0, sp.F16, 8, sp.GATE_TANH_MLP)
    w = sp.W4(ADDR["q"], ADDR["s"], ADDR["z"])
    ec = sp.EC(ADDR["A"], ADDR["B"], 1.0, None, 0.0, None, None, None, None)
    st = sp.LIB.spear_w4ec_linear(ctypes.byref(prob), ADDR["x"], ctypes.byref(w), ctypes.byref(ec),
                                  ADDR["y"], ADDR["W"], 1 << 30, None)
    assert st == -1


def test_dequant_validation():
    prob = sp.problem(0, 256, 100, 0, sp.F16)
    w = sp.W4(ADDR["q"], ADDR["s"], ADDR["z"])
    assert sp.LIB.spear_w4_dequant(ctypes.byref(prob), ctypes.byref(w), ADDR["y"], None) == -2
    prob = sp.problem(0, 256, 256, 0, sp.F16)
    assert sp.LIB.spear_w4_dequant(ctypes.byref(prob), ctypes.byref(w), None, None) == -1
    assert sp.LIB.spear_w4_dequant(ctypes.byref(prob), ctypes.byref(w), ADDR["y"] + 2, None) == -4
    assert sp.LIB.spear_w4_dequant(ctypes.byref(prob), ctypes.byref(w), ADDR["q"], None) == -8
    # N == 0 is a no-op that succeeds without touching anything
    prob = sp.problem(0, 0, 256, 0, sp.F16)
    assert sp.LIB.spear_w4_dequant(ctypes.byref(prob), ctypes.byref(w), None, None) == 0


def test_empty_problem_is_noop():
    prob = sp.problem(0, 256, 256, 0, sp.F16, 8)
    assert _call_ec(prob) == 0
    prob = sp.problem(4, 0, 256, 0, sp.F16, 8)
    assert _call_ec(prob) == 0


def test_wait_poll_hook_roundtrip():
    old = sp.set_wait_polls(5)
    assert sp.set_wait_polls(old) == 5


def test_decode_launch_shape_rules():
    """The measured launch-shape rules at a single token: the fewest row
    tiles whose grid fits one round of 256 blocks, no second K-slice on the
    70B-shaped 8192-row modules, and the producer-fused variant on one row
    tile for layers of 4096+ rows that fit one round, and on one row tile and
    one K-slice for narrower layers."""
    # 1B q: one row tile (16 rows), one K-slice, 128 blocks
    p = _plan(M=1)
    assert (p.tile_n, p.split_k, p.grid) == (16, 1, 128)
    # 1B gate: one row tile would need 512 blocks, so two
    p = _plan(M=1, N=8192)
    assert (p.tile_n, p.grid) == (32, 256)
    # 70B q, 4-bit only: two row tiles, unsplit
    p = _plan(M=1, N=8192, K=8192, rank=0, with_ec=False)
    assert (p.tile_n, p.split_k, p.grid) == (32, 1, 256)
    # 8B q, rank 32: the fused GEMV on one row tile, unsplit
    p = _plan(M=1, N=4096, K=4096, rank=32)
    assert p.path == sp.PATH_FUSED_GEMV and (p.tile_n, p.split_k) == (16, 1)
    # at 16 tokens the earlier shapes stay (1B down: two row tiles, four slices)
    p = _plan(M=16, N=2048, K=8192, rank=0, with_ec=False)
    assert (p.tile_n, p.split_k) == (32, 4)
    # 70B-shaped layers at 16 and 8 tokens: 2048 waves (no second K-slice on
    # q), gate four row tiles of four-wave blocks, the fused gate four row
    # tiles; at 4 tokens gate keeps two row tiles
    p = _plan(M=16, N=8192, K=8192, rank=0, with_ec=False)
    assert (p.tile_n, p.split_k, p.grid) == (32, 1, 256)
    p = _plan(M=16, N=28672, K=8192, rank=0, with_ec=False)
    assert (p.tile_n, p.split_k, p.grid) == (64, 1, 448)
    p = _plan(M=8, N=28672, K=8192, rank=0, with_ec=False)
    assert (p.tile_n, p.split_k) == (64, 1)
    p = _plan(M=4, N=28672, K=8192, rank=0, with_ec=False)
    assert (p.tile_n, p.split_k) == (32, 1)
    # the fused gate takes four row tiles from four tokens on
    p = _plan(M=4, N=28672, K=8192, rank=64)
    assert p.path == sp.PATH_FUSED_GEMV and (p.tile_n, p.split_k) == (64, 1)
    p = _plan(M=16, N=28672, K=8192, rank=64)
    assert p.path == sp.PATH_FUSED_GEMV and (p.tile_n, p.split_k) == (64, 1)
    p = _plan(M=16, N=8192, K=8192, rank=64)
    assert p.path == sp.PATH_FUSED_GEMV and (p.tile_n, p.split_k) == (32, 1)
    # 1B down (2048 x 8192, rank 16) at one token: the producer-fused GEMV
    # on one row tile over all of K, not the local variant; at two tokens
    # the local variant
    p = _plan(M=1, N=2048, K=8192, rank=16)
    assert p.path == sp.PATH_FUSED_GEMV and (p.tile_n, p.split_k) == (16, 1)
    assert _plan(M=2, N=2048, K=8192, rank=16).path == sp.PATH_FUSED_LOCAL
    # two token tiles (32 tokens) on the 70B-shaped layers: four row tiles
    # (two for the 4-bit product on q), K split in two from K = 16384 on
    p = _plan(M=32, N=8192, K=8192, rank=0, with_ec=False)
    assert (p.tile_n, p.split_k, p.grid) == (32, 1, 256)
    p = _plan(M=32, N=28672, K=8192, rank=0, with_ec=False)
    assert (p.tile_n, p.split_k) == (64, 1)
    p = _plan(M=32, N=8192, K=28672, rank=0, with_ec=False)
    assert (p.tile_n, p.split_k) == (64, 2)
    p = _plan(M=32, N=8192, K=8192, rank=64)
    assert p.path == sp.PATH_FUSED_GEMV and (p.tile_n, p.split_k) == (64, 1)
    p = _plan(M=32, N=8192, K=28672, rank=64)
    assert p.path == sp.PATH_FUSED_GEMV and (p.tile_n, p.split_k) == (64, 2)
    # 70B k, rank 64: the fused GEMV on one row tile over all of K (64
    # iterations, ten per wave), 64 consumer workgroups after the producers
    p = _plan(M=1, N=1024, K=8192, rank=64)
    assert p.path == sp.PATH_FUSED_GEMV and (p.tile_n, p.split_k) == (16, 1)
    # 70B gate, rank 64: wide, so two row tiles as before
    p = _plan(M=1, N=28672, K=8192, rank=64)
    assert p.path == sp.PATH_FUSED_GEMV and (p.tile_n, p.split_k) == (32, 1)


def test_prefill_tile_rule():
    """256-token GEMM tiles only above 128 tokens: when they fill the CUs
    (deep K counting extra rounds), or up to 512 tokens on layers of 32M+
    weights once a quarter of the CUs have one."""
    def tm(M, N, K, rank=64):
        return _plan(M=M, N=N, K=K, rank=rank).tile_m
    assert tm(64, 28672, 8192) == 128 and tm(128, 28672, 8192) == 128
    assert tm(192, 28672, 8192) == 256
    assert tm(256, 8192, 8192) == 256          # 70B q: 64M weights
    assert tm(256, 2048, 8192, rank=16) == 128  # 1B down: 16M weights
    assert tm(4096, 2048, 2048, rank=32) == 256


COUNTERS = 131072            # the counter block every workspace starts with
TAG_END = COUNTERS + (1 << 20)  # the fused path's tagged region ends here


def test_tagged_region_is_written_by_the_fused_path_only():
    """Every plan (every path, dtype, gate, rank, token count the fused GEMV
    takes, with and without the EC) keeps its scratch data past the tagged
    region; only the fused GEMV has a tagged region, at the fixed place right
    after the counter block. So a tagged word a consumer reads was written by
    a fused launch (or is still zero) and a stale one carries an older tag."""
    shapes = [(256, 256, 0), (2048, 2048, 128), (512, 2048, 128), (8192, 2048, 128),
              (2048, 8192, 128), (4096, 14336, 0), (8192, 28672, 128), (28672, 8192, 128),
              (1024, 8192, 128)]
    n_fused = 0
    for (N, K, G) in shapes:
        for M in (1, 2, 4, 8, 16, 17, 32, 33, 64, 65, 128, 512, 4096):
            for r in (0, 8, 16, 32, 64, 256):
                for gate in (sp.GATE_ONE, sp.GATE_SIGMOID_LINEAR, sp.GATE_TANH_MLP):
                    for path in range(7):
                        for with_ec in (True, False):
                            pr = sp.problem(M, N, K, G, sp.F16, r, gate, force_path=path)
                            try:
                                plan = sp.dispatch_plan(pr, with_ec)
                            except sp.SpearError:
                                continue
                            (tb, te), (db, de) = sp.workspace_regions(pr, with_ec)
                            fused = with_ec and r > 0 and plan.path == sp.PATH_FUSED_GEMV
                            if fused:
                                n_fused += 1
                                assert tb == COUNTERS and COUNTERS < te <= TAG_END
                            else:
                                assert (tb, te) == (0, 0)
                            ws = plan.workspace_bytes
                            assert ws >= TAG_END
                            if ws > TAG_END:
                                assert (db, de) == (TAG_END, ws)
                            else:
                                assert (db, de) == (0, 0)
    assert n_fused > 100


def test_weight_code_width():
    """3-bit codes (weight_bits = 3) take the same plan as 4-bit ones; any
    other width is rejected; the alias checks cover the 3-bit codes' own
    extent (3K/8 bytes per row)."""
    for M, N, K, G in ((1, 2048, 2048, 128), (16, 8192, 2048, 128), (4096, 4096, 4096, 0),
                       (64, 28672, 8192, 128)):
        for r in (0, 16, 64):
            p4 = sp.dispatch_plan(sp.problem(M, N, K, G, sp.F16, r))
            p3 = sp.dispatch_plan(sp.problem(M, N, K, G, sp.F16, r, weight_bits=3))
            assert (p3.path, p3.split_k, p3.tile_m, p3.tile_n, p3.grid, p3.workspace_bytes) == \
                (p4.path, p4.split_k, p4.tile_m, p4.tile_n, p4.grid, p4.workspace_bytes)
    for bad in (1, 2, 5, 8, -1):
        with pytest.raises(sp.SpearError) as e:
            sp.dispatch_plan(sp.problem(4, 256, 256, 0, sp.F16, 8, weight_bits=bad))
        assert e.value.status == -3
    prob = sp.problem(4, 256, 256, 0, sp.F16, 8, weight_bits=3)
    full = dict(x=ADDR["x"], y=ADDR["y"], q=ADDR["q"], s=ADDR["s"], z=ADDR["z"], A=ADDR["A"],
                B=ADDR["B"], w_g=ADDR["w"], ws=ADDR["W"], ws_bytes=1 << 30)
    args = dict(full)
    args["y"] = ADDR["q"] + 256 * 256 * 3 // 8 - 16  # the last 16 bytes of the 3-bit codes
    assert _call_ec(prob, **args) == -8
    dq = sp.problem(0, 256, 256, 0, sp.F16, weight_bits=3)
    w = sp.W4(ADDR["q"], ADDR["s"], ADDR["z"])
    assert sp.LIB.spear_w4_dequant(ctypes.byref(dq), ctypes.byref(w),
                                   ADDR["q"] + 256 * 256 * 3 // 8 - 16, None) == -8


def test_gemm_wave_roles_rules():
    """Loading and multiplying waves need 256-token tiles and one K-slice;
    the hook refuses them elsewhere (planning returns SPEAR_E_UNSUPPORTED);
    3-bit codes take the same plan as 4-bit ones."""
    q = sp.problem(4096, 8192, 8192, 128, sp.F16, 64, force_path=4)
    base = sp.dispatch_plan(q, True)
    assert (base.tile_m, base.tile_n, base.split_k) == (256, 256, 1)
    kv = sp.dispatch_plan(sp.problem(4096, 1024, 8192, 128, sp.F16, 64, force_path=4), True)
    assert kv.tile_n == 128
    sp.set_gemm_roles(2)
    try:
        assert sp.dispatch_plan(q, True).tile_n == 128
        sp.set_gemm_roles(3)
        assert sp.dispatch_plan(q, True).as_dict() == base.as_dict()
        sp.set_gemm_tile(128)
        with pytest.raises(sp.SpearError):
            sp.dispatch_plan(q, True)
        sp.set_gemm_tile(0)
        q3 = sp.problem(4096, 8192, 8192, 128, sp.F16, 64, force_path=4, weight_bits=3)
        assert sp.dispatch_plan(q3, True).as_dict() == base.as_dict()
        sp.set_gemm_slices(2)
        with pytest.raises(sp.SpearError):
            sp.dispatch_plan(q, True)
    finally:
        sp.set_gemm_roles(0)
        sp.set_gemm_slices(0)
        sp.set_gemm_tile(0)


def test_ceiling_library_exports():
    # the measured-ceiling kernels (measurement only) ship as their own
    # library; host-side argument checks reject bad sizes before any launch
    from paper_2606_11244_amd import ceiling
    lib = ceiling._lib()
    assert hasattr(lib, "spear_ceiling_read") and hasattr(lib, "spear_ceiling_mfma")
    assert lib.spear_ceiling_read(None, 1 << 20, None, None) != 0
    assert lib.spear_ceiling_read(ctypes.c_void_p(1 << 40), 15, ctypes.c_void_p(1 << 40), None) != 0
    assert lib.spear_ceiling_mfma(0, 1, 1, ctypes.c_void_p(1 << 40), None) != 0
