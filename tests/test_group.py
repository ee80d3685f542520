"""Host-side tests of the grouped call (spear_group_workspace,
spear_w4ec_linear_group): workspace layout and validation before any launch.
Every call here is rejected on the host or is the pure workspace query, so
these run without a GPU."""
from __future__ import annotations

import ctypes

from paper_2606_11244_amd import spear as sp

BASE = 0x7F0000000000


def _addr(member, key):
    # distinct, 16-byte aligned, 4 GiB apart per (member, buffer)
    keys = "xyqszABw"
    return BASE + (member * len(keys) + keys.index(key)) * (1 << 32)


def _calls(probs, with_ec=True, override=None):
    """ctypes array of members with fake addresses; override[(i, key)] = addr."""
    override = override or {}
    arr = (sp.LayerCall * max(1, len(probs)))()
    keep = []
    for i, p in enumerate(probs):
        a = {k: override.get((i, k), _addr(i, k)) for k in "xyqszABw"}
        w = sp.W4(a["q"], a["s"], a["z"])
        ec = sp.EC(a["A"], a["B"], 1.0, a["w"], 0.0, None, None, None, None)
        keep += [p, w, ec]
        arr[i].prob = ctypes.pointer(p)
        arr[i].x = a["x"]
        arr[i].w = ctypes.pointer(w)
        arr[i].ec = ctypes.pointer(ec) if with_ec else None
        arr[i].y = a["y"]
    return arr, keep


def _ws(probs, with_ec=True):
    arr, keep = _calls(probs, with_ec)
    out = ctypes.c_size_t(0)
    st = sp.LIB.spear_group_workspace(len(probs), arr, ctypes.byref(out))
    return st, out.value


def _qkv(M=1):
    return [sp.problem(M, 2048, 2048, 128, sp.F16, 16), sp.problem(M, 512, 2048, 128, sp.F16, 16),
            sp.problem(M, 512, 2048, 128, sp.F16, 16)]


COUNTER_BLOCK = 131072 + (1 << 20)  # the counter block and the tagged region of every workspace


def _want(sizes):
    if not any(sizes):
        return 0
    return COUNTER_BLOCK + sum(-(-max(0, b - COUNTER_BLOCK) // 256) * 256 for b in sizes)


def test_workspace_is_counter_block_plus_member_data():
    for probs in (_qkv(1), _qkv(16), [sp.problem(1, 2048, 8192, 128, sp.F16, 16)] * 2,
                  [sp.problem(512, 2048, 2048, 128, sp.F16, 16), sp.problem(1, 512, 2048)]):
        st, got = _ws(probs)
        assert st == 0
        sizes = [sp.dispatch_plan(p, True).workspace_bytes for p in probs]
        assert all(b == 0 or b >= COUNTER_BLOCK for b in sizes)
        assert got == _want(sizes)
        # large enough for any member run on its own at the same base
        assert got >= max(sizes)
    # without an EC each member sizes its 4-bit plan
    probs = _qkv(1)
    st, got = _ws(probs, with_ec=False)
    assert st == 0
    assert got == _want([sp.dispatch_plan(p, False).workspace_bytes for p in probs])


def test_group_size_and_nulls():
    probs = _qkv(1)
    arr, keep = _calls(probs)
    out = ctypes.c_size_t(0)
    assert sp.LIB.spear_group_workspace(0, arr, ctypes.byref(out)) == -2
    assert sp.LIB.spear_group_workspace(sp.GROUP_MAX + 1, arr, ctypes.byref(out)) == -2
    assert sp.LIB.spear_group_workspace(3, None, ctypes.byref(out)) == -1
    assert sp.LIB.spear_group_workspace(3, arr, None) == -1
    assert sp.LIB.spear_w4ec_linear_group(0, arr, BASE, 1 << 30, None) == -2
    assert sp.LIB.spear_w4ec_linear_group(3, None, BASE, 1 << 30, None) == -1
    arr[1].prob = None
    assert sp.LIB.spear_w4ec_linear_group(3, arr, BASE, 1 << 30, None) == -1
    # a member's own shape errors come back as they do from the single call
    bad = _qkv(1)
    bad[2] = sp.problem(1, 512, 2000, 128, sp.F16, 16)
    arr, keep = _calls(bad)
    assert sp.LIB.spear_w4ec_linear_group(3, arr, BASE, 1 << 30, None) == -2


def test_member_checks_before_launch():
    probs = _qkv(1)
    st, need = _ws(probs)
    assert st == 0
    ws = BASE + 200 * (1 << 32)
    # null weights and EC factors of any member
    for i in range(3):
        for key in ("q", "x", "A", "w"):
            arr, keep = _calls(probs, override={(i, key): 0})
            assert sp.LIB.spear_w4ec_linear_group(3, arr, ws, need, None) == -1, (i, key)
    # a later member's NULL weight struct is reported before any member's
    # output is compared with it
    arr, keep = _calls(probs)
    arr[2].w = None
    assert sp.LIB.spear_w4ec_linear_group(3, arr, ws, need, None) == -1
    # workspace size and alignment
    arr, keep = _calls(probs)
    if need > 0:
        assert sp.LIB.spear_w4ec_linear_group(3, arr, None, 0, None) == -5
        assert sp.LIB.spear_w4ec_linear_group(3, arr, ws, need - 1, None) == -5
        assert sp.LIB.spear_w4ec_linear_group(3, arr, ws + 8, need, None) == -4


def test_cross_member_alias_rejected():
    probs = _qkv(1)
    st, need = _ws(probs)
    ws = BASE + 200 * (1 << 32)
    # member 0 writes over member 1's input, weights, factors or output
    for key in ("x", "q", "s", "z", "A", "B", "w", "y"):
        arr, keep = _calls(probs, override={(0, "y"): _addr(1, key) + 16})
        assert sp.LIB.spear_w4ec_linear_group(3, arr, ws, max(need, 256), None) == -8, key
    # a member's output over the group workspace
    assert need > 256
    arr, keep = _calls(probs, override={(2, "y"): ws + 256})
    assert sp.LIB.spear_w4ec_linear_group(3, arr, ws, need, None) == -8


def _launches(probs, ecs):
    """spear_group_launches with member i carrying an EC iff ecs[i]."""
    arr, keep = _calls(probs)
    for i, e in enumerate(ecs):
        if not e:
            arr[i].ec = None
    out = ctypes.c_int32(-1)
    st = sp.LIB.spear_group_launches(len(probs), arr, ctypes.byref(out))
    return st, out.value


def _own(p, ec):
    return sp.dispatch_plan(p, ec).num_launches


def test_group_launches_share_one_launch():
    # 70B-shaped q, k, v and gate, up at one token, 4-bit only: one launch
    # each (k and v re-planned to q's row tiles, which leaves their K-slices
    # and per-wave work unchanged)
    qkv = [sp.problem(1, 8192, 8192, 128, sp.F16, 0), sp.problem(1, 1024, 8192, 128, sp.F16, 0),
           sp.problem(1, 1024, 8192, 128, sp.F16, 0)]
    assert _launches(qkv, [False] * 3) == (0, 1)
    gu = [sp.problem(1, 28672, 8192, 128, sp.F16, 0)] * 2
    assert _launches(gu, [False] * 2) == (0, 1)
    # 1B-shaped q, k, v with the local EC at one and 16 tokens
    for M in (1, 16):
        assert _launches(_qkv(M), [True] * 3) == (0, 1)


def test_group_launches_mixed_members():
    # an EC member on the producer-fused path runs on its own; the two
    # 4-bit-only members share a launch
    probs = [sp.problem(1, 8192, 8192, 128, sp.F16, 64), sp.problem(1, 1024, 8192, 128, sp.F16, 0),
             sp.problem(1, 1024, 8192, 128, sp.F16, 0)]
    assert sp.PATH_NAMES[sp.dispatch_plan(probs[0], True).path] == "fused_gemv"
    st, n = _launches(probs, [True, False, False])
    assert st == 0 and n == _own(probs[0], True) + 1
    # local EC on q and v, k 4-bit only: the larger set (q, v) shares a
    # launch, k runs on its own
    probs = _qkv(1)
    st, n = _launches(probs, [True, False, True])
    assert st == 0 and n == 1 + _own(probs[1], False)
    # every member on its own variant: each its own launches
    probs = [sp.problem(1, 8192, 8192, 128, sp.F16, 64), sp.problem(1, 1024, 8192, 128, sp.F16, 0)]
    st, n = _launches(probs, [True, False])
    assert st == 0 and n == _own(probs[0], True) + _own(probs[1], False)


def test_group_launches_beyond_the_gemv_and_empty_members():
    # prefill token counts take the GEMM: every member on its own
    probs = [sp.problem(4096, 8192, 8192, 128, sp.F16, 64), sp.problem(4096, 1024, 8192, 128, sp.F16, 0),
             sp.problem(4096, 1024, 8192, 128, sp.F16, 0)]
    st, n = _launches(probs, [True, False, False])
    assert st == 0 and n == _own(probs[0], True) + 2 * _own(probs[1], False)
    # an empty member makes no launch and does not join the shared one
    probs = _qkv(1)
    probs[1] = sp.problem(0, 512, 2048, 128, sp.F16, 16)
    assert _launches(probs, [True] * 3) == (0, 1)
    probs = [sp.problem(1, 2048, 2048, 128, sp.F16, 16), sp.problem(0, 512, 2048, 128, sp.F16, 16)]
    st, n = _launches(probs, [True, True])
    assert st == 0 and n == _own(probs[0], True)
    # a NULL out pointer
    arr, keep = _calls(_qkv(1))
    assert sp.LIB.spear_group_launches(3, arr, None) == -1
