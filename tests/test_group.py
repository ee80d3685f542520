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
