"""GPU tests of the grouped call (spear_w4ec_linear_group): each member's
output equals what its own single call writes, bit for bit, and matches the
oracle under the parity bar on sampled rows; covers the one-launch case
(members of one GEMV variant: the 4-bit product alone or the fused local
path, split-K members included), the one-after-another case (mixed
variants, token counts beyond the GEMV), INT8 factors, bf16, shared inputs,
empty members and graph replays, and groups where only some members share
the launch."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import spear_oracle as O
from paper_2606_11244_amd import synth as S

from gpu_util import assert_parity, log, with_fields

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield


def _rows(N, seed):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, N - 1], rng.choice(N, size=min(40, N), replace=False)]))


def _build(specs, M, seed, share_x=True, int8=False, dt=None):
    """specs: [(config id, module, with_ec)] -> (layers, device layers, probs)."""
    from paper_2606_11244_amd import spear as sp
    Ls, dls, probs = [], [], []
    for i, (cid, mod, with_ec) in enumerate(specs):
        L = S.config_layer(cid, mod, M, seed=seed + i, ab_int8=int8 and with_ec)
        if dt is not None and dt != L.act_dtype:
            L = S.make_layer(M=M, N=L.N, K=L.K, group_size=L.group_size, rank=L.rank,
                             act_dtype=dt, seed=seed + i)
        if share_x and Ls and Ls[0].K == L.K:
            L = with_fields(L, x=Ls[0].x)
        dl = sp.DeviceLayer(L)
        if share_x and dls and Ls[0].K == L.K:
            dl.x = dls[0].x
        Ls.append(L)
        dls.append(dl)
        probs.append(dl.problem(rank=None if with_ec else 0))
    return Ls, dls, probs


def _check(specs, M, seed=0, share_x=True, int8=False, dt=None, expect_one=None):
    from paper_2606_11244_amd import spear as sp
    Ls, dls, probs = _build(specs, M, seed, share_x, int8, dt)
    members = [d.member(p, with_ec=p.rank > 0) for d, p in zip(dls, probs)]
    ws = torch.zeros(max(256, sp.group_workspace(members)), dtype=torch.uint8, device="cuda")
    paths = [sp.PATH_NAMES[sp.dispatch_plan(p, p.rank > 0).path] for p in probs]
    log(f"group specs={specs} M={M} seed={seed} int8={int8} dt={dt} paths={paths}")
    sp.w4ec_linear_group(members, ws)
    torch.cuda.synchronize()
    got = [d.y.clone() for d in dls]
    # each member's own call
    for d, p in zip(dls, probs):
        wsi = sp.allocate_workspace(p, p.rank > 0)
        if p.rank > 0:
            d.run_ec(p, wsi)
        else:
            d.run_w4(p, wsi)
    torch.cuda.synchronize()
    for i, (g, d) in enumerate(zip(got, dls)):
        assert torch.equal(g.view(torch.int16), d.y.view(torch.int16)), f"member {i} differs"
    for i, (L, g, p) in enumerate(zip(Ls, got, probs)):
        rows = _rows(L.N, seed + i)
        LL = L if p.rank > 0 else with_fields(L, rank=0)
        ref = O.w4ec_linear_rows(LL, rows)
        y = g.float().cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(y))
        assert_parity(y[:, rows], ref, f"member {i} {specs[i]} M={M}")
    return got


QKV = [(1, "q", True), (1, "k", True), (1, "v", True)]
GATE_UP = [(1, "gate", True), (1, "up", True)]


@pytest.mark.parametrize("M", [1, 4, 16, 32])
def test_qkv_one_launch(M):
    _check(QKV, M)


@pytest.mark.parametrize("M", [1, 16])
def test_gate_up_one_launch(M):
    _check(GATE_UP, M, seed=3)


def test_split_k_members():
    # the 8192-deep module splits K at decode (the local variant at two
    # tokens): each member's partials and counters sit in its own slice of
    # the group workspace
    _check([(1, "down", True), (1, "down", True), (1, "down", True)], 2, seed=5)


def test_four_members_w4_only():
    _check([(1, "q", False), (1, "k", False), (1, "v", False), (1, "o", False)], 1, seed=7)


def test_int8_members():
    _check(QKV, 1, seed=9, int8=True)
    _check(GATE_UP, 16, seed=10, int8=True)


def test_bf16_members():
    _check(QKV, 1, seed=11, dt=S.BF16)


def test_mixed_variants_run_in_order():
    # an EC member next to a 4-bit-only one, and token counts the GEMV does
    # not take: the members run one after another, with the same outputs
    _check([(1, "q", True), (1, "k", False), (1, "v", True)], 1, seed=13)
    _check(QKV, 48, seed=14)
    _check([(2, "q", True), (2, "k", True)], 256, seed=15)


def test_70b_shaped_members_share_a_launch():
    # 4-bit-only q, k, v at one token: k and v re-planned to q's row tiles in
    # one launch; next to a q on the producer-fused EC path, k and v share
    # the launch without it
    from paper_2606_11244_amd import spear as sp
    specs = [(4, "q", False), (4, "k", False), (4, "v", False)]
    _, dls, probs = _build(specs, 1, 31)
    assert sp.group_launches([d.member(p, with_ec=False) for d, p in zip(dls, probs)]) == 1
    _check(specs, 1, seed=31)
    _check([(4, "q", True), (4, "k", False), (4, "v", False)], 1, seed=33)


def test_separate_inputs():
    _check(QKV, 1, seed=17, share_x=False)


def test_empty_member_skipped():
    from paper_2606_11244_amd import spear as sp
    Ls, dls, probs = _build(QKV, 1, 19)
    empty = torch.empty((0, Ls[1].N), dtype=dls[1].y.dtype, device="cuda")
    p0 = sp.problem(0, Ls[1].N, Ls[1].K, Ls[1].group_size, Ls[1].act_dtype, Ls[1].rank)
    members = [dls[0].member(probs[0]), dict(dls[1].member(p0), y=empty), dls[2].member(probs[2])]
    ws = torch.zeros(max(256, sp.group_workspace(members)), dtype=torch.uint8, device="cuda")
    log("group with an empty member")
    sp.w4ec_linear_group(members, ws)
    torch.cuda.synchronize()
    for i in (0, 2):
        rows = _rows(Ls[i].N, i)
        y = dls[i].y.float().cpu().numpy().astype(np.float64)
        assert_parity(y[:, rows], O.w4ec_linear_rows(Ls[i], rows), f"member {i}")


@pytest.mark.parametrize("M", [1, 16])
def test_graph_replay(M):
    """Every replay of a captured group, with new activations written by eager
    work between replays, equals the eager group call bit for bit."""
    from paper_2606_11244_amd import spear as sp
    Ls, dls, probs = _build(QKV, M, 21)
    members = [d.member(p) for d, p in zip(dls, probs)]
    ws = torch.zeros(max(256, sp.group_workspace(members)), dtype=torch.uint8, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        sp.w4ec_linear_group(members, ws, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sp.w4ec_linear_group(members, ws)
    gen = torch.Generator(device="cuda").manual_seed(M + 3)
    x = dls[0].x
    for i in range(4):
        x.copy_(torch.randn(x.shape, generator=gen, device="cuda").to(x.dtype))
        torch.cuda.synchronize()
        log(f"group graph M={M} replay={i}")
        g.replay()
        torch.cuda.synchronize()
        got = [d.y.clone() for d in dls]
        sp.w4ec_linear_group(members, ws)
        torch.cuda.synchronize()
        for j, d in enumerate(dls):
            assert torch.equal(got[j].view(torch.int16), d.y.view(torch.int16)), (i, j)


def test_graph_replay_partly_shared_launch():
    """A group where two members share the launch and one runs on its own
    (a 4-bit-only k between local-EC q and v), captured and replayed with new
    activations between replays: every replay equals the eager call."""
    from paper_2606_11244_amd import spear as sp
    specs = [(1, "q", True), (1, "k", False), (1, "v", True)]
    Ls, dls, probs = _build(specs, 1, 41)
    members = [d.member(p, with_ec=p.rank > 0) for d, p in zip(dls, probs)]
    assert sp.group_launches(members) == 2
    ws = torch.zeros(max(256, sp.group_workspace(members)), dtype=torch.uint8, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        sp.w4ec_linear_group(members, ws, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sp.w4ec_linear_group(members, ws)
    gen = torch.Generator(device="cuda").manual_seed(43)
    x = dls[0].x
    for i in range(3):
        x.copy_(torch.randn(x.shape, generator=gen, device="cuda").to(x.dtype))
        torch.cuda.synchronize()
        log(f"partly shared group graph replay={i}")
        g.replay()
        torch.cuda.synchronize()
        got = [d.y.clone() for d in dls]
        sp.w4ec_linear_group(members, ws)
        torch.cuda.synchronize()
        for j, d in enumerate(dls):
            assert torch.equal(got[j].view(torch.int16), d.y.view(torch.int16)), (i, j)


def test_workspace_shared_with_single_calls():
    """One workspace serves groups and single calls in stream order: groups
    whose members run one after another on the producer/consumer path (rank
    32, beyond the local variant), groups of split-K members in one launch,
    and single calls of both kinds, interleaved over three rounds; every
    output equals the one its call writes with a fresh workspace."""
    from paper_2606_11244_amd import spear as sp

    def dev(L):
        return sp.DeviceLayer(L)

    wide = [dev(S.make_layer(M=1, N=8192, K=2048, group_size=128, rank=32, seed=40 + i))
            for i in range(2)]
    # (the 8192-deep 1B down module at two tokens: the local variant split
    # over K; at one token it takes the producer-fused GEMV)
    deep = [dev(S.config_layer(1, "down", 2, seed=42 + i)) for i in range(2)]
    single = [dev(S.config_layer(1, "down", 2, seed=44)),
              dev(S.make_layer(M=1, N=2048, K=2048, group_size=128, rank=32, seed=45))]
    paths = {n: sp.PATH_NAMES[sp.dispatch_plan(d.problem()).path]
             for n, d in (("wide", wide[0]), ("deep", deep[0]), ("s0", single[0]),
                          ("s1", single[1]))}
    assert paths["wide"] == "fused_gemv" and paths["deep"] == "fused_local", paths
    ref = []
    for d in wide + deep + single:
        d.run_ec(d.problem(), sp.allocate_workspace(d.problem()))
        torch.cuda.synchronize()
        ref.append(d.y.clone())
    gw = [[d.member(d.problem()) for d in grp] for grp in (wide, deep)]
    need = max([sp.group_workspace(m) for m in gw] +
               [sp.dispatch_plan(d.problem()).workspace_bytes for d in single])
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for rnd in range(3):
        for d in wide + deep + single:
            d.y.zero_()
        log(f"shared workspace round {rnd} paths={paths}")
        sp.w4ec_linear_group(gw[0], ws)
        single[0].run_ec(single[0].problem(), ws)
        sp.w4ec_linear_group(gw[1], ws)
        single[1].run_ec(single[1].problem(), ws)
        torch.cuda.synchronize()
        for k, d in enumerate(wide + deep + single):
            assert torch.equal(d.y.view(torch.int16), ref[k].view(torch.int16)), (rnd, k)
