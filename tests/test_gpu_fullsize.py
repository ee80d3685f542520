"""GPU parity at the full workload sizes, on complete outputs.

Decode (1, 4 and 16 tokens): every output element of every module of the
Llama-3.2-1B-, Llama-3-8B- and Llama-2-70B-shaped layer sets, on every decode
path (automatic dispatch, the local and producer-fused GEMVs, the semi-fused
pair, the naive chain) and in grouped calls, against the oracle evaluated in
row chunks. Prefill: every output row for one token of every 16-token tile
(so every 128- and 256-token GEMM tile and every split-K slice is covered),
at the token counts of each workload.

Each check runs twice: on the RTN layer as generated, and on an EC-only
copy of it whose scales are zero (so What == 0 and y is the EC term alone)
with the gate weights scaled so that the logits are of unit size (with
w_g ~ N(0, 0.05) the sigmoid saturates on deep layers and can switch the EC
off for a whole token). On the EC-only copy the parity bar applies to the EC
term itself."""
from __future__ import annotations

import concurrent.futures as cf
import copy

import numpy as np
import pytest
import torch

from oracle import spear_oracle as O
from paper_2606_11244_amd import synth as S

from gpu_util import assert_parity, log, with_fields

pytestmark = pytest.mark.gpu

P_AUTO, P_GEMV, P_MFMA, P_CHAIN, P_2K, P_LOCAL = 0, 1, 2, 3, 4, 5
DECODE_MS = (1, 4, 16)
PREFILL_MS = {1: (512, 2048, 4096), 3: (128, 512, 4096), 4: (64, 512, 2048)}
NAME = {1: "llama1b", 2: "llama1b-prefill", 3: "llama8b", 4: "llama70b"}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield


_CACHE = {}


def _layer(cid, module, M, gate=S.GATE_SIGMOID_LINEAR, rank=None):
    """The generated layer with M tokens (cached: one per config at a time)."""
    key = (cid, module, M, gate, rank)
    if key not in _CACHE:
        _CACHE.clear()
        _CACHE[key] = S.config_layer(cid, module, M, seed=0, gate_kind=gate, rank=rank)
    return _CACHE[key]


def _tokens(L, idx):
    """The layer restricted to the tokens idx (rows of x)."""
    return with_fields(L, x=np.ascontiguousarray(L.x[idx]), M=len(idx))


def _ec_only(L):
    """Zero scales (What == 0, so y is the EC term) and unit-size gate logits."""
    out = with_fields(L, scales=np.zeros_like(L.scales))
    wg = S.from_bits(L.w_g, L.act_dtype) * np.float32(20.0 / np.sqrt(L.K))
    out.w_g = S.to_bits(wg, L.act_dtype)
    return out


def oracle_full(L, chunk=1024, threads=8):
    """Eq. 3 on every output column, in row chunks run on a thread pool."""
    out = np.empty((L.M, L.N), np.float64)

    def one(r0):
        rows = np.arange(r0, min(L.N, r0 + chunk))
        out[:, rows] = O.w4ec_linear_rows(L, rows)

    with cf.ThreadPoolExecutor(threads) as ex:
        list(ex.map(one, range(0, L.N, chunk)))
    return out


class _Dev:
    """One layer's weights on the GPU, reused for every token subset."""

    def __init__(self, L):
        from paper_2606_11244_amd import spear as sp
        self.sp = sp
        self.base = sp.DeviceLayer(L)

    def with_x(self, L):
        d = copy.copy(self.base)
        d.layer = L
        d.M = L.M
        d.x = self.base.x.new_empty((L.M, L.K))
        d.x.copy_(torch.from_numpy(np.ascontiguousarray(L.x).view(np.int16)).view(d.x.dtype))
        d.y = torch.empty((L.M, L.N), dtype=self.base.dtype, device="cuda")
        return d

    def run(self, d, path, with_ec):
        sp = self.sp
        prob = d.problem(force_path=path, rank=None if with_ec else 0)
        ws = torch.zeros(max(256, sp.dispatch_plan(prob, with_ec).workspace_bytes),
                         dtype=torch.uint8, device="cuda")
        if with_ec:
            d.run_ec(prob, ws)
        else:
            d.run_w4(prob, ws)
        torch.cuda.synchronize()
        y = d.y.float().cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(y))
        return y


def _decode_paths(L):
    paths = [P_AUTO, P_GEMV, P_2K, P_CHAIN]
    if L.rank <= 16:
        paths.append(P_LOCAL)
    return paths


def _check_decode(cid, module, gate=S.GATE_SIGMOID_LINEAR, rank=None, ec_only=False):
    base = _layer(cid, module, max(DECODE_MS), gate=gate, rank=rank)
    if ec_only:
        base = _ec_only(base)
    dev = _Dev(base)
    ref16 = oracle_full(base)
    with_ec = base.rank > 0
    for M in DECODE_MS:
        L = _tokens(base, np.arange(M))
        d = dev.with_x(L)
        ref = ref16[:M]
        for p in (_decode_paths(L) if with_ec else [P_AUTO]):
            log(f"full-size decode {NAME[cid]} {module} M={M} rank={L.rank} gate={L.gate_kind} "
                f"path={p} ec_only={ec_only}")
            y = dev.run(d, p, with_ec)
            assert_parity(y, ref, f"{NAME[cid]}/{module}/M={M}/path={p}/ec_only={ec_only}")


def _check_decode_w4(cid, module):
    """The 4-bit product alone (the 70B-shaped model's modules without an EC)."""
    base = with_fields(_layer(cid, module, max(DECODE_MS)), rank=0)
    dev = _Dev(base)
    ref16 = oracle_full(base)
    for M in DECODE_MS:
        L = _tokens(base, np.arange(M))
        d = dev.with_x(L)
        for p in (P_AUTO, P_GEMV):
            log(f"full-size decode W4-only {NAME[cid]} {module} M={M} path={p}")
            assert_parity(dev.run(d, p, False), ref16[:M], f"{NAME[cid]}/{module}/M={M}/w4/{p}")


@pytest.mark.parametrize("module", ["q", "gate", "down"])
def test_decode_two_token_tiles_full_outputs(module):
    """32 tokens (two token tiles) on the 70B-shaped modules, whose launch
    shapes there (four row tiles, K split in two from K = 16384) are their
    own: complete outputs of the 4-bit product alone and of the W4+EC call
    (the producer-fused GEMV) against the oracle, the EC also isolated."""
    base = _layer(4, module, 32)
    for ec_only in (False, True):
        B = _ec_only(base) if ec_only else base
        dev = _Dev(B)
        d = dev.with_x(B)
        ref = oracle_full(B)
        log(f"full-size decode 32 tokens llama70b {module} ec_only={ec_only}")
        assert_parity(dev.run(d, P_AUTO, True), ref, f"llama70b/{module}/M=32/auto/ec_only={ec_only}")
        assert_parity(dev.run(d, P_GEMV, True), ref, f"llama70b/{module}/M=32/gemv/ec_only={ec_only}")
        if not ec_only:
            W4 = with_fields(B, rank=0)
            ref4 = oracle_full(W4)
            assert_parity(dev.run(d, P_AUTO, False), ref4, f"llama70b/{module}/M=32/w4")


def test_decode_two_token_tiles_int8_factors():
    """INT8 EC factors on the four-row-tile fused GEMV at 32 tokens (70B q),
    complete outputs against the oracle."""
    base = S.config_layer(4, "q", 32, seed=0, ab_int8=True)
    for ec_only in (False, True):
        B = _ec_only(base) if ec_only else base
        dev = _Dev(B)
        d = dev.with_x(B)
        ref = oracle_full(B)
        log(f"full-size decode 32 tokens llama70b q int8 ec_only={ec_only}")
        assert_parity(dev.run(d, P_AUTO, True), ref, f"llama70b/q/M=32/int8/ec_only={ec_only}")


def _tile_tokens(M):
    """One token of every 16-token tile, at a different offset in each."""
    t = np.arange((M + 15) // 16)
    return np.minimum(16 * t + (7 * t) % 16, M - 1)


def _check_prefill(cid, module, Ms, gate=S.GATE_SIGMOID_LINEAR, ec_only=False, paths=None):
    base = _layer(cid, module, max(Ms), gate=gate)
    if ec_only:
        base = _ec_only(base)
    dev = _Dev(base)
    # the reference of a token does not depend on how many tokens follow it:
    # one oracle pass over every sampled token of every token count
    every = np.unique(np.concatenate([_tile_tokens(M) for M in Ms]))
    ref_all = oracle_full(_tokens(base, every))
    for M in Ms:
        L = _tokens(base, np.arange(M))
        d = dev.with_x(L)
        idx = _tile_tokens(M)
        ref = ref_all[np.searchsorted(every, idx)]
        ps = paths if paths is not None else (
            [P_AUTO, P_2K] + ([P_MFMA] if L.rank <= 16 else []))
        for p in ps:
            log(f"full-size prefill {NAME[cid]} {module} M={M} tokens={len(idx)} path={p} "
                f"ec_only={ec_only}")
            y = dev.run(d, p, True)
            assert_parity(y[idx], ref, f"{NAME[cid]}/{module}/M={M}/path={p}/ec_only={ec_only}")


# ---- decode: every module, every path, complete outputs --------------------

@pytest.mark.parametrize("ec_only", [False, True])
@pytest.mark.parametrize("module", S.MODULES)
@pytest.mark.parametrize("cid", [1, 3, 4])
def test_decode_full_outputs(cid, module, ec_only):
    _check_decode(cid, module, ec_only=ec_only)
    if cid == 4 and not ec_only:
        # the 70B-shaped model runs three quarters of its modules without an EC
        _check_decode_w4(cid, module)


@pytest.mark.parametrize("ec_only", [False, True])
@pytest.mark.parametrize("module", ["q", "gate"])
def test_decode_full_outputs_tanh_gate(module, ec_only):
    """The paper's rank-space tanh-MLP gate (Eq. 3) on the 1B decode shapes."""
    _check_decode(1, module, gate=S.GATE_TANH_MLP, ec_only=ec_only)


@pytest.mark.parametrize("group", [("q", "k", "v"), ("gate", "up")])
@pytest.mark.parametrize("cid,with_ec", [(1, True), (4, False)])
def test_decode_grouped_full_outputs(cid, group, with_ec):
    """Grouped calls at the workload sizes (the decode pass's launches): every
    member's complete output, EC-only copies included (1B, local EC) and the
    4-bit product alone (70B modules without an EC)."""
    from paper_2606_11244_amd import spear as sp
    gen = {m: S.config_layer(cid, m, max(DECODE_MS), seed=0) for m in group}
    for ec_only in ((False, True) if with_ec else (False,)):
        for M in DECODE_MS:
            Ls, dls = [], []
            x = None
            for m in group:
                L = _tokens(gen[m], np.arange(M))
                if not with_ec:
                    L = with_fields(L, rank=0)
                if ec_only:
                    L = _ec_only(L)
                if x is not None:
                    L = with_fields(L, x=x)  # the members read one hidden state
                x = L.x
                Ls.append(L)
                dls.append(sp.DeviceLayer(L))
            for d in dls[1:]:
                d.x = dls[0].x
            probs = [d.problem(rank=None if with_ec else 0) for d in dls]
            members = [d.member(p, with_ec=with_ec) for d, p in zip(dls, probs)]
            ws = torch.zeros(max(256, sp.group_workspace(members)), dtype=torch.uint8,
                             device="cuda")
            log(f"full-size group {NAME[cid]} {group} M={M} ec={with_ec} ec_only={ec_only}")
            sp.w4ec_linear_group(members, ws)
            torch.cuda.synchronize()
            for L, d in zip(Ls, dls):
                y = d.y.float().cpu().numpy().astype(np.float64)
                assert_parity(y, oracle_full(L), f"group {group} member N={L.N} M={M}")


# ---- prefill: every output row, one token of every 16-token tile ----------

@pytest.mark.parametrize("ec_only", [False, True])
@pytest.mark.parametrize("module", S.MODULES)
@pytest.mark.parametrize("cid", [2, 3, 4])
def test_prefill_full_rows(cid, module, ec_only):
    Ms = PREFILL_MS[1 if cid == 2 else cid]
    if cid == 4 and module in ("gate", "up", "down"):
        Ms = Ms[:2]  # the 28672-wide modules at 64 and 512 tokens
    _check_prefill(cid, module, Ms, ec_only=ec_only)


@pytest.mark.parametrize("ec_only", [False, True])
@pytest.mark.parametrize("module", ["q", "gate"])
def test_prefill_full_rows_tanh_gate(module, ec_only):
    """The tanh-MLP gate on the 8B prefill shapes (rank 32: semi-fused pair
    and chain) and on the 1B ones (rank 16: the fully fused GEMM too)."""
    _check_prefill(3, module, (512, 4096), gate=S.GATE_TANH_MLP, ec_only=ec_only,
                   paths=[P_AUTO, P_2K, P_CHAIN])
    _check_prefill(2, module, (512, 2048), gate=S.GATE_TANH_MLP, ec_only=ec_only,
                   paths=[P_AUTO, P_MFMA, P_2K])


@pytest.mark.parametrize("cid,module,Ms", [(1, "q", (1, 16)), (1, "down", (1,)),
                                           (2, "gate", (512, 4096)), (3, "q", (1, 128)),
                                           (4, "down", (1, 64))])
def test_int8_factors_full_size(cid, module, Ms):
    """INT8 per-channel EC factors at the workload sizes, automatic dispatch,
    every output row (all tokens at decode, one per 16-token tile above)."""
    base = S.config_layer(cid, module, max(Ms), seed=0, ab_int8=True)
    for ec_only in (False, True):
        B = _ec_only(base) if ec_only else base
        dev = _Dev(B)
        for M in Ms:
            L = _tokens(B, np.arange(M))
            d = dev.with_x(L)
            idx = np.arange(M) if M <= 16 else _tile_tokens(M)
            ref = oracle_full(_tokens(B, idx))
            log(f"full-size int8 {NAME[cid]} {module} M={M} ec_only={ec_only}")
            y = dev.run(d, P_AUTO, True)
            assert_parity(y[idx], ref, f"int8 {NAME[cid]}/{module}/M={M}/ec_only={ec_only}")


def test_ec_only_copy_isolates_the_ec():
    """The EC-only copies really isolate a live EC: What is zero, and the gate
    is neither saturated off nor on for the tokens used above."""
    L = _layer(4, "down", max(DECODE_MS))
    E = _ec_only(L)
    assert not np.any(O.dequant(E.qweight[:8], E.scales[:8], E.zeros[:8], E.group_size))
    x = O.bits_to_f64(E.x, E.act_dtype)
    g = O.gate_sigmoid_linear(x, O.bits_to_f64(E.w_g, E.act_dtype), E.b_g)
    assert np.all((g > 0.02) & (g < 0.98)), g
    y = oracle_full(_tokens(E, np.arange(1)))
    assert np.abs(y).max() > 1e-2
