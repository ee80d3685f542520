"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

The bar: int4 unpack/dequant bit-exact; outputs within relative Frobenius
error 5e-3 and max |d| <= 1e-2 * max |y_ref|. Inputs are seeded synthetic
layers from paper_2606_11244_amd.synth.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import spear_oracle as O
from paper_2606_11244_amd import synth as S

from gpu_util import assert_parity, gpu_y, log, scaled_ec, with_fields, zero_weight

pytestmark = pytest.mark.gpu

PATHS = {"auto": 0, "fused_gemv": 1, "fused_mfma": 2, "chain": 3, "2k": 4, "fused_local": 5,
         "overlap": 6}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_11244_amd import spear  # noqa: F401  (fails loudly if not built)
    yield


def _local_ok(L):
    """The local fused variant: M <= 32, rank <= 16, every gate."""
    return L.M <= 32 and L.rank <= 16


def _mfma_ok(L):
    """The fully fused GEMM: rank <= 16, every gate."""
    return L.rank <= 16


def _paths_for(M, L):
    out = []
    for name, p in PATHS.items():
        if name == "fused_gemv" and M > 64:
            continue
        if name == "fused_local" and not _local_ok(L):
            continue
        if name == "fused_mfma" and not _mfma_ok(L):
            continue
        out.append(p)
    return out


# ---------------------------------------------------------------------------
# bit-exact dequantisation
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dt", [S.F16, S.BF16])
@pytest.mark.parametrize("G", [128, 0])
def test_dequant_bit_exact(dt, G):
    from paper_2606_11244_amd import spear as sp
    rng = np.random.default_rng(7)
    N, K = 16 * 16, 256
    g = K if G == 0 else G
    # every code against every zero point, random fp16 scales (incl. subnormal-producing ones)
    q = np.tile(np.arange(16), (N, K // 16))
    z = np.repeat(np.arange(16), 16)[:, None].repeat(K // g, axis=1).astype(np.uint8)
    s = rng.choice([rng.uniform(1e-5, 1e-3), rng.uniform(1e-3, 2.0)], size=(N, K // g))
    s = np.where(rng.random((N, K // g)) < 0.2, 6e-8, s).astype(np.float16)
    qw = S.pack_int4(q)
    want = O.dequant_bits(qw, s.view(np.uint16), z, g, dt)
    log(f"dequant dt={dt} G={g}")
    dq = torch.from_numpy(qw.view(np.int32)).cuda()
    ds = torch.from_numpy(s.view(np.int16)).cuda()
    dz = torch.from_numpy(z).cuda()
    out = torch.empty((N, K), dtype=torch.int16, device="cuda")
    sp.w4_dequant(sp.problem(0, N, K, G, dt), dq, ds, dz, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint16)
    assert np.array_equal(got, want), f"{(got != want).sum()} mismatching bits"


@pytest.mark.parametrize("dt", [S.F16, S.BF16])
@pytest.mark.parametrize("path", ["auto", "fused_gemv", "2k", "chain"])
def test_decode_cancellation_worst_case(dt, path):
    """The decode GEMV never forms a dequantised weight: per 128-wide group it
    sums x (bias + q) and subtracts (bias + z) sum x in fp32 (bias 1024 for
    fp16, 128 for bf16), which cancels. The worst case for that is a long K
    (the 70B down projection, 28672), activations of one sign with outlier
    channels (every group's sum of x large), and codes within one step of the
    zero point (the exact group sums small against the biased ones). The
    result must still meet the parity bar."""
    M, N, K, G = 4, 512, 28672, 128
    L = S.make_layer(M=M, N=N, K=K, group_size=G, rank=16, act_dtype=dt, seed=21)
    rng = np.random.default_rng(21)
    x = np.abs(rng.standard_normal((M, K))).astype(np.float32) + 2.0
    out_idx = rng.choice(K, size=round(0.01 * K), replace=False)
    x[:, out_idx] *= 20.0
    z = rng.integers(1, 15, size=(N, K // G))
    q = np.clip(z[:, np.arange(K) // G] + rng.integers(-1, 2, size=(N, K)), 0, 15)
    L = with_fields(L, x=S.to_bits(x, dt), qweight=S.pack_int4(q), zeros=z.astype(np.uint8))
    ref = O.w4ec_linear(L)
    log(f"cancellation worst case dt={dt} path={path}")
    relf, mx = assert_parity(gpu_y(L, PATHS[path]), ref, f"cancellation/{dt}/{path}")
    log(f"  relF={relf:.2e} max|d|={mx:.2e}")


# ---------------------------------------------------------------------------
# small configurations, every path
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("path", list(PATHS))
def test_tiny_config(seed, path):
    """K=256, N=256, M=4, per-channel, r=8, sigmoid-linear gate, fp16."""
    L = S.config_layer(0, "tiny", 4, seed=seed)
    log(f"tiny seed={seed} path={path}")
    assert_parity(gpu_y(L, PATHS[path]), O.w4ec_linear(L), f"tiny/{path}/{seed}")


@pytest.mark.parametrize("M", [1, 2, 3, 5, 15, 16, 17, 31, 33, 48, 64, 65, 127, 129, 255])
def test_token_counts(M):
    """Ragged token counts across the GEMV/GEMM boundary; N not a tile multiple."""
    L = S.make_layer(M=M, N=320, K=512, group_size=128, rank=16, seed=M)
    ref = O.w4ec_linear(L)
    for p in _paths_for(M, L):
        log(f"M={M} path={p}")
        assert_parity(gpu_y(L, p), ref, f"M={M} path={p}")


@pytest.mark.parametrize("N", [1, 15, 17, 200, 1000])
@pytest.mark.parametrize("M", [1, 16, 100])
def test_ragged_rows(N, M):
    L = S.make_layer(M=M, N=N, K=384, group_size=128, rank=8, seed=N + M)
    ref = O.w4ec_linear(L)
    for p in _paths_for(M, L):
        log(f"N={N} M={M} path={p}")
        assert_parity(gpu_y(L, p), ref, f"N={N} M={M} path={p}")


@pytest.mark.parametrize("gate", [S.GATE_ONE, S.GATE_SIGMOID_LINEAR, S.GATE_TANH_MLP])
@pytest.mark.parametrize("dt", [S.F16, S.BF16])
@pytest.mark.parametrize("M", [1, 8, 40, 200])
def test_gates_and_dtypes(gate, dt, M):
    L = S.make_layer(M=M, N=256, K=1024, group_size=0 if dt == S.BF16 else 128, rank=16,
                     act_dtype=dt, gate_kind=gate, seed=3, ec_std=0.05)
    ref = O.w4ec_linear(L)
    for p in _paths_for(M, L):
        log(f"gate={gate} dt={dt} M={M} path={p}")
        assert_parity(gpu_y(L, p), ref, f"gate={gate} dt={dt} M={M} path={p}")


@pytest.mark.parametrize("r", [0, 1, 7, 8, 16, 32, 64, 100, 256])
@pytest.mark.parametrize("M", [3, 130])
def test_ranks(r, M):
    L = S.make_layer(M=M, N=192, K=512, group_size=128, rank=r, seed=r, ec_std=0.05,
                     gate_kind=S.GATE_TANH_MLP if r in (7, 100) else S.GATE_SIGMOID_LINEAR)
    ref = O.w4ec_linear(L)
    for p in _paths_for(M, L):
        log(f"r={r} M={M} path={p}")
        assert_parity(gpu_y(L, p), ref, f"r={r} M={M} path={p}")


# ---------------------------------------------------------------------------
# cases that isolate the EC term (it is ~1% of y at the workload scales)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dt", [S.F16, S.BF16])
@pytest.mark.parametrize("M", [1, 16, 300])
@pytest.mark.parametrize("gate", [S.GATE_SIGMOID_LINEAR, S.GATE_TANH_MLP])
def test_ec_isolated_zero_weight(dt, M, gate):
    """q == z everywhere: W_hat == 0 exactly, so y is the EC term alone."""
    L = zero_weight(S.make_layer(M=M, N=256, K=1024, group_size=128, rank=16, act_dtype=dt,
                                 gate_kind=gate, seed=11))
    ref = O.w4ec_linear(L)
    assert np.abs(O.w4_linear_layer(L)).max() == 0.0
    for p in _paths_for(M, L):
        log(f"zero-weight dt={dt} M={M} gate={gate} path={p}")
        assert_parity(gpu_y(L, p), ref, f"zero-weight dt={dt} M={M} gate={gate} path={p}")


@pytest.mark.parametrize("M", [2, 16, 257])
def test_ec_scaled_x30(M):
    L = scaled_ec(S.make_layer(M=M, N=512, K=2048, group_size=128, rank=16, seed=5), 30.0)
    ref = O.w4ec_linear(L)
    for p in _paths_for(M, L):
        log(f"x30 M={M} path={p}")
        assert_parity(gpu_y(L, p), ref, f"x30 M={M} path={p}")


@pytest.mark.parametrize("M", [4, 200])
def test_gate_pinned_values(M):
    """b_g = -1e4 gives g = 0 (y = the plain 4-bit product); w_g = 0, b_g = 0
    gives g = 1/2 exactly."""
    L = S.make_layer(M=M, N=256, K=1024, group_size=128, rank=16, seed=9, ec_std=0.2)
    off = with_fields(L, b_g=-1.0e4)
    half = with_fields(L, w_g=np.zeros_like(L.w_g), b_g=0.0)
    y_w4 = gpu_y(L, 0, with_ec=False)
    for p in _paths_for(M, L):
        log(f"gate-pinned M={M} path={p}")
        assert_parity(gpu_y(off, p), O.w4_linear_layer(L), f"g=0 M={M} path={p}")
        assert_parity(gpu_y(half, p), O.w4ec_linear(half), f"g=1/2 M={M} path={p}")
    assert_parity(y_w4, O.w4_linear_layer(L), "w4_linear")


@pytest.mark.parametrize("M", [1, 9, 64, 100])
def test_rank0_equals_w4_linear(M):
    """rank 0 runs exactly the 4-bit kernel: bit-identical to spear_w4_linear."""
    L = S.make_layer(M=M, N=384, K=1024, group_size=128, rank=0, seed=2)
    a = gpu_y(L, 0, with_ec=True)
    b = gpu_y(L, 0, with_ec=False)
    assert np.array_equal(a, b)
    assert_parity(a, O.w4_linear_layer(L), f"r=0 M={M}")


# ---------------------------------------------------------------------------
# robustness of the fused path's cross-workgroup machinery
# ---------------------------------------------------------------------------

def test_fused_wait_fallback():
    """With a zero poll budget every workgroup computes the EC itself: the
    result must still meet the bar."""
    from paper_2606_11244_amd import spear as sp
    L = S.make_layer(M=5, N=1024, K=2048, group_size=128, rank=32, seed=4, ec_std=0.05)
    ref = O.w4ec_linear(L)
    old = sp.set_wait_polls(0)
    try:
        log("fallback fused")
        y = gpu_y(L, PATHS["fused_gemv"])
    finally:
        sp.set_wait_polls(old)
    assert_parity(y, ref, "fused fallback")


@pytest.mark.parametrize("path", ["fused_gemv", "fused_local"])
def test_deterministic_and_workspace_reuse(path):
    """Repeated calls are bit-identical (fixed reduction orders), also when
    calls of other shapes use the same workspace in between: every counter is
    back at zero after a call and every data region is rewritten before it is
    read."""
    from paper_2606_11244_amd import spear as sp
    # K = 16384 spans several K-slices of the 4-bit product and of the EC
    L = S.make_layer(M=3, N=1024, K=16384, group_size=128, rank=16, seed=6)
    other = S.make_layer(M=16, N=700, K=8192, group_size=128, rank=64, seed=7)
    dl, do = sp.DeviceLayer(L), sp.DeviceLayer(other)
    prob = dl.problem(force_path=PATHS[path])
    plan = sp.dispatch_plan(prob)
    assert plan.split_k > 1 and plan.ec_splits > 1
    other_path = PATHS["fused_gemv" if path == "fused_local" else "fused_local"]
    size = max([plan.workspace_bytes, sp.dispatch_plan(dl.problem(force_path=other_path)).workspace_bytes,
                sp.dispatch_plan(dl.problem(), False).workspace_bytes,
                sp.dispatch_plan(do.problem(), False).workspace_bytes] +
               [sp.dispatch_plan(do.problem(force_path=p)).workspace_bytes for p in (0, 3, 4)])
    ws = torch.zeros(size, dtype=torch.uint8, device="cuda")
    log(f"determinism {path}")
    first = gpu_y(L, PATHS[path], workspace=ws, dev=dl)
    for i in range(4):
        for p in (0, 3, 4):
            gpu_y(other, p, workspace=ws, dev=do)
        gpu_y(other, 0, with_ec=False, workspace=ws, dev=do)
        gpu_y(L, 0, with_ec=False, workspace=ws, dev=dl)
        gpu_y(L, other_path, workspace=ws, dev=dl)
        again = gpu_y(L, PATHS[path], workspace=ws, dev=dl)
        assert np.array_equal(first, again), i
    assert_parity(first, O.w4ec_linear(L), f"determinism {path}")


@pytest.mark.parametrize("M", [1, 4])
def test_workspace_shared_by_every_path(M):
    """The fused path's tagged words live in a region no other call writes.
    Between fused calls every other kind of call (the naive chain, the
    semi-fused pair on the GEMV and on the GEMM, the local and fully fused
    variants, the 4-bit product alone on both kernels, split over K) writes
    its partial sums into the same workspace, and then every data region past
    the tagged one is filled with words that carry the next fused launch's
    own tag (the workspace's launch counter tells which): the fused call must
    still return exactly what it returned on a fresh workspace."""
    from paper_2606_11244_amd import spear as sp
    L = S.make_layer(M=M, N=1024, K=4096, group_size=128, rank=32, seed=11 + M)
    dec = S.make_layer(M=3, N=1024, K=16384, group_size=128, rank=16, seed=12)
    pre = S.make_layer(M=96, N=256, K=4096, group_size=128, rank=16, seed=13)
    dl, dd, dp = sp.DeviceLayer(L), sp.DeviceLayer(dec), sp.DeviceLayer(pre)
    fused = dl.problem(force_path=PATHS["fused_gemv"])
    others = [(dd, PATHS[p], True) for p in ("chain", "2k", "fused_local", "fused_gemv")]
    others += [(dp, PATHS[p], True) for p in ("chain", "2k", "fused_mfma")]
    others += [(dd, 0, False), (dp, 0, False)]
    size = max([sp.dispatch_plan(fused).workspace_bytes] +
               [sp.dispatch_plan(d.problem(force_path=p), e).workspace_bytes for d, p, e in others])
    assert sp.dispatch_plan(dd.problem(), False).split_k > 1
    assert sp.dispatch_plan(dp.problem(), False).split_k > 1
    data_base = 131072 + (1 << 20)
    ws = torch.zeros(size, dtype=torch.uint8, device="cuda")
    first = gpu_y(L, PATHS["fused_gemv"], workspace=ws, dev=dl)
    fresh = gpu_y(L, PATHS["fused_gemv"], workspace=torch.zeros_like(ws), dev=dl)
    assert np.array_equal(first, fresh)
    for i in range(3):
        for d, p, e in others:
            log(f"shared workspace M={M} round={i} path={p} ec={e} M'={d.layer.M}")
            gpu_y(d.layer, p, with_ec=e, workspace=ws, dev=d)
        torch.cuda.synchronize()
        gen = int(ws[:8].view(torch.int64).item()) >> 32  # class 0: launches so far
        tag = (gen + 1) & 0xFFFFFFFF
        word = (tag << 32) | 0x3F800000  # fp32 1.0 under the next launch's tag
        if word >= 1 << 63:
            word -= 1 << 64
        n64 = (size - data_base) // 8
        ws[data_base:data_base + 8 * n64].view(torch.int64).fill_(word)
        again = gpu_y(L, PATHS["fused_gemv"], workspace=ws, dev=dl)
        assert np.array_equal(first, again), i
    assert_parity(first, O.w4ec_linear(L), f"shared workspace M={M}")


def test_streams_and_reuse():
    """Calls on a side stream, back to back with different shapes on one
    workspace sized for the largest."""
    from paper_2606_11244_amd import spear as sp
    s = torch.cuda.Stream()
    layers = [S.make_layer(M=M, N=512, K=1024, group_size=128, rank=16, seed=M) for M in (1, 7, 16)]
    devs = [sp.DeviceLayer(L) for L in layers]
    wsz = max(sp.dispatch_plan(d.problem()).workspace_bytes for d in devs)
    ws = torch.zeros(wsz, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        for _ in range(3):
            for d in devs:
                d.run_ec(d.problem(), ws, stream=s)
    s.synchronize()
    for L, d in zip(layers, devs):
        assert_parity(d.y.float().cpu().numpy(), O.w4ec_linear(L), f"stream M={L.M}")


@pytest.mark.parametrize("M,path", [(4, 1), (4, 4), (4, 3), (200, 0), (200, 3), (33, 1), (4, 5),
                                    (17, 5), (200, 2), (4, 2), (4, 6), (200, 6)])
def test_graph_replay(M, path):
    """A captured call replayed several times, with new activations written
    between replays by eager work: every replay equals the eager call on the
    same inputs bit for bit (counters and flags reset themselves, since a
    graph keeps the epoch it was captured with)."""
    from paper_2606_11244_amd import spear as sp
    L = S.make_layer(M=M, N=1024, K=2048, group_size=128, rank=16, seed=M + path)
    dl = sp.DeviceLayer(L)
    prob = dl.problem(force_path=path)
    ws = sp.allocate_workspace(prob)
    y_eager = torch.empty_like(dl.y)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # warm-up outside capture
        dl.run_ec(prob, ws, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dl.run_ec(prob, ws)
    gen = torch.Generator(device="cuda").manual_seed(M)
    for i in range(4):
        dl.x.copy_(torch.randn(dl.x.shape, generator=gen, device="cuda").to(dl.x.dtype))
        torch.cuda.synchronize()
        log(f"graph M={M} path={path} replay={i}")
        g.replay()
        torch.cuda.synchronize()
        y_graph = dl.y.clone()
        dl.run_ec(prob, ws, y=y_eager)
        torch.cuda.synchronize()
        assert torch.equal(y_graph, y_eager), f"replay {i}"


@pytest.mark.parametrize("M", [1, 16, 40])
@pytest.mark.parametrize("K", [128, 8320, 16384, 28672])
def test_long_and_short_k(M, K):
    """K from a single 128-wide iteration to the 70B down projection's 28672:
    one-wave blocks, partial last slices and multi-slice reductions."""
    L = S.make_layer(M=M, N=96, K=K, group_size=128, rank=24, seed=K + M, ec_std=0.05)
    ref = O.w4ec_linear(L)
    for p in _paths_for(M, L):
        log(f"K={K} M={M} path={p}")
        assert_parity(gpu_y(L, p), ref, f"K={K} M={M} path={p}")


GEMV_SHAPES = [(1, 1), (1, 2), (1, 4), (2, 1), (2, 2), (2, 4), (3, 1), (3, 2), (4, 1)]


@pytest.mark.parametrize("shape", GEMV_SHAPES, ids=lambda t: "mt%d_rt%d" % t)
@pytest.mark.parametrize("slices,waves", [(0, 0), (1, 3), (5, 8), (3, 1)])
def test_every_gemv_launch_shape(shape, slices, waves):
    """Each compiled decode launch shape (token tiles, row tiles) with several
    K-slice and wave counts (partial last slices, one-wave blocks) meets the
    bar on ragged rows, for the 4-bit-only and both EC paths."""
    from paper_2606_11244_amd import spear as sp
    mt, rt = shape
    M = {1: 9, 2: 20, 3: 40, 4: 64}[mt]
    sp.set_gemv_shape(rt, slices, waves)
    try:
        for K in (1024, 8192):
            L = S.make_layer(M=M, N=200, K=K, group_size=128, rank=16, seed=K + rt, ec_std=0.05)
            ref = O.w4ec_linear(L)
            for p in (1, 4, 5) if mt <= 2 else (1, 4):
                log(f"shape={shape} slices={slices} waves={waves} K={K} path={p}")
                try:
                    y = gpu_y(L, p)
                except sp.SpearError as e:
                    # the local variant stages its K-slice of A in LDS: long
                    # slices are rejected on the host
                    if p == 5 and e.status == -6:
                        continue
                    raise
                assert_parity(y, ref, f"shape={shape} K={K} path={p}")
            assert_parity(gpu_y(L, 0, with_ec=False), O.w4_linear_layer(L), f"shape={shape} w4")
    finally:
        sp.set_gemv_shape(0, 0, 0)


@pytest.mark.parametrize("slices", [1, 2, 4, 8])
@pytest.mark.parametrize("M", [65, 130, 300])
def test_gemm_split_k(slices, M):
    """The prefill GEMM with its K split into 1..8 slices (each summed in
    slice order by the tile's last workgroup; the fully fused variant sums
    its EC projection the same way) meets the bar on every GEMM path and on
    the 4-bit product alone; ragged tokens and rows."""
    from paper_2606_11244_amd import spear as sp
    L = S.make_layer(M=M, N=200, K=1024, group_size=128, rank=16, seed=M + slices, ec_std=0.05)
    ref = O.w4ec_linear(L)
    sp.set_gemm_slices(slices)
    try:
        for p in (PATHS["2k"], PATHS["chain"], PATHS["fused_mfma"]):
            log(f"gemm slices={slices} M={M} path={p}")
            assert_parity(gpu_y(L, p), ref, f"slices={slices} M={M} path={p}")
        assert_parity(gpu_y(L, 0, with_ec=False), O.w4_linear_layer(L), f"slices={slices} w4")
    finally:
        sp.set_gemm_slices(0)


# ---------------------------------------------------------------------------
# INT8 per-channel symmetric EC factors (the deployed format)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("M,N,K,G,rank,dt,gate", [
    (1, 520, 1024, 128, 16, S.F16, S.GATE_SIGMOID_LINEAR),
    (4, 256, 2048, 0, 8, S.BF16, S.GATE_SIGMOID_LINEAR),
    (17, 200, 1024, 128, 16, S.F16, S.GATE_ONE),
    (3, 256, 1024, 128, 32, S.F16, S.GATE_TANH_MLP),
    (40, 136, 512, 128, 24, S.BF16, S.GATE_SIGMOID_LINEAR),
    (65, 200, 1024, 128, 16, S.F16, S.GATE_SIGMOID_LINEAR),
    (300, 520, 2048, 0, 16, S.BF16, S.GATE_SIGMOID_LINEAR),
    (130, 256, 1024, 128, 24, S.F16, S.GATE_TANH_MLP),
])
def test_int8_factors_all_paths(M, N, K, G, rank, dt, gate):
    """INT8 A and B with fp32 per-channel scales on every path that takes
    the shape: the codes are dequantised in the kernels (to the activation
    dtype where they feed an MFMA, exactly where the sum is fp32) and the
    result meets the bar against the oracle's exact s * q factors. The EC
    term is made large (ec_std 0.05) so that a wrong scale cannot hide."""
    L = S.make_layer(M=M, N=N, K=K, group_size=G, rank=rank, act_dtype=dt, gate_kind=gate,
                     seed=M + N + rank, ec_std=0.05, ab_int8=True)
    ref = O.w4ec_linear(L)
    base = O.w4_linear_layer(L)
    # the EC term is a sizeable part of the output
    assert np.linalg.norm(ref - base) > 0.1 * np.linalg.norm(ref)
    for p in _paths_for(M, L):
        log(f"int8 M={M} N={N} K={K} G={G} r={rank} dt={dt} gate={gate} path={p}")
        assert_parity(gpu_y(L, p), ref, f"int8 path={p}")


def test_int8_factors_split_fused_gemm():
    """The fully fused prefill GEMM with INT8 factors and K split into 2, 4
    and 8 slices."""
    from paper_2606_11244_amd import spear as sp
    L = S.make_layer(M=130, N=200, K=2048, group_size=128, rank=16, seed=5, ec_std=0.05,
                     ab_int8=True)
    ref = O.w4ec_linear(L)
    try:
        for slices in (1, 2, 4, 8):
            sp.set_gemm_slices(slices)
            log(f"int8 fused gemm slices={slices}")
            assert_parity(gpu_y(L, PATHS["fused_mfma"]), ref, f"int8 slices={slices}")
    finally:
        sp.set_gemm_slices(0)


@pytest.mark.parametrize("tile", [128, 256])
@pytest.mark.parametrize("M,N,K,dt,G", [(300, 200, 1024, S.F16, 128), (513, 384, 2048, S.BF16, 0),
                                         (257, 136, 512, S.F16, 128)])
def test_gemm_token_tiles(tile, M, N, K, dt, G):
    """The prefill GEMM with 128-token (four waves) and 256-token (eight
    waves) tiles, whole and split over K, on ragged token and row counts:
    the 4-bit product, the semi-fused EC path and the chain meet the bar."""
    from paper_2606_11244_amd import spear as sp
    L = S.make_layer(M=M, N=N, K=K, group_size=G, rank=16, act_dtype=dt, seed=M + tile,
                     ec_std=0.05)
    ref, ref4 = O.w4ec_linear(L), O.w4_linear_layer(L)
    sp.set_gemm_tile(tile)
    try:
        for slices in (1, 2, 4):
            sp.set_gemm_slices(slices)
            log(f"gemm tile={tile} slices={slices} M={M} N={N} K={K} dt={dt}")
            assert_parity(gpu_y(L, 0, with_ec=False), ref4, f"tile={tile} S={slices} w4")
            for p in (PATHS["2k"], PATHS["chain"]):
                assert_parity(gpu_y(L, p), ref, f"tile={tile} S={slices} path={p}")
    finally:
        sp.set_gemm_slices(0)
        sp.set_gemm_tile(0)


@pytest.mark.parametrize("roles", [1, 2, 3])
@pytest.mark.parametrize("M,N,K,dt,G,rank", [
    (300, 200, 1024, S.F16, 128, 16), (513, 520, 2048, S.BF16, 0, 64), (257, 136, 512, S.F16, 128, 12),
    (256, 256, 1024, S.BF16, 128, 32), (600, 1000, 1536, S.F16, 0, 24), (1, 128, 256, S.F16, 128, 8)])
def test_gemm_wave_roles(roles, M, N, K, dt, G, rank):
    """The 256-token GEMM with every wave loading and multiplying (k_gemm)
    and with four loading and four multiplying waves (k_gemm_ws), on ragged
    token and row counts and ranks that are and are not multiples of eight:
    the 4-bit product, the semi-fused EC path and the chain meet the bar."""
    from paper_2606_11244_amd import spear as sp
    L = S.make_layer(M=M, N=N, K=K, group_size=G, rank=rank, act_dtype=dt, seed=M + N,
                     ec_std=0.05)
    ref, ref4 = O.w4ec_linear(L), O.w4_linear_layer(L)
    sp.set_gemm_tile(256)
    sp.set_gemm_slices(1)
    sp.set_gemm_roles(roles)
    try:
        log(f"gemm roles={roles} M={M} N={N} K={K} dt={dt} G={G} r={rank}")
        assert_parity(gpu_y(L, 0 if M > 64 else PATHS["2k"], with_ec=False), ref4, f"roles={roles} w4")
        for p in (PATHS["2k"], PATHS["chain"]):
            assert_parity(gpu_y(L, p), ref, f"roles={roles} path={p}")
    finally:
        sp.set_gemm_roles(0)
        sp.set_gemm_slices(0)
        sp.set_gemm_tile(0)


# ---------------------------------------------------------------------------
# post-EC tail: residual addition + next-layer RMSNorm
# ---------------------------------------------------------------------------

def _tail_check(L, path, with_ec=True, in_place=False, tile=0):
    from paper_2606_11244_amd import spear as sp
    t = S.make_tail(L, seed=3)
    dt = sp._TORCH_DT[L.act_dtype]
    res = torch.from_numpy(t["residual"].view(np.int16)).view(dt).cuda()
    nw = torch.from_numpy(t["norm_w"].view(np.int16)).view(dt).cuda()
    dl = sp.DeviceLayer(L)
    prob = dl.problem(force_path=path)
    y_norm = torch.empty_like(dl.y)
    if in_place:
        dl.y.copy_(res)
        res = dl.y
    sp.set_gemm_tile(tile)  # before sizing the workspace: the plan depends on it
    try:
        ws = sp.allocate_workspace(prob, with_ec)
        dl.run_tail(prob, ws, residual=res, norm_w=nw, eps=t["eps"], y_norm=y_norm,
                    with_ec=with_ec)
    finally:
        sp.set_gemm_tile(0)
    torch.cuda.synchronize()
    y_ref = O.w4ec_linear(L) if with_ec else O.w4_linear_layer(L)
    h_ref, n_ref = O.post_ec_tail(y_ref, S.from_bits(t["residual"], L.act_dtype),
                                  S.from_bits(t["norm_w"], L.act_dtype), t["eps"])
    assert_parity(dl.y.float().cpu().numpy().astype(np.float64), h_ref, f"tail h path={path}")
    assert_parity(y_norm.float().cpu().numpy().astype(np.float64), n_ref, f"tail norm path={path}")


@pytest.mark.parametrize("M,N,K,G,dt,rank", [
    (1, 520, 1024, 128, S.F16, 16), (4, 256, 2048, 0, S.BF16, 8), (17, 300, 1024, 128, S.F16, 16),
    (3, 256, 1024, 128, S.F16, 32), (65, 200, 1024, 128, S.F16, 16), (300, 520, 2048, 0, S.BF16, 16),
])
def test_post_ec_tail_all_paths(M, N, K, G, dt, rank):
    """The residual is added in every path's final store and the RMSNorm
    follows in the same call: both outputs meet the bar against the oracle's
    float64 tail on the exact layer output; also for the 4-bit layer alone."""
    L = S.make_layer(M=M, N=N, K=K, group_size=G, rank=rank, act_dtype=dt, seed=M + N,
                     ec_std=0.05)
    for p in _paths_for(M, L):
        log(f"tail M={M} N={N} K={K} dt={dt} r={rank} path={p}")
        _tail_check(L, p)
    _tail_check(L, 0, with_ec=False)


@pytest.mark.parametrize("tile", [128, 256])
def test_post_ec_tail_in_place_and_tiles(tile):
    """An in-place residual stream (the residual is y itself) on the prefill
    GEMM with either token tile, and on decode."""
    L = S.make_layer(M=300, N=256, K=1024, group_size=128, rank=16, seed=9, ec_std=0.05)
    _tail_check(L, 4, in_place=True, tile=tile)
    _tail_check(L, 0, with_ec=False, in_place=True, tile=tile)
    Ld = S.make_layer(M=2, N=256, K=1024, group_size=128, rank=16, seed=10, ec_std=0.05)
    _tail_check(Ld, 0, in_place=True)


@pytest.mark.parametrize("M,path,int8,tail", [(1, 5, True, False), (4, 1, True, True),
                                              (200, 2, True, False), (300, 4, False, True),
                                              (2, 5, False, True)])
def test_graph_replay_int8_and_tail(M, path, int8, tail):
    """Graph replays of the INT8-factor paths and of the tail call: every
    replay, with new activations written by eager work between replays,
    equals the eager call bit for bit (the tail's residual is its own
    buffer here, rewritten with the activations)."""
    from paper_2606_11244_amd import spear as sp
    L = S.make_layer(M=M, N=1024, K=2048, group_size=128, rank=16, seed=M + path + 50,
                     ab_int8=int8)
    dl = sp.DeviceLayer(L)
    prob = dl.problem(force_path=path)
    ws = sp.allocate_workspace(prob)
    res = torch.randn(dl.y.shape, device="cuda").to(dl.y.dtype)
    nw = torch.ones((L.N,), device="cuda").to(dl.y.dtype)
    yn = torch.empty_like(dl.y)
    yn_eager = torch.empty_like(dl.y)
    y_eager = torch.empty_like(dl.y)

    def call(y, y_norm, stream=None):
        if tail:
            dl.run_tail(prob, ws, residual=res, norm_w=nw, eps=1e-5, y_norm=y_norm, y=y,
                        stream=stream)
        else:
            dl.run_ec(prob, ws, y=y, stream=stream)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        call(dl.y, yn, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(dl.y, yn)
    gen = torch.Generator(device="cuda").manual_seed(M + 1)
    for i in range(4):
        dl.x.copy_(torch.randn(dl.x.shape, generator=gen, device="cuda").to(dl.x.dtype))
        res.copy_(torch.randn(res.shape, generator=gen, device="cuda").to(res.dtype))
        torch.cuda.synchronize()
        log(f"graph int8={int8} tail={tail} M={M} path={path} replay={i}")
        g.replay()
        torch.cuda.synchronize()
        y_graph, yn_graph = dl.y.clone(), yn.clone()
        call(y_eager, yn_eager)
        torch.cuda.synchronize()
        assert torch.equal(y_graph, y_eager), f"replay {i}"
        if tail:
            assert torch.equal(yn_graph, yn_eager), f"replay {i} norm"


@pytest.mark.parametrize("path", [5, 1, 2, 4])
def test_int8_deterministic(path):
    """INT8-factor calls are bit-identical from call to call."""
    from paper_2606_11244_amd import spear as sp
    M = 130 if path in (2, 4) else 3
    L = S.make_layer(M=M, N=1024, K=8192, group_size=128, rank=16, seed=61, ab_int8=True)
    dl = sp.DeviceLayer(L)
    ws = sp.allocate_workspace(dl.problem(force_path=path))
    first = gpu_y(L, path, workspace=ws, dev=dl)
    for _ in range(3):
        assert np.array_equal(first, gpu_y(L, path, workspace=ws, dev=dl))
    assert_parity(first, O.w4ec_linear(L), f"int8 determinism {path}")


@pytest.mark.parametrize("stages", [4])
@pytest.mark.parametrize("M,N,K,wb", [(1, 1024, 8192, 4), (16, 768, 2048, 4), (3, 512, 28672, 4),
                                      (1, 300, 256, 4), (5, 640, 8192, 3)])
def test_gemv_pipeline_depths(stages, M, N, K, wb):
    """The decode GEMV with 4 and 8 stages of codes in flight per wave (one
    token tile: the 4-bit product alone, the producer-fused and the
    semi-fused variants), including waves with fewer iterations than
    stages, against the oracle and bit-identical across repeats."""
    from paper_2606_11244_amd import spear as sp
    L = S.make_layer(M=M, N=N, K=K, group_size=128, rank=32, seed=stages + M, weight_bits=wb)
    ref, ref4 = O.w4ec_linear(L), O.w4_linear_layer(L)
    sp.set_gemv_stages(stages)
    try:
        for p in (PATHS["fused_gemv"], PATHS["2k"]):
            log(f"gemv stages={stages} M={M} N={N} K={K} wb={wb} path={p}")
            y = gpu_y(L, p)
            assert_parity(y, ref, f"stages={stages} path={p}")
            assert np.array_equal(y, gpu_y(L, p))
        log(f"gemv stages={stages} M={M} N={N} K={K} wb={wb} w4-only")
        assert_parity(gpu_y(L, 0, with_ec=False), ref4, f"stages={stages} w4-only")
    finally:
        sp.set_gemv_stages(0)
