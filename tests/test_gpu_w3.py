"""GPU parity of the 3-bit backbone (Appendix D.1, D.3: the same layer with
3-bit codes, packed 32 to three words): the bit-exact dequantisation, every
execution path on small layers, both prefill tiles split over K, grouped
calls and graph replays, and the 1B- and 8B-shaped layers at full size on
complete outputs (EC-only copies included)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import spear_oracle as O
from paper_2606_11244_amd import synth as S

from gpu_util import assert_parity, gpu_y, log, with_fields

pytestmark = pytest.mark.gpu

PATHS = {"auto": 0, "fused_gemv": 1, "fused_mfma": 2, "chain": 3, "2k": 4, "fused_local": 5}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield


@pytest.mark.parametrize("dt", [S.F16, S.BF16])
@pytest.mark.parametrize("G", [128, 0])
def test_w3_dequant_bit_exact(dt, G):
    """Every 3-bit code against every zero point, random fp16 scales with
    subnormal-producing ones, through the GEMM's dequantisation code."""
    from paper_2606_11244_amd import spear as sp
    rng = np.random.default_rng(17)
    N, K = 8 * 16, 256
    g = K if G == 0 else G
    q = np.tile(np.arange(8), (N, K // 8))
    z = np.repeat(np.arange(8), 16)[:, None].repeat(K // g, axis=1).astype(np.uint8)
    s = rng.choice([rng.uniform(1e-5, 1e-3), rng.uniform(1e-3, 2.0)], size=(N, K // g))
    s = np.where(rng.random((N, K // g)) < 0.2, 6e-8, s).astype(np.float16)
    qw = S.pack_int3(q)
    want = O.dequant_bits(qw, s.view(np.uint16), z, g, dt, bits=3)
    log(f"w3 dequant dt={dt} G={g}")
    out = torch.empty((N, K), dtype=torch.int16, device="cuda")
    sp.w4_dequant(sp.problem(0, N, K, G, dt, weight_bits=3),
                  torch.from_numpy(qw.view(np.int32)).cuda(),
                  torch.from_numpy(s.view(np.int16)).cuda(), torch.from_numpy(z).cuda(), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint16)
    assert np.array_equal(got, want), f"{(got != want).sum()} mismatching bits"


def _w3(**kw):
    return S.make_layer(weight_bits=3, **kw)


@pytest.mark.parametrize("path", list(PATHS))
@pytest.mark.parametrize("M,dt,G,rank", [(4, S.F16, 0, 8), (1, S.F16, 128, 16), (16, S.BF16, 0, 32),
                                         (33, S.F16, 128, 16), (200, S.BF16, 128, 16),
                                         (130, S.F16, 0, 64)])
def test_w3_paths(path, M, dt, G, rank):
    L = _w3(M=M, N=768, K=2048, group_size=G, rank=rank, act_dtype=dt, seed=M + rank)
    p = PATHS[path]
    if path == "fused_gemv" and M > 64:
        pytest.skip("the GEMV takes up to 64 tokens")
    if path == "fused_local" and (M > 32 or rank > 16):
        pytest.skip("local EC: M <= 32, rank <= 16")
    if path == "fused_mfma" and rank > 16:
        pytest.skip("fully fused GEMM: rank <= 16")
    log(f"w3 path={path} M={M} dt={dt} G={G} r={rank}")
    assert_parity(gpu_y(L, p), O.w4ec_linear(L), f"w3/{path}/M={M}")
    assert_parity(gpu_y(L, p, with_ec=False), O.w4_linear_layer(L), f"w3 w4-only/{path}/M={M}")


@pytest.mark.parametrize("roles", [2, 3])
@pytest.mark.parametrize("M,N,K,G", [(300, 384, 4096, 128), (513, 520, 2048, 0), (256, 256, 1024, 128)])
def test_w3_gemm_wave_roles(roles, M, N, K, G):
    """The prefill GEMM with loading and multiplying waves on 3-bit codes
    (256 x 128 and 256 x 256 tiles), ragged token and row counts: the 3-bit
    product and the semi-fused EC path meet the bar."""
    from paper_2606_11244_amd import spear as sp
    L = _w3(M=M, N=N, K=K, group_size=G, rank=24, seed=M + roles)
    sp.set_gemm_tile(256)
    sp.set_gemm_slices(1)
    sp.set_gemm_roles(roles)
    try:
        log(f"w3 gemm roles={roles} M={M} N={N} K={K} G={G}")
        assert_parity(gpu_y(L, 4, with_ec=False), O.w4_linear_layer(L), f"w3 roles={roles} w3-only")
        assert_parity(gpu_y(L, 4), O.w4ec_linear(L), f"w3 roles={roles} 2k")
    finally:
        sp.set_gemm_roles(0)
        sp.set_gemm_slices(0)
        sp.set_gemm_tile(0)


@pytest.mark.parametrize("tile", [128, 256])
@pytest.mark.parametrize("slices", [1, 2, 8])
def test_w3_gemm_tiles_split_k(tile, slices):
    from paper_2606_11244_amd import spear as sp
    L = _w3(M=300, N=384, K=4096, group_size=128, rank=16, seed=5)
    sp.set_gemm_tile(tile)
    sp.set_gemm_slices(slices)
    sp.set_gemm_roles(1)  # every wave loads and multiplies (k_gemm)
    try:
        for p in ((0, 4) if tile == 128 else (4,)):  # the 256-token tile: not fully fused
            log(f"w3 gemm tile={tile} slices={slices} path={p}")
            assert_parity(gpu_y(L, p), O.w4ec_linear(L), f"w3 tile={tile} S={slices} p={p}")
    finally:
        sp.set_gemm_roles(0)
        sp.set_gemm_tile(0)
        sp.set_gemm_slices(0)


def test_w3_grouped_call_and_graph():
    """q, k, v of the 1B shapes as one grouped launch, bit-identical to the
    single calls; then a captured call replayed with new inputs."""
    from paper_2606_11244_amd import spear as sp
    Ls = [S.config_layer(1, m, 1, seed=i, weight_bits=3) for i, m in enumerate(("q", "k", "v"))]
    Ls = [Ls[0]] + [with_fields(L, x=Ls[0].x) for L in Ls[1:]]
    dls = [sp.DeviceLayer(L) for L in Ls]
    for d in dls[1:]:
        d.x = dls[0].x
    members = [d.member(d.problem()) for d in dls]
    ws = torch.zeros(max(256, sp.group_workspace(members)), dtype=torch.uint8, device="cuda")
    log("w3 group")
    sp.w4ec_linear_group(members, ws)
    torch.cuda.synchronize()
    for L, d in zip(Ls, dls):
        y_group = d.y.clone()
        d.run_ec(d.problem(), ws)
        torch.cuda.synchronize()
        assert torch.equal(y_group, d.y)
        assert_parity(d.y.float().cpu().numpy().astype(np.float64), O.w4ec_linear(L), "w3 group")
    # graph replays
    d = dls[0]
    prob = d.problem()
    y_eager = torch.empty_like(d.y)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        d.run_ec(prob, ws, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        d.run_ec(prob, ws)
    gen = torch.Generator(device="cuda").manual_seed(3)
    for i in range(3):
        d.x.copy_(torch.randn(d.x.shape, generator=gen, device="cuda").to(d.x.dtype))
        torch.cuda.synchronize()
        log(f"w3 graph replay {i}")
        g.replay()
        torch.cuda.synchronize()
        y_graph = d.y.clone()
        d.run_ec(prob, ws, y=y_eager)
        torch.cuda.synchronize()
        assert torch.equal(y_graph, y_eager)


def _ec_only(L):
    out = with_fields(L, scales=np.zeros_like(L.scales))
    wg = S.from_bits(L.w_g, L.act_dtype) * np.float32(20.0 / np.sqrt(L.K))
    out.w_g = S.to_bits(wg, L.act_dtype)
    return out


@pytest.mark.parametrize("module", S.MODULES)
@pytest.mark.parametrize("cid,Ms", [(1, (1, 4, 16)), (2, (512, 2048)), (3, (1, 128, 512))])
def test_w3_full_size(cid, module, Ms):
    """Full-size 3-bit layers (1B decode and prefill, 8B bf16 per channel),
    automatic dispatch: every output row, all tokens up to 16, one token of
    every 16-token tile beyond."""
    base = S.config_layer(cid, module, max(Ms), seed=0, weight_bits=3)
    for ec_only in (False, True):
        B = _ec_only(base) if ec_only else base
        for M in Ms:
            L = with_fields(B, x=np.ascontiguousarray(B.x[:M]), M=M)
            idx = np.arange(M) if M <= 16 else np.minimum(16 * np.arange((M + 15) // 16) + 5, M - 1)
            ref = O.w4ec_linear(with_fields(L, x=np.ascontiguousarray(L.x[idx]), M=len(idx)))
            log(f"w3 full-size cid={cid} {module} M={M} ec_only={ec_only}")
            y = gpu_y(L, 0)
            assert np.all(np.isfinite(y))
            assert_parity(y[idx], ref, f"w3 full/{cid}/{module}/M={M}/ec_only={ec_only}")
