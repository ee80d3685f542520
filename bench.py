"""Benchmark of the W4+EC linear layer on one MI355X.

One step = one pass of the hot path over one batch of synthetic input on a
Llama-3.2-1B-shaped model (hidden 2048, MLP 8192; q, k, v, o, gate, up, down
per layer; group-128 4-bit weights, EC rank 16 with the sigmoid-linear gate,
fp16 activations):

  decode   M = 1: all 16 layers x 7 modules through the automatic dispatch
           (the fused single-kernel path), the modules that read one hidden
           state launched together (per layer: q, k, v in one grouped call;
           o; gate, up in one grouped call; down). Two distinct copies of the
           model weights alternate between steps (2 x 0.53 GB), so the
           weights come from HBM rather than the 256 MB Infinity Cache. The
           same pass with one call per module is reported beside it.
  prefill  M = 4096 tokens (1% of input channels scaled x20): the 7 modules of
           one layer through the automatic dispatch (EC pre-kernel + 4-bit
           GEMM with the EC in its epilogue).

Both passes are captured once as HIP graphs and replayed. The printed JSON
line reports decode HBM throughput (algorithmic bytes / time) as `value`, the
prefill MFMA throughput under `prefill`, each with its roofline, the EC
overhead over the same passes without EC, and the CPU oracle timed on a
bounded sample (`cpu_baseline`).

Context line `decode_70b_layer`: one Llama-2-70B-shaped layer (7 modules,
K/N up to 28672, EC rank 64 on every module) at M = 1, fused path, two weight
copies alternating. Its weights are uniform random codes, scales and zero
points drawn on the device (timing only: the kernels' work does not depend on
the values), so that the 0.93 GB do not have to be generated on the host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "W4+EC linear TFLOP/s & HBM GB/s (% roofline) decode M=1 + prefill M=4096"
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
MFMA_F16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16/bf16 MFMA
LAYERS_1B = 16
RANK = 16
GROUP = 128
# per decoder layer, the modules that read one hidden state (q, k, v; gate,
# up) go out as one grouped call; o and down alone
DEC_GROUPS = ((0, 1, 2), (3,), (4, 5), (6,))


def algo_bytes(M, N, K, G, r, ab_int8=False):
    """Algorithmic HBM bytes of one W4+EC call: codes (N K / 2), scales and
    4-bit zeros (2.5 N K / G), A, B, w_g, X and Y in fp16 (A and B as int8
    codes plus fp32 per-channel scales with ab_int8)."""
    ab = (r * K + N * r + 4 * (r + N)) if ab_int8 else (2 * r * K + 2 * N * r)
    return N * K / 2 + 2.5 * N * K / G + (ab if r else 0) + (2 * K if r else 0) + 2 * M * K + 2 * M * N


def algo_flops(M, N, K, r):
    return 2 * M * N * K + (2 * M * K * (r + 1) + 2 * M * N * r if r else 0)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("spear_kernels.hip", "spear_api.cpp", "spear_internal.h"):
        with open(os.path.join(ROOT, "paper_2606_11244_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def stored_traffic():
    """HBM traffic per launch measured with rocprofv3 counters for the current
    kernel sources, if such a measurement is stored under profiles/."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    if d.get("kernel_source_hash") != kernel_source_hash():
        return None
    return d


def cpu_baseline(dec_layers, pre_layer, budget_s=12.0):
    """The float64 oracle on the host cores: the 7 decode modules of one layer
    (repeated), and one prefill module (q, M=4096)."""
    import numpy as np
    from oracle import spear_oracle as O
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        blas = 1
    reps, t_dec, nbytes = 0, 0.0, 0.0
    t0 = time.perf_counter()
    while reps < 1 or (time.perf_counter() - t0 < budget_s * 0.6 and reps < 8):
        for L in dec_layers:
            ts = time.perf_counter()
            y = O.w4ec_linear(L)
            t_dec += time.perf_counter() - ts
            nbytes += algo_bytes(L.M, L.N, L.K, L.group_size, L.rank)
            assert np.isfinite(y).all()
        reps += 1
    ts = time.perf_counter()
    O.w4ec_linear(pre_layer)
    t_pre = time.perf_counter() - ts
    # single-threaded: the tiny workload and the 1B q module at M = 1
    single = None
    try:
        from threadpoolctl import threadpool_limits
        from paper_2606_11244_amd import synth as S
        tiny = S.config_layer(0, "tiny", 4, seed=0)
        with threadpool_limits(limits=1):
            out = {}
            for name, LL, n in (("tiny", tiny, 20), ("1b_q_m1", dec_layers[0], 2)):
                ts = time.perf_counter()
                for _ in range(n):
                    O.w4ec_linear(LL)
                dt = (time.perf_counter() - ts) / n
                out[name] = {"ms_per_call": round(dt * 1e3, 3),
                             "GBps": round(algo_bytes(LL.M, LL.N, LL.K, LL.group_size, LL.rank)
                                           / dt / 1e9, 4)}
        single = out
    except Exception as exc:  # noqa: BLE001
        single = {"error": str(exc)[:80]}
    L = pre_layer
    return {
        "value": round(nbytes / t_dec / 1e9, 4), "unit": "GB/s", "cores": int(blas),
        "kind": "oracle",
        "sample": (f"float64 numpy oracle: one 1B-shaped layer (7 modules, M=1) x {reps} "
                   f"({nbytes / 1e6:.0f} MB algorithmic, {t_dec:.1f} s); prefill q module "
                   f"M={L.M} ({t_pre:.1f} s)"),
        "prefill_tflops": round(algo_flops(L.M, L.N, L.K, L.rank) / t_pre / 1e12, 5),
        "host_cpus": os.cpu_count(),
        "single_thread": single,
    }


def decode_70b_context(sp, torch, steps, warmup, dev):
    """M = 1 decode of one 70B-shaped layer (fused W4+EC and W4-only)."""
    from paper_2606_11244_amd import synth as S
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    r, G = 64, 128
    mods = []
    for c in range(2):
        for m in S.MODULES:
            K, N = S.LLAMA_70B[m]
            q = torch.randint(-2**31, 2**31 - 1, (N, K // 8), dtype=torch.int32, device=dev, generator=g)
            sc = (torch.rand((N, K // G), device=dev, generator=g) * 1e-3 + 1e-4).half().view(torch.int16)
            zr = torch.randint(0, 16, (N, K // G), dtype=torch.uint8, device=dev, generator=g)
            x = torch.randn((1, K), device=dev, generator=g).half()
            A = (torch.randn((r, K), device=dev, generator=g) * 0.01).half()
            B = (torch.randn((N, r), device=dev, generator=g) * 0.01).half()
            wg = (torch.randn((K,), device=dev, generator=g) * 0.05).half()
            y = torch.empty((1, N), dtype=torch.float16, device=dev)
            pr = sp.problem(1, N, K, G, sp.F16, r, sp.GATE_SIGMOID_LINEAR)
            mods.append((c, pr, q, sc, zr, x, A, B, wg, y, K, N))
    ws = torch.zeros(max(max(sp.dispatch_plan(m[1]).workspace_bytes for m in mods), 256),
                     dtype=torch.uint8, device=dev)
    ws4 = torch.zeros(max(max(sp.dispatch_plan(m[1], with_ec=False).workspace_bytes for m in mods), 256),
                      dtype=torch.uint8, device=dev)

    def run(c, ec):
        for (cc, pr, q, sc, zr, x, A, B, wg, y, K, N) in mods:
            if cc != c:
                continue
            if ec:
                sp.w4ec_linear(pr, x, q, sc, zr, A, B, y, w_g=wg, workspace=ws)
            else:
                sp.w4_linear(pr, x, q, sc, zr, y, workspace=ws4)

    def timed(ec):
        graphs = []
        for c in range(2):
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                run(c, ec)
            torch.cuda.current_stream().wait_stream(s)
            torch.cuda.synchronize()
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                run(c, ec)
            graphs.append(gr)
        for i in range(warmup):
            graphs[i % 2].replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(steps):
            graphs[i % 2].replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / steps

    t_ec, t_w4 = timed(True), timed(False)
    nb = sum(algo_bytes(1, N, K, G, r) for (c, pr, q, sc, zr, x, A, B, wg, y, K, N) in mods if c == 0)
    nb4 = sum(algo_bytes(1, N, K, G, 0) for (c, pr, q, sc, zr, x, A, B, wg, y, K, N) in mods if c == 0)
    return {"GBps": round(nb / t_ec / 1e9, 1), "frac": round(nb / t_ec / 1e9 / HBM_PEAK_GBS, 4),
            "us_per_layer": round(t_ec * 1e6, 2), "w4_only_GBps": round(nb4 / t_w4 / 1e9, 1),
            "w4_only_us_per_layer": round(t_w4 * 1e6, 2), "ec_overhead": round(t_ec / t_w4 - 1, 4),
            "rank": r, "path": "fused_gemv", "weights": "device-random (timing only)"}


def model_70b_pass(sp, torch, dev, Ms=(1, 16, 64, 512, 4096, 8192), reps=3):
    """The 70B-shaped model's linear layers as one pass per token count: all
    80 layers x 7 modules resident in HBM (device-random 4-bit weights,
    group 128, about 36 GB), the EC (rank 64, sigmoid-linear gate) on the
    seeded 25% of the (layer, module) pairs and the 4-bit product alone on
    the rest, every call on its AUTO path; the same pass with no EC at all
    gives the model's EC overhead. Each pass is one captured graph."""
    from paper_2606_11244_amd import model70b
    from paper_2606_11244_amd import synth as S
    r, G = model70b.RANK, model70b.GROUP
    layers, sel = model70b.build(dev)
    Kmax, Nmax, Mmax = max(k for k, _ in S.LLAMA_70B.values()), max(n for _, n in S.LLAMA_70B.values()), max(Ms)
    g = torch.Generator(device=dev)
    g.manual_seed(1)
    xbuf = torch.randn((Mmax * Kmax,), device=dev, generator=g).half()
    ybuf = torch.empty((Mmax * Nmax,), dtype=torch.float16, device=dev)
    out = {"weights": "device-random (timing only)",
           "ec": f"rank 64 on a seeded 25% of the (layer, module) pairs ({int(sel.sum())} of {sel.size})",
           "passes": []}
    for M in Ms:
        plans = {}
        ws_need = 256
        for m in S.MODULES:
            K, N = S.LLAMA_70B[m]
            pe = sp.problem(M, N, K, G, sp.F16, r, sp.GATE_SIGMOID_LINEAR)
            p4 = sp.problem(M, N, K, G, sp.F16, 0, sp.GATE_SIGMOID_LINEAR)
            plans[m] = (pe, p4)
            ws_need = max(ws_need, sp.dispatch_plan(pe).workspace_bytes,
                          sp.dispatch_plan(p4, with_ec=False).workspace_bytes)
        ws = torch.zeros(ws_need, dtype=torch.uint8, device=dev)

        def run(with_ec):
            for mods in layers:
                for (m, K, N, q, sc, zr, ec) in mods:
                    x = xbuf[:M * K].view(M, K)
                    y = ybuf[:M * N].view(M, N)
                    pe, p4 = plans[m]
                    if with_ec and ec is not None:
                        sp.w4ec_linear(pe, x, q, sc, zr, ec[0], ec[1], y, w_g=ec[2], workspace=ws)
                    else:
                        sp.w4_linear(p4, x, q, sc, zr, y, workspace=ws)

        def timed(with_ec):
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                run(with_ec)
            torch.cuda.current_stream().wait_stream(s)
            torch.cuda.synchronize()
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                run(with_ec)
            gr.replay()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                gr.replay()
            e1.record()
            torch.cuda.synchronize()
            del gr
            return e0.elapsed_time(e1) * 1e-3 / reps

        t_ec, t_w4 = timed(True), timed(False)
        nbytes = sum(algo_bytes(M, N, K, G, r if ec is not None else 0)
                     for mods in layers for (m, K, N, q, sc, zr, ec) in mods)
        flops = sum(algo_flops(M, N, K, r if ec is not None else 0)
                    for mods in layers for (m, K, N, q, sc, zr, ec) in mods)
        out["passes"].append({
            "M": M, "ms_per_pass": round(t_ec * 1e3, 3), "w4_only_ms": round(t_w4 * 1e3, 3),
            "ec_overhead": round(t_ec / t_w4 - 1, 4), "GBps": round(nbytes / t_ec / 1e9, 1),
            "hbm_frac": round(nbytes / t_ec / 1e9 / HBM_PEAK_GBS, 4),
            "TFLOPs": round(flops / t_ec / 1e12, 1),
            "mfma_frac": round(flops / t_ec / 1e12 / MFMA_F16_PEAK_TFLOPS, 4)})
        print("bench: 70B model pass M=%d: %.3f ms (W4-only %.3f ms)" % (M, t_ec * 1e3, t_w4 * 1e3),
              file=sys.stderr, flush=True)
        del ws
    del layers, xbuf, ybuf
    torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--copies", type=int, default=2, help="decode weight copies rotated per step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-overhead", action="store_true", help="skip the W4-only reference passes")
    ap.add_argument("--no-70b", action="store_true", help="skip the 70B-layer context line")
    ap.add_argument("--no-int8", action="store_true",
                    help="skip the passes with INT8 per-channel EC factors")
    ap.add_argument("--no-ungrouped", action="store_true",
                    help="skip the decode pass with one call per module")
    ap.add_argument("--no-tail", action="store_true",
                    help="skip the passes with the post-EC tail on o and down")
    ap.add_argument("--model70b", action="store_true",
                    help="also time the 70B-shaped model's linear layers (80 layers resident, "
                         "about 36 GB) at M = 1 .. 8192")
    ap.add_argument("--copy-calib-mb", type=int, default=0,
                    help="also run one device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the W4+EC layer is built and timed on a single "
              "MI355X (multi-GPU runs are out of scope); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2606_11244_amd import spear as sp
    from paper_2606_11244_amd import synth as S

    torch.cuda.set_device(0)
    dev = "cuda:0"
    print("bench: generating layers", file=sys.stderr, flush=True)
    dec_base = [S.config_layer(1, m, 1, seed=0) for m in S.MODULES]
    pre_base = [S.config_layer(2, m, 4096, seed=0) for m in S.MODULES]

    # ---- decode: copies x layers x modules, each with its own weights in HBM
    dec_dev = []  # [copy][layer][module] DeviceLayer
    base_dev = [sp.DeviceLayer(L, device=dev) for L in dec_base]
    for c in range(args.copies):
        per_copy = []
        for _l in range(LAYERS_1B):
            mods = []
            for b in base_dev:
                d = sp.DeviceLayer.__new__(sp.DeviceLayer)
                d.__dict__.update(b.__dict__)
                d.qweight = b.qweight.clone()
                d.scales = b.scales.clone()
                d.zeros = b.zeros.clone()
                d.A, d.B, d.w_g = b.A.clone(), b.B.clone(), b.w_g.clone()
                mods.append(d)
            # q, k, v read one hidden state, gate and up another
            for grp in DEC_GROUPS:
                for j in grp[1:]:
                    mods[j].x = mods[grp[0]].x
            per_copy.append(mods)
        dec_dev.append(per_copy)
    dec_ws = max([sp.dispatch_plan(d.problem()).workspace_bytes for d in base_dev] +
                 [sp.group_workspace([base_dev[j].member(base_dev[j].problem(rank=r), with_ec=r != 0)
                                      for j in grp]) for grp in DEC_GROUPS for r in (None, 0)])
    dec_ws_t = torch.zeros(max(dec_ws, 256), dtype=torch.uint8, device=dev)
    pre_dev = [sp.DeviceLayer(L, device=dev) for L in pre_base]
    pre_ws = max(sp.dispatch_plan(d.problem()).workspace_bytes for d in pre_dev)
    pre_ws_t = torch.zeros(max(pre_ws, 256), dtype=torch.uint8, device=dev)
    w4_ws = max(sp.dispatch_plan(d.problem(), with_ec=False).workspace_bytes
                for d in base_dev + pre_dev)
    w4_ws_t = torch.zeros(max(w4_ws, 256), dtype=torch.uint8, device=dev)

    dec_bytes = LAYERS_1B * sum(algo_bytes(1, L.N, L.K, L.group_size, L.rank) for L in dec_base)
    dec_bytes_w4 = LAYERS_1B * sum(algo_bytes(1, L.N, L.K, L.group_size, 0) for L in dec_base)
    pre_flops = sum(algo_flops(L.M, L.N, L.K, L.rank) for L in pre_base)
    pre_flops_w4 = sum(algo_flops(L.M, L.N, L.K, 0) for L in pre_base)
    dec_plan = sp.dispatch_plan(base_dev[0].problem())

    def decode_pass(c, ec=True, grouped=True, devs=None):
        for mods in (dec_dev if devs is None else devs)[c]:
            for grp in (DEC_GROUPS if grouped else [(j,) for j in range(len(mods))]):
                if len(grp) > 1:
                    sp.w4ec_linear_group([mods[j].member(mods[j].problem(rank=None if ec else 0),
                                                         with_ec=ec) for j in grp], dec_ws_t)
                elif ec:
                    mods[grp[0]].run_ec(mods[grp[0]].problem(), dec_ws_t)
                else:
                    mods[grp[0]].run_w4(mods[grp[0]].problem(), w4_ws_t)

    def prefill_pass(ec=True):
        for d in pre_dev:
            if ec:
                d.run_ec(d.problem(), pre_ws_t)
            else:
                d.run_w4(d.problem(), w4_ws_t)

    def capture(fn):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            fn()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        torch.cuda.synchronize()
        return g

    print("bench: capturing graphs", file=sys.stderr, flush=True)
    g_dec = [capture(lambda c=c: decode_pass(c)) for c in range(args.copies)]
    g_pre = capture(prefill_pass)

    def run_steps(n, gdec, gpre, timed):
        ev = []
        for i in range(n):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e2 = torch.cuda.Event(enable_timing=True)
            e0.record()
            gdec[i % len(gdec)].replay()
            e1.record()
            gpre.replay()
            e2.record()
            ev.append((e0, e1, e2))
        return ev

    print("bench: warmup", file=sys.stderr, flush=True)
    run_steps(args.warmup, g_dec, g_pre, False)
    torch.cuda.synchronize()
    print("bench: timed steps", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    ev = run_steps(args.steps, g_dec, g_pre, True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    t_dec = np.array([a.elapsed_time(b) for a, b, _ in ev]) * 1e-3
    t_pre = np.array([b.elapsed_time(c) for _, b, c in ev]) * 1e-3
    dec_s = float(np.mean(t_dec))
    pre_s = float(np.mean(t_pre))
    dec_gbs = dec_bytes / dec_s / 1e9
    pre_tfl = pre_flops / pre_s / 1e12

    # the same decode pass with one call per module
    ungrouped = None
    if not args.no_ungrouped:
        print("bench: decode with one call per module", file=sys.stderr, flush=True)
        g_dec_u = [capture(lambda c=c: decode_pass(c, grouped=False)) for c in range(args.copies)]
        run_steps(args.warmup, g_dec_u, g_pre, False)
        evu = run_steps(args.steps, g_dec_u, g_pre, True)
        torch.cuda.synchronize()
        du = float(np.mean([a.elapsed_time(b) for a, b, _ in evu])) * 1e-3
        del g_dec_u
        ungrouped = {"ms_per_pass": round(du * 1e3, 4), "GBps": round(dec_bytes / du / 1e9, 2),
                     "launches": LAYERS_1B * len(S.MODULES)}

    overhead = None
    if not args.no_overhead:
        print("bench: W4-only reference passes", file=sys.stderr, flush=True)
        g_dec_w4 = [capture(lambda c=c: decode_pass(c, ec=False)) for c in range(args.copies)]
        g_pre_w4 = capture(lambda: prefill_pass(ec=False))
        run_steps(args.warmup, g_dec_w4, g_pre_w4, False)
        ev4 = run_steps(args.steps, g_dec_w4, g_pre_w4, True)
        torch.cuda.synchronize()
        d4 = float(np.mean([a.elapsed_time(b) for a, b, _ in ev4])) * 1e-3
        p4 = float(np.mean([b.elapsed_time(c) for _, b, c in ev4])) * 1e-3
        overhead = {
            "decode": round(dec_s / d4 - 1.0, 4), "prefill": round(pre_s / p4 - 1.0, 4),
            "decode_w4_only_GBps": round(dec_bytes_w4 / d4 / 1e9, 1),
            "prefill_w4_only_TFLOPs": round(pre_flops_w4 / p4 / 1e12, 1),
            "decode_ec_byte_share": round(dec_bytes / dec_bytes_w4 - 1.0, 4),
        }

    # ---- the same passes with the EC factors in INT8 (per-channel symmetric,
    # fp32 scales): same 4-bit weights, activations and gate; A and B swapped
    int8 = None
    if not args.no_int8:
        print("bench: INT8-factor passes", file=sys.stderr, flush=True)
        dec_i8 = [sp.DeviceLayer(S.config_layer(1, m, 1, seed=0, ab_int8=True), device=dev)
                  for m in S.MODULES]
        pre_i8 = [sp.DeviceLayer(S.config_layer(2, m, 4096, seed=0, ab_int8=True), device=dev)
                  for m in S.MODULES]

        def swap(d, src):
            e = sp.DeviceLayer.__new__(sp.DeviceLayer)
            e.__dict__.update(d.__dict__)
            e.layer, e.ab_int8 = src.layer, True
            e.A, e.B = src.A.clone(), src.B.clone()
            e.a_scale, e.b_scale = src.a_scale.clone(), src.b_scale.clone()
            return e

        dec_dev_i8 = [[[swap(d, dec_i8[j]) for j, d in enumerate(mods)] for mods in per_copy]
                      for per_copy in dec_dev]
        pre_dev_i8 = [swap(d, pre_i8[j]) for j, d in enumerate(pre_dev)]

        for per_copy in dec_dev_i8:
            for mods in per_copy:
                for grp in DEC_GROUPS:
                    for j in grp[1:]:
                        mods[j].x = mods[grp[0]].x

        def decode_pass_i8(c):
            decode_pass(c, devs=dec_dev_i8)

        def prefill_pass_i8():
            for d in pre_dev_i8:
                d.run_ec(d.problem(), pre_ws_t)

        g_dec_i8 = [capture(lambda c=c: decode_pass_i8(c)) for c in range(args.copies)]
        g_pre_i8 = capture(prefill_pass_i8)
        run_steps(args.warmup, g_dec_i8, g_pre_i8, False)
        ev8 = run_steps(args.steps, g_dec_i8, g_pre_i8, True)
        torch.cuda.synchronize()
        d8 = float(np.mean([a.elapsed_time(b) for a, b, _ in ev8])) * 1e-3
        p8 = float(np.mean([b.elapsed_time(c) for _, b, c in ev8])) * 1e-3
        dec_bytes_i8 = LAYERS_1B * sum(algo_bytes(1, L.N, L.K, L.group_size, L.rank, True)
                                       for L in dec_base)
        int8 = {
            "format": "A, B int8 per-channel symmetric, fp32 scales; gate fp16",
            "decode_ms_per_pass": round(d8 * 1e3, 4),
            "decode_GBps": round(dec_bytes_i8 / d8 / 1e9, 2),
            "prefill_ms_per_pass": round(p8 * 1e3, 4),
            "prefill_TFLOPs": round(pre_flops / p8 / 1e12, 2),
        }
        if overhead is not None:
            int8["decode_overhead"] = round(d8 / d4 - 1.0, 4)
            int8["prefill_overhead"] = round(p8 / p4 - 1.0, 4)
            int8["decode_ec_byte_share"] = round(dec_bytes_i8 / dec_bytes_w4 - 1.0, 4)

    # ---- the same EC passes with the post-EC tail where a decoder layer has
    # it: after o and down, the residual added in place and the next
    # RMSNorm (the other modules unchanged)
    tail = None
    if not args.no_tail:
        print("bench: post-EC tail passes", file=sys.stderr, flush=True)
        hid = torch.randn((4096 * 2048,), device=dev).half()
        nrm_w = torch.ones((2048,), device=dev).half()
        nrm_out = torch.empty((4096 * 2048,), dtype=torch.float16, device=dev)
        tail_mods = {"o", "down"}

        def call(d, ws_t, M):
            if d.layer_name in tail_mods:
                res = hid[:M * d.N].view(M, d.N)
                d.run_tail(d.problem(), ws_t, residual=res, norm_w=nrm_w, eps=1e-5,
                           y_norm=nrm_out[:M * d.N].view(M, d.N), y=res)
            else:
                d.run_ec(d.problem(), ws_t)

        for c in range(args.copies):
            for mods in dec_dev[c]:
                for j, d in enumerate(mods):
                    d.layer_name = S.MODULES[j]
        for j, d in enumerate(pre_dev):
            d.layer_name = S.MODULES[j]
        def decode_tail(c):
            # the grouped calls as in the decode pass, o and down with the tail
            for mods in dec_dev[c]:
                for grp in DEC_GROUPS:
                    if len(grp) > 1:
                        sp.w4ec_linear_group([mods[j].member(mods[j].problem()) for j in grp],
                                             dec_ws_t)
                    else:
                        call(mods[grp[0]], dec_ws_t, 1)

        g_dec_t = [capture(lambda c=c: decode_tail(c)) for c in range(args.copies)]
        g_pre_t = capture(lambda: [call(d, pre_ws_t, 4096) for d in pre_dev])
        run_steps(args.warmup, g_dec_t, g_pre_t, False)
        evt = run_steps(args.steps, g_dec_t, g_pre_t, True)
        torch.cuda.synchronize()
        dt_ = float(np.mean([a.elapsed_time(b) for a, b, _ in evt])) * 1e-3
        pt_ = float(np.mean([b.elapsed_time(c) for _, b, c in evt])) * 1e-3
        tail = {"modules": "o, down (residual in place + RMSNorm of the 2048-wide hidden state)",
                "decode_ms_per_pass": round(dt_ * 1e3, 4), "prefill_ms_per_pass": round(pt_ * 1e3, 4),
                "decode_added": round(dt_ / dec_s - 1.0, 4), "prefill_added": round(pt_ / pre_s - 1.0, 4)}

    model70 = None
    if args.model70b:
        print("bench: 70B-shaped model pass", file=sys.stderr, flush=True)
        model70 = model_70b_pass(sp, torch, dev)

    ctx70 = None
    if not args.no_70b:
        print("bench: 70B-layer decode context", file=sys.stderr, flush=True)
        ctx70 = decode_70b_context(sp, torch, args.steps, args.warmup, dev)

    if args.copy_calib_mb:
        # counter calibration: one elementwise kernel that reads and writes
        # exactly copy_calib_mb MiB each (fp32 negation)
        n = (args.copy_calib_mb << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        torch.neg(a, out=b)
        torch.cuda.synchronize()

    traffic = stored_traffic()
    n_launch_dec = LAYERS_1B * len(DEC_GROUPS)
    result = {
        "metric": METRIC,
        "value": round(dec_gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": ("llama-3.2-1b-shaped W4+EC linear layers (q,k,v,o 2048->2048/512, "
                         "gate/up 2048->8192, down 8192->2048): decode M=1 over 16 layers x 7 "
                         "modules + prefill M=4096 over 7 modules"),
            "group_size": GROUP, "rank": RANK, "gate": "sigmoid_linear",
            "decode_path": sp.PATH_NAMES[dec_plan.path],
            "prefill_paths": {m: sp.PATH_NAMES[sp.dispatch_plan(d.problem()).path]
                              for m, d in zip(S.MODULES, pre_dev)},
            "decode_weight_copies": args.copies,
            "decode_launches": ("per layer: q,k,v grouped (one launch), o, gate,up grouped "
                                "(one launch), down: %d per pass" % n_launch_dec),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": ("k_gemv_group / k_gemv (one-kernel W4+EC decode GEMV, %s), all "
                       "launches of the decode pass" % sp.PATH_NAMES[dec_plan.path]),
            "achieved": round(dec_bytes / n_launch_dec / (dec_s / n_launch_dec) / 1e9, 2),
            "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(dec_gbs / HBM_PEAK_GBS, 4),
            "traffic": (traffic or {}).get("decode_bytes_per_launch"),
            "algo_bytes_per_launch": round(dec_bytes / n_launch_dec),
            "avg_launch_us": round(dec_s / n_launch_dec * 1e6, 3),
        },
        "prefill": {
            "value": round(pre_tfl, 2), "unit": "TFLOP/s", "ms_per_pass": round(pre_s * 1e3, 4),
            "roofline": {
                "bound": "mfma",
                "kernel": ("the 7 modules on their AUTO paths: k_ec pre-kernel + k_gemm with "
                           "the EC epilogue (unfused_2k), or the fully fused k_gemm (fused_mfma)"),
                "achieved": round(pre_tfl, 2), "peak": MFMA_F16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(pre_tfl / MFMA_F16_PEAK_TFLOPS, 4),
                "traffic": (traffic or {}).get("prefill_bytes_per_launch"),
            },
        },
        "decode_ms_per_pass": round(dec_s * 1e3, 4),
        "decode_one_call_per_module": ungrouped,
        "decode_70b_layer": ctx70,
        "model_70b": model70,
        "ec_overhead": overhead,
        "ec_int8": int8,
        "post_ec_tail": tail,
    }
    if not args.no_cpu_baseline:
        print("bench: CPU oracle baseline", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(dec_base, pre_base[0])
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
