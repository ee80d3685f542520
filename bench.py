"""Benchmark of the W4+EC linear layer on one MI355X.

One step = one pass of the hot path over one batch of synthetic input on the
Llama-2-70B-shaped model that fits one GPU: all 80 layers x 7 linear modules
(q/o 8192->8192, k/v 8192->1024, gate/up 8192->28672, down 28672->8192) of
group-128 4-bit weights resident in HBM (about 36 GB of device-random codes,
scales and zero points), the EC (rank 64, sigmoid-linear gate, fp16) on the
seeded 25% of the (layer, module) pairs and the 4-bit product alone on the
rest, every call on its automatic-dispatch path, the modules of a block that
read one hidden state (q, k, v; gate, up) as grouped calls (members that take
one GEMV variant share a launch; the others run on their own):

  decode   M = 1: every module once;
  prefill  M = 4096 tokens: every module once.

Each pass is captured once as a HIP graph and replayed. The printed JSON line
reports the decode pass's HBM throughput (algorithmic bytes / time) as
`value` with its roofline, the prefill pass's MFMA throughput under
`prefill`, the model's EC overhead over the same passes with no EC, the
decode pass under the paper's timing protocol (200 warm-up and 500 timed
replays, median), and the CPU oracle timed on a bounded sample
(`cpu_baseline`).

Extra fields on the Llama-3.2-1B-shaped layers (`llama1b`): the decode pass
over 16 layers x 7 modules at M = 1 (grouped calls, two weight copies
alternating so that the weights come from HBM), the 7 modules at M = 4096,
their EC overhead, the same passes with INT8 EC factors and with the post-EC
tail.
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
DEC_M, PRE_M = 1, 4096  # the metric's decode and prefill token counts
# per decoder layer, the modules that read one hidden state (q, k, v; gate,
# up) go out as one grouped call; o and down alone
DEC_GROUPS = ((0, 1, 2), (3,), (4, 5), (6,))


# the 70B-shaped model's decode and prefill passes call the modules of a
# block that read one hidden state (q, k, v; gate, up) as grouped calls: the
# members of one GEMV variant share a launch, the others run on their own
GROUPS_70B = (("q", "k", "v"), ("o",), ("gate", "up"), ("down",))


def algo_bytes(M, N, K, G, r, ab_int8=False, wbits=4):
    """Algorithmic HBM bytes of one W4+EC call: codes (N K / 2; 3N K / 8 for
    3-bit codes), scales and 4-bit zeros (2.5 N K / G), A, B, w_g, X and Y in
    fp16 (A and B as int8 codes plus fp32 per-channel scales with ab_int8)."""
    ab = (r * K + N * r + 4 * (r + N)) if ab_int8 else (2 * r * K + 2 * N * r)
    return (N * K * wbits / 8 + 2.5 * N * K / G + (ab if r else 0) + (2 * K if r else 0)
            + 2 * M * K + 2 * M * N)


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


def cpu_baseline(sel, budget_s=20.0):
    """The float64 oracle on the host cores, on a bounded sample of the
    70B-shaped model's decode pass: for each of the 7 module shapes, with the
    EC (rank 64) and without, the oracle evaluates a seeded layer of full K
    restricted to 128 and to 256 output rows at M = 1 (median of three runs
    each); the time of a full-width module is the line through those two
    points at its N, and the pass is the sum over the 80 layers' modules with
    the model's EC selection. The prefill rate comes from the 70B q shape at
    M = 4096 on 256 output rows (time scaled to the full rows)."""
    import numpy as np
    from oracle import spear_oracle as O
    from paper_2606_11244_amd import synth as S
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        blas = 1
    t_start = time.perf_counter()

    def timed(L, reps=3):
        ts = []
        for _ in range(reps):
            t0 = time.perf_counter()
            y = O.w4ec_linear(L)
            ts.append(time.perf_counter() - t0)
            assert np.isfinite(y).all()
        return float(np.median(ts))

    per_module = {}
    for j, m in enumerate(S.MODULES):
        K, N = S.LLAMA_70B[m]
        for r in (0, 64):
            t = {}
            for ns in (512, 1024):
                L = S.make_layer(M=DEC_M, N=ns, K=K, group_size=GROUP, rank=r, seed=0,
                                 config_id=4, module_id=j)
                t[ns] = timed(L)
            slope = max(0.0, (t[1024] - t[512]) / 512.0)
            per_module[(m, r)] = t[512] + slope * (N - 512)
    t_pass, nbytes = 0.0, 0.0
    for l in range(sel.shape[0]):
        for j, m in enumerate(S.MODULES):
            K, N = S.LLAMA_70B[m]
            r = 64 if sel[l, j] else 0
            t_pass += per_module[(m, r)]
            nbytes += algo_bytes(DEC_M, N, K, GROUP, r)
    K, N = S.LLAMA_70B["q"]
    Lp = S.make_layer(M=PRE_M, N=256, K=K, group_size=GROUP, rank=64, seed=0, config_id=4,
                      module_id=0)
    t_pre = timed(Lp, reps=1) * N / 256.0
    return {
        "value": round(nbytes / t_pass / 1e9, 4), "unit": "GB/s", "cores": int(blas),
        "kind": "oracle",
        "sample": ("float64 numpy oracle on the 70B-shaped decode pass (M=1), extrapolated: "
                   "each of the 7 module shapes with and without the EC (rank 64) on 512 and "
                   "1024 output rows of full K, median of 3, the time line evaluated at the "
                   "module's N, summed over 80 layers with the model's EC selection "
                   f"({t_pass:.1f} s per pass, {nbytes / 1e9:.1f} GB algorithmic)"),
        "prefill_tflops": round(algo_flops(PRE_M, N, K, 64) / t_pre / 1e12, 5),
        "prefill_sample": "70B q shape at M=4096, 256 of 8192 output rows, time scaled x32",
        "host_cpus": os.cpu_count(),
        "cpu_seconds": round(time.perf_counter() - t_start, 1),
    }


class Model70B:
    """The 70B-shaped model resident in HBM and one pass of its linear layers
    at M tokens (every module once, each call on its AUTO path)."""

    def __init__(self, sp, torch, dev, Mmax, weight_bits=4):
        from paper_2606_11244_amd import model70b
        from paper_2606_11244_amd import synth as S
        self.sp, self.torch, self.S = sp, torch, S
        self.r, self.G = model70b.RANK, model70b.GROUP
        self.wb = weight_bits
        self.layers, self.sel = model70b.build(dev, weight_bits=weight_bits)
        Kmax = max(k for k, _ in S.LLAMA_70B.values())
        Nmax = max(n for _, n in S.LLAMA_70B.values())
        g = torch.Generator(device=dev)
        g.manual_seed(1)
        self.xbuf = torch.randn((Mmax * Kmax,), device=dev, generator=g).half()
        # each member of a grouped call writes its own slice
        ny = max(sum(S.LLAMA_70B[m][1] for m in grp) for grp in GROUPS_70B)
        self.ybuf = torch.empty((Mmax * max(ny, Nmax),), dtype=torch.float16, device=dev)
        self.dev = dev

    def plans(self, M):
        sp, S = self.sp, self.S
        out = {}
        for m in S.MODULES:
            K, N = S.LLAMA_70B[m]
            out[m] = (sp.problem(M, N, K, self.G, sp.F16, self.r, sp.GATE_SIGMOID_LINEAR,
                                 weight_bits=self.wb),
                      sp.problem(M, N, K, self.G, sp.F16, 0, sp.GATE_SIGMOID_LINEAR,
                                 weight_bits=self.wb))
        return out

    def calls(self, M, with_ec):
        """The pass as a list of calls: ("one", args of a single call) or
        ("group", members of a grouped call: q, k, v and gate, up, which read
        one hidden state)."""
        plans = self.plans(M)
        out = []
        for mods in self.layers:
            byname = {mod[0]: mod for mod in mods}
            for grp in GROUPS_70B:
                members, off = [], 0
                for name in grp:
                    (m, K, N, q, sc, zr, ec) = byname[name]
                    pe, p4 = plans[m]
                    use_ec = with_ec and ec is not None
                    x = self.xbuf[:M * K].view(M, K)
                    y = self.ybuf[off:off + M * N].view(M, N)
                    off += M * N
                    members.append(dict(prob=pe if use_ec else p4, x=x, qweight=q, scales=sc,
                                        zeros=zr, y=y,
                                        ec_args=dict(A=ec[0], B=ec[1], w_g=ec[2]) if use_ec else None))
                if len(members) == 1:
                    out.append(("one", members[0]))
                else:
                    out.append(("group", members))
        return out

    def workspace(self, M):
        sp = self.sp
        need = 256
        for pe, p4 in self.plans(M).values():
            need = max(need, sp.dispatch_plan(pe).workspace_bytes,
                       sp.dispatch_plan(p4, with_ec=False).workspace_bytes)
        for with_ec in (True, False):
            for kind, c in self.calls(M, with_ec):
                if kind == "group":
                    need = max(need, sp.group_workspace(c))
        return self.torch.zeros(need, dtype=self.torch.uint8, device=self.dev)

    def run(self, M, with_ec, ws):
        sp = self.sp
        for kind, c in self.calls(M, with_ec):
            if kind == "group":
                sp.w4ec_linear_group(c, ws)
            elif c["ec_args"] is not None:
                e = c["ec_args"]
                sp.w4ec_linear(c["prob"], c["x"], c["qweight"], c["scales"], c["zeros"], e["A"],
                               e["B"], c["y"], w_g=e["w_g"], workspace=ws)
            else:
                sp.w4_linear(c["prob"], c["x"], c["qweight"], c["scales"], c["zeros"], c["y"],
                             workspace=ws)

    def capture(self, M, with_ec, ws):
        torch = self.torch
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            self.run(M, with_ec, ws)
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            self.run(M, with_ec, ws)
        torch.cuda.synchronize()
        return gr

    def work(self, M, with_ec=True):
        """(algorithmic bytes, algorithmic flops, launches) of one pass."""
        sp = self.sp
        nbytes = flops = 0.0
        launches = 0
        for kind, c in self.calls(M, with_ec):
            for mem in (c if kind == "group" else [c]):
                p = mem["prob"]
                r = p.rank if mem["ec_args"] is not None else 0
                nbytes += algo_bytes(M, p.N, p.K, self.G, r, wbits=self.wb)
                flops += algo_flops(M, p.N, p.K, r)
            if kind == "group":
                launches += sp.group_launches(c)
            else:
                launches += sp.dispatch_plan(c["prob"], with_ec=c["ec_args"] is not None).num_launches
        return nbytes, flops, launches

    def paths(self, M):
        sp = self.sp
        return {m: sp.PATH_NAMES[sp.dispatch_plan(pe).path] for m, (pe, _) in self.plans(M).items()}


def replay_times(torch, graph, n):
    """Event-timed replays of one graph on the current stream (seconds each)."""
    ev = []
    for _ in range(n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        graph.replay()
        e1.record()
        ev.append((e0, e1))
    torch.cuda.synchronize()
    return [a.elapsed_time(b) * 1e-3 for a, b in ev]


def model_70b_sweep(model, Ms=(1, 4, 8, 16, 32, 64, 512, 8192), reps=3):
    """Further token counts of the 70B-shaped model's pass (the sweep of its
    workload), each with its EC overhead."""
    import numpy as np
    torch = model.torch
    out = []
    for M in Ms:
        ws = model.workspace(M)
        t = {}
        for ec in (True, False):
            g = model.capture(M, ec, ws)
            g.replay()
            t[ec] = float(np.median(replay_times(torch, g, reps)))
            del g
        nbytes, flops, _ = model.work(M)
        out.append({"M": M, "ms_per_pass": round(t[True] * 1e3, 3),
                    "w4_only_ms": round(t[False] * 1e3, 3),
                    "ec_overhead": round(t[True] / t[False] - 1, 4),
                    "GBps": round(nbytes / t[True] / 1e9, 1),
                    "hbm_frac": round(nbytes / t[True] / 1e9 / HBM_PEAK_GBS, 4),
                    "TFLOPs": round(flops / t[True] / 1e12, 1),
                    "mfma_frac": round(flops / t[True] / 1e12 / MFMA_F16_PEAK_TFLOPS, 4)})
        print("bench: 70B model pass M=%d: %.3f ms (W4-only %.3f ms)" % (M, t[True] * 1e3, t[False] * 1e3),
              file=sys.stderr, flush=True)
        del ws
    return out


def llama1b_extras(args, sp, S, np, torch, dev):
    """The Llama-3.2-1B-shaped decode and prefill passes (extra fields)."""
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
    # ---- the paper's own gate (tanh-MLP on u = A x, Eq. 3) on the same
    # passes, each module on its AUTO path (one call per module at decode)
    tanh = None
    if not args.no_tanh:
        print("bench: tanh-MLP gate passes", file=sys.stderr, flush=True)

        need = max([sp.dispatch_plan(d.problem(gate_kind=S.GATE_TANH_MLP)).workspace_bytes
                    for d in base_dev + pre_dev])
        tanh_ws = torch.zeros(max(need, 256), dtype=torch.uint8, device=dev)

        def decode_tanh(c):
            for mods in dec_dev[c]:
                for d in mods:
                    d.run_ec(d.problem(gate_kind=S.GATE_TANH_MLP), tanh_ws)

        def prefill_tanh():
            for d in pre_dev:
                d.run_ec(d.problem(gate_kind=S.GATE_TANH_MLP), tanh_ws)

        def decode_sig_single(c):
            for mods in dec_dev[c]:
                for d in mods:
                    d.run_ec(d.problem(), dec_ws_t)

        g_dt = [capture(lambda c=c: decode_tanh(c)) for c in range(args.copies)]
        g_ds = [capture(lambda c=c: decode_sig_single(c)) for c in range(args.copies)]
        g_pt = capture(prefill_tanh)
        run_steps(args.warmup, g_dt, g_pt, False)
        evt = run_steps(args.steps, g_dt, g_pt, True)
        evs = run_steps(args.steps, g_ds, g_pre, True)
        torch.cuda.synchronize()
        dt_ = float(np.median([a.elapsed_time(b) for a, b, _ in evt])) * 1e-3
        pt_ = float(np.median([b.elapsed_time(c) for _, b, c in evt])) * 1e-3
        ds_ = float(np.median([a.elapsed_time(b) for a, b, _ in evs])) * 1e-3
        tanh = {"gate": "tanh-MLP, h = 4r = 64 (Eq. 3), fp16 parameters",
                "decode_paths": sorted({sp.PATH_NAMES[sp.dispatch_plan(
                    d.problem(gate_kind=S.GATE_TANH_MLP)).path] for d in base_dev}),
                "prefill_paths": sorted({sp.PATH_NAMES[sp.dispatch_plan(
                    d.problem(gate_kind=S.GATE_TANH_MLP)).path] for d in pre_dev}),
                "decode_ms_per_pass": round(dt_ * 1e3, 4),
                "decode_sigmoid_same_calls_ms": round(ds_ * 1e3, 4),
                "prefill_ms_per_pass": round(pt_ * 1e3, 4),
                "decode_vs_sigmoid": round(dt_ / ds_ - 1.0, 4),
                "prefill_vs_sigmoid": round(pt_ / pre_s - 1.0, 4)}
        if overhead is not None:
            tanh["decode_overhead_vs_w4"] = round(dt_ / d4 - 1.0, 4)
            tanh["prefill_overhead_vs_w4"] = round(pt_ / p4 - 1.0, 4)
        del g_dt, g_ds, g_pt

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

    # (the stored counter runs cover the 70B-shaped headline workload only)
    n_launch_dec = LAYERS_1B * len(DEC_GROUPS)
    return {
        "workload": ("llama-3.2-1b-shaped W4+EC linear layers (q,k,v,o 2048->2048/512, "
                     "gate/up 2048->8192, down 8192->2048), group 128, rank 16, sigmoid-linear "
                     "gate, fp16: decode M=1 over 16 layers x 7 modules (grouped calls, "
                     "%d weight copies alternating) + prefill M=4096 over 7 modules" % args.copies),
        "decode_GBps": round(dec_gbs, 2), "decode_ms_per_pass": round(dec_s * 1e3, 4),
        "decode_hbm_frac": round(dec_gbs / HBM_PEAK_GBS, 4),
        "decode_path": sp.PATH_NAMES[dec_plan.path],
        "decode_launches": n_launch_dec,
        "decode_avg_launch_us": round(dec_s / n_launch_dec * 1e6, 3),
        "decode_traffic_per_launch": None,
        "decode_algo_bytes_per_launch": round(dec_bytes / n_launch_dec),
        "prefill_TFLOPs": round(pre_tfl, 2), "prefill_ms_per_pass": round(pre_s * 1e3, 4),
        "prefill_mfma_frac": round(pre_tfl / MFMA_F16_PEAK_TFLOPS, 4),
        "prefill_paths": {m: sp.PATH_NAMES[sp.dispatch_plan(d.problem()).path]
                          for m, d in zip(S.MODULES, pre_dev)},
        "prefill_traffic_per_launch": None,
        "decode_one_call_per_module": ungrouped,
        "ec_overhead": overhead,
        "ec_int8": int8,
        "post_ec_tail": tail,
        "tanh_gate": tanh,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--copies", type=int, default=2,
                    help="1B decode: weight copies rotated per step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-overhead", action="store_true", help="skip the W4-only reference passes")
    ap.add_argument("--no-paper-protocol", action="store_true",
                    help="skip the decode pass timed as 200 warm-up + 500 timed replays")
    ap.add_argument("--no-1b", action="store_true", help="skip the Llama-3.2-1B-shaped passes")
    ap.add_argument("--no-w3", action="store_true",
                    help="skip the 70B-shaped model with 3-bit codes")
    ap.add_argument("--no-int8", action="store_true",
                    help="1B: skip the passes with INT8 per-channel EC factors")
    ap.add_argument("--no-ungrouped", action="store_true",
                    help="1B: skip the decode pass with one call per module")
    ap.add_argument("--no-tail", action="store_true",
                    help="1B: skip the passes with the post-EC tail on o and down")
    ap.add_argument("--no-tanh", action="store_true",
                    help="1B: skip the passes with the paper's tanh-MLP gate")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the measured HBM-read and MFMA ceilings")
    ap.add_argument("--model70b", action="store_true",
                    help="also time the 70B-shaped model's pass at M = 1, 4, 8, 16, 32, 64, 512, 8192")
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
    print("bench: building the 70B-shaped model", file=sys.stderr, flush=True)
    # the --model70b sweep reaches 8192 tokens
    model = Model70B(sp, torch, dev, max(PRE_M, 8192) if args.model70b else PRE_M)
    ws_dec, ws_pre = model.workspace(DEC_M), model.workspace(PRE_M)
    print("bench: capturing graphs", file=sys.stderr, flush=True)
    g_dec = model.capture(DEC_M, True, ws_dec)
    g_pre = model.capture(PRE_M, True, ws_pre)
    dec_bytes, dec_flops, dec_launches = model.work(DEC_M)
    pre_bytes, pre_flops, pre_launches = model.work(PRE_M)

    def run_steps(n, gdec, gpre):
        ev = []
        for _ in range(n):
            e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            e0.record()
            gdec.replay()
            e1.record()
            gpre.replay()
            e2.record()
            ev.append((e0, e1, e2))
        torch.cuda.synchronize()
        return (np.array([a.elapsed_time(b) for a, b, _ in ev]) * 1e-3,
                np.array([b.elapsed_time(c) for _, b, c in ev]) * 1e-3)

    print("bench: warmup", file=sys.stderr, flush=True)
    run_steps(args.warmup, g_dec, g_pre)
    print("bench: timed steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    t_dec, t_pre = run_steps(args.steps, g_dec, g_pre)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dec_s, pre_s = float(np.median(t_dec)), float(np.median(t_pre))
    dec_gbs = dec_bytes / dec_s / 1e9
    pre_tfl = pre_flops / pre_s / 1e12
    print("bench: decode %.3f ms, prefill %.3f ms per pass" % (dec_s * 1e3, pre_s * 1e3),
          file=sys.stderr, flush=True)

    overhead = None
    if not args.no_overhead:
        print("bench: W4-only reference passes", file=sys.stderr, flush=True)
        g_dec4 = model.capture(DEC_M, False, ws_dec)
        g_pre4 = model.capture(PRE_M, False, ws_pre)
        run_steps(args.warmup, g_dec4, g_pre4)
        d4, p4 = run_steps(args.steps, g_dec4, g_pre4)
        d4, p4 = float(np.median(d4)), float(np.median(p4))
        b4 = model.work(DEC_M, with_ec=False)[0]
        f4 = model.work(PRE_M, with_ec=False)[1]
        overhead = {"decode": round(dec_s / d4 - 1.0, 4), "prefill": round(pre_s / p4 - 1.0, 4),
                    "decode_w4_only_ms": round(d4 * 1e3, 4), "prefill_w4_only_ms": round(p4 * 1e3, 4),
                    "decode_w4_only_GBps": round(b4 / d4 / 1e9, 1),
                    "prefill_w4_only_TFLOPs": round(f4 / p4 / 1e12, 1),
                    "decode_ec_byte_share": round(dec_bytes / b4 - 1.0, 4)}
        del g_dec4, g_pre4

    paper = None
    if not args.no_paper_protocol:
        print("bench: decode pass, 200 warm-up + 500 timed replays", file=sys.stderr, flush=True)
        replay_times(torch, g_dec, 200)
        tp = float(np.median(replay_times(torch, g_dec, 500)))
        paper = {"protocol": "200 warm-up + 500 timed replays of the decode pass, median",
                 "ms_per_pass": round(tp * 1e3, 4), "GBps": round(dec_bytes / tp / 1e9, 1),
                 "hbm_frac": round(dec_bytes / tp / 1e9 / HBM_PEAK_GBS, 4)}

    sweep = None
    if args.model70b:
        del g_pre
        sweep = model_70b_sweep(model)
    else:
        del g_pre

    if args.copy_calib_mb:
        # counter calibration: one elementwise kernel that reads and writes
        # exactly copy_calib_mb MiB each (fp32 negation)
        n = (args.copy_calib_mb << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        torch.neg(a, out=b)
        torch.cuda.synchronize()
        del a, b

    sel = model.sel
    paths_dec, paths_pre = model.paths(DEC_M), model.paths(PRE_M)
    del model, g_dec, ws_dec, ws_pre
    torch.cuda.empty_cache()

    w3 = None
    if not args.no_w3:
        # the same model with 3-bit codes (the paper's 3-bit backbone)
        print("bench: 70B-shaped model with 3-bit codes", file=sys.stderr, flush=True)
        m3 = Model70B(sp, torch, dev, PRE_M, weight_bits=3)
        wd, wp = m3.workspace(DEC_M), m3.workspace(PRE_M)
        res = {}
        for what, M, ws, n in (("decode", DEC_M, wd, max(5, args.steps)), ("prefill", PRE_M, wp, 3)):
            t = {}
            for ec in (True, False):
                g = m3.capture(M, ec, ws)
                replay_times(torch, g, 2)
                t[ec] = float(np.median(replay_times(torch, g, n)))
                del g
            nb, fl, _ = m3.work(M)
            res[what] = {"ms_per_pass": round(t[True] * 1e3, 4),
                         "w3_only_ms": round(t[False] * 1e3, 4),
                         "ec_overhead": round(t[True] / t[False] - 1.0, 4),
                         "GBps": round(nb / t[True] / 1e9, 1),
                         "hbm_frac": round(nb / t[True] / 1e9 / HBM_PEAK_GBS, 4),
                         "TFLOPs": round(fl / t[True] / 1e12, 1),
                         "mfma_frac": round(fl / t[True] / 1e12 / MFMA_F16_PEAK_TFLOPS, 4)}
        w3 = {"weights": "3-bit codes, 32 to three words; group 128; device-random",
              "decode_M1": res["decode"], "prefill_M4096": res["prefill"]}
        del m3, wd, wp
        torch.cuda.empty_cache()

    extras = None
    if not args.no_1b:
        print("bench: 1B-shaped passes", file=sys.stderr, flush=True)
        extras = llama1b_extras(args, sp, S, np, torch, dev)

    ceil = None
    if not args.no_ceiling:
        # what the chip sustains, beside the published peaks: a streaming read
        # of one 117 MB gate/up/down module's codes, and 32x32x16 fp16 MFMAs
        # with full-entropy operands
        from paper_2606_11244_amd import ceiling
        print("bench: measured ceilings", file=sys.stderr, flush=True)
        rd, _ = ceiling.read_ceiling(torch, 28672 * 8192 // 2)
        mf, _ = ceiling.mfma_ceiling(torch, True)
        ceil = {"hbm_read_GBps": round(rd, 1), "mfma_f16_TFLOPs": round(mf, 1),
                "how": ("python -m paper_2606_11244_amd.ceiling: streaming read of 117 MB "
                        "(rotated copies beyond the Infinity Cache); sustained 32x32x16 fp16 "
                        "MFMAs with full-entropy operands")}
        torch.cuda.empty_cache()

    traffic = stored_traffic()
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
        "data": "synthetic (device-random 4-bit weights, EC factors and activations)",
        "config": {
            "workload": ("llama-2-70b-shaped W4+EC linear layers, the whole model resident: "
                         "80 layers x (q,o 8192->8192; k,v 8192->1024; gate,up 8192->28672; "
                         "down 28672->8192), group-128 int4, EC rank 64 with the sigmoid-linear "
                         "gate on a seeded 25%% of the modules (%d of %d), 4-bit only on the "
                         "rest, fp16 activations; one step = decode pass M=1 + prefill pass "
                         "M=4096, every module once on its AUTO path, q/k/v and gate/up as "
                         "grouped calls" % (int(sel.sum()), sel.size)),
            "group_size": GROUP, "rank": 64, "gate": "sigmoid_linear",
            "decode_M": DEC_M, "prefill_M": PRE_M,
            "decode_paths": paths_dec, "prefill_paths": paths_pre,
            "statistic": "median over the timed steps (per-pass HIP events)",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": ("every launch of the decode pass: the 4-bit GEMV (k_gemv, EPI_NONE; "
                       "k_gemv_group where modules of a grouped call without an EC share a "
                       "launch) on the modules without an EC, the producer-fused W4+EC GEMV (k_gemv, "
                       "EPI_FUSED) on those with one, and on the 28672-deep down modules the EC "
                       "pre-kernel k_ec + k_gemv (EPI_READY)"),
            "achieved": round(dec_bytes / dec_launches / (dec_s / dec_launches) / 1e9, 2),
            "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(dec_gbs / HBM_PEAK_GBS, 4),
            "traffic": (traffic or {}).get("decode_bytes_per_launch"),
            "algo_bytes_per_launch": round(dec_bytes / dec_launches),
            "launches_per_pass": dec_launches,
            "avg_launch_us": round(dec_s / dec_launches * 1e6, 3),
            "measured_ceiling": None if ceil is None else {
                "value": ceil["hbm_read_GBps"], "unit": "GB/s",
                "frac": round(dec_gbs / ceil["hbm_read_GBps"], 4), "how": ceil["how"]},
        },
        "prefill": {
            "value": round(pre_tfl, 2), "unit": "TFLOP/s", "ms_per_pass": round(pre_s * 1e3, 4),
            "roofline": {
                "bound": "mfma",
                "kernel": ("every launch of the prefill pass: the 4-bit GEMM with loading and "
                           "multiplying waves k_gemm_ws (EPI_NONE; 256 x 256 tiles, 256 x 128 "
                           "on q/o-sized layers if 256 x 256 would not fill the CUs) or, on the "
                           "1024-row k and v modules, the split-K k_gemm, without an EC; k_ec + "
                           "the same GEMM with the EC epilogue (EPI_READY) with one"),
                "achieved": round(pre_tfl, 2), "peak": MFMA_F16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(pre_tfl / MFMA_F16_PEAK_TFLOPS, 4),
                "traffic": (traffic or {}).get("prefill_bytes_per_launch"),
                "algo_flops_per_launch": round(pre_flops / pre_launches),
                "launches_per_pass": pre_launches,
                "measured_ceiling": None if ceil is None else {
                    "value": ceil["mfma_f16_TFLOPs"], "unit": "TFLOP/s",
                    "frac": round(pre_tfl / ceil["mfma_f16_TFLOPs"], 4), "how": ceil["how"]},
            },
        },
        "decode_ms_per_pass": round(dec_s * 1e3, 4),
        "decode_mean_ms_per_pass": round(float(np.mean(t_dec)) * 1e3, 4),
        "prefill_mean_ms_per_pass": round(float(np.mean(t_pre)) * 1e3, 4),
        "decode_paper_protocol": paper,
        "ec_overhead": overhead,
        "model_70b_sweep": sweep,
        "w3_model_70b": w3,
        "llama1b": extras,
    }
    if not args.no_cpu_baseline:
        print("bench: CPU oracle baseline", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(sel)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
