"""Dispatch crossover measurement: every execution path of the W4+EC layer,
timed per module shape and token count, next to the path the planner picks.

For each (configuration, module, M) the layer's weights are copied enough
times to exceed the last-level caches (up to 16 copies), each path's calls
over the copies are captured once as a HIP graph and replayed, and the mean
time per call is reported. The markdown written to --out lists, per row, the
4-bit-only time, each EC path's time, the fastest EC path and the planner's
AUTO choice.

Usage (on a GPU):
  python -m paper_2606_11244_amd.crossover --out profiles/dispatch_crossover.md
  python -m paper_2606_11244_amd.crossover --lut profiles/latency_lut_llama1b.json

With --rows it measures the decode kernels of the 1B-shaped modules at each
row-tile count (1, 2, 4 sixteen-row tiles per block, forced with
spear_set_gemv_shape, and the planner's own choice), single calls and the
grouped q,k,v and gate,up calls, and writes a markdown table:
  python -m paper_2606_11244_amd.crossover --rows profiles/decode_row_tiles.md

With --lut it instead measures, for each module of the Llama-3.2-1B-shaped
configuration, the 4-bit-only call and the W4+EC call on the path AUTO picks
over a grid of token counts: the latency tables l_W4(M), l_EC(M) of the
SLO-constrained chunk scheduler (section 4.3, include/spear_sched.h).
"""
from __future__ import annotations

import argparse
import json
import math
import sys

PATHS = [("fused_local", 5), ("fused_gemv", 1), ("fused_mfma", 2), ("unfused_2k", 4),
         ("overlap_2k", 6), ("unfused_chain", 3)]

# (configuration id, module, token counts)
DEFAULT_CASES = [
    (1, "q", [1, 4, 16, 32, 48, 64]), (1, "k", [1, 16, 32, 64]), (1, "gate", [1, 16, 32, 48, 64]),
    (1, "down", [1, 16, 32, 64]),
    (2, "q", [128, 256, 512, 1024, 2048, 4096]), (2, "k", [128, 512, 4096]),
    (2, "gate", [128, 512, 2048, 4096]), (2, "down", [512, 4096]),
    (3, "q", [1, 8, 32, 128, 512]), (3, "down", [1, 8, 32, 512]),
    (4, "k", [1, 16, 64, 512]), (4, "gate", [1, 16, 64]), (4, "down", [1, 16, 64]),
]


LUT_M = [1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 2048, 4096]


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default="profiles/dispatch_crossover.md")
    ap.add_argument("--lut", default=None, help="write latency tables (JSON) instead")
    ap.add_argument("--rows", default=None, help="write the decode row-tile table instead")
    ap.add_argument("--reps", type=int, default=10)
    args = ap.parse_args(argv)

    import numpy as np
    import torch

    from paper_2606_11244_amd import spear as sp
    from paper_2606_11244_amd import synth as S

    torch.cuda.set_device(0)

    def timed(fn, copies, reps):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for c in range(copies):
                fn(c)
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for c in range(copies):
                fn(c)
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps / copies  # us per call

    def weights_copies(base, L):
        copies = int(min(16, max(2, math.ceil(600e6 / (L.N * L.K // 2)))))
        devs = []
        for _ in range(copies):
            d = sp.DeviceLayer.__new__(sp.DeviceLayer)
            d.__dict__.update(base.__dict__)
            d.qweight, d.scales, d.zeros = (base.qweight.clone(), base.scales.clone(),
                                            base.zeros.clone())
            devs.append(d)
        return devs

    if args.rows:
        rows_table(args, sp, S, torch, timed)
        return

    if args.lut:
        # one table per module shape of the 1B configuration: prefill shapes
        # (config 2, outlier activations) above 64 tokens, decode shapes below
        tables = {}
        for mod in S.MODULES:
            Ms, w4, ec, paths = [], [], [], []
            for M in LUT_M:
                L = S.config_layer(2 if M > 64 else 1, mod, M, seed=0)
                base = sp.DeviceLayer(L)
                devs = weights_copies(base, L)
                p4, pe = base.problem(), base.problem()
                ws = torch.zeros(max(sp.dispatch_plan(p4, with_ec=False).workspace_bytes,
                                     sp.dispatch_plan(pe).workspace_bytes, 256),
                                 dtype=torch.uint8, device="cuda")
                Ms.append(M)
                w4.append(round(timed(lambda c: devs[c].run_w4(p4, ws), len(devs), args.reps), 3))
                ec.append(round(timed(lambda c: devs[c].run_ec(pe, ws), len(devs), args.reps), 3))
                paths.append(sp.PATH_NAMES[sp.dispatch_plan(pe).path])
                print(json.dumps({"module": mod, "M": M, "w4_us": w4[-1], "ec_us": ec[-1],
                                  "path": paths[-1]}), flush=True)
                del devs, base
                torch.cuda.empty_cache()
            tables[mod] = {"N": L.N, "K": L.K, "rank": L.rank, "M": Ms, "w4_us": w4,
                           "ec_us": ec, "ec_path": paths}
        out = {"workload": "Llama-3.2-1B-shaped W4+EC linear modules (group 128, rank 16, "
                           "sigmoid-linear gate, fp16); synthetic layers, seed 0",
               "command": f"python -m paper_2606_11244_amd.crossover --lut {args.lut}",
               "unit": "us per call, graph-replayed over rotated weight copies",
               "modules": tables}
        with open(args.lut, "w") as f:
            json.dump(out, f, indent=1)
        print(f"wrote {args.lut}", file=sys.stderr)
        return

    rows = []
    for cid, mod, Ms in DEFAULT_CASES:
        for M in Ms:
            L = S.config_layer(cid, mod, M, seed=0)
            base = sp.DeviceLayer(L)
            wbytes = L.N * L.K // 2
            copies = int(min(16, max(2, math.ceil(600e6 / wbytes))))
            devs = []
            for _ in range(copies):
                d = sp.DeviceLayer.__new__(sp.DeviceLayer)
                d.__dict__.update(base.__dict__)
                d.qweight, d.scales, d.zeros = (base.qweight.clone(), base.scales.clone(),
                                                base.zeros.clone())
                devs.append(d)
            row = {"config": cid, "module": mod, "M": M, "N": L.N, "K": L.K, "rank": L.rank}
            p4 = base.problem()
            ws_size = sp.dispatch_plan(p4, with_ec=False).workspace_bytes
            plans = {}
            for name, code in PATHS:
                try:
                    plans[name] = sp.dispatch_plan(base.problem(force_path=code))
                    ws_size = max(ws_size, plans[name].workspace_bytes)
                except sp.SpearError:
                    pass
            auto = sp.dispatch_plan(base.problem())
            ws = torch.zeros(max(ws_size, auto.workspace_bytes, 256), dtype=torch.uint8,
                             device="cuda")
            row["w4_us"] = round(timed(lambda c: devs[c].run_w4(p4, ws), copies, args.reps), 2)
            # the 4-bit product on the other kernel where both apply
            if M <= 64:
                pg, pv = base.problem(force_path=4), base.problem(force_path=1)
                ws_g = max(sp.dispatch_plan(pg, with_ec=False).workspace_bytes,
                           sp.dispatch_plan(pv, with_ec=False).workspace_bytes)
                if ws_g > ws.numel():
                    ws = torch.zeros(ws_g, dtype=torch.uint8, device="cuda")
                row["w4_gemv_us"] = round(timed(lambda c: devs[c].run_w4(pv, ws), copies, args.reps), 2)
                row["w4_gemm_us"] = round(timed(lambda c: devs[c].run_w4(pg, ws), copies, args.reps), 2)
            for name, code in PATHS:
                if name not in plans:
                    continue
                pr = base.problem(force_path=code)
                row[name + "_us"] = round(timed(lambda c: devs[c].run_ec(pr, ws), copies,
                                                args.reps), 2)
            row["auto"] = sp.PATH_NAMES[auto.path]
            ec_times = {n: row[n + "_us"] for n, _ in PATHS if n + "_us" in row}
            row["best"] = min(ec_times, key=ec_times.get)
            print(json.dumps(row), flush=True)
            rows.append(row)
            del devs, base
            torch.cuda.empty_cache()

    names = [n for n, _ in PATHS]
    w4k = [r for r in rows if "w4_gemm_us" in r]
    lines_w4 = ["", "## The 4-bit product alone at up to 64 tokens: GEMV vs GEMM", "",
                "| config | module | M | GEMV | GEMM | AUTO |", "|---|---|---|---|---|---|"]
    for r in w4k:
        lines_w4.append(f"| {r['config']} | {r['module']} | {r['M']} | {r['w4_gemv_us']} | "
                        f"{r['w4_gemm_us']} | {r['w4_us']} |")
    lines = ["# Dispatch crossover: W4+EC paths by token count", "",
             "Command (from the repository root): `python -m paper_2606_11244_amd.crossover "
             "--out profiles/dispatch_crossover.md`", "",
             "Mean time per call in microseconds (graph-replayed over rotated weight copies; "
             "synthetic layers of the named configurations, seed 0). `-` = path not available "
             "for the shape. EC overhead = fastest EC path / 4-bit-only - 1. config: the "
             "synthetic workload's id, counted from 0 (0 tiny K = N = 256, 1 Llama-3.2-1B "
             "decode, 2 the same layers at prefill, 3 Llama-3-8B, 4 Llama-2-70B).", "",
             "| config | module | N | K | r | M | W4 only | " + " | ".join(names) +
             " | fastest | AUTO | EC overhead |",
             "|---" * (9 + len(names) + 1) + "|"]
    for r in rows:
        cells = [str(r.get(n + "_us", "-")) for n in names]
        best_t = r[r["best"] + "_us"]
        auto_mark = r["auto"] if r["auto"] == r["best"] else r["auto"] + " (*)"
        lines.append(f"| {r['config']} | {r['module']} | {r['N']} | {r['K']} | {r['rank']} | "
                     f"{r['M']} | {r['w4_us']} | " + " | ".join(cells) +
                     f" | {r['best']} | {auto_mark} | {best_t / r['w4_us'] - 1:.1%} |")
    lines += ["", "(*) AUTO differs from the fastest measured path."] + lines_w4 + [""]
    with open(args.out, "w") as f:
        f.write("\n".join(lines))
    print(f"wrote {args.out}", file=sys.stderr)


def rows_table(args, sp, S, torch, timed, copies=24):
    """Decode (M = 1, 16) time per call at each row-tile count."""
    def cp(b):
        out = []
        for _ in range(copies):
            d = sp.DeviceLayer.__new__(sp.DeviceLayer)
            d.__dict__.update(b.__dict__)
            d.qweight, d.scales, d.zeros = b.qweight.clone(), b.scales.clone(), b.zeros.clone()
            d.A, d.B = b.A.clone(), b.B.clone()
            out.append(d)
        return out

    ws = torch.zeros(1 << 24, dtype=torch.uint8, device="cuda")
    names = ["q", "k", "o", "gate", "down", "q,k,v", "gate,up"]
    lines = ["# Decode row tiles: time per call by rows per block", "",
             "Command (from the repository root): `python -m paper_2606_11244_amd.crossover "
             f"--rows {args.rows}`", "",
             "Llama-3.2-1B-shaped modules (group 128, rank 16, sigmoid-linear gate, fp16; "
             "synthetic, seed 0), microseconds per call, graph-replayed over "
             f"{copies} weight copies; `EC / 4-bit only`. Row tiles forced with "
             "spear_set_gemv_shape; `planner` = the automatic choice. `-` = the local EC "
             "variant does not take that shape (the planner would pick another path). "
             "Grouped columns: one spear_w4ec_linear_group call (q,k,v share x; gate,up "
             "share x).", ""]
    for M in (1, 16):
        mods = {m: cp(sp.DeviceLayer(S.config_layer(1, m, M, seed=0)))
                for m in ("q", "k", "v", "o", "gate", "up", "down")}
        for c in range(copies):
            mods["k"][c].x = mods["v"][c].x = mods["q"][c].x
            mods["up"][c].x = mods["gate"][c].x
        lines += [f"## M = {M}", "", "| row tiles | " + " | ".join(names) + " |",
                  "|---" * (len(names) + 1) + "|"]
        for rt in (1, 2, 4, 0):
            sp.set_gemv_shape(rt, 0, 0)
            cells = []
            for nm in names:
                grp = nm.split(",")
                if any(sp.dispatch_plan(mods[m][0].problem()).path != sp.PATH_FUSED_LOCAL
                       for m in grp):
                    cells.append("-")
                    continue
                if len(grp) == 1:
                    m = grp[0]
                    te = timed(lambda c, m=m: mods[m][c].run_ec(mods[m][c].problem(), ws),
                               copies, args.reps)
                    t4 = timed(lambda c, m=m: mods[m][c].run_w4(mods[m][c].problem(rank=0), ws),
                               copies, args.reps)
                else:
                    te = timed(lambda c, g=grp: sp.w4ec_linear_group(
                        [mods[m][c].member(mods[m][c].problem()) for m in g], ws), copies, args.reps)
                    t4 = timed(lambda c, g=grp: sp.w4ec_linear_group(
                        [mods[m][c].member(mods[m][c].problem(rank=0), with_ec=False) for m in g],
                        ws), copies, args.reps)
                cells.append(f"{te:.2f} / {t4:.2f}")
            sp.set_gemv_shape(0, 0, 0)
            lines.append(f"| {rt if rt else 'planner'} | " + " | ".join(cells) + " |")
            print(lines[-1], flush=True)
        lines.append("")
        del mods
        torch.cuda.empty_cache()
    with open(args.rows, "w") as f:
        f.write("\n".join(lines))
    print(f"wrote {args.rows}", file=sys.stderr)


if __name__ == "__main__":
    main()
