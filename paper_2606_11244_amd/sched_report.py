"""SLO-constrained EC-aware chunk scheduling on measured latency tables
(SPEAR section 4.3), for a 16-layer Llama-3.2-1B-shaped model.

Reads the per-module tables written by
`python -m paper_2606_11244_amd.crossover --lut <json>` (4-bit-only and
W4+EC latency per call at a grid of token counts, measured on the GPU) and,
on the host only, evaluates the library's scheduler (include/spear_sched.h):

  * the iteration estimate T_S(M) for three EC selections S: none, a seeded
    40% of the (layer, module) pairs (inside the paper's 15-60% range of
    selected modules), and all of them;
  * the largest prefill chunk c in [c_min, c_max] with T_S(d) + T_S(c) <=
    T_SLO over a grid of decode loads d and latency targets;
  * the host time of one scheduling decision (the C call, binary search
    over the chunk range).

The tables cover the linear layers only: attention, norms and the rest of an
iteration are not modelled (no `extra` table), so T_S is the linear-layer
share of an iteration.

Usage (host only, no GPU needed once the tables exist):
  python -m paper_2606_11244_amd.sched_report profiles/latency_lut_llama1b.json \
      --out profiles/sched_llama1b.md
"""
from __future__ import annotations

import argparse
import json
import sys
import time

LAYERS = 16
C_MIN, C_MAX = 16, 4096
SLO_MS = (1.5, 2.0, 4.0, 8.0, 16.0)
DECODE = (1, 16, 64, 256)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("lut")
    ap.add_argument("--out", default=None)
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args(argv)

    import numpy as np

    from paper_2606_11244_amd import spear as sp

    d = json.load(open(args.lut))
    mods = list(d["modules"])
    luts = [(d["modules"][m]["M"], d["modules"][m]["w4_us"], d["modules"][m]["ec_us"]) for m in mods]
    rng = np.random.default_rng(np.random.SeedSequence([args.seed, 7, 4243]))
    sel40 = np.zeros(LAYERS * len(mods), dtype=bool)
    sel40[rng.choice(sel40.size, size=int(round(0.4 * sel40.size)), replace=False)] = True
    selections = {
        "none": [[0] * len(mods) for _ in range(LAYERS)],
        "40%": sel40.reshape(LAYERS, len(mods)).astype(int).tolist(),
        "all": [[1] * len(mods) for _ in range(LAYERS)],
    }
    models = {k: sp.LatencyModel(luts, v) for k, v in selections.items()}

    lines = ["# SLO-constrained EC-aware chunk scheduling: Llama-3.2-1B-shaped model", "",
             "Command (from the repository root, host only): `python -m "
             f"paper_2606_11244_amd.sched_report {args.lut} --out {args.out}`", "",
             f"Latency tables: `{args.lut}` ({d['workload']}; {d['unit']}; produced by "
             f"`{d['command']}`). {LAYERS} layers x {len(mods)} modules; selections: none, a seeded "
             "40% of the (layer, module) pairs, all. Linear layers only (no attention/norm table), "
             "so T_S is the linear-layer part of an iteration.", "",
             "## Iteration estimate T_S(M) in ms", "",
             "| M | " + " | ".join(f"S = {k}" for k in models) + " |",
             "|---" * (len(models) + 1) + "|"]
    for M in (1, 16, 64, 128, 512, 1024, 2048, 4096):
        row = [f"{sp.sched_latency(m, M) / 1e3:.3f}" for m in models.values()]
        lines.append(f"| {M} | " + " | ".join(row) + " |")
    lines += ["", f"## Largest prefill chunk c in [{C_MIN}, {C_MAX}] (0: none fits)", ""]
    for name, m in models.items():
        lines += [f"Selection {name}:", "", "| d \\ T_SLO (ms) | " +
                  " | ".join(str(t) for t in SLO_MS) + " |", "|---" * (len(SLO_MS) + 1) + "|"]
        for dd in DECODE:
            cs = [str(sp.sched_chunk(m, dd, t * 1e3, C_MIN, C_MAX)) for t in SLO_MS]
            lines.append(f"| {dd} | " + " | ".join(cs) + " |")
        lines.append("")
    # host cost of one decision
    m = models["40%"]
    n = 20000
    t0 = time.perf_counter()
    for i in range(n):
        sp.sched_chunk(m, DECODE[i % len(DECODE)], SLO_MS[i % len(SLO_MS)] * 1e3, C_MIN, C_MAX)
    dt = (time.perf_counter() - t0) / n
    lines += ["## Host cost of one decision", "",
              f"{dt * 1e6:.2f} us per `spear_sched_chunk` call through the Python binding "
              f"(mean of {n}; {LAYERS} x {len(mods)} calls summed per estimate, binary search over "
              f"[{C_MIN}, {C_MAX}]), single host thread.", ""]
    text = "\n".join(lines)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)
        print(f"wrote {args.out}", file=sys.stderr)
    else:
        print(text)


if __name__ == "__main__":
    main()
