"""CPU oracle of SPEAR's SLO-constrained EC-aware chunk scheduling.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute this module: only the tests use it. It shares no code with the
library's scheduler (spear_sched.cpp); the tables are passed in as plain
Python lists.

What it computes (SPEAR, section 4.3): offline, every linear module type has
a latency table measured at a sparse grid of token counts, one for the
4-bit-only call (l_W4) and one with the EC attached (l_EC). Online, the
latency of an iteration at M tokens is estimated by adding up one table
entry per linear call of the model, the EC table for the calls the
selection S compensates and the 4-bit table otherwise, with linear
interpolation for token counts between the measured ones. The scheduler
then takes the largest prefill chunk c in [c_min, c_max] with

    T_S(d) + T_S(c) <= T_SLO,

d being the decode tokens already scheduled.

Everything is computed in exact rational arithmetic (fractions.Fraction of
the given floats), the sum is taken call by call in layer order, and the
chunk is found by testing every candidate c, so none of it depends on
rounding order or on the monotonicity the library's binary search uses.

Readings where the paper is silent (the same readings the library states):
a table is read as its running maximum over M (measured tables carry
noise); below the first entry it takes the first entry, above the last it
continues the last segment linearly (constant for a one-entry table); zero
tokens cost nothing; an optional per-layer table of the iteration's other
work (attention, norms) adds its 4-bit column once per layer; when no
chunk fits, the answer is 0.
"""
from __future__ import annotations

from fractions import Fraction


def _envelope(lat):
    """Running maximum of a latency column, as Fractions."""
    out, best = [], None
    for v in lat:
        f = Fraction(v)
        best = f if best is None or f > best else best
        out.append(best)
    return out


def table_latency(M, lat, x):
    """One column of a table at token count x (section 4.3: linear
    interpolation between measured token counts)."""
    if x <= 0:
        return Fraction(0)
    env = _envelope(lat)
    if x <= M[0]:
        return env[0]
    if len(M) == 1:
        return env[0]
    for i in range(1, len(M)):
        if x <= M[i] or i == len(M) - 1:
            slope = (env[i] - env[i - 1]) / (M[i] - M[i - 1])
            return env[i - 1] + slope * (x - M[i - 1])
    raise AssertionError("unreachable")


def iteration_latency(luts, selection, layers, modules, x, extra=None):
    """T_S(x): one table entry per linear call, layer by layer, the EC table
    where selection[l][j] is set. `luts[j]` = (M, lat_w4, lat_ec)."""
    t = Fraction(0)
    for l in range(layers):
        for j in range(modules):
            M, lw4, lec = luts[j]
            t += table_latency(M, lec if selection[l][j] else lw4, x)
        if extra is not None:
            t += table_latency(extra[0], extra[1], x)
    return t


def chunk(luts, selection, layers, modules, d, t_slo, c_min, c_max, extra=None):
    """The largest c in [c_min, c_max] with T_S(d) + T_S(c) <= T_SLO, by
    testing every candidate; 0 if none fits."""
    td = iteration_latency(luts, selection, layers, modules, d, extra)
    slo = Fraction(t_slo)
    best = 0
    for c in range(c_min, c_max + 1):
        if td + iteration_latency(luts, selection, layers, modules, c, extra) <= slo:
            best = c
    return best
