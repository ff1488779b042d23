"""Writes tests/golden/level_sweep.txt from the oracle alone.

For each record size used by the workloads (n = 128 values, p = 12) it sweeps
the level count M at alpha = 1.4 and records the reconstruction error on
N(0, 1) streams (the procedure of Tab. 2), and, for the level counts the
workloads state, the smallest alpha on a 0.1 grid that makes them fit.

Run from the repository root:  python tests/golden/make_level_sweep.py
"""
import os
import sys
import warnings

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
from oracle import tables, kv  # noqa: E402

warnings.simplefilter("ignore")


def main():
    rng = np.random.default_rng(0)
    x = rng.normal(size=(2000, 128))
    lines = ["# NMSE of the oracle encoder on 2000 N(0,1) streams of 128 values",
             "# (seed 0), alpha = 1.4, p = 12; written by make_level_sweep.py.",
             "# columns: record_bytes  levels  nmse"]
    best = {}
    for C in (32, 36, 48, 64):
        for M in range(3, 64):
            t = tables.build_tables(128, M, 12, 1.4, C)
            if not t.feasible:
                break
            _, syms, s16, o16, _ = kv.encode_streams(x, t)
            xhat = s16.astype(np.float64)[:, None] * syms + o16.astype(np.float64)[:, None]
            nmse = float(((x - xhat) ** 2).sum() / (x ** 2).sum())
            lines.append(f"{C} {M} {nmse:.6f}")
            if C not in best or nmse < best[C][1]:
                best[C] = (M, nmse)
    lines.append("# best level count per record size: record_bytes levels")
    for C, (M, _) in best.items():
        lines.append(f"best {C} {M}")
    lines.append("# smallest feasible alpha (0.1 grid): levels record_bytes alpha")
    for M, C in ((16, 32), (16, 36), (32, 48), (64, 64)):
        for k in range(14, 400):
            if tables.build_tables(128, M, 12, k / 10, C).feasible:
                lines.append(f"alpha {M} {C} {k / 10:.1f}")
                break
    out = os.path.join(os.path.dirname(os.path.abspath(__file__)), "level_sweep.txt")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
