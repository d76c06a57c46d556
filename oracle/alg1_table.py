"""Iterations-versus-error table of Algorithm 1 (Halley-bisection, Sec. 3.1),
run by the oracle in fp64 on rows of the sparsity-sweep workload.

TEST INFRASTRUCTURE: a diagnostic of the paper's solver, computed by the
oracle only.  For each (alpha, c) it takes `rows` evenly spaced query rows of
head 0 of B1 H16 n8192 d128 (the bf16 inputs of synth, widened to fp64),
forms x = (alpha-1) * scale * q k^T, runs Algorithm 1 from its initial
bracket (eo_halley_bisection_trace), and prints, per iteration t, the median
and largest relative error |tau_t - tau| / max(1, |tau|) against the exact
threshold (long bisection).  The paper reports 3 iterations to machine
precision at alpha = 1.5 (Sec. 3.1; its Fig. 2 is not available).

    python oracle/alg1_table.py [--rows 128] [--iters 10]
"""
import argparse
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))

import oracle  # noqa: E402
import synth  # noqa: E402


def table(alpha, c, rows, iters, n=8192, d=128):
    inp = synth.attention_inputs(1, 1, n, d, c=c, dtype="bf16", seed=synth.SEED_BASE)
    q, k = inp["q"].f64()[0, 0], inp["k"].f64()[0, 0]
    a = float(np.float32(alpha))
    scale = float(np.float32(d ** -0.5))
    idx = np.linspace(0, n - 1, rows).astype(int)
    x = (a - 1) * scale * (q[idx] @ k.T)
    err = np.empty((rows, iters + 1))
    for r in range(rows):
        tr = oracle.halley_bisection_trace(x[r], a, iters)
        exact = oracle.entmax_threshold(x[r], a)
        err[r] = np.abs(tr - exact) / max(1.0, abs(exact))
    return err


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--rows", type=int, default=128)
    ap.add_argument("--iters", type=int, default=10)
    args = ap.parse_args()
    points = [(1.5, 0.0625), (1.5, 1.0), (1.5, 32.0), (1.25, 1.0), (2.0, 1.0)]
    print("| alpha | c | " + " | ".join("t=%d" % t for t in range(args.iters + 1)) +
          " | updates to 1e-6 (median / max) |")
    print("|---|---|" + "---|" * (args.iters + 1) + "---|")
    for alpha, c in points:
        err = table(alpha, c, args.rows, args.iters)
        med = np.median(err, axis=0)
        mx = err.max(axis=0)
        cells = ["%.0e / %.0e" % (m, x_) for m, x_ in zip(med, mx)]
        reach = np.array([np.argmax(e <= 1e-6) if (e <= 1e-6).any() else args.iters + 1
                          for e in err])
        print("| %g | %g | %s | %d / %d |" % (alpha, c, " | ".join(cells), int(np.median(reach)),
                                              int(reach.max())))


if __name__ == "__main__":
    main()
