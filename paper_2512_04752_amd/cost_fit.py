"""Fit the verification-cost predictor (RLHFSpec Section 5.2) on measured
verify steps of this library, and read off the instance-throughput threshold
(Section 6.1).

    python -m paper_2512_04752_amd.cost_fit SWEEP.jsonl -o COEFFS.json

SWEEP.jsonl is the output of `bench.py --sweep` (one line per (batch, draft
token num) cell with its measured ms/step).  The model is
    t_sd = c0 + c_seq N_seq + c_draft N_draft + c_tree TK
(N_seq = summed committed lengths, N_draft = summed tree sizes, TK = summed
tree size x committed length), fitted by non-negative least squares on the
relative error (step times span two orders of magnitude, and every term is a
cost, so no coefficient may be negative).  The output also holds
each cell's leave-one-out relative error and the threshold: the largest
measured batch before the marginal accepted-token throughput per added
sample (at each batch's best draft token num) falls below a tenth of its
first value.
"""

import argparse
import json

import numpy as np


def features(row):
    n_draft = row["tokens"]
    n_seq = row["kv_tokens"] - n_draft
    return n_seq, n_draft, row["budget"] * n_seq     # every tree of a cell has `budget` nodes


def solve(F, y):
    from scipy.optimize import nnls
    X = np.column_stack([np.ones(len(y)), F])
    scale = np.abs(X).max(axis=0)
    A = (X / scale) / y[:, None]
    beta, _ = nnls(A, np.ones(len(y)))
    return beta / scale


def fit(rows):
    F = np.array([features(r) for r in rows], dtype=np.float64)
    y = np.array([r["ms_per_step"] for r in rows], dtype=np.float64)
    beta = solve(F, y)
    loo = []
    for i in range(len(rows)):
        keep = np.arange(len(rows)) != i
        b = solve(F[keep], y[keep])
        loo.append(float((b[0] + F[i] @ b[1:]) / y[i] - 1.0))
    return beta, loo


def threshold(rows):
    best = {}
    for r in rows:
        best[r["batch"]] = max(best.get(r["batch"], 0.0), r["accepted_tokens_per_s"])
    batches = sorted(best)
    marg = [(best[b1] - best[b0]) / (b1 - b0) for b0, b1 in zip(batches, batches[1:])]
    thr = batches[-1]
    for k, m in enumerate(marg):
        if m < 0.1 * marg[0]:
            thr = batches[k]
            break
    return thr, {str(b): best[b] for b in batches}, marg


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("sweep")
    ap.add_argument("-o", "--out", required=True)
    ap.add_argument("--bucket-ratio", type=float, default=0.05)
    a = ap.parse_args()
    rows = [json.loads(l) for l in open(a.sweep) if l.strip()]
    beta, loo = fit(rows)
    thr, best, marg = threshold(rows)
    out = {"model": "t_sd_ms = c0 + c_seq*N_seq + c_draft*N_draft + c_tree*TK",
           "c0": float(beta[0]), "c_seq": float(beta[1]), "c_draft": float(beta[2]),
           "c_tree": float(beta[3]), "bucket_ratio": a.bucket_ratio,
           "cells": len(rows),
           "loo_rel_err": {f"b{r['batch']}_n{r['budget']}": round(e, 4) for r, e in zip(rows, loo)},
           "loo_median_abs_rel_err": float(np.median(np.abs(loo))),
           "loo_max_abs_rel_err": float(np.max(np.abs(loo))),
           "threshold_batch": thr, "best_accepted_tokens_per_s_by_batch": best,
           "marginal_tokens_per_s_per_sample": [round(m, 2) for m in marg],
           "source": a.sweep}
    json.dump(out, open(a.out, "w"), indent=1)
    print(json.dumps({k: out[k] for k in ("c0", "c_seq", "c_draft", "c_tree",
                                          "loo_median_abs_rel_err", "loo_max_abs_rel_err",
                                          "threshold_batch")}))


if __name__ == "__main__":
    main()
