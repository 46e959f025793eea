"""The truncation bound of Theorems 1-2 evaluated on the synthetic workloads.

For every sampled (sequence, KV head) group that stops before the end of its
traversal, and every query head of it, this computes what Appendix A's
bound needs, with probe P = I (nu = 1):
- the stop t* (from the oracle) and b = t* - p + 1;
- per block j: the block mass l_j, the prefix mass A_j, the block's own
  attention output u_j and the prefix output o_j, in fp64 (the increment
  identity of Appendix A, pinned against brute force in the oracle tests);
- mu = b l_b / A_b, Delta = max over j in [b, T] of
  |u_j - o_{j-1}| - |u_b - o_{b-1}|, C_v = the largest value norm;
- the conclusion of Lemma 1, l_j / A_j <= mu / j for every j in [b, T],
  which is the hypothesis the proofs use;
- the bound min(tau b + mu Delta, 2 mu C_v) ln(T / t*) against the error
  |o(T) - o(t*)| of the oracle's outputs with termination on and off.

A head whose hypothesis fails is reported as such: the theorems say nothing
about it.  Runs the CPU oracle only; not collected by pytest:

    python tests/study_p7_bound.py --workload qwen3_32b_ragged --groups 64
    python tests/study_p7_bound.py --workload llama3_8b_32k --traversal key_norm
"""
from __future__ import annotations

import argparse
import math
import os
import sys

import numpy as np
import torch

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import oracle  # noqa: E402
from paper_2606_00024_amd import workloads as W  # noqa: E402


def group_arrays(wl, b, kvh):
    """q [g][D], K and V [L][D] of one group in fp64, and its traversal."""
    s = wl.spec
    g = s.group_size
    L = int(wl.seq_lens[b])
    toks = torch.arange(L)
    pages = wl.page_table[b].long()[toks // s.page_size]
    K = wl.k_cache[pages, kvh, toks % s.page_size].double().numpy()
    V = wl.v_cache[pages, kvh, toks % s.page_size].double().numpy()
    q = wl.q[b, kvh * g:(kvh + 1) * g].double().numpy()
    nblk = -(-L // s.block_size)
    if wl.block_list is not None:
        blocks = [int(x) for x in wl.block_list[b, kvh, :int(wl.block_list_len[b, kvh])]]
    elif s.dense_order == 1:
        blocks = list(range(nblk))
    else:
        blocks = list(range(nblk - 1, -1, -1))
    return q, K, V, blocks, L


def block_terms(q, K, V, blocks, L, block_size, scale):
    """Per step t = 1..T (index t): log l_t, log A_t, u_t, o_t; o_0 = 0."""
    g, D = q.shape
    T = len(blocks)
    logl = np.full((T + 1, g), -np.inf)
    logA = np.full((T + 1, g), -np.inf)
    u = np.zeros((T + 1, g, D))
    o = np.zeros((T + 1, g, D))
    for t in range(1, T + 1):
        j0 = blocks[t - 1] * block_size
        idx = np.arange(j0, min(j0 + block_size, L))
        sc = scale * (q @ K[idx].T)
        m = sc.max(axis=1, keepdims=True)
        e = np.exp(sc - m)
        z = e.sum(axis=1, keepdims=True)
        logl[t] = (m + np.log(z))[:, 0]
        u[t] = (e / z) @ V[idx]
        logA[t] = np.logaddexp(logA[t - 1], logl[t])
        w_old = np.exp(logA[t - 1] - logA[t])[:, None]
        w_new = np.exp(logl[t] - logA[t])[:, None]
        o[t] = w_old * o[t - 1] + w_new * u[t]
    return logl, logA, u, o


def evaluate(wl, tau, phi, p, groups, on, off):
    s = wl.spec
    g = s.group_size
    tau32 = float(np.float32(tau))
    rows = []
    for b, kvh in groups:
        q, K, V, blocks, L = group_arrays(wl, b, kvh)
        T = len(blocks)
        ts = int(on["stop"][b, kvh])
        if T == 0 or ts >= T:
            continue
        logl, logA, u, o = block_terms(q, K, V, blocks, L, s.block_size, s.softmax_scale)
        bstart = max(1, ts - p + 1)
        Cv = float(np.linalg.norm(V, axis=1).max())
        for i in range(g):
            ratio = np.exp(logl[1:, i] - logA[1:, i])          # ratio[j - 1] = l_j / A_j
            mu = bstart * ratio[bstart - 1]
            js = np.arange(bstart, T + 1)
            met = bool(np.all(ratio[js - 1] <= mu / js * (1 + 1e-12)))
            upd = np.linalg.norm(u[1:, i] - o[:-1, i], axis=1)  # upd[j - 1] = |u_j - o_{j-1}|
            delta = float((upd[js - 1] - upd[bstart - 1]).max())
            bound = min(tau32 * bstart + mu * delta, 2 * mu * Cv) * math.log(T / ts)
            err = float(np.linalg.norm(off["out"][b, kvh * g + i] - on["out"][b, kvh * g + i]))
            rows.append({"group": (b, kvh), "met": met, "bound": bound, "err": err, "mu": mu})
    return rows


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="qwen3_32b_ragged")
    ap.add_argument("--groups", type=int, default=64, help="groups sampled (seeded)")
    ap.add_argument("--rules", nargs="*", default=["1e-2,1e-2,5", "1e-3,1e-3,5", "1e-4,1e-4,5",
                                                    "1e-5,1e-3,5"])
    ap.add_argument("--traversal", default="dense", choices=["dense", "key_norm"],
                    help="the workload's own order, or every block in descending key norm "
                         "(lists from the list oracle)")
    args = ap.parse_args(argv)
    spec = W.WORKLOADS[args.workload]
    wl = W.make_workload(spec, device="cpu")
    if args.traversal == "key_norm":
        from oracle import lists as OL
        r = OL.block_list(wl.q, wl.k_cache, wl.page_table, wl.seq_lens,
                          block_size=spec.block_size, num_q_heads=spec.num_q_heads,
                          budget=1 << 20)
        wl.block_list = torch.from_numpy(r["list"])
        wl.block_list_len = torch.from_numpy(r["len"])
    all_groups = [(b, h) for b in range(spec.batch) for h in range(spec.num_kv_heads)]
    rng = np.random.default_rng(7)
    pick = rng.choice(len(all_groups), size=min(args.groups, len(all_groups)), replace=False)
    groups = [all_groups[i] for i in sorted(pick)]
    mask = np.zeros((spec.batch, spec.num_kv_heads), dtype=np.int32)
    for b, h in groups:
        mask[b, h] = 1
    off = oracle.decode_workload(wl, tau=0.0, group_mask=mask)
    print(f"workload {spec.name}, {args.traversal} traversal: {len(groups)} groups sampled of "
          f"{len(all_groups)}", flush=True)
    print("| τ, φ, p | groups stopped early | heads | hypothesis met | bound (median, met) | "
          "error (median, met) | max error / bound (met) | error (median, not met) |")
    print("|---|---|---|---|---|---|---|---|")
    for rule in args.rules:
        tau, phi, p = (float(x) for x in rule.split(","))
        p = int(p)
        on = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p, group_mask=mask)
        rows = evaluate(wl, tau, phi, p, groups, on, off)
        stopped = len({r["group"] for r in rows})
        met = [r for r in rows if r["met"]]
        not_met = [r for r in rows if not r["met"]]
        fmt = lambda v: "—" if v is None else f"{v:.3g}"
        med = lambda xs: float(np.median(xs)) if xs else None
        worst = max((r["err"] / r["bound"] for r in met if r["bound"] > 0), default=None)
        print(f"| {tau:g}, {phi:g}, {p} | {stopped} | {len(rows)} | {len(met)} | "
              f"{fmt(med([r['bound'] for r in met]))} | {fmt(med([r['err'] for r in met]))} | "
              f"{fmt(worst)} | {fmt(med([r['err'] for r in not_met]))} |", flush=True)
        assert all(r["err"] <= r["bound"] * (1 + 1e-9) + 1e-12 for r in met), \
            "a head that meets the hypothesis exceeds the bound"


if __name__ == "__main__":
    main()
