"""Reading R3 measured: one stop per (sequence, KV head) group, or one per
query head (the oracle's per_head_stop), on the synthetic workloads.

Runs the CPU oracle only (fp64); prints a markdown table of the blocks the
groups read and of how far each reading's output lies from full attention
(relative L2 per query head).  Not collected by pytest:

    python tests/study_r3_per_head.py [--workloads llama3_8b_32k ...]
"""
from __future__ import annotations

import argparse
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import oracle  # noqa: E402
from paper_2606_00024_amd import workloads as W  # noqa: E402


def _rel(out, ref):
    num = np.linalg.norm(out - ref, axis=-1)
    den = np.linalg.norm(ref, axis=-1)
    return (num / np.where(den > 0, den, 1.0)).ravel()


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--workloads", nargs="*", default=["llama3_8b_32k", "qwen3_32b_ragged"])
    ap.add_argument("--rules", nargs="*", default=["1e-3,1e-4,5", "1e-2,1e-3,5", "1e-5,1e-3,5"])
    ap.add_argument("--traversal", default="dense", choices=["dense", "key_norm"],
                    help="the workload's own order, or every block in descending key norm "
                         "(lists from the list oracle)")
    args = ap.parse_args(argv)
    print("| workload | g | traversal | tau | phi | p | reading | blocks read % | rel L2 mean | "
          "p99 | max |")
    print("|---|---|---|---|---|---|---|---|---|---|---|")
    for name in args.workloads:
        spec = W.WORKLOADS[name]
        wl = W.make_workload(spec, device="cpu")
        if args.traversal == "key_norm":
            from oracle import lists as OL
            r = OL.block_list(wl.q, wl.k_cache, wl.page_table, wl.seq_lens,
                              block_size=spec.block_size, num_q_heads=spec.num_q_heads,
                              budget=1 << 20)
            import torch
            wl.block_list = torch.from_numpy(r["list"])
            wl.block_list_len = torch.from_numpy(r["len"])
        total = int(np.sum(wl.traversal_lengths()))
        full = oracle.decode_workload(wl, tau=0.0)["out"]
        for rule in args.rules:
            tau, phi, p = (float(x) for x in rule.split(","))
            for per_head in (False, True):
                r = oracle.decode_workload(wl, tau=tau, phi=phi, patience=int(p),
                                           per_head_stop=per_head)
                e = _rel(r["out"], full)
                print(f"| {name} | {spec.group_size} | {args.traversal} | {tau:g} | {phi:g} | {int(p)} | "
                      f"{'per query head' if per_head else 'per group (AND)'} | "
                      f"{100 * r['stop'].sum() / total:.1f} | {e.mean():.2e} | "
                      f"{np.percentile(e, 99):.2e} | {e.max():.2e} |", flush=True)


if __name__ == "__main__":
    main()
