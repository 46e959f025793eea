"""Agreement of the subsampled probe with the full-output test (Appendix B).

The stability test of Eq. (2) can look at the whole normalised output of each
query head (P = I) or at a subsample of its coordinates (``probe_stride``).
Appendix B measures how often the cheap probe takes the same stopping decision
as the full-output detector.  This module runs both on the GPU path over
seeded synthetic workloads and classifies every (sequence, KV head) group:

* agree -- both stop at the same block, or neither stops;
* FP    -- the probe stops earlier than the full-output test, or stops where
           it never does (premature: the only case that can cost accuracy);
* FN    -- the full-output test stops earlier, or stops where the probe never
           does (conservative: costs speed only);
* delta_blk -- for groups where both stop but at different blocks, the
           distance between the two stopping blocks.

A stop at the last block of a traversal consumes every block, exactly as no
stop does, and the call reports the same stop_block = T for both; it is
therefore counted as "does not stop".  Groups with an empty traversal are
left out.

Run ``python -m paper_2606_00024_amd.agreement --help`` for the sweep.
"""
from __future__ import annotations

import argparse
import json
import sys
from dataclasses import dataclass, field
from typing import Iterable, Sequence

import numpy as np


@dataclass
class Agreement:
    groups: int = 0
    agree: int = 0
    fp: int = 0
    fn: int = 0
    both_stop_differ: list = field(default_factory=list)  # |stop_probe - stop_full|
    probe_blocks: int = 0      # blocks consumed with the probe
    full_blocks: int = 0       # blocks consumed with the full-output test
    total_blocks: int = 0      # blocks of the traversal sets

    def rates(self) -> dict:
        n = max(1, self.groups)
        d = np.asarray(self.both_stop_differ, dtype=np.float64)
        return {
            "groups": self.groups,
            "agree_pct": 100.0 * self.agree / n,
            "fp_pct": 100.0 * self.fp / n,
            "fn_pct": 100.0 * self.fn / n,
            "delta_blk_mean": float(d.mean()) if d.size else None,
            "delta_blk_std": float(d.std()) if d.size else None,
            "delta_blk_n": int(d.size),
            "skipped_pct_probe": 100.0 * (1 - self.probe_blocks / max(1, self.total_blocks)),
            "skipped_pct_full": 100.0 * (1 - self.full_blocks / max(1, self.total_blocks)),
        }


def classify(stop_probe: Sequence[int], stop_full: Sequence[int], lengths: Sequence[int],
             into: Agreement | None = None) -> Agreement:
    """Classify each group from its two stop_block values and traversal
    length T (all flat sequences of the same size)."""
    a = into or Agreement()
    sp = np.asarray(stop_probe, dtype=np.int64).ravel()
    sf = np.asarray(stop_full, dtype=np.int64).ravel()
    T = np.asarray(lengths, dtype=np.int64).ravel()
    if not (sp.shape == sf.shape == T.shape):
        raise ValueError("stop_probe, stop_full and lengths must have the same size")
    for p, f, t in zip(sp.tolist(), sf.tolist(), T.tolist()):
        if t <= 0:
            continue
        if not (1 <= p <= t and 1 <= f <= t):
            raise ValueError(f"stop values ({p}, {f}) outside [1, {t}]")
        a.groups += 1
        a.probe_blocks += p
        a.full_blocks += f
        a.total_blocks += t
        if p == f:
            a.agree += 1
        elif p < f:
            a.fp += 1
        else:
            a.fn += 1
        if p != f and p < t and f < t:
            a.both_stop_differ.append(abs(p - f))
    return a


def length_sweep_specs(lengths=(1024, 2048, 4096, 8192, 32768), batch=32, seed=40):
    """Needle-in-the-middle workloads of increasing length (Llama-3-8B heads,
    32/8): the eight needles of each (sequence, KV head) lie in the middle
    tenth of the context, as in the length study of Appendix B."""
    from . import workloads as W
    specs = []
    for i, L in enumerate(lengths):
        specs.append(W.WorkloadSpec(
            name=f"niah_mid_{L // 1024}k", batch=batch, num_q_heads=32, num_kv_heads=8,
            seq_lens=(L,) * batch, needle_bands=((8, 0.45, 0.55),), seed=seed + i))
    return specs


def measure(spec, strides: Iterable[int], thresholds: Iterable[tuple], device="cuda:0",
            seeds: Iterable[int] = (0,), rescale_tau: Iterable[bool] = (False, True)) -> list[dict]:
    """Run the GPU path with the full-output test and with each probe stride
    on ``spec`` (once per seed offset) and classify every group.

    d_scale is an absolute norm, and the norm of m of the D coordinates of a
    vector is about sqrt(m / D) of the whole one when its energy is spread
    evenly; never more.  With the same tau the probe's scale test is thus
    looser than the full output's.  ``rescale_tau`` True runs the probe with
    tau * sqrt(m / D) instead, the matched threshold for spread increments
    (d_direction is a ratio and keeps phi)."""
    import torch
    from dataclasses import replace
    from . import api, workloads as W
    rows = []
    strides = list(strides)
    thresholds = list(thresholds)
    rescale_tau = list(rescale_tau)
    acc = {(s, thr, rs): Agreement() for s in strides for thr in thresholds for rs in rescale_tau}
    for sd in seeds:
        wl = W.make_workload(replace(spec, seed=spec.seed + 1000 * sd), device=device)
        T = np.asarray(wl.traversal_lengths(), dtype=np.int64)
        for thr in thresholds:
            tau, phi, p = thr
            full = api.decode_workload(wl, tau=tau, phi=phi, patience=p)[2].cpu().numpy()
            for s in strides:
                for rs in rescale_tau:
                    tau_p = tau * (1.0 / s) ** 0.5 if rs else tau
                    probe = api.decode_workload(wl, tau=tau_p, phi=phi, patience=p,
                                                probe_stride=s)[2].cpu().numpy()
                    classify(probe, full, T, into=acc[(s, thr, rs)])
        del wl
        torch.cuda.empty_cache()
    for (s, thr, rs), a in acc.items():
        r = {"workload": spec.name, "probe_stride": s, "probe_dims": spec.head_dim // s,
             "tau": thr[0], "tau_probe": thr[0] * (1.0 / s) ** 0.5 if rs else thr[0],
             "phi": thr[1], "patience": thr[2]}
        r.update(a.rates())
        rows.append(r)
    return rows


def _fmt(x, nd=2):
    if x is None:
        return "-"
    return f"{x:.{nd}f}"


def markdown(rows: list[dict]) -> str:
    head = ("| workload | m | tau | probe tau | phi | p | groups | agree % | FP % | FN % | "
            "delta_blk (mean ± std, n) | skipped % probe / full |\n"
            "|---|---|---|---|---|---|---|---|---|---|---|---|\n")
    body = ""
    for r in rows:
        d = ("-" if r["delta_blk_mean"] is None else
             f"{r['delta_blk_mean']:.2f} ± {r['delta_blk_std']:.2f} ({r['delta_blk_n']})")
        body += (f"| {r['workload']} | {r['probe_dims']} | {r['tau']:g} | "
                 f"{r.get('tau_probe', r['tau']):.3g} | {r['phi']:g} | "
                 f"{r['patience']} | {r['groups']} | {_fmt(r['agree_pct'])} | {_fmt(r['fp_pct'])} | "
                 f"{_fmt(r['fn_pct'])} | {d} | {_fmt(r['skipped_pct_probe'], 1)} / "
                 f"{_fmt(r['skipped_pct_full'], 1)} |\n")
    return head + body


def main(argv=None) -> int:
    from . import workloads as W
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workloads", nargs="*", default=["lengths", "llama3_8b_32k", "qwen3_32b_ragged"],
                    help="named workloads, or 'lengths' for the needle-in-the-middle length sweep")
    ap.add_argument("--strides", type=int, nargs="*", default=[4, 8, 16])
    ap.add_argument("--seeds", type=int, default=2, help="seed offsets per workload")
    ap.add_argument("--json", default=None, help="also write the rows to this file")
    args = ap.parse_args(argv)
    rows = []
    for name in args.workloads:
        specs = length_sweep_specs() if name == "lengths" else [W.WORKLOADS[name]]
        for spec in specs:
            if spec.name == "qwen3_32b_ragged":
                thrs = [(t, f, spec.patience) for t, f in W.RAGGED_SWEEP]
            else:
                thrs = [(spec.tau, spec.phi, spec.patience), (1e-5, 1e-3, 5)]
            got = measure(spec, args.strides, thrs, seeds=range(args.seeds))
            for r in got:
                print(json.dumps(r), flush=True)
            rows += got
    print(markdown(rows), flush=True)
    if args.json:
        with open(args.json, "w") as f:
            json.dump(rows, f, indent=1)
    return 0


if __name__ == "__main__":
    sys.exit(main())
