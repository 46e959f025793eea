"""Measurement sweeps of the decode call on one GPU.

For a workload, each mode is timed rep by rep: HIP events around every call,
warm-up first, the KV pool rotated over several identical copies so that
consecutive calls do not hit the last-level cache.  The median, p10 and p90
are reported.

  nodet      no stability test at all (no_detector): full attention
  off        the test runs on every block and never passes (tau = 0)
  never      workload thresholds, patience INT32_MAX: the test passes but never stops
  p1 .. p20  workload thresholds with patience 1, 2, 5, 10, 20

The detector's cost is off (or never) against nodet.  The modes that read
different amounts fit time = a + bytes / BW by least squares; the report gives
R^2, the fitted bandwidth and the intercept, and t_on / t_off against the
ideal bytes_on / bytes_off.

`--thresholds` sweeps (tau, phi) instead.  Each point reports the skipped
share, the time, and the relative L2 distance per query head from full
attention (the nodet output): mean, p99 and max.

    python -m paper_2606_00024_amd.sweep --workload llama3_8b_32k
    python -m paper_2606_00024_amd.sweep --workload qwen3_32b_ragged --thresholds
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np

INT32_MAX = 2 ** 31 - 1


class Caller:
    """Pre-marshalled decode calls on the current stream, the KV pool rotated
    over `copies` identical copies."""

    def __init__(self, wl, copies: int, **opt_kw):
        import torch
        from . import _lib, api
        self._lib = _lib
        s = wl.spec
        self.shape = api.make_shape(wl.q, wl.k_cache, wl.v_cache, wl.page_table,
                                    block_size=s.block_size, block_list=wl.block_list)
        self.opts = api.make_opts(softmax_scale=s.softmax_scale, dense_order=s.dense_order,
                                  **opt_kw)
        dev = wl.q.device
        B, Hq, D = wl.q.shape
        self.out = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
        self.lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
        self.stop = torch.empty((B, s.num_kv_heads), dtype=torch.int32, device=dev)
        self.ws = api.new_workspace(api.workspace_bytes(self.shape, self.opts), dev)
        pools = [(wl.k_cache, wl.v_cache)] + [(wl.k_cache.clone(), wl.v_cache.clone())
                                              for _ in range(copies - 1)]
        p = lambda t: 0 if t is None else int(t.data_ptr())
        self.args = [(p(wl.q), p(k), p(v), p(wl.page_table), p(wl.seq_lens), p(wl.block_list),
                      p(wl.block_list_len), p(self.out), p(self.lse), p(self.stop))
                     for k, v in pools]
        self.stream = torch.cuda.current_stream(dev).cuda_stream
        self.i = 0

    def __call__(self):
        a = self.args[self.i % len(self.args)]
        self.i += 1
        st = self._lib.decode_attention(self.shape, self.opts, *a, int(self.ws.data_ptr()),
                                        self.ws.numel(), self.stream)
        if st != 0:
            raise self._lib.ArtError(st, "art_decode_attention")


def time_reps(call, reps: int, warmup: int) -> np.ndarray:
    """Kernel-side milliseconds of each of `reps` calls (HIP events)."""
    import torch
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps)]
    for e0, e1 in evs:
        e0.record()
        call()
        e1.record()
    torch.cuda.synchronize()
    return np.array([e0.elapsed_time(e1) for e0, e1 in evs])


def kv_bytes_read(wl, stop: np.ndarray) -> int:
    """K and V bytes of the blocks consumed (every group, 512 B per token and
    KV head at head_dim 128)."""
    s = wl.spec
    lens = wl.seq_lens.cpu().numpy()
    total = 0
    bl = None if wl.block_list is None else wl.block_list.cpu().numpy()
    for b in range(s.batch):
        L = int(lens[b])
        nblk = (L + s.block_size - 1) // s.block_size
        for h in range(s.num_kv_heads):
            t = int(stop[b, h])
            if bl is None:
                ids = range(nblk - 1, nblk - 1 - t, -1) if s.dense_order == 0 else range(t)
            else:
                ids = bl[b, h, :t]
            for i in ids:
                total += (min((int(i) + 1) * s.block_size, L) - int(i) * s.block_size)
    return total * s.head_dim * 2 * 2


def fit_line(x: np.ndarray, y: np.ndarray) -> dict:
    """Least-squares y = a + b x: intercept a, slope b, R^2."""
    A = np.stack([np.ones_like(x), x], axis=1)
    coef, *_ = np.linalg.lstsq(A, y, rcond=None)
    pred = A @ coef
    ss_res = float(((y - pred) ** 2).sum())
    ss_tot = float(((y - y.mean()) ** 2).sum())
    return {"a": float(coef[0]), "b": float(coef[1]),
            "r2": 1.0 - ss_res / ss_tot if ss_tot > 0 else 1.0}


def _summary(ms: np.ndarray) -> dict:
    return {"median_ms": float(np.median(ms)), "p10_ms": float(np.percentile(ms, 10)),
            "p90_ms": float(np.percentile(ms, 90))}


def patience_sweep(wl, reps: int = 100, warmup: int = 20, copies: int = 4) -> dict:
    import torch
    s = wl.spec
    modes = [("nodet", dict(tau=0.0, phi=0.0, patience=1, no_detector=True)),
             ("off", dict(tau=0.0, phi=s.phi, patience=s.patience)),
             ("never", dict(tau=s.tau, phi=s.phi, patience=INT32_MAX))]
    modes += [(f"p{p}", dict(tau=s.tau, phi=s.phi, patience=p)) for p in (1, 2, 5, 10, 20)]
    total = int(np.sum(wl.traversal_lengths()))
    rows = []
    for name, kw in modes:
        call = Caller(wl, copies, **kw)
        call()
        torch.cuda.synchronize()
        stop = call.stop.cpu().numpy()
        ms = time_reps(call, reps, warmup)
        row = {"mode": name, **{k: v for k, v in kw.items()}, **_summary(ms),
               "blocks_read": int(stop.sum()), "skipped_pct": 100.0 * (1 - stop.sum() / total),
               "kv_bytes": kv_bytes_read(wl, stop)}
        rows.append(row)
        print(json.dumps(row), flush=True)
        del call
        torch.cuda.empty_cache()
    by = {r["mode"]: r for r in rows}
    fit_rows = [r for r in rows if r["mode"] != "nodet"]
    x = np.array([r["kv_bytes"] for r in fit_rows], dtype=np.float64)
    y = np.array([r["median_ms"] for r in fit_rows], dtype=np.float64) * 1e-3
    fit = fit_line(x, y)
    out = {"workload": s.name, "rows": rows,
           "fit": {**fit, "bandwidth_gbps": (1.0 / fit["b"] / 1e9) if fit["b"] > 0 else None,
                   "intercept_ms": fit["a"] * 1e3},
           "detector_overhead_pct": {
               "off_vs_nodet": 100.0 * (by["off"]["median_ms"] / by["nodet"]["median_ms"] - 1),
               "never_vs_nodet": 100.0 * (by["never"]["median_ms"] / by["nodet"]["median_ms"] - 1)},
           "proportionality": [
               {"mode": r["mode"], "t_over_t_off": r["median_ms"] / by["off"]["median_ms"],
                "bytes_over_bytes_off": r["kv_bytes"] / by["off"]["kv_bytes"]}
               for r in rows if r["mode"].startswith("p")]}
    return out


def threshold_sweep(wl, points, reps: int = 50, warmup: int = 10, copies: int = 4) -> dict:
    import torch
    s = wl.spec
    ref = Caller(wl, 1, tau=0.0, phi=0.0, patience=1, no_detector=True)
    ref()
    torch.cuda.synchronize()
    full = ref.out.cpu().numpy().astype(np.float64)
    t_full = _summary(time_reps(ref, reps, warmup))
    del ref
    total = int(np.sum(wl.traversal_lengths()))
    rows = []
    for tau, phi in points:
        call = Caller(wl, copies, tau=tau, phi=phi, patience=s.patience)
        call()
        torch.cuda.synchronize()
        out = call.out.cpu().numpy().astype(np.float64)
        stop = call.stop.cpu().numpy()
        num = np.linalg.norm(out - full, axis=-1)
        den = np.linalg.norm(full, axis=-1)
        rel = (num / np.where(den > 0, den, 1.0)).ravel()
        row = {"tau": tau, "phi": phi, "patience": s.patience,
               **_summary(time_reps(call, reps, warmup)),
               "skipped_pct": 100.0 * (1 - stop.sum() / total),
               "rel_l2_mean": float(rel.mean()), "rel_l2_p99": float(np.percentile(rel, 99)),
               "rel_l2_max": float(rel.max())}
        rows.append(row)
        print(json.dumps(row), flush=True)
        del call
        torch.cuda.empty_cache()
    return {"workload": s.name, "full_attention": t_full, "rows": rows}


def main(argv=None) -> int:
    from . import workloads as W
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="llama3_8b_32k")
    ap.add_argument("--thresholds", action="store_true")
    ap.add_argument("--reps", type=int, default=100)
    ap.add_argument("--json", default=None)
    args = ap.parse_args(argv)
    spec = W.WORKLOADS[args.workload]
    wl = W.make_workload(spec, device="cuda:0")
    if args.thresholds:
        pts = [(t, f) for t, f in W.RAGGED_SWEEP] if spec.name == "qwen3_32b_ragged" else \
            [(1e-2, 1e-2), (1e-3, 1e-3), (1e-4, 1e-4), (1e-5, 1e-3), (spec.tau, spec.phi)]
        res = threshold_sweep(wl, pts, reps=max(10, args.reps // 2))
    else:
        res = patience_sweep(wl, reps=args.reps)
    print(json.dumps({k: v for k, v in res.items() if k != "rows"}), flush=True)
    if args.json:
        with open(args.json, "w") as f:
            json.dump(res, f, indent=1)
    return 0


if __name__ == "__main__":
    sys.exit(main())
