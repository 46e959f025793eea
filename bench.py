#!/usr/bin/env python3
"""Benchmark: ART decode attention on one MI355X.

A step is one call of art_decode_attention (the whole path: block loads,
scores, online softmax, P.V, the per-block stability test, patience and the
early exit) on the Llama-3-8B-shaped decode layer: batch 8, 32 query / 8 KV
heads, head_dim 128, 32768 cached tokens per sequence, KV block 64, paged KV
(page 64, pages permuted in one pool), recency-first order, tau = 1e-3,
phi = 1e-4, patience 5.  Inputs are resident in HBM; the KV pool is rotated
over several identical copies so that consecutive steps do not hit in the
256 MB last-level cache.

Prints one JSON line.  ``value`` is the effective KV tokens*heads/s: tokens
of the traversal set (the whole cache, skipped blocks included) times KV
heads, divided by wall time per step.  The line also carries the rate on
tokens actually read, HBM GB/s on bytes read, the fraction of KV blocks
skipped, the same figures with termination off (tau = 0: the detector runs
every block and never fires), the roofline of the kernel and the CPU oracle
timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0   # MI355X HBM3E, published

# HBM bytes per launch of the decode kernel counted by rocprofv3 (FETCH_SIZE
# scaled by 2.0 plus WRITE_SIZE scaled by 1.0: the factors a plain 1 GiB
# device copy gives for those counters), per workload and mode at the
# workload's default thresholds.  They hold only for the sources they were
# counted on, identified by SHA-256; after any change to those sources the
# figure is reported as null until it is counted again.
COUNTED_TRAFFIC = {
    "sources_sha256": "374e8816aebcec613912408d86293f6d71e1dfcffed62373d7b7235212b9fefa",
    "bytes": {("llama3_8b_32k", "on"): 541698816, ("llama3_8b_32k", "off"): 1120224000},
}
TRAFFIC_SOURCES = ("art_kernels.hip", "art_api.cpp", "art_internal.h")


def sources_digest():
    """SHA-256 of the kernel and host sources with comments and blank space
    removed (so that editing a comment does not invalidate a count)."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, "paper_2606_00024_amd", "csrc", f)) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def counted_traffic(workload, mode):
    if sources_digest() != COUNTED_TRAFFIC["sources_sha256"]:
        return None
    return COUNTED_TRAFFIC["bytes"].get((workload, mode))


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="llama3_8b_32k")
    ap.add_argument("--copies", type=int, default=4, help="KV pool copies rotated across steps")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-off", action="store_true", help="skip the termination-off run")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--tau", type=float, default=None)
    ap.add_argument("--phi", type=float, default=None)
    ap.add_argument("--patience", type=int, default=None)
    ap.add_argument("--chunk-blocks", type=int, default=0)
    ap.add_argument("--list-producer", action="store_true",
                    help="measure the device-side traversal-list producer (block scores and "
                         "selection) on the workload's shape instead of the decode step")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (the reference kernel for "
                         "scaling rocprofv3 FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


class Runner:
    """Pre-marshalled calls of the C ABI on torch's current stream."""

    def __init__(self, wl, copies, tau, phi, patience, chunk_blocks):
        import torch
        from paper_2606_00024_amd import _lib, api
        self._lib = _lib
        s = wl.spec
        self.wl = wl
        self.shape = api.make_shape(wl.q, wl.k_cache, wl.v_cache, wl.page_table,
                                    block_size=s.block_size, block_list=wl.block_list)
        self.opts = api.make_opts(softmax_scale=s.softmax_scale, tau=tau, phi=phi,
                                  patience=patience, dense_order=s.dense_order,
                                  chunk_blocks=chunk_blocks)
        dev = wl.q.device
        B, Hq, D = wl.q.shape
        self.out = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
        self.lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
        self.stop = torch.empty((B, s.num_kv_heads), dtype=torch.int32, device=dev)
        self.ws_bytes = api.workspace_bytes(self.shape, self.opts)
        self.ws = api.new_workspace(self.ws_bytes, dev)
        self.pools = [(wl.k_cache, wl.v_cache)] + [
            (wl.k_cache.clone(), wl.v_cache.clone()) for _ in range(copies - 1)]
        self.stream = torch.cuda.current_stream(dev).cuda_stream
        p = lambda t: 0 if t is None else int(t.data_ptr())
        self.args = [(p(wl.q), p(k), p(v), p(wl.page_table), p(wl.seq_lens), p(wl.block_list),
                      p(wl.block_list_len), p(self.out), p(self.lse), p(self.stop))
                     for k, v in self.pools]
        self.ws_ptr = int(self.ws.data_ptr())
        self.i = 0

    def step(self):
        a = self.args[self.i % len(self.args)]
        self.i += 1
        st = self._lib.decode_attention(self.shape, self.opts, *a, self.ws_ptr,
                                        self.ws.numel(), self.stream)
        if st != 0:
            raise self._lib.ArtError(st, "art_decode_attention")


def algorithmic_bytes(wl, stop):
    """Bytes one launch must move: K+V bf16 of every token in the consumed
    blocks, q, the page-table entries and list entries of those blocks, and
    the outputs (fp32 out, lse, stop_block)."""
    s = wl.spec
    lens = wl.seq_lens.cpu().tolist()
    stop = stop.cpu().tolist()
    Bk, Ps = s.block_size, s.page_size
    tokens = 0
    blocks = 0
    bl = wl.block_list.cpu() if wl.block_list is not None else None
    for b, L in enumerate(lens):
        nblk = -(-L // Bk)
        for h in range(s.num_kv_heads):
            t = stop[b][h]
            blocks += t
            if bl is None:
                order = range(nblk - 1, nblk - 1 - t, -1) if s.dense_order == 0 else range(t)
            else:
                order = bl[b, h, :t].tolist()
            for blk in order:
                tokens += min(Bk, L - blk * Bk)
    kv = tokens * 2 * s.head_dim * 2
    q = s.batch * s.num_q_heads * s.head_dim * 2
    idx = blocks * max(1, Bk // Ps) * 4 + (blocks * 4 if bl is not None else 0)
    outs = s.batch * s.num_q_heads * (s.head_dim * 4 + 4) + s.batch * s.num_kv_heads * 4
    return kv + q + idx + outs, tokens, blocks


def time_steps(runner, steps, warmup):
    import torch
    for _ in range(warmup):
        runner.step()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    t0 = time.perf_counter()
    for e0, e1 in evs:
        e0.record()
        runner.step()
        e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    time_steps.last = {"kernel_ms_p10": per[int(0.1 * (steps - 1))], "kernel_ms_p50": per[(steps - 1) // 2],
                       "kernel_ms_p90": per[int(0.9 * (steps - 1))]}
    return wall, sum(per) / steps


def cpu_baseline(wl, eligible_tokens, tau, phi, patience, budget_s):
    """The oracle (fp64 C, OpenMP over the (sequence, KV head) groups) on the
    same workload, repeated whole until the time budget is used (at least
    once): a bounded sample of steps."""
    import oracle
    s = wl.spec
    host = dict(q=wl.q.cpu(), k=wl.k_cache.cpu(), v=wl.v_cache.cpu(), pt=wl.page_table.cpu(),
                sl=wl.seq_lens.cpu(),
                bl=None if wl.block_list is None else wl.block_list.cpu(),
                bll=None if wl.block_list_len is None else wl.block_list_len.cpu())
    threads = oracle.max_threads()
    reps, elapsed = 0, 0.0
    while reps == 0 or elapsed < budget_s:
        t = time.perf_counter()
        oracle.decode(host["q"], host["k"], host["v"], host["pt"], host["sl"],
                      block_size=s.block_size, scale=s.softmax_scale, tau=tau, phi=phi,
                      patience=patience, dense_order=s.dense_order, block_list=host["bl"],
                      block_list_len=host["bll"], num_threads=threads)
        elapsed += time.perf_counter() - t
        reps += 1
    return {"value": eligible_tokens * reps / elapsed, "unit": "KV tokens·heads/s",
            "cores": threads, "kind": "oracle",
            "sample": f"{reps} whole step(s) of the same workload (all {s.batch * s.num_kv_heads} "
                      f"groups, same thresholds) in {elapsed:.1f}s, {threads} OpenMP threads"}


def list_producer_leg(args):
    """Importance lists (25 % of the blocks, first and last forced) for the
    workload's shape: kernel time per call and the achieved HBM rate on the
    key bytes the scores read (every token of every group: 256 bytes)."""
    import torch
    from paper_2606_00024_amd import _lib, api, workloads as W
    spec = W.WORKLOADS[args.workload]
    print(f"[bench] generating {args.workload}", file=sys.stderr, flush=True)
    wl = W.make_workload(spec, device="cuda:0")
    s = spec
    B, Hkv = s.batch, s.num_kv_heads
    lens = wl.seq_lens.cpu().tolist()
    max_blocks = (int(wl.page_table.shape[1]) * s.page_size + s.block_size - 1) // s.block_size
    budget = max(1, max_blocks // 4)
    bl = torch.full((B, Hkv, max_blocks), -1, dtype=torch.int32, device="cuda:0")
    bll = torch.zeros((B, Hkv), dtype=torch.int32, device="cuda:0")
    scores = torch.empty((B, Hkv, max_blocks), dtype=torch.float64, device="cuda:0")
    shape = api.make_shape(wl.q, wl.k_cache, wl.k_cache, wl.page_table, block_size=s.block_size,
                           block_list=bl)
    stream = torch.cuda.current_stream().cuda_stream
    key_bytes = sum(lens) * Hkv * s.head_dim * 2
    out = {"metric": "traversal-list producer: key bytes read per second", "unit": "GB/s",
           "config": {"workload": args.workload, "batch": B, "kv_heads": Hkv,
                      "q_heads": s.num_q_heads, "seq_lens": sorted(set(lens)),
                      "block_size": s.block_size, "max_blocks": max_blocks, "budget": budget,
                      "sink_blocks": 1, "keep_last": 1},
           "key_bytes": key_bytes, "steps": args.steps, "warmup": args.warmup}
    for name, kind in (("key_norm", _lib.SCORE_KEY_NORM), ("query_bound", _lib.SCORE_QUERY_BOUND)):
        opts = _lib.ListOpts(policy=_lib.LIST_IMPORTANCE, score_kind=kind, budget=budget,
                             sink_blocks=1, keep_last=1)

        def call():
            st = _lib.build_block_list(shape, opts, int(wl.q.data_ptr()), int(wl.k_cache.data_ptr()),
                                       int(wl.page_table.data_ptr()), int(wl.seq_lens.data_ptr()),
                                       int(bl.data_ptr()), int(bll.data_ptr()),
                                       int(scores.data_ptr()), 0, 0, stream)
            if st != 0:
                raise _lib.ArtError(st, "art_build_block_list")
        for _ in range(args.warmup):
            call()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            call()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        out[name] = {"ms_per_call": ms, "key_gbps": key_bytes / (ms * 1e-3) / 1e9,
                     "frac_of_8tbs": key_bytes / (ms * 1e-3) / 8e12}
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the path shards "
              "by (sequence, KV head) group with no exchange, so one GPU's share is the "
              "single-GPU run", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_00024_amd import workloads as W

    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "copies": 3}), flush=True)
        return

    if args.list_producer:
        list_producer_leg(args)
        return

    spec = W.WORKLOADS[args.workload]
    tau = spec.tau if args.tau is None else args.tau
    phi = spec.phi if args.phi is None else args.phi
    pat = spec.patience if args.patience is None else args.patience
    print(f"[bench] generating {args.workload}", file=sys.stderr, flush=True)
    wl = W.make_workload(spec, device="cuda:0")
    torch.cuda.synchronize()
    # tokens*heads in the traversal set (the whole cache for the dense order)
    eligible_tokens = wl.kv_bytes_in_traversal() // (2 * spec.head_dim * 2)

    def measure(t, f, p, steps, warmup):
        run = Runner(wl, args.copies, t, f, p, args.chunk_blocks)
        print(f"[bench] timing tau={t} phi={f} p={p} steps={steps}", file=sys.stderr, flush=True)
        wall, kern_ms = time_steps(run, steps, warmup)
        spread = dict(time_steps.last)
        alg, read_tokens, blocks = algorithmic_bytes(wl, run.stop)
        total_blocks = sum(map(sum, wl.traversal_lengths()))
        ms = wall / steps * 1e3
        res = {
            "ms_per_step": ms,
            "kernel_ms": kern_ms,
            **spread,
            "effective_tokens_heads_per_s": eligible_tokens / (wall / steps),
            "read_tokens_heads_per_s": read_tokens / (wall / steps),
            "hbm_gbps_on_bytes_read": alg / (kern_ms * 1e-3) / 1e9,
            "skipped_pct": 100.0 * (1 - blocks / total_blocks),
            "blocks_read": blocks, "blocks_total": total_blocks,
            "alg_bytes_per_launch": alg,
        }
        del run
        torch.cuda.empty_cache()
        return res

    # a measured ceiling beside the published one: a plain device copy of
    # 1 GiB (read plus written bytes over its HIP-event time, median of 10)
    def copy_rate_gbps():
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        ts = []
        for _ in range(10):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            dst.copy_(src)
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        del src, dst
        torch.cuda.empty_cache()
        return 2 * (1 << 30) / (sorted(ts)[len(ts) // 2] * 1e-3) / 1e9

    copy_gbps = copy_rate_gbps()
    on = measure(tau, phi, pat, args.steps, args.warmup)
    off = None if args.no_off else measure(0.0, phi, pat, max(5, args.steps // 2), max(2, args.warmup // 2))
    cpu = None if args.no_cpu else cpu_baseline(wl, eligible_tokens, tau, phi, pat, args.cpu_seconds)

    defaults = (tau, phi, pat) == (spec.tau, spec.phi, spec.patience) and args.chunk_blocks == 0

    def roofline(r, mode):
        ach = r["hbm_gbps_on_bytes_read"]
        traffic = counted_traffic(args.workload, mode) if defaults else None
        out = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
               "frac": ach / HBM_PEAK_GBPS, "traffic": traffic,
               "kernel": f"art_decode_kernel<{spec.group_size}>", "kernel_ms": r["kernel_ms"],
               "alg_bytes_per_launch": r["alg_bytes_per_launch"],
               "measured_copy_gbps": copy_gbps, "frac_of_measured_copy": ach / copy_gbps}
        if traffic is not None:
            # the rate at which the counted bytes (reads past each stop
            # included) move: how busy HBM is, as opposed to how much of
            # what it moves the result needs
            out["traffic_gbps"] = traffic / (r["kernel_ms"] * 1e-3) / 1e9
            out["traffic_frac"] = out["traffic_gbps"] / HBM_PEAK_GBPS
        return out

    line = {
        "metric": "decode-attn KV tokens·heads/s; achieved HBM GB/s on bytes read; % KV blocks skipped",
        "value": on["effective_tokens_heads_per_s"],
        "unit": "KV tokens·heads/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": on["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "batch": spec.batch, "q_heads": spec.num_q_heads,
                   "kv_heads": spec.num_kv_heads, "head_dim": spec.head_dim,
                   "seq_lens": sorted(set(W.resolve_seq_lens(spec)))[:1] if spec.seq_lens[0] != "uniform" else list(spec.seq_lens),
                   "block_size": spec.block_size, "page_size": spec.page_size,
                   "traversal": "block_list" if wl.block_list is not None else "recent_first",
                   "tau": tau, "phi": phi, "patience": pat, "accumulate": "fp32",
                   "kv_copies_rotated": args.copies},
        "hbm_gbps_on_bytes_read": on["hbm_gbps_on_bytes_read"],
        "skipped_pct": on["skipped_pct"],
        "read_tokens_heads_per_s": on["read_tokens_heads_per_s"],
        "kernel_ms": on["kernel_ms"],
        "kernel_ms_p10": on["kernel_ms_p10"], "kernel_ms_p50": on["kernel_ms_p50"],
        "kernel_ms_p90": on["kernel_ms_p90"],
        "roofline": roofline(on, "on"),
        "cpu_baseline": cpu,
        "termination_off": None if off is None else dict(off, roofline=roofline(off, "off")),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
