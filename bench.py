#!/usr/bin/env python3
"""Benchmark: ART decode attention on one MI355X.

A step is one call of art_decode_attention: the whole path (block loads,
scores, online softmax, P.V, the per-block stability test, patience and the
early exit) over one decode step of a workload.  The headline workload is
the Qwen3-32B-shaped ragged batch: 32 sequences of U{8192..65536} cached
tokens, 64 query / 8 KV heads, head_dim 128, KV block 64, paged KV (page 64,
pages permuted in one pool), recency-first order, tau = phi = 1e-3 (the
middle of the swept thresholds), patience 5.  Inputs are resident in HBM;
workloads smaller than 4 GiB rotate over several identical KV copies so that
consecutive steps do not hit the 256 MB last-level cache.

Prints one JSON line.  ``value`` is the effective KV tokens*heads/s: tokens
of the traversal set (the whole cache, skipped blocks included) times KV
heads, divided by wall time per step.  The line also carries the rate on the
tokens actually read, HBM GB/s on the bytes the result needs, the fraction
of KV blocks skipped, the distance of the output from full attention, the
same figures with termination off (tau = 0: the test runs on every block and
never fires), the threshold sweep, the other workloads, the roofline of the
kernel against the published 8 TB/s and against the read ceiling measured in
the same process, and the CPU oracle timed on bounded samples.
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
HEADLINE = "qwen3_32b_ragged"
# windows of the bounded-speculation runs reported for the other workloads
BOUNDED_WINDOWS = (2, 4, 8)
# the ragged batch's thresholds: the middle of the swept set (tau = phi)
HEADLINE_THRESHOLDS = {"qwen3_32b_ragged": (1e-3, 1e-3)}

# HBM bytes per launch of the decode kernel counted by rocprofv3 (FETCH_SIZE
# scaled by 2.0 plus WRITE_SIZE scaled by 1.0: the factors a plain 1 GiB
# device copy gives for those counters), per workload, thresholds and mode.
# They hold only for the sources they were counted on, identified by
# SHA-256; after any change to those sources the figure is reported as null
# until it is counted again.
COUNTED_TRAFFIC = {
    "sources_sha256": "3137134c6e20c2541cae53f3dcfa1fee65d807cb3caa59ae744aa91886ff435f",
    "bytes": {('qwen3_32b_ragged', 0.001, 0.001, 'on'): 5349924464,
              ('qwen3_32b_ragged', 0.0, 0.001, 'off'): 5360532552,
              ('llama3_8b_32k', 0.001, 0.0001, 'on'): 526330752,
              ('llama3_8b_32k', 0.0, 0.0001, 'off'): 1104039264,
              ('sparse25_128k', 0.001, 0.0001, 'on'): 258422056,
              ('sparse25_128k', 0.0, 0.0001, 'off'): 553799584,
              ('long_512k', 0.001, 0.0001, 'on'): 637014960,
              ('long_512k', 0.0, 0.0001, 'off'): 2176522672,
              ('tiny_4k', 0.001, 0.0001, 'on'): 5259592,
              ('tiny_4k', 0.0, 0.0001, 'off'): 5227968,
              ('llama3_8b_32k', 0.001, 0.0001, 'on_ahead2'): 301494608,
              ('llama3_8b_32k', 0.001, 0.0001, 'on_ahead4'): 336663528,
              ('llama3_8b_32k', 0.001, 0.0001, 'on_ahead8'): 406983560,
              ('sparse25_128k', 0.001, 0.0001, 'on_ahead2'): 36665128,
              ('sparse25_128k', 0.001, 0.0001, 'on_ahead4'): 56437576,
              ('sparse25_128k', 0.001, 0.0001, 'on_ahead8'): 94122560,
              ('long_512k', 0.001, 0.0001, 'on_ahead2'): 192246744,
              ('long_512k', 0.001, 0.0001, 'on_ahead4'): 198173840,
              ('long_512k', 0.001, 0.0001, 'on_ahead8'): 216227440},
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


def counted_traffic(key):
    if sources_digest() != COUNTED_TRAFFIC["sources_sha256"]:
        return None
    return COUNTED_TRAFFIC["bytes"].get(key)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--copies", type=int, default=0,
                    help="KV pool copies rotated across steps (0: enough for 4 GiB, at most 8)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-off", action="store_true", help="skip the termination-off run")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the threshold sweep, the other workloads and the read ceiling")
    ap.add_argument("--only-headline", action="store_true",
                    help="time the headline mode only (for profiling the same launches)")
    ap.add_argument("--tau", type=float, default=None)
    ap.add_argument("--phi", type=float, default=None)
    ap.add_argument("--patience", type=int, default=None)
    ap.add_argument("--chunk-blocks", type=int, default=0)
    ap.add_argument("--max-ahead", type=int, default=0,
                    help="bound the chunks read ahead of the last tested one (0 = unbounded)")
    ap.add_argument("--no-detector", action="store_true",
                    help="the headline mode without the stability test (full attention)")
    ap.add_argument("--list-producer", action="store_true",
                    help="measure the device-side traversal-list producer (block scores and "
                         "selection) on the workload's shape instead of the decode step")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (the reference kernel for "
                         "scaling rocprofv3 FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


def thresholds(spec, args=None):
    tau, phi = HEADLINE_THRESHOLDS.get(spec.name, (spec.tau, spec.phi))
    pat = spec.patience
    if args is not None:
        tau = tau if args.tau is None else args.tau
        phi = phi if args.phi is None else args.phi
        pat = pat if args.patience is None else args.patience
    return tau, phi, pat


class Runner:
    """Pre-marshalled calls of the C ABI on torch's current stream.  Every
    call of a timed run writes its own stop_block buffer, so that the run
    can check afterwards that every call stopped every group alike."""

    def __init__(self, wl, copies, tau, phi, patience, chunk_blocks, no_detector=False,
                 n_stop_bufs=1, max_ahead=0):
        import torch
        from paper_2606_00024_amd import _lib, api
        self._lib = _lib
        self.api = api
        s = wl.spec
        self.wl = wl
        self.shape = api.make_shape(wl.q, wl.k_cache, wl.v_cache, wl.page_table,
                                    block_size=s.block_size, block_list=wl.block_list)
        self.opts = api.make_opts(softmax_scale=s.softmax_scale, tau=tau, phi=phi,
                                  patience=patience, dense_order=s.dense_order,
                                  chunk_blocks=chunk_blocks, no_detector=no_detector,
                                  max_ahead_chunks=max_ahead)
        dev = wl.q.device
        B, Hq, D = wl.q.shape
        self.out = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
        self.lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
        self.stops = torch.full((max(1, n_stop_bufs), B, s.num_kv_heads), -1, dtype=torch.int32,
                                device=dev)
        self.ws_bytes = api.workspace_bytes(self.shape, self.opts)
        self.ws = api.new_workspace(self.ws_bytes, dev)
        self.pools = [(wl.k_cache, wl.v_cache)] + [
            (wl.k_cache.clone(), wl.v_cache.clone()) for _ in range(copies - 1)]
        self.stream = torch.cuda.current_stream(dev).cuda_stream
        p = lambda t: 0 if t is None else int(t.data_ptr())
        self.args = [(p(wl.q), p(k), p(v), p(wl.page_table), p(wl.seq_lens), p(wl.block_list),
                      p(wl.block_list_len), p(self.out), p(self.lse)) for k, v in self.pools]
        self.stop_ptrs = [int(self.stops[i].data_ptr()) for i in range(self.stops.shape[0])]
        self.ws_ptr = int(self.ws.data_ptr())
        self.i = 0

    @property
    def stop(self):
        return self.stops[0]

    def step(self, buf=0):
        a = self.args[self.i % len(self.args)]
        self.i += 1
        st = self._lib.decode_attention(self.shape, self.opts, *a, self.stop_ptrs[buf], self.ws_ptr,
                                        self.ws.numel(), self.stream)
        if st != 0:
            raise self._lib.ArtError(st, "art_decode_attention")

    def check(self, n_bufs):
        """After a timed run: no wait gave up, and every call left the same
        stop_block (a call whose kernel gave up would not)."""
        status = self.api.workspace_status(self.ws)
        if status != self._lib.OK:
            raise RuntimeError(f"timed run: workspace status {self._lib.status_str(status)}")
        import torch
        st = self.stops[:n_bufs]
        if not bool((st == st[0]).all()) or bool((st[0] < 0).any()):
            raise RuntimeError("timed run: stop_block differs between calls")


def default_copies(wl):
    """KV pool copies rotated over consecutive steps: enough that the copies
    together hold 4 GiB (at most 8), so that the blocks one step reads were
    not read by the step before it from the 256 MB last-level cache."""
    pool = (wl.k_cache.numel() + wl.v_cache.numel()) * 2
    return max(1, min(8, math.ceil((4 << 30) / max(pool, 1))))


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
    """HIP events around every launch, on the stream the launches go to."""
    import torch
    for _ in range(warmup):
        runner.step()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    n_bufs = runner.stops.shape[0]
    t0 = time.perf_counter()
    for i, (e0, e1) in enumerate(evs):
        e0.record()
        runner.step(i % n_bufs)
        e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    runner.check(min(steps, n_bufs))
    per = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    spread = {"kernel_ms_p10": per[int(0.1 * (steps - 1))], "kernel_ms_p50": per[(steps - 1) // 2],
              "kernel_ms_p90": per[int(0.9 * (steps - 1))]}
    return wall, sum(per) / steps, spread


def measure(wl, tau, phi, pat, steps, warmup, copies, chunk_blocks=0, no_detector=False,
            keep_out=False, max_ahead=0):
    """One mode of one workload: kernel time, rates, skipped share."""
    import torch
    run = Runner(wl, copies, tau, phi, pat, chunk_blocks, no_detector, n_stop_bufs=steps,
                 max_ahead=max_ahead)
    print(f"[bench] {wl.spec.name}: tau={tau} phi={phi} p={pat} steps={steps}"
          f"{' no_detector' if no_detector else ''}"
          f"{f' max_ahead={max_ahead}' if max_ahead else ''}", file=sys.stderr, flush=True)
    wall, kern_ms, spread = time_steps(run, steps, warmup)
    alg, read_tokens, blocks = algorithmic_bytes(wl, run.stop)
    total_blocks = sum(map(sum, wl.traversal_lengths()))
    eligible = wl.kv_bytes_in_traversal() // (2 * wl.spec.head_dim * 2)
    res = {
        "ms_per_step": wall / steps * 1e3,
        "kernel_ms": kern_ms,
        **spread,
        "effective_tokens_heads_per_s": eligible / (wall / steps),
        "read_tokens_heads_per_s": read_tokens / (wall / steps),
        "hbm_gbps_on_bytes_read": alg / (kern_ms * 1e-3) / 1e9,
        "skipped_pct": 100.0 * (1 - blocks / total_blocks),
        "blocks_read": blocks, "blocks_total": total_blocks,
        "alg_bytes_per_launch": alg,
    }
    out = run.out.clone() if keep_out else None
    # the caching allocator keeps the freed buffers for the next mode's
    # runner: memory handed back to the driver and mapped again made the
    # launches that followed up to 1-2 % slower than steady state
    del run
    return res, out


def distance_from_full(out_on, out_full):
    """Relative L2 distance per query head of the output from full attention
    (termination off): mean, p99, max."""
    import torch
    num = torch.linalg.vector_norm((out_on - out_full).double(), dim=-1).flatten()
    den = torch.linalg.vector_norm(out_full.double(), dim=-1).flatten()
    rel = torch.where(den > 0, num / den.clamp_min(1e-300), num).cpu().numpy()
    import numpy as np
    return {"rel_l2_mean": float(rel.mean()), "rel_l2_p99": float(np.quantile(rel, 0.99)),
            "rel_l2_max": float(rel.max()), "heads": int(rel.size)}


def read_ceiling():
    """The HBM read rate a plain read-only streaming kernel reaches in this
    process (16 KiB pieces, 64 KiB in flight per workgroup): 4 GiB read
    sequentially, and the same pieces in a random order (pages of a pool,
    as the decode kernel reads them).  Median of 10 launches each."""
    import ctypes
    import torch
    from paper_2606_00024_amd import build
    lib = ctypes.CDLL(build.BENCH_LIB)
    lib.art_bench_read.restype = ctypes.c_int
    lib.art_bench_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                   ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    piece = int(lib.art_bench_piece_bytes())
    nbytes = 4 << 30
    n = nbytes // piece
    buf = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    perm = torch.randperm(n, generator=torch.Generator().manual_seed(1)).to(torch.int32).to("cuda:0")
    props = torch.cuda.get_device_properties(0)
    grid = props.multi_processor_count * 8
    sink = torch.empty(grid * 256, dtype=torch.int32, device="cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    out = {"bytes": nbytes, "piece_bytes": piece, "workgroups": grid}
    for name, lst in (("sequential", None), ("random_pieces", perm)):
        def call():
            rc = lib.art_bench_read(int(buf.data_ptr()), n, 0 if lst is None else int(lst.data_ptr()),
                                    grid, int(sink.data_ptr()), stream)
            if rc != 0:
                raise RuntimeError(f"art_bench_read: hip error {rc}")
        call()
        torch.cuda.synchronize()
        ts = []
        for _ in range(10):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            call()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        out[f"{name}_gbps"] = nbytes / (sorted(ts)[len(ts) // 2] * 1e-3) / 1e9
    del buf, perm, sink
    torch.cuda.empty_cache()
    out["gbps"] = max(out["sequential_gbps"], out["random_pieces_gbps"])
    return out


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, tau, phi, pat):
    """The oracle (fp64 C, OpenMP over the (sequence, KV head) groups), as it
    stands, on bounded samples of the same workload: every group with all
    threads, and the first two groups with one thread; termination on (the
    bench thresholds) and off; each the median of three runs.  Rates are KV
    tokens*heads of the traversal set of the sampled groups per second."""
    import numpy as np
    import oracle
    s = wl.spec
    host = dict(q=wl.q.cpu(), k=wl.k_cache.cpu(), v=wl.v_cache.cpu(), pt=wl.page_table.cpu(),
                sl=wl.seq_lens.cpu(),
                bl=None if wl.block_list is None else wl.block_list.cpu(),
                bll=None if wl.block_list_len is None else wl.block_list_len.cpu())
    lens = np.asarray(wl.traversal_lengths())
    Bk = s.block_size
    seq = host["sl"].numpy()

    def tokens_of(mask):
        # tokens in the traversal sets of the masked groups
        tot = 0
        for b in range(s.batch):
            for h in range(s.num_kv_heads):
                if mask[b, h]:
                    if host["bl"] is None:
                        tot += int(seq[b])
                    else:
                        ids = host["bl"][b, h, : int(lens[b, h])].numpy()
                        tot += int(sum(min(Bk, int(seq[b]) - int(i) * Bk) for i in ids))
        return tot

    all_mask = np.ones((s.batch, s.num_kv_heads), dtype=np.uint8)
    two = np.zeros_like(all_mask)
    two.reshape(-1)[:2] = 1
    threads = oracle.max_threads()
    res = {"unit": "KV tokens·heads/s", "kind": "oracle", "cpu_model": cpu_model(),
           "nproc": os.cpu_count(), "threads_all": threads}
    for label, mask, nt in (("all", all_mask, threads), ("one_thread", two, 1)):
        for mode, t in (("on", tau), ("off", 0.0)):
            times = []
            for _ in range(3):
                t0 = time.perf_counter()
                oracle.decode(host["q"], host["k"], host["v"], host["pt"], host["sl"],
                              block_size=Bk, scale=s.softmax_scale, tau=t, phi=phi, patience=pat,
                              dense_order=s.dense_order, block_list=host["bl"],
                              block_list_len=host["bll"], group_mask=mask, num_threads=nt)
                times.append(time.perf_counter() - t0)
            med = sorted(times)[1]
            res[f"{label}_{mode}"] = {"seconds_median": med, "tokens_heads": tokens_of(mask),
                                      "value": tokens_of(mask) / med, "threads": nt,
                                      "groups": int(mask.sum())}
    res["value"] = res["all_on"]["value"]
    res["cores"] = threads
    res["sample"] = (f"whole step (all {s.batch * s.num_kv_heads} groups) with {threads} OpenMP "
                     f"threads and the first 2 groups with 1 thread, termination on "
                     f"(tau={tau}, phi={phi}) and off, median of 3 runs each; "
                     f"value = all groups, termination on")
    return res


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


def workload_config(spec, wl, W, tau, phi, pat, copies):
    lens = W.resolve_seq_lens(spec)
    return {"workload": spec.name, "batch": spec.batch, "q_heads": spec.num_q_heads,
            "kv_heads": spec.num_kv_heads, "head_dim": spec.head_dim,
            "seq_lens": (list(spec.seq_lens) if spec.seq_lens[0] == "uniform"
                         else sorted(set(lens))),
            "tokens_total": int(sum(lens)),
            "block_size": spec.block_size, "page_size": spec.page_size,
            "traversal": "block_list" if wl.block_list is not None else "recent_first",
            "tau": tau, "phi": phi, "patience": pat, "accumulate": "fp32",
            "kv_copies_rotated": copies, "seed": spec.seed}


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
    tau, phi, pat = thresholds(spec, args)
    print(f"[bench] generating {args.workload}", file=sys.stderr, flush=True)
    wl = W.make_workload(spec, device="cuda:0")
    torch.cuda.synchronize()
    copies = args.copies or default_copies(wl)
    # the read ceiling is measured after the decode runs: run before them,
    # its 4 GiB buffer (allocated, read and freed) left the first hundred or
    # so decode launches that followed about 2 % slower than every later one
    ceiling = None

    on, out_on = measure(wl, tau, phi, pat, args.steps, args.warmup, copies, args.chunk_blocks,
                         args.no_detector, keep_out=True, max_ahead=args.max_ahead)
    if args.only_headline:
        print(json.dumps({"workload": spec.name, "tau": tau, "phi": phi, "patience": pat,
                          "no_detector": args.no_detector, "max_ahead": args.max_ahead, **on}),
              flush=True)
        return
    off = None
    out_full = None
    if not args.no_off:
        off, out_full = measure(wl, 0.0, phi, pat, max(10, args.steps // 2),
                                max(5, args.warmup // 2), copies, args.chunk_blocks, keep_out=True)
    defaults = (tau, phi, pat) == thresholds(spec) and args.chunk_blocks == 0 \
        and not args.no_detector and args.max_ahead == 0

    def roofline(r, key):
        ach = r["hbm_gbps_on_bytes_read"]
        traffic = counted_traffic(key) if defaults else None
        out = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
               "frac": ach / HBM_PEAK_GBPS, "traffic": traffic,
               "kernel": f"art_decode_kernel<{spec.group_size}>", "kernel_ms": r["kernel_ms"],
               "alg_bytes_per_launch": r["alg_bytes_per_launch"]}
        if ceiling is not None:
            out["measured_read_gbps"] = ceiling["gbps"]
            out["frac_of_measured_read"] = ach / ceiling["gbps"]
        if traffic is not None:
            # the rate at which the counted bytes (reads past each stop
            # included) move: how busy HBM is, as opposed to how much of
            # what it moves the result needs
            out["traffic_gbps"] = traffic / (r["kernel_ms"] * 1e-3) / 1e9
            out["traffic_frac"] = out["traffic_gbps"] / HBM_PEAK_GBPS
        return out

    quality = None if out_full is None else distance_from_full(out_on, out_full)

    sweep = None
    if not args.no_extra and spec.name == HEADLINE and out_full is not None:
        sweep = []
        for t, f in W.RAGGED_SWEEP:
            r, o = measure(wl, t, f, pat, 30, 10, copies, keep_out=True)
            sweep.append({"tau": t, "phi": f, "kernel_ms": r["kernel_ms"],
                          "skipped_pct": r["skipped_pct"],
                          "hbm_gbps_on_bytes_read": r["hbm_gbps_on_bytes_read"],
                          "frac": r["hbm_gbps_on_bytes_read"] / HBM_PEAK_GBPS,
                          "effective_tokens_heads_per_s": r["effective_tokens_heads_per_s"],
                          **distance_from_full(o, out_full)})
            del o
    cpu = None if args.no_cpu else cpu_baseline(wl, tau, phi, pat)
    cfg = workload_config(spec, wl, W, tau, phi, pat, copies)
    del wl, out_on, out_full
    torch.cuda.empty_cache()

    others = None
    if not args.no_extra:
        others = {}
        for name in ("llama3_8b_32k", "sparse25_128k", "long_512k", "tiny_4k"):
            if name == spec.name:
                continue
            ospec = W.WORKLOADS[name]
            print(f"[bench] generating {name}", file=sys.stderr, flush=True)
            owl = W.make_workload(ospec, device="cuda:0")
            ot, of, op = thresholds(ospec)
            oc = default_copies(owl)
            r_on, _ = measure(owl, ot, of, op, 40, 10, oc)
            r_off, _ = measure(owl, 0.0, of, op, 40, 10, oc)
            entry = {"config": workload_config(ospec, owl, W, ot, of, op, oc)}
            for mode, r, key in (("on", r_on, (name, ot, of, "on")), ("off", r_off, (name, 0.0, of, "off"))):
                entry[mode] = {k: r[k] for k in ("kernel_ms", "kernel_ms_p50", "skipped_pct",
                                                 "hbm_gbps_on_bytes_read",
                                                 "effective_tokens_heads_per_s",
                                                 "alg_bytes_per_launch")}
                entry[mode]["frac"] = r["hbm_gbps_on_bytes_read"] / HBM_PEAK_GBPS
                entry[mode]["traffic"] = counted_traffic(key)
            # bounded speculation (max_ahead_chunks), termination on: the
            # same results, fewer reads past the stops, possibly idle workgroups
            entry["on_max_ahead"] = {}
            for wnd in BOUNDED_WINDOWS:
                r_b, _ = measure(owl, ot, of, op, 40, 10, oc, max_ahead=wnd)
                entry["on_max_ahead"][str(wnd)] = {
                    "kernel_ms": r_b["kernel_ms"], "skipped_pct": r_b["skipped_pct"],
                    "traffic": counted_traffic((name, ot, of, f"on_ahead{wnd}"))}
            others[name] = entry
            del owl
            torch.cuda.empty_cache()

    if not args.no_extra:
        ceiling = read_ceiling()
        for entry in (others or {}).values():
            for mode in ("on", "off"):
                entry[mode]["frac_of_measured_read"] = entry[mode]["hbm_gbps_on_bytes_read"] / ceiling["gbps"]

    line = {
        "metric": "decode-attn KV tokens·heads/s; achieved HBM GB/s on bytes read; % KV blocks skipped",
        "value": on["effective_tokens_heads_per_s"],
        "unit": "KV tokens·heads/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": on["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": cfg,
        "hbm_gbps_on_bytes_read": on["hbm_gbps_on_bytes_read"],
        "skipped_pct": on["skipped_pct"],
        "read_tokens_heads_per_s": on["read_tokens_heads_per_s"],
        "kernel_ms": on["kernel_ms"],
        "kernel_ms_p10": on["kernel_ms_p10"], "kernel_ms_p50": on["kernel_ms_p50"],
        "kernel_ms_p90": on["kernel_ms_p90"],
        "distance_from_full_attention": quality,
        "roofline": roofline(on, (spec.name, tau, phi, "on")),
        "cpu_baseline": cpu,
        "termination_off": None if off is None else dict(off, roofline=roofline(off, (spec.name, 0.0, phi, "off"))),
        "read_ceiling": ceiling,
        "threshold_sweep": sweep,
        "other_workloads": others,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
