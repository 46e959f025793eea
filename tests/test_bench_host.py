"""Host-side pieces of bench.py: the algorithmic byte count, the guard on the
counted traffic, and the one-GPU contract (no GPU needed)."""
from __future__ import annotations

import os
import subprocess
import sys

import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2606_00024_amd import workloads as W  # noqa: E402


def _workload(lens, block_size=64, page_size=64, kv_heads=2, group=4, fraction=None):
    spec = W.WorkloadSpec(name="t", batch=len(lens), num_q_heads=kv_heads * group,
                          num_kv_heads=kv_heads, seq_lens=tuple(lens), block_size=block_size,
                          page_size=page_size, list_fraction=fraction, seed=5)
    return W.make_workload(spec, device="cpu")


def _fixed_bytes(wl, blocks, listed):
    """q, page-table and list entries of the consumed blocks, and the outputs."""
    s = wl.spec
    q = s.batch * s.num_q_heads * s.head_dim * 2
    idx = blocks * max(1, s.block_size // s.page_size) * 4 + (blocks * 4 if listed else 0)
    outs = s.batch * s.num_q_heads * (s.head_dim * 4 + 4) + s.batch * s.num_kv_heads * 4
    return q + idx + outs


def test_full_traversal_reads_every_token():
    lens = [1000, 4096, 65]
    wl = _workload(lens)
    T = [[-(-L // 64)] * 2 for L in lens]
    alg, tokens, blocks = bench.algorithmic_bytes(wl, torch.tensor(T, dtype=torch.int32))
    assert tokens == 2 * sum(lens)
    assert blocks == 2 * sum(-(-L // 64) for L in lens)
    assert alg == tokens * 2 * 128 * 2 + _fixed_bytes(wl, blocks, False)


def test_recency_first_stops_count_the_newest_blocks():
    """A stop after t blocks consumes the last t blocks: the partial tail
    block (recency-first comes first) counts only its tokens."""
    wl = _workload([1000])            # 16 blocks, the last one holds 40 tokens
    stop = torch.tensor([[1, 3]], dtype=torch.int32)
    _, tokens, blocks = bench.algorithmic_bytes(wl, stop)
    assert blocks == 4
    assert tokens == 40 + (40 + 64 + 64)


def test_list_traversal_counts_the_listed_blocks():
    wl = _workload([64 * 40], fraction=0.25)
    bl = wl.block_list
    stop = torch.tensor([[3, 0]], dtype=torch.int32)
    alg, tokens, blocks = bench.algorithmic_bytes(wl, stop)
    assert blocks == 3 and tokens == 3 * 64
    assert alg == tokens * 512 + _fixed_bytes(wl, blocks, True)
    assert int(bl[0, 0, 0]) >= 0


def test_counted_traffic_needs_the_counted_sources(monkeypatch):
    key = ("qwen3_32b_ragged", 1e-3, 1e-3, "on")
    table = {"sources_sha256": bench.sources_digest(), "bytes": {key: 123456}}
    monkeypatch.setattr(bench, "COUNTED_TRAFFIC", table)
    assert bench.counted_traffic(key) == 123456
    assert bench.counted_traffic(("qwen3_32b_ragged", 1e-2, 1e-2, "on")) is None
    monkeypatch.setattr(bench, "COUNTED_TRAFFIC", dict(table, sources_sha256="0" * 64))
    assert bench.counted_traffic(key) is None


def test_headline_is_the_largest_single_gpu_workload():
    """The default workload is the ragged g = 8 batch (the most KV bytes of
    the five), at the middle of its swept thresholds."""
    sizes = {}
    for name, spec in W.WORKLOADS.items():
        lens = W.resolve_seq_lens(spec)
        sizes[name] = sum(lens) * spec.num_kv_heads
    assert max(sizes, key=sizes.get) == bench.HEADLINE == "qwen3_32b_ragged"
    assert bench.thresholds(W.WORKLOADS[bench.HEADLINE]) == (1e-3, 1e-3, 5)
    assert (1e-3, 1e-3) in W.RAGGED_SWEEP


def test_distance_from_full_attention():
    full = torch.zeros((2, 3, 128), dtype=torch.float32)
    full[..., 0] = 1.0
    on = full.clone()
    on[0, 0, 1] = 0.5            # one head moved by half its norm
    d = bench.distance_from_full(on, full)
    assert d["heads"] == 6 and d["rel_l2_max"] == 0.5
    assert abs(d["rel_l2_mean"] - 0.5 / 6) < 1e-12


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_counted_traffic_is_current():
    """The committed counts were taken on the sources as they stand: a kernel
    or host change must come with a recount (else bench reports null)."""
    assert bench.COUNTED_TRAFFIC["sources_sha256"] == bench.sources_digest()
    for w in ("qwen3_32b_ragged", "llama3_8b_32k", "sparse25_128k", "long_512k"):
        tau, phi, _ = bench.thresholds(W.WORKLOADS[w])
        assert bench.counted_traffic((w, tau, phi, "on")) is not None
        assert bench.counted_traffic((w, 0.0, phi, "off")) is not None
