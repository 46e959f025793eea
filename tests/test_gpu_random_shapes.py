"""Seeded random shapes against the oracle (needs a gfx950 GPU).

Each case draws a group size, batch, KV heads, block and page sizes,
sequence lengths (empty and one-token sequences included), a dense order or
random block lists, a chunking, thresholds and the call options
(per-query-head stops, bounded speculation), and compares the GPU call with
the oracle on every group.  Unused pages of the pool hold NaN, so a read of
a wrong page shows in the output."""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest
import torch

from helpers import random_lists, small_workload
from parity import compare_per_head, compare_workload, host_copy
from paper_2606_00024_amd import _lib, api

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
N_CASES = 40
THRESHOLDS = [(1e-3, 1e-4, 5), (0.05, 1e-3, 2), (0.02, math.inf, 1), (0.1, 0.1, 3), (0.0, 1e-4, 5)]


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    _lib.load()
    yield


def _draw(i):
    rng = np.random.default_rng(9000 + i)
    g = int(rng.choice([1, 2, 4, 8, 16]))
    hkv = int(rng.integers(1, 3 if g == 16 else 5))
    batch = int(rng.integers(1, 5))
    bk = int(rng.choice([64, 128, 192, 256]))
    ps = int(rng.choice([16, 32, 64] if bk == 192 else [16, 32, 64, 128, 256]))
    lens = []
    for _ in range(batch):
        r = rng.random()
        lens.append(0 if r < 0.08 else 1 if r < 0.14 else int(rng.integers(2, 3200)))
    if max(lens) == 0:
        lens[0] = int(rng.integers(64, 2000))
    return dict(seed=9000 + i, g=g, hkv=hkv, batch=batch, bk=bk, ps=ps, lens=tuple(lens),
                order=int(rng.integers(0, 2)), lists=bool(rng.random() < 0.3),
                fraction=float(rng.uniform(0.2, 0.9)),
                thr=THRESHOLDS[int(rng.integers(0, len(THRESHOLDS)))],
                chunk=int(rng.choice([0, 0, 1, 2, 3, 5, 9])),
                per_head=bool(rng.random() < 0.15),
                ahead=int(rng.choice([0, 0, 0, 1, 3])))


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_shape(i):
    c = _draw(i)
    wl = small_workload(c["seed"], batch=c["batch"], kv_heads=c["hkv"], group=c["g"],
                        seq_len=c["lens"], block_size=c["bk"], page_size=c["ps"],
                        dense_order=c["order"], needles=2)
    if c["lists"]:
        wl.block_list, wl.block_list_len = random_lists(wl, c["seed"], fraction=c["fraction"])
    for name in ("q", "k_cache", "v_cache", "page_table", "seq_lens", "block_list", "block_list_len"):
        t = getattr(wl, name)
        if t is not None:
            setattr(wl, name, t.to(DEV))
    host = host_copy(wl)
    tau, phi, p = c["thr"]
    _say(f"  case {i}: {c}")
    gpu = api.decode_workload(wl, tau=tau, phi=phi, patience=p, chunk_blocks=c["chunk"],
                              per_head_stop=c["per_head"], max_ahead_chunks=c["ahead"])
    torch.cuda.synchronize()
    if c["per_head"]:
        rep = compare_per_head(wl, gpu, tau=tau, phi=phi, patience=p, host=host,
                               name="random_shapes")
    else:
        rep = compare_workload(wl, gpu, tau=tau, phi=phi, patience=p, host=host,
                               name="random_shapes")
    assert rep.ok(), f"case {i} {c}: {rep}"
