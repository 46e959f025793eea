"""The call's options together, against the oracle (needs a gfx950 GPU).

Each seeded case turns on several options at once: the subsampled probe
(Sec. 3.2's x = P o, probe_stride), the accumulator reading of d_scale,
per-query-head stops, a block list, an explicit chunking and a speculation
window, on a random group size and shape.  The kernel takes each option on
its own path; this checks that they compose (the probe inside the per-head
replay, the accumulator with lists and short chunks, the window with either
reading) and give the oracle's result for the same options."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from helpers import random_lists, small_workload
from parity import compare_per_head, compare_workload
from paper_2606_00024_amd import _lib, api

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
N_CASES = 16
# the accumulator reading's d_scale grows with the mass consumed: its
# near-tie band is relative (as in the accumulator parity tests)
ACC_TAU_REL = 1e-3


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
    rng = np.random.default_rng(7100 + i)
    g = int(rng.choice([1, 2, 4, 8, 16]))
    hkv = int(rng.integers(1, 3))
    batch = int(rng.integers(1, 4))
    bk = int(rng.choice([64, 128]))
    ps = int(rng.choice([16, 32, 64]))
    lens = tuple(int(rng.integers(1, 2600)) for _ in range(batch))
    per_head = bool(rng.random() < 0.4)
    # the accumulator reading is a group-reading option of the oracle
    acc = (not per_head) and bool(rng.random() < 0.5)
    thr = ([(1.0, 1e-3, 2), (10.0, 1e-2, 3), (50.0, 1e-4, 5)] if acc
           else [(1e-3, 1e-4, 5), (0.05, 1e-3, 2), (0.02, 1e-2, 1)])[int(rng.integers(0, 3))]
    return dict(seed=7100 + i, g=g, hkv=hkv, batch=batch, bk=bk, ps=ps, lens=lens,
                lists=bool(rng.random() < 0.5), stride=int(rng.choice([1, 2, 4, 16])),
                acc=acc, per_head=per_head, thr=thr,
                chunk=int(rng.choice([0, 1, 2, 5])), ahead=int(rng.choice([0, 1, 3])))


@pytest.mark.parametrize("i", range(N_CASES))
def test_option_mix(i):
    c = _draw(i)
    wl = small_workload(c["seed"], batch=c["batch"], kv_heads=c["hkv"], group=c["g"],
                        seq_len=c["lens"], block_size=c["bk"], page_size=c["ps"], needles=2)
    if c["lists"]:
        wl.block_list, wl.block_list_len = random_lists(wl, c["seed"], fraction=0.5)
    for name in ("q", "k_cache", "v_cache", "page_table", "seq_lens", "block_list", "block_list_len"):
        t = getattr(wl, name)
        if t is not None:
            setattr(wl, name, t.to(DEV))
    tau, phi, p = c["thr"]
    _say(f"  case {i}: {c}")
    gpu = api.decode_workload(wl, tau=tau, phi=phi, patience=p, chunk_blocks=c["chunk"],
                              probe_stride=c["stride"], scale_of_accumulator=c["acc"],
                              per_head_stop=c["per_head"], max_ahead_chunks=c["ahead"])
    torch.cuda.synchronize()
    if c["per_head"]:
        rep = compare_per_head(wl, gpu, tau=tau, phi=phi, patience=p, probe_stride=c["stride"],
                               name="option_mix")
    else:
        rep = compare_workload(wl, gpu, tau=tau, phi=phi, patience=p, probe_stride=c["stride"],
                               scale_of_accumulator=c["acc"],
                               tau_rel=ACC_TAU_REL if c["acc"] else None, name="option_mix")
    _say("  ", rep)
    assert rep.ok(), f"case {i} {c}: {rep}"
