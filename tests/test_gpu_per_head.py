"""Per-query-head termination (per_head_stop) on the GPU against the
oracle's per-head reading (needs a gfx950 GPU).

Every query head keeps its own patience counter and stops on its own;
stop_block is [batch][num_q_heads] and must equal the oracle's per-head stop
bit for bit except at near-ties of that head; out and lse are those at the
head's own stop (tests/parity.py compare_per_head)."""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest
import torch

from helpers import random_lists, small_workload
from parity import compare_per_head, host_copy
from paper_2606_00024_amd import _lib, api, workloads as W

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    _lib.load()
    yield


def _to_dev(wl):
    for name in ("q", "k_cache", "v_cache", "page_table", "seq_lens", "block_list", "block_list_len"):
        t = getattr(wl, name)
        if t is not None:
            setattr(wl, name, t.to(DEV))
    return wl


CASES = [
    # seed, B, Hkv, g, seq_len(s), Bk, Ps, lists
    (81, 1, 2, 4, 4096, 64, 64, False),
    (82, 2, 2, 1, (700, 1500), 64, 16, False),
    (83, 1, 2, 2, 1500, 128, 64, False),
    (84, 2, 2, 8, (900, 2049), 64, 128, True),
    (85, 1, 2, 16, 3000, 64, 32, False),
    (86, 3, 1, 4, (1, 65, 640), 64, 16, False),
    (87, 2, 2, 4, (3000, 777), 128, 16, True),
]
THRESHOLDS = [(1e-3, 1e-4, 5), (0.05, 1e-3, 2), (0.0, 1e-4, 5), (0.02, math.inf, 1)]


def _case(c):
    seed, B, hkv, g, L, bk, ps, lists = c
    wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, block_size=bk,
                        page_size=ps, needles=2)
    if lists:
        wl.block_list, wl.block_list_len = random_lists(wl, seed, fraction=0.6)
    return _to_dev(wl)


def _run(wl, tau, phi, p, **kw):
    _say(f"  gpu call (per head): {wl.spec.name} B={wl.spec.batch} g={wl.spec.group_size} "
         f"tau={tau} phi={phi} p={p} {kw}")
    r = api.decode_workload(wl, tau=tau, phi=phi, patience=p, per_head_stop=True, **kw)
    torch.cuda.synchronize()
    return r


@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
@pytest.mark.parametrize("thr", THRESHOLDS, ids=["cfg", "relaxed", "off", "scale_only_p1"])
def test_per_head_matrix(case, thr):
    wl = _case(case)
    host = host_copy(wl)
    for chunk in (0, 1, 3):
        gpu = _run(wl, *thr, chunk_blocks=chunk)
        assert gpu[2].shape == (wl.spec.batch, wl.spec.num_q_heads)
        rep = compare_per_head(wl, gpu, tau=thr[0], phi=thr[1], patience=thr[2], host=host,
                               name="per_head_matrix")
        _say("  ", chunk, rep)
        assert rep.ok(), str(rep)


def test_single_head_groups_match_the_group_reading():
    """g = 1: a group is one head, so both readings give the same bits."""
    wl = _case(CASES[1])
    for thr in THRESHOLDS[:2]:
        a = _run(wl, *thr)
        b = api.decode_workload(wl, tau=thr[0], phi=thr[1], patience=thr[2])
        torch.cuda.synchronize()
        for x, y in zip(a, b):
            assert torch.equal(x, y)


def test_heads_stop_no_later_than_the_group():
    """A head's own run of stable steps is at least the group's (the AND over
    heads), so each head stops no later than the group reading stops."""
    wl = _case(CASES[0])
    g = wl.spec.group_size
    for thr in THRESHOLDS[:2]:
        heads = _run(wl, *thr)[2].cpu().numpy()
        group = api.decode_workload(wl, tau=thr[0], phi=thr[1], patience=thr[2])[2].cpu().numpy()
        torch.cuda.synchronize()
        assert np.all(heads.reshape(group.shape[0], group.shape[1], g).max(axis=2) <= group)


@pytest.mark.parametrize("name,tau,phi", [("llama3_8b_32k", 1e-3, 1e-4), ("qwen3_32b_ragged", 1e-2, 1e-2)])
def test_per_head_full_size_every_group(name, tau, phi):
    spec = W.WORKLOADS[name]
    _say(f"  generating {name} on {DEV}")
    wl = W.make_workload(spec, device=DEV)
    torch.cuda.synchronize()
    host = host_copy(wl)
    gpu = _run(wl, tau, phi, spec.patience)
    rep = compare_per_head(wl, gpu, tau=tau, phi=phi, patience=spec.patience, host=host,
                           name=f"full:per_head:{name}")
    _say("  ", rep)
    assert rep.ok(), str(rep)
    assert rep.groups == spec.batch * spec.num_q_heads
    del wl, host
    torch.cuda.empty_cache()
