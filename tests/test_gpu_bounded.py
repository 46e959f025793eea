"""Bounded speculation (max_ahead_chunks) on the GPU (needs a gfx950 GPU).

With a window of n chunks, chunk k of a traversal is loaded only once chunk
k - n has been through the stability test, or a stop before chunk k is
known.  The window changes which blocks are read and when, never the
arithmetic: every output must be bit for bit the unbounded call's, whatever
the window, the chunking, the traversal or the mode.  The small cases are
compared with the oracle as well."""
from __future__ import annotations

import sys

import pytest
import torch

from helpers import random_lists, small_workload
from parity import compare_workload, host_copy
from paper_2606_00024_amd import _lib, api, workloads as W

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
WINDOWS = (1, 2, 4)


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
    (91, 1, 2, 4, 8192, 64, 64, False),
    (92, 2, 2, 1, (700, 3000), 64, 16, False),
    (93, 2, 2, 8, (1900, 4049), 64, 128, True),
    (94, 1, 2, 16, 3000, 64, 32, False),
    (95, 3, 1, 4, (1, 65, 2640), 128, 16, False),
    (96, 2, 2, 4, (6000, 777), 64, 16, True),
]
THRESHOLDS = [(1e-3, 1e-4, 5), (0.05, 1e-3, 2), (0.0, 1e-4, 5)]


def _case(c):
    seed, B, hkv, g, L, bk, ps, lists = c
    wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, block_size=bk,
                        page_size=ps, needles=2)
    if lists:
        wl.block_list, wl.block_list_len = random_lists(wl, seed, fraction=0.6)
    return _to_dev(wl)


def _run(wl, tau, phi, p, **kw):
    _say(f"  gpu call: {wl.spec.name} B={wl.spec.batch} g={wl.spec.group_size} "
         f"tau={tau} phi={phi} p={p} {kw}")
    r = api.decode_workload(wl, tau=tau, phi=phi, patience=p, **kw)
    torch.cuda.synchronize()
    return r


def _same(a, b):
    return all(torch.equal(x, y) for x, y in zip(a, b))


@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
@pytest.mark.parametrize("thr", THRESHOLDS, ids=["cfg", "relaxed", "off"])
def test_window_changes_no_bit(case, thr):
    wl = _case(case)
    host = host_copy(wl)
    for chunk in (0, 1):
        ref = _run(wl, *thr, chunk_blocks=chunk)
        for wnd in WINDOWS:
            got = _run(wl, *thr, chunk_blocks=chunk, max_ahead_chunks=wnd)
            assert _same(ref, got), f"window {wnd}, chunk_blocks {chunk}"
        rep = compare_workload(wl, got, tau=thr[0], phi=thr[1], patience=thr[2], host=host,
                               name="bounded_matrix")
        assert rep.ok(), str(rep)


@pytest.mark.parametrize("mode", ["per_head_stop", "no_detector"])
def test_window_in_the_other_modes(mode):
    wl = _case(CASES[0])
    kw = {mode: True}
    for thr in THRESHOLDS[:2]:
        ref = _run(wl, *thr, chunk_blocks=1, **kw)
        for wnd in WINDOWS:
            assert _same(ref, _run(wl, *thr, chunk_blocks=1, max_ahead_chunks=wnd, **kw)), wnd


@pytest.mark.parametrize("name", ["llama3_8b_32k", "sparse25_128k", "long_512k"])
def test_window_full_size(name):
    """The full-size workloads in the launch configuration the benchmark
    times: every window it reports gives the unbounded call's bits."""
    spec = W.WORKLOADS[name]
    _say(f"  generating {name} on {DEV}")
    wl = W.make_workload(spec, device=DEV)
    torch.cuda.synchronize()
    ref = _run(wl, spec.tau, spec.phi, spec.patience)
    for wnd in (2, 4):
        assert _same(ref, _run(wl, spec.tau, spec.phi, spec.patience, max_ahead_chunks=wnd)), wnd
    del wl
    torch.cuda.empty_cache()
