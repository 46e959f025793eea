"""The cross-workgroup protocol under injected delays (needs a gfx950 GPU).

libart_stress.so is the same library built with ART_RACE_STRESS: at every
point where one workgroup hands data to another (flag publications, the
stop announcement, a loader marking its part of a chunk done) or acts on
what another handed over (after a look-back found its state, before the
stability fold reads the flags again), a wave sleeps a pseudo-random 0 to
7 times 8128 cycles keyed by the call, the group, the chunk and the site.
Chunks of one block, long traversals and repeated calls (each call draws
other delays) make producers and consumers of the look-back meet in orders
a plain run rarely shows.  Every result must still equal the oracle's, and
no wait may give up.  The run stops at the first mismatch (pytest -x)."""
from __future__ import annotations

import math
import sys

import pytest
import torch

from helpers import random_lists, small_workload
from parity import compare_per_head, compare_workload, host_copy
from paper_2606_00024_amd import _lib, api, build

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def stress_lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return _lib.load_variant(build.STRESS_LIB)


def _to_dev(wl):
    for name in ("q", "k_cache", "v_cache", "page_table", "seq_lens", "block_list", "block_list_len"):
        t = getattr(wl, name)
        if t is not None:
            setattr(wl, name, t.to(DEV))
    return wl


CASES = [
    # seed, B, Hkv, g, seq_len(s), lists
    (91, 2, 2, 4, (9000, 6000), False),
    (92, 1, 2, 8, 12000, False),
    (93, 2, 1, 4, (8000, 7000), True),
    (94, 1, 4, 1, 10000, False),
]
THRESHOLDS = [(1e-3, 1e-4, 5), (0.05, 1e-3, 2), (0.0, 1e-4, 5), (0.02, math.inf, 3)]


@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_delayed_handovers_keep_the_sequential_result(stress_lib, case):
    seed, B, hkv, g, L, lists = case
    wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, needles=4)
    if lists:
        wl.block_list, wl.block_list_len = random_lists(wl, seed, fraction=0.7)
    _to_dev(wl)
    host = host_copy(wl)
    ws = api.new_workspace(64 << 20, DEV)
    with _lib.using(stress_lib):
        for thr in THRESHOLDS:
            for chunk in (1, 2):
                for rep_i in range(2):
                    _say(f"  stress call s{seed} thr={thr} chunk={chunk} rep={rep_i}")
                    gpu = api.decode_workload(wl, tau=thr[0], phi=thr[1], patience=thr[2],
                                              chunk_blocks=chunk, workspace=ws)
                    assert api.workspace_status(ws) == _lib.OK
                    rep = compare_workload(wl, gpu, tau=thr[0], phi=thr[1], patience=thr[2],
                                           host=host, name="race_stress")
                    assert rep.ok(), f"thr {thr} chunk {chunk} rep {rep_i}: {rep}"
            gpu = api.decode_workload(wl, tau=thr[0], phi=thr[1], patience=thr[2], chunk_blocks=1,
                                      per_head_stop=True, workspace=ws)
            assert api.workspace_status(ws) == _lib.OK
            rep = compare_per_head(wl, gpu, tau=thr[0], phi=thr[1], patience=thr[2], host=host,
                                   name="race_stress_per_head")
            assert rep.ok(), f"per head, thr {thr}: {rep}"


def test_look_first_under_delays(stress_lib):
    """128 groups of a few chunks each: the launch holds few chunks of a
    group at once, and a chunk then looks back once before it publishes its
    aggregate.  Delayed hand-overs must not change the result."""
    wl = _to_dev(small_workload(96, batch=32, kv_heads=4, group=4, seq_len=1500, needles=2))
    host = host_copy(wl)
    ws = api.new_workspace(64 << 20, DEV)
    with _lib.using(stress_lib):
        for thr in THRESHOLDS:
            for chunk in (0, 1):
                _say(f"  stress call s96 thr={thr} chunk={chunk}")
                gpu = api.decode_workload(wl, tau=thr[0], phi=thr[1], patience=thr[2],
                                          chunk_blocks=chunk, workspace=ws)
                assert api.workspace_status(ws) == _lib.OK
                rep = compare_workload(wl, gpu, tau=thr[0], phi=thr[1], patience=thr[2],
                                       host=host, name="race_stress")
                assert rep.ok(), f"thr {thr} chunk {chunk}: {rep}"


def test_the_stress_build_delays(stress_lib):
    """The delays are really there: the same one-block-chunk call takes
    clearly longer through the stress build than through the library."""
    import time
    wl = _to_dev(small_workload(95, batch=2, kv_heads=2, group=4, seq_len=(9000, 6000), needles=4))
    ws = api.new_workspace(64 << 20, DEV)

    def timed():
        ts = []
        for _ in range(5):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            api.decode_workload(wl, tau=0.0, phi=1e-4, patience=5, chunk_blocks=1, workspace=ws)
            torch.cuda.synchronize()
            ts.append(time.perf_counter() - t0)
        return sorted(ts)[2]
    plain = timed()
    with _lib.using(stress_lib):
        stressed = timed()
    _say(f"  one call: library {plain * 1e6:.0f} us, stress build {stressed * 1e6:.0f} us")
    assert stressed > 2 * plain
