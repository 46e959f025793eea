"""Pins of the oracle's per-query-head stopping (R3 variant): every query
head runs Eq. (3) and Algorithm 1's break on its own stable steps; its
output and lse are those of its own stop, and the group reads blocks until
its last head has stopped."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from bruteforce import Group, float32, prefix_outputs, step_metrics
from helpers import random_lists, small_workload

CASES = [
    (91, 1, 2, 4, 1500, 64, 16, False),
    (92, 2, 1, 8, 1300, 64, 64, False),
    (93, 2, 2, 4, 900, 64, 128, True),
]
RULES = [(0.05, 1e-3, 2), (0.02, 1e-2, 3), (0.2, 0.01, 1)]


def _head_stops(traj, tau, phi, p):
    """Stop of each head of one group from its own stable steps (brute force)."""
    T = len(traj) - 1
    g = traj[0].shape[0]
    stops = [T] * g
    runs = [0] * g
    done = [False] * g
    for t in range(1, T + 1):
        ds, dr = step_metrics(traj[t], traj[t - 1])
        for h in range(g):
            if done[h]:
                continue
            ok = bool(ds[h] < tau and dr[h] < phi)   # NaN direction compares false
            runs[h] = runs[h] + 1 if ok else 0
            if runs[h] >= p:
                stops[h], done[h] = t, True
    return stops


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("rule", RULES)
def test_per_head_stops_and_outputs_match_brute_force(case, rule):
    seed, B, hkv, g, L, bk, ps, lists = case
    tau, phi, p = rule
    wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, block_size=bk,
                        page_size=ps)
    if lists:
        wl.block_list, wl.block_list_len = random_lists(wl, seed)
    r = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p, per_head_stop=True)
    sp = wl.spec
    scale = float32(sp.softmax_scale)
    for b in range(sp.batch):
        for h in range(sp.num_kv_heads):
            grp = Group(wl.q, wl.k_cache, wl.v_cache, wl.page_table, wl.seq_lens, b, h,
                        sp.block_size, sp.dense_order, wl.block_list, wl.block_list_len)
            pre = prefix_outputs(grp, scale)
            stops = _head_stops(pre["o"], float32(tau), float32(phi), p)
            T = len(grp.blocks)
            if T == 0:
                continue
            assert r["head_stop"][b, h * g:(h + 1) * g].tolist() == stops
            assert int(r["stop"][b, h]) == max(stops)
            for i, st in enumerate(stops):
                np.testing.assert_allclose(r["out"][b, h * g + i], pre["o"][st][i], rtol=1e-12,
                                           atol=1e-12)
                np.testing.assert_allclose(r["lse"][b, h * g + i], pre["logA"][st][i], rtol=1e-12,
                                           atol=1e-12)


@pytest.mark.parametrize("rule", RULES)
def test_single_head_groups_are_unchanged(rule):
    wl = small_workload(94, batch=2, kv_heads=2, group=1, seq_len=(1200, 700))
    tau, phi, p = rule
    a = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p)
    b = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p, per_head_stop=True)
    np.testing.assert_array_equal(a["stop"], b["stop"])
    np.testing.assert_array_equal(a["out"], b["out"])
    np.testing.assert_array_equal(a["lse"], b["lse"])
    np.testing.assert_array_equal(b["head_stop"], b["stop"])


@pytest.mark.parametrize("rule", RULES)
def test_each_head_stops_no_later_than_the_group(rule):
    """A head's own run is at least the run of the AND over the group, so it
    stops no later; the group then reads no more blocks than the AND rule."""
    wl = small_workload(95, batch=2, kv_heads=2, group=8, seq_len=(3000, 2200))
    tau, phi, p = rule
    a = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p)
    b = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p, per_head_stop=True)
    g = 8
    for bb in range(2):
        for h in range(2):
            assert (b["head_stop"][bb, h * g:(h + 1) * g] <= a["stop"][bb, h]).all()
            assert b["stop"][bb, h] <= a["stop"][bb, h]


def test_interrupted_run_restarts_the_count():
    """Equal scores (K = 0), one query head, block values a = [1, 1, 1, 4, 1,
    1, 1, 1] * e_0 in traversal order: o(t) is the mean of a_1..a_t, i.e.
    1, 1, 1, 1.75, 1.6, 1.5, 10/7, 11/8, so d_scale(t >= 2) = 0, 0, 0.75,
    0.15, 0.1, 1/14, 3/56 and d_direction = 0.  With tau = 0.2 steps 2, 3 are
    stable, step 4 is not, steps 5.. are: p = 3 stops at 7 (the count restarts
    at step 4), not at 5.  Both readings of R3 agree for a single head."""
    from helpers import uniform_key_case
    vecs = []
    for a in [1, 1, 1, 4, 1, 1, 1, 1]:
        v = np.zeros(128)
        v[0] = a
        vecs.append(v)
    q, k, v, pt, sl = uniform_key_case(vecs)
    for per_head in (False, True):
        r = oracle.decode(q, k, v, pt, sl, block_size=64, scale=0.088, tau=0.2, phi=1e-6,
                          patience=3, per_head_stop=per_head)
        assert int(r["stop"][0, 0]) == 7
        np.testing.assert_allclose(r["out"][0, 0, 0], 10 / 7, rtol=1e-14)
        if per_head:
            assert int(r["head_stop"][0, 0]) == 7
