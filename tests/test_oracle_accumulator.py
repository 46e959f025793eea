"""Pins of the oracle's accumulator reading of d_scale (R2 variant): the
magnitude test on X(t) = l(t) o(t), the unnormalised accumulator with
l(t) = sum of exp(s - running max) over the consumed tokens, each step in
its own reference.  Brute force recomputes l(t) and o(t) from scratch for
every prefix; the closed form uses equal scores, where l(t) counts tokens."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from bruteforce import Group, float32, prefix_outputs, stop_from_trajectory
from helpers import random_lists, small_workload, uniform_key_case


def _accumulator_trajectory(grp: Group, scale: float):
    """X(t) = l(t) o(t) for t = 0..T (X(0) = 0), by direct evaluation."""
    o = prefix_outputs(grp, scale)["o"]
    xs = [o[0]]
    for t in range(1, len(grp.blocks) + 1):
        toks = grp.tokens_of(grp.blocks[:t])
        s = scale * (grp.q @ grp.K[toks].T)                   # [g][n]
        ell = np.exp(s - s.max(axis=1, keepdims=True)).sum(axis=1)
        xs.append(o[t] * ell[:, None])
    return xs


CASES = [
    (81, 1, 2, 4, 1000, 64, 16, False),
    (82, 2, 1, 2, 1300, 64, 64, False),
    (83, 2, 2, 8, 900, 64, 128, True),
]


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("thr", [(5.0, 1e-3, 2), (20.0, 1e-2, 3), (1.0, 0.05, 1)])
def test_bruteforce_stop_and_trace(case, thr):
    seed, B, hkv, g, L, bk, ps, lists = case
    tau, phi, p = thr
    wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, block_size=bk,
                        page_size=ps)
    if lists:
        wl.block_list, wl.block_list_len = random_lists(wl, seed)
    Tmax = max(max(x) for x in wl.traversal_lengths())
    r = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p, trace_steps=Tmax,
                               scale_of_accumulator=True)
    sp = wl.spec
    scale = float32(sp.softmax_scale)
    for b in range(sp.batch):
        for h in range(sp.num_kv_heads):
            grp = Group(wl.q, wl.k_cache, wl.v_cache, wl.page_table, wl.seq_lens, b, h,
                        sp.block_size, sp.dense_order, wl.block_list, wl.block_list_len)
            traj = _accumulator_trajectory(grp, scale)
            ts, mets = stop_from_trajectory(traj, float32(tau), float32(phi), p)
            assert int(r["stop"][b, h]) == ts
            for t in range(1, ts + 1):
                ds, dr = mets[t - 1]
                tr = r["trace"][b, h, t - 1]
                np.testing.assert_allclose(tr[:, 0], ds, rtol=1e-9, atol=1e-12)
                np.testing.assert_allclose(tr[:, 1], dr, rtol=1e-6, atol=1e-12)


@pytest.mark.parametrize("tail", [64, 10])
def test_equal_scores_count_tokens(tail):
    """K = 0: every score is 0, l(t) is the number of tokens consumed, and
    with every value row equal to e_0, X(t) = l(t) e_0.  A full block then
    moves X by 64 (up to the rounding of exp(log l)), so tau = 64.1 lets every
    step after the first pass (stop at p + 1) while tau = 63.9 passes none
    (T); d_direction is 0."""
    T, p = 8, 3
    vec = np.zeros(128)
    vec[0] = 1.0
    q, k, v, pt, sl = uniform_key_case([vec] * T)
    sl = torch.tensor([(T - 1) * 64 + tail], dtype=torch.int32)
    kw = dict(block_size=64, scale=0.088, phi=1e-9, patience=p, scale_of_accumulator=True,
              trace_steps=T)
    r = oracle.decode(q, k, v, pt, sl, tau=64.1, **kw)
    assert int(r["stop"][0, 0]) == p + 1
    # step 1 is the newest (partial) block: X(1) = tail e_0; step 2 adds 64
    np.testing.assert_allclose(r["trace"][0, 0, 1, 0, 0], 64.0, rtol=1e-12)
    r = oracle.decode(q, k, v, pt, sl, tau=63.9, **kw)
    assert int(r["stop"][0, 0]) == T
    # the normalised reading sees no change at all and stops at p + 1 for any tau > 0
    r = oracle.decode(q, k, v, pt, sl, tau=1e-12, phi=1e-9, patience=p, block_size=64,
                      scale=0.088)
    assert int(r["stop"][0, 0]) == p + 1


def test_direction_is_the_same_under_both_readings():
    wl = small_workload(84, batch=1, kv_heads=2, group=4, seq_len=1500)
    T = max(max(x) for x in wl.traversal_lengths())
    a = oracle.decode_workload(wl, tau=0.0, phi=1e-4, patience=5, trace_steps=T)
    b = oracle.decode_workload(wl, tau=0.0, phi=1e-4, patience=5, trace_steps=T,
                               scale_of_accumulator=True)
    np.testing.assert_allclose(a["trace"][..., 1], b["trace"][..., 1], rtol=1e-12, atol=1e-15)
    np.testing.assert_array_equal(a["stop"], b["stop"])
