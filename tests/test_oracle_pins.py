"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every test here runs on the CPU.  None of them re-types the oracle's own
recurrence: expected values come from full-softmax brute force (Eq. 1 over an
explicit token set), hand-derived closed forms (tests/golden/), theorems of
Appendix A, and invariants of the definition.
"""
from __future__ import annotations

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from bruteforce import (Group, prefix_outputs, softmax_attention, step_metrics,
                        stop_from_trajectory, float32)
from helpers import exact_tie_case, random_lists, small_workload, uniform_key_case

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

CASES = [
    # (seed, batch, kv_heads, group, seq_len, block, page, order, lists)
    (11, 1, 2, 4, 1024, 64, 64, 0, False),
    (12, 2, 1, 1, 700, 64, 16, 0, False),      # partial tail, small pages
    (13, 1, 2, 2, 1500, 128, 64, 1, False),    # forward order, block 128
    (14, 2, 2, 8, 900, 64, 128, 0, True),      # random lists, pages > block
    (15, 1, 1, 4, 64, 64, 64, 0, False),       # T = 1
    (16, 1, 2, 4, 2000, 64, 32, 0, True),
]


def _wl(case, **kw):
    seed, B, hkv, g, L, bk, ps, order, lists = case
    wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L,
                        block_size=bk, page_size=ps, dense_order=order, **kw)
    if lists:
        wl.block_list, wl.block_list_len = random_lists(wl, seed)
    return wl


def _groups(wl):
    s = wl.spec
    for b in range(s.batch):
        for h in range(s.num_kv_heads):
            yield b, h, Group(wl.q, wl.k_cache, wl.v_cache, wl.page_table, wl.seq_lens,
                              b, h, s.block_size, s.dense_order, wl.block_list,
                              wl.block_list_len)


def _scale(wl):
    return float32(wl.spec.softmax_scale)


# ---------------------------------------------------------------- p1 / p2

@pytest.mark.parametrize("case", CASES)
def test_termination_off_equals_full_softmax(case):
    """tau = 0: nothing is ever stable, so the result is Eq. (1) over the
    whole traversal set (reordering only changes rounding, Sec. 3.4)."""
    wl = _wl(case)
    r = oracle.decode_workload(wl, tau=0.0)
    g = wl.spec.group_size
    for b, h, grp in _groups(wl):
        toks = grp.tokens_of(grp.blocks)
        out, lse = softmax_attention(grp.q, grp.K[toks], grp.V[toks], _scale(wl))
        np.testing.assert_allclose(r["out"][b, h * g:(h + 1) * g], out, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(r["lse"][b, h * g:(h + 1) * g], lse, rtol=1e-12, atol=1e-12)
        assert r["stop"][b, h] == len(grp.blocks)


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("thr", [(1e-3, 1e-4, 5), (0.05, 1e-3, 2), (0.2, 0.01, 1)])
def test_termination_equals_truncated_softmax(case, thr):
    """out/lse equal Eq. (1) over the tokens of the first t* traversal blocks
    (Algorithm 1 returns o(t*))."""
    tau, phi, p = thr
    wl = _wl(case)
    r = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p)
    g = wl.spec.group_size
    for b, h, grp in _groups(wl):
        ts = int(r["stop"][b, h])
        assert 1 <= ts <= len(grp.blocks) or len(grp.blocks) == 0
        toks = grp.tokens_of(grp.blocks[:ts])
        out, lse = softmax_attention(grp.q, grp.K[toks], grp.V[toks], _scale(wl))
        np.testing.assert_allclose(r["out"][b, h * g:(h + 1) * g], out, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(r["lse"][b, h * g:(h + 1) * g], lse, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- p3

@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("thr", [(1e-3, 1e-4, 5), (0.05, 1e-3, 2), (0.3, 0.05, 1), (0.02, 1e-2, 3)])
def test_bruteforce_stop_and_trace(case, thr):
    """Recompute o(t) for every prefix by full softmax, apply Eq. (2)-(3) and
    Algorithm 1; the stop index and every traced metric must agree."""
    tau, phi, p = thr
    wl = _wl(case)
    Tmax = max(max(x) for x in wl.traversal_lengths())
    assert Tmax <= 32
    r = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p, trace_steps=Tmax)
    for b, h, grp in _groups(wl):
        traj = prefix_outputs(grp, _scale(wl))["o"]
        ts, mets = stop_from_trajectory(traj, float32(tau), float32(phi), p)
        assert int(r["stop"][b, h]) == ts
        for t in range(1, ts + 1):
            ds, dr = mets[t - 1]
            tr = r["trace"][b, h, t - 1]
            np.testing.assert_allclose(tr[:, 0], ds, rtol=1e-9, atol=1e-13)
            np.testing.assert_allclose(tr[:, 1], dr, rtol=1e-6, atol=1e-12)


# ---------------------------------------------------------------- p4 / p5

@pytest.mark.parametrize("case", CASES[:4])
def test_increment_identity_and_convexity(case):
    """o(t) - o(t-1) = (l_t / A_t)(u(t) - o(t-1))  (Appendix A), with l_t,
    A_t and u(t) from brute force and o(t) from the oracle (force_stop = t);
    |o(t)| <= C_v and |u(t) - o(t-1)| <= 2 C_v (Lemma 3)."""
    wl = _wl(case)
    s = wl.spec
    g = s.group_size
    T = max(max(x) for x in wl.traversal_lengths())
    o_prev = {}
    for t in range(1, T + 1):
        fs = np.full((s.batch, s.num_kv_heads), t, dtype=np.int32)
        r = oracle.decode_workload(wl, tau=0.0, force_stop=fs)
        for b, h, grp in _groups(wl):
            if t > len(grp.blocks):
                continue
            bf = prefix_outputs(grp, _scale(wl), upto=t)
            o_t = r["out"][b, h * g:(h + 1) * g]
            o_tm1 = o_prev.get((b, h), np.zeros_like(o_t))
            w = np.exp(bf["logl"][t] - bf["logA"][t])[:, None]
            lhs = o_t - o_tm1
            rhs = w * (bf["u"][t] - o_tm1)
            Cv = np.linalg.norm(grp.V[grp.tokens_of(grp.blocks)], axis=1).max()
            assert np.abs(lhs - rhs).max() <= 1e-12 * max(1.0, Cv)
            assert np.linalg.norm(o_t, axis=1).max() <= Cv * (1 + 1e-12)
            assert np.linalg.norm(bf["u"][t] - o_tm1, axis=1).max() <= 2 * Cv * (1 + 1e-12)
            o_prev[(b, h)] = o_t


# ---------------------------------------------------------------- p6

@settings(max_examples=25, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(seed=st.integers(0, 10_000),
       tau=st.floats(1e-4, 0.5), phi=st.floats(1e-5, 0.1), p=st.integers(1, 6),
       ftau=st.floats(0.0, 1.0), fphi=st.floats(0.0, 1.0), dp=st.integers(0, 3))
def test_monotone_in_thresholds(seed, tau, phi, p, ftau, fphi, dp):
    """Tighter thresholds or more patience never stop earlier: the trajectory
    o(t) does not depend on (tau, phi, p) and Eq. (3) only resets more often."""
    wl = small_workload(seed, batch=1, kv_heads=2, group=2, seq_len=1536,
                        needles=1 + seed % 3)
    a = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p)
    b = oracle.decode_workload(wl, tau=tau * ftau, phi=phi * fphi, patience=p + dp)
    assert (b["stop"] >= a["stop"]).all()


# ---------------------------------------------------------------- p7

def _mass_regulated_case(seed, eps, T=16, g=2, D=128, Bk=64):
    """Nearly equal block masses (keys eps * N(0, I)) and values clustered
    around a common mean: the regime of Assumption 1 (mass-regulated
    traversal), where l_j ~ l and A_j ~ j l."""
    rng = np.random.default_rng(seed)
    q = torch.from_numpy(rng.standard_normal((1, g, D)).astype(np.float32)).to(torch.bfloat16)
    k = torch.from_numpy((eps * rng.standard_normal((T, 1, Bk, D))).astype(np.float32)).to(torch.bfloat16)
    mean = rng.standard_normal(D)
    v = torch.from_numpy((mean + 0.1 * rng.standard_normal((T, 1, Bk, D))).astype(np.float32)).to(torch.bfloat16)
    pt = torch.arange(T, dtype=torch.int32).view(1, T)
    sl = torch.tensor([T * Bk], dtype=torch.int32)
    return q, k, v, pt, sl


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("eps", [0.0, 0.02, 0.05])
def test_truncation_bound(seed, eps):
    """Theorem 1/2 and the Remark of Appendix A (probe P = I, nu = 1):
    |o(T) - o(t*)| <= min(tau b + mu Delta, 2 mu C_v) ln(T / t*), checked for
    every head where the conclusion of Lemma 1 (l_j / A_j <= mu / j for j in
    [b, T]) holds; heads where it does not are skipped (the theorem says
    nothing about them)."""
    tau, phi, p, Bk = 0.05, 1e-3, 3, 64
    q, k, v, pt, sl = _mass_regulated_case(seed, eps)
    g = q.shape[1]
    scale = float32(1 / math.sqrt(128))
    on = oracle.decode(q, k, v, pt, sl, block_size=Bk, scale=scale, tau=tau, phi=phi, patience=p)
    off = oracle.decode(q, k, v, pt, sl, block_size=Bk, scale=scale, tau=0.0, phi=phi, patience=p)
    grp = Group(q, k, v, pt, sl, 0, 0, Bk)
    T = len(grp.blocks)
    ts = int(on["stop"][0, 0])
    assert ts < T, "the case is built to stop early"
    bf = prefix_outputs(grp, scale)
    bstart = ts - p + 1
    Cv = np.linalg.norm(grp.V, axis=1).max()
    checked = 0
    for i in range(g):
        ratio = [math.exp(bf["logl"][j][i] - bf["logA"][j][i]) for j in range(1, T + 1)]
        mu = bstart * ratio[bstart - 1]
        if any(ratio[j - 1] > mu / j * (1 + 1e-12) for j in range(bstart, T + 1)):
            continue
        upd = [np.linalg.norm(bf["u"][j][i] - bf["o"][j - 1][i]) for j in range(1, T + 1)]
        delta = max(upd[j - 1] - upd[bstart - 1] for j in range(bstart, T + 1))
        bound = min(float32(tau) * bstart + mu * delta, 2 * mu * Cv) * math.log(T / ts)
        err = np.linalg.norm(off["out"][0, i] - on["out"][0, i])
        assert err <= bound * (1 + 1e-9) + 1e-12
        checked += 1
    if eps == 0.0:
        assert checked == g  # equal masses: l_j / A_j = 1 / j exactly, mu = 1


# ---------------------------------------------------------------- p8

def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_golden_uniform_keys_scale():
    fx = _load("uniform_keys_scale.json")
    D = 128
    vecs = []
    for a in fx["a"]:
        v = np.zeros(D)
        v[0] = a
        vecs.append(v)
    q, k, v, pt, sl = uniform_key_case(vecs, block_size=fx["block_size"])
    for case in fx["cases"]:
        r = oracle.decode(q, k, v, pt, sl, block_size=fx["block_size"], scale=1 / math.sqrt(D),
                          tau=fx["tau"], phi=fx["phi"], patience=case["patience"],
                          trace_steps=fx["num_blocks"])
        assert int(r["stop"][0, 0]) == case["stop"]
        num, den = case["out0"]
        np.testing.assert_allclose(r["out"][0, 0, 0], num / den, rtol=1e-14)
        assert np.all(r["out"][0, 0, 1:] == 0)
        np.testing.assert_allclose(r["lse"][0, 0], math.log(case["lse_tokens"]), rtol=1e-14)
        for t in range(1, case["stop"] + 1):
            n, d = fx["d_scale"][t - 1]
            np.testing.assert_allclose(r["trace"][0, 0, t - 1, 0, 0], n / d, rtol=1e-13)
            if t >= 2:
                assert r["trace"][0, 0, t - 1, 0, 1] == 0.0
            else:
                assert math.isnan(r["trace"][0, 0, 0, 0, 1])


def test_golden_uniform_keys_direction():
    fx = _load("uniform_keys_direction.json")
    D, T = 128, fx["num_blocks"]
    e0, e1 = np.zeros(D), np.zeros(D)
    e0[0], e1[1] = 1.0, 1.0
    vecs = [e0] + [e1] * (T - 1)
    q, k, v, pt, sl = uniform_key_case(vecs, block_size=fx["block_size"])
    for case in fx["cases"]:
        tau = math.inf if case["tau"] == "inf" else case["tau"]
        phi = math.inf if case["phi"] == "inf" else case["phi"]
        r = oracle.decode(q, k, v, pt, sl, block_size=fx["block_size"], scale=1 / math.sqrt(D),
                          tau=tau, phi=phi, patience=case["patience"], trace_steps=T)
        ts = case["stop"]
        assert int(r["stop"][0, 0]) == ts
        np.testing.assert_allclose(r["out"][0, 0, 0], 1 / ts, rtol=1e-14)
        np.testing.assert_allclose(r["out"][0, 0, 1], (ts - 1) / ts, rtol=1e-14)
        for t in range(2, ts + 1):
            cos = (1 + (t - 1) * (t - 2)) / (math.sqrt(1 + (t - 1) ** 2) * math.sqrt(1 + (t - 2) ** 2))
            np.testing.assert_allclose(r["trace"][0, 0, t - 1, 0, 1], 1 - cos, rtol=1e-9, atol=1e-15)
            np.testing.assert_allclose(r["trace"][0, 0, t - 1, 0, 0], math.sqrt(2) / (t * (t - 1)), rtol=1e-12)


@pytest.mark.parametrize("T,p", [(8, 5), (6, 5), (3, 5), (12, 1), (12, 3)])
def test_constant_values_stop_at_p_plus_1(T, p):
    """Every value row equal to the same v != 0: o(t) = v for all t >= 1, so
    every step t >= 2 has d_scale = 0 and d_direction = 0, step 1 compares
    with o(0) = 0 and is unstable -> t* = min(T, p + 1)."""
    rng = np.random.default_rng(T * 31 + p)
    vec = rng.standard_normal(128)
    q, k, v, pt, sl = uniform_key_case([vec] * T)
    k = torch.from_numpy(rng.standard_normal(k.shape).astype(np.float32)).to(torch.bfloat16)
    r = oracle.decode(q, k, v, pt, sl, block_size=64, scale=0.088, tau=1e-6, phi=1e-9, patience=p)
    assert int(r["stop"][0, 0]) == min(T, p + 1)
    # strict "<": a zero change does not pass a zero threshold
    r0 = oracle.decode(q, k, v, pt, sl, block_size=64, scale=0.088, tau=0.0, phi=1.0, patience=1)
    assert int(r0["stop"][0, 0]) == T


def test_strict_comparison_at_an_exact_tie():
    """Algorithm 1 compares with a strict '<': when o(t) == o(t-1) exactly,
    d_scale == 0 does not pass tau == 0, but passes any tau > 0."""
    q, k, v, pt, sl = exact_tie_case(T=6)
    r = oracle.decode(q, k, v, pt, sl, block_size=64, scale=1 / math.sqrt(128), tau=0.0,
                      phi=1.0, patience=1, trace_steps=6)
    assert np.all(r["trace"][0, 0, 1:, 0, 0] == 0.0)
    assert int(r["stop"][0, 0]) == 6
    r = oracle.decode(q, k, v, pt, sl, block_size=64, scale=1 / math.sqrt(128), tau=1e-30,
                      phi=1.0, patience=1)
    assert int(r["stop"][0, 0]) == 2


def test_patience_at_least_T_never_stops():
    wl = small_workload(7, seq_len=640, tau=10.0, phi=10.0)
    T = max(max(x) for x in wl.traversal_lengths())
    r = oracle.decode_workload(wl, patience=T)
    assert (r["stop"] == T).all()
    r = oracle.decode_workload(wl, patience=2**31 - 1)
    assert (r["stop"] == T).all()


def test_single_block_stops_at_one():
    wl = small_workload(8, seq_len=37, tau=10.0, phi=10.0, patience=1)
    r = oracle.decode_workload(wl)
    assert (r["stop"] == 1).all()


# ---------------------------------------------------------------- p9 / p10

@pytest.mark.parametrize("seed", [21, 22, 23])
def test_order_invariance_when_off(seed):
    """All blocks processed: a permuted traversal list changes only rounding
    (Sec. 3.4)."""
    wl = small_workload(seed, batch=2, kv_heads=2, group=4, seq_len=1100)
    a = oracle.decode_workload(wl, tau=0.0)
    wl.block_list, wl.block_list_len = random_lists(wl, seed, fraction=1.0)
    b = oracle.decode_workload(wl, tau=0.0)
    np.testing.assert_allclose(a["out"], b["out"], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(a["lse"], b["lse"], rtol=1e-12)


@pytest.mark.parametrize("mode", ["no_scale", "no_direction", "no_patience"])
@pytest.mark.parametrize("seed", [31, 32])
def test_ablation_switches(mode, seed):
    """The three ablations of Table 3 through the thresholds: tau = +inf
    drops the scale test, phi = +inf drops the direction test, p = 1 drops
    patience.  Each equals brute force with the reduced rule."""
    wl = small_workload(seed, batch=1, kv_heads=2, group=4, seq_len=1600)
    tau, phi, p = 0.05, 2e-3, 3
    kw = dict(use_scale=True, use_direction=True)
    if mode == "no_scale":
        tau = math.inf
        kw["use_scale"] = False
    elif mode == "no_direction":
        phi = math.inf
        kw["use_direction"] = False
    else:
        p = 1
    r = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p)
    for b, h, grp in _groups(wl):
        traj = prefix_outputs(grp, _scale(wl))["o"]
        ts, _ = stop_from_trajectory(traj, float32(tau), float32(phi), p, **kw)
        assert int(r["stop"][b, h]) == ts


# ---------------------------------------------------------------- edges

def test_empty_traversal_and_empty_sequence():
    wl = small_workload(41, batch=2, kv_heads=2, group=2, seq_len=(0, 300))
    r = oracle.decode_workload(wl)
    assert (r["stop"][0] == 0).all()
    assert np.all(r["out"][0] == 0)
    assert np.all(np.isneginf(r["lse"][0]))
    assert (r["stop"][1] >= 1).all()
    # an empty list for one group
    wl2 = small_workload(42, batch=1, kv_heads=2, group=2, seq_len=300)
    bl, bll = random_lists(wl2, 42)
    bll[0, 1] = 0
    wl2.block_list, wl2.block_list_len = bl, bll
    r2 = oracle.decode_workload(wl2)
    assert r2["stop"][0, 1] == 0 and np.all(np.isneginf(r2["lse"][0, 2:]))


def test_rejects_bad_lists():
    wl = small_workload(43, batch=1, kv_heads=2, group=2, seq_len=300)
    bl, bll = random_lists(wl, 43, fraction=1.0)
    bad = bl.clone()
    bad[0, 1, 0] = 5  # nblk = 5 -> out of range
    wl.block_list, wl.block_list_len = bad, bll
    with pytest.raises(oracle.OracleError) as ei:
        oracle.decode_workload(wl)
    assert ei.value.code == oracle.ERR_INDEX and ei.value.group == 1
    dup = bl.clone()
    dup[0, 0, 1] = dup[0, 0, 0]
    wl.block_list = dup
    with pytest.raises(oracle.OracleError) as ei:
        oracle.decode_workload(wl)
    assert ei.value.group == 0


def test_group_mask_and_threads_deterministic():
    wl = small_workload(44, batch=2, kv_heads=2, group=4, seq_len=900)
    a = oracle.decode_workload(wl, num_threads=1)
    b = oracle.decode_workload(wl, num_threads=4)
    assert np.array_equal(a["out"], b["out"]) and np.array_equal(a["stop"], b["stop"])
    m = np.zeros((2, 2), dtype=np.uint8)
    m[1, 0] = 1
    c = oracle.decode_workload(wl, group_mask=m)
    assert c["stop"][1, 0] == a["stop"][1, 0] and c["stop"][0, 0] == -1
