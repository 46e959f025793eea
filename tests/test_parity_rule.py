"""The near-tie rule of the parity tests (tests/parity.py), checked on the
CPU: which stop mismatches it excuses, and that it excuses nothing else."""
from __future__ import annotations

import math

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from helpers import small_workload
from parity import (NO_STOP, Report, compare_workload, excused, reachable_stops, step_classes,
                    tie_band)


def eq3_stop(stable, patience):
    """Eq. (3) with a plain counter: first t with `patience` consecutive
    stable steps, else T."""
    c = 0
    for t, s in enumerate(stable, start=1):
        c = c + 1 if s else 0
        if c >= patience:
            return t
    return len(stable)


def test_bands():
    assert tie_band(1e-3) == pytest.approx(1e-6, rel=1e-6)
    assert tie_band(1e-2) == pytest.approx(1e-5, rel=1e-6)
    assert tie_band(0.05) == pytest.approx(1e-5, rel=1e-6)   # capped at the rule's 1e-5
    assert tie_band(1e-5) == pytest.approx(1e-7, rel=1e-6)   # the fp32 floor
    assert tie_band(1e-4) == pytest.approx(1e-7, rel=1e-6)
    assert tie_band(0.0) == 0.0 and tie_band(math.inf) == 0.0 and tie_band(-1.0) == 0.0
    assert tie_band(50.0, rel=1e-3) == pytest.approx(0.05, rel=1e-6)


def test_reachable_stops_by_hand():
    # 0 unstable, 1 stable, 2 either way; patience 3
    assert reachable_stops(np.array([0, 1, 1, 2, 1, 1], np.int8), 3) == {4, 6}
    assert reachable_stops(np.array([0, 1, 1, 1, 1, 1], np.int8), 3) == {4}
    assert reachable_stops(np.array([0, 2, 2, 2], np.int8), 2) == {3, 4}
    assert reachable_stops(np.array([0, 0, 0], np.int8), 1) == {3}
    assert reachable_stops(np.array([0, 1], np.int8), 1) == {2}
    assert reachable_stops(np.array([2], np.int8), 1) == {1}


@settings(max_examples=200, deadline=None)
@given(st.lists(st.integers(0, 1), min_size=1, max_size=40), st.integers(1, 6))
def test_sure_classes_reach_exactly_eq3(bits, p):
    assert reachable_stops(np.array(bits, np.int8), p) == {eq3_stop(bits, p)}


@settings(max_examples=200, deadline=None)
@given(st.lists(st.integers(0, 2), min_size=1, max_size=30), st.integers(1, 5))
def test_every_resolution_of_the_ambiguous_steps_is_reachable(cls, p, ):
    cls = np.array(cls, np.int8)
    amb = np.flatnonzero(cls == 2)
    reach = reachable_stops(cls, p)
    rng = np.random.default_rng(len(cls) * 7 + p)
    for _ in range(20):
        choice = cls.copy()
        choice[amb] = rng.integers(0, 2, len(amb))
        assert eq3_stop(choice.tolist(), p) in reach


def _trace(ds_rows, dr=1e-9):
    """trace [T][g][2] from per-step d_scale rows (one value per head)."""
    ds = np.asarray(ds_rows, dtype=np.float64)
    tr = np.empty(ds.shape + (2,))
    tr[..., 0] = ds
    tr[..., 1] = dr
    tr[0, :, 1] = np.nan   # step 1: cos undefined
    return tr


def test_classes_follow_the_band():
    tau = 1e-3                       # band 1e-6
    tr = _trace([[1.0], [5e-4], [1e-3 - 5e-7], [1e-3 + 5e-7], [1e-3 + 2e-6], [1e-3 - 2e-6]])
    assert step_classes(tr, 6, tau, 1e-2).tolist() == [0, 1, 2, 2, 0, 1]
    # one head surely unstable makes the step surely unstable whatever the others
    tr2 = _trace([[1.0, 1.0], [1e-3, 5.0]])
    assert step_classes(tr2, 2, tau, 1e-2).tolist() == [0, 0]


def test_mismatch_far_from_the_band_is_not_excused():
    """A group whose criterion came within the band once, early, and whose
    stops differ at steps far from it: the old any-step-in-band excuse let
    this pass, the replay does not."""
    p = 3
    rows = [[1.0], [1e-3 - 1e-7]] + [[2e-3]] * 5 + [[1e-4]] * 6
    tr = _trace(rows)
    T = len(rows)
    ref = eq3_stop([False, True] + [False] * 5 + [True] * 6, p)
    assert ref == 10
    assert excused(tr, T, ref, ref, 1e-3, 1e-2, p)
    for wrong in (9, 11, T):
        assert not excused(tr, T, wrong, ref, 1e-3, 1e-2, p)


def test_mismatch_at_an_ambiguous_step_is_excused():
    p = 2
    rows = [[1.0], [1e-4], [1e-3 + 3e-7], [1e-4], [1e-4]]
    tr = _trace(rows)
    # exact: steps 2 stable, 3 unstable, 4-5 stable -> stop 5; fp32 may see step 3 stable -> 3
    assert excused(tr, 5, 3, 5, 1e-3, 1e-2, p)
    assert not excused(tr, 5, 4, 5, 1e-3, 1e-2, p)


def test_compare_workload_accepts_the_oracle_and_rejects_a_shifted_stop():
    """The comparison itself, with the oracle's own result standing in for a
    GPU result: it passes; the same result with one group's stop moved by a
    step (and its output left alone) fails."""
    import torch
    wl = small_workload(61, batch=2, kv_heads=2, group=4, seq_len=(3000, 2000), needles=2)
    tau, phi, p = 0.05, 1e-3, 2
    ref = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p)
    gpu = (torch.from_numpy(ref["out"].astype(np.float32)),
           torch.from_numpy(ref["lse"].astype(np.float32)),
           torch.from_numpy(ref["stop"].copy()))
    rep = compare_workload(wl, gpu, tau=tau, phi=phi, patience=p)
    assert rep.ok() and rep.groups == 4 and rep.stop_equal == 4, str(rep)
    bad = gpu[2].clone()
    bad[1, 0] += 1
    rep = compare_workload(wl, (gpu[0], gpu[1], bad), tau=tau, phi=phi, patience=p)
    assert not rep.ok(), str(rep)
    full = oracle.decode_workload(wl, tau=tau, phi=phi, patience=NO_STOP,
                                  trace_steps=max(map(max, wl.traversal_lengths())))
    T1 = wl.traversal_lengths()[1][0]
    assert np.isfinite(full["trace"][1, 0, :T1, :, 0]).all()   # the whole trajectory
    assert np.isnan(full["trace"][1, 0, T1:, :, 0]).all()
    assert Report().near_tie_bound() == 1
