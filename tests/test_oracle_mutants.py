"""Planted mistakes in the oracle (CPU only): every plausible slip in
art_oracle.c must make at least one pin fail.

Each mutant is a textual edit of a private copy of the oracle source, built
into a temporary library; the product oracle is not modified.  The battery
below is a fast subset of tests/test_oracle_pins.py: brute-force stop index
and traced metrics (Eq. 2-3), full and truncated softmax (Eq. 1), and the
hand-derived golden fixtures.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import pytest

import oracle
from bruteforce import Group, prefix_outputs, softmax_attention, stop_from_trajectory, float32
from helpers import exact_tie_case, random_lists, small_workload, uniform_key_case

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

MUTANTS = {
    "recurrence_drops_old_weight": (
        "onew[i * D + d] = keep * o[i * D + d] + w * u[i * D + d];",
        "onew[i * D + d] = o[i * D + d] + w * u[i * D + d];"),
    "value_index_reversed": (
        "u[i * D + d] += e * bf16_to_double(vj[d]);",
        "u[i * D + d] += e * bf16_to_double(vj[D - 1 - d]);"),
    "direction_sign": ("? 1.0 - dot /", "? 1.0 + dot /"),
    "patience_off_by_one": ("c >= O->patience", "c > O->patience"),
    "non_strict_scale": ("(d_scale < O->tau)", "(d_scale <= O->tau)"),
    "forward_instead_of_recent": ("(nblk - 1 - i)", "(i)"),
    "scale_dropped": ("s[i * Bk + j] = O->scale * dot;", "s[i * Bk + j] = dot;"),
    "block_mass_without_max": ("const double logl = mb + log(ssum);",
                               "const double logl = log(ssum);"),
    "gqa_head_interleaved": ("(int64_t)b * S->num_q_heads + kvh * g + i) * D;",
                             "(int64_t)b * S->num_q_heads + kvh + i * S->num_kv_heads) * D;"),
    "only_first_head_decides": ("if (!stable) all_stable = 0;",
                                "if (i == 0) all_stable = stable;"),
    "counter_not_reset": ("c = all_stable ? c + 1 : 0;", "c = all_stable ? c + 1 : c;"),
    "lse_reports_last_block": ("lse[(int64_t)b * S->num_q_heads + h] = (T > 0) ? logA[i] : -INFINITY;",
                               "lse[(int64_t)b * S->num_q_heads + h] = (T > 0) ? logA[i] - 1e-3 : -INFINITY;"),
    "tail_block_not_masked": ("const int j1 = (j0 + Bk < L) ? j0 + Bk : L;",
                              "const int j1 = (j0 + Bk < L) ? j0 + Bk : L - (L > j0 + 1 ? 1 : 0);"),
}


def _battery(lib) -> list[str]:
    """Returns the names of the checks that fail for ``lib``."""
    fails = []
    cases = [
        small_workload(301, batch=1, kv_heads=2, group=4, seq_len=1000, page_size=16),
        small_workload(302, batch=1, kv_heads=2, group=2, seq_len=1300, dense_order=1),
    ]
    wl3 = small_workload(303, batch=1, kv_heads=2, group=4, seq_len=900)
    wl3.block_list, wl3.block_list_len = random_lists(wl3, 303)
    cases.append(wl3)
    for ci, wl in enumerate(cases):
        s = wl.spec
        g = s.group_size
        scale = float32(s.softmax_scale)
        for tau, phi, p in ((0.05, 1e-3, 2), (0.02, 1e-2, 3), (1e-3, 1e-4, 5)):
            T = max(max(x) for x in wl.traversal_lengths())
            r = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p, trace_steps=T, _lib=lib)
            for b in range(s.batch):
                for h in range(s.num_kv_heads):
                    grp = Group(wl.q, wl.k_cache, wl.v_cache, wl.page_table, wl.seq_lens, b, h,
                                s.block_size, s.dense_order, wl.block_list, wl.block_list_len)
                    traj = prefix_outputs(grp, scale)["o"]
                    ts, mets = stop_from_trajectory(traj, float32(tau), float32(phi), p)
                    if int(r["stop"][b, h]) != ts:
                        fails.append(f"stop{ci}")
                    toks = grp.tokens_of(grp.blocks[: int(r["stop"][b, h])])
                    out, lse = softmax_attention(grp.q, grp.K[toks], grp.V[toks], scale)
                    if not np.allclose(r["out"][b, h * g:(h + 1) * g], out, rtol=1e-10, atol=1e-12):
                        fails.append(f"out{ci}")
                    if not np.allclose(r["lse"][b, h * g:(h + 1) * g], lse, rtol=1e-10, atol=1e-12):
                        fails.append(f"lse{ci}")
                    for t in range(1, min(ts, int(r["stop"][b, h])) + 1):
                        ds, dr = mets[t - 1]
                        tr = r["trace"][b, h, t - 1]
                        if not np.allclose(tr[:, 0], ds, rtol=1e-9, atol=1e-13):
                            fails.append(f"trace_scale{ci}")
                            break
                        if not np.allclose(tr[:, 1], dr, rtol=1e-6, atol=1e-12, equal_nan=True):
                            fails.append(f"trace_dir{ci}")
                            break
    # golden closed form (scale term) and the zero-threshold strictness case
    with open(os.path.join(GOLDEN, "uniform_keys_scale.json")) as f:
        fx = json.load(f)
    vecs = []
    for a in fx["a"]:
        v = np.zeros(128)
        v[0] = a
        vecs.append(v)
    q, k, v, pt, sl = uniform_key_case(vecs)
    for case in fx["cases"]:
        r = oracle.decode(q, k, v, pt, sl, block_size=64, scale=1 / math.sqrt(128),
                          tau=fx["tau"], phi=fx["phi"], patience=case["patience"], _lib=lib)
        if int(r["stop"][0, 0]) != case["stop"]:
            fails.append("golden_stop")
    q, k, v, pt, sl = exact_tie_case()
    r = oracle.decode(q, k, v, pt, sl, block_size=64, scale=1 / math.sqrt(128), tau=0.0,
                      phi=1.0, patience=1, trace_steps=6, _lib=lib)
    if int(r["stop"][0, 0]) != 6:
        fails.append("strict_zero_threshold")
    return sorted(set(fails))


ACCUMULATOR_MUTANTS = {
    "accumulator_old_in_new_reference": ("const double xs_old = O->scale_of_accumulator ? l_old : 1.0;",
                                         "const double xs_old = O->scale_of_accumulator ? l_new : 1.0;"),
    "accumulator_without_max_shift": ("const double l_new = exp(logA_new - m_new);",
                                      "const double l_new = exp(logA_new);"),
}


def _accumulator_battery(lib) -> list[str]:
    import test_oracle_accumulator as A
    fails = []
    for fn, args in ((A.test_bruteforce_stop_and_trace, (A.CASES[0], (5.0, 1e-3, 2))),
                     (A.test_equal_scores_count_tokens, (10,))):
        saved = oracle._lib
        try:
            oracle._lib = lib
            fn(*args)
        except AssertionError:
            fails.append(fn.__name__)
        finally:
            oracle._lib = saved
    return fails


@pytest.mark.parametrize("name", sorted(ACCUMULATOR_MUTANTS))
def test_planted_accumulator_mistake_is_caught(name, tmp_path):
    old, new = ACCUMULATOR_MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    lib = oracle.load_library(oracle.build_variant(src.replace(old, new), str(tmp_path / f"{name}.so")))
    assert _accumulator_battery(lib), f"planted mistake '{name}' passed every accumulator pin"


def test_accumulator_battery_passes_on_the_real_oracle():
    assert _accumulator_battery(oracle._load()) == []


PER_HEAD_MUTANTS = {
    "head_counter_not_reset": ("ch[i] = stable ? ch[i] + 1 : 0;", "ch[i] = stable ? ch[i] + 1 : ch[i];"),
    "head_output_at_group_stop": ("if (per_head && hstop[i]) {       /* written at the head's own stop */",
                                  "if (0 && per_head && hstop[i]) {"),
}


def _per_head_battery(lib) -> list[str]:
    import test_oracle_per_head as H
    fails = []
    saved = oracle._lib
    try:
        oracle._lib = lib
        for case in H.CASES:
            for rule in H.RULES:
                try:
                    H.test_per_head_stops_and_outputs_match_brute_force(case, rule)
                except AssertionError:
                    fails.append(f"brute{case[0]}{rule}")
        try:
            H.test_interrupted_run_restarts_the_count()
        except AssertionError:
            fails.append("restart")
    finally:
        oracle._lib = saved
    return fails


@pytest.mark.parametrize("name", sorted(PER_HEAD_MUTANTS))
def test_planted_per_head_mistake_is_caught(name, tmp_path):
    old, new = PER_HEAD_MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    lib = oracle.load_library(oracle.build_variant(src.replace(old, new), str(tmp_path / f"{name}.so")))
    assert _per_head_battery(lib), f"planted mistake '{name}' passed every per-head pin"


def test_per_head_battery_passes_on_the_real_oracle():
    assert _per_head_battery(oracle._load()) == []


PROBE_MUTANTS = {
    "probe_stride_ignored": ("for (int d = 0; d < D; d += ps) {", "for (int d = 0; d < D; d += 1) {"),
    "probe_offset_shifted": ("for (int d = 0; d < D; d += ps) {",
                             "for (int d = ps - 1; d < D; d += ps) {"),
    "probe_on_new_only": ("const double x = onew[i * D + d], x0 = o[i * D + d];",
                          "const double x = onew[i * D + d], x0 = o[i * D + (d ^ 1)];"),
}


def _probe_battery(lib) -> list[str]:
    """Brute force with an explicit selection matrix, plus the closed forms
    of tests/test_oracle_probe.py, at stride 4."""
    fails = []
    s_ = 4
    wl = small_workload(311, batch=1, kv_heads=2, group=4, seq_len=1000, page_size=16)
    sp = wl.spec
    scale = float32(sp.softmax_scale)
    P = np.eye(128)[::s_]
    for tau, phi, p in ((0.05, 1e-3, 2), (0.02, 1e-2, 3)):
        T = max(max(x) for x in wl.traversal_lengths())
        r = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p, trace_steps=T,
                                   probe_stride=s_, _lib=lib)
        for b in range(sp.batch):
            for h in range(sp.num_kv_heads):
                grp = Group(wl.q, wl.k_cache, wl.v_cache, wl.page_table, wl.seq_lens, b, h,
                            sp.block_size, sp.dense_order, None, None)
                traj = prefix_outputs(grp, scale)["o"]
                ts, mets = stop_from_trajectory(traj, float32(tau), float32(phi), p, probe=P)
                if int(r["stop"][b, h]) != ts:
                    fails.append("probe_stop")
                for t in range(1, min(ts, int(r["stop"][b, h])) + 1):
                    ds, dr = mets[t - 1]
                    tr = r["trace"][b, h, t - 1]
                    if not (np.allclose(tr[:, 0], ds, rtol=1e-9, atol=1e-13) and
                            np.allclose(tr[:, 1], dr, rtol=1e-6, atol=1e-12, equal_nan=True)):
                        fails.append("probe_trace")
                        break
    rng = np.random.default_rng(5)
    off = rng.standard_normal(128)
    off[::s_] = 0.0
    q, k, v, pt, sl = uniform_key_case([off] * 10)
    k = k + 0.5  # non-uniform keys are not needed: values are constant
    r = oracle.decode(q, k, v, pt, sl, block_size=64, scale=0.088, tau=1e-6, phi=1e-9,
                      patience=3, probe_stride=s_, _lib=lib)
    if int(r["stop"][0, 0]) != 10:
        fails.append("probe_blind_off_probe")
    return sorted(set(fails))


def test_battery_passes_on_the_real_oracle():
    assert _battery(None) == []
    assert _probe_battery(None) == []


@pytest.mark.parametrize("name", sorted(PROBE_MUTANTS))
def test_planted_probe_mistake_is_caught(name, tmp_path):
    old, new = PROBE_MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    path = oracle.build_variant(src.replace(old, new), str(tmp_path / f"{name}.so"))
    fails = _probe_battery(oracle.load_library(path))
    assert fails, f"planted mistake '{name}' passed every probe pin"


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    path = oracle.build_variant(src.replace(old, new), str(tmp_path / f"{name}.so"))
    lib = oracle.load_library(path)
    fails = _battery(lib)
    assert fails, f"planted mistake '{name}' passed every pin"
