"""HIP path vs the oracle with the subsampled probe (needs a gfx950 GPU).

The stability test runs on every s-th coordinate of each head's output
(probe_stride s); the acceptance rule is the one of tests/parity.py.  The
closed forms of tests/test_oracle_probe.py are checked on the GPU as well,
and the agreement harness is checked against the oracle's own decisions.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
from helpers import random_lists, small_workload, uniform_key_case
from parity import compare_workload, host_copy
from paper_2606_00024_amd import _lib, api, workloads as W
from paper_2606_00024_amd.agreement import classify

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
D = 128


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
    for name in ("q", "k_cache", "v_cache", "page_table", "seq_lens", "block_list",
                 "block_list_len"):
        t = getattr(wl, name)
        if t is not None:
            setattr(wl, name, t.to(DEV))
    return wl


CASES = [
    # seed, B, Hkv, g, seq_len(s), Bk, Ps, lists
    (41, 1, 2, 4, 4096, 64, 64, False),
    (42, 2, 2, 1, (700, 1500), 64, 16, False),
    (43, 2, 2, 8, (900, 2049), 64, 128, True),
    (44, 1, 2, 16, 3000, 64, 32, False),
    (45, 2, 2, 4, (3000, 777), 128, 16, True),
]
THRESHOLDS = [(1e-3, 1e-4, 5), (0.05, 1e-3, 2), (0.02, 1e-2, 1)]


@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
@pytest.mark.parametrize("stride", [2, 4, 16])
def test_probe_matrix(case, stride):
    seed, B, hkv, g, L, bk, ps, lists = case
    wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, block_size=bk,
                        page_size=ps, needles=2)
    if lists:
        wl.block_list, wl.block_list_len = random_lists(wl, seed, fraction=0.6)
    _to_dev(wl)
    for tau, phi, p in THRESHOLDS:
        _say(f"  gpu call: probe s{seed} stride={stride} tau={tau} phi={phi} p={p}")
        gpu = api.decode_workload(wl, tau=tau, phi=phi, patience=p, probe_stride=stride)
        torch.cuda.synchronize()
        rep = compare_workload(wl, gpu, tau=tau, phi=phi, patience=p, probe_stride=stride,
                               name="probe_matrix")
        _say("  ", rep)
        assert rep.ok(), str(rep)


def _run_raw(q, k, v, pt, sl, **kw):
    _say(f"  gpu call: closed form {kw}")
    r = api.decode_attention(q.to(DEV), k.to(DEV), v.to(DEV), pt.to(DEV), sl.to(DEV),
                             block_size=64, **kw)
    torch.cuda.synchronize()
    return r


@pytest.mark.parametrize("stride", [2, 4, 32])
def test_probe_closed_forms(stride):
    """Values that live only off the probe: x = 0, never stable, t* = T while
    the whole-output test stops at p + 1.  Values constant on the probe and
    random elsewhere: the probe stops at p + 1, the whole output runs to T.
    The oracle gives the same stops at these thresholds (checked here too)."""
    T, p = 10, 3
    rng = np.random.default_rng(stride)
    vec = rng.standard_normal(D)
    vec[::stride] = 0.0
    q, k, v, pt, sl = uniform_key_case([vec] * T)
    k = torch.from_numpy(rng.standard_normal(k.shape).astype(np.float32)).to(torch.bfloat16)
    # thresholds well above fp32 rounding of a constant output (|v| ~ 11)
    kw = dict(softmax_scale=0.088, tau=1e-3, phi=1e-6, patience=p)
    assert int(_run_raw(q, k, v, pt, sl, probe_stride=stride, **kw)[2][0, 0]) == T
    assert int(_run_raw(q, k, v, pt, sl, probe_stride=1, **kw)[2][0, 0]) == p + 1
    ok = dict(block_size=64, scale=0.088, tau=kw["tau"], phi=kw["phi"], patience=p)
    assert int(oracle.decode(q, k, v, pt, sl, probe_stride=stride, **ok)["stop"][0, 0]) == T
    assert int(oracle.decode(q, k, v, pt, sl, probe_stride=1, **ok)["stop"][0, 0]) == p + 1

    T, p = 12, 4
    v2 = rng.standard_normal((T, 1, 64, D)).astype(np.float32) * 4.0
    v2[..., ::stride] = 0.75
    v2 = torch.from_numpy(v2).to(torch.bfloat16)
    q2 = torch.from_numpy(rng.standard_normal((1, 1, D)).astype(np.float32)).to(torch.bfloat16)
    k2 = torch.from_numpy(rng.standard_normal((T, 1, 64, D)).astype(np.float32)).to(torch.bfloat16)
    pt2 = torch.arange(T, dtype=torch.int32).view(1, T)
    sl2 = torch.tensor([T * 64], dtype=torch.int32)
    kw = dict(softmax_scale=0.088, tau=1e-4, phi=1e-6, patience=p)
    assert int(_run_raw(q2, k2, v2, pt2, sl2, probe_stride=stride, **kw)[2][0, 0]) == p + 1
    assert int(_run_raw(q2, k2, v2, pt2, sl2, probe_stride=1, **kw)[2][0, 0]) == T
    ok = dict(block_size=64, scale=0.088, tau=kw["tau"], phi=kw["phi"], patience=p)
    assert int(oracle.decode(q2, k2, v2, pt2, sl2, probe_stride=stride, **ok)["stop"][0, 0]) == p + 1
    assert int(oracle.decode(q2, k2, v2, pt2, sl2, probe_stride=1, **ok)["stop"][0, 0]) == T


def test_probe_stride_one_is_the_whole_output():
    """probe_stride 0 and 1 both mean P = I: bit-identical results to the
    default call."""
    wl = _to_dev(small_workload(46, batch=2, kv_heads=2, group=4, seq_len=(3000, 2000),
                                needles=2))
    base = api.decode_workload(wl, tau=0.05, phi=1e-3, patience=2)
    for s in (0, 1):
        again = api.decode_workload(wl, tau=0.05, phi=1e-3, patience=2, probe_stride=s)
        for a, b in zip(base, again):
            assert torch.equal(a, b)
    torch.cuda.synchronize()


def test_probe_full_size_every_group():
    spec = W.WORKLOADS["llama3_8b_32k"]
    _say(f"  generating {spec.name} on {DEV}")
    wl = W.make_workload(spec, device=DEV)
    torch.cuda.synchronize()
    host = host_copy(wl)
    for tau, phi, p in [(spec.tau, spec.phi, spec.patience), (1e-5, 1e-3, 5)]:
        _say(f"  gpu call: {spec.name} probe_stride=4 tau={tau} phi={phi}")
        gpu = api.decode_workload(wl, tau=tau, phi=phi, patience=p, probe_stride=4)
        torch.cuda.synchronize()
        rep = compare_workload(wl, gpu, tau=tau, phi=phi, patience=p, probe_stride=4, host=host,
                               name="full:probe4")
        _say("  ", rep)
        assert rep.ok(), str(rep)
        assert rep.groups == spec.batch * spec.num_kv_heads
    del wl, host
    torch.cuda.empty_cache()


def test_agreement_matches_the_oracle():
    """The harness classifies the GPU's stop decisions; away from near-ties
    they are the oracle's, so the classification is too."""
    wl = small_workload(47, batch=4, kv_heads=2, group=4, seq_len=(4096, 3000, 2500, 4000),
                        needles=2)
    T = np.asarray(wl.traversal_lengths())
    host = {}
    for s in (1, 4):
        host[s] = oracle.decode_workload(wl, tau=0.05, phi=1e-3, patience=2, probe_stride=s,
                                         trace_steps=int(T.max()))
    _to_dev(wl)
    dev = {s: api.decode_workload(wl, tau=0.05, phi=1e-3, patience=2,
                                  probe_stride=s)[2].cpu().numpy() for s in (1, 4)}
    for s in (1, 4):
        rep = compare_workload(wl, (api.decode_workload(wl, tau=0.05, phi=1e-3, patience=2,
                                                        probe_stride=s)),
                               tau=0.05, phi=1e-3, patience=2, probe_stride=s)
        assert rep.ok(), str(rep)
        if rep.near_ties:
            pytest.skip(f"near-tie in the sample: {rep.near_ties}")
    a_dev = classify(dev[4], dev[1], T)
    a_ref = classify(host[4]["stop"], host[1]["stop"], T)
    assert (a_dev.agree, a_dev.fp, a_dev.fn, a_dev.both_stop_differ) == \
        (a_ref.agree, a_ref.fp, a_ref.fn, a_ref.both_stop_differ)


# ---- the accumulator reading of d_scale (scale_of_accumulator) ----------------
# d_scale is then a difference of two unnormalised accumulators l(t) o(t),
# l(t) up to the number of tokens consumed; each carries the fp32 error of
# its merges (about 1e-6 relative after a thousand), so the near-tie band for
# d_scale is relative: 1e-3 of tau.
ACC_TAU_REL = 1e-3


@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_accumulator_reading_matrix(case):
    seed, B, hkv, g, L, bk, ps, lists = case
    wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, block_size=bk,
                        page_size=ps, needles=2)
    if lists:
        wl.block_list, wl.block_list_len = random_lists(wl, seed, fraction=0.6)
    _to_dev(wl)
    for tau, phi, p in [(1.0, 1e-3, 2), (10.0, 1e-2, 3), (50.0, 1e-4, 5), (0.0, 1e-3, 2)]:
        for stride in (1, 4):
            _say(f"  gpu call: accumulator s{seed} stride={stride} tau={tau} phi={phi} p={p}")
            gpu = api.decode_workload(wl, tau=tau, phi=phi, patience=p, probe_stride=stride,
                                      scale_of_accumulator=True)
            torch.cuda.synchronize()
            rep = compare_workload(wl, gpu, tau=tau, phi=phi, patience=p, probe_stride=stride,
                                   scale_of_accumulator=True, tau_rel=ACC_TAU_REL,
                                   name="accumulator")
            _say("  ", rep)
            assert rep.ok(), str(rep)


def test_accumulator_reading_closed_form():
    """Equal scores, every value row e_0: X(t) = l(t) e_0 grows by 64 per
    full block, so tau = 64.1 stops at p + 1 and tau = 63.9 never (the
    normalised reading sees no change at all)."""
    T, p = 8, 3
    vec = np.zeros(D)
    vec[0] = 1.0
    q, k, v, pt, sl = uniform_key_case([vec] * T)
    kw = dict(softmax_scale=0.088, phi=1e-6, patience=p, scale_of_accumulator=True)
    assert int(_run_raw(q, k, v, pt, sl, tau=64.1, **kw)[2][0, 0]) == p + 1
    assert int(_run_raw(q, k, v, pt, sl, tau=63.9, **kw)[2][0, 0]) == T
