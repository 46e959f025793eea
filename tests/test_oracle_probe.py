"""Pins of the oracle's subsampled probe (Sec. 3.2; x = P o in Appendix A).

With ``probe_stride`` s the stability test sees only coordinates 0, s, 2s, ...
of each head's output.  The closed forms below fix both the stride and the
offset of that selection: values that live only off the probe are invisible
to it, values that are constant on the probe look converged to it.  The
brute-force check applies an explicit selection matrix P to prefix outputs
recomputed by full softmax.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from bruteforce import Group, prefix_outputs, stop_from_trajectory, float32
from helpers import random_lists, small_workload, uniform_key_case

D = 128


def _const_value_case(vec, T, seed):
    """Every value row equal to ``vec``; random keys."""
    rng = np.random.default_rng(seed)
    q, k, v, pt, sl = uniform_key_case([vec] * T)
    k = torch.from_numpy(rng.standard_normal(k.shape).astype(np.float32)).to(torch.bfloat16)
    return q, k, v, pt, sl


@pytest.mark.parametrize("s", [2, 4, 8, 32])
def test_values_off_the_probe_are_invisible(s):
    """v is zero on every probe coordinate: x(t) = 0 for all t, the cosine is
    undefined, no step is stable and t* = T.  The whole output o(t) = v is
    constant, so the full-output test (s = 1) stops at p + 1."""
    T, p = 10, 3
    rng = np.random.default_rng(s)
    vec = rng.standard_normal(D)
    vec[::s] = 0.0
    args = _const_value_case(vec, T, seed=s)
    kw = dict(block_size=64, scale=0.088, tau=1e-6, phi=1e-9, patience=p)
    assert int(oracle.decode(*args, probe_stride=s, **kw)["stop"][0, 0]) == T
    assert int(oracle.decode(*args, probe_stride=1, **kw)["stop"][0, 0]) == p + 1


@pytest.mark.parametrize("s", [2, 4, 8, 32])
def test_values_only_on_the_probe_are_seen(s):
    """v is non-zero only on the probe coordinates: x(t) = P v != 0 is constant
    from step 1, so t* = p + 1 for the probe as for the full output."""
    T, p = 10, 3
    rng = np.random.default_rng(100 + s)
    vec = np.zeros(D)
    vec[::s] = rng.standard_normal(D // s)
    args = _const_value_case(vec, T, seed=s)
    kw = dict(block_size=64, scale=0.088, tau=1e-6, phi=1e-9, patience=p)
    assert int(oracle.decode(*args, probe_stride=s, **kw)["stop"][0, 0]) == p + 1
    assert int(oracle.decode(*args, probe_stride=1, **kw)["stop"][0, 0]) == p + 1


@pytest.mark.parametrize("s", [2, 4, 16])
def test_constant_probe_coordinates_look_converged(s):
    """Each value row holds the same constant on the probe coordinates and
    random values elsewhere: o(t) changes from block to block off the probe,
    but x(t) stays the constant vector, so the probe stops at p + 1 while the
    full-output test never passes tau = 1e-6 and runs to T."""
    T, p, L = 12, 4, 12 * 64
    rng = np.random.default_rng(s)
    q = torch.from_numpy(rng.standard_normal((1, 1, D)).astype(np.float32)).to(torch.bfloat16)
    k = torch.from_numpy(rng.standard_normal((T, 1, 64, D)).astype(np.float32)).to(torch.bfloat16)
    v = rng.standard_normal((T, 1, 64, D)).astype(np.float32) * 4.0
    v[..., ::s] = 0.75
    v = torch.from_numpy(v).to(torch.bfloat16)
    pt = torch.arange(T, dtype=torch.int32).view(1, T)
    sl = torch.tensor([L], dtype=torch.int32)
    kw = dict(block_size=64, scale=0.088, tau=1e-6, phi=1e-9, patience=p)
    assert int(oracle.decode(q, k, v, pt, sl, probe_stride=s, **kw)["stop"][0, 0]) == p + 1
    assert int(oracle.decode(q, k, v, pt, sl, probe_stride=1, **kw)["stop"][0, 0]) == T


CASES = [
    # (seed, batch, kv_heads, group, seq_len, block, page, lists)
    (31, 1, 2, 4, 1024, 64, 64, False),
    (32, 2, 1, 2, 700, 64, 16, False),
    (33, 2, 2, 8, 900, 64, 128, True),
]


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("s", [2, 4, 8])
@pytest.mark.parametrize("thr", [(0.05, 1e-3, 2), (0.02, 1e-2, 3), (0.3, 0.05, 1)])
def test_probe_bruteforce_stop_and_trace(case, s, thr):
    """Prefix outputs by full softmax, then x = P o with P the selection
    matrix of rows 0, s, 2s, ... of the identity; Eq. (2)-(3) on x give the
    oracle's stop index and traced metrics."""
    seed, B, hkv, g, L, bk, ps, lists = case
    tau, phi, p = thr
    wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L,
                        block_size=bk, page_size=ps)
    if lists:
        wl.block_list, wl.block_list_len = random_lists(wl, seed)
    Tmax = max(max(x) for x in wl.traversal_lengths())
    r = oracle.decode_workload(wl, tau=tau, phi=phi, patience=p, trace_steps=Tmax,
                               probe_stride=s)
    P = np.eye(D)[::s]
    scale = float32(wl.spec.softmax_scale)
    sp = wl.spec
    for b in range(sp.batch):
        for h in range(sp.num_kv_heads):
            grp = Group(wl.q, wl.k_cache, wl.v_cache, wl.page_table, wl.seq_lens, b, h,
                        sp.block_size, sp.dense_order, wl.block_list, wl.block_list_len)
            traj = prefix_outputs(grp, scale)["o"]
            ts, mets = stop_from_trajectory(traj, float32(tau), float32(phi), p, probe=P)
            assert int(r["stop"][b, h]) == ts
            for t in range(1, ts + 1):
                ds, dr = mets[t - 1]
                tr = r["trace"][b, h, t - 1]
                np.testing.assert_allclose(tr[:, 0], ds, rtol=1e-9, atol=1e-13)
                np.testing.assert_allclose(tr[:, 1], dr, rtol=1e-6, atol=1e-12)


def test_probe_stride_must_divide_head_dim():
    args = _const_value_case(np.ones(D), 3, seed=0)
    kw = dict(block_size=64, scale=0.088, tau=1e-3, phi=1e-4, patience=2)
    for bad in (0, 3, 256):
        with pytest.raises(oracle.OracleError):
            oracle.decode(*args, probe_stride=bad, **kw)
