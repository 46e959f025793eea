"""The GPU path against closed forms and plain NumPy, with no oracle in the
loop (needs a gfx950 GPU).

* Eq. (1) with termination off: the output and lse are those of plain
  softmax attention over the traversal set, computed here in fp64.
* Every value row equal to one vector v: o(t) = v at every step, so d = 0
  and every step from the second is stable (Eq. 2); with patience p the
  stop is step p + 1 (Eq. 3, Algorithm 1), the output v.
* Zero keys (uniform weights) and block-constant values alpha_t e_0: o(t)
  is the token-weighted mean of the alphas seen, d_scale at step t is
  |alpha_t - mean_{t-1}| / t and d_direction is 0; the stop is planned by
  choosing the alphas, and worked out here from their bf16 values.
* Patience beyond the traversal: no stop, stop_block = T."""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest
import torch

from helpers import uniform_key_case
from paper_2606_00024_amd import _lib, api

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


def _run(q, k, v, pt, sl, **kw):
    _say(f"  gpu call: {tuple(q.shape)} {tuple(k.shape)} {kw}")
    out, lse, stop = api.decode_attention(q.to(DEV), k.to(DEV), v.to(DEV), pt.to(DEV), sl.to(DEV),
                                          block_size=64, **kw)
    torch.cuda.synchronize()
    return out.cpu().double().numpy(), lse.cpu().double().numpy(), stop.cpu().numpy()


def _tokens(k, v, pt, L, b, kvh, blocks):
    """Keys and values (fp64) of the given logical blocks of sequence b, in
    token order, through the page table (page size 64 = block size)."""
    ks, vs = [], []
    for blk in blocks:
        page = int(pt[b, blk])
        n = min(64, L - blk * 64)
        ks.append(k[page, kvh, :n].double().numpy())
        vs.append(v[page, kvh, :n].double().numpy())
    return np.concatenate(ks), np.concatenate(vs)


def test_termination_off_is_softmax_attention():
    rng = np.random.default_rng(11)
    B, hkv, g = 2, 2, 4
    lens = [64 * 13 + 17, 64 * 5]
    n_pages = sum((L + 63) // 64 for L in lens) + 3
    q = torch.from_numpy(rng.standard_normal((B, hkv * g, D)).astype(np.float32)).to(torch.bfloat16)
    k = torch.from_numpy(rng.standard_normal((n_pages, hkv, 64, D)).astype(np.float32)).to(torch.bfloat16)
    v = torch.from_numpy(rng.standard_normal((n_pages, hkv, 64, D)).astype(np.float32)).to(torch.bfloat16)
    perm = rng.permutation(n_pages)
    maxp = max((L + 63) // 64 for L in lens)
    pt = torch.zeros((B, maxp), dtype=torch.int32)
    i = 0
    for b, L in enumerate(lens):
        for j in range((L + 63) // 64):
            pt[b, j] = int(perm[i])
            i += 1
    sl = torch.tensor(lens, dtype=torch.int32)
    scale = 1.0 / math.sqrt(D)
    out, lse, stop = _run(q, k, v, pt, sl, softmax_scale=scale, tau=0.0, phi=1e-3, patience=5)
    scale32 = float(np.float32(scale))
    for b, L in enumerate(lens):
        nb = (L + 63) // 64
        for kvh in range(hkv):
            assert stop[b, kvh] == nb
            kk, vv = _tokens(k, v, pt, L, b, kvh, range(nb))
            for i in range(g):
                h = kvh * g + i
                s = scale32 * (kk @ q[b, h].double().numpy())
                m = s.max()
                w = np.exp(s - m)
                o = (w @ vv) / w.sum()
                rel = np.linalg.norm(out[b, h] - o) / np.linalg.norm(o)
                assert rel < 1e-5, (b, h, rel)
                assert abs(lse[b, h] - (m + math.log(w.sum()))) < 1e-5, (b, h)


@pytest.mark.parametrize("p", [1, 3, 5])
def test_constant_values_stop_at_p_plus_one(p):
    T = 12
    rng = np.random.default_rng(p)
    vec = rng.standard_normal(D)
    q, k, v, pt, sl = uniform_key_case([vec] * T)
    k = torch.from_numpy(rng.standard_normal(k.shape).astype(np.float32)).to(torch.bfloat16)
    out, lse, stop = _run(q, k, v, pt, sl, softmax_scale=0.088, tau=1e-3, phi=1e-6, patience=p)
    assert int(stop[0, 0]) == p + 1
    vb = v[0, 0, 0].double().numpy()
    assert np.linalg.norm(out[0, 0] - vb) / np.linalg.norm(vb) < 1e-5
    # lse over the p + 1 blocks consumed (recency-first: the last ones)
    kk, _ = _tokens(k, v, pt, T * 64, 0, 0, range(T - p - 1, T))
    s = float(np.float32(0.088)) * (kk @ q[0, 0].double().numpy())
    m = s.max()
    assert abs(lse[0, 0] - (m + math.log(np.exp(s - m).sum()))) < 1e-5


def _planned_alphas(T, stable_from, tau):
    """alpha_1 = 1, then d_scale 5 tau up to step stable_from - 1 and tau / 5
    from stable_from on (alternating signs), rounded to bf16; returns the
    rounded alphas and the d_scale of every step from them in fp64."""
    a = [1.0]
    mean = 1.0
    for t in range(2, T + 1):
        dsc = 5 * tau if t < stable_from else tau / 5
        sign = 1.0 if t % 2 else -1.0
        a.append(mean + sign * t * dsc)
        a[-1] = float(torch.tensor(a[-1], dtype=torch.float32).to(torch.bfloat16).float())
        mean = sum(a) / len(a)
    ds = [math.nan, math.nan]   # ds[t]: step t (steps from 1; step 1 has no d)
    for t in range(2, T + 1):
        prev = sum(a[:t - 1]) / (t - 1)
        cur = sum(a[:t]) / t
        ds.append(abs(cur - prev))
    return a, ds


@pytest.mark.parametrize("stable_from,p", [(4, 3), (7, 2), (3, 6)])
def test_uniform_keys_planned_stop(stable_from, p):
    T, tau = 14, 1e-2
    a, ds = _planned_alphas(T, stable_from, tau)
    # the stop by Eq. (3) over the fp64 d_scale of the rounded alphas (the
    # direction test always passes: every o(t) is a positive multiple of e_0)
    run, want = 0, T
    for t in range(2, T + 1):
        assert abs(ds[t] - tau) > 0.2 * tau   # far from the threshold
        run = run + 1 if ds[t] < tau else 0
        if run >= p:
            want = t
            break
    vals = []
    for al in a:
        e = np.zeros(D)
        e[0] = al
        vals.append(e)
    q, k, v, pt, sl = uniform_key_case(vals)
    out, lse, stop = _run(q, k, v, pt, sl, softmax_scale=0.088, tau=tau, phi=1e-3, patience=p)
    assert int(stop[0, 0]) == want
    mean = sum(a[:want]) / want
    assert abs(out[0, 0, 0] - mean) < 1e-5 * max(1.0, abs(mean))
    assert np.all(out[0, 0, 1:] == 0.0)
    # zero keys: every score is 0, lse = ln(number of tokens consumed)
    assert abs(lse[0, 0] - math.log(64 * want)) < 1e-5


def test_patience_beyond_the_traversal():
    T = 9
    rng = np.random.default_rng(5)
    q, k, v, pt, sl = uniform_key_case([rng.standard_normal(D) for _ in range(T)])
    out, lse, stop = _run(q, k, v, pt, sl, softmax_scale=0.088, tau=math.inf, phi=math.inf,
                          patience=T)
    assert int(stop[0, 0]) == T
    out2, lse2, stop2 = _run(q, k, v, pt, sl, softmax_scale=0.088, tau=math.inf, phi=math.inf,
                             patience=T - 1)
    assert int(stop2[0, 0]) == T   # stable from step 2: the run reaches T - 1 at step T
    out3, lse3, stop3 = _run(q, k, v, pt, sl, softmax_scale=0.088, tau=math.inf, phi=math.inf,
                             patience=T - 2)
    assert int(stop3[0, 0]) == T - 1
