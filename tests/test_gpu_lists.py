"""Device-built traversal lists vs the list oracle (needs a gfx950 GPU).

Scores are fp64 sums over the head dimension in a fixed order on exact
products of the bf16 inputs, on both sides, so scores, lists and lengths are
compared bit for bit.  The lists then drive the decode call, whose result is
compared with the decode oracle run on the oracle's lists.
"""
from __future__ import annotations

import copy
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle import lists as OL
from helpers import small_workload
from parity import compare_workload
from paper_2606_00024_amd import _lib, api, workloads as W

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


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
    for name in ("q", "k_cache", "v_cache", "page_table", "seq_lens"):
        setattr(wl, name, getattr(wl, name).to(DEV))
    return wl


def _compare(wl, host, policy, kind, budget, sinks, keep_last):
    s = wl.spec
    _say(f"  gpu call: lists {s.name} B={s.batch} Hkv={s.num_kv_heads} g={s.group_size} "
         f"Bk={s.block_size} Ps={s.page_size} policy={policy} kind={kind} budget={budget} "
         f"sinks={sinks} last={keep_last}")
    bl, bll, sc = api.build_block_list(wl.q, wl.k_cache, wl.page_table, wl.seq_lens,
                                       block_size=s.block_size, budget=budget, policy=policy,
                                       score_kind=kind, sink_blocks=sinks, keep_last=keep_last,
                                       return_scores=True)
    torch.cuda.synchronize()
    ref = OL.block_list(host.q, host.k_cache, host.page_table, host.seq_lens,
                        block_size=s.block_size, num_q_heads=s.num_q_heads, policy=policy,
                        score_kind=kind, budget=budget, sink_blocks=sinks, keep_last=keep_last,
                        max_list=bl.shape[-1])
    np.testing.assert_array_equal(bll.cpu().numpy(), ref["len"])
    np.testing.assert_array_equal(bl.cpu().numpy(), ref["list"])
    if policy == OL.IMPORTANCE:
        got = sc.cpu().numpy()
        want = ref["scores"]
        mask = ~np.isnan(want)
        np.testing.assert_array_equal(got[mask], want[mask])
    return bl, bll


CASES = [
    # seed, B, Hkv, g, seq_len(s), Bk, Ps
    (61, 1, 2, 4, 4096, 64, 64),
    (62, 2, 2, 1, (700, 1500), 64, 16),
    (63, 2, 2, 8, (900, 2049), 128, 64),
    (64, 1, 2, 16, 3000, 64, 32),
    (65, 3, 1, 2, (0, 65, 5000), 256, 128),
    (66, 2, 3, 4, (1, 4097), 64, 64),
    # more sequences than the score kernels keep lengths for in LDS (256)
    (67, 300, 1, 4, tuple(int(x) for x in np.random.default_rng(8).integers(0, 700, 300)), 64, 16),
]
SELECT = [(8, 1, True), (3, 0, False), (5, 4, True), (10 ** 4, 0, False), (0, 2, False)]


@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
@pytest.mark.parametrize("kind", [OL.KEY_NORM, OL.QUERY_BOUND], ids=["keynorm", "qbound"])
def test_importance_lists_bit_exact(case, kind):
    seed, B, hkv, g, L, bk, ps = case
    host = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, block_size=bk,
                          page_size=ps, needles=2)
    wl = _to_dev(copy.copy(host))
    for budget, sinks, last in SELECT:
        _compare(wl, host, OL.IMPORTANCE, kind, budget, sinks, last)


@pytest.mark.parametrize("case", CASES[:3], ids=[f"s{c[0]}" for c in CASES[:3]])
def test_streaming_lists_exact(case):
    seed, B, hkv, g, L, bk, ps = case
    host = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, block_size=bk,
                          page_size=ps, needles=2)
    wl = _to_dev(copy.copy(host))
    for budget, sinks in [(4, 1), (0, 2), (3, 0), (10 ** 4, 3), (2, 10 ** 4)]:
        _compare(wl, host, OL.STREAMING, OL.KEY_NORM, budget, sinks, False)


def test_equal_scores_and_longest_sequences():
    """8192 blocks per sequence (the most the selection sorts) with many
    equal scores: keys of only four distinct norms."""
    L, bk = 8192 * 64, 64
    spec = W.WorkloadSpec(name="ties", batch=1, num_q_heads=4, num_kv_heads=1, seq_lens=(L,),
                          block_size=bk, page_size=64, n_needles=0, n_outliers=0, seed=67)
    host = W.make_workload(spec, device="cpu")
    k = host.k_cache.float()
    k.zero_()
    pages = host.page_table[0].long()
    for i in range(8192):          # block i gets norm (i % 4) + 1 on its first token
        k[pages[i], 0, 0, 0] = float(i % 4 + 1)
    host.k_cache = k.to(torch.bfloat16)
    wl = _to_dev(copy.copy(host))
    for budget, sinks, last in [(1000, 1, True), (8192, 0, False), (3, 0, True)]:
        _compare(wl, host, OL.IMPORTANCE, OL.KEY_NORM, budget, sinks, last)


def test_special_key_values():
    """Keys whose channels take every sign case of the extremes: channels
    negative on every token of every block, positive on every token, zeros
    of both signs (whole blocks of -0 too), bf16 subnormals, and magnitudes
    near 1e30; the extremes and the squares are compared bit for bit with
    the oracle's."""
    rng = np.random.default_rng(69)
    host = small_workload(69, batch=2, kv_heads=2, group=4, seq_len=(3000, 1000), block_size=64,
                          page_size=64, needles=0)
    k = host.k_cache.float()
    n_pages, hkv, ps, d = k.shape
    k[..., 0:16] = -k[..., 0:16].abs() - 1e-3
    k[..., 16:32] = k[..., 16:32].abs() + 1e-3
    zeros = torch.from_numpy(rng.integers(0, 2, size=(n_pages, hkv, ps, 16)).astype(np.float32))
    k[..., 32:48] = torch.where(zeros > 0, torch.tensor(-0.0), torch.tensor(0.0))
    k[: n_pages // 2, :, :, 40:48] = -0.0
    sub = torch.from_numpy(rng.integers(1, 127, size=(n_pages, hkv, ps, 16)).astype(np.float32))
    sign = torch.from_numpy(rng.choice([-1.0, 1.0], size=(n_pages, hkv, ps, 16)).astype(np.float32))
    k[..., 48:64] = sign * sub * 2.0 ** -133          # bf16 subnormals (exact in float32)
    k[..., 64:80] = k[..., 64:80] * 1e30
    k[: n_pages // 3, :, :, 80:96] = -7.0             # one value on every token
    host.k_cache = k.to(torch.bfloat16)
    kb = host.k_cache.float()
    assert bool((kb[..., 48:64] != 0).all()) and bool((kb[..., 48:64].abs() < 2.0 ** -126).all())
    assert bool(torch.signbit(kb[..., 32:48]).any()) and bool((~torch.signbit(kb[..., 32:48])).any())
    wl = _to_dev(copy.copy(host))
    for kind in (OL.KEY_NORM, OL.QUERY_BOUND):
        _compare(wl, host, OL.IMPORTANCE, kind, 20, 1, True)


def test_device_lists_drive_the_decode_call():
    """Lists built on the device, then decode over them; the reference is the
    decode oracle over the oracle's lists (the same lists, bit for bit)."""
    seed = 68
    host = small_workload(seed, batch=2, kv_heads=2, group=4, seq_len=(5000, 3000), needles=2)
    wl = _to_dev(copy.copy(host))
    bl, bll = _compare(wl, host, OL.IMPORTANCE, OL.QUERY_BOUND, 40, 1, True)
    wl.block_list, wl.block_list_len = bl, bll
    host.block_list, host.block_list_len = bl.cpu(), bll.cpu()
    for tau, phi, p in [(1e-3, 1e-4, 5), (0.05, 1e-3, 2), (0.0, 1e-4, 5)]:
        _say(f"  gpu call: decode over device lists tau={tau}")
        gpu = api.decode_workload(wl, tau=tau, phi=phi, patience=p)
        torch.cuda.synchronize()
        rep = compare_workload(host, gpu, tau=tau, phi=phi, patience=p, name="device_lists")
        _say("  ", rep)
        assert rep.ok(), str(rep)


def test_full_size_importance_lists():
    """The 128K-token sparse workload's shape: 32 groups of 2048 blocks, 25 %
    kept, the first and the last block forced."""
    spec = W.WORKLOADS["sparse25_128k"]
    _say(f"  generating {spec.name}")
    host = W.make_workload(spec, device="cpu")
    wl = _to_dev(copy.copy(host))
    for kind in (OL.KEY_NORM, OL.QUERY_BOUND):
        _compare(wl, host, OL.IMPORTANCE, kind, 512, 1, True)
    del wl
    torch.cuda.empty_cache()


def test_full_size_ragged_importance_lists():
    """The ragged batch's shape: 32 sequences of 8K-64K tokens (many blocks
    past each sequence's end), 8 KV heads of 8 query heads each."""
    spec = W.WORKLOADS["qwen3_32b_ragged"]
    _say(f"  generating {spec.name} on the device")
    wl = W.make_workload(spec, device=DEV)
    host = copy.copy(wl)
    for name in ("q", "k_cache", "v_cache", "page_table", "seq_lens"):
        setattr(host, name, getattr(wl, name).cpu())
    max_blocks = (int(wl.page_table.shape[1]) * spec.page_size + spec.block_size - 1) // spec.block_size
    for kind in (OL.KEY_NORM, OL.QUERY_BOUND):
        _compare(wl, host, OL.IMPORTANCE, kind, max_blocks // 4, 1, True)
    del wl, host
    torch.cuda.empty_cache()
