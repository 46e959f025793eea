"""The decode call over the library's static scratch
(art_decode_attention_static, for callers that cannot allocate) against the
same call over a caller workspace (art_decode_attention), through the C ABI
(needs a gfx950 GPU).

Both run the same kernels under the same plan, so out, lse and stop_block
must agree bit for bit; each is also checked against the oracle.  Calls come
in a row on one GPU, each smaller than the one before, so every call after
the first finds the scratch holding the previous call's data (another
shape, another layout)."""
from __future__ import annotations

import math
import sys

import pytest
import torch

from helpers import random_lists, small_workload
from parity import compare_workload, host_copy
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
    for name in ("q", "k_cache", "v_cache", "page_table", "seq_lens", "block_list", "block_list_len"):
        t = getattr(wl, name)
        if t is not None:
            setattr(wl, name, t.to(DEV))
    return wl


def _call(wl, static, tau, phi, p):
    s = wl.spec
    shape = api.make_shape(wl.q, wl.k_cache, wl.v_cache, wl.page_table, block_size=s.block_size,
                           block_list=wl.block_list)
    opts = api.make_opts(softmax_scale=s.softmax_scale, tau=tau, phi=phi, patience=p,
                         dense_order=s.dense_order)
    B, Hq, D = wl.q.shape
    out = torch.full((B, Hq, D), float("nan"), dtype=torch.float32, device=DEV)
    lse = torch.full((B, Hq), float("nan"), dtype=torch.float32, device=DEV)
    stop = torch.full((B, s.num_kv_heads), -7, dtype=torch.int32, device=DEV)
    stream = torch.cuda.current_stream().cuda_stream
    ptr = lambda t: 0 if t is None else int(t.data_ptr())
    args = (ptr(wl.q), ptr(wl.k_cache), ptr(wl.v_cache), ptr(wl.page_table), ptr(wl.seq_lens),
            ptr(wl.block_list), ptr(wl.block_list_len), ptr(out), ptr(lse), ptr(stop))
    _say(f"  gpu call ({'static scratch' if static else 'workspace'}): {s.name} B={s.batch} "
         f"Hkv={s.num_kv_heads} g={s.group_size} lens={wl.seq_lens.tolist()[:3]} tau={tau}")
    if static:
        st = _lib.decode_attention_static(shape, opts, *args, stream)
    else:
        ws = api.new_workspace(api.workspace_bytes(shape, opts), DEV)
        st = _lib.decode_attention(shape, opts, *args, ptr(ws), ws.numel(), stream)
    assert st == _lib.OK, _lib.status_str(st)
    torch.cuda.synchronize()
    return out, lse, stop


def _workloads():
    full = W.make_workload(W.WORKLOADS["llama3_8b_32k"], device=DEV)
    mid = _to_dev(small_workload(71, batch=3, kv_heads=2, group=8, seq_len=(9000, 4000, 6100),
                                 needles=2))
    small = _to_dev(small_workload(72, batch=1, kv_heads=2, group=4, seq_len=2500, needles=2))
    small.block_list, small.block_list_len = (t.to(DEV) for t in random_lists(small, 72, 0.6))
    return [full, mid, small]


def test_static_scratch_matches_the_workspace_call():
    for thr in [(1e-3, 1e-4, 5), (0.0, 1e-4, 5)]:
        for wl in _workloads():   # a row of calls, each smaller than the one before
            a = _call(wl, True, *thr)
            b = _call(wl, False, *thr)
            for x, y in zip(a, b):
                assert torch.equal(x, y)
            rep = compare_workload(wl, a, tau=thr[0], phi=thr[1], patience=thr[2],
                                   host=host_copy(wl), name="static_scratch")
            _say("  ", rep)
            assert rep.ok(), str(rep)
            del wl
        torch.cuda.empty_cache()
