"""Bounded waits end the launch (needs a gfx950 GPU).

Every wait of the decode kernel (the look-backs over other workgroups'
chunks, the claim of a work-list index, the hand-over between the loading
and resolving wavefronts of a workgroup) gives up after max_wait_polls
polls.  The first wave that gives up records the call in the workspace's
error word, and every other wait of that call ends within a few polls.  Here
the limit is one poll, so the resolving wavefront of every workgroup gives
up at its first wait (a chunk takes microseconds to load): the call must
return promptly, report ART_ERR_DEVICE_TIMEOUT, and leave the workspace
usable.  The inputs are valid; nothing faults or hangs.
"""
from __future__ import annotations

import sys
import time

import pytest
import torch

from helpers import small_workload
from parity import compare_workload, host_copy
from paper_2606_00024_amd import _lib, api

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


def test_wait_give_up_drains_and_is_reported():
    wl = _to_dev(small_workload(51, batch=2, kv_heads=2, group=4, seq_len=(6000, 5000), needles=2))
    host = host_copy(wl)
    ws = api.new_workspace(16 << 20, DEV)
    torch.cuda.synchronize()
    for chunk in (1, 0):
        _say(f"  gpu call: give-up after one poll, chunk_blocks={chunk}")
        t0 = time.perf_counter()
        api.decode_workload(wl, tau=1e-3, phi=1e-4, patience=5, chunk_blocks=chunk,
                            max_wait_polls=1, workspace=ws)
        status = api.workspace_status(ws)  # synchronises the stream
        dt = time.perf_counter() - t0
        _say(f"   status={_lib.status_str(status)} in {dt * 1e3:.1f} ms")
        assert status == _lib.ERR_DEVICE_TIMEOUT
        assert dt < 2.0
    # the error stays recorded, but later calls on the workspace run normally
    _say("  gpu call: default polls on the same workspace")
    gpu = api.decode_workload(wl, tau=1e-3, phi=1e-4, patience=5, workspace=ws)
    rep = compare_workload(wl, gpu, tau=1e-3, phi=1e-4, patience=5, host=host, name="after_timeout")
    assert rep.ok(), str(rep)
    assert api.workspace_status(ws) == _lib.ERR_DEVICE_TIMEOUT
    # initialised again: no error, and parity
    _lib.workspace_init(int(ws.data_ptr()), ws.numel(), torch.cuda.current_stream().cuda_stream)
    assert api.workspace_status(ws) == _lib.OK
    gpu = api.decode_workload(wl, tau=1e-3, phi=1e-4, patience=5, chunk_blocks=1, workspace=ws)
    rep = compare_workload(wl, gpu, tau=1e-3, phi=1e-4, patience=5, host=host, name="after_timeout")
    assert rep.ok(), str(rep)
    assert api.workspace_status(ws) == _lib.OK
