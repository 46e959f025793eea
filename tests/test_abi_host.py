"""C-ABI checks that need no GPU: the library loads, exports every symbol
include/art.h declares, and rejects malformed calls on the host before
anything is launched."""
from __future__ import annotations

import ctypes
import math
import os
import re

import pytest

from paper_2606_00024_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2606_00024_amd import build
        build.build()
    return _lib.load()


def _declared_symbols():
    with open(os.path.join(ROOT, "include", "art.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(art_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    declared = _declared_symbols()
    assert set(declared) == set(_lib.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def test_version_and_status_strings(lib):
    with open(os.path.join(ROOT, "include", "art.h")) as f:
        declared = int(re.search(r"#define ART_ABI_VERSION (\d+)", f.read()).group(1))
    assert _lib.abi_version() == declared == _lib.ABI_VERSION
    assert _lib.status_str(0) == "ART_OK"
    assert _lib.status_str(3) == "ART_ERR_WORKSPACE_TOO_SMALL"
    assert _lib.status_str(6) == "ART_ERR_DEVICE_TIMEOUT"
    assert _lib.status_str(99) == "ART_ERR_UNKNOWN"


def _shape(**kw):
    d = dict(batch=2, num_q_heads=8, num_kv_heads=2, head_dim=128, block_size=64, page_size=64,
             num_pages=40, max_pages_per_seq=16, max_blocks_per_list=0, list_per_head=1,
             k_stride_page=2 * 64 * 128, k_stride_head=64 * 128, k_stride_token=128,
             v_stride_page=2 * 64 * 128, v_stride_head=64 * 128, v_stride_token=128)
    d.update(kw)
    return _lib.DecodeShape(**d)


def _opts(**kw):
    d = dict(softmax_scale=1 / math.sqrt(128), tau=1e-3, phi=1e-4, patience=5, dense_order=0,
             out_dtype=0, chunk_blocks=0)
    d.update(kw)
    return _lib.DecodeOpts(**d)


def _ws(shape, opts):
    st = ctypes.c_int32(-1)
    n = _lib.load().art_decode_workspace_bytes(ctypes.byref(shape), ctypes.byref(opts), ctypes.byref(st))
    return int(n), st.value


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=64), _lib.ERR_UNSUPPORTED),
    (dict(num_q_heads=12, num_kv_heads=4), _lib.ERR_UNSUPPORTED),   # g = 3
    (dict(num_q_heads=7), _lib.ERR_INVALID_ARG),                    # not a multiple
    (dict(block_size=96), _lib.ERR_UNSUPPORTED),
    (dict(block_size=2048), _lib.ERR_UNSUPPORTED),
    (dict(page_size=8), _lib.ERR_UNSUPPORTED),
    (dict(page_size=48), _lib.ERR_UNSUPPORTED),
    (dict(block_size=0), _lib.ERR_INVALID_ARG),
    (dict(batch=-1), _lib.ERR_INVALID_ARG),
    (dict(num_pages=0), _lib.ERR_INVALID_ARG),
    (dict(list_per_head=2), _lib.ERR_INVALID_ARG),
    (dict(k_stride_token=100), _lib.ERR_UNSUPPORTED),
    (dict(v_stride_page=-8), _lib.ERR_INVALID_ARG),
])
def test_shape_errors(lib, kw, status):
    n, st = _ws(_shape(**kw), _opts())
    assert (n, st) == (0, status)


@pytest.mark.parametrize("kw", [
    dict(tau=float("nan")), dict(phi=float("nan")), dict(patience=0), dict(dense_order=2),
    dict(out_dtype=5), dict(chunk_blocks=-1), dict(chunk_blocks=17),
    dict(softmax_scale=float("inf")), dict(probe_stride=-1), dict(probe_stride=3),
    dict(probe_stride=6), dict(probe_stride=256), dict(scale_of_accumulator=2),
    dict(no_detector=-1), dict(no_detector=2), dict(max_wait_polls=-1),
    dict(per_head_stop=2), dict(per_head_stop=-1), dict(max_ahead_chunks=-1),
])
def test_option_errors(lib, kw):
    n, st = _ws(_shape(), _opts(**kw))
    assert (n, st) == (0, _lib.ERR_INVALID_ARG)


@pytest.mark.parametrize("stride", [0, 1, 2, 4, 8, 32, 128])
def test_probe_strides_accepted(lib, stride):
    """Every power of two dividing head_dim is a valid probe; the workspace
    does not depend on it."""
    n, st = _ws(_shape(), _opts(probe_stride=stride))
    assert st == _lib.OK and n == _ws(_shape(), _opts())[0]


def test_per_head_workspace_holds_the_head_records(lib):
    """Per-head termination adds [groups][chunks][g][8] int32 of per-head
    stability records; without the detector there is nothing to keep."""
    a, st = _ws(_shape(), _opts())
    b, st2 = _ws(_shape(), _opts(per_head_stop=1))
    c, _ = _ws(_shape(), _opts(per_head_stop=1, no_detector=1))
    assert st == st2 == _lib.OK
    assert b > a and c == a


def test_workspace_size_depends_on_shape_only(lib):
    a, st = _ws(_shape(), _opts())
    assert st == 0 and a > 0
    b, _ = _ws(_shape(), _opts(tau=0.5, phi=0.2, patience=1))
    assert a == b
    c, _ = _ws(_shape(max_pages_per_seq=64), _opts())
    assert c > a
    d, _ = _ws(_shape(max_blocks_per_list=200), _opts())
    assert d > a


def _call(shape, opts, ptrs=None, ws_bytes=1 << 30):
    p = dict(q=16, k=16, v=16, pt=16, sl=16, bl=0, bll=0, out=16, lse=16, stop=16, ws=16)
    if ptrs:
        p.update(ptrs)
    return _lib.decode_attention(shape, opts, p["q"], p["k"], p["v"], p["pt"], p["sl"], p["bl"],
                                 p["bll"], p["out"], p["lse"], p["stop"], p["ws"], ws_bytes, 0)


@pytest.mark.parametrize("ptrs,status", [
    (dict(q=0), _lib.ERR_INVALID_ARG),
    (dict(out=0), _lib.ERR_INVALID_ARG),
    (dict(bl=16), _lib.ERR_INVALID_ARG),        # list without lengths
    (dict(bll=16), _lib.ERR_INVALID_ARG),
    (dict(q=18), _lib.ERR_UNSUPPORTED),          # misaligned bf16 rows
    (dict(ws=0), _lib.ERR_WORKSPACE_TOO_SMALL),
])
def test_decode_rejects_before_launch(lib, ptrs, status):
    assert _call(_shape(), _opts(), ptrs) == status


def test_decode_rejects_small_workspace(lib):
    need, _ = _ws(_shape(), _opts())
    assert _call(_shape(), _opts(), ws_bytes=need - 1) == _lib.ERR_WORKSPACE_TOO_SMALL


def test_list_needs_row_stride(lib):
    assert _call(_shape(max_blocks_per_list=0), _opts(), dict(bl=16, bll=16)) == _lib.ERR_INVALID_ARG


def test_launch_failure_is_reported_as_hip_error(lib):
    """A call that passes every host check but whose launch fails returns
    ART_ERR_HIP.  Forced here by the absence of a GPU; on a machine with one
    the placeholder pointers would really be launched, so the test is skipped
    there."""
    if os.path.exists("/dev/kfd"):
        pytest.skip("a GPU is visible: this test launches with placeholder pointers")
    assert _call(_shape(), _opts()) == _lib.ERR_HIP
    assert _call(_shape(), _opts(max_wait_polls=3)) == _lib.ERR_HIP
    assert lib.art_workspace_init(16, 256, None) == _lib.ERR_HIP
    dev = ctypes.c_int32(-1)
    assert lib.art_workspace_status(16, 256, None, ctypes.byref(dev)) == _lib.ERR_HIP


def _call_static(shape, opts, ptrs=None):
    p = dict(q=16, k=16, v=16, pt=16, sl=16, bl=0, bll=0, out=16, lse=16, stop=16)
    if ptrs:
        p.update(ptrs)
    return _lib.decode_attention_static(shape, opts, p["q"], p["k"], p["v"], p["pt"], p["sl"],
                                        p["bl"], p["bll"], p["out"], p["lse"], p["stop"], 0)


def test_static_variant_checks_before_launch(lib):
    """The variant over the library's static scratch takes the decode call's
    host checks, and rejects a shape whose workspace exceeds the scratch
    before anything is set up or launched."""
    assert _call_static(_shape(), _opts(), dict(q=0)) == _lib.ERR_INVALID_ARG
    assert _call_static(_shape(), _opts(tau=float("nan"))) == _lib.ERR_INVALID_ARG
    assert _call_static(_shape(head_dim=64), _opts()) == _lib.ERR_UNSUPPORTED
    assert _call_static(_shape(batch=0), _opts(), dict(q=0, k=0, v=0)) == _lib.OK
    # 256 groups x 1024 blocks of g = 8: about 260 MB of chunk records
    big = _shape(batch=32, num_q_heads=64, num_kv_heads=8, num_pages=40000,
                 max_pages_per_seq=1024, k_stride_page=8 * 64 * 128, v_stride_page=8 * 64 * 128)
    n, st = _ws(big, _opts())
    assert st == _lib.OK and n > _lib.STATIC_SCRATCH_BYTES
    assert _call_static(big, _opts()) == _lib.ERR_WORKSPACE_TOO_SMALL
    n, st = _ws(_shape(), _opts())
    assert st == _lib.OK and n <= _lib.STATIC_SCRATCH_BYTES
    with open(os.path.join(ROOT, "include", "art.h")) as f:
        m = re.search(r"#define ART_STATIC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", f.read())
    assert int(m.group(1)) << int(m.group(2)) == _lib.STATIC_SCRATCH_BYTES


def test_static_variant_launch_failure_is_reported(lib):
    if os.path.exists("/dev/kfd"):
        pytest.skip("a GPU is visible: this test launches with placeholder pointers")
    assert _call_static(_shape(), _opts()) == _lib.ERR_HIP


def test_empty_batch_is_a_no_op(lib):
    assert _call(_shape(batch=0), _opts(), dict(q=0, k=0, v=0)) == _lib.OK


def test_graft_entry_builds(lib):
    import __graft_entry__  # noqa: F401  (import only: build() recompiles every library)


def _lopts(**kw):
    d = dict(policy=_lib.LIST_IMPORTANCE, score_kind=_lib.SCORE_KEY_NORM, budget=4, sink_blocks=1,
             keep_last=1)
    d.update(kw)
    return _lib.ListOpts(**d)


def _lws(shape, opts):
    st = ctypes.c_int32(-1)
    n = _lib.load().art_block_list_workspace_bytes(ctypes.byref(shape), ctypes.byref(opts),
                                                   ctypes.byref(st))
    return n, st.value


def test_block_list_workspace_is_the_score_array(lib):
    # 16 pages of 64 tokens, blocks of 64: 16 blocks per sequence
    n, st = _lws(_shape(max_blocks_per_list=16), _lopts())
    assert (n, st) == (2 * 2 * 16 * 8, _lib.OK)
    n, st = _lws(_shape(max_blocks_per_list=16, block_size=128), _lopts(score_kind=_lib.SCORE_QUERY_BOUND))
    assert (n, st) == (2 * 2 * 8 * 8, _lib.OK)


@pytest.mark.parametrize("kw,status", [
    (dict(budget=-1), _lib.ERR_INVALID_ARG),
    (dict(policy=2), _lib.ERR_INVALID_ARG),
    (dict(score_kind=3), _lib.ERR_INVALID_ARG),
    (dict(keep_last=2), _lib.ERR_INVALID_ARG),
    (dict(sink_blocks=-1), _lib.ERR_INVALID_ARG),
    (dict(budget=17), _lib.OK),                       # capped by the 16 blocks a sequence has
    (dict(policy=_lib.LIST_STREAMING, budget=3, sink_blocks=2), _lib.OK),
])
def test_block_list_option_errors(lib, kw, status):
    assert _lws(_shape(max_blocks_per_list=16), _lopts(**kw))[1] == status


def test_block_list_shape_errors(lib):
    # the row must hold the longest list the options allow
    assert _lws(_shape(max_blocks_per_list=3), _lopts(budget=4))[1] == _lib.ERR_INVALID_ARG
    assert _lws(_shape(max_blocks_per_list=4), _lopts(budget=4))[1] == _lib.OK
    assert _lws(_shape(max_blocks_per_list=4), _lopts(policy=_lib.LIST_STREAMING, budget=3,
                                                      sink_blocks=2))[1] == _lib.ERR_INVALID_ARG
    # per-sequence lists are not produced; more than 8192 blocks per sequence are not sorted
    assert _lws(_shape(max_blocks_per_list=16, list_per_head=0), _lopts())[1] == _lib.ERR_INVALID_ARG
    assert _lws(_shape(max_blocks_per_list=16, max_pages_per_seq=8193), _lopts())[1] == _lib.ERR_UNSUPPORTED
    assert _lws(_shape(max_blocks_per_list=16, page_size=48), _lopts())[1] == _lib.ERR_UNSUPPORTED
    assert _lws(_shape(max_blocks_per_list=16, num_q_heads=6),
                _lopts(score_kind=_lib.SCORE_QUERY_BOUND))[1] == _lib.ERR_UNSUPPORTED


def test_block_list_rejects_null_outputs_before_launch(lib):
    shape = _shape(max_blocks_per_list=16)
    st = lib.art_build_block_list(ctypes.byref(shape), ctypes.byref(_lopts()), None, None, None,
                                  None, None, None, None, None, 0, None)
    assert st == _lib.ERR_INVALID_ARG
    empty = _shape(batch=0, max_blocks_per_list=16)
    assert lib.art_build_block_list(ctypes.byref(empty), ctypes.byref(_lopts()), None, None, None,
                                    None, None, None, None, None, 0, None) == _lib.OK


def test_size_limits_of_the_plan(lib):
    """Traversals of 2^19 blocks and more do not fit the 19-bit stability runs
    of the flag words: refused.  One block less is planned (the workspace is
    sized from the shape alone, so no memory is needed to ask)."""
    big = 1 << 19
    n, st = _ws(_shape(batch=1, num_kv_heads=1, num_q_heads=4, max_pages_per_seq=big,
                       num_pages=big), _opts())
    assert (n, st) == (0, _lib.ERR_UNSUPPORTED)
    n, st = _ws(_shape(batch=1, num_kv_heads=1, num_q_heads=4, max_pages_per_seq=big - 1,
                       num_pages=big), _opts())
    assert st == _lib.OK and n > 0
    # a block list longer than any dense traversal sets the bound too
    n, st = _ws(_shape(batch=1, num_kv_heads=1, num_q_heads=4, max_blocks_per_list=big), _opts())
    assert (n, st) == (0, _lib.ERR_UNSUPPORTED)


def test_work_list_must_fit_a_queue_word(lib):
    """Chunks of all groups are numbered in 24 bits: a launch whose work list
    would not fit (with any chunk size the LDS budget allows) is refused."""
    n, st = _ws(_shape(batch=16384, num_kv_heads=8, num_q_heads=32, max_pages_per_seq=8192,
                       num_pages=1 << 20), _opts())
    assert (n, st) == (0, _lib.ERR_UNSUPPORTED)
    n, st = _ws(_shape(batch=64, num_kv_heads=8, num_q_heads=32, max_pages_per_seq=8192,
                       num_pages=1 << 20), _opts())
    assert st == _lib.OK and n > 0
