"""ctypes view of libart.so (include/art.h).  Argument marshalling only."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# ART_LIBRARY names another build of the same sources (the host-ASan test
# runs the CPU suite against the AddressSanitizer build); default in-tree
LIB_PATH = os.environ.get("ART_LIBRARY") or os.path.join(HERE, "libart.so")

OK = 0
ERR_INVALID_ARG = 1
ERR_UNSUPPORTED = 2
ERR_WORKSPACE_TOO_SMALL = 3
ERR_HIP = 4
ERR_BAD_INDEX = 5
ERR_DEVICE_TIMEOUT = 6

ORDER_RECENT_FIRST = 0
ORDER_FORWARD = 1
OUT_F32 = 0
OUT_BF16 = 1

# every symbol include/art.h declares
EXPORTS = ("art_abi_version", "art_status_str", "art_decode_workspace_bytes",
           "art_workspace_init", "art_decode_attention", "art_validate_inputs",
           "art_workspace_status", "art_block_list_workspace_bytes", "art_build_block_list",
           "art_decode_attention_static")
STATIC_SCRATCH_BYTES = 64 << 20   # ART_STATIC_SCRATCH_BYTES

LIST_IMPORTANCE = 0
LIST_STREAMING = 1
SCORE_KEY_NORM = 0
SCORE_QUERY_BOUND = 1


class DecodeShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "batch", "num_q_heads", "num_kv_heads", "head_dim", "block_size", "page_size",
        "num_pages", "max_pages_per_seq", "max_blocks_per_list", "list_per_head")] + [
        (n, ctypes.c_int64) for n in (
            "k_stride_page", "k_stride_head", "k_stride_token",
            "v_stride_page", "v_stride_head", "v_stride_token")]


# ART_ABI_VERSION of include/art.h that these structure layouts follow
ABI_VERSION = 8


class DecodeOpts(ctypes.Structure):
    _fields_ = [("softmax_scale", ctypes.c_float), ("tau", ctypes.c_float),
                ("phi", ctypes.c_float), ("patience", ctypes.c_int32),
                ("dense_order", ctypes.c_int32), ("out_dtype", ctypes.c_int32),
                ("chunk_blocks", ctypes.c_int32), ("probe_stride", ctypes.c_int32),
                ("scale_of_accumulator", ctypes.c_int32), ("no_detector", ctypes.c_int32),
                ("max_wait_polls", ctypes.c_int32), ("per_head_stop", ctypes.c_int32),
                ("max_ahead_chunks", ctypes.c_int32)]


class ListOpts(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "policy", "score_kind", "budget", "sink_blocks", "keep_last")]


class ArtError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        name = status_str(status) if _lib is not None else str(status)
        super().__init__(f"{what}: {name}" if what else name)


_lib = None


def load() -> ctypes.CDLL:
    """Load the in-tree libart.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        _lib = load_variant(LIB_PATH)
    return _lib


def load_variant(path: str) -> ctypes.CDLL:
    """Load a build of the library at `path` (the in-tree libart.so, or a
    test build of the same sources such as the race-stress build) with the
    argument types of this binding."""
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with `python -m paper_2606_00024_amd.build` "
            "(there is no fallback implementation)")
    lib = ctypes.CDLL(path)
    vp = ctypes.c_void_p
    i32p = ctypes.POINTER(ctypes.c_int32)
    lib.art_abi_version.restype = ctypes.c_int32
    lib.art_abi_version.argtypes = []
    lib.art_status_str.restype = ctypes.c_char_p
    lib.art_status_str.argtypes = [ctypes.c_int32]
    lib.art_decode_workspace_bytes.restype = ctypes.c_size_t
    lib.art_decode_workspace_bytes.argtypes = [ctypes.POINTER(DecodeShape),
                                               ctypes.POINTER(DecodeOpts), i32p]
    lib.art_workspace_init.restype = ctypes.c_int
    lib.art_workspace_init.argtypes = [vp, ctypes.c_size_t, vp]
    lib.art_decode_attention.restype = ctypes.c_int
    lib.art_decode_attention.argtypes = [
        ctypes.POINTER(DecodeShape), ctypes.POINTER(DecodeOpts),
        vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.art_decode_attention_static.restype = ctypes.c_int
    lib.art_decode_attention_static.argtypes = [
        ctypes.POINTER(DecodeShape), ctypes.POINTER(DecodeOpts),
        vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.art_validate_inputs.restype = ctypes.c_int
    lib.art_validate_inputs.argtypes = [
        ctypes.POINTER(DecodeShape), ctypes.POINTER(DecodeOpts), vp, vp, vp, vp, vp,
        ctypes.POINTER(ctypes.c_int64), i32p]
    lib.art_workspace_status.restype = ctypes.c_int
    lib.art_workspace_status.argtypes = [vp, ctypes.c_size_t, vp, i32p]
    lib.art_block_list_workspace_bytes.restype = ctypes.c_size_t
    lib.art_block_list_workspace_bytes.argtypes = [ctypes.POINTER(DecodeShape),
                                                   ctypes.POINTER(ListOpts), i32p]
    lib.art_build_block_list.restype = ctypes.c_int
    lib.art_build_block_list.argtypes = [
        ctypes.POINTER(DecodeShape), ctypes.POINTER(ListOpts), vp, vp, vp, vp, vp, vp, vp,
        vp, ctypes.c_size_t, vp]
    got = int(lib.art_abi_version())
    if got != ABI_VERSION:
        raise RuntimeError(f"{path} has ABI version {got}, this binding needs "
                           f"{ABI_VERSION}: rebuild it")
    return lib


class using:
    """Context manager: calls through this module go to `lib` (a
    load_variant result) inside the block."""

    def __init__(self, lib):
        self.lib = lib

    def __enter__(self):
        global _lib
        load()
        self.saved = _lib
        _lib = self.lib
        return self.lib

    def __exit__(self, *exc):
        global _lib
        _lib = self.saved
        return False


def status_str(status: int) -> str:
    return load().art_status_str(int(status)).decode()


def abi_version() -> int:
    return int(load().art_abi_version())


def workspace_bytes(shape: DecodeShape, opts: DecodeOpts) -> int:
    st = ctypes.c_int32(0)
    n = load().art_decode_workspace_bytes(ctypes.byref(shape), ctypes.byref(opts), ctypes.byref(st))
    if st.value != OK:
        raise ArtError(st.value, "art_decode_workspace_bytes")
    return int(n)


def workspace_init(ptr: int, nbytes: int, stream: int) -> None:
    st = load().art_workspace_init(ptr, nbytes, stream)
    if st != OK:
        raise ArtError(st, "art_workspace_init")


def decode_attention(shape, opts, q, k, v, page_table, seq_lens, block_list, block_list_len,
                     out, lse, stop_block, workspace, workspace_bytes, stream) -> int:
    """Raw call; pointers are ints (0 for NULL).  Returns the status."""
    return int(load().art_decode_attention(
        ctypes.byref(shape), ctypes.byref(opts), q, k, v, page_table, seq_lens,
        block_list or None, block_list_len or None, out, lse, stop_block,
        workspace or None, workspace_bytes, stream or None))


def decode_attention_static(shape, opts, q, k, v, page_table, seq_lens, block_list,
                            block_list_len, out, lse, stop_block, stream) -> int:
    """Raw call of the variant over the library's static scratch (no
    workspace); pointers are ints (0 for NULL).  Returns the status."""
    return int(load().art_decode_attention_static(
        ctypes.byref(shape), ctypes.byref(opts), q, k, v, page_table, seq_lens,
        block_list or None, block_list_len or None, out, lse, stop_block, stream or None))


def validate_inputs(shape, opts, page_table, seq_lens, block_list, block_list_len, stream):
    bad = ctypes.c_int64(-1)
    where = ctypes.c_int32(-1)
    st = load().art_validate_inputs(ctypes.byref(shape), ctypes.byref(opts), page_table,
                                    seq_lens, block_list or None, block_list_len or None,
                                    stream or None, ctypes.byref(bad), ctypes.byref(where))
    return int(st), int(bad.value), int(where.value)


def workspace_status(ptr: int, nbytes: int, stream: int) -> int:
    dev = ctypes.c_int32(-1)
    st = load().art_workspace_status(ptr, nbytes, stream or None, ctypes.byref(dev))
    if st != OK:
        raise ArtError(st, "art_workspace_status")
    return int(dev.value)


def block_list_workspace_bytes(shape: DecodeShape, opts: ListOpts) -> int:
    st = ctypes.c_int32(0)
    n = load().art_block_list_workspace_bytes(ctypes.byref(shape), ctypes.byref(opts),
                                              ctypes.byref(st))
    if st.value != OK:
        raise ArtError(st.value, "art_block_list_workspace_bytes")
    return int(n)


def build_block_list(shape, opts, q, k, page_table, seq_lens, block_list, block_list_len,
                     block_scores, workspace, workspace_bytes, stream) -> int:
    """Raw call; pointers are ints (0 for NULL).  Returns the status."""
    return int(load().art_build_block_list(
        ctypes.byref(shape), ctypes.byref(opts), q or None, k or None, page_table or None,
        seq_lens, block_list, block_list_len, block_scores or None, workspace or None,
        workspace_bytes, stream or None))
