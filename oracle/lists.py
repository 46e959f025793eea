"""CPU fp64 oracle for the traversal lists of Sec. 3.4 -- TEST INFRASTRUCTURE ONLY.

Wraps ``artref_block_list`` from ``art_list_oracle.c`` (plain C, fp64).  Only
``tests/`` may use it; the product path never does.  See the C file for the
readings (score definitions, selection, streaming order).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import _bits, _i32, _ptr

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "art_list_oracle.c")
_DEFAULT_LIB = os.path.join(_HERE, "libart_list_oracle.so")
_LIB = os.environ.get("ART_LIST_ORACLE_LIBRARY") or _DEFAULT_LIB
ASAN_LIB = os.path.join(_HERE, "libart_list_oracle_asan.so")
_lib = None

IMPORTANCE, STREAMING = 0, 1
KEY_NORM, QUERY_BOUND = 0, 1


class ListShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "batch", "num_q_heads", "num_kv_heads", "head_dim", "block_size", "page_size",
        "num_pages", "max_pages_per_seq", "max_blocks_per_list")] + [
        (n, ctypes.c_int64) for n in ("k_stride_page", "k_stride_head", "k_stride_token")]


class ListOpts(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "policy", "score_kind", "budget", "sink_blocks", "keep_last")]


def build(force: bool = True) -> str:
    if _LIB != _DEFAULT_LIB:      # another build was named: leave it alone
        return _LIB
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                               "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def source_text() -> str:
    with open(_SRC) as f:
        return f.read()


def build_variant(src_text: str, out_path: str) -> str:
    """Compile ``src_text`` (a modified copy of art_list_oracle.c)."""
    import shutil
    d = os.path.dirname(out_path)
    c_path = os.path.join(d, "list_variant.c")
    with open(c_path, "w") as f:
        f.write(src_text)
    shutil.copy(os.path.join(_HERE, "art_list_oracle.h"), os.path.join(d, "art_list_oracle.h"))
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-w", "-o", out_path, c_path, "-lm"])
    return out_path


def load_library(path: str):
    lib = ctypes.CDLL(path)
    lib.artref_block_list.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        _lib = load_library(_LIB)
    return _lib


def block_list(q, k_cache, page_table, seq_lens, *, block_size: int, num_q_heads: int,
               policy: int = IMPORTANCE, score_kind: int = KEY_NORM, budget: int,
               sink_blocks: int = 0, keep_last: bool = False, max_list: int | None = None,
               _lib=None):
    """Traversal lists per (sequence, KV head).

    k_cache bf16 [P][Hkv][Ps][D] (contiguous); q bf16 [B][Hq][D] (needed for
    QUERY_BOUND); page_table int32 [B][max_pages]; seq_lens int32 [B].
    Returns dict(list int32 [B][Hkv][max_list] (-1 past the length),
    len int32 [B][Hkv], scores fp64 [B][Hkv][max_blocks] (importance; NaN
    past each sequence's blocks)).
    """
    lib = _lib if _lib is not None else _load()
    kb = _bits(k_cache)
    P, Hkv, Ps, D = kb.shape
    pt = _i32(page_table)
    sl = _i32(seq_lens)
    B = sl.shape[0]
    max_blocks = (pt.shape[1] * Ps + block_size - 1) // block_size
    if max_list is None:
        max_list = max(1, max_blocks)
    qb = None if q is None else _bits(q)
    sh = ListShape(batch=B, num_q_heads=num_q_heads, num_kv_heads=Hkv, head_dim=D,
                   block_size=block_size, page_size=Ps, num_pages=P,
                   max_pages_per_seq=pt.shape[1], max_blocks_per_list=max_list,
                   k_stride_page=Hkv * Ps * D, k_stride_head=Ps * D, k_stride_token=D)
    op = ListOpts(policy=policy, score_kind=score_kind, budget=budget, sink_blocks=sink_blocks,
                  keep_last=1 if keep_last else 0)
    out = np.full((B, Hkv, max_list), -1, dtype=np.int32)
    ln = np.zeros((B, Hkv), dtype=np.int32)
    sc = np.full((B, Hkv, max(1, max_blocks)), np.nan)
    rc = lib.artref_block_list(ctypes.byref(sh), ctypes.byref(op), _ptr(qb, ctypes.c_uint16),
                               _ptr(kb, ctypes.c_uint16), _ptr(pt, ctypes.c_int32),
                               _ptr(sl, ctypes.c_int32), _ptr(out, ctypes.c_int32),
                               _ptr(ln, ctypes.c_int32), _ptr(sc, ctypes.c_double),
                               ctypes.c_int32(max(1, max_blocks)))
    if rc != 0:
        raise ValueError(f"list oracle rejected the input (code {rc})")
    return {"list": out, "len": ln, "scores": sc}
