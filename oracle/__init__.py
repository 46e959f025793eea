"""CPU fp64 oracle for ART decode attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never calls it.

``decode(...)`` wraps ``artref_decode`` from ``art_oracle.c`` (plain C, fp64,
OpenMP across (sequence, KV head) groups); ``build()`` compiles it with gcc.
See ``art_oracle.c`` for the paper passages it follows and the readings taken
where the paper is silent.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "art_oracle.c")
_DEFAULT_LIB = os.path.join(_HERE, "libart_oracle.so")
# ART_ORACLE_LIBRARY names another build of the same source (the host-ASan
# test runs the CPU suite against an AddressSanitizer build)
_LIB = os.environ.get("ART_ORACLE_LIBRARY") or _DEFAULT_LIB
ASAN_LIB = os.path.join(_HERE, "libart_oracle_asan.so")
_lib = None

OK = 0
ERR_ARG = 1
ERR_INDEX = 5


class Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "batch", "num_q_heads", "num_kv_heads", "head_dim", "block_size",
        "page_size", "num_pages", "max_pages_per_seq", "max_blocks_per_list",
        "list_per_head")] + [(n, ctypes.c_int64) for n in (
            "k_stride_page", "k_stride_head", "k_stride_token",
            "v_stride_page", "v_stride_head", "v_stride_token")]


class Opts(ctypes.Structure):
    _fields_ = [("scale", ctypes.c_double), ("tau", ctypes.c_double),
                ("phi", ctypes.c_double), ("patience", ctypes.c_int32),
                ("dense_order", ctypes.c_int32), ("probe_stride", ctypes.c_int32),
                ("scale_of_accumulator", ctypes.c_int32), ("per_head_stop", ctypes.c_int32)]


def build(force: bool = True) -> str:
    """Compile the oracle (and the traversal-list oracle, ``oracle.lists``)
    with gcc (-O2, fp-contract off, OpenMP)."""
    if _LIB != _DEFAULT_LIB:      # another build was named: leave it alone
        return _LIB
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
               "-ffp-contract=off", "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB)
    from . import lists
    lists.build(force=force)
    return _LIB


def build_asan() -> tuple:
    """AddressSanitizer builds of the oracle and the list oracle (gcc; the
    process that loads them preloads gcc's libasan)."""
    from . import lists
    flags = ["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fno-omit-frame-pointer",
             "-fsanitize=address", "-ffp-contract=off", "-Wall"]
    subprocess.check_call([*flags, "-fopenmp", "-o", ASAN_LIB, _SRC, "-lm"])
    subprocess.check_call([*flags, "-o", lists.ASAN_LIB, lists._SRC, "-lm"])
    return ASAN_LIB, lists.ASAN_LIB


def load_library(path: str):
    """Load an oracle build at ``path`` (tests use this for planted-mistake
    builds of the same source)."""
    lib = ctypes.CDLL(path)
    lib.artref_decode.restype = ctypes.c_int
    lib.artref_max_threads.restype = ctypes.c_int
    return lib


def build_variant(src_text: str, out_path: str) -> str:
    """Compile ``src_text`` (a modified copy of art_oracle.c) to ``out_path``."""
    d = os.path.dirname(out_path)
    c_path = os.path.join(d, "variant.c")
    with open(c_path, "w") as f:
        f.write(src_text)
    import shutil
    shutil.copy(os.path.join(_HERE, "art_oracle.h"), os.path.join(d, "art_oracle.h"))
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                           "-ffp-contract=off", "-w", "-o", out_path, c_path, "-lm"])
    return out_path


def source_text() -> str:
    with open(_SRC) as f:
        return f.read()


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        lib.artref_decode.restype = ctypes.c_int
        lib.artref_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def max_threads() -> int:
    return int(_load().artref_max_threads())


def _bits(x) -> np.ndarray:
    """bf16 torch tensor or uint16 numpy array -> contiguous uint16 numpy."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            x = x.detach().cpu().contiguous()
            if x.dtype == torch.bfloat16:
                x = x.view(torch.int16)
            return x.numpy().view(np.uint16)
    except ImportError:  # pragma: no cover
        pass
    a = np.ascontiguousarray(x)
    if a.dtype != np.uint16:
        raise TypeError("bf16 inputs are passed as uint16 bit patterns")
    return a


def _i32(x) -> Optional[np.ndarray]:
    if x is None:
        return None
    try:
        import torch
        if isinstance(x, torch.Tensor):
            x = x.detach().cpu()
            return np.ascontiguousarray(x.numpy().astype(np.int32, copy=False))
    except ImportError:  # pragma: no cover
        pass
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def _ptr(a, ctype):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctype))


class OracleError(RuntimeError):
    def __init__(self, code: int, group: int):
        super().__init__(f"oracle rejected input (code {code}, group {group})")
        self.code = code
        self.group = group


def decode(q, k_cache, v_cache, page_table, seq_lens, *, block_size: int,
           scale: float, tau: float, phi: float, patience: int,
           dense_order: int = 0, block_list=None, block_list_len=None,
           list_per_head: bool = True, force_stop=None, group_mask=None,
           trace_steps: int = 0, num_threads: int = 0, probe_stride: int = 1,
           scale_of_accumulator: bool = False, per_head_stop: bool = False, _lib=None):
    """Run the oracle.

    q: bf16 [B][Hq][D]; k_cache/v_cache: bf16 [P][Hkv][Ps][D] (contiguous);
    page_table int32 [B][max_pages]; seq_lens int32 [B];
    block_list int32 [B][Hkv][n] (list_per_head) or [B][n]; block_list_len
    int32 [B][Hkv] or [B].  ``scale``, ``tau`` and ``phi`` are rounded to
    fp32 first, since the kernel receives fp32 values.  ``probe_stride`` s
    makes the stability test look at coordinates 0, s, 2s, ... of each head's
    output only (1 = the whole output).  ``scale_of_accumulator`` takes
    d_scale on the unnormalised accumulator l(t) o(t) instead of o(t).
    ``per_head_stop`` gives every query head its own counter and stop
    (force_stop is then [B][Hq]); the result then has ``head_stop`` [B][Hq].

    Returns dict(out fp64 [B][Hq][D], lse fp64 [B][Hq], stop int32 [B][Hkv],
    trace fp64 [B][Hkv][trace_steps][g][2] or None).
    """
    lib = _lib if _lib is not None else _load()
    qb, kb, vb = _bits(q), _bits(k_cache), _bits(v_cache)
    if kb.ndim != 4 or vb.shape != kb.shape or qb.ndim != 3:
        raise ValueError("q must be [B][Hq][D], caches [P][Hkv][Ps][D]")
    B, Hq, D = qb.shape
    P, Hkv, Ps, D2 = kb.shape
    if D2 != D:
        raise ValueError("head_dim mismatch")
    pt = _i32(page_table)
    sl = _i32(seq_lens)
    bl = _i32(block_list)
    bll = _i32(block_list_len)
    fs = _i32(force_stop)
    gm = None if group_mask is None else np.ascontiguousarray(np.asarray(group_mask, dtype=np.uint8))
    sh = Shape(batch=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D,
               block_size=block_size, page_size=Ps, num_pages=P,
               max_pages_per_seq=pt.shape[1],
               max_blocks_per_list=0 if bl is None else bl.shape[-1],
               list_per_head=1 if list_per_head else 0,
               k_stride_page=Hkv * Ps * D, k_stride_head=Ps * D, k_stride_token=D,
               v_stride_page=Hkv * Ps * D, v_stride_head=Ps * D, v_stride_token=D)
    op = Opts(scale=float(np.float32(scale)), tau=float(np.float32(tau)),
              phi=float(np.float32(phi)), patience=int(patience),
              dense_order=int(dense_order), probe_stride=int(probe_stride),
              scale_of_accumulator=1 if scale_of_accumulator else 0,
              per_head_stop=1 if per_head_stop else 0)
    g = Hq // Hkv
    out = np.zeros((B, Hq, D), dtype=np.float64)
    lse = np.full((B, Hq), np.nan, dtype=np.float64)
    stop = np.full((B, Hkv), -1, dtype=np.int32)
    head_stop = np.full((B, Hq), -1, dtype=np.int32)
    trace = np.full((B, Hkv, trace_steps, g, 2), np.nan) if trace_steps > 0 else None
    err = ctypes.c_int32(-1)
    rc = lib.artref_decode(
        ctypes.byref(sh), ctypes.byref(op),
        _ptr(qb, ctypes.c_uint16), _ptr(kb, ctypes.c_uint16), _ptr(vb, ctypes.c_uint16),
        _ptr(pt, ctypes.c_int32), _ptr(sl, ctypes.c_int32),
        _ptr(bl, ctypes.c_int32), _ptr(bll, ctypes.c_int32), _ptr(fs, ctypes.c_int32),
        _ptr(gm, ctypes.c_uint8),
        _ptr(out, ctypes.c_double), _ptr(lse, ctypes.c_double), _ptr(stop, ctypes.c_int32),
        _ptr(head_stop, ctypes.c_int32),
        _ptr(trace, ctypes.c_double), ctypes.c_int32(trace_steps),
        ctypes.c_int32(num_threads), ctypes.byref(err))
    if rc != OK:
        raise OracleError(rc, err.value)
    return {"out": out, "lse": lse, "stop": stop, "head_stop": head_stop, "trace": trace}


def decode_workload(wl, *, tau=None, phi=None, patience=None, dense_order=None,
                    force_stop=None, group_mask=None, trace_steps=0, num_threads=0,
                    probe_stride=1, scale_of_accumulator=False, per_head_stop=False,
                    _lib=None):
    """Oracle on a ``paper_2606_00024_amd.workloads.Workload`` (host copies)."""
    s = wl.spec
    return decode(wl.q, wl.k_cache, wl.v_cache, wl.page_table, wl.seq_lens,
                  block_size=s.block_size, scale=s.softmax_scale,
                  tau=s.tau if tau is None else tau,
                  phi=s.phi if phi is None else phi,
                  patience=s.patience if patience is None else patience,
                  dense_order=s.dense_order if dense_order is None else dense_order,
                  block_list=wl.block_list, block_list_len=wl.block_list_len,
                  force_stop=force_stop, group_mask=group_mask,
                  trace_steps=trace_steps, num_threads=num_threads,
                  probe_stride=probe_stride, scale_of_accumulator=scale_of_accumulator,
                  per_head_stop=per_head_stop, _lib=_lib)
