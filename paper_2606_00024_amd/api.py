"""PyTorch-facing binding of the ART decode-attention library.

PyTorch provides device memory and the stream; every step of the computation
runs in the HIP kernels of libart.so (include/art.h).  This module only
checks tensor layouts, builds the ABI structs and passes pointers.
"""
from __future__ import annotations

import math
import threading
from typing import Optional

import torch

from . import _lib
from ._lib import ArtError, DecodeOpts, DecodeShape

_ws_lock = threading.Lock()
_ws_cache: dict = {}


def _ptr(t: Optional[torch.Tensor]) -> int:
    return 0 if t is None else int(t.data_ptr())


def _require_cuda(t: torch.Tensor, name: str, dtype=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")


def make_shape(q, k_cache, v_cache, page_table, *, block_size: int, block_list=None,
               list_per_head: bool = True) -> DecodeShape:
    """ABI shape from tensors: q [B][Hq][D], caches [P][Hkv][Ps][D] (any
    strides with a unit head-dim stride), page_table [B][max_pages]."""
    B, Hq, D = q.shape
    P, Hkv, Ps, D2 = k_cache.shape
    if D2 != D or tuple(v_cache.shape) != tuple(k_cache.shape):
        raise ValueError("k_cache/v_cache must both be [pages][kv_heads][page_size][head_dim]")
    if k_cache.stride(3) != 1 or v_cache.stride(3) != 1:
        raise ValueError("head_dim must be the innermost (unit-stride) dimension")
    ks, vs = k_cache.stride(), v_cache.stride()
    return DecodeShape(
        batch=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, block_size=int(block_size),
        page_size=Ps, num_pages=P, max_pages_per_seq=int(page_table.shape[1]),
        max_blocks_per_list=0 if block_list is None else int(block_list.shape[-1]),
        list_per_head=1 if list_per_head else 0,
        k_stride_page=ks[0], k_stride_head=ks[1], k_stride_token=ks[2],
        v_stride_page=vs[0], v_stride_head=vs[1], v_stride_token=vs[2])


def make_opts(*, softmax_scale: float, tau: float, phi: float, patience: int,
              dense_order: int = 0, out_dtype=torch.float32, chunk_blocks: int = 0,
              probe_stride: int = 1, scale_of_accumulator: bool = False,
              no_detector: bool = False, max_wait_polls: int = 0,
              per_head_stop: bool = False, max_ahead_chunks: int = 0) -> DecodeOpts:
    od = _lib.OUT_BF16 if out_dtype == torch.bfloat16 else _lib.OUT_F32
    if out_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out_dtype must be float32 or bfloat16")
    return DecodeOpts(softmax_scale=float(softmax_scale), tau=float(tau), phi=float(phi),
                      patience=int(patience), dense_order=int(dense_order), out_dtype=od,
                      chunk_blocks=int(chunk_blocks), probe_stride=int(probe_stride),
                      scale_of_accumulator=1 if scale_of_accumulator else 0,
                      no_detector=1 if no_detector else 0,
                      max_wait_polls=int(max_wait_polls),
                      per_head_stop=1 if per_head_stop else 0,
                      max_ahead_chunks=int(max_ahead_chunks))


def workspace_bytes(shape: DecodeShape, opts: DecodeOpts) -> int:
    return _lib.workspace_bytes(shape, opts)


def new_workspace(nbytes: int, device) -> torch.Tensor:
    """A zero-filled workspace (the state art_workspace_init leaves)."""
    n = max(256, (int(nbytes) + 255) // 256 * 256)
    ws = torch.empty(n, dtype=torch.uint8, device=device)
    _lib.workspace_init(_ptr(ws), n, torch.cuda.current_stream(ws.device).cuda_stream)
    return ws


def _cached_workspace(nbytes: int, device, stream) -> torch.Tensor:
    key = (device.index if device.index is not None else torch.cuda.current_device(),
           int(stream))
    with _ws_lock:
        ws = _ws_cache.get(key)
        if ws is None or ws.numel() < nbytes:
            ws = new_workspace(max(nbytes, 1 << 20), device)
            _ws_cache[key] = ws
        return ws


def decode_attention(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                     page_table: torch.Tensor, seq_lens: torch.Tensor, *,
                     block_size: int, tau: float, phi: float, patience: int,
                     softmax_scale: Optional[float] = None, dense_order: int = 0,
                     block_list: Optional[torch.Tensor] = None,
                     block_list_len: Optional[torch.Tensor] = None,
                     list_per_head: bool = True, out_dtype=torch.float32,
                     chunk_blocks: int = 0, probe_stride: int = 1,
                     scale_of_accumulator: bool = False, no_detector: bool = False,
                     max_wait_polls: int = 0, per_head_stop: bool = False,
                     max_ahead_chunks: int = 0,
                     workspace: Optional[torch.Tensor] = None,
                     out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                     stop_block: Optional[torch.Tensor] = None):
    """ART decode attention on the current stream.

    Returns (out [B][Hq][D] out_dtype, lse [B][Hq] fp32, stop_block [B][Hkv]
    int32).  ``workspace`` (uint8, zero-filled before its first use, e.g. by
    ``new_workspace``) defaults to a per-(device, stream) cached buffer.
    ``probe_stride`` s > 1 makes the stability test look at every s-th
    coordinate of each head's output only (Sec. 3.2's subsampled probe).
    ``scale_of_accumulator`` takes d_scale on the unnormalised accumulator
    l(t) o(t) instead of o(t).  ``no_detector`` runs without the stability
    test at all (full attention over the traversal).  ``max_wait_polls``
    n > 0 makes every wait of the kernel give up after n polls (the call then
    reports ART_ERR_DEVICE_TIMEOUT through ``workspace_status``).
    ``per_head_stop`` gives every query head its own patience counter and stop
    (out and lse at the head's own stop; stop_block is then [B][Hq], each
    head's stop).  ``max_ahead_chunks`` n > 0 bounds the reads past a stop:
    a chunk of a traversal is loaded only once the chunk n before it has been
    through the stability test (the results are the same bits).
    """
    _require_cuda(q, "q", torch.bfloat16)
    _require_cuda(k_cache, "k_cache", torch.bfloat16)
    _require_cuda(v_cache, "v_cache", torch.bfloat16)
    _require_cuda(page_table, "page_table", torch.int32)
    _require_cuda(seq_lens, "seq_lens", torch.int32)
    if not q.is_contiguous() or not page_table.is_contiguous() or not seq_lens.is_contiguous():
        raise ValueError("q, page_table and seq_lens must be contiguous")
    if (block_list is None) != (block_list_len is None):
        raise ValueError("block_list and block_list_len go together")
    if block_list is not None:
        _require_cuda(block_list, "block_list", torch.int32)
        _require_cuda(block_list_len, "block_list_len", torch.int32)
        if not block_list.is_contiguous() or not block_list_len.is_contiguous():
            raise ValueError("block_list and block_list_len must be contiguous")
    B, Hq, D = q.shape
    Hkv = k_cache.shape[1]
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(D)
    shape = make_shape(q, k_cache, v_cache, page_table, block_size=block_size,
                       block_list=block_list, list_per_head=list_per_head)
    opts = make_opts(softmax_scale=softmax_scale, tau=tau, phi=phi, patience=patience,
                     dense_order=dense_order, out_dtype=out_dtype, chunk_blocks=chunk_blocks,
                     probe_stride=probe_stride, scale_of_accumulator=scale_of_accumulator,
                     no_detector=no_detector, max_wait_polls=max_wait_polls,
                     per_head_stop=per_head_stop, max_ahead_chunks=max_ahead_chunks)
    dev = q.device
    if out is None:
        out = torch.empty((B, Hq, D), dtype=out_dtype, device=dev)
    if lse is None:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    if stop_block is None:
        stop_block = torch.empty((B, Hq if per_head_stop else Hkv), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    need = workspace_bytes(shape, opts)
    ws = workspace if workspace is not None else _cached_workspace(need, dev, stream)
    st = _lib.decode_attention(shape, opts, _ptr(q), _ptr(k_cache), _ptr(v_cache),
                               _ptr(page_table), _ptr(seq_lens), _ptr(block_list),
                               _ptr(block_list_len), _ptr(out), _ptr(lse), _ptr(stop_block),
                               _ptr(ws), ws.numel(), stream)
    if st != _lib.OK:
        raise ArtError(st, "art_decode_attention")
    return out, lse, stop_block


def decode_workload(wl, *, tau=None, phi=None, patience=None, dense_order=None,
                    out_dtype=torch.float32, chunk_blocks: int = 0, workspace=None, **kw):
    """decode_attention on a ``workloads.Workload`` resident on the GPU."""
    s = wl.spec
    return decode_attention(
        wl.q, wl.k_cache, wl.v_cache, wl.page_table, wl.seq_lens,
        block_size=s.block_size, softmax_scale=s.softmax_scale,
        tau=s.tau if tau is None else tau, phi=s.phi if phi is None else phi,
        patience=s.patience if patience is None else patience,
        dense_order=s.dense_order if dense_order is None else dense_order,
        block_list=wl.block_list, block_list_len=wl.block_list_len,
        out_dtype=out_dtype, chunk_blocks=chunk_blocks, workspace=workspace, **kw)


def validate_inputs(q, k_cache, v_cache, page_table, seq_lens, *, block_size: int,
                    block_list=None, block_list_len=None, list_per_head: bool = True):
    """Checked mode (synchronous): returns (status, bad_index, where)."""
    shape = make_shape(q, k_cache, v_cache, page_table, block_size=block_size,
                       block_list=block_list, list_per_head=list_per_head)
    opts = make_opts(softmax_scale=1.0, tau=0.0, phi=0.0, patience=1)
    stream = torch.cuda.current_stream(q.device).cuda_stream
    return _lib.validate_inputs(shape, opts, _ptr(page_table), _ptr(seq_lens),
                                _ptr(block_list), _ptr(block_list_len), stream)


def workspace_status(ws: torch.Tensor) -> int:
    """ART_OK or ART_ERR_DEVICE_TIMEOUT for calls that used ``ws`` (syncs)."""
    return _lib.workspace_status(_ptr(ws), ws.numel(), torch.cuda.current_stream(ws.device).cuda_stream)


def build_block_list(q: torch.Tensor, k_cache: torch.Tensor, page_table: torch.Tensor,
                     seq_lens: torch.Tensor, *, block_size: int, budget: int,
                     policy: int = _lib.LIST_IMPORTANCE, score_kind: int = _lib.SCORE_KEY_NORM,
                     sink_blocks: int = 0, keep_last: bool = False,
                     max_list: Optional[int] = None, return_scores: bool = False):
    """Traversal lists for decode_attention (Sec. 3.4), built on the current
    stream: importance-first (block scores, top-`budget` with forced sink /
    last blocks, descending score) or streaming (sinks first, then the
    `budget` most recent blocks).

    q bf16 [B][Hq][D] (the shape source; read for the query bound only),
    k_cache bf16 [P][Hkv][Ps][D], page_table int32 [B][max_pages], seq_lens
    int32 [B].  Returns (block_list int32 [B][Hkv][max_list], block_list_len
    int32 [B][Hkv]) and, with return_scores, the fp64 block scores
    [B][Hkv][max_blocks].  Entries past a row's length are -1.
    """
    _require_cuda(q, "q", torch.bfloat16)
    _require_cuda(k_cache, "k_cache", torch.bfloat16)
    _require_cuda(page_table, "page_table", torch.int32)
    _require_cuda(seq_lens, "seq_lens", torch.int32)
    if not q.is_contiguous() or not page_table.is_contiguous() or not seq_lens.is_contiguous():
        raise ValueError("q, page_table and seq_lens must be contiguous")
    B, Hq, D = q.shape
    P, Hkv, Ps, _ = k_cache.shape
    max_blocks = (int(page_table.shape[1]) * Ps + block_size - 1) // block_size
    if max_list is None:
        max_list = max(1, max_blocks)
    dev = q.device
    bl = torch.full((B, Hkv, max_list), -1, dtype=torch.int32, device=dev)
    bll = torch.zeros((B, Hkv), dtype=torch.int32, device=dev)
    shape = make_shape(q, k_cache, k_cache, page_table, block_size=block_size, block_list=bl)
    opts = _lib.ListOpts(policy=int(policy), score_kind=int(score_kind), budget=int(budget),
                         sink_blocks=int(sink_blocks), keep_last=1 if keep_last else 0)
    _lib.block_list_workspace_bytes(shape, opts)  # raises on invalid input
    scores = torch.full((B, Hkv, max(1, max_blocks)), float("nan"), dtype=torch.float64,
                        device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    st = _lib.build_block_list(shape, opts, _ptr(q), _ptr(k_cache), _ptr(page_table),
                               _ptr(seq_lens), _ptr(bl), _ptr(bll), _ptr(scores), 0, 0, stream)
    if st != _lib.OK:
        raise ArtError(st, "art_build_block_list")
    return (bl, bll, scores) if return_scores else (bl, bll)
