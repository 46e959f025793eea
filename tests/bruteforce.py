"""Brute-force references written straight from the paper's definitions.

Independent of the oracle's streaming recurrence: every quantity here is
recomputed from scratch with a full softmax over an explicit token set.

* ``softmax_attention``: Eq. (1), O = softmax(q K^T s) V, plus ln sum exp.
* ``prefix_outputs``: o(t) = attention over the tokens of the first t
  traversal blocks (the quantity the block-streaming kernel holds after t
  blocks, Sec. 3.1), for every t.
* ``stop_from_trajectory``: Eq. (2) metrics against o(0) = 0 (Algorithm 1),
  the stability rule of Sec. 3.2 and the patience rule of Eq. (3).
"""
from __future__ import annotations

import math

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def to_f64(x) -> np.ndarray:
    import torch
    if isinstance(x, torch.Tensor):
        x = x.detach().cpu().contiguous()
        if x.dtype == torch.bfloat16:
            return bf16_bits_to_f64(x.view(torch.int16).numpy().view(np.uint16))
        return x.double().numpy()
    a = np.asarray(x)
    if a.dtype == np.uint16:
        return bf16_bits_to_f64(a)
    return a.astype(np.float64)


def traversal_list(seq_len: int, block_size: int, dense_order: int = 0,
                   block_list=None, list_len=None) -> list[int]:
    nblk = -(-seq_len // block_size) if seq_len > 0 else 0
    if block_list is not None:
        return [int(x) for x in np.asarray(block_list)[: int(list_len)]]
    if dense_order == 1:
        return list(range(nblk))
    return list(range(nblk - 1, -1, -1))


class Group:
    """Dense fp64 copies of one (sequence, KV head) group's inputs."""

    def __init__(self, q, k_cache, v_cache, page_table, seq_lens, b, kvh,
                 block_size, dense_order=0, block_list=None, block_list_len=None):
        qf = to_f64(q)
        kc = to_f64(k_cache)
        vc = to_f64(v_cache)
        pt = np.asarray(page_table.cpu() if hasattr(page_table, "cpu") else page_table)
        sl = np.asarray(seq_lens.cpu() if hasattr(seq_lens, "cpu") else seq_lens)
        Hq = qf.shape[1]
        Hkv = kc.shape[1]
        g = Hq // Hkv
        Ps = kc.shape[2]
        self.L = int(sl[b])
        self.block_size = block_size
        self.q = qf[b, kvh * g:(kvh + 1) * g]                      # [g][D]
        toks = np.arange(self.L)
        pages = pt[b, toks // Ps] if self.L else np.zeros(0, dtype=np.int64)
        self.K = kc[pages, kvh, toks % Ps] if self.L else np.zeros((0, qf.shape[2]))
        self.V = vc[pages, kvh, toks % Ps] if self.L else np.zeros((0, qf.shape[2]))
        bl = None if block_list is None else np.asarray(block_list.cpu() if hasattr(block_list, "cpu") else block_list)[b, kvh]
        bll = None if block_list_len is None else int(np.asarray(block_list_len.cpu() if hasattr(block_list_len, "cpu") else block_list_len)[b, kvh])
        self.blocks = traversal_list(self.L, block_size, dense_order, bl, bll)

    def block_tokens(self, blk: int) -> np.ndarray:
        j0 = blk * self.block_size
        return np.arange(j0, min(j0 + self.block_size, self.L))

    def tokens_of(self, blocks) -> np.ndarray:
        if not blocks:
            return np.zeros(0, dtype=np.int64)
        return np.concatenate([self.block_tokens(b) for b in blocks])


def softmax_attention(qh: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float):
    """Eq. (1) for each query row: (out [g][D], lse [g])."""
    if K.shape[0] == 0:
        return np.zeros((qh.shape[0], V.shape[1])), np.full(qh.shape[0], -np.inf)
    s = scale * (qh @ K.T)                      # [g][n]
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    z = e.sum(axis=1, keepdims=True)
    return (e / z) @ V, (m + np.log(z))[:, 0]


def prefix_outputs(grp: Group, scale: float, upto=None):
    """o(t) for t = 0..T (o(0) = 0) plus per-block mass l(t) and A(t) and
    block outputs u(t) (Appendix A), all by direct evaluation."""
    T = len(grp.blocks) if upto is None else min(upto, len(grp.blocks))
    g, D = grp.q.shape
    o = [np.zeros((g, D))]
    lse = [np.full(g, -np.inf)]
    u, logl = [None], [None]
    for t in range(1, T + 1):
        toks = grp.tokens_of(grp.blocks[:t])
        out, ls = softmax_attention(grp.q, grp.K[toks], grp.V[toks], scale)
        o.append(out)
        lse.append(ls)
        bt = grp.block_tokens(grp.blocks[t - 1])
        ub, lb = softmax_attention(grp.q, grp.K[bt], grp.V[bt], scale)
        u.append(ub)
        logl.append(lb)
    return {"o": o, "logA": lse, "u": u, "logl": logl}


def step_metrics(o_new: np.ndarray, o_old: np.ndarray):
    """Eq. (2) per head: (d_scale, d_direction); d_direction is NaN when a
    vector is zero (the cosine is undefined)."""
    ds = np.linalg.norm(o_new - o_old, axis=1)
    n1 = np.linalg.norm(o_new, axis=1)
    n0 = np.linalg.norm(o_old, axis=1)
    with np.errstate(invalid="ignore", divide="ignore"):
        dr = 1.0 - np.sum(o_new * o_old, axis=1) / (n1 * n0)
    dr = np.where((n1 > 0) & (n0 > 0), dr, np.nan)
    return ds, dr


def stop_from_trajectory(o_traj, tau: float, phi: float, patience: int,
                         use_scale=True, use_direction=True, probe=None):
    """Apply Sec. 3.2 / Eq. (3) / Algorithm 1 to a trajectory o(0..T).
    ``probe`` is an optional linear map P (an m x D matrix): the metrics are
    then taken on x(t) = P o(t) (Appendix A) instead of o(t).
    Returns (t_star, [(d_scale, d_direction) per step])."""
    T = len(o_traj) - 1
    if probe is not None:
        o_traj = [o @ np.asarray(probe).T for o in o_traj]
    c = 0
    mets = []
    for t in range(1, T + 1):
        ds, dr = step_metrics(o_traj[t], o_traj[t - 1])
        mets.append((ds, dr))
        ok = np.ones_like(ds, dtype=bool)
        if use_scale:
            ok &= ds < tau
        if use_direction:
            ok &= dr < phi
        else:
            ok &= ~np.isnan(dr)
        c = c + 1 if bool(ok.all()) else 0
        if c >= patience:
            return t, mets
    return T, mets


def float32(x: float) -> float:
    return float(np.float32(x))


def ln_ratio(T: int, t: int) -> float:
    return math.log(T / t)
