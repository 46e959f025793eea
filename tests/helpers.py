"""Small synthetic inputs for CPU tests (shared by oracle pins and GPU parity)."""
from __future__ import annotations

import numpy as np
import torch

from paper_2606_00024_amd import workloads as W


def small_workload(seed: int, *, batch=1, kv_heads=2, group=4, seq_len=1024,
                   block_size=64, page_size=64, dense_order=0, list_fraction=None,
                   tau=1e-3, phi=1e-4, patience=5, needles=2, device="cpu",
                   nan_fill=True) -> W.Workload:
    spec = W.WorkloadSpec(
        name=f"small{seed}", batch=batch, num_q_heads=kv_heads * group,
        num_kv_heads=kv_heads, seq_lens=seq_len if isinstance(seq_len, tuple) else (seq_len,) * batch,
        block_size=block_size, page_size=page_size, dense_order=dense_order,
        list_fraction=list_fraction, tau=tau, phi=phi, patience=patience,
        n_needles=needles, n_outliers=4, seed=seed)
    return W.make_workload(spec, device=device, nan_fill=nan_fill)


def random_lists(wl: W.Workload, seed: int, fraction=0.5):
    """Random per-(b, kvh) block lists (unique ids, random order)."""
    rng = np.random.default_rng(seed)
    s = wl.spec
    lens = wl.seq_lens.cpu().tolist()
    nbs = [(L + s.block_size - 1) // s.block_size for L in lens]
    nmax = max(1, max(nbs))
    bl = np.full((s.batch, s.num_kv_heads, nmax), -1, dtype=np.int32)
    bll = np.zeros((s.batch, s.num_kv_heads), dtype=np.int32)
    for b, n in enumerate(nbs):
        for h in range(s.num_kv_heads):
            k = max(1, int(round(fraction * n))) if n else 0
            ids = rng.permutation(n)[:k]
            bl[b, h, :k] = ids
            bll[b, h] = k
    return torch.from_numpy(bl), torch.from_numpy(bll)


def uniform_key_case(values_per_step, block_size=64, head_dim=128, group=1,
                     seed=0):
    """K == 0, value rows of the block visited at traversal step t (dense
    recency-first) all equal values_per_step[t-1] (a length-head_dim vector).
    Identity page table, page_size == block_size."""
    T = len(values_per_step)
    L = T * block_size
    rng = np.random.default_rng(seed)
    q = torch.from_numpy(rng.standard_normal((1, group, head_dim)).astype(np.float32)).to(torch.bfloat16)
    k = torch.zeros((T, 1, block_size, head_dim), dtype=torch.bfloat16)
    v = torch.zeros((T, 1, block_size, head_dim), dtype=torch.float32)
    for t, vec in enumerate(values_per_step, start=1):
        blk = T - t  # recency-first: step t visits block T - t
        v[blk, 0, :, :] = torch.as_tensor(np.asarray(vec, dtype=np.float32))
    v = v.to(torch.bfloat16)
    pt = torch.arange(T, dtype=torch.int32).view(1, T)
    sl = torch.tensor([L], dtype=torch.int32)
    return q, k, v, pt, sl


def exact_tie_case(T=6, head_dim=128, block_size=64, seed=0):
    """Step 1 (the last block, recency-first) has zero keys; every other block
    has keys -11314 * e_0 against the query e_0, i.e. scores near -1000 with
    scale 1/sqrt(128).  Their weight exp(-1000 - ln 64) underflows to exactly
    0 in fp64, so o(t) == o(t-1) bit for bit for t >= 2: d_scale is exactly 0."""
    rng = np.random.default_rng(seed)
    q = torch.zeros((1, 1, head_dim), dtype=torch.bfloat16)
    q[0, 0, 0] = 1.0
    k = torch.zeros((T, 1, block_size, head_dim), dtype=torch.float32)
    k[: T - 1, 0, :, 0] = -11314.0
    v = torch.from_numpy(rng.standard_normal((T, 1, block_size, head_dim)).astype(np.float32))
    pt = torch.arange(T, dtype=torch.int32).view(1, T)
    sl = torch.tensor([T * block_size], dtype=torch.int32)
    return q, k.to(torch.bfloat16), v.to(torch.bfloat16), pt, sl
