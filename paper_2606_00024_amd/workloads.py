"""Seeded synthetic decode-attention workloads.

This module produces the *inputs* of one decode-attention step: a bf16 query,
a paged bf16 K/V pool, the page table, per-sequence lengths and (optionally) a
per-(sequence, KV head) block list.  It holds none of the attention or
termination arithmetic; both the HIP path and the CPU oracle consume the exact
arrays it returns.

Structure of the synthetic cache (stand-ins for the paper's long-context
workloads, whose datasets are not available here):

* Q ~ N(0, I_d) per query head; with scale 1/sqrt(d) haystack logits are
  roughly N(0, 1).
* Haystack K and V ~ N(0, I_d).
* Per (sequence, KV head) group a direction u = normalize(sum of the group's
  query heads) is formed.
* "Sink" keys at positions 0..3 and "needle" keys at random positions are
  ``needle_gain * sqrt(d) * u + N(0, I)``: they dominate the attention mass,
  the retrieval-style regime the paper's needle-in-a-haystack study probes
  (Sec. 4, RULER NIAH).
* "Outlier" tokens get keys ``-sqrt(d) * u + N(0, I)`` (low score) and values
  ``10 * N(0, I)``: low-attention tokens with large value norm, the case the
  paper's Fig. 1 discussion uses to argue that key-only importance misses
  value contributions.
* Pages of all sequences are a random permutation inside one pool laid out
  [page][kv_head][token_in_page][d].  Slots past a sequence's length and pages
  no sequence uses are filled with NaN, so that any read of them shows up.
* For the sparse-policy workload a block list per (sequence, KV head) holds
  a fixed fraction of the blocks chosen by a key-norm score (max over the
  block of ||k_j||_2), always including block 0 and the last block, ordered
  by descending score with ties broken by ascending block id: the
  importance-first traversal of Sec. 3.4.

Values are drawn in fp32 and rounded to bf16 (round-to-nearest-even, torch's
conversion).  Generation runs on whatever device is given; the same seed gives
the same arrays on the same device type.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import Optional, Sequence

import torch

HEAD_DIM = 128
BF16_NAN = 0x7FC0

ORDER_RECENT_FIRST = 0
ORDER_FORWARD = 1


@dataclass(frozen=True)
class WorkloadSpec:
    """Shape, thresholds and generator knobs of one synthetic decode step."""

    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    seq_lens: Sequence[int] | tuple  # explicit lengths, or ("uniform", lo, hi)
    block_size: int = 64
    page_size: int = 64
    head_dim: int = HEAD_DIM
    dense_order: int = ORDER_RECENT_FIRST
    list_fraction: Optional[float] = None  # None: dense traversal
    tau: float = 1e-3
    phi: float = 1e-4
    patience: int = 5
    n_sinks: int = 4
    n_needles: int = 8
    n_outliers: int = 16
    needle_gain: float = 3.0
    outlier_vscale: float = 10.0
    # needle placement: None = uniform over the sequence; otherwise a list of
    # (count, lo_fraction, hi_fraction) bands.
    needle_bands: Optional[tuple] = None
    spare_pages: int = 3
    seed: int = 0

    @property
    def group_size(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)


def _c(name, **kw) -> WorkloadSpec:
    return WorkloadSpec(name=name, **kw)


# Named workloads.  Head shapes follow public model cards (Llama-3-8B: 32/8,
# Qwen3-32B: 64/8, head_dim 128).
WORKLOADS = {
    # tiny single-sequence step: 1 x 8/2 heads, 4K context, dense order
    "tiny_4k": _c("tiny_4k", batch=1, num_q_heads=8, num_kv_heads=2,
                  seq_lens=(4096,), seed=1),
    # Llama-3-8B-shaped decode layer: 8 x 32/8, 32K each, paged, dense order
    "llama3_8b_32k": _c("llama3_8b_32k", batch=8, num_q_heads=32,
                        num_kv_heads=8, seq_lens=(32768,) * 8, seed=2),
    # same heads with a sparse 25% importance-ordered block list, 128K context
    "sparse25_128k": _c("sparse25_128k", batch=4, num_q_heads=32,
                        num_kv_heads=8, seq_lens=(131072,) * 4,
                        list_fraction=0.25, seed=3),
    # Qwen3-32B-shaped ragged batch: 32 x 64/8, lengths U{8192..65536}
    "qwen3_32b_ragged": _c("qwen3_32b_ragged", batch=32, num_q_heads=64,
                           num_kv_heads=8, seq_lens=("uniform", 8192, 65536),
                           seed=4),
    # very long single sequence: 1 x 32/8, 512K context, block 128,
    # needles only in the first 5% and the last 1% of positions
    "long_512k": _c("long_512k", batch=1, num_q_heads=32, num_kv_heads=8,
                    seq_lens=(524288,), block_size=128, page_size=128,
                    needle_bands=((4, 0.0, 0.05), (4, 0.99, 1.0)), seed=5),
}

# thresholds swept on the ragged workload (tau = phi = value), plus the
# paper's default operating point (tau=1e-5, phi=1e-3), Sec. 4.1.
RAGGED_SWEEP = ((1e-2, 1e-2), (1e-3, 1e-3), (1e-4, 1e-4), (1e-5, 1e-3))


def scaled(spec: WorkloadSpec, *, batch=None, num_kv_heads=None,
           seq_len=None, **kw) -> WorkloadSpec:
    """A smaller variant of ``spec`` (same structure), for fast tests."""
    b = batch if batch is not None else spec.batch
    hkv = num_kv_heads if num_kv_heads is not None else spec.num_kv_heads
    g = spec.group_size
    if seq_len is None:
        lens = spec.seq_lens
        if isinstance(lens, tuple) and lens and lens[0] == "uniform":
            lens = lens
        else:
            lens = tuple(list(lens)[:1] * b)
    elif isinstance(seq_len, tuple) and seq_len and seq_len[0] == "uniform":
        lens = seq_len
    elif isinstance(seq_len, (list, tuple)):
        lens = tuple(seq_len)
    else:
        lens = (int(seq_len),) * b
    return replace(spec, batch=b, num_kv_heads=hkv, num_q_heads=hkv * g,
                   seq_lens=lens, **kw)


def resolve_seq_lens(spec: WorkloadSpec) -> list[int]:
    lens = spec.seq_lens
    if isinstance(lens, tuple) and lens and lens[0] == "uniform":
        _, lo, hi = lens
        g = torch.Generator(device="cpu").manual_seed(1_000_003 * spec.seed + 17)
        return [int(x) for x in torch.randint(lo, hi + 1, (spec.batch,), generator=g)]
    out = [int(x) for x in lens]
    if len(out) != spec.batch:
        raise ValueError(f"{spec.name}: {len(out)} lengths for batch {spec.batch}")
    return out


@dataclass
class Workload:
    spec: WorkloadSpec
    q: torch.Tensor            # bf16 [B][Hq][D]
    k_cache: torch.Tensor      # bf16 [P][Hkv][Ps][D]
    v_cache: torch.Tensor      # bf16 [P][Hkv][Ps][D]
    page_table: torch.Tensor   # int32 [B][max_pages]
    seq_lens: torch.Tensor     # int32 [B]
    block_list: Optional[torch.Tensor] = None      # int32 [B][Hkv][max_list]
    block_list_len: Optional[torch.Tensor] = None  # int32 [B][Hkv]
    needle_pos: dict = field(default_factory=dict)

    @property
    def num_pages(self) -> int:
        return int(self.k_cache.shape[0])

    @property
    def max_pages_per_seq(self) -> int:
        return int(self.page_table.shape[1])

    @property
    def max_blocks_per_list(self) -> int:
        return 0 if self.block_list is None else int(self.block_list.shape[2])

    def traversal_lengths(self) -> list[list[int]]:
        """T per (b, kvh): the number of blocks in the traversal set."""
        s = self.spec
        lens = self.seq_lens.cpu().tolist()
        if self.block_list_len is not None:
            return self.block_list_len.cpu().tolist()
        return [[(L + s.block_size - 1) // s.block_size] * s.num_kv_heads for L in lens]

    def kv_bytes_in_traversal(self) -> int:
        """bf16 K+V bytes of every token in the traversal set (all groups)."""
        s = self.spec
        lens = self.seq_lens.cpu().tolist()
        total_tokens = 0
        if self.block_list is None:
            total_tokens = sum(lens) * s.num_kv_heads
        else:
            bl = self.block_list.cpu()
            bll = self.block_list_len.cpu()
            for b, L in enumerate(lens):
                for h in range(s.num_kv_heads):
                    ids = bl[b, h, : int(bll[b, h])]
                    toks = torch.clamp(L - ids * s.block_size, max=s.block_size)
                    total_tokens += int(toks.sum())
        return total_tokens * 2 * s.head_dim * 2


def _fill_normal_bf16(t: torch.Tensor, gen: torch.Generator, scale: float = 1.0,
                      chunk_elems: int = 1 << 27) -> None:
    flat = t.view(-1)
    n = flat.numel()
    for s in range(0, n, chunk_elems):
        e = min(n, s + chunk_elems)
        x = torch.randn(e - s, generator=gen, device=t.device, dtype=torch.float32)
        if scale != 1.0:
            x.mul_(scale)
        flat[s:e].copy_(x.to(torch.bfloat16))


def _nan_bf16(shape, device) -> torch.Tensor:
    return torch.full(shape, BF16_NAN, dtype=torch.int16, device=device).view(torch.bfloat16)


def make_workload(spec: WorkloadSpec, device="cpu", seed: Optional[int] = None,
                  nan_fill: bool = True) -> Workload:
    """Generate the inputs of ``spec`` on ``device`` (seeded)."""
    device = torch.device(device)
    seed = spec.seed if seed is None else seed
    s = spec
    D, Ps, Bk = s.head_dim, s.page_size, s.block_size
    B, Hq, Hkv, g = s.batch, s.num_q_heads, s.num_kv_heads, s.group_size
    if Hq % Hkv:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    lens = resolve_seq_lens(s)
    gen = torch.Generator(device=device).manual_seed(int(seed) * 7919 + 11)
    cpu_gen = torch.Generator(device="cpu").manual_seed(int(seed) * 104729 + 3)

    pages_per_seq = [(L + Ps - 1) // Ps for L in lens]
    max_pages = max(1, max(pages_per_seq))
    total_pages = sum(pages_per_seq) + s.spare_pages
    perm = torch.randperm(total_pages, generator=cpu_gen)
    page_table = torch.zeros(B, max_pages, dtype=torch.int32)
    off = 0
    for b, n in enumerate(pages_per_seq):
        page_table[b, :n] = perm[off: off + n].to(torch.int32)
        off += n
    # unused page-table entries point at a spare (NaN-filled) page: a kernel
    # that reads past a sequence's pages sees NaN.
    spare = perm[off:] if s.spare_pages > 0 else perm[:1]
    for b, n in enumerate(pages_per_seq):
        if n < max_pages:
            page_table[b, n:] = int(spare[0])

    q = torch.empty(B, Hq, D, dtype=torch.bfloat16, device=device)
    _fill_normal_bf16(q, gen)
    k_cache = torch.empty(total_pages, Hkv, Ps, D, dtype=torch.bfloat16, device=device)
    v_cache = torch.empty_like(k_cache)
    _fill_normal_bf16(k_cache, gen)
    _fill_normal_bf16(v_cache, gen)

    pt_dev = page_table.to(device)
    needle_pos = {}
    for b, L in enumerate(lens):
        if nan_fill:
            n = pages_per_seq[b]
            tail = n * Ps - L
            if tail > 0 and n > 0:
                last = int(page_table[b, n - 1])
                k_cache[last, :, Ps - tail:, :] = _nan_bf16((Hkv, tail, D), device)
                v_cache[last, :, Ps - tail:, :] = _nan_bf16((Hkv, tail, D), device)
        if L == 0:
            continue
        qf = q[b].float().view(Hkv, g, D)
        u = qf.sum(dim=1)
        u = u / u.norm(dim=1, keepdim=True).clamp_min(1e-30)  # [Hkv][D]
        for h in range(Hkv):
            special = _special_positions(s, L, cpu_gen)
            needle_pos[(b, h)] = special["needles"]
            hot = special["sinks"] + special["needles"]
            cold = special["outliers"]
            if hot:
                idx = torch.tensor(hot, dtype=torch.int64)
                pg = pt_dev[b, (idx // Ps).to(device)].long()
                slot = (idx % Ps).to(device)
                noise = torch.randn(len(hot), D, generator=gen, device=device)
                kk = s.needle_gain * math.sqrt(D) * u[h][None, :] + noise
                k_cache[pg, h, slot, :] = kk.to(torch.bfloat16)
            if cold:
                idx = torch.tensor(cold, dtype=torch.int64)
                pg = pt_dev[b, (idx // Ps).to(device)].long()
                slot = (idx % Ps).to(device)
                noise = torch.randn(len(cold), D, generator=gen, device=device)
                kk = -math.sqrt(D) * u[h][None, :] + noise
                k_cache[pg, h, slot, :] = kk.to(torch.bfloat16)
                vv = s.outlier_vscale * torch.randn(len(cold), D, generator=gen, device=device)
                v_cache[pg, h, slot, :] = vv.to(torch.bfloat16)
    if nan_fill and s.spare_pages > 0:
        sp = spare.to(device).long()
        k_cache[sp] = _nan_bf16((len(sp), Hkv, Ps, D), device)
        v_cache[sp] = _nan_bf16((len(sp), Hkv, Ps, D), device)

    seq_lens = torch.tensor(lens, dtype=torch.int32)
    wl = Workload(spec=s, q=q, k_cache=k_cache, v_cache=v_cache,
                  page_table=pt_dev, seq_lens=seq_lens.to(device),
                  needle_pos=needle_pos)
    if s.list_fraction is not None:
        bl, bll = importance_block_list(wl, s.list_fraction)
        wl.block_list, wl.block_list_len = bl, bll
    return wl


def _special_positions(s: WorkloadSpec, L: int, gen: torch.Generator) -> dict:
    sinks = list(range(min(s.n_sinks, L)))
    taken = set(sinks)
    needles: list[int] = []
    bands = s.needle_bands or ((s.n_needles, 0.0, 1.0),)
    for count, lo_f, hi_f in bands:
        lo = max(len(sinks), int(lo_f * L))
        hi = max(lo + 1, min(L, int(math.ceil(hi_f * L))))
        tries = 0
        got = 0
        while got < count and tries < 100 * max(1, count):
            p = int(torch.randint(lo, hi, (1,), generator=gen))
            tries += 1
            if p in taken:
                continue
            taken.add(p)
            needles.append(p)
            got += 1
    outliers: list[int] = []
    tries = 0
    while len(outliers) < s.n_outliers and tries < 100 * max(1, s.n_outliers) and L > len(taken):
        p = int(torch.randint(0, L, (1,), generator=gen))
        tries += 1
        if p in taken:
            continue
        taken.add(p)
        outliers.append(p)
    return {"sinks": sinks, "needles": sorted(needles), "outliers": sorted(outliers)}


def importance_block_list(wl: Workload, fraction: float):
    """Per (b, kv head): the top ``fraction`` of blocks by max_j ||k_j||_2,
    always with block 0 and the last block, in descending score order (ties:
    ascending id).  Returns (block_list int32 [B][Hkv][n_max], lens [B][Hkv])."""
    s = wl.spec
    Bk, Ps = s.block_size, s.page_size
    lens = wl.seq_lens.cpu().tolist()
    B, Hkv = s.batch, s.num_kv_heads
    nblks = [(L + Bk - 1) // Bk for L in lens]
    counts = []
    for n in nblks:
        c = int(math.ceil(fraction * n)) if n > 0 else 0
        counts.append(min(n, max(c, min(n, 2))))
    n_max = max(1, max(counts))
    out = torch.full((B, Hkv, n_max), -1, dtype=torch.int32)
    out_len = torch.zeros((B, Hkv), dtype=torch.int32)
    for b, L in enumerate(lens):
        n = nblks[b]
        if n == 0:
            continue
        npg = (L + Ps - 1) // Ps
        pages = wl.page_table[b, :npg].long()
        kk = wl.k_cache[pages].float()               # [npg][Hkv][Ps][D]
        norms = kk.norm(dim=-1)                       # [npg][Hkv][Ps]
        norms = norms.permute(1, 0, 2).reshape(Hkv, npg * Ps)[:, :L]
        pad = n * Bk - L
        if pad:
            norms = torch.cat([norms, torch.full((Hkv, pad), -math.inf,
                                                 device=norms.device)], dim=1)
        score = norms.view(Hkv, n, Bk).amax(dim=2).cpu().double()  # [Hkv][n]
        for h in range(Hkv):
            sc = score[h]
            forced = {0, n - 1}
            rest = [i for i in range(n) if i not in forced]
            rest.sort(key=lambda i: (-float(sc[i]), i))
            chosen = sorted(forced) + rest[: max(0, counts[b] - len(forced))]
            chosen = chosen[: counts[b]]
            chosen.sort(key=lambda i: (-float(sc[i]), i))
            out[b, h, : len(chosen)] = torch.tensor(chosen, dtype=torch.int32)
            out_len[b, h] = len(chosen)
    dev = wl.q.device
    return out.to(dev), out_len.to(dev)


def group_subproblem(wl: Workload, b: int, kvh: int) -> dict:
    """Host copies of exactly what group (b, kvh) reads: its query heads, its
    pages (compacted into a private pool), a page table over them and its
    block list.  Used to check sampled groups of full-size runs."""
    s = wl.spec
    g, Ps = s.group_size, s.page_size
    L = int(wl.seq_lens[b])
    npg = (L + Ps - 1) // Ps
    pages = wl.page_table[b, :npg].long()
    k = wl.k_cache[pages, kvh: kvh + 1].cpu().contiguous()
    v = wl.v_cache[pages, kvh: kvh + 1].cpu().contiguous()
    q = wl.q[b: b + 1, kvh * g: (kvh + 1) * g].cpu().contiguous()
    pt = torch.arange(max(1, npg), dtype=torch.int32).view(1, -1)
    sub = {"q": q, "k_cache": k, "v_cache": v, "page_table": pt,
           "seq_lens": torch.tensor([L], dtype=torch.int32),
           "block_list": None, "block_list_len": None}
    if wl.block_list is not None:
        n = int(wl.block_list_len[b, kvh])
        sub["block_list"] = wl.block_list[b: b + 1, kvh: kvh + 1, :].cpu().contiguous()
        sub["block_list_len"] = torch.tensor([[n]], dtype=torch.int32)
    return sub
