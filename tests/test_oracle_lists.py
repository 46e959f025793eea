"""Pins of the traversal-list oracle (Sec. 3.4; readings L1-L4 of
oracle/art_list_oracle.c) against NumPy brute force, closed forms and
planted mistakes.  CPU only."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import lists as OL
from bruteforce import to_f64
from helpers import small_workload


def _dense_keys(wl, b, kvh):
    """fp64 keys [L][D] of sequence b, KV head kvh, in token order."""
    kc = to_f64(wl.k_cache)
    pt = wl.page_table.cpu().numpy()
    L = int(wl.seq_lens[b])
    Ps = kc.shape[2]
    toks = np.arange(L)
    return kc[pt[b, toks // Ps], kvh, toks % Ps] if L else np.zeros((0, kc.shape[3]))


def _brute_scores(wl, kind):
    s = wl.spec
    q = to_f64(wl.q)
    g = s.group_size
    out = {}
    for b in range(s.batch):
        for h in range(s.num_kv_heads):
            K = _dense_keys(wl, b, h)
            n = -(-K.shape[0] // s.block_size)
            sc = []
            for i in range(n):
                Kb = K[i * s.block_size:(i + 1) * s.block_size]
                if kind == OL.KEY_NORM:
                    sc.append(float((Kb ** 2).sum(axis=1).max()))
                else:
                    qh = q[b, h * g:(h + 1) * g]                      # [g][D]
                    lo, hi = Kb.min(axis=0), Kb.max(axis=0)
                    sc.append(float(np.maximum(qh * lo, qh * hi).sum(axis=1).max()))
            out[(b, h)] = np.array(sc)
    return out


def _brute_select(scores, budget, sinks, keep_last):
    n = len(scores)
    forced = set(range(min(sinks, n)))
    if keep_last and n:
        forced.add(n - 1)
    order = sorted(range(n), key=lambda i: (-scores[i], i))
    others = budget - len(forced)
    chosen = []
    for i in order:
        if i in forced:
            chosen.append(i)
        elif others > 0:
            chosen.append(i)
            others -= 1
    return chosen


def _run(wl, **kw):
    s = wl.spec
    return OL.block_list(wl.q, wl.k_cache, wl.page_table, wl.seq_lens, block_size=s.block_size,
                         num_q_heads=s.num_q_heads, **kw)


CASES = [
    # seed, batch, kv_heads, group, seq_len(s), block, page
    (51, 1, 2, 4, 1000, 64, 16),     # partial tail block
    (52, 2, 2, 2, (700, 2049), 64, 64),
    (53, 1, 1, 8, 3000, 128, 64),
    (54, 2, 2, 4, (0, 640), 64, 32),  # an empty sequence
]


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("kind", [OL.KEY_NORM, OL.QUERY_BOUND])
def test_scores_match_numpy(case, kind):
    seed, B, hkv, g, L, bk, ps = case
    wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, block_size=bk,
                        page_size=ps, needles=2)
    r = _run(wl, score_kind=kind, budget=4)
    ref = _brute_scores(wl, kind)
    for (b, h), sc in ref.items():
        got = r["scores"][b, h, :len(sc)]
        np.testing.assert_allclose(got, sc, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("kind", [OL.KEY_NORM, OL.QUERY_BOUND])
@pytest.mark.parametrize("sel", [(4, 0, False), (5, 1, True), (7, 3, False), (2, 4, True), (10 ** 6, 0, False)])
def test_selection_matches_brute_force(case, kind, sel):
    budget, sinks, keep_last = sel
    seed, B, hkv, g, L, bk, ps = case
    wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, block_size=bk,
                        page_size=ps, needles=2)
    r = _run(wl, score_kind=kind, budget=budget, sink_blocks=sinks, keep_last=keep_last)
    for (b, h), sc in _brute_scores(wl, kind).items():
        want = _brute_select(sc, budget, sinks, keep_last)
        n = int(r["len"][b, h])
        assert r["list"][b, h, :n].tolist() == want
        assert np.all(r["list"][b, h, n:] == -1)


def test_query_bound_is_an_upper_bound_and_tight_for_one_token():
    """For every head, the bound is >= q . k_j for every token of the block,
    and equals the largest q . k_j when the block holds one token."""
    wl = small_workload(55, batch=1, kv_heads=2, group=4, seq_len=900, block_size=64, needles=2)
    q = to_f64(wl.q)
    r = _run(wl, score_kind=OL.QUERY_BOUND, budget=3)
    for h in range(2):
        K = _dense_keys(wl, 0, h)
        for i in range(-(-K.shape[0] // 64)):
            dots = q[0, 4 * h:4 * h + 4] @ K[i * 64:(i + 1) * 64].T
            assert r["scores"][0, h, i] >= dots.max() - 1e-9
    one = small_workload(56, batch=1, kv_heads=1, group=4, seq_len=1, block_size=64, needles=0)
    r1 = _run(one, score_kind=OL.QUERY_BOUND, budget=1)
    k0 = _dense_keys(one, 0, 0)[0]
    assert r1["scores"][0, 0, 0] == pytest.approx(float((to_f64(one.q)[0] @ k0).max()), rel=1e-12)


def _ramp_keys(n_blocks, block=64, D=128, rising=True):
    """Keys c_i * e_0 in block i: the block scores rise (or fall) with the id."""
    k = torch.zeros((n_blocks, 1, block, D), dtype=torch.float32)
    for i in range(n_blocks):
        k[i, 0, :, 0] = float(i + 1 if rising else n_blocks - i)
    q = torch.ones((1, 1, D), dtype=torch.float32)
    pt = torch.arange(n_blocks, dtype=torch.int32).view(1, n_blocks)
    sl = torch.tensor([n_blocks * block], dtype=torch.int32)
    return q.to(torch.bfloat16), k.to(torch.bfloat16), pt, sl


@pytest.mark.parametrize("kind", [OL.KEY_NORM, OL.QUERY_BOUND])
def test_closed_form_ramp(kind):
    """Block scores rising with the id: the top k blocks are the last k,
    newest first; forced block 0 comes last (smallest score), the forced
    last block is among the top anyway."""
    q, k, pt, sl = _ramp_keys(10)
    r = OL.block_list(q, k, pt, sl, block_size=64, num_q_heads=1, score_kind=kind, budget=4)
    assert r["list"][0, 0, :4].tolist() == [9, 8, 7, 6] and r["len"][0, 0] == 4
    r = OL.block_list(q, k, pt, sl, block_size=64, num_q_heads=1, score_kind=kind, budget=4,
                      sink_blocks=1, keep_last=True)
    assert r["list"][0, 0, :4].tolist() == [9, 8, 7, 0]
    if kind == OL.KEY_NORM:
        np.testing.assert_array_equal(r["scores"][0, 0, :10], [(i + 1.0) ** 2 for i in range(10)])
    q, k, pt, sl = _ramp_keys(10, rising=False)
    r = OL.block_list(q, k, pt, sl, block_size=64, num_q_heads=1, score_kind=kind, budget=3,
                      keep_last=True)
    assert r["list"][0, 0, :3].tolist() == [0, 1, 9]


def test_equal_scores_prefer_smaller_ids():
    q, k, pt, sl = _ramp_keys(8)
    k = torch.zeros_like(k)
    k[..., 0] = 1.0
    r = OL.block_list(q, k, pt, sl, block_size=64, num_q_heads=1, budget=3, keep_last=True)
    assert r["list"][0, 0, :3].tolist() == [0, 1, 7]


@pytest.mark.parametrize("n,sinks,budget,want", [
    (10, 2, 3, [0, 1, 9, 8, 7]),
    (4, 2, 5, [0, 1, 3, 2]),
    (3, 5, 2, [0, 1, 2]),
    (6, 0, 2, [5, 4]),
    (1, 0, 0, []),
    (0, 2, 2, []),
])
def test_streaming_lists(n, sinks, budget, want):
    q, k, pt, sl = _ramp_keys(max(n, 1))
    sl = torch.tensor([n * 64], dtype=torch.int32)
    r = OL.block_list(None, k, pt, sl, block_size=64, num_q_heads=1, policy=OL.STREAMING,
                      budget=budget, sink_blocks=sinks)
    assert r["list"][0, 0, :r["len"][0, 0]].tolist() == want


def test_rejects_bad_options():
    q, k, pt, sl = _ramp_keys(4)
    for kw in (dict(budget=-1), dict(policy=3, budget=1), dict(score_kind=5, budget=1),
               dict(budget=1, sink_blocks=-2)):
        with pytest.raises(ValueError):
            OL.block_list(q, k, pt, sl, block_size=64, num_q_heads=1, **kw)
    with pytest.raises(ValueError):   # a list longer than its row stride
        OL.block_list(q, k, pt, sl, block_size=64, num_q_heads=1, budget=4, max_list=3)
    with pytest.raises(ValueError):   # the query bound needs q
        OL.block_list(None, k, pt, sl, block_size=64, num_q_heads=1, score_kind=OL.QUERY_BOUND,
                      budget=1)


LIST_MUTANTS = {
    "tie_prefers_larger_id": ("return (x->id > y->id) - (x->id < y->id);",
                              "return (x->id < y->id) - (x->id > y->id);"),
    "keep_last_ignored": ("if (O->keep_last && n > 0 && !forced[n - 1])",
                          "if (0 && O->keep_last && n > 0 && !forced[n - 1])"),
    "bound_uses_min_only": ("s += a > c ? a : c;", "s += a;"),
    "tail_off_by_one": ("const int j0 = blk * Bk, j1 = (j0 + Bk < L) ? j0 + Bk : L;",
                        "const int j0 = blk * Bk, j1 = (j0 + Bk < L) ? j0 + Bk : L - 1;"),
    "streaming_oldest_first": ("for (int i = n - 1, taken = 0; i >= ns && taken < O->budget; --i, ++taken) {",
                               "for (int i = ns, taken = 0; i < n && taken < O->budget; ++i, ++taken) {"),
    "norm_not_squared": ("for (int d = 0; d < D; ++d) s += bf16(k[d]) * bf16(k[d]);",
                         "for (int d = 0; d < D; ++d) s += bf16(k[d]);"),
}


def _list_battery(lib) -> list[str]:
    fails = []
    for case in CASES[:2]:
        seed, B, hkv, g, L, bk, ps = case
        wl = small_workload(seed, batch=B, kv_heads=hkv, group=g, seq_len=L, block_size=bk,
                            page_size=ps, needles=2)
        for kind in (OL.KEY_NORM, OL.QUERY_BOUND):
            s = wl.spec
            r = OL.block_list(wl.q, wl.k_cache, wl.page_table, wl.seq_lens, block_size=bk,
                              num_q_heads=s.num_q_heads, score_kind=kind, budget=5, sink_blocks=1,
                              keep_last=True, _lib=lib)
            for (b, h), sc in _brute_scores(wl, kind).items():
                if not np.allclose(r["scores"][b, h, :len(sc)], sc, rtol=1e-12, atol=1e-12):
                    fails.append("scores")
                if r["list"][b, h, :r["len"][b, h]].tolist() != _brute_select(sc, 5, 1, True):
                    fails.append("select")
    q, k, pt, sl = _ramp_keys(8)
    k = torch.zeros_like(k)
    k[..., 0] = 1.0
    r = OL.block_list(q, k, pt, sl, block_size=64, num_q_heads=1, budget=3, _lib=lib)
    if r["list"][0, 0, :3].tolist() != [0, 1, 2]:
        fails.append("ties")
    q, k, pt, sl = _ramp_keys(10)
    r = OL.block_list(None, k, pt, sl, block_size=64, num_q_heads=1, policy=OL.STREAMING,
                      budget=3, sink_blocks=2, _lib=lib)
    if r["list"][0, 0, :5].tolist() != [0, 1, 9, 8, 7]:
        fails.append("streaming")
    return sorted(set(fails))


def test_list_battery_passes_on_the_real_oracle():
    assert _list_battery(None) == []


@pytest.mark.parametrize("name", sorted(LIST_MUTANTS))
def test_planted_list_mistake_is_caught(name, tmp_path):
    old, new = LIST_MUTANTS[name]
    src = OL.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    lib = OL.load_library(OL.build_variant(src.replace(old, new), str(tmp_path / f"{name}.so")))
    assert _list_battery(lib), f"planted mistake '{name}' passed every list pin"
