"""The ablation harness (Table 3's settings): host logic on the CPU, and on
the GPU the exact relations between the settings' stopping blocks."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

from paper_2606_00024_amd.ablation import deviation, markdown, settings


def test_settings_remove_one_part_each():
    s = settings(1e-3, 1e-4, 5)
    assert [x[0] for x in s] == ["full", "w/o d_scale", "w/o d_direction", "w/o patience"]
    assert s[1][1] == math.inf and s[1][2:] == (1e-4, 5)
    assert s[2][2] == math.inf and (s[2][1], s[2][3]) == (1e-3, 5)
    assert s[3][3] == 1 and s[3][1:3] == (1e-3, 1e-4)


def test_deviation_per_head():
    ref = np.zeros((1, 2, 4))
    ref[0, 0, 0] = 1.0
    ref[0, 1, 1] = 2.0
    out = ref.copy()
    out[0, 1, 1] = 2.2           # 10 % off on head 1
    d = deviation(out, ref)
    assert d["rel_l2_max"] == pytest.approx(0.1)
    assert d["rel_l2_mean"] == pytest.approx(0.05)
    assert d["heads_over_1pct"] == 0.5


def test_markdown_row():
    row = {"workload": "w", "setting": "full", "tau": 1e-3, "phi": 1e-4, "patience": 5, "ms": 0.1,
           "delta_time_pct": 0.0, "skipped_pct": 50.0, "rel_l2_mean": 1e-3, "rel_l2_p99": 2e-3,
           "rel_l2_max": 3e-3, "heads_over_1pct": 0.0}
    assert "| w | dense | full |" in markdown([row])


@pytest.mark.gpu
def test_ablations_only_ever_stop_earlier():
    """Dropping a condition (tau or phi to +inf) or the patience (p = 1) can
    only make steps stable sooner: every group stops at or before the full
    rule's block, and the full rule's output distance is what the oracle-
    checked kernel gives (a sanity bound here)."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import sys
    from helpers import small_workload
    from paper_2606_00024_amd.ablation import measure
    wl = small_workload(71, batch=2, kv_heads=2, group=4, seq_len=(6000, 4000), needles=2)
    for n in ("q", "k_cache", "v_cache", "page_table", "seq_lens"):
        setattr(wl, n, getattr(wl, n).to("cuda:0"))
    print("  gpu call: ablation settings on a small workload", flush=True)
    rows = measure(wl, (0.05, 1e-3, 3), steps=2, warmup=1)
    full = rows[0]["stop"]
    for r in rows[1:]:
        assert (r["stop"] <= full).all(), r["setting"]
        assert r["skipped_pct"] >= rows[0]["skipped_pct"]
    assert all(np.isfinite(r["rel_l2_max"]) for r in rows)
