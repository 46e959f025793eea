"""Host logic of the measurement sweeps: the least-squares fit and the
bytes each stop reads."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from helpers import small_workload
from paper_2606_00024_amd.sweep import fit_line, kv_bytes_read


def test_fit_recovers_a_line():
    x = np.array([1e8, 3e8, 5e8, 1e9])
    y = 2e-5 + x / 5e12
    f = fit_line(x, y)
    assert f["a"] == pytest.approx(2e-5) and f["b"] == pytest.approx(1 / 5e12)
    assert f["r2"] == pytest.approx(1.0)
    f = fit_line(x, y + np.array([1e-6, -1e-6, 1e-6, -1e-6]))
    assert 0.99 < f["r2"] < 1.0


def test_bytes_read_follow_the_traversal():
    # 1000 tokens, blocks of 64: 16 blocks, the newest holds 40 tokens
    wl = small_workload(101, batch=1, kv_heads=2, group=4, seq_len=1000)
    stop = np.array([[1, 3]])
    # recency-first: group 0 reads the 40-token tail; group 1 also 2 full blocks
    assert kv_bytes_read(wl, stop) == (40 + 40 + 128) * 128 * 4
    wl.block_list = torch.tensor([[[0, 5, 15], [15, 2, 1]]], dtype=torch.int32)
    wl.block_list_len = torch.tensor([[3, 3]], dtype=torch.int32)
    assert kv_bytes_read(wl, np.array([[3, 1]])) == (64 + 64 + 40 + 40) * 128 * 4
