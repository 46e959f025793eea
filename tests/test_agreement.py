"""Host logic of the probe-agreement harness (Appendix B's categories)."""
from __future__ import annotations

import pytest

from paper_2606_00024_amd.agreement import Agreement, classify, length_sweep_specs, markdown


def test_categories():
    # (probe, full, T)
    cases = [
        (5, 5, 10),    # same block: agree
        (10, 10, 10),  # neither stops: agree
        (4, 7, 10),    # probe earlier: FP, both stop -> delta 3
        (6, 10, 10),   # probe stops, full never: FP
        (9, 6, 10),    # full earlier: FN, delta 3
        (12, 7, 12),   # full stops, probe never: FN
        (3, 3, 3),     # stop at the last block = no stop: agree
    ]
    a = classify([c[0] for c in cases], [c[1] for c in cases], [c[2] for c in cases])
    assert (a.groups, a.agree, a.fp, a.fn) == (7, 3, 2, 2)
    assert sorted(a.both_stop_differ) == [3, 3]
    r = a.rates()
    assert r["agree_pct"] == pytest.approx(300 / 7)
    assert r["delta_blk_mean"] == 3 and r["delta_blk_std"] == 0
    assert a.total_blocks == 10 * 5 + 12 + 3
    assert a.probe_blocks == 5 + 10 + 4 + 6 + 9 + 12 + 3


def test_empty_traversals_are_left_out_and_bad_stops_rejected():
    a = classify([0, 2], [0, 2], [0, 4])
    assert a.groups == 1 and a.agree == 1
    with pytest.raises(ValueError):
        classify([0], [1], [4])
    with pytest.raises(ValueError):
        classify([5], [1], [4])
    with pytest.raises(ValueError):
        classify([1, 2], [1], [4, 4])


def test_accumulates_and_formats():
    a = Agreement()
    classify([1, 2], [1, 3], [4, 4], into=a)
    classify([4], [2], [4], into=a)
    assert (a.groups, a.agree, a.fp, a.fn) == (3, 1, 1, 1)
    row = {"workload": "w", "probe_stride": 4, "probe_dims": 32, "tau": 1e-3, "phi": 1e-4,
           "patience": 5}
    row.update(a.rates())
    text = markdown([row])
    assert "| w | 32 |" in text


def test_length_sweep_places_needles_mid_context():
    specs = length_sweep_specs(lengths=(1024, 4096))
    assert [s.seq_lens[0] for s in specs] == [1024, 4096]
    assert all(s.needle_bands == ((8, 0.45, 0.55),) for s in specs)
