"""CPU check of the wavefront-timeline statistics on a synthetic table with known readings."""

import numpy as np

from paper_2510_13223_amd import timeline


def test_summarize_known_table():
    n = 8
    t = np.full((n + 4, 4), timeline.UNSET, dtype=np.uint64)  # 4 unused slots at the end
    base = 1_000_000
    for i in range(n):  # entry at 100 ns steps; ready 1 us later; first block 2 us + i us later; exit 10 us + i us
        e = base + 10 * i
        t[i] = (e, e + 100, e + 200 + 100 * i, base + 1000 + 100 * i)
    t[3, 2] = timeline.UNSET  # a wavefront with no block: no first-block reading
    s = timeline.summarize(t)
    assert s["waves"] == n
    assert abs(s["entry_spread_us"] - 0.7) < 1e-9
    assert abs(s["span_us"] - (1000 + 700) * timeline.TICK_US) < 1e-9
    assert abs(s["ready_after_entry_p50_us"] - 1.0) < 1e-9
    first = np.array([2.0 + i for i in range(n) if i != 3])
    assert abs(s["first_block_after_entry_p50_us"] - np.percentile(first, 50)) < 1e-9
    exits = np.array([10.0 + i for i in range(n)])
    assert abs(s["exit_p90_us"] - np.percentile(exits, 90)) < 1e-9
    # quarters in slot order: two slots each
    assert abs(s["q0_exit_p50_us"] - 10.5) < 1e-9 and abs(s["q3_exit_p50_us"] - 16.5) < 1e-9
    assert abs(s["q1_first_block_p50_us"] - 4.0) < 1e-9  # slot 2 only (slot 3 has no reading)


def test_summarize_without_exits_or_entries():
    import pytest

    t = np.full((4, 4), timeline.UNSET, dtype=np.uint64)
    with pytest.raises(ValueError):
        timeline.summarize(t)
    t[0] = (100, 110, timeline.UNSET, timeline.UNSET)  # entered and scheduled, never finished
    s = timeline.summarize(t)
    assert s["waves"] == 1 and np.isnan(s["span_us"]) and np.isnan(s["exit_p50_us"])
