"""Host logic of bench.py's work-group timeline summaries, on synthetic records (no GPU)."""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _records(starts, ends, types, xcds, cus):
    n = len(starts)
    r = np.zeros((n, 4), dtype=np.uint64)
    r[:, 0] = np.asarray(starts, dtype=np.uint64) + np.uint64(10 ** 9)
    r[:, 1] = np.asarray(ends, dtype=np.uint64) + np.uint64(10 ** 9)
    r[:, 2] = (np.asarray(xcds, dtype=np.uint64) << np.uint64(32)) | (
        np.asarray(cus, dtype=np.uint64) << np.uint64(8))
    r[:, 3] = (np.uint64(n) << np.uint64(8)) | np.asarray(types, dtype=np.uint64)
    return r


def test_timeline_summary_types_span_and_refill():
    # ticks of 10 ns: C 0-1000 and 0-800, A 100-600, B 800-1100 (refills the CU of the C that
    # ended at 800, 0 us later) and 900-1200 on XCD 1
    r = _records([0, 0, 100, 800, 900], [1000, 800, 600, 1100, 1200], [0, 0, 1, 2, 2],
                 [0, 0, 0, 0, 1], [3, 3, 3, 3, 5])
    total = {0: 2000, 1: 1000, 2: 3000}
    lines = bench.timeline_summary([r], total, ["head"])
    text = "\n".join(lines)
    assert lines[0] == "head"
    assert "median over calls: 12.00 us" in text
    row_c = next(ln for ln in lines if ln.split()[:1] == ["C"])
    f = row_c.split()
    assert f[1] == "2" and f[3] == "9.00"          # 2 work-groups, mean (10 + 8) / 2 us
    row_b = next(ln for ln in lines if ln.split()[:1] == ["B"])
    assert row_b.split()[8] == "12.00"             # last end of B
    # one refill on (XCD 0, CU 3): B started at 8 us, the C there ended at 8 us; A at 1 us had
    # no earlier end
    assert "1 work-groups, median 0.00 us" in text
    assert "XCD1:     1     9.00" in text


def test_tail_summary_offsets_from_stream_end():
    r = _records([0, 50], [1000, 900], [0, 2], [0, 1], [0, 0])
    p = _records([1150, 1170], [1550, 1600], [3, 3], [0, 1], [0, 0])
    d = np.array([1700 + 10 ** 9, 1930 + 10 ** 9, 0, 4], dtype=np.uint64)
    lines = bench.tail_summary([r], [(p, d)])
    text = "\n".join(lines)
    assert "first start 1.50, last start 1.70, last end 6.00" in text
    assert "XCD0 1.50  XCD1 1.70" in text
    assert "decision: start 7.00, end 9.30 (duration 2.30)" in text
    assert "decision end 19.30" in text


def test_tail_summary_skips_stale_records():
    r = _records([0], [1000], [0], [0], [0])
    p = _records([-500 + 10 ** 6], [-100 + 10 ** 6], [3], [0], [0])
    p[:, 0] -= np.uint64(10 ** 6)
    p[:, 1] -= np.uint64(10 ** 6)
    d = np.array([10, 20, 0, 4], dtype=np.uint64)
    assert bench.tail_summary([r], [(p, d)]) == []
