"""Host aggregations of the load metrics (closed forms on constructed records)."""
import numpy as np

from paper_2609_39137_amd.metrics import LoadRecord, bias_drift


def test_summary_means_and_worst():
    rec = LoadRecord()
    for t in range(2000):
        # two layers: MaxVio 1 + t/1000 and 3; MinVio 0.5 and 0.25
        rec.add(np.array([[1.0 + t / 1000.0, 0.5], [3.0, 0.25]]))
    s = rec.summary(last=1000)
    assert s["steps"] == 2000 and s["layers"] == 2
    # layer mean of MaxVio at step t: (4 + t/1000) / 2; last 1000 steps t = 1000..1999
    assert abs(s["maxvio_last"] - np.mean([(4 + t / 1000.0) / 2 for t in range(1000, 2000)])) < 1e-12
    assert abs(s["maxvio_avg"] - np.mean([(4 + t / 1000.0) / 2 for t in range(2000)])) < 1e-12
    assert s["maxvio_worst"] == 3.0
    assert s["minvio_last"] == 0.375 and s["minvio_avg"] == 0.375


def test_cumulative_excess_counts_only_the_part_above_threshold():
    rec = LoadRecord()
    for v in (0.5, 1.5, 2.0, 0.9, 1.25):
        rec.add(np.array([v, 0.0]))
    assert rec.cumulative_excess(1.0) == 0.5 + 1.0 + 0.25
    assert rec.cumulative_excess(1.0, start=3) == 0.25


def test_bias_drift():
    a = np.array([[0.0, 1.0], [2.0, -2.0]], np.float32)
    b = np.array([[0.5, 1.0], [1.0, -1.0]], np.float32)
    assert bias_drift(a, b) == (0.5 + 0.0 + 1.0 + 1.0) / 4
