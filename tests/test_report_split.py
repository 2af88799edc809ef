"""Host logic of the report's Sec. V-B split of an iteration (no GPU)."""
import numpy as np

from paper_2101_07968_amd.report import breakdown


def test_breakdown_of_a_hand_timeline():
    ms = 1_000_000
    # per layer: pull start/end, forward start/end, backward start/end, push start/end
    tl = np.array([[0, 10, 10, 15, 30, 40, 40, 50],
                   [10, 20, 20, 25, 25, 30, 30, 38]], dtype=np.int64) * ms
    s = breakdown(tl)
    # forward: link [0, 20], compute [10, 15] + [20, 25]
    assert s["fwd"] == [5.0, 5.0, 15.0]
    # backward: link [30, 38] + [40, 50], compute [25, 40]
    assert s["bwd"] == [7.0, 8.0, 10.0]


def test_breakdown_segments_repeat_per_layer():
    ms = 1_000_000
    # one pull segment covering both layers appears on both rows; it counts once
    tl = np.array([[0, 10, 10, 12, 14, 16, 16, 20],
                   [0, 10, 12, 14, 12, 14, 16, 20]], dtype=np.int64) * ms
    s = breakdown(tl)
    assert s["fwd"] == [4.0, 0.0, 10.0]
    assert s["bwd"] == [4.0, 0.0, 4.0]
