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


def test_link_rates_count_each_segment_once():
    from paper_2101_07968_amd.report import link_rates
    # two layers in one pull segment (0..10 us), one push segment per layer
    tl = np.array([[0, 10_000, 0, 0, 0, 0, 30_000, 32_000],
                   [0, 10_000, 0, 0, 0, 0, 20_000, 30_000]], dtype=np.int64)
    pull, push = link_rates(tl, [1000, 3000], dt_ns=2_000)
    assert pull == 4000 / 8_000 * 1e9
    # 1000 B in 2 us - 2 us overhead -> clamped to 1 ns; 3000 B in 10 - 2 us
    assert push == 4000 / (1 + 8_000) * 1e9
