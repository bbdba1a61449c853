"""Host checks of the assumption diagnostics (paper_2605_31598_amd/diagnostics.py) on
hand-made score vectors whose answers follow from the definitions."""
import numpy as np
import pytest

from paper_2605_31598_amd import diagnostics as dg


def test_concentration_counts_historical_mass_only():
    s = np.array([5.0, 3.0, 1.0, 7.0])  # position 3 is the current frame: excluded
    p = np.array([0, 1, 2, 3])
    assert dg.concentration(s, p, 3, 1) == pytest.approx(5 / 9)
    assert dg.concentration(s, p, 3, 2) == pytest.approx(8 / 9)
    assert dg.concentration(s, p, 3, 3) == pytest.approx(1.0)
    assert dg.concentration(s, p, 3, 10) == pytest.approx(1.0)


def test_top_b_ties_go_to_the_lower_position():
    s = np.array([2.0, 2.0, 2.0, 1.0])
    p = np.array([7, 3, 5, 1])
    assert dg.top_b(s, p, 2) == {3, 5}


def test_evolution_recall_retention_churn():
    prev_s = np.array([9.0, 8.0, 1.0, 1.0])  # positions 0..3 seen up to frame n; S_n (B=2) = {0, 1}
    prev_p = np.arange(4)
    s = np.array([9.0, 0.5, 4.0, 0.1, 6.0, 0.2])  # frame n+1 = positions 4, 5; S_{n+1} = {0, 4}
    p = np.arange(6)
    e = dg.evolution(prev_s, prev_p, s, p, np.array([4, 5]), 2)
    assert e == pytest.approx({"recall": 1.0, "weighted_recall": 1.0, "retention": 0.5, "churn": 0.5})
    # with B = 3: S_n = {0, 1, 2}, S_{n+1} = {0, 4, 2}; pool = {0, 1, 2, 4, 5} holds all of it
    e3 = dg.evolution(prev_s, prev_p, s, p, np.array([4, 5]), 3)
    assert e3["recall"] == 1.0 and e3["retention"] == pytest.approx(2 / 3)
    # a key outside both the previous state and the frame lowers recall, weighted by its mass
    s2 = np.array([9.0, 0.5, 0.4, 5.0, 6.0, 0.2])  # S_{n+1} (B=2) = {0, 4}; B=3 adds position 3
    e4 = dg.evolution(prev_s, prev_p, s2, p, np.array([4, 5]), 3)
    assert e4["recall"] == pytest.approx(2 / 3)
    assert e4["weighted_recall"] == pytest.approx(15 / 20)
    assert e4["churn"] == pytest.approx(2 / 3)


def test_summarise_averages_over_frames():
    frames = [(np.array([1.0, 1.0]), np.array([0, 1]), 0),
              (np.array([3.0, 1.0, 5.0]), np.array([0, 1, 2]), 2),
              (np.array([3.0, 1.0, 2.0, 9.0]), np.array([0, 1, 2, 3]), 3)]
    out = dg.summarise(frames, [1])
    assert out[1]["concentration"] == pytest.approx(np.mean([3 / 4, 3 / 6]))
