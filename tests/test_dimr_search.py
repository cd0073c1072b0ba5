"""Host logic of the routing-mask search (Eq. 13), with synthetic costs.

The search must only propose masks of the right size that keep the fixed
layers, never evaluate a mask twice, report the minimum it evaluated, be
reproducible from its seed, and find a planted optimum of a cost whose
structure a surrogate can learn (distance to a hidden mask).
"""
import pytest

from paper_2606_12243_amd.dimr import MaskSearch


def hamming_cost(target):
    t = set(target)
    return lambda m: float(len(t.symmetric_difference(m)))


def test_search_invariants_and_reproducibility():
    target = (0, 1, 5, 9, 12, 15)
    runs = []
    for _ in range(2):
        s = MaskSearch(16, 6, hamming_cost(target), seed=3, theta=3, max_steps=40, patience=40, fixed=(0, 15))
        best, c = s.run()
        runs.append((best, c, [h[0] for h in s.history]))
        masks = [h[0] for h in s.history]
        assert len(masks) == len(set(masks)), "no mask is evaluated twice"
        assert all(len(m) == 6 and 0 in m and 15 in m and list(m) == sorted(m) for m in masks)
        assert c == min(h[1] for h in s.history) and best in masks
        assert any(h[2] == "bayes" for h in s.history) and any(h[2] == "random" for h in s.history)
    assert runs[0] == runs[1], "the search is reproducible from its seed"


def test_bayesian_steps_find_a_planted_optimum():
    target = (0, 2, 3, 7, 8, 11, 13, 15)
    s = MaskSearch(16, 8, hamming_cost(target), seed=1, theta=2, max_steps=60, patience=60)
    best, c = s.run()
    assert best == target and c == 0.0


def test_patience_stops_the_search():
    s = MaskSearch(12, 4, lambda m: 1.0, seed=0, theta=4, max_steps=50, patience=5)
    s.run()
    assert len(s.history) == 6  # the first evaluation, then five without improvement


def test_small_space_is_exhausted_cleanly():
    s = MaskSearch(4, 3, lambda m: float(sum(m)), seed=0, theta=2, max_steps=50, patience=50)
    best, c = s.run()
    assert len(s.history) == 4 and best == (0, 1, 2) and c == 3.0


def test_rejects_bad_sizes():
    with pytest.raises(ValueError):
        MaskSearch(4, 0, lambda m: 0.0)
    with pytest.raises(ValueError):
        MaskSearch(4, 2, lambda m: 0.0, fixed=(0, 1, 2))
