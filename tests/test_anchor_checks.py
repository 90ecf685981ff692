"""The anchor-set acceptance rule used by the GPU tests (host logic)."""

import numpy as np
import pytest

from oracle import acache_oracle as O
from tests.oracle_side import check_anchors


def _scores(n=300, seed=0):
    return np.random.default_rng(seed).permutation(np.linspace(2.0, 1.0, n))


def test_swap_inside_the_band_is_accepted_for_small_k():
    s = _scores(100)
    k = 60
    order = np.argsort(-s, kind="stable")
    s[order[k]] = s[order[k - 1]] - 1e-7      # K-th and (K+1)-th nearly tied
    g = s.copy()
    g[order[k]], g[order[k - 1]] = s[order[k - 1]], s[order[k]]  # rounding swaps them
    got = O.topk_anchors(g, k)
    ov = check_anchors(got, s, k, score_err=np.max(np.abs(g - s)))
    assert ov == pytest.approx(59 / 60)


def test_swap_outside_the_band_is_rejected():
    s = _scores(100)
    k = 60
    order = np.argsort(-s, kind="stable")
    got = np.concatenate([order[:k - 1], [order[k + 5]]])   # a clearly lower score swapped in
    with pytest.raises(AssertionError):
        check_anchors(got, s, k, score_err=1e-6)


def test_large_k_needs_99_percent_even_inside_the_band():
    s = _scores(300)
    k = 150
    order = np.argsort(-s, kind="stable")
    got = np.concatenate([order[:k - 2], order[k:k + 2]])    # two swaps of 150: 98.7%
    err = 1.0                                                # a band wide enough for any swap
    with pytest.raises(AssertionError):
        check_anchors(got, s, k, score_err=err)
    got1 = np.concatenate([order[:k - 1], order[k:k + 1]])   # one swap: 99.3%
    assert check_anchors(got1, s, k, score_err=err) == pytest.approx(149 / 150)


def test_exact_scores_need_identical_sets():
    s = _scores(200)
    k = 40
    assert check_anchors(O.topk_anchors(s, k), s, k, score_err=0.0) == 1.0
    order = np.argsort(-s, kind="stable")
    got = np.concatenate([order[:k - 1], [order[k]]])
    with pytest.raises(AssertionError):
        check_anchors(got, s, k, score_err=0.0)
