"""The anchor-set acceptance rule used by the GPU tests (host logic)."""

import numpy as np
import pytest

from tests.oracle_side import anchors_agree, assert_overlap


def test_near_tie_swap_is_accepted():
    s = np.linspace(2.0, 1.0, 100)
    k = 60
    s[k] = s[k - 1] * (1 - 1e-5)          # K-th and (K+1)-th nearly tied
    ref = np.argsort(-s, kind="stable")[:k]
    got = np.concatenate([ref[:-1], [k]])  # the near-tied neighbour instead of the K-th
    ov = anchors_agree(got, ref, s, k, 2e-2)
    assert ov == pytest.approx(59 / 60)
    assert_overlap(ov, s, k, 2e-2)


def test_swap_at_a_clear_boundary_is_rejected():
    s = np.linspace(2.0, 1.0, 100)
    k = 60
    s[k:] -= 0.5                           # clear gap below the K-th score
    ref = np.argsort(-s, kind="stable")[:k]
    with pytest.raises(AssertionError):
        assert_overlap(59 / 60, s, k, 2e-2)
    got = np.concatenate([ref[:-1], [k]])
    with pytest.raises(AssertionError):   # the swapped-in anchor is outside the tie band
        anchors_agree(got, ref, s, k, 2e-2)
