"""The parity helpers themselves (CPU): the near-tie top-k rule accepts every
valid answer and rejects wrong ones."""
import numpy as np
import pytest

from gpu_util import topk_agreement


def test_topk_agreement_accepts_exact_and_boundary_ties():
    row = np.array([5.0, 1.0, 3.0, 3.0 + 1e-9, 0.5, 2.0])
    tau = np.full(row.shape, 1e-6)
    assert topk_agreement(np.array([0, 3, 2]), row, tau, 3) == (1, 0)    # ranks 1, 2 tie: only rank 0 checked
    assert topk_agreement(np.array([0, 2, 3]), row, tau, 3) == (1, 0)    # the tie in either order
    # a boundary tie: index 2 or 3 may take the last slot
    assert topk_agreement(np.array([0, 2]), row, tau, 2)[1] == 1
    assert topk_agreement(np.array([0, 3]), row, tau, 2)[1] == 0


def test_topk_agreement_rejects_wrong_answers():
    row = np.array([5.0, 1.0, 3.0, 4.0, 0.5, 2.0])
    tau = np.full(row.shape, 1e-6)
    assert topk_agreement(np.array([0, 3, 2]), row, tau, 3) == (3, 0)
    with pytest.raises(AssertionError):
        topk_agreement(np.array([0, 2, 3]), row, tau, 3)      # ranks swapped
    with pytest.raises(AssertionError):
        topk_agreement(np.array([0, 3, 5]), row, tau, 3)      # a member that is no near-tie
