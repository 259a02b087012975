"""Frames with k rho != d (Sec. 3.2 construction; the appendix's (6, 3, 11) example is one, redundant
and with T(x) blocks between its rows): the oracle's frame P equals L^T Pv, where Pv is the oracle's
block frame of dimension k rho and L places row r of the Spectral Tetris frame F at the positions
r k + (j mod k) with weights F[r][j].  The library applies every such frame in this factored form,
so this pins that reading with the oracle's own constructions; L is built here from F alone."""
import numpy as np
import pytest

from oracle import frameft_oracle as O


def lift_matrix(k, rho, d):
    """Real (k rho) x d lift of the Spectral Tetris rows, or None when two entries of one row agree
    mod k (the rows' windows do not fit in k positions)."""
    F = O.spectral_tetris(rho // 2, d // 2)
    L = np.zeros((k * rho, d))
    for r in range(F.shape[0]):
        for j in np.nonzero(F[r])[0]:
            v = r * k + j % k
            if L[2 * v].any():
                return None
            L[2 * v, 2 * j] = L[2 * v + 1, 2 * j + 1] = F[r, j]
    return L


# the appendix's example (complex (6, 3, 11)); a redundant frame with an integer ratio; frames of
# Llama width with d / rho = 42.67 and 85.33; the block-diagonal case k rho = d (L = I)
CASES = [(6, 6, 22), (8, 4, 16), (12, 6, 22), (48, 96, 4096), (88, 48, 4096), (64, 64, 4096)]


@pytest.mark.parametrize("k,rho,d", CASES)
def test_frame_is_lifted_block_frame(k, rho, d):
    P = O.tight_fusion_frame(k, rho, d)
    Pv = O.tight_fusion_frame(k, rho, k * rho)
    L = lift_matrix(k, rho, d)
    assert L is not None
    if d == k * rho:
        np.testing.assert_array_equal(L, np.eye(d))
    diff = abs(P - (Pv.T @ L).T)
    assert diff.max() <= 1e-15
    # each user coordinate lies in one or two rows of F
    per_col = np.count_nonzero(L, axis=0)
    assert per_col.min() >= 1 and per_col.max() <= 2


@pytest.mark.parametrize("k,rho,d", [(5, 6, 22), (4, 6, 22), (40, 96, 4096)])
def test_window_wider_than_k_is_not_tight(k, rho, d):
    """When a row of F does not fit in k positions the lift collides, and the frame is not tight."""
    assert lift_matrix(k, rho, d) is None
    with pytest.raises(O.NotATightFusionFrame):
        O.tight_fusion_frame(k, rho, d)
