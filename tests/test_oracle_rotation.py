"""Pins of the oracle's activation rotation (reading R17): the Walsh matrix
against scipy's Hadamard construction, orthogonality, hand-computed small
cases, blockwise structure, and the inverse."""
import numpy as np
import pytest
from scipy.linalg import hadamard

from oracle import rotation as R
from paper_2609_02652_amd import synth


@pytest.mark.parametrize("n", [1, 2, 4, 8, 16, 64, 256, 1024, 4096])
def test_walsh_matrix_is_sylvester_hadamard(n):
    assert np.array_equal(R.walsh_matrix(n), hadamard(n).astype(np.float64))


def test_walsh_rows_orthogonal():
    H = R.walsh_matrix(128)
    assert np.array_equal(H @ H.T, 128 * np.eye(128))


def test_block_length():
    assert [R.pow2_block(K) for K in (4096, 14336, 5120, 17408, 24, 7)] == \
        [4096, 2048, 1024, 1024, 8, 1]


def test_four_point_by_hand():
    # H4 (Sylvester) rows: ++++, +-+-, ++--, +--+ ; scaled by 1/2
    assert np.array_equal(R.rotate64([1, 2, 3, 4], [1, 1, 1, 1]), [5, -1, -2, 0])
    # a sign flip on coordinate 1 negates column 1 of H4
    assert np.array_equal(R.rotate64([1, 2, 3, 4], [1, -1, 1, 1]), [3, 1, -4, 2])


def test_blockwise_structure():
    """K = 12 = 4·3: three independent 4-point transforms."""
    x = np.arange(1, 13, dtype=np.float64)
    s = np.ones(12)
    out = R.rotate64(x, s)
    for b in range(3):
        assert np.array_equal(out[4 * b:4 * b + 4], R.rotate64(x[4 * b:4 * b + 4], s[:4]))


def test_orthogonal_and_inverse():
    K = 5120
    x = synth.make_activation(K, seed=3, name="rot").astype(np.float64)[:K]
    s = synth.make_signs(K, seed=3, name="rot")
    y = R.rotate64(x, s)
    assert abs(np.linalg.norm(y) - np.linalg.norm(x)) <= 1e-12 * np.linalg.norm(x)
    # inverse: x = diag(s) · H^T y / sqrt(n), blockwise
    n = R.pow2_block(K)
    H = R.walsh_matrix(n)
    back = (y.reshape(-1, n) @ H / np.sqrt(n)).reshape(K) * s
    assert np.max(np.abs(back - x)) <= 1e-12 * np.max(np.abs(x))


def test_padding_and_signs():
    s = synth.make_signs(48, seed=1, name="p")
    assert set(np.unique(s)) == {-1, 1}
    out = R.rotate_padded64(np.ones(40), np.ones(40), 48)
    assert out.shape == (48,) and np.all(out[40:] == 0)
    with pytest.raises(ValueError):
        R.rotate64(np.ones(8), np.zeros(8))


def test_planted_natural_order_is_caught():
    """A naturally ordered (bit-reversed rows) Hadamard matrix is a plausible
    mistake; the scipy pin separates it from the Sylvester order."""
    n = 8
    rev = [int(f"{i:03b}"[::-1], 2) for i in range(n)]
    wrong = R.walsh_matrix(n)[rev]
    assert not np.array_equal(wrong, hadamard(n))


def test_sampled_rows_match_full_rotation():
    """rotate64_at picks single rows of H_n: it equals rotate64 at those indices
    (blockwise, across several blocks)."""
    K = 3 * 256
    x = np.random.default_rng(11).standard_normal(K)
    s = np.where(np.random.default_rng(12).integers(0, 2, K) == 1, 1.0, -1.0)
    idx = np.array([0, 1, 255, 256, 300, 511, 512, 767])
    assert np.allclose(R.rotate64_at(x, s, idx), R.rotate64(x, s)[idx], rtol=0, atol=1e-12)
