"""Pins for the oracle's decode and matvec (oracle/decode.py).

Checks against hand-derived blocks, brute-force sums on tiny matrices, the
unit-norm property of every decoded direction, one-hot column extraction, and
planted mistakes that the pins must catch.
"""
import numpy as np
import pytest

from oracle import decode as D
from oracle import lattice as L
from paper_2609_02652_amd import synth


@pytest.fixture(scope="module")
def pts():
    return synth.sample_ball_points(synth.rng_for(7, "oracle-decode"), 3000)


def test_hand_decoded_block():
    # z = (−3, 1^23): the odd shell-2 class; levels ascending (1, 3)
    z = [-3] + [1] * 23
    cid, sm, lv = D.fields_of_point(z)
    cls = L.ball_classes()[cid]
    assert cls.mags_desc == (3,) + (1,) * 23 and cls.shell == 2
    assert sm == 1 and lv == [1] + [0] * 23
    assert D.decode_block(cid, sm, lv) == z
    # weight: scale · centroid · z / (4 √2)
    w = D.weights64(np.array([[cid]]), np.array([[1]]), np.array([[0.5]], np.float16),
                    np.array([[z]]), centroids=(1.0, 2.0))
    assert w.shape == (1, 24)
    assert w[0, 0] == pytest.approx(0.5 * 2.0 * -3 / (4 * 2 ** 0.5), rel=1e-15)
    assert w[0, 1] == pytest.approx(0.5 * 2.0 * 1 / (4 * 2 ** 0.5), rel=1e-15)


def test_hand_decoded_even_block():
    # (−8, 0^23): class of shell 4 with levels (0, 8); the sign sits on coordinate 5
    z = [0] * 24
    z[5] = -8
    cid, sm, lv = D.fields_of_point(z)
    assert L.ball_classes()[cid].levels == (0, 8)
    assert sm == 1 << 5
    assert lv == [1 if i == 5 else 0 for i in range(24)]


def test_round_trip_scalar_and_vector(pts):
    cid, sm, lv = D.fields_from_points(pts)
    for b in range(0, len(pts), 37):
        c1, s1, l1 = D.fields_of_point(pts[b])
        assert (c1, s1, l1) == (int(cid[b]), int(sm[b]), [int(v) for v in lv[b]])
        assert D.decode_block(c1, s1, l1) == [int(v) for v in pts[b]]
    z = D.decode_fields(cid, sm, lv)
    assert z.dtype == np.int8
    assert (z == pts).all()


@pytest.mark.parametrize("mutate", ["class", "level", "zero_sign", "multiset", "high_sign"])
def test_invalid_fields_raise(pts, mutate):
    cid, sm, lv = D.fields_from_points(pts[:64])
    cid, sm, lv = cid.copy(), sm.copy(), lv.copy()
    classes = L.ball_classes()
    if mutate == "class":
        cid[3] = 301
    elif mutate == "level":
        lv[3, 0] = classes[int(cid[3])].n_levels
    elif mutate == "zero_sign":
        b = next(b for b in range(64) if classes[int(cid[b])].levels[0] == 0)
        i = int(np.nonzero(lv[b] == 0)[0][0])
        sm[b] |= np.uint32(1 << i)
    elif mutate == "multiset":
        b = next(b for b in range(64) if classes[int(cid[b])].n_levels >= 2)
        i = int(np.argmin(lv[b]))
        lv[b, i] += 1                      # one coordinate moves to the next level
    elif mutate == "high_sign":
        sm[0] |= np.uint32(1 << 24)
    with pytest.raises(ValueError):
        D.decode_fields(cid, sm, lv)


def test_every_direction_has_unit_norm(pts):
    """‖w_b‖₂ = scale · centroid for every block: the level values divide by the
    shell's norm 4√m (§2.3 folds this per-class constant into the levels)."""
    n = 240
    cid, sm, lv = D.fields_from_points(pts[:n])
    M, nb = 10, 24
    scale = np.linspace(0.01, 0.2, n).astype(np.float16).reshape(M, nb)
    gain = (np.arange(n) % 2).astype(np.uint8).reshape(M, nb)
    W = D.weights64(cid.reshape(M, nb), gain, scale, pts[:n].reshape(M, nb, 24), centroids=(0.75, 1.25))
    blocks = W.reshape(M, nb, 24)
    want = scale.astype(np.float64) * np.where(gain == 1, 1.25, 0.75)
    assert np.allclose(np.sqrt((blocks ** 2).sum(-1)), want, rtol=1e-14, atol=0)
    assert np.allclose(D.row_norms_from_scales(cid.reshape(M, nb), gain, scale, (0.75, 1.25)),
                       np.sqrt((W ** 2).sum(1)), rtol=1e-14)


@pytest.mark.parametrize("M,K", [(2, 48), (3, 72), (5, 30)])
def test_tiny_matvec_brute_force(M, K):
    inp = synth.make_gemv_inputs(M, K, seed=3, name=f"tiny{M}x{K}")
    cid, sm, lv = D.fields_from_points(inp.z)
    z = D.decode_fields(cid, sm, lv)
    W = D.weights64(cid, inp.gain, inp.scale, z, centroids=(0.9, 1.1))
    assert W.shape == (M, inp.Kpad)
    y = D.gemv64(W, inp.x)
    # brute force: explicit loops over every block and coordinate
    yb = np.zeros(M)
    classes = L.ball_classes()
    for r in range(M):
        for b in range(inp.nb):
            c = classes[int(cid[r, b])]
            cen = float(np.float32(1.1)) if inp.gain[r, b] else float(np.float32(0.9))  # f32 centroids
            f = float(inp.scale[r, b]) * cen / (4 * c.shell ** 0.5)
            for i in range(24):
                yb[r] += f * int(z[r, b, i]) * float(inp.x[24 * b + i])
    assert np.allclose(y, yb, rtol=1e-13, atol=1e-15)
    assert np.allclose(D.gemv64_naive(W, inp.x), y, rtol=1e-13, atol=1e-15)
    assert (inp.x[K:] == 0).all()


def test_one_hot_extracts_columns():
    inp = synth.make_gemv_inputs(4, 96, seed=5, name="onehot")
    cid, sm, lv = D.fields_from_points(inp.z)
    W = D.weights64(cid, inp.gain, inp.scale, D.decode_fields(cid, sm, lv))
    for j in (0, 1, 23, 24, 50, 95):
        e = np.zeros(inp.Kpad, np.float16)
        e[j] = 1
        assert (D.gemv64(W, e) == W[:, j]).all()


def test_error_metrics():
    inp = synth.make_gemv_inputs(3, 48, seed=9, name="err")
    cid, sm, lv = D.fields_from_points(inp.z)
    W = D.weights64(cid, inp.gain, inp.scale, D.decode_fields(cid, sm, lv))
    y64 = D.gemv64(W, inp.x)
    assert D.errors(y64, y64, W, inp.x) == {"max_norm_err": 0.0, "max_abs_err": 0.0}
    y = y64.copy()
    y[1] += 1e-3
    e = D.errors(y, y64, W, inp.x)
    x = inp.x.astype(np.float64)
    assert e["max_norm_err"] == pytest.approx(1e-3 / (np.linalg.norm(W[1]) * np.linalg.norm(x)), rel=1e-6)
    assert e["max_abs_err"] == pytest.approx(1e-3 / (np.abs(W[1]) @ np.abs(x)), rel=1e-6)


# ----------------------------------------------------------------------------
# Planted mistakes: each plausible slip in the decode must trip a pin.
# ----------------------------------------------------------------------------
def test_planted_sign_shift_is_caught(pts):
    """Reading sign bit i+1 for coordinate i breaks membership for odd blocks,
    whose signs the codeword forces.  (Inverting every sign is not caught by
    membership, since −z is a lattice point too; the GPU parity tests compare
    decoded z with the drawn z exactly, which catches it.)"""
    odd = [b for b in range(200) if pts[b, 0] % 2]
    cid, sm, lv = D.fields_from_points(pts[odd])
    full = np.uint32((1 << 24) - 1)
    bad = ((sm >> np.uint32(1)) | (sm << np.uint32(23))) & full
    with pytest.raises(ValueError):
        D.decode_fields(cid, bad, lv)
    z = D.decode_fields(cid, sm, lv)
    assert (z == pts[odd]).all()


def test_planted_level_order_is_caught(pts):
    """Levels read in descending instead of ascending order give another
    multiset than the class's for every class with two or more levels."""
    cid, sm, lv = D.fields_from_points(pts[:200])
    nlev = np.array([c.n_levels for c in L.ball_classes()])[cid.astype(int)]
    flipped = (nlev[:, None] - 1 - lv.astype(int)).astype(np.uint8)
    with pytest.raises(ValueError):
        D.decode_fields(cid, sm, flipped)


def test_planted_normalisation_is_caught(pts):
    """Dividing by √(2m) (the standard-scaling norm) instead of 4√m changes
    every block norm, which the unit-norm pin catches."""
    cid, sm, lv = D.fields_from_points(pts[:24])
    z = pts[:24].astype(np.float64)
    shell = np.array([L.ball_classes()[int(c)].shell for c in cid])
    wrong = z / np.sqrt(2 * shell)[:, None]
    assert not np.allclose(np.sqrt((wrong ** 2).sum(1)), 1.0)
    right = z / (4 * np.sqrt(shell))[:, None]
    assert np.allclose(np.sqrt((right ** 2).sum(1)), 1.0, rtol=1e-15)


def test_weights_from_points_equal_class_weights():
    inp = synth.make_gemv_inputs(6, 240, seed=13, name="wfp")
    cid, sm, lv = D.fields_from_points(inp.z)
    W1 = D.weights64(cid, inp.gain, inp.scale, inp.z, centroids=(0.5, 2.0))
    W2 = D.weights64_from_points(inp.z, inp.gain, inp.scale, centroids=(0.5, 2.0))
    assert np.allclose(W1, W2, rtol=1e-15, atol=0)
