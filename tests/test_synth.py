"""The seeded input generator: every sample is a ball point (checked by the
oracle), classes appear in proportion to their sizes, and inputs are
reproducible from the seed."""
import numpy as np
import pytest

from oracle import decode as D
from oracle import lattice as L
from paper_2609_02652_amd import synth


def test_multisets_agree_with_oracle_classes():
    ms = synth.ball_multisets()
    cls = {c.mags_desc: c.size for c in L.ball_classes()}
    assert {m.mags: m.count for m in ms} == cls


@pytest.fixture(scope="module")
def big_sample():
    return synth.sample_ball_points(synth.rng_for(0, "stats"), 400_000)


def test_samples_are_ball_points(big_sample):
    z = big_sample[:20000]
    for b in range(0, 20000, 499):
        assert L.is_leech_point(z[b])
    D.fields_from_points(z)        # raises on any non-member


def test_class_frequencies_follow_sizes(big_sample):
    cid, _, _ = D.fields_from_points(big_sample)
    classes = L.ball_classes()
    p = np.array([c.size for c in classes], dtype=np.float64)
    p /= p.sum()
    n = len(big_sample)
    obs = np.bincount(cid.astype(int), minlength=len(classes))
    # pool classes with expected count < 20 into one bin, then chi-square
    exp = p * n
    big = exp >= 20
    o = np.append(obs[big], obs[~big].sum())
    e = np.append(exp[big], exp[~big].sum())
    chi2 = ((o - e) ** 2 / e).sum()
    dof = len(o) - 1
    assert chi2 < dof + 6 * np.sqrt(2 * dof), (chi2, dof)
    # aggregate statistics of the ball
    five = sum(c.size for c in classes if c.n_levels == 5) / L.ball_size()
    assert abs(obs[[c.class_id for c in classes if c.n_levels == 5]].sum() / n - five) < 5 * np.sqrt(five / n)
    odd = sum(c.size for c in classes if c.parity) / L.ball_size()
    assert abs((big_sample[:, 0] % 2 != 0).mean() - odd) < 5 * np.sqrt(0.25 / n)


def test_coordinates_are_exchangeable(big_sample):
    """A uniform member of a class puts every magnitude equally often on every
    coordinate."""
    a = np.abs(big_sample.astype(np.int64))
    means = a.mean(axis=0)
    assert np.ptp(means) < 0.02 * means.mean()
    neg = (big_sample < 0).mean(axis=0)
    assert np.ptp(neg) < 0.01


def test_inputs_reproducible_and_padded():
    a = synth.make_gemv_inputs(5, 100, seed=11, name="r")
    b = synth.make_gemv_inputs(5, 100, seed=11, name="r")
    c = synth.make_gemv_inputs(5, 100, seed=12, name="r")
    assert a.Kpad == 120 and a.nb == 5
    for f in ("z", "gain", "scale", "x"):
        assert (getattr(a, f) == getattr(b, f)).all()
    assert (a.z != c.z).any()
    assert (a.x[100:] == 0).all() and (a.x[:100] != 0).all()
    assert a.scale.dtype == np.float16 and (a.scale >= 0).all()
    assert set(np.unique(a.gain)) <= {0, 1}


def test_scale_distribution():
    inp = synth.make_gemv_inputs(256, 4096, seed=0, name="scales")
    s = inp.scale.astype(np.float64).ravel()
    # |N(0,1)|·0.02 has mean 0.02·√(2/π)
    assert abs(s.mean() - 0.02 * np.sqrt(2 / np.pi)) < 3e-4
    sub = (inp.scale != 0) & (np.abs(inp.scale) < np.float16(6.104e-05))
    assert sub.any()               # fp16 subnormal scales occur (about 0.24 %)
