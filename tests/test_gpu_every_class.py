"""GPU parity over every class of the ball and over the whole kissing shell.

§2.4 ("Verification") locks the codebook over the whole ball and decodes every
block of a transcoded matrix bit for bit; §2.2 unfolds every index at load
time.  Draws proportional to class size never reach the rare classes (no
shell 2 or 3 point, no |z| of 12 or 13, no one-level class among the blocks
of a 4096×4104 draw), so these matrices are built from the oracle's format-v1
index instead:

* every class id 0..300: its first and last index and four uniform members,
  each once with gain bit 0 and once with gain bit 1, in a seeded shuffle, and
  a second matrix with the same blocks sorted by class (the five-level classes,
  i.e. the exceptions, then pile up in a few tiles);
* every one of the 196,560 minimal vectors (shell 2, §2.4's lock).

Block scales are fp16 |N(0,1)|·0.02 with every fifth one an fp16 subnormal
(k·2^-24) and two exact zeros.  Through the C ABI, for every layout: decoded
z, class id and gain bit equal the oracle's point and fields bit for bit; y is
within the tolerance of the oracle's f64 matvec (2e-3 of ‖W_r‖‖x‖, and the
paper's 1e-5 of Σ|w x|); y is bit-identical across the four layouts and both
exception decoders; the batched, grouped and rotated entry points give the
single GEMV's bits (or the two-call bits) and the oracle's values (batches on
the matrix cores: within the dot units' rounding of the single GEMV, and its
bits in the v_dot2 mode).
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2609_02652_amd as P  # noqa: E402
from paper_2609_02652_amd import synth  # noqa: E402
from oracle import decode as D  # noqa: E402
from oracle import index as I  # noqa: E402
from oracle import lattice as L  # noqa: E402
from oracle import rotation as R  # noqa: E402

pytestmark = pytest.mark.gpu

TOL_NORM = 2e-3
TOL_PAPER = 1e-5
CEN = (0.75, 1.25)
N_CLASSES = 301


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def dcb(dev):
    return P.DeviceCodebook(P.Codebook(12), dev)


def every_class_points(seed: int) -> np.ndarray:
    """First, last and four uniform indices of every class, as points."""
    offs = I.class_offsets()
    rng = synth.rng_for(seed, "every-class/index")
    idx = []
    for c in range(N_CLASSES):
        lo, hi = offs[c], offs[c + 1]
        idx += [lo, hi - 1] + [lo + int(rng.integers(0, hi - lo)) for _ in range(4)]
    return np.array([I.point_of_index(i) for i in idx], dtype=np.int8)


def scales(shape, seed: int) -> np.ndarray:
    s = (np.abs(synth.rng_for(seed, "every-class/scale").standard_normal(shape)) * 0.02)
    s = s.astype(np.float16).ravel()
    k = synth.rng_for(seed, "every-class/subnormal").integers(1, 1024, s.size)
    sub = (k.astype(np.float64) * 2.0 ** -24).astype(np.float16)
    s[::5] = sub[::5]
    s[1] = 0
    s[-2] = 0
    assert np.all(np.abs(s[::5][s[::5] != 0]) < np.float16(2.0 ** -14))   # subnormal
    return s.reshape(shape)


def build(M: int, nb: int, seed: int, sort_by_class: bool):
    """(z [M, nb, 24], gain [M, nb], scale [M, nb], x [Kpad]) holding every
    class twice (both gain bits), the rest of the matrix uniform points."""
    pts = every_class_points(seed)
    z = np.concatenate([pts, pts])
    gain = np.concatenate([np.zeros(len(pts), np.uint8), np.ones(len(pts), np.uint8)])
    n = M * nb
    assert n >= len(z)
    extra = synth.sample_ball_points(synth.rng_for(seed, "every-class/extra"), n - len(z))
    z = np.concatenate([z, extra])
    gain = np.concatenate([gain, synth.rng_for(seed, "every-class/gain").integers(
        0, 2, n - len(gain)).astype(np.uint8)])
    if sort_by_class:
        cid, _, _ = D.fields_from_points(z)
        order = np.argsort(cid, kind="stable")
    else:
        order = synth.rng_for(seed, "every-class/perm").permutation(n)
    z, gain = z[order].reshape(M, nb, 24), gain[order].reshape(M, nb)
    x = synth.make_activation(nb * 24, seed, "every-class")
    return z, gain, scales((M, nb), seed), x


SHAPES = [(151, 24, False), (151, 24, True), (9, 402, False)]
_cache = {}


def case(M, nb, sort_by_class):
    key = (M, nb, sort_by_class)
    if key not in _cache:
        z, gain, sc, x = build(M, nb, 5, sort_by_class)
        cls, sm, lv = D.fields_from_points(z)                  # the oracle's fields
        W = D.weights64(cls, gain, sc, D.decode_fields(cls, sm, lv), CEN)
        _cache[key] = (z, gain, sc, x, (cls, sm, lv), W)
    return _cache[key]


def test_matrix_holds_every_class():
    z, gain, _, _, (cls, _, _), _ = case(151, 24, False)
    present = {(int(c), int(g)) for c, g in zip(cls.ravel(), gain.ravel())}
    assert all((c, g) in present for c in range(N_CLASSES) for g in (0, 1))
    mags = np.abs(z.astype(np.int64))
    assert mags.max() == 13 and (mags == 12).any()
    shells = (z.astype(np.int64) ** 2).sum(-1) // 16
    assert set(range(2, 13)) <= set(shells.ravel().tolist())
    one_level = [c.class_id for c in L.ball_classes() if c.n_levels == 1]
    assert one_level and all(c in cls for c in one_level)


@pytest.mark.parametrize("M,nb,sort_by_class", SHAPES)
def test_every_class_all_layouts(dev, dcb, M, nb, sort_by_class):
    z, gain, sc, x, (cls, sm, lv), W = case(M, nb, sort_by_class)
    pc, psm, plv = dcb.cb.fields_from_points(z)                 # the library's fields
    assert (pc == cls).all() and (psm == sm).all() and (plv == lv).all()
    xd = torch.from_numpy(x).to(dev)
    y64 = D.gemv64(W, x)
    ys = {}
    for name, lay in P.LAYOUTS.items():
        say(f"[every class] {M}x{nb * 24} sorted={sort_by_class} layout={name}")
        mat = P.LeechMatrix.from_fields(dcb, lay, cls, gain, sm, lv, sc, dev)
        zz, cc, gg = mat.decode()
        assert np.array_equal(zz.cpu().numpy(), z), name
        assert np.array_equal(cc.cpu().numpy().astype(np.uint16), cls), name
        assert np.array_equal(gg.cpu().numpy(), gain), name
        modes = (P.EXC_HOISTED, P.EXC_INLINE) if name in ("planes12x", "golay70") else (None,)
        for mode in modes:
            if mode is not None:
                P.set_exception_mode(mode)
            try:
                y = mat.gemv(xd, centroids=CEN).cpu().numpy()
            finally:
                P.set_exception_mode(P.EXC_HOISTED)
            ys[(name, mode)] = y
            e = D.errors(y, y64, W, x)
            say(f"    mode={mode} errors {e}")
            assert e["max_norm_err"] <= TOL_NORM and e["max_abs_err"] <= TOL_PAPER, (name, mode, e)
        del mat
    ref = ys[("planes14", None)].view(np.uint32)
    for k, y in ys.items():
        assert np.array_equal(y.view(np.uint32), ref), k


@pytest.mark.parametrize("M,nb,sort_by_class", SHAPES)
def test_every_class_batched_grouped_rotated(dev, dcb, M, nb, sort_by_class):
    z, gain, sc, x, (cls, sm, lv), W = case(M, nb, sort_by_class)
    Kpad = nb * 24
    mat = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, gain, sm, lv, sc, dev)
    say(f"[every class: batch] {M}x{Kpad}")
    X = np.stack([x] + [synth.make_activation(Kpad, 6 + b, "every-class-batch") for b in range(2)])
    Xd = torch.from_numpy(X).to(dev)
    Y = mat.gemv_batch(Xd, centroids=CEN).cpu().numpy()
    P.set_batch_mode(P.BATCH_DOT2)
    try:
        Yd = mat.gemv_batch(Xd, centroids=CEN).cpu().numpy()
    finally:
        P.set_batch_mode(P.BATCH_AUTO)
    # matrix-core products: within 2^-15 · Σ|w x| of the single GEMV (the dot
    # units' measured rounding); v_dot2 products: the single GEMV's bits
    for b in range(3):
        yb = mat.gemv(Xd[b].contiguous(), centroids=CEN).cpu().numpy()
        assert np.array_equal(Yd[b].view(np.uint32), yb.view(np.uint32)), b
        bound = 2.0 ** -15 * (np.abs(W) @ np.abs(X[b].astype(np.float64)))
        assert (np.abs(Y[b].astype(np.float64) - yb) <= bound).all(), b
        e = D.errors(Y[b], D.gemv64(W, X[b]), W, X[b])
        assert e["max_norm_err"] <= TOL_NORM and e["max_abs_err"] <= TOL_PAPER, (b, e)
    if M > 64:
        say(f"[every class: grouped] {M}x{Kpad}")
        rows = [64, M - 64]
        cens = [CEN, (1.1, 0.9)]
        xd = torch.from_numpy(x).to(dev)
        y64 = np.empty(M)
        Wg = np.empty_like(W)
        for g, (r0, r1) in enumerate(((0, 64), (64, M))):
            Wg[r0:r1] = D.weights64(cls[r0:r1], gain[r0:r1], sc[r0:r1],
                                    D.decode_fields(cls[r0:r1], sm[r0:r1], lv[r0:r1]), cens[g])
        y64 = D.gemv64(Wg, x)
        yl = {}
        for name, lay in P.LAYOUTS.items():
            m = mat if name == "planes14" else P.LeechMatrix.from_fields(dcb, lay, cls, gain, sm, lv, sc, dev)
            yl[name] = m.gemv_grouped(xd, rows, cens).cpu().numpy()
            e = D.errors(yl[name], y64, Wg, x)
            assert e["max_norm_err"] <= TOL_NORM and e["max_abs_err"] <= TOL_PAPER, (name, e)
        for name, y in yl.items():
            assert np.array_equal(y.view(np.uint32), yl["planes14"].view(np.uint32)), name
    say(f"[every class: rotated] {M}x{Kpad}")
    K = Kpad
    s = synth.make_signs(K, seed=7, name="every-class-rot")
    xr_raw = torch.from_numpy(x[:K].copy()).to(dev)
    sd = torch.from_numpy(s).to(dev)
    y_one = mat.gemv_rotated(xr_raw, sd, group_centroids=(CEN,)).cpu().numpy()
    y_two = mat.gemv(P.rotate_x(xr_raw, sd, Kpad), centroids=CEN).cpu().numpy()
    assert np.array_equal(y_one.view(np.uint32), y_two.view(np.uint32))
    xr16 = R.rotate_padded64(x[:K], s, Kpad).astype(np.float16)
    e = D.errors(y_one, D.gemv64(W, xr16), W, xr16)
    assert e["max_norm_err"] <= TOL_NORM, e


def test_every_minimal_vector_all_layouts(dev, dcb):
    """All 196,560 points of shell 2 (three classes), 8190 rows × 24 blocks."""
    n = 196560
    offs = I.class_offsets()
    shell2 = [c.class_id for c in L.ball_classes() if c.shell == 2]
    assert offs[max(shell2) + 1] == n
    pts = np.array([I.point_of_index(i) for i in range(n)], dtype=np.int8)
    assert len({p.tobytes() for p in pts}) == n
    perm = synth.rng_for(9, "kissing/perm").permutation(n)
    M, nb = 8190, 24
    z = pts[perm].reshape(M, nb, 24)
    gain = synth.rng_for(9, "kissing/gain").integers(0, 2, (M, nb)).astype(np.uint8)
    sc = scales((M, nb), 9)
    x = synth.make_activation(nb * 24, 9, "kissing")
    cls, sm, lv = D.fields_from_points(z)
    W = D.weights64(cls, gain, sc, D.decode_fields(cls, sm, lv), CEN)
    y64 = D.gemv64(W, x)
    xd = torch.from_numpy(x).to(dev)
    ref = None
    for name, lay in P.LAYOUTS.items():
        say(f"[kissing shell] layout={name}")
        mat = P.LeechMatrix.from_fields(dcb, lay, cls, gain, sm, lv, sc, dev)
        zz, cc, gg = mat.decode()
        assert np.array_equal(zz.cpu().numpy(), z), name
        assert np.array_equal(cc.cpu().numpy().astype(np.uint16), cls), name
        assert np.array_equal(gg.cpu().numpy(), gain), name
        y = mat.gemv(xd, centroids=CEN).cpu().numpy()
        e = D.errors(y, y64, W, x)
        assert e["max_norm_err"] <= TOL_NORM and e["max_abs_err"] <= TOL_PAPER, (name, e)
        if ref is None:
            ref = y.view(np.uint32).copy()
        assert np.array_equal(y.view(np.uint32), ref), name
        del mat
