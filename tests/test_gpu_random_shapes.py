"""GPU parity on seeded random shapes: M and K drawn from 1 to a few thousand,
so tiles, column groups, lane_cols, the last tile's height and the last
column group's width take many combinations the fixed cases do not.  For each
shape every layout must decode bit-exactly to the drawn points, all four
layouts must give bit-identical y, y must be within the GEMV tolerance of the
oracle on sampled rows, and, on a third of the shapes, the batched, grouped
and rotated entry points must give the single GEMV's or the two-call bits
(batches on the matrix cores: within the dot units' rounding of the single
GEMV, and its bits in the v_dot2 mode).
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2609_02652_amd as P  # noqa: E402
from paper_2609_02652_amd import synth  # noqa: E402
from oracle import decode as D  # noqa: E402
from oracle import rotation as R  # noqa: E402

pytestmark = pytest.mark.gpu

CEN = (0.75, 1.25)
_rng = np.random.default_rng(2609)
# (M, K): a few fixed extremes, then draws; K need not be a multiple of 24 or 8
SHAPES = [(1, 1), (1, 23), (2, 25), (63, 24 * 64), (64, 24 * 65 + 1), (129, 7)]
SHAPES += [(int(m), int(k)) for m, k in zip(_rng.integers(1, 3000, 18), _rng.integers(1, 3000, 18))]


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


@pytest.mark.parametrize("i", range(len(SHAPES)))
def test_random_shape(dev, dcb, i):
    M, K = SHAPES[i]
    say(f"[random shape {i}] {M}x{K}")
    inp = synth.make_gemv_inputs(M, K, seed=100 + i, name="random-shape")
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    x = torch.from_numpy(inp.x).to(dev)
    rows = np.sort(np.random.default_rng(i).choice(M, min(M, 64), replace=False))
    W = D.weights64_from_points(inp.z[rows], inp.gain[rows], inp.scale[rows], CEN)
    y64 = D.gemv64(W, inp.x)
    ys = {}
    for name, layout in P.LAYOUTS.items():
        mat = P.LeechMatrix.from_fields(dcb, layout, cls, inp.gain, sm, lv, inp.scale, dev)
        z, c, g = mat.decode()
        assert np.array_equal(z.cpu().numpy(), inp.z), name
        assert np.array_equal(c.cpu().numpy().astype(np.uint16), cls), name
        assert np.array_equal(g.cpu().numpy(), inp.gain), name
        ys[name] = mat.gemv(x, centroids=CEN).cpu().numpy()
        if name == "planes14":
            p14 = mat
    for name, y in ys.items():
        assert np.array_equal(y.view(np.uint32), ys["planes14"].view(np.uint32)), name
    e = D.errors(ys["planes14"][rows], y64, W, inp.x)
    assert e["max_norm_err"] <= 2e-3, e

    if i % 3:
        return
    y1 = ys["planes14"]
    # batched: three activations, the first being x
    X = np.stack([inp.x] + [synth.make_activation(K, seed=1000 + i + b, name="random-shape")
                            for b in range(2)])
    Xd = torch.from_numpy(X).to(dev)
    Y = p14.gemv_batch(Xd, centroids=CEN).cpu().numpy()
    # matrix-core products: within 2^-15 · Σ|w x| of the single GEMV (the dot
    # units' measured rounding), and the v_dot2 mode gives its bits
    bound = 2.0 ** -15 * (np.abs(W) @ np.abs(inp.x.astype(np.float64)))
    assert (np.abs(Y[0][rows].astype(np.float64) - y1[rows]) <= bound).all()
    P.set_batch_mode(P.BATCH_DOT2)
    try:
        Y = p14.gemv_batch(Xd, centroids=CEN).cpu().numpy()
    finally:
        P.set_batch_mode(P.BATCH_AUTO)
    assert np.array_equal(Y[0].view(np.uint32), y1.view(np.uint32))
    # grouped, one group: the plain call's bits
    yg = p14.gemv_grouped(x, [M], [CEN]).cpu().numpy()
    assert np.array_equal(yg.view(np.uint32), y1.view(np.uint32))
    # rotated, where K is a multiple of 8 and fits the prologue
    if K % 8 == 0 and K <= 2560:
        raw = x[:K].contiguous()
        s = torch.from_numpy(synth.make_signs(K, seed=i, name="random-shape")).to(dev)
        y_rot = p14.gemv_rotated(raw, s, group_centroids=(CEN,)).cpu().numpy()
        y_two = p14.gemv(P.rotate_x(raw, s, inp.Kpad), centroids=CEN).cpu().numpy()
        assert np.array_equal(y_rot.view(np.uint32), y_two.view(np.uint32))
        xr = R.rotate_padded64(inp.x[:K], s.cpu().numpy(), inp.Kpad).astype(np.float16)
        Wr = D.weights64_from_points(inp.z[rows], inp.gain[rows], inp.scale[rows], CEN)
        er = D.errors(y_rot[rows], D.gemv64(Wr, xr), Wr, xr)
        assert er["max_norm_err"] <= 2e-3, er
