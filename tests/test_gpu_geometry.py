"""GPU parity across tile geometries (lane_cols × tile_rows) and row groups
that share a tile, through the C ABI.

* Geometries of every lane_cols the kernels serve, the library's choices on
  the workload shapes among them (3 × 20, 4 × 16, 2 × 32, 1 × 64, 8 × 8, ...),
  plus small ones, on a matrix with a ragged last tile and a ragged last column group:
  each layout decodes bit-exactly to the drawn points, all four layouts (and
  both exception decoders) give bit-identical y, and y is within the GEMV
  tolerance of the oracle's f64 matvec on every row.
* The batched and rotated entry points on 3 × 20, 2 × 24 and 1 × 60 give
  the single GEMV's bits (batches: in the v_dot2 mode; on the matrix cores,
  within the dot units' rounding) and the two-call bits.
* Row groups whose boundaries fall inside tiles (each such tile holds rows of
  two groups, every lane reading its own row's centroids): every row matches
  the oracle with its own group's centroids, in every layout, bit-identical
  across layouts; the same launch rotated in the prologue gives the two-call
  bits.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2609_02652_amd as P  # noqa: E402
from paper_2609_02652_amd import synth  # noqa: E402
from oracle import decode as D  # noqa: E402

pytestmark = pytest.mark.gpu

TOL_NORM = 2e-3
TOL_PAPER = 1e-5
CEN = (0.75, 1.25)
# (lane_cols, tile_rows)
GEOMETRIES = [(3, 20), (3, 12), (3, 4), (2, 28), (2, 24), (2, 12), (1, 60), (1, 56), (1, 44),
              (1, 4), (4, 12), (8, 8), (16, 4), (4, 16)]


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


@pytest.fixture(scope="module")
def ragged():
    """203 rows (ragged last tile in every geometry here) × 37 blocks (ragged
    last column group for lane_cols 2, 3, 4, 8, 16)."""
    return synth.make_gemv_inputs(203, 24 * 37 - 5, seed=31, name="geometry")


@pytest.mark.parametrize("geo", GEOMETRIES, ids=[f"{c}x{r}" for c, r in GEOMETRIES])
def test_geometry_all_layouts(dev, dcb, ragged, geo):
    inp = ragged
    say(f"[geometry] {geo} {inp.M}x{inp.K}")
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    x = torch.from_numpy(inp.x).to(dev)
    W = D.weights64_from_points(inp.z, inp.gain, inp.scale, CEN)
    y64 = D.gemv64(W, inp.x)
    ys = {}
    for name, layout in P.LAYOUTS.items():
        mat = P.LeechMatrix.from_fields(dcb, layout, cls, inp.gain, sm, lv, inp.scale, dev,
                                        geometry=geo)
        assert (mat.desc.lane_cols, mat.desc.tile_rows) == geo
        z, c, g = mat.decode()
        assert np.array_equal(z.cpu().numpy(), inp.z), name
        assert np.array_equal(c.cpu().numpy().astype(np.uint16), cls), name
        assert np.array_equal(g.cpu().numpy(), inp.gain), name
        modes = (P.EXC_HOISTED, P.EXC_INLINE) if name in ("planes12x", "golay70") else (None,)
        for mode in modes:
            if mode is not None:
                P.set_exception_mode(mode)
            try:
                ys[(name, mode)] = mat.gemv(x, centroids=CEN).cpu().numpy()
            finally:
                P.set_exception_mode(P.EXC_HOISTED)
    ref = ys[("planes14", None)]
    for key, y in ys.items():
        assert np.array_equal(y.view(np.uint32), ref.view(np.uint32)), key
    e = D.errors(ref, y64, W, inp.x)
    say(f"    errors {e}")
    assert e["max_norm_err"] <= TOL_NORM and e["max_abs_err"] <= TOL_PAPER, e


@pytest.mark.parametrize("geo", [(3, 20), (2, 24), (1, 60)], ids=["3x20", "2x24", "1x60"])
def test_geometry_batched_and_rotated(dev, dcb, geo):
    M, K = 301, 24 * 50
    inp = synth.make_gemv_inputs(M, K, seed=32, name="geometry-batch")
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    mat = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev,
                                    geometry=geo)
    X = np.stack([synth.make_activation(K, seed=40 + b, name="geometry-batch") for b in range(5)])
    Xt = torch.from_numpy(X).to(dev)
    Y = mat.gemv_batch(Xt, centroids=CEN).cpu().numpy()
    P.set_batch_mode(P.BATCH_DOT2)
    try:
        Yd = mat.gemv_batch(Xt, centroids=CEN).cpu().numpy()
    finally:
        P.set_batch_mode(P.BATCH_AUTO)
    W = D.weights64_from_points(inp.z, inp.gain, inp.scale, CEN)
    for b in range(5):
        y1 = mat.gemv(Xt[b].contiguous(), centroids=CEN).cpu().numpy()
        assert np.array_equal(Yd[b].view(np.uint32), y1.view(np.uint32)), b
        # matrix-core products: within the dot units' rounding (2^-15 · Σ|w x|)
        bound = 2.0 ** -15 * (np.abs(W) @ np.abs(X[b].astype(np.float64)))
        assert (np.abs(Y[b].astype(np.float64) - y1) <= bound).all(), b
    raw = Xt[0, :K].contiguous()
    s = torch.from_numpy(synth.make_signs(K, seed=3, name="geometry-batch")).to(dev)
    y_rot = mat.gemv_rotated(raw, s, group_centroids=(CEN,)).cpu().numpy()
    y_two = mat.gemv(P.rotate_x(raw, s, inp.Kpad), centroids=CEN).cpu().numpy()
    assert np.array_equal(y_rot.view(np.uint32), y_two.view(np.uint32))


# (group rows, geometry): boundaries inside tiles, on tile starts, and a group
# shorter than a tile that starts on a tile boundary
STRADDLE = [([100, 37, 90], (3, 20)), ([4096 - 8, 8 + 1024, 1024], (2, 24)),
            ([13, 51, 64, 7], (1, 64)), ([24, 10, 30], (4, 12))]


@pytest.mark.parametrize("case", range(len(STRADDLE)))
def test_groups_sharing_tiles(dev, dcb, case):
    parts, geo = STRADDLE[case]
    K = 24 * 23
    ins = [synth.make_gemv_inputs(M, K, seed=600 + 10 * case + i, name=f"straddle{i}")
           for i, M in enumerate(parts)]
    cens = [(0.75, 1.25), (0.9, 1.1), (1.3, 0.6), (1.05, 0.85)][:len(parts)]
    z = np.concatenate([i.z for i in ins])
    gain = np.concatenate([i.gain for i in ins])
    scale = np.concatenate([i.scale for i in ins])
    x = ins[0].x
    cls, sm, lv = dcb.cb.fields_from_points(z)
    xt = torch.from_numpy(x).to(dev)
    ref = None
    for name, layout in P.LAYOUTS.items():
        say(f"[groups] {parts} geometry {geo} {name}")
        mat = P.LeechMatrix.from_fields(dcb, layout, cls, gain, sm, lv, scale, dev, geometry=geo)
        y = mat.gemv_grouped(xt, parts, cens).cpu().numpy()
        r0 = 0
        for inp, c in zip(ins, cens):
            W = D.weights64_from_points(inp.z, inp.gain, inp.scale, c)
            e = D.errors(y[r0:r0 + inp.M], D.gemv64(W, x), W, x)
            assert e["max_norm_err"] <= TOL_NORM and e["max_abs_err"] <= TOL_PAPER, (name, e)
            r0 += inp.M
        if ref is None:
            ref = y
        if name == "planes14":
            raw = xt[:K].contiguous()
            y_rot = mat.gemv_rotated(raw, None, parts, cens).cpu().numpy()
            y_two = mat.gemv_grouped(P.rotate_x(raw, None, mat.Kpad), parts, cens).cpu().numpy()
            assert np.array_equal(y_rot.view(np.uint32), y_two.view(np.uint32))
        assert np.array_equal(y.view(np.uint32), ref.view(np.uint32)), name
