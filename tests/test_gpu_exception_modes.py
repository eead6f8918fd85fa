"""The two exception decoders of Planes12x and Golay70 (hoisted: each exception
kept as a table entry of its own; in line: decoded in the loop) through the C
ABI: bit-identical y to each other and to Planes14, and to the oracle within
tolerance, on the usual shapes, on a tile made only of exceptions, and on a
grouped launch whose two table copies with 3072 exception entries each exceed
the LDS budget (decoded in line whichever mode is asked for)."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2609_02652_amd as P  # noqa: E402
from paper_2609_02652_amd import synth  # noqa: E402
from oracle import decode as D  # noqa: E402

pytestmark = pytest.mark.gpu
CEN = (0.75, 1.25)


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


def y_in_mode(mat, x, mode):
    P.set_exception_mode(mode)
    try:
        y = mat.gemv(x, centroids=CEN).cpu().numpy()
    finally:
        P.set_exception_mode(P.EXC_HOISTED)
    return y


def check(dev, dcb, inp, label, layout):
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    g70 = P.LeechMatrix.from_fields(dcb, layout, cls, inp.gain, sm, lv, inp.scale, dev)
    p14 = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
    assert (p14.desc.lane_cols, p14.desc.tile_rows) == (g70.desc.lane_cols, g70.desc.tile_rows)
    say(f"[exception modes] {P.LAYOUT_NAMES[layout]} {label}: {g70.desc.n_exceptions} "
        f"exceptions of {inp.M * inp.nb}")
    x = torch.from_numpy(inp.x).to(dev)
    yh = y_in_mode(g70, x, P.EXC_HOISTED)
    yi = y_in_mode(g70, x, P.EXC_INLINE)
    yp = p14.gemv(x, centroids=CEN).cpu().numpy()
    assert np.array_equal(yh.view(np.uint32), yi.view(np.uint32)), "modes differ"
    assert np.array_equal(yh.view(np.uint32), yp.view(np.uint32)), "differs from Planes14"
    W = D.weights64_from_points(inp.z, inp.gain, inp.scale, CEN)
    e = D.errors(yh, D.gemv64(W, inp.x), W, inp.x)
    assert e["max_norm_err"] <= 2e-3 and e["max_abs_err"] <= 1e-5, e
    return g70


EXC_LAYOUTS = [P.PLANES12X, P.GOLAY70]


@pytest.mark.parametrize("layout", EXC_LAYOUTS, ids=["planes12x", "golay70"])
@pytest.mark.parametrize("M,K", [(1, 24), (65, 408), (257, 792), (768, 1536), (14337, 120)])
def test_modes_agree(dev, dcb, M, K, layout):
    check(dev, dcb, synth.make_gemv_inputs(M, K, seed=M + K, name="excmodes"), f"{M}x{K}",
          layout)


def exception_points(cb, layout, n, seed):
    """n drawn points that are exceptions of the layout.  Planes12x: points of
    five-level classes.  Golay70: points its 2-bit code cannot hold, which the
    host expansion of a one-column matrix flags (an exception record's entry
    field, bits [0, 12), is 1024 or more; with one block per row the storage
    slot of row r is r)."""
    pool = synth.sample_ball_points(synth.rng_for(seed, "exc-pool"), 40 * n)
    cls, sm, lv = cb.fields_from_points(pool)
    if layout == P.PLANES12X:
        flags = lv.max(axis=1) == 4
    else:
        gain = np.zeros(len(pool), np.uint8)
        d, main, _, _ = P.expand_layout(cb, P.GOLAY70, cls[:, None], gain[:, None], sm[:, None],
                                        lv[:, None, :])
        rec = main[: 9 * len(pool)].reshape(-1, 9).astype(np.uint32)
        flags = ((rec[:, 0] | rec[:, 1] << 8) & 0xFFF) >= 1024
    picked = pool[flags]
    assert len(picked) >= n, "pool too small"
    return picked[:n]


@pytest.mark.parametrize("layout", EXC_LAYOUTS, ids=["planes12x", "golay70"])
def test_tile_of_exceptions(dev, dcb, layout):
    """8 × 14400: geometry 16 × 4, two tiles of 4 rows × 600 blocks.  The first
    tile holds only exceptions (2400 entries after the table's 1024 class
    entries); the second is an ordinary tile."""
    M, K = 8, 14400
    inp = synth.make_gemv_inputs(M, K, seed=31, name="exc-heavy")
    z = inp.z.copy()
    z[:4] = exception_points(dcb.cb, layout, 4 * inp.nb, seed=31).reshape(4, inp.nb, 24)
    inp = synth.GemvInputs(M, inp.K, inp.Kpad, inp.nb, z, inp.gain, inp.scale, inp.x, inp.seed,
                           inp.name)
    mat = check(dev, dcb, inp, "heavy tile", layout)
    assert mat.desc.n_exceptions >= 4 * inp.nb
    z_dev, _, _ = mat.decode()
    assert np.array_equal(z_dev.cpu().numpy(), z)


def test_mode_is_validated():
    with pytest.raises(P.LeechError, match="LEECH_E_ARG"):
        P.set_exception_mode(7)


@pytest.mark.parametrize("layout", EXC_LAYOUTS, ids=["planes12x", "golay70"])
def test_exceptions_over_the_lds_budget(dev, dcb, layout):
    """8 × 18432 (768 blocks a row), geometry 16 × 4, the first tile all
    exceptions (3072, the most a tile may hold), launched as two row groups
    [2, 6] so that tile 0 holds rows of both groups: two table copies of
    (1024 + 3072) entries (128 KiB) and the activation exceed the 160 KiB of
    LDS, so the exceptions are decoded in line in either mode.  Every row
    matches the oracle with its own group's centroids, and both modes and
    Planes14 give the same bits."""
    M, K = 8, 18432
    inp = synth.make_gemv_inputs(M, K, seed=33, name="exc-budget")
    z = inp.z.copy()
    z[:4] = exception_points(dcb.cb, layout, 4 * inp.nb, seed=33).reshape(4, inp.nb, 24)
    cls, sm, lv = dcb.cb.fields_from_points(z)
    mat = P.LeechMatrix.from_fields(dcb, layout, cls, inp.gain, sm, lv, inp.scale, dev)
    p14 = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
    assert mat.desc.tile_exc_max == 3072 and mat.desc.tile_rows == 4
    say(f"[exception modes] {P.LAYOUT_NAMES[layout]} over the budget: "
        f"{mat.desc.n_exceptions} exceptions")
    x = torch.from_numpy(inp.x).to(dev)
    rows, cens = [2, 6], [(0.75, 1.25), (1.1, 0.9)]
    ys = []
    for mode in (P.EXC_HOISTED, P.EXC_INLINE):
        P.set_exception_mode(mode)
        try:
            ys.append(mat.gemv_grouped(x, rows, cens).cpu().numpy())
        finally:
            P.set_exception_mode(P.EXC_HOISTED)
    yp = p14.gemv_grouped(x, rows, cens).cpu().numpy()
    assert np.array_equal(ys[0].view(np.uint32), ys[1].view(np.uint32))
    assert np.array_equal(ys[0].view(np.uint32), yp.view(np.uint32))
    r0 = 0
    for n, c in zip(rows, cens):
        W = D.weights64_from_points(z[r0:r0 + n], inp.gain[r0:r0 + n], inp.scale[r0:r0 + n], c)
        e = D.errors(ys[0][r0:r0 + n], D.gemv64(W, inp.x), W, inp.x)
        assert e["max_norm_err"] <= 2e-3 and e["max_abs_err"] <= 1e-5, e
        r0 += n
