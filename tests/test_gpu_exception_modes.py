"""The two exception decoders of Planes12x and Golay70 (hoisted pre-pass, in
line) through the C ABI: bit-identical y to each other and to Planes14, and to
the oracle within tolerance, on the usual shapes and on a tile whose exception
records exceed the LDS budget (decoded from global memory in both modes)."""
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
    host expansion of a one-column matrix flags (record bit 70; with one block
    per row the storage slot of row r is r)."""
    pool = synth.sample_ball_points(synth.rng_for(seed, "exc-pool"), 40 * n)
    cls, sm, lv = cb.fields_from_points(pool)
    if layout == P.PLANES12X:
        flags = lv.max(axis=1) == 4
    else:
        gain = np.zeros(len(pool), np.uint8)
        d, main, _, _ = P.expand_layout(cb, P.GOLAY70, cls[:, None], gain[:, None], sm[:, None],
                                        lv[:, None, :])
        flags = ((main[: 9 * len(pool)].reshape(-1, 9)[:, 8] >> 6) & 1) == 1
    picked = pool[flags]
    assert len(picked) >= n, "pool too small"
    return picked[:n]


@pytest.mark.parametrize("layout", EXC_LAYOUTS, ids=["planes12x", "golay70"])
def test_tile_over_the_lds_budget(dev, dcb, layout):
    """8 × 14400: lane_cols 16, two tiles of 4 rows × 600 blocks.  The first
    tile holds only exceptions (2400 records, more than the 32 KiB staged in
    LDS): it is decoded in line from global memory in both modes; the second
    is an ordinary tile."""
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
