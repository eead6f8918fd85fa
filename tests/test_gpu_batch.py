"""Batched GEMV (Planes14) through the C ABI.  With v_dot2 products
(BATCH_DOT2) every output vector is bit-identical to the single GEMV of its
activation; with the matrix-core products (BATCH_AUTO, every geometry) each
vector is within tolerance of the oracle's f64 product and of its single
GEMV, and bit-identical whatever the batch size and its position in the
batch.  Batches not a power of two, above 16, wide K (narrower chunks), every
geometry the matrix-core path takes (ragged tiles, lanes without a column),
strided activations and outputs."""
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


def activations(K, B, seed):
    return np.stack([synth.make_activation(K, seed=seed + b, name="batch") for b in range(B)])


def oracle_check(inp, rows, X, Y, bs):
    sub = synth.GemvInputs(len(rows), inp.K, inp.Kpad, inp.nb, inp.z[rows], inp.gain[rows],
                           inp.scale[rows], inp.x, inp.seed, inp.name)
    W = D.weights64_from_points(sub.z, sub.gain, sub.scale, CEN)
    for b in bs:
        e = D.errors(Y[b][rows], D.gemv64(W, X[b]), W, X[b])
        assert e["max_norm_err"] <= 2e-3 and e["max_abs_err"] <= 1e-5, (b, e)
    return W


def sample_rows(M):
    return np.arange(M) if M <= 1024 else np.sort(np.random.default_rng(M).choice(M, 256, False))


def build(dev, dcb, M, K, seed, geometry=None):
    inp = synth.make_gemv_inputs(M, K, seed=seed, name="batch")
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    mat = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev,
                                    geometry=geometry)
    return inp, mat


def matrix_cores(mat, B):
    return B > 1


@pytest.fixture
def dot2_mode():
    P.set_batch_mode(P.BATCH_DOT2)
    yield
    P.set_batch_mode(P.BATCH_AUTO)


SHAPES = [(1, 24, 2), (65, 408, 3), (257, 792, 8), (768, 1536, 5), (4096, 4096, 11),
          (14337, 120, 4), (1024, 17408, 8), (300, 24 * 30, 1), (768, 1536, 21), (257, 792, 16)]


@pytest.mark.parametrize("M,K,B", SHAPES)
def test_dot2_batch_bit_identical_to_single(dev, dcb, dot2_mode, M, K, B):
    say(f"[batch dot2] {M}x{K} B={B}")
    inp, mat = build(dev, dcb, M, K, M + B)
    X = activations(K, B, seed=K)
    Xd = torch.from_numpy(X).to(dev)
    Y = mat.gemv_batch(Xd, centroids=CEN).cpu().numpy()
    for b in range(B):
        y1 = mat.gemv(Xd[b].contiguous(), centroids=CEN).cpu().numpy()
        assert np.array_equal(Y[b].view(np.uint32), y1.view(np.uint32)), f"vector {b}"
    oracle_check(inp, sample_rows(M), X, Y, (0, B - 1))


def check_auto(dev, mat, inp, X, Y):
    """Y from BATCH_AUTO: bit-identical to single GEMVs where the products are
    v_dot2; on the matrix cores within tolerance of the oracle and, row by
    row, within 2^-15 · Σ|w x| of the single GEMV.  The bound: a block's
    24-product dot of the decoded (subnormal) weights with an N(0,1) binary16
    activation errs by at most 119 (v_dot2) and 155 (matrix core) units of
    2^-24 · Σ|h x| over 512,000 measured dot products, so two paths differ by
    under 2^-15 · Σ|h x| a block; the blocks' f32 accumulation adds a few
    more units."""
    B = X.shape[0]
    Xd = torch.from_numpy(X).to(dev)
    rows = sample_rows(inp.M)
    if not matrix_cores(mat, B):
        for b in range(B):
            y1 = mat.gemv(Xd[b].contiguous(), centroids=CEN).cpu().numpy()
            assert np.array_equal(Y[b].view(np.uint32), y1.view(np.uint32)), f"vector {b}"
        oracle_check(inp, rows, X, Y, (0, B - 1))
        return
    W = oracle_check(inp, rows, X, Y, range(B))
    for b in (0, B - 1):
        y1 = mat.gemv(Xd[b].contiguous(), centroids=CEN).cpu().numpy()
        bound = 2.0 ** -15 * (np.abs(W) @ np.abs(X[b].astype(np.float64)))
        diff = np.abs(Y[b][rows].astype(np.float64) - y1[rows])
        assert (diff <= bound).all(), (b, float((diff / np.maximum(bound, 1e-300)).max()))


@pytest.mark.parametrize("M,K,B", SHAPES)
def test_batch_matches_oracle_and_single(dev, dcb, M, K, B):
    say(f"[batch] {M}x{K} B={B}")
    inp, mat = build(dev, dcb, M, K, M + B)
    say(f"[batch] geometry {mat.desc.lane_cols}x{mat.desc.tile_rows}, "
        f"matrix cores {matrix_cores(mat, B)}")
    X = activations(K, B, seed=K)
    Y = mat.gemv_batch(torch.from_numpy(X).to(dev), centroids=CEN).cpu().numpy()
    check_auto(dev, mat, inp, X, Y)


# lane placements of the matrix-core path: every lane_cols (1, 2, 3, 4, 8, 16),
# tile_rows from 4 to 64, lanes past the last column (R · C < 64), ragged last
# tiles (rows of a 4-lane block partly past the matrix) and last column groups
MX_GEOMETRIES = [((1, 64), 1000, 24 * 37), ((2, 32), 777, 24 * 41), ((4, 16), 301, 24 * 43),
                 ((3, 16), 333, 24 * 29), ((1, 16), 70, 24 * 11), ((1, 48), 100, 24 * 7),
                 ((2, 16), 50, 24 * 9), ((1, 32), 33, 24), ((4, 16), 4096, 4104),
                 ((2, 28), 1000, 24 * 45), ((2, 24), 301, 24 * 50), ((1, 20), 333, 24 * 13),
                 ((4, 12), 100, 24 * 23), ((1, 60), 777, 24 * 17), ((3, 12), 200, 24 * 31),
                 ((4, 4), 37, 24 * 9), ((3, 20), 301, 24 * 50), ((8, 8), 100, 24 * 37),
                 ((16, 4), 30, 24 * 70), ((8, 4), 66, 24 * 20), ((3, 20), 5120, 5136)]


@pytest.mark.parametrize("geo,M,K", MX_GEOMETRIES)
def test_matrix_core_geometries(dev, dcb, geo, M, K):
    inp, mat = build(dev, dcb, M, K, M + K, geometry=geo)
    assert (mat.desc.lane_cols, mat.desc.tile_rows) == geo
    for B in (2, 3, 5, 16, 17):
        say(f"[batch mx] {geo} {M}x{K} B={B}")
        X = activations(K, B, seed=K + B)
        Y = mat.gemv_batch(torch.from_numpy(X).to(dev), centroids=CEN).cpu().numpy()
        check_auto(dev, mat, inp, X, Y)


@pytest.mark.parametrize("geo,M,K", [((4, 16), 301, 24 * 43), ((2, 32), 777, 24 * 41),
                                     ((1, 64), 1000, 24 * 37), ((2, 28), 1000, 24 * 45),
                                     ((3, 20), 301, 24 * 50), ((8, 8), 100, 24 * 37)])
def test_matrix_core_bits_independent_of_batch(dev, dcb, geo, M, K):
    """One activation's y is the same bits alone in a 2-wide launch, in
    every position of 4-, 8- and 16-wide launches and in a trailing chunk."""
    inp, mat = build(dev, dcb, M, K, 3 * M + K, geometry=geo)
    X = activations(K, 17, seed=K)
    Xd = torch.from_numpy(X).to(dev)
    ref = mat.gemv_batch(Xd[:2], centroids=CEN).cpu().numpy()
    for B in (3, 4, 8, 16, 17):
        say(f"[batch bits] {geo} B={B}")
        Y = mat.gemv_batch(Xd[:B], centroids=CEN).cpu().numpy()
        assert np.array_equal(Y[:2].view(np.uint32), ref.view(np.uint32)), B
    full = mat.gemv_batch(Xd, centroids=CEN).cpu().numpy()
    for shift in (1, 5, 13, 16):
        say(f"[batch bits] {geo} shift {shift}")
        Y = mat.gemv_batch(torch.roll(Xd, shift, 0).contiguous(), centroids=CEN).cpu().numpy()
        assert np.array_equal(Y.view(np.uint32), np.roll(full, shift, 0).view(np.uint32)), shift


def test_batch_mode_rejects_unknown(dev):
    with pytest.raises(P.LeechError):
        P.set_batch_mode(7)
    P.set_batch_mode(P.BATCH_AUTO)


def test_strided_activations_and_outputs(dev, dcb):
    M, K, B = 257, 792, 6
    inp = synth.make_gemv_inputs(M, K, seed=5, name="batch-stride")
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    mat = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
    X = activations(K, B, seed=9)
    big = torch.zeros((B, inp.Kpad + 40), dtype=torch.float16, device=dev)
    big[:, :inp.Kpad] = torch.from_numpy(X).to(dev)
    Ybig = torch.full((B, M + 3), 123.0, dtype=torch.float32, device=dev)
    mat.gemv_batch(big[:, :inp.Kpad], Ybig[:, :M], centroids=CEN)
    Yc = mat.gemv_batch(torch.from_numpy(X).to(dev), centroids=CEN)
    assert torch.equal(Ybig[:, :M], Yc)
    assert torch.all(Ybig[:, M:] == 123.0)
