"""GPU parity at the full workload shapes, through the C ABI, in the launch
configuration the benchmark times.

* the seven projections of one 8B-class decoder layer (K padded to a multiple
  of 24): q, o 4096×4104; k, v 1024×4104; gate, up 14336×4104; down 4096×14352;
* the seven projection shapes of the 14B-class model: q, o 5120×5136; k, v
  1024×5136; gate, up 17408×5136; down 5120×17424.

Each matrix is drawn with its own seed, served as Planes14, decoded on the GPU
and compared with the drawn points in full (bit-exact), and its GEMV is
compared with the oracle's f64 matvec on sampled rows, which the oracle
computes one by one.  These shapes take the geometries (lane_cols × tile_rows)
1 × 64, 2 × 24, 3 × 20, 4 × 16 and 16 × 4; the fused 8B launches 4 × 16 (two
tiles per CU) and 1 × 64.  A tall matrix with a one-row last
tile at 1 × 64 exercises the kernel variant whose unit bases are not
4-aligned, for every layout.
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

LAYER_8B = [("q", 4096, 4096), ("k", 1024, 4096), ("v", 1024, 4096), ("o", 4096, 4096),
            ("gate", 14336, 4096), ("up", 14336, 4096), ("down", 4096, 14336)]
MODEL_14B = [("q", 5120, 5120), ("k", 1024, 5120), ("v", 1024, 5120), ("o", 5120, 5120),
             ("gate", 17408, 5120), ("up", 17408, 5120), ("down", 5120, 17408)]


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


def check_matrix(dev, dcb, name, M, K, seed, layouts=("planes14",), rows_sampled=128,
                 geometry=None):
    inp = synth.make_gemv_inputs(M, K, seed=seed, name=name)
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    x = torch.from_numpy(inp.x).to(dev)
    rng = np.random.default_rng(seed)
    rows = np.sort(rng.choice(M, min(rows_sampled, M), replace=False))
    sub = synth.GemvInputs(len(rows), inp.K, inp.Kpad, inp.nb, inp.z[rows], inp.gain[rows],
                           inp.scale[rows], inp.x, inp.seed, inp.name)
    W = D.weights64_from_points(sub.z, sub.gain, sub.scale, CEN)
    y64 = D.gemv64(W, inp.x)
    ys = {}
    for lay in layouts:
        say(f"[workload] {name} {M}x{K} layout={lay} seed={seed}")
        mat = P.LeechMatrix.from_fields(dcb, P.LAYOUTS[lay], cls, inp.gain, sm, lv, inp.scale, dev,
                                        geometry=geometry)
        z, c, g = mat.decode()
        y = mat.gemv(x, centroids=CEN)
        torch.cuda.synchronize()
        assert torch.equal(z.cpu(), torch.from_numpy(inp.z)), f"{name}: decoded z differ"
        assert (g.cpu().numpy() == inp.gain).all()
        yh = y.cpu().numpy()
        e = D.errors(yh[rows], y64, W, inp.x)
        say(f"    geometry={mat.desc.lane_cols}x{mat.desc.tile_rows} errors {e}")
        assert e["max_norm_err"] <= TOL_NORM and e["max_abs_err"] <= TOL_PAPER, (name, lay, e)
        ys[lay] = yh
        del mat, z, c, g
        torch.cuda.empty_cache()
    ref = ys[layouts[0]].view(np.uint32)
    for lay, y in ys.items():
        assert (y.view(np.uint32) == ref).all(), f"{name}: {lay} not bit-identical"


@pytest.mark.parametrize("proj", LAYER_8B, ids=[p[0] for p in LAYER_8B])
def test_layer_8b(dev, dcb, proj):
    name, M, K = proj
    check_matrix(dev, dcb, f"8b-{name}", M, K, seed=100 + LAYER_8B.index(proj))


@pytest.mark.parametrize("proj", MODEL_14B, ids=[p[0] for p in MODEL_14B])
def test_model_14b_shapes(dev, dcb, proj):
    name, M, K = proj
    check_matrix(dev, dcb, f"14b-{name}", M, K, seed=200 + MODEL_14B.index(proj))


def test_odd_last_tile_all_layouts(dev, dcb):
    """Geometry 1 × 64 with a one-row last tile: unit bases that are not 4-aligned."""
    check_matrix(dev, dcb, "tall-odd", 14337, 24 * 5, seed=7,
                 layouts=("planes14", "slot32", "planes12x", "golay70"), rows_sampled=256,
                 geometry=(1, 64))


# ----------------------------------------------------------- fused launches
def fused_inputs(parts, seed0):
    """Row concatenation of independently drawn matrices sharing one K (and x)."""
    ins = [synth.make_gemv_inputs(M, K, seed=seed0 + i, name=f"fused{i}")
           for i, (M, K) in enumerate(parts)]
    x = ins[0].x
    cat = lambda f: np.concatenate([getattr(i, f) for i in ins], axis=0)  # noqa: E731
    return ins, cat("z"), cat("gain"), cat("scale"), x


def check_fused(dev, dcb, parts, cens, seed0, layouts, rows_per_part=None):
    ins, z, gain, scale, x = fused_inputs(parts, seed0)
    cls, sm, lv = dcb.cb.fields_from_points(z)
    xt = torch.from_numpy(x).to(dev)
    group_rows = [M for M, _ in parts]
    ref_bits = None
    for lay in layouts:
        say(f"[fused] parts={parts} layout={lay}")
        mat = P.LeechMatrix.from_fields(dcb, P.LAYOUTS[lay], cls, gain, sm, lv, scale, dev)
        y = mat.gemv_grouped(xt, group_rows, cens).cpu().numpy()
        r0 = 0
        for i, (inp, c) in enumerate(zip(ins, cens)):
            M = inp.M
            rows = np.arange(M) if rows_per_part is None else \
                np.sort(np.random.default_rng(i).choice(M, min(rows_per_part, M), replace=False))
            sub = synth.GemvInputs(len(rows), inp.K, inp.Kpad, inp.nb, inp.z[rows], inp.gain[rows],
                                   inp.scale[rows], x, inp.seed, inp.name)
            W = D.weights64_from_points(sub.z, sub.gain, sub.scale, c)
            e = D.errors(y[r0 + rows], D.gemv64(W, x), W, x)
            say(f"    group {i} ({M} rows, centroids {c}): {e}")
            assert e["max_norm_err"] <= TOL_NORM and e["max_abs_err"] <= TOL_PAPER
            r0 += M
        if ref_bits is None:
            ref_bits = y.view(np.uint32).copy()
        assert (y.view(np.uint32) == ref_bits).all(), f"{lay} not bit-identical"
        del mat
        torch.cuda.empty_cache()


def test_fused_qkv_small_all_layouts(dev, dcb):
    check_fused(dev, dcb, [(256, 408), (64, 408), (64, 408)],
                [(0.75, 1.25), (0.9, 1.1), (1.3, 0.6)], seed0=300,
                layouts=("planes14", "slot32", "planes12x", "golay70"))


def test_fused_layer_8b(dev, dcb):
    """q/k/v in one launch and gate/up in one launch, as served (Planes14)."""
    check_fused(dev, dcb, [(4096, 4096), (1024, 4096), (1024, 4096)],
                [(0.75, 1.25), (0.9, 1.1), (1.3, 0.6)], seed0=400, layouts=("planes14",),
                rows_per_part=64)
    check_fused(dev, dcb, [(14336, 4096), (14336, 4096)], [(0.8, 1.2), (1.1, 0.95)], seed0=500,
                layouts=("planes14",), rows_per_part=64)


def test_fused_single_group_matches_plain_gemv(dev, dcb):
    """One group with the plain call's centroids gives the plain call's bits."""
    inp = synth.make_gemv_inputs(768, 1536, seed=9, name="one-group")
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    mat = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
    x = torch.from_numpy(inp.x).to(dev)
    a = mat.gemv(x, centroids=CEN).cpu().numpy()
    b = mat.gemv_grouped(x, [768], [CEN]).cpu().numpy()
    assert (a.view(np.uint32) == b.view(np.uint32)).all()
