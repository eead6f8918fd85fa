"""The GEMV's prologue modes (leech_set_prologue_mode) change only the order
in which a wave requests its weight records, never the summation order: y is
bit-identical in every mode, for every layout, at shapes whose waves stream
from one unit to many (ragged row tiles and column groups included), and
within tolerance of the oracle (§2.3; §2.4's tolerance)."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2609_02652_amd as P  # noqa: E402
from paper_2609_02652_amd import synth  # noqa: E402
from oracle import decode as D  # noqa: E402

pytestmark = pytest.mark.gpu
CEN = (0.75, 1.25)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def dcb(dev):
    return P.DeviceCodebook(P.Codebook(12), dev)


# units a wave streams: 0 (one column group), 1, ~6, ~13, ~21 and ~45
SHAPES = [(3, 24), (65, 408), (257, 3000), (4096, 4096), (640, 5120), (1024, 8192),
          (300, 17408)]


@pytest.mark.parametrize("M,K", SHAPES)
def test_modes_bit_identical(dev, dcb, M, K):
    inp = synth.make_gemv_inputs(M, K, seed=M + 3 * K, name="prologue")
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    x = torch.from_numpy(inp.x).to(dev)
    rows = np.arange(M) if M <= 700 else np.random.default_rng(M).choice(M, 200, replace=False)
    W = D.weights64_from_points(inp.z[rows], inp.gain[rows], inp.scale[rows], CEN)
    y64 = D.gemv64(W, inp.x)
    ref = None
    try:
        for name, lay in P.LAYOUTS.items():
            mat = P.LeechMatrix.from_fields(dcb, lay, cls, inp.gain, sm, lv, inp.scale, dev)
            for mode in (P.PROLOGUE_AUTO, 0, 1, 2):
                print(f"[prologue] {M}x{K} layout={name} mode={mode}", flush=True)
                P.set_prologue_mode(mode)
                y = mat.gemv(x, centroids=CEN).cpu().numpy()
                if ref is None:
                    ref = y.view(np.uint32).copy()
                    e = D.errors(y[rows], y64, W, inp.x)
                    assert e["max_norm_err"] <= 2e-3 and e["max_abs_err"] <= 1e-5, e
                assert np.array_equal(y.view(np.uint32), ref), (name, mode)
            del mat
    finally:
        P.set_prologue_mode(P.PROLOGUE_AUTO)


def test_bad_mode_is_refused():
    with pytest.raises(P.LeechError):
        P.set_prologue_mode(3)
    P.set_prologue_mode(P.PROLOGUE_AUTO)
