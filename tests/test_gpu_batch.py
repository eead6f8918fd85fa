"""Batched GEMV (Planes14) through the C ABI: every output vector is
bit-identical to the single GEMV of its activation and within tolerance of
the oracle's f64 product; batches not a power of two, batches above 8, wide K
(narrower chunks), strided activations and outputs."""
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


@pytest.mark.parametrize("M,K,B", [(1, 24, 2), (65, 408, 3), (257, 792, 8), (768, 1536, 5),
                                   (4096, 4096, 11), (14337, 120, 4), (1024, 17408, 8),
                                   (300, 24 * 30, 1), (768, 1536, 21), (257, 792, 16)])
def test_batch_matches_single_and_oracle(dev, dcb, M, K, B):
    say(f"[batch] {M}x{K} B={B}")
    inp = synth.make_gemv_inputs(M, K, seed=M + B, name="batch")
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    mat = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
    X = activations(K, B, seed=K)
    Xd = torch.from_numpy(X).to(dev)
    Y = mat.gemv_batch(Xd, centroids=CEN).cpu().numpy()
    for b in range(B):
        y1 = mat.gemv(Xd[b].contiguous(), centroids=CEN).cpu().numpy()
        assert np.array_equal(Y[b].view(np.uint32), y1.view(np.uint32)), f"vector {b}"
    rows = np.arange(M) if M <= 1024 else np.sort(np.random.default_rng(M).choice(M, 256, False))
    sub = synth.GemvInputs(len(rows), inp.K, inp.Kpad, inp.nb, inp.z[rows], inp.gain[rows],
                           inp.scale[rows], inp.x, inp.seed, inp.name)
    W = D.weights64_from_points(sub.z, sub.gain, sub.scale, CEN)
    for b in (0, B - 1):
        e = D.errors(Y[b][rows], D.gemv64(W, X[b]), W, X[b])
        assert e["max_norm_err"] <= 2e-3 and e["max_abs_err"] <= 1e-5, (b, e)


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
