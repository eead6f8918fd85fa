"""GPU parity of the activation rotation against the oracle (reading R17),
through the C ABI, and the rotation feeding the GEMV."""
import math
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2609_02652_amd as P  # noqa: E402
from paper_2609_02652_amd import synth  # noqa: E402
from oracle import decode as D  # noqa: E402
from oracle import rotation as R  # noqa: E402

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch.device("cuda:0")


def check_rotation(dev, K, Kpad, offset=0):
    """Rotate through the C ABI and compare with the oracle.  offset > 0 hands
    the kernel x, signs and both outputs as views `offset` elements into larger
    buffers, so no pointer is 16-byte aligned (the element-wise path)."""
    say(f"[rotate] K={K} Kpad={Kpad} offset={offset}")
    x = synth.make_activation(K, seed=K, name="rot")[:K]
    s = synth.make_signs(K, seed=K, name="rot")
    xt = torch.zeros(K + offset, dtype=torch.float16, device=dev)
    st = torch.ones(K + offset, dtype=torch.int8, device=dev)
    xt[offset:] = torch.from_numpy(x).to(dev)
    st[offset:] = torch.from_numpy(s).to(dev)
    o16 = torch.full((Kpad + offset,), 7.0, dtype=torch.float16, device=dev)[offset:]
    o32 = torch.empty(K + offset, dtype=torch.float32, device=dev)[offset:]
    P._lib.rotate_x(K, Kpad, xt[offset:].data_ptr(), st[offset:].data_ptr(), o16.data_ptr(),
                    o32.data_ptr())
    torch.cuda.synchronize()
    y16 = o16.cpu().numpy()
    y32 = o32.cpu().numpy().astype(np.float64)
    n = R.pow2_block(K)
    k = int(math.log2(n))
    # f32 butterflies: k stages, each error ≤ 2^-24 · |partial| ≤ 2^-24 · 2^t · max|x|,
    # reaching every output through 2^(k-t) paths; then one rounding of the scale
    bound = (k * 2 ** (k / 2) + 1) * 2.0 ** -24 * np.max(np.abs(x.astype(np.float64)))
    if n <= 4096:
        idx = np.arange(K)
        y64 = R.rotate64(x, s)
    else:       # long blocks: 1024 sampled outputs, each from its own row of H_n
        idx = np.sort(np.random.default_rng(K).choice(K, 1024, replace=False))
        y64 = R.rotate64_at(x, s, idx)
    err = np.max(np.abs(y32[idx] - y64))
    say(f"    max |f32 - f64| = {err:.3e} over {idx.size} outputs (bound {bound:.3e})")
    assert err <= bound
    # every output: the rotation is orthogonal, so the norm is kept
    xn = np.linalg.norm(x.astype(np.float64))
    assert abs(np.linalg.norm(y32) - xn) <= bound * math.sqrt(K)
    # the binary16 output is the f32 value rounded to nearest even, zero past K
    assert np.array_equal(y16[:K].view(np.uint16), y32.astype(np.float32).astype(np.float16).view(np.uint16))
    assert np.all(y16[K:] == 0)


# block lengths 2^0 .. 2^15: K = 1, 6, 12 take the blocks shorter than one
# thread's eight coordinates; 24576 and 49152 the 8192- and 16384-point blocks
ROT_KS = [1, 6, 12, 24, 44, 1000, 4096, 5120, 14336, 17408, 24576, 49152, 32768]


@pytest.mark.parametrize("K", ROT_KS)
def test_rotation_matches_oracle(dev, K):
    check_rotation(dev, K, synth.padded_k(K))


@pytest.mark.parametrize("K,Kpad", [(7, 13), (4096, 4101), (14336, 14343), (5120, 5120)])
def test_rotation_unaligned_and_odd_padding(dev, K, Kpad):
    check_rotation(dev, K, Kpad, offset=1)


def test_rotation_without_signs_is_plain_walsh(dev):
    K = 256
    x = synth.make_activation(K, seed=5, name="plain")[:K]
    out = P.rotate_x(torch.from_numpy(x).to(dev), None, K, with_f32=True)[1].cpu().numpy()
    assert np.max(np.abs(out - R.rotate64(x, np.ones(K)))) <= 1e-5 * np.max(np.abs(x))


def test_rotation_feeds_gemv(dev):
    """x -> rotation -> GEMV: y equals the oracle's W·(rotated x), with the GEMV
    fed the rotation's binary16 output."""
    M, K = 768, 1536
    inp = synth.make_gemv_inputs(M, K, seed=3, name="rot-gemv")
    s = synth.make_signs(K, seed=3, name="rot-gemv")
    cb = P.Codebook(12)
    dcb = P.DeviceCodebook(cb, dev)
    cls, sm, lv = cb.fields_from_points(inp.z)
    mat = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
    xr = P.rotate_x(torch.from_numpy(inp.x[:K]).to(dev), torch.from_numpy(s).to(dev), inp.Kpad)
    y = mat.gemv(xr).cpu().numpy()
    xr_h = xr.cpu().numpy()
    assert np.max(np.abs(xr_h[:K].astype(np.float64) - R.rotate64(inp.x[:K], s))) <= \
        2.0 ** -10 * np.max(np.abs(R.rotate64(inp.x[:K], s)))
    W = D.weights64_from_points(inp.z, inp.gain, inp.scale, (1.0, 1.0))
    e = D.errors(y, D.gemv64(W, xr_h), W, xr_h)
    say(f"    rotated GEMV errors {e}")
    assert e["max_norm_err"] <= 2e-3 and e["max_abs_err"] <= 1e-5


# ------------------------------------------------ rotation fused into the GEMV
# k = log2 of the largest power of two dividing K: 9, 12, 11, 10, 3, 3, 3, then
# one case for each other k the fused path admits (4..8, 13, 14), since each
# k has its own schedule of LDS passes
FUSED = [(768, 1536, True), (4096, 4096, True), (1024, 14336, True), (5120, 17408, True),
         (64, 408, True), (3, 24, False), (257, 1000, False),
         (256, 48, True), (256, 96, True), (256, 320, True), (256, 384, True), (200, 768, True),
         (512, 8192, True), (256, 16384, True)]


@pytest.mark.parametrize("M,K,with_signs", FUSED)
def test_fused_rotation_equals_rotate_then_gemv(dev, M, K, with_signs):
    """leech_gemv_rotated gives the bits of leech_rotate_x followed by the GEMV."""
    say(f"[fused rotation] {M}x{K} signs={with_signs}")
    inp = synth.make_gemv_inputs(M, K, seed=M + K, name="fused-rot")
    cb = P.Codebook(12)
    dcb = P.DeviceCodebook(cb, dev)
    cls, sm, lv = cb.fields_from_points(inp.z)
    mat = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
    x = torch.from_numpy(inp.x[:K].copy()).to(dev)
    s = torch.from_numpy(synth.make_signs(K, seed=K, name="fused-rot")).to(dev) if with_signs else None
    cen = (0.75, 1.25)
    y_fused = mat.gemv_rotated(x, s, group_centroids=(cen,)).cpu().numpy()
    xr = P.rotate_x(x, s, inp.Kpad)
    y_two = mat.gemv(xr, centroids=cen).cpu().numpy()
    assert np.array_equal(y_fused.view(np.uint32), y_two.view(np.uint32))
    # and against the oracle: W · R(x) with R from the oracle's rotation
    if M <= 1024:
        xr64 = R.rotate_padded64(inp.x[:K], s.cpu().numpy() if with_signs else np.ones(K), inp.Kpad)
        xr16 = xr64.astype(np.float16)
        W = D.weights64_from_points(inp.z, inp.gain, inp.scale, cen)
        e = D.errors(y_fused, D.gemv64(W, xr16), W, xr16)
        assert e["max_norm_err"] <= 2e-3, e


def test_fused_rotation_grouped(dev):
    """q/k/v fused and rotated in one launch, bit-identical to rotate + grouped."""
    parts = [(256, 1536), (64, 1536), (64, 1536)]
    ins = [synth.make_gemv_inputs(M, K, seed=40 + i, name=f"frg{i}") for i, (M, K) in enumerate(parts)]
    z = np.concatenate([i.z for i in ins])
    gain = np.concatenate([i.gain for i in ins])
    scale = np.concatenate([i.scale for i in ins])
    cb = P.Codebook(12)
    dcb = P.DeviceCodebook(cb, dev)
    cls, sm, lv = cb.fields_from_points(z)
    mat = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, gain, sm, lv, scale, dev)
    K = 1536
    x = torch.from_numpy(ins[0].x[:K].copy()).to(dev)
    s = torch.from_numpy(synth.make_signs(K, seed=4, name="frg")).to(dev)
    cens = [(0.75, 1.25), (0.9, 1.1), (1.3, 0.6)]
    rows = [M for M, _ in parts]
    y1 = mat.gemv_rotated(x, s, rows, cens).cpu().numpy()
    y2 = mat.gemv_grouped(P.rotate_x(x, s, mat.Kpad), rows, cens).cpu().numpy()
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))
