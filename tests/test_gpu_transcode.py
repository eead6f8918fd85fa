"""GPU load-time transcoder (format-v1 codes -> Planes14 stream) through the C
ABI: on small shapes the codes come from the oracle's index and the stream
decodes (with the GEMV's own decoder) to the oracle's points; on every shape
the stream equals the host expansion byte for byte and its GEMV equals the
host-expanded matrix's bit for bit; invalid codes are counted."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2609_02652_amd as P  # noqa: E402
from paper_2609_02652_amd import _lib, synth  # noqa: E402
from oracle import index as I  # noqa: E402

pytestmark = pytest.mark.gpu


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


def transcode_and_compare(dev, dcb, inp, codes, oracle_rows=None):
    M, nb = inp.M, inp.nb
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    ref = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
    mat = P.LeechMatrix.from_codes(dcb, torch.from_numpy(codes.view(np.int64)).to(dev), inp.scale)
    assert mat.desc.as_dict() == ref.desc.as_dict()
    assert torch.equal(mat.main, ref.main), "transcoded stream differs from the host expansion"
    z, c, g = mat.decode()
    zc = z.cpu().numpy()
    if oracle_rows is None:
        assert np.array_equal(zc, inp.z)
    else:
        r, j = oracle_rows
        want = np.array([I.point_of_index(int(codes[a, b]) & ((1 << 47) - 1))
                         for a, b in zip(r, j)], dtype=np.int8)
        assert np.array_equal(zc[r, j], want)
    assert np.array_equal(g.cpu().numpy(), inp.gain)
    x = torch.from_numpy(inp.x).to(dev)
    y0 = ref.gemv(x, centroids=(0.75, 1.25)).cpu().numpy()
    y1 = mat.gemv(x, centroids=(0.75, 1.25)).cpu().numpy()
    assert np.array_equal(y0.view(np.uint32), y1.view(np.uint32))


@pytest.mark.parametrize("M,K", [(1, 24), (65, 408), (257, 792)])
def test_transcode_oracle_codes(dev, dcb, M, K):
    say(f"[transcode] oracle codes {M}x{K}")
    inp = synth.make_gemv_inputs(M, K, seed=M, name="transcode")
    codes = np.array([[I.code_of(I.index_of_point(inp.z[r, j]), int(inp.gain[r, j]))
                       for j in range(inp.nb)] for r in range(M)], dtype=np.uint64)
    transcode_and_compare(dev, dcb, inp, codes)


@pytest.mark.parametrize("M,K", [(14337, 120), (4096, 4096), (17408, 5120), (1024, 17408)])
def test_transcode_full_shapes(dev, dcb, M, K):
    """Tall odd-tile (lane_cols 1), the 8B q/o shape, the 14B gate/up shape
    and a wide one; codes from the host encoder, 512 blocks against the oracle."""
    say(f"[transcode] host codes {M}x{K}")
    inp = synth.make_gemv_inputs(M, K, seed=7, name="transcode-full")
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    codes = P.index_encode(dcb.cb, cls, inp.gain, sm, lv)
    rng = np.random.default_rng(M)
    rows = (rng.integers(0, M, 512), rng.integers(0, inp.nb, 512))
    transcode_and_compare(dev, dcb, inp, codes, oracle_rows=rows)


def test_invalid_codes_are_counted_and_zeroed(dev, dcb):
    inp = synth.make_gemv_inputs(65, 408, seed=9, name="transcode-bad")
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    codes = P.index_encode(dcb.cb, cls, inp.gain, sm, lv)
    N = I.class_offsets()[-1]
    planted = {(0, 0): 1 << 48, (10, 5): N, (64, 16): (1 << 47) - 1}
    for (r, j), v in planted.items():
        codes[r, j] = v
    with pytest.raises(P.LeechError, match="3 of"):
        P.LeechMatrix.from_codes(dcb, torch.from_numpy(codes.view(np.int64)).to(dev), inp.scale)
    desc = P.planes14_desc(65, 408)
    d_codes = torch.from_numpy(codes.view(np.int64)).to(dev)
    main = torch.full((desc.main_bytes,), 0xAB, dtype=torch.uint8, device=dev)
    bad = torch.full((1,), 77, dtype=torch.int32, device=dev)
    _lib.transcode_planes14(desc, dcb.index.data_ptr(), d_codes.data_ptr(), main.data_ptr(),
                            bad.data_ptr())
    torch.cuda.synchronize()
    assert int(bad.item()) == 3
    ref = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
    got, want = main.cpu().numpy(), ref.main.cpu().numpy()
    geo_index = host_storage_index(desc)
    for (r, j) in planted:
        s = geo_index(r, j)
        assert np.all(got[14 * s:14 * s + 14] == 0)
        want[14 * s:14 * s + 14] = 0
    assert np.array_equal(got, want)


def host_storage_index(desc):
    """Storage slot of block (r, j) in the wave-tile order (rows grouped in
    tiles of tile_rows, units of lane_cols columns, stored row by row)."""
    C = desc.lane_cols
    R = desc.tile_rows
    M, nb = desc.M, desc.nb

    def index(r, j):
        t, g = r // R, j // C
        rows = min(R, M - t * R)
        cols = min(C, nb - g * C)
        return t * R * nb + g * rows * C + (r % R) * cols + (j % C)
    return index
