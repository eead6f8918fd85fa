"""The phase-stamp measurement launch (leech_gemv_phases) through the C ABI:
its y is the plain GEMV's bit for bit, and every workgroup's stamps are in
order (start ≤ staging barrier passed ≤ each wave's last unit ≤ last store),
on a single-tile and a many-tile shape and both even and uneven unit bases."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2609_02652_amd as P  # noqa: E402
from paper_2609_02652_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def dcb(dev):
    return P.DeviceCodebook(P.Codebook(12), dev)


@pytest.mark.parametrize("M,K,geo", [(64, 24, None), (4096, 4096, None), (777, 1000, (1, 64)),
                                     (1030, 2400, (3, 20))])
def test_phase_stamps(dev, dcb, M, K, geo):
    inp = synth.make_gemv_inputs(M, K, seed=M + K, name="phases")
    cls, sm, lv = dcb.cb.fields_from_points(inp.z)
    mat = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev,
                                    geometry=geo)
    x = torch.from_numpy(inp.x).to(dev)
    y0 = mat.gemv(x, centroids=(0.75, 1.25)).cpu().numpy()
    tiles = -(-M // mat.desc.tile_rows)
    waves = min(8, -(-mat.desc.nb // mat.desc.lane_cols))
    st = torch.full((tiles, 11), -1, dtype=torch.int64, device=dev)
    y = torch.empty(M, dtype=torch.float32, device=dev)
    mat.gemv_phases(x, y, st, centroids=(0.75, 1.25))
    torch.cuda.synchronize()
    assert np.array_equal(y.cpu().numpy().view(np.uint32), y0.view(np.uint32))
    s = st.cpu().numpy()
    assert (s[:, :2] > 0).all() and (s[:, 2:2 + waves] > 0).all() and (s[:, 10] > 0).all()
    assert (s[:, 2 + waves:10] == -1).all()
    assert (s[:, 0] <= s[:, 1]).all()
    assert (s[:, 1][:, None] <= s[:, 2:2 + waves]).all()
    assert (s[:, 2:2 + waves].max(axis=1) <= s[:, 10]).all()
