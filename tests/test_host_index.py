"""Host format-v1 encode/decode (libleech, C++) against the oracle's index
(reading R19): codes of drawn points equal the oracle's indices bit for bit,
decoding the oracle's codes gives the oracle's points, boundaries of every
class, error paths, and the Planes14 descriptor without fields."""
import numpy as np
import pytest

import paper_2609_02652_amd as P
from oracle import decode as D
from oracle import index as I
from oracle import lattice as L
from paper_2609_02652_amd import _lib, synth

N = 111_043_117_458_000


@pytest.fixture(scope="module")
def cb():
    return P.Codebook(12)


def test_index_table_size(cb):
    t = cb.table(_lib.TABLE_INDEX)
    assert t.size == 16 + 512 * 48 + 2 * 4096 * 4 + 32 * 4 + 25 * 32 * 4
    assert int(t[:8].view(np.uint64)[0]) == N


def test_encode_matches_oracle(cb):
    z = synth.sample_ball_points(synth.rng_for(21, "host-index"), 3000)
    gain = synth.rng_for(21, "host-index-gain").integers(0, 2, 3000).astype(np.uint8)
    cls, sm, lv = cb.fields_from_points(z)
    code = P.index_encode(cb, cls, gain, sm, lv)
    want = np.array([I.code_of(I.index_of_point(x), int(g)) for x, g in zip(z, gain)],
                    dtype=np.uint64)
    assert np.array_equal(code, want)


def test_decode_matches_oracle(cb):
    rng = np.random.default_rng(22)
    idx = [int(v) for v in rng.integers(0, N, 3000, dtype=np.int64)]
    gain = rng.integers(0, 2, len(idx))
    code = np.array([I.code_of(i, int(g)) for i, g in zip(idx, gain)], dtype=np.uint64)
    cls, g, sm, lv = P.index_decode(cb, code)
    assert np.array_equal(g, gain.astype(np.uint8))
    z = D.decode_fields(cls, sm, lv)
    want = np.array([I.point_of_index(i) for i in idx], dtype=np.int64)
    assert np.array_equal(z.astype(np.int64), want)


def test_class_boundaries(cb):
    offs = I.class_offsets()
    idx = [o for c in range(301) for o in (offs[c], offs[c + 1] - 1)]
    cls, g, sm, lv = P.index_decode(cb, np.array(idx, dtype=np.uint64))
    z = D.decode_fields(cls, sm, lv)
    for i, x in zip(idx, z):
        assert list(map(int, x)) == I.point_of_index(i)
    assert np.array_equal(cls, np.repeat(np.arange(301), 2))


def test_round_trip_many(cb):
    z = synth.sample_ball_points(synth.rng_for(23, "host-index-rt"), 200_000)
    gain = (np.arange(len(z)) % 2).astype(np.uint8)
    cls, sm, lv = cb.fields_from_points(z)
    code = P.index_encode(cb, cls, gain, sm, lv)
    assert code.max() < 1 << 48 and (code & ((1 << 47) - 1)).max() < N
    c2, g2, s2, l2 = P.index_decode(cb, code)
    assert np.array_equal(c2, cls) and np.array_equal(g2, gain)
    assert np.array_equal(s2, sm) and np.array_equal(l2, lv)
    assert len(np.unique(code & np.uint64((1 << 47) - 1))) == len(np.unique(z, axis=0))


def test_decode_rejects_non_codes(cb):
    for bad in (1 << 48, N, (1 << 47) - 1, N | 1 << 47):
        with pytest.raises(P.LeechError, match="LEECH_E_FIELD"):
            P.index_decode(cb, np.array([0, bad], dtype=np.uint64))


def test_encode_rejects_bad_fields(cb):
    z = synth.sample_ball_points(synth.rng_for(24, "host-index-bad"), 4)
    cls, sm, lv = cb.fields_from_points(z)
    gain = np.zeros(4, np.uint8)
    bad_sm = sm.copy()
    bad_sm[2] ^= 1 << 30
    with pytest.raises(P.LeechError, match="block 2"):
        P.index_encode(cb, cls, gain, bad_sm, lv)
    bad_g = gain.copy()
    bad_g[1] = 2
    with pytest.raises(P.LeechError, match="block 1"):
        P.index_encode(cb, cls, bad_g, sm, lv)


def test_no_index_for_balls_past_2_47():
    big = P.Codebook(13)
    assert big.info()["n_points"] > 1 << 47
    with pytest.raises(P.LeechError):
        big.table(_lib.TABLE_INDEX)


@pytest.mark.parametrize("M,K", [(1, 24), (65, 408), (257, 792), (14337, 120), (4096, 4104)])
def test_planes14_desc_matches_expansion(cb, M, K):
    d = P.planes14_desc(M, K)
    if M * K > 2_000_000:
        assert d.main_bytes == M * (K // 24) * 14 + 16 and d.layout == P.PLANES14
        return
    inp = synth.make_gemv_inputs(M, K, seed=3, name="desc")
    cls, sm, lv = cb.fields_from_points(inp.z)
    e, _, _, _ = P.expand_layout(cb, P.PLANES14, cls, inp.gain, sm, lv)
    assert d.as_dict() == e.as_dict()


def test_planes14_desc_rejects_bad_shape():
    with pytest.raises(P.LeechError, match="LEECH_E_SHAPE"):
        P.planes14_desc(4, 25)
