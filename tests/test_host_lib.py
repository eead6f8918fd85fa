"""Host half of libleech against the oracle (no GPU needed).

The library's codebook, decoded fields and layout expansion are checked
against the oracle and the seeded generator: class tables entry for entry,
fields bit for bit, and every layout's host decode back to the drawn points.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2609_02652_amd as P
from paper_2609_02652_amd import _lib, synth
from oracle import decode as D
from oracle import lattice as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def cb():
    return P.Codebook(12)


def test_library_exports_every_declared_symbol():
    with open(os.path.join(ROOT, "include", "leech.h")) as f:
        text = f.read()
    declared = set(re.findall(r"^\s*(?:const char\*|int|void)\s+(leech_\w+)\s*\(", text, re.M))
    assert declared == set(_lib.EXPORTS)
    lib = ctypes.CDLL(_lib.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name


def test_codebook_matches_oracle(cb):
    info = cb.info()
    assert info == {"n_classes": 301, "n_points": L.ball_size(), "index_bits": 47}
    for c in L.ball_classes():
        got = cb.class_info(c.class_id)
        assert got == {"shell": c.shell, "parity": c.parity, "n_levels": c.n_levels,
                       "levels": c.levels, "size": c.size}, c.class_id
    assert P.Codebook(13).info()["n_points"] == L.ball_size(13)


def test_class_level_table_bit_exact(cb):
    raw = cb.table(_lib.TABLE_CLASS_LEVELS)
    assert raw.size == 512 * 24
    rec = raw.reshape(512, 24)
    levels = rec[:, :20].copy().view(np.float32).reshape(512, 5)
    counts = rec[:, 20:].copy().view(np.uint32).ravel()
    want = L.level_table_f32()
    assert (levels[:301].view(np.uint32) == want.view(np.uint32)).all()
    assert (levels[301:] == 0).all() and (counts[301:] == 0).all()
    assert list(counts[:301]) == [c.n_levels for c in L.ball_classes()]


def test_codeword_table(cb):
    cw = cb.table(_lib.TABLE_CODEWORDS).view(np.uint32)
    assert list(cw) == list(L.golay_codewords())
    # the generator table: entry (m & 63) ^ entry 64 + (m >> 6) over all 4096
    # messages gives every codeword once
    gen = cb.table(_lib.TABLE_GOLAY_GEN).view(np.uint32)
    assert gen.size == 128
    words = sorted(int(gen[m & 63] ^ gen[64 + (m >> 6)]) for m in range(4096))
    assert words == sorted(L.golay_codewords())


def test_fields_match_oracle(cb):
    z = synth.sample_ball_points(synth.rng_for(1, "host-fields"), 20000)
    c1, s1, l1 = cb.fields_from_points(z)
    c2, s2, l2 = D.fields_from_points(z)
    assert (c1 == c2).all() and (s1 == s2).all() and (l1 == l2).all()


def test_fields_reject_non_points(cb):
    z = synth.sample_ball_points(synth.rng_for(2, "host-reject"), 10)
    bad = z.copy()
    bad[4, 0] = -bad[4, 0] if bad[4, 0] % 2 else bad[4, 0] + 2   # break membership
    with pytest.raises(P.LeechError) as e:
        cb.fields_from_points(bad)
    assert e.value.code == -5 and "block 4" in str(e.value)
    big = np.zeros((1, 24), np.int8)
    big[0, 0] = 16                                                 # outside the ball
    with pytest.raises(P.LeechError):
        cb.fields_from_points(big)


SHAPES = [(1, 24), (3, 48), (64, 24 * 5), (100, 500), (65, 24 * 17), (768, 1536), (1000, 96)]


@pytest.mark.parametrize("layout", list(P.LAYOUTS))
@pytest.mark.parametrize("M,K", SHAPES)
def test_expand_round_trip(cb, layout, M, K):
    inp = synth.make_gemv_inputs(M, K, seed=M * 131 + K, name=f"rt{M}x{K}")
    cls, sm, lv = cb.fields_from_points(inp.z)
    d, main, s0, s1 = P.expand_layout(cb, P.LAYOUTS[layout], cls, inp.gain, sm, lv)
    assert d.M == M and d.Kpad == inp.Kpad and d.nb == inp.nb
    z, c, g = P.host_decode_layout(cb, d, main, s0, s1)
    assert (z == inp.z).all() and (c == cls).all() and (g == inp.gain).all()
    # storage order of scales is a permutation of the row-major scales
    sc = P.layout_scales(d, inp.scale)
    assert sorted(sc.view(np.uint16).tolist()) == sorted(inp.scale.view(np.uint16).ravel().tolist())


def test_record_sizes_and_exceptions(cb):
    inp = synth.make_gemv_inputs(256, 24 * 40, seed=4, name="sizes")
    cls, sm, lv = cb.fields_from_points(inp.z)
    n = 256 * 40
    nlev = np.array([c.n_levels for c in L.ball_classes()])[cls.astype(int)]
    five = int((nlev == 5).sum())
    d14 = P.expand_layout(cb, P.PLANES14, cls, inp.gain, sm, lv)[0]
    assert d14.main_bytes == 14 * n + 16 and d14.side_bytes[0] == d14.side_bytes[1] == 0
    assert d14.served_bytes == d14.main_bytes + 2 * n
    d12 = P.expand_layout(cb, P.PLANES12X, cls, inp.gain, sm, lv)[0]
    assert d12.n_exceptions == five
    assert d12.main_bytes == 12 * n + 16 and d12.side_bytes[0] == 16 * five + 16
    assert d12.side_bytes[1] == 4 * -(-256 // d12.tile_rows)
    ds = P.expand_layout(cb, P.SLOT32, cls, inp.gain, sm, lv)[0]
    assert ds.main_bytes == 16 * n + 4 * five + 16
    dg = P.expand_layout(cb, P.GOLAY70, cls, inp.gain, sm, lv)[0]
    assert dg.main_bytes == 9 * n + 16 and dg.side_bytes[0] == 16 * dg.n_exceptions + 16
    assert dg.side_bytes[1] == 4 * -(-256 // dg.tile_rows)
    assert d12.tile_exc_max >= -(-five // -(-256 // d12.tile_rows)) and dg.tile_exc_max > 0
    assert 0 < dg.n_exceptions < 0.08 * n


def _fields(cb, M=8, K=96, seed=5):
    inp = synth.make_gemv_inputs(M, K, seed=seed, name="bad")
    cls, sm, lv = cb.fields_from_points(inp.z)
    return inp, cls.copy(), sm.copy(), lv.copy()


@pytest.mark.parametrize("what,code", [("class", -4), ("level", -4), ("zero_sign", -4),
                                       ("multiset", -4), ("gain", -4), ("high_sign", -4),
                                       ("lattice", -5)])
def test_expand_rejects_bad_fields(cb, what, code):
    inp, cls, sm, lv = _fields(cb)
    classes = L.ball_classes()
    b = (2, 3)
    if what == "class":
        cls[b] = 301
    elif what == "level":
        lv[b][0] = classes[int(cls[b])].n_levels
    elif what == "zero_sign":
        rc = next((r, j) for r in range(8) for j in range(4) if classes[int(cls[r, j])].levels[0] == 0)
        i = int(np.nonzero(lv[rc] == 0)[0][0])
        sm[rc] |= np.uint32(1 << i)
        b = rc
    elif what == "multiset":
        rc = next((r, j) for r in range(8) for j in range(4) if classes[int(cls[r, j])].n_levels > 1)
        i = int(np.argmin(lv[rc]))
        lv[rc][i] += 1
        sm[rc] &= np.uint32(~(1 << i) & 0xFFFFFF)
        b = rc
    elif what == "gain":
        inp.gain[b] = 2
    elif what == "high_sign":
        sm[b] |= np.uint32(1 << 30)
    elif what == "lattice":
        # flip one sign of an odd block: same multiset, not a lattice point
        rc = next((r, j) for r in range(8) for j in range(4) if classes[int(cls[r, j])].parity == 1)
        sm[rc] ^= np.uint32(1)
        b = rc
    for layout in P.LAYOUTS.values():
        with pytest.raises(P.LeechError) as e:
            P.expand_layout(cb, layout, cls, inp.gain, sm, lv)
        assert e.value.code == code
        assert f"row {b[0]}, column block {b[1]}" in str(e.value)


def test_expand_rejects_bad_shapes(cb):
    inp, cls, sm, lv = _fields(cb)
    import ctypes as C
    d = P.LayoutDesc()
    args = [_lib._ptr(np.ascontiguousarray(a)) for a in (cls, inp.gain, sm, lv)]
    rc = _lib.lib.leech_expand_layout(cb.handle, P.PLANES14, 8, 100, *args, None, None, None, C.byref(d))
    assert rc == -3
    rc = _lib.lib.leech_expand_layout(cb.handle, 7, 8, 96, *args, None, None, None, C.byref(d))
    assert rc == -2
    assert "unknown layout" in _lib.lib.leech_last_error().decode()
    rc = _lib.lib.leech_expand_layout(cb.handle, P.PLANES14, 0, 96, *args, None, None, None, C.byref(d))
    assert rc == -3


def test_device_calls_validate_before_launch():
    """Argument checks run on the host; no GPU is touched when they fail."""
    d = P.LayoutDesc()
    d.layout, d.lane_cols, d.M, d.Kpad, d.nb = P.PLANES14, 16, 8, 100, 4
    with pytest.raises(P.LeechError) as e:
        _lib.noweights_ctrl(d, 16, 16)
    assert e.value.code == -3
    with pytest.raises(P.LeechError) as e:
        _lib.fp16_gemv_ref(4, 12, 16, 16, 16)
    assert e.value.code == -3
    with pytest.raises(P.LeechError) as e:
        _lib.fp16_gemv_ref(4, 16, 0, 16, 16)
    assert e.value.code == -1


def test_grouped_gemv_validates_groups_before_launch():
    """Row groups are checked on the host; every case here fails before any
    launch (the device pointers are stand-ins that are never dereferenced)."""
    d = P.LayoutDesc()
    d.layout, d.M, d.Kpad, d.nb = P.PLANES14, 128, 48, 2
    d.lane_cols, d.tile_rows = 16, 4     # what the library picks for M = 128
    fake = 256
    cases = [
        ([], [], -1),                                 # no group
        ([16] * 8 + [0], [(1, 1)] * 9, -1),           # more than 8 groups
        ([64, 32], [(1, 1), (1, 1)], -3),             # rows do not sum to M
        ([2, 1, 125], [(1, 1)] * 3, -3),              # tile 0 would hold three groups
        ([65, 1, 62], [(1, 1)] * 3, -3),              # so would tile 16
        ([64, 64], [(1, float("nan")), (1, 1)], -1),  # non-finite centroid
        ([64, 0, 64], [(1, 1)] * 3, -3),              # empty group
    ]
    for rows, cens, code in cases:
        with pytest.raises(P.LeechError) as e:
            _lib.gemv_grouped(d, fake, 0, 0, fake, 0, fake, rows, cens, fake, fake)
        assert e.value.code == code, (rows, cens, _lib.lib.leech_last_error())


def test_batch_gemv_validates_before_launch():
    """Batch arguments are checked on the host before any launch (stand-in
    device pointers, never dereferenced)."""
    d = P.LayoutDesc()
    d.layout, d.M, d.Kpad, d.nb = P.PLANES14, 128, 48, 2
    d.lane_cols, d.tile_rows = 16, 4
    fake = 256
    cases = [
        (P.PLANES14, 0, 48, 128, -1),       # empty batch
        (P.PLANES14, 2, 40, 128, -1),       # ldx below Kpad
        (P.PLANES14, 2, 52, 128, -1),       # ldx not a multiple of 8
        (P.PLANES14, 2, 48, 100, -1),       # ldy below M
        (P.GOLAY70, 2, 48, 128, -2),        # batched launches serve Planes14
    ]
    for layout, batch, ldx, ldy, code in cases:
        d.layout = layout
        with pytest.raises(P.LeechError) as e:
            _lib.gemv_batch(d, fake, 0, 0, fake, fake, fake, (1, 1), batch, fake, ldx, fake, ldy)
        assert e.value.code == code, (layout, batch, ldx, ldy, _lib.lib.leech_last_error())


def test_rotated_gemv_validates_before_launch():
    d = P.LayoutDesc()
    d.layout, d.M, d.Kpad, d.nb = P.PLANES14, 128, 48, 2
    d.lane_cols, d.tile_rows = 16, 4
    fake = 256
    cases = [
        (P.PLANES14, 0, -3),          # K = 0
        (P.PLANES14, 72, -3),         # K above Kpad
        (P.PLANES14, 44, -3),         # K not a multiple of 8
        (P.GOLAY70, 48, -2),          # rotated launches serve Planes14
    ]
    for layout, K, code in cases:
        d.layout = layout
        with pytest.raises(P.LeechError) as e:
            _lib.gemv_rotated(d, fake, 0, 0, fake, fake, fake, [128], [(1, 1)], K, fake, 0, fake)
        assert e.value.code == code, (layout, K, _lib.lib.leech_last_error())
    d.layout, d.M, d.Kpad, d.nb = P.PLANES14, 8, 24 * 1000, 1000
    with pytest.raises(P.LeechError) as e:        # K above 40 × 512 threads
        _lib.gemv_rotated(d, fake, 0, 0, fake, fake, fake, [8], [(1, 1)], 24 * 1000, fake, 0, fake)
    assert e.value.code == -3


def test_phase_launch_validates_before_launch():
    """leech_gemv_phases serves Planes14 only and needs its stamp buffer; both
    are checked on the host (stand-in device pointers, never dereferenced)."""
    d = P.LayoutDesc()
    d.layout, d.M, d.Kpad, d.nb = P.GOLAY70, 128, 48, 2
    d.lane_cols, d.tile_rows = 16, 4
    fake = 256
    with pytest.raises(P.LeechError) as e:
        _lib.gemv_phases(d, fake, fake, fake, fake, fake, fake, (1, 1), fake, fake, fake)
    assert e.value.code == -2
    d.layout = P.PLANES14
    with pytest.raises(P.LeechError) as e:
        _lib.gemv_phases(d, fake, 0, 0, fake, 0, fake, (1, 1), fake, fake, 0)
    assert e.value.code == -1


def test_rotate_validates_before_launch():
    fake = 256
    for K, Kpad, code in ((0, 24, -3), (48, 24, -3), (65536, 65544, -3)):
        with pytest.raises(P.LeechError) as e:
            _lib.rotate_x(K, Kpad, fake, fake, fake)
        assert e.value.code == code
    with pytest.raises(P.LeechError) as e:
        _lib.rotate_x(24, 24, 0, 0, fake)
    assert e.value.code == -1


def test_geometry_fills_the_gpu():
    """The library's geometry has the least L · 5 + max(L · units per wave,
    tiles · units per tile / 1792), L = ceil(tiles / 256), plus for three to
    six rounds 1.5 · (L − tiles / 256) · units per wave; ties to more blocks per
    unit, then to more tiles; a choice of one round with 9 to 17 units per
    wave moves to two tiles per CU of at most half the units per wave (plus
    one).  5120-row projections take 256 tiles of 3 × 20 rather than 160 of
    2 × 32; 6144, 7168 and 8192 rows of 171 or 214 blocks take 4 × 16 (two
    tiles per CU); 34816 rows take 2 × 28 (a fuller last round than 2 × 32);
    the other decoder shapes full 64-block units."""
    cases = {(1, 24): (1, 64), (64, 24): (16, 4), (768, 1536): (16, 4), (1024, 4104): (16, 4),
             (4096, 4104): (4, 16), (5120, 5136): (3, 20), (5120, 17424): (3, 20),
             (6144, 4104): (4, 16), (7168, 5136): (4, 16), (8192, 8208): (2, 32),
             (8192, 4104): (4, 16), (4096, 8208): (8, 8), (10240, 5136): (3, 20),
             (14336, 4104): (1, 64), (14337, 120): (1, 64), (17408, 5136): (2, 24),
             (28672, 4104): (1, 64), (34816, 5136): (2, 28), (16384, 16392): (1, 64),
             (152064, 5136): (1, 64), (65536, 8208): (1, 64)}
    for (M, Kpad), want in cases.items():
        assert P.layout_geometry(M, Kpad) == want, (M, Kpad)
    cb_ = P.Codebook(12)
    inp = synth.make_gemv_inputs(5120, 5136, seed=0, name="geom")
    cls, sm, lv = cb_.fields_from_points(inp.z)
    d = P.expand_layout(cb_, P.PLANES14, cls, inp.gain, sm, lv)[0]
    assert (d.lane_cols, d.tile_rows) == (3, 20)
    assert (P.planes14_desc(5120, 5136).lane_cols, P.planes14_desc(5120, 5136).tile_rows) == (3, 20)


def test_geometry_is_validated(cb):
    """A caller's geometry must be one the kernels serve: lane_cols in
    {1, 2, 3, 4, 8, 16}, tile_rows a positive multiple of 4, at most 64 blocks
    per unit."""
    inp = synth.make_gemv_inputs(40, 48, seed=0, name="geomv")
    cls, sm, lv = cb.fields_from_points(inp.z)
    for geo in ((5, 4), (3, 22), (3, 24), (16, 8), (2, 0), (0, 8), (1, 68)):
        with pytest.raises(P.LeechError) as e:
            P.expand_layout(cb, P.PLANES14, cls, inp.gain, sm, lv, geometry=geo)
        assert e.value.code == -3, geo
        with pytest.raises(P.LeechError) as e:
            P.planes14_desc(40, 48, geometry=geo)
        assert e.value.code == -3, geo
    for geo in ((3, 20), (1, 64), (16, 4), (2, 12)):
        d = P.expand_layout(cb, P.PLANES14, cls, inp.gain, sm, lv, geometry=geo)[0]
        assert (d.lane_cols, d.tile_rows) == geo


def test_paper_byte_accounting(cb):
    """Record widths reproduce the paper's kernel rates on Qwen3-4B's 252
    projections (Table "layout scale", §3.2; 150,681,600 blocks and 1,105,920
    rows, §2.4), billed the paper's way: records + exception entries of 18 B
    (a 14-B record and a 4-B position) + f32 tail columns + f32 row scales."""
    inp = synth.make_gemv_inputs(4, 96, seed=0, name="acct")
    cls, sm, lv = cb.fields_from_points(inp.z)
    width = {}
    for name, lay in P.LAYOUTS.items():
        d = P.expand_layout(cb, lay, cls, inp.gain, sm, lv)[0]
        width[name] = (d.main_bytes - 16) / (4 * 4)
    assert width["planes14"] == 14 and width["planes12x"] == 12 and width["golay70"] == 9
    layer = [(4096, 2560), (1024, 2560), (1024, 2560), (2560, 4096), (9728, 2560), (9728, 2560),
             (2560, 9728)]
    blocks = 36 * sum(M * (K // 24) for M, K in layer)
    rows = 36 * sum(M for M, _ in layer)
    params = 36 * sum(M * K for M, K in layer)
    tail = 36 * sum(M * (K % 24) * 4 for M, K in layer) + rows * 4
    assert blocks == 150_681_600 and rows == 1_105_920
    exc12, exc70 = 0.0338, 0.0744          # exception rates on the paper's artifact (§3.2)
    rate = {
        "fp16": 16.0,
        "planes14": 8 * (14 * blocks + tail) / params,
        "planes12x": 8 * (12 * blocks + 18 * exc12 * blocks + tail) / params,
        "golay70": 8 * (9 * blocks + 18 * exc70 * blocks + tail) / params,
        "noweights": 8 * tail / params,
    }
    paper = {"fp16": 16.000, "planes14": 4.804, "planes12x": 4.342, "golay70": 3.589,
             "noweights": 0.159}
    for k, v in paper.items():
        assert abs(rate[k] - v) < 0.0015, (k, rate[k])
    gb = {"fp16": 2 * params, "planes14": 14 * blocks + tail}
    assert round(gb["fp16"] / 1e9, 2) == 7.27 and round(gb["planes14"] / 1e9, 2) == 2.18


def test_mode_setters_reject_unknown_values():
    """The process-wide mode setters are host code: unknown values fail with
    LEECH_E_ARG and leave the mode as it was."""
    with pytest.raises(P.LeechError):
        P.set_batch_mode(2)
    with pytest.raises(P.LeechError):
        P.set_prologue_mode(3)
    with pytest.raises(P.LeechError):
        P.set_exception_mode(5)
    P.set_batch_mode(P.BATCH_DOT2)
    P.set_batch_mode(P.BATCH_AUTO)
