"""The table every GPU kernel reads (LEECH_TABLE_DEVICE), entry by entry,
against the oracle (no GPU needed).

Each 32-byte record of a class id holds (§2.3 "The kernel": the class table
the decode looks levels up in; §3.2 "The layout scale": Golay70's in-class
value code):

* the byte-permute table: byte 0 = 0x80 (the binary16 sign byte), byte 1 + k
  = the k-th distinct magnitude of the class in ascending order, zeros after;
* f32 of 1 / (4 √m), bit for bit (the unit-norm direction, §2.3);
* n_levels | parity << 8 | shell << 16 | Golay70 sign bits << 24;
* Golay70's signed values per (side, 2-bit code) and their magnitudes.

The Golay70 values follow reading R14: per side of the codeword (even points:
|z_i| ≡ 2 mod 4 on the codeword; odd points: z_i ≡ 3 mod 4), the four signed
values most frequent over the class's points, ties to the smaller |v| and
then to v > 0.  Their frequencies are taken two ways here: from the lattice
symmetry (a sign is uniform where flipping it, or flipping it with a partner
on the support, keeps the point in the lattice, and forced otherwise), and by
brute force over every point of eight small classes, enumerated with the
oracle's format-v1 index; the two must agree before the table is judged.
Slots 301..511 are zero.
"""
import math
from collections import Counter

import numpy as np
import pytest

import paper_2609_02652_amd as P
from paper_2609_02652_amd import _lib
from oracle import index as I
from oracle import lattice as L

SMALL_CLASSES = (0, 1, 2, 12, 34, 75, 150, 256)   # 264,688 points in all


@pytest.fixture(scope="module")
def table():
    raw = P.Codebook(12).table(_lib.TABLE_DEVICE)
    assert raw.size == 512 * 32
    return raw.reshape(512, 32)


def side_of(z_i: int, parity: int) -> int:
    """Codeword bit of a coordinate: |z| ≡ 2 (mod 4) for even points, z ≡ 3
    (mod 4) for odd points (the two congruence sets of the membership test)."""
    return int(abs(z_i) % 4 == 2) if parity == 0 else int(z_i % 4 == 3)


def symmetric_frequencies(c: L.LeechClass) -> list[Counter]:
    """Twice the expected count, per coordinate of a uniform point of the
    class, of each signed value on each side (constant factors dropped)."""
    mult = Counter(c.mags_desc)
    out = [Counter(), Counter()]
    for a, m in mult.items():
        if c.parity == 0:
            side = int(a % 4 == 2)
            if a == 0:
                out[side][0] += 2 * m
            else:                                # sign uniform: ±a half each
                out[side][a] += m
                out[side][-a] += m
        else:                                    # a uniform codeword holds each
            for v in (a, -a):                    # coordinate half the time; the
                out[side_of(v, 1)][v] += m       # sign is then forced
    return out


def brute_frequencies(c: L.LeechClass) -> list[Counter]:
    offs = I.class_offsets()
    out = [Counter(), Counter()]
    for idx in range(offs[c.class_id], offs[c.class_id + 1]):
        for v in I.point_of_index(idx):
            out[side_of(v, c.parity)][v] += 1
    return out


def top4(freq: Counter) -> list[int]:
    ranked = sorted(freq, key=lambda v: (-freq[v], abs(v), -v))
    return (ranked + [0, 0, 0, 0])[:4]


@pytest.mark.parametrize("cid", SMALL_CLASSES)
def test_golay70_frequencies_brute_force(cid):
    """The symmetry argument against every point of a small class (ratios)."""
    c = L.ball_classes()[cid]
    sym, brute = symmetric_frequencies(c), brute_frequencies(c)
    for side in (0, 1):
        assert set(sym[side]) == set(brute[side]), (cid, side)
        tot_s, tot_b = sum(sym[side].values()), sum(brute[side].values())
        for v in sym[side]:
            assert sym[side][v] * tot_b == brute[side][v] * tot_s, (cid, side, v)
        assert top4(sym[side]) == top4(brute[side])


def test_permute_table_and_norm_bit_exact(table):
    for c in L.ball_classes():
        rec = table[c.class_id]
        want = [0x80] + list(c.levels) + [0] * (7 - c.n_levels)
        assert list(rec[:8]) == want, c.class_id
        inv = rec[8:12].copy().view(np.float32)[0]
        assert inv.view(np.uint32) == np.float32(1.0 / (4.0 * math.sqrt(c.shell))).view(np.uint32)


def test_info_word(table):
    for c in L.ball_classes():
        info = int(table[c.class_id, 12:16].copy().view(np.uint32)[0])
        assert info & 0xFF == c.n_levels
        assert (info >> 8) & 0xFF == c.parity
        assert (info >> 16) & 0xFF == c.shell
        vals = table[c.class_id, 16:24].copy().view(np.int8)
        neg = sum(1 << k for k in range(8) if vals[k] < 0)
        assert info >> 24 == neg, c.class_id


def test_golay70_values(table):
    for c in L.ball_classes():
        rec = table[c.class_id]
        vals = rec[16:24].copy().view(np.int8).reshape(2, 4)
        freq = symmetric_frequencies(c)
        for side in (0, 1):
            assert list(vals[side]) == top4(freq[side]), (c.class_id, side)
            # every stored value is a signed value of the class on its side
            for v in vals[side]:
                assert v == 0 or (abs(int(v)) in c.levels and side_of(int(v), c.parity) == side)
        assert list(rec[24:32]) == [abs(int(v)) for v in vals.ravel()]


def test_unused_slots_zero(table):
    assert (table[301:] == 0).all()
