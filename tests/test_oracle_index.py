"""Pins of the oracle's format-v1 index (reading R19): the class offsets against
the printed N, the radices against the class sizes (themselves pinned by the
theta series), colex ranks against itertools' enumeration, exhaustive
bijections on small classes enumerated by brute force, round trips through
points drawn by the independent input generator, and a stored fingerprint of
the whole map."""
import itertools
import json
import os
import random
from collections import Counter
from math import comb, factorial

import numpy as np
import pytest

from oracle import index as I
from oracle import lattice as L
from paper_2609_02652_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "format_v1_fingerprint.json")
N = 111_043_117_458_000


def test_offsets_end_at_printed_count():
    offs = I.class_offsets()
    assert len(offs) == 302 and offs[0] == 0 and offs[-1] == N
    assert 2 ** 46 < N < 2 ** I.INDEX_BITS
    assert all(b > a for a, b in zip(offs, offs[1:]))


def test_radix_products_are_class_sizes():
    for c in L.ball_classes():
        prod = 1
        for _, R in I.class_radices(c):
            prod *= R
        assert prod == c.size, c.class_id


@pytest.mark.parametrize("n,c", [(1, 1), (5, 2), (7, 3), (9, 4), (10, 0), (8, 8)])
def test_colex_rank_is_colex_order(n, c):
    # colex order: compare the largest element first, then the next largest
    subsets = sorted(itertools.combinations(range(n), c), key=lambda s: tuple(reversed(s)))
    for r, s in enumerate(subsets):
        assert I.colex_rank(s) == r
        assert I.colex_unrank(r, c, n) == list(s)
    assert len(subsets) == comb(n, c)


@pytest.mark.parametrize("mags", [[0, 0, 1, 1, 2], [3, 3, 3], [0, 4, 4, 8, 8, 8], [1, 2, 3, 4]])
def test_arrangements_biject(mags):
    seqs = sorted(set(itertools.permutations(mags)))
    m = factorial(len(mags))
    for k in Counter(mags).values():
        m //= factorial(k)
    assert len(seqs) == m
    ranks = sorted(I.arrangement_rank(list(s)) for s in seqs)
    assert ranks == list(range(m))
    for s in seqs:
        assert tuple(I.arrangement_unrank(mags, I.arrangement_rank(list(s)))) == s


def brute_force_class(cls):
    """Every lattice point of a class: all distinct arrangements of its
    magnitudes and all signs of the nonzero coordinates, kept when the
    membership test of §2.1 accepts them."""
    out = set()
    mags = list(cls.mags_desc)
    for perm in _arrangements(mags):
        nz = [i for i, a in enumerate(perm) if a]
        for signs in range(1 << len(nz)):
            x = list(perm)
            for j, i in enumerate(nz):
                if signs >> j & 1:
                    x[i] = -x[i]
            if L.is_leech_point(x):
                out.add(tuple(x))
    return out


def _arrangements(mags):
    """Distinct arrangements of a multiset with few nonzero entries: choose the
    positions of the nonzero magnitudes, then their order."""
    nonzero = [a for a in mags if a]
    seen = set()
    for pos in itertools.combinations(range(L.DIM), len(nonzero)):
        for order in set(itertools.permutations(nonzero)):
            x = [0] * L.DIM
            for p, a in zip(pos, order):
                x[p] = a
            t = tuple(x)
            if t not in seen:
                seen.add(t)
                yield t


# the six classes whose arrangements × sign patterns number ≤ 50,000
SMALL_CLASSES = [12, 1, 75, 150, 256, 34]


@pytest.mark.parametrize("cid", SMALL_CLASSES)
def test_small_class_exhaustive_bijection(cid):
    cls = L.ball_classes()[cid]
    pts = brute_force_class(cls)
    assert len(pts) == cls.size
    off = I.class_offsets()[cid]
    mapped = [tuple(I.point_of_index(off + r)) for r in range(cls.size)]
    assert set(mapped) == pts                     # onto the class, one index each
    for r in range(0, cls.size, max(1, cls.size // 500)):
        assert I.index_of_point(mapped[r]) == off + r


def test_odd_class_prefix_is_injective():
    """The odd class (±3, ±1^23): its first 64 codewords × 24 arrangements map
    to distinct lattice points of the class, each with its ±3 where the
    arrangement digit puts it."""
    cid = next(c.class_id for c in L.ball_classes() if c.mags_desc[:2] == (3, 1))
    cls = L.ball_classes()[cid]
    off = I.class_offsets()[cid]
    seen = set()
    for r in range(64 * 24):
        x = I.point_of_index(off + r)
        assert L.is_leech_point(x) and L.class_of_point(x).class_id == cid
        seen.add(tuple(x))
    assert len(seen) == 64 * 24
    assert cls.size == 4096 * 24


def test_boundaries_of_every_class():
    offs = I.class_offsets()
    for c in L.ball_classes():
        for idx in (offs[c.class_id], offs[c.class_id + 1] - 1):
            x = I.point_of_index(idx)
            assert L.is_leech_point(x)
            assert L.class_of_point(x).class_id == c.class_id
            assert I.index_of_point(x) == idx
    with pytest.raises(ValueError):
        I.point_of_index(N)
    with pytest.raises(ValueError):
        I.point_of_index(-1)


def test_random_indices_round_trip():
    rng = random.Random(2609)
    for _ in range(1500):
        idx = rng.randrange(N)
        x = I.point_of_index(idx)
        assert L.is_leech_point(x) and 2 <= L.shell_of(x) <= 12
        assert I.index_of_point(x) == idx


def test_points_from_the_input_generator_round_trip():
    """Points drawn by the generator (its own Golay code and sampler) index and
    come back unchanged; their classes follow the index's class ranges."""
    z = synth.sample_ball_points(synth.rng_for(5, "index-rt"), 800)
    offs = I.class_offsets()
    for x in z:
        idx = I.index_of_point(x)
        cid = L.class_of_point(x).class_id
        assert offs[cid] <= idx < offs[cid + 1]
        assert I.point_of_index(idx) == [int(v) for v in x]


def test_codes_carry_the_gain_bit():
    assert I.code_of(N - 1, 1) == (N - 1) | 1 << 47
    assert I.split_code(I.code_of(12345, 1)) == (12345, 1)
    with pytest.raises(ValueError):
        I.split_code(1 << 48)
    with pytest.raises(ValueError):
        I.code_of(1 << 47, 0)


def fingerprint_indices():
    """First and last index of every class, then 256 seeded random indices."""
    offs = I.class_offsets()
    idx = []
    for c in range(len(offs) - 1):
        idx += [offs[c], offs[c + 1] - 1]
    rng = np.random.default_rng(2609)
    idx += [int(v) for v in rng.integers(0, N, 256, dtype=np.int64)]
    return idx


def test_fingerprint_matches_stored():
    stored = json.load(open(GOLDEN))
    assert stored["n_indices"] == len(fingerprint_indices())
    assert I.fingerprint(fingerprint_indices()) == stored["sha256"]


def test_planted_order_change_changes_fingerprint(monkeypatch):
    """A different composition order (support and off-support arrangements
    swapped) is still a bijection, so only the fingerprint catches it."""
    orig = I.class_radices

    def swapped(cls):
        r = orig(cls)
        if cls.parity == 0:
            r[1], r[2] = r[2], r[1]
        return r
    base = I.fingerprint(fingerprint_indices()[:300])
    monkeypatch.setattr(I, "class_radices", swapped)
    x = I.point_of_index(I.class_offsets()[5] + 12345)
    assert L.is_leech_point(x)
    assert I.fingerprint(fingerprint_indices()[:300]) != base
