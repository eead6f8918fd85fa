"""Pins for the oracle's lattice math (oracle/lattice.py).

Each test ties the oracle to something fixed outside it: counts the paper
prints (tests/golden/paper_counts.json), the theta series of the Leech lattice
computed from σ11 and Ramanujan's τ, the textbook construction of the minimal
vectors, and brute-force enumerations of small classes.
"""
import json
import os
from itertools import combinations, permutations, product
from math import ceil, log2

import pytest

from oracle import lattice as L


@pytest.fixture(scope="module")
def paper(golden_dir):
    with open(os.path.join(golden_dir, "paper_counts.json")) as f:
        return {k: v["value"] for k, v in json.load(f).items() if not k.startswith("_")}


# ----------------------------------------------------------------------------
# Golay code
# ----------------------------------------------------------------------------
def test_golay_weight_enumerator(paper):
    cw = L.golay_codewords()
    assert len(cw) == paper["golay_codewords"] == 4096
    hist = {}
    for c in cw:
        w = bin(c).count("1")
        hist[w] = hist.get(w, 0) + 1
    # the extended Golay code's weight enumerator 1 + 759 y^8 + 2576 y^12 + 759 y^16 + y^24
    assert hist == {0: 1, 8: 759, 12: 2576, 16: 759, 24: 1}


def test_golay_is_linear_and_self_dual():
    cw = L.golay_codewords()
    s = set(cw)
    import random
    rnd = random.Random(1)
    for _ in range(2000):
        a, b = rnd.choice(cw), rnd.choice(cw)
        assert a ^ b in s                              # closed under addition
        assert bin(a & b).count("1") % 2 == 0          # self-orthogonal


# ----------------------------------------------------------------------------
# Theta series: N_m = (65520/691)(σ11(m) − τ(m)) for the Leech lattice
# ----------------------------------------------------------------------------
def _tau(nmax):
    """Ramanujan τ(1..nmax) from Δ = q ∏ (1 − q^n)^24, integer power series."""
    coeffs = [0] * (nmax + 1)
    coeffs[0] = 1
    for n in range(1, nmax + 1):
        for _ in range(24):                 # multiply by (1 − q^n), 24 times
            for k in range(nmax, n - 1, -1):
                coeffs[k] -= coeffs[k - n]
    return {n: coeffs[n - 1] for n in range(1, nmax + 1)}


def _sigma11(n):
    return sum(d ** 11 for d in range(1, n + 1) if n % d == 0)


def test_tau_known_values():
    t = _tau(6)
    assert [t[n] for n in range(1, 7)] == [1, -24, 252, -1472, 4830, -6048]


def test_shell_sizes_match_theta_series():
    tau = _tau(13)
    sizes = L.shell_sizes(13)
    for m in range(2, 14):
        num = 65520 * (_sigma11(m) - tau[m])
        assert num % 691 == 0
        assert sizes[m] == num // 691, m
    # and no norm-2 vectors (no roots): the m = 1 coefficient vanishes
    assert 65520 * (_sigma11(1) - tau[1]) == 0


def test_paper_counts(paper):
    classes = L.ball_classes()
    assert len(classes) == paper["n_classes"]
    assert L.ball_size() == paper["ball_points_N"]
    assert ceil(log2(paper["ball_points_N"])) == paper["index_bits"]
    assert 2 ** 46 < L.ball_size() < 2 ** 47
    shells = L.shell_sizes()
    assert len(shells) == paper["n_shells"]
    assert shells[2] == paper["kissing_number"]
    assert shells[3] == paper["second_shell"]
    assert L.ball_size(13) == paper["ball13_points"]
    assert max(c.n_levels for c in classes) == paper["max_levels_per_class"]
    assert len(classes) <= paper["class_table_records"]


def test_class_table_structure():
    classes = L.ball_classes()
    per_shell = [sum(1 for c in classes if c.shell == m) for m in range(2, 13)]
    assert per_shell == [3, 4, 8, 9, 17, 17, 30, 33, 47, 54, 79]
    by_levels = [sum(1 for c in classes if c.n_levels == k) for k in range(1, 6)]
    assert by_levels == [1, 34, 126, 124, 16]
    assert max(max(c.mags_desc) for c in classes) == 13          # int8 holds every z
    assert min(c.size for c in classes) == 48                     # (±8, 0^23)
    biggest = max(classes, key=lambda c: c.size)
    assert biggest.mags_desc == (6, 6) + (4,) * 5 + (2,) * 10 + (0,) * 7
    assert biggest.size == 8824597512192
    # canonical order (reading R4): shell, parity, descending magnitudes
    keys = [(c.shell, c.parity, c.mags_desc) for c in classes]
    assert keys == sorted(keys)
    assert [c.class_id for c in classes] == list(range(301))


def test_level_table_f32():
    t = L.level_table_f32()
    assert t.shape == (301, 5)
    c = L.ball_classes()[2]                     # (3, 1^23), shell 2
    assert c.levels == (1, 3)
    import numpy as np
    assert t[2, 0] == np.float32(1 / (4 * 2 ** 0.5))
    assert t[2, 1] == np.float32(3 / (4 * 2 ** 0.5))
    assert (t[2, 2:] == 0).all()


# ----------------------------------------------------------------------------
# Membership, against the textbook construction of the minimal vectors
# (Conway & Sloane's shapes (±2^8 0^16), (∓3 ±1^23), (±4^2 0^22))
# ----------------------------------------------------------------------------
def _minimal_vectors():
    cw = L.golay_codewords()
    octads = [c for c in cw if bin(c).count("1") == 8]
    out = []
    for o in octads:                                  # ±2 on an octad, even # of minus
        pos = [i for i in range(24) if o >> i & 1]
        for signs in range(256):
            if bin(signs).count("1") % 2:
                continue
            v = [0] * 24
            for k, i in enumerate(pos):
                v[i] = -2 if signs >> k & 1 else 2
            out.append(tuple(v))
    for c in cw:                                      # upper signs on a codeword
        for p in range(24):
            v = [(1 if c >> i & 1 else -1) for i in range(24)]
            v[p] = -3 if c >> p & 1 else 3
            out.append(tuple(v))
    for i, j in combinations(range(24), 2):           # ±4 ±4
        for si, sj in product((4, -4), repeat=2):
            v = [0] * 24
            v[i], v[j] = si, sj
            out.append(tuple(v))
    return out


def test_minimal_vectors_are_members():
    mv = _minimal_vectors()
    assert len(mv) == len(set(mv)) == 196560
    assert all(sum(a * a for a in v) == 32 for v in mv)
    assert all(L.is_leech_point(v) for v in mv)


def test_near_misses_are_rejected():
    cw = set(L.golay_codewords())
    # ±2 on a weight-8 set that is not an octad
    for pos in [(0, 1, 2, 3, 4, 5, 6, 7), (0, 2, 4, 6, 8, 10, 12, 14)]:
        m = sum(1 << i for i in pos)
        v = [2 if i in pos else 0 for i in range(24)]
        assert L.is_leech_point(v) == (m in cw)
    # an octad with an odd number of minus signs
    o = next(c for c in cw if bin(c).count("1") == 8)
    v = [2 if o >> i & 1 else 0 for i in range(24)]
    assert L.is_leech_point(v)
    v[next(i for i in range(24) if o >> i & 1)] = -2
    assert not L.is_leech_point(v)
    # (4, 0^23) has norm 16 (a root): Λ24 has none
    assert not L.is_leech_point([4] + [0] * 23)
    assert L.is_leech_point([8] + [0] * 23)
    # mixed parity
    assert not L.is_leech_point([3, 2] + [1] * 22)
    # an odd vector whose ≡3 set is not a codeword
    assert not L.is_leech_point([3] + [1] * 23)
    assert L.is_leech_point([-3] + [1] * 23)


def test_brute_force_octad_class():
    """Every ±2 pattern on every 8-subset: exactly 759·2^7 members."""
    members = 0
    supports = 0
    for pos in combinations(range(24), 8):
        v = [0] * 24
        for i in pos:
            v[i] = 2
        if not L.is_leech_point(v):
            continue
        supports += 1
        for signs in range(256):
            w = list(v)
            for k, i in enumerate(pos):
                if signs >> k & 1:
                    w[i] = -2
            members += L.is_leech_point(w)
    assert supports == 759
    assert members == 97152 == L.class_size((2,) * 8 + (0,) * 16)


@pytest.mark.parametrize("mult", [
    {4: 2}, {8: 1}, {8: 1, 4: 2}, {8: 2}, {12: 1, 4: 1}, {8: 3},   # classes
    {4: 3}, {4: 1}, {8: 1, 4: 1}, {12: 1},                         # not classes
])
def test_brute_force_small_multisets(mult):
    vals = sorted((a for a, k in mult.items() for _ in range(k)), reverse=True)
    n = len(vals)
    members = 0
    # choose positions for the nonzero values (distinct arrangements), then signs
    seen = set()
    for pos in combinations(range(24), n):
        for perm in set(permutations(vals)):
            key = tuple(zip(pos, perm))
            if key in seen:
                continue
            seen.add(key)
            for signs in range(1 << n):
                v = [0] * 24
                for k, (i, a) in enumerate(key):
                    v[i] = -a if signs >> k & 1 else a
                members += L.is_leech_point(v)
    mags = tuple(vals) + (0,) * (24 - n)
    assert members == L.class_size(mags)
