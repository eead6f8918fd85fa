"""Format-v1 direction index for the oracle (paper §2.1 "What a Λ24 index is":
the 47-bit index enumerates the classes, then the arrangements and signs inside
a class, in a fixed order, as a bijection onto the ball; one gain bit makes the
48-bit block code; §2.2 "Unfolding at load time": the transcoder expands the
index into decoded fields once, at load time).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Reading R19.  The paper fixes the structure (classes, then arrangements and
signs, mixed radix) but prints neither the order nor the radices.  The order
taken here:

* code = index | gain << 47, with index < N = 111,043,117,458,000 < 2^47;
* index = offset(c) + r, where offset(c) is the number of points in the
  classes with smaller id (class-id order R4) and r ∈ [0, size(c));
* r is a mixed-radix number whose digits, most significant first, are
  - even class (w = number of coordinates with |x_i| ≡ 2 mod 4):
      1. the rank of the support codeword {i : |x_i| ≡ 2 mod 4} among the
         codewords of weight w in ascending order of their 24-bit value
         (bit i = coordinate i);
      2. the arrangement of the ≡ 2 (mod 4) magnitudes over the support;
      3. the arrangement of the ≡ 0 (mod 4) magnitudes over the other
         coordinates;
      4. the signs of the nonzero off-support coordinates, bit j for the j-th
         of them in increasing coordinate order (1 = negative), radix 2^f0;
      5. the signs of the first w − 1 support coordinates, likewise, radix
         2^(w−1) (radix 1 when w = 0); the last support coordinate takes the
         sign that makes Σx ≡ 0 (mod 8);
  - odd class:
      1. the rank of the codeword {i : x_i ≡ 3 mod 4} among all 4096 codewords
         in ascending order of value;
      2. the arrangement of the 24 magnitudes over all coordinates; the signs
         follow from the codeword (sign(x_i) = −1 iff bit i of the codeword
         differs from [|x_i| ≡ 3 mod 4]).
* an arrangement of a multiset over an ordered list of n positions is itself
  a mixed-radix number: one digit per distinct magnitude in ascending order,
  the colex rank Σ_j C(q_j, j) of that magnitude's positions q_1 < … < q_c,
  counted among the positions still free after the smaller magnitudes took
  theirs, with radix C(free, c).  (The positions of the largest magnitude are
  forced: radix 1.)  The product of the radices is the multinomial
  coefficient, so every digit string names exactly one arrangement.

Parity with the paper's own codes is unpinned: the paper prints none.  The
tests pin this map by what any such index must satisfy (a bijection onto the
ball, round trips of every class's first and last index, the class sizes)
and fix its order with a stored fingerprint written from this module.
"""
from __future__ import annotations

import hashlib
from bisect import bisect_right
from collections import Counter
from functools import lru_cache
from math import comb

from .lattice import BALL_M, DIM, ball_classes, class_of_point, golay_codewords

INDEX_BITS = 47
GAIN_SHIFT = 47


@lru_cache(maxsize=None)
def class_offsets(m_max: int = BALL_M) -> tuple[int, ...]:
    """offset(c) for every class id, and N as the last entry."""
    out = [0]
    for c in ball_classes(m_max):
        out.append(out[-1] + c.size)
    return tuple(out)


@lru_cache(maxsize=None)
def codewords_sorted() -> tuple[int, ...]:
    """All 4096 codewords in ascending value."""
    return tuple(sorted(golay_codewords()))


@lru_cache(maxsize=None)
def codewords_of_weight(w: int) -> tuple[int, ...]:
    return tuple(c for c in codewords_sorted() if bin(c).count("1") == w)


# ------------------------------------------------------------ arrangements
def colex_rank(subset) -> int:
    """Σ_j C(q_j, j) over the sorted relative positions q_1 < … < q_c."""
    return sum(comb(q, j + 1) for j, q in enumerate(sorted(subset)))


def colex_unrank(r: int, c: int, n: int) -> list[int]:
    """The c-subset of {0..n−1} with colex rank r (0 ≤ r < C(n, c))."""
    if not 0 <= r < comb(n, c):
        raise ValueError("rank out of range")
    out = []
    q = n - 1
    for j in range(c, 0, -1):
        while comb(q, j) > r:
            q -= 1
        out.append(q)
        r -= comb(q, j)
        q -= 1
    return sorted(out)


def arrangement_radices(mags) -> list[int]:
    """Radices of an arrangement of the multiset `mags` (ascending magnitudes)."""
    cnt = Counter(mags)
    free = len(mags)
    rad = []
    for a in sorted(cnt):
        rad.append(comb(free, cnt[a]))
        free -= cnt[a]
    return rad


def arrangement_rank(seq) -> int:
    """Rank of the sequence of magnitudes `seq` (one per position, in order)."""
    free = list(range(len(seq)))
    r = 0
    for a in sorted(set(seq)):
        mine = [k for k, p in enumerate(free) if seq[p] == a]
        r = r * comb(len(free), len(mine)) + colex_rank(mine)
        free = [p for p in free if seq[p] != a]
    return r


def arrangement_unrank(mags, r: int) -> list[int]:
    """The sequence of magnitudes with rank r among the arrangements of `mags`."""
    cnt = Counter(mags)
    levels = sorted(cnt)
    rad = arrangement_radices(mags)
    digits = []
    for R in reversed(rad):            # least significant digit last
        digits.append(r % R)
        r //= R
    if r:
        raise ValueError("arrangement rank out of range")
    digits.reverse()
    n = len(mags)
    seq = [None] * n
    free = list(range(n))
    for a, d in zip(levels, digits):
        picked = colex_unrank(d, cnt[a], len(free))
        for k in picked:
            seq[free[k]] = a
        free = [p for k, p in enumerate(free) if k not in set(picked)]
    return seq


def _product(xs) -> int:
    out = 1
    for x in xs:
        out *= x
    return out


# ------------------------------------------------------------- the index
def class_radices(cls) -> list[tuple[str, int]]:
    """The mixed-radix digits of a class, most significant first (R19)."""
    mags = list(cls.mags_desc)
    if cls.parity == 0:
        two = [a for a in mags if a % 4 == 2]
        zero = [a for a in mags if a % 4 == 0]
        w = len(two)
        f0 = sum(1 for a in zero if a > 0)
        return [("codeword", len(codewords_of_weight(w))),
                ("support", _product(arrangement_radices(two))),
                ("off_support", _product(arrangement_radices(zero))),
                ("free_signs", 2 ** f0), ("support_signs", 2 ** max(w - 1, 0))]
    return [("codeword", len(codewords_sorted())),
            ("arrangement", _product(arrangement_radices(mags)))]


def point_of_index(index: int, m_max: int = BALL_M) -> list[int]:
    """The lattice point with the given 47-bit direction index."""
    offs = class_offsets(m_max)
    if not 0 <= index < offs[-1]:
        raise ValueError("index out of range")
    c = bisect_right(offs, index) - 1
    cls = ball_classes(m_max)[c]
    r = index - offs[c]
    radices = class_radices(cls)
    digits = {}
    for name, R in reversed(radices):
        digits[name] = r % R
        r //= R
    assert r == 0
    mags = list(cls.mags_desc)
    x = [0] * DIM
    if cls.parity == 0:
        two = [a for a in mags if a % 4 == 2]
        zero = [a for a in mags if a % 4 == 0]
        cw = codewords_of_weight(len(two))[digits["codeword"]]
        sup = [i for i in range(DIM) if cw >> i & 1]
        off = [i for i in range(DIM) if not cw >> i & 1]
        for i, a in zip(sup, arrangement_unrank(two, digits["support"])):
            x[i] = a
        for i, a in zip(off, arrangement_unrank(zero, digits["off_support"])):
            x[i] = a
        nz = [i for i in off if x[i] != 0]
        for j, i in enumerate(nz):
            if digits["free_signs"] >> j & 1:
                x[i] = -x[i]
        for j, i in enumerate(sup[:-1]):
            if digits["support_signs"] >> j & 1:
                x[i] = -x[i]
        if sup and sum(x) % 8 != 0:
            x[sup[-1]] = -x[sup[-1]]
    else:
        cw = codewords_sorted()[digits["codeword"]]
        for i, a in enumerate(arrangement_unrank(mags, digits["arrangement"])):
            x[i] = -a if (cw >> i & 1) != (a % 4 == 3) else a
    return x


def index_of_point(x, m_max: int = BALL_M) -> int:
    """The 47-bit direction index of a lattice point of the ball."""
    x = [int(v) for v in x]
    cls = class_of_point(x, m_max)
    radices = class_radices(cls)
    if cls.parity == 0:
        cw = sum(1 << i for i in range(DIM) if x[i] % 4 == 2)
        sup = [i for i in range(DIM) if cw >> i & 1]
        off = [i for i in range(DIM) if not cw >> i & 1]
        nz = [i for i in off if x[i] != 0]
        digits = {
            "codeword": codewords_of_weight(len(sup)).index(cw),
            "support": arrangement_rank([abs(x[i]) for i in sup]),
            "off_support": arrangement_rank([abs(x[i]) for i in off]),
            "free_signs": sum(1 << j for j, i in enumerate(nz) if x[i] < 0),
            "support_signs": sum(1 << j for j, i in enumerate(sup[:-1]) if x[i] < 0),
        }
    else:
        cw = sum(1 << i for i in range(DIM) if x[i] % 4 == 3)
        digits = {"codeword": codewords_sorted().index(cw),
                  "arrangement": arrangement_rank([abs(v) for v in x])}
    r = 0
    for name, R in radices:
        if not 0 <= digits[name] < R:
            raise AssertionError("digit out of range")
        r = r * R + digits[name]
    return class_offsets(m_max)[cls.class_id] + r


def code_of(index: int, gain: int) -> int:
    """48-bit block code: direction index and gain bit."""
    if not 0 <= index < 1 << INDEX_BITS or gain not in (0, 1):
        raise ValueError("bad index or gain")
    return index | gain << GAIN_SHIFT


def split_code(code: int) -> tuple[int, int]:
    """(index, gain) of a 48-bit block code."""
    if code >> 48:
        raise ValueError("bits above 47 set")
    return code & ((1 << INDEX_BITS) - 1), code >> GAIN_SHIFT


def fingerprint(indices, m_max: int = BALL_M) -> str:
    """sha256 over the class radices (in composition order) of every class and
    the points of the given indices: it pins the whole map, order included."""
    h = hashlib.sha256()
    for cls in ball_classes(m_max):
        h.update(repr((cls.class_id, class_radices(cls))).encode())
    for i in indices:
        h.update(repr((int(i), point_of_index(int(i), m_max))).encode())
    return h.hexdigest()


