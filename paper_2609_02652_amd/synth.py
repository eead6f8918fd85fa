"""Seeded synthetic inputs for the Leech GEMV (shared by tests and the bench).

This module only draws inputs.  It holds none of the method's arithmetic: no
decoded fields, no class ids, no layouts, no weights, no matvec.  It emits

* lattice points z (int8 [M, nb, 24]) drawn uniformly from the ball Λ24(12):
  a class with probability proportional to its size, then a uniform member of
  it (random arrangement, signs obeying the Golay constraints);
* one gain bit per block (uniform), one fp16 scale per block fp16(|N(0,1)|·0.02),
* an activation x = fp16(N(0,1)) of length K, zero-padded to Kpad = 24·⌈K/24⌉.

To draw uniform ball points it needs the ball's magnitude multisets and how
many points each holds; it derives them here, independently of any other
module, from the lattice's definition (√8 scaling: coordinates all even or all
odd; the positions with x ≡ 2 (mod 4), resp. x ≡ 3 (mod 4), form an extended
Golay codeword; Σx ≡ 0, resp. 4 (mod 8); shells Σx² = 16m, m = 2..12).

Every stream is a numpy PCG64 generator keyed by (seed, stream name), so a
workload is reproducible from its seed alone.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass
from functools import lru_cache
from math import comb, isqrt

import numpy as np

DIM = 24
SCALE_SIGMA = 0.02


# ----------------------------------------------------------------------------
# Extended Golay code: generator matrix = 12 shifts of the cyclic generator
# g(x) = 1 + x^2 + x^4 + x^5 + x^6 + x^10 + x^11, plus an overall parity bit.
# ----------------------------------------------------------------------------
@lru_cache(maxsize=None)
def _codewords() -> np.ndarray:
    g = sum(1 << e for e in (0, 2, 4, 5, 6, 10, 11))
    rows = []
    for s in range(12):
        r = g << s
        rows.append(r | ((bin(r).count("1") & 1) << 23))
    words = np.zeros(1, dtype=np.int64)
    for r in rows:                       # span of the rows, doubling each time
        words = np.concatenate([words, words ^ r])
    return np.sort(words)


@lru_cache(maxsize=None)
def _codewords_by_weight() -> dict[int, np.ndarray]:
    cw = _codewords()
    wt = np.array([bin(int(c)).count("1") for c in cw])
    return {int(w): cw[wt == w] for w in np.unique(wt)}


# ----------------------------------------------------------------------------
# Magnitude multisets of the ball and their point counts
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class _Multiset:
    mags: tuple[int, ...]        # 24 magnitudes, sorted descending
    count: int                   # lattice points with these magnitudes


def _arrangements(values) -> int:
    """Distinct orderings of a list of values."""
    n, out = len(values), 1
    for v in set(values):
        k = values.count(v)
        out *= comb(n, k)
        n -= k
    return out


def _points_with_magnitudes(mags: tuple[int, ...]) -> int:
    nw = {w: len(c) for w, c in _codewords_by_weight().items()}
    if all(a % 2 == 0 for a in mags):
        two = [a for a in mags if a % 4 == 2]
        rest = [a for a in mags if a % 4 == 0]
        w = len(two)
        if w not in nw:
            return 0
        if w:
            signs = 2 ** (w - 1)                   # half the support signs fit mod 8
        else:
            signs = 1 if sum(1 for a in mags if a % 8 == 4) % 2 == 0 else 0
        signs *= 2 ** sum(1 for a in rest if a)    # signs of 0-mod-4 entries are free
        return nw[w] * _arrangements(two) * _arrangements(rest) * signs
    if all(a % 2 == 1 for a in mags):
        if sum(1 for a in mags if a % 8 in (3, 5)) % 2 == 0:
            return 0
        return 4096 * _arrangements(list(mags))   # signs forced by the codeword
    return 0


@lru_cache(maxsize=None)
def ball_multisets(m_max: int = 12) -> tuple[_Multiset, ...]:
    """All magnitude multisets of the ball with nonzero point count."""
    out = []

    def extend(prefix, largest, remaining, slots):
        if slots == 0:
            if remaining == 0:
                yield tuple(prefix)
            return
        for a in range(min(largest, isqrt(remaining)), -1, -1):
            if (a - prefix[0]) % 2 if prefix else False:
                continue
            yield from extend(prefix + [a], a, remaining - a * a, slots - 1)

    for m in range(2, m_max + 1):
        for first in range(isqrt(16 * m), 0, -1):
            for mags in extend([first], first, 16 * m - first * first, DIM - 1):
                cnt = _points_with_magnitudes(mags)
                if cnt:
                    out.append(_Multiset(mags, cnt))
    return tuple(out)


# ----------------------------------------------------------------------------
# Sampling
# ----------------------------------------------------------------------------
def rng_for(seed: int, stream: str) -> np.random.Generator:
    """Independent PCG64 stream keyed by (seed, stream name)."""
    key = int.from_bytes(hashlib.sha256(stream.encode()).digest()[:8], "little")
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), key])))


def sample_ball_points(rng: np.random.Generator, n: int, m_max: int = 12) -> np.ndarray:
    """n points drawn uniformly from the ball; int8 [n, 24]."""
    sets = ball_multisets(m_max)
    counts = np.array([s.count for s in sets], dtype=np.int64)
    cum = np.cumsum(counts)
    u = rng.integers(0, int(cum[-1]), size=n, dtype=np.int64)
    which = np.searchsorted(cum, u, side="right")
    z = np.zeros((n, DIM), dtype=np.int8)
    by_weight = _codewords_by_weight()
    allcw = _codewords()
    bitpos = np.arange(DIM, dtype=np.int64)
    order = np.argsort(which, kind="stable")
    bounds = np.searchsorted(which[order], np.arange(len(sets) + 1))
    for k in range(len(sets)):
        idx = order[bounds[k]:bounds[k + 1]]
        nk = idx.size
        if nk == 0:
            continue
        mags = np.array(sets[k].mags, dtype=np.int64)
        if mags[0] % 2 == 0:
            two = mags[mags % 4 == 2]
            rest = mags[mags % 4 == 0]
            w = two.size
            cw = by_weight[w]
            support = ((cw[rng.integers(0, cw.size, nk)][:, None] >> bitpos) & 1).astype(bool)
            # support positions first, each part in uniformly random order
            keys = rng.random((nk, DIM)) + (~support) * 2.0
            pos = np.argsort(keys, axis=1)
            vals = np.concatenate([two, rest])
            blk = np.zeros((nk, DIM), dtype=np.int64)
            np.put_along_axis(blk, pos, np.broadcast_to(vals, (nk, DIM)), axis=1)
            neg = rng.integers(0, 2, (nk, DIM)).astype(bool) & (blk != 0)
            blk = np.where(neg, -blk, blk)
            if w:
                bad = np.mod(blk.sum(axis=1), 8) != 0       # flip one support sign
                first = pos[:, 0]
                rows = np.nonzero(bad)[0]
                blk[rows, first[rows]] *= -1
        else:
            c = allcw[rng.integers(0, allcw.size, nk)]
            bits = (c[:, None] >> bitpos) & 1
            pos = np.argsort(rng.random((nk, DIM)), axis=1)
            blk = np.zeros((nk, DIM), dtype=np.int64)
            np.put_along_axis(blk, pos, np.broadcast_to(mags, (nk, DIM)), axis=1)
            # x_i ≡ 3 (mod 4) exactly on the codeword's support
            positive = (blk % 4 == 3) == (bits == 1)
            blk = np.where(positive, blk, -blk)
        z[idx] = blk.astype(np.int8)
    return z


@dataclass
class GemvInputs:
    M: int
    K: int
    Kpad: int
    nb: int
    z: np.ndarray          # int8 [M, nb, 24]
    gain: np.ndarray       # uint8 [M, nb]
    scale: np.ndarray      # float16 [M, nb]
    x: np.ndarray          # float16 [Kpad], zero past K
    seed: int
    name: str


def padded_k(K: int) -> int:
    return DIM * ((K + DIM - 1) // DIM)


def make_gemv_inputs(M: int, K: int, seed: int = 0, name: str = "gemv") -> GemvInputs:
    """One synthetic GEMV: M×K Leech-coded weights (K padded to 24·nb) and x."""
    if M <= 0 or K <= 0:
        raise ValueError("M and K must be positive")
    Kpad = padded_k(K)
    nb = Kpad // DIM
    z = sample_ball_points(rng_for(seed, f"{name}/z"), M * nb).reshape(M, nb, DIM)
    gain = rng_for(seed, f"{name}/gain").integers(0, 2, (M, nb)).astype(np.uint8)
    scale = (np.abs(rng_for(seed, f"{name}/scale").standard_normal((M, nb))) * SCALE_SIGMA).astype(np.float16)
    x = np.zeros(Kpad, dtype=np.float16)
    x[:K] = rng_for(seed, f"{name}/x").standard_normal(K).astype(np.float16)
    return GemvInputs(M, K, Kpad, nb, z, gain, scale, x, seed, name)


def make_activation(K: int, seed: int, name: str) -> np.ndarray:
    Kpad = padded_k(K)
    x = np.zeros(Kpad, dtype=np.float16)
    x[:K] = rng_for(seed, f"{name}/x").standard_normal(K).astype(np.float16)
    return x


def make_signs(K: int, seed: int, name: str) -> np.ndarray:
    """Uniform ±1 signs (int8, length K) for the activation rotation."""
    return np.where(rng_for(seed, f"{name}/signs").integers(0, 2, K) == 1, 1, -1).astype(np.int8)


# Workload shapes (M, K) of the benchmark configurations.
CONFIG_SHAPES = {
    "c1_768x1536": [("w", 768, 1536)],
    "c2_4096x4096": [("w", 4096, 4096)],
    "c3_8b_layer": [("q", 4096, 4096), ("k", 1024, 4096), ("v", 1024, 4096), ("o", 4096, 4096),
                    ("gate", 14336, 4096), ("up", 14336, 4096), ("down", 4096, 14336)],
    "c4_8192x8192": [("w", 8192, 8192)],
}
