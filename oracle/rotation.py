"""Activation rotation for the oracle (paper §2.3 "The kernel": the activation
is rotated by a Walsh–Hadamard transform before the matvec; §6 "The rotated
basis and the shared-memory wall": weights are stored in the rotated basis, so
every consumer rotates its activation).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Reading R17.  The paper names a Walsh–Hadamard transform of the whole
activation but fixes neither its length nor its signs.  For K = 2^k · m with m
odd (the shapes served here include 14336 = 2^11·7, 5120 = 2^10·5 and
17408 = 2^10·17, widths with no Hadamard matrix of the full order), the
rotation is taken blockwise:

    x_rot[b·n + i] = n^(-1/2) · Σ_j H_n[i, j] · s[b·n + j] · x[b·n + j],  n = 2^k,

for every block b = 0..m−1, where H_n is the Sylvester-ordered Walsh–Hadamard
matrix, H_n[i, j] = (−1)^popcount(i AND j), and s ∈ {−1, +1}^K is a sign vector
the caller supplies (random signs make the map an incoherence rotation; they
are an input, drawn by the input generator).  The map is orthogonal.  The
rotated activation is zero-padded to Kpad for the matvec.
"""
from __future__ import annotations

import numpy as np


def pow2_block(K: int) -> int:
    """n = 2^k, the largest power of two dividing K (the block length)."""
    if K <= 0:
        raise ValueError("K must be positive")
    return K & -K


def _parity16() -> np.ndarray:
    """popcount(v) mod 2 for v = 0..65535, bit by bit."""
    v = np.arange(1 << 16, dtype=np.int64)
    p = np.zeros_like(v)
    while v.any():
        p ^= v & 1
        v >>= 1
    return p


_PARITY16 = _parity16()


def walsh_at(n: int, rows) -> np.ndarray:
    """The given rows of H_n: H_n[i, j] = (−1)^popcount(i & j), as f64 (the
    textbook definition; the parity of i & j is read 16 bits at a time)."""
    if n <= 0 or n & (n - 1) or n > 1 << 32:
        raise ValueError("n must be a power of two ≤ 2^32")
    i = np.asarray(rows, dtype=np.int64)
    j = np.arange(n, dtype=np.int64)
    ij = i[:, None] & j[None, :]
    parity = _PARITY16[ij & 0xFFFF] ^ _PARITY16[ij >> 16]
    return np.where(parity == 1, -1.0, 1.0)


def walsh_rows(n: int, r0: int, r1: int) -> np.ndarray:
    """Rows r0..r1-1 of H_n."""
    return walsh_at(n, np.arange(r0, r1))


def walsh_matrix(n: int) -> np.ndarray:
    """H_n, all n rows."""
    return walsh_rows(n, 0, n)


def rotate64(x, signs) -> np.ndarray:
    """The rotation R17 in f64: x (length K, any float type) and signs (±1,
    length K) -> x_rot (f64, length K)."""
    x = np.asarray(x, dtype=np.float64)
    s = np.asarray(signs, dtype=np.float64)
    K = x.size
    if s.size != K or not np.all(np.abs(s) == 1.0):
        raise ValueError("signs must be ±1 of the activation's length")
    n = pow2_block(K)
    blocks = (s * x).reshape(K // n, n)
    out = np.empty((K // n, n))
    step = max(1, (1 << 22) // n)          # rows of H_n per piece (bounded memory)
    for r0 in range(0, n, step):
        r1 = min(n, r0 + step)
        out[:, r0:r1] = blocks @ walsh_rows(n, r0, r1).T
    return (out / np.sqrt(n)).reshape(K)


def rotate64_at(x, signs, idx) -> np.ndarray:
    """Entries idx of rotate64(x, signs), each from its own row of H_n (for
    checking sampled outputs of long blocks)."""
    x = np.asarray(x, dtype=np.float64)
    s = np.asarray(signs, dtype=np.float64)
    K = x.size
    if s.size != K or not np.all(np.abs(s) == 1.0):
        raise ValueError("signs must be ±1 of the activation's length")
    n = pow2_block(K)
    idx = np.asarray(idx, dtype=np.int64)
    sx = s * x
    out = np.empty(idx.size)
    for b in np.unique(idx // n):
        sel = idx // n == b
        H = walsh_at(n, idx[sel] % n)
        out[sel] = H @ sx[b * n:(b + 1) * n]
    return out / np.sqrt(n)


def rotate_padded64(x, signs, Kpad: int) -> np.ndarray:
    """rotate64 followed by zero padding to Kpad (the matvec's input length)."""
    r = rotate64(x, signs)
    out = np.zeros(Kpad, dtype=np.float64)
    out[: r.size] = r
    return out
