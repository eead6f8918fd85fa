"""Decoded fields -> lattice points -> f64 weights -> y64 = W x.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's transcoder turns each 24-weight block into a record of decoded
fields: class identifier, gain bit, sign mask and the magnitude level of each
coordinate (§2.2).  The matvec never decodes the 47-bit index; it reads those
fields (§2.2, §2.3).  This module states, in f64, what any correct reading of
the fields computes:

  z_i   = (−1)^{s_i} · a_{c, ℓ_i}                     (integer coordinates)
  w_b,i = f64(scale_b) · centroid[g_b] · z_i / (4√m_c) (shape–gain weight)
  y64_r = Σ_b Σ_i w_{r,b,i} · f64(x_{24b+i})          (the matvec)

Readings (also in the design notes):
* R7 signs: bit i of the sign mask is 1 iff z_i < 0; it must be 0 where the
  magnitude is 0 (§2.2 names a sign mask without fixing its convention).
* R8 scales: the workloads give every block an fp16 scale; the paper's
  per-tensor gain centroids (§2.1: one gain bit picks one of two centroids) are
  kept as a pair of f32 values selected by the gain bit, and multiply the
  block's scale.  The paper's f32 row scale and f32 tail columns (§2.3) are
  replaced by these per-block scales and by zero-padding K to a multiple of 24.
* R9 tolerance: the primary check is max_r |y_r − y64_r| / (‖W_r‖₂·‖x‖₂); the
  paper's own per-row check |y_r − y64_r| ≤ 1e-5 · Σ_j |W_rj x_j| (§2.4) is
  reported beside it.
"""
from __future__ import annotations

from math import sqrt

import numpy as np

from .lattice import DIM, BALL_M, ball_classes, class_of_point, is_leech_point


# ----------------------------------------------------------------------------
# One block, written out plainly (§2.2 decoded-field record)
# ----------------------------------------------------------------------------
def decode_block(class_id: int, sign_mask: int, levels, m_max: int = BALL_M) -> list[int]:
    """Integer coordinates of one block from its decoded fields.

    Raises ValueError for any field the ball cannot hold: a class id out of
    range, a level beyond the class's level count, a sign on a zero coordinate,
    or a level pattern whose magnitudes do not form the class's multiset.
    """
    classes = ball_classes(m_max)
    if not 0 <= int(class_id) < len(classes):
        raise ValueError(f"class id {class_id} out of range")
    cls = classes[int(class_id)]
    z = []
    for i in range(DIM):
        lv = int(levels[i])
        if not 0 <= lv < cls.n_levels:
            raise ValueError(f"level {lv} out of range for class {class_id}")
        a = cls.levels[lv]
        neg = (int(sign_mask) >> i) & 1
        if a == 0 and neg:
            raise ValueError("sign bit set on a zero coordinate")
        z.append(-a if neg else a)
    if int(sign_mask) >> DIM:
        raise ValueError("sign mask has bits above coordinate 23")
    if tuple(sorted((abs(v) for v in z), reverse=True)) != cls.mags_desc:
        raise ValueError("levels do not form the class's magnitude multiset")
    if not is_leech_point(z):
        raise ValueError("decoded block is not a Leech lattice point")
    return z


def fields_of_point(z, m_max: int = BALL_M) -> tuple[int, int, list[int]]:
    """Inverse of decode_block: (class id, sign mask, levels) of a ball point."""
    cls = class_of_point(z, m_max)
    sign_mask = 0
    levels = []
    for i, v in enumerate(z):
        v = int(v)
        if v < 0:
            sign_mask |= 1 << i
        levels.append(cls.levels.index(abs(v)))
    return cls.class_id, sign_mask, levels


# ----------------------------------------------------------------------------
# Whole matrices.  Same arithmetic, vectorised with numpy gathers so that the
# oracle can follow the workloads' sizes; tests check it against the per-block
# functions above on small inputs.
# ----------------------------------------------------------------------------
def _class_arrays(m_max: int = BALL_M):
    classes = ball_classes(m_max)
    mags = np.zeros((len(classes), 8), dtype=np.int64)
    nlev = np.zeros(len(classes), dtype=np.int64)
    shell = np.zeros(len(classes), dtype=np.int64)
    for c in classes:
        mags[c.class_id, : c.n_levels] = c.levels
        nlev[c.class_id] = c.n_levels
        shell[c.class_id] = c.shell
    return mags, nlev, shell


def fields_from_points(z: np.ndarray, m_max: int = BALL_M):
    """Decoded fields of many ball points.

    z: int array [..., 24].  Returns (class_id uint16, sign_mask uint32,
    level uint8 [..., 24]).  Every point is checked for membership.
    """
    z = np.asarray(z)
    flat = z.reshape(-1, DIM).astype(np.int64)
    n = flat.shape[0]
    classes = ball_classes(m_max)
    index = {c.mags_desc: c.class_id for c in classes}
    mags_sorted = -np.sort(-np.abs(flat), axis=1)
    class_id = np.empty(n, dtype=np.int64)
    for b in range(n):
        key = tuple(int(v) for v in mags_sorted[b])
        if key not in index:
            raise ValueError(f"block {b} is not in the ball")
        class_id[b] = index[key]
    mags, _, _ = _class_arrays(m_max)
    absz = np.abs(flat)
    # level = position of |z_i| among the class's ascending distinct magnitudes
    level = np.full((n, DIM), -1, dtype=np.int64)
    for lv in range(8):
        hit = absz == mags[class_id, lv][:, None]
        hit &= (lv < np.array([classes[c].n_levels for c in range(len(classes))])[class_id])[:, None]
        level = np.where(hit & (level < 0), lv, level)
    assert (level >= 0).all()
    bits = (flat < 0).astype(np.uint64) << np.arange(DIM, dtype=np.uint64)
    sign_mask = bits.sum(axis=1).astype(np.uint32)
    _check_membership(flat)
    shp = z.shape[:-1]
    return (class_id.astype(np.uint16).reshape(shp), sign_mask.reshape(shp),
            level.astype(np.uint8).reshape(shp + (DIM,)))


def _check_membership(flat: np.ndarray) -> None:
    """Vectorised restatement of is_leech_point (checked against it in tests)."""
    from .lattice import golay_codewords
    mu = flat[:, 0] & 1
    if ((flat & 1) != mu[:, None]).any():
        raise ValueError("mixed parities")
    residue = np.where(mu == 0, 2, 3)
    sel = (np.mod(flat, 4) == residue[:, None]).astype(np.int64)
    masks = (sel << np.arange(DIM)).sum(axis=1)
    ok = np.isin(masks, np.array(golay_codewords(), dtype=np.int64))
    ok &= np.mod(flat.sum(axis=1), 8) == 4 * mu
    if not ok.all():
        raise ValueError(f"{int((~ok).sum())} blocks are not Leech points")


def decode_fields(class_id, sign_mask, level, m_max: int = BALL_M) -> np.ndarray:
    """Integer coordinates int8 [..., 24] of many blocks (§2.2), validated."""
    class_id = np.asarray(class_id).astype(np.int64)
    sign_mask = np.asarray(sign_mask).astype(np.int64)
    level = np.asarray(level).astype(np.int64)
    shp = class_id.shape
    cid = class_id.reshape(-1)
    sm = sign_mask.reshape(-1)
    lv = level.reshape(-1, DIM)
    mags, nlev, _ = _class_arrays(m_max)
    if ((cid < 0) | (cid >= len(nlev))).any():
        raise ValueError("class id out of range")
    if (lv >= nlev[cid][:, None]).any() or (lv < 0).any():
        raise ValueError("level out of range")
    if (sm >> DIM).any():
        raise ValueError("sign mask has bits above coordinate 23")
    a = mags[cid[:, None], lv]
    neg = (sm[:, None] >> np.arange(DIM)) & 1
    if ((a == 0) & (neg == 1)).any():
        raise ValueError("sign bit set on a zero coordinate")
    z = np.where(neg == 1, -a, a)
    classes = ball_classes(m_max)
    want = np.array([c.mags_desc for c in classes], dtype=np.int64)[cid]
    if (-np.sort(-np.abs(z), axis=1) != want).any():
        raise ValueError("levels do not form the class's magnitude multiset")
    _check_membership(z)
    return z.astype(np.int8).reshape(shp + (DIM,))


def weights64(class_id, gain, scale_f16, z, centroids=(1.0, 1.0), m_max: int = BALL_M) -> np.ndarray:
    """f64 weights [M, Kpad] of a matrix of blocks (shape–gain, reading R8).

    class_id, gain, scale_f16: [M, nb]; z: int [M, nb, 24]; centroids: two f32
    values picked by the gain bit.  w = scale · centroid[g] · z / (4√m).
    """
    _, _, shell = _class_arrays(m_max)
    cid = np.asarray(class_id).astype(np.int64)
    g = np.asarray(gain).astype(np.int64)
    if ((g != 0) & (g != 1)).any():
        raise ValueError("gain bit must be 0 or 1")
    s = np.asarray(scale_f16, dtype=np.float16).astype(np.float64)
    cen = np.asarray(centroids, dtype=np.float32).astype(np.float64)
    norm = 4.0 * np.sqrt(shell[cid].astype(np.float64))
    factor = s * cen[g] / norm                                  # [M, nb]
    w = np.asarray(z).astype(np.float64) * factor[..., None]    # [M, nb, 24]
    M, nb = cid.shape
    return w.reshape(M, nb * DIM)


def gemv64(W64: np.ndarray, x_f16) -> np.ndarray:
    """y64 = W x in f64 with x converted exactly from fp16."""
    x = np.asarray(x_f16, dtype=np.float16).astype(np.float64)
    if W64.shape[1] != x.shape[0]:
        raise ValueError("shape mismatch")
    return W64 @ x


def gemv64_naive(W64: np.ndarray, x_f16) -> np.ndarray:
    """The same product as plain Python sums (for tiny matrices in tests)."""
    x = [float(v) for v in np.asarray(x_f16, dtype=np.float16).astype(np.float64)]
    return np.array([sum(float(w) * xv for w, xv in zip(row, x)) for row in W64])


def errors(y, y64, W64, x_f16) -> dict:
    """Both tolerance normalisations of reading R9, maxima over rows."""
    y = np.asarray(y, dtype=np.float64)
    x = np.asarray(x_f16, dtype=np.float16).astype(np.float64)
    d = np.abs(y - y64)
    rownorm = np.sqrt((W64 * W64).sum(axis=1))
    xnorm = float(np.sqrt((x * x).sum()))
    abssum = np.abs(W64) @ np.abs(x)
    with np.errstate(divide="ignore", invalid="ignore"):
        e_norm = np.where(rownorm * xnorm > 0, d / (rownorm * xnorm), np.where(d > 0, np.inf, 0.0))
        e_abs = np.where(abssum > 0, d / abssum, np.where(d > 0, np.inf, 0.0))
    return {"max_norm_err": float(e_norm.max(initial=0.0)),
            "max_abs_err": float(e_abs.max(initial=0.0))}


def row_norms_from_scales(class_id, gain, scale_f16, centroids=(1.0, 1.0)) -> np.ndarray:
    """‖W_r‖₂ without materialising W: every block's direction has unit norm
    (§2.3: every point of a shell has the same norm), so
    ‖W_r‖² = Σ_b (scale_b · centroid[g_b])²."""
    g = np.asarray(gain).astype(np.int64)
    s = np.asarray(scale_f16, dtype=np.float16).astype(np.float64)
    cen = np.asarray(centroids, dtype=np.float32).astype(np.float64)
    return np.sqrt(((s * cen[g]) ** 2).sum(axis=1))


def block_norm(z) -> float:
    return sqrt(float(sum(int(v) * int(v) for v in z)))


def weights64_from_points(z, gain, scale_f16, centroids=(1.0, 1.0)) -> np.ndarray:
    """Same weights as weights64, with each block's shell read off its point:
    Σ z_i² = 16 m (§2.1), so the norm 4√m is √(Σ z_i²).  Lets the oracle follow
    the full workload sizes without a per-block class lookup."""
    z = np.asarray(z).astype(np.int64)
    n2 = (z * z).sum(axis=-1)
    if (n2 % 16).any() or (n2 < 32).any() or (n2 > 16 * BALL_M).any():
        raise ValueError("a block is not a ball point")
    g = np.asarray(gain).astype(np.int64)
    s = np.asarray(scale_f16, dtype=np.float16).astype(np.float64)
    cen = np.asarray(centroids, dtype=np.float32).astype(np.float64)
    factor = s * cen[g] / np.sqrt(n2.astype(np.float64))
    w = z.astype(np.float64) * factor[..., None]
    M, nb = g.shape
    return w.reshape(M, nb * DIM)
