"""ctypes binding of libleech (include/leech.h): argument marshalling only.

Every step of the GEMV path runs in the library: host calls in its C++ half,
device calls in its HIP kernels.  PyTorch supplies device memory and streams.
If libleech.so is missing this module raises at import: there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libleech.so")

SLOT32, PLANES14, PLANES12X, GOLAY70 = 0, 1, 2, 3
LAYOUTS = {"slot32": SLOT32, "planes14": PLANES14, "planes12x": PLANES12X, "golay70": GOLAY70}
LAYOUT_NAMES = {v: k for k, v in LAYOUTS.items()}
TABLE_CLASS_LEVELS, TABLE_CODEWORDS, TABLE_DEVICE, TABLE_INDEX, TABLE_GOLAY_GEN = 0, 1, 2, 3, 4
INDEX_BITS = 47
ERRORS = {0: "OK", -1: "LEECH_E_ARG", -2: "LEECH_E_LAYOUT", -3: "LEECH_E_SHAPE",
          -4: "LEECH_E_FIELD", -5: "LEECH_E_NOT_LATTICE", -6: "LEECH_E_HIP",
          -7: "LEECH_E_CAPACITY"}
EXPORTS = ["leech_last_error", "leech_codebook_build", "leech_codebook_free",
           "leech_codebook_info", "leech_codebook_class", "leech_codebook_table",
           "leech_fields_from_points", "leech_expand_layout", "leech_layout_scales",
           "leech_host_decode_layout", "leech_gemv", "leech_gemv_grouped", "leech_decode_blocks",
           "leech_fp16_gemv_ref", "leech_noweights_ctrl", "leech_rotate_x",
           "leech_index_encode", "leech_index_decode", "leech_planes14_desc",
           "leech_transcode_planes14", "leech_set_exception_mode", "leech_gemv_batch",
           "leech_gemv_rotated", "leech_set_prologue_mode", "leech_set_batch_mode",
           "leech_expand_layout_tiled", "leech_layout_geometry", "leech_gemv_phases"]


class LeechError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class LayoutDesc(C.Structure):
    _fields_ = [("layout", C.c_int32), ("lane_cols", C.c_int32), ("tile_rows", C.c_int32),
                ("tile_exc_max", C.c_uint32), ("M", C.c_int64),
                ("Kpad", C.c_int64), ("nb", C.c_int64), ("main_bytes", C.c_uint64),
                ("side_bytes", C.c_uint64 * 2), ("n_exceptions", C.c_uint64),
                ("served_bytes", C.c_uint64)]

    def as_dict(self) -> dict:
        return {"layout": LAYOUT_NAMES.get(self.layout, self.layout), "lane_cols": self.lane_cols,
                "tile_rows": self.tile_rows, "M": self.M, "Kpad": self.Kpad, "nb": self.nb,
                "main_bytes": self.main_bytes,
                "side_bytes": [self.side_bytes[0], self.side_bytes[1]],
                "n_exceptions": self.n_exceptions, "served_bytes": self.served_bytes}


def _load() -> C.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2609_02652_amd.build` (no CPU fallback exists)")
    # The library must resolve its HIP runtime to the one PyTorch loaded, so
    # that PyTorch's device memory and streams are the library's: loaded the
    # other way round, the process holds two HIP runtimes and the library's
    # sees no device.  PyTorch is therefore loaded first when it is installed.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = C.CDLL(LIB_PATH)
    P, I64, U64, I, I32 = C.c_void_p, C.c_int64, C.c_uint64, C.c_int, C.c_int32
    sig = {
        "leech_last_error": (C.c_char_p, []),
        "leech_codebook_build": (I, [I, C.POINTER(P)]),
        "leech_codebook_free": (None, [P]),
        "leech_codebook_info": (I, [P, C.POINTER(I), C.POINTER(U64), C.POINTER(I)]),
        "leech_codebook_class": (I, [P, I, C.POINTER(I), C.POINTER(I), C.POINTER(I), P,
                                     C.POINTER(U64)]),
        "leech_codebook_table": (I, [P, I, C.POINTER(P), C.POINTER(C.c_size_t)]),
        "leech_fields_from_points": (I, [P, I64, P, P, P, P]),
        "leech_expand_layout": (I, [P, I, I64, I64, P, P, P, P, P, P, P, C.POINTER(LayoutDesc)]),
        "leech_expand_layout_tiled": (I, [P, I, I64, I64, I32, I32, P, P, P, P, P, P, P,
                                          C.POINTER(LayoutDesc)]),
        "leech_layout_geometry": (I, [I64, I64, C.POINTER(I32), C.POINTER(I32)]),
        "leech_layout_scales": (I, [C.POINTER(LayoutDesc), P, P]),
        "leech_host_decode_layout": (I, [P, C.POINTER(LayoutDesc), P, P, P, P, P, P]),
        "leech_gemv": (I, [C.POINTER(LayoutDesc), P, P, P, P, P, P, P, P, P, P]),
        "leech_gemv_phases": (I, [C.POINTER(LayoutDesc), P, P, P, P, P, P, P, P, P, P, P]),
        "leech_gemv_grouped": (I, [C.POINTER(LayoutDesc), P, P, P, P, P, P, I, P, P, P, P, P]),
        "leech_decode_blocks": (I, [C.POINTER(LayoutDesc), P, P, P, P, P, P, P, P, P]),
        "leech_fp16_gemv_ref": (I, [I64, I64, P, P, P, P]),
        "leech_noweights_ctrl": (I, [C.POINTER(LayoutDesc), P, P, P]),
        "leech_rotate_x": (I, [I64, I64, P, P, P, P, P]),
        "leech_index_encode": (I, [P, I64, P, P, P, P, P]),
        "leech_index_decode": (I, [P, I64, P, P, P, P, P]),
        "leech_planes14_desc": (I, [I64, I64, I32, I32, C.POINTER(LayoutDesc)]),
        "leech_transcode_planes14": (I, [C.POINTER(LayoutDesc), P, P, P, P, P]),
        "leech_set_exception_mode": (I, [I]),
        "leech_set_prologue_mode": (I, [I]),
        "leech_set_batch_mode": (I, [I]),
        "leech_gemv_batch": (I, [C.POINTER(LayoutDesc), P, P, P, P, P, P, P, I, P, I64, P, I64,
                                 P]),
        "leech_gemv_rotated": (I, [C.POINTER(LayoutDesc), P, P, P, P, P, P, I, P, P, I64, P, P,
                                   P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


def check(rc: int) -> None:
    if rc != 0:
        raise LeechError(rc, lib.leech_last_error().decode(errors="replace"))


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    if not a.flags["C_CONTIGUOUS"]:
        raise ValueError("array must be C-contiguous")
    return a.ctypes.data_as(C.c_void_p)


# ------------------------------------------------------------------ codebook
class Codebook:
    """Host codebook of the ball (leech_codebook_*)."""

    def __init__(self, ball_m: int = 12):
        h = C.c_void_p()
        check(lib.leech_codebook_build(ball_m, C.byref(h)))
        self._h = h
        self.ball_m = ball_m

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            lib.leech_codebook_free(h)
            self._h = None

    @property
    def handle(self):
        return self._h

    def info(self) -> dict:
        n, pts, bits = C.c_int(), C.c_uint64(), C.c_int()
        check(lib.leech_codebook_info(self._h, C.byref(n), C.byref(pts), C.byref(bits)))
        return {"n_classes": n.value, "n_points": pts.value, "index_bits": bits.value}

    def class_info(self, cid: int) -> dict:
        sh, par, nl, sz = C.c_int(), C.c_int(), C.c_int(), C.c_uint64()
        lv = (C.c_uint8 * 5)()
        check(lib.leech_codebook_class(self._h, cid, C.byref(sh), C.byref(par), C.byref(nl),
                                       C.cast(lv, C.c_void_p), C.byref(sz)))
        return {"shell": sh.value, "parity": par.value, "n_levels": nl.value,
                "levels": tuple(lv[: nl.value]), "size": sz.value}

    def table(self, which: int) -> np.ndarray:
        p, n = C.c_void_p(), C.c_size_t()
        check(lib.leech_codebook_table(self._h, which, C.byref(p), C.byref(n)))
        return np.ctypeslib.as_array(C.cast(p, C.POINTER(C.c_uint8)), shape=(n.value,)).copy()

    def fields_from_points(self, z: np.ndarray):
        z = np.ascontiguousarray(z, dtype=np.int8)
        shp = z.shape[:-1]
        n = int(np.prod(shp)) if shp else 1
        cls = np.empty(n, np.uint16)
        sm = np.empty(n, np.uint32)
        lv = np.empty((n, 24), np.uint8)
        check(lib.leech_fields_from_points(self._h, n, _ptr(z), _ptr(cls), _ptr(sm), _ptr(lv)))
        return cls.reshape(shp), sm.reshape(shp), lv.reshape(shp + (24,))


# ----------------------------------------------------- format-v1 block codes
def index_encode(cb: Codebook, class_id, gain, sign_mask, level) -> np.ndarray:
    """Decoded fields (any leading shape) -> u64 block codes of that shape."""
    class_id = np.ascontiguousarray(class_id, np.uint16)
    shp = class_id.shape
    n = class_id.size
    gain = np.ascontiguousarray(gain, np.uint8).reshape(n)
    sign_mask = np.ascontiguousarray(sign_mask, np.uint32).reshape(n)
    level = np.ascontiguousarray(level, np.uint8).reshape(n, 24)
    code = np.empty(n, np.uint64)
    check(lib.leech_index_encode(cb.handle, n, _ptr(class_id.reshape(n)), _ptr(gain),
                                 _ptr(sign_mask), _ptr(level), _ptr(code)))
    return code.reshape(shp)


def index_decode(cb: Codebook, code):
    """u64 block codes -> (class_id, gain, sign_mask, level[..., 24])."""
    code = np.ascontiguousarray(code, np.uint64)
    shp = code.shape
    n = code.size
    cls = np.empty(n, np.uint16)
    g = np.empty(n, np.uint8)
    sm = np.empty(n, np.uint32)
    lv = np.empty((n, 24), np.uint8)
    check(lib.leech_index_decode(cb.handle, n, _ptr(code.reshape(n)), _ptr(cls), _ptr(g),
                                 _ptr(sm), _ptr(lv)))
    return cls.reshape(shp), g.reshape(shp), sm.reshape(shp), lv.reshape(shp + (24,))


def layout_geometry(M: int, Kpad: int) -> tuple:
    """The library's (lane_cols, tile_rows) for an M × Kpad matrix."""
    c, r = C.c_int32(), C.c_int32()
    check(lib.leech_layout_geometry(M, Kpad, C.byref(c), C.byref(r)))
    return c.value, r.value


def planes14_desc(M: int, Kpad: int, geometry=None) -> LayoutDesc:
    """Planes14 descriptor; geometry = (lane_cols, tile_rows) or None for the
    library's choice."""
    lc, tr = geometry or (0, 0)
    d = LayoutDesc()
    check(lib.leech_planes14_desc(M, Kpad, lc, tr, C.byref(d)))
    return d


# ------------------------------------------------------------------- layouts
def expand_layout(cb: Codebook, layout: int, class_id, gain, sign_mask, level, geometry=None):
    """Fields (row-major [M, nb]) -> (desc, main, side0, side1) host byte arrays;
    geometry = (lane_cols, tile_rows), or None for the library's choice."""
    class_id = np.ascontiguousarray(class_id, np.uint16)
    gain = np.ascontiguousarray(gain, np.uint8)
    sign_mask = np.ascontiguousarray(sign_mask, np.uint32)
    level = np.ascontiguousarray(level, np.uint8)
    M, nb = class_id.shape
    d = LayoutDesc()
    lc, tr = geometry or (0, 0)
    args = (cb.handle, layout, M, nb * 24, lc, tr, _ptr(class_id), _ptr(gain), _ptr(sign_mask),
            _ptr(level))
    check(lib.leech_expand_layout_tiled(*args, None, None, None, C.byref(d)))
    main = np.zeros(d.main_bytes, np.uint8)
    s0 = np.zeros(max(d.side_bytes[0], 1), np.uint8)
    s1 = np.zeros(max(d.side_bytes[1], 1), np.uint8)
    check(lib.leech_expand_layout_tiled(*args, _ptr(main), _ptr(s0), _ptr(s1), C.byref(d)))
    return d, main, s0[: d.side_bytes[0]], s1[: d.side_bytes[1]]


def layout_scales(desc: LayoutDesc, scale_rowmajor: np.ndarray) -> np.ndarray:
    s = np.ascontiguousarray(scale_rowmajor, np.float16).view(np.uint16)
    out = np.empty(desc.M * desc.nb, np.uint16)
    check(lib.leech_layout_scales(C.byref(desc), _ptr(s), _ptr(out)))
    return out.view(np.float16)


def host_decode_layout(cb: Codebook, desc: LayoutDesc, main, side0, side1):
    n = desc.M * desc.nb
    z = np.empty((n, 24), np.int8)
    cls = np.empty(n, np.uint16)
    g = np.empty(n, np.uint8)
    s0 = _ptr(side0) if side0 is not None and side0.size else None
    s1 = _ptr(side1) if side1 is not None and side1.size else None
    check(lib.leech_host_decode_layout(cb.handle, C.byref(desc), _ptr(main), s0, s1,
                                       _ptr(z), _ptr(cls), _ptr(g)))
    shp = (desc.M, desc.nb)
    return z.reshape(shp + (24,)), cls.reshape(shp), g.reshape(shp)


# -------------------------------------------------------------- device calls
# Device pointers are integers (torch tensor .data_ptr()); stream is a raw
# hipStream_t integer (torch.cuda.Stream.cuda_stream) or 0.
def gemv(desc, d_main, d_side0, d_side1, d_table, d_codewords, d_scale, centroids, d_x, d_y,
         stream=0):
    cen = (C.c_float * 2)(float(centroids[0]), float(centroids[1]))
    check(lib.leech_gemv(C.byref(desc), d_main, d_side0 or None, d_side1 or None, d_table,
                         d_codewords or None, d_scale, C.cast(cen, C.c_void_p), d_x, d_y,
                         stream or None))


PHASE_STAMPS = 11


def gemv_phases(desc, d_main, d_side0, d_side1, d_table, d_codewords, d_scale, centroids, d_x,
                d_y, d_stamps, stream=0):
    cen = (C.c_float * 2)(float(centroids[0]), float(centroids[1]))
    check(lib.leech_gemv_phases(C.byref(desc), d_main, d_side0 or None, d_side1 or None, d_table,
                                d_codewords or None, d_scale, C.cast(cen, C.c_void_p), d_x, d_y,
                                d_stamps, stream or None))


def gemv_batch(desc, d_main, d_side0, d_side1, d_table, d_codewords, d_scale, centroids, batch,
               d_X, ldx, d_Y, ldy, stream=0):
    cen = (C.c_float * 2)(float(centroids[0]), float(centroids[1]))
    check(lib.leech_gemv_batch(C.byref(desc), d_main, d_side0 or None, d_side1 or None, d_table,
                               d_codewords or None, d_scale, C.cast(cen, C.c_void_p), batch, d_X,
                               ldx, d_Y, ldy, stream or None))


def gemv_rotated(desc, d_main, d_side0, d_side1, d_table, d_codewords, d_scale, group_rows,
                 group_centroids, K, d_x, d_signs, d_y, stream=0):
    n = len(group_rows)
    rows = (C.c_int64 * max(n, 1))(*[int(r) for r in group_rows])
    cen = (C.c_float * max(2 * n, 2))(*[float(c) for pair in group_centroids for c in pair])
    check(lib.leech_gemv_rotated(C.byref(desc), d_main, d_side0 or None, d_side1 or None, d_table,
                                 d_codewords or None, d_scale, n, C.cast(rows, C.c_void_p),
                                 C.cast(cen, C.c_void_p), K, d_x, d_signs or None, d_y,
                                 stream or None))


MAX_GROUPS = 8


def gemv_grouped(desc, d_main, d_side0, d_side1, d_table, d_codewords, d_scale, group_rows,
                 group_centroids, d_x, d_y, stream=0):
    n = len(group_rows)
    rows = (C.c_int64 * max(n, 1))(*[int(r) for r in group_rows])
    cen = (C.c_float * max(2 * n, 2))(*[float(c) for pair in group_centroids for c in pair])
    check(lib.leech_gemv_grouped(C.byref(desc), d_main, d_side0 or None, d_side1 or None,
                                 d_table, d_codewords or None, d_scale, n,
                                 C.cast(rows, C.c_void_p), C.cast(cen, C.c_void_p), d_x, d_y,
                                 stream or None))


def decode_blocks(desc, d_main, d_side0, d_side1, d_table, d_codewords, d_z, d_cls, d_gain,
                  stream=0):
    check(lib.leech_decode_blocks(C.byref(desc), d_main, d_side0 or None, d_side1 or None,
                                  d_table, d_codewords or None, d_z or None, d_cls or None,
                                  d_gain or None, stream or None))


def fp16_gemv_ref(M, K, d_W, d_x, d_y, stream=0):
    check(lib.leech_fp16_gemv_ref(M, K, d_W, d_x, d_y, stream or None))


def noweights_ctrl(desc, d_x, d_y, stream=0):
    check(lib.leech_noweights_ctrl(C.byref(desc), d_x, d_y, stream or None))


def rotate_x(K, Kpad, d_x, d_signs, d_xr, d_xr32=0, stream=0):
    check(lib.leech_rotate_x(K, Kpad, d_x, d_signs or None, d_xr, d_xr32 or None, stream or None))


def transcode_planes14(desc, d_index_table, d_code, d_main, d_bad, stream=0):
    check(lib.leech_transcode_planes14(C.byref(desc), d_index_table, d_code, d_main, d_bad,
                                       stream or None))


EXC_HOISTED, EXC_INLINE = 0, 1


def set_exception_mode(mode: int) -> None:
    """Process-wide: how Golay70 GEMVs enqueued afterwards decode exceptions."""
    check(lib.leech_set_exception_mode(mode))


BATCH_AUTO, BATCH_DOT2 = 0, 1


def set_batch_mode(mode: int) -> None:
    """Process-wide: the products of batched GEMVs enqueued afterwards
    (BATCH_AUTO: the matrix cores, 16-block 4x4x4 MFMAs; BATCH_DOT2: v_dot2,
    bit-identical to single GEMVs)."""
    check(lib.leech_set_batch_mode(mode))


PROLOGUE_AUTO = -1


def set_prologue_mode(mode: int) -> None:
    """Process-wide: the order in which single GEMVs enqueued afterwards request
    their records (PROLOGUE_AUTO, or 0, 1, 2); y does not depend on it."""
    check(lib.leech_set_prologue_mode(mode))
