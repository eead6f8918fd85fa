"""MI355X-native fused Λ24(12) dequantize + GEMV (batch-1 decode).

The compute path lives in libleech.so (include/leech.h): a C++ host half
(codebook, decoded fields, offline layout expansion) and HIP kernels for
gfx950 (fused GEMV per layout, verification decode, FP16 and no-weights
controls).  This package is its thin binding; PyTorch only provides device
memory and streams.  Importing it fails loudly if the library is not built.
"""
from __future__ import annotations

import numpy as np

from . import _lib
from ._lib import (GOLAY70, LAYOUT_NAMES, LAYOUTS, PLANES12X, PLANES14, SLOT32, Codebook,
                   LayoutDesc, LeechError, expand_layout, host_decode_layout, index_decode,
                   index_encode, layout_geometry, layout_scales, planes14_desc,
                   set_exception_mode,
                   EXC_HOISTED, EXC_INLINE, set_prologue_mode, PROLOGUE_AUTO,
                   set_batch_mode, BATCH_AUTO, BATCH_DOT2)

__all__ = ["Codebook", "DeviceCodebook", "LeechMatrix", "LayoutDesc", "LeechError", "LAYOUTS",
           "LAYOUT_NAMES", "SLOT32", "PLANES14", "PLANES12X", "GOLAY70", "expand_layout",
           "host_decode_layout", "layout_scales", "fp16_gemv", "noweights_ctrl", "rotate_x",
           "index_encode", "index_decode", "planes14_desc", "layout_geometry", "set_exception_mode",
           "EXC_HOISTED", "EXC_INLINE", "set_prologue_mode", "PROLOGUE_AUTO",
           "set_batch_mode", "BATCH_AUTO", "BATCH_DOT2"]


def _torch():
    import torch
    return torch


def _stream(stream):
    torch = _torch()
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dev(arr: np.ndarray, device):
    torch = _torch()
    t = torch.from_numpy(np.ascontiguousarray(arr).view(np.uint8))
    return t.to(device)


class DeviceCodebook:
    """Device copies of the class table, the Golay codeword and generator
    tables and the format-v1 index table."""

    def __init__(self, cb: Codebook, device="cuda"):
        self.cb = cb
        self.table = _dev(cb.table(_lib.TABLE_DEVICE), device)
        self.codewords = _dev(cb.table(_lib.TABLE_CODEWORDS), device)
        self.golay_gen = _dev(cb.table(_lib.TABLE_GOLAY_GEN), device)
        self.index = _dev(cb.table(_lib.TABLE_INDEX), device)


class LeechMatrix:
    """One Leech-coded matrix resident in device memory in one layout."""

    def __init__(self, desc: LayoutDesc, main, side0, side1, scale, dcb: DeviceCodebook):
        self.desc, self.main, self.side0, self.side1, self.scale, self.dcb = (
            desc, main, side0, side1, scale, dcb)

    @classmethod
    def from_fields(cls, dcb: DeviceCodebook, layout: int, class_id, gain, sign_mask, level,
                    scale_rowmajor, device="cuda", geometry=None):
        """Expand decoded fields into `layout` (geometry: (lane_cols, tile_rows),
        or None for the library's choice) and upload the streams."""
        desc, main, s0, s1 = expand_layout(dcb.cb, layout, class_id, gain, sign_mask, level,
                                           geometry)
        sc = layout_scales(desc, scale_rowmajor)
        torch = _torch()
        empty = torch.empty(0, dtype=torch.uint8, device=device)
        return cls(desc, _dev(main, device), _dev(s0, device) if s0.size else empty,
                   _dev(s1, device) if s1.size else empty, _dev(sc, device), dcb)

    @classmethod
    def from_codes(cls, dcb: DeviceCodebook, codes, scale_rowmajor, stream=None):
        """Planes14 matrix from format-v1 block codes, transcoded on the device
        (§2.2): codes is an int64 device tensor [M, nb] holding the u64 codes;
        scale_rowmajor the fp16 block scales [M, nb] (host)."""
        torch = _torch()
        if codes.dtype != torch.int64 or codes.dim() != 2 or not codes.is_contiguous():
            raise ValueError("codes must be a contiguous int64 tensor [M, nb]")
        M, nb = codes.shape
        desc = planes14_desc(M, nb * 24)
        dev = codes.device
        main = torch.empty(desc.main_bytes, dtype=torch.uint8, device=dev)
        bad = torch.empty(1, dtype=torch.int32, device=dev)
        _lib.transcode_planes14(desc, dcb.index.data_ptr(), codes.data_ptr(), main.data_ptr(),
                                bad.data_ptr(), _stream(stream))
        n_bad = int(bad.item())
        if n_bad:
            raise LeechError(-4, f"{n_bad} of {M * nb} block codes are not format-v1 codes")
        sc = layout_scales(desc, scale_rowmajor)
        empty = torch.empty(0, dtype=torch.uint8, device=dev)
        return cls(desc, main, empty, empty, _dev(sc, dev), dcb)

    @property
    def M(self):
        return self.desc.M

    @property
    def Kpad(self):
        return self.desc.Kpad

    def _ptrs(self):
        return (self.main.data_ptr(), self.side0.data_ptr() if self.side0.numel() else 0,
                self.side1.data_ptr() if self.side1.numel() else 0)

    def gemv(self, x, y=None, centroids=(1.0, 1.0), stream=None):
        """y = W x; x: fp16 [Kpad] device tensor, y: f32 [M] device tensor."""
        torch = _torch()
        if x.dtype != torch.float16 or x.numel() != self.Kpad or not x.is_contiguous():
            raise ValueError("x must be a contiguous fp16 tensor of length Kpad")
        if y is None:
            y = torch.empty(self.M, dtype=torch.float32, device=x.device)
        elif y.dtype != torch.float32 or y.numel() != self.M or not y.is_contiguous():
            raise ValueError("y must be a contiguous f32 tensor of length M")
        m, s0, s1 = self._ptrs()
        _lib.gemv(self.desc, m, s0, s1, self.dcb.table.data_ptr(), self.dcb.golay_gen.data_ptr(),
                  self.scale.data_ptr(), centroids, x.data_ptr(), y.data_ptr(), _stream(stream))
        return y

    def gemv_phases(self, x, y, stamps, centroids=(1.0, 1.0), stream=None):
        """gemv with per-workgroup phase stamps (leech_gemv_phases): stamps is a
        contiguous int64 device tensor of at least 11 · tiles entries."""
        torch = _torch()
        tiles = -(-self.M // self.desc.tile_rows)
        if (stamps.dtype != torch.int64 or not stamps.is_contiguous()
                or stamps.numel() < _lib.PHASE_STAMPS * tiles):
            raise ValueError("stamps must be a contiguous int64 tensor of 11 * tiles entries")
        if x.dtype != torch.float16 or x.numel() != self.Kpad or not x.is_contiguous():
            raise ValueError("x must be a contiguous fp16 tensor of length Kpad")
        if y.dtype != torch.float32 or y.numel() != self.M or not y.is_contiguous():
            raise ValueError("y must be a contiguous f32 tensor of length M")
        m, s0, s1 = self._ptrs()
        _lib.gemv_phases(self.desc, m, s0, s1, self.dcb.table.data_ptr(),
                         self.dcb.golay_gen.data_ptr(), self.scale.data_ptr(), centroids,
                         x.data_ptr(), y.data_ptr(), stamps.data_ptr(), _stream(stream))
        return y

    def gemv_batch(self, X, Y=None, centroids=(1.0, 1.0), stream=None):
        """Y[b] = W X[b]: X fp16 [B, Kpad] device tensor (row stride a multiple
        of 8), Y f32 [B, M]; each block decoded once for up to 16 activations,
        multiplied on the matrix cores or with v_dot2 (set_batch_mode)."""
        torch = _torch()
        if X.dtype != torch.float16 or X.dim() != 2 or X.shape[1] != self.Kpad or X.stride(1) != 1:
            raise ValueError("X must be an fp16 [B, Kpad] tensor with unit column stride")
        B = X.shape[0]
        if Y is None:
            Y = torch.empty((B, self.M), dtype=torch.float32, device=X.device)
        elif Y.dtype != torch.float32 or Y.shape != (B, self.M) or Y.stride(1) != 1:
            raise ValueError("Y must be an f32 [B, M] tensor with unit column stride")
        m, s0, s1 = self._ptrs()
        _lib.gemv_batch(self.desc, m, s0, s1, self.dcb.table.data_ptr(),
                        self.dcb.golay_gen.data_ptr(), self.scale.data_ptr(), centroids, B,
                        X.data_ptr(), X.stride(0), Y.data_ptr(), Y.stride(0), _stream(stream))
        return Y

    def gemv_grouped(self, x, group_rows, group_centroids, y=None, stream=None):
        """y = W x for a row concatenation of matrices sharing x (§3.4): group g
        covers the next group_rows[g] rows and uses gain centroids
        group_centroids[g] = (c0, c1); group boundaries are multiples of 64 rows."""
        torch = _torch()
        if x.dtype != torch.float16 or x.numel() != self.Kpad or not x.is_contiguous():
            raise ValueError("x must be a contiguous fp16 tensor of length Kpad")
        if y is None:
            y = torch.empty(self.M, dtype=torch.float32, device=x.device)
        elif y.dtype != torch.float32 or y.numel() != self.M or not y.is_contiguous():
            raise ValueError("y must be a contiguous f32 tensor of length M")
        m, s0, s1 = self._ptrs()
        _lib.gemv_grouped(self.desc, m, s0, s1, self.dcb.table.data_ptr(),
                          self.dcb.golay_gen.data_ptr(), self.scale.data_ptr(), group_rows,
                          group_centroids, x.data_ptr(), y.data_ptr(), _stream(stream))
        return y

    def gemv_rotated(self, x, signs=None, group_rows=None, group_centroids=((1.0, 1.0),), y=None,
                     stream=None):
        """y = W · R(x) in one launch: x the raw fp16 activation [K] (K ≤ Kpad,
        a multiple of 8), signs int8 ±1 [K] or None; R is rotate_x's rotation,
        done by each workgroup in LDS.  Row groups as gemv_grouped (None: one
        group of all rows)."""
        torch = _torch()
        if x.dtype != torch.float16 or x.dim() != 1 or not x.is_contiguous():
            raise ValueError("x must be a contiguous 1-D fp16 tensor")
        K = x.numel()
        if signs is not None and (signs.dtype != torch.int8 or signs.numel() != K
                                  or not signs.is_contiguous()):
            raise ValueError("signs must be a contiguous int8 tensor of length K")
        if y is None:
            y = torch.empty(self.M, dtype=torch.float32, device=x.device)
        rows = [self.M] if group_rows is None else group_rows
        m, s0, s1 = self._ptrs()
        _lib.gemv_rotated(self.desc, m, s0, s1, self.dcb.table.data_ptr(),
                          self.dcb.golay_gen.data_ptr(), self.scale.data_ptr(), rows,
                          group_centroids, K, x.data_ptr(),
                          signs.data_ptr() if signs is not None else 0, y.data_ptr(),
                          _stream(stream))
        return y

    def decode(self, stream=None):
        """Device decode: (z int8 [M, nb, 24], class_id int16 [M, nb], gain uint8 [M, nb])."""
        torch = _torch()
        M, nb = self.desc.M, self.desc.nb
        dev = self.main.device
        z = torch.empty((M, nb, 24), dtype=torch.int8, device=dev)
        c = torch.empty((M, nb), dtype=torch.int16, device=dev)
        g = torch.empty((M, nb), dtype=torch.uint8, device=dev)
        m, s0, s1 = self._ptrs()
        _lib.decode_blocks(self.desc, m, s0, s1, self.dcb.table.data_ptr(),
                           self.dcb.golay_gen.data_ptr(), z.data_ptr(), c.data_ptr(), g.data_ptr(),
                           _stream(stream))
        return z, c, g


def fp16_gemv(W, x, y=None, stream=None):
    """FP16 GEMV control: W fp16 [M, K] (K % 8 == 0), x fp16 [K] -> y f32 [M]."""
    torch = _torch()
    M, K = W.shape
    if W.dtype != torch.float16 or x.dtype != torch.float16 or not W.is_contiguous():
        raise ValueError("W and x must be contiguous fp16")
    if y is None:
        y = torch.empty(M, dtype=torch.float32, device=W.device)
    _lib.fp16_gemv_ref(M, K, W.data_ptr(), x.data_ptr(), y.data_ptr(), _stream(stream))
    return y


def noweights_ctrl(desc: LayoutDesc, x, y=None, stream=None):
    """No-weights control over the GEMV geometry of desc: y[r] = Σ x."""
    torch = _torch()
    if y is None:
        y = torch.empty(desc.M, dtype=torch.float32, device=x.device)
    _lib.noweights_ctrl(desc, x.data_ptr(), y.data_ptr(), _stream(stream))
    return y


def rotate_x(x, signs=None, Kpad=None, with_f32=False, out=None, stream=None):
    """Blockwise Walsh–Hadamard rotation of an fp16 activation (§2.3, §6):
    x fp16 [K], signs int8 ±1 [K] (None: all +1) -> fp16 [Kpad] (zero past K),
    and the f32 values before rounding when with_f32.  `out` (fp16 [Kpad],
    contiguous) receives the result in place of a new tensor."""
    torch = _torch()
    if x.dtype != torch.float16 or x.dim() != 1 or not x.is_contiguous():
        raise ValueError("x must be a contiguous 1-D fp16 tensor")
    K = x.numel()
    Kpad = K if Kpad is None else int(Kpad)
    if signs is not None and (signs.dtype != torch.int8 or signs.numel() != K
                              or not signs.is_contiguous()):
        raise ValueError("signs must be a contiguous int8 tensor of length K")
    if out is None:
        xr = torch.empty(Kpad, dtype=torch.float16, device=x.device)
    else:
        if (out.dtype != torch.float16 or out.dim() != 1 or out.numel() != Kpad
                or not out.is_contiguous() or out.device != x.device):
            raise ValueError("out must be a contiguous fp16 tensor of length Kpad on x's device")
        xr = out
    xr32 = torch.empty(K, dtype=torch.float32, device=x.device) if with_f32 else None
    _lib.rotate_x(K, Kpad, x.data_ptr(), signs.data_ptr() if signs is not None else 0,
                  xr.data_ptr(), xr32.data_ptr() if with_f32 else 0, _stream(stream))
    return (xr, xr32) if with_f32 else xr
