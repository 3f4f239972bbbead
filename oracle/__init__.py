"""CPU oracle of the PIC synthesis decoder (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library neither imports nor
links it.  It wraps ``pic_oracle.c`` (plain C, fp64 and an fp32 model, see that
file's header) with numpy marshalling; the arithmetic lives in the C file.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

import numpy as np

from . import build as _build

OUT_RAW, OUT_CLAMPED, OUT_U8 = 0, 1, 2


def _bind(path):
    lib = ctypes.CDLL(path)
    # (H, W, L, nl, widths, batch, latents, weights, is_bf16, w_stride,
    #  biases, b_stride, out_kind, out, nthreads, y_begin, y_end)
    argt = [ctypes.c_int] * 4 + [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_int, ctypes.c_long,
                                 ctypes.c_void_p, ctypes.c_long,
                                 ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                                 ctypes.c_int, ctypes.c_int]
    for name in ("pic_oracle_decode_f64", "pic_oracle_decode_f32"):
        fn = getattr(lib, name)
        fn.restype = ctypes.c_int
        fn.argtypes = argt
    lib.pic_oracle_upsample_f64.restype = ctypes.c_int
    lib.pic_oracle_upsample_f64.argtypes = [ctypes.c_int] * 4 + [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
    lib.pic_oracle_fuse_modulation_f64.restype = ctypes.c_int
    lib.pic_oracle_fuse_modulation_f64.argtypes = [ctypes.c_int, ctypes.c_int] + [ctypes.c_void_p] * 8
    lib.pic_oracle_level_dim.restype = ctypes.c_int
    lib.pic_oracle_level_dim.argtypes = [ctypes.c_int, ctypes.c_int]
    return lib


class Oracle:
    """numpy front end of one build of pic_oracle.c."""

    def __init__(self, path: str):
        self.path = path
        self._lib = _bind(path)

    def level_dim(self, n: int, k: int) -> int:
        return self._lib.pic_oracle_level_dim(n, k)

    def _latent_ptrs(self, latents, batch, H, W):
        L = len(latents)
        arrs = []
        for k, a in enumerate(latents):
            a = np.ascontiguousarray(a, dtype=np.float32)
            want = (batch, self.level_dim(H, k), self.level_dim(W, k))
            if a.shape != want:
                raise ValueError(f"level {k}: shape {a.shape}, expected {want}")
            arrs.append(a)
        ptrs = (ctypes.c_void_p * L)(*[a.ctypes.data for a in arrs])
        return arrs, ptrs

    def upsample(self, latents: Sequence[np.ndarray], height: int, width: int,
                 nthreads: int = 0) -> np.ndarray:
        """fp64 upsampled pyramid [batch][L][H][W] (channel k = level k)."""
        batch = latents[0].shape[0]
        keep, ptrs = self._latent_ptrs(latents, batch, height, width)
        out = np.empty((batch, len(latents), height, width), dtype=np.float64)
        rc = self._lib.pic_oracle_upsample_f64(height, width, len(latents), batch, ptrs,
                                               out.ctypes.data, nthreads)
        if rc:
            raise ValueError("oracle rejected the arguments")
        del keep
        return out

    def decode(self, latents: Sequence[np.ndarray], weights: np.ndarray, biases: np.ndarray,
               widths: Sequence[int], height: int, width: int, out: str = "clamped",
               precision: str = "f64", weights_bf16: np.ndarray = None,
               shared: bool = False, nthreads: int = 0, rows: tuple = None) -> np.ndarray:
        """Decode a batch on the CPU.

        latents: L float32 arrays [batch][H_k][W_k]; weights float32 [batch][nw]
        (or [nw] with ``shared``); biases float32 [batch][nb] (or [nb]);
        ``weights_bf16`` (uint16 bit patterns, same shape as weights) replaces
        the float32 weights when given.  ``out`` is "raw", "clamped" or "u8";
        ``precision`` is "f64" (the definition) or "f32" (binary32 model).
        ``rows`` = (y_begin, y_end) computes only those output rows.
        Returns [batch][3][rows][W] float64 / float32 / uint8.
        """
        widths = [int(w) for w in widths]
        L, nl = len(latents), len(widths) - 1
        batch = latents[0].shape[0]
        keep, ptrs = self._latent_ptrs(latents, batch, height, width)
        if weights_bf16 is not None:
            w = np.ascontiguousarray(weights_bf16, dtype=np.uint16)
            is_bf16 = 1
        else:
            w = np.ascontiguousarray(weights, dtype=np.float32)
            is_bf16 = 0
        b = np.ascontiguousarray(biases, dtype=np.float32)
        nw = sum(widths[i] * widths[i + 1] for i in range(nl))
        nb = sum(widths[1:])
        if shared:
            w_stride = b_stride = 0
            if w.reshape(-1).size < nw or b.reshape(-1).size < nb:
                raise ValueError("parameter arrays too small")
        else:
            w_stride, b_stride = nw, nb
            if w.shape != (batch, nw) or b.shape != (batch, nb):
                raise ValueError(f"weights {w.shape} / biases {b.shape}, "
                                 f"expected ({batch},{nw}) / ({batch},{nb})")
        kind = {"raw": OUT_RAW, "clamped": OUT_CLAMPED, "u8": OUT_U8}[out]
        if kind == OUT_U8:
            dt = np.uint8
        else:
            dt = np.float64 if precision == "f64" else np.float32
        y0, y1 = (0, height) if rows is None else (int(rows[0]), int(rows[1]))
        res = np.empty((batch, 3, max(0, y1 - y0), width), dtype=dt)
        wid = (ctypes.c_int * len(widths))(*widths)
        fn = {"f64": self._lib.pic_oracle_decode_f64,
              "f32": self._lib.pic_oracle_decode_f32}[precision]
        rc = fn(height, width, L, nl, wid, batch, ptrs, w.ctypes.data, is_bf16, w_stride,
                b.ctypes.data, b_stride, kind, res.ctypes.data, nthreads, y0, y1)
        if rc:
            raise ValueError("oracle rejected the arguments")
        del keep
        return res

    def fuse_modulation(self, W, b, gamma, beta, mu, sigma):
        """App. A fusion for one image (W [out][in]); returns (W', b') in fp64."""
        W = np.ascontiguousarray(W, dtype=np.float32)
        out, fin = W.shape
        arrs = [np.ascontiguousarray(a, dtype=np.float32) for a in (b, gamma, beta, mu, sigma)]
        wf = np.empty((out, fin), dtype=np.float64)
        bf = np.empty(out, dtype=np.float64)
        rc = self._lib.pic_oracle_fuse_modulation_f64(fin, out, W.ctypes.data, *[a.ctypes.data for a in arrs],
                                                      wf.ctypes.data, bf.ctypes.data)
        if rc:
            raise ValueError("oracle rejected the arguments")
        return wf, bf

    def decode_inputs(self, inp, out: str = "clamped", precision: str = "f64",
                      nthreads: int = 0, batch_slice: slice = None, rows: tuple = None) -> np.ndarray:
        """decode() on a synth.Inputs bundle (optionally some images / rows)."""
        sl = batch_slice or slice(None)
        lat = [a[sl] for a in inp.latents]
        wb = inp.weights_bf16[sl] if inp.weights_bf16 is not None else None
        return self.decode(lat, inp.weights[sl], inp.biases[sl], inp.widths, inp.height,
                           inp.width, out=out, precision=precision, weights_bf16=wb,
                           nthreads=nthreads, rows=rows)


_default = None


def default() -> Oracle:
    """The oracle built from oracle/pic_oracle.c (built on first use)."""
    global _default
    if _default is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _default = Oracle(_build.LIB)
    return _default


def level_dim(n, k):
    return default().level_dim(n, k)


def upsample(*a, **kw):
    return default().upsample(*a, **kw)


def decode(*a, **kw):
    return default().decode(*a, **kw)


def decode_inputs(*a, **kw):
    return default().decode_inputs(*a, **kw)


def fuse_modulation(*a, **kw):
    return default().fuse_modulation(*a, **kw)
