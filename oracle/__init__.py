"""CPU oracle of the PIC synthesis decoder (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library neither imports nor
links it.  It wraps ``pic_oracle.c`` (the synthesis step: plain C, fp64 and an fp32
model), ``zpr_oracle.c`` (latents from the ZpR symbol stream, fp64) and
``huff_oracle.c`` (symbols from the Huffman bitstream) with numpy
marshalling; the arithmetic lives in the C files (see their headers).
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
    # latent decoding from the ZpR symbol stream (zpr_oracle.c)
    lib.pic_oracle_zigzag.restype = None
    lib.pic_oracle_zigzag.argtypes = [ctypes.c_void_p]
    lib.pic_oracle_zpr_blocks.restype = ctypes.c_long
    lib.pic_oracle_zpr_blocks.argtypes = [ctypes.c_int] * 3
    lib.pic_oracle_eob_offsets.restype = ctypes.c_long
    lib.pic_oracle_eob_offsets.argtypes = [ctypes.c_void_p, ctypes.c_long, ctypes.c_int32,
                                           ctypes.c_void_p, ctypes.c_long]
    lib.pic_oracle_expand_symbols.restype = ctypes.c_int
    lib.pic_oracle_expand_symbols.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                              ctypes.c_long, ctypes.c_void_p]
    lib.pic_oracle_idct8x8_f64.restype = None
    lib.pic_oracle_idct8x8_f64.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    lib.pic_oracle_unpatchify_f64.restype = ctypes.c_int
    lib.pic_oracle_unpatchify_f64.argtypes = [ctypes.c_int] * 4 + [ctypes.c_void_p, ctypes.c_void_p]
    lib.pic_oracle_zpr_decode_f64.restype = ctypes.c_int
    lib.pic_oracle_zpr_decode_f64.argtypes = [ctypes.c_int] * 4 + [ctypes.c_void_p, ctypes.c_long,
                                                                    ctypes.c_int32, ctypes.c_void_p]
    # entropy decoding (huff_oracle.c)
    lib.pic_oracle_huffman_codes.restype = ctypes.c_int
    lib.pic_oracle_huffman_codes.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    lib.pic_oracle_huffman_decode.restype = ctypes.c_int
    lib.pic_oracle_huffman_decode.argtypes = [ctypes.c_void_p, ctypes.c_long, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_int, ctypes.c_long, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_void_p]
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

    # ---------------------------------------------- ZpR stream -> latents

    def zigzag(self) -> np.ndarray:
        """JPEG zigzag scan: entry p is the row-major index of the p-th coefficient."""
        zz = np.empty(64, dtype=np.int32)
        self._lib.pic_oracle_zigzag(zz.ctypes.data)
        return zz

    def zpr_blocks(self, H: int, W: int, L: int) -> int:
        """8x8 blocks of one image's pyramid."""
        return int(self._lib.pic_oracle_zpr_blocks(H, W, L))

    def eob_offsets(self, symbols, eob: int) -> np.ndarray:
        """Positions of the eob markers in the stream (the copy_if step)."""
        s = np.ascontiguousarray(symbols, dtype=np.int32)
        n = int(self._lib.pic_oracle_eob_offsets(s.ctypes.data, s.size, int(eob), None, 0))
        off = np.empty(max(n, 1), dtype=np.int64)
        self._lib.pic_oracle_eob_offsets(s.ctypes.data, s.size, int(eob), off.ctypes.data, n)
        return off[:n]

    def expand_symbols(self, symbols, eob: int, offsets) -> tuple:
        """Alg. 1 over every block the offsets delimit: (coefficients int32
        [n_blocks][64] row-major, error flags)."""
        s = np.ascontiguousarray(symbols, dtype=np.int32)
        off = np.ascontiguousarray(offsets, dtype=np.int64)
        co = np.empty((max(off.size, 1), 64), dtype=np.int32)
        err = self._lib.pic_oracle_expand_symbols(s.ctypes.data, int(eob), off.ctypes.data, off.size,
                                                  co.ctypes.data)
        return co[:off.size], int(err)

    def idct8x8(self, S) -> np.ndarray:
        """Orthonormal 8x8 inverse DCT of one coefficient block (fp64 [8][8])."""
        S = np.ascontiguousarray(S, dtype=np.float64).reshape(64)
        f = np.empty(64, dtype=np.float64)
        self._lib.pic_oracle_idct8x8_f64(S.ctypes.data, f.ctypes.data)
        return f.reshape(8, 8)

    def _split_levels(self, flat, H, W, L, batch):
        out, o = [], 0
        for k in range(L):
            h, w = self.level_dim(H, k), self.level_dim(W, k)
            out.append(flat[o:o + batch * h * w].reshape(batch, h, w))
            o += batch * h * w
        return out

    def _level_total(self, H, W, L, batch):
        return sum(batch * self.level_dim(H, k) * self.level_dim(W, k) for k in range(L))

    def unpatchify(self, blocks, H: int, W: int, L: int, batch: int) -> list:
        """Place [n_blocks][64] fp64 samples into the L grids [batch][h_k][w_k]."""
        bl = np.ascontiguousarray(blocks, dtype=np.float64)
        if bl.size != 64 * batch * self.zpr_blocks(H, W, L):
            raise ValueError("block count does not match the pyramid")
        flat = np.zeros(self._level_total(H, W, L, batch), dtype=np.float64)
        if self._lib.pic_oracle_unpatchify_f64(H, W, L, batch, bl.ctypes.data, flat.ctypes.data):
            raise ValueError("oracle rejected the arguments")
        return self._split_levels(flat, H, W, L, batch)

    def zpr_decode(self, symbols, eob: int, H: int, W: int, L: int, batch: int, fill=0.0) -> tuple:
        """The whole step: (L fp64 grids [batch][h_k][w_k], error flags).
        Grid samples no decoded block covers keep ``fill``."""
        s = np.ascontiguousarray(symbols, dtype=np.int32)
        flat = np.full(self._level_total(H, W, L, batch), fill, dtype=np.float64)
        err = self._lib.pic_oracle_zpr_decode_f64(H, W, L, batch, s.ctypes.data, s.size, int(eob),
                                                  flat.ctypes.data)
        if err < 0:
            raise ValueError("oracle rejected the arguments")
        return self._split_levels(flat, H, W, L, batch), int(err)

    # ---------------------------------------------- Huffman bitstream -> symbols

    def huffman_codes(self, lengths) -> tuple:
        """Canonical codes of the given lengths: (codes uint32 [n], error flags)."""
        ln = np.ascontiguousarray(lengths, dtype=np.uint8)
        codes = np.zeros(max(ln.size, 1), dtype=np.uint32)
        err = self._lib.pic_oracle_huffman_codes(ln.ctypes.data, ln.size, codes.ctypes.data)
        return codes[:ln.size], int(err)

    def huffman_decode(self, data, n_bits: int, values, lengths, n_out: int) -> tuple:
        """Decode n_out symbols from the MSB-first bitstream `data` (bytes or
        uint8 array; its first n_bits bits): (symbols int32 [decoded], error
        flags, bits used)."""
        buf = np.frombuffer(bytes(data), dtype=np.uint8) if not isinstance(data, np.ndarray) else \
            np.ascontiguousarray(data, dtype=np.uint8)
        vals = np.ascontiguousarray(values, dtype=np.int32)
        ln = np.ascontiguousarray(lengths, dtype=np.uint8)
        out = np.zeros(max(int(n_out), 1), dtype=np.int32)
        nd, used = ctypes.c_long(0), ctypes.c_long(0)
        err = self._lib.pic_oracle_huffman_decode(buf.ctypes.data if buf.size else None, int(n_bits),
                                                  vals.ctypes.data, ln.ctypes.data, ln.size, int(n_out),
                                                  out.ctypes.data, ctypes.byref(nd), ctypes.byref(used))
        return out[:nd.value], int(err), int(used.value)

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
    """The oracle built from oracle/pic_oracle.c (built on first use).  The
    environment variable PIC_ORACLE_LIB names another build of the same
    sources to use instead (the sanitizer test's)."""
    global _default
    if _default is None:
        alt = os.environ.get("PIC_ORACLE_LIB")
        if alt:
            _default = Oracle(alt)
        else:
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


def zpr_decode(*a, **kw):
    return default().zpr_decode(*a, **kw)
