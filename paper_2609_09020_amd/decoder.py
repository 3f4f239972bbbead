"""Thin ctypes binding of libpic_decode.so (include/pic_decode.h).

The ``pic_decode_*``, ``pic_zpr_*``, ``pic_huff_*``, ``pic_fuse_modulation`` and
``pic_status_string`` functions mirror the C entry points one to one and only
marshal arguments; every step runs in the HIP kernels behind them.
``Decoder`` (synthesis), ``ZprDecoder`` (latents from the ZpR symbol stream)
and ``HuffDecoder`` (ZpR symbols from the Huffman bitstream) wrap handles for
use with torch tensors (torch supplies device memory and streams, nothing
else).

There is no fallback: if the library is missing or fails to load, every call
raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libpic_decode.so")

PIC_OK, PIC_E_INVALID, PIC_E_UNSUPPORTED, PIC_E_NODEVICE, PIC_E_HIP, PIC_E_NOMEM = range(6)
PIC_F32, PIC_BF16, PIC_U8 = 0, 1, 2
PIC_VARIANT_AUTO, PIC_VARIANT_VALU, PIC_VARIANT_MFMA_F32, PIC_VARIANT_MFMA_BF16, PIC_VARIANT_MFMA_F16X3 = range(5)
PIC_MAX_LEVELS, PIC_MAX_LAYERS, PIC_MAX_WIDTH, PIC_MAX_BATCH = 12, 8, 128, 65535
PIC_NOALLOC_MAX_BATCH = 4096
PIC_FLAG_NO_CLAMP = 1

VARIANTS = {"auto": PIC_VARIANT_AUTO, "valu": PIC_VARIANT_VALU,
            "mfma_f32": PIC_VARIANT_MFMA_F32, "mfma_bf16": PIC_VARIANT_MFMA_BF16,
            "mfma_f16x3": PIC_VARIANT_MFMA_F16X3}
VARIANT_NAMES = {v: k for k, v in VARIANTS.items()}

# Every symbol include/pic_decode.h and include/pic_zpr.h declare.
EXPORTS = ("pic_decode_create", "pic_decode_run", "pic_decode_run_noalloc", "pic_decode_run_layers",
           "pic_decode_query", "pic_decode_destroy", "pic_status_string", "pic_fuse_modulation",
           "pic_zpr_create", "pic_zpr_decode", "pic_zpr_expand", "pic_zpr_query", "pic_zpr_destroy",
           "pic_huff_create", "pic_huff_decode", "pic_huff_query", "pic_huff_destroy")

PIC_HUFF_ERR_BITS, PIC_HUFF_ERR_CODE, PIC_HUFF_ERR_TABLE = 1, 2, 4
PIC_HUFF_MAX_LEN, PIC_HUFF_MAX_TABLE = 24, 4096

PIC_ZPR_ERR_COUNT, PIC_ZPR_ERR_OVERFLOW, PIC_ZPR_ERR_SYMBOL = 1, 2, 4


class pic_decode_desc(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32),
                ("height", ctypes.c_int32), ("width", ctypes.c_int32),
                ("num_levels", ctypes.c_int32), ("num_layers", ctypes.c_int32),
                ("widths", ctypes.c_int32 * (PIC_MAX_LAYERS + 1)),
                ("weight_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("max_batch", ctypes.c_int32),
                ("variant", ctypes.c_int32)]


class pic_decode_info(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("variant", ctypes.c_int32),
                ("weights_per_image", ctypes.c_int64), ("biases_per_image", ctypes.c_int64),
                ("device", ctypes.c_int32), ("pixels_per_wave_step", ctypes.c_int32),
                ("kernel_name", ctypes.c_char * 64)]


class pic_zpr_desc(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("height", ctypes.c_int32), ("width", ctypes.c_int32),
                ("num_levels", ctypes.c_int32), ("max_batch", ctypes.c_int32)]


class pic_zpr_info(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("device", ctypes.c_int32),
                ("blocks_per_image", ctypes.c_int64), ("max_symbols", ctypes.c_int64),
                ("scratch_bytes", ctypes.c_int64), ("symbols_per_chunk", ctypes.c_int32)]


class pic_huff_desc(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("reserved", ctypes.c_int32), ("max_bits", ctypes.c_int64)]


class pic_huff_info(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("device", ctypes.c_int32), ("max_bits", ctypes.c_int64),
                ("scratch_bytes", ctypes.c_int64), ("bits_per_thread", ctypes.c_int32),
                ("lut_bits", ctypes.c_int32)]


class PicError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {pic_status_string(status)} (status {status})")


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libpic_decode.so; raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2609_09020_amd.build` "
                           "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(path)
    lib.pic_decode_create.restype = ctypes.c_int
    lib.pic_decode_create.argtypes = [ctypes.POINTER(pic_decode_desc), ctypes.POINTER(ctypes.c_void_p)]
    lib.pic_decode_run.restype = ctypes.c_int
    lib.pic_decode_run.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                   ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                   ctypes.c_void_p, ctypes.c_void_p]
    lib.pic_decode_run_noalloc.restype = ctypes.c_int
    lib.pic_decode_run_noalloc.argtypes = [ctypes.POINTER(pic_decode_desc), ctypes.c_int32, ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                           ctypes.c_void_p, ctypes.c_void_p]
    lib.pic_decode_run_layers.restype = ctypes.c_int
    lib.pic_decode_run_layers.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.pic_fuse_modulation.restype = ctypes.c_int
    lib.pic_fuse_modulation.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.pic_decode_query.restype = ctypes.c_int
    lib.pic_decode_query.argtypes = [ctypes.c_void_p, ctypes.POINTER(pic_decode_info)]
    lib.pic_decode_destroy.restype = None
    lib.pic_decode_destroy.argtypes = [ctypes.c_void_p]
    lib.pic_status_string.restype = ctypes.c_char_p
    lib.pic_status_string.argtypes = [ctypes.c_int32]
    lib.pic_zpr_create.restype = ctypes.c_int
    lib.pic_zpr_create.argtypes = [ctypes.POINTER(pic_zpr_desc), ctypes.POINTER(ctypes.c_void_p)]
    for name in ("pic_zpr_decode", "pic_zpr_expand"):
        fn = getattr(lib, name)
        fn.restype = ctypes.c_int
        fn.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.pic_zpr_query.restype = ctypes.c_int
    lib.pic_zpr_query.argtypes = [ctypes.c_void_p, ctypes.POINTER(pic_zpr_info)]
    lib.pic_zpr_destroy.restype = None
    lib.pic_zpr_destroy.argtypes = [ctypes.c_void_p]
    lib.pic_huff_create.restype = ctypes.c_int
    lib.pic_huff_create.argtypes = [ctypes.POINTER(pic_huff_desc), ctypes.POINTER(ctypes.c_void_p)]
    lib.pic_huff_decode.restype = ctypes.c_int
    lib.pic_huff_decode.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_void_p]
    lib.pic_huff_query.restype = ctypes.c_int
    lib.pic_huff_query.argtypes = [ctypes.c_void_p, ctypes.POINTER(pic_huff_info)]
    lib.pic_huff_destroy.restype = None
    lib.pic_huff_destroy.argtypes = [ctypes.c_void_p]
    _lib = lib
    return lib


# ------------------------------------------------------------- C mirrors

def pic_status_string(status: int) -> str:
    return load_library().pic_status_string(int(status)).decode()


def make_desc(height: int, width: int, widths: Sequence[int], weight_dtype: int = PIC_F32,
              out_dtype: int = PIC_F32, flags: int = 0, max_batch: int = 1,
              variant: int = PIC_VARIANT_AUTO) -> pic_decode_desc:
    d = pic_decode_desc()
    d.struct_size = ctypes.sizeof(pic_decode_desc)
    d.height, d.width = int(height), int(width)
    widths = [int(w) for w in widths]
    d.num_levels = widths[0]
    d.num_layers = len(widths) - 1
    for i, w in enumerate(widths[:PIC_MAX_LAYERS + 1]):
        d.widths[i] = w
    d.weight_dtype, d.out_dtype, d.flags = int(weight_dtype), int(out_dtype), int(flags)
    d.max_batch, d.variant = int(max_batch), int(variant)
    return d


def pic_decode_create(desc: pic_decode_desc) -> int:
    """Returns the handle (an integer address); raises PicError."""
    h = ctypes.c_void_p()
    st = load_library().pic_decode_create(ctypes.byref(desc), ctypes.byref(h))
    if st != PIC_OK:
        raise PicError(st, "pic_decode_create")
    return h.value


def pic_decode_run(handle: int, batch: int, latent_ptrs: Sequence[int], weights_ptr: int,
                   weights_img_stride: int, biases_ptr: int, biases_img_stride: int,
                   out_ptr: int, stream: int = 0) -> int:
    """Raw-pointer call; returns the status (no raise, for argument tests)."""
    arr = (ctypes.c_void_p * max(1, len(latent_ptrs)))(*latent_ptrs)
    return load_library().pic_decode_run(handle, batch, arr if latent_ptrs is not None else None,
                                         weights_ptr, weights_img_stride, biases_ptr,
                                         biases_img_stride, out_ptr, stream)


def pic_decode_run_noalloc(desc: pic_decode_desc, batch: int, latent_ptrs: Sequence[int], weights_ptr: int,
                           weights_img_stride: int, biases_ptr: int, biases_img_stride: int,
                           out_ptr: int, stream: int = 0) -> int:
    """Raw-pointer call of the entry point that allocates nothing (no handle:
    the descriptor is passed each time); returns the status."""
    arr = (ctypes.c_void_p * max(1, len(latent_ptrs)))(*latent_ptrs)
    return load_library().pic_decode_run_noalloc(ctypes.byref(desc), batch, arr, weights_ptr, weights_img_stride,
                                                 biases_ptr, biases_img_stride, out_ptr, stream)


def pic_decode_run_layers(handle: int, batch: int, latent_ptrs: Sequence[int], layer_weight_ptrs: Sequence[int],
                          layer_weight_strides: Sequence[int], layer_bias_ptrs: Sequence[int],
                          layer_bias_strides: Sequence[int], out_ptr: int, stream: int = 0) -> int:
    """Raw-pointer call with per-layer parameter pointers and strides; returns the status."""
    n = len(layer_weight_ptrs)
    lat = (ctypes.c_void_p * max(1, len(latent_ptrs)))(*latent_ptrs)
    wp = (ctypes.c_void_p * n)(*layer_weight_ptrs)
    ws = (ctypes.c_int64 * n)(*layer_weight_strides)
    bp = (ctypes.c_void_p * n)(*layer_bias_ptrs)
    bs = (ctypes.c_int64 * n)(*layer_bias_strides)
    return load_library().pic_decode_run_layers(handle, batch, lat, wp, ws, bp, bs, out_ptr, stream)


def pic_fuse_modulation(fan_in: int, fan_out: int, batch: int, w_ptr: int, w_stride: int, b_ptr: int,
                        b_stride: int, gamma_ptr: int, beta_ptr: int, mu_ptr: int, sigma_ptr: int,
                        stat_stride: int, w_fused_ptr: int, b_fused_ptr: int, stream: int = 0) -> int:
    """Raw-pointer call of the App. A fusion; returns the status."""
    return load_library().pic_fuse_modulation(fan_in, fan_out, batch, w_ptr, w_stride, b_ptr, b_stride,
                                              gamma_ptr, beta_ptr, mu_ptr, sigma_ptr, stat_stride,
                                              w_fused_ptr, b_fused_ptr, stream)


def fuse_modulation(w, b, gamma, beta, mu, sigma, stream=None):
    """torch front end of pic_fuse_modulation: w [batch][out][in], b [batch][out],
    gamma/beta/mu/sigma [batch][in] (fp32 device tensors; a missing batch
    dimension means shared).  Returns (w_fused [batch][out][in], b_fused [batch][out])."""
    import torch
    fan_out, fan_in = w.shape[-2], w.shape[-1]
    batch = max(t.shape[0] if t.dim() > d else 1 for t, d in
                ((w, 2), (b, 1), (gamma, 1), (beta, 1), (mu, 1), (sigma, 1)))
    stats = [gamma, beta, mu, sigma]
    if len({t.dim() for t in stats}) != 1:
        raise ValueError("gamma, beta, mu and sigma must share one layout")
    for t in (w, b, *stats):
        if t.dtype != torch.float32 or not t.is_contiguous() or t.device.type != "cuda":
            raise ValueError("fuse_modulation takes contiguous float32 device tensors")
    wf = torch.empty((batch, fan_out, fan_in), dtype=torch.float32, device=w.device)
    bf = torch.empty((batch, fan_out), dtype=torch.float32, device=w.device)
    if stream is None:
        stream = torch.cuda.current_stream(w.device).cuda_stream
    st = pic_fuse_modulation(fan_in, fan_out, batch, w.data_ptr(), fan_in * fan_out if w.dim() == 3 else 0,
                             b.data_ptr(), fan_out if b.dim() == 2 else 0, gamma.data_ptr(), beta.data_ptr(),
                             mu.data_ptr(), sigma.data_ptr(), fan_in if gamma.dim() == 2 else 0,
                             wf.data_ptr(), bf.data_ptr(), int(stream))
    if st != PIC_OK:
        raise PicError(st, "pic_fuse_modulation")
    return wf, bf


def pic_decode_query(handle: int) -> dict:
    info = pic_decode_info()
    info.struct_size = ctypes.sizeof(pic_decode_info)
    st = load_library().pic_decode_query(handle, ctypes.byref(info))
    if st != PIC_OK:
        raise PicError(st, "pic_decode_query")
    return dict(variant=VARIANT_NAMES.get(info.variant, info.variant),
                weights_per_image=info.weights_per_image, biases_per_image=info.biases_per_image,
                device=info.device, pixels_per_wave_step=info.pixels_per_wave_step,
                kernel_name=info.kernel_name.decode())


def pic_decode_destroy(handle: int) -> None:
    load_library().pic_decode_destroy(handle)


def make_zpr_desc(height: int, width: int, levels: int, max_batch: int = 1) -> pic_zpr_desc:
    d = pic_zpr_desc()
    d.struct_size = ctypes.sizeof(pic_zpr_desc)
    d.height, d.width, d.num_levels, d.max_batch = int(height), int(width), int(levels), int(max_batch)
    return d


def pic_zpr_create(desc: pic_zpr_desc) -> int:
    """Returns the handle (an integer address); raises PicError."""
    h = ctypes.c_void_p()
    st = load_library().pic_zpr_create(ctypes.byref(desc), ctypes.byref(h))
    if st != PIC_OK:
        raise PicError(st, "pic_zpr_create")
    return h.value


def pic_zpr_decode(handle: int, batch: int, symbols_ptr: int, n_symbols: int, eob: int,
                   latent_ptrs: Optional[Sequence[int]], status_ptr: int, stream: int = 0) -> int:
    """Raw-pointer call; returns the status (no raise, for argument tests).
    ``latent_ptrs`` is indexed by level k (finest first), as in the header."""
    arr = None if latent_ptrs is None else (ctypes.c_void_p * len(latent_ptrs))(*latent_ptrs)
    return load_library().pic_zpr_decode(handle, int(batch), symbols_ptr, int(n_symbols), int(eob), arr,
                                         status_ptr, stream)


def pic_zpr_expand(handle: int, batch: int, symbols_ptr: int, n_symbols: int, eob: int, coeffs_ptr: int,
                   status_ptr: int, stream: int = 0) -> int:
    """Raw-pointer call; returns the status."""
    return load_library().pic_zpr_expand(handle, int(batch), symbols_ptr, int(n_symbols), int(eob), coeffs_ptr,
                                         status_ptr, stream)


def pic_zpr_query(handle: int) -> dict:
    info = pic_zpr_info()
    info.struct_size = ctypes.sizeof(pic_zpr_info)
    st = load_library().pic_zpr_query(handle, ctypes.byref(info))
    if st != PIC_OK:
        raise PicError(st, "pic_zpr_query")
    return dict(device=info.device, blocks_per_image=info.blocks_per_image, max_symbols=info.max_symbols,
                scratch_bytes=info.scratch_bytes, symbols_per_chunk=info.symbols_per_chunk)


def pic_zpr_destroy(handle: int) -> None:
    load_library().pic_zpr_destroy(handle)


def make_huff_desc(max_bits: int) -> pic_huff_desc:
    d = pic_huff_desc()
    d.struct_size = ctypes.sizeof(pic_huff_desc)
    d.max_bits = int(max_bits)
    return d


def pic_huff_create(desc: pic_huff_desc) -> int:
    """Returns the handle (an integer address); raises PicError."""
    h = ctypes.c_void_p()
    st = load_library().pic_huff_create(ctypes.byref(desc), ctypes.byref(h))
    if st != PIC_OK:
        raise PicError(st, "pic_huff_create")
    return h.value


def pic_huff_decode(handle: int, data_ptr: int, n_bits: int, values_ptr: int, lengths_ptr: int, n_table: int,
                    n_symbols: int, out_ptr: int, status_ptr: int, stream: int = 0) -> int:
    """Raw-pointer call; returns the status (no raise, for argument tests)."""
    return load_library().pic_huff_decode(handle, data_ptr, int(n_bits), values_ptr, lengths_ptr, int(n_table),
                                          int(n_symbols), out_ptr, status_ptr, stream)


def pic_huff_query(handle: int) -> dict:
    info = pic_huff_info()
    info.struct_size = ctypes.sizeof(pic_huff_info)
    st = load_library().pic_huff_query(handle, ctypes.byref(info))
    if st != PIC_OK:
        raise PicError(st, "pic_huff_query")
    return dict(device=info.device, max_bits=info.max_bits, scratch_bytes=info.scratch_bytes,
                bits_per_thread=info.bits_per_thread, lut_bits=info.lut_bits)


def pic_huff_destroy(handle: int) -> None:
    load_library().pic_huff_destroy(handle)


# ------------------------------------------------------------ torch layer

class Decoder:
    """One decoder handle for a fixed image size and MLP shape.

    ``run`` takes torch tensors on the handle's device: ``latents`` (L fp32
    tensors [batch][ceil(H/2^k)][ceil(W/2^k)]), ``weights`` ([batch][nw] fp32,
    or uint16/bfloat16 for bf16 weights; [nw] when shared), ``biases``
    ([batch][nb] fp32 or [nb] shared).  It enqueues on torch's current stream
    (or ``stream``) and returns ``out`` ([batch][3][H][W], float32 or uint8).
    """

    def __init__(self, height: int, width: int, widths: Sequence[int], weight_dtype: str = "f32",
                 out_dtype: str = "f32", clamp: bool = True, max_batch: int = 1,
                 variant: str = "auto"):
        self.height, self.width = int(height), int(width)
        self.widths = tuple(int(w) for w in widths)
        self.levels = self.widths[0]
        self.weight_dtype, self.out_dtype, self.clamp = weight_dtype, out_dtype, clamp
        self.max_batch = int(max_batch)
        self.desc = make_desc(height, width, self.widths,
                              PIC_BF16 if weight_dtype == "bf16" else PIC_F32,
                              PIC_U8 if out_dtype == "u8" else PIC_F32,
                              0 if clamp else PIC_FLAG_NO_CLAMP, max_batch, VARIANTS[variant])
        self.handle = pic_decode_create(self.desc)
        self.nw = sum(self.widths[i] * self.widths[i + 1] for i in range(len(self.widths) - 1))
        self.nb = sum(self.widths[1:])

    def level_shape(self, k: int):
        f = 1 << k
        return (-(-self.height // f), -(-self.width // f))

    def info(self) -> dict:
        return pic_decode_query(self.handle)

    def alloc_out(self, batch: int, device=None):
        import torch
        dt = torch.uint8 if self.out_dtype == "u8" else torch.float32
        return torch.empty((batch, 3, self.height, self.width), dtype=dt, device=device)

    def run(self, latents, weights, biases, out=None, batch: Optional[int] = None, stream=None):
        import torch
        batch = latents[0].shape[0] if batch is None else int(batch)
        if len(latents) != self.levels:
            raise ValueError(f"expected {self.levels} latent levels, got {len(latents)}")
        dev = latents[0].device
        if dev.type != "cuda":
            raise ValueError("latents must be device tensors")
        for k, t in enumerate(latents):
            if t.dtype != torch.float32 or not t.is_contiguous() or t.device != dev:
                raise ValueError(f"level {k}: need a contiguous float32 tensor on {dev}")
            if tuple(t.shape[1:]) != self.level_shape(k) or t.shape[0] < batch:
                raise ValueError(f"level {k}: shape {tuple(t.shape)}, expected "
                                 f"[>= {batch}][{self.level_shape(k)}]")
        wdt = (torch.uint16, torch.bfloat16, torch.int16) if self.weight_dtype == "bf16" else (torch.float32,)
        if weights.dtype not in wdt or not weights.is_contiguous() or weights.device != dev:
            raise ValueError(f"weights: need a contiguous {wdt[0]} tensor on {dev}")
        if biases.dtype != torch.float32 or not biases.is_contiguous() or biases.device != dev:
            raise ValueError(f"biases: need a contiguous float32 tensor on {dev}")
        ws = 0 if weights.dim() == 1 else self.nw
        bs = 0 if biases.dim() == 1 else self.nb
        if weights.numel() < (self.nw if ws == 0 else batch * self.nw):
            raise ValueError("weights tensor too small")
        if biases.numel() < (self.nb if bs == 0 else batch * self.nb):
            raise ValueError("biases tensor too small")
        if out is None:
            out = self.alloc_out(batch, dev)
        want_dt = torch.uint8 if self.out_dtype == "u8" else torch.float32
        if out.dtype != want_dt or not out.is_contiguous() or out.device != dev or \
                tuple(out.shape[1:]) != (3, self.height, self.width) or out.shape[0] < batch:
            raise ValueError("out: wrong dtype, shape, layout or device")
        if stream is None:
            stream = torch.cuda.current_stream(dev).cuda_stream
        st = pic_decode_run(self.handle, batch, [t.data_ptr() for t in latents], weights.data_ptr(), ws,
                            biases.data_ptr(), bs, out.data_ptr(), int(stream))
        if st != PIC_OK:
            raise PicError(st, "pic_decode_run")
        return out

    def run_layers(self, latents, layer_weights, layer_biases, out=None, batch: Optional[int] = None,
                   stream=None):
        """Per-layer parameters: layer_weights[l] is [batch][out][in] (per image)
        or [out][in] (shared by the batch); layer_biases[l] likewise."""
        import torch
        batch = latents[0].shape[0] if batch is None else int(batch)
        nl = len(self.widths) - 1
        if len(layer_weights) != nl or len(layer_biases) != nl:
            raise ValueError(f"expected {nl} layers")
        dev = latents[0].device
        ws, bs = [], []
        for l in range(nl):
            w, b = layer_weights[l], layer_biases[l]
            shape = (self.widths[l + 1], self.widths[l])
            if tuple(w.shape[-2:]) != shape or not w.is_contiguous() or w.device != dev:
                raise ValueError(f"layer {l}: weights must be [..][{shape[0]}][{shape[1]}] on {dev}")
            if b.shape[-1] != shape[0] or not b.is_contiguous() or b.dtype != torch.float32:
                raise ValueError(f"layer {l}: bias must be contiguous float32 [..][{shape[0]}]")
            ws.append(0 if w.dim() == 2 else shape[0] * shape[1])
            bs.append(0 if b.dim() == 1 else shape[0])
        if out is None:
            out = self.alloc_out(batch, dev)
        if stream is None:
            stream = torch.cuda.current_stream(dev).cuda_stream
        st = pic_decode_run_layers(self.handle, batch, [t.data_ptr() for t in latents],
                                   [w.data_ptr() for w in layer_weights], ws,
                                   [b.data_ptr() for b in layer_biases], bs, out.data_ptr(), int(stream))
        if st != PIC_OK:
            raise PicError(st, "pic_decode_run_layers")
        return out

    def close(self):
        if getattr(self, "handle", None):
            pic_decode_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


class ZprDecoder:
    """One latent-decoding handle (include/pic_zpr.h) for a fixed pyramid shape.

    ``decode`` takes the symbol stream as a contiguous int32 device tensor and
    returns the L latent grids (fp32 [batch][ceil(H/2^k)][ceil(W/2^k)], level
    k = 0 finest, the layout ``Decoder.run`` takes) and a one-element int32
    status tensor (PIC_ZPR_ERR_* bits).  ``expand`` returns Alg. 1's
    coefficient blocks instead ([batch * blocks_per_image][64] int32).  Both
    enqueue on torch's current stream (or ``stream``) and do not synchronise.
    """

    def __init__(self, height: int, width: int, levels: int, max_batch: int = 1):
        self.height, self.width, self.levels = int(height), int(width), int(levels)
        self.max_batch = int(max_batch)
        self.handle = pic_zpr_create(make_zpr_desc(height, width, levels, max_batch))
        self.blocks_per_image = self.info()["blocks_per_image"]

    def info(self) -> dict:
        return pic_zpr_query(self.handle)

    def level_shape(self, k: int):
        f = 1 << k
        return (-(-self.height // f), -(-self.width // f))

    def _check(self, symbols, status, batch):
        import torch
        if symbols.dtype != torch.int32 or symbols.dim() != 1 or not symbols.is_contiguous() \
                or symbols.device.type != "cuda":
            raise ValueError("symbols: need a contiguous 1-D int32 device tensor")
        dev = symbols.device
        if status is None:
            status = torch.empty(1, dtype=torch.int32, device=dev)
        if status.dtype != torch.int32 or status.device != dev or not status.is_contiguous():
            raise ValueError("status: need an int32 device tensor")
        if not 0 <= batch <= self.max_batch:
            raise ValueError(f"batch {batch} outside 0 .. {self.max_batch}")
        return dev, status

    def decode(self, symbols, eob: int, batch: int = 1, latents=None, status=None, stream=None):
        import torch
        batch = int(batch)
        dev, status = self._check(symbols, status, batch)
        if latents is None:
            latents = [torch.empty((batch,) + self.level_shape(k), dtype=torch.float32, device=dev)
                       for k in range(self.levels)]
        if len(latents) != self.levels:
            raise ValueError(f"expected {self.levels} latent levels")
        for k, t in enumerate(latents):
            if t.dtype != torch.float32 or not t.is_contiguous() or t.device != dev or \
                    tuple(t.shape[1:]) != self.level_shape(k) or t.shape[0] < batch:
                raise ValueError(f"level {k}: need contiguous float32 [>= {batch}][{self.level_shape(k)}]")
        if stream is None:
            stream = torch.cuda.current_stream(dev).cuda_stream
        st = pic_zpr_decode(self.handle, batch, symbols.data_ptr(), symbols.numel(), eob,
                            [t.data_ptr() for t in latents], status.data_ptr(), int(stream))
        if st != PIC_OK:
            raise PicError(st, "pic_zpr_decode")
        return latents, status

    def expand(self, symbols, eob: int, batch: int = 1, coeffs=None, status=None, stream=None):
        import torch
        batch = int(batch)
        dev, status = self._check(symbols, status, batch)
        nb = batch * self.blocks_per_image
        if coeffs is None:
            coeffs = torch.empty((nb, 64), dtype=torch.int32, device=dev)
        if coeffs.dtype != torch.int32 or not coeffs.is_contiguous() or coeffs.device != dev or \
                coeffs.numel() < nb * 64:
            raise ValueError(f"coeffs: need contiguous int32 [{nb}][64] on {dev}")
        if stream is None:
            stream = torch.cuda.current_stream(dev).cuda_stream
        st = pic_zpr_expand(self.handle, batch, symbols.data_ptr(), symbols.numel(), eob, coeffs.data_ptr(),
                            status.data_ptr(), int(stream))
        if st != PIC_OK:
            raise PicError(st, "pic_zpr_expand")
        return coeffs, status

    def close(self):
        if getattr(self, "handle", None):
            pic_zpr_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


class HuffDecoder:
    """One entropy-decoding handle (include/pic_huff.h).

    ``decode`` takes the bitstream (contiguous uint8 device tensor, MSB
    first), its bit count, the code table (int32 values and uint8 lengths,
    device tensors) and the number of symbols, and returns the symbols (int32
    device tensor, the input of ``ZprDecoder``) and a one-element int32 status
    tensor (PIC_HUFF_ERR_* bits).  It enqueues on torch's current stream (or
    ``stream``) and does not synchronise.
    """

    def __init__(self, max_bits: int):
        self.max_bits = int(max_bits)
        self.handle = pic_huff_create(make_huff_desc(max_bits))

    def info(self) -> dict:
        return pic_huff_query(self.handle)

    def decode(self, data, n_bits: int, values, lengths, n_symbols: int, out=None, status=None, stream=None):
        import torch
        dev = values.device
        if data.dtype != torch.uint8 or not data.is_contiguous() or data.device != dev or \
                data.numel() * 8 < int(n_bits):
            raise ValueError("data: need a contiguous uint8 device tensor holding n_bits bits")
        if values.dtype != torch.int32 or not values.is_contiguous() or values.device.type != "cuda":
            raise ValueError("values: need a contiguous int32 device tensor")
        if lengths.dtype != torch.uint8 or not lengths.is_contiguous() or lengths.device != dev or \
                lengths.numel() != values.numel():
            raise ValueError("lengths: need a contiguous uint8 device tensor like values")
        if out is None:
            out = torch.empty(max(int(n_symbols), 1), dtype=torch.int32, device=dev)
        if out.dtype != torch.int32 or not out.is_contiguous() or out.device != dev or out.numel() < n_symbols:
            raise ValueError("out: need a contiguous int32 device tensor of n_symbols entries")
        if status is None:
            status = torch.empty(1, dtype=torch.int32, device=dev)
        if stream is None:
            stream = torch.cuda.current_stream(dev).cuda_stream
        st = pic_huff_decode(self.handle, data.data_ptr() if data.numel() else 0, n_bits, values.data_ptr(),
                             lengths.data_ptr(), values.numel(), n_symbols, out.data_ptr(), status.data_ptr(),
                             int(stream))
        if st != PIC_OK:
            raise PicError(st, "pic_huff_decode")
        return out[:int(n_symbols)], status

    def close(self):
        if getattr(self, "handle", None):
            pic_huff_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
