"""Seeded synthetic inputs for the PIC synthesis decoder.

This module only *draws* inputs: latent pyramids and MLP parameters with the
shapes and value distributions of the decoder's workloads (PIC, Sec. 3.1
Eq. (2) for the pyramid; Sec. 4.1 "Implementation Details" and App. A for the
per-image MLP).  It holds none of the decoder's arithmetic (no upsampling, no
MLP evaluation), so both the HIP path and the CPU oracle can consume its
output without sharing any of the method's code.

Layouts produced here are the ones the C ABI takes:

* level k (k = 0 is full resolution, factor 2**k) is a float32 array
  ``[batch][ceil(H / 2**k)][ceil(W / 2**k)]``;
* weights are float32 ``[batch][sum_l out_l * in_l]``: layer l's matrix is
  stored ``[out][in]`` row-major and the layers are concatenated;
* biases are float32 ``[batch][sum_l out_l]``, layers concatenated.

Draw order with one ``numpy.random.default_rng(seed)`` (PCG64): images in
batch order; per image the latent levels 0..L-1 (each row-major), then each
layer's weight matrix row-major; biases are drawn last (per image, per layer)
only when a workload asks for nonzero biases.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np


def level_shape(height: int, width: int, k: int) -> tuple:
    """Grid size of latent level k: ceil(H / 2**k) x ceil(W / 2**k)."""
    f = 1 << k
    return (-(-height // f), -(-width // f))


def param_counts(widths: Sequence[int]) -> tuple:
    """(number of weights, number of biases) of an MLP with these widths."""
    nw = sum(int(widths[i]) * int(widths[i + 1]) for i in range(len(widths) - 1))
    nb = sum(int(widths[i + 1]) for i in range(len(widths) - 1))
    return nw, nb


@dataclass(frozen=True)
class Workload:
    """A synthetic decode workload: image size, pyramid depth, MLP widths and
    the distributions its inputs are drawn from."""

    name: str
    height: int
    width: int
    levels: int
    widths: tuple            # (L, N1, ..., 3)
    batch: int
    latent: str              # "uniform_int" | "laplace_int" | "normal"
    latent_scale: float      # half-range for uniform_int, Laplace scale b, or normal std
    latent_clip: float       # clip bound for laplace_int (ignored otherwise)
    bias: str = "zero"       # "zero" | "normal"
    weight_dtype: str = "f32"  # "f32" | "bf16"
    seed: int = 0
    note: str = ""

    @property
    def pixels(self) -> int:
        return self.batch * self.height * self.width

    def with_batch(self, batch: int) -> "Workload":
        return Workload(**{**self.__dict__, "batch": batch,
                           "name": f"{self.name.split('_b')[0]}_b{batch}"})


# The five decode workloads.  768x512 stands in for the Kodak set (24 images
# of that size, Sec. 4.1); 2048x1536 stands in for the high-resolution CLIC
# images; 64x64 and 3840x2160 bracket them.
WORKLOADS = {
    "pic64": Workload("pic64", 64, 64, 4, (4, 16, 16, 3), 1,
                      "uniform_int", 8, 0, note="64x64, 4 levels, integer latents in [-8, 8]"),
    "kodak768": Workload("kodak768", 512, 768, 7, (7, 40, 40, 3), 1,
                         "laplace_int", 2.0, 32, note="768x512 single image"),
    "kodak768_b64": Workload("kodak768_b64", 512, 768, 7, (7, 40, 40, 3), 64,
                             "laplace_int", 2.0, 32, note="64 independent 768x512 decodes in one call"),
    "clic2048": Workload("clic2048", 1536, 2048, 7, (7, 48, 48, 3), 1,
                         "laplace_int", 2.0, 32, note="2048x1536 single image"),
    "clic2048_b16": Workload("clic2048_b16", 1536, 2048, 7, (7, 48, 48, 3), 16,
                             "laplace_int", 2.0, 32, note="16 independent 2048x1536 decodes"),
    "uhd4k": Workload("uhd4k", 2160, 3840, 8, (8, 64, 64, 3), 1,
                      "laplace_int", 3.0, 64, note="3840x2160, fp32 weights"),
    "uhd4k_bf16": Workload("uhd4k_bf16", 2160, 3840, 8, (8, 64, 64, 3), 1,
                           "laplace_int", 3.0, 64, weight_dtype="bf16",
                           note="3840x2160, bf16 weights (fp32 draws rounded to nearest-even)"),
    # The paper's own synthesis net: 8 levels, four linear layers of width 16.
    "kodak768_paper": Workload("kodak768_paper", 512, 768, 8, (8, 16, 16, 16, 3), 1,
                               "laplace_int", 2.0, 32,
                               note="768x512, the paper's 4-layer width-16 synthesis net"),
}


@dataclass
class Inputs:
    """Host-side (numpy) inputs of one decode call."""

    height: int
    width: int
    levels: int
    widths: tuple
    batch: int
    latents: List[np.ndarray]            # L arrays, float32 [batch][h_k][w_k]
    weights: np.ndarray                  # float32 [batch][nw]
    biases: np.ndarray                   # float32 [batch][nb]
    weights_bf16: Optional[np.ndarray] = None   # uint16 bf16 bit patterns [batch][nw]
    meta: dict = field(default_factory=dict)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even) and
    return the 16-bit patterns.  A storage-format conversion, used to hand the
    bf16-weight variant its input; inputs must be finite."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if not np.all(np.isfinite(a)):
        raise ValueError("bf16 conversion expects finite values")
    u = a.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to the float32 values they denote."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _draw_latent(rng, shape, kind, scale, clip):
    if kind == "uniform_int":
        s = int(scale)
        return rng.integers(-s, s + 1, size=shape).astype(np.float32)
    if kind == "laplace_int":
        v = np.rint(rng.laplace(0.0, scale, size=shape))
        return np.clip(v, -clip, clip).astype(np.float32)
    if kind == "normal":
        return rng.normal(0.0, scale, size=shape).astype(np.float32)
    raise ValueError(f"unknown latent distribution {kind!r}")


def make_inputs(height: int, width: int, levels: int, widths: Sequence[int],
                batch: int = 1, seed: int = 0, latent: str = "laplace_int",
                latent_scale: float = 2.0, latent_clip: float = 32.0,
                bias: str = "zero", weight_dtype: str = "f32",
                shared_weights: bool = False) -> Inputs:
    """Draw one decode call's inputs.

    Weights are N(0, 1/fan_in) (variance 1/fan_in).  ``bias="normal"`` draws
    N(0, 0.5**2) biases so tests exercise the bias path; ``shared_weights``
    draws one parameter set and repeats it for every image (the case of a
    zero image stride at the ABI).
    """
    widths = tuple(int(w) for w in widths)
    if widths[0] != levels:
        raise ValueError("widths[0] must equal the number of levels")
    rng = np.random.default_rng(seed)
    nw, nb = param_counts(widths)
    shapes = [level_shape(height, width, k) for k in range(levels)]
    lat = [np.empty((batch,) + s, dtype=np.float32) for s in shapes]
    W = np.empty((batch, nw), dtype=np.float32)
    B = np.zeros((batch, nb), dtype=np.float32)
    for b in range(batch):
        for k in range(levels):
            lat[k][b] = _draw_latent(rng, shapes[k], latent, latent_scale, latent_clip)
        if shared_weights and b > 0:
            W[b] = W[0]
            continue
        off = 0
        for l in range(len(widths) - 1):
            fin, fout = widths[l], widths[l + 1]
            W[b, off:off + fin * fout] = rng.normal(
                0.0, 1.0 / np.sqrt(fin), size=(fout, fin)).astype(np.float32).ravel()
            off += fin * fout
    if bias == "normal":
        for b in range(batch):
            if shared_weights and b > 0:
                B[b] = B[0]
            else:
                B[b] = rng.normal(0.0, 0.5, size=nb).astype(np.float32)
    elif bias != "zero":
        raise ValueError(f"unknown bias mode {bias!r}")
    inp = Inputs(height, width, levels, widths, batch, lat, W, B)
    if weight_dtype == "bf16":
        inp.weights_bf16 = f32_to_bf16_bits(W)
    elif weight_dtype != "f32":
        raise ValueError(f"unknown weight dtype {weight_dtype!r}")
    inp.meta = dict(seed=seed, latent=latent, latent_scale=latent_scale,
                    latent_clip=latent_clip, bias=bias, weight_dtype=weight_dtype)
    return inp


def workload_inputs(w: Workload, batch: Optional[int] = None, seed: Optional[int] = None) -> Inputs:
    """Inputs of a named workload (optionally with a smaller batch or another seed)."""
    return make_inputs(w.height, w.width, w.levels, w.widths,
                       batch=w.batch if batch is None else batch,
                       seed=w.seed if seed is None else seed,
                       latent=w.latent, latent_scale=w.latent_scale,
                       latent_clip=w.latent_clip, bias=w.bias,
                       weight_dtype=w.weight_dtype)


# ------------------------------------------------------------------ ZpR streams
#
# Symbol streams as the entropy decoder hands them to the latent-decoding step
# (PIC, Sec. 3.3 and Fig. 2; App. B Alg. 1).  The stream format: one code per
# 8x8 block, blocks in the order image, level (coarsest first), patch row,
# patch column; a block's code is a sequence of tokens, each either one
# nonzero coefficient value (a literal) or a run code eob - 17 + r standing
# for r zeros (r = 1 .. 16), and it ends with the marker eob.  The tokens
# cover the block's zigzag positions from the first up to its last nonzero
# coefficient; nothing is coded after it.
#
# The generator draws the run-length description directly: for each block the
# zigzag positions that carry a nonzero value and those values.  It then
# serialises it: the gap before each nonzero position as whole runs of 16 and
# a remainder, the value, and finally the marker.  No coefficient block is
# built and no transform is applied here.
#
# Distribution (a stand-in for quantised DCT coefficients of trained latents
# at a few tenths of a bit per pixel):
#   - 10 % of blocks are empty; 2 % are dense (every position nonzero with
#     probability 0.7);
#   - otherwise position 0 (DC) is nonzero with probability 0.9 and position
#     p >= 1 with probability 0.55 exp(-(p - 1) / 5), about 3 AC values;
#   - |DC| = 1 + Geometric(0.12), |AC| = 1 + Geometric(0.55) (mostly 1 or
#     2), random sign, clipped to max_abs; eob = max_abs + 17, so the run
#     codes are max_abs + 1 .. max_abs + 16.
# That gives about 9 symbols per block, the empty blocks 1.


def zpr_blocks_per_image(height: int, width: int, levels: int) -> int:
    """8x8 patches of one image's pyramid (each level padded to whole patches)."""
    n = 0
    for k in range(levels):
        h, w = level_shape(height, width, k)
        n += (-(-h // 8)) * (-(-w // 8))
    return n


@dataclass
class ZprStream:
    """One latent-decoding call's input: the symbol stream of `batch` images."""

    height: int
    width: int
    levels: int
    batch: int
    eob: int
    symbols: np.ndarray          # int32 [n_symbols]
    blocks: int                  # blocks in the stream (batch * per image)


def make_zpr_stream(height: int, width: int, levels: int, batch: int = 1, seed: int = 0,
                    max_abs: int = 60, empty_frac: float = 0.10, dense_frac: float = 0.02) -> ZprStream:
    """Draw a seeded symbol stream for `batch` images of this pyramid shape."""
    rng = np.random.default_rng(seed)
    nb = batch * zpr_blocks_per_image(height, width, levels)
    pos = np.arange(64)
    prob = np.where(pos == 0, 0.9, 0.55 * np.exp(-(pos - 1) / 5.0))
    kind = rng.random(nb)
    p = np.broadcast_to(prob, (nb, 64)).copy()
    p[kind < empty_frac] = 0.0
    p[(kind >= empty_frac) & (kind < empty_frac + dense_frac)] = 0.7
    mask = rng.random((nb, 64)) < p
    mag_dc = 1 + rng.geometric(0.12, size=nb) - 1
    mag_ac = 1 + rng.geometric(0.55, size=(nb, 64)) - 1
    mag = np.where(pos[None, :] == 0, mag_dc[:, None], mag_ac)
    sign = np.where(rng.random((nb, 64)) < 0.5, -1, 1)
    val = np.clip(sign * mag, -max_abs, max_abs).astype(np.int64)
    eob = max_abs + 17

    g, q = np.nonzero(mask)                       # block, zigzag position (row-major order)
    first = np.ones(g.size, dtype=bool)
    first[1:] = g[1:] != g[:-1]
    prev = np.empty(g.size, dtype=np.int64)
    prev[first] = -1
    prev[~first] = q[:-1][~first[1:]]
    gap = q - prev - 1
    n16, rem = gap // 16, gap % 16
    ntok = n16 + (rem > 0) + 1                     # runs, then the literal
    per_block = np.bincount(g, weights=ntok, minlength=nb).astype(np.int64) + 1
    start = np.concatenate([[0], np.cumsum(per_block)[:-1]])
    total = int(per_block.sum())
    sym = np.empty(total, dtype=np.int64)
    # offset of each nonzero's tokens inside its block
    cum = np.cumsum(ntok) - ntok
    block_first = np.concatenate([[0], np.cumsum(np.bincount(g, minlength=nb))[:-1]])
    within = cum - cum[block_first[g]] if g.size else cum
    at = start[g] + within
    # runs of 16
    r16 = np.repeat(at, n16) + (np.arange(n16.sum()) - np.repeat(np.cumsum(n16) - n16, n16))
    sym[r16] = eob - 17 + 16
    has_rem = rem > 0
    sym[at[has_rem] + n16[has_rem]] = eob - 17 + rem[has_rem]
    sym[at + n16 + has_rem] = val[g, q]
    sym[start + per_block - 1] = eob
    return ZprStream(height, width, levels, batch, eob, sym.astype(np.int32), nb)


def workload_zpr_stream(w: Workload, batch: Optional[int] = None, seed: Optional[int] = None) -> ZprStream:
    """The symbol stream of a named workload's pyramid shape."""
    return make_zpr_stream(w.height, w.width, w.levels, w.batch if batch is None else batch,
                           w.seed + 1000 if seed is None else seed)


# ------------------------------------------------------------ Huffman streams
#
# The bitstream the entropy decoder reads (PIC, Sec. 3.3: an image-specific
# Huffman code whose stored table lists only the symbols used).  Format, as
# the decoder takes it: a table of (symbol value, code length) pairs, one per
# distinct symbol in increasing value order; the canonical code of those
# lengths (codes of one length consecutive in table order, shorter lengths
# first); the codewords packed most significant bit first.  The generator
# draws nothing new: it codes a ZpR stream with a Huffman code built from
# that stream's own symbol histogram (the two rarest subtrees merged
# repeatedly), its longest codeword kept at or below max_len bits by raising
# the rarest counts.


@dataclass
class HuffStream:
    """One entropy-decoding call's input."""

    data: np.ndarray            # uint8 [ceil(n_bits / 8)], MSB first
    n_bits: int
    values: np.ndarray          # int32 [n_table], increasing
    lengths: np.ndarray         # uint8 [n_table]
    n_symbols: int
    symbols: np.ndarray         # int32 [n_symbols]: what the bits code


def _huff_depths(freqs):
    import heapq
    n = len(freqs)
    if n == 1:
        return np.ones(1, dtype=np.int64)
    depth = np.zeros(n, dtype=np.int64)
    heap = [(int(f), i, (i,)) for i, f in enumerate(freqs)]
    heapq.heapify(heap)
    uid = n
    while len(heap) > 1:
        f1, _, a = heapq.heappop(heap)
        f2, _, b = heapq.heappop(heap)
        members = a + b
        depth[list(members)] += 1
        heapq.heappush(heap, (f1 + f2, uid, members))
        uid += 1
    return depth


def make_huff_stream(symbols: np.ndarray, max_len: int = 20) -> HuffStream:
    """Huffman-code `symbols` (int32) with a code built from their histogram."""
    symbols = np.ascontiguousarray(symbols, dtype=np.int32)
    values, inverse, counts = np.unique(symbols, return_inverse=True, return_counts=True)
    floor = 0
    while True:
        depth = _huff_depths(np.maximum(counts, floor))
        if depth.max() <= max_len:
            break
        floor = max(1, floor * 2, int(counts.sum()) >> (max_len - 2))
    lengths = depth.astype(np.int64)
    # canonical codes: by (length, table order)
    order = np.lexsort((np.arange(lengths.size), lengths))
    codes = np.zeros(lengths.size, dtype=np.int64)
    code, prev = 0, int(lengths[order[0]])
    for k, i in enumerate(order):
        if k:
            code = (code + 1) << (int(lengths[i]) - prev)
        codes[i] = code
        prev = int(lengths[i])
    ln = lengths[inverse]
    cw = codes[inverse]
    start = np.concatenate([[0], np.cumsum(ln)[:-1]])
    n_bits = int(ln.sum())
    bitarr = np.zeros(n_bits + (-n_bits % 8), dtype=np.uint8)
    for j in range(int(lengths.max())):
        sel = ln > j
        bitarr[start[sel] + j] = (cw[sel] >> (ln[sel] - 1 - j)) & 1
    data = np.packbits(bitarr)
    return HuffStream(data, n_bits, values.astype(np.int32), lengths.astype(np.uint8), int(symbols.size),
                      symbols)


def workload_huff_stream(w: Workload, batch: Optional[int] = None, seed: Optional[int] = None) -> HuffStream:
    """The Huffman bitstream of a named workload's ZpR stream."""
    return make_huff_stream(workload_zpr_stream(w, batch, seed).symbols)
