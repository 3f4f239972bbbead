"""Pins of the ZpR part of the CPU oracle (latents from the symbol stream).

Each ``check_*`` takes an oracle object and raises AssertionError on a
mismatch; they join ``pins.ALL_CHECKS`` so the mutant test runs them too.

What pins what (PIC, Sec. 3.2 Eq. (5)-(7), Sec. 3.3 and Fig. 2, App. B
Alg. 1):
  * zigzag order      -- the JPEG table (tests/golden/jpeg_zigzag.txt, from
                         ITU-T T.81) and an independent construction by sorting
                         the positions by anti-diagonal with alternating
                         direction;
  * eob offsets       -- numpy's flatnonzero of the marker test;
  * Alg. 1 expansion  -- hand-worked blocks, and a round trip through a ZpR
                         encoder written here from the description of Fig. 2
                         (zigzag, trailing zeros dropped, zero runs as run
                         codes; runs split in several ways, literal zeros too);
  * inverse DCT       -- scipy's orthonormal idctn, the DC-only closed form,
                         Parseval, and scipy's dctn undoing it;
  * un-patchify       -- a numpy patchify (pad, reshape, transpose) of random
                         pyramids with ragged sizes undone exactly;
  * whole step        -- random sparse coefficient blocks encoded here, the
                         expected pyramid built with scipy and numpy;
  * error flags       -- streams broken in each of the flagged ways.
"""
from __future__ import annotations

import os

import numpy as np
import scipy.fft

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _zigzag_table():
    vals = []
    for line in open(os.path.join(GOLDEN, "jpeg_zigzag.txt")):
        if not line.startswith("#"):
            vals += [int(t) for t in line.split()]
    return np.array(vals, dtype=np.int64)


ZZ = _zigzag_table()


# ------------------------------------------------- a ZpR encoder (Fig. 2)

def zpr_encode_block(coeffs, eob, rng=None, split="greedy", literal_zero_prob=0.0):
    """ZpR code of one 8x8 block of integer coefficients (row-major 64):
    reorder by the zigzag table, drop the trailing zeros, replace each run of
    zeros by run codes eob - 17 + r (r in 1..16), end with eob.  ``split``
    chooses how a run longer than 16 (or any run, with "random") is cut into
    pieces; ``literal_zero_prob`` emits some zeros as literal 0 instead."""
    z = [int(coeffs[ZZ[p]]) for p in range(64)]
    last = max([p for p in range(64) if z[p] != 0], default=-1)
    out, p = [], 0
    while p <= last:
        if z[p] != 0:
            out.append(z[p])
            p += 1
            continue
        run = 0
        while p + run <= last and z[p + run] == 0:
            run += 1
        pieces = []
        left = run
        while left > 0:
            if split == "random" and rng is not None:
                r = int(rng.integers(1, min(16, left) + 1))
            else:
                r = min(16, left)
            pieces.append(r)
            left -= r
        for r in pieces:
            if rng is not None and literal_zero_prob > 0 and r == 1 and rng.random() < literal_zero_prob:
                out.append(0)
            else:
                out.append(eob - 17 + r)
        p += run
    out.append(eob)
    return out


def random_blocks(rng, n, density, max_abs):
    """n integer 8x8 blocks (row-major), each position nonzero with the
    given probability, values in [-max_abs, max_abs] \\ {0}."""
    mask = rng.random((n, 64)) < density
    vals = rng.integers(1, max_abs + 1, size=(n, 64)) * np.where(rng.random((n, 64)) < 0.5, -1, 1)
    return np.where(mask, vals, 0).astype(np.int64)


# ------------------------------------------------- patchify (Eq. (5)-(6))

def patchify(levels, L, batch):
    """Blocks [n][64] of a pyramid in the stream order: image, level coarsest
    first, patch row, patch column, row-major inside the patch.  Padding
    samples are filled with NaN (the decoder must drop them)."""
    out = []
    for b in range(batch):
        for k in range(L - 1, -1, -1):
            g = levels[k][b]
            h, w = g.shape
            ph, pw = -(-h // 8), -(-w // 8)
            pad = np.full((ph * 8, pw * 8), np.nan)
            pad[:h, :w] = g
            out.append(pad.reshape(ph, 8, pw, 8).transpose(0, 2, 1, 3).reshape(ph * pw, 64))
    return np.concatenate(out, axis=0)


def place_blocks(blocks, H, W, L, batch):
    """Inverse of ``patchify`` written with reshapes (cropping the padding)."""
    levels = [np.empty((batch, -(-H // (1 << k)), -(-W // (1 << k)))) for k in range(L)]
    g = 0
    for b in range(batch):
        for k in range(L - 1, -1, -1):
            h, w = levels[k].shape[1:]
            ph, pw = -(-h // 8), -(-w // 8)
            tiles = blocks[g:g + ph * pw].reshape(ph, pw, 8, 8).transpose(0, 2, 1, 3).reshape(ph * 8, pw * 8)
            levels[k][b] = tiles[:h, :w]
            g += ph * pw
    return levels


def _level_sizes(H, W, L):
    return [(-(-H // (1 << k)), -(-W // (1 << k))) for k in range(L)]


# ------------------------------------------------------------------ checks

def check_zigzag(orc):
    zz = orc.zigzag()
    assert np.array_equal(zz, ZZ), "zigzag differs from the JPEG table"
    # independent construction: sort (row, col) by anti-diagonal d = r + c,
    # rows increasing on odd d and decreasing on even d
    pos = [(r, c) for r in range(8) for c in range(8)]
    pos.sort(key=lambda rc: (rc[0] + rc[1], rc[0] if (rc[0] + rc[1]) % 2 else -rc[0]))
    assert np.array_equal(zz, [r * 8 + c for r, c in pos])


def check_eob_offsets(orc):
    rng = np.random.default_rng(5)
    s = rng.integers(-30, 40, size=5000).astype(np.int32)
    eob = 33
    assert np.array_equal(orc.eob_offsets(s, eob), np.flatnonzero(s == eob))
    assert orc.eob_offsets(np.zeros(0, np.int32), eob).size == 0


def check_expand_handmade(orc):
    # eob = 20: run codes 4 .. 19 stand for 1 .. 16 zeros; literals are <= 3.
    eob = 20
    stream = [3, 19, 2, 20,          # block 0: 3, sixteen zeros, 2
              20,                    # block 1: empty
              -5, 4, -1, 20,         # block 2: -5, one zero, -1
              3, 4, 4, 4, 1, 20]     # block 3: 3, three single zeros, 1
    off = orc.eob_offsets(np.array(stream, np.int32), eob)
    assert list(off) == [3, 4, 8, 14]
    co, err = orc.expand_symbols(np.array(stream, np.int32), eob, off)
    assert err == 0
    want = np.zeros((4, 64), np.int64)
    want[0, 0] = 3          # zigzag position 0 -> natural 0
    want[0, 19] = 2         # position 17 -> natural 19 (row 2, column 3)
    want[2, 0] = -5
    want[2, 8] = -1         # position 2 -> natural 8 (row 1, column 0)
    want[3, 0] = 3
    want[3, 9] = 1          # position 4 -> natural 9 (row 1, column 1)
    assert np.array_equal(co, want), "hand-worked Alg. 1 blocks differ"
    # a full block of 64 literals 1 .. 64: coefficient at natural index ZZ[p] is p + 1
    eob = 100
    stream = list(range(1, 65)) + [eob]
    co, err = orc.expand_symbols(np.array(stream, np.int32), eob, [64])
    want = np.zeros(64, np.int64)
    want[ZZ] = np.arange(1, 65)
    assert err == 0 and np.array_equal(co[0], want)
    # literal zeros are coefficients too
    co, err = orc.expand_symbols(np.array([0, 0, 7, eob], np.int32), eob, [3])
    assert err == 0 and co[0, ZZ[2]] == 7 and np.count_nonzero(co[0]) == 1


def check_expand_roundtrip(orc):
    rng = np.random.default_rng(11)
    for density, max_abs, split, lz in ((0.05, 3, "greedy", 0.0), (0.3, 60, "random", 0.0),
                                        (0.9, 200, "greedy", 0.3), (0.0, 1, "greedy", 0.0),
                                        (1.0, 5, "random", 0.0), (0.02, 9, "random", 0.5)):
        blocks = random_blocks(rng, 300, density, max_abs)
        blocks[0] = 0
        blocks[1] = 0
        blocks[1, 63] = max_abs                     # a single value at the last position
        blocks[2] = 0
        blocks[2, 0] = -1                           # DC only
        eob = max_abs + 17 + int(rng.integers(0, 3))
        stream = []
        for blk in blocks:
            stream += zpr_encode_block(blk, eob, rng, split, lz)
        s = np.array(stream, np.int32)
        off = orc.eob_offsets(s, eob)
        assert off.size == blocks.shape[0]
        co, err = orc.expand_symbols(s, eob, off)
        assert err == 0
        assert np.array_equal(co, blocks), f"round trip failed (density {density}, split {split})"


def check_idct(orc):
    rng = np.random.default_rng(3)
    for _ in range(20):
        S = rng.integers(-50, 51, size=(8, 8)).astype(np.float64) * (rng.random((8, 8)) < 0.4)
        f = orc.idct8x8(S)
        assert np.allclose(f, scipy.fft.idctn(S, norm="ortho"), rtol=0, atol=1e-12)
        assert np.isclose((f * f).sum(), (S * S).sum(), rtol=1e-12, atol=1e-12)     # Parseval
        assert np.allclose(scipy.fft.dctn(f, norm="ortho"), S, rtol=0, atol=1e-11)
    S = np.zeros((8, 8))
    S[0, 0] = 40.0
    assert np.allclose(orc.idct8x8(S), 5.0, rtol=0, atol=1e-13)                  # DC / 8
    # a horizontal-only frequency varies along columns only (u rows, v columns)
    S = np.zeros((8, 8))
    S[0, 3] = 1.0
    f = orc.idct8x8(S)
    assert np.allclose(f, f[0:1, :], atol=1e-14) and not np.allclose(f, f[:, 0:1], atol=1e-3)


def check_unpatchify(orc):
    rng = np.random.default_rng(7)
    for H, W, L, batch in ((37, 53, 4, 2), (8, 8, 1, 1), (64, 24, 3, 1), (5, 130, 6, 3)):
        levels = [rng.normal(size=(batch, h, w)) for h, w in _level_sizes(H, W, L)]
        blocks = patchify(levels, L, batch)
        assert blocks.shape[0] == batch * orc.zpr_blocks(H, W, L)
        got = orc.unpatchify(np.nan_to_num(blocks, nan=1e300), H, W, L, batch)
        for k in range(L):
            assert np.array_equal(got[k], levels[k]), f"level {k} of {H}x{W}"


def check_zpr_decode_chain(orc):
    rng = np.random.default_rng(13)
    for H, W, L, batch in ((40, 24, 3, 2), (17, 33, 4, 1), (64, 64, 1, 1)):
        n = batch * orc.zpr_blocks(H, W, L)
        co = random_blocks(rng, n, 0.15, 40)
        eob = 40 + 17
        stream = np.array([t for blk in co for t in zpr_encode_block(blk, eob, rng, "random")], np.int32)
        want = place_blocks(scipy.fft.idctn(co.reshape(n, 8, 8).astype(np.float64), axes=(1, 2),
                                            norm="ortho").reshape(n, 64), H, W, L, batch)
        got, err = orc.zpr_decode(stream, eob, H, W, L, batch)
        assert err == 0
        for k in range(L):
            assert np.allclose(got[k], want[k], rtol=0, atol=1e-11), f"level {k}"


def check_zpr_errors(orc):
    H, W, L = 16, 16, 2                 # 4 + 1 blocks per image
    eob = 30
    good = [1, 2, eob] * 5
    assert orc.zpr_decode(np.array(good, np.int32), eob, H, W, L, 1)[1] == 0
    assert orc.zpr_decode(np.array(good[:-1], np.int32), eob, H, W, L, 1)[1] & 1      # last marker missing
    assert orc.zpr_decode(np.array(good + [eob], np.int32), eob, H, W, L, 1)[1] & 1   # one block too many
    assert orc.zpr_decode(np.array(good + [3], np.int32), eob, H, W, L, 1)[1] & 1     # trailing symbol
    long_blk = [1] * 65 + [eob]                                                       # 65 coefficients
    assert orc.zpr_decode(np.array(long_blk + good[3:], np.int32), eob, H, W, L, 1)[1] == 2
    runs = [eob - 1] * 4 + [1, eob]                                                   # 16 * 4 zeros + 1
    assert orc.zpr_decode(np.array(runs + good[3:], np.int32), eob, H, W, L, 1)[1] == 2
    assert orc.zpr_decode(np.array([eob + 1] + good, np.int32), eob, H, W, L, 1)[1] == 4
    # 66 symbols that produce only 60 coefficients: too many symbols all the same
    many = [eob + 1] * 6 + [1] * 60 + [eob]
    assert orc.zpr_decode(np.array(many + good[3:], np.int32), eob, H, W, L, 1)[1] == 6


ZPR_CHECKS = [check_zigzag, check_eob_offsets, check_expand_handmade, check_expand_roundtrip,
              check_idct, check_unpatchify, check_zpr_decode_chain, check_zpr_errors]
