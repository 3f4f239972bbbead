"""Pins of the Huffman part of the CPU oracle (symbols from the bitstream).

What pins what (PIC, Sec. 3.3 and Sec. 4.1; the readings are in
oracle/huff_oracle.c):
  * canonical code  -- DEFLATE's fixed literal/length code, whose codewords
                       RFC 1951 prints (tests/golden/deflate_fixed_code.txt),
                       and an independent construction here (sort by length
                       then table order, count upwards, shift on each longer
                       length) on random complete and incomplete codes;
  * decoding        -- a hand-worked stream, and round trips through a
                       Huffman encoder written here (heap merging of symbol
                       frequencies, MSB-first packing) on skewed alphabets of
                       several sizes, including a one-symbol alphabet;
  * error flags     -- truncated streams, a pattern outside an incomplete
                       code, invalid and over-subscribed tables.
"""
from __future__ import annotations

import heapq
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ------------------------------------------------- a Huffman encoder

def huffman_lengths(freqs, max_len=24):
    """Code lengths of a Huffman code for the given (positive) frequencies:
    repeatedly merge the two least frequent subtrees; a symbol's length is
    its depth.  One symbol gets length 1.  Raises if a length exceeds max_len."""
    n = len(freqs)
    if n == 1:
        return [1]
    heap = [(f, i, [i]) for i, f in enumerate(freqs)]
    heapq.heapify(heap)
    depth = [0] * n
    uid = n
    while len(heap) > 1:
        f1, _, s1 = heapq.heappop(heap)
        f2, _, s2 = heapq.heappop(heap)
        for i in s1 + s2:
            depth[i] += 1
        heapq.heappush(heap, (f1 + f2, uid, s1 + s2))
        uid += 1
    if max(depth) > max_len:
        raise ValueError("code too long for the test")
    return depth


def canonical_codes(lengths):
    """Codes by sorting: symbols in (length, table order); the first gets 0;
    each next code is the previous plus one, shifted left by the growth in
    length."""
    lengths = [int(l) for l in lengths]
    order = sorted(range(len(lengths)), key=lambda i: (lengths[i], i))
    codes = [0] * len(lengths)
    code, prev_len = 0, lengths[order[0]]
    for k, i in enumerate(order):
        if k > 0:
            code = (code + 1) << (lengths[i] - prev_len)
        codes[i] = code
        prev_len = lengths[i]
    return codes


def encode(symbol_indices, lengths):
    """MSB-first bitstream of the symbols (indices into the table):
    (bytes, number of bits)."""
    lengths = [int(l) for l in lengths]
    codes = canonical_codes(lengths)
    bits = []
    for s in symbol_indices:
        c, l = codes[s], lengths[s]
        bits.extend((c >> (l - 1 - j)) & 1 for j in range(l))
    n_bits = len(bits)
    bits += [0] * (-n_bits % 8)
    arr = np.packbits(np.array(bits, dtype=np.uint8)) if bits else np.zeros(0, np.uint8)
    return arr.tobytes(), n_bits


def skewed_stream(rng, n_sym, n, zipf=1.3):
    """n symbol indices over an alphabet of n_sym, Zipf-like frequencies,
    every symbol used at least once."""
    p = 1.0 / np.arange(1, n_sym + 1) ** zipf
    p /= p.sum()
    idx = rng.choice(n_sym, size=n, p=p)
    idx[:n_sym] = np.arange(n_sym)
    rng.shuffle(idx)
    return idx


def table_for(idx, n_sym, rng=None):
    """Values and lengths of a Huffman table for the symbol indices; values
    are distinct arbitrary int32s (a shuffled range when rng is given)."""
    freqs = np.bincount(idx, minlength=n_sym)
    lengths = huffman_lengths(list(freqs))
    values = np.arange(n_sym, dtype=np.int64) * 7 - 3 * n_sym
    if rng is not None:
        values = rng.permutation(values)
    return values.astype(np.int32), np.array(lengths, dtype=np.uint8)


# ------------------------------------------------------------------ checks

def check_huffman_rfc_fixed(orc):
    rows = [l.split() for l in open(os.path.join(GOLDEN, "deflate_fixed_code.txt")) if not l.startswith("#")]
    lengths = np.zeros(288, np.uint8)
    for a, b, ln, _, _ in rows:
        lengths[int(a):int(b) + 1] = int(ln)
    codes, err = orc.huffman_codes(lengths)
    assert err == 0
    for a, b, ln, c0, c1 in rows:
        assert format(int(codes[int(a)]), f"0{ln}b") == c0, f"first code of {a}..{b}"
        assert format(int(codes[int(b)]), f"0{ln}b") == c1, f"last code of {a}..{b}"


def check_huffman_canonical(orc):
    rng = np.random.default_rng(2)
    for n_sym in (1, 2, 3, 17, 100, 300):
        idx = skewed_stream(rng, n_sym, 4 * n_sym + 50)
        _, lengths = table_for(idx, n_sym)
        codes, err = orc.huffman_codes(lengths)
        assert err == 0
        assert list(codes) == canonical_codes(list(lengths))
        # prefix-free
        words = sorted(format(int(c), f"0{l}b") for c, l in zip(codes, lengths))
        assert all(not b.startswith(a) for a, b in zip(words, words[1:]))
    # an incomplete code (Kraft sum below 1) is still canonical
    lengths = [2, 3, 3, 5, 6]
    codes, err = orc.huffman_codes(lengths)
    assert err == 0 and list(codes) == canonical_codes(lengths)


def check_huffman_handmade(orc):
    # lengths 1, 2, 3, 3 -> codes 0, 10, 110, 111
    values, lengths = [10, 20, 30, 40], [1, 2, 3, 3]
    bits = "0" + "10" + "110" + "111" + "0"
    data = int(bits + "0" * (-len(bits) % 8), 2).to_bytes((len(bits) + 7) // 8, "big")
    out, err, used = orc.huffman_decode(data, len(bits), values, lengths, 5)
    assert err == 0 and list(out) == [10, 20, 30, 40, 10] and used == 10
    # table order decides among equal lengths: lengths 2, 1, 2 -> codes 10, 0, 11
    out, err, _ = orc.huffman_decode(bytes([0b10011000]), 5, [7, 8, 9], [2, 1, 2], 3)
    assert err == 0 and list(out) == [7, 8, 9]


def check_huffman_roundtrip(orc):
    rng = np.random.default_rng(4)
    for n_sym, n, zipf in ((1, 200, 1.0), (2, 500, 1.0), (5, 3000, 2.0), (90, 20000, 1.2), (700, 30000, 0.8)):
        idx = skewed_stream(rng, n_sym, n, zipf)
        values, lengths = table_for(idx, n_sym, rng)
        data, n_bits = encode(idx, list(lengths))
        out, err, used = orc.huffman_decode(data, n_bits, values, lengths, n)
        assert err == 0 and used == n_bits, (n_sym, err)
        assert np.array_equal(out, values[idx]), f"round trip failed ({n_sym} symbols)"


def check_huffman_errors(orc):
    values, lengths = [10, 20, 30, 40], [1, 2, 3, 3]
    data = bytes([0b01011011, 0b10000000])
    assert orc.huffman_decode(data, 10, values, lengths, 6)[1] == 1          # runs out of bits
    assert orc.huffman_decode(data, 9, values, lengths, 5)[1] == 1           # ends inside a codeword
    # incomplete code {0, 10}: the pattern 11 starts no codeword
    assert orc.huffman_decode(bytes([0b01100000]), 8, [1, 2], [1, 2], 3)[1] == 2
    assert orc.huffman_decode(data, 10, [1, 2], [0, 1], 1)[1] == 4            # length 0
    assert orc.huffman_decode(data, 10, [1, 2], [25, 1], 1)[1] == 4           # length 25
    assert orc.huffman_decode(data, 10, [1, 2, 3], [1, 1, 1], 1)[1] == 4      # over-subscribed
    out, err, _ = orc.huffman_decode(data, 10, values, lengths, 0)            # nothing asked
    assert err == 0 and out.size == 0


HUFF_CHECKS = [check_huffman_rfc_fixed, check_huffman_canonical, check_huffman_handmade,
               check_huffman_roundtrip, check_huffman_errors]
