"""GPU parity of the entropy-decoding step (include/pic_huff.h) against the
CPU oracle (oracle/huff_oracle.c), through the C ABI.

Bar: bit-exact.  Symbols equal the oracle's, status bits equal its error
flags, and on a malformed stream the GPU writes exactly the symbols the
oracle decoded before the error (the rest of `out` is left as it was).

Inputs: the workloads' ZpR streams coded by ``synth.make_huff_stream``, and
streams written by the test-side encoder of ``tests/pins_huff.py``:
- skewed alphabets from 1 to 4096 symbols;
- codes up to 24 bits long, beyond the 11-bit first-level table;
- fixed-length codes, which never resynchronise, so every subsequence goes
  through the repair kernel;
- streams from a few bits to a few million.
"""
import zlib

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import paper_2609_09020_amd as pkg  # noqa: E402
from paper_2609_09020_amd import decoder as D  # noqa: E402
from paper_2609_09020_amd import synth  # noqa: E402
from tests import pins_huff as H  # noqa: E402

DEV = "cuda:0"
FILL = -123456


@pytest.fixture(scope="module")
def orc():
    return oracle.default()


def _print_case(*a):
    print("case:", *a, flush=True)


def _gpu(data, n_bits, values, lengths, n_symbols, max_bits=None):
    data = np.frombuffer(bytes(data), np.uint8).copy() if not isinstance(data, np.ndarray) else data
    with pkg.HuffDecoder(max_bits or max(int(n_bits), 1)) as h:
        d = torch.from_numpy(np.ascontiguousarray(data, np.uint8)).to(DEV) if data.size else \
            torch.zeros(1, dtype=torch.uint8, device=DEV)
        v = torch.from_numpy(np.ascontiguousarray(values, np.int32)).to(DEV)
        ln = torch.from_numpy(np.ascontiguousarray(lengths, np.uint8)).to(DEV)
        out = torch.full((max(n_symbols, 1),), FILL, dtype=torch.int32, device=DEV)
        st = torch.full((1,), -7, dtype=torch.int32, device=DEV)
        out, st = h.decode(d, n_bits, v, ln, n_symbols, out=out, status=st)
        torch.cuda.synchronize()
        return out.cpu().numpy(), int(st.item())


def _check(orc, data, n_bits, values, lengths, n_symbols, max_bits=None):
    got, st = _gpu(data, n_bits, values, lengths, n_symbols, max_bits)
    want, err, _ = orc.huffman_decode(data, n_bits, values, lengths, n_symbols)
    assert st == err, f"status {st}, oracle flags {err}"
    k = want.size
    assert np.array_equal(got[:k], want), f"first mismatch at {np.flatnonzero(got[:k] != want)[:3]}"
    assert np.all(got[k:n_symbols] == FILL), "symbols written past the decodable ones"
    return got


WORKLOADS = [("pic64", 1), ("kodak768", 1), ("kodak768", 3), ("uhd4k", 1)]


@pytest.mark.parametrize("name,batch", WORKLOADS, ids=[f"{w}_b{b}" for w, b in WORKLOADS])
def test_workload_streams(orc, name, batch):
    wl = synth.WORKLOADS[name]
    hs = synth.workload_huff_stream(wl, batch=batch)
    _print_case(name, batch, hs.n_bits, hs.n_symbols, int(hs.lengths.max()))
    got = _check(orc, hs.data, hs.n_bits, hs.values, hs.lengths, hs.n_symbols)
    assert np.array_equal(got[:hs.n_symbols], hs.symbols)


ALPHABETS = [(1, 3000, 1.0), (2, 5000, 1.0), (3, 70, 1.0), (17, 40000, 1.5), (120, 100000, 1.1),
             (700, 200000, 0.9), (4096, 150000, 0.6)]


@pytest.mark.parametrize("n_sym,n,zipf", ALPHABETS, ids=[f"{a[0]}sym" for a in ALPHABETS])
def test_skewed_alphabets(orc, n_sym, n, zipf):
    rng = np.random.default_rng(zlib.crc32(f"{n_sym}".encode()))
    idx = H.skewed_stream(rng, n_sym, n, zipf)
    values, lengths = H.table_for(idx, n_sym, rng)
    data, n_bits = H.encode(idx, list(lengths))
    _print_case("alphabet", n_sym, n_bits, int(lengths.max()))
    got = _check(orc, data, n_bits, values, lengths, n)
    assert np.array_equal(got[:n], values[idx])


def _long_code_lengths():
    # Kraft sum exactly 1: lengths 1, 2, ..., 23, 24, 24
    return np.array(list(range(1, 25)) + [24], dtype=np.uint8)


def test_codes_up_to_24_bits(orc):
    lengths = _long_code_lengths()
    n_sym = lengths.size
    rng = np.random.default_rng(3)
    # every symbol, with the long ones frequent enough to straddle subsequences
    idx = np.concatenate([np.arange(n_sym), rng.integers(0, n_sym, 20000)])
    rng.shuffle(idx)
    values = (np.arange(n_sym) * 1000 - 7).astype(np.int32)
    data, n_bits = H.encode(idx, list(lengths))
    _print_case("long codes", n_bits)
    got = _check(orc, data, n_bits, values, lengths, idx.size)
    assert np.array_equal(got[:idx.size], values[idx])


@pytest.mark.parametrize("length", [3, 5, 7])
def test_fixed_length_codes_take_the_repair_path(orc, length):
    # a misaligned parse of a fixed-length code never falls into step: every
    # subsequence whose first bit is not a codeword start is repaired
    n_sym = 1 << length
    rng = np.random.default_rng(length)
    idx = rng.integers(0, n_sym, 30000)
    values = rng.permutation(n_sym).astype(np.int32) - 5
    lengths = np.full(n_sym, length, np.uint8)
    data, n_bits = H.encode(idx, list(lengths))
    _print_case("fixed length", length, n_bits)
    got = _check(orc, data, n_bits, values, lengths, idx.size)
    assert np.array_equal(got[:idx.size], values[idx])


@pytest.mark.parametrize("n", [1, 2, 10, 31, 32, 33, 64, 200])
def test_short_streams(orc, n):
    rng = np.random.default_rng(n)
    idx = H.skewed_stream(rng, 5, max(n, 5), 1.2)[:n]
    values, lengths = H.table_for(np.concatenate([idx, np.arange(5)]), 5, rng)
    data, n_bits = H.encode(idx, list(lengths))
    got = _check(orc, data, n_bits, values, lengths, n)
    assert np.array_equal(got[:n], values[idx])


def test_exact_subsequence_multiples(orc):
    # 128 two-bit codewords: 256 bits, two whole subsequences
    lengths = np.array([2, 2, 2, 2], np.uint8)
    rng = np.random.default_rng(1)
    idx = rng.integers(0, 4, 128)
    values = np.array([5, 6, 7, 8], np.int32)
    data, n_bits = H.encode(idx, list(lengths))
    assert n_bits == 256
    got = _check(orc, data, n_bits, values, lengths, 128)
    assert np.array_equal(got[:128], values[idx])


MALFORMED = ["truncated", "too_many_requested", "no_bits", "incomplete_code", "bad_length", "oversubscribed",
             "fewer_requested"]


@pytest.mark.parametrize("name", MALFORMED)
def test_malformed(orc, name):
    rng = np.random.default_rng(5)
    idx = H.skewed_stream(rng, 40, 20000, 1.2)
    values, lengths = H.table_for(idx, 40, rng)
    data, n_bits = H.encode(idx, list(lengths))
    n = idx.size
    if name == "truncated":
        n_bits = n_bits // 2
        data = data[:(n_bits + 7) // 8]
    elif name == "too_many_requested":
        n = n + 50
    elif name == "no_bits":
        data, n_bits = b"", 0
    elif name == "incomplete_code":
        # drop the table's longest entry: its codewords (and their prefixes
        # shared with nothing else) no longer start any codeword
        last = int(np.argmax(lengths))
        keep = np.ones(lengths.size, bool)
        keep[last] = False
        values, lengths = values[keep], lengths[keep]
    elif name == "bad_length":
        lengths = lengths.copy()
        lengths[3] = 0
    elif name == "oversubscribed":
        lengths = lengths.copy()
        lengths[:3] = 1
    elif name == "fewer_requested":
        n = n // 3
    _print_case("malformed", name)
    _check(orc, data, n_bits, values, lengths, n, max_bits=max(n_bits, 1))


def test_large_stream_sampled(orc):
    # the bench's input: 64 Kodak-size images' symbols, every symbol checked
    wl = synth.WORKLOADS["kodak768_b64"]
    hs = synth.workload_huff_stream(wl)
    _print_case("kodak768_b64", hs.n_bits, hs.n_symbols)
    got, st = _gpu(hs.data, hs.n_bits, hs.values, hs.lengths, hs.n_symbols)
    assert st == 0 and np.array_equal(got[:hs.n_symbols], hs.symbols)


# 2^24 + 1000 byte-long codewords: 1,048,639 subsequences, more workgroups
# than the write kernel sums by itself, so the fix kernel turns the
# per-workgroup counts into prefixes
N_PREFIX = (1 << 24) + 1000


def test_many_workgroups_identity_code():
    # 256 codes of 8 bits: the decoded stream is the byte stream, mapped
    rng = np.random.default_rng(11)
    data = rng.integers(0, 256, N_PREFIX, dtype=np.uint8)
    values = (np.arange(256, dtype=np.int32) * 3 - 100)
    lengths = np.full(256, 8, np.uint8)
    _print_case("identity code", N_PREFIX * 8)
    got, st = _gpu(data, N_PREFIX * 8, values, lengths, N_PREFIX)
    assert st == 0 and np.array_equal(got[:N_PREFIX], values[data])


def test_many_workgroups_bad_pattern_near_the_end():
    # 255 codes of 8 bits: the byte 0xff starts no codeword; decoding stops
    # at the one planted near the end (the same construction, small, is
    # checked against the oracle below)
    rng = np.random.default_rng(12)
    for n, k in ((N_PREFIX, N_PREFIX - 5000), (3000, 2100)):
        data = rng.integers(0, 255, n, dtype=np.uint8)
        data[k] = 255
        values = (np.arange(255, dtype=np.int32) * 7 + 1)
        lengths = np.full(255, 8, np.uint8)
        _print_case("bad pattern", n * 8, k)
        got, st = _gpu(data, n * 8, values, lengths, n)
        assert st == D.PIC_HUFF_ERR_CODE
        assert np.array_equal(got[:k], values[data[:k]]) and np.all(got[k:n] == FILL)
        if n < 10000:
            want, err, used = oracle.default().huffman_decode(data, n * 8, values, lengths, n)
            assert err == D.PIC_HUFF_ERR_CODE and want.size == k and used == 8 * k


def test_reuse_and_batch_of_calls(orc):
    rng = np.random.default_rng(8)
    with pkg.HuffDecoder(1 << 22) as h:
        for n_sym, n in ((30, 50000), (3, 100), (300, 120000)):
            idx = H.skewed_stream(rng, n_sym, n, 1.1)
            values, lengths = H.table_for(idx, n_sym, rng)
            data, n_bits = H.encode(idx, list(lengths))
            d = torch.from_numpy(np.frombuffer(data, np.uint8).copy()).to(DEV)
            out, st = h.decode(d, n_bits, torch.from_numpy(values).to(DEV), torch.from_numpy(lengths).to(DEV), n)
            torch.cuda.synchronize()
            assert int(st.item()) == 0 and np.array_equal(out.cpu().numpy(), values[idx])


def test_two_handles_on_two_streams():
    # two handles decoding at the same time on two streams, each with its own
    # one-launch hand-off words, eight calls each, not synchronised between
    rng = np.random.default_rng(12)
    jobs = []
    for n in (60000, 45000):
        idx = H.skewed_stream(rng, 40, n, 1.1)
        values, lengths = H.table_for(idx, 40, rng)
        data, n_bits = H.encode(idx, list(lengths))
        jobs.append((torch.from_numpy(np.frombuffer(data, np.uint8).copy()).to(DEV), n_bits,
                     torch.from_numpy(values).to(DEV), torch.from_numpy(lengths).to(DEV), n, values[idx]))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    handles = [pkg.HuffDecoder(1 << 20), pkg.HuffDecoder(1 << 20)]
    outs = [[], []]
    torch.cuda.synchronize()
    for _ in range(8):
        for j in range(2):
            d, n_bits, v, ln, n, _ = jobs[j]
            with torch.cuda.stream(streams[j]):
                outs[j].append(handles[j].decode(d, n_bits, v, ln, n, stream=streams[j].cuda_stream))
    torch.cuda.synchronize()
    for j in range(2):
        for out, st in outs[j]:
            assert int(st.item()) == 0 and np.array_equal(out.cpu().numpy(), jobs[j][5])
    for h in handles:
        h.close()


def test_argument_rejection():
    with pkg.HuffDecoder(4096) as h:
        buf = torch.zeros(1024, dtype=torch.uint8, device=DEV)
        v = torch.zeros(8, dtype=torch.int32, device=DEV)
        ln = torch.ones(8, dtype=torch.uint8, device=DEV)
        out = torch.zeros(64, dtype=torch.int32, device=DEV)
        st = torch.zeros(1, dtype=torch.int32, device=DEV)
        args = [h.handle, buf.data_ptr(), 100, v.data_ptr(), ln.data_ptr(), 8, 10, out.data_ptr(), st.data_ptr()]
        assert D.pic_huff_decode(*args) == D.PIC_OK
        torch.cuda.synchronize()
        bad = [(2, 4097), (2, -1), (5, 0), (5, 4097), (6, -1), (3, v.data_ptr() + 2), (7, out.data_ptr() + 2),
               (8, 0), (1, 0)]
        for pos, val in bad:
            a = list(args)
            a[pos] = val
            assert D.pic_huff_decode(*a) == D.PIC_E_INVALID, (pos, val)
        a = list(args)
        a[6] = 0
        assert D.pic_huff_decode(*a) == D.PIC_OK                 # nothing to decode
        info = h.info()
        assert info["bits_per_thread"] == 64 and info["lut_bits"] == 11 and info["max_bits"] == 4096


def test_full_decoder_chain(orc):
    # bits -> symbols -> latents -> image, every stage on the GPU, checked
    # against the stage's own oracle on the stage's GPU input
    wl = synth.WORKLOADS["kodak768"]
    H_, W_, L = wl.height, wl.width, wl.levels
    zs = synth.workload_zpr_stream(wl)
    hs = synth.make_huff_stream(zs.symbols)
    inp = synth.workload_inputs(wl)
    with pkg.HuffDecoder(hs.n_bits) as hd, pkg.ZprDecoder(H_, W_, L) as zd, \
            pkg.Decoder(H_, W_, wl.widths) as dec:
        sym, st1 = hd.decode(torch.from_numpy(hs.data).to(DEV), hs.n_bits, torch.from_numpy(hs.values).to(DEV),
                             torch.from_numpy(hs.lengths).to(DEV), hs.n_symbols)
        lat, st2 = zd.decode(sym, zs.eob, 1)
        img = dec.run(lat, torch.from_numpy(inp.weights).to(DEV), torch.from_numpy(inp.biases).to(DEV))
        torch.cuda.synchronize()
        assert int(st1.item()) == 0 and int(st2.item()) == 0
        assert np.array_equal(sym.cpu().numpy(), zs.symbols)
        lat_np = [t.cpu().numpy() for t in lat]
        want_lat, _ = orc.zpr_decode(zs.symbols, zs.eob, H_, W_, L, 1)
        for k in range(L):
            assert np.abs(lat_np[k] - want_lat[k]).max() <= 1e-6 * 64 * 60 * 8
        ref = orc.decode(lat_np, inp.weights, inp.biases, wl.widths, H_, W_, out="clamped")
        assert np.abs(img.cpu().numpy() - ref).max() <= 1e-5
