"""GPU parity of the latent-decoding step (include/pic_zpr.h) against the CPU
oracle (oracle/zpr_oracle.c), through the C ABI.

Bars:
  * pic_zpr_expand (Alg. 1's integer output) -- bit-exact;
  * status bits -- equal to the oracle's error flags;
  * pic_zpr_decode (fp32 separable inverse DCT) -- per sample
        |gpu - oracle| <= 1e-6 * sum |S| of the sample's block  (+ 1e-30)
    The kernel forms T = S B^T (eight fp32 fused multiply-adds per value,
    |basis| <= 1/2) and then B T (eight more), with the basis rounded to fp32.
    Each stage adds at most 8 u_32 of its absolute sum, so the error is at most
    about (8 + 8 + 2) * 2^-24 * (1/2 * 1/2) * sum|S| = 2.7e-7 * sum|S|.  The
    test allows 1e-6 * sum|S|;
  * samples and blocks a malformed stream does not delimit stay untouched.

Inputs are the seeded streams of ``synth.make_zpr_stream`` (the workloads'
pyramid shapes) and streams written by the test-side ZpR encoder of
``tests/pins_zpr.py`` (dense blocks, long runs, literal zeros, negative
markers).
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
from tests import pins_zpr  # noqa: E402

DEV = "cuda:0"


@pytest.fixture(scope="module")
def orc():
    return oracle.default()


def _print_case(*a):
    print("case:", *a, flush=True)


def _gpu_expand(H, W, L, batch, symbols, eob, max_batch=None):
    with pkg.ZprDecoder(H, W, L, max_batch or max(batch, 1)) as z:
        sym = torch.from_numpy(np.ascontiguousarray(symbols, np.int32)).to(DEV)
        co, st = z.expand(sym, eob, batch)
        torch.cuda.synchronize()
        return co.cpu().numpy(), int(st.item())


def _gpu_decode(H, W, L, batch, symbols, eob, fill=None, max_batch=None):
    with pkg.ZprDecoder(H, W, L, max_batch or max(batch, 1)) as z:
        sym = torch.from_numpy(np.ascontiguousarray(symbols, np.int32)).to(DEV)
        lat = None
        if fill is not None:
            lat = [torch.full((batch,) + z.level_shape(k), fill, dtype=torch.float32, device=DEV)
                   for k in range(L)]
        lat, st = z.decode(sym, eob, batch, latents=lat)
        torch.cuda.synchronize()
        return [t.cpu().numpy() for t in lat], int(st.item())


def _oracle_expand(orc, symbols, eob, n_blocks):
    off = orc.eob_offsets(symbols, eob)[:n_blocks]
    return orc.expand_symbols(symbols, eob, off)


def _block_abs_sums(orc, symbols, eob, H, W, L, batch):
    """Per-sample sum |S| of the sample's block (for the decode tolerance)."""
    nb = batch * orc.zpr_blocks(H, W, L)
    co, _ = _oracle_expand(orc, symbols, eob, nb)
    sums = np.zeros((nb, 64))
    sums[:co.shape[0]] = np.abs(co.astype(np.float64)).sum(axis=1, keepdims=True)
    return pins_zpr.place_blocks(sums, H, W, L, batch)


def _assert_block_bound(orc, got, want, symbols, eob, H, W, L, batch):
    """Every sample within 1e-6 * sum|S| of its block (the bound in the module
    docstring); a sample no decoded block covers has sum 0, so it must equal
    the oracle's (the fill value) exactly."""
    sums = _block_abs_sums(orc, symbols, eob, H, W, L, batch)
    for k in range(L):
        diff = np.abs(got[k].astype(np.float64) - want[k])
        tol = 1e-6 * sums[k] + 1e-30
        bad = diff > tol
        assert not bad.any(), (f"level {k}: {bad.sum()} samples off, max diff {diff.max():.3g}, "
                               f"max ratio {(diff / tol).max():.3g}")


def _check_decode(orc, H, W, L, batch, symbols, eob):
    got, st = _gpu_decode(H, W, L, batch, symbols, eob)
    want, err = orc.zpr_decode(symbols, eob, H, W, L, batch)
    assert st == err
    _assert_block_bound(orc, got, want, symbols, eob, H, W, L, batch)


SHAPES = [("pic64", 64, 64, 4, 1), ("ragged", 37, 53, 4, 3), ("tiny", 8, 8, 1, 1), ("one_px", 1, 1, 3, 2),
          ("kodak768", 512, 768, 7, 1), ("kodak768_L8", 512, 768, 8, 2), ("tall", 300, 17, 5, 2)]


@pytest.mark.parametrize("name,H,W,L,batch", SHAPES, ids=[s[0] for s in SHAPES])
def test_expand_bit_exact(orc, name, H, W, L, batch):
    s = synth.make_zpr_stream(H, W, L, batch, seed=zlib.crc32(name.encode()) % 1000)
    _print_case("expand", name, s.symbols.size)
    got, st = _gpu_expand(H, W, L, batch, s.symbols, s.eob)
    want, err = _oracle_expand(orc, s.symbols, s.eob, s.blocks)
    assert st == 0 and err == 0
    assert np.array_equal(got, want)


@pytest.mark.parametrize("name,H,W,L,batch", SHAPES, ids=[s[0] for s in SHAPES])
def test_decode_matches_oracle(orc, name, H, W, L, batch):
    s = synth.make_zpr_stream(H, W, L, batch, seed=zlib.crc32(name.encode()) % 1000 + 1)
    _print_case("decode", name, s.symbols.size)
    _check_decode(orc, H, W, L, batch, s.symbols, s.eob)


ENCODED = [  # (name, density, max_abs, split, literal-zero prob, eob offset)
    ("dense_full", 1.0, 9, "greedy", 0.0, 0), ("dense_random", 0.9, 300, "random", 0.2, 3),
    ("sparse_long_runs", 0.02, 5, "greedy", 0.0, 0), ("runs_random_split", 0.2, 40, "random", 0.5, 1),
    ("empty", 0.0, 1, "greedy", 0.0, 0), ("big_values", 0.3, 2_000_000, "random", 0.0, 0),
]


@pytest.mark.parametrize("name,density,max_abs,split,lz,eoff", ENCODED, ids=[e[0] for e in ENCODED])
def test_encoded_streams(orc, name, density, max_abs, split, lz, eoff):
    H, W, L, batch = 48, 80, 4, 2
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    nb = batch * orc.zpr_blocks(H, W, L)
    co = pins_zpr.random_blocks(rng, nb, density, max_abs)
    eob = max_abs + 17 + eoff
    stream = np.array([t for blk in co for t in pins_zpr.zpr_encode_block(blk, eob, rng, split, lz)], np.int32)
    _print_case("encoded", name, stream.size)
    got, st = _gpu_expand(H, W, L, batch, stream, eob)
    assert st == 0 and np.array_equal(got, co)
    _check_decode(orc, H, W, L, batch, stream, eob)


def test_negative_marker(orc):
    # eob = -3: run codes -19 .. -4, literals below -19
    H, W, L = 24, 24, 2
    rng = np.random.default_rng(1)
    nb = orc.zpr_blocks(H, W, L)
    co = -20 - np.abs(pins_zpr.random_blocks(rng, nb, 0.3, 50))
    co[pins_zpr.random_blocks(rng, nb, 0.5, 1) == 0] = 0
    eob = -3
    stream = np.array([t for blk in co for t in pins_zpr.zpr_encode_block(blk, eob)], np.int32)
    got, st = _gpu_expand(H, W, L, 1, stream, eob)
    assert st == 0 and np.array_equal(got, co)
    _check_decode(orc, H, W, L, 1, stream, eob)


@pytest.mark.parametrize("batch", [1, 40], ids=["short", "long"])
def test_marker_only_stream_spans_many_chunks(orc, batch):
    # every block empty: the stream is all markers (a full chunk of them each)
    H, W, L = 512, 768, 7
    nb = batch * orc.zpr_blocks(H, W, L)
    eob = 77
    stream = np.full(nb, eob, np.int32)
    got, st = _gpu_decode(H, W, L, batch, stream, eob, fill=5.0)
    assert st == 0
    for g in got:
        assert not np.any(g)


def test_long_stream_dense_blocks(orc):
    # 1024-symbol chunks whose blocks are all 64 literals long (65 symbols)
    H, W, L, batch = 256, 256, 3, 4
    rng = np.random.default_rng(9)
    nb = batch * orc.zpr_blocks(H, W, L)
    co = pins_zpr.random_blocks(rng, nb, 1.0, 30)
    eob = 30 + 17
    stream = np.array([t for blk in co for t in pins_zpr.zpr_encode_block(blk, eob)], np.int32)
    assert stream.size >= 262144
    got, st = _gpu_expand(H, W, L, batch, stream, eob)
    assert st == 0 and np.array_equal(got, co)
    _check_decode(orc, H, W, L, batch, stream, eob)


MALFORMED = ["missing_last_marker", "extra_marker", "trailing_symbols", "symbol_above_eob",
             "too_many_markers", "empty_stream", "block_too_long", "run_overflow", "first_block_too_long"]


def _malformed(name, good, eob):
    g = list(good)
    if name == "missing_last_marker":
        return g[:-1]
    if name == "extra_marker":
        return g + [eob]
    if name == "trailing_symbols":
        return g + [1, 2]
    if name == "symbol_above_eob":
        return [eob + 5] + g[:40] + [eob + 1] + g[40:]
    if name == "too_many_markers":
        return g + [eob] * 300
    if name == "empty_stream":
        return []
    if name == "block_too_long":
        i = len(g) // 2
        while g[i] != eob:
            i += 1
        return g[:i + 1] + [3] * 70 + [eob] + g[i + 1:]
    if name == "run_overflow":
        i = len(g) // 3
        while g[i] != eob:
            i += 1
        return g[:i + 1] + [eob - 1] * 5 + [eob] + g[i + 1:]
    if name == "first_block_too_long":
        return [2] * 66 + g
    raise KeyError(name)


# (H, W, L, batch): a short stream (256-symbol chunks) and a long one (1024)
MALFORMED_SHAPES = [(64, 96, 4, 2), (512, 768, 7, 6)]


@pytest.mark.parametrize("shape", MALFORMED_SHAPES, ids=["short", "long"])
@pytest.mark.parametrize("name", MALFORMED)
def test_malformed_streams(orc, name, shape):
    H, W, L, batch = shape
    s = synth.make_zpr_stream(H, W, L, batch, seed=7)
    stream = np.array(_malformed(name, s.symbols, s.eob), np.int32)
    _print_case("malformed", name, stream.size)
    fill = 1234.5
    got, st = _gpu_decode(H, W, L, batch, stream, s.eob, fill=fill)
    want, err = orc.zpr_decode(stream, s.eob, H, W, L, batch, fill=fill)
    assert st == err and err != 0
    if err & D.PIC_ZPR_ERR_OVERFLOW:
        return   # the values of an over-long block are unspecified; the flag is the contract
    _assert_block_bound(orc, got, want, stream, s.eob, H, W, L, batch)


def _replace_blocks(symbols, eob, body, every):
    """The stream with every `every`-th block's symbols replaced by `body`."""
    out, cur, k = [], [], 0
    for t in symbols:
        if t != eob:
            cur.append(t)
            continue
        out += (body if k % every == every - 1 else cur) + [eob]
        cur, k = [], k + 1
    return out + cur


# block bodies at the 64-symbol / 64-coefficient limits (Alg. 1: a block
# holds 64 coefficients): exactly 64 is a whole block, 65 is flagged
LIMIT_BODIES = {
    "values_64": (lambda eob: [((v * 7) % 23) - 11 or 1 for v in range(64)], 0),
    "runs_64": (lambda eob: [eob - 1] * 4, 0),
    "runs_and_values_64": (lambda eob: [5, eob - 1, -3] + [eob - 2] * 3 + [4], 0),
    "values_65": (lambda eob: [2] * 65, D.PIC_ZPR_ERR_OVERFLOW),
    "runs_65": (lambda eob: [eob - 1] * 4 + [1], D.PIC_ZPR_ERR_OVERFLOW),
}


@pytest.mark.parametrize("shape", MALFORMED_SHAPES, ids=["short", "long"])
@pytest.mark.parametrize("name", list(LIMIT_BODIES))
def test_blocks_at_the_length_limit(orc, name, shape):
    H, W, L, batch = shape
    s = synth.make_zpr_stream(H, W, L, batch, seed=11)
    body_of, flag = LIMIT_BODIES[name]
    body = body_of(s.eob)
    assert all(t != s.eob for t in body)
    stream = np.array(_replace_blocks(s.symbols, s.eob, body, every=13), np.int32)
    _print_case("limit", name, stream.size)
    fill = -77.25
    got, st = _gpu_decode(H, W, L, batch, stream, s.eob, fill=fill)
    want, err = orc.zpr_decode(stream, s.eob, H, W, L, batch, fill=fill)
    assert err == flag and st == err
    if flag:
        return   # the values of an over-long block are unspecified; the flag is the contract
    _assert_block_bound(orc, got, want, stream, s.eob, H, W, L, batch)


def test_full_size_batch(orc):
    # the launch the benchmark times (768x512, 7 levels, 64 images): every
    # sample of every image compared with the oracle's decode of the batch
    wl = synth.WORKLOADS["kodak768_b64"]
    s = synth.workload_zpr_stream(wl)
    H, W, L, batch = wl.height, wl.width, wl.levels, wl.batch
    _print_case("full size", wl.name, s.symbols.size)
    got, st = _gpu_decode(H, W, L, batch, s.symbols, s.eob)
    want, err = orc.zpr_decode(s.symbols, s.eob, H, W, L, batch)
    assert st == 0 and err == 0
    _assert_block_bound(orc, got, want, s.symbols, s.eob, H, W, L, batch)


def test_two_runs_reuse_scratch(orc):
    # the arrival counter and prefix scratch are reused: a second, smaller run
    H, W, L = 64, 64, 4
    with pkg.ZprDecoder(H, W, L, 4) as z:
        for batch, seed in ((4, 1), (1, 2), (3, 3)):
            s = synth.make_zpr_stream(H, W, L, batch, seed=seed)
            co, st = z.expand(torch.from_numpy(s.symbols).to(DEV), s.eob, batch)
            torch.cuda.synchronize()
            want, err = _oracle_expand(orc, s.symbols, s.eob, s.blocks)
            assert int(st.item()) == 0 and np.array_equal(co.cpu().numpy(), want)


def test_side_stream_and_batch_zero(orc):
    H, W, L = 40, 40, 3
    s = synth.make_zpr_stream(H, W, L, 2, seed=4)
    with pkg.ZprDecoder(H, W, L, 2) as z:
        sym = torch.from_numpy(s.symbols).to(DEV)
        st = torch.full((1,), -7, dtype=torch.int32, device=DEV)
        z.decode(sym, s.eob, 0, status=st)                     # enqueues nothing
        torch.cuda.synchronize()
        assert int(st.item()) == -7
        side = torch.cuda.Stream()
        with torch.cuda.stream(side):
            lat, st2 = z.decode(sym, s.eob, 2)
        side.synchronize()
        want, err = orc.zpr_decode(s.symbols, s.eob, H, W, L, 2)
        assert int(st2.item()) == 0 and err == 0
        _assert_block_bound(orc, [t.cpu().numpy() for t in lat], want, s.symbols, s.eob, H, W, L, 2)


def test_argument_rejection():
    with pkg.ZprDecoder(64, 64, 4, 2) as z:
        h = z.handle
        bpi = z.blocks_per_image
        sym = torch.zeros(1024, dtype=torch.int32, device=DEV)
        st = torch.zeros(4, dtype=torch.int32, device=DEV)
        co = torch.zeros((2 * bpi + 1, 64), dtype=torch.int32, device=DEV)
        p = sym.data_ptr()
        ok = D.pic_zpr_expand(h, 1, p, 10, 20, co.data_ptr(), st.data_ptr())
        torch.cuda.synchronize()
        assert ok == D.PIC_OK
        assert D.pic_zpr_expand(h, 3, p, 10, 20, co.data_ptr(), st.data_ptr()) == D.PIC_E_INVALID  # batch
        assert D.pic_zpr_expand(h, 1, p, 65 * bpi + 1, 20, co.data_ptr(), st.data_ptr()) == D.PIC_E_INVALID
        assert D.pic_zpr_expand(h, 1, p, -1, 20, co.data_ptr(), st.data_ptr()) == D.PIC_E_INVALID
        assert D.pic_zpr_expand(h, 1, p, 10, -2**31, co.data_ptr(), st.data_ptr()) == D.PIC_E_INVALID
        assert D.pic_zpr_expand(h, 1, p, 10, 2**31 - 1, co.data_ptr(), st.data_ptr()) == D.PIC_E_INVALID
        assert D.pic_zpr_expand(h, 1, p, 10, 20, co.data_ptr() + 4, st.data_ptr()) == D.PIC_E_INVALID
        assert D.pic_zpr_expand(h, 1, p + 2, 10, 20, co.data_ptr(), st.data_ptr()) == D.PIC_E_INVALID
        assert D.pic_zpr_expand(h, 1, p, 10, 20, co.data_ptr(), 0) == D.PIC_E_INVALID
        assert D.pic_zpr_expand(h, 1, 0, 10, 20, co.data_ptr(), st.data_ptr()) == D.PIC_E_INVALID
        lat = [0] * 4
        assert D.pic_zpr_decode(h, 1, p, 10, 20, lat, st.data_ptr()) == D.PIC_E_INVALID
        assert D.pic_zpr_decode(h, 1, p, 10, 20, None, st.data_ptr()) == D.PIC_E_INVALID
        info = z.info()
        assert info["blocks_per_image"] == bpi == oracle.default().zpr_blocks(64, 64, 4)
        assert info["symbols_per_chunk"] == 256 and info["scratch_bytes"] > 0


def test_latents_feed_the_synthesis(orc):
    # symbols -> latents (GPU) -> image (GPU), checked step by step: the
    # latents against the oracle's, and the image against the synthesis
    # oracle applied to the GPU's own latents (the synthesis parity bar)
    wl = synth.WORKLOADS["kodak768"]
    H, W, L = wl.height, wl.width, wl.levels
    s = synth.workload_zpr_stream(wl)
    inp = synth.workload_inputs(wl)
    got, st = _gpu_decode(H, W, L, 1, s.symbols, s.eob)
    assert st == 0
    want, _ = orc.zpr_decode(s.symbols, s.eob, H, W, L, 1)
    sums = _block_abs_sums(orc, s.symbols, s.eob, H, W, L, 1)
    for k in range(L):
        assert (np.abs(got[k] - want[k]) <= 1e-6 * sums[k] + 1e-30).all()
    lat_dev = [torch.from_numpy(g).to(DEV) for g in got]
    with pkg.Decoder(H, W, wl.widths, clamp=False) as dec:
        img = dec.run(lat_dev, torch.from_numpy(inp.weights).to(DEV), torch.from_numpy(inp.biases).to(DEV))
        torch.cuda.synchronize()
    ref = orc.decode(got, inp.weights, inp.biases, wl.widths, H, W, out="raw")
    assert np.abs(img.cpu().numpy() - ref).max() <= 1e-5 * max(1.0, np.abs(ref).max())


def test_many_chunks_long_stream(orc):
    # over 9000 chunks of 1024 symbols (every block 64 coefficient values and
    # its marker): the group-count prefix across many groups
    H, W, L, batch = 1024, 1024, 2, 7
    rng = np.random.default_rng(21)
    nb = batch * orc.zpr_blocks(H, W, L)
    co = pins_zpr.random_blocks(rng, nb, 1.0, 50)
    eob = 50 + 17
    stream = np.concatenate([co[:, pins_zpr.ZZ], np.full((nb, 1), eob)], axis=1).astype(np.int32).ravel()
    assert stream.size > 8192 * 1024
    _print_case("many chunks", stream.size)
    got, st = _gpu_expand(H, W, L, batch, stream, eob)
    assert st == 0 and np.array_equal(got, co)
    _check_decode(orc, H, W, L, batch, stream, eob)


def test_scan_path_very_long_stream(orc):
    # beyond 16384 chunks of 1024 symbols the one-workgroup scan kernel turns
    # the counts into prefixes first: 85M symbols, every block 64 values and
    # its marker, checked bit for bit in expand mode (the blocks are known)
    H, W, L, batch = 4096, 4096, 1, 5
    nb = batch * orc.zpr_blocks(H, W, L)
    rng = np.random.default_rng(23)
    co = rng.integers(1, 51, size=(nb, 64), dtype=np.int32)
    co *= np.where(rng.random((nb, 64)) < 0.5, -1, 1).astype(np.int32)
    eob = 50 + 17
    stream = np.empty((nb, 65), np.int32)
    stream[:, :64] = co[:, pins_zpr.ZZ]
    stream[:, 64] = eob
    stream = stream.ravel()
    assert stream.size > 16384 * 1024
    _print_case("scan path", stream.size)
    got, st = _gpu_expand(H, W, L, batch, stream, eob)
    assert st == 0 and np.array_equal(got, co)
    # and the count check still works on this path
    got, st = _gpu_expand(H, W, L, batch, stream[:-1], eob)
    assert st == D.PIC_ZPR_ERR_COUNT
