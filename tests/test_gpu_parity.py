"""GPU parity: the HIP decode path (through the C ABI) against the CPU oracle.

Bars (the 8-bit band follows from the 1e-5 bar: an fp32 error within it can
move 255 c + 1/2 across an integer only from inside the band):
  * fp32 output clamped to [0, 1]: max |gpu - oracle_f64| <= 1e-5;
  * raw output (PIC_FLAG_NO_CLAMP): |gpu - oracle_f64| <= 1e-5 * max(1, |oracle|);
  * 8-bit output, reference (VALU) family: identical to the oracle's binary32
    model, which takes the same rounding decision in the same precision;
  * 8-bit output, matrix-core family: identical to the fp64 oracle wherever
    255 c + 1/2 lies more than 255e-5 from an integer, at most one code apart
    inside that band;
  * reference family raw output: equal, value for value, to the binary32
    model for any inputs (same operations in the same order).
Full-size workloads run on the GPU at full size in the launch configuration
the benchmark times, and every pixel of every image is compared with the
oracle (which runs on all host cores; one workload's oracle results are kept
while its families and output kinds are checked, then dropped).
"""
import numpy as np
import pytest

import oracle
from paper_2609_09020_amd import synth

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

TOL = 1e-5
U8_BAND = 255 * TOL
BF16_TOL = 4e-3


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_09020_amd as pkg
    pkg.load_library()


def _to_dev(inp, dev="cuda"):
    lat = [torch.from_numpy(a).to(dev) for a in inp.latents]
    if inp.weights_bf16 is not None:
        w = torch.from_numpy(inp.weights_bf16.view(np.int16)).to(dev)
    else:
        w = torch.from_numpy(inp.weights).to(dev)
    b = torch.from_numpy(inp.biases).to(dev)
    return lat, w, b


def gpu_decode(inp, variant="auto", out_dtype="f32", clamp=True, shared=False, stream=None):
    from paper_2609_09020_amd import Decoder
    wdt = "bf16" if inp.weights_bf16 is not None else "f32"
    dec = Decoder(inp.height, inp.width, inp.widths, weight_dtype=wdt, out_dtype=out_dtype,
                  clamp=clamp, max_batch=inp.batch, variant=variant)
    lat, w, b = _to_dev(inp)
    if shared:
        w, b = w[0].contiguous(), b[0].contiguous()
    out = dec.alloc_out(inp.batch, "cuda")
    if out.dtype == torch.float32:
        out.fill_(float("nan"))             # every pixel must be written
    torch.cuda.synchronize()                # (the run may be on another stream)
    dec.run(lat, w, b, out=out, stream=stream)
    torch.cuda.synchronize()
    info = dec.info()
    dec.close()
    got = out.cpu().numpy()
    if got.dtype == np.float32:
        assert np.isfinite(got).all(), "pixels left unwritten"
    return got, info


def _check_float(got, ref, raw, what):
    """Max error over the whole output, image by image (bounded temporaries)."""
    err = 0.0
    for b in range(got.shape[0]):
        g, r = got[b], ref[b]
        if raw:
            e = np.max(np.abs(g - r) / np.maximum(1.0, np.abs(r)))
        else:
            e = np.max(np.abs(g - r))
        err = max(err, float(e))
    print(f"PARITY {what}: max err {err:.3e} over {got.size} values", flush=True)
    assert err <= TOL, what


def _check_u8_band(got, ref_clamped, ref_u8, what):
    n_band = n_band_samples = 0
    for b in range(got.shape[0]):
        t = 255.0 * ref_clamped[b] + 0.5
        safe = np.abs(t - np.round(t)) > U8_BAND
        diff = got[b].astype(np.int32) - ref_u8[b].astype(np.int32)
        n_band += int(np.count_nonzero(diff[~safe]))
        n_band_samples += int(np.count_nonzero(~safe))
        assert np.array_equal(got[b][safe], ref_u8[b][safe]), f"{what} image {b}"
        assert np.all(np.abs(diff) <= 1), f"{what} image {b}"
    print(f"PARITY {what}: u8 codes differing inside the rounding band: {n_band} "
          f"of {n_band_samples} band samples; {got.size} codes", flush=True)


class _Workload:
    """The inputs and whole-output oracle results of one workload at a time."""
    name = None
    inp = None
    refs = {}

    @classmethod
    def get(cls, name):
        if cls.name != name:
            cls.name, cls.inp, cls.refs = None, None, {}
            cls.inp = synth.workload_inputs(synth.WORKLOADS[name])
            cls.name = name
        return cls.inp

    @classmethod
    def ref(cls, out, precision="f64"):
        key = (out, precision)
        if key not in cls.refs:
            cls.refs[key] = oracle.decode_inputs(cls.inp, out=out, precision=precision)
        return cls.refs[key]


FULL = ["pic64", "kodak768", "kodak768_b64", "clic2048", "clic2048_b16", "uhd4k", "kodak768_paper"]
F32_VARIANTS = ["valu", "mfma_f32", "mfma_f16x3"]
KINDS = ["clamped", "raw", "u8"]
# every (workload, kind, family), grouped by workload so its oracle results
# are computed once
WORKLOAD_CASES = [(n, k, v) for n in FULL for k in KINDS for v in F32_VARIANTS] + \
                 [("uhd4k_bf16", k, "mfma_bf16") for k in KINDS]


@pytest.mark.parametrize("case", WORKLOAD_CASES, ids=["-".join(c) for c in WORKLOAD_CASES])
def test_workload_whole_output(case):
    name, kind, variant = case
    inp = _Workload.get(name)
    print(f"case: {name} {kind} {variant}", flush=True)
    if kind == "u8":
        got, info = gpu_decode(inp, variant=variant, out_dtype="u8")
    else:
        got, info = gpu_decode(inp, variant=variant, clamp=(kind == "clamped"))
    assert info["variant"] == variant
    what = f"{name} {variant} {kind}"
    if variant == "mfma_bf16":
        # 4e-3 against the oracle fed the same bf16 weights
        if kind == "u8":
            # an error within 4e-3 of c moves the code by at most 2
            refc = _Workload.ref("clamped")
            n = 0
            for b in range(got.shape[0]):
                d = np.abs(got[b].astype(np.int32) - np.floor(255 * refc[b] + 0.5).astype(np.int32))
                n = max(n, int(d.max()))
            print(f"PARITY {what}: max code difference {n}", flush=True)
            assert n <= 2
            return
        ref = _Workload.ref(kind)
        err = 0.0
        for b in range(got.shape[0]):
            d = np.abs(got[b] - ref[b])
            if kind == "raw":
                d = d / np.maximum(1.0, np.abs(ref[b]))
            err = max(err, float(d.max()))
        print(f"PARITY {what}: max err {err:.3e} over {got.size} values", flush=True)
        assert err <= BF16_TOL
        return
    if kind == "u8":
        if variant == "valu":
            # the reference family takes the 8-bit decision in the oracle's
            # binary32 model's precision and order: every code equal
            ref = _Workload.ref("u8", "f32")
            n = int(np.count_nonzero(got != ref))
            print(f"PARITY {what}: {n} of {got.size} codes differ from the binary32 model", flush=True)
            assert n == 0
        else:
            _check_u8_band(got, _Workload.ref("clamped"), _Workload.ref("u8"), what)
        return
    _check_float(got, _Workload.ref(kind), kind == "raw", what)


# ------------------------------------------------------------------ fuzz

def _fuzz_cases(n, seed):
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        H = int(rng.integers(1, 71))
        W = int(rng.integers(1, 71))
        L = int(rng.integers(1, 9))
        nl = int(rng.integers(1, 5))
        hidden = [int(rng.integers(1, 65)) for _ in range(nl - 1)]
        widths = (L, *hidden, 3)
        batch = int(rng.integers(1, 4))
        cases.append((H, W, widths, batch, int(rng.integers(0, 2**31)), bool(rng.integers(0, 2))))
    return cases


EDGE_CASES = [
    (1, 1, (1, 3), 1, 1, False),
    (1, 1, (3, 5, 3), 2, 2, False),
    (3, 5, (2, 4, 3), 1, 3, True),
    (16, 15, (4, 16, 16, 3), 1, 4, False),
    (16, 16, (4, 16, 16, 3), 1, 5, False),
    (16, 17, (4, 16, 16, 3), 3, 6, False),
    (33, 47, (12, 64, 64, 3), 2, 7, False),      # largest level count and width
    (40, 64, (12, 17, 3), 1, 8, True),
    (9, 70, (8, 64, 64, 64, 3), 1, 9, False),    # two hidden layers at width 64
    (20, 30, (8, 16, 16, 16, 3), 2, 10, False),  # the paper's 4-layer width-16 shape
    (25, 31, (5, 1, 3), 1, 11, False),
    (7, 200, (6, 40, 3), 1, 12, False),
    # the last hidden layer wider than the earlier ones, in the K-step count
    # of 33..40-wide nets and beyond it
    (30, 70, (7, 40, 48, 3), 2, 13, False),
    (33, 65, (4, 8, 41, 3), 1, 14, False),
    (17, 90, (5, 40, 40, 44, 3), 1, 15, False),
    (21, 40, (7, 33, 47, 3), 1, 16, True),
    # hidden widths past the matrix-core families (four 16-neuron blocks):
    # the reference family decodes them, the others report them unsupported
    (19, 37, (7, 65, 3), 1, 17, False),
    (23, 29, (8, 96, 96, 3), 2, 18, False),
    (13, 70, (12, 128, 128, 3), 1, 19, False),
    (9, 33, (3, 128, 20, 128, 3), 1, 20, True),
]


def _run_case(case, variant):
    H, W, widths, batch, seed, shared = case
    from paper_2609_09020_amd import decoder as D
    inp = synth.make_inputs(H, W, widths[0], widths, batch=batch, seed=seed, latent="normal",
                            latent_scale=1.5, bias="normal", shared_weights=shared)
    nl = len(widths) - 1
    if variant in ("mfma_f32", "mfma_f16x3") and not (2 <= nl <= 4 and max(widths[1:-1]) <= 64):
        with pytest.raises(D.PicError) as e:
            gpu_decode(inp, variant=variant)
        assert e.value.status == D.PIC_E_UNSUPPORTED
        return None
    got, _ = gpu_decode(inp, variant=variant, clamp=False, shared=shared)
    ref = oracle.decode_inputs(inp, out="raw")
    _check_float(got, ref, True, f"fuzz {case} {variant}")
    return inp, got


@pytest.mark.parametrize("variant", F32_VARIANTS)
@pytest.mark.parametrize("case", EDGE_CASES + _fuzz_cases(24, 2024), ids=str)
def test_fuzz_raw(case, variant):
    _run_case(case, variant)


# The longest image sides the descriptor accepts, 2^23 - 1 (pixel centres
# and source coordinates exact in fp32, a texel's index in one 24-bit
# multiply), one pixel across: a single row of 2^17 tiles, where tiles x tiles
# across >= 2^32 so the tile row comes from the division rather than the
# multiply-high, and a single column of 2^20 tiles.
_LONG_REF = {}


@pytest.mark.parametrize("variant", F32_VARIANTS)
@pytest.mark.parametrize("hw", [(1, (1 << 23) - 1), ((1 << 23) - 1, 1)], ids=["row", "column"])
def test_longest_sides(hw, variant):
    H, W = hw
    widths = (4, 16, 16, 3)
    inp = synth.make_inputs(H, W, widths[0], widths, batch=1, seed=41, latent="normal", latent_scale=1.5,
                            bias="normal")
    got, _ = gpu_decode(inp, variant=variant, clamp=False)
    if hw not in _LONG_REF:
        _LONG_REF[hw] = oracle.decode_inputs(inp, out="raw")
    _check_float(got, _LONG_REF[hw], True, f"sides {H}x{W} {variant}")


@pytest.mark.parametrize("hw", [(1, (1 << 23) - 1), ((1 << 23) - 1, 1)], ids=["row", "column"])
def test_longest_sides_bf16(hw):
    """The bf16-weight matrix family at the longest sides the boundary takes
    (its tile rows then come from the division, not the multiply-high), the
    whole output against the fp64 oracle on the same bf16 weights."""
    H, W = hw
    widths = (4, 16, 16, 3)
    inp = synth.make_inputs(H, W, widths[0], widths, batch=1, seed=43, latent="normal", latent_scale=1.5,
                            bias="normal", weight_dtype="bf16")
    got, info = gpu_decode(inp, variant="mfma_bf16", clamp=False)
    assert info["variant"] == "mfma_bf16"
    ref = oracle.decode_inputs(inp, out="raw")
    err = np.max(np.abs(got - ref) / np.maximum(1.0, np.abs(ref)))
    print(f"PARITY bf16 sides {H}x{W}: max err {err:.3e}", flush=True)
    assert err <= BF16_TOL


@pytest.mark.parametrize("case", EDGE_CASES + _fuzz_cases(12, 77), ids=str)
def test_reference_family_matches_binary32_model(case):
    r = _run_case(case, "valu")
    inp, got = r
    ref32 = oracle.decode_inputs(inp, out="raw", precision="f32")
    n = int(np.count_nonzero(got != ref32))
    assert n == 0, f"{n} values differ from the binary32 model"


# Batches large enough for the fp32 matrix-core family's 16-row tiles (it
# takes them when every workgroup averages two or more: with 64 images,
# 16 workgroups per image at 4 per CU, and an image of 200 x 300 has
# 5 x 13 = 65 such tiles), at sizes ragged against both tile dimensions
# (200 = 12 x 16 + 8 rows, 300 = 4 x 64 + 44 columns), raw outputs.
@pytest.mark.parametrize("case", [(200, 300, (7, 40, 40, 3), 64, 31, False),
                                  (200, 300, (4, 16, 16, 3), 64, 32, True),
                                  (136, 330, (8, 48, 48, 3), 64, 33, False)], ids=str)
def test_tall_tiles_ragged_batch(case):
    _run_case(case, "mfma_f32")


# The bf16 family's 16-row tiles (same rule), ragged likewise.
@pytest.mark.parametrize("case", [(200, 300, (8, 64, 64, 3), 64, 34, False),
                                  (136, 330, (7, 40, 40, 3), 64, 35, True)], ids=str)
def test_tall_tiles_ragged_batch_bf16(case):
    test_fuzz_bf16_weights(case, "mfma_bf16")


def test_shared_weights_stride_zero_matches_repeated():
    inp = synth.make_inputs(37, 53, 6, (6, 24, 24, 3), batch=3, seed=5, latent="normal",
                            bias="normal", shared_weights=True)
    for variant in F32_VARIANTS:
        a, _ = gpu_decode(inp, variant=variant, clamp=False, shared=True)
        b, _ = gpu_decode(inp, variant=variant, clamp=False, shared=False)
        assert np.array_equal(a, b)


@pytest.mark.parametrize("variant", ["mfma_f32", "mfma_f16x3"])
def test_handle_reuse_with_changing_batch(variant):
    # the matrix-core kernels take tiles from per-image counters that each
    # run clears for the next one: runs of different batch sizes on one
    # handle must each decode exactly what a fresh handle decodes
    from paper_2609_09020_amd import Decoder
    inp = synth.make_inputs(70, 150, 7, (7, 40, 40, 3), batch=5, seed=31, latent="normal", latent_scale=2.0,
                            bias="normal")
    lat, w, b = _to_dev(inp)
    want, _ = gpu_decode(inp, variant=variant, clamp=False)
    dec = Decoder(inp.height, inp.width, inp.widths, clamp=False, max_batch=5, variant=variant)
    for n in (5, 2, 5, 1, 3, 5, 4):
        out = dec.run([t[:n] for t in lat], w[:n], b[:n])
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        print(f"PARITY handle reuse {variant} batch {n}", flush=True)
        assert np.array_equal(got, want[:n]), n
    dec.close()


@pytest.mark.parametrize("variant", ["mfma_f32", "mfma_f16x3", "mfma_bf16"])
def test_one_image_tile_ranges_per_xcd(variant):
    # a one-image grid takes each XCD's tiles from a contiguous range and a
    # counter of its own; 1920x1080 has 4050 tiles (not a multiple of 8) and
    # more tiles than workgroups, so the ranges are uneven and the counters
    # run.  Every pixel must be written (the output starts as NaN) and match
    # the oracle, on two runs of one handle.
    from paper_2609_09020_amd import Decoder
    H, W = 1080, 1920
    wdt = "bf16" if variant == "mfma_bf16" else "f32"
    inp = synth.make_inputs(H, W, 7, (7, 40, 40, 3), seed=5, bias="normal", weight_dtype=wdt)
    lat, w, b = _to_dev(inp)
    dec = Decoder(H, W, inp.widths, weight_dtype=wdt, clamp=False, max_batch=1, variant=variant)
    ref = oracle.decode_inputs(inp, out="raw")
    for run in range(2):
        out = torch.full((1, 3, H, W), float("nan"), device="cuda")
        dec.run(lat, w, b, out=out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        print(f"PARITY xcd ranges {variant} run {run}: unwritten {int(np.count_nonzero(~np.isfinite(got)))}",
              flush=True)
        assert np.isfinite(got).all()
        if wdt == "bf16":
            err = np.max(np.abs(got - ref) / np.maximum(1.0, np.abs(ref)))
            print(f"PARITY xcd ranges {variant} run {run}: max err {err:.3e}", flush=True)
            assert err <= BF16_TOL
        else:
            _check_float(got, ref, True, f"xcd ranges {variant} run {run}")
    dec.close()


def test_batch_zero_enqueues_nothing():
    from paper_2609_09020_amd import Decoder
    inp = synth.make_inputs(8, 8, 2, (2, 4, 3), batch=1, seed=0)
    lat, w, b = _to_dev(inp)
    dec = Decoder(8, 8, (2, 4, 3), max_batch=1)
    out = torch.full((1, 3, 8, 8), 7.0, device="cuda")
    dec.run(lat, w, b, out=out, batch=0)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)


def test_runs_on_caller_stream():
    inp = synth.workload_inputs(synth.WORKLOADS["kodak768"])
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        got, _ = gpu_decode(inp, variant="mfma_f32", stream=s.cuda_stream)
    ref, _ = gpu_decode(inp, variant="mfma_f32")
    assert np.array_equal(got, ref)


def test_two_handles_on_two_streams():
    """Two handles decoding batches at the same time on two streams (each
    batch takes tiles from its handle's counters), eight calls each with no
    synchronisation between them: every output equals a run on its own."""
    from paper_2609_09020_amd import Decoder
    inps = [synth.make_inputs(256, 384, 7, (7, 40, 40, 3), batch=8, seed=s, latent_scale=2.0, bias="normal")
            for s in (41, 42)]
    decs = [Decoder(256, 384, (7, 40, 40, 3), clamp=False, max_batch=8, variant="mfma_f32") for _ in range(2)]
    devin = [_to_dev(inp) for inp in inps]
    want = []
    for j in range(2):
        o = decs[j].alloc_out(8, "cuda")
        decs[j].run(*devin[j], out=o)
        torch.cuda.synchronize()
        want.append(o.cpu().numpy())
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [[decs[j].alloc_out(8, "cuda") for _ in range(8)] for j in range(2)]
    torch.cuda.synchronize()
    for k in range(8):
        for j in range(2):
            with torch.cuda.stream(streams[j]):
                decs[j].run(*devin[j], out=outs[j][k], stream=streams[j].cuda_stream)
    torch.cuda.synchronize()
    for j in range(2):
        for k in range(8):
            assert np.array_equal(outs[j][k].cpu().numpy(), want[j]), (j, k)
        decs[j].close()


def test_create_does_not_wait_for_other_streams():
    """Creating a decode or an entropy-decoding handle clears its device
    memory on a private stream and waits for that alone: about 50 ms of
    decodes queued on another stream are still running when both creates
    return (an event recorded after them has not completed)."""
    from paper_2609_09020_amd import Decoder, HuffDecoder
    inp = synth.workload_inputs(synth.WORKLOADS["uhd4k"])
    lat, w, b = _to_dev(inp)
    dec = Decoder(inp.height, inp.width, inp.widths, max_batch=1, variant="mfma_f32")
    out = dec.alloc_out(1, "cuda")
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    done = torch.cuda.Event()
    with torch.cuda.stream(s):
        for _ in range(80):                  # 0.6 ms each
            dec.run(lat, w, b, out=out, stream=s.cuda_stream)
        done.record(s)
    d2 = Decoder(512, 768, (7, 40, 40, 3), max_batch=4)
    h2 = HuffDecoder(1 << 20)
    pending = not done.query()
    torch.cuda.synchronize()
    d2.close()
    h2.close()
    dec.close()
    assert pending, "a handle's creation waited for work queued on another stream"


def test_run_rejects_bad_arguments_before_launch():
    from paper_2609_09020_amd import decoder as D
    inp = synth.make_inputs(8, 8, 2, (2, 4, 3), batch=2, seed=0)
    lat, w, b = _to_dev(inp)
    dec = D.Decoder(8, 8, (2, 4, 3), max_batch=2)
    out = dec.alloc_out(2, "cuda")
    ptrs = [t.data_ptr() for t in lat]
    h = dec.handle
    run = D.pic_decode_run
    assert run(h, 3, ptrs, w.data_ptr(), 20, b.data_ptr(), 7, out.data_ptr()) == D.PIC_E_INVALID
    assert run(h, -1, ptrs, w.data_ptr(), 20, b.data_ptr(), 7, out.data_ptr()) == D.PIC_E_INVALID
    assert run(h, 2, ptrs, 0, 20, b.data_ptr(), 7, out.data_ptr()) == D.PIC_E_INVALID
    assert run(h, 2, ptrs, w.data_ptr(), 19, b.data_ptr(), 7, out.data_ptr()) == D.PIC_E_INVALID
    assert run(h, 2, ptrs, w.data_ptr(), 20, b.data_ptr(), -1, out.data_ptr()) == D.PIC_E_INVALID
    assert run(h, 2, ptrs, w.data_ptr() + 2, 20, b.data_ptr(), 7, out.data_ptr()) == D.PIC_E_INVALID
    assert run(h, 2, [ptrs[0], 0], w.data_ptr(), 20, b.data_ptr(), 7, out.data_ptr()) == D.PIC_E_INVALID
    assert run(h, 2, ptrs, w.data_ptr(), 20, b.data_ptr(), 7, out.data_ptr()) == D.PIC_OK
    torch.cuda.synchronize()
    dec.close()


# ------------------------------------------------------- bf16-weight family


@pytest.mark.parametrize("variant", ["mfma_bf16", "mfma_f32", "valu"])
@pytest.mark.parametrize("case", EDGE_CASES + _fuzz_cases(16, 4242), ids=str)
def test_fuzz_bf16_weights(case, variant):
    H, W, widths, batch, seed, shared = case
    from paper_2609_09020_amd import decoder as D
    inp = synth.make_inputs(H, W, widths[0], widths, batch=batch, seed=seed, latent="normal",
                            latent_scale=1.5, bias="normal", shared_weights=shared, weight_dtype="bf16")
    nl = len(widths) - 1
    if variant != "valu" and not (2 <= nl <= 4 and max(widths[1:-1]) <= 64):
        with pytest.raises(D.PicError) as e:
            gpu_decode(inp, variant=variant)
        assert e.value.status == D.PIC_E_UNSUPPORTED
        return
    got, _ = gpu_decode(inp, variant=variant, clamp=False, shared=shared)
    ref = oracle.decode_inputs(inp, out="raw")     # fp64 with the same bf16 weights
    err = np.max(np.abs(got - ref) / np.maximum(1.0, np.abs(ref)))
    tol = BF16_TOL if variant == "mfma_bf16" else TOL
    print(f"PARITY bf16-weights {case} {variant}: max err {err:.3e}", flush=True)
    assert err <= tol


def test_bf16_family_u8_band():
    inp = synth.make_inputs(300, 500, 8, (8, 64, 64, 3), batch=2, seed=3, weight_dtype="bf16",
                            latent_scale=3.0, latent_clip=64)
    got, _ = gpu_decode(inp, variant="mfma_bf16", out_dtype="u8")
    refc = oracle.decode_inputs(inp, out="clamped")
    # a 4e-3 bar on c puts the 8-bit code within one step of the oracle's
    diff = np.abs(got.astype(np.int32) - np.floor(255 * refc + 0.5).astype(np.int32))
    assert diff.max() <= 2


# ------------------------------------------------- AUTO on narrow fp32 nets

@pytest.mark.parametrize("widths,want", [
    ((8, 8, 8, 8, 3), "valu"), ((4, 8, 3), "valu"), ((7, 5, 8, 3), "valu"),
    ((8, 9, 3), "mfma_f32"), ((8, 8, 16, 3), "mfma_f32"), ((8, 16, 16, 16, 3), "mfma_f32")])
def test_auto_family_for_narrow_nets(widths, want):
    """AUTO runs fp32 nets whose hidden layers are all at most 8 wide on the
    vector family (the matrix family pads them to 16-neuron blocks), wider
    ones on the fp32 matrix family; the result matches the oracle either
    way (200x300, ragged against the tiles)."""
    inp = synth.make_inputs(200, 300, widths[0], widths, batch=2, seed=31, latent_scale=1.5, bias="normal")
    got, info = gpu_decode(inp, clamp=False)
    assert info["variant"] == want
    ref = oracle.decode_inputs(inp, out="raw")
    err = np.max(np.abs(got - ref) / np.maximum(1.0, np.abs(ref)))
    print(f"PARITY auto {widths} -> {want}: max err {err:.3e}", flush=True)
    assert err <= TOL


# ------------------------------------------ per-layer parameters, App. A fusion

def test_run_layers_shared_and_per_image():
    """The paper's split: the first layers shared by the batch (stride 0), the
    last layer per image, through pic_decode_run_layers."""
    from paper_2609_09020_amd import Decoder, synth as sy
    for variant, wdt in (("mfma_f32", "f32"), ("valu", "f32"), ("mfma_bf16", "bf16")):
        widths = (8, 16, 16, 16, 3)
        batch = 3
        inp = sy.make_inputs(48, 80, 8, widths, batch=batch, seed=21, latent="normal", latent_scale=2.0,
                             bias="normal", weight_dtype=wdt)
        nl = len(widths) - 1
        sizes = [widths[l] * widths[l + 1] for l in range(nl)]
        offs = np.cumsum([0] + sizes)
        boffs = np.cumsum([0] + list(widths[1:]))
        src_w = inp.weights_bf16 if wdt == "bf16" else inp.weights
        # shared layers take image 0's parameters; the reference repeats them
        ref_w = src_w.copy()
        ref_b = inp.biases.copy()
        for l in range(nl - 1):
            ref_w[:, offs[l]:offs[l + 1]] = src_w[0, offs[l]:offs[l + 1]]
            ref_b[:, boffs[l]:boffs[l + 1]] = inp.biases[0, boffs[l]:boffs[l + 1]]
        dev = "cuda"
        lat = [torch.from_numpy(a).to(dev) for a in inp.latents]
        lw, lb = [], []
        for l in range(nl):
            blk = src_w[:, offs[l]:offs[l + 1]].reshape(batch, widths[l + 1], widths[l])
            bb = inp.biases[:, boffs[l]:boffs[l + 1]]
            if l < nl - 1:
                blk, bb = blk[0], bb[0]
            if wdt == "bf16":
                lw.append(torch.from_numpy(np.ascontiguousarray(blk).view(np.int16)).to(dev))
            else:
                lw.append(torch.from_numpy(np.ascontiguousarray(blk)).to(dev))
            lb.append(torch.from_numpy(np.ascontiguousarray(bb)).to(dev))
        dec = Decoder(48, 80, widths, weight_dtype=wdt, clamp=False, max_batch=batch, variant=variant)
        got = dec.run_layers(lat, lw, lb)
        torch.cuda.synchronize()
        dec.close()
        if wdt == "bf16":
            ref = oracle.decode(inp.latents, None, ref_b, widths, 48, 80, out="raw", weights_bf16=ref_w)
        else:
            ref = oracle.decode(inp.latents, ref_w, ref_b, widths, 48, 80, out="raw")
        err = np.max(np.abs(got.cpu().numpy() - ref) / np.maximum(1.0, np.abs(ref)))
        print(f"PARITY run_layers {variant}: max err {err:.3e}", flush=True)
        assert err <= (BF16_TOL if wdt == "bf16" else TOL)


def test_fuse_modulation_matches_oracle():
    from paper_2609_09020_amd import fuse_modulation
    rng = np.random.default_rng(31)
    for fin, fout, batch, shared in ((16, 3, 4, False), (40, 40, 2, True), (64, 64, 3, False), (1, 5, 1, False)):
        W = rng.normal(0, 0.5, size=(batch, fout, fin)).astype(np.float32)
        b = rng.normal(0, 0.5, size=(batch, fout)).astype(np.float32)
        g, be, mu = (rng.normal(m, s, size=(batch, fin)).astype(np.float32) for m, s in ((1, .5), (0, .5), (0, 2)))
        sg = (np.abs(rng.normal(1, .5, size=(batch, fin))) + 0.1).astype(np.float32)
        T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
        if shared:
            wf, bf = fuse_modulation(T(W[0]), T(b[0]), T(g), T(be), T(mu), T(sg))
        else:
            wf, bf = fuse_modulation(T(W), T(b), T(g), T(be), T(mu), T(sg))
        torch.cuda.synchronize()
        wf, bf = wf.cpu().numpy(), bf.cpu().numpy()
        for i in range(batch):
            src = 0 if shared else i
            rw, rb = oracle.fuse_modulation(W[src], b[src], g[i], be[i], mu[i], sg[i])
            # one rounding of the fp64 value to fp32
            assert np.max(np.abs(wf[i] - rw) / np.maximum(np.abs(rw), 1e-30)) <= 2 ** -24
            scale = np.abs(b[src]) + np.abs(W[src]).astype(np.float64) @ (np.abs(be[i]) + np.abs(g[i] * mu[i] / sg[i]))
            assert np.all(np.abs(bf[i] - rb) <= 2 ** -23 * scale + 1e-30)


def test_fused_network_decodes_like_modulated_network():
    """End to end (App. A): decoding with the fused last layer equals the oracle
    decode whose last layer is the oracle's fusion of the same statistics."""
    from paper_2609_09020_amd import Decoder, fuse_modulation
    rng = np.random.default_rng(41)
    widths = (7, 40, 40, 3)
    H, W_, batch = 64, 96, 2
    inp = synth.make_inputs(H, W_, 7, widths, batch=batch, seed=9, latent="normal", latent_scale=2.0,
                            bias="normal")
    nl = 3
    offs = np.cumsum([0] + [widths[l] * widths[l + 1] for l in range(nl)])
    boffs = np.cumsum([0] + list(widths[1:]))
    W3 = inp.weights[:, offs[2]:offs[3]].reshape(batch, 3, 40)
    b3 = inp.biases[:, boffs[2]:boffs[3]]
    g = rng.normal(1, .3, size=(batch, 40)).astype(np.float32)
    be = rng.normal(0, .3, size=(batch, 40)).astype(np.float32)
    mu = rng.normal(1, .5, size=(batch, 40)).astype(np.float32)
    sg = (np.abs(rng.normal(1, .3, size=(batch, 40))) + 0.2).astype(np.float32)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    wf, bf = fuse_modulation(T(W3), T(b3), T(g), T(be), T(mu), T(sg))
    ref_w = inp.weights.copy()
    ref_b = inp.biases.copy()
    for i in range(batch):
        rw, rb = oracle.fuse_modulation(W3[i], b3[i], g[i], be[i], mu[i], sg[i])
        ref_w[i, offs[2]:offs[3]] = rw.astype(np.float32).ravel()
        ref_b[i, boffs[2]:boffs[3]] = rb.astype(np.float32)
    lat = [torch.from_numpy(a).cuda() for a in inp.latents]
    lw = [T(inp.weights[:, offs[l]:offs[l + 1]].reshape(batch, widths[l + 1], widths[l])) for l in range(2)] + [wf]
    lb = [T(inp.biases[:, boffs[l]:boffs[l + 1]]) for l in range(2)] + [bf]
    dec = Decoder(H, W_, widths, clamp=False, max_batch=batch, variant="mfma_f32")
    got = dec.run_layers(lat, lw, lb)
    torch.cuda.synchronize()
    dec.close()
    ref = oracle.decode(inp.latents, ref_w, ref_b, widths, H, W_, out="raw")
    err = np.max(np.abs(got.cpu().numpy() - ref) / np.maximum(1.0, np.abs(ref)))
    print(f"PARITY fused network: max err {err:.3e}", flush=True)
    assert err <= TOL


def test_run_layers_and_fuse_reject_bad_arguments():
    from paper_2609_09020_amd import decoder as D
    dec = D.Decoder(8, 8, (2, 4, 3), max_batch=2)
    lat = [torch.zeros((2, 8, 8), device="cuda"), torch.zeros((2, 4, 4), device="cuda")]
    w0 = torch.zeros((2, 4, 2), device="cuda")
    w1 = torch.zeros((2, 3, 4), device="cuda")
    b0 = torch.zeros((2, 4), device="cuda")
    b1 = torch.zeros((2, 3), device="cuda")
    out = dec.alloc_out(2, "cuda")
    run = D.pic_decode_run_layers
    lp = [t.data_ptr() for t in lat]
    good = dict(lw=[w0.data_ptr(), w1.data_ptr()], ws=[8, 12], lb=[b0.data_ptr(), b1.data_ptr()], bs=[4, 3])
    assert run(dec.handle, 2, lp, good["lw"], good["ws"], good["lb"], good["bs"], out.data_ptr()) == D.PIC_OK
    assert run(dec.handle, 2, lp, good["lw"], [7, 12], good["lb"], good["bs"], out.data_ptr()) == D.PIC_E_INVALID
    assert run(dec.handle, 2, lp, good["lw"], good["ws"], good["lb"], [4, -1], out.data_ptr()) == D.PIC_E_INVALID
    assert run(dec.handle, 2, lp, [w0.data_ptr(), 0], good["ws"], good["lb"], good["bs"], out.data_ptr()) == D.PIC_E_INVALID
    assert run(dec.handle, 3, lp, good["lw"], good["ws"], good["lb"], good["bs"], out.data_ptr()) == D.PIC_E_INVALID
    f = D.pic_fuse_modulation
    p = w0.data_ptr()
    assert f(0, 4, 1, p, 0, p, 0, p, p, p, p, 0, p, p) == D.PIC_E_INVALID
    assert f(4, 129, 1, p, 0, p, 0, p, p, p, p, 0, p, p) == D.PIC_E_INVALID
    assert f(4, 4, 1, p, 3, p, 0, p, p, p, p, 0, p, p) == D.PIC_E_INVALID
    assert f(4, 4, 1, p, 0, p, 0, p, p, p, 0, 0, p, p) == D.PIC_E_INVALID
    torch.cuda.synchronize()
    dec.close()
