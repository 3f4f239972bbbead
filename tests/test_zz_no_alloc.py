"""The entry point that allocates nothing (pic_decode_run_noalloc), through
the C ABI, against pic_decode_run on a handle: the same kernels, so every
output value must be identical, on two calls in a row, the second with a
smaller input (the library's counter array keeps the first call's contents).
The first call of each case is also checked against the oracle."""
import numpy as np
import pytest

import oracle
from paper_2609_09020_amd import decoder as D
from paper_2609_09020_amd import synth

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    D.load_library()


def _dev(inp):
    lat = [torch.from_numpy(a).cuda() for a in inp.latents]
    if inp.weights_bf16 is not None:
        w = torch.from_numpy(inp.weights_bf16.view(np.int16)).cuda()
    else:
        w = torch.from_numpy(inp.weights).cuda()
    return lat, w, torch.from_numpy(inp.biases).cuda()


def _with_handle(inp, variant, wdt, max_batch):
    dec = D.Decoder(inp.height, inp.width, inp.widths, weight_dtype=wdt, clamp=False, max_batch=max_batch,
                    variant=variant)
    lat, w, b = _dev(inp)
    out = torch.full((inp.batch, 3, inp.height, inp.width), float("nan"), device="cuda")
    dec.run(lat, w, b, out=out)
    torch.cuda.synchronize()
    dec.close()
    return out.cpu().numpy()


def _noalloc(inp, variant, wdt, max_batch):
    desc = D.make_desc(inp.height, inp.width, inp.widths, weight_dtype=D.PIC_BF16 if wdt == "bf16" else D.PIC_F32,
                       flags=D.PIC_FLAG_NO_CLAMP,
                       max_batch=max_batch, variant=D.VARIANTS[variant])
    lat, w, b = _dev(inp)
    nw, nb = synth.param_counts(inp.widths)
    out = torch.full((inp.batch, 3, inp.height, inp.width), float("nan"), device="cuda")
    torch.cuda.synchronize()
    st = D.pic_decode_run_noalloc(desc, inp.batch, [t.data_ptr() for t in lat], w.data_ptr(), nw, b.data_ptr(),
                                  nb, out.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert st == D.PIC_OK, D.pic_status_string(st)
    torch.cuda.synchronize()
    return out.cpu().numpy()


# (variant, weights, first call (H, W, batch), second call (smaller)); one
# image at 1920x1080 has more tiles than workgroups (per-XCD counters run)
CASES = [
    ("mfma_f32", "f32", (1080, 1920, 1), (480, 640, 1)),
    ("mfma_f32", "f32", (300, 500, 5), (300, 500, 2)),
    ("mfma_bf16", "bf16", (1080, 1920, 1), (200, 330, 3)),
    ("mfma_f16x3", "f32", (300, 500, 5), (64, 64, 1)),
    ("valu", "f32", (300, 500, 3), (37, 53, 2)),
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-{c[2]}-{c[3]}" for c in CASES])
def test_noalloc_matches_handle_on_two_calls(case):
    variant, wdt, first, second = case
    max_batch = max(first[2], second[2])
    for call, (H, W, batch) in enumerate((first, second)):
        print(f"case: noalloc {variant} call {call} {H}x{W} x{batch}", flush=True)
        inp = synth.make_inputs(H, W, 7, (7, 40, 40, 3), batch=batch, seed=100 + call, latent="normal",
                                latent_scale=2.0, bias="normal", weight_dtype=wdt)
        got = _noalloc(inp, variant, wdt, max_batch)
        want = _with_handle(inp, variant, wdt, max_batch)
        assert np.isfinite(got).all(), "pixels left unwritten"
        n = int(np.count_nonzero(got != want))
        print(f"PARITY noalloc {variant} call {call}: {n} of {got.size} values differ from pic_decode_run",
              flush=True)
        assert n == 0
        if call == 0:
            ref = oracle.decode_inputs(inp, out="raw")
            err = float(np.max(np.abs(got - ref) / np.maximum(1.0, np.abs(ref))))
            print(f"PARITY noalloc {variant} call {call}: max err vs oracle {err:.3e}", flush=True)
            assert err <= (4e-3 if wdt == "bf16" else 1e-5)


def test_noalloc_rejects_before_enqueueing():
    # nothing here reaches the device: every status comes from the host checks
    desc = D.make_desc(64, 64, (4, 16, 16, 3), max_batch=5000)
    assert D.pic_decode_run_noalloc(desc, D.PIC_NOALLOC_MAX_BATCH + 1, [1, 2, 3, 4], 4, 0, 4, 0, 4) == \
        D.PIC_E_UNSUPPORTED
    assert D.pic_decode_run_noalloc(desc, 5001, [1, 2, 3, 4], 4, 0, 4, 0, 4) == D.PIC_E_INVALID
    bad = D.make_desc(64, 64, (4, 129, 3))
    assert D.pic_decode_run_noalloc(bad, 1, [1, 2, 3, 4], 4, 0, 4, 0, 4) == D.PIC_E_INVALID
    assert D.pic_decode_run_noalloc(desc, 0, [1, 2, 3, 4], 4, 0, 4, 0, 4) == D.PIC_OK
