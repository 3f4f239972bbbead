#!/usr/bin/env python3
"""Benchmark of the PIC synthesis decoder on one MI355X.

A step is one pic_decode_run call: the whole synthesis path (upsample of every
latent level + the per-pixel MLP + epilogue) over one batch of synthetic,
device-resident inputs.  W untimed warm-up steps, then exactly K timed steps
bracketed by torch.cuda.synchronize(); the average device time per launch is
measured live with two HIP events recorded, around the timed steps, on the
stream the kernel is launched on.

Prints ONE JSON line: decoded Mpixel/s (value), FPS, ms per step, the
roofline of the dominant kernel and the CPU oracle's throughput on a bounded
sample of the same workload (rank 0, N = 1 only).

The same line carries `per_config`: every other workload of the benchmark
suite (64x64; 768x512 x64; 2048x1536 x1 and x16; 3840x2160 with fp32 and
with bf16 weights; the paper's 4-layer net at 768x512; 768x512 and 3840x2160
again in the fp16-split matrix-core family), each timed with HIP events over
back-to-back launches, with its roofline fraction.  They run after the
headline's inputs are resident and before its warm-up and timed calls, so
that those follow real work on the GPU rather than seconds of host-side
input generation; and `paper_context`: the paper's own decoding speed with
the hardware it was measured on (context, not the target).

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload kodak768]
                  [--variant auto|valu|mfma_f32|mfma_bf16|mfma_f16x3]
                  [--out-dtype f32|u8] [--no-cpu-baseline] [--no-per-config]
                  [--copy-calib]
  python bench.py --peaks        peak issue rates of the matrix and vector
                                 units and the device-copy bandwidth
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decoded Mpixel/s (and FPS at 768x512) on 1 MI355X; % of roofline"
# MI355X published peaks.
PEAK_FP32_TFLOPS = 157.3        # fp32 vector (packed) and fp32 matrix
PEAK_BF16_TFLOPS = 2500.0       # dense bf16 matrix
PEAK_FP16_TFLOPS = 2500.0       # dense fp16 matrix
PEAK_HBM_GBS = 8000.0
CLOCK_HZ = 2.4e9                # peak engine clock


def flops_per_pixel(widths):
    """Algorithmic work per pixel: 2 * sum(in * out) for the MLP (bias folded
    into the accumulator start) + 8 * (L - 1) for the bilinear upsample of the
    L - 1 coarser levels (3 lerps of a multiply and an add, plus weights)."""
    L = widths[0]
    return 2 * sum(widths[i] * widths[i + 1] for i in range(len(widths) - 1)) + 8 * (L - 1)


def bytes_per_call(wl, out_dtype):
    """Compulsory HBM bytes: every latent read once, every output written once,
    every image's parameters read once."""
    from paper_2609_09020_amd import synth
    lat = sum(h * w for h, w in (synth.level_shape(wl.height, wl.width, k) for k in range(wl.levels)))
    nw, nb = synth.param_counts(wl.widths)
    wbytes = 2 if wl.weight_dtype == "bf16" else 4
    out_b = 1 if out_dtype == "u8" else 4
    return wl.batch * (4 * lat + 3 * out_b * wl.height * wl.width + wbytes * nw + 4 * nb)


def load_traffic(kernel, workload, out_dtype):
    """Measured HBM traffic per launch from the committed counter summary, if
    it was taken on the current kernel source (else None)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_{out_dtype}_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    h = hashlib.sha256()
    for name in kv.get("source", "").split():
        src = os.path.join(ROOT, "paper_2609_09020_amd", "csrc", name)
        if not os.path.exists(src):
            return None
        h.update(open(src, "rb").read())
    sha = h.hexdigest()[:16]
    if sha != kv.get("source_sha256_16"):
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(wl, inp, target_s=12.0):
    """The fp64 oracle, as it stands, on the host cores: whole images of the
    workload, repeated until about target_s seconds of CPU work."""
    import oracle
    threads = len(os.sched_getaffinity(0))
    orc = oracle.default()
    n_img = 0
    t0 = time.perf_counter()
    while True:
        b = n_img % inp.batch
        orc.decode_inputs(inp, out="clamped", batch_slice=slice(b, b + 1), nthreads=threads)
        n_img += 1
        if time.perf_counter() - t0 >= target_s:
            break
    dt = time.perf_counter() - t0
    px = n_img * wl.height * wl.width
    # the same on one core, for a shorter while
    n1 = 0
    t1 = time.perf_counter()
    while True:
        orc.decode_inputs(inp, out="clamped", batch_slice=slice(n1 % inp.batch, n1 % inp.batch + 1), nthreads=1)
        n1 += 1
        if time.perf_counter() - t1 >= target_s / 3:
            break
    dt1 = time.perf_counter() - t1
    return {"value": round(px / dt / 1e6, 3), "unit": "Mpixel/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{n_img} whole {wl.width}x{wl.height} image decode(s) of this workload by the "
                      f"fp64 C oracle (OpenMP over rows), {dt:.1f} s",
            "value_1core": round(n1 * wl.height * wl.width / dt1 / 1e6, 3),
            "sample_1core": f"{n1} image decode(s) on one thread, {dt1:.1f} s",
            "cpu_model": cpu_model()}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def time_calls(run, K, W, stream):
    """Average device time per call over K back-to-back calls (HIP events on
    the launch stream) and the wall time of the K calls."""
    import torch
    for _ in range(W):
        run()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(K):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / K, time.perf_counter() - t0


def variant_peak(variant):
    """(bound, peak, unit) of the dominant instructions of a kernel family."""
    if variant == "mfma_bf16":
        return "mfma", PEAK_BF16_TFLOPS, "TFLOP/s"
    if variant == "mfma_f32":
        return "mfma", PEAK_FP32_TFLOPS, "TFLOP/s"
    if variant == "mfma_f16x3":
        # fp32 arithmetic carried out on the fp16 matrix cores: against the
        # peak of the instructions it runs on (its fp32-equivalent rate beside)
        return "mfma", PEAK_FP16_TFLOPS, "TFLOP/s"
    return "alu", PEAK_FP32_TFLOPS, "TFLOP/s"


# The paper's own decoding speed (Table 1; Sec. 4.1): the whole decoder,
# entropy decoding included, per Kodak image, serially, on its GPU.
PAPER_CONTEXT = {
    "fps": 2392, "ms_per_image": 0.418, "mpixel_s": round(768 * 512 / 0.418e-3 / 1e6, 1),
    "hardware": "1x NVIDIA RTX 4090D", "precision": "TF32 tensor cores",
    "workload": "Kodak (24 images of 768x512), whole decoder (entropy decoding, latent decoding, "
                "synthesis), L = 8 levels, g_s 4 layers of width 16, images decoded one at a time",
    "source": "Table 1 (decode time), Sec. 4.1",
    "note": "context only: another machine and the whole decoder; `bench.py --full` times the "
            "whole decoder here",
}

# Workloads of the benchmark suite timed beside the headline one (per_config).
PER_CONFIG = ["pic64", "kodak768_b64", "clic2048", "clic2048_b16", "uhd4k", "uhd4k_bf16", "kodak768_paper"]
# fp32-weight workloads also timed in the fp16-split matrix-core family (fp32
# accuracy from fp16 matrix instructions): key "<workload>@mfma_f16x3"
PER_CONFIG_F16X3 = ["kodak768", "uhd4k"]


def time_workload(name, variant="auto", out_dtype="f32", target_s=0.3):
    """Kernel time of one workload: HIP events on the launch stream around
    back-to-back pic_decode_run calls (about target_s seconds of them)."""
    import ctypes
    import numpy as np
    import torch
    from paper_2609_09020_amd import synth
    from paper_2609_09020_amd import decoder as D
    wl = synth.WORKLOADS[name]
    inp = synth.workload_inputs(wl)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    lat = [torch.from_numpy(a).to(dev) for a in inp.latents]
    w = torch.from_numpy(inp.weights_bf16.view(np.int16) if inp.weights_bf16 is not None else inp.weights).to(dev)
    b = torch.from_numpy(inp.biases).to(dev)
    dec = D.Decoder(wl.height, wl.width, wl.widths, weight_dtype=wl.weight_dtype, out_dtype=out_dtype,
                    max_batch=wl.batch, variant=variant)
    out = dec.alloc_out(wl.batch, dev)
    lib = D.load_library()
    lat_arr = (ctypes.c_void_p * len(lat))(*[t.data_ptr() for t in lat])
    run_args = (ctypes.c_void_p(dec.handle), ctypes.c_int32(wl.batch), lat_arr, ctypes.c_void_p(w.data_ptr()),
                ctypes.c_int64(dec.nw), ctypes.c_void_p(b.data_ptr()), ctypes.c_int64(dec.nb),
                ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(stream.cuda_stream))

    def launches(n):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(n):
            st = lib.pic_decode_run(*run_args)
            if st != D.PIC_OK:
                raise D.PicError(st, "pic_decode_run")
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    launches(10)                                   # warm-up
    est = launches(5)
    n = int(min(4000, max(20, target_s * 1e3 / max(est, 1e-4))))
    ms = launches(n)
    info = dec.info()
    dec.close()
    px = wl.batch * wl.height * wl.width
    fpp = flops_per_pixel(wl.widths)
    bound, peak, unit = variant_peak(info["variant"])
    achieved = px * fpp / (ms * 1e-3) / 1e12
    return {"workload": f"{wl.name}: {wl.note}", "widths": list(wl.widths), "batch": wl.batch,
            "weights": wl.weight_dtype, "variant": info["variant"], "kernel": info["kernel_name"],
            "launches": n, "kernel_avg_ms": round(ms, 5), "mpixel_s": round(px / ms / 1e3, 1),
            "fps": round(wl.batch / ms * 1e3, 1),
            "roofline": {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
                         "frac": round(achieved / peak, 4),
                         "fp32_equivalent_frac": round(achieved / PEAK_FP32_TFLOPS, 4),
                         "flop_per_pixel": fpp}}


def peaks(args):
    """Peak issue rates on this GPU (microbenchmarks that ground the kernel
    design): fp32 / bf16 / fp16 matrix instructions and fp32 vector
    FMAs, each with independent accumulators, the fp32 and bf16 matrix
    instructions interleaved with vector FMAs in the same wavefronts, a
    device-to-device copy, and what an empty kernel launch costs back to back
    (from a host loop and from a graph).  One JSON line per measurement."""
    import ctypes
    import torch
    from paper_2609_09020_amd import build as B
    lib = ctypes.CDLL(B.PEAKS_LIB)
    lib.pic_peaks_launch.restype = ctypes.c_int
    lib.pic_peaks_launch.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    props = torch.cuda.get_device_properties(dev)
    cus = props.multi_processor_count
    # (name, matrix FLOP per iteration per wavefront, vector FLOP per iteration per wavefront)
    kinds = [("fp32 matrix v_mfma_f32_16x16x4_f32", 8 * 2048, 0),
             ("bf16 matrix v_mfma_f32_16x16x32_bf16", 8 * 16384, 0),
             ("fp16 matrix v_mfma_f32_16x16x32_f16", 8 * 16384, 0),
             ("fp32 vector v_fma_f32 (not packed)", 0, 32 * 128),
             ("fp32 matrix + fp32 vector, interleaved", 8 * 2048, 32 * 128),
             ("bf16 matrix + fp32 vector, interleaved", 8 * 16384, 32 * 128)]
    alone = {}
    for waves_per_simd in (1, 2, 4):
        blocks = cus * waves_per_simd                  # 4 wavefronts per workgroup: one per SIMD
        out = torch.empty(blocks * 256, dtype=torch.float32, device=dev)
        for kind, (what, mf, vf) in enumerate(kinds):
            iters = 20000 if kind != 3 else 40000

            def launch():
                st = lib.pic_peaks_launch(kind, blocks, iters, ctypes.c_void_p(out.data_ptr()),
                                          ctypes.c_void_p(stream.cuda_stream))
                if st:
                    raise RuntimeError(f"pic_peaks_launch({kind}) failed: {st}")
            launch()
            torch.cuda.synchronize()
            ms, _ = time_calls(launch, 5, 1, stream)
            waves = blocks * 4
            mt = mf * iters * waves / (ms * 1e-3) / 1e12
            vt = vf * iters * waves / (ms * 1e-3) / 1e12
            # cycles at the published 2.4 GHz engine clock
            cyc = ms * 1e-3 * CLOCK_HZ / (waves_per_simd * iters)
            rec = {"peaks": what, "waves_per_simd": waves_per_simd, "ms": round(ms, 4),
                   "matrix_tflops": round(mt, 1), "vector_tflops": round(vt, 1),
                   "cycles_per_iteration_per_simd": round(cyc * waves_per_simd, 1),
                   "cycles_per_iteration_per_wave": round(cyc, 1)}
            # per-iteration cycles per SIMD: the mixed kernels against the sum
            # of their parts (0: the parts serialise, 1: the shorter is hidden)
            if kind < 4:
                alone[(kind, waves_per_simd)] = cyc * waves_per_simd
            else:
                a = alone[(0 if kind == 4 else 1, waves_per_simd)]
                v = alone[(3, waves_per_simd)]
                both = cyc * waves_per_simd
                rec["sum_of_parts_cycles_per_simd"] = round(a + v, 1)
                rec["overlap_frac"] = round((a + v - both) / min(a, v), 3)
            print(json.dumps(rec), flush=True)
    n = 1 << 30
    src = torch.full((n,), 7, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    ms, _ = time_calls(lambda: dst.copy_(src), 20, 3, stream)
    print(json.dumps({"peaks": "device copy (torch copy_ of 1 GiB)", "ms": round(ms, 4),
                      "read_plus_write_gbs": round(2 * n / (ms * 1e-3) / 1e9, 1)}), flush=True)
    del src, dst
    # What a launch costs with nothing in it: an empty kernel, 200 launches
    # back to back, from a host loop and replayed from a graph.
    lib.pic_peaks_launch_cadence.restype = ctypes.c_int
    lib.pic_peaks_launch_cadence.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                             ctypes.POINTER(ctypes.c_float)]
    buf = torch.empty(4096, dtype=torch.float32, device=dev)
    for blocks in (1, 256, 768, 3072):
        rec = {"peaks": "empty kernel launch", "workgroups": blocks, "threads": 256}
        for graph in (0, 1):
            us = ctypes.c_float(0.0)
            st = lib.pic_peaks_launch_cadence(blocks, 200, graph, ctypes.c_void_p(buf.data_ptr()), ctypes.byref(us))
            if st:
                raise RuntimeError(f"pic_peaks_launch_cadence failed: {st}")
            rec["graph_us_per_launch" if graph else "host_loop_us_per_launch"] = round(us.value, 3)
        print(json.dumps(rec), flush=True)


def width_sweep(args):
    """Decode speed against synthesis width for the paper's net shape: L = 8
    levels, three hidden layers of width W, 3 outputs, 768x512 (the Kodak image
    size), fp32, in the fp32 matrix-core, fp16-split matrix-core and vector
    families.  Width 8 runs in 16-wide matrix blocks (zero padded)."""
    import ctypes
    import torch
    from paper_2609_09020_amd import synth
    from paper_2609_09020_amd import decoder as D
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    H, W = 512, 768
    for width in (8, 16, 24, 32, 40, 48, 64):
        widths = (8, width, width, width, 3)
        inp = synth.make_inputs(H, W, 8, widths, batch=1, seed=0, latent="laplace_int",
                                latent_scale=2.0, latent_clip=32)
        lat = [torch.from_numpy(a).to(dev) for a in inp.latents]
        wt = torch.from_numpy(inp.weights).to(dev)
        bt = torch.from_numpy(inp.biases).to(dev)
        lib = D.load_library()
        lat_arr = (ctypes.c_void_p * len(lat))(*[t.data_ptr() for t in lat])
        for variant in ("mfma_f32", "mfma_f16x3", "valu"):
            dec = D.Decoder(H, W, widths, max_batch=1, variant=variant)
            out = dec.alloc_out(1, dev)
            # the pre-marshalled raw call, as in the main measurement: the
            # Python wrapper's checks would make a call of this size host-bound
            run_args = (ctypes.c_void_p(dec.handle), ctypes.c_int32(1), lat_arr,
                        ctypes.c_void_p(wt.data_ptr()), ctypes.c_int64(dec.nw),
                        ctypes.c_void_p(bt.data_ptr()), ctypes.c_int64(dec.nb),
                        ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(stream.cuda_stream))

            def run():
                st = lib.pic_decode_run(*run_args)
                if st != D.PIC_OK:
                    raise D.PicError(st, "pic_decode_run")
            ms, wall = time_calls(run, args.steps, args.warmup, stream)
            fpp = flops_per_pixel(widths)
            print(json.dumps({"sweep": "width", "widths": list(widths), "variant": variant,
                              "kernel_avg_ms": round(ms, 5), "mpixel_s": round(H * W / ms / 1e3, 1),
                              "fps": round(1e3 / ms, 1), "flop_per_pixel": fpp,
                              "fp32_frac": round(fpp * H * W / (ms * 1e-3) / 1e12 / PEAK_FP32_TFLOPS, 4)}),
                  flush=True)
            dec.close()


def zpr_bytes_per_call(wl, n_symbols):
    """Compulsory HBM bytes of one latent-decoding call: the symbol stream read
    once (4 B per symbol) and every latent sample written once (4 B)."""
    from paper_2609_09020_amd import synth
    lat = sum(h * w for h, w in (synth.level_shape(wl.height, wl.width, k) for k in range(wl.levels)))
    return 4 * n_symbols + 4 * wl.batch * lat


def zpr_cpu_baseline(wl, stream, target_s=12.0):
    """The oracle's latent decoding of the workload's first image, repeated
    until about target_s seconds of CPU work."""
    import numpy as np
    import oracle
    threads = len(os.sched_getaffinity(0))
    orc = oracle.default()
    bpi = orc.zpr_blocks(wl.height, wl.width, wl.levels)
    marks = np.flatnonzero(stream.symbols == stream.eob)
    first = stream.symbols[:marks[bpi - 1] + 1]
    n_img = 0
    t0 = time.perf_counter()
    while True:
        orc.zpr_decode(first, stream.eob, wl.height, wl.width, wl.levels, 1)
        n_img += 1
        if time.perf_counter() - t0 >= target_s:
            break
    dt = time.perf_counter() - t0
    return {"value": round(n_img * wl.height * wl.width / dt / 1e6, 3), "unit": "Mpixel/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{n_img} decodes of the first image's symbol stream ({first.size} symbols, "
                      f"{bpi} blocks) by the fp64 C oracle (OpenMP over blocks), {dt:.1f} s"}


def huff_cpu_baseline(hs, wl, target_s=12.0):
    """The oracle's Huffman decoding of the workload's whole stream, repeated
    until about target_s seconds of CPU work (it is single-threaded)."""
    import oracle
    orc = oracle.default()
    n = 0
    t0 = time.perf_counter()
    while True:
        orc.huffman_decode(hs.data, hs.n_bits, hs.values, hs.lengths, hs.n_symbols)
        n += 1
        if time.perf_counter() - t0 >= target_s:
            break
    dt = time.perf_counter() - t0
    return {"value": round(n * wl.batch * wl.height * wl.width / dt / 1e6, 3), "unit": "Mpixel/s", "cores": 1,
            "kind": "oracle",
            "sample": f"{n} decodes of the workload's {hs.n_bits}-bit stream ({hs.n_symbols} symbols) by the "
                      f"C oracle (one thread), {dt:.1f} s"}


STAGE_NAMES = {
    ("huff",): "PIC entropy decoding (Huffman bitstream -> ZpR symbols)",
    ("zpr",): "PIC latent decoding (ZpR symbol stream -> latent pyramid)",
    ("zpr", "synth"): "PIC decode without entropy decoding (ZpR stream -> latents -> RGB)",
    ("huff", "zpr", "synth"): "PIC full decode (Huffman bitstream -> ZpR symbols -> latents -> RGB)",
}
STAGE_KERNELS = {"huff": "k_huff_table + k_huff_parse + k_huff_check + k_huff_fix + k_huff_count + k_huff_write",
                 "zpr": "k_zpr_count + k_zpr_expand", "synth": "pic_decode_run"}


def stage_bench(args, stages):
    """Time the decoder stages before (and with) the synthesis, each step
    running `stages` in order on device-resident inputs:
      huff   Huffman bitstream -> ZpR symbols   (pic_huff_decode)
      zpr    ZpR symbols -> latent pyramid      (pic_zpr_decode)
      synth  latent pyramid -> RGB              (pic_decode_run)"""
    import ctypes
    import numpy as np
    import torch
    from paper_2609_09020_amd import synth
    from paper_2609_09020_amd import decoder as D
    stages = tuple(stages)
    wl = synth.WORKLOADS[args.workload]
    zs = synth.workload_zpr_stream(wl)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    lib = D.load_library()
    sv = ctypes.c_void_p(stream.cuda_stream)
    calls, handles, checks = [], [], []
    sym = torch.from_numpy(zs.symbols).to(dev)
    hs = None
    if "huff" in stages:
        hs = synth.make_huff_stream(zs.symbols)
        hdata = torch.from_numpy(hs.data).to(dev)
        hvals = torch.from_numpy(hs.values).to(dev)
        hlens = torch.from_numpy(hs.lengths).to(dev)
        hst = torch.zeros(1, dtype=torch.int32, device=dev)
        hd = D.HuffDecoder(hs.n_bits)
        handles.append(hd)
        sym = torch.empty(hs.n_symbols, dtype=torch.int32, device=dev)
        calls.append((lib.pic_huff_decode, (ctypes.c_void_p(hd.handle), ctypes.c_void_p(hdata.data_ptr()),
                                            ctypes.c_int64(hs.n_bits), ctypes.c_void_p(hvals.data_ptr()),
                                            ctypes.c_void_p(hlens.data_ptr()), ctypes.c_int32(hs.values.size),
                                            ctypes.c_int64(hs.n_symbols), ctypes.c_void_p(sym.data_ptr()),
                                            ctypes.c_void_p(hst.data_ptr()), sv)))
        checks.append(("entropy decoding", hst))
    lat_arr = None
    if "zpr" in stages:
        z = D.ZprDecoder(wl.height, wl.width, wl.levels, wl.batch)
        handles.append(z)
        lat = [torch.empty((wl.batch,) + z.level_shape(k), dtype=torch.float32, device=dev)
               for k in range(wl.levels)]
        zst = torch.zeros(1, dtype=torch.int32, device=dev)
        lat_arr = (ctypes.c_void_p * wl.levels)(*[t.data_ptr() for t in lat])
        calls.append((lib.pic_zpr_decode, (ctypes.c_void_p(z.handle), ctypes.c_int32(wl.batch),
                                           ctypes.c_void_p(sym.data_ptr()), ctypes.c_int64(zs.symbols.size),
                                           ctypes.c_int32(zs.eob), lat_arr, ctypes.c_void_p(zst.data_ptr()), sv)))
        checks.append(("latent decoding", zst))
    dec = None
    if "synth" in stages:
        inp = synth.workload_inputs(wl)
        w = torch.from_numpy(inp.weights_bf16.view(np.int16) if inp.weights_bf16 is not None
                             else inp.weights).to(dev)
        b = torch.from_numpy(inp.biases).to(dev)
        dec = D.Decoder(wl.height, wl.width, wl.widths, weight_dtype=wl.weight_dtype,
                        out_dtype=args.out_dtype, max_batch=wl.batch, variant=args.variant)
        handles.append(dec)
        out = dec.alloc_out(wl.batch, dev)
        calls.append((lib.pic_decode_run,
                      (ctypes.c_void_p(dec.handle), ctypes.c_int32(wl.batch), lat_arr,
                       ctypes.c_void_p(w.data_ptr()), ctypes.c_int64(dec.nw), ctypes.c_void_p(b.data_ptr()),
                       ctypes.c_int64(dec.nb), ctypes.c_void_p(out.data_ptr()), sv)))

    def step():
        for fn, a in calls:
            r = fn(*a)
            if r != D.PIC_OK:
                raise D.PicError(r, fn.__name__)

    step()
    torch.cuda.synchronize()
    for what, st in checks:
        if int(st.item()) != 0:
            raise RuntimeError(f"{what} reported status {int(st.item())} on the benchmark stream")
    ms, wall = time_calls(step, args.steps, args.warmup, stream)
    # latency mode (the paper's serial protocol): synchronise, decode, synchronise
    lat_n = min(200, max(20, args.steps // 10))
    tl = 0.0
    for _ in range(lat_n):
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        step()
        torch.cuda.synchronize()
        tl += time.perf_counter() - t1
    px = wl.batch * wl.height * wl.width
    res = {
        "metric": STAGE_NAMES[stages], "value": round(px * args.steps / wall / 1e6, 2), "unit": "Mpixel/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(1e3 * wall / args.steps, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "fps": round(wl.batch * args.steps / wall, 1), "kernel_avg_ms": round(ms, 5),
        "latency_ms": round(1e3 * tl / lat_n, 4),
        "config": {"workload": f"{wl.name}: {wl.note}", "height": wl.height, "width": wl.width,
                   "levels": wl.levels, "batch": wl.batch, "symbols": int(zs.symbols.size),
                   "blocks": int(zs.blocks), "eob": int(zs.eob),
                   "kernels": " ; ".join(STAGE_KERNELS[s] for s in stages), "parallelism": "single GPU"},
    }
    if hs is not None:
        res["config"].update({"bitstream_bits": hs.n_bits, "table_entries": int(hs.values.size),
                              "longest_code": int(hs.lengths.max())})
    if dec is not None:
        res["config"].update({"widths": list(wl.widths), "weights": wl.weight_dtype,
                              "out_dtype": args.out_dtype, "synthesis_kernel": dec.info()["kernel_name"]})
    if stages == ("zpr",):
        nbytes = zpr_bytes_per_call(wl, zs.symbols.size)
        achieved = nbytes / (ms * 1e-3) / 1e9
        res["roofline"] = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                           "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                           "traffic": load_traffic("k_zpr", args.workload, "latents"),
                           "bytes_per_launch": nbytes, "kernels": STAGE_KERNELS["zpr"]}
        if not args.no_cpu_baseline:
            res["cpu_baseline"] = zpr_cpu_baseline(wl, zs)
    if stages == ("huff",):
        nbytes = (hs.n_bits + 7) // 8 + 4 * hs.n_symbols
        achieved = nbytes / (ms * 1e-3) / 1e9
        res["roofline"] = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                           "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None,
                           "bytes_per_launch": nbytes, "kernels": STAGE_KERNELS["huff"],
                           "note": "the bitstream read once and the symbols written once; the step is "
                                   "bound by its serial codeword chains and launch count, not by HBM"}
        res["symbols_per_s"] = round(hs.n_symbols / (ms * 1e-3), 1)
        if not args.no_cpu_baseline:
            res["cpu_baseline"] = huff_cpu_baseline(hs, wl)
    if stages == ("huff", "zpr", "synth"):
        # the same step with the bitstream copied in from pinned host memory
        # first (context for the paper's per-image figure; not the value)
        host = torch.from_numpy(hs.data).pin_memory()
        tl = 0.0
        for _ in range(lat_n):
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            hdata.copy_(host, non_blocking=True)
            step()
            torch.cuda.synchronize()
            tl += time.perf_counter() - t1
        res["latency_ms_with_h2d"] = round(1e3 * tl / lat_n, 4)
    if args.copy_calib:
        src = torch.full((256 << 20,), 7, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
    for h in handles:
        h.close()
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="kodak768")
    ap.add_argument("--variant", default="auto")
    ap.add_argument("--out-dtype", default="f32", choices=["f32", "u8"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-per-config", action="store_true",
                    help="leave out the other workloads' timings (per_config)")
    ap.add_argument("--peaks", action="store_true",
                    help="instead of the benchmark line, measure peak issue rates and copy bandwidth")
    ap.add_argument("--copy-calib", action="store_true",
                    help="also run a plain device copy of known size (counter calibration)")
    ap.add_argument("--width-sweep", action="store_true",
                    help="instead of the benchmark line, time the paper's 4-layer net shape "
                         "(8 -> W -> W -> W -> 3) at 768x512 for several widths W; one JSON line each")
    ap.add_argument("--zpr", action="store_true",
                    help="instead of the synthesis, time the latent decoding from the ZpR symbol "
                         "stream (pic_zpr_decode) on the workload's pyramid shape")
    ap.add_argument("--pipeline", action="store_true",
                    help="time the latent decoding followed by the synthesis as one step")
    ap.add_argument("--huff", action="store_true",
                    help="time the Huffman entropy decoding (pic_huff_decode) of the workload's stream")
    ap.add_argument("--full", action="store_true",
                    help="time the whole decoder as one step: Huffman bitstream -> symbols -> latents -> RGB")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: runs on exactly one GPU (the decoder has no multi-GPU "
              "path); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_09020_amd import synth
    from paper_2609_09020_amd import decoder as D

    if args.width_sweep:
        width_sweep(args)
        return
    if args.peaks:
        peaks(args)
        return
    for flag, stages in ((args.full, ("huff", "zpr", "synth")), (args.pipeline, ("zpr", "synth")),
                         (args.huff, ("huff",)), (args.zpr, ("zpr",))):
        if flag:
            stage_bench(args, stages)
            return

    wl = synth.WORKLOADS[args.workload]
    inp = synth.workload_inputs(wl)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lat = [torch.from_numpy(a).to(dev) for a in inp.latents]
    if inp.weights_bf16 is not None:
        w = torch.from_numpy(inp.weights_bf16.view(np.int16)).to(dev)
    else:
        w = torch.from_numpy(inp.weights).to(dev)
    b = torch.from_numpy(inp.biases).to(dev)
    dec = D.Decoder(wl.height, wl.width, wl.widths, weight_dtype=wl.weight_dtype,
                    out_dtype=args.out_dtype, max_batch=wl.batch, variant=args.variant)
    out = dec.alloc_out(wl.batch, dev)
    stream = torch.cuda.current_stream(dev)

    # The other workloads of the suite first (their inputs are made and freed
    # one at a time); the headline's inputs are resident already, and its
    # warm-up and timed calls follow with no host work in between.
    per_config = None
    if not args.no_per_config:
        per_config = {name: time_workload(name, out_dtype=args.out_dtype)
                      for name in PER_CONFIG if name != args.workload}
        for name in PER_CONFIG_F16X3:
            per_config[f"{name}@mfma_f16x3"] = time_workload(name, variant="mfma_f16x3",
                                                             out_dtype=args.out_dtype)
        torch.cuda.empty_cache()

    # Pre-marshalled raw call: the loop measures the library, not Python checks.
    import ctypes
    lib = D.load_library()
    lat_arr = (ctypes.c_void_p * len(lat))(*[t.data_ptr() for t in lat])
    run_args = (ctypes.c_void_p(dec.handle), ctypes.c_int32(wl.batch), lat_arr,
                ctypes.c_void_p(w.data_ptr()), ctypes.c_int64(dec.nw),
                ctypes.c_void_p(b.data_ptr()), ctypes.c_int64(dec.nb),
                ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(stream.cuda_stream))
    run = lib.pic_decode_run

    for _ in range(args.warmup):
        st = run(*run_args)
        if st != D.PIC_OK:
            raise D.PicError(st, "pic_decode_run")
    torch.cuda.synchronize()

    # Timed region: K back-to-back launches on the launch stream, bracketed by
    # synchronisation; two HIP events on that stream around the whole region
    # give the average device time per launch (kernel + dispatch gap).
    K = args.steps
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(K):
        run(*run_args)
    ev1.record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    kern_avg_ms = ev0.elapsed_time(ev1) / K

    # Latency mode (synchronise, decode, synchronise) over single calls.
    lat_n = min(200, max(20, K // 10))
    tl = 0.0
    for _ in range(lat_n):
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        run(*run_args)
        torch.cuda.synchronize()
        tl += time.perf_counter() - t1
    latency_ms = 1e3 * tl / lat_n

    if args.copy_calib:
        # Reference for the HBM byte counters: 5 copies of 256 MiB (read 256 MiB,
        # write 256 MiB each), from a source that has been written.
        src = torch.full((256 << 20,), 7, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()

    info = dec.info()
    px = wl.batch * wl.height * wl.width
    ms_per_step = 1e3 * elapsed / K
    mpx_s = px * K / elapsed / 1e6
    fpp = flops_per_pixel(wl.widths)
    flop = px * fpp
    kernel = info["kernel_name"]
    bound, peak, unit = variant_peak(info["variant"])
    achieved = flop / (kern_avg_ms * 1e-3) / 1e12
    traffic = load_traffic(kernel, args.workload, args.out_dtype)
    res = {
        "metric": METRIC, "value": round(mpx_s, 2), "unit": "Mpixel/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if wl.weight_dtype == "bf16" else "f32", "data": "synthetic",
        "fps": round(wl.batch * K / elapsed, 1),
        "latency_ms": round(latency_ms, 4),
        "kernel_avg_ms": round(kern_avg_ms, 5),
        "config": {"workload": f"{wl.name}: {wl.note}", "height": wl.height, "width": wl.width,
                   "levels": wl.levels, "widths": list(wl.widths), "batch": wl.batch,
                   "weights": wl.weight_dtype, "out_dtype": args.out_dtype,
                   "variant": info["variant"], "kernel": kernel, "parallelism": "single GPU"},
        "roofline": {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
                     "frac": round(achieved / peak, 4), "traffic": traffic,
                     "fp32_equivalent_frac": round(achieved / PEAK_FP32_TFLOPS, 4),
                     "flop_per_launch": flop, "flop_per_pixel": fpp,
                     "compulsory_bytes_per_launch": bytes_per_call(wl, args.out_dtype),
                     "hbm_frac_at_compulsory_bytes": round(
                         bytes_per_call(wl, args.out_dtype) / (kern_avg_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)},
    }
    dec.close()
    del lat, w, b, out
    res["paper_context"] = PAPER_CONTEXT
    if per_config is not None:
        res["per_config"] = per_config
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl, inp)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
