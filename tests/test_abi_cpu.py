"""C ABI checks that need no GPU: the library loads, exports exactly what
include/pic_decode.h and include/pic_zpr.h declare, struct layouts agree with
the headers, and invalid descriptors are rejected before any device is
touched."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2609_09020_amd as pkg
from paper_2609_09020_amd import decoder as D

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pic_decode.h")
HEADERS = [HEADER, os.path.join(ROOT, "include", "pic_zpr.h"), os.path.join(ROOT, "include", "pic_huff.h")]


def _declared():
    txt = "".join(open(h).read() for h in HEADERS)
    return sorted(set(re.findall(r"PIC_API\s+[\w\s\*]*?\b(pic_\w+)\s*\(", txt)))


def test_library_loads():
    assert os.path.exists(D.LIB_PATH), "build the library first"
    pkg.load_library()


def test_exports_match_header():
    declared = _declared()
    assert declared == sorted(D.EXPORTS)
    out = subprocess.run(["nm", "-D", "--defined-only", D.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = sorted(l.split()[-1] for l in out.splitlines()
                      if l.split()[-1].startswith("pic_") and " T " in l)
    assert exported == declared
    lib = pkg.load_library()
    for name in declared:
        assert hasattr(lib, name)


def test_struct_layout_matches_header(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "pic_decode.h"\n'
                   'int main(void){printf("%zu %zu %zu %zu %zu %zu\\n", sizeof(pic_decode_desc),'
                   ' offsetof(pic_decode_desc, widths), offsetof(pic_decode_desc, variant),'
                   ' sizeof(pic_decode_info), offsetof(pic_decode_info, kernel_name),'
                   ' offsetof(pic_decode_info, weights_per_image));return 0;}\n')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)],
                   check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    want = [ctypes.sizeof(D.pic_decode_desc), D.pic_decode_desc.widths.offset,
            D.pic_decode_desc.variant.offset, ctypes.sizeof(D.pic_decode_info),
            D.pic_decode_info.kernel_name.offset, D.pic_decode_info.weights_per_image.offset]
    assert got == want


def test_status_strings():
    for s in range(6):
        assert isinstance(pkg.pic_status_string(s), str) and pkg.pic_status_string(s)
    assert "unknown" in pkg.pic_status_string(99)


def _create_status(_raw=None, **kw):
    args = dict(height=64, width=64, widths=(4, 16, 16, 3))
    args.update(kw)
    desc = D.make_desc(**args)
    for k, v in (_raw or {}).items():
        setattr(desc, k, v)
    h = ctypes.c_void_p()
    st = pkg.load_library().pic_decode_create(ctypes.byref(desc), ctypes.byref(h))
    if st == D.PIC_OK:
        pkg.pic_decode_destroy(h.value)
    else:
        assert h.value is None
    return st


def _gpu_present():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.mark.parametrize("kw", [
    dict(height=0), dict(width=-1), dict(widths=(4, 16, 16, 4)),
    dict(widths=(3, 16, 16, 3), _raw={"num_levels": 4}), dict(_raw={"num_layers": 0}),
    dict(_raw={"num_layers": 9}),
    dict(widths=(4, 129, 3)), dict(widths=(4, 16, 129, 3)), dict(widths=(4, 0, 3)), dict(weight_dtype=2), dict(out_dtype=1),
    dict(flags=2), dict(flags=D.PIC_FLAG_NO_CLAMP, out_dtype=D.PIC_U8), dict(max_batch=0),
    dict(max_batch=70000), dict(variant=9), dict(variant=5), dict(height=65536, width=32768),
    dict(height=1, width=1 << 23), dict(height=1 << 23, width=1),
    dict(widths=(13,) + (16,) * 2 + (3,)),
])
def test_invalid_descriptors(kw):
    assert _create_status(**kw) == D.PIC_E_INVALID


def test_bad_struct_size_and_null_out():
    desc = D.make_desc(64, 64, (4, 16, 16, 3))
    desc.struct_size = 12
    h = ctypes.c_void_p()
    assert pkg.load_library().pic_decode_create(ctypes.byref(desc), ctypes.byref(h)) == D.PIC_E_INVALID
    desc = D.make_desc(64, 64, (4, 16, 16, 3))
    assert pkg.load_library().pic_decode_create(ctypes.byref(desc), None) == D.PIC_E_INVALID


def test_unsupported_combinations():
    # the bf16 matrix-core family needs bf16 weights, the fp16-split one fp32
    assert _create_status(variant=D.PIC_VARIANT_MFMA_BF16) == D.PIC_E_UNSUPPORTED
    assert _create_status(variant=D.PIC_VARIANT_MFMA_F16X3, weight_dtype=D.PIC_BF16) == D.PIC_E_UNSUPPORTED
    # the matrix-core families take 2 to 4 linear layers
    assert _create_status(variant=D.PIC_VARIANT_MFMA_F16X3, widths=(4, 3)) == D.PIC_E_UNSUPPORTED
    # ... and hidden widths up to 64 (four 16-neuron blocks); wider nets run on
    # the reference family, which AUTO then picks
    for v in (D.PIC_VARIANT_MFMA_F32, D.PIC_VARIANT_MFMA_F16X3):
        for widths in ((4, 65, 3), (8, 64, 96, 3), (8, 128, 128, 3)):
            assert _create_status(variant=v, widths=widths) == D.PIC_E_UNSUPPORTED
    assert _create_status(variant=D.PIC_VARIANT_MFMA_BF16, weight_dtype=D.PIC_BF16,
                          widths=(8, 128, 3)) == D.PIC_E_UNSUPPORTED


@pytest.mark.skipif(_gpu_present(), reason="checks the no-device path")
def test_widest_descriptors_pass_validation():
    # the largest hidden width, level count and depth are valid descriptors:
    # validation passes, and the CPU host then has no device
    assert _create_status(widths=(4, 128, 3)) == D.PIC_E_NODEVICE
    assert _create_status(widths=(12,) + (128,) * 7 + (3,)) == D.PIC_E_NODEVICE
    assert _create_status(widths=(12,) + (128,) * 7 + (3,), variant=D.PIC_VARIANT_VALU) == D.PIC_E_NODEVICE
    # and so are the longest image sides, 2^23 - 1
    assert _create_status(height=1, width=(1 << 23) - 1) == D.PIC_E_NODEVICE
    assert _create_status(height=(1 << 23) - 1, width=1) == D.PIC_E_NODEVICE


@pytest.mark.skipif(_gpu_present(), reason="checks the no-device path")
def test_nodevice_on_cpu_host():
    assert _create_status() == D.PIC_E_NODEVICE
    with pytest.raises(pkg.PicError) as e:
        pkg.Decoder(64, 64, (4, 16, 16, 3))
    assert e.value.status == D.PIC_E_NODEVICE


def test_null_handle_is_rejected():
    lib = pkg.load_library()
    assert lib.pic_decode_run(None, 1, None, None, 0, None, 0, None, None) == D.PIC_E_INVALID
    info = D.pic_decode_info()
    info.struct_size = ctypes.sizeof(D.pic_decode_info)
    assert lib.pic_decode_query(None, ctypes.byref(info)) == D.PIC_E_INVALID
    lib.pic_decode_destroy(None)   # accepted


def test_fuse_modulation_argument_checks_without_device():
    f = D.pic_fuse_modulation
    p = 4096   # never dereferenced: every call below returns before any launch
    assert f(0, 4, 1, p, 0, p, 0, p, p, p, p, 0, p, p) == D.PIC_E_INVALID
    assert f(4, 4, -1, p, 0, p, 0, p, p, p, p, 0, p, p) == D.PIC_E_INVALID
    assert f(4, 4, 1, p, 15, p, 0, p, p, p, p, 0, p, p) == D.PIC_E_INVALID      # stride < in*out
    assert f(4, 4, 1, p + 2, 0, p, 0, p, p, p, p, 0, p, p) == D.PIC_E_INVALID   # misaligned
    assert f(4, 4, 0, p, 0, p, 0, p, p, p, p, 0, p, p) == D.PIC_OK              # empty batch
    if not _gpu_present():
        assert f(4, 4, 1, p, 0, p, 0, p, p, p, p, 0, p, p) == D.PIC_E_NODEVICE


def test_run_layers_null_handle():
    assert D.pic_decode_run_layers(None, 1, [0], [0], [0], [0], [0], 0) == D.PIC_E_INVALID


def test_zpr_struct_layout_matches_header(tmp_path):
    src = tmp_path / "layout_zpr.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "pic_zpr.h"\n'
                   'int main(void){printf("%zu %zu %zu %zu %zu %zu\\n", sizeof(pic_zpr_desc),'
                   ' offsetof(pic_zpr_desc, max_batch), sizeof(pic_zpr_info),'
                   ' offsetof(pic_zpr_info, blocks_per_image), offsetof(pic_zpr_info, scratch_bytes),'
                   ' offsetof(pic_zpr_info, symbols_per_chunk));'
                   'printf("%d %d %d\\n", PIC_ZPR_ERR_COUNT, PIC_ZPR_ERR_OVERFLOW, PIC_ZPR_ERR_SYMBOL);'
                   'return 0;}\n')
    exe = tmp_path / "layout_zpr"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)],
                   check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    want = [ctypes.sizeof(D.pic_zpr_desc), D.pic_zpr_desc.max_batch.offset, ctypes.sizeof(D.pic_zpr_info),
            D.pic_zpr_info.blocks_per_image.offset, D.pic_zpr_info.scratch_bytes.offset,
            D.pic_zpr_info.symbols_per_chunk.offset,
            D.PIC_ZPR_ERR_COUNT, D.PIC_ZPR_ERR_OVERFLOW, D.PIC_ZPR_ERR_SYMBOL]
    assert got == want


def _zpr_create_status(**raw):
    desc = D.make_zpr_desc(64, 64, 4, 1)
    for k, v in raw.items():
        setattr(desc, k, v)
    h = ctypes.c_void_p()
    st = pkg.load_library().pic_zpr_create(ctypes.byref(desc), ctypes.byref(h))
    if st == D.PIC_OK:
        pkg.pic_zpr_destroy(h.value)
    else:
        assert h.value is None
    return st


@pytest.mark.parametrize("raw", [dict(height=0), dict(width=-3), dict(num_levels=0), dict(num_levels=13),
                                 dict(max_batch=0), dict(max_batch=65536), dict(struct_size=8),
                                 dict(height=65536, width=32768)])
def test_zpr_invalid_descriptors(raw):
    assert _zpr_create_status(**raw) == D.PIC_E_INVALID


def test_zpr_unsupported_size():
    # 4K at 65535 images: more than 2^31 blocks in one stream
    assert _zpr_create_status(height=2160, width=3840, num_levels=8, max_batch=65535) == D.PIC_E_UNSUPPORTED


def test_zpr_null_arguments():
    lib = pkg.load_library()
    assert lib.pic_zpr_create(None, None) == D.PIC_E_INVALID
    assert D.pic_zpr_decode(None, 1, 4096, 4, 20, [4096], 4096) == D.PIC_E_INVALID
    assert D.pic_zpr_expand(None, 1, 4096, 4, 20, 4096, 4096) == D.PIC_E_INVALID
    info = D.pic_zpr_info()
    info.struct_size = ctypes.sizeof(D.pic_zpr_info)
    assert lib.pic_zpr_query(None, ctypes.byref(info)) == D.PIC_E_INVALID
    lib.pic_zpr_destroy(None)   # accepted


@pytest.mark.skipif(_gpu_present(), reason="checks the no-device path")
def test_zpr_nodevice_on_cpu_host():
    assert _zpr_create_status() == D.PIC_E_NODEVICE
    with pytest.raises(pkg.PicError) as e:
        pkg.ZprDecoder(64, 64, 4)
    assert e.value.status == D.PIC_E_NODEVICE


def test_huff_struct_layout_matches_header(tmp_path):
    src = tmp_path / "layout_huff.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "pic_huff.h"\n'
                   'int main(void){printf("%zu %zu %zu %zu %zu %zu\\n", sizeof(pic_huff_desc),'
                   ' offsetof(pic_huff_desc, max_bits), sizeof(pic_huff_info),'
                   ' offsetof(pic_huff_info, scratch_bytes), offsetof(pic_huff_info, bits_per_thread),'
                   ' offsetof(pic_huff_info, lut_bits));'
                   'printf("%d %d %d %d %d\\n", PIC_HUFF_ERR_BITS, PIC_HUFF_ERR_CODE, PIC_HUFF_ERR_TABLE,'
                   ' PIC_HUFF_MAX_LEN, PIC_HUFF_MAX_TABLE);return 0;}\n')
    exe = tmp_path / "layout_huff"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    want = [ctypes.sizeof(D.pic_huff_desc), D.pic_huff_desc.max_bits.offset, ctypes.sizeof(D.pic_huff_info),
            D.pic_huff_info.scratch_bytes.offset, D.pic_huff_info.bits_per_thread.offset,
            D.pic_huff_info.lut_bits.offset, D.PIC_HUFF_ERR_BITS, D.PIC_HUFF_ERR_CODE, D.PIC_HUFF_ERR_TABLE,
            D.PIC_HUFF_MAX_LEN, D.PIC_HUFF_MAX_TABLE]
    assert got == want


@pytest.mark.parametrize("raw", [dict(max_bits=0), dict(max_bits=2**31), dict(struct_size=4), dict(reserved=1)])
def test_huff_invalid_descriptors(raw):
    desc = D.make_huff_desc(1 << 20)
    for k, v in raw.items():
        setattr(desc, k, v)
    h = ctypes.c_void_p()
    assert pkg.load_library().pic_huff_create(ctypes.byref(desc), ctypes.byref(h)) == D.PIC_E_INVALID
    assert h.value is None


def test_huff_null_arguments():
    lib = pkg.load_library()
    assert lib.pic_huff_create(None, None) == D.PIC_E_INVALID
    assert D.pic_huff_decode(None, 4096, 8, 4096, 4096, 1, 1, 4096, 4096) == D.PIC_E_INVALID
    info = D.pic_huff_info()
    info.struct_size = ctypes.sizeof(D.pic_huff_info)
    assert lib.pic_huff_query(None, ctypes.byref(info)) == D.PIC_E_INVALID
    lib.pic_huff_destroy(None)


@pytest.mark.skipif(_gpu_present(), reason="checks the no-device path")
def test_huff_nodevice_on_cpu_host():
    h = ctypes.c_void_p()
    desc = D.make_huff_desc(1 << 20)
    assert pkg.load_library().pic_huff_create(ctypes.byref(desc), ctypes.byref(h)) == D.PIC_E_NODEVICE
