"""Host sanitizer builds (AddressSanitizer + UndefinedBehaviorSanitizer), no
GPU:

- the C oracle built by gcc with both sanitizers, and the oracle's pin tests
  run against that build (tests/test_oracle_pins.py in a child process with
  gcc's runtime preloaded);
- the host side of the C ABI (pic_decode.hip, pic_zpr.hip, pic_huff.hip:
  argument validation, handle set-up, status strings) built by hipcc with
  both sanitizers on the host pass only, linked with the ordinary kernel
  objects, and the ABI tests (tests/test_abi_cpu.py) run against it with
  clang's runtime preloaded.

Each run is preceded by a positive control: a tiny library with a planted
heap overflow, built the same way, must be reported, so that a silent
sanitizer cannot pass the test.  Leak detection is off (the Python
interpreter itself does not free everything at exit)."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2609_09020_amd", "csrc")
BUILD = os.path.join(ROOT, "_build")
HIPCC = "/opt/rocm/bin/hipcc"
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0", "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"}

PLANTED = r"""
#include <stdlib.h>
int planted_overflow(int n) {
    int *a = (int *)malloc(sizeof(int) * n);
    for (int i = 0; i <= n; ++i) a[i] = i;   /* one past the end */
    int s = a[0];
    free(a);
    return s;
}
"""


def _run_child(code, preload, extra_env=None, timeout=600):
    env = dict(os.environ, LD_PRELOAD=preload, **SAN_ENV, **(extra_env or {}))
    return subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env,
                          timeout=timeout, cwd=ROOT)


def _planted_is_reported(compile_cmd, lib, preload):
    subprocess.run(compile_cmd, check=True, capture_output=True)
    r = _run_child(f"import ctypes; ctypes.CDLL({lib!r}).planted_overflow(8)", preload)
    return r.returncode != 0 and "heap-buffer-overflow" in r.stderr


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_pins_under_asan_ubsan(tmp_path):
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("gcc has no AddressSanitizer runtime")
    flags = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]
    # positive control
    src = tmp_path / "planted.c"
    src.write_text(PLANTED)
    ctl = str(tmp_path / "libplanted_gcc.so")
    assert _planted_is_reported(["gcc", "-O1", "-fPIC", "-shared", *flags, str(src), "-o", ctl], ctl, asan)
    # the oracle, sanitized
    sys.path.insert(0, ROOT)
    from oracle import build as obuild
    lib = obuild.build(out=str(tmp_path / "liboracle_san.so"), extra_flags=flags)
    code = ("import sys, pytest; sys.exit(pytest.main(['tests/test_oracle_pins.py', '-q', '-s', "
            "'-p', 'no:cacheprovider']))")
    r = _run_child(code, asan, {"PIC_ORACLE_LIB": lib})
    print(r.stdout[-2000:])
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert "runtime error" not in r.stdout + r.stderr
    assert "AddressSanitizer" not in r.stdout + r.stderr


def _clang_asan_runtime():
    rt = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return rt[-1] if rt else None


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="needs hipcc")
def test_abi_host_code_under_asan_ubsan(tmp_path):
    rt = _clang_asan_runtime()
    if rt is None:
        pytest.skip("no clang AddressSanitizer runtime")
    kernel_objs = [o for o in sorted(glob.glob(os.path.join(BUILD, "k_*.hip.o"))) if "k_peaks" not in o]
    if not kernel_objs:
        pytest.skip("build the library first (the kernel objects are linked as built)")
    clangxx = "/opt/rocm/llvm/bin/clang++"
    # positive control, same runtime
    src = tmp_path / "planted.cpp"
    src.write_text(PLANTED.replace("int planted_overflow", 'extern "C" int planted_overflow'))
    ctl = str(tmp_path / "libplanted_clang.so")
    assert _planted_is_reported([clangxx, "-O1", "-fPIC", "-shared", "-fsanitize=address,undefined",
                                 "-shared-libsan", str(src), "-o", ctl], ctl, rt)
    # the ABI's host translation units, sanitized on the host pass only
    flags = ["-O1", "-g", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-fvisibility=hidden",
             "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC,
             "-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=all",
             "-Xarch_host", "-fno-omit-frame-pointer"]
    objs = []
    procs = []
    for tu in ("pic_decode", "pic_zpr", "pic_huff"):
        o = str(tmp_path / f"{tu}.o")
        objs.append(o)
        procs.append(subprocess.Popen([HIPCC, *flags, "-c", os.path.join(CSRC, tu + ".hip"), "-o", o],
                                      stdout=subprocess.PIPE, stderr=subprocess.PIPE))
    for p in procs:
        _, err = p.communicate(timeout=600)
        assert p.returncode == 0, err.decode()[-2000:]
    lib = str(tmp_path / "libpic_decode_san.so")
    subprocess.run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", lib, *objs, *kernel_objs],
                   check=True, capture_output=True)
    code = ("import sys\n"
            "from paper_2609_09020_amd import decoder as D\n"
            f"D.LIB_PATH = {lib!r}\n"
            f"D.load_library.__defaults__ = ({lib!r},)\n"
            "import pytest\n"
            "sys.exit(pytest.main(['tests/test_abi_cpu.py', '-q', '-s', '-p', 'no:cacheprovider']))\n")
    r = _run_child(code, rt)
    print(r.stdout[-2000:])
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert "runtime error" not in r.stdout + r.stderr
    assert "AddressSanitizer" not in r.stdout + r.stderr
