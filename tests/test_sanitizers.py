"""AddressSanitizer and UndefinedBehaviorSanitizer runs of the host code.

Two libraries are rebuilt with the sanitizers into a temporary directory and
loaded into a child Python process with the sanitizer runtime preloaded:
- the oracle (gcc), running the oracle's pin tests;
- libw2v (hipcc; the sanitizers apply to the host pass only, device code is
  unchanged), running the C ABI's argument-check tests, which exercise the
  host-side validation and never launch a kernel.
A first test plants an out-of-bounds write in a scratch library and checks
that the harness reports it, so a clean run means something.
"""
import os
import shutil
import subprocess
import sys
import textwrap

import pytest

pytestmark = pytest.mark.slow
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0", "UBSAN_OPTIONS": "print_stacktrace=1"}


def gcc_asan_runtime():
    if not shutil.which("gcc"):
        pytest.skip("gcc not found")
    p = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(p) or not os.path.exists(p):
        pytest.skip("gcc's libasan not found")
    return p


def clang_asan_runtime():
    import glob
    rts = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rts or not os.path.exists(HIPCC):
        pytest.skip("hipcc or clang's ASan runtime not found")
    return rts[-1]


def child(code, preload, extra_env=None, timeout=600):
    env = dict(os.environ, LD_PRELOAD=preload, **SAN_ENV, **(extra_env or {}))
    return subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=timeout)


def gcc_san(src, out):
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           "-fno-omit-frame-pointer", src, "-o", out, "-lm"])


def test_harness_reports_a_planted_overflow(tmp_path):
    rt = gcc_asan_runtime()
    src = tmp_path / "bad.c"
    src.write_text("#include <stdlib.h>\nint bad(int n) { int *a = malloc(4 * n); a[n] = 1; int r = a[0]; "
                   "free(a); return r; }\n")
    lib = str(tmp_path / "libbad.so")
    gcc_san(str(src), lib)
    r = child(f"import ctypes; ctypes.CDLL({lib!r}).bad(8)", rt)
    assert r.returncode != 0 and "AddressSanitizer: heap-buffer-overflow" in r.stderr


def test_oracle_pins_under_asan_ubsan(tmp_path):
    rt = gcc_asan_runtime()
    lib = str(tmp_path / "liboracle_san.so")
    gcc_san(os.path.join(ROOT, "oracle", "w2v_oracle.c"), lib)
    code = textwrap.dedent("""
        import sys, glob, pytest
        files = sorted(glob.glob('tests/test_oracle_*.py'))
        sys.exit(pytest.main(files + ['-q', '-x', '-p', 'no:cacheprovider', '-m', 'not gpu']))
    """)
    r = child(code, rt, {"W2V_ORACLE_LIB": lib})
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out
    assert " passed" in r.stdout


def test_abi_checks_under_asan_ubsan(tmp_path):
    rt = clang_asan_runtime()
    csrc = os.path.join(ROOT, "paper_1606_07822_amd", "csrc")
    import paper_1606_07822_amd._build as b
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-fPIC", "-std=c++17", "-munsafe-fp-atomics",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
             "-I" + os.path.join(ROOT, "include")]
    procs, objs = [], []
    for src in b.SOURCES:
        obj = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        objs.append(obj)
        procs.append(subprocess.Popen([HIPCC, *flags, "-c", os.path.join(csrc, src), "-o", obj],
                                      stdout=subprocess.DEVNULL, stderr=subprocess.PIPE, text=True))
    for p in procs:
        _, err = p.communicate()
        assert p.returncode == 0, err[-3000:]
    lib = str(tmp_path / "libw2v_san.so")
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Xarch_host", "-fsanitize=address",
                           "-Xarch_host", "-fsanitize=undefined", *objs, "-o", lib])
    code = textwrap.dedent("""
        import sys, pytest
        sys.exit(pytest.main(['tests/test_abi.py', '-q', '-x', '-p', 'no:cacheprovider']))
    """)
    r = child(code, rt, {"W2V_TEST_LIB": lib})
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out
    assert " passed" in r.stdout
