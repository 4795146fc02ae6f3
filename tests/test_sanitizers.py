"""Host-side sanitizer runs (CPU only).

The oracle is rebuilt with AddressSanitizer and UndefinedBehaviorSanitizer and
its pins run against that build; the library is rebuilt with both sanitizers
on its host code (device code is unchanged) and the C-ABI argument checks run
against it.  Each build also gets one planted mistake that the sanitizer must
report, so a run that passes is known to have had the checks live.  Every
sanitized run is its own process with the sanitizer runtime preloaded (a
Python interpreter is not built with it).
"""
import glob
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_SRC = os.path.join(ROOT, "oracle", "scone_oracle.cpp")
CSRC = os.path.join(ROOT, "paper_2502_01637_amd", "csrc")
LIB_SOURCES = ["runtime", "table_build", "lookup", "gather", "embed", "decode", "gather_split",
               "discover", "fgram_model", "pipeline"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def gcc_asan_runtime():
    p = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = p.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def clang_asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def run_sanitized(runtime, script, *args):
    env = dict(os.environ, **SAN_ENV)
    env["LD_PRELOAD"] = ":".join(p for p in (runtime, os.environ.get("LD_PRELOAD", "")) if p)
    return subprocess.run([sys.executable, "-c", script, *args], env=env, capture_output=True,
                          text=True, timeout=600, cwd=ROOT)


ORACLE_PINS = textwrap.dedent("""
    import ctypes, sys
    sys.path[:0] = [{root!r}, {tests!r}]
    import oracle
    oracle._lib = oracle.bind(ctypes.CDLL(sys.argv[1]))
    import pytest
    sys.exit(pytest.main(["-q", "-p", "no:cacheprovider", {pins!r}]))
""").format(root=ROOT, tests=os.path.join(ROOT, "tests"),
            pins=os.path.join(ROOT, "tests", "test_oracle_pins.py"))

ORACLE_ROW_PAST_END = textwrap.dedent("""
    import ctypes, sys
    sys.path[:0] = [{root!r}]
    import numpy as np
    import oracle
    oracle._lib = oracle.bind(ctypes.CDLL(sys.argv[1]))
    table = np.arange(4 * 16, dtype=np.uint8).reshape(4, 16)
    oracle.gather(np.array([0, 4], dtype=np.int32), table)   # row 4 of 4
""").format(root=ROOT)


def build_oracle(tmp_path, src_text):
    src = tmp_path / "oracle.cpp"
    src.write_text(src_text)
    so = tmp_path / "liboracle_san.so"
    subprocess.check_call(["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           "-shared", "-fPIC", "-o", str(so), str(src)])
    return str(so)


@pytest.fixture(scope="module")
def gcc_asan():
    rt = gcc_asan_runtime()
    if rt is None:
        pytest.skip("g++ has no AddressSanitizer runtime here")
    return rt


def test_oracle_pins_pass_under_asan_and_ubsan(gcc_asan, tmp_path):
    so = build_oracle(tmp_path, open(ORACLE_SRC).read())
    r = run_sanitized(gcc_asan, ORACLE_PINS, so)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "passed" in r.stdout


def test_oracle_sanitizer_reports_a_planted_row_overrun(gcc_asan, tmp_path):
    src = open(ORACLE_SRC).read()
    assert src.count("r >= n_rows") == 1
    so = build_oracle(tmp_path, src.replace("r >= n_rows", "r > n_rows"))
    r = run_sanitized(gcc_asan, ORACLE_ROW_PAST_END, so)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr, r.stderr[-3000:]


# ------------------------------------------------------------- library ----

LIB_ABI = textwrap.dedent("""
    import ctypes, sys
    sys.path[:0] = [{root!r}, {tests!r}]
    import paper_2502_01637_amd as S
    S.scone._lib = S.scone._declare(ctypes.CDLL(sys.argv[1]))
    import pytest
    sys.exit(pytest.main(["-q", "-p", "no:cacheprovider", {abi!r}]))
""").format(root=ROOT, tests=os.path.join(ROOT, "tests"),
            abi=os.path.join(ROOT, "tests", "test_abi_cpu.py"))

LIB_HUGE_SPLIT = textwrap.dedent("""
    import ctypes, sys
    lib = ctypes.CDLL(sys.argv[1])
    P, I64 = ctypes.c_void_p, ctypes.c_int64
    lib.scone_gather_split.argtypes = [P, I64, P, I64, P, I64, I64, P, P, I64, P, P]
    f = ctypes.c_void_p(1 << 32)
    print(lib.scone_gather_split(f, 1 << 61, f, 1, f, 1, 16, f, f, 1 << 40, None, None))
""")


def hipcc_object(src, obj, include_dirs):
    # host code only is sanitized: each -fsanitize= flag follows -Xarch_host
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-c", src, "-o", obj]
    for d in include_dirs:
        cmd[1:1] = ["-I", d]
    return subprocess.Popen(cmd, stdout=subprocess.DEVNULL, stderr=subprocess.PIPE)


def hipcc_link(objs, so):
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC",
                           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                           "-shared-libasan", "-o", so] + objs,
                          stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)


@pytest.fixture(scope="module")
def sanitized_objects(tmp_path_factory):
    if clang_asan_runtime() is None or not os.path.exists(HIPCC):
        pytest.skip("hipcc or clang's AddressSanitizer runtime is missing")
    import torch
    if torch.cuda.device_count() > 0:
        # the library checks run test_abi_cpu.py, which passes fake device
        # addresses and is meant for a process without a GPU
        pytest.skip("a GPU is visible")
    d = tmp_path_factory.mktemp("libsan")
    inc = [os.path.join(ROOT, "include"), CSRC]
    objs, procs = [], []
    for name in LIB_SOURCES:
        obj = str(d / f"{name}.o")
        procs.append((name, hipcc_object(os.path.join(CSRC, name + ".hip"), obj, inc)))
        objs.append(obj)
    for name, p in procs:
        _, err = p.communicate()
        assert p.returncode == 0, (name, err.decode()[-2000:])
    return d, objs


def test_library_host_checks_pass_under_asan_and_ubsan(sanitized_objects):
    d, objs = sanitized_objects
    so = str(d / "libscone_san.so")
    hipcc_link(objs, so)
    r = run_sanitized(clang_asan_runtime(), LIB_ABI, so)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "passed" in r.stdout


def test_library_sanitizer_reports_a_planted_overflow(sanitized_objects):
    """Without the size bound, the byte count of a huge split gather overflows
    64 bits in the argument checks, which UBSan must report."""
    d, objs = sanitized_objects
    src = open(os.path.join(CSRC, "gather_split.hip")).read()
    bound = "(int64_t)1 << 31) || n_tok > ((int64_t)1 << 40) / row_bytes"
    assert src.count(bound) == 1
    mut = d / "gather_split_mutant.hip"
    mut.write_text(src.replace(bound, "(int64_t)1 << 31)"))
    obj = str(d / "gather_split_mutant.o")
    p = hipcc_object(str(mut), obj, [os.path.join(ROOT, "include"), CSRC])
    _, err = p.communicate()
    assert p.returncode == 0, err.decode()[-2000:]
    so = str(d / "libscone_mutant.so")
    hipcc_link([o for o in objs if not o.endswith("gather_split.o")] + [obj], so)
    r = run_sanitized(clang_asan_runtime(), LIB_HUGE_SPLIT, so)
    assert r.returncode != 0 and "overflow" in r.stderr, r.stdout[-2000:] + r.stderr[-2000:]
