"""Host-side sanitizers (CPU only).  The float64 oracle and the host code of
the C ABI (argument validation, workspace carving, the store-file reader and
writer: abi.cpp, store_file.cpp) are rebuilt with AddressSanitizer and
UndefinedBehaviorSanitizer -- the host pass only; device code is linked from
the regular build -- and the CPU tests that drive them (every validation path
of the ABI, store-file round trips and errors, the oracle's pins) run against
those builds in a child process.  Any sanitizer report fails the test."""
import glob
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2405_13954_amd", "csrc")
OBJ = os.path.join(ROOT, "_build", "obj")


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"


@pytest.fixture(scope="module")
def sanitized(tmp_path_factory):
    d = tmp_path_factory.mktemp("sanitized")
    rt = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rt:
        pytest.fail("clang's AddressSanitizer runtime is not installed under /opt/rocm/llvm")
    oracle_so = str(d / "liblogra_oracle_san.so")
    _run(["/opt/rocm/llvm/bin/clang", "-std=c99", "-O1", "-g", "-fno-omit-frame-pointer",
          "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-shared-libsan", "-fPIC", "-shared",
          os.path.join(ROOT, "oracle", "logra_oracle.c"), "-o", oracle_so, "-lm"])
    # the device-side objects of the regular build (built here if missing)
    from paper_2405_13954_amd import build as hb
    hip_objs = []
    for src in sorted(glob.glob(os.path.join(CSRC, "*.hip"))):
        obj = os.path.join(OBJ, os.path.basename(src) + ".o")
        if not os.path.exists(obj):
            os.makedirs(OBJ, exist_ok=True)
            _run(["hipcc", *hb.flags_for(src), "-c", src, "-o", obj])
        hip_objs.append(obj)
    host_flags = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                  "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-shared-libsan",
                  "-Xarch_host", "-fno-omit-frame-pointer"]
    san_objs = []
    for src in ("abi.cpp", "store_file.cpp"):
        obj = str(d / (src + ".o"))
        _run(["hipcc", *[f for f in hb.FLAGS if f != "-O3"], "-O1", "-g", *host_flags, "-c",
              os.path.join(CSRC, src), "-o", obj])
        san_objs.append(obj)
    lib_so = str(d / "libpaper_logra_san.so")
    _run(["hipcc", f"--offload-arch={hb.ARCH}", "-shared", "-fPIC", *host_flags, *san_objs, *hip_objs, "-o", lib_so])
    return rt[-1], oracle_so, lib_so, d


def test_abi_host_code_and_oracle_under_sanitizers(sanitized):
    rt, oracle_so, lib_so, d = sanitized
    runner = d / "run.py"
    runner.write_text(textwrap.dedent(f"""
        import os, sys
        sys.path.insert(0, {ROOT!r})
        import paper_2405_13954_amd as P
        P.LIB_PATH = {lib_so!r}          # the sanitized build of the same sources
        import pytest
        sys.exit(pytest.main(["-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu", "-k", "not peaks",
                              os.path.join({ROOT!r}, "tests", "test_abi_cpu.py"),
                              os.path.join({ROOT!r}, "tests", "test_store_file_cpu.py"),
                              os.path.join({ROOT!r}, "tests", "test_oracle_pins.py")]))
    """))
    env = dict(os.environ, LD_PRELOAD=rt, LOGRA_ORACLE_LIB=oracle_so,
               ASAN_OPTIONS="detect_leaks=0:protect_shadow_gap=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="4")
    r = subprocess.run([sys.executable, str(runner)], capture_output=True, text=True, env=env, cwd=str(d),
                       timeout=900)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out
    print(out.strip().splitlines()[-1])
