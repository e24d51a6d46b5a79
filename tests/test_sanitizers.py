"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Two builds in a temporary directory, each exercised in a process of its own
with its sanitizer runtime preloaded (the Python interpreter itself is not
instrumented):

  * the C-ABI library's host code (planner, coordinator, argument checks,
    id bitmaps), built by hipcc with the sanitizers on the host pass only
    (each -fsanitize= right after -Xarch_host; the device code is built as
    usual but never runs here), under the host, coordinator, property and
    driver-record tests;
  * the oracle, built by gcc with both sanitizers, under every pin.

Any report fails the run (halt_on_error); leak checking is off, since the
interpreter keeps objects alive until exit.  Skipped when a compiler or a
runtime is missing."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TESTS = os.path.join(ROOT, "tests")
PKG = os.path.join(ROOT, "paper_2406_03243_amd")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG_ASAN = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
ENV = {"ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0",
       "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _gcc_runtime(name):
    try:
        path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                              check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return path if os.path.isabs(path) and os.path.exists(path) else None


def _run(code, preload, timeout):
    env = dict(os.environ, **ENV, LD_PRELOAD=preload)
    return subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=timeout,
                          cwd=ROOT)


@pytest.mark.skipif(not os.path.exists(HIPCC) or not CLANG_ASAN, reason="hipcc or clang's ASan runtime missing")
def test_library_host_code_under_sanitizers(tmp_path):
    pkg = tmp_path / "paper_2406_03243_amd"
    pkg.mkdir()
    for f in glob.glob(os.path.join(PKG, "*.py")):
        shutil.copy(f, pkg)
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-shared",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"), "-o", str(pkg / "libllmig.so"),
           os.path.join(PKG, "csrc", "llmig.hip")]
    build = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert build.returncode == 0, build.stderr[-3000:]
    files = [os.path.join(TESTS, f) for f in ("test_host.py", "test_coordinator.py", "test_properties.py",
                                              "test_migrate_records.py")]
    code = (f"import sys; sys.path.insert(0, {str(tmp_path)!r}); sys.path.insert(1, {ROOT!r}); "
            f"sys.path.insert(2, {TESTS!r})\n"
            "import paper_2406_03243_amd.llmig as m\n"
            f"assert m.LIBRARY.startswith({str(tmp_path)!r}), m.LIBRARY\n"
            "import pytest\n"
            # the plain-C client test links the library with gcc, which cannot resolve the ASan runtime
            f"sys.exit(pytest.main(['-q', '-x', '-p', 'no:cacheprovider', '-m', 'not gpu', '-k', "
            f"'not test_header_is_plain_c', *{files!r}]))\n")
    res = _run(code, CLANG_ASAN[-1], 900)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in out


@pytest.mark.skipif(shutil.which("gcc") is None or _gcc_runtime("libasan.so") is None,
                    reason="gcc or its ASan runtime missing")
def test_oracle_under_sanitizers(tmp_path):
    lib = tmp_path / "liboracle_san.so"
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-shared", "-fPIC", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-o", str(lib),
           os.path.join(ROOT, "oracle", "llmig_oracle.c"), "-lm"]
    build = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert build.returncode == 0, build.stderr[-3000:]
    code = (f"import sys; sys.path[:0] = [{ROOT!r}, {TESTS!r}]\n"
            "import pins\n"
            "from oracle import Oracle\n"
            f"orc = Oracle({str(lib)!r})\n"
            "for pin in pins.ALL_PINS:\n"
            "    pin(orc)\n"
            "print('pins passed:', len(pins.ALL_PINS))\n")
    preload = " ".join(p for p in (_gcc_runtime("libasan.so"), _gcc_runtime("libubsan.so")) if p)
    res = _run(code, preload, 900)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert "pins passed:" in out
