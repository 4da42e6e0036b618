"""AddressSanitizer + UBSan runs on the CPU (no GPU needed).

The oracle (``oracle/hill_oracle.c``) and the library's host layer
(``hill_api.cpp``: descriptor validation, workspace layouts, launch set-up)
are built a second time with ``-fsanitize=address,undefined
-fno-sanitize-recover=all`` (clang; host code only), and the oracle's pins and
the ABI's error-path tests run again in a child process that preloads the
sanitizer runtime, so that any out-of-bounds access, use after free or
undefined behaviour in that code aborts the child.  A canary built with the
same flags shows that the harness catches a planted out-of-bounds read.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402


def _runtime():
    try:
        res = subprocess.run([O.CLANG, "-print-resource-dir"], capture_output=True, text=True, check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    hits = sorted(glob.glob(os.path.join(res, "lib", "*", "libclang_rt.asan-x86_64.so")) +
                  glob.glob(os.path.join(res, "lib", "*", "libclang_rt.asan.so")))
    return hits[0] if hits else None


RT = _runtime()
pytestmark = pytest.mark.skipif(RT is None, reason="clang's AddressSanitizer runtime is not installed")


def _env(**extra):
    env = dict(os.environ)
    env.update({"LD_PRELOAD": RT, "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
                "UBSAN_OPTIONS": "print_stacktrace=1", "PYTHONDONTWRITEBYTECODE": "1"})
    env.update(extra)
    return env


def _run(args, env, timeout=900):
    return subprocess.run([sys.executable] + args, cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=timeout)


def test_canary_out_of_bounds_read_is_caught(tmp_path):
    src = tmp_path / "canary.c"
    src.write_text("#include <stdlib.h>\n"
                   "int canary(int i) { int* p = malloc(4 * sizeof(int)); int v = p[i]; free(p); return v; }\n")
    lib = tmp_path / "libcanary.so"
    subprocess.run([O.CLANG, "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-shared",
                    "-fPIC", "-o", str(lib), str(src)], check=True)
    code = "import ctypes; ctypes.CDLL(%r).canary(%d)"
    ok = _run(["-c", code % (str(lib), 1)], _env())
    assert ok.returncode == 0, ok.stderr[-2000:]
    bad = _run(["-c", code % (str(lib), 4)], _env())
    assert bad.returncode != 0 and "heap-buffer-overflow" in bad.stderr


def test_oracle_pins_under_sanitizers():
    lib = O.build(sanitize=True)
    env = _env(HILL_ORACLE_LIB=lib)
    probe = _run(["-c", "from oracle import oracle as O; O._load(); print(open('/proc/self/maps').read())"], env)
    assert probe.returncode == 0, probe.stderr[-2000:]
    assert "libhill_oracle_san.so" in probe.stdout and "libclang_rt.asan" in probe.stdout
    r = _run(["-m", "pytest", "tests/test_oracle.py", "tests/test_app.py", "-x", "-q", "-m", "not gpu",
              "-p", "no:cacheprovider"], env)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert " passed" in r.stdout and "failed" not in r.stdout


def test_abi_error_paths_under_sanitizers():
    from paper_2602_18750_amd import _build
    lib = _build.HOSTSAN_LIB
    srcs = [os.path.join(_build.CSRC, f) for f in os.listdir(_build.CSRC)] + [os.path.join(_build.INCLUDE, "hill.h")]
    if not os.path.exists(lib) or os.path.getmtime(lib) < max(os.path.getmtime(p) for p in srcs):
        if not os.path.exists(_build.LIB):
            pytest.skip("libhill.so is not built")
        _build.build_host_sanitized()
    env = _env(HILL_LIBRARY=lib)
    probe = _run(["-c", "import paper_2602_18750_amd as H; H.load_library(); print(open('/proc/self/maps').read())"],
                 env)
    assert probe.returncode == 0, probe.stderr[-2000:]
    assert "libhill_hostsan.so" in probe.stdout and "libclang_rt.asan" in probe.stdout
    r = _run(["-m", "pytest", "tests/test_abi.py", "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider"], env)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert " passed" in r.stdout and "failed" not in r.stdout
