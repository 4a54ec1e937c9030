"""CPU sanitizer tier.

The oracle's C code (built with gcc) and the host side of the C ABI (argument checks, workspace
sizing and the no-allocation entry point's limits in the HIP library, built with host-only
sanitizer flags) are exercised under AddressSanitizer and UndefinedBehaviorSanitizer.  Each suite
runs in a fresh Python process with the matching sanitizer runtime preloaded; a sanitizer report
ends that process with a non-zero status.  A first test plants an overflow and a signed overflow in a
throw-away C file, so a sanitizer set-up that stopped reporting would fail here too.
"""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
pytestmark = pytest.mark.timeout(900)

ASAN_OPTIONS = "detect_leaks=0:halt_on_error=1:abort_on_error=0:exitcode=86"
UBSAN_OPTIONS = "halt_on_error=1:print_stacktrace=1:exitcode=87"


def _gcc_runtime() -> str:
    return subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True,
                          check=True).stdout.strip()


def _env(preload: str, **extra) -> dict:
    env = dict(os.environ)
    env["LD_PRELOAD"] = preload + (":" + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    env["ASAN_OPTIONS"] = ASAN_OPTIONS
    env["UBSAN_OPTIONS"] = UBSAN_OPTIONS
    env["PYTHONDONTWRITEBYTECODE"] = "1"
    env.update(extra)
    return env


def _run(args, env, timeout=600):
    return subprocess.run([sys.executable, *args], cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=timeout)


def _mapped(env, code: str) -> str:
    """Run `code` in a fresh interpreter under `env`, then return its /proc/self/maps."""
    r = _run(["-c", code + "\nprint(open('/proc/self/maps').read())"], env, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    return r.stdout


@pytest.fixture(scope="module")
def gcc_asan():
    if not os.path.exists(_gcc_runtime()):
        pytest.skip("gcc's libasan is not installed")
    return _gcc_runtime()


def test_planted_errors_are_reported(tmp_path, gcc_asan):
    src = tmp_path / "planted.c"
    src.write_text(textwrap.dedent("""
        #include <stdlib.h>
        int read_past_end(int n) { int* a = malloc(n * sizeof(int)); int v = a[n]; free(a); return v; }
        int add_overflow(int a) { return a + 1; }
    """))
    lib = tmp_path / "libplanted.so"
    subprocess.run(["gcc", "-O0", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    "-fPIC", "-shared", "-o", str(lib), str(src)], check=True)
    env = _env(gcc_asan)
    load = f"import ctypes; L = ctypes.CDLL({str(lib)!r}); "
    r = _run(["-c", load + "L.read_past_end(4)"], env)
    assert r.returncode == 86 and "heap-buffer-overflow" in r.stderr, r.stderr[-2000:]
    r = _run(["-c", load + "L.add_overflow(2**31 - 1)"], env)
    assert r.returncode != 0 and "signed integer overflow" in r.stderr, r.stderr[-2000:]
    r = _run(["-c", load + "print(L.add_overflow(41))"], env)
    assert r.returncode == 0 and r.stdout.strip() == "42"


def test_oracle_pins_under_asan_ubsan(tmp_path, gcc_asan):
    import oracle

    lib = oracle.build_sanitized(str(tmp_path / "liboracle_san.so"))
    env = _env(gcc_asan, TACG_ORACLE_LIBRARY=lib)
    maps = _mapped(env, "import oracle, numpy as np; oracle.coact(np.zeros((1, 3, 2), np.int16) + "
                        "np.array([0, 1], np.int16), [0, 3], 4)")
    assert lib in maps and "libasan" in maps
    tests = sorted(os.path.join("tests", f) for f in os.listdir(os.path.join(ROOT, "tests"))
                   if f.startswith("test_oracle_") and f.endswith(".py")) + ["tests/test_golden_comm_trace.py"]
    r = _run(["-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu", *tests], env, timeout=800)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr
    assert " passed" in r.stdout


def test_abi_host_checks_under_asan_ubsan(tmp_path):
    from paper_2606_01007_amd import build as b

    runtime = b.host_asan_runtime()
    if not os.path.exists(runtime):
        pytest.skip("clang's ASan runtime is not installed")
    lib = b.build(sanitize=True, out=str(tmp_path / "libtacg_san.so"))
    env = _env(runtime, TACG_LIBRARY=lib)
    maps = _mapped(env, "import paper_2606_01007_amd as t; t.lib().tacg_strerror(-1)")
    assert lib in maps and "libclang_rt.asan" in maps
    r = _run(["-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu", "tests/test_abi_host.py"],
             env, timeout=600)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr
    assert " passed" in r.stdout and "skipped" not in r.stdout
