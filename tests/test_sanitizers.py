"""The CPU test-suite again, with the oracle and the library's host layer
(the C ABI: argument validation, workspace layout, launch set-up) built
with AddressSanitizer and UndefinedBehaviorSanitizer.

The oracle is compiled by clang with -fsanitize=address,undefined; api.hip
is compiled by hipcc with the sanitizers on its host pass only (device code
is unchanged) and linked with the regular objects of the other sources.  A
child process preloads clang's shared sanitizer runtime, loads both
instrumented libraries (ILW_ORACLE_LIBRARY, ILW_LIBRARY_PATH) and runs every
`not gpu` test; any report aborts it.  No GPU is needed: the host layer
rejects its inputs or sizes its workspaces before any device call.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.sanitize


def _clang():
    for cand in ("/opt/rocm/llvm/bin/clang", shutil.which("clang")):
        if cand and os.path.exists(cand):
            return cand
    return None


def _undefined_asan_symbols(path):
    out = subprocess.run(["nm", "-D", "--undefined-only", path], capture_output=True,
                         text=True, check=True).stdout
    return [ln.split()[-1] for ln in out.splitlines() if "__asan_report" in ln]


def test_cpu_suite_under_asan_ubsan(tmp_path):
    import oracle
    from paper_2607_24981_amd import build

    clang = _clang()
    try:
        build.hipcc()
        runtime = build.sanitizer_runtime()
    except RuntimeError as e:
        pytest.skip(f"no sanitizer toolchain: {e}")
    if clang is None:
        pytest.skip("no clang for the oracle")

    orc = oracle.build_sanitized(str(tmp_path / "libilw_oracle_san.so"), clang)
    lib = build.build_sanitized(str(tmp_path / "libilw_san.so"))
    # both really are instrumented
    assert _undefined_asan_symbols(orc) and _undefined_asan_symbols(lib)

    env = dict(os.environ)
    env.update(LD_PRELOAD=runtime, ILW_ORACLE_LIBRARY=orc, ILW_LIBRARY_PATH=lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               PYTHONPATH=ROOT)
    # the child loads the instrumented copies, not the regular ones
    probe = ("import oracle; from paper_2607_24981_amd import ilw; oracle.lib(); ilw.lib(); "
             "maps = open('/proc/self/maps').read(); "
             f"assert {orc!r} in maps and {lib!r} in maps, 'instrumented libraries not loaded'")
    r = subprocess.run([sys.executable, "-c", probe], env=env, cwd=ROOT, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr

    r = subprocess.run([sys.executable, "-m", "pytest", "tests", "-x", "-q", "-s",
                        "-p", "no:cacheprovider", "-m", "not gpu and not sanitize"],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=1200)
    log = r.stdout + r.stderr
    assert "runtime error:" not in log and "AddressSanitizer" not in log, log[-6000:]
    assert r.returncode == 0, log[-6000:]
    assert " passed" in log
