"""The host tree under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

The library is rebuilt with both sanitizers on its host code (the device code
as usual) into a temporary directory, and the table tests, which run every
tree operation through the C ABI in table-only mode against the oracle, are
run again against it in a child process with the clang ASan runtime
preloaded. Any sanitizer report stops that process with an error.
"""
import os
import shutil
import subprocess
import sys

import pytest

from paper_2402_15220_amd import build as libbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin", "clang")


def _asan_runtime():
    if not os.path.exists(CLANG):
        return None
    r = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                       text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def test_table_tests_under_asan_and_ubsan(tmp_path):
    runtime = _asan_runtime()
    if runtime is None or shutil.which(libbuild.HIPCC) is None and not os.path.exists(libbuild.HIPCC):
        pytest.skip("no clang ASan runtime or hipcc in this image")
    lib = libbuild.build(sanitize=True, lib=str(tmp_path / "libchunkattn_san.so"))
    # the build really carries both sanitizers (their runtime entry points are
    # referenced by the instrumented host code)
    syms = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True).stdout
    assert "__asan_report_load" in syms and "__ubsan_handle_" in syms, syms[:2000]
    env = dict(os.environ)
    env.update(CA_LIBRARY=lib, LD_PRELOAD=runtime,
               # Python's own allocations are not instrumented; leak reports
               # would be about the interpreter
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # The address-space cap of the allocation-failure test cannot work under
    # ASan (its shadow memory is reserved up front), so that test is left out;
    # so are the static-config and segment-length tests, which run the same
    # host code as the random scripts and the replay on bigger trees (a third
    # of the sanitized run's time).
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_tables.py"),
                        "-k", "not host_allocation_failure and not static_configs_bit_exact "
                              "and not automatic_segment_length"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert " passed" in r.stdout and " failed" not in r.stdout, out[-2000:]
