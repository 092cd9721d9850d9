"""The ABI tests again, against a build of the host-side sources under
AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

``build.build_sanitized()`` compiles the C-ABI's host code (validation,
workspace layout, launch sequence, error strings) with the sanitizers for the
host only and links it with the regular kernel objects.  tests/test_abi.py
then runs in a child process with clang's sanitizer runtime preloaded (Python
itself is not instrumented) and every finding fatal.  Out-of-range enum values
from C callers, overreads of caller structs, bad format arguments in error
messages and signed overflow in size arithmetic all stop the run.
"""
import os
import subprocess
import sys

import pytest

from paper_2506_12035_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _have_toolchain():
    try:
        build.hipcc()
    except RuntimeError:
        return False
    return build.asan_runtime() is not None


@pytest.mark.skipif(not _have_toolchain(), reason="hipcc or clang's ASan runtime not installed")
def test_abi_under_address_and_undefined_behavior_sanitizers(tmp_path):
    lib = build.build_sanitized()
    nm = subprocess.run(["nm", "-D", lib], capture_output=True, text=True, check=True).stdout
    assert "__asan_report" in nm and "__ubsan_handle" in nm, "sanitizer instrumentation missing"
    log = tmp_path / "san"
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": ":".join(p for p in (build.asan_runtime(), os.environ.get("LD_PRELOAD")) if p),
        # Python and its extensions are not instrumented: their allocations
        # are not ours to judge (leaks at exit, mismatched allocators)
        "ASAN_OPTIONS": f"detect_leaks=0:alloc_dealloc_mismatch=0:verify_asan_link_order=0:"
                        f"halt_on_error=1:log_path={log}",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "MARCHE_LIB_PATH": lib,
    })
    r = subprocess.run([sys.executable, "-m", "pytest", "tests/test_abi.py", "-q", "-p",
                        "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=600)
    reports = "".join(p.read_text() for p in tmp_path.glob("san*"))
    assert r.returncode == 0 and not reports, (r.stdout[-3000:] + r.stderr[-3000:] + reports[:4000])
    assert " passed" in r.stdout
