"""The C-ABI's host-side code under AddressSanitizer and
UndefinedBehaviorSanitizer: every check of tests/test_abi_cpu.py (validation
before any HIP call, the overlap test on strided lattices, workspace sizes and
their arithmetic, the no-allocation entry point's size check) run against a
build of relation_api.cpp with both sanitizers on the host side, in a process
that preloads the ASan runtime. No GPU is used; no kernel is launched."""
from __future__ import annotations

import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.timeout(900) if hasattr(pytest.mark, "timeout") else []


def test_host_code_under_asan_and_ubsan(tmp_path):
    from paper_2608_20172_amd import build
    if not os.path.exists(os.path.join(ROOT, "paper_2608_20172_amd", "librelation.so")):
        build.build()
    lib = build.build_host_sanitized()
    rt = build.asan_runtime()
    driver = tmp_path / "run_abi_tests.py"
    driver.write_text(textwrap.dedent(f"""
        import sys
        sys.path.insert(0, {ROOT!r})
        import pytest
        from paper_2608_20172_amd import binding as R
        R.load_library({lib!r})  # cached: the tests' load_library() returns this build
        sys.exit(pytest.main([{os.path.join(ROOT, "tests", "test_abi_cpu.py")!r}, "-q", "-p", "no:cacheprovider",
                              "-m", "not gpu"]))
    """))
    env = dict(os.environ)
    env["LD_PRELOAD"] = rt + ((" " + env["LD_PRELOAD"]) if env.get("LD_PRELOAD") else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, str(driver)], env=env, capture_output=True, text=True, timeout=800,
                       cwd=ROOT)
    out = r.stdout + r.stderr
    print(out[-3000:])
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-3000:]
    assert r.returncode == 0, out[-3000:]
    assert " passed" in r.stdout
