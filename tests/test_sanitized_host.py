"""The boundary's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

Builds libproxyattn_san.so (host code instrumented, device code as usual) and
runs the host-only boundary tests (test_abi_host.py: exports, struct layout,
problem validation, work-order settings, workspace and blocked-copy sizes,
argument rejection before launch, binding checks) against it in a process
that preloads the ASan runtime.  Any ASan report or UBSan finding aborts that
process and fails this test.  No GPU is needed: every call these tests make
returns before any HIP call.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_boundary_host_code_under_asan_and_ubsan():
    from paper_2509_24745_amd import build as B
    try:
        B.build_sanitized(verbose=False)
    except (OSError, RuntimeError) as e:
        pytest.skip(f"sanitized build unavailable: {e}")
    out = subprocess.run(["nm", "-D", "--undefined-only", B.LIB_SAN], capture_output=True,
                         text=True, check=True).stdout
    assert "__asan_" in out and "__ubsan_" in out, "the library is not instrumented"
    env = B.sanitizer_env()
    probe = ("import paper_2509_24745_amd.proxyattn as pa; pa.lib(); "
             "maps = open('/proc/self/maps').read(); "
             "assert pa.LIB_PATH.endswith('libproxyattn_san.so'), pa.LIB_PATH; "
             "assert 'libproxyattn_san.so' in maps and 'libclang_rt.asan' in maps; print('ok')")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "tests/test_abi_host.py", "-q",
                        "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert "passed" in r.stdout and "failed" not in r.stdout
