"""The host side of the C ABI under AddressSanitizer and UndefinedBehaviorSanitizer.

Builds the library with abi.cpp's host code instrumented (build.build_sanitized;
device code is not), then runs every host-side ABI test (tests/test_abi_host.py:
argument checks, error codes, plans, workspace queries, exports) against it in
a child process with the ASan runtime preloaded.  Any sanitizer report halts
the child with a non-zero status.  No GPU is needed: every call in those tests
returns before the first HIP call.
"""

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_abi_under_asan_and_ubsan():
    sys.path.insert(0, ROOT)
    from paper_2509_26538_amd import build
    lib = build.build_sanitized()
    rt = build.sanitizer_runtime()
    assert os.path.exists(rt), rt
    env = dict(os.environ, HILBERTA_LIB=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # the child loads the sanitized build (it would not load without the
    # preloaded runtime: its __asan_* symbols are undefined)
    probe = ("import sys; sys.path.insert(0, %r); from paper_2509_26538_amd import hilberta as hb; hb.load(); "
             "print([l.split()[-1] for l in open('/proc/self/maps') if 'libhilberta' in l][0])" % ROOT)
    r = subprocess.run([sys.executable, "-c", probe], env=env, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr[-2000:]
    assert r.stdout.strip() == lib, r.stdout
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(ROOT, "tests", "test_abi_host.py")],
                       env=env, capture_output=True, text=True, timeout=300, cwd=ROOT)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-3000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-3000:]
