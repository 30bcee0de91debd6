"""The library's host entry points under AddressSanitizer and
UndefinedBehaviorSanitizer: a build whose api.hip host code (the entry points
and their argument checks) is instrumented runs the ABI argument checks in a
child process with clang's ASan runtime preloaded; any finding ends it with a
non-zero status.  Device code is not instrumented (no GPU sanitizers here)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/lib/llvm/bin/clang"

CHILD = r"""
import sys
from paper_2609_35629_amd import _lib
_lib.load(sys.argv[1])
import tests.test_abi as T
T.test_budget_rule()
T.test_host_argument_checks()
T.test_kmeans_and_label_table_argument_checks()
print("sanitized api ok")
"""


def _asan_runtime():
    if not os.path.exists(CLANG):
        return None
    out = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                         text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


def test_api_host_checks_under_asan_and_ubsan(tmp_path):
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("clang's ASan runtime is not installed")
    from paper_2609_35629_amd import build as B
    so = B.build_host_sanitized(str(tmp_path / "libsantapp_san.so"))
    env = dict(os.environ, LD_PRELOAD=rt, PYTHONPATH=ROOT,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-c", CHILD, so], env=env, capture_output=True, text=True,
                       timeout=600, cwd=ROOT)
    assert r.returncode == 0 and "sanitized api ok" in r.stdout, r.stdout[-2000:] + r.stderr[-4000:]
