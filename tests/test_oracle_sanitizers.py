"""The C oracle under AddressSanitizer and UndefinedBehaviorSanitizer (host
code only): an instrumented build runs every oracle entry point on edge
cases in a child process with the ASan runtime preloaded, and any finding
ends it with a non-zero status."""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# every oracle entry point on small edge cases: a ragged last parent, more
# representatives than a parent has members, a one-token prompt, a parent
# longer than the prompt, budgets below, at and beyond the team count, an
# empty suffix, a suffix with no prompt rows, centroid routing keys,
# k-means parents and the teams of their labels
SCRIPT = r"""
import numpy as np
import oracle
rng = np.random.default_rng(5)
keys = lambda n, d: rng.standard_normal((n, d))
for N, d, P, R in ((37, 8, 10, 3), (23, 8, 4, 6), (1, 8, 4, 2), (9, 16, 64, 5)):
    K, V = keys(N, d), keys(N, d)
    t = oracle.build_teams(K, P, R)
    assert t.M >= 1 and int(t.sizes.sum()) == N
    q = rng.standard_normal(d)
    means = oracle.team_means(K, t)
    for T in (0, 3):
        sK, sV = keys(T, d), keys(T, d)
        for Kb in sorted({1, max(1, t.M - 1), t.M, t.M + 3}):
            r = oracle.decode_head(q, K, V, t, sK, sV, Kb, seed=7, step=2, b=0, h=1, scale=0.3)
            assert np.all(np.isfinite(r.out))
            oracle.decode_head(q, K, V, t, sK, sV, Kb, seed=7, step=3, b=0, h=1, scale=0.3,
                               route_keys=means)
        oracle.dense_head(q, K, V, sK, sV, 0.3)
    oracle.philox([1, 2, 3, 4], [5, 6])
    oracle.team_gumbel(1, 2, 0, 1, 3)
oracle.dense_head(rng.standard_normal(8), np.zeros((0, 8)), np.zeros((0, 8)), keys(3, 8), keys(3, 8), 0.3)
X = keys(96, 8)
for ratio in (0.0, 0.5):
    th = oracle.KMeansSettings(batch=16, max_iter=3, max_no_improvement=2, reassignment_ratio=ratio)
    res = oracle.kmeans(X, 4, th)
    t = oracle.build_teams_from_labels(X, res.labels, 3)
    assert int(t.sizes.sum()) == 96
print("sanitized oracle ok")
"""


def _runtime(name):
    out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


def test_oracle_under_asan_and_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None or _runtime("libubsan.so") is None:
        pytest.skip("gcc has no ASan/UBSan runtime here")
    so = oracle.build(out=str(tmp_path / "liboracle_san.so"), sanitize=True)
    env = dict(os.environ, LD_PRELOAD=asan, SANTAPP_ORACLE_LIB=so, PYTHONPATH=ROOT,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-c", SCRIPT], env=env, capture_output=True, text=True,
                       timeout=300, cwd=ROOT)
    assert r.returncode == 0 and "sanitized oracle ok" in r.stdout, r.stdout[-2000:] + r.stderr[-4000:]
