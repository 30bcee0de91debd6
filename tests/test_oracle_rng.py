"""Pins for the oracle's counter-based generator and Gumbel noise.

The sampler needs independent standard Gumbel noise per (head, team) at each
decode step (section "Sampling and correcting team contributions"; paragraph
"Conditional inclusion correction" fixes the CDF Pr(G <= x) = exp(-exp(-x))).
The oracle draws it from Philox4x64-10; these tests pin that generator to its
published known-answer vectors and to numpy's independent implementation, and
the Gumbel transform to its CDF.
"""
import math
import os

import numpy as np
import pytest
from scipy import stats

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x64_10_kat.txt")


def _kat_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            w = [int(x, 16) for x in line.split()]
            rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


def test_philox_known_answers():
    rows = _kat_rows()
    assert len(rows) == 3
    for ctr, key, want in rows:
        got = [int(x) for x in oracle.philox(ctr, key)]
        assert got == want


def _numpy_block(ctr, key):
    # numpy's Philox advances its 256-bit counter before producing a block,
    # so the block for counter c comes from a generator started at c - 1.
    c = (sum(int(x) << (64 * i) for i, x in enumerate(ctr)) - 1) % (1 << 256)
    start = np.array([(c >> (64 * i)) & (2**64 - 1) for i in range(4)], dtype=np.uint64)
    bg = np.random.Philox(counter=start, key=np.array(key, dtype=np.uint64))
    return [int(x) for x in bg.random_raw(4)]


def test_philox_matches_numpy():
    rng = np.random.default_rng(123)
    for _ in range(500):
        ctr = [int(x) for x in rng.integers(0, 2**64 - 1, 4, dtype=np.uint64, endpoint=True)]
        key = [int(x) for x in rng.integers(0, 2**64 - 1, 2, dtype=np.uint64, endpoint=True)]
        assert [int(x) for x in oracle.philox(ctr, key)] == _numpy_block(ctr, key)


def test_team_gumbel_counter_layout():
    # team g of head h, sequence b, step t: counter (g // 4, h, b, t), key (seed, 0),
    # output word g % 4
    for (seed, step, b, h, g) in [(0, 0, 0, 0, 0), (7, 3, 2, 27, 513), (2**63 + 5, 99, 7, 13, 8191)]:
        words = _numpy_block([g >> 2, h, b, step], [seed, 0])
        x = words[g & 3]
        u = ((x >> 12) + 0.5) * 2.0**-52
        assert oracle.team_gumbel(seed, step, b, h, g) == pytest.approx(-math.log(-math.log(u)), rel=1e-15, abs=1e-15)


def test_gumbel_extremes_are_finite():
    lo = oracle.gumbel(0)
    hi = oracle.gumbel(2**64 - 1)
    assert math.isfinite(lo) and math.isfinite(hi)
    # U = 2^-53 gives -log(-log U) = -log(53 log 2); U = 1 - 2^-53 gives
    # -log(-log1p(-2^-53)) = 53 log 2 (to fp64 accuracy)
    assert lo == pytest.approx(-math.log(53 * math.log(2.0)), rel=1e-12)
    assert hi == pytest.approx(53 * math.log(2.0), rel=1e-9)


def test_gumbel_law_ks():
    # 2e5 draws over distinct counters against the standard Gumbel CDF
    draws = np.array([oracle.team_gumbel(11, 0, 0, h, g) for h in range(50) for g in range(4000)])
    res = stats.kstest(draws, "gumbel_r")
    assert res.pvalue > 1e-4
    assert abs(draws.mean() - np.euler_gamma) < 4 * math.pi / math.sqrt(6) / math.sqrt(len(draws))
