"""Pins for the oracle's decode estimator.

What the paper fixes, and how each is checked here:

* Full budget: with every team selected all corrections are one and the
  output is dense attention (Alg. "SANTA++ attention for one query head",
  first branch; end of paragraph "Unnormalized sums").  Checked against
  softmax attention written out with numpy.
* Unbiasedness of the unnormalised sums (eq. app-unbiased-sums) and the
  per-team identity E[1{g in S} / c_g] = 1 behind it
  (eq. app-conditional-sum with X_g = 1): Monte Carlo over seeds.
* The sampler draws teams without replacement in proportion to the routing
  weights n_g exp(q.l_g / sqrt(d)) (eq. method-routing and the Gumbel-top-K
  paragraph): inclusion frequencies against the exact Plackett-Luce law,
  enumerated by brute force on six teams.
* Limiting case: with one key per team the routing logit is the exact
  attention logit and the first draw follows the exact attention distribution
  (Introduction; SANTA as the limiting case).  Chi-square test.
"""
import itertools
import math

import numpy as np
import pytest
from scipy import stats

import datagen
import oracle


def softmax_attention(q, K, V, scale):
    """Textbook softmax attention over the rows of K, V (fp64)."""
    s = scale * (K @ q)
    w = np.exp(s - s.max())
    return (w[:, None] * V).sum(axis=0) / w.sum()


@pytest.fixture(scope="module")
def tiny():
    b = datagen.get("tiny")
    wl = b.wl
    K = b.f64(b.K)
    V = b.f64(b.V)
    sK = b.f64(b.sK)
    sV = b.f64(b.sV)
    q = b.q.astype(np.float64)
    teams = oracle.build_all(K, wl.P, wl.R)
    return wl, q, K, V, sK, sV, teams


def test_tiny_workload_shape(tiny):
    wl, q, K, V, sK, sV, teams = tiny
    t = teams[0][0]
    assert t.M == 32  # 4 parents of 256 keys, 8 representatives each
    assert t.sizes.sum() == 1024


@pytest.mark.parametrize("Kbudget", [32, 33, 1000])
def test_full_budget_is_dense_attention(tiny, Kbudget):
    wl, q, K, V, sK, sV, teams = tiny
    r = oracle.decode_head(q[0, 0], K[0, 0], V[0, 0], teams[0][0], sK[0, 0], sV[0, 0],
                           Kbudget, 0, 0, 0, 0, wl.scale)
    want = softmax_attention(q[0, 0], np.concatenate([K[0, 0], sK[0, 0]]),
                             np.concatenate([V[0, 0], sV[0, 0]]), wl.scale)
    np.testing.assert_allclose(r.out, want, rtol=1e-12, atol=1e-13)
    assert len(r.sel) == 32 and (r.c == 1.0).all() and r.tau == -np.inf


def test_dense_oracle_is_softmax_attention(tiny):
    wl, q, K, V, sK, sV, teams = tiny
    out = oracle.dense(q, K, V, sK, sV, wl.scale)
    want = softmax_attention(q[0, 0], np.concatenate([K[0, 0], sK[0, 0]]),
                             np.concatenate([V[0, 0], sV[0, 0]]), wl.scale)
    np.testing.assert_allclose(out[0, 0], want, rtol=1e-12, atol=1e-13)
    # no suffix
    out0, _, _, _ = oracle.dense_head(q[0, 0], K[0, 0], V[0, 0], sK[0, 0][:0], sV[0, 0][:0], wl.scale)
    np.testing.assert_allclose(out0, softmax_attention(q[0, 0], K[0, 0], V[0, 0], wl.scale), rtol=1e-12, atol=1e-13)


def test_tiny_sampled_step(tiny):
    wl, q, K, V, sK, sV, teams = tiny
    r = oracle.decode_head(q[0, 0], K[0, 0], V[0, 0], teams[0][0], sK[0, 0], sV[0, 0],
                           wl.K, wl.seed, 0, 0, 0, wl.scale)
    assert len(r.sel) == wl.K
    assert (np.diff(r.sel) > 0).all()
    assert ((r.c > 0) & (r.c <= 1)).all()
    # tau is the (K+1)-th largest perturbed score; selected ones lie above it
    order = np.argsort(-r.Y, kind="stable")
    assert r.tau == r.Y[order[wl.K]]
    assert set(order[:wl.K].tolist()) == set(r.sel.tolist())
    # the routing logit of team g is log n_g + scale q.l_g
    t = teams[0][0]
    phi = np.log(t.sizes) + wl.scale * (K[0, 0][t.rep_token] @ q[0, 0])
    np.testing.assert_allclose(r.phi, phi, rtol=1e-13, atol=1e-13)
    # suffix-free call is legal (first sparse call)
    r0 = oracle.decode_head(q[0, 0], K[0, 0], V[0, 0], t, sK[0, 0][:0], sV[0, 0][:0],
                            wl.K, wl.seed, 0, 0, 0, wl.scale)
    assert np.isfinite(r0.out).all()


def test_budget_must_be_positive(tiny):
    wl, q, K, V, sK, sV, teams = tiny
    with pytest.raises(ValueError):
        oracle.decode_head(q[0, 0], K[0, 0], V[0, 0], teams[0][0], sK[0, 0], sV[0, 0], 0, 0, 0, 0, 0, wl.scale)


# ---------------------------------------------------------------------------
# Statistical pins on a six-team case
# ---------------------------------------------------------------------------
def _six_team_case():
    q, K, V, sK, sV = datagen.small_case(seed=42, N=14, d=4, T=2, logit_scale=1.2)
    q, K, V, sK, sV = q[0, 0], K[0, 0], V[0, 0], sK[0, 0], sV[0, 0]
    teams = oracle.build_teams(K, 5, 2)  # parents of 5, 5, 4 rows -> 6 teams
    assert teams.M == 6
    return q, K, V, sK, sV, teams


def _plackett_luce_inclusion(w, k):
    """Exact Pr(g in S) when k items are drawn without replacement with
    probability proportional to w among the remaining ones."""
    M = len(w)
    pi = np.zeros(M)
    for seq in itertools.permutations(range(M), k):
        p, rest = 1.0, w.sum()
        for g in seq:
            p *= w[g] / rest
            rest -= w[g]
        for g in seq:
            pi[g] += p
    return pi


N_SEEDS = 40000


@pytest.fixture(scope="module")
def six_team_draws():
    q, K, V, sK, sV, teams = _six_team_case()
    scale = 0.5
    k = 2
    incl = np.zeros((N_SEEDS, teams.M))
    ht = np.zeros((N_SEEDS, teams.M))
    Uh = np.zeros((N_SEEDS, K.shape[1]))
    Zh = np.zeros(N_SEEDS)
    for s in range(N_SEEDS):
        r = oracle.decode_head(q, K, V, teams, sK, sV, k, s, 0, 0, 0, scale, ref_shift=0.0)
        incl[s, r.sel] = 1.0
        ht[s, r.sel] = 1.0 / r.c
        Uh[s] = r.U
        Zh[s] = r.Z
    return dict(q=q, K=K, V=V, sK=sK, sV=sV, teams=teams, scale=scale, k=k,
                incl=incl, ht=ht, Uh=Uh, Zh=Zh)


@pytest.mark.slow
def test_inclusion_matches_plackett_luce(six_team_draws):
    D = six_team_draws
    t = D["teams"]
    w = t.sizes * np.exp(D["scale"] * (D["K"][t.rep_token] @ D["q"]))
    pi = _plackett_luce_inclusion(w, D["k"])
    assert abs(pi.sum() - D["k"]) < 1e-12
    freq = D["incl"].mean(axis=0)
    se = np.sqrt(pi * (1 - pi) / N_SEEDS)
    assert (np.abs(freq - pi) < 4.5 * se).all(), (freq, pi)


@pytest.mark.slow
def test_horvitz_thompson_identity(six_team_draws):
    ht = six_team_draws["ht"]
    m = ht.mean(axis=0)
    se = ht.std(axis=0, ddof=1) / math.sqrt(N_SEEDS)
    assert (np.abs(m - 1.0) < 4.5 * se).all(), (m, se)


@pytest.mark.slow
def test_unnormalised_sums_unbiased(six_team_draws):
    D = six_team_draws
    Kall = np.concatenate([D["K"], D["sK"]])
    Vall = np.concatenate([D["V"], D["sV"]])
    e = np.exp(D["scale"] * (Kall @ D["q"]))
    Z = e.sum()
    U = (e[:, None] * Vall).sum(axis=0)
    zm = D["Zh"].mean()
    zse = D["Zh"].std(ddof=1) / math.sqrt(N_SEEDS)
    assert abs(zm - Z) < 4.5 * zse, (zm, Z, zse)
    um = D["Uh"].mean(axis=0)
    use = D["Uh"].std(axis=0, ddof=1) / math.sqrt(N_SEEDS)
    assert (np.abs(um - U) < 4.5 * use).all(), (um, U, use)
    # the estimator really is random here (otherwise the test proves nothing)
    assert zse > 1e-3 * Z


@pytest.mark.slow
def test_limiting_case_first_draw_is_attention():
    q, K, V, sK, sV = datagen.small_case(seed=7, N=16, d=4, T=0, logit_scale=1.0)
    q, K, V = q[0, 0], K[0, 0], V[0, 0]
    teams = oracle.build_teams(K, 1, 1)
    scale = 0.5
    s = scale * (K @ q)
    p = np.exp(s - s.max())
    p /= p.sum()
    n = 50000
    counts = np.zeros(16)
    for seed in range(n):
        r = oracle.decode_head(q, K, V, teams, sK[0, 0][:0], sV[0, 0][:0], 1, seed, 0, 0, 0, scale)
        if seed == 0:
            np.testing.assert_allclose(r.phi, s, rtol=1e-14, atol=1e-14)
        counts[r.sel[0]] += 1
    chi = stats.chisquare(counts, n * p)
    assert chi.pvalue > 1e-4, (counts / n, p)
