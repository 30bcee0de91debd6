"""Pins of the oracle's centroid routing keys and KL routing diagnostic
(section "Attention-distribution diagnostic"; appendix "Dense-trajectory KL
and task-variant evaluation", eq. diagnostic-kl)."""
import math

import numpy as np
import pytest

import oracle


def _bf16_grid():
    """Every finite bf16 value, ascending, with its bit pattern."""
    bits = np.arange(1 << 16, dtype=np.uint32) << 16
    with np.errstate(invalid="ignore"):
        v = bits.view(np.float32).astype(np.float64)
    ok = np.isfinite(v)
    v, b = v[ok], (bits[ok] >> 16)
    order = np.argsort(v, kind="stable")
    v, b = v[order], b[order]
    keep = np.concatenate([[True], np.diff(v) > 0])  # +0 and -0 collapse
    return v[keep], b[keep]


def test_round_to_bf16_hand_cases():
    one = 1.0
    cases = {
        one: one,
        one + 2 ** -8: one,                        # halfway, the even neighbour is 1
        one + 3 * 2 ** -8: one + 2 ** -6,          # halfway, the even neighbour is above
        one + 2 ** -8 + 2 ** -30: one + 2 ** -7,   # just above halfway
        -(one + 2 ** -8): -one,
        2.0 ** -133: 2.0 ** -133,                  # smallest bf16 subnormal
        2.0 ** -135: 0.0,                          # below half of it
        3.0e38: float(np.array([0x7F62_0000], np.uint32).view(np.float32)[0]),
        3.4e38: math.inf,                          # beyond bf16's largest value
    }
    got = oracle.round_to_bf16(np.array(list(cases.keys())))
    np.testing.assert_array_equal(got, np.array(list(cases.values())))
    assert np.isnan(oracle.round_to_bf16(np.array([np.nan])))[0]


def test_round_to_bf16_matches_brute_force_nearest():
    grid, bits = _bf16_grid()
    rng = np.random.default_rng(7)
    x = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
        # exact midpoints between neighbours, where the tie rule decides
        (grid[1000:1200] + grid[1001:1201]) / 2,
        (grid[-300:-250] + grid[-299:-249]) / 2,
    ])
    got = oracle.round_to_bf16(x)
    for xi, gi in zip(x, got):
        j = np.searchsorted(grid, xi)
        cands = [c for c in (j - 1, j) if 0 <= c < len(grid)]
        dist = [abs(grid[c] - xi) for c in cands]
        best = [c for c, dd in zip(cands, dist) if dd == min(dist)]
        if len(best) > 1:
            best = [c for c in best if bits[c] & 1 == 0]
        assert gi == grid[best[0]], (xi, gi, grid[best[0]])


def test_team_means_hand_and_identical_rows():
    K = np.array([[1.0, 2.0], [3.0, 4.0], [5.0, 9.0], [7.0, -1.0]])
    teams = oracle.Teams(members=np.array([0, 1, 2, 3], np.int32),
                         team_ptr=np.array([0, 3, 4], np.int32),
                         rep_token=np.array([1, 3], np.int32))
    np.testing.assert_array_equal(oracle.team_means(K, teams), [[3.0, 5.0], [7.0, -1.0]])
    row = np.array([0.1, -2.7, 3.3])
    Kd = np.tile(row, (5, 1))
    t1 = oracle.Teams(np.arange(5, dtype=np.int32), np.array([0, 5], np.int32), np.array([2], np.int32))
    np.testing.assert_array_equal(oracle.team_means(Kd, t1)[0], row)


def test_team_means_close_to_numpy_mean():
    rng = np.random.default_rng(3)
    K = rng.standard_normal((600, 32))
    teams = oracle.build_teams(K, 200, 5)
    m = oracle.team_means(K, teams)
    for g in range(teams.M):
        mem = teams.members[teams.team_ptr[g]:teams.team_ptr[g + 1]]
        np.testing.assert_allclose(m[g], K[mem].mean(axis=0), rtol=0, atol=1e-14)


def _case(N=256, d=16, seed=0, spread=2.0):
    rng = np.random.default_rng(seed)
    K = rng.standard_normal((N, d)) * spread
    q = rng.standard_normal(d)
    return q, K


def test_kl_zero_when_every_key_is_a_team():
    # P = R = 1: one token per team, its own key routes it, so q equals p
    q, K = _case()
    teams = oracle.build_teams(K, 1, 1)
    keys = oracle.routing_keys(K, teams, "representative", "fp32")
    kl = oracle.routing_kl(q, K, teams, keys, 0.25)
    assert abs(kl) < 1e-12
    # the team mean of a one-token team is the token's key: zero as well
    keys_c = oracle.team_means(K, teams)
    assert abs(oracle.routing_kl(q, K, teams, keys_c, 0.25)) < 1e-12


def test_kl_one_group_is_log_n_minus_entropy():
    # one group covering every token: q is uniform, KL(p || 1/N) = log N - H(p)
    q, K = _case(N=300)
    teams = oracle.build_teams(K, 300, 1)
    assert teams.M == 1
    scale = 0.3
    s = scale * (K @ q)
    p = np.exp(s - s.max())
    p /= p.sum()
    H = -float(np.sum(p * np.log(p)))
    for kind in ("representative", "centroid"):
        keys = oracle.routing_keys(K, teams, kind, "fp32")
        kl = oracle.routing_kl(q, K, teams, keys, scale)
        assert abs(kl - (math.log(300) - H)) < 1e-12


@pytest.mark.parametrize("P,R", [(16, 4), (64, 8), (4, 1), (16, 1)])
def test_kl_is_nonnegative(P, R):
    for seed in range(3):
        q, K = _case(N=512, seed=seed)
        teams = oracle.build_teams(K, P, R)
        for kind in ("representative", "centroid"):
            keys = oracle.routing_keys(K, teams, kind, "bf16")
            assert oracle.routing_kl(q, K, teams, keys, 0.25) >= -1e-12


def test_decode_with_explicit_representative_keys_is_unchanged():
    q, K = _case(N=512, d=16, seed=5)
    rng = np.random.default_rng(5)
    V = rng.standard_normal(K.shape)
    teams = oracle.build_teams(K, 64, 4)
    keys = oracle.routing_keys(K, teams, "representative", "fp32")
    sK = np.zeros((0, 16))
    a = oracle.decode_head(q, K, V, teams, sK, sK, 5, 11, 3, 0, 2, 0.25)
    b = oracle.decode_head(q, K, V, teams, sK, sK, 5, 11, 3, 0, 2, 0.25, route_keys=keys)
    np.testing.assert_array_equal(a.out, b.out)
    np.testing.assert_array_equal(a.sel, b.sel)
    # centroid keys change the routing logits by the team means' scores
    c = oracle.decode_head(q, K, V, teams, sK, sK, 5, 11, 3, 0, 2, 0.25,
                           route_keys=oracle.team_means(K, teams))
    np.testing.assert_allclose(c.phi, np.log(teams.sizes) + 0.25 * (oracle.team_means(K, teams) @ q),
                               rtol=1e-13, atol=1e-13)
