"""Pins for the oracle's team construction.

Follows the paper's Alg. "Contiguous parent partition" and Alg. "Build
actual-key teams from a parent partition" (section "Preparing parent groups
and teams"; paragraph "Shared team construction" fixes the tie rules).  The
paper prints no worked build, so the pins are hand-worked cases
(tests/golden/build_hand_cases.txt), an independent brute-force restatement on
small random inputs, and the algorithm's invariants.
"""
import os

import numpy as np
import pytest

import datagen
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "build_hand_cases.txt")


def _cases():
    out = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, pr, keys, teams = [x.strip() for x in line.split("|")]
            P, R = (int(x) for x in pr.split())
            K = np.array([[float(c) for c in row.split(",")] for row in keys.split(";")])
            want = []
            for t in teams.split(";"):
                mem, rep = [], None
                for tok in t.split():
                    if tok.startswith("["):
                        rep = int(tok.strip("[]"))
                        mem.append(rep)
                    else:
                        mem.append(int(tok))
                want.append((sorted(mem), rep))
            out.append((name, P, R, K, want))
    return out


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c[0])
def test_hand_cases(case):
    name, P, R, K, want = case
    t = oracle.build_teams(K, P, R)
    got = [(sorted(t.members[t.team_ptr[g]:t.team_ptr[g + 1]].tolist()), int(t.rep_token[g]))
           for g in range(t.M)]
    assert got == want


def brute_force_teams(K, P, R):
    """Alg. 2 on contiguous parents restated directly with numpy: full
    distance matrices, argmin/argmax taking the first (lowest) index."""
    N = K.shape[0]
    teams = []
    for start in range(0, N, P):
        idx = np.arange(start, min(start + P, N))
        X = K[idx]
        r = min(R, len(idx))
        mu = X.mean(axis=0)
        reps = [int(np.argmin(((X - mu) ** 2).sum(axis=1)))]
        D = ((X[:, None, :] - X[None, :, :]) ** 2).sum(axis=2)
        while len(reps) < r:
            near = D[:, reps].min(axis=1)
            near[reps] = -np.inf
            reps.append(int(np.argmax(near)))
        owner = np.argmin(D[:, reps], axis=1)
        for u, j in enumerate(reps):
            owner[j] = u
        for u, j in enumerate(reps):
            teams.append((idx[owner == u].tolist(), int(idx[j])))
    return teams


@pytest.mark.parametrize("seed,N,d,P,R", [(0, 40, 3, 10, 4), (1, 57, 5, 8, 3), (2, 64, 8, 16, 16),
                                          (3, 33, 2, 33, 5), (4, 20, 4, 1, 1), (5, 50, 6, 7, 9)])
def test_matches_brute_force(seed, N, d, P, R):
    rng = np.random.default_rng(seed)
    K = rng.standard_normal((N, d))
    t = oracle.build_teams(K, P, R)
    got = [(t.members[t.team_ptr[g]:t.team_ptr[g + 1]].tolist(), int(t.rep_token[g])) for g in range(t.M)]
    assert got == brute_force_teams(K, P, R)


def test_invariants_on_workload_keys():
    b = datagen.get("qwen8k")
    K = b.f64(b.K[0, 1])
    P, R = 1024, 16
    t = oracle.build_teams(K, P, R)
    N = K.shape[0]
    assert t.M == (N // P) * R
    # the teams partition [0, N) and none is empty
    assert sorted(t.members.tolist()) == list(range(N))
    assert (t.sizes >= 1).all()
    for g in range(t.M):
        mem = t.members[t.team_ptr[g]:t.team_ptr[g + 1]]
        assert (np.diff(mem) > 0).all()
        assert t.rep_token[g] in mem
        # every member lies in the representative's parent
        assert (mem // P == t.rep_token[g] // P).all()
    # nearest-representative property within each parent
    for p in range(N // P):
        reps = t.rep_token[p * R:(p + 1) * R]
        L = K[reps]
        for u in range(R):
            g = p * R + u
            mem = t.members[t.team_ptr[g]:t.team_ptr[g + 1]]
            dd = ((K[mem][:, None, :] - L[None, :, :]) ** 2).sum(axis=2)
            mine = dd[:, u]
            assert (mine <= dd.min(axis=1) * (1 + 1e-12) + 1e-12).all()
    # the first representative of each parent is the member nearest the mean
    for p in range(N // P):
        X = K[p * P:(p + 1) * P]
        j1 = p * P + int(np.argmin(((X - X.mean(axis=0)) ** 2).sum(axis=1)))
        assert t.rep_token[p * R] == j1


def test_limiting_case_every_key_its_own_team():
    rng = np.random.default_rng(9)
    K = rng.standard_normal((37, 4))
    t = oracle.build_teams(K, 1, 1)
    assert t.M == 37
    assert t.members.tolist() == list(range(37))
    assert t.rep_token.tolist() == list(range(37))


def test_rejects_bad_arguments():
    with pytest.raises(ValueError):
        oracle.build_teams(np.zeros((4, 2)), 0, 1)
    with pytest.raises(ValueError):
        oracle.build_teams(np.zeros((4, 2)), 2, 0)
