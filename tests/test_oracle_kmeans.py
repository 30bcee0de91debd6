"""Pins of the oracle's k-means parents and its team construction from any
parent partition (Alg. "Global minibatch k-means parent partition" and the
settings that follow it; Alg. "Build actual-key teams from a parent
partition").

Each pin checks the oracle against something other than itself: clusters
known by construction, the running-mean property of the cumulative-count
update recomputed from the drawn minibatches, the nearest-center rule of the
final labels, the behaviour of seeding and reassignment on inputs whose
outcome is forced, the team construction of the already pinned contiguous
builder on each parent's own keys, and the inertia scikit-learn's
MiniBatchKMeans reaches on the same data with the paper's settings.
"""
import numpy as np
import pytest

import oracle

def blobs(rng, centers, per, sigma):
    X = np.concatenate([c + sigma * rng.standard_normal((per, len(c))) for c in centers])
    truth = np.repeat(np.arange(len(centers)), per)
    return X, truth


def same_partition(a, b):
    """True when labels a and b define the same partition (up to renaming)."""
    pairs = set(zip(a.tolist(), b.tolist()))
    return len(pairs) == len(set(a.tolist())) == len(set(b.tolist()))


def batch_indices(seed, step, batch, N):
    """Token indices of a minibatch: Philox4x64-10 (pinned against its
    published answers elsewhere), key (seed, 1), counter (j / 4, 3, step, 0),
    word j mod 4, index floor(w N / 2^64)."""
    out = []
    for j in range(batch):
        w = int(oracle.philox([j >> 2, 3, step, 0], [seed, 1])[j & 3])
        out.append((w * N) >> 64)
    return np.array(out)


def test_parent_count():
    # M_parent = min(N, max(2, floor(N / P)))
    assert oracle.kmeans_parent_count(32768, 1024) == 32
    assert oracle.kmeans_parent_count(100, 1024) == 2
    assert oracle.kmeans_parent_count(2, 1) == 2
    assert oracle.kmeans_parent_count(10, 3) == 3
    assert oracle.kmeans_parent_count(5, 1) == 5
    with pytest.raises(ValueError):
        oracle.kmeans_parent_count(1, 1)


def test_separated_blobs_are_recovered():
    rng = np.random.default_rng(1)
    centers = 20.0 * np.eye(8)[:6]
    X, truth = blobs(rng, centers, 200, 0.3)
    r = oracle.kmeans_parents(X, 200, oracle.KMeansSettings(batch=256))
    assert r.centers.shape == (6, 8)
    assert same_partition(r.labels, truth)
    # every final center sits at its blob's centre
    for u in range(6):
        c = X[r.labels == u].mean(axis=0)
        assert np.linalg.norm(r.centers[u] - c) < 0.2


def test_labels_are_nearest_final_center():
    rng = np.random.default_rng(2)
    X = rng.standard_normal((1500, 12))
    r = oracle.kmeans(X, 15, oracle.KMeansSettings(batch=300))
    d2 = ((X[:, None, :] - r.centers[None, :, :]) ** 2).sum(axis=2)
    assert np.array_equal(r.labels, d2.argmin(axis=1))
    assert r.labels.min() >= 0 and r.labels.max() < 15


@pytest.mark.parametrize("steps", [1, 2, 3])
def test_cumulative_count_update_is_a_running_mean(steps):
    """With reassignment off, after s steps each center equals the mean of
    every minibatch point assigned to it so far (or stays at its seed)."""
    rng = np.random.default_rng(3)
    N, d, M, batch, seed = 600, 6, 7, 600, 11
    X = rng.standard_normal((N, d))
    th = oracle.KMeansSettings(batch=batch, max_iter=steps, max_no_improvement=0,
                               reassignment_ratio=0.0, seed=seed)
    r = oracle.kmeans(X, M, th)
    assert r.steps == steps
    C = r.init_centers.copy()
    sums = np.zeros((M, d))
    cnt = np.zeros(M)
    for s in range(steps):
        xb = X[batch_indices(seed, s, batch, N)]
        a = (((xb[:, None, :] - C[None]) ** 2).sum(axis=2)).argmin(axis=1)
        for u in range(M):
            sel = a == u
            if sel.any():
                sums[u] += xb[sel].sum(axis=0)
                cnt[u] += sel.sum()
                C[u] = sums[u] / cnt[u]
    np.testing.assert_allclose(r.centers, C, rtol=1e-12, atol=1e-12)


def test_stopping_rule_follows_the_smoothed_batch_inertia():
    """A second statement of the loop in numpy (reassignment off): the batch
    inertia I_s, its smoothing with alpha = min(1, 2 batch / (N + 1)) and the
    no-improvement count give the same stopping step and centers."""
    rng = np.random.default_rng(12)
    N, d, M, batch, seed, patience = 500, 4, 5, 50, 0, 4
    X = rng.standard_normal((N, d))
    r = oracle.kmeans(X, M, oracle.KMeansSettings(batch=batch, max_iter=20, max_no_improvement=patience,
                                                  reassignment_ratio=0.0, seed=seed))
    C = r.init_centers.copy()
    sums, cnt = np.zeros((M, d)), np.zeros(M)
    alpha = min(1.0, 2.0 * batch / (N + 1.0))
    ewa, best, stale, steps = None, np.inf, 0, 0
    for s in range(20 * N // batch):
        xb = X[batch_indices(seed, s, batch, N)]
        d2 = ((xb[:, None, :] - C[None]) ** 2).sum(axis=2)
        a = d2.argmin(axis=1)
        inert = d2.min(axis=1).mean()
        for u in range(M):
            if (a == u).any():
                sums[u] += xb[a == u].sum(axis=0)
                cnt[u] += (a == u).sum()
                C[u] = sums[u] / cnt[u]
        steps = s + 1
        ewa = inert if ewa is None else ewa * (1 - alpha) + inert * alpha
        if ewa < best:
            best, stale = ewa, 0
        else:
            stale += 1
        if stale >= patience:
            break
    assert steps < 20 * N // batch
    assert r.steps == steps
    np.testing.assert_allclose(r.centers, C, rtol=1e-12, atol=1e-12)


def test_seeding_picks_distinct_points():
    """D^2 sampling never draws a point at distance 0, so the seeds are M
    distinct input points."""
    rng = np.random.default_rng(4)
    X = rng.standard_normal((200, 5))
    r = oracle.kmeans(X, 20, oracle.KMeansSettings(batch=100, max_iter=0))
    assert r.steps == 0
    rows = {tuple(x) for x in X}
    seeds = [tuple(c) for c in r.init_centers]
    assert all(c in rows for c in seeds)
    assert len(set(seeds)) == 20
    # with no steps the final centers are the seeds
    np.testing.assert_array_equal(r.centers, r.init_centers)


def test_seeding_spreads_over_blobs():
    rng = np.random.default_rng(5)
    X, truth = blobs(rng, [np.zeros(4), np.full(4, 50.0)], 100, 0.5)
    for seed in range(5):
        r = oracle.kmeans(X, 2, oracle.KMeansSettings(batch=64, max_iter=0, seed=seed))
        owners = {int(np.argmin(((X - c) ** 2).sum(axis=1))) for c in r.init_centers}
        assert {int(truth[o]) for o in owners} == {0, 1}


def test_reassignment_moves_a_starved_center():
    """Five copies of one far point draw the second seed; they are 0.5 % of
    the data, so that center gets too few points: with the reassignment
    ratio it moves off the far point into the main cloud (the far points,
assigned to it later, pull it only a little way back), without it it stays
there."""
    rng = np.random.default_rng(6)
    X = np.concatenate([rng.standard_normal((1000, 3)), np.tile([[1000.0, 0.0, 0.0]], (5, 1))])
    base = dict(batch=128, max_iter=5, max_no_improvement=0, init_size=3000)
    kept = oracle.kmeans(X, 2, oracle.KMeansSettings(reassignment_ratio=0.0, **base))
    assert np.isclose(kept.init_centers[:, 0], 1000.0).any()
    assert np.isclose(kept.centers[:, 0], 1000.0).any()
    moved = oracle.kmeans(X, 2, oracle.KMeansSettings(reassignment_ratio=0.01, **base))
    assert np.all(np.abs(moved.centers) < 100.0)


def test_stopping_rule():
    rng = np.random.default_rng(7)
    X, _ = blobs(rng, 10.0 * np.eye(6), 300, 0.2)
    full = oracle.kmeans(X, 6, oracle.KMeansSettings(batch=200, max_no_improvement=0))
    assert full.steps == 100 * X.shape[0] // 200
    early = oracle.kmeans(X, 6, oracle.KMeansSettings(batch=200, max_no_improvement=10))
    assert 10 <= early.steps < full.steps


def test_inertia_matches_sklearn_minibatch_kmeans():
    """The library the paper names, with its settings, reaches the same
    within-cluster sum of squares.  Both runs land in the global optimum or in
    a local one depending on their random draws, so the means over 150 seeds
    are compared, and the best runs of both."""
    sk = pytest.importorskip("sklearn.cluster")
    rng = np.random.default_rng(8)
    M, d = 16, 16
    X, _ = blobs(rng, 3.0 * rng.standard_normal((M, d)), 512, 1.0)
    X = X[rng.permutation(len(X))]

    def inertia(labels):
        return sum(((X[labels == u] - X[labels == u].mean(axis=0)) ** 2).sum() for u in np.unique(labels))

    ours, ref = [], []
    for seed in range(150):
        ours.append(inertia(oracle.kmeans(X, M, oracle.KMeansSettings(batch=1024, seed=seed)).labels))
        fit = sk.MiniBatchKMeans(n_clusters=M, batch_size=1024, n_init=1, max_iter=100,
                                 max_no_improvement=10, reassignment_ratio=0.01, tol=0.0,
                                 random_state=seed).fit(X)
        ref.append(inertia(fit.labels_))
    assert np.mean(ours) <= 1.05 * np.mean(ref), (np.mean(ours), np.mean(ref))
    assert min(ours) <= 1.0001 * min(ref)


def test_teams_from_labels_build_each_parent_on_its_own():
    rng = np.random.default_rng(9)
    N, d, R = 700, 8, 5
    K = rng.standard_normal((N, d))
    labels = rng.integers(0, 9, N)
    labels[labels == 4] = 5  # label 4 stays empty
    t = oracle.build_teams_from_labels(K, labels, R)
    g = 0
    for u in range(9):
        idx = np.flatnonzero(labels == u)
        if len(idx) == 0:
            continue
        sub = oracle.build_teams(K[idx], len(idx), R)
        for h in range(sub.M):
            got = t.members[t.team_ptr[g]:t.team_ptr[g + 1]]
            want = idx[sub.members[sub.team_ptr[h]:sub.team_ptr[h + 1]]]
            assert np.array_equal(got, want)
            assert t.rep_token[g] == idx[sub.rep_token[h]]
            g += 1
    assert g == t.M
    assert np.array_equal(np.sort(t.members), np.arange(N))


def test_contiguous_labels_reproduce_contiguous_parents():
    rng = np.random.default_rng(10)
    K = rng.standard_normal((333, 8))
    a = oracle.build_teams(K, 50, 3)
    b = oracle.build_teams_from_labels(K, np.arange(333) // 50, 3)
    assert np.array_equal(a.members, b.members)
    assert np.array_equal(a.team_ptr, b.team_ptr)
    assert np.array_equal(a.rep_token, b.rep_token)


def test_smallest_input():
    X = np.array([[0.0, 1.0], [2.0, 3.0]])
    r = oracle.kmeans_parents(X, 4, oracle.KMeansSettings(batch=4))
    assert sorted(r.labels.tolist()) == [0, 1]
