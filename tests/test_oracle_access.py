"""The oracle's logical-access counter (eq. qwen-logical-access, appendix
"Reference logical-access counter"): per decoding call and KV head, m routing
keys, then one key and one value for each of the u distinct prompt rows the
sharing query heads selected and for each of the e suffix rows, over two
reads per row of the whole cache N.

Pinned on hand-worked cases and on a brute-force recount of the selected
rows of real oracle steps."""
import types

import numpy as np
import pytest

import datagen
import oracle


def _teams(sizes):
    """Teams of the given sizes over tokens 0.. in order (representative:
    each team's first token)."""
    ptr = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    return oracle.Teams(np.arange(ptr[-1], dtype=np.int32), ptr, ptr[:-1].copy())


def _step(sels):
    """A stand-in for a step result: heads[b][h].sel only."""
    return types.SimpleNamespace(heads=[[types.SimpleNamespace(sel=np.array(s, np.int32)) for s in row]
                                        for row in sels])


def test_union_counts_overlap_once():
    t = _teams([3, 5, 2, 7])
    # head A reads teams {0, 2}, head B {2, 3}: team 2's two rows count once
    assert oracle.union_rows(t, [[0, 2], [2, 3]]) == 3 + 2 + 7
    assert oracle.union_rows(t, [[1], [1], [1]]) == 5
    assert oracle.union_rows(t, [[], []]) == 0
    assert oracle.union_rows(t, [[0, 1, 2, 3]]) == 17


def test_access_counts_hand_worked():
    # B = 1, Hkv = 2, G = 2: KV head 0 has teams of 3, 5, 2, 7 rows (N = 17),
    # KV head 1 teams of 4, 4 rows (N = 8); suffix T = 3
    teams = [[_teams([3, 5, 2, 7]), _teams([4, 4])]]
    step = _step([[[0, 2], [2, 3], [1], [0]]])
    # K = 2 < M for both heads' tables: every table is routed (m = M)
    rows = oracle.access_counts(step, teams, Hkv=2, T=3, Kbudget=2)
    assert rows[0] == (4, 12, 3, 20)
    # K = 2 = M of KV head 1: every team taken, no routing pass (m = 0)
    assert rows[1] == (0, 8, 3, 11)
    num = (4 + 2 * (12 + 3)) + (0 + 2 * (8 + 3))
    den = 2 * 20 + 2 * 11
    assert oracle.kv_access_fraction(rows) == pytest.approx(num / den, rel=0, abs=1e-15)
    # a budget above M also takes every team
    rows = oracle.access_counts(_step([[[0, 1, 2, 3], [0, 1, 2, 3], [0, 1], [0, 1]]]), teams, 2, 3, 9)
    assert [r[0] for r in rows] == [0, 0]
    # full budget everywhere and no routing: exactly the dense count
    assert oracle.kv_access_fraction(rows) == 1.0


def test_suffix_counted_once_per_kv_head():
    # the suffix belongs to the KV head, not to each query head: e rows (two
    # reads each) whatever the group size
    for G in (1, 3, 7):
        teams = [[_teams([2, 2, 2])]]
        step = _step([[[0]] * G])
        rows = oracle.access_counts(step, teams, Hkv=1, T=5, Kbudget=1)
        assert rows == [(3, 2, 5, 11)]
        assert oracle.kv_access_fraction(rows) == pytest.approx((3 + 2 * 7) / 22)


def test_counter_matches_a_recount_of_real_steps():
    # the selected rows of oracle steps counted row by row (member lists, not
    # team sizes), on a GQA layout with unequal teams
    wl = datagen.WORKLOADS["qwen8k"].with_(name="acc", N=1500, P=300, R=7, Hq=6, Hkv=2, K=5, T=9)
    b = datagen.generate(wl)
    teams = oracle.build_all(b.f64(b.K), wl.P, wl.R)
    for step_id in (0, 1):
        st = oracle.decode(b.q, b.f64(b.K), b.f64(b.V), b.f64(b.sK), b.f64(b.sV), teams, wl.K, wl.seed,
                           step_id, wl.scale)
        rows = oracle.access_counts(st, teams, wl.Hkv, wl.T, wl.K)
        num = den = 0
        for kv in range(wl.Hkv):
            tm = teams[0][kv]
            read = set()
            for h in range(kv * wl.G, (kv + 1) * wl.G):
                for g in st.heads[0][h].sel:
                    read.update(int(x) for x in tm.members[tm.team_ptr[g]:tm.team_ptr[g + 1]])
            assert rows[kv] == (tm.M, len(read), wl.T, wl.N + wl.T)
            num += tm.M + 2 * (len(read) + wl.T)
            den += 2 * (wl.N + wl.T)
        assert oracle.kv_access_fraction(rows) == pytest.approx(num / den, rel=1e-15)
        assert 0 < oracle.kv_access_fraction(rows) < 1
