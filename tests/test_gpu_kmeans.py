"""GPU parity of the k-means parents (Alg. "Global minibatch k-means parent
partition"), of team tables built from label-defined parents, and of decoding
with such tables, all through the C ABI against the CPU oracle.

Bars: labels and steps run bit-exact (every nearest-center decision and the
stopping step are taken in fp64 on both sides; sums over many points may
differ in the last bits, which moves no decision here); team tables bit-exact,
absent teams empty; decode outputs within the relative L2 bar of the other
decode tests, selections equal on the real teams up to near-ties.
"""
import numpy as np
import pytest
import torch

import datagen
import oracle
import paper_2609_35629_amd as sp
from tests.gpu_util import dev_batch, log

pytestmark = pytest.mark.gpu

REL_BAR = 1e-2

CASES = {
    # bf16 d = 128, eight parents, batch not a multiple of the 64-point tile
    "bf16_d128": dict(base="qwen8k", N=3000, Hq=8, Hkv=2, P=375, batch=300, max_iter=20),
    # fp32 d = 64, two sequences, batch of 512
    "fp32_d64": dict(base="tiny", N=2500, B=2, Hq=2, Hkv=1, P=250, batch=512, max_iter=30, data_seeds=(0, 5)),
}


def _workload(c):
    kw = {k: v for k, v in c.items() if k not in ("base", "batch", "max_iter")}
    return datagen.WORKLOADS[c["base"]].with_(**kw)


def _theta(c):
    return oracle.KMeansSettings(batch=c["batch"], max_iter=c["max_iter"])


@pytest.mark.parametrize("name", sorted(CASES))
def test_kmeans_labels_match_oracle(name):
    c = CASES[name]
    wl = _workload(c)
    log(f"[gpu] kmeans {name}: B={wl.B} Hkv={wl.Hkv} N={wl.N} d={wl.d} P={wl.P}")
    b = datagen.generate(wl)
    db = dev_batch(b)
    th = _theta(c)
    labels, mp, steps = sp.kmeans_parents(db.K, wl.P, batch_size=th.batch, max_iter=th.max_iter)
    torch.cuda.synchronize()
    labels = labels.cpu().numpy()
    assert mp == oracle.kmeans_parent_count(wl.N, wl.P)
    for bi in range(wl.B):
        for kv in range(wl.Hkv):
            r = oracle.kmeans_parents(b.f64(b.K[bi, kv]), wl.P, th)
            log(f"[gpu]   b={bi} kv={kv} steps gpu={steps[bi * wl.Hkv + kv]} oracle={r.steps}")
            assert steps[bi * wl.Hkv + kv] == r.steps
            np.testing.assert_array_equal(labels[bi, kv], r.labels, err_msg=f"labels b={bi} kv={kv}")


def test_kmeans_reassignment_and_no_early_stop():
    """Reassignment exercised (many centers, small batch) and the stopping rule
    off: the full step count runs."""
    wl = datagen.WORKLOADS["qwen8k"].with_(N=2048, Hq=4, Hkv=1, P=32)
    b = datagen.generate(wl)
    db = dev_batch(b)
    th = oracle.KMeansSettings(batch=64, max_iter=3, max_no_improvement=0, reassignment_ratio=0.2)
    labels, mp, steps = sp.kmeans_parents(db.K, wl.P, batch_size=64, max_iter=3, max_no_improvement=0,
                                          reassignment_ratio=0.2)
    r = oracle.kmeans_parents(b.f64(b.K[0, 0]), wl.P, th)
    assert mp == 64 and steps[0] == r.steps == 3 * 2048 // 64
    np.testing.assert_array_equal(labels.cpu().numpy()[0, 0], r.labels)


def _labels_with_gaps(wl, seed):
    rng = np.random.default_rng(seed)
    lab = rng.integers(0, 12, size=(wl.B, wl.Hkv, wl.N)).astype(np.int32)
    lab[lab == 3] = 4            # label 3 empty everywhere
    lab[0, 0][lab[0, 0] == 7] = 8  # and label 7 empty in one pair only
    lab[0, 0, :5] = 11           # a parent smaller than R in that pair
    lab[0, 0, 5:][lab[0, 0, 5:] == 11] = 10
    return lab


@pytest.mark.parametrize("dtype_base", ["qwen8k", "tiny"])
def test_tables_from_labels_match_oracle(dtype_base):
    wl = datagen.WORKLOADS[dtype_base].with_(N=1500, B=1, Hq=4, Hkv=2, R=8)
    b = datagen.generate(wl)
    db = dev_batch(b)
    lab = _labels_with_gaps(wl, 1)
    log(f"[gpu] tables from labels base={dtype_base}")
    teams = sp.build_teams_from_labels(db.K, db.V, torch.from_numpy(lab).cuda(), 12, wl.R)
    torch.cuda.synchronize()
    perm, tb, ts, rt = (teams.perm().cpu().numpy(), teams.team_begin().cpu().numpy(),
                        teams.team_size().cpu().numpy(), teams.rep_token().cpu().numpy())
    tc = teams.team_count().cpu().numpy()
    Mmax = 0
    for kv in range(wl.Hkv):
        t = oracle.build_teams_from_labels(b.f64(b.K[0, kv]), lab[0, kv], wl.R)
        Mmax = max(Mmax, t.M)
        assert tc[0, kv] == t.M
        np.testing.assert_array_equal(perm[0, kv], t.members)
        np.testing.assert_array_equal(tb[0, kv, :t.M], t.team_ptr[:-1])
        np.testing.assert_array_equal(ts[0, kv, :t.M], t.sizes)
        np.testing.assert_array_equal(rt[0, kv, :t.M], t.rep_token)
        assert (ts[0, kv, t.M:] == 0).all() and (tb[0, kv, t.M:] == wl.N).all()
    assert teams.M == Mmax
    assert tc.min() < tc.max()  # the pairs' team counts differ
    pk = teams.packed_K().view(torch.int16 if db.K.dtype == torch.bfloat16 else torch.int32)
    K = db.K.view(pk.dtype)
    for kv in range(wl.Hkv):
        assert torch.equal(pk[0, kv], K[0, kv][torch.from_numpy(perm[0, kv]).long().cuda()])


def test_label_out_of_range_is_rejected():
    wl = datagen.WORKLOADS["tiny"].with_(N=300)
    b = datagen.generate(wl)
    db = dev_batch(b)
    lab = np.zeros((1, 1, 300), np.int32)
    lab[0, 0, 17] = 5
    with pytest.raises(sp.SantappError):
        sp.build_teams_from_labels(db.K, db.V, torch.from_numpy(lab).cuda(), 5, 2)


@pytest.mark.parametrize("Kb", [4, 12])
def test_decode_with_kmeans_tables(Kb):
    """Decode over k-means teams; with K = 12 one pair has at most K real
    teams, so its absent teams are sampled and every real team is taken with
    correction 1."""
    wl = datagen.WORKLOADS["qwen8k"].with_(N=4096, Hq=8, Hkv=2, P=512, R=4, T=32)
    b = datagen.generate(wl)
    db = dev_batch(b)
    th = oracle.KMeansSettings(batch=512, max_iter=10)
    labels, mp, _ = sp.kmeans_parents(db.K, wl.P, batch_size=512, max_iter=10)
    lab = labels.cpu().numpy()
    if Kb == 12:  # force one pair to hold few teams: two parents only
        lab[0, 1] = lab[0, 1] % 2
        labels = torch.from_numpy(lab).cuda()
    teams = sp.build_teams_from_labels(db.K, db.V, labels, mp, wl.R)
    ot = [[oracle.build_teams_from_labels(b.f64(b.K[0, kv]), lab[0, kv], wl.R) for kv in range(wl.Hkv)]]
    for kv in range(wl.Hkv):
        if Kb == 4:
            r = oracle.kmeans_parents(b.f64(b.K[0, kv]), wl.P, th)
            np.testing.assert_array_equal(lab[0, kv], r.labels)
    tc = teams.team_count().cpu().numpy()
    log(f"[gpu] decode kmeans K={Kb} team counts={tc.tolist()} M={teams.M}")
    ws = sp.decode_workspace(teams, wl.Hq, wl.T, Kb)
    dbg = sp.DebugOut(wl.B, wl.Hq, wl.Hkv, teams.M, min(Kb, teams.M)) if Kb < teams.M else None
    out = sp.decode(teams, db.q, db.sK, db.sV, Kb, seed=wl.seed, step=0, scale=wl.scale, workspace=ws,
                    debug=dbg)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    assert np.isfinite(out).all()
    so = oracle.decode(b.q, b.f32(b.K), b.f32(b.V), b.f32(b.sK), b.f32(b.sV), ot, Kb, wl.seed, 0, wl.scale)
    sel = dbg.sel.cpu().numpy() if dbg is not None else None
    for h in range(wl.Hq):
        r = so.heads[0][h]
        kv = h // wl.G
        rel = oracle.rel_l2(out[0, h], r.out)
        assert rel <= REL_BAR, (h, rel)
        if sel is not None:
            real = np.sort(sel[0, h][sel[0, h] < tc[0, kv]])
            if not np.array_equal(real, r.sel):
                ys = np.sort(r.Y)[::-1]
                gap = ys[Kb - 1] - ys[Kb] if len(ys) > Kb else np.inf
                assert gap <= 1e-6 * max(1.0, abs(r.tau)), (h, real, r.sel)
        if tc[0, kv] <= Kb:  # every real team taken: the exact attention
            assert len(r.sel) == tc[0, kv]


def test_kmeans_full_size_headline_layer():
    """The 32768-token layer the benchmark times (4 KV heads, d = 128, bf16,
    P = 1024, the paper's settings): labels, steps run and the team table of
    two of the pairs against the oracle, element by element."""
    wl = datagen.WORKLOADS["qwen32k"]
    b = datagen.generate(wl)
    db = dev_batch(b)
    log("[gpu] kmeans full size qwen32k")
    labels, mp, steps = sp.kmeans_parents(db.K, wl.P)
    teams = sp.build_teams_from_labels(db.K, db.V, labels, mp, wl.R)
    torch.cuda.synchronize()
    lab = labels.cpu().numpy()
    perm, tb, ts, rt = (teams.perm().cpu().numpy(), teams.team_begin().cpu().numpy(),
                        teams.team_size().cpu().numpy(), teams.rep_token().cpu().numpy())
    tc = teams.team_count().cpu().numpy()
    for kv in (0, 3):
        r = oracle.kmeans_parents(b.f64(b.K[0, kv]), wl.P)
        log(f"[gpu]   kv={kv} steps gpu={steps[kv]} oracle={r.steps}")
        assert steps[kv] == r.steps
        np.testing.assert_array_equal(lab[0, kv], r.labels)
        t = oracle.build_teams_from_labels(b.f64(b.K[0, kv]), r.labels, wl.R)
        assert tc[0, kv] == t.M
        np.testing.assert_array_equal(perm[0, kv], t.members)
        np.testing.assert_array_equal(tb[0, kv, :t.M], t.team_ptr[:-1])
        np.testing.assert_array_equal(ts[0, kv, :t.M], t.sizes)
        np.testing.assert_array_equal(rt[0, kv, :t.M], t.rep_token)
