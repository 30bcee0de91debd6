"""GPU parity of the routing-key variants and the KL routing diagnostic
(section "Attention-distribution diagnostic"; eq. diagnostic-kl) against the
CPU oracle, through the C ABI.

Bars: centroid keys bit-exact (both sides take the fp64 mean in team order
and round it to nearest-even bf16, or to fp32); KL within 1e-9 absolute plus
1e-9 relative (fp64 on both sides, different summation orders); decoding
with centroid keys held to the decode bars of test_gpu_parity."""
import numpy as np
import pytest
import torch

import datagen
import oracle
import paper_2609_35629_amd as sp
from tests.gpu_util import compare_step, dev_batch, gpu_tables, log, oracle_teams

pytestmark = pytest.mark.gpu


def _bits_bf16(vals: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of values that are exact bf16 numbers."""
    return (np.asarray(vals, np.float64).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _oracle_keys(b, ot, kind):
    return [[oracle.routing_keys(b.f64(b.K[bi, kv]), ot[bi][kv], kind, b.wl.dtype)
             for kv in range(b.wl.Hkv)] for bi in range(b.wl.B)]


def _check_keys(teams, b, keys):
    got = teams.reps().cpu()
    for bi in range(b.wl.B):
        for kv in range(b.wl.Hkv):
            if b.wl.dtype == datagen.BF16:
                g = got[bi, kv].view(torch.int16).numpy().view(np.uint16)
                np.testing.assert_array_equal(g, _bits_bf16(keys[bi][kv]), err_msg=f"b={bi} kv={kv}")
            else:
                np.testing.assert_array_equal(got[bi, kv].numpy(), keys[bi][kv].astype(np.float32))


@pytest.mark.parametrize("name", ["qwen8k", "tiny"])
def test_centroid_and_representative_keys(name):
    wl = datagen.WORKLOADS[name]
    log(f"[gpu] route keys {name}")
    b = datagen.generate(wl)
    db = dev_batch(b)
    ot = oracle_teams(b)
    teams = sp.build_teams(db.K, db.V, wl.P, wl.R)
    sp.set_route_keys(teams, "centroid")
    torch.cuda.synchronize()
    _check_keys(teams, b, _oracle_keys(b, ot, "centroid"))
    sp.set_route_keys(teams, "representative")
    torch.cuda.synchronize()
    _check_keys(teams, b, _oracle_keys(b, ot, "representative"))


def test_centroid_rounding_ties():
    # two-token teams (P = 2, R = 1) of bf16 values in [1, 2): the mean of
    # two such values is a rounding tie whenever their sum is odd in the
    # last place, so about half of all key entries exercise ties-to-even
    wl = datagen.WORKLOADS["qwen8k"].with_(name="ties", N=4096, P=2, R=1, Hq=2, Hkv=1)
    b = datagen.generate(wl)
    rng = np.random.default_rng(11)
    mant = rng.integers(0, 128, size=b.K.shape, dtype=np.uint16)
    b.K[...] = np.uint16(0x3F80) | mant  # 1 + m / 128
    log("[gpu] centroid rounding ties")
    db = dev_batch(b)
    ot = oracle_teams(b)
    keys = _oracle_keys(b, ot, "centroid")
    m = oracle.team_means(b.f64(b.K[0, 0]), ot[0][0])
    tie = (oracle.round_to_bf16(m) != m)
    assert tie.mean() > 0.3  # the case really is full of ties
    teams = sp.build_teams(db.K, db.V, wl.P, wl.R)
    sp.set_route_keys(teams, "centroid")
    torch.cuda.synchronize()
    _check_keys(teams, b, keys)


@pytest.mark.parametrize("name", ["qwen8k", "tiny", "limit"])
def test_routing_kl_matches_oracle(name):
    wl = datagen.WORKLOADS[name]
    log(f"[gpu] routing KL {name}")
    b = datagen.generate(wl)
    db = dev_batch(b)
    ot = oracle_teams(b)
    teams = sp.build_teams(db.K, db.V, wl.P, wl.R)
    kinds = ("representative",) if name == "limit" else ("representative", "centroid")
    for kind in kinds:
        sp.set_route_keys(teams, kind)
        kl = sp.routing_kl(teams, db.q, scale=wl.scale)
        torch.cuda.synchronize()
        kl = kl.cpu().numpy()
        keys = _oracle_keys(b, ot, kind)
        for bi in range(wl.B):
            for h in range(wl.Hq):
                kv = h // wl.G
                ref = oracle.routing_kl(b.q[bi, h], b.f64(b.K[bi, kv]), ot[bi][kv], keys[bi][kv], wl.scale)
                assert abs(kl[bi, h] - ref) <= 1e-9 + 1e-9 * abs(ref), (kind, bi, h, kl[bi, h], ref)
        log(f"[gpu]   {kind}: mean KL {kl.mean():.4f} nats")
        if name == "limit":
            # every key its own team: routing equals dense attention
            assert np.abs(kl).max() < 1e-9


def test_decode_with_centroid_keys():
    wl = datagen.WORKLOADS["qwen8k"]
    log("[gpu] decode with centroid routing keys")
    b = datagen.generate(wl)
    db = dev_batch(b)
    ot = oracle_teams(b)
    teams = sp.build_teams(db.K, db.V, wl.P, wl.R)
    sp.set_route_keys(teams, "centroid")
    keys = _oracle_keys(b, ot, "centroid")
    ws = sp.decode_workspace(teams, wl.Hq, wl.T, wl.K)
    dbg = sp.DebugOut(wl.B, wl.Hq, wl.Hkv, teams.M, wl.K)
    out = sp.decode(teams, db.q, db.sK, db.sV, wl.K, seed=wl.seed, step=3, scale=wl.scale, workspace=ws,
                    debug=dbg)
    torch.cuda.synchronize()
    pairs = [(bi, h) for bi in range(wl.B) for h in range(wl.Hq)]
    so = oracle.decode(b.q, b.f32(b.K), b.f32(b.V), b.f32(b.sK), b.f32(b.sV), ot, wl.K, wl.seed, 3,
                       wl.scale, route_keys=keys)
    cmp = compare_step(wl, wl.K, out.cpu().numpy(), dbg, so, pairs, True)
    log(f"[gpu]   sel_equal={cmp.sel_equal}/{cmp.heads} max_rel_l2={cmp.rel_l2.max():.2e} "
        f"max_phi_rel={cmp.max_phi_rel:.1e}")
    assert not cmp.unexcused
    assert cmp.max_phi_rel < 1e-10
    assert cmp.rel_l2.max() <= 1e-2
