"""A multi-layer decode loop (NEXT-4, weight-free): the first call of every
layer has an empty suffix, each step appends the generated row of every
(b, kv), and every step of every layer is checked against the oracle with
the suffix rows generated so far (paragraph "Cache state and budget"; the
exact suffix E of Alg. "SANTA++ attention for one query head")."""
from collections import Counter

import numpy as np
import pytest
import torch

import datagen
import oracle
from paper_2609_35629_amd.decode_loop import DecodeLoop
from tests.gpu_util import compare_step, log, oracle_teams, to_dev
import paper_2609_35629_amd as sp

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dense", [False, True])
def test_decode_loop_two_layers_64_steps(dense):
    steps, layers = 64, 2
    wl = datagen.WORKLOADS["qwen8k"]
    trace = datagen.decode_trace(wl, layers, steps)
    log(f"[gpu] decode loop: {layers} layers x {steps} steps, {wl.name}, dense={dense}")
    prompts = [(to_dev(b.K, wl.dtype), to_dev(b.V, wl.dtype)) for b, _ in trace]
    loop = DecodeLoop(prompts, capacity=steps, Hq=wl.Hq, budget=wl.K, P=wl.P, R=wl.R, seed=wl.seed, dense=dense)
    rows = [(to_dev(b.sK, wl.dtype), to_dev(b.sV, wl.dtype)) for b, _ in trace]  # [B, Hkv, steps, d]
    qdev = [torch.from_numpy(qs).cuda() for _, qs in trace]
    ot = [oracle_teams(b) for b, _ in trace]
    x64 = [[b.f64(x) for x in (b.K, b.V, b.sK, b.sV)] for b, _ in trace]
    M = None if dense else loop.layers[0].teams.M
    dbgs = None if dense else [sp.DebugOut(wl.B, wl.Hq, wl.Hkv, M, wl.K) for _ in range(layers)]
    tot = Counter()
    worst = 0.0
    for t in range(steps):
        assert all(layer.T == t for layer in loop.layers)
        outs = loop.step([q[t] for q in qdev], [r[0][:, :, t] for r in rows], [r[1][:, :, t] for r in rows],
                         scale=wl.scale, debugs=dbgs)
        torch.cuda.synchronize()
        for li, (b, qs) in enumerate(trace):
            K64, V64, sK64, sV64 = x64[li]
            got = outs[li].cpu().numpy()
            assert np.isfinite(got).all()
            if dense:
                want = oracle.dense(qs[t], K64, V64, sK64[:, :, :t], sV64[:, :, :t], wl.scale)
                rel = max(oracle.rel_l2(got[bi, h], want[bi, h]) for bi in range(wl.B) for h in range(wl.Hq))
                assert rel <= 1e-4, (t, li, rel)
                worst = max(worst, rel)
                continue
            so = oracle.decode(qs[t], K64, V64, sK64[:, :, :t], sV64[:, :, :t], ot[li], wl.K, wl.seed + li, t,
                               wl.scale)
            pairs = [(bi, h) for bi in range(wl.B) for h in range(wl.Hq)]
            cmp = compare_step(wl, wl.K, got, dbgs[li], so, pairs, True)
            assert not cmp.unexcused, (t, li, cmp.unexcused)
            assert cmp.rel_l2.max() <= 1e-2
            if cmp.equal.any():
                assert cmp.rel_l2_equal.max() <= 1e-4, (t, li)
            assert cmp.max_logc_abs <= 1e-5
            tot.update(heads=cmp.heads, equal=cmp.sel_equal, excused=cmp.excused)
            worst = max(worst, float(cmp.rel_l2.max()))
    assert all(layer.T == steps for layer in loop.layers)
    if not dense:
        assert tot["equal"] >= int(np.ceil(0.999 * tot["heads"])), tot
    log(f"[gpu]   layer-steps={layers * steps} instances={tot['heads']} equal={tot['equal']} "
        f"excused={tot['excused']} worst rel-L2={worst:.3e}")
    with pytest.raises(ValueError):
        loop.layers[0].append(rows[0][0][:, :, 0], rows[0][1][:, :, 0])  # the cache holds `steps` rows
    loop.close()
