"""santapp_decode_static (the entry point for callers that cannot allocate)
against santapp_decode with a workspace of its own: bit-identical outputs and
diagnostics on two calls in a row, the second on a smaller input, and the
size limit of the static scratch."""
import numpy as np
import pytest
import torch

import datagen
import oracle
import paper_2609_35629_amd as sp
from tests.gpu_util import dev_batch, log, oracle_teams

pytestmark = pytest.mark.gpu


def _case(name, **kw):
    wl = datagen.WORKLOADS[name].with_(**kw) if kw else datagen.WORKLOADS[name]
    b = datagen.generate(wl)
    db = dev_batch(b)
    teams = sp.build_teams(db.K, db.V, wl.P, wl.R)
    return wl, b, db, teams


def test_static_scratch_matches_workspace_entry_point():
    # the 32K layer first, then a smaller table and suffix (the scratch keeps
    # the first call's contents; the second must not see them)
    for name, kw, step in (("qwen32k", {}, 11), ("qwen8k", dict(N=4096, T=17, K=20), 3)):
        wl, b, db, teams = _case(name, **kw)
        log(f"[gpu] static scratch: workload={wl.name} N={wl.N} M={teams.M} K={wl.K} T={wl.T} step={step}")
        ws = sp.decode_workspace(teams, wl.Hq, wl.T, wl.K)
        dbg_a = sp.DebugOut(wl.B, wl.Hq, wl.Hkv, teams.M, min(wl.K, teams.M))
        dbg_b = sp.DebugOut(wl.B, wl.Hq, wl.Hkv, teams.M, min(wl.K, teams.M))
        want = sp.decode(teams, db.q, db.sK, db.sV, wl.K, seed=wl.seed, step=step, scale=wl.scale,
                         workspace=ws, debug=dbg_a)
        got = torch.full_like(want, float("nan"))
        sp.decode_static(teams, db.q, db.sK, db.sV, wl.K, got, seed=wl.seed, step=step, scale=wl.scale,
                         debug=dbg_b)
        torch.cuda.synchronize()
        assert torch.equal(got, want)
        for f in ("sel", "logc", "tau", "union_teams", "union_rows"):
            assert torch.equal(getattr(dbg_a, f), getattr(dbg_b, f)), f
        # and the oracle's bar on a few heads
        pairs = [(0, 0), (0, wl.Hq - 1)]
        ot = oracle_teams(b, sorted(set((bi, h // wl.G) for bi, h in pairs)))
        so = oracle.decode(b.q, b.f64(b.K), b.f64(b.V), b.f64(b.sK), b.f64(b.sV), ot, wl.K, wl.seed, step,
                           wl.scale, heads=pairs)
        g = got.cpu().numpy()
        for bi, h in pairs:
            assert oracle.rel_l2(g[bi, h], so.heads[bi][h].out) <= 1e-4
        teams.close()


def test_static_scratch_limit():
    # every key its own team (M = 8192) for 8 sequences: log c alone needs
    # 8 x 28 x 8192 x 4 bytes, beyond the 4 MiB scratch
    wl, b, db, teams = _case("limit", B=8, data_seeds=tuple(range(20, 28)))
    need = sp.decode_workspace(teams, wl.Hq, wl.T, wl.K).numel()
    assert need > 4 << 20
    out = torch.empty((wl.B, wl.Hq, wl.d), dtype=torch.float32, device="cuda")
    with pytest.raises(sp.SantappError) as e:
        sp.decode_static(teams, db.q, db.sK, db.sV, wl.K, out, seed=1, step=0)
    assert e.value.status == sp._lib.ELIMIT
    assert b"static scratch" in sp._lib.load().santapp_last_error()
    teams.close()
