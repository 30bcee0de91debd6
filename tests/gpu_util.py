"""Helpers shared by the GPU parity tests: move a datagen batch to the GPU,
run the library, run the oracle on the same bytes, and compare."""
from __future__ import annotations

import dataclasses
import sys
from typing import List, Optional

import numpy as np
import torch

import datagen
import oracle
import paper_2609_35629_amd as sp


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == datagen.BF16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


@dataclasses.dataclass
class DevBatch:
    batch: datagen.Batch
    q: torch.Tensor
    K: torch.Tensor
    V: torch.Tensor
    sK: Optional[torch.Tensor]
    sV: Optional[torch.Tensor]


def dev_batch(b: datagen.Batch) -> DevBatch:
    dt = b.wl.dtype
    sK = to_dev(b.sK, dt) if b.wl.T > 0 else None
    sV = to_dev(b.sV, dt) if b.wl.T > 0 else None
    return DevBatch(b, torch.from_numpy(b.q).cuda(), to_dev(b.K, dt), to_dev(b.V, dt), sK, sV)


def oracle_teams(b: datagen.Batch, kv_pairs=None):
    """teams[b][kv] from the oracle (only the listed (b, kv) pairs if given)."""
    B, Hkv = b.wl.B, b.wl.Hkv
    out = [[None] * Hkv for _ in range(B)]
    for bi in range(B):
        for kv in range(Hkv):
            if kv_pairs is None or (bi, kv) in kv_pairs:
                out[bi][kv] = oracle.build_teams(b.f64(b.K[bi, kv]), b.wl.P, b.wl.R)
    return out


def gpu_tables(teams: sp.Teams):
    return (teams.perm().cpu().numpy(), teams.team_begin().cpu().numpy(),
            teams.team_size().cpu().numpy(), teams.rep_token().cpu().numpy())


def assert_tables_equal(gpu, ot, bi, kv):
    perm, tb, ts, rt = gpu
    t = ot[bi][kv]
    assert tb.shape[2] == t.M
    np.testing.assert_array_equal(perm[bi, kv], t.members, err_msg=f"perm b={bi} kv={kv}")
    np.testing.assert_array_equal(tb[bi, kv], t.team_ptr[:-1], err_msg=f"team_begin b={bi} kv={kv}")
    np.testing.assert_array_equal(ts[bi, kv], t.sizes, err_msg=f"team_size b={bi} kv={kv}")
    np.testing.assert_array_equal(rt[bi, kv], t.rep_token, err_msg=f"rep_token b={bi} kv={kv}")


@dataclasses.dataclass
class Compare:
    heads: int
    sel_equal: int
    excused: int
    unexcused: List[tuple]
    rel_l2: np.ndarray      # per compared head
    max_phi_rel: float
    max_tau_abs: float
    equal: np.ndarray = None        # per compared head: same team set as the oracle
    max_logc_abs: float = 0.0       # |log c_gpu - log c_oracle| over heads with equal sets
    max_tau_rel_equal: float = 0.0  # |tau_gpu - tau_oracle| / max(1, |tau|) over the same heads

    @property
    def rel_l2_equal(self) -> np.ndarray:
        """rel-L2 of the heads whose selection equals the oracle's (the
        fixed-selection comparison of the appendix "Kernel evaluation
        protocol")."""
        return self.rel_l2[self.equal] if self.equal is not None else self.rel_l2

    def assert_selection_bar(self):
        """At least 99.9% of the instances select the oracle's team set (so
        every one of fewer than 1000), and every mismatch is a near-tie of
        the oracle's K-th and (K+1)-th perturbed scores."""
        assert not self.unexcused, self.unexcused
        assert self.sel_equal + self.excused == self.heads
        assert self.sel_equal >= int(np.ceil(0.999 * self.heads)), (self.sel_equal, self.heads)


def compare_step(wl: datagen.Workload, Kb: int, out_gpu: np.ndarray, dbg: Optional[sp.DebugOut],
                 step_or: oracle.StepResult, pairs, sampled: bool) -> Compare:
    rel, unexc, equal = [], [], []
    eq = exc = 0
    max_phi = max_tau = max_lc = max_tau_eq = 0.0
    if sampled:
        sel = dbg.sel.cpu().numpy()
        phi = dbg.phi.cpu().numpy()
        tau = dbg.tau.cpu().numpy()
        logc = dbg.logc.cpu().numpy()
    for (bi, h) in pairs:
        r = step_or.heads[bi][h]
        rel.append(oracle.rel_l2(out_gpu[bi, h], r.out))
        if not sampled:
            equal.append(True)
            continue
        max_phi = max(max_phi, float(np.max(np.abs(phi[bi, h] - r.phi) / np.maximum(1.0, np.abs(r.phi)))))
        max_tau = max(max_tau, abs(float(tau[bi, h]) - r.tau))
        if np.array_equal(sel[bi, h], r.sel):  # both ascending
            eq += 1
            equal.append(True)
            max_lc = max(max_lc, float(np.max(np.abs(logc[bi, h].astype(np.float64) - np.log(r.c)))))
            max_tau_eq = max(max_tau_eq, abs(float(tau[bi, h]) - r.tau) / max(1.0, abs(r.tau)))
        else:
            equal.append(False)
            ys = np.sort(r.Y)[::-1]
            gap = ys[Kb - 1] - ys[Kb]
            if gap <= 1e-6 * max(1.0, abs(r.tau)):
                exc += 1
            else:
                unexc.append((bi, h, gap))
    return Compare(len(pairs), eq, exc, unexc, np.array(rel), max_phi, max_tau, np.array(equal, bool), max_lc,
                   max_tau_eq)


def union_stats(teams_or, sels, G: int):
    """Per (b, kv): the number of distinct teams the pair's G query heads
    selected and their prompt rows (eq. qwen-logical-access's u), from
    selections sels[b][h] (ascending team ids)."""
    B = len(sels)
    Hkv = len(sels[0]) // G
    ut = np.zeros((B, Hkv), np.int64)
    ur = np.zeros((B, Hkv), np.int64)
    for b in range(B):
        for kv in range(Hkv):
            hs = [sels[b][h] for h in range(kv * G, (kv + 1) * G)]
            ut[b, kv] = len(set(int(g) for s in hs for g in s))
            ur[b, kv] = oracle.union_rows(teams_or[b][kv], hs)
    return ut, ur
