#!/usr/bin/env python3
"""Benchmark: SANTA++ decode attention on one MI355X.

One step = one ``santapp_decode`` call: routing, sampling, GQA read plan,
split-K attention over the sampled teams and the exact suffix, and the split
merge, for every query head of one Qwen2.5-7B-shaped layer (28 Q / 4 KV heads,
d = 128, bf16 K/V) at a 32768-token prompt, 32 sampled teams per head, 128
suffix rows, batch 1.  The step index advances every step, so every step
draws fresh Gumbel noise and reads a different set of teams.

Timing: the inputs are resident in HBM; before every step a 1 GiB buffer is
rewritten (outside the timed interval) so that the 256 MB last-level cache
holds none of the step's data; each step is bracketed by HIP events on the
stream the library launches on.  ``value`` is the mean step time in
microseconds.  The dense flash-decode baseline over all 32768 + 128 rows is
timed the same way.  The CPU oracle is timed on a bounded sample of the same
steps on the host (single thread).

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, GB/s


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default="qwen32k")
    p.add_argument("--K", type=int, default=None, help="teams per query head (default: workload's)")
    p.add_argument("--B", type=int, default=None)
    p.add_argument("--no-evict", action="store_true", help="keep the last-level cache warm")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="budget of the oracle CPU-baseline sample (0 disables it)")
    p.add_argument("--no-dense", action="store_true")
    p.add_argument("--parents", choices=("contiguous", "kmeans"), default="contiguous",
                   help="parent partition of the team table (Alg. contiguous / minibatch k-means)")
    p.add_argument("--kl-table", action="store_true",
                   help="print the routing KL diagnostic of several groupings of the workload and exit")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="only run a plain 256 MiB device-to-device copy five times (the reference "
                        "kernel for scaling the FETCH_SIZE / WRITE_SIZE counters) and exit")
    return p.parse_args()


def make_table(wl, db, parents, P=None, R=None):
    """Team table of the workload's keys: contiguous parents, or minibatch
    k-means parents with the paper's settings (batch 4096, at most 100
    iterations, 10-step no-improvement rule, reassignment ratio 0.01, seed 0).
    Returns (table, minibatch steps per (b, kv) or None)."""
    import paper_2609_35629_amd as sp
    P = wl.P if P is None else P
    R = wl.R if R is None else R
    if parents == "contiguous":
        return sp.build_teams(db["K"], db["V"], P, R), None
    labels, mp, steps = sp.kmeans_parents(db["K"], P)
    return sp.build_teams_from_labels(db["K"], db["V"], labels, mp, R), steps


def kl_table(wl, db):
    """Mean KL(p || q) in nats (eq. diagnostic-kl) over every (sequence, query
    head) of the workload, for teams and for centroid-guided sampling over
    contiguous groups (one team of B tokens per parent, routed by its mean),
    the groupings the paper's routing table compares (there with k-means
    groups on recorded model states)."""
    import paper_2609_35629_amd as sp
    variants = [("teams P=16 R=4 (representative keys)", 16, 4, "representative"),
                ("teams P=16 R=4 (team means)", 16, 4, "centroid"),
                ("centroid-guided B=4 (contiguous)", 4, 1, "centroid"),
                ("centroid-guided B=16 (contiguous)", 16, 1, "centroid"),
                (f"teams P={wl.P} R={wl.R} (representative keys)", wl.P, wl.R, "representative"),
                (f"teams P={wl.P} R={wl.R} (team means)", wl.P, wl.R, "centroid")]
    variants = [v + ("contiguous",) for v in variants]
    # k-means parents (the paper's main policy), and centroid-guided sampling
    # over k-means groups where their count stays within the k-means limit
    variants.append((f"teams P={wl.P} R={wl.R}, k-means parents (representative keys)", wl.P, wl.R,
                     "representative", "kmeans"))
    for Bg in (16, 32):
        if wl.N // Bg <= 1024:
            variants.append((f"centroid-guided B={Bg} (k-means groups)", Bg, 1, "centroid", "kmeans"))
    rows = []
    for name, P, R, kind, parents in variants:
        t, _ = make_table(wl, db, parents, P, R)
        sp.set_route_keys(t, kind)
        kl = sp.routing_kl(t, db["q"], scale=wl.scale)
        rows.append({"variant": name, "P": P, "R": R, "M": t.M, "route_keys": kind,
                     "mean_kl_nats": round(float(kl.mean().item()), 4)})
        t.close()
    print(json.dumps({"workload": wl.name, "N": wl.N, "B": wl.B, "Hq": wl.Hq, "kl_table": rows}))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: this build has no multi-GPU path "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import datagen
    import paper_2609_35629_amd as sp

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy()
        return
    sp._lib.load()  # raises when the HIP library is not built

    wl = datagen.WORKLOADS[args.workload]
    if args.K is not None:
        wl = wl.with_(K=args.K)
    if args.B is not None:
        wl = wl.with_(B=args.B, data_seeds=tuple(range(100, 100 + args.B)))
    print(f"[bench] workload={wl.name} B={wl.B} N={wl.N} K={wl.K} T={wl.T}", file=sys.stderr, flush=True)
    batch = datagen.generate(wl)
    db = upload(batch)
    if args.kl_table:
        kl_table(wl, db)
        return
    teams, km_steps = make_table(wl, db, args.parents)
    M = teams.M
    ws = sp.decode_workspace(teams, wl.Hq, wl.T, wl.K)
    out = torch.empty((wl.B, wl.Hq, wl.d), dtype=torch.float32, device="cuda")
    evict = torch.empty(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB

    def run_sparse(step, dbg=None):
        sp.decode(teams, db["q"], db["sK"], db["sV"], wl.K, seed=wl.seed, step=step, scale=wl.scale,
                  out=out, workspace=ws, debug=dbg)

    dense_ws = sp.dense_workspace(wl.B, wl.Hq, wl.Hkv, wl.N, wl.T, wl.d)
    dense_out = torch.empty_like(out)

    def run_dense(step, dbg=None):
        sp.dense_decode(db["q"], db["K"], db["V"], db["sK"], db["sV"], scale=wl.scale, out=dense_out,
                        workspace=dense_ws)

    hev = HipEvents(sp._lib.load())

    def timed(fn, n, warm, with_stages):
        for i in range(warm):
            fn(i)
        warm = max(warm, args.warmup)
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        ev0 = [hev.make() for _ in range(n)]
        ev1 = [hev.make() for _ in range(n)]
        marks = [[hev.make() for _ in range(4)] for _ in range(n)] if with_stages else None
        dbgs = [None] * n
        if with_stages:
            dbgs = [sp.DebugOut(wl.B, wl.Hq, wl.Hkv, M, wl.K, arrays=False) for _ in range(n)]
            for d, mk in zip(dbgs, marks):
                d.raw_events = mk
        torch.cuda.synchronize()
        for i in range(n):
            if not args.no_evict:
                evict.add_(1.0)
            hev.record(ev0[i], stream)
            fn(warm + i, dbgs[i])
            hev.record(ev1[i], stream)
        torch.cuda.synchronize()
        times = np.array([hev.us(a, b) for a, b in zip(ev0, ev1)])
        stages = []
        if with_stages:
            stages = np.array([[hev.us(mk[k], mk[k + 1]) for k in range(3)] for mk in marks])
        return times, stages

    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    sparse_us, _ = timed(run_sparse, args.steps, args.warmup, False)
    t_wall1 = time.perf_counter()
    dense_us = None
    if not args.no_dense:
        dense_us, _ = timed(run_dense, args.steps, args.warmup, False)
    # second pass over the same steps with the library's stage markers on
    # (each marker adds a few microseconds, so the step time above has none)
    _, stages_us = timed(run_sparse, args.steps, 0, True)

    # bytes each timed step read: the union rows of every (b, kv) (replayed
    # with the diagnostics on; same seed and step give the same selection)
    row_bytes = 2 * wl.d * 2
    union_rows = np.zeros(args.steps)
    for i in range(args.steps):
        dbg = sp.DebugOut(wl.B, wl.Hq, wl.Hkv, M, wl.K)
        run_sparse(args.warmup + i, dbg)
        torch.cuda.synchronize()
        union_rows[i] = dbg.union_rows.sum().item()
    sampled = wl.K < M
    BH = wl.B * wl.Hkv
    rep_bytes = BH * M * wl.d * 2 if sampled else 0
    suffix_bytes = BH * wl.T * row_bytes
    small_bytes = wl.B * wl.Hq * wl.d * 4 * 2  # q in, out
    if not sampled:
        union_rows[:] = BH * wl.N
    attend_bytes = union_rows * row_bytes + suffix_bytes
    step_bytes = rep_bytes + attend_bytes + small_bytes
    dense_bytes = BH * (wl.N + wl.T) * row_bytes + small_bytes

    attend_us = stages_us[:, 1]
    achieved = float(np.mean(attend_bytes) / np.mean(attend_us) / 1e3)  # GB/s
    value = float(np.mean(sparse_us))
    # eq. qwen-logical-access: one key per representative, key + value per row read
    read_fraction = float(np.mean(rep_bytes + attend_bytes) / (BH * (wl.N + wl.T) * row_bytes))

    # HBM bytes per launch of the attention kernel (rocprofv3 counters,
    # copy-calibrated), for the workload they were measured on, while the
    # kernel's sources are unchanged since
    traffic = None
    if wl.name == "qwen32k" and wl.K == 32 and wl.B == 1 and not args.no_evict and args.parents == "contiguous":
        traffic = measured_traffic()

    # preparation per prompt, excluded from the step as in the paper: host
    # time of the table build (k-means when chosen, device allocations, team
    # build, packed copies; the calls return once their kernels are done),
    # median of three
    prep_us = []
    for _ in range(3):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        extra, _ = make_table(wl, db, args.parents)
        prep_us.append((time.perf_counter() - t0) * 1e6)
        extra.close()

    # routing diagnostic (eq. diagnostic-kl) of this table on the step's
    # queries, routed by the representative keys and by the team means
    routing_kl = {}
    for kind in ("representative", "centroid"):
        sp.set_route_keys(teams, kind)
        routing_kl[kind] = round(float(sp.routing_kl(teams, db["q"], scale=wl.scale).mean().item()), 4)
    sp.set_route_keys(teams, "representative")

    cpu = None
    if args.cpu_seconds > 0 and args.parents == "contiguous":
        cpu = cpu_baseline(wl, batch, args.cpu_seconds)

    res = {
        "metric": "SANTA++ decode-attn us/step/layer + achieved HBM GB/s, 32K ctx, 32 teams",
        "value": round(value, 3),
        "unit": "us/step/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(value / 1e3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == datagen.BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: Qwen2.5-7B-shaped layer, {wl.N}-token prompt, B={wl.B}",
                   "B": wl.B, "Hq": wl.Hq, "Hkv": wl.Hkv, "d": wl.d, "N": wl.N, "T": wl.T,
                   "P": wl.P, "R": wl.R, "M": M, "K": wl.K, "parents": args.parents,
                   "evict_1GiB": not args.no_evict},
        "roofline": {"bound": "hbm", "kernel": "k_attend_mfma<128, false>", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic},
        "prep_us": round(float(np.median(prep_us)), 1),
        "routing_kl_nats": routing_kl,
        "step_gbs": round(float(np.mean(step_bytes) / value / 1e3), 1),
        "step_hbm_frac": round(float(np.mean(step_bytes) / value / 1e3) / HBM_PEAK_GBS, 4),
        "step_bytes_mean": int(np.mean(step_bytes)),
        "union_rows_mean": float(np.mean(union_rows)),
        "read_fraction": round(read_fraction, 4),
        "median_us": round(float(np.median(sparse_us)), 3),
        "stage_us_mean": {"route_select": round(float(np.mean(stages_us[:, 0])), 3),
                          "attend": round(float(np.mean(stages_us[:, 1])), 3),
                          "merge": round(float(np.mean(stages_us[:, 2])), 3)},
        "wall_s_sparse_loop": round(t_wall1 - t_wall0, 3),
    }
    if km_steps is not None:
        res["kmeans_steps"] = km_steps
    if dense_us is not None:
        d = float(np.mean(dense_us))
        res["dense_us"] = round(d, 3)
        res["dense_gbs"] = round(dense_bytes / d / 1e3, 1)
        res["speedup_vs_dense"] = round(d / value, 3)
    if cpu is not None:
        res["cpu_baseline"] = cpu
    print(json.dumps(res), flush=True)


class HipEvents:
    """HIP events recorded with a device-scope release: the default event
    record also writes back and invalidates the caches at system scope, which
    adds several microseconds to every bracketed interval."""
    RELEASE_TO_DEVICE = 0x40000000

    def __init__(self, lib):
        import ctypes
        self.c = ctypes
        self.L = lib
        vp = ctypes.c_void_p
        lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp), ctypes.c_uint]
        lib.hipEventRecord.argtypes = [vp, vp]
        lib.hipEventSynchronize.argtypes = [vp]
        lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
        lib.hipEventDestroy.argtypes = [vp]
        for f in (lib.hipEventCreateWithFlags, lib.hipEventRecord, lib.hipEventSynchronize,
                  lib.hipEventElapsedTime, lib.hipEventDestroy):
            f.restype = ctypes.c_int

    def make(self):
        e = self.c.c_void_p()
        if self.L.hipEventCreateWithFlags(self.c.byref(e), self.RELEASE_TO_DEVICE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")
        return e

    def record(self, e, stream):
        if self.L.hipEventRecord(e, stream) != 0:
            raise RuntimeError("hipEventRecord failed")

    def us(self, a, b):
        t = self.c.c_float()
        self.L.hipEventSynchronize(b)
        if self.L.hipEventElapsedTime(self.c.byref(t), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return t.value * 1e3


def measured_traffic():
    """Read + write bytes per launch of the sparse attention kernel from
    profiles/traffic_k_attend_qwen32k_K32.md, or None when the kernel's
    sources no longer hash to the value recorded there."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", "traffic_k_attend_qwen32k_K32.md")
    try:
        text = open(path).read()
    except OSError:
        return None
    vals = dict(re.findall(r"^(sources_sha256|read_bytes_per_launch|write_bytes_per_launch): (\S+)$", text, re.M))
    if len(vals) != 3:
        return None
    csrc = os.path.join(ROOT, "paper_2609_35629_amd", "csrc")
    src = b"".join(open(os.path.join(csrc, f), "rb").read() for f in ("decode_kernels.hip", "common.h", "internal.h"))
    if hashlib.sha256(src).hexdigest() != vals["sources_sha256"]:
        return None
    return int(vals["read_bytes_per_launch"]) + int(vals["write_bytes_per_launch"])


def calibrate_copy():
    """A plain copy of known size: 256 MiB read and 256 MiB written per
    launch (torch's device-to-device copy kernel), five launches."""
    import torch
    n = 64 << 20  # floats
    src = torch.empty(n, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy": {"bytes_read": n * 4, "bytes_written": n * 4, "launches": 5}}),
          flush=True)


def upload(batch):
    """Copy a datagen batch to the GPU (bf16 bit patterns become bfloat16)."""
    import numpy as np
    import torch

    import datagen

    def dev(a):
        if batch.wl.dtype == datagen.BF16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()

    T = batch.wl.T
    return {"q": torch.from_numpy(batch.q).cuda(), "K": dev(batch.K), "V": dev(batch.V),
            "sK": dev(batch.sK) if T else None, "sV": dev(batch.sV) if T else None}


def cpu_baseline(wl, batch, budget_s):
    """The oracle (test infrastructure) on the host: whole decode steps (all
    query heads), as many as fit in the time budget; team construction is
    excluded, as for the GPU."""
    import numpy as np

    import oracle
    Kf = batch.f32(batch.K)
    teams = oracle.build_all(Kf, wl.P, wl.R)
    Vf = batch.f32(batch.V)
    sKf = batch.f32(batch.sK)
    sVf = batch.f32(batch.sV)
    steps = 0
    t0 = time.perf_counter()
    while True:
        oracle.decode(batch.q, Kf, Vf, sKf, sVf, teams, wl.K, wl.seed, steps, wl.scale)
        steps += 1
        if time.perf_counter() - t0 > budget_s:
            break
    el = time.perf_counter() - t0
    return {"value": round(el / steps * 1e6, 1), "unit": "us/step/layer", "cores": 1,
            "kind": "oracle",
            "sample": f"{steps} full decode steps ({wl.B}x{wl.Hq} heads each) of the same workload, "
                      f"fp64 C oracle, one thread, team build excluded"}


if __name__ == "__main__":
    main()
