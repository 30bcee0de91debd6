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
    p.add_argument("--check-steps", type=int, default=-1,
                   help="timed steps the cpu_baseline leg checks against the oracle afterwards (-1: as "
                        "many as fit in about 20 s of oracle time, 0: none)")
    p.add_argument("--loop-steps", type=int, default=64,
                   help="steps of the two-layer decode loop timed as the suffix grows (0: skip)")
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
                        workspace=dense_ws, debug=dbg)

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
    dense_stages_us = None
    if not args.no_dense:
        _, dense_stages_us = timed(run_dense, args.steps, 0, True)

    # bytes each timed step read: the union rows of every (b, kv) (replayed
    # with the diagnostics on; same seed and step give the same selection)
    row_bytes = 2 * wl.d * (2 if wl.dtype == datagen.BF16 else 4)
    union_rows = np.zeros(args.steps)
    replays = []
    for i in range(args.steps):
        dbg = sp.DebugOut(wl.B, wl.Hq, wl.Hkv, M, wl.K)
        run_sparse(args.warmup + i, dbg)
        torch.cuda.synchronize()
        union_rows[i] = dbg.union_rows.sum().item()
        replays.append((out.cpu().numpy(), dbg.sel.cpu().numpy()))
    sampled = wl.K < M
    BH = wl.B * wl.Hkv
    rep_bytes = BH * M * wl.d * (2 if wl.dtype == datagen.BF16 else 4) if sampled else 0
    suffix_bytes = BH * wl.T * row_bytes
    small_bytes = wl.B * wl.Hq * wl.d * 4 * 2  # q in, out
    if not sampled:
        union_rows[:] = BH * wl.N
    attend_bytes = union_rows * row_bytes + suffix_bytes
    step_bytes = rep_bytes + attend_bytes + small_bytes
    dense_bytes = BH * (wl.N + wl.T) * row_bytes + small_bytes

    # the launch the stage events bracket: the single step kernel (every
    # byte of the step: routing keys, union rows, suffix, q and out) or the
    # attention launch of the three-launch kernels (union rows and suffix)
    kernels, _ = sp.decode_launch_info(teams, wl.Hq, wl.T, wl.K)
    single = kernels == 1 and os.environ.get("SANTAPP_DECODE_LAUNCH") != "fused"
    kernel_us = stages_us[:, 1]
    kernel_bytes = step_bytes if single else attend_bytes
    achieved = float(np.mean(kernel_bytes) / np.mean(kernel_us) / 1e3)  # GB/s
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

    # the cpu_baseline leg: the oracle (test infrastructure) on the host
    # cores, outside the timed region -- timed over whole decode steps, and
    # the checker of the replayed timed steps (output rel-L2 per head and
    # team-set agreement)
    check = cpu = None
    if args.cpu_seconds > 0 and args.parents == "contiguous":
        host = HostOracle(wl, batch)
        if args.check_steps != 0:
            check = host.check(replays, args.warmup, args.check_steps, sampled=wl.K < M)
        cpu = host.time_steps(args.cpu_seconds)

    ceiling = hbm_read_ceiling(evict)
    loop = None
    if args.loop_steps > 0 and args.parents == "contiguous":
        loop = loop_timing(wl, args.loop_steps, 2, evict, hev, args.no_evict)

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
        "roofline": {"bound": "hbm", "kernel": attend_kernel_name(wl, M, single), "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic},
        "hbm_read_ceiling": ceiling,
        "prep_us": round(float(np.median(prep_us)), 1),
        "routing_kl_nats": routing_kl,
        "step_gbs": round(float(np.mean(step_bytes) / value / 1e3), 1),
        "step_hbm_frac": round(float(np.mean(step_bytes) / value / 1e3) / HBM_PEAK_GBS, 4),
        "step_frac_of_measured_ceiling": round(float(np.mean(step_bytes) / value / 1e3) / ceiling["read_gbs"], 4),
        "attend_frac_of_measured_ceiling": round(achieved / ceiling["read_gbs"], 4),
        "step_bytes_mean": int(np.mean(step_bytes)),
        "union_rows_mean": float(np.mean(union_rows)),
        "read_fraction": round(read_fraction, 4),
        "median_us": round(float(np.median(sparse_us)), 3),
        "stage_us_mean": ({"before_kernel": round(float(np.mean(stages_us[:, 0])), 3),
                           "kernel": round(float(np.mean(stages_us[:, 1])), 3),
                           "after_kernel": round(float(np.mean(stages_us[:, 2])), 3)} if single else
                          {"route_select": round(float(np.mean(stages_us[:, 0])), 3),
                           "attend": round(float(np.mean(stages_us[:, 1])), 3),
                           "merge": round(float(np.mean(stages_us[:, 2])), 3)}),
        "wall_s_sparse_loop": round(t_wall1 - t_wall0, 3),
    }
    if km_steps is not None:
        res["kmeans_steps"] = km_steps
    if dense_us is not None:
        d = float(np.mean(dense_us))
        res["dense_us"] = round(d, 3)
        res["dense_gbs"] = round(dense_bytes / d / 1e3, 1)
        res["speedup_vs_dense"] = round(d / value, 3)
        # the dense launch by its own start/end events: its rows' bytes over
        # the kernel's execution time
        dk = float(np.mean(dense_stages_us[:, 1]))
        dense_kernel = (f"k_step<{wl.d}, 2, true>" if wl.dtype == datagen.BF16 and wl.B * wl.Hkv <= 256
                        else "k_decode (dense)")
        res["dense_roofline"] = {"kernel": dense_kernel, "kernel_us": round(dk, 3),
                                 "achieved": round(dense_bytes / dk / 1e3, 1), "peak": 8000.0, "unit": "GB/s",
                                 "frac": round(dense_bytes / dk / 1e3 / 8000.0, 4)}
    if check is not None:
        res.update(check)
    if loop is not None:
        res["decode_loop"] = loop
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
    profiles/traffic_k_step_qwen32k_K32.md, or None when the kernel's
    sources no longer hash to the value recorded there."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", "traffic_k_step_qwen32k_K32.md")
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


def loop_timing(wl, steps, layers, evict, hev, no_evict):
    """A two-layer decode loop at the workload's shape: every layer starts
    with an empty suffix and appends one generated row per (b, kv) and step.
    Each layer's attention call is timed on its own (events on the stream,
    the 1 GiB eviction between steps); reported as the mean over the layers
    and the steps of each quarter of the loop, sampled and dense."""
    import numpy as np
    import torch

    import datagen
    from paper_2609_35629_amd.decode_loop import DecodeLoop
    trace = datagen.decode_trace(wl, layers, steps)
    dev = lambda a: upload_rows(a, wl.dtype)
    prompts = [(dev(b.K), dev(b.V)) for b, _ in trace]
    rows = [(dev(b.sK), dev(b.sV)) for b, _ in trace]
    qdev = [torch.from_numpy(qs).cuda() for _, qs in trace]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    out = {"layers": layers, "steps": steps, "workload": f"{wl.name} shape, T = 0 .. {steps - 1}"}
    q4 = max(1, steps // 4)
    for dense in (False, True):
        loop = DecodeLoop(prompts, steps, wl.Hq, wl.K, wl.P, wl.R, seed=wl.seed, dense=dense)
        ev = [[(hev.make(), hev.make()) for _ in range(layers)] for _ in range(steps)]
        torch.cuda.synchronize()
        for t in range(steps):
            if not no_evict:
                evict.add_(1.0)
            for li, layer in enumerate(loop.layers):
                hev.record(ev[t][li][0], stream)
                layer.attend(qdev[li][t], loop.seed + li, t, wl.scale)
                hev.record(ev[t][li][1], stream)
                layer.append(rows[li][0][:, :, t], rows[li][1][:, :, t])
        torch.cuda.synchronize()
        us = np.array([[hev.us(a, b) for a, b in ev[t]] for t in range(steps)]).mean(axis=1)
        key = "dense_us_per_layer_step" if dense else "us_per_layer_step"
        out[key] = {f"T{lo}-{min(lo + q4, steps) - 1}": round(float(us[lo:lo + q4].mean()), 2)
                    for lo in range(0, steps, q4)}
        loop.close()
    return out


def upload_rows(a, dtype):
    import numpy as np
    import torch
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def attend_kernel_name(wl, M, single):
    """The launch the stage events bracket: the single step kernel (template
    arguments: head dimension, keys per lane of the selecting waves, dense),
    the attention kernel of the split launch, or the single kernel of the
    fused one (row type, head dimension, teams per sampler thread, launch
    mode, dense)."""
    if single:
        return f"k_step<{wl.d}, {2 if M <= 128 else 8}, {'true' if wl.K >= M else 'false'}>"
    dt = "bf16_t" if wl.dtype == "bf16" else "float"
    mode = "kFused" if os.environ.get("SANTAPP_DECODE_LAUNCH") == "fused" and wl.dtype == "bf16" else "kAttend"
    hk = 1 if M <= 512 else (4 if M <= 2048 else 16)
    return f"k_decode<{dt}, {wl.d}, {hk}, {mode}, false>"


def hbm_read_ceiling(buf):
    """Measured streaming rates of this GPU over the 1 GiB buffer: a plain
    read of all of it (the package's streaming-read probe, best of five
    launches at each of four grid sizes) and a 512 MiB device copy (read +
    write, best of five)."""
    import torch
    from paper_2609_35629_amd import build as pkg_build
    probe = ctypes.CDLL(pkg_build.PROBE_LIB)
    probe.santapp_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int,
                                         ctypes.c_void_p]
    probe.santapp_probe_read.restype = ctypes.c_int
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    nbytes = buf.numel() * buf.element_size()

    def best_of(fn, reps=5):
        fn()
        best = None
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            best = ms if best is None else min(best, ms)
        return best

    def read(grid):
        rc = probe.santapp_probe_read(ctypes.c_void_p(buf.data_ptr()), nbytes, ctypes.c_void_p(sink.data_ptr()),
                                      grid, stream)
        if rc != 0:
            raise RuntimeError(f"streaming-read probe failed ({rc})")

    grids = (256, 512, 1024, 2048)
    read_ms = {g: best_of(lambda: read(g)) for g in grids}
    g_best = min(read_ms, key=read_ms.get)
    half = buf.numel() // 2
    src, dst = buf[:half], buf[half:]
    copy_ms = best_of(lambda: dst.copy_(src))
    return {"read_gbs": round(nbytes / (read_ms[g_best] * 1e-3) / 1e9, 1),
            "copy_gbs": round(2 * half * buf.element_size() / (copy_ms * 1e-3) / 1e9, 1),
            "read_grid": g_best,
            "method": "1 GiB streaming read (16-byte non-temporal loads, 512-thread workgroups, best grid of "
                      "256/512/1024/2048, best of 5) and a 512 MiB torch device copy (read + write, best of 5)"}


class HostOracle:
    """The oracle (test infrastructure) on the host, over the same batch:
    team tables built once, inputs widened to fp64 once."""

    def __init__(self, wl, batch):
        import oracle
        self.oracle = oracle
        self.wl = wl
        self.batch = batch
        self.teams = oracle.build_all(batch.f64(batch.K), wl.P, wl.R)
        self.x64 = [batch.f64(x) for x in (batch.K, batch.V, batch.sK, batch.sV)]

    def _head(self, b, h, step):
        wl = self.wl
        kv = h // wl.G
        K, V, sK, sV = self.x64
        return self.oracle.decode_head(self.batch.q[b, h], K[b, kv], V[b, kv], self.teams[b][kv], sK[b, kv],
                                       sV[b, kv], wl.K, wl.seed, step, b, h, wl.scale)

    def step(self, step, pool=None):
        wl = self.wl
        heads = [(b, h) for b in range(wl.B) for h in range(wl.Hq)]
        if pool is None:
            return [self._head(b, h, step) for (b, h) in heads]
        return list(pool.map(lambda bh: self._head(bh[0], bh[1], step), heads))

    def check(self, replays, first_step, max_steps, sampled):
        """rel-L2 of every head of the replayed timed steps and the share of
        (query, head) instances whose team set equals the oracle's."""
        import numpy as np
        wl = self.wl
        n = len(replays)
        if max_steps < 0:
            t0 = time.perf_counter()
            self.step(first_step)
            per = max(time.perf_counter() - t0, 1e-3)
            max_steps = max(1, min(n, int(20.0 / per)))
        n = min(n, max_steps)
        rel, equal, total = [], 0, 0
        for i in range(n):
            out, sel = replays[i]
            res = self.step(first_step + i)
            for j, r in enumerate(res):
                b, h = divmod(j, wl.Hq)
                rel.append(self.oracle.rel_l2(out[b, h], r.out))
                if sampled:
                    total += 1
                    equal += int(np.array_equal(sel[b, h], r.sel))
        rel = np.array(rel)
        outd = {"rel_l2_vs_oracle": {"max": float(f"{rel.max():.3e}"), "mean": float(f"{rel.mean():.3e}"),
                                     "heads": int(rel.size), "steps": n}}
        if sampled:
            outd["team_set_agreement"] = {"equal": equal, "instances": total,
                                          "fraction": round(equal / max(total, 1), 6)}
        return outd

    def time_steps(self, budget_s):
        """Whole decode steps (all query heads) on the host cores: one thread,
        then a thread per core over the (b, h) heads (the C oracle runs with
        the GIL released); each figure is the median of five repetitions of
        a fixed number of steps, sized so that the whole leg takes about
        budget_s seconds."""
        import statistics
        from concurrent.futures import ThreadPoolExecutor
        try:
            nproc = len(os.sched_getaffinity(0))
        except AttributeError:
            nproc = os.cpu_count() or 1
        threads = max(1, min(nproc, 16))
        t0 = time.perf_counter()
        self.step(0)
        per = max(time.perf_counter() - t0, 1e-4)
        k = max(1, int(budget_s / 2 / 5 / per))  # steps per single-thread repetition

        def reps(pool):
            times = []
            s = 0
            for _ in range(5):
                t = time.perf_counter()
                for _ in range(k):
                    self.step(s, pool)
                    s += 1
                times.append((time.perf_counter() - t) / k)
            return statistics.median(times)

        single = reps(None)
        with ThreadPoolExecutor(max_workers=threads) as pool:
            multi = reps(pool)
        wl = self.wl
        return {"value": round(multi * 1e6, 1), "unit": "us/step/layer", "cores": threads, "kind": "oracle",
                "single_thread_us": round(single * 1e6, 1), "multi_thread_us": round(multi * 1e6, 1),
                "nproc": nproc,
                "sample": f"median of 5 repetitions of {k} full decode steps ({wl.B}x{wl.Hq} heads each) of "
                          f"the same workload, fp64 C oracle, team build and input widening excluded; "
                          f"multi-thread: {threads} threads over the (b, h) heads"}


if __name__ == "__main__":
    main()
