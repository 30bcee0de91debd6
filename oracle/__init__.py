"""CPU oracle for SANTA++ decode attention.

TEST INFRASTRUCTURE ONLY: the fp64 statement of what the decode path computes,
written from the paper.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it; the GPU library never
does, and this package imports nothing from the GPU library.

The arithmetic lives in ``santapp_oracle.c`` (plain C, fp64, compiled with
``-ffp-contract=off``); this module marshals numpy arrays into it and adds the
bookkeeping of the paper's logical KV-access counter (eq. qwen-logical-access).
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
import subprocess
from typing import List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "santapp_oracle.c")
# SANTAPP_ORACLE_LIB names another build of the same source to load (the
# sanitizer test's instrumented copy)
_SO = os.environ.get("SANTAPP_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

_d = ctypes.POINTER(ctypes.c_double)
_i = ctypes.POINTER(ctypes.c_int)
_u64 = ctypes.POINTER(ctypes.c_uint64)


def build(out: Optional[str] = None, sanitize: bool = False) -> str:
    """Compile the oracle into ``oracle/liboracle.so``, or ``out`` (always
    recompiles).  ``sanitize``: a host build with AddressSanitizer and
    UndefinedBehaviorSanitizer, every finding fatal, for the sanitizer test
    (loaded with the ASan runtime preloaded)."""
    out = out or _SO
    tmp = out + ".tmp"
    cmd = ["gcc", "-O2", "-std=gnu11", "-fPIC", "-shared", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-o", tmp, _SRC, "-lm"]
    if sanitize:
        cmd[1:2] = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        L.philox4x64_10.argtypes = [_u64, _u64, _u64]
        L.philox4x64_10.restype = None
        L.oracle_gumbel.argtypes = [ctypes.c_uint64]
        L.oracle_gumbel.restype = ctypes.c_double
        L.oracle_team_gumbel.argtypes = [ctypes.c_uint64] * 5
        L.oracle_team_gumbel.restype = ctypes.c_double
        L.oracle_build_teams.argtypes = [_d, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                         ctypes.c_int, _i, _i, _i]
        L.oracle_build_teams.restype = ctypes.c_int
        L.oracle_decode_head.argtypes = (
            [_d, ctypes.c_int, _d, _d, ctypes.c_int, _i, _i, _i, _d, ctypes.c_int,
             _d, _d, ctypes.c_int, ctypes.c_int, ctypes.c_uint64, ctypes.c_uint64,
             ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double, ctypes.c_double,
             _d, _d, _d, _d, _d, _d, _i, _d, _d])
        L.oracle_decode_head.restype = ctypes.c_int
        L.oracle_dense_head.argtypes = [_d, ctypes.c_int, _d, _d, ctypes.c_int, _d, _d,
                                        ctypes.c_int, ctypes.c_double, _d, _d, _d, _d]
        L.oracle_dense_head.restype = ctypes.c_int
        L.oracle_team_means.argtypes = [_d, ctypes.c_int, _i, _i, ctypes.c_int, _d]
        L.oracle_team_means.restype = ctypes.c_int
        L.oracle_build_teams_parents.argtypes = [_d, ctypes.c_int, ctypes.c_int, _i, _i, ctypes.c_int,
                                                 ctypes.c_int, _i, _i, _i]
        L.oracle_build_teams_parents.restype = ctypes.c_int
        L.oracle_kmeans.argtypes = [_d, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_int, ctypes.c_int, ctypes.c_double, ctypes.c_int,
                                    ctypes.c_uint64, _d, _i, _i, _d]
        L.oracle_kmeans.restype = ctypes.c_int
        _lib = L
    return _lib


def _pd(a: np.ndarray):
    return a.ctypes.data_as(_d)


def _pi(a: np.ndarray):
    return a.ctypes.data_as(_i)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


# --------------------------------------------------------------------------
# Counter-based generator and Gumbel noise
# --------------------------------------------------------------------------
def philox(counter, key) -> np.ndarray:
    """Philox4x64-10 of one 4x64-bit counter under a 2x64-bit key."""
    c = (ctypes.c_uint64 * 4)(*[int(x) & (2**64 - 1) for x in counter])
    k = (ctypes.c_uint64 * 2)(*[int(x) & (2**64 - 1) for x in key])
    o = (ctypes.c_uint64 * 4)()
    lib().philox4x64_10(c, k, o)
    return np.array(list(o), dtype=np.uint64)


def gumbel(word: int) -> float:
    return lib().oracle_gumbel(int(word))


def team_gumbel(seed: int, step: int, b: int, h: int, g: int) -> float:
    return lib().oracle_team_gumbel(seed, step, b, h, g)


# --------------------------------------------------------------------------
# Team construction (contiguous parents, actual-key representatives)
# --------------------------------------------------------------------------
@dataclasses.dataclass
class Teams:
    """Team records of one (sequence, KV head), in team order.

    ``members`` lists the token indices of team 0 (ascending), then team 1,
    ...; ``team_ptr`` holds the CSR offsets; ``rep_token[g]`` is the token
    whose key represents team g.
    """
    members: np.ndarray
    team_ptr: np.ndarray
    rep_token: np.ndarray

    @property
    def M(self) -> int:
        return len(self.rep_token)

    @property
    def sizes(self) -> np.ndarray:
        return np.diff(self.team_ptr)


def build_teams(K: np.ndarray, P: int, R: int) -> Teams:
    """Contiguous parents of P tokens, then up to R representatives each.

    ``K`` is one KV head's prompt keys ``[N, d]`` (exact values).
    """
    K = _f64(K)
    N, d = K.shape
    members = np.empty(N, np.int32)
    team_ptr = np.empty(N + 1, np.int32)
    rep_token = np.empty(N, np.int32)
    M = lib().oracle_build_teams(_pd(K), N, d, P, R, _pi(members), _pi(team_ptr), _pi(rep_token))
    if M < 0:
        raise ValueError("oracle_build_teams rejected its arguments")
    return Teams(members, team_ptr[:M + 1].copy(), rep_token[:M].copy())


def build_teams_from_labels(K: np.ndarray, labels: np.ndarray, R: int) -> Teams:
    """Teams of any parent partition given as one label per token: parent u
    is ``{i : labels[i] == u}``, parents in ascending label order, empty ones
    omitted (Alg. "Global minibatch k-means parent partition", last step),
    then Alg. "Build actual-key teams from a parent partition" per parent."""
    K = _f64(K)
    N, d = K.shape
    labels = np.asarray(labels)
    if labels.shape != (N,) or labels.min() < 0:
        raise ValueError("labels must be [N] and non-negative")
    order = np.argsort(labels, kind="stable").astype(np.int32)
    counts = np.bincount(labels, minlength=int(labels.max()) + 1)
    pptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    members = np.empty(N, np.int32)
    team_ptr = np.empty(N + 1, np.int32)
    rep_token = np.empty(N, np.int32)
    M = lib().oracle_build_teams_parents(_pd(K), N, d, _pi(order), _pi(pptr), len(counts), R,
                                         _pi(members), _pi(team_ptr), _pi(rep_token))
    if M < 0:
        raise ValueError("oracle_build_teams_parents rejected its arguments")
    return Teams(members, team_ptr[:M + 1].copy(), rep_token[:M].copy())


# --------------------------------------------------------------------------
# K-means parents (Alg. "Global minibatch k-means parent partition")
# --------------------------------------------------------------------------
@dataclasses.dataclass
class KMeansSettings:
    """theta of the paper's reported runs (minibatch 4096, at most 100
    iterations, 10-minibatch no-improvement rule, reassignment ratio 0.01,
    default seeding sample) and the seed xi = 0."""
    batch: int = 4096
    max_iter: int = 100
    max_no_improvement: int = 10
    reassignment_ratio: float = 0.01
    init_size: int = 0
    seed: int = 0


def kmeans_parent_count(N: int, P: int) -> int:
    """M_parent = min(N, max(2, floor(N / P))) (N >= 2)."""
    if N < 2 or P < 1:
        raise ValueError("k-means parents need N >= 2 and P >= 1")
    return min(N, max(2, N // P))


@dataclasses.dataclass
class KMeansResult:
    labels: np.ndarray        # [N] nearest final center of every token
    centers: np.ndarray       # [M, d] final centers
    init_centers: np.ndarray  # [M, d] the seeding result
    steps: int                # minibatch steps run


def kmeans(X: np.ndarray, M: int, theta: KMeansSettings = KMeansSettings()) -> KMeansResult:
    X = _f64(X)
    N, d = X.shape
    centers = np.empty((M, d))
    init = np.empty((M, d))
    labels = np.empty(N, np.int32)
    steps = np.zeros(1, np.int32)
    rc = lib().oracle_kmeans(_pd(X), N, d, M, theta.batch, theta.max_iter, theta.max_no_improvement,
                             float(theta.reassignment_ratio), theta.init_size, int(theta.seed),
                             _pd(centers), _pi(labels), _pi(steps), _pd(init))
    if rc != 0:
        raise ValueError("oracle_kmeans rejected its arguments")
    return KMeansResult(labels, centers, init, int(steps[0]))


def kmeans_parents(K: np.ndarray, P: int, theta: KMeansSettings = KMeansSettings()) -> KMeansResult:
    """Parents of one KV head's prompt keys ``[N, d]``: k-means with
    M_parent centers; ``labels`` define the parents."""
    K = _f64(K)
    return kmeans(K, kmeans_parent_count(K.shape[0], P), theta)


def build_all(K: np.ndarray, P: int, R: int) -> List[List[Teams]]:
    """``K`` is ``[B, Hkv, N, d]``; returns teams[b][kv]."""
    return [[build_teams(K[b, kv], P, R) for kv in range(K.shape[1])] for b in range(K.shape[0])]


# --------------------------------------------------------------------------
# Decode: one query head, or a whole [B, Hq] step
# --------------------------------------------------------------------------
@dataclasses.dataclass
class HeadResult:
    out: np.ndarray        # [d] attention output o^ = U^ / Z^
    U: np.ndarray          # [d] U^ in the shifted scale
    Z: float               # Z^ in the shifted scale
    shift: float           # U^ e^shift and Z^ e^shift are the unshifted sums
    phi: np.ndarray        # [M] routing logits (NaN when every team is taken)
    Y: np.ndarray          # [M] perturbed routing scores (NaN likewise)
    sel: np.ndarray        # selected team ids, ascending
    c: np.ndarray          # their conditional inclusion corrections
    tau: float             # (K'+1)-th largest perturbed score, -inf if K' = M


def decode_head(q, K, V, teams: Teams, sK, sV, Kbudget: int, seed: int, step: int,
                b: int, h: int, scale: float, ref_shift: float = float("nan"),
                route_keys: Optional[np.ndarray] = None) -> HeadResult:
    """``route_keys [M, d]``: the keys the teams are routed by (default: the
    representative keys; the team means for the centroid-guided variant)."""
    q = _f64(q)
    K = _f64(K)
    V = _f64(V)
    d = q.shape[0]
    sK = _f64(sK).reshape(-1, d)
    sV = _f64(sV).reshape(-1, d)
    T = sK.shape[0]
    M = teams.M
    out = np.empty(d)
    U = np.empty(d)
    Z = np.empty(1)
    sh = np.empty(1)
    phi = np.empty(M)
    Y = np.empty(M)
    sel = np.empty(M, np.int32)
    c = np.empty(M)
    tau = np.empty(1)
    members = np.ascontiguousarray(teams.members, np.int32)
    tptr = np.ascontiguousarray(teams.team_ptr, np.int32)
    reps = np.ascontiguousarray(teams.rep_token, np.int32)
    rk = None
    if route_keys is not None:
        rk = _f64(route_keys)
        if rk.shape != (M, d):
            raise ValueError("route_keys must be [M, d]")
    ns = lib().oracle_decode_head(
        _pd(q), d, _pd(K), _pd(V), K.shape[0], _pi(members), _pi(tptr), _pi(reps),
        _pd(rk) if rk is not None else None, M,
        _pd(sK), _pd(sV), T, int(Kbudget), seed, step, b, h, float(scale), float(ref_shift),
        _pd(out), _pd(U), _pd(Z), _pd(sh), _pd(phi), _pd(Y), _pi(sel), _pd(c), _pd(tau))
    if ns < 0:
        raise ValueError("oracle_decode_head rejected its arguments")
    return HeadResult(out, U, float(Z[0]), float(sh[0]), phi, Y, sel[:ns].copy(), c[:ns].copy(),
                      float(tau[0]))


def dense_head(q, K, V, sK, sV, scale: float):
    q = _f64(q)
    d = q.shape[0]
    K = _f64(K).reshape(-1, d)
    V = _f64(V).reshape(-1, d)
    sK = _f64(sK).reshape(-1, d)
    sV = _f64(sV).reshape(-1, d)
    out = np.empty(d)
    U = np.empty(d)
    Z = np.empty(1)
    sh = np.empty(1)
    rc = lib().oracle_dense_head(_pd(q), d, _pd(K), _pd(V), K.shape[0], _pd(sK), _pd(sV),
                                 sK.shape[0], float(scale), _pd(out), _pd(U), _pd(Z), _pd(sh))
    if rc != 0:
        raise ValueError("oracle_dense_head rejected its arguments")
    return out, U, float(Z[0]), float(sh[0])


@dataclasses.dataclass
class StepResult:
    out: np.ndarray                 # [B, Hq, d]
    heads: List[List[HeadResult]]   # [b][h]


def decode(q, K, V, sK, sV, teams, Kbudget: int, seed: int, step: int, scale: float,
           heads: Optional[List[tuple]] = None, route_keys=None) -> StepResult:
    """Alg. 1 for every (b, h) (or only the listed ``heads`` pairs).

    ``q [B,Hq,d]``, ``K,V [B,Hkv,N,d]``, ``sK,sV [B,Hkv,T,d]`` hold exact
    values (any float dtype); ``teams[b][kv]`` from :func:`build_all`.
    Query head h reads KV head ``h // (Hq // Hkv)``.
    """
    B, Hq, d = q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    out = np.full((B, Hq, d), np.nan)
    res = [[None] * Hq for _ in range(B)]
    pairs = heads if heads is not None else [(b, h) for b in range(B) for h in range(Hq)]
    cache = {}
    for (b, h) in pairs:
        kv = h // G
        if (b, kv) not in cache:
            cache = {(b, kv): (_f64(K[b, kv]), _f64(V[b, kv]), _f64(sK[b, kv]), _f64(sV[b, kv]))}
        Kb, Vb, sKb, sVb = cache[(b, kv)]
        r = decode_head(q[b, h], Kb, Vb, teams[b][kv], sKb, sVb, Kbudget, seed, step, b, h, scale,
                        route_keys=None if route_keys is None else route_keys[b][kv])
        out[b, h] = r.out
        res[b][h] = r
    return StepResult(out, res)


def dense(q, K, V, sK, sV, scale: float, heads: Optional[List[tuple]] = None) -> np.ndarray:
    B, Hq, d = q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    out = np.full((B, Hq, d), np.nan)
    pairs = heads if heads is not None else [(b, h) for b in range(B) for h in range(Hq)]
    for (b, h) in pairs:
        kv = h // G
        out[b, h] = dense_head(q[b, h], K[b, kv], V[b, kv], sK[b, kv], sV[b, kv], scale)[0]
    return out


# --------------------------------------------------------------------------
# Logical KV-access counter (eq. qwen-logical-access)
# --------------------------------------------------------------------------
# --------------------------------------------------------------------------
# Routing keys of the centroid-guided variant and the KL routing diagnostic
# (section "Attention-distribution diagnostic", appendix "Dense-trajectory KL
# and task-variant evaluation", eq. diagnostic-kl)
# --------------------------------------------------------------------------
def team_means(K: np.ndarray, teams: Teams) -> np.ndarray:
    """``[M, d]`` arithmetic mean of each team's keys (fp64; per dimension the
    members are summed in team order, then divided by n_g)."""
    K = _f64(K)
    d = K.shape[1]
    out = np.empty((teams.M, d))
    members = np.ascontiguousarray(teams.members, np.int32)
    tptr = np.ascontiguousarray(teams.team_ptr, np.int32)
    if lib().oracle_team_means(_pd(K), d, _pi(members), _pi(tptr), teams.M, _pd(out)) != 0:
        raise ValueError("oracle_team_means rejected its arguments")
    return out


_BF16_MAX = float(np.array([0x7F7F0000], np.uint32).view(np.float32)[0])
_BF16_OVERFLOW = _BF16_MAX + 2.0 ** (127 - 8)  # halfway to the next binade: rounds to inf


def round_to_bf16(x) -> np.ndarray:
    """Each fp64 value rounded to the nearest bf16 value, ties to an even
    significand (round-to-nearest-even), returned as fp64 values.

    The nearest bf16 lies within one bf16 step of the bf16 truncation of the
    value's nearest fp32; of those three candidates the nearest is taken (the
    distances are exact: each candidate is within a factor of two of x)."""
    x = _f64(x)
    with np.errstate(invalid="ignore", over="ignore"):
        f = x.astype(np.float32).view(np.uint32).astype(np.int64)
        t = f & 0xFFFF0000
        cand = np.stack([t - 0x10000, t, t + 0x10000]) & 0xFFFFFFFF
        cv = cand.astype(np.uint32).view(np.float32).astype(np.float64)
    dist = np.where(np.isfinite(cv), np.abs(cv - x[None]), np.inf)
    best = np.argmin(dist, axis=0)
    bd = np.take_along_axis(dist, best[None], 0)[0]
    tied = (dist == bd[None]) & np.isfinite(dist)
    even = ((cand >> 16) & 1) == 0
    # among tied candidates prefer the even one (at most two can tie)
    pick = np.where(tied.sum(0) > 1, np.argmax(tied & even, axis=0), best)
    out = np.take_along_axis(cv, pick[None], 0)[0]
    out = np.where(np.abs(x) >= _BF16_OVERFLOW, np.copysign(np.inf, x), out)
    out = np.where(np.isnan(x), np.nan, out)
    return np.where(x == 0, x, out)


def routing_keys(K: np.ndarray, teams: Teams, kind: str, dtype: str) -> np.ndarray:
    """``[M, d]`` keys the teams are routed by: ``"representative"`` (the
    representative's key) or ``"centroid"`` (the team mean, stored in the
    cache's element type: rounded to nearest-even bf16, or to fp32)."""
    K = _f64(K)
    if kind == "representative":
        return K[teams.rep_token]
    if kind != "centroid":
        raise ValueError(kind)
    m = team_means(K, teams)
    if dtype == "bf16":
        return round_to_bf16(m)
    return m.astype(np.float32).astype(np.float64)


def _logsumexp(v: np.ndarray) -> float:
    mx = np.max(v)
    return float(mx + np.log(np.sum(np.exp(v - mx))))


def routing_kl(q, K, teams: Teams, route_keys, scale: float) -> float:
    """eq. diagnostic-kl for one query head: KL(p || q) in nats, with p the
    dense attention over the N prompt tokens and q_i = P(g(i)) / n_g(i), where
    P is the softmax over teams of log n_g + scale q . key_g."""
    q = _f64(q)
    K = _f64(K)
    s = scale * (K @ q)
    logp = s - _logsumexp(s)
    n = teams.sizes.astype(np.float64)
    phi = np.log(n) + scale * (_f64(route_keys) @ q)
    logP = phi - _logsumexp(phi)
    group = np.empty(K.shape[0], np.int64)
    for g in range(teams.M):
        group[teams.members[teams.team_ptr[g]:teams.team_ptr[g + 1]]] = g
    logq = logP[group] - np.log(n[group])
    return float(np.sum(np.exp(logp) * (logp - logq)))


def union_rows(teams: Teams, selections) -> int:
    """Prompt rows read for one KV head: the union of the selected teams of
    the query heads sharing it (teams are disjoint, so sizes add)."""
    u = set()
    for s in selections:
        u.update(int(g) for g in s)
    sizes = teams.sizes
    return int(sum(int(sizes[g]) for g in u))


def access_counts(step: StepResult, teams, Hkv: int, T: int, Kbudget: int):
    """Per (b, kv): (m, u, e, N) of the counter; m = 0 when every team is
    taken (no routing pass is needed then)."""
    B = len(step.heads)
    Hq = len(step.heads[0])
    G = Hq // Hkv
    rows = []
    for b in range(B):
        for kv in range(Hkv):
            tm = teams[b][kv]
            sels = [step.heads[b][h].sel for h in range(kv * G, (kv + 1) * G)]
            m = tm.M if min(Kbudget, tm.M) < tm.M else 0
            rows.append((m, union_rows(tm, sels), T, int(tm.team_ptr[-1]) + T))
    return rows


def kv_access_fraction(counts) -> float:
    num = sum(m + 2 * (u + e) for (m, u, e, _) in counts)
    den = sum(2 * n for (_, _, _, n) in counts)
    return num / den


def rel_l2(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def scale_for(d: int) -> float:
    return 1.0 / math.sqrt(d)
