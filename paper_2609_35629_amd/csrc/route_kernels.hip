// Routing, sampling and the GQA read plan of one decode step.
//
// k_route   eq. method-routing: phi_g = log n_g + scale q.l_g for every query
//           head sharing the KV head (one representative load serves all of
//           them), plus the Gumbel perturbation Y_g = phi_g + G_g.  The dot
//           products accumulate in fp64 (every bf16 x fp32 product is exact in
//           fp64), so phi differs from an fp64 reference only by summation
//           order.
// k_select  Gumbel-top-K per query head: tau = the (K+1)-th largest Y (radix
//           select over order-preserving 64-bit keys), S = the K largest
//           (ties to the lower team index), log c_g for g in S
//           (eq. method-inclusion); then the union of the heads' selections
//           per KV head with an 8-bit head mask and per-head log c, the row
//           prefix of the union, and the row map the attention kernel reads:
//           for each union row its packed row and its union slot.
#include <math.h>

#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

constexpr int kRouteThreads = 256;
constexpr int kRouteGroups = kRouteThreads / 16;  // 16 lanes per representative
constexpr int kRouteTeamsPerBlock = kRouteGroups;  // one representative per lane group
constexpr int kSelectThreads = 512;
constexpr int kSelectWaves = kSelectThreads / kWave;

template <typename T, int DPL>
struct RepChunk;

template <>
struct RepChunk<bf16_t, 8> {
    using raw = uint4;
    static __device__ __forceinline__ raw load(const bf16_t* p) {
        return *reinterpret_cast<const uint4*>(p);
    }
    static __device__ __forceinline__ float get(const raw& r, int e) {
        const uint32_t w = (e < 2) ? r.x : (e < 4) ? r.y : (e < 6) ? r.z : r.w;
        return (e & 1) ? bf16hi(w) : bf16lo(w);
    }
};

template <>
struct RepChunk<bf16_t, 4> {
    using raw = uint2;
    static __device__ __forceinline__ raw load(const bf16_t* p) {
        return *reinterpret_cast<const uint2*>(p);
    }
    static __device__ __forceinline__ float get(const raw& r, int e) {
        const uint32_t w = (e < 2) ? r.x : r.y;
        return (e & 1) ? bf16hi(w) : bf16lo(w);
    }
};

template <>
struct RepChunk<float, 8> {
    struct raw {
        float4 a, b;
    };
    static __device__ __forceinline__ raw load(const float* p) {
        raw r;
        r.a = *reinterpret_cast<const float4*>(p);
        r.b = *reinterpret_cast<const float4*>(p + 4);
        return r;
    }
    static __device__ __forceinline__ float get(const raw& r, int e) {
        const float4& v = (e < 4) ? r.a : r.b;
        const int k = e & 3;
        return k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w;
    }
};

template <>
struct RepChunk<float, 4> {
    using raw = float4;
    static __device__ __forceinline__ raw load(const float* p) {
        return *reinterpret_cast<const float4*>(p);
    }
    static __device__ __forceinline__ float get(const raw& r, int e) {
        return e == 0 ? r.x : e == 1 ? r.y : e == 2 ? r.z : r.w;
    }
};

template <typename T, int D, int G>
__global__ __launch_bounds__(kRouteThreads) void k_route(
    const T* __restrict__ reps, const double* __restrict__ log_n, const float* __restrict__ q,
    int M, int Hkv, int Hq, double scale, uint64_t seed, uint64_t step, double* __restrict__ phi,
    double* __restrict__ Y) {
    constexpr int DPL = D / 16;
    using Chunk = RepChunk<T, DPL>;
    __shared__ double s_gum[G][kRouteTeamsPerBlock];
    const int bh = blockIdx.y;
    const int b = bh / Hkv, kv = bh - b * Hkv;
    const int tid = threadIdx.x, grp = tid >> 4, sub = tid & 15;
    const int g0 = blockIdx.x * kRouteTeamsPerBlock;

    // 1) every load of the block is issued first: one representative per
    //    16-lane group (clamped in range), its log n, this lane's query dims
    const int gmine = min(g0 + grp, M - 1);
    const typename Chunk::raw raw =
        Chunk::load(reps + (static_cast<size_t>(bh) * M + gmine) * D + sub * DPL);
    const double lnn = log_n[static_cast<size_t>(bh) * M + gmine];
    double qd[G][DPL];
    const float* qb = q + (static_cast<size_t>(b) * Hq + kv * G) * D + sub * DPL;
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < DPL; ++e) qd[h][e] = static_cast<double>(qb[h * D + e]);

    // 2) the Gumbel noise does not depend on the loads: one (head, team)
    //    draw per thread while they are in flight
    for (int p = tid; p < G * kRouteTeamsPerBlock; p += kRouteThreads) {
        const int h = p / kRouteTeamsPerBlock, gi = p - h * kRouteTeamsPerBlock;
        const int g = g0 + gi;
        if (g < M) s_gum[h][gi] = team_gumbel(seed, step, b, kv * G + h, g);
    }
    __syncthreads();

    // 3) fp64 dot products of the representative with the G queries
    const int g = g0 + grp;
    if (g >= M) return;  // uniform across the 16-lane group; no barrier follows
    double acc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        double a = 0.0;
#pragma unroll
        for (int e = 0; e < DPL; ++e) a = fma(qd[h][e], static_cast<double>(Chunk::get(raw, e)), a);
        acc[h] = row16_sum(a);
    }
    if (sub < G) {
        double dot = 0.0;
#pragma unroll
        for (int h = 0; h < G; ++h)
            if (h == sub) dot = acc[h];
        const double ph = lnn + scale * dot;
        const size_t o = (static_cast<size_t>(b) * Hq + kv * G + sub) * M + g;
        phi[o] = ph;
        Y[o] = ph + s_gum[sub][grp];
    }
}

// log c for c = 1 - exp(-exp(x)) in fp32 (eq. method-inclusion).  x >= -37
// for a selected team (its perturbed score beats tau and a Gumbel draw is at
// most 53 log 2), so e^x stays a normal fp32.  For e^x < 1/16 a four-term
// series avoids the cancellation of 1 - exp(-e); its truncation error is below
// e^4 / 120 relative.
__device__ __forceinline__ float log_inclusion(float x) {
    constexpr float kL2e = 1.4426950408889634f, kLn2 = 0.6931471805599453f;
    const float e = __builtin_amdgcn_exp2f(x * kL2e);
    const float c = (e < 0.0625f)
                        ? e * (1.f - e * (0.5f - e * (1.f / 6.f - e * (1.f / 24.f))))
                        : 1.f - __builtin_amdgcn_exp2f(-e * kL2e);
    return __builtin_amdgcn_logf(c) * kLn2;
}

// Exclusive scan of two counters over the workgroup; returns the totals.
__device__ __forceinline__ void block_scan2(int a, int c, int& ea, int& ec, int& ta, int& tc,
                                            int* s_w /* [2 * kSelectWaves] */) {
    const int lane = lane_id(), w = wave_id();
    const int ia = wave_incl_scan(a), ic = wave_incl_scan(c);
    if (lane == kWave - 1) {
        s_w[w] = ia;
        s_w[kSelectWaves + w] = ic;
    }
    __syncthreads();
    int pa = 0, pc = 0;
    ta = 0;
    tc = 0;
#pragma unroll
    for (int v = 0; v < kSelectWaves; ++v) {
        const int xa = s_w[v], xc = s_w[kSelectWaves + v];
        if (v < w) {
            pa += xa;
            pc += xc;
        }
        ta += xa;
        tc += xc;
    }
    ea = pa + ia - a;
    ec = pc + ic - c;
    __syncthreads();
}

// The perturbed scores of one head, as order-preserving keys.  PL > 0 keeps
// element i = j * 64 + lane in register j (M <= 64 * PL); PL == 0 re-reads
// them from global memory on every pass.
template <int PL>
struct KeySet {
    uint64_t k[PL];
    double ph[PL];
    const double* y;
    const double* p;
    int M;
    // every load is issued before the first use (clamped addresses, no branch)
    __device__ __forceinline__ void init(const double* yy, const double* pp, int MM) {
        y = yy;
        p = pp;
        M = MM;
        const int lane = lane_id();
        double v[PL];
#pragma unroll
        for (int j = 0; j < PL; ++j) {
            const int i = min(j * kWave + lane, M - 1);
            v[j] = y[i];
            ph[j] = p[i];
        }
#pragma unroll
        for (int j = 0; j < PL; ++j) k[j] = order_key(v[j]);
    }
    __device__ __forceinline__ int count() const { return PL; }
    __device__ __forceinline__ bool valid(int j) const { return j * kWave + lane_id() < M; }
    __device__ __forceinline__ uint64_t key(int j) const { return k[j]; }
    __device__ __forceinline__ double phi(int j) const { return ph[j]; }
};

template <>
struct KeySet<0> {
    const double* y;
    const double* p;
    int M;
    __device__ __forceinline__ void init(const double* yy, const double* pp, int MM) {
        y = yy;
        p = pp;
        M = MM;
    }
    __device__ __forceinline__ int count() const { return (M + kWave - 1) / kWave; }
    __device__ __forceinline__ bool valid(int j) const { return j * kWave + lane_id() < M; }
    __device__ __forceinline__ uint64_t key(int j) const {
        return order_key(y[min(j * kWave + lane_id(), M - 1)]);
    }
    __device__ __forceinline__ double phi(int j) const { return p[j * kWave + lane_id()]; }
};

// Per-wave candidate bookkeeping of the selection: the value bucket of a key
// (monotone in the key's value) and the candidates of the current pass.
struct Buckets {
    double ymin, scale;
    __device__ __forceinline__ int of(uint64_t k) const {
        const double t = (key_value(k) - ymin) * scale;
        return min(255, static_cast<int>(t));
    }
};

// Rank `want` (0-based, descending) among the lane bins of one LDS histogram:
// lane l owns bins 255 - 4 l .. 252 - 4 l.  Returns the bin, and through
// `above` / `cnt` the candidates in higher bins and in the bin itself.
__device__ __forceinline__ int hist_select(const uint32_t* hist, int want, int& above, int& cnt) {
    const int lane = lane_id();
    const uint4 hv = reinterpret_cast<const uint4*>(hist)[63 - lane];
    const int c[4] = {static_cast<int>(hv.w), static_cast<int>(hv.z), static_cast<int>(hv.y),
                      static_cast<int>(hv.x)};
    const int mine = c[0] + c[1] + c[2] + c[3];
    const int incl = wave_incl_scan(mine);
    const int ab = incl - mine;
    const bool owner = (ab <= want) && (want < incl);
    int digit = 0, cum = ab, cn = 0;
    if (owner) {
        bool done = false;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (!done && cum + c[e] > want) {
                digit = 255 - (4 * lane + e);
                cn = c[e];
                done = true;
            }
            if (!done) cum += c[e];
        }
    }
    const int src = __ffsll(static_cast<unsigned long long>(__ballot(owner))) - 1;
    above = readlane(cum, src);
    cnt = readlane(cn, src);
    return readlane(digit, src);
}

template <int PL>
__global__ __launch_bounds__(kSelectThreads) void k_select(
    const double* __restrict__ phi, const double* __restrict__ Y,
    const int* __restrict__ team_begin, const int* __restrict__ team_size, int M, int Kp,
    int Hkv, int G, int Hq, int T, int max_split, float* __restrict__ lc,
    int* __restrict__ hdr, int* __restrict__ ubeg, int* __restrict__ urs,
    float* __restrict__ ulogc, int* __restrict__ split_team, int* __restrict__ dbg_sel,
    float* __restrict__ dbg_logc, double* __restrict__ dbg_tau, int* __restrict__ dbg_uteams,
    int* __restrict__ dbg_urows) {
    // dynamic LDS: 8-bit head mask per team, then (kLdsLc) log c per head and
    // team; larger team counts keep log c in global memory
    constexpr bool kLdsLc = PL > 0 && PL <= 16;
    extern __shared__ uint32_t s_dyn[];
    const int mask_words = (M + 3) >> 2;
    uint32_t* s_mask = s_dyn;
    float* s_lc = reinterpret_cast<float*>(s_dyn + mask_words);  // [G][M] when kLdsLc
    __shared__ __align__(16) uint32_t s_hist[kSelectWaves][256];
    __shared__ uint64_t s_cand[kSelectWaves][kWave];
    __shared__ int s_w[2 * kSelectWaves];

    const int bh = blockIdx.x;
    const int b = bh / Hkv, kv = bh - b * Hkv;
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    for (int i = tid; i < mask_words; i += kSelectThreads) s_mask[i] = 0;
    // team sizes and starts of the first chunk of teams, fetched while the
    // heads select
    const size_t tb0 = static_cast<size_t>(bh) * M;
    const int gc0 = min(tid, M - 1);
    const int size0 = team_size[tb0 + gc0];
    const int begin0 = team_begin[tb0 + gc0];
    __syncthreads();

    if (w < G) {
        const int hq = kv * G + w;
        const size_t hoff = (static_cast<size_t>(b) * Hq + hq) * M;
        KeySet<PL> ks;
        ks.init(Y + hoff, phi + hoff, M);
        const int nj = ks.count();
        uint32_t* hist = s_hist[w];
        int want = Kp;  // rank of tau among the keys, 0-based from the top
        uint64_t tkey = 0;

        // pass 1: 256 value buckets over [min Y, max Y]
        uint64_t kmin = ~0ull, kmax = 0;
#pragma unroll
        for (int j = 0; j < nj; ++j) {
            if (ks.valid(j)) {
                kmin = min(kmin, ks.key(j));
                kmax = max(kmax, ks.key(j));
            }
        }
        kmin = wave_min64(kmin);
        kmax = wave_max64(kmax);
        Buckets bk;
        bk.ymin = key_value(kmin);
        const double range = key_value(kmax) - bk.ymin;
        bool found = !(range > 0.0);  // every key equal
        if (found) tkey = kmin;
        bk.scale = found ? 0.0 : 255.999 / range;
        int bucket = -1;
        if (!found) {
            reinterpret_cast<uint4*>(hist)[lane] = make_uint4(0, 0, 0, 0);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int j = 0; j < nj; ++j)
                if (ks.valid(j)) atomicAdd(&hist[bk.of(ks.key(j))], 1u);
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            __builtin_amdgcn_wave_barrier();
            int above, cnt;
            bucket = hist_select(hist, want, above, cnt);
            want -= above;
            if (cnt <= kWave) {
                // few candidates left: gather them and rank them directly
                const uint64_t lt = lanemask_lt();
                int n = 0;
#pragma unroll
                for (int j = 0; j < nj; ++j) {
                    const bool cand = ks.valid(j) && bk.of(ks.key(j)) == bucket;
                    const uint64_t cb = __ballot(cand);
                    if (cand) s_cand[w][n + __popcll(cb & lt)] = ks.key(j);
                    n += __popcll(cb);
                }
                __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                __builtin_amdgcn_wave_barrier();
                const uint64_t mine = s_cand[w][min(lane, n - 1)];
                int gt = 0, ge = 0;
                for (int t = 0; t < n; ++t) {
                    const uint64_t o = s_cand[w][t];
                    gt += o > mine ? 1 : 0;
                    ge += o >= mine ? 1 : 0;
                }
                const bool owner = lane < n && gt <= want && want < ge;
                tkey = readlane(mine, __ffsll(static_cast<unsigned long long>(__ballot(owner))) - 1);
                found = true;
            }
        }
        if (!found) {
            // many equal-bucket keys: exact radix over their 64-bit keys
            uint64_t kand = ~0ull, kor = 0;
#pragma unroll
            for (int j = 0; j < nj; ++j) {
                if (ks.valid(j) && bk.of(ks.key(j)) == bucket) {
                    kand &= ks.key(j);
                    kor |= ks.key(j);
                }
            }
            const uint64_t all_and = wave_and64(kand), all_or = wave_or64(kor);
            const uint64_t diff = all_or & ~all_and;
            uint64_t prefix = 0, pmask = 0;
            const int top = diff ? 63 - __clzll(static_cast<long long>(diff)) : 7;
            int shift = top >= 7 ? top - 7 : 0;
            if (shift + 8 < 64) {
                pmask = ~0ull << (shift + 8);
                prefix = all_and & pmask;
            }
            for (; !found; shift -= 8) {
                reinterpret_cast<uint4*>(hist)[lane] = make_uint4(0, 0, 0, 0);
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
#pragma unroll
                for (int j = 0; j < nj; ++j) {
                    const uint64_t k = ks.key(j);
                    if (ks.valid(j) && bk.of(k) == bucket && (k & pmask) == prefix)
                        atomicAdd(&hist[(k >> shift) & 255], 1u);
                }
                __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                __builtin_amdgcn_wave_barrier();
                int above, cnt;
                const int digit = hist_select(hist, want, above, cnt);
                want -= above;
                prefix |= static_cast<uint64_t>(digit) << shift;
                pmask |= 0xffull << shift;
                if (cnt == 1 || shift == 0) {
                    // the rank element is determined: fetch one key equal to it
                    uint64_t kk = 0;
                    bool have = false;
#pragma unroll
                    for (int j = 0; j < nj; ++j) {
                        const uint64_t k = ks.key(j);
                        if (ks.valid(j) && bk.of(k) == bucket && (k & pmask) == prefix) {
                            kk = k;
                            have = true;
                        }
                    }
                    tkey = readlane(kk, __ffsll(static_cast<unsigned long long>(__ballot(have))) - 1);
                    found = true;
                }
                if (shift < 8) shift = 8;  // the last digit may overlap earlier bits
            }
        }
        const double tau = key_value(tkey);

        int above_cnt = 0;
#pragma unroll
        for (int j = 0; j < nj; ++j) above_cnt += (ks.valid(j) && ks.key(j) > tkey) ? 1 : 0;
        const int need_ties = Kp - wave_sum(above_cnt);

        // log c of every key in flight at once (independent chains), then
        // the selection in index order: i = j * 64 + lane
        float lcv[PL > 0 ? PL : 1];
#pragma unroll
        for (int j = 0; j < (PL > 0 ? PL : 0); ++j)
            lcv[j] = log_inclusion(static_cast<float>(ks.phi(j) - tau));
        const uint64_t lt = lanemask_lt();
        int nsel = 0, nties = 0;
#pragma unroll
        for (int j = 0; j < nj; ++j) {
            const int i = j * kWave + lane;
            const bool valid = ks.valid(j);
            const uint64_t k = ks.key(j);
            const bool tie = valid && k == tkey;
            const uint64_t tb = __ballot(tie);
            const int trank = nties + __popcll(tb & lt);
            nties += __popcll(tb);
            const bool sel = valid && (k > tkey || (tie && trank < need_ties));
            const uint64_t sb = __ballot(sel);
            const int pos = nsel + __popcll(sb & lt);
            nsel += __popcll(sb);
            if (sel) {
                float v;
                if constexpr (PL > 0)
                    v = lcv[j];
                else
                    v = log_inclusion(static_cast<float>(ks.phi(j) - tau));
                if constexpr (kLdsLc)
                    s_lc[w * M + i] = v;
                else
                    lc[hoff + i] = v;
                atomicOr(&s_mask[i >> 2], 1u << ((i & 3) * 8 + w));
                if (pos < Kp) {
                    if (dbg_sel) dbg_sel[(static_cast<size_t>(b) * Hq + hq) * Kp + pos] = i;
                    if (dbg_logc) dbg_logc[(static_cast<size_t>(b) * Hq + hq) * Kp + pos] = v;
                }
            }
        }
        if (lane == 0 && dbg_tau) dbg_tau[static_cast<size_t>(b) * Hq + hq] = tau;
    }
    __syncthreads();

    // union of the heads' selections in ascending team order, its row prefix,
    // and the first union team of every kSplitRows-row range of the rows
    int* sp = split_team + static_cast<size_t>(bh) * max_split;
    const size_t rs0 = static_cast<size_t>(bh) * (M + 1);
    int run_u = 0, run_rows = 0;
    for (int base = 0; base < M; base += kSelectThreads) {
        const int g = base + tid;
        int tsz = size0, tbeg = begin0;
        if (base > 0) {
            const int gc = min(g, M - 1);
            tsz = team_size[tb0 + gc];
            tbeg = team_begin[tb0 + gc];
        }
        const uint32_t m = (g < M) ? ((s_mask[g >> 2] >> ((g & 3) * 8)) & 0xffu) : 0u;
        const int f = m ? 1 : 0;
        const int sz = f ? tsz : 0;
        int ef, es, tf, ts;
        block_scan2(f, sz, ef, es, tf, ts, s_w);
        if (f) {
            const int slot = run_u + ef, rs = run_rows + es;
            float v[kLogcStride];
#pragma unroll
            for (int h = 0; h < kLogcStride; ++h) {
                const int hc = min(h, G - 1);
                if constexpr (kLdsLc)
                    v[h] = s_lc[hc * M + g];
                else
                    v[h] = lc[(static_cast<size_t>(b) * Hq + kv * G + hc) * M + g];
            }
#pragma unroll
            for (int h = 0; h < kLogcStride; ++h)
                if (!(h < G && ((m >> h) & 1u))) v[h] = 1.0e30f;  // no weight for this head
            float4* L = reinterpret_cast<float4*>(ulogc + (tb0 + slot) * kLogcStride);
            L[0] = make_float4(v[0], v[1], v[2], v[3]);
            L[1] = make_float4(v[4], v[5], v[6], v[7]);
            ubeg[tb0 + slot] = tbeg;
            urs[rs0 + slot] = rs;
            // row ranges whose first row falls inside this team
            for (int r = (rs + kSplitRows - 1) / kSplitRows * kSplitRows; r < rs + tsz; r += kSplitRows)
                sp[r / kSplitRows] = slot;
        }
        run_u += tf;
        run_rows += ts;
    }
    // ranges that start in the suffix
    const int nsp = (run_rows + T + kSplitRows - 1) / kSplitRows;
    for (int q0 = (run_rows + kSplitRows - 1) / kSplitRows + tid; q0 < nsp; q0 += kSelectThreads)
        sp[q0] = run_u;
    if (tid == 0) {
        urs[rs0 + run_u] = run_rows;
        hdr[bh * 4 + 0] = run_u;
        hdr[bh * 4 + 1] = run_rows;
        if (dbg_uteams) dbg_uteams[bh] = run_u;
        if (dbg_urows) dbg_urows[bh] = run_rows;
    }
}

template <typename T, int D>
hipError_t route_dispatch_d(const RouteArgs& a, hipStream_t s) {
    const dim3 grid((a.M + kRouteTeamsPerBlock - 1) / kRouteTeamsPerBlock, a.B * a.Hkv);
    double* phi = reinterpret_cast<double*>(a.ws + a.lay->phi);
    double* Y = reinterpret_cast<double*>(a.ws + a.lay->Y);
    const T* reps = static_cast<const T*>(a.reps);
#define SANTAPP_ROUTE(GG)                                                                  \
    k_route<T, D, GG><<<grid, kRouteThreads, 0, s>>>(reps, a.log_n, a.q, a.M, a.Hkv, a.Hq,  \
                                                      a.scale, a.seed, a.step, phi, Y)
    switch (a.G) {
        case 1: SANTAPP_ROUTE(1); break;
        case 2: SANTAPP_ROUTE(2); break;
        case 3: SANTAPP_ROUTE(3); break;
        case 4: SANTAPP_ROUTE(4); break;
        case 5: SANTAPP_ROUTE(5); break;
        case 6: SANTAPP_ROUTE(6); break;
        case 7: SANTAPP_ROUTE(7); break;
        case 8: SANTAPP_ROUTE(8); break;
        default: return hipErrorInvalidValue;
    }
#undef SANTAPP_ROUTE
    return hipGetLastError();
}

template <typename T>
hipError_t route_dispatch(const RouteArgs& a, hipStream_t s) {
    switch (a.d) {
        case 64: return route_dispatch_d<T, 64>(a, s);
        case 128: return route_dispatch_d<T, 128>(a, s);
        default: return hipErrorInvalidValue;
    }
}

template <int PL>
void select_launch(const RouteArgs& a, hipStream_t s) {
    size_t lds = sizeof(uint32_t) * ((a.M + 3) / 4);
    if (PL > 0 && PL <= 16) lds += sizeof(float) * static_cast<size_t>(a.G) * a.M;
    const santapp_decode_debug* d = a.dbg;
    const DecodeLayout& L = *a.lay;
    k_select<PL><<<a.B * a.Hkv, kSelectThreads, lds, s>>>(
        reinterpret_cast<const double*>(a.ws + L.phi), reinterpret_cast<const double*>(a.ws + L.Y),
        a.team_begin, a.team_size, a.M, a.Kp, a.Hkv, a.G, a.Hq, a.T, L.max_split,
        reinterpret_cast<float*>(a.ws + L.lc), reinterpret_cast<int*>(a.ws + L.hdr),
        reinterpret_cast<int*>(a.ws + L.ubeg), reinterpret_cast<int*>(a.ws + L.urs),
        reinterpret_cast<float*>(a.ws + L.ulogc), reinterpret_cast<int*>(a.ws + L.split),
        d ? d->sel : nullptr, d ? d->logc : nullptr, d ? d->tau : nullptr,
        d ? d->union_teams : nullptr, d ? d->union_rows : nullptr);
}

}  // namespace

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
    return a.dtype == SANTAPP_BF16 ? route_dispatch<bf16_t>(a, s) : route_dispatch<float>(a, s);
}

hipError_t launch_select(const RouteArgs& a, hipStream_t s) {
    if (a.M <= 8 * kWave)
        select_launch<8>(a, s);
    else if (a.M <= 16 * kWave)
        select_launch<16>(a, s);
    else if (a.M <= 32 * kWave)
        select_launch<32>(a, s);
    else
        select_launch<0>(a, s);
    return hipGetLastError();
}

}  // namespace santapp
