// Routing, sampling and the GQA read plan of one decode step.
//
// k_route   eq. method-routing: phi_g = log n_g + scale q.l_g for every query
//           head sharing the KV head (one representative load serves all of
//           them), and the Gumbel perturbation Y_g = phi_g + G_g.  The dot
//           products accumulate in fp64 (every bf16 x fp32 product is exact
//           in fp64), so phi differs from an fp64 reference only by summation
//           order.
// k_select  Alg. "SANTA++ attention for one query head", eq.
//           method-inclusion, one workgroup per (sequence, KV head): one wave
//           per query head finds tau = the (K+1)-th largest Y with a
//           two-level value histogram and an exact finish over the
//           order-preserving 64-bit keys, selects the K largest (ties to the
//           lower team index) and computes log c_g for the selected teams.
//           Then the read plan: the union of the heads' selections in
//           ascending team order with each team's per-head corrections, cut
//           into chunks of at most kChunkRows consecutive packed rows (each
//           chunk is one unit of attention work), followed by the chunks of
//           the exactly attended suffix.  Each (sequence, KV head) pair owns a
//           fixed region of the unit list, so the plan needs no global
//           atomics.
// k_select_head  past 2048 teams per KV head: the head waves' part of
//           k_select by one workgroup per query head (the head's scores no
//           longer fit one wave's registers); k_select then only builds the
//           plan from the heads' results.
#include <math.h>

#include <atomic>
#include <type_traits>

#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

constexpr int kRouteThreads = 256;
constexpr int kRouteTeams = kRouteThreads / 16;  // one representative per 16-lane group
constexpr int kSelectThreads = 512;
constexpr int kSelectWaves = kSelectThreads / kWave;
constexpr int kFineBits = 16;                 // value-histogram resolution of the sampler
constexpr int kSelectUnits = 4096;            // units of a plan pass resolved through an LDS table
constexpr int kSelectRecs = 2048;             // union teams of a plan pass (M <= 2048: one pass)

template <typename T, int DPL>
struct RepChunk;

template <>
struct RepChunk<bf16_t, 8> {
    using raw = uint4;
    static __device__ __forceinline__ raw load(const bf16_t* p) { return load_stream(p); }
    static __device__ __forceinline__ float get(const raw& r, int e) {
        const uint32_t w = (e < 2) ? r.x : (e < 4) ? r.y : (e < 6) ? r.z : r.w;
        return (e & 1) ? bf16hi(w) : bf16lo(w);
    }
};

template <>
struct RepChunk<bf16_t, 4> {
    using raw = uint2;
    static __device__ __forceinline__ raw load(const bf16_t* p) { return load_stream8(p); }
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
        r.a = load_stream_f(p);
        r.b = load_stream_f(p + 4);
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
    static __device__ __forceinline__ raw load(const float* p) { return load_stream_f(p); }
    static __device__ __forceinline__ float get(const raw& r, int e) {
        return e == 0 ? r.x : e == 1 ? r.y : e == 2 ? r.z : r.w;
    }
};

// Value-histogram bucket of a key in [0, 2^kFineBits): keys below the range
// (absent teams) land in bucket 0.
__device__ __forceinline__ int fine_bucket(double y, double ymin, double fs) {
    return static_cast<int>(fmin(static_cast<double>((1 << kFineBits) - 1), fmax(0.0, (y - ymin) * fs)));
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

// Exclusive scan of NV counters over the workgroup; returns the totals.
// s_w holds NV x kSelectWaves wave totals.
template <int NV>
__device__ __forceinline__ void block_scan(const int (&x)[NV], int (&ex)[NV], int (&tot)[NV],
                                           int* s_w /* [NV * kSelectWaves] */) {
    static_assert(kSelectWaves == 8, "wave totals are read as two int4 per counter");
    const int lane = lane_id(), w = wave_id();
    int inc[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        inc[k] = wave_incl_scan(x[k]);
        if (lane == kWave - 1) s_w[k * kSelectWaves + w] = inc[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int4 a = reinterpret_cast<const int4*>(s_w)[2 * k];
        const int4 c = reinterpret_cast<const int4*>(s_w)[2 * k + 1];
        const int y[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
        int pre = 0, t = 0;
#pragma unroll
        for (int v = 0; v < kSelectWaves; ++v) {
            pre += (v < w) ? y[v] : 0;
            t += y[v];
        }
        ex[k] = pre + inc[k] - x[k];
        tot[k] = t;
    }
    __syncthreads();
}

// The perturbed scores of one head as order-preserving keys, with each key's
// fine value bucket: element i = j * 64 + lane in register j (M <= 64 PL).
template <int PL>
struct KeySet {
    // phi stays in registers only for small PL; larger sets re-read it for
    // the few selected keys
    static constexpr bool kPhiRegs = PL <= 8;
    uint64_t k[PL];
    double ph[kPhiRegs ? PL : 1];
    int fine[PL];
    const double* p;
    int M;
    __device__ __forceinline__ void init(const double* y, const double* pp, int MM) {
        M = MM;
        p = pp;
        const int lane = lane_id();
        double v[PL];
        // clamped indices: no branch around the loads; the keys' loads
        // first, phi (needed only once tau is known) after them
#pragma unroll
        for (int j = 0; j < PL; ++j) v[j] = y[min(j * kWave + lane, M - 1)];
        if constexpr (kPhiRegs) {
#pragma unroll
            for (int j = 0; j < PL; ++j) ph[j] = pp[min(j * kWave + lane, M - 1)];
        }
#pragma unroll
        for (int j = 0; j < PL; ++j) k[j] = order_key(v[j]);
    }
    __device__ __forceinline__ int count() const { return PL; }
    __device__ __forceinline__ bool valid(int j) const { return j * kWave + lane_id() < M; }
    __device__ __forceinline__ uint64_t key(int j) const { return k[j]; }
    __device__ __forceinline__ double phi(int j) const {
        if constexpr (kPhiRegs)
            return ph[j];
        else
            return p[min(j * kWave + lane_id(), M - 1)];
    }
    __device__ __forceinline__ void set_fine(double ymin, double fs) {
#pragma unroll
        for (int j = 0; j < PL; ++j)
            fine[j] = fine_bucket(key_value(k[j]), ymin, fs);
    }
    __device__ __forceinline__ int fine_of(int j, double, double) const { return fine[j]; }
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

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// tau's key for one head: the key of rank `want` (0-based, descending) among
// the valid keys.  Value histograms over [min Y, max Y] at 2^16 buckets (two
// passes of 256); at most 64 candidates left are ranked directly; beyond that
// (many nearly equal keys) an exact 8-bit radix over the 64-bit keys finishes.
template <int PL>
__device__ uint64_t select_key(KeySet<PL>& ks, int want, uint32_t* hist, uint64_t* cand) {
    const int lane = lane_id();
    const int nj = ks.count();
    // the histogram spans the real teams' keys (absent teams, far below,
    // fall into bucket 0) unless those are all equal
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
    const uint64_t kreal = order_key(kAbsentBelow);
    if (kmin < kreal) {  // wave-uniform: only tables with absent teams
        uint64_t rmin = ~0ull;
#pragma unroll
        for (int j = 0; j < nj; ++j)
            if (ks.valid(j) && ks.key(j) >= kreal) rmin = min(rmin, ks.key(j));
        rmin = wave_min64(rmin);
        if (rmin < kmax) kmin = rmin;
    }
    const double ymin = key_value(kmin);
    const double range = key_value(kmax) - ymin;
    if (!(range > 0.0)) return kmin;  // every key equal
    const double fs = (static_cast<double>(1 << kFineBits) - 0.001) / range;
    ks.set_fine(ymin, fs);

    // pass 0: the top 8 bits of the fine bucket over every key; pass 1: its
    // low 8 bits over the keys of the chosen top bin.  `target` is the part
    // of the fine bucket fixed so far.
    int target = 0;
    for (int pass = 0; pass < 2; ++pass) {
        const int shift = pass == 0 ? 8 : 0;
        reinterpret_cast<uint4*>(hist)[lane] = make_uint4(0, 0, 0, 0);
        wave_lds_sync();
#pragma unroll
        for (int j = 0; j < nj; ++j) {
            const int f = ks.fine_of(j, ymin, fs);
            if (ks.valid(j) && (pass == 0 || (f >> 8) == target)) atomicAdd(&hist[(f >> shift) & 255], 1u);
        }
        wave_lds_sync();
        int above, cnt;
        const int bin = hist_select(hist, want, above, cnt);
        want -= above;
        target = pass == 0 ? bin : (target << 8) | bin;
        if (cnt <= kWave) {
            // few candidates: gather them and rank them directly
            const uint64_t lt = lanemask_lt();
            int n = 0;
#pragma unroll
            for (int j = 0; j < nj; ++j) {
                const bool c = ks.valid(j) && (ks.fine_of(j, ymin, fs) >> shift) == target;
                const uint64_t cb = __ballot(c);
                if (c) cand[n + __popcll(cb & lt)] = ks.key(j);
                n += __popcll(cb);
            }
            wave_lds_sync();
            const uint64_t mine = cand[min(lane, n - 1)];
            int gt = 0, ge = 0;
            for (int t = 0; t < n; ++t) {  // n is wave-uniform
                const uint64_t o = readlane(mine, t);
                gt += o > mine ? 1 : 0;
                ge += o >= mine ? 1 : 0;
            }
            const bool owner = lane < n && gt <= want && want < ge;
            const uint64_t r = readlane(mine, __ffsll(static_cast<unsigned long long>(__ballot(owner))) - 1);
            wave_lds_sync();  // cand is reused by the caller
            return r;
        }
    }

    // many keys in one fine bucket: exact radix over their 64-bit keys
    auto in_bucket = [&](int j) { return ks.valid(j) && ks.fine_of(j, ymin, fs) == target; };
    uint64_t kand = ~0ull, kor = 0;
#pragma unroll
    for (int j = 0; j < nj; ++j) {
        if (in_bucket(j)) {
            kand &= ks.key(j);
            kor |= ks.key(j);
        }
    }
    const uint64_t all_and = wave_and64(kand), all_or = wave_or64(kor);
    const uint64_t diff = all_or & ~all_and;
    uint64_t prefix = 0, pmask = 0;
    const int top = diff ? 63 - __clzll(static_cast<long long>(diff)) : 7;
    int sh = top >= 7 ? top - 7 : 0;
    if (sh + 8 < 64) {
        pmask = ~0ull << (sh + 8);
        prefix = all_and & pmask;
    }
    for (;;) {
        reinterpret_cast<uint4*>(hist)[lane] = make_uint4(0, 0, 0, 0);
        wave_lds_sync();
#pragma unroll
        for (int j = 0; j < nj; ++j) {
            const uint64_t k = ks.key(j);
            if (in_bucket(j) && (k & pmask) == prefix) atomicAdd(&hist[(k >> sh) & 255], 1u);
        }
        wave_lds_sync();
        int above, cnt;
        const int digit = hist_select(hist, want, above, cnt);
        want -= above;
        prefix |= static_cast<uint64_t>(digit) << sh;
        pmask |= 0xffull << sh;
        if (cnt == 1 || sh == 0) {
            // the rank element is determined: fetch one key equal to it
            uint64_t kk = 0;
            bool have = false;
#pragma unroll
            for (int j = 0; j < nj; ++j) {
                const uint64_t k = ks.key(j);
                if (in_bucket(j) && (k & pmask) == prefix) {
                    kk = k;
                    have = true;
                }
            }
            return readlane(kk, __ffsll(static_cast<unsigned long long>(__ballot(have))) - 1);
        }
        sh = sh >= 8 ? sh - 8 : 0;  // the last digit may overlap bits fixed before
    }
}

template <typename T, int D, int G>
__global__ __launch_bounds__(kRouteThreads) void k_route(
    const T* __restrict__ reps, const double* __restrict__ log_n, const float* __restrict__ q,
    int M, int Hkv, int Hq, double scale, uint64_t seed, uint64_t step, double* __restrict__ phi,
    double* __restrict__ Y) {
    constexpr int DPL = D / 16;
    using RC = RepChunk<T, DPL>;
    __shared__ double s_gum[G][kRouteTeams];
    __shared__ uint64_t s_word[G][kRouteTeams];
    const int bh = blockIdx.y;
    const int b = bh / Hkv, kv = bh - b * Hkv;
    const int tid = threadIdx.x, grp = tid >> 4, sub = tid & 15;
    const int g0 = blockIdx.x * kRouteTeams;
    const size_t tb0 = static_cast<size_t>(bh) * M;

    // every load first: one representative per 16-lane group (clamped in
    // range), its log n, this lane's query dims
    const int gmine = min(g0 + grp, M - 1);
    const typename RC::raw raw = RC::load(reps + (tb0 + gmine) * D + sub * DPL);
    const double lnn = log_n[tb0 + gmine];
    double qd[G][DPL];
    const float* qb = q + (static_cast<size_t>(b) * Hq + kv * G) * D + sub * DPL;
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < DPL; ++e) qd[h][e] = static_cast<double>(qb[h * D + e]);
    // the Gumbel noise does not depend on the loads, so it is drawn while
    // they are in flight: one Philox block per (head, 4 teams) (the block at
    // counter (g / 4, h, b, step) holds the words of teams 4 (g / 4) ..
    // + 3), then one (head, team) variate per thread from its word
    static_assert(kRouteTeams % 4 == 0, "a workgroup's teams are whole Philox blocks");
    for (int p = tid; p < G * (kRouteTeams / 4); p += kRouteThreads) {
        const int h = p / (kRouteTeams / 4), qd = p - h * (kRouteTeams / 4);
        const u64x4 r = philox4x64_10(static_cast<uint64_t>(g0 / 4 + qd), static_cast<uint64_t>(kv * G + h),
                                      static_cast<uint64_t>(b), step, seed, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e) s_word[h][4 * qd + e] = r.v[e];
    }
    __syncthreads();
    for (int p = tid; p < G * kRouteTeams; p += kRouteThreads) {
        const int h = p / kRouteTeams, gi = p - h * kRouteTeams;
        if (g0 + gi < M) s_gum[h][gi] = gumbel_of_word(s_word[h][gi]);
    }
    __syncthreads();
    const int g = g0 + grp;
    if (g >= M) return;  // uniform across the 16-lane group; no barrier follows
    double acc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        double a = 0.0;
#pragma unroll
        for (int e = 0; e < DPL; ++e) a = fma(qd[h][e], static_cast<double>(RC::get(raw, e)), a);
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

// ---------------------------------------------------------------------------
// One query head per workgroup, for team counts past the register path of
// k_select (M > 32 x 64): the same selection as k_select's head waves (tau,
// the selected teams with ties to the lower index, log c and each selected
// team's first position in the head's list), with the workgroup's 512 threads
// sharing the head's keys (kHeadKeys each).  Results go to the workspace:
// selection bits in team order (kSelWords words per head), log c and
// positions (lc, lpos) and the head's unit count; k_select<G, 0, true> then
// builds the plan.
constexpr int kHeadKeys = kMaxTeams / kSelectThreads;

template <bool kMax>
__device__ __forceinline__ uint64_t block_ext64(uint64_t v, uint64_t* s_red) {
    v = kMax ? wave_max64(v) : wave_min64(v);
    if (lane_id() == 0) s_red[wave_id()] = v;
    __syncthreads();
    uint64_t r = s_red[0];
    for (int w = 1; w < kSelectWaves; ++w) r = kMax ? max(r, s_red[w]) : min(r, s_red[w]);
    __syncthreads();
    return r;
}

template <bool kOr>
__device__ __forceinline__ uint64_t block_bits64(uint64_t v, uint64_t* s_red) {
    v = kOr ? wave_or64(v) : wave_and64(v);
    if (lane_id() == 0) s_red[wave_id()] = v;
    __syncthreads();
    uint64_t r = s_red[0];
    for (int w = 1; w < kSelectWaves; ++w) r = kOr ? (r | s_red[w]) : (r & s_red[w]);
    __syncthreads();
    return r;
}

template <int G>
__global__ __launch_bounds__(kSelectThreads) void k_select_head(
    const double* __restrict__ phi, const double* __restrict__ Y, const int* __restrict__ team_size,
    int M, int Hkv, int Hq, int Kp, float* __restrict__ lc, unsigned short* __restrict__ lpos,
    uint64_t* __restrict__ sbits, int* __restrict__ hunits, int* __restrict__ dbg_sel,
    float* __restrict__ dbg_logc, double* __restrict__ dbg_tau) {
    __shared__ __align__(16) uint32_t s_hist[256];
    __shared__ uint64_t s_red[kSelectWaves];
    __shared__ uint64_t s_cand[kWave];
    __shared__ int s_ncand;
    __shared__ int s_bc[3];  // a histogram's bin, the count above it, its count
    __shared__ uint64_t s_sel[kSelWords];
    __shared__ uint64_t s_tie[kSelWords];
    __shared__ __align__(16) int s_w[3 * kSelectWaves];

    const int bq = blockIdx.x;  // b * Hq + query head
    const int b = bq / Hq, hq = bq - b * Hq;
    const size_t tb0 = (static_cast<size_t>(b) * Hkv + hq / G) * M;
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    const double* y = Y + static_cast<size_t>(bq) * M;
    const double* ph = phi + static_cast<size_t>(bq) * M;
    const int nwords = (M + kWave - 1) / kWave;

    // key j of this thread is team j * 512 + tid (word 8 j + w of the bits)
    uint64_t k[kHeadKeys];
#pragma unroll
    for (int j = 0; j < kHeadKeys; ++j) {
        const int g = j * kSelectThreads + tid;
        k[j] = g < M ? order_key(y[g]) : 0;
    }
    auto valid = [&](int j) { return j * kSelectThreads + tid < M; };

    // tau's key: rank Kp (0-based, descending) among the M keys
    // histogram range: the real teams' keys unless those are all equal
    uint64_t kmin = ~0ull, kmax = 0;
#pragma unroll
    for (int j = 0; j < kHeadKeys; ++j) {
        if (valid(j)) {
            kmin = min(kmin, k[j]);
            kmax = max(kmax, k[j]);
        }
    }
    kmin = block_ext64<false>(kmin, s_red);
    kmax = block_ext64<true>(kmax, s_red);
    const uint64_t kreal = order_key(kAbsentBelow);
    if (kmin < kreal) {  // uniform: only tables with absent teams
        uint64_t rmin = ~0ull;
#pragma unroll
        for (int j = 0; j < kHeadKeys; ++j)
            if (valid(j) && k[j] >= kreal) rmin = min(rmin, k[j]);
        rmin = block_ext64<false>(rmin, s_red);
        if (rmin < kmax) kmin = rmin;
    }
    const double ymin = key_value(kmin);
    const double range = key_value(kmax) - ymin;
    int want = Kp;
    uint64_t tkey = kmin;
    if (range > 0.0) {  // uniform; else every key is equal
        const double fs = (static_cast<double>(1 << kFineBits) - 0.001) / range;
        int fine[kHeadKeys];
#pragma unroll
        for (int j = 0; j < kHeadKeys; ++j)
            fine[j] = valid(j) ? fine_bucket(key_value(k[j]), ymin, fs) : -1;
        // a 256-bin histogram of the (selected) keys' bins, and the bin that
        // holds rank `want`
        auto hist_pass = [&](auto bin_of) {
            if (tid < 64) reinterpret_cast<uint4*>(s_hist)[tid] = make_uint4(0, 0, 0, 0);
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kHeadKeys; ++j) {
                const int bn = bin_of(j);
                if (bn >= 0) atomicAdd(&s_hist[bn], 1u);
            }
            __syncthreads();
            if (w == 0) {
                int above, cnt;
                const int bin = hist_select(s_hist, want, above, cnt);
                if (lane == 0) {
                    s_bc[0] = bin;
                    s_bc[1] = above;
                    s_bc[2] = cnt;
                }
            }
            __syncthreads();
            const int bin = s_bc[0];
            want -= s_bc[1];
            const int cnt = s_bc[2];
            __syncthreads();  // s_bc and s_hist are reused
            return make_int2(bin, cnt);
        };
        // at most 64 keys left: gather them and rank them directly
        auto rank_direct = [&](auto in) {
            if (tid == 0) s_ncand = 0;
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kHeadKeys; ++j)
                if (in(j)) s_cand[atomicAdd(&s_ncand, 1)] = k[j];
            __syncthreads();
            const int n = s_ncand;
            if (w == 0) {
                const uint64_t mine = s_cand[min(lane, n - 1)];
                int gt = 0, ge = 0;
                for (int t = 0; t < n; ++t) {
                    const uint64_t o = readlane(mine, t);
                    gt += o > mine ? 1 : 0;
                    ge += o >= mine ? 1 : 0;
                }
                const bool owner = lane < n && gt <= want && want < ge;
                const uint64_t r = readlane(mine, __ffsll(static_cast<unsigned long long>(__ballot(owner))) - 1);
                if (lane == 0) s_red[0] = r;
            }
            __syncthreads();
            const uint64_t r = s_red[0];
            __syncthreads();
            return r;
        };
        const int2 p0 = hist_pass([&](int j) { return fine[j] >= 0 ? fine[j] >> 8 : -1; });
        const int top = p0.x;
        if (p0.y <= kWave) {
            tkey = rank_direct([&](int j) { return fine[j] >= 0 && (fine[j] >> 8) == top; });
        } else {
            const int2 p1 = hist_pass([&](int j) { return fine[j] >= 0 && (fine[j] >> 8) == top ? fine[j] & 255 : -1; });
            const int target = (top << 8) | p1.x;
            auto in_bucket = [&](int j) { return fine[j] == target; };
            if (p1.y <= kWave) {
                tkey = rank_direct(in_bucket);
            } else {
                // many keys in one fine bucket: exact radix over their 64-bit keys
                uint64_t kand = ~0ull, kor = 0;
#pragma unroll
                for (int j = 0; j < kHeadKeys; ++j) {
                    if (in_bucket(j)) {
                        kand &= k[j];
                        kor |= k[j];
                    }
                }
                const uint64_t all_and = block_bits64<false>(kand, s_red);
                const uint64_t all_or = block_bits64<true>(kor, s_red);
                const uint64_t diff = all_or & ~all_and;
                const int topbit = diff ? 63 - __clzll(static_cast<long long>(diff)) : 7;
                int sh = topbit >= 7 ? topbit - 7 : 0;
                uint64_t prefix = 0, pmask = 0;
                if (sh + 8 < 64) {
                    pmask = ~0ull << (sh + 8);
                    prefix = all_and & pmask;
                }
                for (;;) {  // uniform
                    const int2 pr = hist_pass([&](int j) {
                        return in_bucket(j) && (k[j] & pmask) == prefix ? static_cast<int>((k[j] >> sh) & 255) : -1;
                    });
                    prefix |= static_cast<uint64_t>(pr.x) << sh;
                    pmask |= 0xffull << sh;
                    if (pr.y == 1 || sh == 0) {
                        // one key, or equal keys: any key with the prefix
#pragma unroll
                        for (int j = 0; j < kHeadKeys; ++j)
                            if (in_bucket(j) && (k[j] & pmask) == prefix) s_red[0] = k[j];
                        __syncthreads();
                        tkey = s_red[0];
                        __syncthreads();
                        break;
                    }
                    sh = sh >= 8 ? sh - 8 : 0;  // the last digit may overlap bits fixed before
                }
            }
        }
    }
    const double tau = key_value(tkey);

    // the keys above tau's, and the first need_ties keys equal to it in
    // team order
    int above = 0;
#pragma unroll
    for (int j = 0; j < kHeadKeys; ++j) above += (valid(j) && k[j] > tkey) ? 1 : 0;
    {
        const int x[1] = {above};
        int ex[1], tot[1];
        block_scan<1>(x, ex, tot, s_w);
        above = tot[0];
    }
    const int need_ties = Kp - above;
#pragma unroll
    for (int j = 0; j < kHeadKeys; ++j) {
        const bool v = valid(j);
        const uint64_t sb = __ballot(v && k[j] > tkey);
        const uint64_t tb = __ballot(v && k[j] == tkey);
        if (lane == 0 && j * kSelectWaves + w < kSelWords) {
            s_sel[j * kSelectWaves + w] = sb;
            s_tie[j * kSelectWaves + w] = tb;
        }
    }
    __syncthreads();
    if (need_ties > 0) {  // uniform; exactly equal perturbed scores
        const int tc = tid < nwords ? static_cast<int>(__popcll(s_tie[tid])) : 0;
        const int x[1] = {tc};
        int ex[1], tot[1];
        block_scan<1>(x, ex, tot, s_w);
        if (tid < nwords && ex[0] < need_ties) {
            uint64_t t = s_tie[tid];
            for (int left = need_ties - ex[0]; left > 0 && t; --left) {
                const uint64_t lowest = t & (~t + 1);
                s_sel[tid] |= lowest;
                t ^= lowest;
            }
        }
        __syncthreads();
    }

    // thread t < nwords takes word t (teams 64 t ..): its selected teams'
    // log c and first positions in the head's list, in team order
    const uint64_t word = tid < nwords ? s_sel[tid] : 0;
    int nunits = 0;
    for (uint64_t t = word; t; t &= t - 1) nunits += chunk_count(team_size[tb0 + tid * kWave + __ffsll(static_cast<unsigned long long>(t)) - 1]);
    const int x[2] = {static_cast<int>(__popcll(word)), nunits};
    int ex[2], tot[2];
    block_scan<2>(x, ex, tot, s_w);
    int rank = ex[0], pos = ex[1];
    for (uint64_t t = word; t; t &= t - 1) {
        const int g = tid * kWave + __ffsll(static_cast<unsigned long long>(t)) - 1;
        const float v = log_inclusion(static_cast<float>(ph[g] - tau));
        lc[static_cast<size_t>(bq) * M + g] = v;
        lpos[static_cast<size_t>(bq) * M + g] = static_cast<unsigned short>(pos);
        if (dbg_sel) dbg_sel[static_cast<size_t>(bq) * Kp + rank] = g;
        if (dbg_logc) dbg_logc[static_cast<size_t>(bq) * Kp + rank] = v;
        ++rank;
        pos += chunk_count(team_size[tb0 + g]);
    }
    if (tid < nwords) sbits[static_cast<size_t>(bq) * kSelWords + tid] = word;
    if (tid == 0) {
        hunits[bq] = tot[1];
        if (dbg_tau) dbg_tau[bq] = tau;
    }
}

// FROM_HEADS (PL = 0 only): the heads' selections, corrections, positions
// and unit counts come from k_select_head (sbits, hunits), and only the read
// plan is built here.
// HTPT (FROM_HEADS only): teams per thread and plan pass.  16 covers 8192
// teams in one pass; the host takes it only when no pass can hold more
// union teams than the records (G K <= kSelectRecs).
template <int G, int PL, bool FROM_HEADS = false, int HTPT = 4>
__global__ __launch_bounds__(kSelectThreads) void k_select(
    const double* __restrict__ phi, const double* __restrict__ Y, const int* __restrict__ team_begin,
    const int* __restrict__ team_size, int M, int Hkv, int Hq, int Kp, int T_suf, int max_chunks,
    float* __restrict__ lc, unsigned short* __restrict__ lpos, PlanHeader* __restrict__ hdr,
    Chunk* __restrict__ chunks, float* __restrict__ ulogc, int* __restrict__ dbg_sel,
    float* __restrict__ dbg_logc, double* __restrict__ dbg_tau, int* __restrict__ dbg_uteams,
    int* __restrict__ dbg_urows, const uint64_t* __restrict__ sbits, const int* __restrict__ hunits) {
    static_assert(FROM_HEADS == (PL == 0), "head waves hold their keys in registers; PL = 0 only builds the plan");
    // Team sizes and starts, and per (head, team) log c and the team's
    // first position in the head's list of units: in LDS when the heads'
    // keys are in registers (up to 2048 teams); with the heads' results
    // (FROM_HEADS) sizes and starts come from the table and the per-head
    // values from the workspace.
    constexpr bool kLds = PL > 0;
    extern __shared__ int s_dyn[];  // kLds: [M] sizes, [M] starts, [G][M] floats, [G][M] ushorts
    __shared__ __align__(16) uint32_t s_hist[kSelectWaves][256];
    __shared__ __align__(16) uint64_t s_cand[kSelectWaves][kWave];
    __shared__ uint64_t s_bits[kMaxGroup][kMaxTeams / kWave];  // selection bits per head
    __shared__ __align__(16) int s_w[3 * kSelectWaves];
    __shared__ int s_hunits[kMaxGroup];  // units of each head's teams
    __shared__ int2 s_rec[kSelectRecs];      // union teams of a pass: first unit, team index
    __shared__ unsigned short s_u2t[kSelectUnits];  // union slot of each unit of a pass

    const int bh = blockIdx.x;
    const int b = bh / Hkv, kv = bh - b * Hkv;
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    const size_t tb0 = static_cast<size_t>(bh) * M;
    const size_t hq0 = static_cast<size_t>(b) * Hq + kv * G;  // first query head of the pair
    int* const s_size = s_dyn;
    int* const s_begin = s_dyn + M;
    float* const s_lc = reinterpret_cast<float*>(s_dyn + 2 * M);
    unsigned short* const s_pos = reinterpret_cast<unsigned short*>(s_lc + G * M);
    auto lc_at = [&](int h, int g) -> float& {
        if constexpr (kLds) return s_lc[h * M + g];
        else return lc[(hq0 + h) * M + g];
    };
    auto pos_at = [&](int h, int g) -> unsigned short& {
        if constexpr (kLds) return s_pos[h * M + g];
        else return lpos[(hq0 + h) * M + g];
    };

    auto size_of = [&](int g) { return kLds ? s_size[g] : team_size[tb0 + g]; };
    auto begin_of = [&](int g) { return kLds ? s_begin[g] : team_begin[tb0 + g]; };
    if constexpr (FROM_HEADS) {
        // the heads' selection bits (team order) and unit counts
        const int nwords = (M + kWave - 1) / kWave;
        for (int i = tid; i < G * nwords; i += kSelectThreads) {
            const int h = i / nwords, wd = i - h * nwords;
            s_bits[h][wd] = sbits[(hq0 + h) * kSelWords + wd];
        }
        if (tid < G) s_hunits[tid] = hunits[hq0 + tid];
        __syncthreads();
    } else {
    // loads first: each head wave's perturbed scores, then the team table
    // (into LDS once the heads have found tau, so that its load overlaps
    // the search: the search waits only for the earlier loads)
    const int hq = kv * G + min(w, G - 1);
    const size_t hoff = (static_cast<size_t>(b) * Hq + hq) * M;
    KeySet<PL> ks;
    if (w < G) ks.init(Y + hoff, phi + hoff, M);
    asm volatile("" ::: "memory");  // the scores' loads are issued before the table's
    constexpr int NT = kLds ? (PL * kWave + kSelectThreads - 1) / kSelectThreads : 1;  // teams per thread
    int sz[NT], bg[NT];
    if constexpr (kLds) {
#pragma unroll
        for (int k = 0; k < NT; ++k) {
            const int g = min(tid + k * kSelectThreads, M - 1);
            sz[k] = team_size[tb0 + g];
            bg[k] = team_begin[tb0 + g];
        }
    }

    const int nj = ks.count();
    uint64_t tkey = 0;
    double tau = 0.0;
    int need_ties = 0;
    if (w < G) {
        tkey = select_key<PL>(ks, Kp, s_hist[w], s_cand[w]);
        tau = key_value(tkey);
        int above_cnt = 0;
#pragma unroll
        for (int j = 0; j < nj; ++j) above_cnt += (ks.valid(j) && ks.key(j) > tkey) ? 1 : 0;
        need_ties = Kp - wave_sum(above_cnt);
    }
    if constexpr (kLds) {
#pragma unroll
        for (int k = 0; k < NT; ++k) {
            const int g = tid + k * kSelectThreads;
            if (g < M) {
                s_size[g] = sz[k];
                s_begin[g] = bg[k];
            }
        }
    }
    __syncthreads();

    if (w < G) {

        // selection in index order i = j * 64 + lane: the keys above tau's
        // key and the first need_ties keys equal to it (exactly equal Y
        // values; the tie path is kept out of the common loop), compacted
        // in team order into batches of 64 (LDS)
        const uint64_t lt = lanemask_lt();
        uint32_t* cidx = reinterpret_cast<uint32_t*>(s_cand[w]);  // [64] team index
        float* cx = reinterpret_cast<float*>(s_cand[w]) + kWave;  // [64] phi - tau
        int nsel = 0, npos = 0;
        // per batch of 64 selected teams, one per lane in team order: log c
        // and the team's first position in the head's list (a scan of the
        // selected teams' unit counts)
        auto flush = [&](int cnt) {
            wave_lds_sync();
            const bool on = lane < cnt;
            const int i = on ? static_cast<int>(cidx[lane]) : 0;
            // phi - tau: kept from the pass when phi sits in registers, else
            // one gather per batch
            const float x = KeySet<PL>::kPhiRegs ? cx[lane] : static_cast<float>(phi[hoff + i] - tau);
            const int nc = on ? chunk_count(size_of(i)) : 0;
            const int incl = wave_incl_scan(nc);
            if (on) {
                const float v = log_inclusion(x);
                lc_at(w, i) = v;
                pos_at(w, i) = static_cast<unsigned short>(npos + incl - nc);
                const size_t r = (static_cast<size_t>(b) * Hq + hq) * Kp + nsel + lane;
                if (dbg_sel) dbg_sel[r] = i;
                if (dbg_logc) dbg_logc[r] = v;
            }
            npos += __builtin_amdgcn_readlane(incl, kWave - 1);
            nsel += cnt;
            wave_lds_sync();  // cidx / cx are refilled
        };
        auto select_pass = [&](auto with_ties) {
            int nties = 0, fill = 0;
            auto ballot_word = [&](int j) {
                const bool valid = ks.valid(j);
                const uint64_t k = ks.key(j);
                bool sel = valid && k > tkey;
                if constexpr (decltype(with_ties)::value) {
                    const bool tie = valid && k == tkey;
                    const uint64_t tb = __ballot(tie);
                    sel = sel || (tie && nties + __popcll(tb & lt) < need_ties);
                    nties += __popcll(tb);
                }
                const uint64_t sb = __ballot(sel);
                if (lane == 0) s_bits[w][j] = sb;
                return sb;
            };
            auto compact = [&](int j, uint64_t sb) {
                const bool sel = (sb >> lane) & 1ull;
                const int cnt = __popcll(sb);
                if (fill + cnt > kWave) {  // uniform: the batch is full
                    flush(fill);
                    fill = 0;
                }
                if (sel) {
                    const int p = fill + __popcll(sb & lt);
                    cidx[p] = static_cast<uint32_t>(j * kWave + lane);
                    if constexpr (KeySet<PL>::kPhiRegs) cx[p] = static_cast<float>(ks.phi(j) - tau);
                }
                fill += cnt;
            };
            if constexpr (KeySet<PL>::kPhiRegs) {
#pragma unroll
                for (int j = 0; j < nj; ++j) compact(j, ballot_word(j));
            } else {
                // ballots first (unrolled over the registers), then the
                // compaction (rolled, so that the batch flush is one copy)
#pragma unroll
                for (int j = 0; j < nj; ++j) ballot_word(j);
                wave_lds_sync();
#pragma unroll 1
                for (int j = 0; j < nj; ++j) compact(j, s_bits[w][j]);
            }
            if (fill > 0) flush(fill);
        };
        if (need_ties > 0)  // uniform
            select_pass(std::true_type{});
        else
            select_pass(std::false_type{});
        if (lane == 0) {
            s_hunits[w] = npos;
            if (dbg_tau) dbg_tau[static_cast<size_t>(b) * Hq + hq] = tau;
        }
    }
    __syncthreads();
    }  // !FROM_HEADS

    // ---- union of the heads' selections in ascending team order -------------
    // One pass per kPass teams (all of them when the team table is in LDS),
    // thread tid owning TPT consecutive teams: a scan gives every union team
    // its slot, its first unit and its rows; the team writes its corrections
    // and enters itself in LDS (its record, and its slot at each of its
    // units); then thread c writes unit c of the pass to the pair's own
    // region of the unit list (max_chunks entries, which bound the units of
    // any union of this size).  Passes whose units exceed the LDS table fall
    // back to a search over the records.  A unit's position in the list of a
    // head that reads it is the team's first position there plus the unit's
    // index within the team.
    auto heads_of = [&](int g) {
        int hm = 0;
        if (g < M) {
#pragma unroll
            for (int h = 0; h < G; ++h) hm |= static_cast<int>((s_bits[h][g >> 6] >> (g & 63)) & 1ull) << h;
        }
        return hm;
    };
    // teams per thread and pass: M <= 512 TPT with LDS tables; HTPT with the
    // heads' results
    constexpr int TPT = kLds ? PL / 8 : (FROM_HEADS ? HTPT : 1);
    constexpr int kPass = kSelectThreads * TPT;
    static_assert(kPass <= kSelectRecs || (FROM_HEADS && HTPT * kSelectThreads == kMaxTeams),
                  "a pass's union teams fit the LDS records (single pass: G K <= kSelectRecs, checked on the host)");
    Chunk* const cb = chunks + static_cast<size_t>(bh) * max_chunks;
    int run_u = 0, run_rows = 0, run_c = 0;
    for (int base = 0; base < M; base += kPass) {
        int hmk[TPT], nck[TPT];
        int lf = 0, lnc = 0, lrows = 0;
#pragma unroll
        for (int k = 0; k < TPT; ++k) {
            const int g = base + tid * TPT + k;
            hmk[k] = heads_of(g);  // 0 past the last team
            const int tsz = hmk[k] ? size_of(g) : 0;
            nck[k] = hmk[k] ? chunk_count(tsz) : 0;
            lf += hmk[k] ? 1 : 0;
            lnc += nck[k];
            lrows += tsz;
        }
        const int x[3] = {lf, lnc, lrows};
        int ex[3], tot[3];
        block_scan<3>(x, ex, tot, s_w);
        const bool table = tot[1] <= kSelectUnits;  // uniform
        int slot = ex[0], ust = ex[1];
#pragma unroll
        for (int k = 0; k < TPT; ++k) {
            if (hmk[k]) {
                const int g = base + tid * TPT + k;
                float lv[kLogcStride];
#pragma unroll
                for (int h = 0; h < kMaxGroup; ++h) lv[h] = (h < G && ((hmk[k] >> h) & 1)) ? lc_at(h, g) : 0.f;
                float4* L = reinterpret_cast<float4*>(ulogc + (tb0 + run_u + slot) * kLogcStride);
                L[0] = make_float4(lv[0], lv[1], lv[2], lv[3]);
                L[1] = make_float4(lv[4], lv[5], lv[6], lv[7]);
                if (slot < kSelectRecs) s_rec[slot] = make_int2(ust, g);
                if (table)
                    for (int c = 0; c < nck[k]; ++c) s_u2t[ust + c] = static_cast<unsigned short>(slot);
                ++slot;
                ust += nck[k];
            }
        }
        __syncthreads();
        for (int c = tid; c < tot[1]; c += kSelectThreads) {
            int sl;
            if (table) {
                sl = s_u2t[c];
            } else {  // the last record whose first unit is at or before c
                int lo = 0, hi = tot[0] - 1;
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (s_rec[mid].x <= c)
                        lo = mid;
                    else
                        hi = mid - 1;
                }
                sl = lo;
            }
            const int2 rc = s_rec[sl];
            const int g = rc.y, p = c - rc.x;
            const int hm = heads_of(g), tsz = size_of(g);
            const int ci = run_c + c;
            if (ci < max_chunks) {
                Chunk ch;
                ch.begin = begin_of(g) + p * kChunkRows;
                ch.slot = run_u + sl;
                ch.meta = chunk_meta(min(kChunkRows, tsz - p * kChunkRows), hm, bh);
                ch.ci = ci;
                int ps[kMaxGroup];
#pragma unroll
                for (int h = 0; h < kMaxGroup; ++h)
                    ps[h] = (h < G && ((hm >> h) & 1)) ? static_cast<int>(pos_at(h, g)) + p : 0;
                set_chunk_pos(ch, ps);
                cb[ci] = ch;
            }
        }
        run_u += tot[0];
        run_c += tot[1];
        run_rows += tot[2];
        if (base + kPass < M) __syncthreads();  // the LDS records are rewritten by the next pass
    }
    const int nsc = chunk_count(T_suf);
    const int utotal = min(run_c + nsc, max_chunks);
    // the suffix: every head, no correction, after each head's teams
    for (int p = tid; p < nsc; p += kSelectThreads) {
        const int ci = run_c + p;
        if (ci < max_chunks) {
            Chunk ch;
            ch.begin = p * kChunkRows;
            ch.slot = -1;
            ch.meta = chunk_meta(min(kChunkRows, T_suf - p * kChunkRows), (1 << G) - 1, bh);
            ch.ci = ci;
            int ps[kMaxGroup];
#pragma unroll
            for (int h = 0; h < kMaxGroup; ++h) ps[h] = h < G ? s_hunits[h] + p : 0;
            set_chunk_pos(ch, ps);
            cb[ci] = ch;
        }
    }
    if (tid == 0) {
        PlanHeader ph;
        ph.teams = run_u;
        ph.rows = run_rows;
        ph.chunks = utotal;
        ph.pad = 0;
#pragma unroll
        for (int h = 0; h < kMaxGroup; ++h) ph.hunits[h] = h < G ? s_hunits[h] + nsc : 0;
        hdr[bh] = ph;
        if (dbg_uteams) dbg_uteams[bh] = run_u;
        if (dbg_urows) dbg_urows[bh] = run_rows;
    }
}

// Raise a kernel's dynamic LDS limit to `bytes` (once per kernel and limit;
// the select kernel keeps up to ~115 KB of team tables in LDS).
template <typename F>
hipError_t allow_dynamic_lds(F* kernel, size_t bytes) {
    static std::atomic<size_t> granted{0};
    if (bytes <= granted.load(std::memory_order_relaxed)) return hipSuccess;
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(bytes));
    if (e == hipSuccess) {
        size_t cur = granted.load(std::memory_order_relaxed);
        while (bytes > cur && !granted.compare_exchange_weak(cur, bytes)) {
        }
    }
    return e;
}

template <typename T, int D, int G>
hipError_t route_g(const RouteArgs& a, hipStream_t s) {
    const DecodeLayout& L = *a.lay;
    const santapp_decode_debug* d = a.dbg;
    double* phi = reinterpret_cast<double*>(a.ws + L.phi);
    double* Y = reinterpret_cast<double*>(a.ws + L.Y);
    k_route<T, D, G><<<dim3((a.M + kRouteTeams - 1) / kRouteTeams, a.B * a.Hkv), kRouteThreads, 0, s>>>(
        static_cast<const T*>(a.reps), a.log_n, a.q, a.M, a.Hkv, a.Hq, a.scale, a.seed, a.step, phi, Y);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    float* lc = reinterpret_cast<float*>(a.ws + L.lc);
    PlanHeader* hdr = reinterpret_cast<PlanHeader*>(a.ws + L.hdr);
    Chunk* ch = reinterpret_cast<Chunk*>(a.ws + L.chunk);
    float* ulogc = reinterpret_cast<float*>(a.ws + L.ulogc);
#define SANTAPP_SEL(PLV)                                                                          \
    do {                                                                                          \
        const size_t dyn = PLV > 0 ? (2 * sizeof(int) + (sizeof(float) + sizeof(unsigned short)) * G) * a.M : 0; \
        hipError_t ea = allow_dynamic_lds(k_select<G, PLV>, dyn);                                 \
        if (ea != hipSuccess) return ea;                                                          \
        k_select<G, PLV><<<a.B * a.Hkv, kSelectThreads, dyn, s>>>(                                \
            phi, Y, a.team_begin, a.team_size, a.M, a.Hkv, a.Hq, a.Kp, a.T, L.max_chunks, lc,   \
            reinterpret_cast<unsigned short*>(a.ws + L.lpos), hdr, ch, ulogc, d ? d->sel : nullptr, \
            d ? d->logc : nullptr, d ? d->tau : nullptr, d ? d->union_teams : nullptr,            \
            d ? d->union_rows : nullptr, nullptr, nullptr);                                       \
    } while (0)
    if (a.M <= 8 * kWave) {
        SANTAPP_SEL(8);
    } else if (a.M <= 32 * kWave) {
        SANTAPP_SEL(32);
    } else {
        // one workgroup per query head for the selection, then the plan
        uint64_t* sbits = reinterpret_cast<uint64_t*>(a.ws + L.sbits);
        int* hunits = reinterpret_cast<int*>(a.ws + L.hunits);
        unsigned short* lpos = reinterpret_cast<unsigned short*>(a.ws + L.lpos);
        k_select_head<G><<<a.B * a.Hq, kSelectThreads, 0, s>>>(
            phi, Y, a.team_size, a.M, a.Hkv, a.Hq, a.Kp, lc, lpos, sbits, hunits, d ? d->sel : nullptr,
            d ? d->logc : nullptr, d ? d->tau : nullptr);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        auto plan = static_cast<long long>(G) * a.Kp <= kSelectRecs ? k_select<G, 0, true, 16> : k_select<G, 0, true, 4>;
        plan<<<a.B * a.Hkv, kSelectThreads, 0, s>>>(
            phi, Y, a.team_begin, a.team_size, a.M, a.Hkv, a.Hq, a.Kp, a.T, L.max_chunks, lc, lpos, hdr, ch,
            ulogc, nullptr, nullptr, nullptr, d ? d->union_teams : nullptr, d ? d->union_rows : nullptr,
            sbits, hunits);
    }
#undef SANTAPP_SEL
    return hipGetLastError();
}

template <typename T, int D>
hipError_t route_d(const RouteArgs& a, hipStream_t s) {
    switch (a.G) {
        case 1: return route_g<T, D, 1>(a, s);
        case 2: return route_g<T, D, 2>(a, s);
        case 3: return route_g<T, D, 3>(a, s);
        case 4: return route_g<T, D, 4>(a, s);
        case 5: return route_g<T, D, 5>(a, s);
        case 6: return route_g<T, D, 6>(a, s);
        case 7: return route_g<T, D, 7>(a, s);
        case 8: return route_g<T, D, 8>(a, s);
        default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t route_t(const RouteArgs& a, hipStream_t s) {
    switch (a.d) {
        case 64: return route_d<T, 64>(a, s);
        case 128: return route_d<T, 128>(a, s);
        default: return hipErrorInvalidValue;
    }
}

template <typename T, int D>
hipError_t route_phi_d(const RouteArgs& a, double* phi, double* Y, hipStream_t s) {
    const dim3 grid((a.M + kRouteTeams - 1) / kRouteTeams, a.B * a.Hkv);
#define SANTAPP_PHI(GG)                                                                             \
    case GG:                                                                                        \
        k_route<T, D, GG><<<grid, kRouteThreads, 0, s>>>(static_cast<const T*>(a.reps), a.log_n, a.q, \
                                                         a.M, a.Hkv, a.Hq, a.scale, a.seed, a.step,   \
                                                         phi, Y);                                     \
        break
    switch (a.G) {
        SANTAPP_PHI(1); SANTAPP_PHI(2); SANTAPP_PHI(3); SANTAPP_PHI(4);
        SANTAPP_PHI(5); SANTAPP_PHI(6); SANTAPP_PHI(7); SANTAPP_PHI(8);
        default: return hipErrorInvalidValue;
    }
#undef SANTAPP_PHI
    return hipGetLastError();
}

}  // namespace

hipError_t launch_route_phi(const RouteArgs& a, double* phi, double* Y, hipStream_t s) {
    if (a.dtype == SANTAPP_BF16) {
        if (a.d == 128) return route_phi_d<bf16_t, 128>(a, phi, Y, s);
        if (a.d == 64) return route_phi_d<bf16_t, 64>(a, phi, Y, s);
    } else {
        if (a.d == 128) return route_phi_d<float, 128>(a, phi, Y, s);
        if (a.d == 64) return route_phi_d<float, 64>(a, phi, Y, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_route_select(const RouteArgs& a, hipStream_t s) {
    return a.dtype == SANTAPP_BF16 ? route_t<bf16_t>(a, s) : route_t<float>(a, s);
}

}  // namespace santapp
