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
constexpr int kRouteTPG = 1;                      // representatives per lane group
constexpr int kRouteTeamsPerBlock = kRouteGroups * kRouteTPG;
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
    const T* __restrict__ reps, const int* __restrict__ team_size, const float* __restrict__ q,
    int M, int Hkv, int Hq, double scale, uint64_t seed, uint64_t step, double* __restrict__ phi,
    double* __restrict__ Y) {
    constexpr int DPL = D / 16;
    using Chunk = RepChunk<T, DPL>;
    const int bh = blockIdx.y;
    const int b = bh / Hkv, kv = bh - b * Hkv;
    const int tid = threadIdx.x, grp = tid >> 4, sub = tid & 15;

    // every representative load of the group is issued before any arithmetic
    typename Chunk::raw raw[kRouteTPG];
    int nsz[kRouteTPG];
    const T* rb = reps + static_cast<size_t>(bh) * M * D + sub * DPL;
#pragma unroll
    for (int t = 0; t < kRouteTPG; ++t) {
        const int g = min(blockIdx.x * kRouteTeamsPerBlock + t * kRouteGroups + grp, M - 1);
        raw[t] = Chunk::load(rb + static_cast<size_t>(g) * D);
        nsz[t] = team_size[static_cast<size_t>(bh) * M + g];
    }
    double qd[G][DPL];
    const float* qb = q + (static_cast<size_t>(b) * Hq + kv * G) * D + sub * DPL;
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < DPL; ++e) qd[h][e] = static_cast<double>(qb[h * D + e]);

#pragma unroll
    for (int t = 0; t < kRouteTPG; ++t) {
        const int g = blockIdx.x * kRouteTeamsPerBlock + t * kRouteGroups + grp;
        if (g >= M) break;  // uniform across the 16-lane group
        double acc[G];
#pragma unroll
        for (int h = 0; h < G; ++h) {
            double a = 0.0;
#pragma unroll
            for (int e = 0; e < DPL; ++e)
                a = fma(qd[h][e], static_cast<double>(Chunk::get(raw[t], e)), a);
            acc[h] = a;
        }
#pragma unroll
        for (int h = 0; h < G; ++h) acc[h] = row16_sum(acc[h]);
        if (sub < G) {
            double dot = 0.0;
#pragma unroll
            for (int h = 0; h < G; ++h)
                if (h == sub) dot = acc[h];
            const int hq = kv * G + sub;
            const double ph = log(static_cast<double>(nsz[t])) + scale * dot;
            const size_t o = (static_cast<size_t>(b) * Hq + hq) * M + g;
            phi[o] = ph;
            Y[o] = ph + team_gumbel(seed, step, b, hq, g);
        }
    }
}

// Exclusive scan of two counters over the workgroup; returns the totals.
__device__ __forceinline__ void block_scan2(int a, int c, int& ea, int& ec, int& ta, int& tc,
                                            int* s_w /* [2 * kSelectWaves] */) {
    const int lane = lane_id(), w = wave_id();
    int ia = a, ic = c;
    for (int off = 1; off < kWave; off <<= 1) {
        const int xa = __shfl_up(ia, off), xc = __shfl_up(ic, off);
        if (lane >= off) {
            ia += xa;
            ic += xc;
        }
    }
    if (lane == kWave - 1) {
        s_w[w] = ia;
        s_w[kSelectWaves + w] = ic;
    }
    __syncthreads();
    int pa = 0, pc = 0;
    ta = 0;
    tc = 0;
    for (int v = 0; v < kSelectWaves; ++v) {
        if (v < w) {
            pa += s_w[v];
            pc += s_w[kSelectWaves + v];
        }
        ta += s_w[v];
        tc += s_w[kSelectWaves + v];
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

template <int PL>
__global__ __launch_bounds__(kSelectThreads) void k_select(
    const double* __restrict__ phi, const double* __restrict__ Y,
    const int* __restrict__ team_begin, const int* __restrict__ team_size, int M, int N, int Kp,
    int Hkv, int G, int Hq, float* __restrict__ lc, int* __restrict__ hdr,
    float* __restrict__ ulogc, int2* __restrict__ rowmap, int* __restrict__ dbg_sel,
    float* __restrict__ dbg_logc,
    double* __restrict__ dbg_tau, int* __restrict__ dbg_uteams, int* __restrict__ dbg_urows) {
    extern __shared__ uint32_t s_mask[];  // [ceil(M / 4)]: 8-bit head mask per team
    __shared__ uint32_t s_hist[kSelectWaves][256];
    __shared__ int s_w[2 * kSelectWaves];

    const int bh = blockIdx.x;
    const int b = bh / Hkv, kv = bh - b * Hkv;
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    const int mask_words = (M + 3) >> 2;
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
        // radix select of the element of rank Kp (0-based, descending)
        uint64_t prefix = 0, pmask = 0, tkey = 0;
        int want = Kp;
        bool found = false;
        for (int shift = 56; shift >= 0 && !found; shift -= 8) {
            for (int e = lane; e < 256; e += kWave) hist[e] = 0;
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int j = 0; j < nj; ++j) {
                const uint64_t k = ks.key(j);
                if (ks.valid(j) && (k & pmask) == prefix) atomicAdd(&hist[(k >> shift) & 255], 1u);
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            __builtin_amdgcn_wave_barrier();
            int c[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) c[e] = static_cast<int>(hist[lane * 4 + e]);
            const int mine = c[0] + c[1] + c[2] + c[3];
            int suf = mine;  // candidates in this lane's bins and all higher ones
            for (int off = 1; off < kWave; off <<= 1) {
                const int t = __shfl_down(suf, off);
                if (lane + off < kWave) suf += t;
            }
            const int above = suf - mine;
            const bool owner = (above <= want) && (want < suf);
            int digit = 0, cum = above, cnt = 0;
            if (owner) {
#pragma unroll
                for (int e = 3; e >= 0; --e) {
                    if (cum + c[e] > want) {
                        digit = lane * 4 + e;
                        cnt = c[e];
                        break;
                    }
                    cum += c[e];
                }
            }
            const uint64_t ob = __ballot(owner);
            const int src = __ffsll(static_cast<unsigned long long>(ob)) - 1;
            digit = __shfl(digit, src);
            cum = __shfl(cum, src);
            cnt = __shfl(cnt, src);
            want -= cum;
            prefix |= static_cast<uint64_t>(digit) << shift;
            pmask |= 0xffull << shift;
            if (cnt == 1) {
                // the rank-Kp element is the only candidate left: fetch it
                uint64_t kk = 0;
                bool have = false;
#pragma unroll
                for (int j = 0; j < nj; ++j) {
                    const uint64_t k = ks.key(j);
                    if (ks.valid(j) && (k & pmask) == prefix) {
                        kk = k;
                        have = true;
                    }
                }
                const uint64_t hb = __ballot(have);
                tkey = __shfl(kk, __ffsll(static_cast<unsigned long long>(hb)) - 1);
                found = true;
            }
        }
        if (!found) tkey = prefix;
        const double tau = key_value(tkey);

        int above_cnt = 0;
#pragma unroll
        for (int j = 0; j < nj; ++j) above_cnt += (ks.valid(j) && ks.key(j) > tkey) ? 1 : 0;
        for (int off = kWave / 2; off > 0; off >>= 1) above_cnt += __shfl_xor(above_cnt, off);
        const int need_ties = Kp - above_cnt;

        const uint64_t lt = lanemask_lt();
        int nsel = 0, nties = 0;
#pragma unroll
        for (int j = 0; j < nj; ++j) {  // index order: i = j * 64 + lane
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
                // log c = log(1 - exp(-exp(phi - tau))), without cancellation
                const double x = ks.phi(j) - tau;
                const float lcv = static_cast<float>(log(-expm1(-exp(x))));
                lc[hoff + i] = lcv;
                atomicOr(&s_mask[i >> 2], 1u << ((i & 3) * 8 + w));
                if (pos < Kp) {
                    if (dbg_sel) dbg_sel[(static_cast<size_t>(b) * Hq + hq) * Kp + pos] = i;
                    if (dbg_logc) dbg_logc[(static_cast<size_t>(b) * Hq + hq) * Kp + pos] = lcv;
                }
            }
        }
        if (lane == 0 && dbg_tau) dbg_tau[static_cast<size_t>(b) * Hq + hq] = tau;
    }
    __syncthreads();

    // union of the heads' selections in ascending team order, its row prefix,
    // and the row map (each wave writes the rows of its own union teams)
    int2* rm = rowmap + static_cast<size_t>(bh) * N;
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
        const int slot = run_u + ef, rs = run_rows + es;
        if (f) {
            float* L = ulogc + (tb0 + slot) * kLogcStride;
#pragma unroll
            for (int h = 0; h < kLogcStride; ++h) {
                float v = 1.0e30f;  // heads that did not select the team give its rows no weight
                if (h < G && ((m >> h) & 1u))
                    v = lc[(static_cast<size_t>(b) * Hq + kv * G + h) * M + g];
                L[h] = v;
            }
        }
        uint64_t fb = __ballot(f);
        while (fb) {
            const int j = __ffsll(static_cast<unsigned long long>(fb)) - 1;
            fb &= fb - 1;
            const int trs = __shfl(rs, j), tn = __shfl(sz, j), tb = __shfl(tbeg, j),
                      tslot = __shfl(slot, j);
            for (int k = lane; k < tn; k += kWave) rm[trs + k] = make_int2(tb + k, tslot);
        }
        run_u += tf;
        run_rows += ts;
    }
    if (tid == 0) {
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
    k_route<T, D, GG><<<grid, kRouteThreads, 0, s>>>(reps, a.team_size, a.q, a.M, a.Hkv,  \
                                                      a.Hq, a.scale, a.seed, a.step, phi, Y)
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
    const size_t lds = sizeof(uint32_t) * ((a.M + 3) / 4);
    const santapp_decode_debug* d = a.dbg;
    const DecodeLayout& L = *a.lay;
    k_select<PL><<<a.B * a.Hkv, kSelectThreads, lds, s>>>(
        reinterpret_cast<const double*>(a.ws + L.phi), reinterpret_cast<const double*>(a.ws + L.Y),
        a.team_begin, a.team_size, a.M, a.N, a.Kp, a.Hkv, a.G, a.Hq,
        reinterpret_cast<float*>(a.ws + L.lc), reinterpret_cast<int*>(a.ws + L.hdr),
        reinterpret_cast<float*>(a.ws + L.ulogc), reinterpret_cast<int2*>(a.ws + L.rowmap),
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
    else if (a.M <= 32 * kWave)
        select_launch<32>(a, s);
    else
        select_launch<0>(a, s);
    return hipGetLastError();
}

}  // namespace santapp
