// Routing, sampling and the GQA read plan of one decode step.
//
// k_route   eq. method-routing: phi_g = log n_g + scale q.l_g for every query
//           head sharing the KV head (one representative load serves all of
//           them), plus the Gumbel perturbation Y_g = phi_g + G_g.  fp64.
// k_select  Gumbel-top-K per query head: tau = the (K+1)-th largest Y (radix
//           select over order-preserving 64-bit keys), S = the K largest
//           (ties to the lower team index), log c_g for g in S
//           (eq. method-inclusion); then the union of the heads' selections
//           per KV head with an 8-bit head mask and per-head log c, a prefix
//           sum of the union's rows, and the row split of the next kernel.
#include <math.h>

#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

constexpr int kRouteThreads = 256;
constexpr int kRouteGroups = kRouteThreads / 16;  // 16 lanes per representative
constexpr int kRouteTeamsPerBlock = 64;
constexpr int kSelectThreads = 512;
constexpr int kSelectWaves = kSelectThreads / kWave;

template <typename T, int G>
__global__ __launch_bounds__(kRouteThreads) void k_route(
    const T* __restrict__ reps, const int* __restrict__ team_size, const float* __restrict__ q,
    int M, int d, int Hkv, int Hq, double scale, uint64_t seed, uint64_t step,
    double* __restrict__ phi, double* __restrict__ Y) {
    __shared__ float s_q[G][kMaxHeadDim];
    const int bh = blockIdx.y;
    const int b = bh / Hkv, kv = bh - b * Hkv;
    const int tid = threadIdx.x;
    const float* qb = q + (static_cast<size_t>(b) * Hq + kv * G) * d;
    for (int i = tid; i < G * d; i += kRouteThreads) s_q[i / d][i % d] = qb[i];
    __syncthreads();

    const int grp = tid >> 4, sub = tid & 15;
    const T* rb = reps + static_cast<size_t>(bh) * M * d;
    for (int it = 0; it < kRouteTeamsPerBlock / kRouteGroups; ++it) {
        const int g = blockIdx.x * kRouteTeamsPerBlock + it * kRouteGroups + grp;
        if (g >= M) break;  // uniform across the 16-lane group
        double acc[G];
#pragma unroll
        for (int h = 0; h < G; ++h) acc[h] = 0.0;
        const T* row = rb + static_cast<size_t>(g) * d;
        for (int j = sub; j < d; j += 16) {
            const double k = static_cast<double>(load_elem(row, j));
#pragma unroll
            for (int h = 0; h < G; ++h) acc[h] = fma(static_cast<double>(s_q[h][j]), k, acc[h]);
        }
#pragma unroll
        for (int h = 0; h < G; ++h) {
#pragma unroll
            for (int off = 8; off > 0; off >>= 1) acc[h] += __shfl_xor(acc[h], off, 16);
        }
        if (sub < G) {
            double dot = 0.0;
#pragma unroll
            for (int h = 0; h < G; ++h)
                if (h == sub) dot = acc[h];
            const int hq = kv * G + sub;
            const double ph = log(static_cast<double>(team_size[static_cast<size_t>(bh) * M + g])) +
                              scale * dot;
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

__global__ __launch_bounds__(kSelectThreads) void k_select(
    const double* __restrict__ phi, const double* __restrict__ Y,
    const int* __restrict__ team_begin, const int* __restrict__ team_size, int M, int Kp, int Hkv,
    int G, int Hq, int T, int n_split, float* __restrict__ lc, int* __restrict__ hdr,
    int* __restrict__ ubeg, int* __restrict__ urs, float* __restrict__ ulogc,
    int* __restrict__ split_team, int* __restrict__ dbg_sel, float* __restrict__ dbg_logc,
    double* __restrict__ dbg_tau, int* __restrict__ dbg_uteams, int* __restrict__ dbg_urows) {
    extern __shared__ uint32_t s_dyn[];
    const int mask_words = (M + 3) >> 2;
    uint32_t* s_mask = s_dyn;
    int* s_rs = reinterpret_cast<int*>(s_dyn + mask_words);  // [M + 1]
    __shared__ uint32_t s_hist[kSelectWaves][256];
    __shared__ int s_w[2 * kSelectWaves];

    const int bh = blockIdx.x;
    const int b = bh / Hkv, kv = bh - b * Hkv;
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    for (int i = tid; i < mask_words; i += kSelectThreads) s_mask[i] = 0;
    __syncthreads();

    if (w < G) {
        const int hq = kv * G + w;
        const size_t hoff = (static_cast<size_t>(b) * Hq + hq) * M;
        const double* y = Y + hoff;
        uint32_t* hist = s_hist[w];
        // radix select of the element of rank Kp (0-based, descending)
        uint64_t prefix = 0, pmask = 0, tkey = 0;
        int want = Kp;
        bool found = false;
        for (int shift = 56; shift >= 0 && !found; shift -= 8) {
            for (int e = lane; e < 256; e += kWave) hist[e] = 0;
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            for (int i = lane; i < M; i += kWave) {
                const uint64_t k = order_key(y[i]);
                if ((k & pmask) == prefix) atomicAdd(&hist[(k >> shift) & 255], 1u);
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            __builtin_amdgcn_wave_barrier();
            int c[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) c[e] = static_cast<int>(hist[lane * 4 + e]);
            const int mine = c[0] + c[1] + c[2] + c[3];
            int suf = mine;  // sum over lanes >= lane
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
                for (int i = lane; i < M; i += kWave) {
                    const uint64_t k = order_key(y[i]);
                    if ((k & pmask) == prefix) kk = k;
                }
                const uint64_t hb = __ballot(kk != 0);
                tkey = __shfl(kk, __ffsll(static_cast<unsigned long long>(hb)) - 1);
                found = true;
            }
        }
        if (!found) tkey = prefix;
        const double tau = key_value(tkey);

        int above_cnt = 0;
        for (int i = lane; i < M; i += kWave) above_cnt += (order_key(y[i]) > tkey) ? 1 : 0;
        for (int off = kWave / 2; off > 0; off >>= 1) above_cnt += __shfl_xor(above_cnt, off);
        const int need_ties = Kp - above_cnt;

        const uint64_t lt = lanemask_lt();
        int nsel = 0, nties = 0;
        for (int base = 0; base < M; base += kWave) {
            const int i = base + lane;
            const bool valid = i < M;
            const uint64_t k = valid ? order_key(y[i]) : 0;
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
                const double x = phi[hoff + i] - tau;
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

    // union of the heads' selections, ascending team index, and its row prefix
    const size_t tb0 = static_cast<size_t>(bh) * M;
    int run_u = 0, run_rows = 0;
    for (int base = 0; base < M; base += kSelectThreads) {
        const int g = base + tid;
        const uint32_t m = (g < M) ? ((s_mask[g >> 2] >> ((g & 3) * 8)) & 0xffu) : 0u;
        const int f = m ? 1 : 0;
        const int sz = f ? team_size[tb0 + g] : 0;
        int ef, es, tf, ts;
        block_scan2(f, sz, ef, es, tf, ts, s_w);
        if (f) {
            const int slot = run_u + ef;
            ubeg[tb0 + slot] = team_begin[tb0 + g];
            s_rs[slot] = run_rows + es;
            float* L = ulogc + (tb0 + slot) * kLogcStride;
#pragma unroll
            for (int h = 0; h < kLogcStride; ++h) {
                float v = INFINITY;  // heads that did not select the team ignore its rows
                if (h < G && ((m >> h) & 1u))
                    v = lc[(static_cast<size_t>(b) * Hq + kv * G + h) * M + g];
                L[h] = v;
            }
        }
        run_u += tf;
        run_rows += ts;
    }
    if (tid == 0) s_rs[run_u] = run_rows;
    __syncthreads();
    const size_t rs0 = static_cast<size_t>(bh) * (M + 1);
    for (int j = tid; j <= run_u; j += kSelectThreads) urs[rs0 + j] = s_rs[j];
    if (tid == 0) {
        hdr[bh * 4 + 0] = run_u;
        hdr[bh * 4 + 1] = run_rows;
        if (dbg_uteams) dbg_uteams[bh] = run_u;
        if (dbg_urows) dbg_urows[bh] = run_rows;
    }
    // first union team of every split of the rows [0, run_rows + T)
    const int total = run_rows + T;
    const int L = (total + n_split - 1) / n_split;
    for (int s = tid; s < n_split; s += kSelectThreads) {
        const int r0 = s * L;
        int t = run_u;
        if (r0 < run_rows) {
            int lo = 0, hi = run_u - 1;  // largest t with s_rs[t] <= r0
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (s_rs[mid] <= r0)
                    lo = mid;
                else
                    hi = mid - 1;
            }
            t = lo;
        }
        split_team[static_cast<size_t>(bh) * n_split + s] = t;
    }
}

template <typename T>
hipError_t route_dispatch(const RouteArgs& a, hipStream_t s) {
    const dim3 grid((a.M + kRouteTeamsPerBlock - 1) / kRouteTeamsPerBlock, a.B * a.Hkv);
    double* phi = reinterpret_cast<double*>(a.ws + a.lay->phi);
    double* Y = reinterpret_cast<double*>(a.ws + a.lay->Y);
    const T* reps = static_cast<const T*>(a.reps);
#define SANTAPP_ROUTE(GG)                                                                   \
    k_route<T, GG><<<grid, kRouteThreads, 0, s>>>(reps, a.team_size, a.q, a.M, a.d, a.Hkv, \
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

}  // namespace

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
    return a.dtype == SANTAPP_BF16 ? route_dispatch<bf16_t>(a, s) : route_dispatch<float>(a, s);
}

hipError_t launch_select(const RouteArgs& a, hipStream_t s) {
    const size_t lds = sizeof(uint32_t) * (((a.M + 3) / 4) + (a.M + 1));
    const santapp_decode_debug* d = a.dbg;
    k_select<<<a.B * a.Hkv, kSelectThreads, lds, s>>>(
        reinterpret_cast<const double*>(a.ws + a.lay->phi),
        reinterpret_cast<const double*>(a.ws + a.lay->Y), a.team_begin, a.team_size, a.M, a.Kp,
        a.Hkv, a.G, a.Hq, a.T, a.lay->n_split, reinterpret_cast<float*>(a.ws + a.lay->lc),
        reinterpret_cast<int*>(a.ws + a.lay->hdr), reinterpret_cast<int*>(a.ws + a.lay->ubeg),
        reinterpret_cast<int*>(a.ws + a.lay->urs), reinterpret_cast<float*>(a.ws + a.lay->ulogc),
        reinterpret_cast<int*>(a.ws + a.lay->split), d ? d->sel : nullptr,
        d ? d->logc : nullptr, d ? d->tau : nullptr, d ? d->union_teams : nullptr,
        d ? d->union_rows : nullptr);
    return hipGetLastError();
}

}  // namespace santapp
