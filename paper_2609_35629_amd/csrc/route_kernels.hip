// Routing logits of every team for every query head (eq. method-routing),
// for the routing diagnostic.
//
// k_route   phi_g = log n_g + scale q.l_g for every query head sharing the KV
//           head (one representative load serves all of them), and the Gumbel
//           perturbation Y_g = phi_g + G_g.  The dot products accumulate in
//           fp64 (every bf16 x fp32 product is exact in fp64), so phi differs
//           from an fp64 reference only by summation order.
#include <math.h>

#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

constexpr int kRouteThreads = 256;
constexpr int kRouteTeams = kRouteThreads / 16;  // one representative per 16-lane group

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

}  // namespace santapp
