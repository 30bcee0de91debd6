// Routing-key variants and the KL routing diagnostic (section
// "Attention-distribution diagnostic"; appendix "Dense-trajectory KL and
// task-variant evaluation", eq. diagnostic-kl).
//
// k_team_centroid   the team mean as routing key (centroid-guided sampling)
// k_team_repkey     the representative's key again (the table's default)
// k_kl_team         per (query head, team): max, sum of e^(s - max) and of
//                   e^(s - max) s over the team's prompt rows, fp64
// k_kl_merge        per query head: KL(p || q) from those sums and the
//                   routing logits phi
#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

// fp64 -> bf16, round to nearest with ties to even: round to fp32 with
// round-to-odd (toward zero, then the last bit set when inexact), then to
// bf16 to nearest even.  fp32 keeps 16 more significand bits than bf16, so
// the two steps round correctly (no double-rounding error).
__device__ __forceinline__ uint16_t f64_to_bf16(double x) {
    if (x != x) return 0x7fc0;
    const float f = static_cast<float>(x);
    uint32_t u = __float_as_uint(f);
    if (static_cast<double>(f) != x) {
        if (fabs(static_cast<double>(f)) > fabs(x)) u -= 1u;  // one step toward zero
        u |= 1u;
    }
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ void store_mean(bf16_t* p, double v) { p->bits = f64_to_bf16(v); }
__device__ __forceinline__ void store_mean(float* p, double v) { *p = static_cast<float>(v); }

// Team means: thread j sums dimension j over the team's rows in packed
// order (ascending token index), then divides by n_g.
template <typename T, int D>
__global__ __launch_bounds__(D) void k_team_centroid(const T* __restrict__ packed_K,
                                                     const int* __restrict__ team_begin,
                                                     const int* __restrict__ team_size, int N, int M,
                                                     T* __restrict__ reps) {
#pragma clang fp contract(off)
    const int g = blockIdx.x, bh = blockIdx.y, j = threadIdx.x;
    const size_t t = static_cast<size_t>(bh) * M + g;
    const int begin = team_begin[t], n = team_size[t];
    const T* col = packed_K + (static_cast<size_t>(bh) * N + begin) * D + j;
    double s = 0.0;
    int i = 0;
    for (; i + 8 <= n; i += 8) {  // eight loads in flight, then the adds in order
        float v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = load_elem(col, static_cast<size_t>(i + k) * D);
#pragma unroll
        for (int k = 0; k < 8; ++k) s = s + static_cast<double>(v[k]);
    }
    for (; i < n; ++i) s = s + static_cast<double>(load_elem(col, static_cast<size_t>(i) * D));
    // an absent team (no rows) keeps a zero key; its log n excludes it
    store_mean(reps + t * D + j, n > 0 ? s / static_cast<double>(n) : 0.0);
}

// The representative's key: its packed row is found among the team's rows
// (perm maps packed rows to tokens) and copied.
template <typename T, int D>
__global__ __launch_bounds__(kWave) void k_team_repkey(const T* __restrict__ packed_K,
                                                       const int* __restrict__ team_begin,
                                                       const int* __restrict__ team_size,
                                                       const int* __restrict__ rep_token,
                                                       const int* __restrict__ perm, int N, int M,
                                                       T* __restrict__ reps) {
    const int g = blockIdx.x, bh = blockIdx.y, lane = lane_id();
    const size_t t = static_cast<size_t>(bh) * M + g;
    const int begin = team_begin[t], n = team_size[t], tok = rep_token[t];
    const int* pm = perm + static_cast<size_t>(bh) * N + begin;
    int found = -1;
    for (int base = 0; base < n && found < 0; base += kWave) {  // uniform
        const int i = base + lane;
        const uint64_t hit = __ballot(i < n && pm[i] == tok);
        if (hit) found = base + __ffsll(static_cast<unsigned long long>(hit)) - 1;
    }
    if (found < 0) return;  // a table's representative is always a member of its team
    constexpr int kChunks = D * static_cast<int>(sizeof(T)) / 16;
    const uint4* src = reinterpret_cast<const uint4*>(packed_K + (static_cast<size_t>(bh) * N + begin + found) * D);
    uint4* dst = reinterpret_cast<uint4*>(reps + t * D);
    for (int c = lane; c < kChunks; c += kWave) dst[c] = src[c];
}

struct KlPart {
    double m;  // max score of the team's rows
    double z;  // sum of e^(s - m)
    double s;  // sum of e^(s - m) s
};

// Add score x to a running (max, sum e^(s-max), sum e^(s-max) s).
__device__ __forceinline__ void kl_push(double& m, double& z, double& sm, double x) {
    if (x > m) {
        const double c = exp(m - x);
        z = z * c + 1.0;
        sm = sm * c + x;
        m = x;
    } else {
        const double e = exp(x - m);
        z += e;
        sm += e * x;
    }
}

__device__ __forceinline__ void kl_combine(double& m, double& z, double& s, double m2, double z2, double s2) {
    const double mm = fmax(m, m2);
    if (mm == -INFINITY) return;
    const double c1 = exp(m - mm), c2 = exp(m2 - mm);
    z = z * c1 + z2 * c2;
    s = s * c1 + s2 * c2;
    m = mm;
}

// Eight consecutive elements of a row (16 bytes of bf16, 32 of fp32).
__device__ __forceinline__ void load8(const bf16_t* p, float (&v)[8]) {
    const uint4 w = *reinterpret_cast<const uint4*>(p);
    const uint32_t x[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        v[2 * k] = bf16lo(x[k]);
        v[2 * k + 1] = bf16hi(x[k]);
    }
}

__device__ __forceinline__ void load8(const float* p, float (&v)[8]) {
    const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// One wave per (b, kv, team): lane l takes the team's rows l, l + 64, ...,
// scores them for the G query heads of kv in fp64 and keeps each head's
// running sums; the wave then combines its lanes.
template <typename T, int D, int G>
__global__ __launch_bounds__(kWave) void k_kl_team(const T* __restrict__ packed_K,
                                                   const int* __restrict__ team_begin,
                                                   const int* __restrict__ team_size,
                                                   const float* __restrict__ q, int N, int M, int Hkv,
                                                   int Hq, double scale, KlPart* __restrict__ part) {
    __shared__ double s_q[G][D];
    const int g = blockIdx.x, bh = blockIdx.y, lane = lane_id();
    const int b = bh / Hkv, kv = bh - b * Hkv;
    const float* qb = q + (static_cast<size_t>(b) * Hq + kv * G) * D;
    for (int i = lane; i < G * D; i += kWave) s_q[i / D][i % D] = static_cast<double>(qb[i]);
    __syncthreads();
    const size_t t = static_cast<size_t>(bh) * M + g;
    const int begin = team_begin[t], n = team_size[t];
    double m[G], z[G], sm[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        m[h] = -INFINITY;
        z[h] = 0.0;
        sm[h] = 0.0;
    }
    for (int r = lane; r < n; r += kWave) {
        const T* row = packed_K + (static_cast<size_t>(bh) * N + begin + r) * D;
        double acc[G];
#pragma unroll
        for (int h = 0; h < G; ++h) acc[h] = 0.0;
#pragma unroll 1
        for (int j = 0; j < D; j += 8) {  // rolled: unrolling hoists every query read from LDS
            float v[8];
            load8(row + j, v);
#pragma unroll
            for (int e = 0; e < 8; ++e)
#pragma unroll
                for (int h = 0; h < G; ++h) acc[h] = fma(s_q[h][j + e], static_cast<double>(v[e]), acc[h]);
        }
#pragma unroll
        for (int h = 0; h < G; ++h) kl_push(m[h], z[h], sm[h], scale * acc[h]);
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
        for (int off = kWave / 2; off > 0; off >>= 1)
            kl_combine(m[h], z[h], sm[h], __shfl_xor(m[h], off), __shfl_xor(z[h], off), __shfl_xor(sm[h], off));
        if (lane == 0) part[(static_cast<size_t>(b) * Hq + kv * G + h) * M + g] = KlPart{m[h], z[h], sm[h]};
    }
}

constexpr int kKlThreads = 256;

template <bool kMax>
__device__ double kl_block_reduce(double v, double* s_red) {
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const double o = __shfl_xor(v, off);
        v = kMax ? fmax(v, o) : v + o;
    }
    if (lane_id() == 0) s_red[wave_id()] = v;
    __syncthreads();
    double r = s_red[0];
    for (int w = 1; w < kKlThreads / kWave; ++w) r = kMax ? fmax(r, s_red[w]) : r + s_red[w];
    __syncthreads();
    return r;
}

// KL(p || q) = E_p[s] - E_p[r] - LSE(s) + LSE(phi), with r_g = phi_g - log n_g
// the routing score of team g (log q_i = r_g(i) - LSE(phi)).
__global__ __launch_bounds__(kKlThreads) void k_kl_merge(const double* __restrict__ phi,
                                                         const KlPart* __restrict__ part,
                                                         const double* __restrict__ log_n, int M,
                                                         int Hkv, int Hq, double* __restrict__ kl) {
    __shared__ double s_red[kKlThreads / kWave];
    const int bhq = blockIdx.x, tid = threadIdx.x;
    const int b = bhq / Hq, hq = bhq - b * Hq, G = Hq / Hkv;
    const int bh = b * Hkv + hq / G;
    const double* ph = phi + static_cast<size_t>(bhq) * M;
    const KlPart* pt = part + static_cast<size_t>(bhq) * M;
    const double* ln = log_n + static_cast<size_t>(bh) * M;
    double pmax = -INFINITY, mmax = -INFINITY;
    for (int g = tid; g < M; g += kKlThreads) {
        pmax = fmax(pmax, ph[g]);
        mmax = fmax(mmax, pt[g].m);
    }
    pmax = kl_block_reduce<true>(pmax, s_red);
    mmax = kl_block_reduce<true>(mmax, s_red);
    double ep = 0.0, Z = 0.0, S = 0.0, Rr = 0.0;
    for (int g = tid; g < M; g += kKlThreads) {
        ep += exp(ph[g] - pmax);
        const double c = exp(pt[g].m - mmax);
        Z += pt[g].z * c;
        S += pt[g].s * c;
        Rr += (ph[g] - ln[g]) * pt[g].z * c;
    }
    ep = kl_block_reduce<false>(ep, s_red);
    Z = kl_block_reduce<false>(Z, s_red);
    S = kl_block_reduce<false>(S, s_red);
    Rr = kl_block_reduce<false>(Rr, s_red);
    if (tid == 0) kl[bhq] = (S - Rr) / Z - (mmax + log(Z)) + (pmax + log(ep));
}

template <typename T, int D>
hipError_t route_keys_d(const void* packed_K, const int* team_begin, const int* team_size,
                        const int* rep_token, const int* perm, int BH, int N, int M, bool centroid,
                        void* reps, hipStream_t s) {
    const dim3 grid(M, BH);
    if (centroid)
        k_team_centroid<T, D><<<grid, D, 0, s>>>(static_cast<const T*>(packed_K), team_begin, team_size, N, M,
                                                 static_cast<T*>(reps));
    else
        k_team_repkey<T, D><<<grid, kWave, 0, s>>>(static_cast<const T*>(packed_K), team_begin, team_size,
                                                   rep_token, perm, N, M, static_cast<T*>(reps));
    return hipGetLastError();
}

template <typename T, int D>
hipError_t kl_d(const KlArgs& a, hipStream_t s) {
    KlPart* part = static_cast<KlPart*>(a.part);
    const dim3 grid(a.M, a.B * a.Hkv);
#define SANTAPP_KL(GG)                                                                                \
    case GG:                                                                                          \
        k_kl_team<T, D, GG><<<grid, kWave, 0, s>>>(static_cast<const T*>(a.packed_K), a.team_begin,  \
                                                   a.team_size, a.q, a.N, a.M, a.Hkv, a.Hq, a.scale, \
                                                   part);                                             \
        break
    switch (a.Hq / a.Hkv) {
        SANTAPP_KL(1); SANTAPP_KL(2); SANTAPP_KL(3); SANTAPP_KL(4);
        SANTAPP_KL(5); SANTAPP_KL(6); SANTAPP_KL(7); SANTAPP_KL(8);
        default: return hipErrorInvalidValue;
    }
#undef SANTAPP_KL
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    k_kl_merge<<<a.B * a.Hq, kKlThreads, 0, s>>>(a.phi, part, a.log_n, a.M, a.Hkv, a.Hq, a.kl);
    return hipGetLastError();
}

}  // namespace

size_t kl_part_bytes() { return sizeof(KlPart); }

hipError_t launch_route_keys(const void* packed_K, const int* team_begin, const int* team_size,
                             const int* rep_token, const int* perm, int BH, int N, int M, int d,
                             santapp_dtype dtype, bool centroid, void* reps, hipStream_t s) {
    if (dtype == SANTAPP_BF16) {
        if (d == 128) return route_keys_d<bf16_t, 128>(packed_K, team_begin, team_size, rep_token, perm, BH, N, M, centroid, reps, s);
        if (d == 64) return route_keys_d<bf16_t, 64>(packed_K, team_begin, team_size, rep_token, perm, BH, N, M, centroid, reps, s);
    } else {
        if (d == 128) return route_keys_d<float, 128>(packed_K, team_begin, team_size, rep_token, perm, BH, N, M, centroid, reps, s);
        if (d == 64) return route_keys_d<float, 64>(packed_K, team_begin, team_size, rep_token, perm, BH, N, M, centroid, reps, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_routing_kl(const KlArgs& a, hipStream_t s) {
    if (a.dtype == SANTAPP_BF16) {
        if (a.d == 128) return kl_d<bf16_t, 128>(a, s);
        if (a.d == 64) return kl_d<bf16_t, 64>(a, s);
    } else {
        if (a.d == 128) return kl_d<float, 128>(a, s);
        if (a.d == 64) return kl_d<float, 64>(a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace santapp
