// Minibatch k-means parents (Alg. "Global minibatch k-means parent partition"
// and the settings stated after it: greedy k-means++ seeding on a sample,
// minibatches drawn with replacement, cumulative-count center updates,
// reassignment of starved centers, a no-improvement rule on the smoothed
// minibatch inertia), and the parent member lists that feed the team build.
//
// Every (sequence, KV head) runs its own k-means on its prompt keys; all
// heads share the random draws (one seed serves every head's fit).  Draws:
// Philox4x64-10, key (seed, 1), counter (a / 4, tag, s, 0), word a mod 4; an
// index in [0, n) is floor(w n / 2^64), a uniform in [0, 1) is (w >> 11) 2^-53.
//   tag 0  seeding sample position a        tag 1  first center (a = 0)
//   tag 2  trial a of seeding round s        tag 3  batch position a of step s
//   tag 4  the a-th reassigned center of step s
//
// A distance between a key and a center is an fp64 sum over dimensions in
// index order with no fused multiply-add, so it equals the plain definition's
// value bit for bit when the center does.  Sums over many points (center
// updates, seeding potentials, the batch inertia) are blocked: per workgroup
// in point order, then over workgroups in order.  For bf16 keys these sums
// are exact in fp64 unless the keys span more than about 40 binary orders of
// magnitude, so they equal a sequential sum; otherwise they differ from it in
// the last bits.
//
// Kernels (one launch serves every (sequence, KV head); y = the pair)
//   k_kpp_sample   the seeding sample (token indices) and the first candidate
//   k_kpp_dist     seeding round c: min(D^2_j, |x_j - cand_t|^2) per sample
//                  point and candidate, and per-workgroup potential sums
//   k_kpp_pick     round c: the candidate with the smallest potential becomes
//                  center c, D^2 follows it, the next round's candidates are
//                  drawn from the running sums of D^2
//   k_km_assign    nearest center of each batch point (FINAL: of every
//                  token, written as its label); per-workgroup center sums
//   k_km_update    cumulative-count update of one center
//   k_km_control   reassignment, smoothed inertia and the stopping rule
//   k_parent_lists members of each parent in token order, parent and team
//                  offsets (Alg. "Build actual-key teams from a parent
//                  partition" numbers teams parent by parent)
#include <math.h>

#include <algorithm>

#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

constexpr int kKppThreads = 256;
constexpr int kPickThreads = 1024;
constexpr int kPickCache = 16;  // sample values per thread k_kpp_pick keeps in registers
constexpr int kAsgThreads = 256;
constexpr int kAsgPts = 64;   // batch points per assignment workgroup
constexpr int kAsgCen = 32;   // centers per LDS tile
constexpr int kUpdBatch = 32; // workgroup partials the center update loads at once
constexpr int kListThreads = 1024;
constexpr int kListWaves = kListThreads / kWave;

__device__ __forceinline__ uint64_t km_word(uint64_t seed, uint64_t a, uint64_t tag, uint64_t s) {
    const u64x4 r = philox4x64_10(a >> 2, tag, s, 0, seed, 1);
    const int e = static_cast<int>(a & 3);
    return e == 0 ? r.v[0] : e == 1 ? r.v[1] : e == 2 ? r.v[2] : r.v[3];
}

__device__ __forceinline__ int draw_index(uint64_t w, int n) {
    return static_cast<int>(__umul64hi(w, static_cast<uint64_t>(n)));
}

__device__ __forceinline__ double draw_unit(uint64_t w) {
    return static_cast<double>(w >> 11) * 0x1.0p-53;
}

// 16 bytes of a key row as floats (8 bf16 or 4 fp32 values, in order).
__device__ __forceinline__ void load_row16(const bf16_t* p, float (&v)[8]) {
    const uint4 w = *reinterpret_cast<const uint4*>(p);
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        v[2 * q] = bf16lo(ws[q]);
        v[2 * q + 1] = bf16hi(ws[q]);
    }
}

__device__ __forceinline__ void load_row16(const float* p, float (&v)[4]) {
    const uint4 w = *reinterpret_cast<const uint4*>(p);
    v[0] = __uint_as_float(w.x);
    v[1] = __uint_as_float(w.y);
    v[2] = __uint_as_float(w.z);
    v[3] = __uint_as_float(w.w);
}

// Per-workgroup sum of one value per thread: waves by xor shuffles, then the
// wave totals in wave order.
template <int W>
__device__ __forceinline__ double block_sum(double v, double* s_w) {
    for (int off = kWave / 2; off > 0; off >>= 1) v = v + __shfl_xor(v, off);
    if (lane_id() == 0) s_w[wave_id()] = v;
    __syncthreads();
    double r = 0.0;
    for (int w = 0; w < W; ++w) r = r + s_w[w];
    __syncthreads();
    return r;
}

__global__ __launch_bounds__(kKppThreads) void k_kpp_sample(int* __restrict__ samp, int s0, int N,
                                                            int* __restrict__ cand, int L, int BH,
                                                            uint64_t seed) {
    const int j = blockIdx.x * kKppThreads + threadIdx.x;
    if (j < s0) samp[j] = draw_index(km_word(seed, static_cast<uint64_t>(j), 0, 0), N);
    if (j == 0) {
        const int pos0 = draw_index(km_word(seed, 0, 1, 0), s0);
        for (int bh = 0; bh < BH; ++bh) cand[bh * L] = pos0;
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kKppThreads) void k_kpp_dist(
    const T* __restrict__ K, int N, const int* __restrict__ samp, int s0, const int* __restrict__ cand,
    int L, int c, double* __restrict__ D2, double* __restrict__ Dt, double* __restrict__ part) {
#pragma clang fp contract(off)
    __shared__ double s_cand[kKmMaxTrials][D];
    __shared__ double s_w[kKppThreads / kWave];
    const int bh = blockIdx.y, tid = threadIdx.x;
    const int nc = c == 0 ? 1 : L;
    const T* X = K + static_cast<size_t>(bh) * N * D;
    __shared__ int s_ctok[kKmMaxTrials];
    if (tid < nc) s_ctok[tid] = samp[cand[bh * L + tid]];
    __syncthreads();
    {
        constexpr int kPer = 16 / static_cast<int>(sizeof(T));
        for (int e = tid; e < nc * (D / kPer); e += kKppThreads) {
            const int t = e / (D / kPer), k0 = (e % (D / kPer)) * kPer;
            float v[kPer];
            load_row16(X + static_cast<size_t>(s_ctok[t]) * D + k0, v);
#pragma unroll
            for (int r = 0; r < kPer; ++r) s_cand[t][k0 + r] = static_cast<double>(v[r]);
        }
    }
    __syncthreads();
    const int j = blockIdx.x * kKppThreads + tid;
    const bool valid = j < s0;
    const T* x = X + static_cast<size_t>(valid ? samp[j] : 0) * D;
    const double dcur = (valid && c > 0) ? D2[static_cast<size_t>(bh) * s0 + j] : 0.0;
    // one pass over the point's row, all of it loaded up front; candidate
    // t's sum runs in dimension order
    double acc[kKmMaxTrials];
#pragma unroll
    for (int t = 0; t < kKmMaxTrials; ++t) acc[t] = 0.0;
    constexpr int kPer = 16 / static_cast<int>(sizeof(T));
    uint4 raw[D / kPer];
#pragma unroll
    for (int q = 0; q < D / kPer; ++q) raw[q] = reinterpret_cast<const uint4*>(x)[q];
#pragma unroll
    for (int k0 = 0; k0 < D; k0 += kPer) {
        float xv[kPer];
        load_row16(reinterpret_cast<const T*>(&raw[k0 / kPer]), xv);
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
#pragma unroll
            for (int t = 0; t < kKmMaxTrials; ++t) {
                if (t < nc) {
                    const double e = static_cast<double>(xv[q]) - s_cand[t][k0 + q];
                    acc[t] = acc[t] + e * e;
                }
            }
        }
    }
    const int nblk = gridDim.x;
#pragma unroll
    for (int t = 0; t < kKmMaxTrials; ++t) {
        if (t < nc) {  // uniform
            double m = 0.0;
            if (valid) {
                m = (c == 0) ? acc[t] : (acc[t] < dcur ? acc[t] : dcur);
                Dt[(static_cast<size_t>(bh) * L + t) * s0 + j] = m;
            }
            const double tot = block_sum<kKppThreads / kWave>(m, s_w);
            if (tid == 0) part[(static_cast<size_t>(bh) * nblk + blockIdx.x) * L + t] = tot;
        }
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kPickThreads) void k_kpp_pick(
    const T* __restrict__ K, int N, const int* __restrict__ samp, int s0, int* __restrict__ cand,
    int L, int c, int M, int nblk, double* __restrict__ D2, const double* __restrict__ Dt,
    const double* __restrict__ part, double* __restrict__ cent, uint64_t seed) {
#pragma clang fp contract(off)
    __shared__ double s_pot[kKmMaxTrials];
    __shared__ double s_tot[kPickThreads / kWave];
    __shared__ int s_best;
    __shared__ int s_first[kKmMaxTrials];
    __shared__ double s_u[kKmMaxTrials];
    const int bh = blockIdx.x, tid = threadIdx.x;
    const int nc = c == 0 ? 1 : L;
    const T* X = K + static_cast<size_t>(bh) * N * D;
    if (wave_id() < nc) {  // wave t sums trial t's workgroup partials
        const int t = wave_id();
        double p = 0.0;
        for (int b = lane_id(); b < nblk; b += kWave) p = p + part[(static_cast<size_t>(bh) * nblk + b) * L + t];
        for (int off = kWave / 2; off > 0; off >>= 1) p = p + __shfl_xor(p, off);
        if (lane_id() == 0) s_pot[t] = p;
    }
    if (tid < kKmMaxTrials) s_first[tid] = s0 - 1;
    __syncthreads();
    if (tid == 0) {
        int best = 0;
        for (int t = 1; t < nc; ++t)
            if (s_pot[t] < s_pot[best]) best = t;
        s_best = best;
    }
    __syncthreads();
    const int best = s_best;
    const int tok = samp[cand[bh * L + best]];
    for (int k = tid; k < D; k += kPickThreads)
        cent[(static_cast<size_t>(bh) * M + c) * D + k] = static_cast<double>(load_elem(X + static_cast<size_t>(tok) * D, k));
    const double* src = Dt + (static_cast<size_t>(bh) * L + best) * s0;
    double* dst = D2 + static_cast<size_t>(bh) * s0;
    if (c + 1 >= M) {
        for (int j = tid; j < s0; j += kPickThreads) dst[j] = src[j];
        return;
    }
    // running sums of D^2 over the sample in index order: thread tid owns
    // the contiguous range [tid per, (tid + 1) per)
    const int per = (s0 + kPickThreads - 1) / kPickThreads;
    const int j0 = min(s0, tid * per), j1 = min(s0, j0 + per);
    // the range's first kPickCache values, loaded together (indices clamped
    // into the sample, so no load is conditional) and kept for both passes;
    // the sums still run in index order
    double vals[kPickCache];
#pragma unroll
    for (int q = 0; q < kPickCache; ++q) vals[q] = src[min(j0 + q, s0 - 1)];
    double loc = 0.0;
#pragma unroll
    for (int q = 0; q < kPickCache; ++q) {
        if (j0 + q < j1) {
            dst[j0 + q] = vals[q];
            loc = loc + vals[q];
        }
    }
    for (int j = j0 + kPickCache; j < j1; ++j) {
        const double v = src[j];
        dst[j] = v;
        loc = loc + v;
    }
    // scan of the thread sums in thread order
    double inc = loc;
    for (int off = 1; off < kWave; off <<= 1) {
        const double y = __shfl_up(inc, off);
        if (lane_id() >= off) inc = y + inc;
    }
    double exc = __shfl_up(inc, 1);
    if (lane_id() == 0) exc = 0.0;
    if (lane_id() == kWave - 1) s_tot[wave_id()] = inc;
    __syncthreads();
    double wpre = 0.0, total = 0.0;
    for (int w = 0; w < kPickThreads / kWave; ++w) {
        if (w < wave_id()) wpre = wpre + s_tot[w];
        total = total + s_tot[w];
    }
    const double pre = wpre + exc;
    if (tid < L) s_u[tid] = draw_unit(km_word(seed, static_cast<uint64_t>(tid), 2, static_cast<uint64_t>(c + 1)));
    __syncthreads();
    double target[kKmMaxTrials];
#pragma unroll
    for (int t = 0; t < kKmMaxTrials; ++t) target[t] = t < L ? s_u[t] * total : 0.0;
    int found[kKmMaxTrials];
#pragma unroll
    for (int t = 0; t < kKmMaxTrials; ++t) found[t] = s0;
    double run = pre;
#pragma unroll
    for (int q = 0; q < kPickCache; ++q) {
        if (j0 + q < j1) {
            run = run + vals[q];
#pragma unroll
            for (int t = 0; t < kKmMaxTrials; ++t)
                if (t < L && found[t] == s0 && run > target[t]) found[t] = j0 + q;
        }
    }
    for (int j = j0 + kPickCache; j < j1; ++j) {
        run = run + src[j];
#pragma unroll
        for (int t = 0; t < kKmMaxTrials; ++t)
            if (t < L && found[t] == s0 && run > target[t]) found[t] = j;
    }
    // the first crossing of each trial: every thread past it has found a
    // position too, so the wave's minimum goes to LDS, one atomic per wave
#pragma unroll
    for (int t = 0; t < kKmMaxTrials; ++t) {
        if (t < L) {  // uniform
            const int f = static_cast<int>(wave_min64(static_cast<uint64_t>(found[t])));
            if (lane_id() == 0 && f < s0) atomicMin(&s_first[t], f);
        }
    }
    __syncthreads();
    if (tid < L) cand[bh * L + tid] = s_first[tid];
}

// Nearest center of 64 points per workgroup against center tiles of 32 in
// LDS.  Thread (pg, cg) = (tid / 16, tid % 16) scores points 4 pg .. 4 pg + 3
// against tile centers 2 cg, 2 cg + 1; rows are padded to D + 1 doubles so
// that the 16 center rows and the 4 point rows a wave reads per dimension sit
// in distinct banks.
template <typename T, int D, bool FINAL>
__global__ __launch_bounds__(kAsgThreads) void k_km_assign(
    const T* __restrict__ K, int N, int M, int batch, int step, uint64_t seed,
    const double* __restrict__ cent, const KmState* __restrict__ state, int* __restrict__ labels,
    double* __restrict__ bpart, int* __restrict__ bcnt, double* __restrict__ binert) {
#pragma clang fp contract(off)
    __shared__ float s_x[kAsgPts][D + 1];  // exact key values
    __shared__ double s_c[kAsgCen][D + 1];
    __shared__ int s_tok[kAsgPts];
    __shared__ int s_lab[kAsgPts];
    __shared__ double s_e[kAsgPts];
    __shared__ int s_ord[kAsgPts];
    const int bh = blockIdx.y, tid = threadIdx.x;
    if (!FINAL && state[bh].stop) return;
    const T* X = K + static_cast<size_t>(bh) * N * D;
    const int npts = FINAL ? N : batch;
    const int p0 = blockIdx.x * kAsgPts;
    if (tid < kAsgPts) {
        const int j = p0 + tid;
        int tok = -1;
        if (j < npts) tok = FINAL ? j : draw_index(km_word(seed, static_cast<uint64_t>(j), 3, static_cast<uint64_t>(step)), N);
        s_tok[tid] = tok;
    }
    __syncthreads();
    // point rows, 16 bytes per load: every load of a thread is independent
    {
        constexpr int kPer = 16 / static_cast<int>(sizeof(T));
        constexpr int kChunks = kAsgPts * D / kPer;
        static_assert(kChunks % kAsgThreads == 0, "whole 16-byte chunks per thread");
        float v[kChunks / kAsgThreads][kPer];
#pragma unroll
        for (int q = 0; q < kChunks / kAsgThreads; ++q) {
            const int e = q * kAsgThreads + tid;
            const int p = e / (D / kPer), k0 = (e % (D / kPer)) * kPer;
            const int tok = s_tok[p];
            load_row16(X + static_cast<size_t>(tok >= 0 ? tok : 0) * D + k0, v[q]);
        }
#pragma unroll
        for (int q = 0; q < kChunks / kAsgThreads; ++q) {
            const int e = q * kAsgThreads + tid;
            const int p = e / (D / kPer), k0 = (e % (D / kPer)) * kPer;
            const bool ok = s_tok[p] >= 0;
#pragma unroll
            for (int r = 0; r < kPer; ++r) s_x[p][k0 + r] = ok ? v[q][r] : 0.f;
        }
    }
    const int pg = tid >> 4, cg = tid & 15;
    double bd[4];
    int bu[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        bd[i] = INFINITY;
        bu[i] = 0x7fffffff;
    }
    const double* cb = cent + static_cast<size_t>(bh) * M * D;
    for (int ct = 0; ct < M; ct += kAsgCen) {
        __syncthreads();  // the previous tile is no longer read
        const int nct = min(kAsgCen, M - ct);
        {
            // the tile's values, all loads in flight before the LDS stores
            // (rows past the last center read center 0 and store zero)
            static_assert(kAsgCen * D % kAsgThreads == 0, "whole tile elements per thread");
            constexpr int kPer = kAsgCen * D / kAsgThreads;
            double v[kPer];
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                const int e = q * kAsgThreads + tid, u = e / D, k = e % D;
                v[q] = cb[static_cast<size_t>(u < nct ? ct + u : 0) * D + k];
            }
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                const int e = q * kAsgThreads + tid, u = e / D, k = e % D;
                s_c[u][k] = u < nct ? v[q] : 0.0;
            }
        }
        __syncthreads();
        double acc[4][2];
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i][0] = acc[i][1] = 0.0;
#pragma unroll 4
        for (int k = 0; k < D; ++k) {
            double xv[4], cv[2];
#pragma unroll
            for (int i = 0; i < 4; ++i) xv[i] = static_cast<double>(s_x[4 * pg + i][k]);
#pragma unroll
            for (int e = 0; e < 2; ++e) cv[e] = s_c[2 * cg + e][k];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const double t = xv[i] - cv[e];
                    acc[i][e] = acc[i][e] + t * t;
                }
            }
        }
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int u = ct + 2 * cg + e;
            if (2 * cg + e < nct) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (acc[i][e] < bd[i] || (acc[i][e] == bd[i] && u < bu[i])) {
                        bd[i] = acc[i][e];
                        bu[i] = u;
                    }
            }
        }
    }
    // the 16 center groups of a point: lowest distance, then lowest index
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const double od = __shfl_xor(bd[i], off);
            const int ou = __shfl_xor(bu[i], off);
            if (od < bd[i] || (od == bd[i] && ou < bu[i])) {
                bd[i] = od;
                bu[i] = ou;
            }
        }
    }
    if (cg == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            // no winner (NaN keys): center 0, so every label stays in range
            s_lab[4 * pg + i] = bu[i] < M ? bu[i] : 0;
            s_e[4 * pg + i] = bd[i];
        }
    }
    __syncthreads();
    if (FINAL) {
        if (tid < kAsgPts && s_tok[tid] >= 0) labels[static_cast<size_t>(bh) * N + s_tok[tid]] = s_lab[tid];
        return;
    }
    const int nv = min(kAsgPts, npts - p0);  // valid points: 0 .. nv - 1
    const size_t blk = static_cast<size_t>(bh) * gridDim.x + blockIdx.x;
    if (tid == 0) {
        double s = 0.0;
        for (int p = 0; p < nv; ++p) s = s + s_e[p];
        binert[blk] = s;
    }
    // points ordered by (center, position): a stable counting sort
    if (tid < nv) {
        const int u = s_lab[tid];
        int r = 0;
        for (int q = 0; q < nv; ++q) {
            const int v = s_lab[q];
            r += (v < u || (v == u && q < tid)) ? 1 : 0;
        }
        s_ord[r] = tid;
    }
    for (int u = tid; u < M; u += kAsgThreads) {
        int n = 0;
        for (int q = 0; q < nv; ++q) n += s_lab[q] == u ? 1 : 0;
        bcnt[blk * M + u] = n;
    }
    __syncthreads();
    // each present center's sum, in point order, one thread per dimension;
    // 16 sorted points' positions, labels and values are read ahead of
    // their additions (indices clamped into the valid points)
    if (tid < D) {
        int cur = -1;
        double acc = 0.0;
        for (int r0 = 0; r0 < nv; r0 += 16) {
            int pp[16], uu[16];
            float xx[16];
#pragma unroll
            for (int q = 0; q < 16; ++q) pp[q] = s_ord[min(r0 + q, nv - 1)];
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                uu[q] = s_lab[pp[q]];
                xx[q] = s_x[pp[q]][tid];
            }
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                if (r0 + q < nv) {
                    if (uu[q] != cur) {
                        if (cur >= 0) bpart[(blk * M + cur) * D + tid] = acc;
                        cur = uu[q];
                        acc = 0.0;
                    }
                    acc = acc + static_cast<double>(xx[q]);
                }
            }
        }
        if (cur >= 0) bpart[(blk * M + cur) * D + tid] = acc;
    }
}

template <int D>
__global__ __launch_bounds__(D) void k_km_update(int M, int nblk, const double* __restrict__ bpart,
                                                 const int* __restrict__ bcnt, double* __restrict__ cent,
                                                 double* __restrict__ w, const KmState* __restrict__ state) {
#pragma clang fp contract(off)
    const int u = blockIdx.x, bh = blockIdx.y, k = threadIdx.x;
    if (state[bh].stop) return;
    // kUpdBatch workgroups' counts and partial sums loaded together (a
    // partial of a center the workgroup did not see is stale and not added),
    // then added in workgroup order
    double S = 0.0;
    int n = 0;
    for (int b0 = 0; b0 < nblk; b0 += kUpdBatch) {
        int c[kUpdBatch];
        double v[kUpdBatch];
#pragma unroll
        for (int q = 0; q < kUpdBatch; ++q) {
            const size_t blk = static_cast<size_t>(bh) * nblk + min(b0 + q, nblk - 1);
            c[q] = b0 + q < nblk ? bcnt[blk * M + u] : 0;
            v[q] = bpart[(blk * M + u) * D + k];
        }
#pragma unroll
        for (int q = 0; q < kUpdBatch; ++q) {
            if (c[q]) {
                S = S + v[q];
                n += c[q];
            }
        }
    }
    if (n == 0) return;  // uniform over the workgroup
    const double wu = w[static_cast<size_t>(bh) * M + u];
    double* m = cent + (static_cast<size_t>(bh) * M + u) * D + k;
    *m = (*m * wu + S) / (wu + static_cast<double>(n));
    __syncthreads();  // every thread has read w before it changes
    if (k == 0) w[static_cast<size_t>(bh) * M + u] = wu + static_cast<double>(n);
}

template <typename T, int D>
__global__ __launch_bounds__(256) void k_km_control(
    const T* __restrict__ K, int N, int M, int batch, int step, uint64_t seed, int nblk, double alpha,
    double ratio, int max_no_improvement, const double* __restrict__ binert, double* __restrict__ cent,
    double* __restrict__ w, KmState* __restrict__ state) {
#pragma clang fp contract(off)
    __shared__ int s_mark[kKmMaxCenters];
    __shared__ double s_wb[kKmMaxCenters];
    __shared__ int s_count;
    __shared__ double s_wkeep;
    const int bh = blockIdx.x, tid = threadIdx.x;
    KmState* st = state + bh;
    if (st->stop) return;
    double* wb = w + static_cast<size_t>(bh) * M;
    // the weights staged in LDS by every thread, then scanned in index order
    // by one
    for (int u = tid; u < M; u += 256) s_wb[u] = wb[u];
    __syncthreads();
    if (tid == 0) {
        int count = 0;
        double wkeep = INFINITY;
        if (ratio > 0.0) {
            double wmax = s_wb[0];
            for (int u = 1; u < M; ++u)
                if (s_wb[u] > wmax) wmax = s_wb[u];
            const double thr = ratio * wmax;
            for (int u = 0; u < M; ++u) {
                if (s_wb[u] < thr && count < batch / 2)
                    s_mark[count++] = u;
                else if (s_wb[u] < wkeep)
                    wkeep = s_wb[u];
            }
        }
        s_count = count;
        s_wkeep = wkeep;
    }
    __syncthreads();
    const int count = s_count;
    const T* X = K + static_cast<size_t>(bh) * N * D;
    for (int r = 0; r < count; ++r) {
        const int u = s_mark[r];
        const int j = draw_index(km_word(seed, static_cast<uint64_t>(r), 4, static_cast<uint64_t>(step)), batch);
        const int tok = draw_index(km_word(seed, static_cast<uint64_t>(j), 3, static_cast<uint64_t>(step)), N);
        for (int k = tid; k < D; k += 256)
            cent[(static_cast<size_t>(bh) * M + u) * D + k] = static_cast<double>(load_elem(X + static_cast<size_t>(tok) * D, k));
        if (tid == 0) wb[u] = s_wkeep;
    }
    if (tid == 0) {
        double I = 0.0;
        for (int b0 = 0; b0 < nblk; b0 += 8) {
            double v[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] = binert[static_cast<size_t>(bh) * nblk + min(b0 + q, nblk - 1)];
#pragma unroll
            for (int q = 0; q < 8; ++q)
                if (b0 + q < nblk) I = I + v[q];
        }
        I = I / static_cast<double>(batch);
        KmState s = *st;
        s.ewa = step == 0 ? I : s.ewa * (1.0 - alpha) + I * alpha;
        if (s.ewa < s.ewa_min) {
            s.ewa_min = s.ewa;
            s.no_imp = 0;
        } else {
            s.no_imp += 1;
        }
        s.steps = step + 1;
        if (max_no_improvement > 0 && s.no_imp >= max_no_improvement) s.stop = 1;
        *st = s;
    }
}

__global__ __launch_bounds__(256) void k_km_init_state(KmState* __restrict__ state, double* __restrict__ w,
                                                       int BH, int M) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i < BH) {
        KmState s;
        s.ewa = 0.0;
        s.ewa_min = INFINITY;
        s.no_imp = 0;
        s.stop = 0;
        s.steps = 0;
        s.pad = 0;
        state[i] = s;
    }
    if (i < BH * M) w[i] = 0.0;
}

// Parents of one (sequence, KV head) from its labels: wave w counts and then
// places the tokens of its own contiguous segment, so members of a parent
// land in token order.  Outputs: members [N] (parent by parent), pbeg
// [Mp + 1] (first member position of each parent), toff [Mp + 1] (first team
// of each parent: sum of min(R, |C|) over the parents before it), and the
// pair's team count.  A label outside [0, Mp) sets *bad and is skipped.
__global__ __launch_bounds__(kListThreads) void k_parent_lists(
    const int* __restrict__ labels, int N, int Mp, int R, int* __restrict__ members,
    int* __restrict__ pbeg, int* __restrict__ toff, int* __restrict__ team_count, int* __restrict__ bad) {
    __shared__ int s_off[kListWaves][kMaxLabels];
    __shared__ int s_wt[2][kListWaves];
    __shared__ int s_carry[2];
    const int bh = blockIdx.x, tid = threadIdx.x, w = wave_id(), lane = lane_id();
    const int* lab = labels + static_cast<size_t>(bh) * N;
    int* mem = members + static_cast<size_t>(bh) * N;
    for (int e = tid; e < kListWaves * Mp; e += kListThreads) s_off[e / Mp][e % Mp] = 0;
    if (tid < 2) s_carry[tid] = 0;
    __syncthreads();
    const int seg = (N + kListWaves - 1) / kListWaves;
    const int i0 = min(N, w * seg), i1 = min(N, i0 + seg);
    for (int i = i0 + lane; i < i1; i += kWave) {
        const int L = lab[i];
        if (L < 0 || L >= Mp)
            atomicOr(bad, 1);
        else
            atomicAdd(&s_off[w][L], 1);
    }
    __syncthreads();
    // parent sizes and team counts, scanned over labels in chunks
    for (int base = 0; base < Mp; base += kListThreads) {
        const int u = base + tid;
        int cnt[kListWaves];
        int tot = 0;
#pragma unroll
        for (int v = 0; v < kListWaves; ++v) {
            cnt[v] = u < Mp ? s_off[v][u] : 0;
            tot += cnt[v];
        }
        const int x[2] = {tot, min(R, tot)};
        int ex[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int inc = wave_incl_scan(x[q]);
            if (lane == kWave - 1) s_wt[q][w] = inc;
            ex[q] = inc - x[q];
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            int pre = s_carry[q];
            for (int v = 0; v < w; ++v) pre += s_wt[q][v];
            ex[q] += pre;
        }
        if (u < Mp) {
            pbeg[static_cast<size_t>(bh) * (Mp + 1) + u] = ex[0];
            toff[static_cast<size_t>(bh) * (Mp + 1) + u] = ex[1];
            int run = ex[0];
#pragma unroll
            for (int v = 0; v < kListWaves; ++v) {
                s_off[v][u] = run;
                run += cnt[v];
            }
        }
        __syncthreads();
        if (tid < 2) {
            int add = 0;
            for (int v = 0; v < kListWaves; ++v) add += s_wt[tid][v];
            s_carry[tid] += add;
        }
        __syncthreads();
    }
    if (tid == 0) {
        pbeg[static_cast<size_t>(bh) * (Mp + 1) + Mp] = s_carry[0];
        toff[static_cast<size_t>(bh) * (Mp + 1) + Mp] = s_carry[1];
        team_count[bh] = s_carry[1];
    }
    // placement: per 64-token group, one ballot per distinct label
    const uint64_t lt = lanemask_lt();
    for (int g0 = i0; g0 < i1; g0 += kWave) {
        const int i = g0 + lane;
        const int L = i < i1 ? lab[i] : -1;
        const bool ok = L >= 0 && L < Mp;
        uint64_t pending = __ballot(ok);
        while (pending) {
            const int leader = __ffsll(static_cast<unsigned long long>(pending)) - 1;
            const int Lv = readlane(L, leader);
            const uint64_t m = __ballot(ok && L == Lv) & pending;
            const int base = s_off[w][Lv];
            if ((m >> lane) & 1ull) mem[base + __popcll(m & lt)] = i;
            // the new offset depends on the value every lane read, and a
            // wave's LDS accesses complete in order
            if (lane == leader) s_off[w][Lv] = base + static_cast<int>(__popcll(m));
            pending &= ~m;
        }
    }
}

// Absent teams past each pair's team count: no rows, log n = kAbsentLogN.
__global__ __launch_bounds__(256) void k_pad_teams(const int* __restrict__ team_count, int M, int N,
                                                   int BH, int* __restrict__ team_begin,
                                                   int* __restrict__ team_size, double* __restrict__ log_n,
                                                   int* __restrict__ rep_token) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= BH * M) return;
    const int bh = i / M, g = i % M;
    if (g < team_count[bh]) return;
    team_begin[i] = N;
    team_size[i] = 0;
    log_n[i] = kAbsentLogN;
    rep_token[i] = 0;
}

}  // namespace

KmLayout kmeans_layout(int BH, int N, int d, int M, int batch, int s0) {
    KmLayout L{};
    L.M = M;
    L.s0 = s0;
    L.L = 2 + static_cast<int>(floor(log(static_cast<double>(M))));
    L.nkpp = (s0 + kKppThreads - 1) / kKppThreads;
    L.nasg = (batch + kAsgPts - 1) / kAsgPts;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off += (bytes + 255) / 256 * 256;
        return o;
    };
    L.samp = take(sizeof(int) * static_cast<size_t>(s0));
    L.cand = take(sizeof(int) * static_cast<size_t>(BH) * L.L);
    L.D2 = take(sizeof(double) * static_cast<size_t>(BH) * s0);
    L.Dt = take(sizeof(double) * static_cast<size_t>(BH) * L.L * s0);
    L.part = take(sizeof(double) * static_cast<size_t>(BH) * L.nkpp * L.L);
    L.cent = take(sizeof(double) * static_cast<size_t>(BH) * M * d);
    L.w = take(sizeof(double) * static_cast<size_t>(BH) * M);
    L.state = take(sizeof(KmState) * static_cast<size_t>(BH));
    L.bpart = take(sizeof(double) * static_cast<size_t>(BH) * L.nasg * M * d);
    L.bcnt = take(sizeof(int) * static_cast<size_t>(BH) * L.nasg * M);
    L.binert = take(sizeof(double) * static_cast<size_t>(BH) * L.nasg);
    L.total = off;
    return L;
}

hipError_t launch_kmeans_seed(const void* K, santapp_dtype dtype, int BH, int N, int d,
                              const KmLayout& L, char* ws, uint64_t seed, hipStream_t s) {
    int* samp = reinterpret_cast<int*>(ws + L.samp);
    int* cand = reinterpret_cast<int*>(ws + L.cand);
    double* D2 = reinterpret_cast<double*>(ws + L.D2);
    double* Dt = reinterpret_cast<double*>(ws + L.Dt);
    double* part = reinterpret_cast<double*>(ws + L.part);
    double* cent = reinterpret_cast<double*>(ws + L.cent);
    k_kpp_sample<<<L.nkpp, kKppThreads, 0, s>>>(samp, L.s0, N, cand, L.L, BH, seed);
    for (int c = 0; c < L.M; ++c) {
#define SANTAPP_KPP(TT, DD)                                                                       \
    do {                                                                                         \
        k_kpp_dist<TT, DD><<<dim3(L.nkpp, BH), kKppThreads, 0, s>>>(                             \
            static_cast<const TT*>(K), N, samp, L.s0, cand, L.L, c, D2, Dt, part);              \
        k_kpp_pick<TT, DD><<<BH, kPickThreads, 0, s>>>(static_cast<const TT*>(K), N, samp, L.s0, \
                                                       cand, L.L, c, L.M, L.nkpp, D2, Dt, part,  \
                                                       cent, seed);                              \
    } while (0)
        if (dtype == SANTAPP_BF16 && d == 128) SANTAPP_KPP(bf16_t, 128);
        else if (dtype == SANTAPP_BF16) SANTAPP_KPP(bf16_t, 64);
        else if (d == 128) SANTAPP_KPP(float, 128);
        else SANTAPP_KPP(float, 64);
#undef SANTAPP_KPP
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    k_km_init_state<<<(BH * L.M + 255) / 256, 256, 0, s>>>(reinterpret_cast<KmState*>(ws + L.state),
                                                           reinterpret_cast<double*>(ws + L.w), BH, L.M);
    return hipGetLastError();
}

hipError_t launch_kmeans_steps(const void* K, santapp_dtype dtype, int BH, int N, int d,
                               const KmLayout& L, char* ws, int batch, int first, int count,
                               double alpha, double ratio, int max_no_improvement, uint64_t seed,
                               hipStream_t s) {
    double* cent = reinterpret_cast<double*>(ws + L.cent);
    double* w = reinterpret_cast<double*>(ws + L.w);
    KmState* st = reinterpret_cast<KmState*>(ws + L.state);
    double* bpart = reinterpret_cast<double*>(ws + L.bpart);
    int* bcnt = reinterpret_cast<int*>(ws + L.bcnt);
    double* binert = reinterpret_cast<double*>(ws + L.binert);
    for (int step = first; step < first + count; ++step) {
#define SANTAPP_STEP(TT, DD)                                                                          \
    do {                                                                                             \
        k_km_assign<TT, DD, false><<<dim3(L.nasg, BH), kAsgThreads, 0, s>>>(                        \
            static_cast<const TT*>(K), N, L.M, batch, step, seed, cent, st, nullptr, bpart, bcnt,  \
            binert);                                                                                 \
        k_km_update<DD><<<dim3(L.M, BH), DD, 0, s>>>(L.M, L.nasg, bpart, bcnt, cent, w, st);        \
        k_km_control<TT, DD><<<BH, 256, 0, s>>>(static_cast<const TT*>(K), N, L.M, batch, step,     \
                                                seed, L.nasg, alpha, ratio, max_no_improvement,     \
                                                binert, cent, w, st);                               \
    } while (0)
        if (dtype == SANTAPP_BF16 && d == 128) SANTAPP_STEP(bf16_t, 128);
        else if (dtype == SANTAPP_BF16) SANTAPP_STEP(bf16_t, 64);
        else if (d == 128) SANTAPP_STEP(float, 128);
        else SANTAPP_STEP(float, 64);
#undef SANTAPP_STEP
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_kmeans_labels(const void* K, santapp_dtype dtype, int BH, int N, int d,
                                const KmLayout& L, char* ws, int* labels, hipStream_t s) {
    const double* cent = reinterpret_cast<const double*>(ws + L.cent);
    const dim3 grid((N + kAsgPts - 1) / kAsgPts, BH);
#define SANTAPP_LAB(TT, DD)                                                                            \
    k_km_assign<TT, DD, true><<<grid, kAsgThreads, 0, s>>>(static_cast<const TT*>(K), N, L.M, 0, 0, 0, \
                                                           cent, nullptr, labels, nullptr, nullptr,   \
                                                           nullptr)
    if (dtype == SANTAPP_BF16 && d == 128) SANTAPP_LAB(bf16_t, 128);
    else if (dtype == SANTAPP_BF16) SANTAPP_LAB(bf16_t, 64);
    else if (d == 128) SANTAPP_LAB(float, 128);
    else SANTAPP_LAB(float, 64);
#undef SANTAPP_LAB
    return hipGetLastError();
}

hipError_t launch_parent_lists(const int* labels, int BH, int N, int Mp, int R, int* members, int* pbeg,
                               int* toff, int* team_count, int* bad, hipStream_t s) {
    k_parent_lists<<<BH, kListThreads, 0, s>>>(labels, N, Mp, R, members, pbeg, toff, team_count, bad);
    return hipGetLastError();
}

hipError_t launch_pad_teams(const int* team_count, int BH, int M, int N, int* team_begin, int* team_size,
                            double* log_n, int* rep_token, hipStream_t s) {
    const int total = BH * M;
    k_pad_teams<<<(total + 255) / 256, 256, 0, s>>>(team_count, M, N, BH, team_begin, team_size, log_n,
                                                    rep_token);
    return hipGetLastError();
}

}  // namespace santapp
