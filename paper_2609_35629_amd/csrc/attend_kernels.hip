// Split-K attention over the read plan, and the split merge.
//
// k_attend  eq. method-estimate in log space: every row read gets the logit
//           w_{h,i} = scale q_h.k_i - log c_{g(i),h} for each query head h of
//           the KV head (no weight when h did not select the team; no
//           correction for suffix rows and on the dense path), and an online
//           softmax accumulates (m, l, acc) per head.  The rows of one KV head,
//           [union rows ; suffix rows], are cut into ranges of kSplitRows
//           rows; one workgroup owns one range and writes one partial per
//           head.  The query heads sharing the KV head share every K/V load.
// k_merge   rescales the partials of a head to a common maximum and divides
//           the weighted value sum by the mass.
//
// Scores on the matrix cores: for a tile of 16 rows, S[head][row] = Q K^T
// with the query heads of the KV head (padded to 16) as the M dimension.
// bf16 keys use v_mfma_f32_16x16x32_bf16 with the fp32 query split into
// three bf16 terms (exact to fp32 precision), fp32 keys v_mfma_f32_16x16x4_f32.
// The softmax runs on the 16x16 accumulator (lanes = rows, registers =
// heads); the value sum runs on the vector ALUs with 16 lanes per row, each
// owning d/16 dimensions of all heads, and the probabilities broadcast
// through LDS.
// Exponentials are base 2 with log2(e) folded into the query and the
// corrections.  "No weight" is the finite logit kNeg, so differences of
// logits never form inf - inf; a state that only ever saw kNeg logits gets
// weight exp2(kNeg - m) = 0 as soon as it meets a real logit, and every head
// has at least one real logit.
#include <math.h>

#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kAttThreads = 256;
constexpr int kAttWaves = kAttThreads / kWave;
constexpr int kWaveRows = kSplitRows / kAttWaves;  // 32 rows per wave
constexpr int kTiles = kWaveRows / 16;             // two 16-row MFMA tiles
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNeg = -1.0e30f;   // logit of a row that carries no weight
constexpr float kSkip = 1.0e30f;   // correction of a head that did not select the team
constexpr int kMergeThreads = 256;
constexpr int kMergeDims = 32;  // output dimensions per merge workgroup

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Scale factor of a state with maximum m when rebased to mn.
__device__ __forceinline__ float rebase(float m, float mn) { return fast_exp2(m - mn); }

template <int CTRL>
__device__ __forceinline__ float dpp_max_step(float v) {
    return fmaxf(v, dpp_f32<CTRL>(v));
}

__device__ __forceinline__ float row16_max(float v) {
    v = dpp_max_step<0x128>(v);
    v = dpp_max_step<0x124>(v);
    v = dpp_max_step<0x122>(v);
    v = dpp_max_step<0x121>(v);
    return v;
}

// Scores of one 16-row tile.  Lane l = 16 c + j feeds row j of the tile and
// holds head 4 c + r of row j in accumulator register r.
template <typename T, int D>
struct QK;

template <int D>
struct QK<bf16_t, D> {
    // block kb, lane group c: 16-byte chunk 4 kb + c of the row (dims
    // 8 (4 kb + c) .. + 8); the same dims of the query head l % 16
    static constexpr int KB = D / 32;
    using frag = uint4;
    bf16x8 qa[KB][3];

    __device__ __forceinline__ void load_q(const float* qrow, float scale, int c) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            const float4* p = reinterpret_cast<const float4*>(qrow + 8 * (4 * kb + c));
            const float4 u = p[0], v = p[1];
            const float x[8] = {u.x, u.y, u.z, u.w, v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float f = x[e] * scale;
                const __bf16 a = static_cast<__bf16>(f);
                const float r1 = f - static_cast<float>(a);
                const __bf16 b = static_cast<__bf16>(r1);
                const float r2 = r1 - static_cast<float>(b);
                qa[kb][0][e] = a;
                qa[kb][1][e] = b;
                qa[kb][2][e] = static_cast<__bf16>(r2);
            }
        }
    }
    __device__ __forceinline__ void load_k(const bf16_t* row, int c, frag* f) const {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) f[kb] = *reinterpret_cast<const uint4*>(row + 8 * (4 * kb + c));
    }
    __device__ __forceinline__ f32x4 scores(const frag* f) const {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            const bf16x8 k = __builtin_bit_cast(bf16x8, f[kb]);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[kb][2], k, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[kb][1], k, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[kb][0], k, acc, 0, 0, 0);
        }
        return acc;
    }
};

template <int D>
struct QK<float, D> {
    // block kb, lane group c: dim (D / 4) c + kb
    static constexpr int KB = D / 4;
    using frag = float4;
    float qa[KB];

    __device__ __forceinline__ void load_q(const float* qrow, float scale, int c) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) qa[kb] = qrow[(D / 4) * c + kb] * scale;
    }
    __device__ __forceinline__ void load_k(const float* row, int c, frag* f) const {
#pragma unroll
        for (int i = 0; i < KB / 4; ++i) f[i] = *reinterpret_cast<const float4*>(row + (D / 4) * c + 4 * i);
    }
    __device__ __forceinline__ f32x4 scores(const frag* f) const {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < KB / 4; ++i) {
            const float k[4] = {f[i].x, f[i].y, f[i].z, f[i].w};
#pragma unroll
            for (int e = 0; e < 4; ++e)
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[4 * i + e], k[e], acc, 0, 0, 0);
        }
        return acc;
    }
};

template <typename T, int D>
constexpr int frag_count() {
    return sizeof(T) == 2 ? D / 32 : D / 16;
}

// d / 16 consecutive value dims of a row for one of 16 lanes.
template <typename T, int VPL>
struct RowChunk;

template <>
struct RowChunk<bf16_t, 8> {  // d = 128: 8 bf16 = 16 bytes per lane
    using raw = uint4;
    static __device__ __forceinline__ raw load(const bf16_t* p) {
        return *reinterpret_cast<const uint4*>(p);
    }
    static __device__ __forceinline__ void unpack(const raw& u, float* x) {
        x[0] = bf16lo(u.x); x[1] = bf16hi(u.x); x[2] = bf16lo(u.y); x[3] = bf16hi(u.y);
        x[4] = bf16lo(u.z); x[5] = bf16hi(u.z); x[6] = bf16lo(u.w); x[7] = bf16hi(u.w);
    }
};

template <>
struct RowChunk<bf16_t, 4> {  // d = 64
    using raw = uint2;
    static __device__ __forceinline__ raw load(const bf16_t* p) {
        return *reinterpret_cast<const uint2*>(p);
    }
    static __device__ __forceinline__ void unpack(const raw& u, float* x) {
        x[0] = bf16lo(u.x); x[1] = bf16hi(u.x); x[2] = bf16lo(u.y); x[3] = bf16hi(u.y);
    }
};

template <>
struct RowChunk<float, 8> {
    struct raw {
        float4 a, b;
    };
    static __device__ __forceinline__ raw load(const float* p) {
        raw r;
        r.a = *reinterpret_cast<const float4*>(p);
        r.b = *reinterpret_cast<const float4*>(p + 4);
        return r;
    }
    static __device__ __forceinline__ void unpack(const raw& r, float* x) {
        x[0] = r.a.x; x[1] = r.a.y; x[2] = r.a.z; x[3] = r.a.w;
        x[4] = r.b.x; x[5] = r.b.y; x[6] = r.b.z; x[7] = r.b.w;
    }
};

template <>
struct RowChunk<float, 4> {
    using raw = float4;
    static __device__ __forceinline__ raw load(const float* p) {
        return *reinterpret_cast<const float4*>(p);
    }
    static __device__ __forceinline__ void unpack(const raw& r, float* x) {
        x[0] = r.x; x[1] = r.y; x[2] = r.z; x[3] = r.w;
    }
};

// Rows of one KV head are [prompt rows ; suffix rows]; the prompt part holds
// rows_u rows (the union rows of the plan, or all N rows on the dense path).
__device__ __forceinline__ int split_count(int rows_u, int T_suf) {
    return (rows_u + T_suf + kSplitRows - 1) / kSplitRows;
}

template <typename T, int D, int G, bool DENSE>
__global__ __launch_bounds__(kAttThreads) void k_attend(
    const T* __restrict__ K, const T* __restrict__ V, const T* __restrict__ sK,
    const T* __restrict__ sV, const float* __restrict__ q, int N, int T_suf, int M, int Hkv,
    int Hq, int Greal, float scale_log2, int max_split, const int* __restrict__ hdr,
    const int* __restrict__ split_team, const int* __restrict__ ubeg,
    const int* __restrict__ urs, const float* __restrict__ ulogc, float* __restrict__ part_o,
    float* __restrict__ part_ml) {
    constexpr int NF = frag_count<T, D>();
    constexpr int VPL = D / 16;  // value dims per lane (16 lanes per row)
    using QKT = QK<T, D>;
    using VC = RowChunk<T, VPL>;
    __shared__ int s_src[kSplitRows];          // prompt row, or -(suffix row) - 1
    __shared__ float4 s_lc[kSplitRows][2];     // log2 corrections of heads 0..7
    __shared__ int s_trs[kSplitRows + 1];      // union slice: first row of each team
    __shared__ int s_tbeg[kSplitRows];         //   its first packed row
    __shared__ float4 s_tlc[kSplitRows][2];    //   its corrections
    __shared__ float4 s_p[kAttWaves][16][2];   // probabilities of one tile
    __shared__ float4 s_a[kAttWaves][2];       // rescale factors of one tile
    __shared__ float s_m[kAttWaves][8];
    __shared__ float s_l[kAttWaves][8];
    __shared__ float s_o[kAttWaves][G][D];

    const int bh = blockIdx.x;  // KV heads vary fastest: active ranges dispatch first
    const int s = blockIdx.y;
    const int b = bh / Hkv, kv = bh - b * Hkv;
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    const int c = lane >> 4, j16 = lane & 15;

    // plan header and the first union team of this range, in one round trip
    int rows_u = N, U = 0, t0 = 0;
    if (!DENSE) {
        U = hdr[bh * 4 + 0];
        rows_u = hdr[bh * 4 + 1];
        t0 = split_team[static_cast<size_t>(bh) * max_split + s];
    }
    // query fragments: head l % 16 of this KV head (zero for padding heads)
    QKT qk;
    {
        const int h = j16;
        const int hq = kv * Greal + (h < Greal ? h : 0);
        qk.load_q(q + (static_cast<size_t>(b) * Hq + hq) * D, h < Greal ? scale_log2 : 0.f, c);
    }
    const int total = rows_u + T_suf;
    if (s >= split_count(rows_u, T_suf)) return;  // uniform: nothing to read here
    const int r0 = s * kSplitRows;
    const int nrows = min(kSplitRows, total - r0);

    if (!DENSE && r0 < rows_u) {
        // union teams t0 .. t0 + kSplitRows - 1 hold every union row of the range
        const int* ursb = urs + static_cast<size_t>(bh) * (M + 1);
        for (int j = tid; j <= kSplitRows; j += kAttThreads) {
            const int t = t0 + j;
            s_trs[j] = (t <= U) ? ursb[t] : 0x7fffffff;
        }
        if (tid < kSplitRows) {
            const int t = min(t0 + tid, U - 1);
            s_tbeg[tid] = ubeg[static_cast<size_t>(bh) * M + t];
            const float4* L = reinterpret_cast<const float4*>(ulogc + (static_cast<size_t>(bh) * M + t) * kLogcStride);
            s_tlc[tid][0] = L[0];
            s_tlc[tid][1] = L[1];
        }
        __syncthreads();
    }
    if (tid < kSplitRows) {
        // rows past the range repeat the last row with no weight for any head
        const int r = r0 + min(tid, nrows - 1);
        float lcv[8];
#pragma unroll
        for (int h = 0; h < 8; ++h) lcv[h] = (h < Greal && tid < nrows) ? 0.f : kSkip;
        int src;
        if (r < rows_u) {
            if (DENSE) {
                src = r;
            } else {
                int lo = 0, hi = min(kSplitRows, U - t0) - 1;  // largest j with s_trs[j] <= r
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (s_trs[mid] <= r)
                        lo = mid;
                    else
                        hi = mid - 1;
                }
                src = s_tbeg[lo] + (r - s_trs[lo]);
                const float4 u = s_tlc[lo][0], v = s_tlc[lo][1];
                const float x[8] = {u.x, u.y, u.z, u.w, v.x, v.y, v.z, v.w};
#pragma unroll
                for (int h = 0; h < 8; ++h)
                    if (h < Greal && tid < nrows) lcv[h] = x[h] * kLog2e;
            }
        } else {
            src = -(r - rows_u) - 1;
        }
        s_src[tid] = src;
        s_lc[tid][0] = make_float4(lcv[0], lcv[1], lcv[2], lcv[3]);
        s_lc[tid][1] = make_float4(lcv[4], lcv[5], lcv[6], lcv[7]);
    }
    __syncthreads();

    const T* Kb = K + static_cast<size_t>(bh) * N * D;
    const T* Vb = V + static_cast<size_t>(bh) * N * D;
    const T* sKb = sK + static_cast<size_t>(bh) * T_suf * D;
    const T* sVb = sV + static_cast<size_t>(bh) * T_suf * D;
    const int wrow = w * kWaveRows;

    // every K and V load of the wave's 32 rows is issued before any math:
    // K as MFMA fragments (lane (c, j) -> row j of a 16-row tile), V with 16
    // lanes per row (lane (c, j) -> dims VPL j .. of rows c, c + 4, ...)
    typename QKT::frag kf[kTiles][NF];
    typename VC::raw vr[kWaveRows / 4];
#pragma unroll
    for (int t = 0; t < kTiles; ++t) {
        const int src = s_src[wrow + 16 * t + j16];
        const T* row = (src >= 0) ? Kb + static_cast<size_t>(src) * D
                                  : sKb + static_cast<size_t>(-src - 1) * D;
        qk.load_k(row, c, kf[t]);
    }
#pragma unroll
    for (int k = 0; k < kWaveRows / 4; ++k) {
        const int src = s_src[wrow + 4 * k + c];
        const T* row = (src >= 0) ? Vb + static_cast<size_t>(src) * D
                                  : sVb + static_cast<size_t>(-src - 1) * D;
        vr[k] = VC::load(row + VPL * j16);
    }

    float m[4], l[4], acc[G][VPL];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        m[r] = kNeg;
        l[r] = 0.f;
    }
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < VPL; ++e) acc[h][e] = 0.f;

#pragma unroll
    for (int t = 0; t < kTiles; ++t) {
        const f32x4 sc = qk.scores(kf[t]);
        // lane (c, j16): row j16 of the tile, heads 4 c .. 4 c + 3
        const float4 lc = s_lc[wrow + 16 * t + j16][c & 1];
        const float lcr[4] = {lc.x, lc.y, lc.z, lc.w};
        float a[4], p[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float x = (c < 2) ? sc[r] - lcr[r] : kNeg;
            const float mn = fmaxf(m[r], row16_max(x));
            a[r] = rebase(m[r], mn);
            p[r] = fast_exp2(x - mn);
            l[r] = l[r] * a[r] + row16_sum(p[r]);
            m[r] = mn;
        }
        if (c < 2) {
            s_p[w][j16][c] = make_float4(p[0], p[1], p[2], p[3]);
            if (j16 == 0) s_a[w][c] = make_float4(a[0], a[1], a[2], a[3]);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        {
            const float4 a0 = s_a[w][0], a1 = s_a[w][1];
            const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
#pragma unroll
            for (int h = 0; h < G; ++h)
#pragma unroll
                for (int e = 0; e < VPL; ++e) acc[h][e] *= av[h];
        }
        // this lane group's rows of the tile: c, c + 4, c + 8, c + 12
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            float v[VPL];
            VC::unpack(vr[4 * t + kk], v);
            const float4 p0 = s_p[w][4 * kk + c][0], p1 = s_p[w][4 * kk + c][1];
            const float pv[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
            for (int h = 0; h < G; ++h)
#pragma unroll
                for (int e = 0; e < VPL; ++e) acc[h][e] = fmaf(pv[h], v[e], acc[h][e]);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }

    // the four lane groups share each head's maximum: their sums simply add
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < VPL; ++e) {
            float x = acc[h][e];
            x += __shfl_xor(x, 16);
            x += __shfl_xor(x, 32);
            acc[h][e] = x;
        }
    if (c < 2 && j16 == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            s_m[w][4 * c + r] = m[r];
            s_l[w][4 * c + r] = l[r];
        }
    }
    if (c == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
            for (int e = 0; e < VPL; ++e) s_o[w][h][VPL * j16 + e] = acc[h][e];
    }
    __syncthreads();
    for (int idx = tid; idx < Greal * D; idx += kAttThreads) {
        const int h = idx / D, jd = idx - h * D;
        float mx = s_m[0][h];
#pragma unroll
        for (int v = 1; v < kAttWaves; ++v) mx = fmaxf(mx, s_m[v][h]);
        float lsum = 0.f, osum = 0.f;
#pragma unroll
        for (int v = 0; v < kAttWaves; ++v) {
            const float a = rebase(s_m[v][h], mx);
            lsum += s_l[v][h] * a;
            osum += s_o[v][h][jd] * a;
        }
        const size_t pidx = (static_cast<size_t>(b) * Hq + kv * Greal + h) * max_split + s;
        part_o[pidx * D + jd] = osum;
        if (jd == 0) {
            part_ml[pidx * 2 + 0] = mx;
            part_ml[pidx * 2 + 1] = lsum;
        }
    }
}

// One workgroup per (sequence, query head, 32 output dimensions).
__global__ __launch_bounds__(kMergeThreads) void k_merge(
    const float* __restrict__ part_o, const float* __restrict__ part_ml,
    const int* __restrict__ hdr, int N, int T_suf, int Hq, int Hkv, int max_split, int D,
    float* __restrict__ out) {
    __shared__ float s_red[kMergeThreads / kWave];
    __shared__ float s_acc[kMergeThreads / kMergeDims][kMergeDims];
    const int bhq = blockIdx.x;
    const int b = bhq / Hq, h = bhq - b * Hq;
    const int bh = b * Hkv + h / (Hq / Hkv);
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    const int rows_u = hdr ? hdr[bh * 4 + 1] : N;
    const int n = split_count(rows_u, T_suf);
    const float* ml = part_ml + static_cast<size_t>(bhq) * max_split * 2;
    const float* po = part_o + static_cast<size_t>(bhq) * max_split * D;

    float mx = -INFINITY;
    for (int s = tid; s < n; s += kMergeThreads) mx = fmaxf(mx, ml[2 * s]);
    for (int off = kWave / 2; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    if (lane == 0) s_red[w] = mx;
    __syncthreads();
    mx = s_red[0];
    for (int v = 1; v < kMergeThreads / kWave; ++v) mx = fmaxf(mx, s_red[v]);
    __syncthreads();

    float lsum = 0.f;
    for (int s = tid; s < n; s += kMergeThreads) lsum += ml[2 * s + 1] * rebase(ml[2 * s], mx);
    for (int off = kWave / 2; off > 0; off >>= 1) lsum += __shfl_xor(lsum, off);
    if (lane == 0) s_red[w] = lsum;
    __syncthreads();
    lsum = 0.f;
    for (int v = 0; v < kMergeThreads / kWave; ++v) lsum += s_red[v];

    const int j = blockIdx.y * kMergeDims + (tid % kMergeDims);
    const int sl = tid / kMergeDims;
    constexpr int kLanes = kMergeThreads / kMergeDims;
    float acc = 0.f;
#pragma unroll 4
    for (int s = sl; s < n; s += kLanes) acc += po[static_cast<size_t>(s) * D + j] * rebase(ml[2 * s], mx);
    s_acc[sl][tid % kMergeDims] = acc;
    __syncthreads();
    if (tid < kMergeDims) {
        float t = 0.f;
#pragma unroll
        for (int v = 0; v < kLanes; ++v) t += s_acc[v][tid];
        out[static_cast<size_t>(bhq) * D + blockIdx.y * kMergeDims + tid] = t / lsum;
    }
}

__global__ void k_zero(uint4* __restrict__ p, size_t n16, unsigned char* __restrict__ tail,
                       int ntail) {
    const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < n16; i += stride)
        p[i] = make_uint4(0, 0, 0, 0);
    if (blockIdx.x == 0 && static_cast<int>(threadIdx.x) < ntail) tail[threadIdx.x] = 0;
}

template <typename T, int D, int G>
hipError_t attend_g(const AttendArgs& a, hipStream_t s) {
    const dim3 grid(a.B * a.Hkv, a.max_split);
    const float sl2 = a.scale * kLog2e;
    const T* K = static_cast<const T*>(a.K);
    const T* V = static_cast<const T*>(a.V);
    const T* sK = static_cast<const T*>(a.sK);
    const T* sV = static_cast<const T*>(a.sV);
    if (a.dense) {
        k_attend<T, D, G, true><<<grid, kAttThreads, 0, s>>>(
            K, V, sK, sV, a.q, a.N, a.T, 0, a.Hkv, a.Hq, a.G, sl2, a.max_split, nullptr, nullptr,
            nullptr, nullptr, nullptr, a.part_o, a.part_ml);
    } else {
        const DecodeLayout& L = *a.lay;
        k_attend<T, D, G, false><<<grid, kAttThreads, 0, s>>>(
            K, V, sK, sV, a.q, a.N, a.T, a.M, a.Hkv, a.Hq, a.G, sl2, a.max_split,
            reinterpret_cast<const int*>(a.ws + L.hdr), reinterpret_cast<const int*>(a.ws + L.split),
            reinterpret_cast<const int*>(a.ws + L.ubeg), reinterpret_cast<const int*>(a.ws + L.urs),
            reinterpret_cast<const float*>(a.ws + L.ulogc), a.part_o, a.part_ml);
    }
    return hipGetLastError();
}

template <typename T, int D>
hipError_t attend_d(const AttendArgs& a, hipStream_t s) {
    switch (a.G) {
        case 1: return attend_g<T, D, 1>(a, s);
        case 2: return attend_g<T, D, 2>(a, s);
        case 3:
        case 4: return attend_g<T, D, 4>(a, s);
        case 5:
        case 6:
        case 7: return attend_g<T, D, 7>(a, s);
        case 8: return attend_g<T, D, 8>(a, s);
        default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t attend_t(const AttendArgs& a, hipStream_t s) {
    switch (a.d) {
        case 64: return attend_d<T, 64>(a, s);
        case 128: return attend_d<T, 128>(a, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_attend(const AttendArgs& a, hipStream_t s) {
    return a.dtype == SANTAPP_BF16 ? attend_t<bf16_t>(a, s) : attend_t<float>(a, s);
}

hipError_t launch_merge(const AttendArgs& a, hipStream_t s) {
    const int* hdr = a.dense ? nullptr : reinterpret_cast<const int*>(a.ws + a.lay->hdr);
    const dim3 grid(a.B * a.Hq, a.d / kMergeDims);
    k_merge<<<grid, kMergeThreads, 0, s>>>(a.part_o, a.part_ml, hdr, a.N, a.T, a.Hq, a.Hkv,
                                           a.max_split, a.d, a.out);
    return hipGetLastError();
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
    const size_t n16 = bytes / 16;
    const int ntail = static_cast<int>(bytes - n16 * 16);
    const size_t want = (n16 + 255) / 256;
    const unsigned blocks = static_cast<unsigned>(want == 0 ? 1 : (want < 4096 ? want : 4096));
    k_zero<<<blocks, 256, 0, s>>>(static_cast<uint4*>(p), n16,
                                  static_cast<unsigned char*>(p) + n16 * 16, ntail);
    return hipGetLastError();
}

}  // namespace santapp
