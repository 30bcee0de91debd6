// Attention over the read plan, and the merge of the chunk partials.
//
// k_attend_mfma (bf16) / k_attend (fp32)
//           eq. method-estimate in log space.  A wave reads one chunk at a
//           time: up to kChunkRows consecutive packed rows of one union team,
//           or of the suffix.  Every query head h of the KV head that selected the
//           team gets the logits w_{h,i} = scale q_h.k_i over the chunk's rows
//           and an online softmax state (m, l, acc); all rows of a chunk
//           belong to one team, so the team's correction -log c_{g,h} enters
//           as a shift of the state's maximum.  Heads that did not select the
//           team skip the value sum and leave an empty state.  The query heads
//           sharing the KV head share every K/V load.  The dense path (and the
//           full budget) cuts [prompt rows ; suffix rows] into chunks with
//           every head and no correction.
// k_merge   rescales the chunk states of a head to a common maximum and
//           divides the weighted value sum by the mass.
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
// weight exp2(kNeg - m) = 0 as soon as it meets a real logit.
#include <math.h>

#include <algorithm>

#include <hip/hip_ext.h>

#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

static_assert(kChunkRows % 32 == 0, "a sampled unit is whole 32-row steps");
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNeg = -1.0e30f;   // logit of a row that carries no weight
constexpr float kEmpty = -1.0e29f; // chunk states with a maximum below this are empty

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

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
    // 8 (4 kb + c) .. + 8); the same dims of the query head of M row
    // l % 16, as three bf16 terms per fp32 value (exact to fp32).
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
                const __bf16 h0 = static_cast<__bf16>(f);
                const float r1 = f - static_cast<float>(h0);
                const __bf16 h1 = static_cast<__bf16>(r1);
                const float r2 = r1 - static_cast<float>(h1);
                qa[kb][0][e] = h0;
                qa[kb][1][e] = h1;
                qa[kb][2][e] = static_cast<__bf16>(r2);
            }
        }
    }
    static __device__ __forceinline__ void load_k(const bf16_t* row, int c, frag* f) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) f[kb] = load_stream(row + 8 * (4 * kb + c));
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
    // block kb, lane group c: dim (D / 4) c + kb; the query stays in registers
    static constexpr int KB = D / 4;
    using frag = float4;
    float qa[KB];

    __device__ __forceinline__ void load_q(const float* qrow, float scale, int c) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) qa[kb] = qrow[(D / 4) * c + kb] * scale;
    }
    __device__ __forceinline__ void load_k(const float* row, int c, frag* f) const {
#pragma unroll
        for (int i = 0; i < KB / 4; ++i) f[i] = load_stream_f(row + (D / 4) * c + 4 * i);
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
    static __device__ __forceinline__ raw load(const bf16_t* p) { return load_stream(p); }
    static __device__ __forceinline__ void unpack(const raw& u, float* x) {
        x[0] = bf16lo(u.x); x[1] = bf16hi(u.x); x[2] = bf16lo(u.y); x[3] = bf16hi(u.y);
        x[4] = bf16lo(u.z); x[5] = bf16hi(u.z); x[6] = bf16lo(u.w); x[7] = bf16hi(u.w);
    }
};

template <>
struct RowChunk<bf16_t, 4> {  // d = 64
    using raw = uint2;
    static __device__ __forceinline__ raw load(const bf16_t* p) { return load_stream8(p); }
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
        r.a = load_stream_f(p);
        r.b = load_stream_f(p + 4);
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
    static __device__ __forceinline__ raw load(const float* p) { return load_stream_f(p); }
    static __device__ __forceinline__ void unpack(const raw& r, float* x) {
        x[0] = r.x; x[1] = r.y; x[2] = r.z; x[3] = r.w;
    }
};

// Value sum of a 32-row step on the matrix cores (bf16 values):
// O[h][dim] += sum_row P[h][row] V[row][dim] as v_mfma_f32_16x16x32_bf16
// with the step's rows as the K dimension, one product per 16 dims.
//   A (probabilities): M row i < 8 holds the bf16 high part of head i, row
//     i + 8 the bf16 low part (p - high), so a product carries p to 16
//     significant bits; the two halves of the accumulator are added when
//     the unit ends.
//   B (values): 8 consecutive rows of one dim per lane, read from an LDS
//     copy of the 32 x D tile with the transposing read ds_read_b64_tr_b16:
//     lane 4 a + e of a 16-lane block receives element e of the 8-byte
//     words that lanes a, a + 4, a + 8, a + 12 of the block address, so
//     when lane s addresses row s / 4, dims 4 (s % 4) .. + 4 of a 16-dim
//     block, lane n gets four consecutive rows of dim n.
//   The tile's 32-byte pieces are XOR-swizzled per row so that the eight
//   rows one half-wave reads fall in distinct LDS banks.
template <int D>
struct VTile {
    static constexpr int NB = D / 16;  // 16-dim blocks = products per step
    static constexpr int kBytes = 32 * D * 2;
    static __device__ __forceinline__ int swz(int row) { return ((row & 3) | ((row >> 1) & 4)) & (NB - 1); }
    static __device__ __forceinline__ int offset(int row, int byte) {
        return row * (2 * D) + ((((byte >> 5) ^ swz(row))) << 5) + (byte & 31);
    }
    // B operand of block nb for lane l
    static __device__ __forceinline__ bf16x8 operand(const char* tile, int nb, int lane) {
        const int blk = lane >> 4, s = lane & 15;
        const int r = 8 * blk + (s >> 2);
        const int byte = 32 * nb + 8 * (s & 3);
        typedef short v4i16 __attribute__((ext_vector_type(4)));
        typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(tile + offset(r, byte)));
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(tile + offset(r + 4, byte)));
        return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
};

// One wave per workgroup (the fp32 kernel).  The sampled path's units are
// chunks of at most kChunkRows consecutive rows of one union team or of the
// suffix; the dense path's units are kDenseRows rows; both are walked 32 rows
// at a time with the softmax state carried along.  Each (sequence, KV head)
// pair's units sit in that pair's region of the sampler's list; wave w serves
// pair w % BH and takes its units w / BH, + gridDim.x / BH, ... (a loop
// bounded by the pair's count).  A unit's state for head h goes to position
// pos[h] of that head's list (its unit index on the dense path, where every
// head reads every unit).
//
// Register layout of the softmax: lane l = 16 c + j holds, in register r,
// M row 4 c + r of the score tile, i.e. query head (4 c + r) % 8 of row j
// (for bf16 the query fills M rows 8..15 with a copy of heads 0..7, so lane
// groups 2 and 3 repeat the states of groups 0 and 1 and every lane has the
// state of the heads its value accumulators hold).
template <typename T, int D, int GT, bool DENSE>
__global__ __launch_bounds__(kWave, 2) void k_attend(
    const T* __restrict__ K, const T* __restrict__ V, const T* __restrict__ sK,
    const T* __restrict__ sV, const float* __restrict__ q, int N, int T_suf, int BH, int Hkv,
    int Hq, int G, int M, float scale_log2, int max_chunks, int max_hunits,
    const PlanHeader* __restrict__ hdr, const Chunk* __restrict__ chunks,
    const float* __restrict__ ulogc, float* __restrict__ part_o, float* __restrict__ part_ml) {
    constexpr int NF = frag_count<T, D>();
    constexpr int VPL = D / 16;  // value dims per lane (16 lanes per row)
    constexpr int UR = DENSE ? kDenseRows : kChunkRows;
    constexpr bool kMfmaPV = sizeof(T) == 2;
    using QKT = QK<T, D>;
    using VC = RowChunk<T, VPL>;
    using VT = VTile<D>;
    constexpr int NB = VT::NB;
    __shared__ __attribute__((aligned(16))) char s_v[kMfmaPV ? VT::kBytes : 16];  // value tile
    __shared__ float4 s_pt[8][8];  // probabilities [head][row / 4] (bf16 values)
    __shared__ float4 s_p[16][2];  // probabilities [row][head / 4] of one tile (fp32 values)
    __shared__ float4 s_a[2];      // rescale factors of one tile (fp32 values)

    const int lane = lane_id();
    const int c = lane >> 4, j16 = lane & 15;
    const int hsel = 4 * (c & 1);  // first head of this lane's registers
    const int ncp = (N + UR - 1) / UR;
    const int nchd = ncp + (T_suf + UR - 1) / UR;  // dense units per (b, kv)
    // the sampled path's wave serves one (b, kv) pair: entries
    // blockIdx.x / BH, + gridDim.x / BH, ... of the pair's region of the
    // sampler's unit list; the dense path walks its (b, kv)-major list
    const int pbh = DENSE ? 0 : static_cast<int>(blockIdx.x) % BH;
    const Chunk* const pchunks = chunks + static_cast<size_t>(pbh) * max_chunks;
    const int total = DENSE ? BH * nchd : min(hdr[pbh].chunks, max_chunks);
    auto descriptor = [&](int u) {
        if (DENSE) {
            const int bhx = u / nchd, cix = u - bhx * nchd;
            const bool suf = cix >= ncp;
            const int begin = (suf ? cix - ncp : cix) * UR;
            Chunk d;
            d.begin = begin;
            d.slot = suf ? -1 : 0;
            d.meta = chunk_meta(min(UR, (suf ? T_suf : N) - begin), (1 << G) - 1, bhx);
            d.ci = cix;
            d.p01 = d.p23 = d.p45 = d.p67 = 0u;
            return d;
        }
        return pchunks[min(u, max_chunks - 1)];
    };
    // the sampled path fetches the next unit's descriptor while it processes
    // one; the dense path computes it in place
    const int stride = DENSE ? static_cast<int>(gridDim.x) : static_cast<int>(gridDim.x) / BH;
    const int u0 = DENSE ? static_cast<int>(blockIdx.x) : static_cast<int>(blockIdx.x) / BH;

    Chunk ck = descriptor(DENSE ? 0 : u0);
    int qbh = -1;  // the (b, kv) pair whose query the registers hold
    QKT qk;

    for (int u = u0; u < total; u += stride) {
        if (DENSE) ck = descriptor(u);
        const int bh = DENSE ? meta_bh(ck.meta) : pbh, ci = ck.ci;
        if (bh >= BH || ci < 0 || ci >= max_chunks) {  // uniform; never for a plan of this step
            ck = descriptor(min(u + stride, total - 1));
            continue;
        }
        const int b = bh / Hkv, kv = bh - b * Hkv;
        if (bh != qbh) {  // uniform
            // query of M row l % 16: head (l % 16) % 8 of this KV head
            // (zero for heads past the group)
            const int h = kMfmaPV ? (j16 & 7) : j16;
            const int hq = kv * G + (h < G ? h : 0);
            qk.load_q(q + (static_cast<size_t>(b) * Hq + hq) * D, h < G ? scale_log2 : 0.f, c);
            qbh = bh;
        }
        const Chunk nx = DENSE ? ck : descriptor(min(u + stride, total - 1));
        int begin = ck.begin, rows = meta_rows(ck.meta), slot = ck.slot;
        const int hmask = meta_hmask(ck.meta) & ((1 << G) - 1);
        const bool suffix = slot < 0;
        const int lim = suffix ? T_suf : N;
        if (!DENSE) {
            // a descriptor only ever addresses rows inside its buffer,
            // whatever the workspace holds
            rows = min(max(rows, 1), min(UR, max(lim, 1)));
            begin = min(max(begin, 0), max(lim - rows, 0));
            slot = min(slot, M - 1);
        }
        const bool live_unit = lim >= 1;  // uniform
        const T* Kb = suffix ? sK + (static_cast<size_t>(bh) * T_suf + begin) * D
                             : K + (static_cast<size_t>(bh) * N + begin) * D;
        const T* Vb = suffix ? sV + (static_cast<size_t>(bh) * T_suf + begin) * D
                             : V + (static_cast<size_t>(bh) * N + begin) * D;
        // the correction of this unit's team for heads 0..3 (lc03) and 4..7
        // (lc47), zero for the suffix
        float4 lc03 = make_float4(0.f, 0.f, 0.f, 0.f), lc47 = lc03;
        if (!DENSE && !suffix) {
            const float4* L = reinterpret_cast<const float4*>(ulogc + (static_cast<size_t>(bh) * M + slot) * kLogcStride);
            lc03 = L[0];
            lc47 = L[1];
        }

        float m[4], l[4], acc[GT][VPL];
        f32x4 oacc[NB];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            m[r] = kNeg;
            l[r] = 0.f;
        }
#pragma unroll
        for (int h = 0; h < GT; ++h)
#pragma unroll
            for (int e = 0; e < VPL; ++e) acc[h][e] = 0.f;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) oacc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};

        // 32 rows at a time: two 16-row tiles whose K and V loads are all
        // issued before any math.  K as MFMA fragments (lane (c, j) -> row j
        // of the tile), V with 16 lanes per row (lane (c, j) -> dims VPL j ..
        // of rows c, c + 4, ...).  Rows past the unit repeat its last row and
        // get no weight.
        for (int r0 = 0; live_unit && r0 < rows; r0 += 32) {
            const bool has1 = r0 + 16 < rows;
            typename QKT::frag kf[2][NF];
            typename VC::raw vr[2][4];
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                if (k == 0 || has1) {
                    const int t0 = r0 + 16 * k;
                    qk.load_k(Kb + static_cast<size_t>(min(t0 + j16, rows - 1)) * D, c, kf[k]);
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk)
                        vr[k][kk] = VC::load(Vb + static_cast<size_t>(min(t0 + 4 * kk + c, rows - 1)) * D + VPL * j16);
                }
            }
            if constexpr (kMfmaPV) {
                // softmax over the step's 32 rows at once
                const f32x4 s0 = qk.scores(kf[0]);
                f32x4 s1 = {kNeg, kNeg, kNeg, kNeg};
                if (has1) s1 = qk.scores(kf[1]);
                const bool live0 = r0 + j16 < rows, live1 = r0 + 16 + j16 < rows;
                float a[4], p0[4], p1[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float x0 = live0 ? s0[r] : kNeg;
                    const float x1 = live1 ? s1[r] : kNeg;
                    const float mn = fmaxf(m[r], row16_max(fmaxf(x0, x1)));
                    a[r] = rebase(m[r], mn);
                    p0[r] = fast_exp2(x0 - mn);
                    p1[r] = fast_exp2(x1 - mn);
                    l[r] = l[r] * a[r] + row16_sum(p0[r] + p1[r]);
                    m[r] = mn;
                }
                wave_lds_sync();  // the previous step's reads of the tiles are done
                // the value tile (zeros for a missing second tile: its rows
                // carry no weight, and 0 x garbage could be NaN)
#pragma unroll
                for (int k = 0; k < 2; ++k)
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk) {
                        const int row = 16 * k + 4 * kk + c;
                        typename VC::raw v = vr[k][kk];
                        if (k == 1 && !has1) v = typename VC::raw{};
                        *reinterpret_cast<typename VC::raw*>(s_v + VT::offset(row, 2 * VPL * j16)) = v;
                    }
                if (c < 2) {
                    float* pt = reinterpret_cast<float*>(s_pt);
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        pt[(hsel + r) * 32 + j16] = p0[r];
                        pt[(hsel + r) * 32 + 16 + j16] = p1[r];
                    }
                }
                wave_lds_sync();
                // A operand: rows 8 c .. 8 c + 7 of head (l % 16) % 8, high
                // or low bf16 part
                bf16x8 pa;
                {
                    const float4 x0 = s_pt[j16 & 7][2 * c], x1 = s_pt[j16 & 7][2 * c + 1];
                    const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
                    const bool low = j16 >= 8;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const __bf16 hi = static_cast<__bf16>(x[e]);
                        pa[e] = low ? static_cast<__bf16>(x[e] - static_cast<float>(hi)) : hi;
                    }
                }
                if (r0 > 0) {  // uniform; the first step starts from zero
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                        for (int r = 0; r < 4; ++r) oacc[nb][r] *= a[r];
                }
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
                    oacc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, VT::operand(s_v, nb, lane), oacc[nb], 0, 0, 0);
            } else {
#pragma unroll
                for (int k = 0; k < 2; ++k) {
                    if (k == 1 && !has1) continue;  // uniform
                    const int t0 = r0 + 16 * k;
                    const f32x4 sc = qk.scores(kf[k]);
                    // lane (c, j16): row j16 of the tile, heads 4 c .. 4 c + 3
                    const bool live = c < 2 && t0 + j16 < rows;
                    float a[4], p[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float x = live ? sc[r] : kNeg;
                        const float mn = fmaxf(m[r], row16_max(x));
                        a[r] = rebase(m[r], mn);
                        p[r] = fast_exp2(x - mn);
                        l[r] = l[r] * a[r] + row16_sum(p[r]);
                        m[r] = mn;
                    }
                    if (c < 2) {
                        s_p[j16][c] = make_float4(p[0], p[1], p[2], p[3]);
                        if (j16 == 0) s_a[c] = make_float4(a[0], a[1], a[2], a[3]);
                    }
                    wave_lds_sync();
                    float av[8];
                    {
                        const float4 a0 = s_a[0], a1 = s_a[1];
                        av[0] = a0.x; av[1] = a0.y; av[2] = a0.z; av[3] = a0.w;
                        av[4] = a1.x; av[5] = a1.y; av[6] = a1.z; av[7] = a1.w;
                    }
                    // only the heads that read this unit accumulate
#pragma unroll
                    for (int h = 0; h < GT; ++h) {
                        if (!((hmask >> h) & 1)) continue;  // uniform
#pragma unroll
                        for (int e = 0; e < VPL; ++e) acc[h][e] *= av[h];
                    }
                    // this lane group's rows of the tile: c, c + 4, c + 8, c + 12
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk) {
                        float vv[VPL];
                        VC::unpack(vr[k][kk], vv);
                        const float4 pp0 = s_p[4 * kk + c][0], pp1 = s_p[4 * kk + c][1];
                        const float pv[8] = {pp0.x, pp0.y, pp0.z, pp0.w, pp1.x, pp1.y, pp1.z, pp1.w};
#pragma unroll
                        for (int h = 0; h < GT; ++h) {
                            if (!((hmask >> h) & 1)) continue;
#pragma unroll
                            for (int e = 0; e < VPL; ++e) acc[h][e] = fmaf(pv[h], vv[e], acc[h][e]);
                        }
                    }
                    wave_lds_sync();
                }
            }
        }

        // the unit's state for each head that reads it, at the unit's
        // position in that head's list (rows of this pair's lists)
        float* const po_bh = part_o + static_cast<size_t>(bh) * G * max_hunits * D;
        float* const pml_bh = part_ml + static_cast<size_t>(bh) * G * max_hunits * 2;
        auto list_row = [&](int h, int pos) { return h * max_hunits + min(DENSE ? ci : pos, max_hunits - 1); };
        // positions of this lane's register heads hsel .. hsel + 3: the
        // descriptor words as wave-uniform values, picked by selects (an
        // indexed read would move the descriptor to scratch memory)
        int hp[4];
        {
            const unsigned w01 = __builtin_amdgcn_readfirstlane(ck.p01), w23 = __builtin_amdgcn_readfirstlane(ck.p23);
            const unsigned w45 = __builtin_amdgcn_readfirstlane(ck.p45), w67 = __builtin_amdgcn_readfirstlane(ck.p67);
            const unsigned wa = hsel ? w45 : w01, wb = hsel ? w67 : w23;
            hp[0] = static_cast<int>(wa & 0xffffu);
            hp[1] = static_cast<int>(wa >> 16);
            hp[2] = static_cast<int>(wb & 0xffffu);
            hp[3] = static_cast<int>(wb >> 16);
        }
        if constexpr (kMfmaPV) {
            // high + low halves: lane groups c and c ^ 2 hold the same
            // heads; group c < 2 finishes dim blocks 0 .. NB/2 - 1, group
            // c >= 2 blocks NB/2 .. NB - 1
            const bool lower = c < 2;
            const int dim0 = (lower ? 0 : D / 2) + j16;
#pragma unroll
            for (int nb = 0; nb < NB / 2; ++nb) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float keep = lower ? oacc[nb][r] : oacc[nb + NB / 2][r];
                    const float send = lower ? oacc[nb + NB / 2][r] : oacc[nb][r];
                    const float x = keep + __shfl_xor(send, 32);
                    const int h = hsel + r;
                    if (live_unit && h < G && ((hmask >> h) & 1))
                        __builtin_nontemporal_store(x, po_bh + list_row(h, hp[r]) * D + dim0 + 16 * nb);
                }
            }
        } else {
            // the four lane groups share each head's maximum, so their value
            // sums simply add
#pragma unroll
            for (int h = 0; h < GT; ++h) {
                if (!(live_unit && h < G && ((hmask >> h) & 1))) continue;  // uniform
                float x[VPL];
#pragma unroll
                for (int e = 0; e < VPL; ++e) {
                    float t = acc[h][e];
                    t += __shfl_xor(t, 16);
                    t += __shfl_xor(t, 32);
                    x[e] = t;
                }
                if (c == 0) {
                    float* o = po_bh + list_row(h, chunk_pos(ck, h)) * D + VPL * j16;
#pragma unroll
                    for (int e = 0; e < VPL; e += 4) store_stream(o + e, make_float4(x[e], x[e + 1], x[e + 2], x[e + 3]));
                }
            }
        }
        if (c < 2 && j16 == 0) {
            // register r of lane group c is head 4 c + r; the correction
            // enters as a shift of the unit's maximum (every row of the unit
            // belongs to the same team).  Written out per register so that
            // every index is a constant (a lane-dependent index into a
            // register array would put the array in scratch memory).
            auto put = [&](int r, float lc_lo, float lc_hi, float mr, float lr, int pos) {
                const int h = 4 * c + r;
                if (live_unit && h < G && ((hmask >> h) & 1))
                    store_stream2(pml_bh + list_row(h, pos) * 2, make_float2(mr - (c ? lc_hi : lc_lo) * kLog2e, lr));
            };
            put(0, lc03.x, lc47.x, m[0], l[0], hp[0]);
            put(1, lc03.y, lc47.y, m[1], l[1], hp[1]);
            put(2, lc03.z, lc47.z, m[2], l[2], hp[2]);
            put(3, lc03.w, lc47.w, m[3], l[3], hp[3]);
        }
        ck = nx;
    }
}

// bf16 keys and values: the units, arithmetic and results of k_attend, with
// the loads software-pipelined across the 32-row steps of a wave's units
// (unit after unit).  Each step waits for its own data, issues the next
// step's, and computes while those fly: K as MFMA fragments into the other
// of two register sets, V by the LDS DMA (global_load_lds, 16 bytes per
// lane, lane l to byte 16 l of a 1 KB block, each lane fetching the
// 16-byte segment that the tile's swizzle puts at its position) into the
// other of two tiles.  Loads complete in issue order and a step's V copies
// go out before its K loads, so waiting for its K fragments covers its
// value tile too.  Rows past a unit's end repeat its last row: finite, and
// weighted 0.
// Order of this wave's LDS accesses for the compiler only: the LDS executes
// one wave's instructions in order, so no wait is needed (a fence would also
// wait for the value copies in flight).
__device__ __forceinline__ void lds_order() { asm volatile("" ::: "memory"); }

// Workgroups of kAttendWaves independent waves, one workgroup per compute
// unit: the waves share nothing but the workgroup's LDS allocation (each has
// its own tiles) and never synchronise.  Wave k of workgroup b is wave
// k gridDim.x + b of the launch, so the launch's first waves, which get work
// first, are spread over every compute unit (one-wave workgroups were
// placed several to a compute unit, leaving others idle).
constexpr int kAttendWaves = 8;

template <int D, bool DENSE>
__global__ __launch_bounds__(kAttendWaves * kWave, 1) void k_attend_mfma(
    const bf16_t* __restrict__ K, const bf16_t* __restrict__ V, const bf16_t* __restrict__ sK,
    const bf16_t* __restrict__ sV, const float* __restrict__ q, int N, int T_suf, int BH, int Hkv,
    int Hq, int G, int M, float scale_log2, int max_chunks, int max_hunits,
    const PlanHeader* __restrict__ hdr, const Chunk* __restrict__ chunks,
    const float* __restrict__ ulogc, float* __restrict__ part_o, float* __restrict__ part_ml) {
    constexpr int UR = DENSE ? kDenseRows : kChunkRows;
    using QKT = QK<bf16_t, D>;
    using VT = VTile<D>;
    constexpr int NF = QKT::KB;         // K fragments per 16-row tile
    constexpr int NB = VT::NB;
    constexpr int SPR = D / 8;          // 16-byte segments per row
    constexpr int RPI = kWave / SPR;    // rows per DMA instruction (1 KB)
    constexpr int NDMA = 32 / RPI;      // DMA instructions per step
    static_assert(RPI * SPR == kWave && NDMA * RPI == 32, "a step's tile is whole 1 KB DMA blocks");
    constexpr int kNT = 2;              // cache policy of the value copies: streaming
    // value tiles, double-buffered (two objects, so that the compiler can
    // tell the copies into one from the reads of the other)
    __shared__ __attribute__((aligned(16))) char s_v0[kAttendWaves][VT::kBytes];
    __shared__ __attribute__((aligned(16))) char s_v1[kAttendWaves][VT::kBytes];
    __shared__ float4 s_pt[kAttendWaves][8][8];  // probabilities [head][row / 4]

    const int lane = lane_id();
    const int wv = __builtin_amdgcn_readfirstlane(wave_id());  // uniform: keeps the tile bases scalar
    const int c = lane >> 4, j16 = lane & 15;
    const int hsel = 4 * (c & 1);  // first head of this lane's registers
    const int ncp = (N + UR - 1) / UR;
    const int nchd = ncp + (T_suf + UR - 1) / UR;
    const int gw = wv * static_cast<int>(gridDim.x) + static_cast<int>(blockIdx.x);  // wave of the launch
    const int nw = kAttendWaves * static_cast<int>(gridDim.x);                       // waves of the launch
    // Wave gw takes units gw, gw + nw, ... of the step's list: the dense
    // path's (b, kv)-major list, or the sampled path's units of all pairs in
    // pair order (each pair's units sit in its own region of the sampler's
    // list; every wave reads the pairs' unit counts and maps a unit to its
    // pair by a prefix sum).  Every compute unit so gets the same number of
    // units to within one, however the pairs' counts differ.
    const int stride = nw;
    char* const tile0 = s_v0[wv];
    char* const tile1 = s_v1[wv];
    float4 (*const ptile)[8] = s_pt[wv];
    int pc_cnt = 0, pc_incl = 0;  // sampled path: lane p's pair count and inclusive prefix (p < 64)
    auto descriptor = [&](int u) {
        if (DENSE) {
            const int bhx = u / nchd, cix = u - bhx * nchd;
            const bool suf = cix >= ncp;
            const int begin = (suf ? cix - ncp : cix) * UR;
            Chunk d;
            d.begin = begin;
            d.slot = suf ? -1 : 0;
            d.meta = chunk_meta(min(UR, (suf ? T_suf : N) - begin), (1 << G) - 1, bhx);
            d.ci = cix;
            d.p01 = d.p23 = d.p45 = d.p67 = 0u;
            return d;
        }
        // unit u of the pairs' concatenated lists: lanes hold the counts of
        // 64 pairs at a time and their inclusive prefix sums (kept in
        // registers from the start when there are at most 64 pairs)
        int base = 0, p = BH - 1, idx = 0;
        if (BH <= kWave) {  // uniform
            const int nb = __popcll(__ballot(lane < BH && pc_incl <= u));  // pairs wholly before unit u
            p = min(nb, BH - 1);
            idx = u - (__builtin_amdgcn_readlane(pc_incl, p) - __builtin_amdgcn_readlane(pc_cnt, p));
        } else for (int p0 = 0; p0 < BH; p0 += kWave) {  // uniform
            const int cnt = p0 + lane < BH ? min(max(hdr[p0 + lane].chunks, 0), max_chunks) : 0;
            const int incl = wave_incl_scan(cnt) + base;
            const uint64_t before = __ballot(p0 + lane < BH && incl <= u);  // pairs wholly before unit u
            const int nb = __popcll(before);
            if (nb < kWave && p0 + nb < BH) {  // unit u is in pair p0 + nb
                p = p0 + nb;
                idx = u - (__builtin_amdgcn_readlane(incl, nb) - __builtin_amdgcn_readlane(cnt, nb));
                break;
            }
            base = __builtin_amdgcn_readlane(incl, kWave - 1);
        }
        Chunk d = chunks[static_cast<size_t>(p) * max_chunks + min(max(idx, 0), max_chunks - 1)];
        d.meta = (d.meta & 0xffff) | (p << 16);  // the pair the unit was found in
        return d;
    };
    // units of the step: the dense list's length, or the sum of the pairs'
    // counts (a wave-wide sum over the headers; the first 64 pairs' counts
    // and prefix sums stay in registers for the unit lookups)
    auto unit_total = [&]() {
        if (DENSE) return BH * nchd;
        int t = 0;
        for (int p0 = 0; p0 < BH; p0 += kWave) {  // uniform
            const int cnt = p0 + lane < BH ? min(max(hdr[p0 + lane].chunks, 0), max_chunks) : 0;
            const int incl = wave_incl_scan(cnt);
            if (p0 == 0) {
                pc_cnt = cnt;
                pc_incl = incl;
            }
            t += __builtin_amdgcn_readlane(incl, kWave - 1);
        }
        return t;
    };
    // a unit's rows, clamped to its buffer whatever the workspace holds
    struct Unit {
        const bf16_t* Kb;
        const bf16_t* Vb;
        int bh, rows, slot, hmask, ci;
        bool suffix, live;
        unsigned p01, p23, p45, p67;
    };
    auto unit_of = [&](const Chunk& ck) {
        Unit U;
        U.bh = min(max(meta_bh(ck.meta), 0), BH - 1);
        U.ci = ck.ci;
        int begin = ck.begin, rows = meta_rows(ck.meta);
        U.slot = min(ck.slot, M - 1);
        U.hmask = meta_hmask(ck.meta) & ((1 << G) - 1);
        U.suffix = ck.slot < 0;
        const int lim = U.suffix ? T_suf : N;
        U.live = lim >= 1;
        rows = min(max(rows, 1), min(UR, max(lim, 1)));
        begin = min(max(begin, 0), max(lim - rows, 0));
        U.rows = rows;
        U.Kb = U.suffix ? sK + (static_cast<size_t>(U.bh) * T_suf + begin) * D : K + (static_cast<size_t>(U.bh) * N + begin) * D;
        U.Vb = U.suffix ? sV + (static_cast<size_t>(U.bh) * T_suf + begin) * D : V + (static_cast<size_t>(U.bh) * N + begin) * D;
        U.p01 = __builtin_amdgcn_readfirstlane(ck.p01);
        U.p23 = __builtin_amdgcn_readfirstlane(ck.p23);
        U.p45 = __builtin_amdgcn_readfirstlane(ck.p45);
        U.p67 = __builtin_amdgcn_readfirstlane(ck.p67);
        return U;
    };
    auto corrections = [&](const Unit& U, float4& lo, float4& hi) {
        lo = make_float4(0.f, 0.f, 0.f, 0.f);
        hi = lo;
        if (!DENSE && !U.suffix) {
            const float4* L = reinterpret_cast<const float4*>(ulogc + (static_cast<size_t>(U.bh) * M + U.slot) * kLogcStride);
            lo = L[0];
            hi = L[1];
        }
    };
    // V copies, then K loads, of rows r0 .. r0 + 31 of unit U.  Every step
    // issues the same loads whether or not a next step exists (then every
    // lane fetches the unit's first 16 bytes: one cache line per
    // instruction), so that the compiler's count of loads in flight, and
    // with it the wait before each step, is the same on every path.
    auto issue = [&](const Unit& U, int r0, char* tile, typename QKT::frag (&kf)[2][NF], bool real) {
        const int ls = real ? lane : 0;
#pragma unroll
        for (int j = 0; j < NDMA; ++j) {
            const int row = real ? RPI * j + lane / SPR : 0;
            const int seg = real ? (ls % SPR) ^ (2 * VT::swz(row)) : 0;
            const bf16_t* src = U.Vb + static_cast<size_t>(min(r0 + row, U.rows - 1)) * D + 8 * seg;
            __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)(tile + 1024 * j), 16, 0, kNT);
        }
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const bf16_t* row = U.Kb + (real ? static_cast<size_t>(min(r0 + 16 * k + j16, U.rows - 1)) * D : 0);
            QKT::load_k(row, real ? c : 0, kf[k]);
        }
    };

    int u = gw;
    const int total = unit_total();
    if (u >= total) return;  // uniform
    Unit cur = unit_of(descriptor(u));
    // the sampled path fetches the next unit's descriptor while it
    // processes one; the dense path computes it when it needs it
    Chunk nxck = DENSE ? Chunk{} : descriptor(min(u + stride, total - 1));
    float4 lc_lo, lc_hi;
    corrections(cur, lc_lo, lc_hi);
    QKT qk;
    int qbh = cur.bh;
    {
        const int h = j16 & 7;
        const int b = cur.bh / Hkv, kv = cur.bh - b * Hkv;
        qk.load_q(q + (static_cast<size_t>(b) * Hq + kv * G + (h < G ? h : 0)) * D, h < G ? scale_log2 : 0.f, c);
    }
    typename QKT::frag kf0[2][NF], kf1[2][NF];
    issue(cur, 0, tile0, kf0, true);

    float m[4], l[4];
    f32x4 oacc[NB];
    auto reset = [&]() {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            m[r] = kNeg;
            l[r] = 0.f;
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) oacc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    };
    reset();
    int r0 = 0;
    bool done = false;

    // one step from tile `tile` and fragments kf (rows r0 .. of unit cur),
    // with the next step issued into the other buffer first
    auto step = [&](char* tile, typename QKT::frag (&kf)[2][NF], char* ntile, typename QKT::frag (&nkf)[2][NF]) {
        // the next step: the same unit's next 32 rows, or the next unit's first
        const bool more = r0 + 32 < cur.rows;
        const int un = u + stride;
        const bool has_next = more || un < total;
        Unit nxt = cur;
        int nr0 = r0 + 32;
        if (!more && has_next) {
            nxt = unit_of(DENSE ? descriptor(un) : nxck);
            nr0 = 0;
        }
        // this step's data first: its K fragments, and with them (issued
        // before them) its value copies; nothing later is in flight yet, so
        // the wait is exact.  Then the next step goes out and flies while
        // this one computes.  No load or read of a tile moves above here.
        asm volatile("" ::"v"(kf[1][NF - 1].w) : "memory");
        issue(nxt, has_next ? nr0 : 0, ntile, nkf, has_next);

        // scores and softmax over the step's 32 rows
        const f32x4 s0 = qk.scores(kf[0]);
        const f32x4 s1 = qk.scores(kf[1]);
        const bool live0 = r0 + j16 < cur.rows, live1 = r0 + 16 + j16 < cur.rows;
        float a[4], p0[4], p1[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float x0 = live0 ? s0[r] : kNeg;
            const float x1 = live1 ? s1[r] : kNeg;
            const float mn = fmaxf(m[r], row16_max(fmaxf(x0, x1)));
            a[r] = rebase(m[r], mn);
            p0[r] = fast_exp2(x0 - mn);
            p1[r] = fast_exp2(x1 - mn);
            l[r] = l[r] * a[r] + row16_sum(p0[r] + p1[r]);
            m[r] = mn;
        }
        lds_order();  // the previous step's reads of s_pt come first
        if (c < 2) {
            float* pt = reinterpret_cast<float*>(ptile);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                pt[(hsel + r) * 32 + j16] = p0[r];
                pt[(hsel + r) * 32 + 16 + j16] = p1[r];
            }
        }
        lds_order();
        bf16x8 pa;
        {
            const float4 x0 = ptile[j16 & 7][2 * c], x1 = ptile[j16 & 7][2 * c + 1];
            const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
            const bool low = j16 >= 8;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const __bf16 hi = static_cast<__bf16>(x[e]);
                pa[e] = low ? static_cast<__bf16>(x[e] - static_cast<float>(hi)) : hi;
            }
        }
        if (r0 > 0) {  // uniform; a unit's first step starts from zero
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int r = 0; r < 4; ++r) oacc[nb][r] *= a[r];
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
            oacc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, VT::operand(tile, nb, lane), oacc[nb], 0, 0, 0);

        if (!more) {
            // the unit's state for each head that reads it, at the unit's
            // position in that head's list
            float* const po_bh = part_o + static_cast<size_t>(cur.bh) * G * max_hunits * D;
            float* const pml_bh = part_ml + static_cast<size_t>(cur.bh) * G * max_hunits * 2;
            auto list_row = [&](int h, int pos) { return h * max_hunits + min(DENSE ? cur.ci : pos, max_hunits - 1); };
            const unsigned wa = hsel ? cur.p45 : cur.p01, wb = hsel ? cur.p67 : cur.p23;
            const int hp[4] = {static_cast<int>(wa & 0xffffu), static_cast<int>(wa >> 16),
                               static_cast<int>(wb & 0xffffu), static_cast<int>(wb >> 16)};
            // high + low halves: lane groups c and c ^ 2 hold the same heads
            const bool lower = c < 2;
            const int dim0 = (lower ? 0 : D / 2) + j16;
#pragma unroll
            for (int nb = 0; nb < NB / 2; ++nb) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float keep = lower ? oacc[nb][r] : oacc[nb + NB / 2][r];
                    const float send = lower ? oacc[nb + NB / 2][r] : oacc[nb][r];
                    const float x = keep + __shfl_xor(send, 32);
                    const int h = hsel + r;
                    if (cur.live && h < G && ((cur.hmask >> h) & 1))
                        __builtin_nontemporal_store(x, po_bh + list_row(h, hp[r]) * D + dim0 + 16 * nb);
                }
            }
            if (c < 2 && j16 == 0) {
                // the correction enters as a shift of the unit's maximum
                // (every row of the unit belongs to the same team); written
                // out per register so that every index is a constant
                auto put = [&](int r, float lc0, float lc1, float mr, float lr, int pos) {
                    const int h = 4 * c + r;
                    if (cur.live && h < G && ((cur.hmask >> h) & 1))
                        store_stream2(pml_bh + list_row(h, pos) * 2, make_float2(mr - (c ? lc1 : lc0) * kLog2e, lr));
                };
                put(0, lc_lo.x, lc_hi.x, m[0], l[0], hp[0]);
                put(1, lc_lo.y, lc_hi.y, m[1], l[1], hp[1]);
                put(2, lc_lo.z, lc_hi.z, m[2], l[2], hp[2]);
                put(3, lc_lo.w, lc_hi.w, m[3], l[3], hp[3]);
            }
        }
        if (!has_next) {
            done = true;
            return;
        }
        if (!more) {  // the next unit becomes current
            cur = nxt;
            u = un;
            if (!DENSE) nxck = descriptor(min(u + stride, total - 1));
            corrections(cur, lc_lo, lc_hi);
            if (cur.bh != qbh) {
                const int h = j16 & 7;
                const int b = cur.bh / Hkv, kv = cur.bh - b * Hkv;
                qk.load_q(q + (static_cast<size_t>(b) * Hq + kv * G + (h < G ? h : 0)) * D, h < G ? scale_log2 : 0.f, c);
                qbh = cur.bh;
            }
            reset();
        }
        r0 = nr0;
    };
    for (;;) {
        step(tile0, kf0, tile1, kf1);
        if (done) break;
        step(tile1, kf1, tile0, kf0);
        if (done) break;
    }
}

// Merge of one query head's list of n unit states (m_p: log2-domain maximum
// with the team's correction folded in, l_p: mass) and value sums o_p:
// out = sum_p 2^(m_p - mx) o_p / sum_p 2^(m_p - mx) l_p with mx = max_p m_p.
// Workgroup = (sequence and query head, slice of kMergeDims output dims).
// A pass covers 32 NPL positions: thread t loads the states of positions
// t, t + 256, ... (to LDS, weights computed once per position) and 16 bytes
// of values (four dims) of positions t / 8 + 32 k, k < NPL, so a pass is
// NPL + 1 loads per thread, all issued before any is used.  Positions are
// clamped to the list (the sampled path reads its list length from the
// plan header first), so a pass reads each of the list's states once
// whatever NPL is; the host picks NPL from the longest list a step can
// have, so one pass covers every list in the common case.  The value sums
// reduce over the 32 position groups in a fixed order.
constexpr int kMergeDims = 32;
constexpr int kMergeQuads = kMergeDims / 4;             // threads per position (16 bytes each)
constexpr int kMergeRowsPerLoad = kMergeThreads / kMergeQuads;  // positions per load instruction (32)

template <bool DENSE, int NPL>
__global__ __launch_bounds__(kMergeThreads) void k_merge(const float* __restrict__ part_o,
                                                         const float* __restrict__ part_ml,
                                                         const PlanHeader* __restrict__ hdr,
                                                         int n_dense, int Hkv, int Hq, int max_hunits,
                                                         int D, float* __restrict__ out) {
    constexpr int PP = kMergeRowsPerLoad * NPL;                              // positions per pass
    constexpr int NST = (PP + kMergeThreads - 1) / kMergeThreads;            // states per thread
    constexpr int NW = kMergeThreads / kWave;
    __shared__ float2 s_st[PP];       // (weight exponent, mass) of the pass's positions
    __shared__ float s_red[2][NW];
    __shared__ float4 s_acc[NW][kMergeQuads];
    const int bhq = blockIdx.x;
    const int b = bhq / Hq, hq = bhq - b * Hq;
    const int G = Hq / Hkv;
    const int kv = hq / G, h = hq - kv * G;
    const int bh = b * Hkv + kv;
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    const int dq = tid % kMergeQuads, pg = tid / kMergeQuads;
    const size_t row0 = (static_cast<size_t>(bh) * G + h) * max_hunits;
    const float2* ml = reinterpret_cast<const float2*>(part_ml) + row0;
    const float* po = part_o + row0 * D + blockIdx.y * kMergeDims + 4 * dq;
    // the list length (a uniform load of the plan header on the sampled
    // path); the loads touch only the list's positions
    const int n_list = DENSE ? n_dense : hdr[bh].hunits[h];
    const int lim = max(1, min(n_list, max_hunits));

    float mx = kNeg, lsum = 0.f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    float2 st[NST];
    float4 v[NPL];
    auto load = [&](int p0) {
#pragma unroll
        for (int k = 0; k < NST; ++k) st[k] = ml[min(p0 + tid + k * kMergeThreads, lim - 1)];
#pragma unroll
        for (int k = 0; k < NPL; ++k)
            v[k] = load_stream_f(po + static_cast<size_t>(min(p0 + pg + k * kMergeRowsPerLoad, lim - 1)) * D);
    };
    auto consume = [&](int p0, int n) {
        float pm = kNeg;
#pragma unroll
        for (int k = 0; k < NST; ++k) {
            const int i = tid + k * kMergeThreads;
            if (i < PP) pm = fmaxf(pm, p0 + i < n ? st[k].x : kNeg);
        }
        for (int off = kWave / 2; off > 0; off >>= 1) pm = fmaxf(pm, __shfl_xor(pm, off));
        if (lane == 0) s_red[0][w] = pm;
        __syncthreads();
#pragma unroll
        for (int k = 0; k < NW; ++k) pm = fmaxf(pm, s_red[0][k]);
        const float nmx = fmaxf(mx, pm);
        const float sc = rebase(mx, nmx);
        acc.x *= sc;
        acc.y *= sc;
        acc.z *= sc;
        acc.w *= sc;
        lsum *= sc;
        // each state's weight once, by the thread that loaded it
#pragma unroll
        for (int k = 0; k < NST; ++k) {
            const int i = tid + k * kMergeThreads;
            if (i < PP) {
                const float wt = p0 + i < n ? rebase(st[k].x, nmx) : 0.f;
                lsum = fmaf(wt, p0 + i < n ? st[k].y : 0.f, lsum);
                s_st[i].x = wt;
            }
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < NPL; ++k) {
            const float wt = s_st[pg + k * kMergeRowsPerLoad].x;  // zero past the list
            acc.x = fmaf(wt, v[k].x, acc.x);
            acc.y = fmaf(wt, v[k].y, acc.y);
            acc.z = fmaf(wt, v[k].z, acc.z);
            acc.w = fmaf(wt, v[k].w, acc.w);
        }
        mx = nmx;
    };
    load(0);
    const int n = min(n_list, max_hunits);
    consume(0, n);
    for (int p0 = PP; p0 < n; p0 += PP) {  // uniform; lists longer than one pass
        __syncthreads();  // s_st and s_red are rewritten
        load(p0);
        consume(p0, n);
    }
    // value sums: lanes l, l + 8, ..., l + 56 of a wave hold the same four
    // dims; then the waves in order
#pragma unroll
    for (int off = kMergeQuads; off < kWave; off <<= 1) {
        acc.x += __shfl_xor(acc.x, off);
        acc.y += __shfl_xor(acc.y, off);
        acc.z += __shfl_xor(acc.z, off);
        acc.w += __shfl_xor(acc.w, off);
    }
    if (lane < kMergeQuads) s_acc[w][lane] = acc;
    for (int off = kWave / 2; off > 0; off >>= 1) lsum += __shfl_xor(lsum, off);
    if (lane == 0) s_red[1][w] = lsum;
    __syncthreads();
    if (tid < kMergeQuads) {
        float4 o = s_acc[0][tid];
#pragma unroll
        for (int k = 1; k < NW; ++k) {
            o.x += s_acc[k][tid].x;
            o.y += s_acc[k][tid].y;
            o.z += s_acc[k][tid].z;
            o.w += s_acc[k][tid].w;
        }
        float L = 0.f;
#pragma unroll
        for (int k = 0; k < NW; ++k) L += s_red[1][k];
        const float inv = 1.f / L;
        *reinterpret_cast<float4*>(out + static_cast<size_t>(bhq) * D + blockIdx.y * kMergeDims + 4 * tid) =
            make_float4(o.x * inv, o.y * inv, o.z * inv, o.w * inv);
    }
}

__global__ void k_zero(uint4* __restrict__ p, size_t n16, unsigned char* __restrict__ tail,
                       int ntail) {
    const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < n16; i += stride)
        p[i] = make_uint4(0, 0, 0, 0);
    if (blockIdx.x == 0 && static_cast<int>(threadIdx.x) < ntail) tail[threadIdx.x] = 0;
}

// Launch an attention kernel; with stage events, the launch itself stamps
// them at the kernel's start and end (so they time the kernel's execution,
// not the dispatch gap before it).
template <typename F, typename... Args>
hipError_t launch_timed(const AttendArgs& a, F kernel, dim3 grid, dim3 block, hipStream_t s, Args... args) {
    if (a.ev_start || a.ev_stop)
        hipExtLaunchKernelGGL(kernel, grid, block, 0, s, a.ev_start, a.ev_stop, 0, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
    return hipGetLastError();
}

// Waves of an attention launch: one per unit on the dense path; on the
// sampled path W per (b, kv) pair, where W spreads the device's resident
// waves over the pairs and never exceeds the units a pair can have.
long long attend_waves(const AttendArgs& a) {
    const long long BH = static_cast<long long>(a.B) * a.Hkv;
    if (a.dense) return BH * a.max_chunks;
    long long W = a.max_chunks;
    if (a.grid_waves > 0) W = std::min<long long>(W, std::max<long long>(1, a.grid_waves / BH));
    return BH * W;
}

// Workgroups of an attention launch on the matrix cores: one per compute
// unit, fewer when the step cannot have that many units of work.
long long attend_blocks(const AttendArgs& a) {
    const long long units = static_cast<long long>(a.B) * a.Hkv * a.max_chunks;
    const long long blocks = a.cus > 0 ? std::min<long long>(a.cus, units) : (units + kAttendWaves - 1) / kAttendWaves;
    return std::max<long long>(blocks, 1);
}

template <int D>
hipError_t attend_mfma(const AttendArgs& a, hipStream_t s) {
    const long long blocks = attend_blocks(a);
    if (blocks > 0x7fffffffLL / kAttendWaves) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(blocks));
    constexpr int kThreads = kAttendWaves * kWave;
    const float sl2 = a.scale * kLog2e;
    const bf16_t* K = static_cast<const bf16_t*>(a.K);
    const bf16_t* V = static_cast<const bf16_t*>(a.V);
    const bf16_t* sK = static_cast<const bf16_t*>(a.sK);
    const bf16_t* sV = static_cast<const bf16_t*>(a.sV);
    const int BH = a.B * a.Hkv;
    if (a.dense) {
        return launch_timed(a, k_attend_mfma<D, true>, grid, dim3(kThreads), s, K, V, sK, sV, a.q, a.N, a.T, BH,
                            a.Hkv, a.Hq, a.G, 0, sl2, a.max_chunks, a.max_hunits,
                            static_cast<const PlanHeader*>(nullptr), static_cast<const Chunk*>(nullptr),
                            static_cast<const float*>(nullptr), a.part_o, a.part_ml);
    } else {
        const DecodeLayout& L = *a.lay;
        return launch_timed(a, k_attend_mfma<D, false>, grid, dim3(kThreads), s, K, V, sK, sV, a.q, a.N, a.T,
                            BH, a.Hkv, a.Hq, a.G, a.M, sl2, a.max_chunks, a.max_hunits,
                            reinterpret_cast<const PlanHeader*>(a.ws + L.hdr),
                            reinterpret_cast<const Chunk*>(a.ws + L.chunk),
                            reinterpret_cast<const float*>(a.ws + L.ulogc), a.part_o, a.part_ml);
    }
    return hipGetLastError();
}

template <typename T, int D, int GT>
hipError_t attend_g(const AttendArgs& a, hipStream_t s) {
    // one list of units over every (b, kv) pair; the sampled path runs as
    // many one-wave workgroups as the chip keeps resident (each looping over
    // its share), the dense path one workgroup per unit
    const long long waves = attend_waves(a);
    if (waves < 1 || waves > 0x7fffffffLL) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(waves));
    const float sl2 = a.scale * kLog2e;
    const T* K = static_cast<const T*>(a.K);
    const T* V = static_cast<const T*>(a.V);
    const T* sK = static_cast<const T*>(a.sK);
    const T* sV = static_cast<const T*>(a.sV);
    const int BH = a.B * a.Hkv;
    if (a.dense) {
        return launch_timed(a, k_attend<T, D, GT, true>, grid, dim3(kWave), s, K, V, sK, sV, a.q, a.N, a.T, BH,
                            a.Hkv, a.Hq, a.G, 0, sl2, a.max_chunks, a.max_hunits,
                            static_cast<const PlanHeader*>(nullptr), static_cast<const Chunk*>(nullptr),
                            static_cast<const float*>(nullptr), a.part_o, a.part_ml);
    } else {
        const DecodeLayout& L = *a.lay;
        return launch_timed(a, k_attend<T, D, GT, false>, grid, dim3(kWave), s, K, V, sK, sV, a.q, a.N, a.T, BH,
                            a.Hkv, a.Hq, a.G, a.M, sl2, a.max_chunks, a.max_hunits,
                            reinterpret_cast<const PlanHeader*>(a.ws + L.hdr),
                            reinterpret_cast<const Chunk*>(a.ws + L.chunk),
                            reinterpret_cast<const float*>(a.ws + L.ulogc), a.part_o, a.part_ml);
    }
    return hipGetLastError();
}

template <typename T, int D>
hipError_t attend_d(const AttendArgs& a, hipStream_t s) {
    if constexpr (sizeof(T) == 2) {
        // the matrix-core value sum computes every head of the group at once
        return a.G >= 1 && a.G <= kMaxGroup ? attend_mfma<D>(a, s) : hipErrorInvalidValue;
    } else {
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
    if (a.d % kMergeDims != 0) return hipErrorInvalidValue;
    const dim3 grid(a.B * a.Hq, a.d / kMergeDims);
    // positions per pass: enough for the longest list the step can have, up
    // to 640 (longer lists take several passes)
    const int longest = a.dense ? a.max_chunks : a.max_hunits;
    const PlanHeader* hdr = a.dense ? nullptr : reinterpret_cast<const PlanHeader*>(a.ws + a.lay->hdr);
    const int nd = a.dense ? a.max_chunks : 0;
#define SANTAPP_MERGE(DN, NPL)                                                                      \
    k_merge<DN, NPL><<<grid, kMergeThreads, 0, s>>>(a.part_o, a.part_ml, hdr, nd, a.Hkv, a.Hq, \
                                                    a.max_hunits, a.d, a.out)
    const int npl = longest <= 5 * kMergeRowsPerLoad ? 5 : longest <= 10 * kMergeRowsPerLoad ? 10 : 20;
    if (a.dense) {
        if (npl == 5) SANTAPP_MERGE(true, 5);
        else if (npl == 10) SANTAPP_MERGE(true, 10);
        else SANTAPP_MERGE(true, 20);
    } else {
        if (npl == 5) SANTAPP_MERGE(false, 5);
        else if (npl == 10) SANTAPP_MERGE(false, 10);
        else SANTAPP_MERGE(false, 20);
    }
#undef SANTAPP_MERGE
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
