// Team construction and packing (section "Preparing parent groups and teams";
// Alg. "Contiguous parent partition", Alg. "Build actual-key teams from a
// parent partition"; packed team-contiguous copy of the prompt K/V as in the
// appendix "Triton decode kernels").
//
// One workgroup builds one contiguous parent of one (sequence, KV head).  The
// farthest-first rounds and the nearest-representative assignment share one
// running minimum per member: after round u, mind[i] = min_{v<=u} |k_i-k_{j_v}|^2
// and owner[i] is the first v attaining it, which is exactly the assignment
// rule (ties to the earliest-chosen representative) once all r rounds ran.
// Distances are fp64 sums in dimension order with no fused multiply-add, so
// every comparison sees the value the definition gives.
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

constexpr int kBuildThreads = 256;
constexpr int kBuildWaves = kBuildThreads / kWave;
// label-defined parents hold about N / M members each (k-means: about P),
// one workgroup per parent: four times the threads for fewer rounds per
// member sweep
constexpr int kListBuildThreads = 1024;

// (value, index) reductions with ties broken toward the lower index.
struct ArgVal {
    double v;
    int i;
};

__device__ __forceinline__ ArgVal pick_min(ArgVal a, ArgVal b) {
    return (b.v < a.v || (b.v == a.v && b.i < a.i)) ? b : a;
}

__device__ __forceinline__ ArgVal pick_max(ArgVal a, ArgVal b) {
    return (b.v > a.v || (b.v == a.v && b.i < a.i)) ? b : a;
}

template <bool kMax, int W = kBuildWaves>
__device__ ArgVal block_arg(ArgVal x, ArgVal* s_red) {
    for (int off = kWave / 2; off > 0; off >>= 1) {
        ArgVal y;
        y.v = __shfl_xor(x.v, off);
        y.i = __shfl_xor(x.i, off);
        x = kMax ? pick_max(x, y) : pick_min(x, y);
    }
    if (lane_id() == 0) s_red[wave_id()] = x;
    __syncthreads();
    ArgVal r = s_red[0];
    for (int w = 1; w < W; ++w) r = kMax ? pick_max(r, s_red[w]) : pick_min(r, s_red[w]);
    __syncthreads();
    return r;
}

// |k_i - c|^2 with c held in LDS as fp64, summed in dimension order; the row
// is read 16 bytes at a time (rows are 16-byte aligned, d a multiple of 8).
template <typename T>
__device__ double sqdist_to(const T* __restrict__ row, const double* __restrict__ c, int d) {
#pragma clang fp contract(off)
    double acc = 0.0;
    constexpr int kPer = 16 / static_cast<int>(sizeof(T));
    for (int j = 0; j < d; j += kPer) {
        const uint4 w = *reinterpret_cast<const uint4*>(row + j);
        float v[kPer];
        if constexpr (sizeof(T) == 2) {
            const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                v[2 * q] = bf16lo(ws[q]);
                v[2 * q + 1] = bf16hi(ws[q]);
            }
        } else {
            v[0] = __uint_as_float(w.x);
            v[1] = __uint_as_float(w.y);
            v[2] = __uint_as_float(w.z);
            v[3] = __uint_as_float(w.w);
        }
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const double t = static_cast<double>(v[q]) - c[j + q];
            acc = acc + t * t;
        }
    }
    return acc;
}

// NT threads per workgroup.  LIST: the parent's members are the token
// indices mem[0 .. n) (ascending)
// of a label-defined partition; otherwise the contiguous span [pP, pP + n).
template <typename T, bool LIST, int NT>
__global__ __launch_bounds__(NT) void k_build_parent(
    const T* __restrict__ K, int N, int d, int P, int R, int M, double* __restrict__ mind_all,
    int* __restrict__ owner_all, int* __restrict__ team_begin, int* __restrict__ team_size,
    double* __restrict__ log_n, int* __restrict__ rep_token, int* __restrict__ perm,
    const int* __restrict__ members, const int* __restrict__ pbeg, const int* __restrict__ toff, int Mp,
    int* __restrict__ team_count) {
#pragma clang fp contract(off)
    // contiguous parents: every pair has M teams
    if (!LIST && blockIdx.x == 0 && threadIdx.x == 0) team_count[blockIdx.y] = M;
    __shared__ double s_vec[kMaxHeadDim];
    __shared__ ArgVal s_red[(NT / kWave)];
    __shared__ int s_reps[kMaxReps];
    __shared__ int s_cnt[kMaxReps];
    __shared__ int s_off[kMaxReps];
    __shared__ int s_wcnt[(NT / kWave)][kMaxReps];

    const int p = blockIdx.x;
    const int bh = blockIdx.y;
    const int tid = threadIdx.x;
    int start, n, team0;
    if constexpr (LIST) {
        start = pbeg[static_cast<size_t>(bh) * (Mp + 1) + p];
        n = pbeg[static_cast<size_t>(bh) * (Mp + 1) + p + 1] - start;
        team0 = toff[static_cast<size_t>(bh) * (Mp + 1) + p];
        if (n == 0) return;  // empty parents are omitted (uniform over the workgroup)
    } else {
        start = p * P;
        n = min(P, N - start);
        team0 = p * min(R, P);  // every earlier parent is full-size
    }
    const int r = min(R, n);
    const int* mem = LIST ? members + static_cast<size_t>(bh) * N + start : nullptr;
    // token of member i, and its key row
    auto tok = [&](int i) { return LIST ? mem[i] : start + i; };
    const T* Kb = K + static_cast<size_t>(bh) * N * d;
    auto row = [&](int i) { return Kb + static_cast<size_t>(tok(i)) * d; };
    double* mind = mind_all + static_cast<size_t>(bh) * N + start;
    int* owner = owner_all + static_cast<size_t>(bh) * N + start;

    // parent mean, summed over members in token order
    for (int j = tid; j < d; j += NT) {
        double s = 0.0;
        for (int i = 0; i < n; ++i) s = s + static_cast<double>(load_elem(row(i), j));
        s_vec[j] = s / static_cast<double>(n);
    }
    __syncthreads();

    // first representative: the member nearest the mean
    ArgVal best{INFINITY, 0x7fffffff};
    for (int i = tid; i < n; i += NT) {
        ArgVal c{sqdist_to(row(i), s_vec, d), i};
        best = pick_min(best, c);
    }
    best = block_arg<false, NT / kWave>(best, s_red);
    // a reduction without a winner (NaN keys) falls back to member 0, so
    // that every index stays inside the parent
    int rep = best.i < n ? best.i : 0;

    for (int u = 0; u < r; ++u) {
        if (tid == 0) s_reps[u] = rep;
        for (int j = tid; j < d; j += NT) s_vec[j] = static_cast<double>(load_elem(row(rep), j));
        __syncthreads();
        // fold the new representative into the running minimum; a chosen
        // representative gets -1 so that it is never chosen again
        ArgVal far{-INFINITY, 0x7fffffff};
        for (int i = tid; i < n; i += NT) {
            double m, dd = sqdist_to(row(i), s_vec, d);
            int o;
            if (u == 0) {
                m = dd;
                o = 0;
            } else {
                m = mind[i];
                o = owner[i];
                if (dd < m) {
                    m = dd;
                    o = u;
                }
            }
            if (i == rep) {
                m = -1.0;
                o = u;
            }
            mind[i] = m;
            owner[i] = o;
            far = pick_max(far, ArgVal{m, i});
        }
        if (u + 1 < r) {
            far = block_arg<true, NT / kWave>(far, s_red);
            rep = far.i < n ? far.i : 0;
        } else {
            __syncthreads();
        }
    }

    // team sizes and offsets inside the parent
    for (int u = tid; u < r; u += NT) s_cnt[u] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += NT) atomicAdd(&s_cnt[owner[i]], 1);
    __syncthreads();
    if (tid == 0) {
        int acc = 0;
        for (int u = 0; u < r; ++u) {
            s_off[u] = acc;
            acc += s_cnt[u];
        }
    }
    __syncthreads();
    const size_t tbase = static_cast<size_t>(bh) * M + team0;
    for (int u = tid; u < r; u += NT) {
        team_begin[tbase + u] = start + s_off[u];
        team_size[tbase + u] = s_cnt[u];
        log_n[tbase + u] = log(static_cast<double>(s_cnt[u]));
        rep_token[tbase + u] = tok(s_reps[u]);
    }

    // packed position of each member: team offset + rank among the team's
    // members in token order (ballots per representative, chunk by chunk)
    int* pperm = perm + static_cast<size_t>(bh) * N + start;
    const int w = wave_id();
    const uint64_t lt = lanemask_lt();
    for (int base = 0; base < n; base += NT) {
        const int i = base + tid;
        const int o = (i < n) ? owner[i] : -1;
        int rank_in_wave = 0;
        for (int u = 0; u < r; ++u) {
            const uint64_t m = __ballot(o == u);
            if (o == u) rank_in_wave = __popcll(m & lt);
            if (lane_id() == 0) s_wcnt[w][u] = __popcll(m);
        }
        __syncthreads();
        if (i < n) {
            int pos = s_off[o] + rank_in_wave;
            for (int v = 0; v < w; ++v) pos += s_wcnt[v][o];
            pperm[pos] = tok(i);
        }
        __syncthreads();
        for (int u = tid; u < r; u += NT) {
            int add = 0;
            for (int v = 0; v < (NT / kWave); ++v) add += s_wcnt[v][u];
            s_off[u] += add;
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Register-resident variant of the same construction for parents of at most
// kRegThreads members whose rows fit 64 registers (d * element size <= 256 B).
// Thread i holds member i's key row in registers for the whole build, so each
// round reads only the new representative (an LDS broadcast) instead of every
// member's row from memory.  The arithmetic, its order and the tie rules are
// those of k_build_parent, so both kernels produce identical tables.
constexpr int kRegThreads = 512;
constexpr int kRegWaves = kRegThreads / kWave;
constexpr int kRankBlock = kWave;  // representatives ranked per ballot block

// A member row as 32-bit words: packed bf16 pairs, or fp32 values.
template <typename T, int D>
struct RegRow;

template <int D>
struct RegRow<bf16_t, D> {
    static constexpr int kWords = D / 2;
    uint32_t w[kWords];
    __device__ __forceinline__ void load(const bf16_t* row) {
        const uint4* p = reinterpret_cast<const uint4*>(row);
#pragma unroll
        for (int k = 0; k < kWords / 4; ++k) {
            const uint4 v = p[k];
            w[4 * k] = v.x;
            w[4 * k + 1] = v.y;
            w[4 * k + 2] = v.z;
            w[4 * k + 3] = v.w;
        }
    }
    __device__ __forceinline__ float elem(int j) const {
        return (j & 1) ? bf16hi(w[j >> 1]) : bf16lo(w[j >> 1]);
    }
    // hides the words from code motion: widening the row to fp64 ahead of
    // its use would need 4 D registers
    __device__ __forceinline__ void opaque() {
#pragma unroll
        for (int k = 0; k < kWords; ++k) asm volatile("" : "+v"(w[k]));
    }
    // the same for the words of dimensions j0 .. j0 + 7
    __device__ __forceinline__ void opaque8(int j0) {
#pragma unroll
        for (int k = 0; k < 4; ++k) asm volatile("" : "+v"(w[j0 / 2 + k]));
    }
    __device__ __forceinline__ void store(bf16_t* row) const {
        uint4* p = reinterpret_cast<uint4*>(row);
#pragma unroll
        for (int k = 0; k < kWords / 4; ++k) p[k] = make_uint4(w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]);
    }
    // the row as kWords / 4 chunks of 16 bytes, chunk c at position c ^ sw
    __device__ __forceinline__ void store_swizzled(uint4* dst, int sw) const {
#pragma unroll
        for (int k = 0; k < kWords / 4; ++k) dst[k ^ sw] = make_uint4(w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]);
    }
    // element j of a row stored by store_swizzled
    static __device__ __forceinline__ float swizzled_elem(const uint4* src, int j, int sw) {
        const uint16_t* c = reinterpret_cast<const uint16_t*>(src + ((j >> 3) ^ sw));
        return __uint_as_float(static_cast<uint32_t>(c[j & 7]) << 16);
    }
    // lane l < kWords widens the stored row's word l (dimensions 2l, 2l + 1)
    // to fp64
    static __device__ __forceinline__ void widen(const uint32_t* words, double* out, int lane) {
        if (lane < kWords) {
            const uint32_t x = words[lane];
            *reinterpret_cast<double2*>(out + 2 * lane) =
                make_double2(static_cast<double>(bf16lo(x)), static_cast<double>(bf16hi(x)));
        }
    }
};

template <int D>
struct RegRow<float, D> {
    static constexpr int kWords = D;
    float w[kWords];
    __device__ __forceinline__ void load(const float* row) {
        const float4* p = reinterpret_cast<const float4*>(row);
#pragma unroll
        for (int k = 0; k < kWords / 4; ++k) {
            const float4 v = p[k];
            w[4 * k] = v.x;
            w[4 * k + 1] = v.y;
            w[4 * k + 2] = v.z;
            w[4 * k + 3] = v.w;
        }
    }
    __device__ __forceinline__ float elem(int j) const { return w[j]; }
    __device__ __forceinline__ void opaque() {
#pragma unroll
        for (int k = 0; k < kWords; ++k) asm volatile("" : "+v"(w[k]));
    }
    __device__ __forceinline__ void opaque8(int j0) {
#pragma unroll
        for (int k = 0; k < 8; ++k) asm volatile("" : "+v"(w[j0 + k]));
    }
    __device__ __forceinline__ void store(float* row) const {
        float4* p = reinterpret_cast<float4*>(row);
#pragma unroll
        for (int k = 0; k < kWords / 4; ++k) p[k] = make_float4(w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]);
    }
    __device__ __forceinline__ void store_swizzled(uint4* dst, int sw) const {
#pragma unroll
        for (int k = 0; k < kWords / 4; ++k)
            dst[k ^ sw] = make_uint4(__float_as_uint(w[4 * k]), __float_as_uint(w[4 * k + 1]),
                                     __float_as_uint(w[4 * k + 2]), __float_as_uint(w[4 * k + 3]));
    }
    static __device__ __forceinline__ float swizzled_elem(const uint4* src, int j, int sw) {
        return reinterpret_cast<const float*>(src + ((j >> 2) ^ sw))[j & 3];
    }
    // lane l < kWords widens the stored row's dimension l to fp64
    static __device__ __forceinline__ void widen(const uint32_t* words, double* out, int lane) {
        if (lane < kWords) out[lane] = static_cast<double>(__uint_as_float(words[lane]));
    }
};

// |k - c|^2 with c an fp64 vector in LDS (read as broadcasts), summed in
// dimension order without contraction.
template <typename T, int D>
__device__ __forceinline__ double reg_sqdist(const RegRow<T, D>& r, const double* c) {
#pragma clang fp contract(off)
    double acc = 0.0;
#pragma unroll
    for (int j = 0; j < D; j += 2) {
        // LDS reads are kept in groups of four (eight dims): hoisting them
        // all would need 256 registers for c
        if (j % 8 == 0) asm volatile("" ::: "memory");
        const double2 cc = *reinterpret_cast<const double2*>(c + j);
        const double t0 = static_cast<double>(r.elem(j)) - cc.x;
        acc = acc + t0 * t0;
        const double t1 = static_cast<double>(r.elem(j + 1)) - cc.y;
        acc = acc + t1 * t1;
    }
    return acc;
}

// (value, index) extremum over the wave (wave-uniform): DPP row rotations
// within each 16-lane row, then the four rows' results.  The order is total
// (value, then the smaller index; NaN never reaches it), so any reduction
// order gives the same winner.
template <bool kMax>
__device__ __forceinline__ ArgVal wave_arg(ArgVal x) {
#define SANTAPP_ARGSTEP(CTRL)                                                  \
    {                                                                          \
        ArgVal y;                                                              \
        y.v = dpp_f64<CTRL>(x.v);                                              \
        y.i = __builtin_amdgcn_update_dpp(0, x.i, CTRL, 0xF, 0xF, false);     \
        x = kMax ? pick_max(x, y) : pick_min(x, y);                            \
    }
    SANTAPP_ARGSTEP(0x128)
    SANTAPP_ARGSTEP(0x124)
    SANTAPP_ARGSTEP(0x122)
    SANTAPP_ARGSTEP(0x121)
#undef SANTAPP_ARGSTEP
    const uint64_t vb = static_cast<uint64_t>(__double_as_longlong(x.v));
    ArgVal r{__longlong_as_double(static_cast<long long>(readlane(vb, 0))), readlane(x.i, 0)};
#pragma unroll
    for (int row = 1; row < 4; ++row) {
        const ArgVal y{__longlong_as_double(static_cast<long long>(readlane(vb, 16 * row))), readlane(x.i, 16 * row)};
        r = kMax ? pick_max(r, y) : pick_min(r, y);
    }
    return r;
}

// (value, index) reduction over the workgroup's waves; s_red holds one
// entry per wave.  The caller separates reuses of s_red by a barrier.
template <bool kMax>
__device__ __forceinline__ ArgVal reg_block_arg(ArgVal x, ArgVal* s_red, int nw) {
    x = wave_arg<kMax>(x);
    if (lane_id() == 0) s_red[wave_id()] = x;
    __syncthreads();
    ArgVal r = s_red[0];
#pragma unroll
    for (int w = 1; w < kRegWaves; ++w)
        if (w < nw) r = kMax ? pick_max(r, s_red[w]) : pick_min(r, s_red[w]);
    return r;
}

// Thread t owns members t + k * blockDim.x, k < MPT, and is launched with
// max(D, ceil(members / MPT) rounded up to a wave) threads.  Two members per
// thread let one LDS read of the representative serve two distances.  The
// kernel also writes the parent's rows of the packed copies: each member's
// key from its registers and its value row, at its packed position, and the
// representative key of each of its teams.
template <typename T, int D, int MPT>
__global__ __launch_bounds__(kRegThreads) void k_build_parent_regs(
    const T* __restrict__ K, const T* __restrict__ V, int N, int P, int R, int M,
    int* __restrict__ team_begin, int* __restrict__ team_size, double* __restrict__ log_n,
    int* __restrict__ rep_token, int* __restrict__ perm, T* __restrict__ packed_K,
    T* __restrict__ packed_V, T* __restrict__ reps, int* __restrict__ team_count) {
#pragma clang fp contract(off)
    __shared__ __align__(16) double s_mean[D];
    __shared__ __align__(16) uint32_t s_raw[RegRow<T, D>::kWords];  // the new representative's words
    __shared__ __align__(16) double s_cw[kRegWaves][D];  // each wave's fp64 copy of it
    // one slot's rows (member t + k nt in row t), for the mean; 16-byte
    // chunk c of row t sits at position c ^ (t mod chunks) so that the
    // lanes' row stores spread over the banks
    constexpr int kChunks = RegRow<T, D>::kWords / 4;
    __shared__ __align__(16) uint4 s_rows[kRegThreads][kChunks];
    __shared__ ArgVal s_red[2][kRegWaves];
    __shared__ int s_reps[kMaxReps];
    __shared__ int s_cnt[kMaxReps];
    __shared__ int s_off[kMaxReps];
    __shared__ int s_wsum[kRegWaves];
    __shared__ int s_wcnt[MPT][kRegWaves][kRankBlock];

    const int p = blockIdx.x;
    const int bh = blockIdx.y;
    const int tid = threadIdx.x;
    const int nt = blockDim.x;
    const int nw = nt / kWave;
    const int w = wave_id(), lane = lane_id();
    const int start = p * P;
    const int n = min(P, N - start);
    const int r = min(R, n);
    const int team0 = p * min(R, P);  // every earlier parent is full-size
    const T* Kc = K + (static_cast<size_t>(bh) * N + start) * D;
    if (p == 0 && tid == 0) team_count[bh] = M;  // every pair has M teams

    RegRow<T, D> row[MPT];
    bool member[MPT];
#pragma unroll
    for (int k = 0; k < MPT; ++k) {
        const int i = tid + k * nt;
        member[k] = i < n;
        if (member[k]) row[k].load(Kc + static_cast<size_t>(i) * D);
    }

    // parent mean, summed over members in token order: each slot's rows
    // pass through LDS at once, and thread j < D adds dimension j of each
    // staged row in turn, the reads 16 rows ahead of their (serial)
    // additions
    double msum = 0.0;
#pragma unroll
    for (int k = 0; k < MPT; ++k) {
        const int cnt = min(nt, n - k * nt);  // members of slot k
        if (cnt <= 0) break;
        if (k > 0) __syncthreads();  // the previous slot's reads are done
        row[k].opaque();
        if (member[k]) row[k].store_swizzled(s_rows[tid], tid & (kChunks - 1));
        __syncthreads();
        if (tid < D) {
            int i0 = 0;
            for (; i0 + 16 <= cnt; i0 += 16) {
                float x[16];
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    x[i] = RegRow<T, D>::swizzled_elem(s_rows[i0 + i], tid, (i0 + i) & (kChunks - 1));
#pragma unroll
                for (int i = 0; i < 16; ++i) msum = msum + static_cast<double>(x[i]);
                asm volatile("" : "+v"(msum)::"memory");  // one batch of reads in flight at a time
            }
            for (; i0 < cnt; ++i0)
                msum = msum + static_cast<double>(RegRow<T, D>::swizzled_elem(s_rows[i0], tid, i0 & (kChunks - 1)));
        }
    }
    if (tid < D) s_mean[tid] = msum / static_cast<double>(n);
    __syncthreads();

    // distances of this thread's members to the vector c in LDS: |k - c|^2
    // summed in dimension order without contraction, one LDS read of c for
    // all MPT members, eight dimensions per scheduling group (hoisting the
    // reads or the widening of all dimensions would need 4 D registers)
    auto distances = [&](const double* c, double (&dd)[MPT]) {
#pragma unroll
        for (int k = 0; k < MPT; ++k) {
            row[k].opaque();
            dd[k] = 0.0;
        }
#pragma unroll
        for (int j = 0; j < D; j += 2) {
            if (j % 8 == 0) {
                // the sums so far are complete before the group's LDS reads
                // and widening (no group's work moves past another's)
#pragma unroll
                for (int k = 0; k < MPT; ++k) {
                    asm volatile("" : "+v"(dd[k])::"memory");
                    row[k].opaque8(j);
                }
            }
            const double2 cc = *reinterpret_cast<const double2*>(c + j);
#pragma unroll
            for (int k = 0; k < MPT; ++k) {
                const double t0 = static_cast<double>(row[k].elem(j)) - cc.x;
                dd[k] = dd[k] + t0 * t0;
                const double t1 = static_cast<double>(row[k].elem(j + 1)) - cc.y;
                dd[k] = dd[k] + t1 * t1;
            }
        }
    };

    // first representative: the member nearest the mean
    double dd[MPT];
    distances(s_mean, dd);
    ArgVal best{INFINITY, 0x7fffffff};
#pragma unroll
    for (int k = 0; k < MPT; ++k)
        if (member[k]) best = pick_min(best, ArgVal{dd[k], tid + k * nt});
    int rep = reg_block_arg<false>(best, s_red[0], nw).i;
    if (rep >= n) rep = 0;  // no winner (NaN keys): stay inside the parent

    // farthest-first rounds with a running minimum; a chosen representative
    // gets -1 so that it is never chosen again.  Round u uses buffer
    // (u + 1) & 1 of s_red (the mean used buffer 0): a buffer is rewritten
    // two rounds after it was read, past both barriers of the round between.
    // The new representative's owner stores its raw words to s_raw, and
    // after the barrier every wave widens them into its own fp64 copy
    // (wave-private, so no second barrier); s_raw is rewritten only after
    // the round's reduction barrier, which every wave reaches after its
    // widening.
    double m[MPT];
    int o[MPT];
#pragma unroll
    for (int k = 0; k < MPT; ++k) {
        m[k] = 0.0;
        o[k] = 0;
    }
    for (int u = 0; u < r; ++u) {
        const int b = (u + 1) & 1;
        const int rk = rep / nt;
        if (tid == rep - rk * nt) {
            s_reps[u] = rep;
#pragma unroll
            for (int k = 0; k < MPT; ++k)
                if (k == rk) row[k].store(reinterpret_cast<T*>(s_raw));
        }
        __syncthreads();
        double* cw = s_cw[w];
        RegRow<T, D>::widen(s_raw, cw, lane);
        distances(cw, dd);
        ArgVal far{-INFINITY, 0x7fffffff};
#pragma unroll
        for (int k = 0; k < MPT; ++k) {
            const int i = tid + k * nt;
            if (member[k]) {
                if (u == 0 || dd[k] < m[k]) {
                    m[k] = dd[k];
                    o[k] = u;
                }
                if (i == rep) {
                    m[k] = -1.0;
                    o[k] = u;
                }
                far = pick_max(far, ArgVal{m[k], i});
            }
        }
        if (u + 1 < r) {
            rep = reg_block_arg<true>(far, s_red[b], nw).i;
            if (rep >= n) rep = 0;
        }
    }
    __syncthreads();

    // team sizes and their exclusive scan (r <= blockDim.x: one team per
    // thread)
    for (int u = tid; u < r; u += nt) s_cnt[u] = 0;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < MPT; ++k)
        if (member[k]) atomicAdd(&s_cnt[o[k]], 1);
    __syncthreads();
    for (int base = 0; base < r; base += nt) {
        const int u = base + tid;
        const int c = u < r ? s_cnt[u] : 0;
        const int inc = wave_incl_scan(c);
        if (lane == kWave - 1) s_wsum[w] = inc;
        __syncthreads();
        int pre = base > 0 ? s_off[base - 1] + s_cnt[base - 1] : 0;
        for (int v = 0; v < w; ++v) pre += s_wsum[v];
        if (u < r) s_off[u] = pre + inc - c;
        __syncthreads();
    }
    const size_t tbase = static_cast<size_t>(bh) * M + team0;
    for (int u = tid; u < r; u += nt) {
        team_begin[tbase + u] = start + s_off[u];
        team_size[tbase + u] = s_cnt[u];
        log_n[tbase + u] = log(static_cast<double>(s_cnt[u]));
        rep_token[tbase + u] = start + s_reps[u];
    }

    // packed position of each member: its team's offset plus its rank among
    // the team's members in token order (slot k of wave v holds members
    // k nt + 64 v ..), per block of 64 representatives with one ballot per
    // representative, slot and wave
    int* pperm = perm + static_cast<size_t>(bh) * N + start;
    const uint64_t lt = lanemask_lt();
    int pos[MPT];
#pragma unroll
    for (int k = 0; k < MPT; ++k) pos[k] = 0;
    for (int ub = 0; ub < r; ub += kRankBlock) {
        const int nb = min(kRankBlock, r - ub);
        int rank_in_wave[MPT];
#pragma unroll
        for (int k = 0; k < MPT; ++k) {
            const int ok = member[k] ? o[k] : -1;
            rank_in_wave[k] = 0;
            for (int q = 0; q < nb; ++q) {
                const uint64_t bm = __ballot(ok == ub + q);
                if (ok == ub + q) rank_in_wave[k] = __popcll(bm & lt);
                if (lane == 0) s_wcnt[k][w][q] = __popcll(bm);
            }
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < MPT; ++k) {
            const int ok = member[k] ? o[k] : -1;
            if (ok >= ub && ok < ub + nb) {
                int ps = s_off[ok] + rank_in_wave[k];
                for (int kk = 0; kk < k; ++kk)
                    for (int v = 0; v < nw; ++v) ps += s_wcnt[kk][v][ok - ub];
                for (int v = 0; v < w; ++v) ps += s_wcnt[k][v][ok - ub];
                pperm[ps] = start + tid + k * nt;
                pos[k] = ps;
            }
        }
        __syncthreads();
    }

    // packed copies: key rows from registers, value rows copied, and each
    // team's representative key (its member's row, re-read from memory)
    const size_t prow0 = static_cast<size_t>(bh) * N + start;
#pragma unroll
    for (int k = 0; k < MPT; ++k) {
        if (member[k]) {
            const size_t prow = prow0 + pos[k];
            row[k].store(packed_K + prow * D);
            const uint4* src = reinterpret_cast<const uint4*>(V + (prow0 + tid + k * nt) * D);
            uint4* dst = reinterpret_cast<uint4*>(packed_V + prow * D);
#pragma unroll
            for (int c = 0; c < kChunks; ++c) dst[c] = src[c];
        }
    }
    for (int c = tid; c < r * kChunks; c += nt) {
        const int u = c / kChunks, q = c - u * kChunks;
        reinterpret_cast<uint4*>(reps + (tbase + u) * D)[q] =
            reinterpret_cast<const uint4*>(Kc + static_cast<size_t>(s_reps[u]) * D)[q];
    }
}

// Row gather into team order: packed[bh][pos] = src[bh][perm[bh][pos]], and the
// representative keys reps[bh][g] = K[bh][rep_token[bh][g]].  One thread per
// 16-byte chunk of a row.
__global__ __launch_bounds__(256) void k_gather_rows(const uint4* __restrict__ src,
                                                     uint4* __restrict__ dst,
                                                     const int* __restrict__ index, int rows_out,
                                                     int rows_in, int chunks_per_row, int BH) {
    const size_t total = static_cast<size_t>(BH) * rows_out * chunks_per_row;
    for (size_t t = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; t < total;
         t += static_cast<size_t>(gridDim.x) * blockDim.x) {
        const size_t row = t / chunks_per_row;
        const int c = static_cast<int>(t - row * chunks_per_row);
        const size_t bh = row / rows_out;
        const int srow = index[row];
        dst[t] = src[(bh * rows_in + srow) * chunks_per_row + c];
    }
}

}  // namespace

bool build_packs_in_place(int N, int d, santapp_dtype dtype, int P, int R) {
    const int members = std::min(P, N);
    return members <= 2 * kRegThreads && R <= kMaxReps &&
           ((dtype == SANTAPP_BF16 && (d == 128 || d == 64)) || (dtype == SANTAPP_FP32 && d == 64));
}

hipError_t launch_build_parents(const void* K, const void* V, santapp_dtype dtype, int BH, int N,
                                int d, int P, int R, int M, double* mind, int* owner,
                                int* team_begin, int* team_size, double* log_n, int* rep_token,
                                int* perm, void* packed_K, void* packed_V, void* reps, int* team_count,
                                bool* packed, hipStream_t s) {
    *packed = false;
    const dim3 grid((N + P - 1) / P, BH);
    // register-resident kernel where a parent fits 2 kRegThreads members and
    // a row 64 registers (two members per thread above kRegThreads); the
    // general kernel otherwise.  At least one thread per dimension: they sum
    // the parent mean.
    const int members = std::min(P, N);
    if (build_packs_in_place(N, d, dtype, P, R)) {
        const int mpt = members > kRegThreads ? 2 : 1;
        const int threads = std::max(d, ((members + mpt - 1) / mpt + kWave - 1) / kWave * kWave);
#define SANTAPP_REGS(TT, DD)                                                                       \
    do {                                                                                          \
        auto kern = mpt == 1 ? k_build_parent_regs<TT, DD, 1> : k_build_parent_regs<TT, DD, 2>;  \
        kern<<<grid, threads, 0, s>>>(static_cast<const TT*>(K), static_cast<const TT*>(V), N, P, R, \
                                      M, team_begin, team_size, log_n, rep_token, perm,           \
                                      static_cast<TT*>(packed_K), static_cast<TT*>(packed_V),    \
                                      static_cast<TT*>(reps), team_count);                        \
        *packed = true;                                                                           \
        return hipGetLastError();                                                                 \
    } while (0)
        if (dtype == SANTAPP_BF16 && d == 128) SANTAPP_REGS(bf16_t, 128);
        if (dtype == SANTAPP_BF16 && d == 64) SANTAPP_REGS(bf16_t, 64);
        if (dtype == SANTAPP_FP32 && d == 64) SANTAPP_REGS(float, 64);
#undef SANTAPP_REGS
    }
    if (dtype == SANTAPP_BF16)
        k_build_parent<bf16_t, false, kBuildThreads><<<grid, kBuildThreads, 0, s>>>(
            static_cast<const bf16_t*>(K), N, d, P, R, M, mind, owner, team_begin, team_size,
            log_n, rep_token, perm, nullptr, nullptr, nullptr, 0, team_count);
    else
        k_build_parent<float, false, kBuildThreads><<<grid, kBuildThreads, 0, s>>>(
            static_cast<const float*>(K), N, d, P, R, M, mind, owner, team_begin, team_size,
            log_n, rep_token, perm, nullptr, nullptr, nullptr, 0, team_count);
    return hipGetLastError();
}

hipError_t launch_build_parent_lists(const void* K, santapp_dtype dtype, int BH, int N, int d, int Mp,
                                     int R, int M, const int* members, const int* pbeg, const int* toff,
                                     double* mind, int* owner, int* team_begin, int* team_size,
                                     double* log_n, int* rep_token, int* perm, hipStream_t s) {
    const dim3 grid(Mp, BH);
    if (dtype == SANTAPP_BF16)
        k_build_parent<bf16_t, true, kListBuildThreads><<<grid, kListBuildThreads, 0, s>>>(
            static_cast<const bf16_t*>(K), N, d, 0, R, M, mind, owner, team_begin, team_size, log_n,
            rep_token, perm, members, pbeg, toff, Mp, nullptr);
    else
        k_build_parent<float, true, kListBuildThreads><<<grid, kListBuildThreads, 0, s>>>(
            static_cast<const float*>(K), N, d, 0, R, M, mind, owner, team_begin, team_size, log_n,
            rep_token, perm, members, pbeg, toff, Mp, nullptr);
    return hipGetLastError();
}

hipError_t launch_gather_rows(const void* src, void* dst, const int* index, int BH, int rows_out,
                              int rows_in, size_t row_bytes, hipStream_t s) {
    const int chunks = static_cast<int>(row_bytes / 16);
    const size_t total = static_cast<size_t>(BH) * rows_out * chunks;
    const size_t want = (total + 255) / 256;
    const unsigned blocks = static_cast<unsigned>(want < 65536 ? want : 65536);
    k_gather_rows<<<blocks, 256, 0, s>>>(static_cast<const uint4*>(src), static_cast<uint4*>(dst),
                                         index, rows_out, rows_in, chunks, BH);
    return hipGetLastError();
}

}  // namespace santapp
