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
#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

constexpr int kBuildThreads = 256;
constexpr int kBuildWaves = kBuildThreads / kWave;

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

template <bool kMax>
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
    for (int w = 1; w < kBuildWaves; ++w) r = kMax ? pick_max(r, s_red[w]) : pick_min(r, s_red[w]);
    __syncthreads();
    return r;
}

// |k_i - c|^2 with c held in LDS as fp64, summed in dimension order.
template <typename T>
__device__ double sqdist_to(const T* __restrict__ row, const double* __restrict__ c, int d) {
#pragma clang fp contract(off)
    double acc = 0.0;
    for (int j = 0; j < d; ++j) {
        const double t = static_cast<double>(load_elem(row, j)) - c[j];
        acc = acc + t * t;
    }
    return acc;
}

template <typename T>
__global__ __launch_bounds__(kBuildThreads) void k_build_parent(
    const T* __restrict__ K, int N, int d, int P, int R, int M, double* __restrict__ mind_all,
    int* __restrict__ owner_all, int* __restrict__ team_begin, int* __restrict__ team_size,
    double* __restrict__ log_n, int* __restrict__ rep_token, int* __restrict__ perm) {
#pragma clang fp contract(off)
    __shared__ double s_vec[kMaxHeadDim];
    __shared__ ArgVal s_red[kBuildWaves];
    __shared__ int s_reps[kMaxReps];
    __shared__ int s_cnt[kMaxReps];
    __shared__ int s_off[kMaxReps];
    __shared__ int s_wcnt[kBuildWaves][kMaxReps];

    const int p = blockIdx.x;
    const int bh = blockIdx.y;
    const int tid = threadIdx.x;
    const int start = p * P;
    const int n = min(P, N - start);
    const int r = min(R, n);
    const int team0 = p * min(R, P);  // every earlier parent is full-size
    const T* Kc = K + (static_cast<size_t>(bh) * N + start) * d;
    double* mind = mind_all + static_cast<size_t>(bh) * N + start;
    int* owner = owner_all + static_cast<size_t>(bh) * N + start;

    // parent mean, summed over members in token order
    for (int j = tid; j < d; j += kBuildThreads) {
        double s = 0.0;
        for (int i = 0; i < n; ++i) s = s + static_cast<double>(load_elem(Kc, static_cast<size_t>(i) * d + j));
        s_vec[j] = s / static_cast<double>(n);
    }
    __syncthreads();

    // first representative: the member nearest the mean
    ArgVal best{INFINITY, 0x7fffffff};
    for (int i = tid; i < n; i += kBuildThreads) {
        ArgVal c{sqdist_to(Kc + static_cast<size_t>(i) * d, s_vec, d), i};
        best = pick_min(best, c);
    }
    best = block_arg<false>(best, s_red);
    int rep = best.i;

    for (int u = 0; u < r; ++u) {
        if (tid == 0) s_reps[u] = rep;
        for (int j = tid; j < d; j += kBuildThreads)
            s_vec[j] = static_cast<double>(load_elem(Kc, static_cast<size_t>(rep) * d + j));
        __syncthreads();
        // fold the new representative into the running minimum; a chosen
        // representative gets -1 so that it is never chosen again
        ArgVal far{-INFINITY, 0x7fffffff};
        for (int i = tid; i < n; i += kBuildThreads) {
            double m, dd = sqdist_to(Kc + static_cast<size_t>(i) * d, s_vec, d);
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
            far = block_arg<true>(far, s_red);
            rep = far.i;
        } else {
            __syncthreads();
        }
    }

    // team sizes and offsets inside the parent
    for (int u = tid; u < r; u += kBuildThreads) s_cnt[u] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += kBuildThreads) atomicAdd(&s_cnt[owner[i]], 1);
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
    for (int u = tid; u < r; u += kBuildThreads) {
        team_begin[tbase + u] = start + s_off[u];
        team_size[tbase + u] = s_cnt[u];
        log_n[tbase + u] = log(static_cast<double>(s_cnt[u]));
        rep_token[tbase + u] = start + s_reps[u];
    }

    // packed position of each member: team offset + rank among the team's
    // members in token order (ballots per representative, chunk by chunk)
    int* pperm = perm + static_cast<size_t>(bh) * N + start;
    const int w = wave_id();
    const uint64_t lt = lanemask_lt();
    for (int base = 0; base < n; base += kBuildThreads) {
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
            pperm[pos] = start + i;
        }
        __syncthreads();
        for (int u = tid; u < r; u += kBuildThreads) {
            int add = 0;
            for (int v = 0; v < kBuildWaves; ++v) add += s_wcnt[v][u];
            s_off[u] += add;
        }
        __syncthreads();
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

hipError_t launch_build_parents(const void* K, santapp_dtype dtype, int BH, int N, int d, int P,
                                int R, int M, double* mind, int* owner, int* team_begin,
                                int* team_size, double* log_n, int* rep_token, int* perm,
                                hipStream_t s) {
    const dim3 grid((N + P - 1) / P, BH);
    if (dtype == SANTAPP_BF16)
        k_build_parent<bf16_t><<<grid, kBuildThreads, 0, s>>>(
            static_cast<const bf16_t*>(K), N, d, P, R, M, mind, owner, team_begin, team_size,
            log_n, rep_token, perm);
    else
        k_build_parent<float><<<grid, kBuildThreads, 0, s>>>(
            static_cast<const float*>(K), N, d, P, R, M, mind, owner, team_begin, team_size,
            log_n, rep_token, perm);
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
