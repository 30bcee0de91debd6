// One SANTA++ decode step, and the dense baseline.
//
// Phase A, sampling (one workgroup per query head; eq. method-routing,
//   Alg. "SANTA++ attention for one query head", eq. method-inclusion):
//   the routing logits phi_g = log n_g + scale q.l_g of the head's teams in
//   fp64 (every bf16 x fp32 product is exact in fp64, so phi differs from an
//   fp64 reference only by summation order), the Gumbel perturbation
//   Y_g = phi_g + G_g, tau = the (K+1)-th largest Y (a value histogram, and
//   an exact finish over order-preserving 64-bit keys), the K largest as the
//   sample (ties to the lower team index) and log c_g.  The head publishes
//   its sample as bits in team order and the log c of its sampled teams.
// Phase B, attention (eq. method-estimate), on workgroups bound to one
//   (sequence, KV head) pair.  Each workgroup builds the pair's read plan in
//   LDS from its G heads' sample bits: the union of the samples in team
//   order, each union team cut into units of at most kUnitRows packed rows
//   that carry the mask of the heads that sampled the team.  Every wave walks
//   its share of the pair's units (the exact suffix first, then the union)
//   carrying one online-softmax state per query head from unit to unit: a
//   unit's rows enter head h's state with the base-2 logit
//   log2(e) (scale q_h.k_i - log c_{g,h}) when head h sampled the unit's team
//   g, and do not enter it otherwise; suffix rows enter every head with no
//   correction.  The query heads of the group share every K/V load: scores
//   and value sums run on the matrix cores for bf16 rows.
// Phase C, merge: the waves' states are combined in LDS and each workgroup
//   publishes one state per query head; for every head one designated
//   workgroup of the pair waits for all of them and rescales them to a
//   common maximum, giving U^ / Z^ (App. "Triton decode kernels",
//   split-softmax reducer).
//
// Launch modes: the sampling kernel followed by the attention kernel
// (split), or all three phases in one launch (fused), in which a pair's
// attention waits for the pair's G sampling workgroups to arrive.  The dense
// baseline (and a budget that takes every team) runs phases B and C over
// every row.
//
// Hand-offs between workgroups use agent-scope (coherent) stores and loads
// for the data and a per-pair counter: the producer waits for its coherent
// stores to complete before it increments the counter, and the consumer
// reads the data with coherent loads after it has seen the count.  No cache
// write-back or invalidation is needed (the write-back of a release fence
// also drains whatever earlier kernels left dirty in the L2).  Every counter
// is reset by its last reader, so each call leaves the workspace counters at
// zero.  Waits are bounded: a wait that runs out poisons the affected
// outputs with NaN instead of hanging.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include <hip/hip_ext.h>

#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

constexpr int kThreads = kDecodeThreads;
constexpr int kWaves = kThreads / kWave;
static_assert(kWaves == 8, "block scans read eight wave totals");
constexpr int kFineBits = 16;       // value-histogram resolution of the general sampler
constexpr int kPlanRecs = kThreads; // union teams of one plan pass
constexpr int kPlanUnits = 3072;    // units of a plan pass resolved through an LDS table
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNeg = -1.0e30f;    // logit of a row that carries no weight
constexpr float kEmpty = -1.0e29f;  // states with a maximum below this hold no row
constexpr int kSpinLimit = 1 << 18; // polls of a counter before a wait gives up

enum Mode { kSample = 0, kAttend = 1, kFused = 2 };

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Order of this wave's LDS accesses for the compiler only: the LDS executes
// one wave's instructions in order, so no wait is needed (a fence would also
// wait for the value copies in flight).
__device__ __forceinline__ void lds_order() { asm volatile("" ::: "memory"); }

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Every memory access of every thread of the workgroup is complete, then the
// workgroup synchronises (the barrier alone does not wait for stores).
__device__ __forceinline__ void drain_and_sync() {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
}

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

__device__ __forceinline__ float wave_max_f(float v) {
    for (int off = kWave / 2; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
    return v;
}

__device__ __forceinline__ float wave_sum_f(float v) {
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

// Wave-uniform copies (scalar registers) of values every lane holds alike.
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Agent-scope (coherent) accesses: a store is performed at agent scope once
// it completes, and a load never returns a stale cached copy.
__device__ __forceinline__ void store_u64_coherent(void* p, unsigned long long x) {
    __hip_atomic_store(static_cast<unsigned long long*>(p), x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_f32_coherent(float* p, float x) {
    __hip_atomic_store(reinterpret_cast<unsigned*>(p), __float_as_uint(x), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long load_u64_coherent(const void* p) {
    return __hip_atomic_load(static_cast<const unsigned long long*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_f32_coherent(const float* p) {
    return __uint_as_float(__hip_atomic_load(reinterpret_cast<const unsigned*>(p), __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ int load_i32_coherent(const int* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_f2_coherent(float* p, float x, float y) {
    store_u64_coherent(p, (static_cast<unsigned long long>(__float_as_uint(y)) << 32) | __float_as_uint(x));
}
__device__ __forceinline__ float2 load_f2_coherent(const float* p) {
    const unsigned long long u = load_u64_coherent(p);
    return make_float2(__uint_as_float(static_cast<unsigned>(u)), __uint_as_float(static_cast<unsigned>(u >> 32)));
}
__device__ __forceinline__ void store_f4_coherent(float* p, float4 v) {
    store_f2_coherent(p, v.x, v.y);
    store_f2_coherent(p + 2, v.z, v.w);
}
__device__ __forceinline__ float4 load_f4_coherent(const float* p) {
    const float2 a = load_f2_coherent(p), b = load_f2_coherent(p + 2);
    return make_float4(a.x, a.y, b.x, b.y);
}

// 16-byte and 8-byte device-coherent accesses through a buffer resource
// (cache policy sc1: a store writes through to memory, a load never returns a
// copy cached in this XCD's L2).  The resource is built from a wave-uniform
// base and covers `bytes` bytes; accesses outside it read zero and store
// nothing.
typedef unsigned u32x4v __attribute__((ext_vector_type(4)));
typedef unsigned u32x2v __attribute__((ext_vector_type(2)));
constexpr int kCoherentPolicy = 16;  // sc1

__device__ __forceinline__ __amdgpu_buffer_rsrc_t coherent_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), 0x00020000);
}
__device__ __forceinline__ u32x4v load16_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(off), 0, kCoherentPolicy);
}
__device__ __forceinline__ void store16_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off, u32x4v x) {
    __builtin_amdgcn_raw_buffer_store_b128(x, r, static_cast<int>(off), 0, kCoherentPolicy);
}
__device__ __forceinline__ u32x2v load8_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b64(r, static_cast<int>(off), 0, kCoherentPolicy);
}
__device__ __forceinline__ void store8_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off, u32x2v x) {
    __builtin_amdgcn_raw_buffer_store_b64(x, r, static_cast<int>(off), 0, kCoherentPolicy);
}
__device__ __forceinline__ uint32_t load_u32_coherent(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_u32_coherent(uint32_t* p, uint32_t x) {
    __hip_atomic_store(p, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Thread 0 polls a counter until it reaches `target` (bounded); returns
// whether it did, to the whole workgroup.  The caller's other threads wait at
// the barrier.
__device__ __forceinline__ bool wait_count(const int* ctr, int target, int* s_flag) {
    if (threadIdx.x == 0) {
        int ok = 0;
        for (int it = 0; it < kSpinLimit; ++it) {
            if (load_i32_coherent(ctr) >= target) {
                ok = 1;
                break;
            }
            __builtin_amdgcn_s_sleep(2);
        }
        s_flag[0] = ok;
    }
    __syncthreads();
    const bool ok = s_flag[0] != 0;
    __syncthreads();
    return ok;
}

// Sum over the eight lanes of each lane octet (quad swaps, then the mirror
// within each half row); every lane of the octet receives it.
__device__ __forceinline__ double row8_sum(double v) {
    v += dpp_f64<0xB1>(v);   // quad_perm [1,0,3,2]
    v += dpp_f64<0x4E>(v);   // quad_perm [2,3,0,1]
    v += dpp_f64<0x141>(v);  // row_half_mirror
    return v;
}

// ---------------------------------------------------------------------------
// Phase A helpers
// ---------------------------------------------------------------------------

// Value-histogram bucket of a key in [0, 2^kFineBits): keys below the range
// (absent teams) land in bucket 0.
__device__ __forceinline__ int fine_bucket(double y, double ymin, double fs) {
    return static_cast<int>(fmin(static_cast<double>((1 << kFineBits) - 1), fmax(0.0, (y - ymin) * fs)));
}

// log c for c = 1 - exp(-exp(x)) in fp32 (eq. method-inclusion).  x >= -37
// for a sampled team (its perturbed score beats tau and a Gumbel draw is at
// most 53 log 2), so e^x stays a normal fp32.  For e^x < 1/16 a four-term
// series avoids the cancellation of 1 - exp(-e); its truncation error is below
// e^4 / 120 relative.
__device__ __forceinline__ float log_inclusion(float x) {
    constexpr float kLn2 = 0.6931471805599453f;
    const float e = __builtin_amdgcn_exp2f(x * kLog2e);
    const float c = (e < 0.0625f)
                        ? e * (1.f - e * (0.5f - e * (1.f / 6.f - e * (1.f / 24.f))))
                        : 1.f - __builtin_amdgcn_exp2f(-e * kLog2e);
    return __builtin_amdgcn_logf(c) * kLn2;
}

// Exclusive scan of NV counters over the workgroup; returns the totals.
template <int NV>
__device__ __forceinline__ void block_scan(const int (&x)[NV], int (&ex)[NV], int (&tot)[NV],
                                           int* s_w /* [NV * kWaves] */) {
    const int lane = lane_id(), w = wave_id();
    int inc[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        inc[k] = wave_incl_scan(x[k]);
        if (lane == kWave - 1) s_w[k * kWaves + w] = inc[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int4 a = reinterpret_cast<const int4*>(s_w)[2 * k];
        const int4 c = reinterpret_cast<const int4*>(s_w)[2 * k + 1];
        const int y[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
        int pre = 0, t = 0;
#pragma unroll
        for (int v = 0; v < kWaves; ++v) {
            pre += (v < w) ? y[v] : 0;
            t += y[v];
        }
        ex[k] = pre + inc[k] - x[k];
        tot[k] = t;
    }
    __syncthreads();
}

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

// LDS scratch of the sampler (beyond its score arrays).
struct SelScratch {
    uint32_t hist[256];
    uint64_t red[kWaves];
    uint64_t cand[kWave];
    uint64_t sel[kSelWords];
    uint64_t tie[kSelWords];
    int w[3 * kWaves];
    int ncand;
    int bc[3];
    int flag;
};

template <bool kMax>
__device__ __forceinline__ uint64_t block_ext64(uint64_t v, uint64_t* s_red) {
    v = kMax ? wave_max64(v) : wave_min64(v);
    if (lane_id() == 0) s_red[wave_id()] = v;
    __syncthreads();
    uint64_t r = s_red[0];
    for (int w = 1; w < kWaves; ++w) r = kMax ? max(r, s_red[w]) : min(r, s_red[w]);
    __syncthreads();
    return r;
}

template <bool kOr>
__device__ __forceinline__ uint64_t block_bits64(uint64_t v, uint64_t* s_red) {
    v = kOr ? wave_or64(v) : wave_and64(v);
    if (lane_id() == 0) s_red[wave_id()] = v;
    __syncthreads();
    uint64_t r = s_red[0];
    for (int w = 1; w < kWaves; ++w) r = kOr ? (r | s_red[w]) : (r & s_red[w]);
    __syncthreads();
    return r;
}

// Key of rank `want` (0-based, descending) among the M perturbed scores held
// as order-preserving keys, HK per thread (key j of thread t is team
// j * kThreads + t).  Value histograms over [min Y, max Y] at 2^16 buckets
// (two passes of 256; absent teams, far below the real ones, fall into bucket
// 0 unless only they differ); at most 64 keys left are ranked directly; many
// keys in one fine bucket are finished by an exact 8-bit radix over the keys.
template <int HK>
__device__ uint64_t select_rank_key(const uint64_t (&k)[HK], int M, int want, SelScratch& S) {
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    auto valid = [&](int j) { return j * kThreads + tid < M; };
    uint64_t kmin = ~0ull, kmax = 0;
#pragma unroll
    for (int j = 0; j < HK; ++j) {
        if (valid(j)) {
            kmin = min(kmin, k[j]);
            kmax = max(kmax, k[j]);
        }
    }
    kmin = block_ext64<false>(kmin, S.red);
    kmax = block_ext64<true>(kmax, S.red);
    const uint64_t kreal = order_key(kAbsentBelow);
    if (kmin < kreal) {  // uniform: only tables with absent teams
        uint64_t rmin = ~0ull;
#pragma unroll
        for (int j = 0; j < HK; ++j)
            if (valid(j) && k[j] >= kreal) rmin = min(rmin, k[j]);
        rmin = block_ext64<false>(rmin, S.red);
        if (rmin < kmax) kmin = rmin;
    }
    const double ymin = key_value(kmin);
    const double range = key_value(kmax) - ymin;
    if (!(range > 0.0)) return kmin;  // uniform: every key equal
    const double fs = (static_cast<double>(1 << kFineBits) - 0.001) / range;
    int fine[HK];
#pragma unroll
    for (int j = 0; j < HK; ++j) fine[j] = valid(j) ? fine_bucket(key_value(k[j]), ymin, fs) : -1;
    // a 256-bin histogram of the keys' bins (-1: not counted), and the bin
    // that holds rank `want`
    auto hist_pass = [&](auto bin_of) {
        if (tid < 64) reinterpret_cast<uint4*>(S.hist)[tid] = make_uint4(0, 0, 0, 0);
        __syncthreads();
#pragma unroll
        for (int j = 0; j < HK; ++j) {
            const int bn = bin_of(j);
            if (bn >= 0) atomicAdd(&S.hist[bn], 1u);
        }
        __syncthreads();
        if (w == 0) {
            int above, cnt;
            const int bin = hist_select(S.hist, want, above, cnt);
            if (lane == 0) {
                S.bc[0] = bin;
                S.bc[1] = above;
                S.bc[2] = cnt;
            }
        }
        __syncthreads();
        const int bin = S.bc[0];
        want -= S.bc[1];
        const int cnt = S.bc[2];
        __syncthreads();  // bc and hist are reused
        return make_int2(bin, cnt);
    };
    // at most 64 keys left: gather them and rank them directly
    auto rank_direct = [&](auto in) {
        if (tid == 0) S.ncand = 0;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < HK; ++j)
            if (in(j)) S.cand[atomicAdd(&S.ncand, 1)] = k[j];
        __syncthreads();
        const int n = S.ncand;
        if (w == 0) {
            const uint64_t mine = S.cand[min(lane, n - 1)];
            int gt = 0, ge = 0;
            for (int t = 0; t < n; ++t) {
                const uint64_t o = readlane(mine, t);
                gt += o > mine ? 1 : 0;
                ge += o >= mine ? 1 : 0;
            }
            const bool owner = lane < n && gt <= want && want < ge;
            const uint64_t r = readlane(mine, __ffsll(static_cast<unsigned long long>(__ballot(owner))) - 1);
            if (lane == 0) S.red[0] = r;
        }
        __syncthreads();
        const uint64_t r = S.red[0];
        __syncthreads();
        return r;
    };
    const int2 p0 = hist_pass([&](int j) { return fine[j] >= 0 ? fine[j] >> 8 : -1; });
    const int top = p0.x;
    if (p0.y <= kWave) return rank_direct([&](int j) { return fine[j] >= 0 && (fine[j] >> 8) == top; });
    const int2 p1 = hist_pass([&](int j) { return fine[j] >= 0 && (fine[j] >> 8) == top ? fine[j] & 255 : -1; });
    const int target = (top << 8) | p1.x;
    auto in_bucket = [&](int j) { return fine[j] == target; };
    if (p1.y <= kWave) return rank_direct(in_bucket);
    // many keys in one fine bucket: exact radix over their 64-bit keys
    uint64_t kand = ~0ull, kor = 0;
#pragma unroll
    for (int j = 0; j < HK; ++j) {
        if (in_bucket(j)) {
            kand &= k[j];
            kor |= k[j];
        }
    }
    const uint64_t all_and = block_bits64<false>(kand, S.red);
    const uint64_t all_or = block_bits64<true>(kor, S.red);
    const uint64_t diff = all_or & ~all_and;
    const int topbit = diff ? 63 - __clzll(static_cast<long long>(diff)) : 7;
    int sh = topbit >= 7 ? topbit - 7 : 0;
    uint64_t prefix = 0, pmask = 0;
    if (sh + 8 < 64) {
        pmask = ~0ull << (sh + 8);
        prefix = all_and & pmask;
    }
    for (;;) {  // uniform; at most eight digits
        const int2 pr = hist_pass([&](int j) {
            return in_bucket(j) && (k[j] & pmask) == prefix ? static_cast<int>((k[j] >> sh) & 255) : -1;
        });
        prefix |= static_cast<uint64_t>(pr.x) << sh;
        pmask |= 0xffull << sh;
        if (pr.y == 1 || sh == 0) {
            // one key, or equal keys: any key with the prefix
#pragma unroll
            for (int j = 0; j < HK; ++j)
                if (in_bucket(j) && (k[j] & pmask) == prefix) S.red[0] = k[j];
            __syncthreads();
            const uint64_t r = S.red[0];
            __syncthreads();
            return r;
        }
        sh = sh >= 8 ? sh - 8 : 0;  // the last digit may overlap bits fixed before
    }
}

// The common case of select_rank_key: one value histogram of 256 bins over
// [min Y, max Y] and a direct ranking of the keys in the bin that holds rank
// `want`, in three workgroup barriers.  The caller has cleared S.hist and
// S.ncand before an earlier barrier.  Returns the key and, through `above`,
// the count of keys strictly greater than it.  Tables with absent teams and
// bins of more than 64 keys take the general path (above = -1).
template <int HK>
__device__ uint64_t select_rank_key_fast(const uint64_t (&k)[HK], int M, int want, SelScratch& S, int& above) {
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    auto valid = [&](int j) { return j * kThreads + tid < M; };
    uint64_t kmin = ~0ull, kmax = 0;
#pragma unroll
    for (int j = 0; j < HK; ++j) {
        if (valid(j)) {
            kmin = min(kmin, k[j]);
            kmax = max(kmax, k[j]);
        }
    }
    kmin = wave_min64(kmin);
    kmax = wave_max64(kmax);
    if (lane == 0) {
        S.red[w] = kmin;
        S.cand[w] = kmax;
    }
    __syncthreads();
    kmin = S.red[0];
    kmax = S.cand[0];
#pragma unroll
    for (int v = 1; v < kWaves; ++v) {
        kmin = min(kmin, S.red[v]);
        kmax = max(kmax, S.cand[v]);
    }
    above = -1;
    if (kmin < order_key(kAbsentBelow)) {  // uniform
        __syncthreads();                   // red / cand are reused
        return select_rank_key<HK>(k, M, want, S);
    }
    const double ymin = key_value(kmin);
    const double range = key_value(kmax) - ymin;
    if (!(range > 0.0)) {  // uniform: every key equal
        above = 0;
        return kmin;
    }
    const double fs = 255.999 / range;
    int bin[HK];
#pragma unroll
    for (int j = 0; j < HK; ++j) {
        bin[j] = valid(j) ? static_cast<int>(fmin(255.0, (key_value(k[j]) - ymin) * fs)) : -1;
        if (bin[j] >= 0) atomicAdd(&S.hist[bin[j]], 1u);
    }
    __syncthreads();  // also orders the reads of red / cand above before the writes of cand below
    // every wave finds the same bin (no broadcast needed)
    int hi_cnt, cnt;
    const int sb = hist_select(S.hist, want, hi_cnt, cnt);
    if (cnt > kWave) {  // uniform
        __syncthreads();
        return select_rank_key<HK>(k, M, want, S);
    }
    const int rest = want - hi_cnt;
#pragma unroll
    for (int j = 0; j < HK; ++j)
        if (bin[j] == sb) S.cand[atomicAdd(&S.ncand, 1)] = k[j];
    __syncthreads();
    // every wave ranks the bin's keys (one per lane) and finds the same key
    const int n = S.ncand;
    const uint64_t mine = S.cand[min(lane, n - 1)];
    int gt = 0, ge = 0;
    for (int t = 0; t < n; ++t) {
        const uint64_t o = readlane(mine, t);
        gt += o > mine ? 1 : 0;
        ge += o >= mine ? 1 : 0;
    }
    const bool owner = lane < n && gt <= rest && rest < ge;
    const int src = __ffsll(static_cast<unsigned long long>(__ballot(owner))) - 1;
    above = hi_cnt + readlane(gt, src);
    return readlane(mine, src);
}

// Workspace views of a step.
struct Views {
    int* arrive;        // [BH] sampling workgroups that finished
    int* done;          // [BH, G] attention workgroups that published a head's state
    uint64_t* sbits;    // [B Hq, swords] sample bits per head, team order
    float* lc;          // [B Hq, M] log c of the sampled teams
    float* part;        // [BH, maxwp, G, d + 4] partial states
};

__device__ __forceinline__ Views views_of(const DecodeArgs& a) {
    const int BH = a.B * a.Hkv;
    Views v;
    int* ctr = reinterpret_cast<int*>(a.ws + a.lay.ctr);
    v.arrive = ctr;
    v.done = ctr + BH;
    v.sbits = reinterpret_cast<uint64_t*>(a.ws + a.lay.sbits);
    v.lc = reinterpret_cast<float*>(a.ws + a.lay.lc);
    v.part = reinterpret_cast<float*>(a.ws + a.lay.part);
    return v;
}

// A lane's EPL = d / 8 consecutive elements of a routing-key row (8 lanes per
// row) as LPL 16-byte words, and element e of them widened to fp32.
template <typename T, int D>
struct RepLanes {
    static constexpr int EPL = D / 8;
    static constexpr int LPL = EPL * static_cast<int>(sizeof(T)) / 16;
    static __device__ __forceinline__ float elem(const uint4 (&r)[LPL], int e) {
        if constexpr (sizeof(T) == 2) {
            const uint4 u = r[e >> 3];
            const int q = (e & 7) >> 1;
            const uint32_t wd = q == 0 ? u.x : q == 1 ? u.y : q == 2 ? u.z : u.w;
            return (e & 1) ? bf16hi(wd) : bf16lo(wd);
        } else {
            const uint4 u = r[e >> 2];
            const int q = e & 3;
            return __uint_as_float(q == 0 ? u.x : q == 1 ? u.y : q == 2 ? u.z : u.w);
        }
    }
};

// ---------------------------------------------------------------------------
// Phase A: query head j of pair p.  LDS: the head's routing logits (HK *
// kThreads doubles, in the first value-tile set), its Philox words or Gumbel
// variates (in the second) and the select scratch.
// ---------------------------------------------------------------------------
template <typename T, int D, int HK, bool FUSED>
__device__ void sample_head(const DecodeArgs& a, const Views& v, int p, int j, char* t0, char* t1, char* misc) {
    using RL = RepLanes<T, D>;
    constexpr int EPL = RL::EPL, LPL = RL::LPL;
    double* const s_dot = reinterpret_cast<double*>(t0);
    uint64_t* const s_word = reinterpret_cast<uint64_t*>(t1);
    SelScratch& S = *reinterpret_cast<SelScratch*>(misc);
    const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
    const int M = a.M, Kp = a.Kp;
    const int b = p / a.Hkv, kv = p - b * a.Hkv, hq = kv * a.G + j;
    const size_t bq = static_cast<size_t>(b) * a.Hq + hq;
    const size_t tb0 = static_cast<size_t>(p) * M;
    const T* reps = static_cast<const T*>(a.reps);
    const int nblk = (M + 3) / 4;

    // the select scratch starts empty (read only after the barriers below)
    if (tid < 64) reinterpret_cast<uint4*>(S.hist)[tid] = make_uint4(0, 0, 0, 0);
    if (tid == 0) S.ncand = 0;

    // The Philox block at counter (g / 4, h, b, step), key (seed, 0), holds
    // the words of teams 4 (g / 4) .. + 3.
    auto philox_words = [&](int bi) {
        const u64x4 r = philox4x64_10(static_cast<uint64_t>(bi), static_cast<uint64_t>(hq), static_cast<uint64_t>(b),
                                      a.step, a.seed, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (4 * bi + e < M) s_word[4 * bi + e] = r.v[e];
    };
    // the same block's four Gumbel variates, stored in place of its words
    auto philox_gumbels = [&](int bi) {
        const u64x4 r = philox4x64_10(static_cast<uint64_t>(bi), static_cast<uint64_t>(hq), static_cast<uint64_t>(b),
                                      a.step, a.seed, 0);
        double* const s_gum = reinterpret_cast<double*>(s_word);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (4 * bi + e < M) s_gum[4 * bi + e] = gumbel_of_word(r.v[e]);
    };
    // phi_g = log n_g + scale q.l_g for the team of octet `grp` in each
    // round (8 lanes per routing key, `per` keys per round): the dot product
    // in fp64 (exact products; two partial sums per lane, then the octet's
    // sum), stored by the octet's first lane
    // the query dims are loaded before the routing keys and widened after
    // them, so that the first round waits only for its own loads (the
    // hardware counts loads in issue order)
    auto query_load = [&](int sub, float (&qf)[EPL]) {
        const float* qrow = a.q + bq * D + sub * EPL;
#pragma unroll
        for (int e = 0; e < EPL; e += 4) {
            const float4 x = *reinterpret_cast<const float4*>(qrow + e);
            qf[e] = x.x;
            qf[e + 1] = x.y;
            qf[e + 2] = x.z;
            qf[e + 3] = x.w;
        }
    };
    auto query_dims = [&](const float (&qf)[EPL], double (&qd)[EPL]) {
#pragma unroll
        for (int e = 0; e < EPL; ++e) qd[e] = static_cast<double>(qf[e]);
    };
    auto load_batch = [&](auto& raw, auto& ln, int grp, int sub, int per, int r0) {
        constexpr int RB = sizeof(ln) / sizeof(double);
#pragma unroll
        for (int rr = 0; rr < RB; ++rr) {
            const int g = min((r0 + rr) * per + grp, M - 1);
            const uint4* src = reinterpret_cast<const uint4*>(reps + (tb0 + g) * D + sub * EPL);
#pragma unroll
            for (int l = 0; l < LPL; ++l) raw[rr][l] = load_stream(src + l);
            ln[rr] = a.log_n[tb0 + g];
        }
        // keep every load here, in this order (the compiler would otherwise
        // sink a round's loads into the block that uses them, behind the
        // waits of the rounds before it)
        asm volatile("" ::: "memory");
    };
    auto logits_batch = [&](const auto& raw, const auto& ln, const double (&qd)[EPL], int grp, int sub, int per,
                            int r0) {
        constexpr int RB = sizeof(ln) / sizeof(double);
#pragma unroll
        for (int rr = 0; rr < RB; ++rr) {
            if ((r0 + rr) * per < M) {  // uniform
                double acc0 = 0.0, acc1 = 0.0;
#pragma unroll
                for (int e = 0; e < EPL; e += 2) {
                    acc0 = fma(qd[e], static_cast<double>(RL::elem(raw[rr], e)), acc0);
                    acc1 = fma(qd[e + 1], static_cast<double>(RL::elem(raw[rr], e + 1)), acc1);
                }
                const double acc = row8_sum(acc0 + acc1);
                const int g = (r0 + rr) * per + grp;
                if (sub == 0 && g < M) {
                    const double ph = ln[rr] + a.scale * acc;
                    s_dot[g] = ph;
                    if (a.dbg_phi) a.dbg_phi[bq * M + g] = ph;
                }
            }
        }
    };
    if constexpr (HK == 1) {
        // M <= 512: two waves draw the Philox words and turn them into
        // Gumbel variates while the other six compute the logits, 48 teams
        // per round, every round's loads in flight together (two batches for
        // fp32 keys)
        constexpr int kPhiloxThreads = 2 * kWave;
        constexpr int kPer = (kThreads - kPhiloxThreads) / 8;
        constexpr int kRounds = (kThreads + kPer - 1) / kPer;
        constexpr int kBatch = LPL <= 2 ? kRounds : 24 / LPL;
        if (tid < kPhiloxThreads) {
            for (int bi = tid; bi < nblk; bi += kPhiloxThreads) philox_gumbels(bi);
        } else {
            const int lt = tid - kPhiloxThreads, grp = lt >> 3, sub = lt & 7;
            const int rounds = (M + kPer - 1) / kPer;
            uint4 raw[kBatch][LPL];
            double ln[kBatch], qd[EPL];
            float qf[EPL];
            query_load(sub, qf);
            load_batch(raw, ln, grp, sub, kPer, 0);
            query_dims(qf, qd);
            logits_batch(raw, ln, qd, grp, sub, kPer, 0);
            for (int r0 = kBatch; r0 < rounds; r0 += kBatch) {
                load_batch(raw, ln, grp, sub, kPer, r0);
                logits_batch(raw, ln, qd, grp, sub, kPer, r0);
            }
        }
    } else {
        // every thread: the Philox words while the first keys load, then the
        // logits with two batches of four rounds in flight
        constexpr int RB = 4;
        const int grp = tid >> 3, sub = tid & 7, per = kThreads / 8;
        const int rounds = (M + per - 1) / per;
        uint4 ra[RB][LPL], rb[RB][LPL];
        double la[RB], lb[RB], qd[EPL];
        float qf[EPL];
        query_load(sub, qf);
        load_batch(ra, la, grp, sub, per, 0);
        query_dims(qf, qd);
        for (int bi = tid; bi < nblk; bi += kThreads) philox_words(bi);
        for (int r0 = 0; r0 < rounds; r0 += 2 * RB) {
            if (r0 + RB < rounds) load_batch(rb, lb, grp, sub, per, r0 + RB);
            logits_batch(ra, la, qd, grp, sub, per, r0);
            if (r0 + 2 * RB < rounds) load_batch(ra, la, grp, sub, per, r0 + 2 * RB);
            if (r0 + RB < rounds) logits_batch(rb, lb, qd, grp, sub, per, r0 + RB);
        }
    }
    __syncthreads();

    // the perturbed score Y_g = phi_g + G_g as an order-preserving key: key
    // jj of this thread is team jj * kThreads + tid
    auto valid = [&](int jj) { return jj * kThreads + tid < M; };
    double phi[HK];
    uint64_t k[HK];
#pragma unroll
    for (int jj = 0; jj < HK; ++jj) {
        const int g = jj * kThreads + tid;
        phi[jj] = 0.0;
        k[jj] = 0;
        if (g < M) {
            phi[jj] = s_dot[g];
            const double gm = HK == 1 ? reinterpret_cast<const double*>(s_word)[g] : gumbel_of_word(s_word[g]);
            const double y = phi[jj] + gm;
            k[jj] = order_key(y);
            if (a.dbg_Y) a.dbg_Y[bq * M + g] = y;
        }
    }

    // tau: the key of rank Kp (0-based, descending)
    int above;
    const uint64_t tkey = select_rank_key_fast<HK>(k, M, Kp, S, above);
    const double tau = key_value(tkey);
    if (above < 0) {  // uniform: the general select does not count
        int x[1] = {0};
#pragma unroll
        for (int jj = 0; jj < HK; ++jj) x[0] += (valid(jj) && k[jj] > tkey) ? 1 : 0;
        int ex[1], tot[1];
        block_scan<1>(x, ex, tot, S.w);
        above = tot[0];
    }

    // the sample: the keys above tau's, and the first need_ties keys equal to
    // it in team order (exactly equal perturbed scores)
    const int need_ties = Kp - above;
    const int nwords = (M + kWave - 1) / kWave;
#pragma unroll
    for (int jj = 0; jj < HK; ++jj) {
        const bool vj = valid(jj);
        const uint64_t sb = __ballot(vj && k[jj] > tkey);
        const uint64_t tb = need_ties > 0 ? __ballot(vj && k[jj] == tkey) : 0;
        if (lane == 0 && jj * kWaves + w < kSelWords) {
            S.sel[jj * kWaves + w] = sb;
            S.tie[jj * kWaves + w] = tb;
        }
    }
    __syncthreads();
    if (need_ties > 0) {  // uniform
        const int tc = tid < nwords ? static_cast<int>(__popcll(S.tie[tid])) : 0;
        const int x[1] = {tc};
        int ex[1], tot[1];
        block_scan<1>(x, ex, tot, S.w);
        if (tid < nwords && ex[0] < need_ties) {
            uint64_t t = S.tie[tid];
            for (int left = need_ties - ex[0]; left > 0 && t; --left) {
                const uint64_t lowest = t & (~t + 1);
                S.sel[tid] |= lowest;
                t ^= lowest;
            }
        }
        __syncthreads();
    }

    // log c of every sampled team, by the thread that holds its key (and,
    // for the diagnostics, its rank in the head's ascending sample); thread
    // t < nwords publishes sample word t (teams 64 t ..)
    const bool ranks = a.dbg_sel || a.dbg_logc;
#pragma unroll
    for (int jj = 0; jj < HK; ++jj) {
        const int g = jj * kThreads + tid;
        const int wd = jj * kWaves + w;
        const bool taken = valid(jj) && (k[jj] > tkey || (need_ties > 0 && k[jj] == tkey &&
                                                          ((S.sel[wd] >> lane) & 1ull)));
        if (taken) {
            const float lcv = log_inclusion(static_cast<float>(phi[jj] - tau));
            if (FUSED)
                store_f32_coherent(v.lc + bq * M + g, lcv);
            else
                v.lc[bq * M + g] = lcv;
            if (ranks) {
                int rank = static_cast<int>(__popcll(S.sel[wd] & ((1ull << lane) - 1ull)));
                for (int x = 0; x < wd; ++x) rank += static_cast<int>(__popcll(S.sel[x]));
                if (rank < Kp) {  // always: exactly Kp teams are sampled
                    if (a.dbg_sel) a.dbg_sel[bq * Kp + rank] = g;
                    if (a.dbg_logc) a.dbg_logc[bq * Kp + rank] = lcv;
                }
            }
        }
    }
    if (tid < nwords) {
        const uint64_t word = S.sel[tid];
        if (FUSED)
            store_u64_coherent(v.sbits + bq * a.lay.swords + tid, word);
        else
            v.sbits[bq * a.lay.swords + tid] = word;
    }
    if (tid == 0 && a.dbg_tau) a.dbg_tau[bq] = tau;
    if (FUSED) {
        // arrival, once every store above is complete
        drain_and_sync();
        if (tid == 0) atomicAdd(&v.arrive[p], 1);
    }
    __syncthreads();  // the LDS is reused by the next task
}

// Scores of one 16-row tile.  Lane l = 16 c + j feeds row j of the tile and
// holds head 4 c + r of row j in accumulator register r (M rows 8 .. 15 repeat
// heads 0 .. 7, so lane groups 2 and 3 repeat the states of groups 0 and 1).
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

// Value sum of a 32-row step on the matrix cores (bf16 values):
// O[h][dim] += sum_row P[h][row] V[row][dim] as v_mfma_f32_16x16x32_bf16
// with the step's rows as the K dimension, one product per 16 dims.
//   A (probabilities): M row i < 8 holds the bf16 high part of head i, row
//     i + 8 the bf16 low part (p - high), so a product carries p to 16
//     significant bits; the two halves of the accumulator are added when
//     the state is written out.
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

// d / 16 consecutive value dims of a row for one of 16 lanes (fp32 rows).
template <int VPL>
struct RowChunkF;

template <>
struct RowChunkF<8> {
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
struct RowChunkF<4> {
    using raw = float4;
    static __device__ __forceinline__ raw load(const float* p) { return load_stream_f(p); }
    static __device__ __forceinline__ void unpack(const raw& r, float* x) {
        x[0] = r.x; x[1] = r.y; x[2] = r.z; x[3] = r.w;
    }
};

// One attention unit of pair p: its rows and the query heads that read them.
template <typename T>
struct Unit {
    const T* Kb;
    const T* Vb;
    int rows;
    int hmask;
    int g;  // the unit's team, -1 for suffix and dense rows
};

// The read plan of one pass in LDS: per union team of the pass (in team
// order) its first unit, packed begin row, size and (team | head mask << 16);
// and, when the pass has at most kPlanUnits units, the union slot of every
// unit.
struct PlanLds {
    int4 rec[kPlanRecs];
    unsigned short u2t[kPlanUnits];
    int w[3 * kWaves];
    int flag[4];
};

// The records of one plan pass from this thread's teams g0 .. g0 + PT - 1:
// their head masks hm (cleared here beyond the table), sizes and packed
// begins.  Returns (union teams, units, rows) of the pass (rows only when
// `rows`, else 0); the records are in place on return.  The union teams
// (< 4096) and units (< 2^20) of the pass are scanned as one packed count.
template <int PT>
__device__ int3 plan_records(int g0, int M, int (&hm)[PT], const int (&sz)[PT], const int (&bg)[PT], PlanLds& P,
                             bool rows = true) {
    const int lane = lane_id(), w = wave_id();
    int nck[PT], lf = 0, lnc = 0, lrows = 0;
#pragma unroll
    for (int k = 0; k < PT; ++k) {
        if (g0 + k >= M) hm[k] = 0;
        nck[k] = hm[k] ? chunk_count(sz[k]) : 0;
        lf += hm[k] ? 1 : 0;
        lnc += nck[k];
        lrows += hm[k] ? sz[k] : 0;
    }
    // exclusive prefix over the workgroup: wave scans, then the waves' totals
    const int x0 = lf | (lnc << 12);
    const int inc0 = wave_incl_scan(x0);
    const int inc1 = rows ? wave_incl_scan(lrows) : 0;
    if (lane == kWave - 1) {
        P.w[w] = inc0;
        P.w[kWaves + w] = inc1;
    }
    __syncthreads();
    int pre0 = 0, tot0 = 0, tot1 = 0;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) {
        const int y = P.w[v];
        pre0 += v < w ? y : 0;
        tot0 += y;
        tot1 += rows ? P.w[kWaves + v] : 0;
    }
    const int ex0 = pre0 + inc0 - x0;
    const int totf = tot0 & 0xfff, totu = tot0 >> 12;
    const bool table = totu <= kPlanUnits;  // uniform
    int slot = ex0 & 0xfff, ust = ex0 >> 12;
#pragma unroll
    for (int k = 0; k < PT; ++k) {
        if (hm[k]) {
            if (slot < kPlanRecs) P.rec[slot] = make_int4(ust, bg[k], sz[k], (g0 + k) | (hm[k] << 16));
            if (table)
                for (int c = 0; c < nck[k]; ++c) P.u2t[ust + c] = static_cast<unsigned short>(slot);
            ++slot;
            ust += nck[k];
        }
    }
    __syncthreads();
    return make_int3(totf, totu, tot1);
}

// Pass `base` of pair p's plan: the teams base + t PT + k of thread t (their
// sizes and begins sz / bg loaded by the caller), head masks from the heads'
// sample words in the workspace.
template <int PT, bool COHERENT>
__device__ int3 plan_pass(const DecodeArgs& a, const Views& v, int p, int base, const int (&sz)[PT], const int (&bg)[PT],
                          PlanLds& P) {
    const int tid = threadIdx.x, G = a.G, M = a.M;
    const int b = p / a.Hkv, kv = p - b * a.Hkv;
    const size_t hq0 = static_cast<size_t>(b) * a.Hq + kv * G;
    // the heads' sample words that hold this thread's teams (PT divides 64)
    static_assert(64 % PT == 0, "a thread's teams share one sample word");
    const int g0 = base + tid * PT;
    int hm[PT];
#pragma unroll
    for (int k = 0; k < PT; ++k) hm[k] = 0;
    if (g0 < M) {
        for (int h = 0; h < G; ++h) {
            const uint64_t* wp = v.sbits + (hq0 + h) * a.lay.swords + (g0 >> 6);
            const uint64_t wd = COHERENT ? load_u64_coherent(wp) : *wp;
#pragma unroll
            for (int k = 0; k < PT; ++k) hm[k] |= static_cast<int>((wd >> ((g0 + k) & 63)) & 1ull) << h;
        }
    }
    return plan_records<PT>(g0, M, hm, sz, bg, P);
}

// Unit i (0-based within the pass) of a pass with `teams` union teams and
// `units` units: its rows, heads and team, clamped to the packed rows.
template <typename T>
__device__ __forceinline__ Unit<T> plan_unit(const DecodeArgs& a, const PlanLds& P, int p, int i, int teams,
                                             int units) {
    int sl;
    if (units <= kPlanUnits) {
        sl = P.u2t[min(i, kPlanUnits - 1)];
    } else {  // the last record whose first unit is at or before i
        int lo = 0, hi = min(teams, kPlanRecs) - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (P.rec[mid].x <= i)
                lo = mid;
            else
                hi = mid - 1;
        }
        sl = lo;
    }
    const int4 r = P.rec[min(sl, kPlanRecs - 1)];
    const int first = uni(r.x), begin0 = uni(r.y), size = uni(r.z), gm = uni(r.w);
    const int pc = i - first;
    Unit<T> U;
    U.rows = min(max(size - pc * kUnitRows, 1), min(kUnitRows, max(a.N, 1)));
    const int begin = min(max(begin0 + pc * kUnitRows, 0), max(a.N - U.rows, 0));
    U.hmask = (gm >> 16) & ((1 << a.G) - 1);
    U.g = min(gm & 0xffff, a.M - 1);
    const size_t o = (static_cast<size_t>(p) * a.N + begin) * a.d;
    U.Kb = static_cast<const T*>(a.K) + o;
    U.Vb = static_cast<const T*>(a.V) + o;
    return U;
}

// Suffix unit u, or dense prompt unit u - nsuf.
template <typename T>
__device__ __forceinline__ Unit<T> index_unit(const DecodeArgs& a, int p, int nsuf, int u) {
    Unit<T> U;
    U.hmask = (1 << a.G) - 1;
    U.g = -1;
    if (u < nsuf) {
        const int begin = u * kUnitRows;
        U.rows = max(1, min(kUnitRows, a.T - begin));
        const size_t o = (static_cast<size_t>(p) * a.sstride + begin) * a.d;
        U.Kb = static_cast<const T*>(a.sK) + o;
        U.Vb = static_cast<const T*>(a.sV) + o;
    } else {
        const int begin = (u - nsuf) * kUnitRows;
        U.rows = max(1, min(kUnitRows, a.N - begin));
        const size_t o = (static_cast<size_t>(p) * a.N + begin) * a.d;
        U.Kb = static_cast<const T*>(a.K) + o;
        U.Vb = static_cast<const T*>(a.V) + o;
    }
    return U;
}

// Canonical per-wave state in LDS: [wave][head][d + 4] floats, the value sum
// then (maximum, mass).
__device__ __forceinline__ float* wave_state(char* lds, int wv, int h, int D) {
    return reinterpret_cast<float*>(lds) + (static_cast<size_t>(wv) * kMaxGroup + h) * state_stride(D);
}

// The pair's units as the waves see them: the suffix units and each pass of
// the plan (a workgroup-wide step) with its units.  `run(lo, hi, unit, rev)`
// walks the wave's units u in [lo, hi), u == s (mod waves of the pair), with
// unit(u) giving each one; s is the wave's index among the pair's waves, or
// that index counted from the last wave when `rev`.  In the single launch the
// suffix units go to the pair's last waves while the samples are drawn; in
// the split launch (the samples are there when it starts) they join the
// first plan pass's units, so that they neither hold up a workgroup's plan
// (its passes wait for all its waves) nor follow a wave's union units.
template <typename T, bool DENSE, bool FUSED, int PT, typename Run>
__device__ __forceinline__ bool walk_units(const DecodeArgs& a, const Views& v, int p, int iw, char* plan_lds,
                                           Run&& run) {
    PlanLds& P = *reinterpret_cast<PlanLds*>(plan_lds);
    const int nsuf = (a.T + kUnitRows - 1) / kUnitRows;
    auto by_index = [&](int u) { return index_unit<T>(a, p, nsuf, u); };
    if (DENSE) {
        run(0, nsuf, by_index, false);
        run(nsuf, nsuf + (a.N + kUnitRows - 1) / kUnitRows, by_index, false);
        return true;
    }
    if (FUSED) run(0, nsuf, by_index, true);
    const int tid = threadIdx.x, M = a.M;
    const size_t tb0 = static_cast<size_t>(p) * M;
    int sz[PT], bg[PT];
    auto fetch = [&](int base) {
#pragma unroll
        for (int k = 0; k < PT; ++k) {
            const int g = min(base + tid * PT + k, M - 1);
            sz[k] = a.team_size[tb0 + g];
            bg[k] = a.team_begin[tb0 + g];
        }
    };
    fetch(0);
    bool ok = true;
    if (FUSED) ok = wait_count(v.arrive + p, a.G, P.flag);  // the pair's samples are published
    int run_u = nsuf, run_teams = 0, run_rows = 0;
    if (ok) {
        for (int base = 0; base < M; base += kThreads * PT) {
            if (base > 0) fetch(base);
            const int3 t = plan_pass<PT, FUSED>(a, v, p, base, sz, bg, P);
            // the split launch reads the suffix units in the first pass's run
            // (units 0 .. nsuf - 1), so that no wave reads them after its
            // union units
            const int lo = (!FUSED && base == 0) ? 0 : run_u, first = run_u;
            run(lo, run_u + t.y,
                [&](int u) { return u < first ? by_index(u) : plan_unit<T>(a, P, p, u - first, t.x, t.y); }, false);
            run_u += t.y;
            run_teams += t.x;
            run_rows += t.z;
            if (base + kThreads * PT < M) __syncthreads();  // the records are rewritten by the next pass
        }
    }
    if (iw == 0 && tid == 0) {
        if (a.dbg_uteams) a.dbg_uteams[p] = run_teams;
        if (a.dbg_urows) a.dbg_urows[p] = run_rows;
    }
    return ok;
}

// ---------------------------------------------------------------------------
// Single-launch step: the selection of every head of the pair in LDS.
// ---------------------------------------------------------------------------

// The pair's selection in LDS: per team the mask of the heads that sampled
// it, and per head tau's order key -- its high half, and either the team
// whose published low half completes it (tau_g >= 0) or the low half itself
// (tau_g < 0); `ok` is cleared when a head's published scores did not all
// arrive.
struct StepSel {
    uint32_t hm[kStepMaxTeams / 4];  // byte g % 4 of word g / 4: the heads that sampled team g
    uint32_t tau_hi[kMaxGroup];
    int tau_g[kMaxGroup];
    uint32_t tau_lo[kMaxGroup];
    int ok;
    int pad[3];
};

// Where a unit of the step finds its corrections: the pair's exchange words
// and the call's tag.
struct StepCtx {
    const uint64_t* xk;  // the pair's [G, 3, M] exchange words
    uint32_t tag;
    const float* q;      // the pair's G query rows staged in LDS (sampled steps), else null
};

// The correction of a unit for one lane's head in flight: phi of the unit's
// team and the low half of tau's key, as loaded (need = 0: no correction).
struct CorrWords {
    u32x2v ph, tl;
    int need, g;
};

// The pair's units for the single-launch step: as walk_units in the split
// launch, with the heads' samples taken from LDS and the first pass's team
// sizes and begins from the LDS copy s_tab (size, begin per team) made when
// the step started (later passes read the table in memory).
template <typename T, bool DENSE, int PT, typename Run>
__device__ __forceinline__ bool step_walk_units(const DecodeArgs& a, int p, int iw, char* plan_lds, const StepSel* SS,
                                                const int* s_tab, Run&& run) {
    PlanLds& P = *reinterpret_cast<PlanLds*>(plan_lds);
    const int nsuf = (a.T + kUnitRows - 1) / kUnitRows;
    auto by_index = [&](int u) { return index_unit<T>(a, p, nsuf, u); };
    if (DENSE) {
        run(0, nsuf, by_index, false);
        run(nsuf, nsuf + (a.N + kUnitRows - 1) / kUnitRows, by_index, false);
        return true;
    }
    const int tid = threadIdx.x, M = a.M;
    const size_t tb0 = static_cast<size_t>(p) * M;
    int run_u = nsuf, run_teams = 0, run_rows = 0;
    for (int base = 0; base < M; base += kThreads * PT) {
        const int g0 = base + tid * PT;
        int sz[PT], bg[PT], hm[PT];
#pragma unroll
        for (int k = 0; k < PT; ++k) {
            const int g = min(g0 + k, M - 1);
            if (base == 0) {
                sz[k] = s_tab[2 * g];
                bg[k] = s_tab[2 * g + 1];
            } else {
                sz[k] = a.team_size[tb0 + g];
                bg[k] = a.team_begin[tb0 + g];
            }
            hm[k] = 0;
        }
        if (g0 < M) {
#pragma unroll
            for (int k = 0; k < PT; ++k) {
                const int g = min(g0 + k, M - 1);
                hm[k] = static_cast<int>((SS->hm[g >> 2] >> (8 * (g & 3))) & 0xffu);
            }
        }
        const int3 t = plan_records<PT>(g0, M, hm, sz, bg, P, a.dbg_urows != nullptr);
        // the suffix units come first in the first pass's run
        const int lo = base == 0 ? 0 : run_u, first = run_u;
        run(lo, run_u + t.y,
            [&](int u) { return u < first ? by_index(u) : plan_unit<T>(a, P, p, u - first, t.x, t.y); }, false);
        run_u += t.y;
        run_teams += t.x;
        run_rows += t.z;
        if (base + kThreads * PT < M) __syncthreads();  // the records are rewritten by the next pass
    }
    if (iw == 0 && tid == 0) {
        if (a.dbg_uteams) a.dbg_uteams[p] = run_teams;
        if (a.dbg_urows) a.dbg_urows[p] = run_rows;
    }
    return SS->ok != 0;
}

// ---------------------------------------------------------------------------
// Phase B for bf16 rows.
// ---------------------------------------------------------------------------
template <int D, bool DENSE, bool FUSED, int PT, bool STEP = false>
__device__ void attend_mfma(const DecodeArgs& a, const Views& v, int p, int iw, int nwp, char* t0, char* t1,
                            char* misc, const StepSel* SS = nullptr, const int* s_tab = nullptr,
                            const StepCtx* sc = nullptr) {
    using QKT = QK<bf16_t, D>;
    using VT = VTile<D>;
    constexpr int NF = QKT::KB;         // K fragments per 16-row tile
    constexpr int NB = VT::NB;
    constexpr int SPR = D / 8;          // 16-byte segments per row
    constexpr int RPI = kWave / SPR;    // rows per DMA instruction (1 KB)
    constexpr int NDMA = 32 / RPI;      // DMA instructions per step
    static_assert(RPI * SPR == kWave && NDMA * RPI == 32, "a step's tile is whole 1 KB DMA blocks");
    static_assert(kUnitRows == 32, "one unit is one 32-row step");
    constexpr int kNT = 2;              // cache policy of the value copies: streaming
    const int lane = lane_id();
    const int wv = __builtin_amdgcn_readfirstlane(wave_id());  // uniform: keeps the tile bases scalar
    const int c = lane >> 4, j16 = lane & 15;
    const int hsel = 4 * (c & 1);  // first head of this lane's registers
    // the two value-tile sets are distinct LDS objects, so that the compiler
    // can tell the copies into one set from the reads of the other
    char* const tile0 = t0 + wv * VT::kBytes;
    char* const tile1 = t1 + wv * VT::kBytes;
    float4(*const ptile)[8] = reinterpret_cast<float4(*)[8]>(misc + wv * 1024);
    char* const plan_lds = misc + kWaves * 1024;
    const int G = a.G;
    const int b = p / a.Hkv, kv = p - b * a.Hkv;
    const size_t hq0 = static_cast<size_t>(b) * a.Hq + kv * G;
    const int NW = nwp * kWaves;
    const int gwp = wv * nwp + iw;  // this wave's index among the pair's waves

    QKT qk;
    bool qready = false;
    auto ensure_q = [&]() {
        if (!qready) {  // uniform
            const int h = j16 & 7;
            const int hc = h < G ? h : 0;
            if constexpr (STEP && !DENSE)
                qk.load_q(sc->q + hc * D, h < G ? a.scale_log2 : 0.f, c);
            else
                qk.load_q(a.q + (hq0 + hc) * D, h < G ? a.scale_log2 : 0.f, c);
            qready = true;
        }
    };
    float m[4], l[4];
    f32x4 oacc[NB];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        m[r] = kNeg;
        l[r] = 0.f;
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) oacc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // V copies, then K loads, of unit U into `tile` / kf.  The K loads go
    // last, so that waiting for them waits for the whole unit.  A stand-in
    // issue (real = false) has every lane fetch the unit's first 16 bytes:
    // one cache line per instruction.
    auto issue = [&](const Unit<bf16_t>& U, char* tile, typename QKT::frag(&kf)[2][NF], bool real) {
        const int ls = real ? lane : 0;
#pragma unroll
        for (int jd = 0; jd < NDMA; ++jd) {
            const int row = real ? RPI * jd + lane / SPR : 0;
            const int seg = real ? (ls % SPR) ^ (2 * VT::swz(row)) : 0;
            const bf16_t* src = U.Vb + static_cast<size_t>(min(row, U.rows - 1)) * D + 8 * seg;
            __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)(tile + 1024 * jd), 16, 0,
                                             kNT);
        }
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const bf16_t* row = U.Kb + (real ? static_cast<size_t>(min(16 * kk + j16, U.rows - 1)) * D : 0);
            QKT::load_k(row, real ? c : 0, kf[kk]);
        }
    };
    // log c of the unit's team for head lane % 8 (0 where that head did not
    // sample it, or for suffix and dense rows); a step spreads the values to
    // the lanes that hold each head's state
    // In the single-launch step the corrections are read from the exchange
    // words with the unit's rows (phi of the unit's team and the low half of
    // tau's key for head lane % 8) and resolved to log c when the unit
    // computes.
    const __amdgpu_buffer_rsrc_t rx =
        coherent_rsrc(STEP && !DENSE ? static_cast<const void*>(sc->xk) : static_cast<const void*>(a.q),
                      STEP && !DENSE ? static_cast<uint32_t>(a.G) * a.M * 24u : 0u);
    auto corrections = [&](const Unit<bf16_t>& U) {
        const int h = lane & 7;
        if constexpr (STEP) {
            CorrWords c;
            c.need = 0;
            c.g = max(U.g, 0);
            c.ph = u32x2v{0u, 0u};
            c.tl = u32x2v{0u, 0u};
            if (!DENSE && U.g >= 0 && ((U.hmask >> h) & 1)) {
                c.need = 1;
                const uint32_t hb = static_cast<uint32_t>(h) * 24u * a.M;
                c.ph = load8_coherent(rx, hb + 16u * a.M + 8u * U.g);
                const int tg = SS->tau_g[h];
                if (tg >= 0)
                    c.tl = load8_coherent(rx, hb + 8u * a.M + 8u * tg);
                else
                    c.tl = u32x2v{SS->tau_lo[h], sc->tag};
            }
            return c;
        } else {
            float cr = 0.f;
            if (!DENSE && U.g >= 0 && ((U.hmask >> h) & 1)) {
                const float* src = v.lc + (hq0 + h) * a.M + U.g;
                cr = FUSED ? load_f32_coherent(src) : *src;
            }
            return cr;
        }
    };
    // log c of a correction in flight (eq. method-inclusion); a word that
    // does not yet carry the tag is read again
    auto corr_value = [&](const auto& c) -> float {
        if constexpr (STEP) {
            if (!c.need) return 0.f;
            const int h = lane & 7;
            u32x2v ph = c.ph, tl = c.tl;
            if (ph.y != sc->tag || tl.y != sc->tag) {
                const uint32_t hb = static_cast<uint32_t>(h) * 24u * a.M;
                const int tg = max(SS->tau_g[h], 0);
                for (int it = 0; it < kSpinLimit && (ph.y != sc->tag || tl.y != sc->tag); ++it) {
                    __builtin_amdgcn_s_sleep(1);
                    if (ph.y != sc->tag) ph = load8_coherent(rx, hb + 16u * a.M + 8u * static_cast<uint32_t>(c.g));
                    if (tl.y != sc->tag) tl = load8_coherent(rx, hb + 8u * a.M + 8u * tg);
                }
            }
            const double tau = key_value((static_cast<uint64_t>(SS->tau_hi[h]) << 32) | tl.x);
            return log_inclusion(static_cast<float>(static_cast<double>(__uint_as_float(ph.x)) - tau));
        } else {
            return c;
        }
    };

    typename QKT::frag kf0[2][NF], kf1[2][NF];
    // The wave's units u in [lo, hi), u == gwp (mod NW), one 32-row step each.
    // A unit's corrections go out first, then its rows; its log c is formed
    // while the rows fly (the wait for the corrections leaves the rows in
    // flight).  A step waits for its own rows, issues the next unit's loads
    // into the other buffers and computes while those fly; the two buffer
    // sets alternate between two inlined copies of the step, so that each
    // copy names its registers statically.  In the loop every step issues
    // loads whether or not a next unit exists (then a stand-in issue), so
    // that the loop's register needs are the same on every path; a wave
    // with a single unit takes a copy of the step of its own that issues
    // nothing.
    auto run = [&](int lo_u, int hi_u, auto&& unit, bool rev) {
        const int gs = rev ? NW - 1 - gwp : gwp;
        int u = lo_u + (((gs - lo_u) % NW) + NW) % NW;
        if (u >= hi_u) return;  // uniform
        Unit<bf16_t> cur = unit(u);
        auto ccr = corrections(cur);
        issue(cur, tile0, kf0, true);
        ensure_q();
        float cv = corr_value(ccr);
        auto step = [&](char* tile, typename QKT::frag(&kf)[2][NF], char* ntile, typename QKT::frag(&nkf)[2][NF],
                        auto last) {
            constexpr bool has_next = !decltype(last)::value;
            // this step's rows: the K fragments were issued last, so the
            // wait for them covers the value copies too
            asm volatile("" ::"v"(kf[1][NF - 1].w) : "memory");
            float bias[4];
            bool on[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                bias[r] = -__shfl(cv, hsel + r) * kLog2e;
                on[r] = ((cur.hmask >> (hsel + r)) & 1) != 0;
            }
            const bool more = has_next && u + NW < hi_u;
            Unit<bf16_t> nxt = cur;
            auto ncr = ccr;
            if constexpr (has_next) {
                nxt = more ? unit(u + NW) : cur;
                ncr = corrections(nxt);
                issue(nxt, ntile, nkf, more);
            }

            // scores and the online softmax over the step's 32 rows
            const f32x4 s0 = qk.scores(kf[0]);
            const f32x4 s1 = qk.scores(kf[1]);
            const bool live0 = j16 < cur.rows, live1 = 16 + j16 < cur.rows;
            float aa[4], p0[4], p1[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const bool v0 = live0 && on[r], v1 = live1 && on[r];
                const float x0 = v0 ? s0[r] + bias[r] : kNeg;
                const float x1 = v1 ? s1[r] + bias[r] : kNeg;
                const float mn = fmaxf(m[r], row16_max(fmaxf(x0, x1)));
                aa[r] = fast_exp2(m[r] - mn);
                p0[r] = v0 ? fast_exp2(x0 - mn) : 0.f;
                p1[r] = v1 ? fast_exp2(x1 - mn) : 0.f;
                l[r] = l[r] * aa[r] + row16_sum(p0[r] + p1[r]);
                m[r] = mn;
            }
            lds_order();  // the previous step's reads of ptile come first
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
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int r = 0; r < 4; ++r) oacc[nb][r] *= aa[r];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                oacc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, VT::operand(tile, nb, lane), oacc[nb], 0, 0, 0);
            if constexpr (has_next) {
                if (!more) return false;
                // the next unit's log c: its corrections were issued before
                // its rows, which stay in flight
                cv = corr_value(ncr);
                u += NW;
                cur = nxt;
                ccr = ncr;
            }
            return true;
        };
        if (u + NW >= hi_u) {  // uniform: a single unit
            step(tile0, kf0, tile1, kf1, std::true_type{});
        } else {
            for (;;) {
                if (!step(tile0, kf0, tile1, kf1, std::false_type{})) break;
                if (!step(tile1, kf1, tile0, kf0, std::false_type{})) break;
            }
        }
        // nothing is left in flight once the last step has waited for its
        // rows; the drain is kept for the tiles' reuse after the walk
        __builtin_amdgcn_s_waitcnt(0);
    };

    bool ok;
    if constexpr (STEP)
        ok = step_walk_units<bf16_t, DENSE, PT>(a, p, iw, plan_lds, SS, s_tab, run);
    else
        ok = walk_units<bf16_t, DENSE, FUSED, PT>(a, v, p, iw, plan_lds, run);

    // the wave's state per head, in canonical form, over the (now free) tiles
    char* const lds = t0;
    __syncthreads();
    {
        const bool lower = c < 2;
        const int dim0 = (lower ? 0 : D / 2) + j16;
#pragma unroll
        for (int nb = 0; nb < NB / 2; ++nb) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float keep = lower ? oacc[nb][r] : oacc[nb + NB / 2][r];
                const float send = lower ? oacc[nb + NB / 2][r] : oacc[nb][r];
                const float x = keep + __shfl_xor(send, 32);
                wave_state(lds, wv, hsel + r, D)[dim0 + 16 * nb] = x;
            }
        }
        if (c < 2 && j16 == 0) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float* st = wave_state(lds, wv, hsel + r, D);
                st[D] = ok ? m[r] : __builtin_nanf("");
                st[D + 1] = l[r];
            }
        }
    }
}

// Phase B for fp32 rows (the small fp32 workloads): scores on the matrix cores
// as for bf16; the value sums on the vector ALUs with 16 lanes per row, each
// owning d / 16 dims of every head, and the probabilities broadcast through
// LDS.  No software pipelining.
template <int D, bool DENSE, int PT>
__device__ void attend_f32(const DecodeArgs& a, const Views& v, int p, int iw, int nwp, char* t0, char* misc) {
    using QKT = QK<float, D>;
    constexpr int NF = QKT::KB / 4;
    constexpr int VPL = D / 16;
    using VC = RowChunkF<VPL>;
    constexpr int GT = kMaxGroup;
    const int lane = lane_id();
    const int wv = __builtin_amdgcn_readfirstlane(wave_id());
    const int c = lane >> 4, j16 = lane & 15;
    float4(*const s_p)[2] = reinterpret_cast<float4(*)[2]>(misc + wv * 640);       // [16][2]
    float4* const s_a = reinterpret_cast<float4*>(misc + wv * 640 + 512);            // [2]
    char* const plan_lds = misc + kWaves * 1024;
    char* const lds = t0;  // the wave states
    const int G = a.G;
    const int b = p / a.Hkv, kv = p - b * a.Hkv;
    const size_t hq0 = static_cast<size_t>(b) * a.Hq + kv * G;
    const int NW = nwp * kWaves;
    const int gwp = wv * nwp + iw;

    QKT qk;
    {
        const int h = j16 & 7;
        qk.load_q(a.q + (hq0 + (h < G ? h : 0)) * D, h < G ? a.scale_log2 : 0.f, c);
    }
    float m[4], l[4], acc[GT][VPL];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        m[r] = kNeg;
        l[r] = 0.f;
    }
#pragma unroll
    for (int h = 0; h < GT; ++h)
#pragma unroll
        for (int e = 0; e < VPL; ++e) acc[h][e] = 0.f;

    auto run = [&](int lo_u, int hi_u, auto&& unit, bool rev) {
        const int gs = rev ? NW - 1 - gwp : gwp;
        for (int u = lo_u + (((gs - lo_u) % NW) + NW) % NW; u < hi_u; u += NW) {
            const Unit<float> U = unit(u);
            float bias[4];
            bool on[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int h = 4 * (c & 1) + r;
                on[r] = c < 2 && ((U.hmask >> h) & 1) != 0;
                bias[r] = (!DENSE && U.g >= 0 && on[r]) ? -v.lc[(hq0 + h) * a.M + U.g] * kLog2e : 0.f;
            }
            typename QKT::frag kf[2][NF];
            typename VC::raw vr[2][4];
            const bool has1 = 16 < U.rows;
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const int t0 = 16 * k;
                qk.load_k(U.Kb + static_cast<size_t>(min(t0 + j16, U.rows - 1)) * D, c, kf[k]);
#pragma unroll
                for (int kk = 0; kk < 4; ++kk)
                    vr[k][kk] = VC::load(U.Vb + static_cast<size_t>(min(t0 + 4 * kk + c, U.rows - 1)) * D + VPL * j16);
            }
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                if (k == 1 && !has1) continue;  // uniform
                const int t0 = 16 * k;
                const f32x4 sc = qk.scores(kf[k]);
                const bool live = t0 + j16 < U.rows;
                float aa[4], pp[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const bool vr_ = live && on[r];
                    const float x = vr_ ? sc[r] + bias[r] : kNeg;
                    const float mn = fmaxf(m[r], row16_max(x));
                    aa[r] = fast_exp2(m[r] - mn);
                    pp[r] = vr_ ? fast_exp2(x - mn) : 0.f;
                    l[r] = l[r] * aa[r] + row16_sum(pp[r]);
                    m[r] = mn;
                }
                if (c < 2) {
                    s_p[j16][c] = make_float4(pp[0], pp[1], pp[2], pp[3]);
                    if (j16 == 0) s_a[c] = make_float4(aa[0], aa[1], aa[2], aa[3]);
                }
                wave_lds_sync();
                float av[8];
                {
                    const float4 a0 = s_a[0], a1 = s_a[1];
                    av[0] = a0.x; av[1] = a0.y; av[2] = a0.z; av[3] = a0.w;
                    av[4] = a1.x; av[5] = a1.y; av[6] = a1.z; av[7] = a1.w;
                }
#pragma unroll
                for (int h = 0; h < GT; ++h)
#pragma unroll
                    for (int e = 0; e < VPL; ++e) acc[h][e] *= av[h];
                // this lane group's rows of the tile: c, c + 4, c + 8, c + 12
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) {
                    float vv[VPL];
                    VC::unpack(vr[k][kk], vv);
                    const float4 pp0 = s_p[4 * kk + c][0], pp1 = s_p[4 * kk + c][1];
                    const float pv[8] = {pp0.x, pp0.y, pp0.z, pp0.w, pp1.x, pp1.y, pp1.z, pp1.w};
#pragma unroll
                    for (int h = 0; h < GT; ++h)
#pragma unroll
                        for (int e = 0; e < VPL; ++e) acc[h][e] = fmaf(pv[h], vv[e], acc[h][e]);
                }
                wave_lds_sync();
            }
        }
    };
    const bool ok = walk_units<float, DENSE, false, PT>(a, v, p, iw, plan_lds, run);

    __syncthreads();  // s_p / s_a are overwritten by the states
    // the four lane groups share each head's maximum: their value sums add
#pragma unroll
    for (int h = 0; h < GT; ++h) {
        float x[VPL];
#pragma unroll
        for (int e = 0; e < VPL; ++e) {
            float t = acc[h][e];
            t += __shfl_xor(t, 16);
            t += __shfl_xor(t, 32);
            x[e] = t;
        }
        if (c == 0) {
            float* st = wave_state(lds, wv, h, D);
#pragma unroll
            for (int e = 0; e < VPL; ++e) st[VPL * j16 + e] = x[e];
        }
    }
    if (c < 2 && j16 == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float* st = wave_state(lds, wv, 4 * c + r, D);
            st[D] = ok ? m[r] : __builtin_nanf("");
            st[D + 1] = l[r];
        }
    }
}

// Head h of pair p from the nwp workgroup states of the pair: thread
// (slice, quad) folds the states slice, slice + NSL, ... into a running
// (maximum, mass, value quad); the slices are then rescaled to a common
// maximum in LDS and the quads of out = U^ / Z^ written.  `ok` false (a wait
// that ran out) or a NaN maximum poisons the head with NaN.
template <int D, bool COHERENT>
__device__ void merge_head(const DecodeArgs& a, const float* part_p, int p, int h, int nwp, bool ok, float4* s_acc,
                           float2* s_ml) {
    constexpr int NQ = D / 4;
    constexpr int SS = D + 4;
    constexpr int NSL = kThreads / NQ;
    const int tid = threadIdx.x, G = a.G;
    const int sl = tid / NQ, dq = tid - sl * NQ;
    // this thread's states w = sl, sl + NSL, ...: KL of them loaded together
    // (one memory round trip per KL), then folded in
    constexpr int KL = 8;
    float mx = kNeg, L = 0.f;
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
    bool nan = false;
    const __amdgpu_buffer_rsrc_t rs = coherent_rsrc(part_p, static_cast<uint32_t>(nwp) * G * SS * 4u);
    for (int w0 = sl; w0 < nwp; w0 += NSL * KL) {
        float2 ml[KL];
        float4 x[KL];
#pragma unroll
        for (int k = 0; k < KL; ++k) {
            const int w = w0 + k * NSL;
            ml[k] = make_float2(kNeg, 0.f);
            x[k] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (w < nwp) {
                const uint32_t off = static_cast<uint32_t>((w * G + h) * SS) * 4u;
                if (COHERENT) {
                    const u32x2v m2 = load8_coherent(rs, off + 4u * D);
                    const u32x4v x4 = load16_coherent(rs, off + 16u * dq);
                    ml[k] = make_float2(__uint_as_float(m2.x), __uint_as_float(m2.y));
                    x[k] = make_float4(__uint_as_float(x4.x), __uint_as_float(x4.y), __uint_as_float(x4.z),
                                       __uint_as_float(x4.w));
                } else {
                    const float* st = part_p + (static_cast<size_t>(w) * G + h) * SS;
                    ml[k] = *reinterpret_cast<const float2*>(st + D);
                    x[k] = reinterpret_cast<const float4*>(st)[dq];
                }
            }
        }
#pragma unroll
        for (int k = 0; k < KL; ++k) {
            nan = nan || ml[k].x != ml[k].x;
            if (ml[k].x > kEmpty) {
                const float mn = fmaxf(mx, ml[k].x);
                const float sa = fast_exp2(mx - mn), sb = fast_exp2(ml[k].x - mn);
                L = L * sa + ml[k].y * sb;
                o.x = o.x * sa + x[k].x * sb;
                o.y = o.y * sa + x[k].y * sb;
                o.z = o.z * sa + x[k].z * sb;
                o.w = o.w * sa + x[k].w * sb;
                mx = mn;
            }
        }
    }
    if (nan) mx = __builtin_nanf("");
    s_acc[sl * NQ + dq] = o;
    if (dq == 0) s_ml[sl] = make_float2(mx, L);
    __syncthreads();
    if (tid < NQ) {
        float M2 = kNeg;
        bool bad = !ok;
        for (int s = 0; s < NSL; ++s) {
            const float ms = s_ml[s].x;
            bad = bad || ms != ms;
            M2 = fmaxf(M2, ms);
        }
        float L2 = 0.f;
        float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int s = 0; s < NSL; ++s) {
            const float2 ml = s_ml[s];
            const float wt = ml.x > kEmpty ? fast_exp2(ml.x - M2) : 0.f;
            L2 = fmaf(wt, ml.y, L2);
            const float4 x = s_acc[s * NQ + tid];
            O.x = fmaf(wt, x.x, O.x);
            O.y = fmaf(wt, x.y, O.y);
            O.z = fmaf(wt, x.z, O.z);
            O.w = fmaf(wt, x.w, O.w);
        }
        const float inv = bad ? __builtin_nanf("") : 1.f / L2;
        const int b = p / a.Hkv, kv = p - b * a.Hkv;
        float* out = a.out + (static_cast<size_t>(b) * a.Hq + kv * G + h) * D;
        reinterpret_cast<float4*>(out)[tid] = make_float4(O.x * inv, O.y * inv, O.z * inv, O.w * inv);
    }
}

// ---------------------------------------------------------------------------
// Phase C: the workgroup's waves' states (canonical form in LDS) -> one state
// per query head in the workspace; workgroup iw of the pair then merges the
// heads h == iw (mod nwp) once every workgroup of the pair has published.
// ---------------------------------------------------------------------------
template <int D, bool INKERNEL>
__device__ void combine_and_merge(const DecodeArgs& a, const Views& v, int p, int iw, int nwp, char* lds) {
    constexpr int NQ = D / 4;  // 16-byte quads of a state's value sum
    constexpr int SS = D + 4;
    constexpr int NSL = kThreads / NQ;  // workgroups' states one merge pass reads at once
    const int tid = threadIdx.x;
    const int G = a.G;
    __syncthreads();
    // 1. combine the eight waves' states of each head and publish it
    float* const part_p = v.part + static_cast<size_t>(p) * a.lay.maxwp * G * SS;
    if (tid < G * NQ) {
        const int h = tid / NQ, dq = tid - h * NQ;
        float mx = kNeg;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) mx = fmaxf(mx, wave_state(lds, w, h, D)[D]);
        float L = 0.f;
        float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const float* st = wave_state(lds, w, h, D);
            const float mw = st[D];
            const float wt = mw > kEmpty ? fast_exp2(mw - mx) : 0.f;
            L = fmaf(wt, st[D + 1], L);
            const float4 x = reinterpret_cast<const float4*>(st)[dq];
            o.x = fmaf(wt, x.x, o.x);
            o.y = fmaf(wt, x.y, o.y);
            o.z = fmaf(wt, x.z, o.z);
            o.w = fmaf(wt, x.w, o.w);
        }
        float* dst = part_p + (static_cast<size_t>(iw) * G + h) * SS;
        if (INKERNEL) {
            store_f4_coherent(dst + 4 * dq, o);
            if (dq == 0) store_f2_coherent(dst + D, mx, L);
        } else {
            reinterpret_cast<float4*>(dst)[dq] = o;
            if (dq == 0) reinterpret_cast<float4*>(dst + D)[0] = make_float4(mx, L, 0.f, 0.f);
        }
    }
    if (!INKERNEL) return;  // the merge kernel follows
    drain_and_sync();
    if (tid < G) atomicAdd(&v.done[static_cast<size_t>(p) * G + tid], 1);
    // 2. this workgroup's heads: wait for the pair's states, then merge
    int* const s_flag = reinterpret_cast<int*>(lds);
    float4* const s_acc = reinterpret_cast<float4*>(lds + 64);   // [NSL][NQ]
    float2* const s_ml = reinterpret_cast<float2*>(lds + 64 + NSL * NQ * 16);  // [NSL]
    for (int h = iw; h < G; h += nwp) {
        int* const ctr = v.done + static_cast<size_t>(p) * G + h;
        const bool ok = wait_count(ctr, nwp, s_flag);
        merge_head<D, true>(a, part_p, p, h, nwp, ok, s_acc, s_ml);
        if (tid == 0) {
            // for the next call: every workgroup of the pair has published
            // this head (so, for head 0, every one has passed its wait for
            // the samples)
            __hip_atomic_store(ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (h == 0) __hip_atomic_store(v.arrive + p, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        __syncthreads();  // s_acc / s_ml are reused
    }
}

// ===========================================================================
// Single-launch step.  One launch of B Hkv nwp workgroups, nwp per (b, kv)
// pair, all resident at once (one per compute unit):
//   1. routing, split over the pair's workgroups: workgroup iw takes the
//      pair's teams [iw S, iw S + S) and computes, for every query head of the
//      group, phi_g = log n_g + scale q.l_g in fp64, the head's Gumbel variate
//      and Y_g = phi_g + G_g; it publishes Y's order key and phi (fp32) as
//      tagged words;
//   2. selection, redundantly in every workgroup of the pair (wave h for head
//      h): the wave reads the head's M keys once all carry this call's tag,
//      finds tau (the key of rank K) and the sample (ties to the lower team),
//      and log c of its sampled teams; every workgroup of the pair holds the
//      same selection, so no further exchange is needed;
//   3. the read plan (the union of the heads' samples in team order) and the
//      attention over the workgroup's share of the units, as in the split
//      launch;
//   4. each workgroup publishes one tagged state per head; workgroup h of the
//      pair merges head h once every state of it carries the tag, and the
//      merger of head 0 advances the pair's epoch.
// ===========================================================================
// The exchange words of pair p, head h: three rows of M tagged 64-bit words
// (value, tag): the high 32 bits of Y's order key, its low 32 bits, and phi
// in fp32.
struct StepViews {
    uint32_t* epoch;  // [BH]
    uint64_t* xk;     // [BH, G, 3, M] tagged exchange words
    float* part;      // [BH, maxwp, G] published states of step_state_bytes(d) each
};

__device__ __forceinline__ StepViews step_views(const DecodeArgs& a) {
    StepViews v;
    v.epoch = reinterpret_cast<uint32_t*>(a.ws + a.lay.epoch);
    v.xk = reinterpret_cast<uint64_t*>(a.ws + a.lay.xk);
    v.part = reinterpret_cast<float*>(a.ws + a.lay.part);
    return v;
}

// Publish Y (as its order key, high and low 32 bits) and phi of (head h,
// team g) to the pair's exchange words (rx covers the pair's G * 3 * M words).
__device__ __forceinline__ void publish_item(__amdgpu_buffer_rsrc_t rx, int M, int h, int g, double phi, double y,
                                             uint32_t tag) {
    const uint64_t key = order_key(y);
    const uint32_t o = (static_cast<uint32_t>(h) * 3u * M + g) * 8u;
    store8_coherent(rx, o, u32x2v{static_cast<uint32_t>(key >> 32), tag});
    store8_coherent(rx, o + 8u * M, u32x2v{static_cast<uint32_t>(key), tag});
    store8_coherent(rx, o + 16u * M, u32x2v{__float_as_uint(static_cast<float>(phi)), tag});
}

// Teams of a workgroup's routing slice: a multiple of four (whole Philox
// blocks), the pair's M teams covered by its nwp workgroups.
__device__ __forceinline__ int step_slice(int M, int nwp) { return 4 * ((M + 4 * nwp - 1) / (4 * nwp)); }

// Phase 1 for workgroup iw of pair p: the slice's teams in chunks of 64.
// Octet o (threads 8 o .. 8 o + 7) takes team c0 + o: each lane holds d / 8
// dims of the routing key (route_issue), every head's dot product is summed
// over the octet (fp64, exact products), and lane h keeps phi of head h
// (route_finish); lane h also draws the Gumbel variate of (h, team) while the
// routing keys load (route_gumbel).
template <int D>
struct RouteRegs {
    static constexpr int LPL = RepLanes<bf16_t, D>::LPL;
    uint4 raw[LPL];
    double ln;
};

template <int D>
__device__ __forceinline__ RouteRegs<D> route_issue(const DecodeArgs& a, int p, int c0, int nt) {
    using RL = RepLanes<bf16_t, D>;
    RouteRegs<D> r;
    const int o = threadIdx.x >> 3, sub = threadIdx.x & 7;
    r.ln = 0.0;
#pragma unroll
    for (int l = 0; l < RL::LPL; ++l) r.raw[l] = make_uint4(0, 0, 0, 0);
    if (o < nt) {
        const size_t g = static_cast<size_t>(p) * a.M + c0 + o;
        const uint4* src = reinterpret_cast<const uint4*>(static_cast<const bf16_t*>(a.reps) + g * D + sub * RL::EPL);
#pragma unroll
        for (int l = 0; l < RL::LPL; ++l) r.raw[l] = load_stream(src + l);
        r.ln = a.log_n[g];
    }
    return r;
}

// The Gumbel variate of (head sub, team c0 + o) for lane sub < G of octet o
// (0 elsewhere): word (c0 + o) % 4 of the Philox block at counter
// ((c0 + o) / 4, h, b, step), key (seed, 0).
__device__ __forceinline__ double route_gumbel(const DecodeArgs& a, int p, int c0, int nt) {
    const int G = a.G, b = p / a.Hkv, kv = p - b * a.Hkv;
    const int o = threadIdx.x >> 3, h = threadIdx.x & 7;
    if (o >= nt || h >= G) return 0.0;
    const int g = c0 + o;
    const u64x4 r = philox4x64_10(static_cast<uint64_t>(g >> 2), static_cast<uint64_t>(kv * G + h),
                                  static_cast<uint64_t>(b), a.step, a.seed, 0);
    const int e = g & 3;
    return gumbel_of_word(e == 0 ? r.v[0] : e == 1 ? r.v[1] : e == 2 ? r.v[2] : r.v[3]);
}

template <int D>
__device__ __forceinline__ void route_finish(const DecodeArgs& a, int p, int c0, int nt, uint32_t tag,
                                             const RouteRegs<D>& r, const double* s_qd, double gum,
                                             __amdgpu_buffer_rsrc_t rx) {
    using RL = RepLanes<bf16_t, D>;
    constexpr int EPL = RL::EPL;
    const int G = a.G, M = a.M;
    const int o = threadIdx.x >> 3, sub = threadIdx.x & 7;
    if (o >= nt) return;
    double phi = 0.0;
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
        if (h < G) {  // uniform
            const double* qh = s_qd + h * D + sub * EPL;
            double a0 = 0.0, a1 = 0.0;
#pragma unroll
            for (int e = 0; e < EPL; e += 2) {
                a0 = fma(qh[e], static_cast<double>(RL::elem(r.raw, e)), a0);
                a1 = fma(qh[e + 1], static_cast<double>(RL::elem(r.raw, e + 1)), a1);
            }
            const double sum = row8_sum(a0 + a1);
            if (sub == h) phi = r.ln + a.scale * sum;
        }
    }
    if (sub < G) {
        const int g = c0 + o, h = sub;
        const double y = phi + gum;
        publish_item(rx, M, h, g, phi, y, tag);
        const int b = p / a.Hkv, kv = p - b * a.Hkv;
        const size_t bq = static_cast<size_t>(b) * a.Hq + kv * G + h;
        if (a.dbg_phi) a.dbg_phi[bq * M + g] = phi;
        if (a.dbg_Y) a.dbg_Y[bq * M + g] = y;
    }
}

__device__ __forceinline__ double readlane_f64(double v, int l) {
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane(static_cast<int>(b & 0xffffffff), l);
    const int hi = __builtin_amdgcn_readlane(static_cast<int>(b >> 32), l);
    return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<unsigned>(lo));
}

// Routing of a slice of at most eight teams, in two roles that run at once:
// waves 0-3 form the dot products (two teams per wave, 32 lanes per team, d /
// 32 dims of the routing key and of every query head per lane, read directly;
// a head's sum over the team's lanes in fp64 with exact products), wave 4
// draws the slice's Gumbel variates (lane 8 t + h for head h of team t).
// Both land in s_pg (phi [8][8], then the variates [8][8]); route_publish
// forms Y after the workgroup barrier that follows.
template <int D>
__device__ __forceinline__ void route_split(const DecodeArgs& a, int p, int c0, int nt, double* s_pg) {
    constexpr int EPL = D / 32;  // 4 (d = 128) or 2 (d = 64)
    static_assert(EPL == 2 || EPL == 4, "two or four dims per lane");
    const int lane = lane_id(), w = wave_id();
    const int G = a.G, M = a.M, b = p / a.Hkv, kv = p - b * a.Hkv;
    if (w < 4) {
        if (2 * w >= nt) return;  // uniform
        const int t = 2 * w + (lane >> 5), l = lane & 31;
        const int g = c0 + min(t, nt - 1);
        const size_t tg = static_cast<size_t>(p) * M + g;
        // every load first (heads beyond G read head G - 1's dims)
        const bf16_t* row = static_cast<const bf16_t*>(a.reps) + tg * D + l * EPL;
        uint32_t kr[EPL / 2];
        if constexpr (EPL == 4) {
            const uint2 x = *reinterpret_cast<const uint2*>(row);
            kr[0] = x.x;
            kr[1] = x.y;
        } else {
            kr[0] = *reinterpret_cast<const uint32_t*>(row);
        }
        const double ln = a.log_n[tg];
        const float* qg = a.q + (static_cast<size_t>(b) * a.Hq + kv * G) * D + l * EPL;
        float qv[kMaxGroup][EPL];
#pragma unroll
        for (int h = 0; h < kMaxGroup; ++h) {
            const float* qh = qg + min(h, G - 1) * D;
            if constexpr (EPL == 4) {
                const float4 x = *reinterpret_cast<const float4*>(qh);
                qv[h][0] = x.x;
                qv[h][1] = x.y;
                qv[h][2] = x.z;
                qv[h][3] = x.w;
            } else {
                const float2 x = *reinterpret_cast<const float2*>(qh);
                qv[h][0] = x.x;
                qv[h][1] = x.y;
            }
        }
        double kd[EPL];
#pragma unroll
        for (int e = 0; e < EPL; ++e) kd[e] = static_cast<double>((e & 1) ? bf16hi(kr[e >> 1]) : bf16lo(kr[e >> 1]));
        const double lnA = readlane_f64(ln, 0), lnB = readlane_f64(ln, 32);
#pragma unroll
        for (int h = 0; h < kMaxGroup; ++h) {
            if (h < G) {  // uniform
                double part = static_cast<double>(qv[h][0]) * kd[0];
#pragma unroll
                for (int e = 1; e < EPL; ++e) part = fma(static_cast<double>(qv[h][e]), kd[e], part);
                part = row16_sum(part);
                const double sA = readlane_f64(part, 0) + readlane_f64(part, 16);
                const double sB = readlane_f64(part, 32) + readlane_f64(part, 48);
                if (lane == 0) {
                    s_pg[(2 * w) * 8 + h] = lnA + a.scale * sA;
                    s_pg[(2 * w + 1) * 8 + h] = lnB + a.scale * sB;
                }
            }
        }
    } else if (w == 4) {
        const int t = lane >> 3, h = lane & 7;
        if (t < nt && h < G) {
            const int g = c0 + t;
            const u64x4 r = philox4x64_10(static_cast<uint64_t>(g >> 2), static_cast<uint64_t>(kv * G + h),
                                          static_cast<uint64_t>(b), a.step, a.seed, 0);
            const int e = g & 3;
            s_pg[64 + t * 8 + h] = gumbel_of_word(e == 0 ? r.v[0] : e == 1 ? r.v[1] : e == 2 ? r.v[2] : r.v[3]);
        }
    }
}

// Y = phi + G of the slice's (team, head) items (lane 8 t + h of wave 0),
// published as tagged words with phi.
__device__ __forceinline__ void route_publish(const DecodeArgs& a, int p, int c0, int nt, uint32_t tag,
                                              const double* s_pg, __amdgpu_buffer_rsrc_t rx) {
    const int lane = lane_id();
    const int t = lane >> 3, h = lane & 7;
    if (wave_id() != 0 || t >= nt || h >= a.G) return;
    const int G = a.G, M = a.M, b = p / a.Hkv, kv = p - b * a.Hkv;
    const int g = c0 + t;
    const double phi = s_pg[t * 8 + h];
    const double y = phi + s_pg[64 + t * 8 + h];
    publish_item(rx, M, h, g, phi, y, tag);
    const size_t bq = static_cast<size_t>(b) * a.Hq + kv * G + h;
    if (a.dbg_phi) a.dbg_phi[bq * M + g] = phi;
    if (a.dbg_Y) a.dbg_Y[bq * M + g] = y;
}

// LDS of one wave's selection: a 256-bin histogram and up to 64 candidates.
struct WaveSel {
    uint32_t hist[256];
    uint64_t cand[kWave];
};

// Key of rank `want` (0-based, descending) among the wave's keys (key j of
// lane l is team 64 j + l; teams >= M do not count), by an exact radix over
// the 64-bit keys, eight bits at a time from the top; `above` receives the
// count of keys strictly greater.
template <int KPL>
__device__ uint64_t wave_rank_exact(const uint64_t (&k)[KPL], int M, int want, WaveSel& W, int& above) {
    const int lane = lane_id();
    uint64_t prefix = 0, pmask = 0;
    above = 0;
    int cnt = 0;
    for (int sh = 56;; sh -= 8) {  // uniform
        reinterpret_cast<uint4*>(W.hist)[lane] = make_uint4(0, 0, 0, 0);
        lds_order();
#pragma unroll
        for (int j = 0; j < KPL; ++j)
            if (64 * j + lane < M && (k[j] & pmask) == prefix) atomicAdd(&W.hist[(k[j] >> sh) & 255], 1u);
        lds_order();
        int hi;
        const int dg = hist_select(W.hist, want, hi, cnt);
        lds_order();
        want -= hi;
        above += hi;
        prefix |= static_cast<uint64_t>(dg) << sh;
        pmask |= 0xffull << sh;
        if (cnt == 1 || sh == 0) break;
    }
    if (cnt == 1) {  // the one key with this prefix
        uint64_t r = 0;
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            const bool m = 64 * j + lane < M && (k[j] & pmask) == prefix;
            const uint64_t bal = __ballot(m);
            if (bal) r = readlane(k[j], __ffsll(static_cast<unsigned long long>(bal)) - 1);
        }
        return r;
    }
    return prefix;  // every bit fixed: equal keys
}

// Minimum / maximum of a float over the wave (rotations within each 16-lane
// row, then the four rows' results); wave-uniform.
template <bool kMin>
__device__ __forceinline__ float wave_ext_f(float v) {
    auto op = [](float x, float y) { return kMin ? fminf(x, y) : fmaxf(x, y); };
    v = op(v, dpp_f32<0x128>(v));
    v = op(v, dpp_f32<0x124>(v));
    v = op(v, dpp_f32<0x122>(v));
    v = op(v, dpp_f32<0x121>(v));
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return op(op(r0, r1), op(r2, r3));
}

// Key of rank `want` among the wave's keys, and the count above it: a value
// histogram of 256 bins over [min Y, max Y] with Y rounded to fp32 (rounding
// keeps the order, so a bin above another holds only larger or equal keys),
// then a direct ranking of the exact keys in the bin that holds rank `want`;
// the exact radix where that bin holds more than 64 keys, the keys span no
// finite fp32 range (absent teams) or all are equal.
template <int KPL>
__device__ uint64_t wave_rank(const uint64_t (&k)[KPL], int M, int want, WaveSel& W, int& above) {
    const int lane = lane_id();
    float y[KPL];
    float lo = __builtin_inff(), hi = -__builtin_inff();
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        y[j] = static_cast<float>(key_value(k[j]));
        if (64 * j + lane < M) {
            lo = fminf(lo, y[j]);
            hi = fmaxf(hi, y[j]);
        }
    }
    lo = wave_ext_f<true>(lo);
    hi = wave_ext_f<false>(hi);
    const float range = hi - lo;
    if (!(range > 0.f) || !(range < 3.0e38f)) return wave_rank_exact<KPL>(k, M, want, W, above);
    const float fs = 255.99f / range;
    reinterpret_cast<uint4*>(W.hist)[lane] = make_uint4(0, 0, 0, 0);
    lds_order();
    int bin[KPL];
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        bin[j] = 64 * j + lane < M ? static_cast<int>(fminf(255.f, (y[j] - lo) * fs)) : -1;
        if (bin[j] >= 0) atomicAdd(&W.hist[bin[j]], 1u);
    }
    lds_order();
    int hcnt, cnt;
    const int sb = hist_select(W.hist, want, hcnt, cnt);
    lds_order();
    if (cnt > kWave) return wave_rank_exact<KPL>(k, M, want, W, above);
    int n = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        const bool in = bin[j] == sb;
        const uint64_t bal = __ballot(in);
        if (in) W.cand[n + static_cast<int>(__popcll(bal & lanemask_lt()))] = k[j];
        n += static_cast<int>(__popcll(bal));
    }
    lds_order();
    const int rest = want - hcnt;
    const uint64_t mine = W.cand[min(lane, n - 1)];
    int gt = 0, ge = 0;
    for (int t = 0; t < n; ++t) {
        const uint64_t o = readlane(mine, t);
        gt += o > mine ? 1 : 0;
        ge += o >= mine ? 1 : 0;
    }
    const bool owner = lane < n && gt <= rest && rest < ge;
    const int src = __ffsll(static_cast<unsigned long long>(__ballot(owner))) - 1;
    above = hcnt + readlane(gt, src);
    return readlane(mine, src);
}

// Monotone fp32 value of a 32-bit key (the high half of a double's order
// key): the double truncated to its 20 high mantissa bits, then rounded.
__device__ __forceinline__ float key32_value(uint32_t k) {
    const uint32_t hi = (k >> 31) ? (k & 0x7fffffffu) : ~k;
    return static_cast<float>(__hiloint2double(static_cast<int>(hi), 0));
}

// Exact radix select over 32-bit keys (four 8-bit digits from the top), as
// wave_rank_exact for 64-bit keys.
template <int KPL>
__device__ uint32_t wave_rank32_exact(const uint32_t (&k)[KPL], int M, int want, WaveSel& W, int& above) {
    const int lane = lane_id();
    uint32_t prefix = 0, pmask = 0;
    above = 0;
    int cnt = 0;
    for (int sh = 24;; sh -= 8) {  // uniform
        reinterpret_cast<uint4*>(W.hist)[lane] = make_uint4(0, 0, 0, 0);
        lds_order();
#pragma unroll
        for (int j = 0; j < KPL; ++j)
            if (64 * j + lane < M && (k[j] & pmask) == prefix) atomicAdd(&W.hist[(k[j] >> sh) & 255u], 1u);
        lds_order();
        int hi;
        const int dg = hist_select(W.hist, want, hi, cnt);
        lds_order();
        want -= hi;
        above += hi;
        prefix |= static_cast<uint32_t>(dg) << sh;
        pmask |= 0xffu << sh;
        if (cnt == 1 || sh == 0) break;
    }
    if (cnt == 1) {  // the one key with this prefix
        uint32_t r = 0;
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            const uint64_t bal = __ballot(64 * j + lane < M && (k[j] & pmask) == prefix);
            if (bal) r = static_cast<uint32_t>(readlane(static_cast<int>(k[j]), __ffsll(static_cast<unsigned long long>(bal)) - 1));
        }
        return r;
    }
    return prefix;  // every bit fixed: equal keys
}

// Key of rank `want` (0-based, descending) among the wave's 32-bit keys and
// the count strictly above it: a 256-bin value histogram over [min, max] of
// the keys' fp32 values, then a direct ranking of the keys in the bin that
// holds rank `want`; the exact radix where that bin holds more than 64 keys
// or the keys span no finite fp32 range.
template <int KPL>
__device__ uint32_t wave_rank32(const uint32_t (&k)[KPL], int M, int want, WaveSel& W, int& above) {
    const int lane = lane_id();
    float y[KPL];
    float lo = __builtin_inff(), hi = -__builtin_inff();
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        y[j] = key32_value(k[j]);
        if (64 * j + lane < M) {
            lo = fminf(lo, y[j]);
            hi = fmaxf(hi, y[j]);
        }
    }
    lo = wave_ext_f<true>(lo);
    hi = wave_ext_f<false>(hi);
    const float range = hi - lo;
    if (!(range > 0.f) || !(range < 3.0e38f)) return wave_rank32_exact<KPL>(k, M, want, W, above);
    const float fs = 255.99f / range;
    reinterpret_cast<uint4*>(W.hist)[lane] = make_uint4(0, 0, 0, 0);
    lds_order();
    int bin[KPL];
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        bin[j] = 64 * j + lane < M ? static_cast<int>(fminf(255.f, (y[j] - lo) * fs)) : -1;
        if (bin[j] >= 0) atomicAdd(&W.hist[bin[j]], 1u);
    }
    lds_order();
    int hcnt, cnt;
    const int sb = hist_select(W.hist, want, hcnt, cnt);
    lds_order();
    if (cnt > kWave) return wave_rank32_exact<KPL>(k, M, want, W, above);
    uint32_t* const cand = reinterpret_cast<uint32_t*>(W.cand);
    int n = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        const bool in = bin[j] == sb;
        const uint64_t bal = __ballot(in);
        if (in) cand[n + static_cast<int>(__popcll(bal & lanemask_lt()))] = k[j];
        n += static_cast<int>(__popcll(bal));
    }
    lds_order();
    const int rest = want - hcnt;
    const uint32_t mine = cand[min(lane, n - 1)];
    int gt = 0, ge = 0;
    for (int t = 0; t < n; ++t) {
        const uint32_t o = static_cast<uint32_t>(readlane(static_cast<int>(mine), t));
        gt += o > mine ? 1 : 0;
        ge += o >= mine ? 1 : 0;
    }
    const bool owner = lane < n && gt <= rest && rest < ge;
    const int src = __ffsll(static_cast<unsigned long long>(__ballot(owner))) - 1;
    above = hcnt + readlane(gt, src);
    return static_cast<uint32_t>(readlane(static_cast<int>(mine), src));
}

// Poll `n` rows-of-words loads: lane's words at byte offsets off[j] (for the
// bits of `pend`) until each carries `tag`; returns false at the spin limit.
template <int KPL>
__device__ __forceinline__ bool poll_words(__amdgpu_buffer_rsrc_t r, const uint32_t (&off)[KPL], uint32_t pend,
                                           uint32_t tag, uint32_t (&val)[KPL]) {
    constexpr int kBatch = KPL < 16 ? KPL : 16;
    for (int it = 0;; ++it) {
#pragma unroll
        for (int j0 = 0; j0 < KPL; j0 += kBatch) {
            u32x2v w[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j)
                if ((pend >> (j0 + j)) & 1u) w[j] = load8_coherent(r, off[j0 + j]);
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                if (((pend >> (j0 + j)) & 1u) && w[j].y == tag) {
                    val[j0 + j] = w[j].x;
                    pend &= ~(1u << (j0 + j));
                }
            }
        }
        if (__ballot(pend != 0) == 0) return true;  // uniform
        if (it >= kSpinLimit) return false;
        __builtin_amdgcn_s_sleep(1);
    }
}

// Phase 2 for wave h (a query head of the pair).  The wave reads the high
// halves of the head's M keys once all carry the tag and finds the key of
// rank K among them.  When that high half is unique (the common case) the
// sample is every key above it, and a second read fetches the low half of
// tau's key and phi of the sampled teams; otherwise the low halves of all
// keys are read and the exact 64-bit keys ranked (ties of equal keys to the
// lower team index).  The sample goes to SS as bit words, head bits of the
// team masks and phi - tau by rank.  Returns false when a word did not arrive
// within the spin limit.
template <int KPL>
__device__ bool step_select(const DecodeArgs& a, const StepViews& v, int p, int iw, uint32_t tag, WaveSel& W,
                            StepSel& SS) {
    const int lane = lane_id(), h = wave_id(), G = a.G, M = a.M, Kp = a.Kp;
    const int b = p / a.Hkv, kv = p - b * a.Hkv;
    const size_t hb = (static_cast<size_t>(p) * G + h) * 3 * M;
    const __amdgpu_buffer_rsrc_t rh = coherent_rsrc(v.xk + hb, static_cast<uint32_t>(M) * 24u);
    const uint32_t row1 = 8u * M, row2 = 16u * M;
    uint32_t off[KPL], k[KPL], valid = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        off[j] = static_cast<uint32_t>(64 * j + lane) * 8u;
        k[j] = 0;
        if (64 * j + lane < M) valid |= 1u << j;
    }
    bool ok = poll_words<KPL>(rh, off, valid, tag, k);
    int above;
    const uint32_t th = wave_rank32<KPL>(k, M, Kp, W, above);
    int bcnt = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) bcnt += static_cast<int>(__popcll(__ballot(((valid >> j) & 1u) && k[j] == th)));
    uint64_t selw[KPL];
    int tau_g = -1;
    uint32_t tau_lo = 0;
    if (bcnt == 1) {  // uniform: the sample is every key whose high half exceeds th
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            selw[j] = __ballot(((valid >> j) & 1u) && k[j] > th);
            const uint64_t t = __ballot(((valid >> j) & 1u) && k[j] == th);
            if (t) tau_g = 64 * j + __ffsll(static_cast<unsigned long long>(t)) - 1;
        }
    } else {  // several keys share tau's high half: rank the exact keys
        uint32_t offl[KPL], lo[KPL];
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            offl[j] = row1 + off[j];
            lo[j] = 0;
        }
        ok = poll_words<KPL>(rh, offl, valid, tag, lo) && ok;
        uint64_t k64[KPL];
#pragma unroll
        for (int j = 0; j < KPL; ++j) k64[j] = (static_cast<uint64_t>(k[j]) << 32) | lo[j];
        int above64;
        const uint64_t tkey = wave_rank<KPL>(k64, M, Kp, W, above64);
        tau_lo = static_cast<uint32_t>(tkey);
        int need = Kp - above64;
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            const bool vj = (valid >> j) & 1u;
            uint64_t sb = __ballot(vj && k64[j] > tkey);
            if (need > 0) {  // uniform
                uint64_t tb = __ballot(vj && k64[j] == tkey);
                while (need > 0 && tb) {
                    const uint64_t low = tb & (~tb + 1);
                    sb |= low;
                    tb ^= low;
                    --need;
                }
            }
            selw[j] = sb;
        }
    }
    // tau for the corrections: its high half, and where its low half is
    if (lane == 0) {
        SS.tau_hi[h] = th;  // also the high half of the exact path's key (truncation keeps the order)
        SS.tau_g[h] = tau_g;
        SS.tau_lo[h] = tau_lo;
    }
    // the head's bit in the masks of its sampled teams
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        if ((selw[j] >> lane) & 1ull) {
            const int g = 64 * j + lane;
            atomicOr(&SS.hm[g >> 2], 1u << (h + 8 * (g & 3)));
        }
    }
    // diagnostics (one workgroup of the pair): tau, the sample in ascending
    // team order and its log c, from the exchange words
    const size_t bq = static_cast<size_t>(b) * a.Hq + kv * G + h;
    double tau = 0.0;
    if (iw == 0 && (a.dbg_tau || a.dbg_sel || a.dbg_logc)) {  // uniform
        uint32_t tl = tau_lo;
        if (tau_g >= 0) {
            uint32_t o1[1] = {row1 + static_cast<uint32_t>(tau_g) * 8u}, v1[1] = {0};
            ok = poll_words<1>(rh, o1, 1u, tag, v1) && ok;
            tl = v1[0];
        }
        tau = key_value((static_cast<uint64_t>(th) << 32) | tl);
        uint32_t offp[KPL], ph[KPL], mine = 0;
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            offp[j] = row2 + off[j];
            ph[j] = 0;
            if ((selw[j] >> lane) & 1ull) mine |= 1u << j;
        }
        ok = poll_words<KPL>(rh, offp, mine, tag, ph) && ok;
        int cum = 0;
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            const uint64_t sb = selw[j];
            if ((sb >> lane) & 1ull) {
                const int rank = cum + static_cast<int>(__popcll(sb & lanemask_lt()));
                if (rank < Kp) {
                    if (a.dbg_sel) a.dbg_sel[bq * Kp + rank] = 64 * j + lane;
                    if (a.dbg_logc)
                        a.dbg_logc[bq * Kp + rank] =
                            log_inclusion(static_cast<float>(static_cast<double>(__uint_as_float(ph[j])) - tau));
                }
            }
            cum += static_cast<int>(__popcll(sb));
        }
    }
    if (iw == 0 && lane == 0 && a.dbg_tau) a.dbg_tau[bq] = tau;
    return ok;
}

// Sum of a float over the wave (rotations within each 16-lane row, then the
// four rows' sums); wave-uniform.
__device__ __forceinline__ float wave_sum_dpp(float v) {
    v = row16_sum(v);
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return (r0 + r1) + (r2 + r3);
}

// Phase 4.  A published state (one per workgroup and head) is d / 2 + 1
// 16-byte chunks: chunk c < d / 2 holds (acc[2c], tag, acc[2c + 1], tag), the
// last (maximum, tag, mass, tag).  Each 8-byte half carries the tag, so a
// reader that sees the tag in both halves of a chunk has the chunk's values
// of this call, and no ordering between the chunks is needed.
//
// The workgroup combines its waves' states of each head (canonical form in
// LDS) and publishes them.  Each (head, sixteenth of the dims) is then merged
// by one wave of the pair: lane w reads state w (nwp <= 64) -- the sixteenth's
// value chunks and the (maximum, mass) chunk -- until all carry the tag, and
// the states are rescaled to the common maximum by wave sums.  The merger of
// (head 0, first sixteenth) advances the pair's epoch once all its states
// carry the tag (every workgroup of the pair has then read the epoch).
template <int D>
__device__ void step_publish_merge(const DecodeArgs& a, const StepViews& v, int p, int iw, int nwp, uint32_t tag,
                                   char* lds) {
    constexpr int NC = D / 2 + 1;  // chunks per state
    constexpr int kParts = 32;     // merge tasks per head
    constexpr int DW = D / kParts; // dims per merge task
    const int tid = threadIdx.x, G = a.G, lane = lane_id(), wv = wave_id();
    __syncthreads();
    char* const part_p = reinterpret_cast<char*>(v.part) + static_cast<size_t>(p) * a.lay.maxwp * G * NC * 16;
    const __amdgpu_buffer_rsrc_t rs = coherent_rsrc(part_p, static_cast<uint32_t>(a.lay.maxwp) * G * NC * 16u);
    for (int i = tid; i < G * NC; i += kThreads) {
        const int h = i / NC, c = i - h * NC;
        float mx = kNeg;
        bool nan = false;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const float mw = wave_state(lds, w, h, D)[D];
            nan = nan || mw != mw;
            mx = fmaxf(mx, mw);
        }
        float x0 = 0.f, x1 = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const float* st = wave_state(lds, w, h, D);
            const float mw = st[D];
            const float wt = mw > kEmpty ? fast_exp2(mw - mx) : 0.f;
            if (c < D / 2) {
                x0 = fmaf(wt, st[2 * c], x0);
                x1 = fmaf(wt, st[2 * c + 1], x1);
            } else {
                x1 = fmaf(wt, st[D + 1], x1);
            }
        }
        if (c == D / 2) x0 = nan ? __builtin_nanf("") : mx;
        store16_coherent(rs, static_cast<uint32_t>((iw * G + h) * NC + c) * 16u,
                         u32x4v{__float_as_uint(x0), tag, __float_as_uint(x1), tag});
    }
    // merge tasks: task t = 16 h + c (head h, dims [c D / 16, (c + 1) D / 16))
    // runs on workgroup t mod nwp, wave (t / nwp) mod 8, so that the merge of
    // a pair is spread over many compute units and each poll is small
    // The merge waves hold off their first poll for about 0.8 us: the pair's
    // last states land that long or more after this workgroup's, and polls
    // issued meanwhile load the memory-side cache that the pair's last
    // workgroups still read their rows through (measured: the step, sampled
    // and dense, ends sooner with the pause than without it or with 2 us).
    __builtin_amdgcn_s_sleep(30);
    for (int t = iw + wv * nwp; t < kParts * G; t += kWaves * nwp) {
        const int h = t / kParts, c = t % kParts;
        const bool live = lane < nwp;
        const uint32_t base = static_cast<uint32_t>((lane * G + h) * NC) * 16u;
        float acc[DW], mw = kNeg, lw = 0.f;
        uint32_t pend = live ? ((1u << (DW / 2 + 1)) - 1u) : 0u;  // bit DW / 2: the (maximum, mass) chunk
#pragma unroll
        for (int i = 0; i < DW; ++i) acc[i] = 0.f;
        bool ok = true;
        for (int it = 0;; ++it) {
            u32x4v x[DW / 2 + 1];
#pragma unroll
            for (int k = 0; k <= DW / 2; ++k) {
                const int cc = k < DW / 2 ? c * (DW / 2) + k : D / 2;
                if ((pend >> k) & 1u) x[k] = load16_coherent(rs, base + 16u * cc);
            }
#pragma unroll
            for (int k = 0; k <= DW / 2; ++k) {
                if (((pend >> k) & 1u) && x[k].y == tag && x[k].w == tag) {
                    if (k < DW / 2) {
                        acc[2 * k] = __uint_as_float(x[k].x);
                        acc[2 * k + 1] = __uint_as_float(x[k].z);
                    } else {
                        mw = __uint_as_float(x[k].x);
                        lw = __uint_as_float(x[k].z);
                    }
                    pend &= ~(1u << k);
                }
            }
            if (__ballot(pend != 0) == 0) break;  // uniform
            if (it >= kSpinLimit) {
                ok = false;
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        const bool bad = !ok || __ballot(mw != mw) != 0;
        const float m_all = wave_ext_f<false>(live ? mw : kNeg);
        const float wt = live && mw > kEmpty ? fast_exp2(mw - m_all) : 0.f;
        const float L = wave_sum_dpp(wt * lw);
        const float inv = bad ? __builtin_nanf("") : 1.f / L;
        const int b = p / a.Hkv, kv = p - b * a.Hkv;
        float* const out = a.out + (static_cast<size_t>(b) * a.Hq + kv * G + h) * D + c * DW;
        float r[DW];
#pragma unroll
        for (int i = 0; i < DW; ++i) r[i] = wave_sum_dpp(wt * acc[i]) * inv;
        if (lane == 0) {
#pragma unroll
            for (int i = 0; i < DW; i += 4) *reinterpret_cast<float4*>(out + i) = make_float4(r[i], r[i + 1], r[i + 2], r[i + 3]);
            if (t == 0) store_u32_coherent(v.epoch + p, tag);
        }
    }
}

// LDS of the single-launch step.  t0 and t1 hold the value tiles during the
// attention; before it, t0 holds the widened queries, the Gumbel variates and
// the waves' select scratch, and t1 the first plan pass's team table.  misc
// holds the probability tiles, the plan records, the selection state and the
// attention's fp32 copy of the pair's queries.
template <int D>
struct StepLds {
    static constexpr int tiles = kWaves * VTile<D>::kBytes;
    static constexpr int states = kWaves * kMaxGroup * (D + 4) * 4;
    static constexpr int merge = 64 + kThreads * 16 + (kThreads / (D / 4)) * 8;
    static constexpr int qd = kMaxGroup * D * 8;
    static constexpr int gum = kMaxGroup * 64 * 8;
    static constexpr int sel = kWaves * static_cast<int>(sizeof(WaveSel));
    static constexpr int max2(int x, int y) { return x > y ? x : y; }
    static constexpr int t0 = max2(max2(tiles, states), max2(merge, qd + gum + sel));
    static constexpr int t1 = max2(tiles, 2 * kStepMaxTeams * 4);
    static constexpr int plan_off = kWaves * 1024;
    static constexpr int sel_off = (plan_off + static_cast<int>(sizeof(PlanLds)) + 15) / 16 * 16;
    static constexpr int q_off = (sel_off + static_cast<int>(sizeof(StepSel)) + 15) / 16 * 16;
    static constexpr int misc = q_off + kMaxGroup * D * 4;
};

template <int D, int KPL, bool DENSE>
__global__ __launch_bounds__(kThreads, 1) void k_step(DecodeArgs a) {
    using L = StepLds<D>;
    static_assert(L::t0 + L::t1 + L::misc <= 160 * 1024, "the step's LDS fits one compute unit");
    __shared__ __attribute__((aligned(16))) char s_t0[L::t0];
    __shared__ __attribute__((aligned(16))) char s_t1[L::t1];
    __shared__ __attribute__((aligned(16))) char s_misc[L::misc];
    const StepViews v = step_views(a);
    const PairSlot sl = pair_slot(blockIdx.x, gridDim.x, a.B * a.Hkv);
    const int p = sl.p, iw = sl.iw, nwp = sl.nwp;
    // the call's tag (epoch + 1) is formed where it is first needed, so that
    // the epoch load does not hold up the loads issued after it
    const uint32_t epoch = load_u32_coherent(v.epoch + p);
    StepSel* const SS = reinterpret_cast<StepSel*>(s_misc + L::sel_off);
    int* const s_tab = reinterpret_cast<int*>(s_t1);
    const int tid = threadIdx.x;
    // the plan passes take PT teams per thread when the heads' union fits one
    // pass's records, else one
    constexpr int PT = KPL >= 8 ? KPL / 8 : 1;
    const bool wide = !DENSE && static_cast<long long>(a.G) * a.Kp <= kPlanRecs;
    if constexpr (!DENSE) {
        const int G = a.G, M = a.M;
        const int b = p / a.Hkv, kv = p - b * a.Hkv;
        double* const s_qd = reinterpret_cast<double*>(s_t0);
        WaveSel* const s_ws = reinterpret_cast<WaveSel*>(s_t0 + L::qd);
        const int S = step_slice(M, nwp);
        const int t0 = iw * S, t1 = min(M, t0 + S);
        const __amdgpu_buffer_rsrc_t rx = coherent_rsrc(v.xk + 3 * static_cast<size_t>(p) * G * M,
                                                        static_cast<uint32_t>(G) * M * 24u);
        // everything the routing needs is requested at once: the slice's
        // routing keys, the queries and the first plan pass's table
        const size_t tb0 = static_cast<size_t>(p) * M;
        const int first = min(M, kThreads * (wide ? PT : 1));
        int tsz[PT], tbg[PT];
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const int g = min(tid + i * kThreads, M - 1);
            tsz[i] = a.team_size[tb0 + g];
            tbg[i] = a.team_begin[tb0 + g];
        }
        // the pair's queries: widened for the octet routing, and the
        // attention's fp32 copy; stored once the routing's loads are out
        constexpr int kQ = kMaxGroup * D / kThreads;
        float qv[kQ];
        {
            const float* qg = a.q + (static_cast<size_t>(b) * a.Hq + kv * G) * D;
#pragma unroll
            for (int i = 0; i < kQ; ++i) qv[i] = tid + i * kThreads < G * D ? qg[tid + i * kThreads] : 0.f;
        }
        const bool by_wave = S <= kWaves;  // uniform: the split routing of at most eight teams
        RouteRegs<D> rr;
        double gum = 0.0;
        if (by_wave) {
            route_split<D>(a, p, t0, max(0, t1 - t0), s_qd);
        } else {
            rr = route_issue<D>(a, p, t0, max(0, min(64, t1 - t0)));
            gum = route_gumbel(a, p, t0, min(64, t1 - t0));
#pragma unroll
            for (int i = 0; i < kQ; ++i)
                if (tid + i * kThreads < G * D) s_qd[tid + i * kThreads] = static_cast<double>(qv[i]);
        }
        {
            float* const s_q = reinterpret_cast<float*>(s_misc + L::q_off);
#pragma unroll
            for (int i = 0; i < kQ; ++i)
                if (tid + i * kThreads < G * D) s_q[tid + i * kThreads] = qv[i];
        }
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const int g = tid + i * kThreads;
            if (g < first) {
                s_tab[2 * g] = tsz[i];
                s_tab[2 * g + 1] = tbg[i];
            }
        }
        for (int i = tid; i < (M + 3) / 4; i += kThreads) SS->hm[i] = 0;
        if (tid == 0) SS->ok = 1;
        __syncthreads();
        const uint32_t tag = epoch + 1u;
        if (by_wave) {
            route_publish(a, p, t0, max(0, t1 - t0), tag, s_qd, rx);
        } else {
            for (int c0 = t0; c0 < t1; c0 += 64) {  // uniform
                const int nt = min(64, t1 - c0);
                if (c0 > t0) {
                    rr = route_issue<D>(a, p, c0, nt);
                    gum = route_gumbel(a, p, c0, nt);
                }
                route_finish<D>(a, p, c0, nt, tag, rr, s_qd, gum, rx);
            }
        }
        if (wave_id() < G) {
            // as for the merge: a pause of about 0.5 us before the first poll
            // of the pair's keys, which the other workgroups are still
            // publishing
            __builtin_amdgcn_s_sleep(20);
            const bool ok = step_select<KPL>(a, v, p, iw, tag, s_ws[wave_id()], *SS);
            if (!ok && lane_id() == 0) SS->ok = 0;
        }
        __syncthreads();
    }
    const uint32_t tag = epoch + 1u;
    const Views none{};
    const StepCtx ctx{v.xk + 3 * static_cast<size_t>(p) * a.G * a.M, tag,
                      DENSE ? nullptr : reinterpret_cast<const float*>(s_misc + L::q_off)};
    if (wide)
        attend_mfma<D, DENSE, false, PT, true>(a, none, p, iw, nwp, s_t0, s_t1, s_misc, SS, s_tab, &ctx);
    else
        attend_mfma<D, DENSE, false, 1, true>(a, none, p, iw, nwp, s_t0, s_t1, s_misc, SS, s_tab, &ctx);
    step_publish_merge<D>(a, v, p, iw, nwp, tag, s_t0);
}

template <typename T, int D, int HK>
struct Lds {
    static constexpr int tiles = sizeof(T) == 2 ? kWaves * VTile<D>::kBytes : 16;
    static constexpr int states = kWaves * kMaxGroup * (D + 4) * 4;
    static constexpr int merge = 64 + kThreads * 16 + (kThreads / (D / 4)) * 8;
    static constexpr int words = HK * kThreads * 8;
    static constexpr int max2(int x, int y) { return x > y ? x : y; }
    static constexpr int t0 = max2(max2(tiles, states), max2(merge, words));
    static constexpr int t1 = max2(tiles, words);
    static constexpr int misc = max2(kWaves * 1024 + static_cast<int>(sizeof(PlanLds)), static_cast<int>(sizeof(SelScratch)));
};

template <typename T, int D, bool DENSE, bool FUSED, int PT>
__device__ __forceinline__ void attend_pair(const DecodeArgs& a, const Views& v, int p, int iw, int nwp, char* t0,
                                            char* t1, char* misc) {
    if constexpr (sizeof(T) == 2)
        attend_mfma<D, DENSE, FUSED, PT>(a, v, p, iw, nwp, t0, t1, misc);
    else
        attend_f32<D, DENSE, PT>(a, v, p, iw, nwp, t0, misc);
    combine_and_merge<D, FUSED>(a, v, p, iw, nwp, t0);
}

// Phase B and C for every pair this workgroup serves: pair w mod BH (or the
// pairs w, w + grid, ... when there are more pairs than workgroups).  The
// plan passes cover HK teams per thread when the heads' union fits one
// pass's records (G K <= kPlanRecs), else one team per thread.
template <typename T, int D, int HK, bool DENSE, bool FUSED>
__device__ __forceinline__ void attend_all(const DecodeArgs& a, const Views& v, char* t0, char* t1, char* misc) {
    const int w = blockIdx.x, nwg = gridDim.x;
    const int BH = a.B * a.Hkv;
    auto one = [&](int p, int iw, int nwp) {
        if (HK > 1 && !DENSE && static_cast<long long>(a.G) * a.Kp <= kPlanRecs)
            attend_pair<T, D, DENSE, FUSED, HK>(a, v, p, iw, nwp, t0, t1, misc);
        else
            attend_pair<T, D, DENSE, FUSED, 1>(a, v, p, iw, nwp, t0, t1, misc);
    };
    if (BH <= nwg) {
        const PairSlot sl = pair_slot(w, nwg, BH);
        one(sl.p, sl.iw, sl.nwp);
    } else {
        for (int p = w; p < BH; p += nwg) one(p, 0, 1);
    }
}

// MODE kSample: one workgroup per (pair, head) task, placed so that the G
// heads of a pair share an XCD (workgroup w runs on XCD w mod 8): task
// (p, j) is workgroup 8 (G (p / 8) + j) + p mod 8.
// MODE kAttend: the attention grid.
// MODE kFused: the sampling tasks of workgroup w (the same placement, the
// grid's rows of eight workgroups reused), then its attention work.
template <typename T, int D, int HK, int MODE, bool DENSE>
__global__ __launch_bounds__(kThreads, 1) void k_decode(DecodeArgs a) {
    using L = Lds<T, D, HK>;
    __shared__ __attribute__((aligned(16))) char s_t0[L::t0];
    __shared__ __attribute__((aligned(16))) char s_t1[L::t1];
    __shared__ __attribute__((aligned(16))) char s_misc[L::misc];
    const Views v = views_of(a);
    const int w = blockIdx.x, nwg = gridDim.x;
    const int BH = a.B * a.Hkv, G = a.G;
    if constexpr (MODE == kSample) {
        const int q = w >> 3, p = 8 * (q / G) + (w & 7), j = q % G;
        if (p < BH) sample_head<T, D, HK, false>(a, v, p, j, s_t0, s_t1, s_misc);
    } else {
        if constexpr (MODE == kFused && !DENSE) {
            const int rows = (BH + 7) / 8 * G;
            for (int q = w >> 3; q < rows; q += nwg >> 3) {
                const int p = 8 * (q / G) + (w & 7), j = q % G;
                if (p < BH) sample_head<T, D, HK, true>(a, v, p, j, s_t0, s_t1, s_misc);
            }
        }
        attend_all<T, D, HK, DENSE, MODE == kFused>(a, v, s_t0, s_t1, s_misc);
    }
}

// The merge launch of the split mode: one workgroup per (pair, head), over
// the states the attention launch published.
template <int D>
__global__ __launch_bounds__(kThreads) void k_merge(DecodeArgs a) {
    constexpr int NSL = kThreads / (D / 4);
    __shared__ float4 s_acc[kThreads];
    __shared__ float2 s_ml[NSL];
    const Views v = views_of(a);
    const int BH = a.B * a.Hkv, G = a.G, nwg = a.lay.nwg;
    const int p = blockIdx.x / G, h = blockIdx.x - p * G;
    const int nwp = BH <= nwg ? pair_wgs(p, nwg, BH) : 1;
    const float* part_p = v.part + static_cast<size_t>(p) * a.lay.maxwp * G * state_stride(D);
    merge_head<D, false>(a, part_p, p, h, nwp, true, s_acc, s_ml);
}

__global__ void k_zero(uint4* __restrict__ p, size_t n16, unsigned char* __restrict__ tail, int ntail) {
    const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < n16; i += stride)
        p[i] = make_uint4(0, 0, 0, 0);
    if (blockIdx.x == 0 && static_cast<int>(threadIdx.x) < ntail) tail[threadIdx.x] = 0;
}

// Launch a kernel; with stage events, the launch itself stamps them at the
// kernel's start and end (so they time the kernel's execution, not the
// dispatch gap before it).
template <typename F>
hipError_t launch_one(const DecodeArgs& a, F kernel, int grid, bool timed, hipStream_t s) {
    if (timed && (a.ev_start || a.ev_stop))
        hipExtLaunchKernelGGL(kernel, dim3(grid), dim3(kThreads), 0, s, a.ev_start, a.ev_stop, 0, a);
    else
        hipLaunchKernelGGL(kernel, dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

template <int D>
hipError_t launch_merge(const DecodeArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(k_merge<D>, dim3(a.B * a.Hkv * a.G), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

template <typename T, int D, int HK>
hipError_t decode_sampled(const DecodeArgs& a, hipStream_t s) {
    const int BH = a.B * a.Hkv;
    if (a.fused) {
        if constexpr (sizeof(T) == 2)
            return launch_one(a, k_decode<T, D, HK, kFused, false>, a.lay.nwg, true, s);
        return hipErrorInvalidValue;
    }
    const int tasks = 8 * ((BH + 7) / 8) * a.G;
    hipError_t e = launch_one(a, k_decode<T, D, HK, kSample, false>, tasks, false, s);
    if (e == hipSuccess) e = launch_one(a, k_decode<T, D, HK, kAttend, false>, a.lay.nwg, true, s);
    if (e == hipSuccess) e = launch_merge<D>(a, s);
    return e;
}

// The single-launch step (bf16): keys per lane of the selecting waves by the
// team count.
template <int D>
hipError_t decode_step(const DecodeArgs& a, hipStream_t s) {
    const int grid = a.lay.nwg;
    if (a.dense) return launch_one(a, k_step<D, 2, true>, grid, true, s);
    if (a.M <= 128) return launch_one(a, k_step<D, 2, false>, grid, true, s);
    if (a.M <= kStepMaxTeams) return launch_one(a, k_step<D, 8, false>, grid, true, s);
    return hipErrorInvalidValue;
}

template <typename T, int D>
hipError_t decode_d(const DecodeArgs& a, hipStream_t s) {
    if constexpr (sizeof(T) == 2) {
        if (a.lay.step) return decode_step<D>(a, s);
    }
    if (a.dense) {
        if (a.fused) {
            if constexpr (sizeof(T) == 2)
                return launch_one(a, k_decode<T, D, 1, kFused, true>, a.lay.nwg, true, s);
            return hipErrorInvalidValue;
        }
        hipError_t e = launch_one(a, k_decode<T, D, 1, kAttend, true>, a.lay.nwg, true, s);
        if (e == hipSuccess) e = launch_merge<D>(a, s);
        return e;
    }
    if (a.M <= kThreads) return decode_sampled<T, D, 1>(a, s);
    if (a.M <= 4 * kThreads) return decode_sampled<T, D, 4>(a, s);
    if (a.M <= 16 * kThreads) return decode_sampled<T, D, 16>(a, s);
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, hipStream_t s) {
    if (a.dtype == SANTAPP_BF16) {
        if (a.d == 128) return decode_d<bf16_t, 128>(a, s);
        if (a.d == 64) return decode_d<bf16_t, 64>(a, s);
    } else {
        if (a.d == 128) return decode_d<float, 128>(a, s);
        if (a.d == 64) return decode_d<float, 64>(a, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
    const size_t n16 = bytes / 16;
    const int ntail = static_cast<int>(bytes - n16 * 16);
    const size_t want = (n16 + 255) / 256;
    const unsigned blocks = static_cast<unsigned>(want == 0 ? 1 : (want < 4096 ? want : 4096));
    k_zero<<<blocks, 256, 0, s>>>(static_cast<uint4*>(p), n16, static_cast<unsigned char*>(p) + n16 * 16, ntail);
    return hipGetLastError();
}

}  // namespace santapp
