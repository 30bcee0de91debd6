// C ABI of libsantapp: argument checks, buffer ownership, workspace layout and
// launch sequencing.  All arithmetic runs in the kernels.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <functional>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

struct santapp_teams {
    int B, Hkv, N, d;
    santapp_dtype dtype;
    int P, R, M;
    void* packed_K;
    void* packed_V;
    void* reps;
    int* team_begin;
    int* team_size;
    double* log_n;
    int* rep_token;
    int* perm;
    int* team_count;  // [B*Hkv] teams of each pair (M for contiguous parents)
    void* block;      // the one device allocation every array above is carved from
    // cap[x]: the most attention chunks any x distinct teams of one (b, kv)
    // need (sum of their x largest chunk counts, maximum over (b, kv))
    std::vector<int> cap;
    int cus;  // compute units of the device the handle was built on
};

namespace {

thread_local std::string g_err;

santapp_status fail(santapp_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

santapp_status ok() {
    g_err.clear();
    return SANTAPP_OK;
}

santapp_status hip_fail(hipError_t e, const char* what) {
    return fail(SANTAPP_EHIP, "%s: %s", what, hipGetErrorString(e));
}

size_t elem_size(santapp_dtype dt) { return dt == SANTAPP_BF16 ? 2 : 4; }

bool dtype_ok(santapp_dtype dt) { return dt == SANTAPP_BF16 || dt == SANTAPP_FP32; }

size_t align_up(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

constexpr int kWaves8 = santapp::kDecodeThreads / 64;  // waves of a decode workgroup

// Device buffers are read and written with 16-byte vector accesses.
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Compute units of the current device (0 if the query fails), looked up once
// per device.
int device_cus() {
    constexpr int kDevs = 64;
    static std::atomic<int> cache[kDevs];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    if (dev < 0 || dev >= kDevs) return 0;
    int n = cache[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 0) {
        (void)hipGetLastError();
        return 0;
    }
    cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

// Teams per (b, kv) for contiguous parents: every parent but the last has P
// members and min(R, P) teams.
long long team_count(int N, int P, int R) {
    const long long np = (static_cast<long long>(N) + P - 1) / P;
    const long long last = N - (np - 1) * static_cast<long long>(P);
    return (np - 1) * std::min<long long>(R, P) + std::min<long long>(R, last);
}

// Release device memory on clean-up paths, where a failure to free cannot be
// reported any better than the error already being returned.
void release(void* p) {
    if (p) (void)hipFree(p);
}

void free_teams(santapp_teams* t) {
    if (!t) return;
    release(t->block);
    delete t;
}

santapp_status finish_table(santapp_teams* t, hipStream_t s, santapp_teams** out);

}  // namespace

namespace santapp {

int decode_wgs(int cus, long long BH, long long units_per_pair) {
    if (cus < 1) cus = 8;
    long long want = (BH * units_per_pair + kWaves8 - 1) / kWaves8;  // a unit per wave
    want = std::max<long long>(want, std::min<long long>(BH, cus));   // every pair a workgroup
    want = std::min<long long>(want, cus);
    if (cus % 8 == 0) want = std::min<long long>(cus, (want + 7) / 8 * 8);
    return static_cast<int>(std::max<long long>(want, 1));
}

namespace {

struct Carver {
    size_t off = 0;
    size_t take(size_t bytes) {
        const size_t at = off;
        off = align_up(off + bytes);
        return at;
    }
};

// Every device array of a table (t->B, Hkv, N, M, d and dtype set) from one
// allocation, each 256-byte aligned.
hipError_t alloc_table(santapp_teams* t) {
    const size_t BH = static_cast<size_t>(t->B) * t->Hkv;
    const size_t N = static_cast<size_t>(t->N), M = static_cast<size_t>(t->M);
    const size_t row = static_cast<size_t>(t->d) * elem_size(t->dtype);
    Carver c;
    const size_t oK = c.take(BH * N * row), oV = c.take(BH * N * row), oR = c.take(BH * M * row);
    const size_t ob = c.take(BH * M * sizeof(int)), os = c.take(BH * M * sizeof(int));
    const size_t ol = c.take(BH * M * sizeof(double)), ot = c.take(BH * M * sizeof(int));
    const size_t op = c.take(BH * N * sizeof(int)), oc = c.take(BH * sizeof(int));
    char* b = nullptr;
    const hipError_t e = hipMalloc(reinterpret_cast<void**>(&b), c.off);
    if (e != hipSuccess) return e;
    t->block = b;
    t->packed_K = b + oK;
    t->packed_V = b + oV;
    t->reps = b + oR;
    t->team_begin = reinterpret_cast<int*>(b + ob);
    t->team_size = reinterpret_cast<int*>(b + os);
    t->log_n = reinterpret_cast<double*>(b + ol);
    t->rep_token = reinterpret_cast<int*>(b + ot);
    t->perm = reinterpret_cast<int*>(b + op);
    t->team_count = reinterpret_cast<int*>(b + oc);
    return hipSuccess;
}

}  // namespace

namespace {

// Launch mode asked for by SANTAPP_DECODE_LAUNCH (read once per process):
// "split" or "fused" take the three-launch kernels (fused: in one launch);
// anything else takes the single-launch step wherever it applies.
enum class LaunchMode { kStep, kSplit, kFused };

LaunchMode launch_mode() {
    static const LaunchMode m = [] {
        const char* e = getenv("SANTAPP_DECODE_LAUNCH");
        if (e != nullptr && strcmp(e, "fused") == 0) return LaunchMode::kFused;
        if (e != nullptr && strcmp(e, "split") == 0) return LaunchMode::kSplit;
        return LaunchMode::kStep;
    }();
    return m;
}

// The single-launch step's own workspace: epochs, the tagged exchange words
// (sampled steps) and the tagged partial states.
void step_regions(DecodeLayout& L, size_t BH, int G, int M, int d, bool dense, size_t& off) {
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = (off + bytes + 255) & ~static_cast<size_t>(255);
        return at;
    };
    L.epoch = take(BH * sizeof(uint32_t));
    if (!dense) {
        L.xk = take(BH * G * 3 * static_cast<size_t>(M) * 8);
    }
    L.part = take(BH * L.maxwp * G * static_cast<size_t>(step_state_bytes(d)));
}

bool fused_wanted() { return launch_mode() == LaunchMode::kFused; }

}  // namespace

bool step_mode(santapp_dtype dt, int d, long long BH, int M, int Kp, bool dense, int cus) {
    if (launch_mode() != LaunchMode::kStep) return false;
    if (dt != SANTAPP_BF16 || (d != 64 && d != 128) || cus < 8 || BH < 1 || BH > cus) return false;
    return dense || (M <= kStepMaxTeams && Kp <= kStepMaxKp);
}

int step_wgs(int cus, long long BH) {
    if (cus % 8 == 0 && BH * 8 <= cus) {
        const long long per = std::min<long long>(kStepMaxWgs, 8 * (cus / (8 * BH)));
        return static_cast<int>(BH * per);
    }
    return static_cast<int>(BH * std::min<long long>(kStepMaxWgs, cus / BH));
}

DecodeLayout decode_layout(int B, int Hq, int Hkv, int T, int d, int M, int Kp, const int* cap, int cus,
                           santapp_dtype dt) {
    DecodeLayout L;
    const size_t BH = static_cast<size_t>(B) * Hkv, BQ = static_cast<size_t>(B) * Hq;
    const int G = Hq / Hkv;
    if (step_mode(dt, d, static_cast<long long>(BH), M, Kp, false, cus)) {
        L.step = true;
        L.nwg = step_wgs(cus, static_cast<long long>(BH));
        L.maxwp = pair_wgs(0, L.nwg, static_cast<int>(BH));
        L.swords = (M + 63) / 64;
        size_t off = 0;
        step_regions(L, BH, G, M, d, false, off);
        L.total = off;
        return L;
    }
    const long long xs = std::min<long long>(M, static_cast<long long>(G) * Kp);
    L.nwg = decode_wgs(cus, static_cast<long long>(BH), chunk_count(T) + static_cast<long long>(std::max(1, cap[xs])));
    L.maxwp = BH <= static_cast<size_t>(L.nwg) ? pair_wgs(0, L.nwg, static_cast<int>(BH)) : 1;
    L.swords = (M + 63) / 64;
    Carver c;
    L.ctr = c.take((BH + BH * G) * sizeof(int));
    L.sbits = c.take(BQ * L.swords * sizeof(uint64_t));
    L.lc = c.take(BQ * M * sizeof(float));
    L.part = c.take(BH * L.maxwp * G * state_stride(d) * sizeof(float));
    L.total = c.off;
    return L;
}

DecodeLayout dense_layout(int B, int Hq, int Hkv, int N, int T, int d, int cus, santapp_dtype dt) {
    DecodeLayout L;
    const size_t BH = static_cast<size_t>(B) * Hkv;
    const int G = Hq / Hkv;
    if (step_mode(dt, d, static_cast<long long>(BH), 0, 0, true, cus)) {
        L.step = true;
        L.nwg = step_wgs(cus, static_cast<long long>(BH));
        L.maxwp = pair_wgs(0, L.nwg, static_cast<int>(BH));
        size_t off = 0;
        step_regions(L, BH, G, 0, d, true, off);
        L.total = off;
        return L;
    }
    L.nwg = decode_wgs(cus, static_cast<long long>(BH), chunk_count(N) + static_cast<long long>(chunk_count(T)));
    L.maxwp = BH <= static_cast<size_t>(L.nwg) ? pair_wgs(0, L.nwg, static_cast<int>(BH)) : 1;
    Carver c;
    L.ctr = c.take((BH + BH * G) * sizeof(int));
    L.part = c.take(BH * L.maxwp * G * state_stride(d) * sizeof(float));
    L.total = c.off;
    return L;
}

}  // namespace santapp

using namespace santapp;

extern "C" {

const char* santapp_last_error(void) { return g_err.c_str(); }

santapp_status santapp_budget_to_K(int S, int P, int R, int M, int* K) {
    if (!K) return fail(SANTAPP_EINVAL, "K is NULL");
    if (S < 1 || P < 1 || R < 1 || M < 1)
        return fail(SANTAPP_EINVAL, "S, P, R and M must be positive (got %d, %d, %d, %d)", S, P, R, M);
    if (P % R != 0) return fail(SANTAPP_EINVAL, "P (%d) must be divisible by R (%d)", P, R);
    const int per = P / R;
    if (S % per != 0) return fail(SANTAPP_EINVAL, "S (%d) must be divisible by P/R (%d)", S, per);
    *K = std::min(M, S / per);
    return ok();
}

santapp_status santapp_build_teams(const void* K, const void* V, int B, int Hkv, int N, int d,
                                   santapp_dtype dtype, int parent_size, int reps_per_parent,
                                   void* stream, santapp_teams** out) {
    if (!out) return fail(SANTAPP_EINVAL, "out is NULL");
    *out = nullptr;
    if (!K || !V) return fail(SANTAPP_EINVAL, "K and V must be device pointers");
    if (!aligned16(K) || !aligned16(V)) return fail(SANTAPP_EINVAL, "K and V must be 16-byte aligned");
    if (B < 1 || Hkv < 1 || N < 1) return fail(SANTAPP_EINVAL, "B, Hkv, N must be >= 1");
    if (parent_size < 1) return fail(SANTAPP_EINVAL, "parent_size must be >= 1");
    if (reps_per_parent < 1) return fail(SANTAPP_EINVAL, "reps_per_parent must be >= 1");
    if (!dtype_ok(dtype)) return fail(SANTAPP_EDTYPE, "unsupported dtype %d", static_cast<int>(dtype));
    if (d != 64 && d != 128) return fail(SANTAPP_ELIMIT, "head dim %d not supported (64 or 128)", d);
    if (reps_per_parent > kMaxReps)
        return fail(SANTAPP_ELIMIT, "reps_per_parent %d exceeds %d", reps_per_parent, kMaxReps);
    const long long M = team_count(N, parent_size, reps_per_parent);
    const size_t BH = static_cast<size_t>(B) * Hkv;
    if (BH * static_cast<size_t>(N) > static_cast<size_t>(0x7fffffff))
        return fail(SANTAPP_ELIMIT, "B*Hkv*N exceeds 2^31");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const size_t esz = elem_size(dtype);
    const size_t row = static_cast<size_t>(d) * esz;

    santapp_teams* t = new santapp_teams();
    t->B = B;
    t->Hkv = Hkv;
    t->N = N;
    t->d = d;
    t->dtype = dtype;
    t->P = parent_size;
    t->R = reps_per_parent;
    t->M = static_cast<int>(M);
    double* mind = nullptr;
    int* owner = nullptr;
    hipError_t e = alloc_table(t);
    auto alloc = [&](void** p, size_t bytes) {
        if (e == hipSuccess) e = hipMalloc(p, bytes);
    };
    if (!build_packs_in_place(N, d, dtype, parent_size, reps_per_parent)) {
        // running minimum and owner per token, for the general build kernel
        alloc(reinterpret_cast<void**>(&mind), BH * N * sizeof(double));
        alloc(reinterpret_cast<void**>(&owner), BH * N * sizeof(int));
    }
    if (e != hipSuccess) {
        release(mind);
        release(owner);
        free_teams(t);
        (void)hipGetLastError();
        return fail(SANTAPP_ENOMEM, "device allocation failed: %s", hipGetErrorString(e));
    }
    const char* what = "team build";
    bool packed = false;
    e = launch_build_parents(K, V, dtype, static_cast<int>(BH), N, d, parent_size, reps_per_parent,
                             t->M, mind, owner, t->team_begin, t->team_size, t->log_n,
                             t->rep_token, t->perm, t->packed_K, t->packed_V, t->reps, t->team_count,
                             &packed, s);
    if (e == hipSuccess && !packed) {
        what = "packing K";
        e = launch_gather_rows(K, t->packed_K, t->perm, static_cast<int>(BH), N, N, row, s);
    }
    if (e == hipSuccess && !packed) {
        what = "packing V";
        e = launch_gather_rows(V, t->packed_V, t->perm, static_cast<int>(BH), N, N, row, s);
    }
    if (e == hipSuccess && !packed) {
        what = "gathering representatives";
        e = launch_gather_rows(K, t->reps, t->rep_token, static_cast<int>(BH), t->M, N, row, s);
    }
    if (e != hipSuccess) {
        // a launch failed: nothing of this call is left queued that uses the
        // buffers (hipFree waits for the device)
        release(mind);
        release(owner);
        free_teams(t);
        return hip_fail(e, what);
    }
    const santapp_status st = finish_table(t, s, out);  // waits for the build
    release(mind);
    release(owner);
    return st;
}

namespace {

// Waits for the build queued on s, then sets the chunk capacities and the
// device's compute units of the table; frees it on failure.
santapp_status finish_table(santapp_teams* t, hipStream_t s, santapp_teams** out) {
    const size_t BH = static_cast<size_t>(t->B) * t->Hkv;
    std::vector<int> sizes(BH * t->M);
    hipError_t e = hipMemcpyAsync(sizes.data(), t->team_size, sizes.size() * sizeof(int), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        free_teams(t);
        return hip_fail(e, "team build");
    }
    int dev = 0;
    t->cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&t->cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        t->cus = 0;
    (void)hipGetLastError();
    t->cap.assign(t->M + 1, 0);
    std::vector<int> cnt(t->M);
    for (size_t bh = 0; bh < BH; ++bh) {
        for (int g = 0; g < t->M; ++g) cnt[g] = chunk_count(sizes[bh * t->M + g]);
        std::sort(cnt.begin(), cnt.end(), std::greater<int>());
        int run = 0;
        for (int x = 1; x <= t->M; ++x) {
            run += cnt[x - 1];
            t->cap[x] = std::max(t->cap[x], run);
        }
    }
    *out = t;
    return ok();
}

}  // namespace

santapp_status santapp_kmeans_parents(const void* K, int B, int Hkv, int N, int d, santapp_dtype dtype,
                                      int parent_size, const santapp_kmeans_settings* theta, int* labels,
                                      int* num_parents, int* steps, void* stream) {
    if (!K || !labels || !theta) return fail(SANTAPP_EINVAL, "K, labels and theta must not be NULL");
    if (!aligned16(K) || !aligned16(labels)) return fail(SANTAPP_EINVAL, "K and labels must be 16-byte aligned");
    if (B < 1 || Hkv < 1 || N < 2) return fail(SANTAPP_EINVAL, "B, Hkv must be >= 1 and N >= 2");
    if (parent_size < 1) return fail(SANTAPP_EINVAL, "parent_size must be >= 1");
    if (theta->batch_size < 1 || theta->max_iter < 0 || theta->max_no_improvement < 0 ||
        theta->init_size < 0 || !(theta->reassignment_ratio >= 0.0 && theta->reassignment_ratio < 1.0))
        return fail(SANTAPP_EINVAL, "invalid k-means settings");
    if (!dtype_ok(dtype)) return fail(SANTAPP_EDTYPE, "unsupported dtype %d", static_cast<int>(dtype));
    if (d != 64 && d != 128) return fail(SANTAPP_ELIMIT, "head dim %d not supported (64 or 128)", d);
    const int M = std::min(N, std::max(2, N / parent_size));
    if (M > kKmMaxCenters) return fail(SANTAPP_ELIMIT, "%d k-means parents exceed %d", M, kKmMaxCenters);
    const size_t BH = static_cast<size_t>(B) * Hkv;
    if (BH * static_cast<size_t>(N) > static_cast<size_t>(0x7fffffff))
        return fail(SANTAPP_ELIMIT, "B*Hkv*N exceeds 2^31");
    const long long steps_total = static_cast<long long>(theta->max_iter) * N / theta->batch_size;
    if (steps_total > 0x7fffffff) return fail(SANTAPP_ELIMIT, "too many minibatch steps");
    int s0 = theta->init_size > 0 ? theta->init_size : 3 * theta->batch_size;
    if (s0 < M) s0 = 3 * M;
    if (s0 > N) s0 = N;
    const KmLayout L = kmeans_layout(static_cast<int>(BH), N, d, M, theta->batch_size, s0);
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* ws = nullptr;
    hipError_t e = hipMalloc(reinterpret_cast<void**>(&ws), L.total);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(SANTAPP_ENOMEM, "k-means scratch (%zu bytes): %s", L.total, hipGetErrorString(e));
    }
    const char* what = "k-means seeding";
    e = launch_kmeans_seed(K, dtype, static_cast<int>(BH), N, d, L, ws, theta->seed, s);
    const double alpha = std::min(1.0, 2.0 * theta->batch_size / (static_cast<double>(N) + 1.0));
    std::vector<KmState> st(BH);
    // minibatch steps in groups; stopped pairs skip the rest, and the loop
    // ends once every pair has stopped
    constexpr int kGroup = 16;
    for (long long first = 0; e == hipSuccess && first < steps_total; first += kGroup) {
        const int count = static_cast<int>(std::min<long long>(kGroup, steps_total - first));
        what = "k-means steps";
        e = launch_kmeans_steps(K, dtype, static_cast<int>(BH), N, d, L, ws, theta->batch_size,
                                static_cast<int>(first), count, alpha, theta->reassignment_ratio,
                                theta->max_no_improvement, theta->seed, s);
        if (e == hipSuccess && theta->max_no_improvement > 0) {
            what = "k-means state";
            e = hipMemcpyAsync(st.data(), ws + L.state, BH * sizeof(KmState), hipMemcpyDeviceToHost, s);
            if (e == hipSuccess) e = hipStreamSynchronize(s);
            if (e == hipSuccess &&
                std::all_of(st.begin(), st.end(), [](const KmState& x) { return x.stop != 0; }))
                break;
        }
    }
    if (e == hipSuccess) {
        what = "k-means labels";
        e = launch_kmeans_labels(K, dtype, static_cast<int>(BH), N, d, L, ws, labels, s);
    }
    if (e == hipSuccess) {
        what = "k-means state";
        e = hipMemcpyAsync(st.data(), ws + L.state, BH * sizeof(KmState), hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
    }
    release(ws);
    if (e != hipSuccess) return hip_fail(e, what);
    if (num_parents) *num_parents = M;
    if (steps)
        for (size_t i = 0; i < BH; ++i) steps[i] = st[i].steps;
    return ok();
}

santapp_status santapp_build_teams_from_labels(const void* K, const void* V, int B, int Hkv, int N, int d,
                                               santapp_dtype dtype, const int* labels, int num_labels,
                                               int reps_per_parent, void* stream, santapp_teams** out) {
    if (!out) return fail(SANTAPP_EINVAL, "out is NULL");
    *out = nullptr;
    if (!K || !V || !labels) return fail(SANTAPP_EINVAL, "K, V and labels must be device pointers");
    if (!aligned16(K) || !aligned16(V) || !aligned16(labels))
        return fail(SANTAPP_EINVAL, "K, V and labels must be 16-byte aligned");
    if (B < 1 || Hkv < 1 || N < 1) return fail(SANTAPP_EINVAL, "B, Hkv, N must be >= 1");
    if (num_labels < 1) return fail(SANTAPP_EINVAL, "num_labels must be >= 1");
    if (reps_per_parent < 1) return fail(SANTAPP_EINVAL, "reps_per_parent must be >= 1");
    if (!dtype_ok(dtype)) return fail(SANTAPP_EDTYPE, "unsupported dtype %d", static_cast<int>(dtype));
    if (d != 64 && d != 128) return fail(SANTAPP_ELIMIT, "head dim %d not supported (64 or 128)", d);
    if (num_labels > kMaxLabels) return fail(SANTAPP_ELIMIT, "num_labels %d exceeds %d", num_labels, kMaxLabels);
    if (reps_per_parent > kMaxReps)
        return fail(SANTAPP_ELIMIT, "reps_per_parent %d exceeds %d", reps_per_parent, kMaxReps);
    const size_t BH = static_cast<size_t>(B) * Hkv;
    if (BH * static_cast<size_t>(N) > static_cast<size_t>(0x7fffffff))
        return fail(SANTAPP_ELIMIT, "B*Hkv*N exceeds 2^31");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const size_t esz = elem_size(dtype);
    const size_t row = static_cast<size_t>(d) * esz;
    const int Mp = num_labels;

    // parent lists, then the team counts that size the table; the build's
    // scratch arrays are carved from one allocation
    Carver sc;
    const size_t o_mem = sc.take(BH * N * sizeof(int)), o_pbeg = sc.take(BH * (Mp + 1) * sizeof(int));
    const size_t o_toff = sc.take(BH * (Mp + 1) * sizeof(int)), o_tcount = sc.take(BH * sizeof(int));
    const size_t o_bad = sc.take(sizeof(int)), o_mind = sc.take(BH * N * sizeof(double));
    const size_t o_owner = sc.take(BH * N * sizeof(int));
    char* scratch = nullptr;
    hipError_t e = hipMalloc(reinterpret_cast<void**>(&scratch), sc.off);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(SANTAPP_ENOMEM, "device allocation failed: %s", hipGetErrorString(e));
    }
    auto cleanup = [&]() { release(scratch); };
    int* members = reinterpret_cast<int*>(scratch + o_mem);
    int* pbeg = reinterpret_cast<int*>(scratch + o_pbeg);
    int* toff = reinterpret_cast<int*>(scratch + o_toff);
    int* tcount = reinterpret_cast<int*>(scratch + o_tcount);
    int* bad = reinterpret_cast<int*>(scratch + o_bad);
    double* mind = reinterpret_cast<double*>(scratch + o_mind);
    int* owner = reinterpret_cast<int*>(scratch + o_owner);
    const char* what = "parent lists";
    e = hipMemsetAsync(bad, 0, sizeof(int), s);
    if (e == hipSuccess)
        e = launch_parent_lists(labels, static_cast<int>(BH), N, Mp, reps_per_parent, members, pbeg, toff,
                                tcount, bad, s);
    std::vector<int> counts(BH);
    int flag = 0;
    if (e == hipSuccess) e = hipMemcpyAsync(counts.data(), tcount, BH * sizeof(int), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(&flag, bad, sizeof(int), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        cleanup();
        return hip_fail(e, what);
    }
    if (flag) {
        cleanup();
        return fail(SANTAPP_EINVAL, "a label lies outside [0, %d)", Mp);
    }
    const int M = *std::max_element(counts.begin(), counts.end());

    santapp_teams* t = new santapp_teams();
    t->B = B;
    t->Hkv = Hkv;
    t->N = N;
    t->d = d;
    t->dtype = dtype;
    t->P = 0;
    t->R = reps_per_parent;
    t->M = M;
    e = alloc_table(t);
    if (e != hipSuccess) {
        cleanup();
        free_teams(t);
        (void)hipGetLastError();
        return fail(SANTAPP_ENOMEM, "device allocation failed: %s", hipGetErrorString(e));
    }
    what = "team counts";
    e = hipMemcpyAsync(t->team_count, tcount, BH * sizeof(int), hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess) {
        what = "absent teams";
        e = launch_pad_teams(tcount, static_cast<int>(BH), M, N, t->team_begin, t->team_size, t->log_n,
                             t->rep_token, s);
    }
    if (e == hipSuccess) {
        what = "team build";
        e = launch_build_parent_lists(K, dtype, static_cast<int>(BH), N, d, Mp, reps_per_parent, M, members,
                                      pbeg, toff, mind, owner, t->team_begin, t->team_size, t->log_n,
                                      t->rep_token, t->perm, s);
    }
    if (e == hipSuccess) {
        what = "packing K";
        e = launch_gather_rows(K, t->packed_K, t->perm, static_cast<int>(BH), N, N, row, s);
    }
    if (e == hipSuccess) {
        what = "packing V";
        e = launch_gather_rows(V, t->packed_V, t->perm, static_cast<int>(BH), N, N, row, s);
    }
    if (e == hipSuccess) {
        what = "gathering representatives";
        e = launch_gather_rows(K, t->reps, t->rep_token, static_cast<int>(BH), M, N, row, s);
    }
    if (e != hipSuccess) {
        cleanup();
        free_teams(t);
        return hip_fail(e, what);
    }
    const santapp_status st = finish_table(t, s, out);  // waits for the build
    cleanup();
    return st;
}

santapp_status santapp_teams_info(const santapp_teams* t, santapp_teams_desc* d) {
    if (!t || !d) return fail(SANTAPP_EINVAL, "NULL argument");
    d->B = t->B;
    d->Hkv = t->Hkv;
    d->N = t->N;
    d->d = t->d;
    d->dtype = t->dtype;
    d->parent_size = t->P;
    d->reps_per_parent = t->R;
    d->M = t->M;
    d->packed_K = t->packed_K;
    d->packed_V = t->packed_V;
    d->reps = t->reps;
    d->team_begin = t->team_begin;
    d->team_size = t->team_size;
    d->log_n = t->log_n;
    d->rep_token = t->rep_token;
    d->perm = t->perm;
    d->team_count = t->team_count;
    return ok();
}

void santapp_teams_destroy(santapp_teams* t) { free_teams(t); }

santapp_status santapp_teams_set_route_keys(santapp_teams* t, santapp_route_key kind, void* stream) {
    if (!t) return fail(SANTAPP_EINVAL, "teams is NULL");
    if (kind != SANTAPP_ROUTE_REPRESENTATIVE && kind != SANTAPP_ROUTE_CENTROID)
        return fail(SANTAPP_EINVAL, "unknown routing key kind %d", static_cast<int>(kind));
    const hipError_t e = launch_route_keys(t->packed_K, t->team_begin, t->team_size, t->rep_token, t->perm,
                                           t->B * t->Hkv, t->N, t->M, t->d, t->dtype,
                                           kind == SANTAPP_ROUTE_CENTROID, t->reps, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ok() : hip_fail(e, "routing keys");
}

namespace {

// KL workspace: phi, Y (unused by the diagnostic, written by the routing
// kernel) and the per-team sums, each [B, Hq, M].
struct KlLayout {
    size_t phi, Y, part, total;
};

KlLayout kl_layout(int B, int Hq, int M) {
    const size_t n = static_cast<size_t>(B) * Hq * M;
    KlLayout L;
    L.phi = 0;
    L.Y = align_up(L.phi + n * sizeof(double));
    L.part = align_up(L.Y + n * sizeof(double));
    L.total = align_up(L.part + n * kl_part_bytes());
    return L;
}

}  // namespace

santapp_status santapp_routing_kl_workspace_bytes(const santapp_teams* t, int Hq, size_t* bytes) {
    if (!t || !bytes) return fail(SANTAPP_EINVAL, "NULL argument");
    if (Hq < 1 || Hq % t->Hkv != 0) return fail(SANTAPP_EINVAL, "Hq must be a positive multiple of Hkv");
    *bytes = kl_layout(t->B, Hq, t->M).total;
    return ok();
}

santapp_status santapp_routing_kl(const santapp_teams* t, const float* q, int Hq, double scale, double* kl,
                                  void* workspace, size_t ws_bytes, void* stream) {
    if (!t) return fail(SANTAPP_EINVAL, "teams is NULL");
    if (!q || !kl) return fail(SANTAPP_EINVAL, "q and kl must be device pointers");
    if (Hq < 1 || Hq % t->Hkv != 0) return fail(SANTAPP_EINVAL, "Hq (%d) must be a positive multiple of Hkv (%d)", Hq, t->Hkv);
    if (Hq / t->Hkv > kMaxGroup) return fail(SANTAPP_ELIMIT, "%d query heads per KV head exceed %d", Hq / t->Hkv, kMaxGroup);
    if (!(scale >= 0.0) || !isfinite(scale)) return fail(SANTAPP_EINVAL, "scale must be finite and >= 0");
    if (scale == 0.0) scale = 1.0 / sqrt(static_cast<double>(t->d));
    const KlLayout L = kl_layout(t->B, Hq, t->M);
    if (!workspace || ws_bytes < L.total)
        return fail(SANTAPP_EWORKSPACE, "workspace of %zu bytes needed (got %zu)", L.total, ws_bytes);
    if (!aligned16(q) || !aligned16(kl) || !aligned16(workspace))
        return fail(SANTAPP_EINVAL, "q, kl and workspace must be 16-byte aligned");
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* ws = static_cast<char*>(workspace);
    double* phi = reinterpret_cast<double*>(ws + L.phi);
    RouteArgs R{};
    R.reps = t->reps;
    R.log_n = t->log_n;
    R.q = q;
    R.B = t->B;
    R.Hkv = t->Hkv;
    R.Hq = Hq;
    R.G = Hq / t->Hkv;
    R.d = t->d;
    R.M = t->M;
    R.dtype = t->dtype;
    R.scale = scale;
    hipError_t e = launch_route_phi(R, phi, reinterpret_cast<double*>(ws + L.Y), s);
    if (e != hipSuccess) return hip_fail(e, "routing kernel");
    KlArgs A{};
    A.packed_K = t->packed_K;
    A.team_begin = t->team_begin;
    A.team_size = t->team_size;
    A.log_n = t->log_n;
    A.q = q;
    A.phi = phi;
    A.part = ws + L.part;
    A.kl = kl;
    A.B = t->B;
    A.Hkv = t->Hkv;
    A.Hq = Hq;
    A.N = t->N;
    A.M = t->M;
    A.d = t->d;
    A.dtype = t->dtype;
    A.scale = scale;
    e = launch_routing_kl(A, s);
    return e == hipSuccess ? ok() : hip_fail(e, "KL kernels");
}

santapp_status santapp_workspace_zero(void* ws, size_t bytes, void* stream) {
    if (bytes == 0) return ok();
    if (!ws) return fail(SANTAPP_EINVAL, "workspace is NULL");
    const hipError_t e = launch_zero(ws, bytes, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ok() : hip_fail(e, "workspace zero");
}

santapp_status santapp_decode_workspace_bytes(const santapp_teams* t, int Hq, int T, int K,
                                              size_t* bytes) {
    if (!t || !bytes) return fail(SANTAPP_EINVAL, "NULL argument");
    if (Hq < 1 || Hq % t->Hkv != 0) return fail(SANTAPP_EINVAL, "Hq must be a positive multiple of Hkv");
    if (T < 0 || K < 1) return fail(SANTAPP_EINVAL, "T must be >= 0 and K >= 1");
    const int Kp = std::min(K, t->M);
    *bytes = Kp == t->M ? dense_layout(t->B, Hq, t->Hkv, t->N, T, t->d, t->cus, t->dtype).total
                        : decode_layout(t->B, Hq, t->Hkv, T, t->d, t->M, Kp, t->cap.data(), t->cus, t->dtype).total;
    return ok();
}

santapp_status santapp_decode_launch_info(const santapp_teams* t, int Hq, int T, int K, int* kernels,
                                         int* workgroups) {
    if (!t || !kernels || !workgroups) return fail(SANTAPP_EINVAL, "NULL argument");
    if (Hq < 1 || Hq % t->Hkv != 0) return fail(SANTAPP_EINVAL, "Hq must be a positive multiple of Hkv");
    if (T < 0 || K < 1) return fail(SANTAPP_EINVAL, "T must be >= 0 and K >= 1");
    const int Kp = std::min(K, t->M);
    const bool dense = Kp == t->M;
    const DecodeLayout L = dense ? dense_layout(t->B, Hq, t->Hkv, t->N, T, t->d, t->cus, t->dtype)
                                 : decode_layout(t->B, Hq, t->Hkv, T, t->d, t->M, Kp, t->cap.data(), t->cus,
                                                 t->dtype);
    const bool fused = !L.step && t->dtype == SANTAPP_BF16 && fused_wanted() && L.nwg % 8 == 0;
    *kernels = L.step || fused ? 1 : (dense ? 2 : 3);
    *workgroups = L.nwg;
    return ok();
}

santapp_status santapp_dense_workspace_bytes(int B, int Hq, int Hkv, int N, int T, int d,
                                             size_t* bytes) {
    if (!bytes) return fail(SANTAPP_EINVAL, "NULL argument");
    if (B < 1 || Hkv < 1 || Hq < 1 || Hq % Hkv != 0 || N < 0 || T < 0 || N + T < 1 || d < 1)
        return fail(SANTAPP_EINVAL, "invalid sizes");
    // the larger of the two element types' layouts (the call's type is not an argument)
    const int cus = device_cus();
    *bytes = std::max(dense_layout(B, Hq, Hkv, N, T, d, cus, SANTAPP_BF16).total,
                      dense_layout(B, Hq, Hkv, N, T, d, cus, SANTAPP_FP32).total);
    return ok();
}

namespace {

santapp_status check_suffix(const void* sK, const void* sV, int T, int& stride) {
    if (T < 0) return fail(SANTAPP_EINVAL, "T must be >= 0");
    if (stride == 0) stride = T;
    if (stride < T) return fail(SANTAPP_EINVAL, "suffix_stride (%d) is smaller than T (%d)", stride, T);
    if (T > 0 && (!sK || !sV)) return fail(SANTAPP_EINVAL, "suffix K/V are NULL with T > 0");
    if (T > 0 && (!aligned16(sK) || !aligned16(sV))) return fail(SANTAPP_EINVAL, "suffix K/V must be 16-byte aligned");
    return SANTAPP_OK;
}

}  // namespace

santapp_status santapp_decode(const santapp_teams* t, const float* q, const void* suffix_K,
                              const void* suffix_V, int T, int suffix_stride, int Hq, int K, uint64_t seed,
                              uint64_t step, double scale, float* out, void* workspace,
                              size_t ws_bytes, const santapp_decode_debug* dbg, void* stream) {
    if (!t) return fail(SANTAPP_EINVAL, "teams is NULL");
    if (!q || !out) return fail(SANTAPP_EINVAL, "q and out must be device pointers");
    if (Hq < 1 || Hq % t->Hkv != 0) return fail(SANTAPP_EINVAL, "Hq (%d) must be a positive multiple of Hkv (%d)", Hq, t->Hkv);
    const int G = Hq / t->Hkv;
    if (G > kMaxGroup) return fail(SANTAPP_ELIMIT, "%d query heads per KV head exceed %d", G, kMaxGroup);
    if (santapp_status st = check_suffix(suffix_K, suffix_V, T, suffix_stride)) return st;
    if (!aligned16(q) || !aligned16(out) || !aligned16(workspace))
        return fail(SANTAPP_EINVAL, "q, out and workspace must be 16-byte aligned");
    if (K < 1) return fail(SANTAPP_EINVAL, "K must be >= 1 (got %d)", K);
    if (!(scale >= 0.0) || !isfinite(scale)) return fail(SANTAPP_EINVAL, "scale must be finite and >= 0");
    if (scale == 0.0) scale = 1.0 / sqrt(static_cast<double>(t->d));
    const int Kp = std::min(K, t->M);
    const bool dense = Kp == t->M;
    if (!dense && t->M > kMaxTeams) return fail(SANTAPP_ELIMIT, "%d teams per KV head exceed %d", t->M, kMaxTeams);
    const DecodeLayout L = dense ? dense_layout(t->B, Hq, t->Hkv, t->N, T, t->d, t->cus, t->dtype)
                                 : decode_layout(t->B, Hq, t->Hkv, T, t->d, t->M, Kp, t->cap.data(), t->cus,
                                                 t->dtype);
    if (!workspace || ws_bytes < L.total)
        return fail(SANTAPP_EWORKSPACE, "workspace of %zu bytes needed (got %zu)", L.total, ws_bytes);
    hipStream_t s = static_cast<hipStream_t>(stream);

    DecodeArgs A{};
    A.reps = t->reps;
    A.log_n = t->log_n;
    A.team_begin = t->team_begin;
    A.team_size = t->team_size;
    A.K = t->packed_K;
    A.V = t->packed_V;
    A.sK = suffix_K;
    A.sV = suffix_V;
    A.q = q;
    A.out = out;
    A.B = t->B;
    A.Hkv = t->Hkv;
    A.Hq = Hq;
    A.G = G;
    A.d = t->d;
    A.N = t->N;
    A.T = T;
    A.sstride = suffix_stride;
    A.M = t->M;
    A.Kp = Kp;
    A.dtype = t->dtype;
    A.dense = dense;
    A.scale = scale;
    A.scale_log2 = static_cast<float>(scale * 1.4426950408889634);
    A.seed = seed;
    A.step = step;
    A.lay = L;
    A.ws = static_cast<char*>(workspace);
    if (dbg) {
        A.dbg_phi = dbg->phi;
        A.dbg_Y = dbg->Y;
        A.dbg_sel = dbg->sel;
        A.dbg_logc = dbg->logc;
        A.dbg_tau = dbg->tau;
        A.dbg_uteams = dbg->union_teams;
        A.dbg_urows = dbg->union_rows;
        // events 1 and 2 are stamped by the attention launch itself, at the
        // kernel's start and end
        A.ev_start = static_cast<hipEvent_t>(dbg->events[1]);
        A.ev_stop = static_cast<hipEvent_t>(dbg->events[2]);
    }
    A.fused = t->dtype == SANTAPP_BF16 && fused_wanted() && L.nwg % 8 == 0;

    hipError_t e;
    auto mark = [&](int i) -> hipError_t {
        if (dbg && dbg->events[i]) return hipEventRecord(static_cast<hipEvent_t>(dbg->events[i]), s);
        return hipSuccess;
    };
    if ((e = mark(0)) != hipSuccess) return hip_fail(e, "event record");
    if ((e = launch_decode(A, s)) != hipSuccess) return hip_fail(e, "decode kernels");
    if ((e = mark(3)) != hipSuccess) return hip_fail(e, "event record");
    return ok();
}

// ---------------------------------------------------------------------------
// santapp_decode_static: santapp_decode over a scratch buffer the library
// owns, a file-scope device array of kStaticScratchBytes that every GPU the
// library runs on holds until the process ends.  Its device address is taken
// once per device (with that device current) and used for every launch; its
// first use on a device clears it with the fill kernel (the counters must
// start at zero; every completed call leaves them at zero).
// ---------------------------------------------------------------------------
namespace {

constexpr size_t kStaticScratchBytes = size_t(4) << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

struct ScratchSlot {
    void* ptr = nullptr;  // device address of `scratch` on this device
    bool cleared = false;
};
static ScratchSlot g_scratch[kMaxDevices];
static std::mutex g_scratch_mu;

static santapp_status static_scratch(hipStream_t s, void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(SANTAPP_ELIMIT, "device %d beyond the %d devices supported", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    ScratchSlot& sl = g_scratch[dev];
    if (!sl.ptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "hipGetSymbolAddress(scratch)");
        sl.ptr = p;
    }
    if (!sl.cleared) {
        e = launch_zero(sl.ptr, kStaticScratchBytes, s);
        if (e != hipSuccess) return hip_fail(e, "static scratch clear");
        sl.cleared = true;
    }
    *out = sl.ptr;
    return SANTAPP_OK;
}

}  // namespace

santapp_status santapp_decode_static(const santapp_teams* t, const float* q, const void* suffix_K,
                                     const void* suffix_V, int T, int suffix_stride, int Hq, int K,
                                     uint64_t seed, uint64_t step, double scale, float* out,
                                     const santapp_decode_debug* dbg, void* stream) {
    if (!t) return fail(SANTAPP_EINVAL, "teams is NULL");
    size_t need = 0;
    if (santapp_status st = santapp_decode_workspace_bytes(t, Hq, T, K, &need)) return st;
    if (need > kStaticScratchBytes)
        return fail(SANTAPP_ELIMIT, "this step needs %zu bytes of scratch; the static scratch holds %zu "
                    "(use santapp_decode with a workspace)", need, kStaticScratchBytes);
    void* ws = nullptr;
    if (santapp_status st = static_scratch(static_cast<hipStream_t>(stream), &ws)) return st;
    return santapp_decode(t, q, suffix_K, suffix_V, T, suffix_stride, Hq, K, seed, step, scale, out, ws,
                          kStaticScratchBytes, dbg, stream);
}

santapp_status santapp_dense_decode(const float* q, const void* K, const void* V, int B, int Hkv,
                                    int N, int d, santapp_dtype dtype, const void* suffix_K,
                                    const void* suffix_V, int T, int suffix_stride, int Hq, double scale,
                                    float* out, void* workspace, size_t ws_bytes,
                                    const santapp_decode_debug* dbg, void* stream) {
    if (!q || !out) return fail(SANTAPP_EINVAL, "q and out must be device pointers");
    if (B < 1 || Hkv < 1 || N < 0 || T < 0 || N + T < 1)
        return fail(SANTAPP_EINVAL, "invalid sizes");
    if (N > 0 && (!K || !V)) return fail(SANTAPP_EINVAL, "K and V are NULL with N > 0");
    if (santapp_status st = check_suffix(suffix_K, suffix_V, T, suffix_stride)) return st;
    if (!aligned16(q) || !aligned16(out) || !aligned16(workspace) || (N > 0 && (!aligned16(K) || !aligned16(V))))
        return fail(SANTAPP_EINVAL, "q, out, K/V and workspace must be 16-byte aligned");
    if (Hq < 1 || Hq % Hkv != 0) return fail(SANTAPP_EINVAL, "Hq must be a positive multiple of Hkv");
    if (Hq / Hkv > kMaxGroup) return fail(SANTAPP_ELIMIT, "more than %d query heads per KV head", kMaxGroup);
    if (!dtype_ok(dtype)) return fail(SANTAPP_EDTYPE, "unsupported dtype %d", static_cast<int>(dtype));
    if (d != 64 && d != 128) return fail(SANTAPP_ELIMIT, "head dim %d not supported (64 or 128)", d);
    if (!(scale >= 0.0) || !isfinite(scale)) return fail(SANTAPP_EINVAL, "scale must be finite and >= 0");
    if (scale == 0.0) scale = 1.0 / sqrt(static_cast<double>(d));
    const DecodeLayout L = dense_layout(B, Hq, Hkv, N, T, d, device_cus(), dtype);
    if (!workspace || ws_bytes < L.total)
        return fail(SANTAPP_EWORKSPACE, "workspace of %zu bytes needed (got %zu)", L.total, ws_bytes);
    DecodeArgs A{};
    A.K = K;
    A.V = V;
    A.sK = suffix_K;
    A.sV = suffix_V;
    A.q = q;
    A.out = out;
    A.B = B;
    A.Hkv = Hkv;
    A.Hq = Hq;
    A.G = Hq / Hkv;
    A.d = d;
    A.N = N;
    A.T = T;
    A.sstride = suffix_stride;
    A.M = 0;
    A.Kp = 0;
    A.dtype = dtype;
    A.dense = true;
    A.scale = scale;
    A.scale_log2 = static_cast<float>(scale * 1.4426950408889634);
    A.lay = L;
    A.ws = static_cast<char*>(workspace);
    A.fused = dtype == SANTAPP_BF16 && fused_wanted() && L.nwg % 8 == 0;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (dbg) {  // the stage events only
        A.ev_start = static_cast<hipEvent_t>(dbg->events[1]);
        A.ev_stop = static_cast<hipEvent_t>(dbg->events[2]);
    }
    auto mark = [&](int i) -> hipError_t {
        if (dbg && dbg->events[i]) return hipEventRecord(static_cast<hipEvent_t>(dbg->events[i]), s);
        return hipSuccess;
    };
    hipError_t e;
    if ((e = mark(0)) != hipSuccess) return hip_fail(e, "event record");
    if ((e = launch_decode(A, s)) != hipSuccess) return hip_fail(e, "dense decode kernels");
    if ((e = mark(3)) != hipSuccess) return hip_fail(e, "event record");
    return ok();
}

}  // extern "C"
