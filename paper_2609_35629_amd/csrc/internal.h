// Internal interface between the C-ABI layer (api.hip) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "santapp.h"

namespace santapp {

constexpr int kMaxHeadDim = 256;   // LDS vector in the team builder
constexpr int kMaxReps = 1024;     // representatives per parent
constexpr int kMaxTeams = 8192;    // teams per (b, kv) the sampler keeps in LDS
constexpr int kMaxGroup = 8;       // query heads per KV head (8-bit head masks)
constexpr int kLogcStride = 8;     // floats per union team in the read plan

// Workspace layout of santapp_decode; byte offsets into the caller's buffer.
// Rows of one KV head are [union rows ; suffix rows]; the attention kernel
// splits them into ranges of at most kSplitRows rows, so the number of
// partials per head is at most max_split = ceil((N + T) / kSplitRows).
struct DecodeLayout {
    int max_split = 0;
    size_t phi = 0, Y = 0, lc = 0, hdr = 0, ubeg = 0, urs = 0, ulogc = 0, split = 0, po = 0,
           pml = 0, total = 0;
};

constexpr int kSplitRows = 128;  // rows per attention workgroup (16 groups x 8 rows)

DecodeLayout decode_layout(int B, int Hq, int Hkv, int N, int T, int d, int M);
DecodeLayout dense_layout(int B, int Hq, int Hkv, int N, int T, int d);

hipError_t launch_build_parents(const void* K, santapp_dtype dtype, int BH, int N, int d, int P,
                                int R, int M, double* mind, int* owner, int* team_begin,
                                int* team_size, double* log_n, int* rep_token, int* perm,
                                hipStream_t s);

hipError_t launch_gather_rows(const void* src, void* dst, const int* index, int BH, int rows_out,
                              int rows_in, size_t row_bytes, hipStream_t s);

struct RouteArgs {
    const void* reps;       // [BH, M, d]
    const int* team_size;   // [BH, M]
    const int* team_begin;  // [BH, M]
    const double* log_n;    // [BH, M]
    const float* q;         // [B, Hq, d]
    int B, Hkv, Hq, G, d, N, M, Kp, T;
    santapp_dtype dtype;
    double scale;
    uint64_t seed, step;
    const DecodeLayout* lay;
    char* ws;
    const santapp_decode_debug* dbg;
};

hipError_t launch_route(const RouteArgs& a, hipStream_t s);
hipError_t launch_select(const RouteArgs& a, hipStream_t s);

struct AttendArgs {
    const void* K;    // [BH, N, d] packed (sampled path) or original (dense path)
    const void* V;
    const void* sK;   // [BH, T, d]
    const void* sV;
    const float* q;   // [B, Hq, d]
    int B, Hkv, Hq, G, d, N, T, M, max_split;
    santapp_dtype dtype;
    float scale;
    bool dense;                 // every row, every head, correction 1
    const char* ws;             // plan (sampled path)
    const DecodeLayout* lay;    // plan offsets (sampled path)
    float* part_o;              // [B, Hq, max_split, d]
    float* part_ml;             // [B, Hq, max_split, 2]
    float* out;                 // [B, Hq, d]
};

hipError_t launch_attend(const AttendArgs& a, hipStream_t s);
hipError_t launch_merge(const AttendArgs& a, hipStream_t s);
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);

}  // namespace santapp
