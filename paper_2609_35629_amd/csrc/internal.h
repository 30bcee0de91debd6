// Internal interface between the C-ABI layer (api.hip) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "santapp.h"

namespace santapp {

constexpr int kMaxHeadDim = 256;   // LDS vector in the team builder
constexpr int kMaxReps = 1024;     // representatives per parent
constexpr int kMaxTeams = 8192;    // teams per (b, kv) the sampler handles
constexpr int kMaxGroup = 8;       // query heads per KV head (8-bit head masks)
constexpr int kLogcStride = 8;     // floats per union team in the read plan
constexpr int kChunkRows = 32;     // rows per sampled attention unit (one wave)
constexpr int kDenseRows = 128;    // rows per dense attention unit
constexpr int kAttendWavesPerCU = 8; // resident attention waves per compute unit

// Attention work unit: up to kChunkRows consecutive rows of one union team of
// the packed cache, or of the suffix (slot < 0); the dense path cuts its rows
// into units of kDenseRows.  The sampler appends the units of each (b, kv)
// to one list shared by all pairs; `meta` packs the row count (bits 0-7),
// the mask of query heads of the KV head that read the rows (bits 8-15) and
// the (b, kv) pair (bits 16-31).
struct Chunk {
    int begin;  // first packed row, or first suffix row when slot < 0
    int slot;   // union slot (index of the team's corrections), -1 = suffix
    int ci;     // index of the unit within its (b, kv) pair
    int meta;
};

__host__ __device__ inline int chunk_meta(int rows, int hmask, int bh) {
    return rows | (hmask << 8) | (bh << 16);
}
__host__ __device__ inline int meta_rows(int m) { return m & 255; }
__host__ __device__ inline int meta_hmask(int m) { return (m >> 8) & 255; }
__host__ __device__ inline int meta_bh(int m) { return static_cast<int>(static_cast<unsigned>(m) >> 16); }
constexpr int kMaxPairs = 65536;  // (b, kv) pairs a unit can name

// Plan header per (b, kv), written by the sampler.
struct PlanHeader {
    int teams;   // union teams U
    int rows;    // union rows (excluding the suffix)
    int chunks;  // chunks of the union and the suffix
    int pad;
};

// Workspace layout of santapp_decode; byte offsets into the caller's buffer.
// max_chunks bounds the chunks of any (b, kv): the largest chunk count any
// union of up to min(M, G K) teams can have, plus the suffix chunks.
struct DecodeLayout {
    int max_chunks = 0;
    size_t counter = 0, phi = 0, Y = 0, lc = 0, hdr = 0, chunk = 0, ulogc = 0, po = 0, pml = 0,
           total = 0;
};

// cap: host table with cap[x] = most chunks any x distinct teams of one
// (b, kv) can need (x = 0 .. M); nullptr for the dense layout.
DecodeLayout decode_layout(int B, int Hq, int Hkv, int T, int d, int M, int Kp, const int* cap);
DecodeLayout dense_layout(int B, int Hq, int Hkv, int N, int T, int d);

__host__ __device__ inline int chunk_count(int rows) { return (rows + kChunkRows - 1) / kChunkRows; }
__host__ __device__ inline int dense_count(int rows) { return (rows + kDenseRows - 1) / kDenseRows; }

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
    int B, Hkv, Hq, G, d, M, Kp, T;
    santapp_dtype dtype;
    double scale;
    uint64_t seed, step;
    const DecodeLayout* lay;
    char* ws;
    const santapp_decode_debug* dbg;
};

// Routing (k_route), then Gumbel-top-K, corrections and the read plan
// (k_select): two launches on the stream.
hipError_t launch_route_select(const RouteArgs& a, hipStream_t s);

struct AttendArgs {
    const void* K;    // [BH, N, d] packed (sampled path) or original (dense path)
    const void* V;
    const void* sK;   // [BH, T, d]
    const void* sV;
    const float* q;   // [B, Hq, d]
    int B, Hkv, Hq, G, d, N, T, M, max_chunks;
    int grid_waves;             // one-wave workgroups on the sampled path (0: one per unit)
    santapp_dtype dtype;
    float scale;
    bool dense;                 // every row, every head, correction 1
    const char* ws;             // plan (sampled path)
    const DecodeLayout* lay;    // plan offsets (sampled path)
    float* part_o;              // [BH, G, max_chunks, d]
    float* part_ml;             // [BH, G, max_chunks, 2]
    float* out;                 // [B, Hq, d]
};

hipError_t launch_attend(const AttendArgs& a, hipStream_t s);
hipError_t launch_merge(const AttendArgs& a, hipStream_t s);
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);

}  // namespace santapp
