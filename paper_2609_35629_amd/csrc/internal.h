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
constexpr int kSelWords = kMaxTeams / 64;  // 64-team selection words per query head
constexpr int kMaxGroup = 8;       // query heads per KV head (8-bit head masks)
constexpr int kLogcStride = 8;     // floats per union team in the read plan
constexpr int kChunkRows = 64;     // rows per sampled attention unit (two 32-row steps of one wave)
constexpr int kDenseRows = 128;    // rows per dense attention unit
constexpr int kAttendWavesPerCU = 8; // resident attention waves per compute unit
constexpr int kMergeThreads = 256;   // threads of a merge workgroup
constexpr int kKmMaxCenters = 1024;  // k-means parents per (b, kv)
constexpr int kKmMaxTrials = 8;      // seeding candidates per round: 2 + floor(ln 1024)
constexpr int kMaxLabels = 1024;     // parents of a label-defined partition
// log n of an absent team (tables whose (b, kv) pairs have different team
// counts pad the shorter ones): a finite stand-in for log 0, far below every
// real routing score, so that no score is infinite and sampling never takes
// such a team while its pair has more than K real ones
constexpr double kAbsentLogN = -1e300;
constexpr double kAbsentBelow = -1e299;  // routing scores below this are absent teams

// Attention work unit: up to kChunkRows consecutive rows of one union team of
// the packed cache, or of the suffix (slot < 0); the dense path cuts its rows
// into units of kDenseRows.  The sampler writes the units of each (b, kv)
// to that pair's region of the unit list; `meta` packs the row count (bits 0-7),
// the mask of query heads of the KV head that read the rows (bits 8-15) and
// the (b, kv) pair (bits 16-31); pos[h] is the unit's position in the list
// of units head h reads (for the heads of the mask), where its partial
// state goes.
struct Chunk {
    int begin;  // first packed row, or first suffix row when slot < 0
    int slot;   // union slot (index of the team's corrections), -1 = suffix
    int meta;
    int ci;     // index of the unit within its (b, kv) pair
    // head h's position in bits 16 (h % 2) .. of p01 (h < 2), p23, p45, p67
    unsigned p01, p23, p45, p67;
};
static_assert(sizeof(Chunk) == 32, "unit descriptors are two 16-byte words");

// Position of a unit in head h's list (h may differ across lanes: named
// fields and selects, so the descriptor stays in registers).
__host__ __device__ inline int chunk_pos(const Chunk& c, int h) {
    const unsigned lo = (h & 2) ? c.p23 : c.p01;
    const unsigned hi = (h & 2) ? c.p67 : c.p45;
    const unsigned wd = (h & 4) ? hi : lo;
    return static_cast<int>((wd >> (16 * (h & 1))) & 0xffffu);
}
// Positions of heads 0 .. 7 (a head outside the unit's mask gets 0).
__host__ __device__ inline void set_chunk_pos(Chunk& c, const int (&p)[8]) {
    auto pack = [](int a, int b) {
        return static_cast<unsigned>(a & 0xffff) | (static_cast<unsigned>(b & 0xffff) << 16);
    };
    c.p01 = pack(p[0], p[1]);
    c.p23 = pack(p[2], p[3]);
    c.p45 = pack(p[4], p[5]);
    c.p67 = pack(p[6], p[7]);
}

__host__ __device__ inline int chunk_meta(int rows, int hmask, int bh) {
    return rows | (hmask << 8) | (bh << 16);
}
__host__ __device__ inline int meta_rows(int m) { return m & 255; }
__host__ __device__ inline int meta_hmask(int m) { return (m >> 8) & 255; }
__host__ __device__ inline int meta_bh(int m) { return static_cast<int>(static_cast<unsigned>(m) >> 16); }
constexpr int kMaxPairs = 65536;       // (b, kv) pairs a unit can name
constexpr int kMaxHeadUnits = 65535;   // units one head can read (16-bit positions)

// Plan header per (b, kv), written by the sampler.
struct PlanHeader {
    int teams;   // union teams U
    int rows;    // union rows (excluding the suffix)
    int chunks;  // units of the union and the suffix
    int pad;
    int hunits[kMaxGroup];  // units each query head reads (its teams and the suffix)
};

// Workspace layout of santapp_decode; byte offsets into the caller's buffer.
// max_chunks bounds the units of any (b, kv): the largest unit count any
// union of up to min(M, G K) teams can have, plus the suffix units;
// max_hunits bounds the units one head reads (K teams and the suffix), the
// length of each head's partial-state list.
struct DecodeLayout {
    int max_chunks = 0, max_hunits = 0;
    size_t phi = 0, Y = 0, lc = 0, lpos = 0, hdr = 0, chunk = 0, ulogc = 0, po = 0,
           pml = 0, total = 0;
    size_t sbits = 0, hunits = 0;  // per query head: selection words, unit count (M > 2048)
};

// cap: host table with cap[x] = most chunks any x distinct teams of one
// (b, kv) can need (x = 0 .. M); nullptr for the dense layout.
DecodeLayout decode_layout(int B, int Hq, int Hkv, int T, int d, int M, int Kp, const int* cap);
DecodeLayout dense_layout(int B, int Hq, int Hkv, int N, int T, int d);

__host__ __device__ inline int chunk_count(int rows) { return (rows + kChunkRows - 1) / kChunkRows; }
__host__ __device__ inline int dense_count(int rows) { return (rows + kDenseRows - 1) / kDenseRows; }

// Whether launch_build_parents takes the register-resident kernel (which
// needs no per-token scratch and writes the packed copies itself).
bool build_packs_in_place(int N, int d, santapp_dtype dtype, int P, int R);

// Team table of every parent.  Where the register-resident kernel runs it
// also writes the packed copies (packed_K, packed_V, reps) and sets *packed;
// otherwise the caller gathers them from perm and rep_token.
hipError_t launch_build_parents(const void* K, const void* V, santapp_dtype dtype, int BH, int N,
                                int d, int P, int R, int M, double* mind, int* owner,
                                int* team_begin, int* team_size, double* log_n, int* rep_token,
                                int* perm, void* packed_K, void* packed_V, void* reps, bool* packed,
                                hipStream_t s);

hipError_t launch_gather_rows(const void* src, void* dst, const int* index, int BH, int rows_out,
                              int rows_in, size_t row_bytes, hipStream_t s);

// Team table of label-defined parents: parent u of pair bh has the members
// members[bh N + pbeg[bh (Mp+1) + u] ..] (token order) and its first team is
// toff[bh (Mp+1) + u]; team_begin is a position in that member order.
hipError_t launch_build_parent_lists(const void* K, santapp_dtype dtype, int BH, int N, int d, int Mp,
                                     int R, int M, const int* members, const int* pbeg, const int* toff,
                                     double* mind, int* owner, int* team_begin, int* team_size,
                                     double* log_n, int* rep_token, int* perm, hipStream_t s);

// k-means state of one (b, kv): smoothed batch inertia and its minimum, the
// count of steps without a new minimum, the stop flag and the steps run.
struct KmState {
    double ewa, ewa_min;
    int no_imp, stop, steps, pad;
};

// Scratch of santapp_kmeans_parents (byte offsets into one buffer).
struct KmLayout {
    int M = 0, s0 = 0, L = 0, nkpp = 0, nasg = 0;
    size_t samp = 0, cand = 0, D2 = 0, Dt = 0, part = 0, cent = 0, w = 0, state = 0, bpart = 0,
           bcnt = 0, binert = 0, total = 0;
};
KmLayout kmeans_layout(int BH, int N, int d, int M, int batch, int s0);

// Seeding (every round), then `count` minibatch steps from step `first`,
// then the final labels [BH, N].
hipError_t launch_kmeans_seed(const void* K, santapp_dtype dtype, int BH, int N, int d,
                              const KmLayout& L, char* ws, uint64_t seed, hipStream_t s);
hipError_t launch_kmeans_steps(const void* K, santapp_dtype dtype, int BH, int N, int d,
                               const KmLayout& L, char* ws, int batch, int first, int count,
                               double alpha, double ratio, int max_no_improvement, uint64_t seed,
                               hipStream_t s);
hipError_t launch_kmeans_labels(const void* K, santapp_dtype dtype, int BH, int N, int d,
                                const KmLayout& L, char* ws, int* labels, hipStream_t s);

// Members of each parent in token order, parent offsets pbeg [BH, Mp+1],
// team offsets toff [BH, Mp+1], team counts [BH]; *bad is set (never
// cleared) when a label lies outside [0, Mp).
hipError_t launch_parent_lists(const int* labels, int BH, int N, int Mp, int R, int* members, int* pbeg,
                               int* toff, int* team_count, int* bad, hipStream_t s);

// Absent teams g >= team_count[bh] of every pair: size 0, begin N,
// log n = kAbsentLogN, representative token 0.
hipError_t launch_pad_teams(const int* team_count, int BH, int M, int N, int* team_begin, int* team_size,
                            double* log_n, int* rep_token, hipStream_t s);

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

// Routing logits only (k_route): phi and Y for every (b, h, team).
hipError_t launch_route_phi(const RouteArgs& a, double* phi, double* Y, hipStream_t s);

// Routing keys of a table: the team means (centroid) or the representatives'
// keys, written to reps [BH, M, d].
hipError_t launch_route_keys(const void* packed_K, const int* team_begin, const int* team_size,
                             const int* rep_token, const int* perm, int BH, int N, int M, int d,
                             santapp_dtype dtype, bool centroid, void* reps, hipStream_t s);

struct KlArgs {
    const void* packed_K;    // [BH, N, d]
    const int* team_begin;   // [BH, M]
    const int* team_size;    // [BH, M]
    const double* log_n;     // [BH, M]
    const float* q;          // [B, Hq, d]
    const double* phi;       // [B, Hq, M] routing logits
    void* part;              // [B, Hq, M] per-team sums (kl_part_bytes() each)
    double* kl;              // [B, Hq]
    int B, Hkv, Hq, N, M, d;
    santapp_dtype dtype;
    double scale;
};

size_t kl_part_bytes();

// Per-team sums over the prompt rows, then KL(p || q) per query head.
hipError_t launch_routing_kl(const KlArgs& a, hipStream_t s);

struct AttendArgs {
    const void* K;    // [BH, N, d] packed (sampled path) or original (dense path)
    const void* V;
    const void* sK;   // [BH, T, d]
    const void* sV;
    const float* q;   // [B, Hq, d]
    int B, Hkv, Hq, G, d, N, T, M, max_chunks, max_hunits;
    int grid_waves;             // resident one-wave workgroups of the device (0: one per unit)
    int cus;                    // compute units of the device (0: unknown)
    santapp_dtype dtype;
    float scale;
    bool dense;                 // every row, every head, correction 1
    const char* ws;             // plan (sampled path)
    const DecodeLayout* lay;    // plan offsets (sampled path)
    float* part_o;              // [BH, G, max_hunits, d]
    float* part_ml;             // [BH, G, max_hunits, 2]
    float* out;                 // [B, Hq, d]
    hipEvent_t ev_start;        // stamped at the attention kernel's start (nullable)
    hipEvent_t ev_stop;         // stamped at its end (nullable)
};

hipError_t launch_attend(const AttendArgs& a, hipStream_t s);
hipError_t launch_merge(const AttendArgs& a, hipStream_t s);
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);

}  // namespace santapp
