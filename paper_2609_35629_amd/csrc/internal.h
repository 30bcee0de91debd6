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
constexpr int kUnitRows = 32;      // rows per attention unit (one 32-row step of a wave)
constexpr int kDecodeThreads = 512;  // threads of every decode workgroup (eight waves)
constexpr int kStepMaxTeams = 512;   // teams per (b, kv) of the single-launch step
constexpr int kStepMaxKp = kStepMaxTeams;  // budget of the single-launch step: any below M
constexpr int kStepMaxWgs = 64;      // workgroups per (b, kv) pair of the single-launch step
constexpr int kKmMaxCenters = 1024;  // k-means parents per (b, kv)
constexpr int kKmMaxTrials = 8;      // seeding candidates per round: 2 + floor(ln 1024)
constexpr int kMaxLabels = 1024;     // parents of a label-defined partition
// log n of an absent team (tables whose (b, kv) pairs have different team
// counts pad the shorter ones): a finite stand-in for log 0, far below every
// real routing score, so that no score is infinite and sampling never takes
// such a team while its pair has more than K real ones
constexpr double kAbsentLogN = -1e300;
constexpr double kAbsentBelow = -1e299;  // routing scores below this are absent teams

// Floats per partial state (one query head of one workgroup): the weighted
// value sum [d], then the maximum, the mass and two pad floats, so that every
// state starts 16-byte aligned.
__host__ __device__ inline int state_stride(int d) { return d + 4; }

// Workspace layout of santapp_decode / santapp_dense_decode; byte offsets
// into the caller's buffer.  `ctr` holds per (b, kv) pair the count of its
// sampling workgroups that finished, then per (b, kv, head) the count of
// attention workgroups that published that head's state; they must be zero
// before a workspace is first used and every call leaves them zero.  nwg is
// the attention grid, maxwp the most attention workgroups one pair can have
// (the partial states per pair and head) and swords the 64-team sample words
// per head.
//
// The single-launch step (`step`) uses instead: per pair a 32-bit epoch (the
// calls the pair has completed, modulo 2^32); per (pair, head, team) three
// tagged 64-bit words (`xk`): the high and the low 32 bits of the perturbed
// score's order key and phi in fp32; and the tagged partial states.  Every word a
// call publishes carries the tag epoch + 1, so words left by earlier calls are
// never taken for this call's; the workspace must be zero before its first
// use and needs no reset between calls.
struct DecodeLayout {
    int nwg = 0, maxwp = 0, swords = 0;
    bool step = false;
    size_t ctr = 0, sbits = 0, lc = 0, part = 0, total = 0;
    size_t epoch = 0, xk = 0;
};

// Bytes of one published state of the single-launch step: d / 2 + 1 chunks
// of 16 bytes, each holding two values and two copies of the call's tag.
__host__ __device__ inline int step_state_bytes(int d) { return (d / 2 + 1) * 16; }

// Whether a step takes the single-launch kernel: bf16 rows of 64 or 128 dims,
// at most kStepMaxTeams teams (any budget below the team count), and
// at most one (b, kv) pair per compute unit; unless SANTAPP_DECODE_LAUNCH asks
// for the split or fused launches.
bool step_mode(santapp_dtype dt, int d, long long BH, int M, int Kp, bool dense, int cus);
// Workgroups of a single-launch step: the same number for every pair, at most
// kStepMaxWgs, one per compute unit at most; a multiple of eight per pair where
// the compute units allow it, so that each pair spans all eight XCDs.
int step_wgs(int cus, long long BH);

// Workgroup w of an attention grid of nwg workgroups serving BH (b, kv)
// pairs (BH <= nwg): its pair p, its index iw among the pair's workgroups and
// their count nwp.  A launch places workgroup w on XCD w mod 8.  When the
// grid holds at least one group of eight consecutive workgroups per pair, the
// groups go to the pairs in turn, so every pair's workgroups span all eight
// XCDs (each XCD has its own share of the memory bandwidth); otherwise
// workgroup w serves pair w mod BH.
struct PairSlot {
    int p, iw, nwp;
};
__host__ __device__ inline PairSlot pair_slot(int w, int nwg, int BH) {
    const int groups = nwg / 8;
    PairSlot s;
    if (nwg % 8 == 0 && groups >= BH) {
        const int j = w / 8;
        s.p = j % BH;
        s.iw = 8 * (j / BH) + w % 8;
        s.nwp = 8 * ((groups - 1 - s.p) / BH + 1);
    } else {
        s.p = w % BH;
        s.iw = w / BH;
        s.nwp = (nwg - 1 - s.p) / BH + 1;
    }
    return s;
}
// The workgroups of pair p (the nwp of its slots).
__host__ __device__ inline int pair_wgs(int p, int nwg, int BH) {
    const int groups = nwg / 8;
    if (nwg % 8 == 0 && groups >= BH) return 8 * ((groups - 1 - p) / BH + 1);
    return (nwg - 1 - p) / BH + 1;
}

// Attention workgroups of a step: one per compute unit (a multiple of eight,
// the XCDs a launch spreads over), fewer when the step has few units.
int decode_wgs(int cus, long long BH, long long units_per_pair);

// cap: host table with cap[x] = most units any x distinct teams of one
// (b, kv) can need (x = 0 .. M).
DecodeLayout decode_layout(int B, int Hq, int Hkv, int T, int d, int M, int Kp, const int* cap, int cus,
                           santapp_dtype dt);
DecodeLayout dense_layout(int B, int Hq, int Hkv, int N, int T, int d, int cus, santapp_dtype dt);

__host__ __device__ inline int chunk_count(int rows) { return (rows + kUnitRows - 1) / kUnitRows; }

// Whether launch_build_parents takes the register-resident kernel (which
// needs no per-token scratch and writes the packed copies itself).
bool build_packs_in_place(int N, int d, santapp_dtype dtype, int P, int R);

// Team table of every parent, and team_count[bh] = M.  Where the
// register-resident kernel runs it also writes the packed copies (packed_K,
// packed_V, reps) and sets *packed; otherwise the caller gathers them from
// perm and rep_token.
hipError_t launch_build_parents(const void* K, const void* V, santapp_dtype dtype, int BH, int N,
                                int d, int P, int R, int M, double* mind, int* owner,
                                int* team_begin, int* team_size, double* log_n, int* rep_token,
                                int* perm, void* packed_K, void* packed_V, void* reps, int* team_count,
                                bool* packed, hipStream_t s);

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

// Routing logits of the KL diagnostic (k_route): phi and Y for every
// (b, h, team).
struct RouteArgs {
    const void* reps;       // [BH, M, d]
    const double* log_n;    // [BH, M]
    const float* q;         // [B, Hq, d]
    int B, Hkv, Hq, G, d, M;
    santapp_dtype dtype;
    double scale;
    uint64_t seed, step;
};

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

// One decode step (sampled, or dense when `dense`): everything the kernels
// read, as plain pointers and sizes.
struct DecodeArgs {
    // team table (sampled path) or the original cache (dense path)
    const void* reps;        // [BH, M, d] routing keys
    const double* log_n;     // [BH, M]
    const int* team_begin;   // [BH, M]
    const int* team_size;    // [BH, M]
    const void* K;           // [BH, N, d] packed (sampled) or original (dense) keys
    const void* V;           // [BH, N, d]
    const void* sK;          // suffix rows: pair p's row t at (p sstride + t) d
    const void* sV;
    const float* q;          // [B, Hq, d]
    float* out;              // [B, Hq, d]
    int B, Hkv, Hq, G, d, N, T, sstride, M, Kp;
    santapp_dtype dtype;
    bool dense;
    double scale;            // softmax scale (routing in fp64)
    float scale_log2;        // scale log2(e) (attention logits, base-2 exponentials)
    uint64_t seed, step;
    DecodeLayout lay;
    char* ws;                // workspace base
    // optional diagnostics (device pointers, each may be null)
    double* dbg_phi;
    double* dbg_Y;
    int* dbg_sel;
    float* dbg_logc;
    double* dbg_tau;
    int* dbg_uteams;
    int* dbg_urows;
    hipEvent_t ev_start;     // stamped at the attention launch's start (nullable)
    hipEvent_t ev_stop;      // stamped at its end (nullable)
    bool fused;              // sampling, attention and merge in one launch
};

hipError_t launch_decode(const DecodeArgs& a, hipStream_t s);
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);

}  // namespace santapp
