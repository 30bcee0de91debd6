/*
 * santapp -- SANTA++ decode-time attention on AMD Instinct MI355X (gfx950).
 *
 * C ABI of libsantapp.so.  The operations follow the paper "SANTA++: Sampling
 * Attention through Representative Keys":
 *
 *   santapp_build_teams   section "Preparing parent groups and teams",
 *                         Alg. "Contiguous parent partition" and
 *                         Alg. "Build actual-key teams from a parent
 *                         partition", plus the team-contiguous packed copy of
 *                         the prompt K/V described for the GPU implementation
 *                         (appendix "Triton decode kernels", first paragraph).
 *   santapp_decode        Alg. "SANTA++ attention for one query head" for every
 *                         query head of one decode step: eq. method-routing,
 *                         the Gumbel-top-K sampler, eq. method-inclusion,
 *                         eq. method-estimate, GQA sharing of the reads.
 *   santapp_dense_decode  eq. method-attention over the whole current cache
 *                         (the dense baseline).
 *   santapp_teams_set_route_keys, santapp_routing_kl
 *                         section "Attention-distribution diagnostic":
 *                         centroid routing keys and eq. diagnostic-kl.
 *   santapp_kmeans_parents  Alg. "Global minibatch k-means parent partition"
 *                         with the settings stated after it.
 *   santapp_build_teams_from_labels  Alg. "Build actual-key teams from a
 *                         parent partition" for any parent partition.
 *
 * Conventions
 *   - Every tensor argument is a DEVICE pointer owned by the caller unless
 *     stated otherwise; layouts are dense row-major.  Tensor and workspace
 *     pointers must be 16-byte aligned (else SANTAPP_EINVAL).
 *   - K/V element type is bf16 (raw 16-bit patterns) or fp32, chosen by
 *     santapp_dtype; queries are fp32; outputs are fp32.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Every call only enqueues work on that stream; none synchronises except
 *     santapp_build_teams, which waits for its own kernels before returning.
 *   - Every call returns a santapp_status.  On failure nothing is enqueued
 *     after the failing step and santapp_last_error() returns a message for
 *     the calling thread.  No call aborts the process.
 *   - santapp_decode and santapp_dense_decode never allocate: the caller
 *     provides a workspace of the queried size, zeroed once before its
 *     first use.
 */
#ifndef SANTAPP_H
#define SANTAPP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SANTAPP_OK = 0,
    SANTAPP_EINVAL = 1,     /* invalid argument (size, budget, null pointer, scale) */
    SANTAPP_EDTYPE = 2,     /* unsupported element type                             */
    SANTAPP_ENOMEM = 3,     /* device allocation failed (santapp_build_teams only)  */
    SANTAPP_EHIP = 4,       /* a HIP runtime call or kernel launch failed           */
    SANTAPP_EWORKSPACE = 5, /* workspace missing or smaller than required           */
    SANTAPP_ELIMIT = 6      /* valid but beyond this library's supported sizes      */
} santapp_status;

/* The input enumerations below span the whole int range (their last two
 * enumerators are never valid arguments), so that a caller may pass any int
 * and an unknown value is answered with an error status instead of being
 * undefined behaviour in the library. */
typedef enum {
    SANTAPP_BF16 = 0,
    SANTAPP_FP32 = 1,
    SANTAPP_DTYPE_INT_MIN_ = -2147483647 - 1,
    SANTAPP_DTYPE_INT_MAX_ = 2147483647
} santapp_dtype;

/* Opaque team table of one layer: owns its device buffers. */
typedef struct santapp_teams santapp_teams;

/* Read-only view of a team table.  All pointers are device pointers owned by
 * the table; every per-(b,kv) array is laid out [B][Hkv][...]. */
typedef struct {
    int B, Hkv, N, d;
    santapp_dtype dtype;
    int parent_size, reps_per_parent;
    int M;                   /* teams per (b, kv); identical for all (b, kv) */
    const void* packed_K;    /* [B,Hkv,N,d] prompt keys in team order        */
    const void* packed_V;    /* [B,Hkv,N,d] prompt values in team order      */
    const void* reps;        /* [B,Hkv,M,d] routing key of each team (its    */
                             /* representative's key unless changed by       */
                             /* santapp_teams_set_route_keys)                */
    const int* team_begin;   /* [B,Hkv,M] first packed row of each team      */
    const int* team_size;    /* [B,Hkv,M] n_g                                */
    const double* log_n;     /* [B,Hkv,M] log n_g (fp64)                     */
    const int* rep_token;    /* [B,Hkv,M] original token index of l_g        */
    const int* perm;         /* [B,Hkv,N] packed row -> original token index */
    const int* team_count;   /* [B,Hkv] real teams of each (b, kv); teams    */
                             /* g >= team_count are absent (see below)       */
} santapp_teams_desc;

/*
 * Build the team table of one layer (done once after prefill).
 *
 * K, V:      [B,Hkv,N,d] post-RoPE prompt keys / values (device, caller-owned,
 *            not modified; they may be freed after the call returns).
 * parent_size (P >= 1):     contiguous parents [uP, min((u+1)P, N)).
 * reps_per_parent (R >= 1): representatives per parent, r = min(R, |C|).
 * Per parent: the first representative is the member nearest the parent
 * mean; each later one is the member farthest from its nearest chosen
 * representative (ties: lowest token index); every member joins its nearest
 * representative (ties: earliest chosen); representatives own themselves.
 * Distances are squared Euclidean in fp64 on the exact input values.
 * Teams are numbered parent by parent in representative order; members of a
 * team are stored contiguously in ascending token order.
 *
 * Limits: d in {64, 128}; R <= 1024 (else SANTAPP_ELIMIT).  Sampled decoding
 * (K < M) supports M <= 8192 teams per (b, kv).
 * On success *out receives a new table (free with santapp_teams_destroy).
 * Allocates device memory; synchronises `stream` before returning.
 */
santapp_status santapp_build_teams(const void* K, const void* V, int B, int Hkv, int N, int d,
                                   santapp_dtype dtype, int parent_size, int reps_per_parent,
                                   void* stream, santapp_teams** out);

/*
 * Minibatch k-means settings theta (the paper's reported runs: batch 4096,
 * max_iter 100, max_no_improvement 10, reassignment_ratio 0.01, init_size 0,
 * seed 0).
 */
typedef struct {
    int batch_size;             /* points per minibatch, drawn with replacement  */
    int max_iter;               /* steps = floor(max_iter * N / batch_size)      */
    int max_no_improvement;     /* stop after this many steps without a new      */
                                /* minimum of the smoothed batch inertia (0: no) */
    double reassignment_ratio;  /* in [0, 1): centers with a cumulative count    */
                                /* below ratio * the largest move to a batch     */
                                /* point                                         */
    int init_size;              /* seeding sample; 0: 3 * batch_size (at least   */
                                /* 3 M, at most N)                               */
    uint64_t seed;              /* xi                                            */
} santapp_kmeans_settings;

/*
 * K-means parents of one layer (Alg. "Global minibatch k-means parent
 * partition"): for every (b, kv), M = min(N, max(2, floor(N / parent_size)))
 * centers fitted to the post-RoPE keys by greedy k-means++ seeding and
 * minibatch steps with cumulative-count updates, then labels[b,kv,i] = the
 * nearest center of token i (ties: lowest index).  Every (b, kv) pair uses
 * the same random draws (Philox4x64-10, key (seed, 1)); distances are fp64 on
 * the exact key values.
 *
 * K:      [B,Hkv,N,d] keys (device, not modified).
 * labels: [B,Hkv,N] int32 output (device, caller-owned).
 * num_parents (host, may be NULL): receives M.
 * steps (host [B*Hkv], may be NULL): minibatch steps each pair ran.
 * Limits: N >= 2, d in {64, 128}, M <= 1024 (else SANTAPP_ELIMIT).
 * Allocates scratch device memory; synchronises `stream` before returning.
 */
santapp_status santapp_kmeans_parents(const void* K, int B, int Hkv, int N, int d, santapp_dtype dtype,
                                      int parent_size, const santapp_kmeans_settings* theta, int* labels,
                                      int* num_parents, int* steps, void* stream);

/*
 * Team table of label-defined parents: parent u of (b, kv) is
 * {i : labels[b,kv,i] == u}; parents are taken in ascending label order,
 * empty ones omitted, and each is split into teams as in
 * santapp_build_teams (representatives, assignment, ties, member order).
 * labels: [B,Hkv,N] int32 in [0, num_labels) (device; else SANTAPP_EINVAL).
 * The pairs' team counts differ in general: the table's M is the largest,
 * and the teams g >= team_count[b,kv] of a pair are absent: no rows
 * (team_size 0, team_begin N), rep_token 0 and log_n = -1e300, a finite
 * stand-in for log 0 that keeps every routing score finite.  Decoding never
 * samples an absent team while its pair has more than K real teams; when it
 * has at most K, every real team is taken with correction 1 and absent ones
 * add nothing.  The table's parent_size is 0.
 * Limits: d in {64, 128}; num_labels <= 1024; R <= 1024.
 * Allocates device memory; synchronises `stream` before returning.
 */
santapp_status santapp_build_teams_from_labels(const void* K, const void* V, int B, int Hkv, int N, int d,
                                               santapp_dtype dtype, const int* labels, int num_labels,
                                               int reps_per_parent, void* stream, santapp_teams** out);

/*
 * Keys the teams are routed by (the table's `reps`; section
 * "Attention-distribution diagnostic" and its appendix, which compare
 * routing by an actual representative key with centroid-guided sampling):
 *   SANTAPP_ROUTE_REPRESENTATIVE  each team's representative key (the state
 *                                 santapp_build_teams leaves);
 *   SANTAPP_ROUTE_CENTROID        the arithmetic mean of the team's keys: per
 *                                 dimension the members' values summed in fp64
 *                                 in team order (ascending token index),
 *                                 divided by n_g, rounded to the table's
 *                                 element type (nearest, ties to even).
 * With contiguous parents of B tokens and one representative each
 * (parent_size = B, reps_per_parent = 1) the centroid keys give the paper's
 * centroid-guided sampling over contiguous groups.  Decoding with a table
 * uses whichever keys it holds; the team partition is unchanged.  Enqueued
 * on `stream`; never allocates.
 */
typedef enum {
    SANTAPP_ROUTE_REPRESENTATIVE = 0,
    SANTAPP_ROUTE_CENTROID = 1,
    SANTAPP_ROUTE_INT_MIN_ = -2147483647 - 1,
    SANTAPP_ROUTE_INT_MAX_ = 2147483647
} santapp_route_key;

santapp_status santapp_teams_set_route_keys(santapp_teams* teams, santapp_route_key kind, void* stream);

/* Fill *desc with the table's sizes and device pointers. */
santapp_status santapp_teams_info(const santapp_teams* teams, santapp_teams_desc* desc);

/* Free a table and its device buffers (NULL is ignored).  The caller must
 * make sure no enqueued decode still reads it. */
void santapp_teams_destroy(santapp_teams* teams);

/*
 * eq. method-budget: K = min(M, S / (P / R)) for a nominal row budget S.
 * Requires P % R == 0 and S % (P / R) == 0 (else SANTAPP_EINVAL).  Host-only.
 */
santapp_status santapp_budget_to_K(int S, int P, int R, int M, int* K);

/* Optional diagnostic outputs of santapp_decode (device pointers; each may be
 * NULL).  The arrays are written only when the step samples (K < M).
 * events[0..3], when non-NULL, are hipEvent_t handles created by the caller:
 * events[0] is recorded on `stream` before the step's launches, events[1]
 * and events[2] are stamped by the attention launch at that kernel's start
 * and end (its execution time, without the dispatch gap before it; in the
 * one-launch mode that kernel also samples), and events[3] is recorded after
 * the step, so that hipEventElapsedTime gives the time of each stage. */
typedef struct {
    double* phi;      /* [B,Hq,M] routing logits log n_g + scale q.l_g          */
    double* Y;        /* [B,Hq,M] perturbed routing scores phi_g + G_g          */
    int* sel;         /* [B,Hq,K] selected team ids per head, ascending         */
    float* logc;      /* [B,Hq,K] log c_g of those teams                        */
    double* tau;      /* [B,Hq]   (K+1)-th largest perturbed score              */
    int* union_teams; /* [B,Hkv]  teams read for the kv head (union over heads) */
    int* union_rows;  /* [B,Hkv]  prompt rows read for the kv head              */
    void* events[4];  /* hipEvent_t stage markers (each may be NULL)            */
} santapp_decode_debug;

/*
 * Workspace for santapp_decode with these sizes (bytes, host-only query).
 * It holds what the workgroups of a step hand to each other: the perturbed
 * routing scores, the samples and partial results, with per (b, kv) pair
 * either a call counter whose value tags every word a call publishes (the
 * single-launch step) or counters that every completed call leaves at zero
 * (the three-launch kernels).  A workspace must be zeroed once before its
 * first use (santapp_workspace_zero) and needs nothing between calls.  Calls
 * that share a workspace must not overlap in time (use one workspace per
 * stream).  The size depends on the compute units of the device the table
 * was built on.
 */
santapp_status santapp_decode_workspace_bytes(const santapp_teams* teams, int Hq, int T, int K,
                                              size_t* bytes);

/*
 * How santapp_decode runs a step with these sizes (host-only query): the
 * kernel launches of one step in *kernels (1 for the single-launch step,
 * which bf16 tables of at most 512 teams per KV head and budgets of at most
 * 128 teams take, and for the launches SANTAPP_DECODE_LAUNCH=fused asks for;
 * 3 otherwise for a sampled step, 2 for a budget that takes every team) and
 * the workgroups of its main launch in *workgroups.  Errors as
 * santapp_decode_workspace_bytes.
 */
santapp_status santapp_decode_launch_info(const santapp_teams* teams, int Hq, int T, int K, int* kernels,
                                         int* workgroups);

/* Zero `bytes` bytes of device memory at `ws` on `stream` (a fill kernel,
 * safe inside HIP graph capture). */
santapp_status santapp_workspace_zero(void* ws, size_t bytes, void* stream);

/*
 * One SANTA++ decode step for every sequence b < B and query head h < Hq of
 * one layer (query head h reads KV head h / (Hq / Hkv)).
 *
 * q:        [B,Hq,d] fp32 post-RoPE queries.
 * suffix_K, suffix_V: the generated rows attended exactly (section "Cache
 *           state and budget": empty on the first sparse call, one row more
 *           per generated token); same dtype as the table; may be NULL when
 *           T == 0.  Row t < T of pair p = b Hkv + kv starts at element
 *           (p suffix_stride + t) d, so a caller can append rows in place to a
 *           buffer [B,Hkv,capacity,d] (suffix_stride = capacity); 0 means T
 *           (a dense [B,Hkv,T,d] tensor).  suffix_stride < T is EINVAL.
 * K:        teams to sample per query head (>= 1).  K >= M selects every team
 *           with correction 1 (dense attention over the cache).
 * seed, step: Gumbel noise of team g for head h of sequence b is word g % 4 of
 *           Philox4x64-10(key = {seed, 0}, counter = {g / 4, h, b, step});
 *           U = ((w >> 12) + 1/2) 2^-52, G = -log(-log U).
 * scale:    softmax scale; 0 means 1/sqrt(d).  Used for routing too.
 * out:      [B,Hq,d] fp32 estimate U^ / Z^.
 * Routing logits, the perturbed scores, the selection and tau are computed in
 * fp64; attention scores and the online softmax in fp32.
 * A step on a bf16 table with d of 64 or 128, at most 512 teams per (b, kv)
 * and at most one (b, kv) pair per compute unit runs as one launch, whose
 * workgroups hand the perturbed scores and their partial results to each
 * other through tagged words in the workspace; any other step runs as three
 * launches (sampling, attention, merge).  santapp_decode_launch_info reports
 * which.  The environment variable SANTAPP_DECODE_LAUNCH (read at the first
 * call of a process) set to "split" forces the three launches, "fused" their
 * one-launch form with counters in the workspace.
 * Never allocates and never synchronises.
 */
santapp_status santapp_decode(const santapp_teams* teams, const float* q, const void* suffix_K,
                              const void* suffix_V, int T, int suffix_stride, int Hq, int K, uint64_t seed,
                              uint64_t step, double scale, float* out, void* workspace,
                              size_t ws_bytes, const santapp_decode_debug* dbg, void* stream);

/*
 * santapp_decode for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same step, the same arguments except the workspace, over a scratch
 * buffer the library owns -- a static device array of 4 MiB on every GPU the
 * library runs on, held until the process ends.  The call allocates nothing
 * and never synchronises; its first use on a device enqueues a clear of that
 * device's array on `stream` ahead of the step.  Steps whose workspace
 * (santapp_decode_workspace_bytes) exceeds 4 MiB return SANTAPP_ELIMIT.
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * contents: calls that overlap in time on one GPU (other streams, other host
 * threads) race and must be serialised by the caller.
 */
santapp_status santapp_decode_static(const santapp_teams* teams, const float* q, const void* suffix_K,
                                     const void* suffix_V, int T, int suffix_stride, int Hq, int K,
                                     uint64_t seed, uint64_t step, double scale, float* out,
                                     const santapp_decode_debug* dbg, void* stream);

/* Workspace for santapp_dense_decode (bytes, host-only query). */
santapp_status santapp_dense_workspace_bytes(int B, int Hq, int Hkv, int N, int T, int d,
                                             size_t* bytes);

/*
 * Dense softmax attention over K, V [B,Hkv,N,d] followed by the suffix rows
 * (eq. method-attention), with the same GQA mapping, suffix layout, dtypes
 * and scale convention as santapp_decode.  The workspace follows the same
 * rules (zeroed before first use; nothing between calls).  dbg may be NULL;
 * only its events are used, as for santapp_decode (events[1] and events[2]
 * stamped by the attention launch at its start and end).  Never allocates or
 * synchronises.
 */
santapp_status santapp_dense_decode(const float* q, const void* K, const void* V, int B, int Hkv,
                                    int N, int d, santapp_dtype dtype, const void* suffix_K,
                                    const void* suffix_V, int T, int suffix_stride, int Hq, double scale,
                                    float* out, void* workspace, size_t ws_bytes,
                                    const santapp_decode_debug* dbg, void* stream);

/* Workspace for santapp_routing_kl (bytes, host-only query). */
santapp_status santapp_routing_kl_workspace_bytes(const santapp_teams* teams, int Hq, size_t* bytes);

/*
 * Routing diagnostic of eq. diagnostic-kl for every sequence b and query head
 * h: KL(p || q) in nats, with p the dense softmax attention over the N prompt
 * tokens (the suffix excluded) and q_i = P(g(i)) / n_g(i), where P is the
 * softmax over the teams of log n_g + scale q . key_g with the table's
 * current routing keys (no sampling).  Scores, sums and logarithms in fp64.
 * q: [B,Hq,d] fp32; kl: [B,Hq] fp64 (device).  scale 0 means 1/sqrt(d).
 * Never allocates; the workspace needs no initialisation.
 */
santapp_status santapp_routing_kl(const santapp_teams* teams, const float* q, int Hq, double scale,
                                  double* kl, void* workspace, size_t ws_bytes, void* stream);

/* Message of the last failed call on this thread ("" if none). */
const char* santapp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SANTAPP_H */
