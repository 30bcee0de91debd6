/*
 * SANTA++ decode attention -- CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, fp64 statement of
 * what the decode path computes, written from the paper (SANTA++: Sampling
 * Attention through Representative Keys).  Only the test suite, the smoke
 * check and the CPU-baseline leg of the benchmark may load it.  It shares no
 * code, header, table or constant generator with the GPU library.
 *
 * Everything is fp64 on inputs that are exact fp32/bf16 values.  Loops run in
 * plain index order; the file is compiled with -ffp-contract=off so that each
 * product and sum is rounded exactly as written.
 *
 * Contents
 *   philox4x64_10        counter-based generator (Salmon et al., SC'11)
 *   oracle_gumbel        U in (0,1) from one 64-bit word, G = -log(-log U)
 *   oracle_build_teams   Alg. "Contiguous parent partition" followed by
 *                        Alg. "Build actual-key teams from a parent partition"
 *   oracle_build_teams_parents  the same team construction for any parent
 *                        partition
 *   oracle_kmeans        Alg. "Global minibatch k-means parent partition"
 *   oracle_decode_head   Alg. "SANTA++ attention for one query head",
 *                        eq. method-routing, method-inclusion, method-estimate
 *   oracle_dense_head    eq. method-attention over the whole current cache
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Philox4x64-10: 10 rounds of the Philox S-box with 64-bit words.           */
/* Round: (x0,x1,x2,x3) -> (hi(M1*x2)^x1^k0, lo(M1*x2), hi(M0*x0)^x3^k1,     */
/* lo(M0*x0)); the key is bumped by the Weyl constants before rounds 2..10.  */
/* ------------------------------------------------------------------------ */
#define PHILOX_M0 0xD2E7470EE14C6C93ULL
#define PHILOX_M1 0xCA5A826395121157ULL
#define PHILOX_W0 0x9E3779B97F4A7C15ULL
#define PHILOX_W1 0xBB67AE8584CAA73BULL

void philox4x64_10(const uint64_t ctr_in[4], const uint64_t key_in[2], uint64_t out[4])
{
    uint64_t x0 = ctr_in[0], x1 = ctr_in[1], x2 = ctr_in[2], x3 = ctr_in[3];
    uint64_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += PHILOX_W0;
            k1 += PHILOX_W1;
        }
        unsigned __int128 p0 = (unsigned __int128)PHILOX_M0 * x0;
        unsigned __int128 p1 = (unsigned __int128)PHILOX_M1 * x2;
        uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
        uint64_t y0 = hi1 ^ x1 ^ k0;
        uint64_t y1 = lo1;
        uint64_t y2 = hi0 ^ x3 ^ k1;
        uint64_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* Standard Gumbel draw from one 64-bit word: U = ((x >> 12) + 1/2) 2^-52 is
 * exact in fp64 and lies in [2^-53, 1 - 2^-53], strictly inside (0, 1); the
 * inverse CDF of Pr(G <= x) = exp(-exp(-x)) is G = -log(-log U). */
double oracle_gumbel(uint64_t x)
{
    double u = ((double)(x >> 12) + 0.5) * 0x1.0p-52;
    return -log(-log(u));
}

/* The Gumbel noise of team g for query head h of sequence b at decode step
 * `step`: Philox4x64-10 with key (seed, 0) and counter (g/4, h, b, step);
 * team g takes output word g mod 4.  Every (b, h, g, step) therefore gets its
 * own independent draw. */
double oracle_team_gumbel(uint64_t seed, uint64_t step, uint64_t b, uint64_t h, uint64_t g)
{
    uint64_t ctr[4] = { g >> 2, h, b, step };
    uint64_t key[2] = { seed, 0 };
    uint64_t out[4];
    philox4x64_10(ctr, key, out);
    return oracle_gumbel(out[g & 3]);
}

/* Squared Euclidean distance between two rows, summed in index order. */
static double sqdist(const double* a, const double* b, int d)
{
    double acc = 0.0;
    for (int j = 0; j < d; ++j) {
        double t = a[j] - b[j];
        acc = acc + t * t;
    }
    return acc;
}

/* ------------------------------------------------------------------------ */
/* Team construction for one parent (Alg. "Build actual-key teams from a     */
/* parent partition").                                                       */
/*                                                                           */
/* The parent C is given by its member token indices idx[0..n) in ascending  */
/* order.  r = min(R, n), mu = mean of the member keys,                      */
/*   j_1 = argmin_i |k_i - mu|^2,                                            */
/*   j_u = argmax over non-representatives of min_{j in L} |k_i - k_j|^2,    */
/*   b_i = argmin_u |k_i - k_{j_u}|^2, then b_{j_u} = u (self-ownership),     */
/*   teams appended in representative order u = 1..r.                        */
/* Ties: representative choice by lowest token index, assignment by          */
/* representative-selection order.  Scratch: mu[d], reps[R], is_rep[n],      */
/* owner[n], D[R * n].  Appends to members / team_ptr / rep_token at team    */
/* *M and member position *filled.                                           */
/* ------------------------------------------------------------------------ */
static void build_parent(const double* K, int d, const int* idx, int n, int R,
                         double* mu, int* reps, int* is_rep, int* owner, double* D,
                         int* members, int* team_ptr, int* rep_token, int* M, int* filled)
{
    int r = R < n ? R : n;
#define ROW(i) (K + (size_t)idx[i] * d)
    for (int j = 0; j < d; ++j) {
        double s = 0.0;
        for (int i = 0; i < n; ++i) s = s + ROW(i)[j];
        mu[j] = s / (double)n;
    }
    for (int i = 0; i < n; ++i) is_rep[i] = 0;

    /* first representative: the member nearest the parent mean */
    int best = 0;
    double best_d = sqdist(ROW(0), mu, d);
    for (int i = 1; i < n; ++i) {
        double t = sqdist(ROW(i), mu, d);
        if (t < best_d) { best_d = t; best = i; }
    }
    reps[0] = best;
    is_rep[best] = 1;
    for (int i = 0; i < n; ++i) D[i] = sqdist(ROW(i), ROW(best), d);

    /* farthest-first: maximise the distance to the nearest chosen rep */
    for (int u = 1; u < r; ++u) {
        int pick = -1;
        double pick_d = -1.0;
        for (int i = 0; i < n; ++i) {
            if (is_rep[i]) continue;
            double m = D[i];
            for (int v = 1; v < u; ++v)
                if (D[(size_t)v * n + i] < m) m = D[(size_t)v * n + i];
            if (pick < 0 || m > pick_d) { pick = i; pick_d = m; }
        }
        reps[u] = pick;
        is_rep[pick] = 1;
        for (int i = 0; i < n; ++i) D[(size_t)u * n + i] = sqdist(ROW(i), ROW(pick), d);
    }

    /* nearest-representative assignment, then representative self-ownership */
    for (int i = 0; i < n; ++i) {
        int bu = 0;
        double bd = D[i];
        for (int u = 1; u < r; ++u)
            if (D[(size_t)u * n + i] < bd) { bd = D[(size_t)u * n + i]; bu = u; }
        owner[i] = bu;
    }
    for (int u = 0; u < r; ++u) owner[reps[u]] = u;

    /* emit teams in representative order, members ascending */
    for (int u = 0; u < r; ++u) {
        for (int i = 0; i < n; ++i)
            if (owner[i] == u) members[(*filled)++] = idx[i];
        rep_token[*M] = idx[reps[u]];
        team_ptr[*M + 1] = *filled;
        ++*M;
    }
#undef ROW
}

/* ------------------------------------------------------------------------ */
/* Teams of one (sequence, KV head) from any parent partition: parent p has  */
/* the members pmem[pptr[p] .. pptr[p+1]) (ascending token indices); empty   */
/* parents are skipped; parents are taken in the order given.                */
/*                                                                           */
/* K: [N, d] row-major.  Outputs, in team order: members[N] (the token       */
/* indices of team 0 ascending, then team 1, ...), team_ptr[M+1] (CSR        */
/* offsets into members) and rep_token[M].  The caller sizes team_ptr and    */
/* rep_token for at most N teams.  Returns M, or -1 on bad arguments.        */
/* ------------------------------------------------------------------------ */
int oracle_build_teams_parents(const double* K, int N, int d, const int* pmem, const int* pptr,
                               int n_parents, int R, int* members, int* team_ptr, int* rep_token)
{
    if (N < 1 || d < 1 || R < 1 || n_parents < 1 || pptr[0] != 0 || pptr[n_parents] != N) return -1;
    int nmax = 0;
    for (int p = 0; p < n_parents; ++p) {
        int n = pptr[p + 1] - pptr[p];
        if (n < 0) return -1;
        if (n > nmax) nmax = n;
        for (int i = pptr[p]; i < pptr[p + 1]; ++i)
            if (pmem[i] < 0 || pmem[i] >= N || (i > pptr[p] && pmem[i] <= pmem[i - 1])) return -1;
    }
    int rmax = R < nmax ? R : nmax;
    double* mu = (double*)malloc(sizeof(double) * (size_t)d);
    int* reps = (int*)malloc(sizeof(int) * (size_t)rmax);
    int* is_rep = (int*)malloc(sizeof(int) * (size_t)nmax);
    int* owner = (int*)malloc(sizeof(int) * (size_t)nmax);
    /* D[u * n + i] = |k_i - k_{j_u}|^2 for member i of the current parent */
    double* D = (double*)malloc(sizeof(double) * (size_t)rmax * (size_t)nmax);
    if (!mu || !reps || !is_rep || !owner || !D) {
        free(mu); free(reps); free(is_rep); free(owner); free(D);
        return -1;
    }
    int M = 0, filled = 0;
    team_ptr[0] = 0;
    for (int p = 0; p < n_parents; ++p) {
        int n = pptr[p + 1] - pptr[p];
        if (n > 0)
            build_parent(K, d, pmem + pptr[p], n, R, mu, reps, is_rep, owner, D,
                         members, team_ptr, rep_token, &M, &filled);
    }
    free(mu); free(reps); free(is_rep); free(owner); free(D);
    return M;
}

/* Alg. "Contiguous parent partition" (C_u = [uP, min((u+1)P, N)), 0-indexed)
 * followed by the team construction above. */
int oracle_build_teams(const double* K, int N, int d, int P, int R,
                       int* members, int* team_ptr, int* rep_token)
{
    if (N < 1 || d < 1 || P < 1 || R < 1) return -1;
    int n_parents = (N + P - 1) / P;
    int* pmem = (int*)malloc(sizeof(int) * (size_t)N);
    int* pptr = (int*)malloc(sizeof(int) * (size_t)(n_parents + 1));
    if (!pmem || !pptr) {
        free(pmem); free(pptr);
        return -1;
    }
    for (int i = 0; i < N; ++i) pmem[i] = i;
    for (int p = 0; p <= n_parents; ++p) pptr[p] = (p * (long long)P < N) ? p * P : N;
    int M = oracle_build_teams_parents(K, N, d, pmem, pptr, n_parents, R, members, team_ptr, rep_token);
    free(pmem); free(pptr);
    return M;
}

/* ------------------------------------------------------------------------ */
/* Alg. "SANTA++ attention for one query head".                             */
/*                                                                           */
/* q[d]; K, V: [N, d] original (unpacked) prompt cache of the KV head;       */
/* teams as produced by oracle_build_teams; sK, sV: [T, d] exact suffix.     */
/* Routing (eq. method-routing): phi_g = log n_g + scale * q . l_g.           */
/* Sampling: Y_g = phi_g + G_g; S = the K' largest Y (ties: lower g);         */
/* tau = the (K'+1)-th largest Y.                                            */
/* Correction (eq. method-inclusion): c_g = 1 - exp(-exp(phi_g - tau)),      */
/* evaluated as -expm1(-exp(phi_g - tau)), the same quantity without the     */
/* cancellation of 1 - (value near 1).                                       */
/* Estimate (eq. method-estimate): U^ = U_E + sum_{g in S} U_g / c_g,        */
/* Z^ = Z_E + sum_{g in S} Z_g / c_g, o = U^ / Z^.                           */
/*                                                                           */
/* All exponentials are taken relative to a common shift m (the largest raw  */
/* score s_i among the rows read, or ref_shift when it is not NaN); U_hat    */
/* and Z_hat are returned in that shifted scale and *shift_out = m, so that  */
/* the unshifted sums are U_hat * e^m and Z_hat * e^m.                       */
/*                                                                           */
/* route_keys [M, d] (NULL: the representative keys K[rep_token[g]]) gives   */
/* the key each team is routed by: the centroid-guided variant routes by    */
/* the team mean (section "Attention-distribution diagnostic").              */
/* Optional outputs (NULL to skip): phi[M], Y[M]; sel[M] receives the        */
/* selected team ids in ascending order and c_sel[M] their corrections;      */
/* *tau_out is -inf when every team is selected.  Returns |S|, or -1.        */
/* ------------------------------------------------------------------------ */
typedef struct { double y; int g; } ranked_t;

static int rank_cmp(const void* a, const void* b)
{
    const ranked_t* x = (const ranked_t*)a;
    const ranked_t* y = (const ranked_t*)b;
    if (x->y > y->y) return -1;
    if (x->y < y->y) return 1;
    return (x->g < y->g) ? -1 : (x->g > y->g);
}

int oracle_decode_head(const double* q, int d,
                       const double* K, const double* V, int N,
                       const int* members, const int* team_ptr, const int* rep_token,
                       const double* route_keys, int M,
                       const double* sK, const double* sV, int T,
                       int Kbudget, uint64_t seed, uint64_t step, uint64_t b, uint64_t h,
                       double scale, double ref_shift,
                       double* out, double* U_hat, double* Z_hat, double* shift_out,
                       double* phi, double* Y, int* sel, double* c_sel, double* tau_out)
{
    if (d < 1 || N < 1 || M < 1 || T < 0 || Kbudget < 1) return -1;
    int Kp = Kbudget < M ? Kbudget : M;
    double* c = (double*)malloc(sizeof(double) * (size_t)M);      /* c_g of selected teams */
    char* in_S = (char*)malloc((size_t)M);                        /* g in S */
    double* ph = (double*)malloc(sizeof(double) * (size_t)M);
    double* yy = (double*)malloc(sizeof(double) * (size_t)M);
    ranked_t* rk = (ranked_t*)malloc(sizeof(ranked_t) * (size_t)M);
    if (!c || !in_S || !ph || !yy || !rk) {
        free(c); free(in_S); free(ph); free(yy); free(rk);
        return -1;
    }
    double tau = -INFINITY;

    if (Kp == M) {
        for (int g = 0; g < M; ++g) { c[g] = 1.0; in_S[g] = 1; ph[g] = NAN; yy[g] = NAN; }
    } else {
        for (int g = 0; g < M; ++g) {
            /* routing key: the representative's key, or route_keys[g] when given */
            const double* l = route_keys ? route_keys + (size_t)g * d : K + (size_t)rep_token[g] * d;
            double dot = 0.0;
            for (int j = 0; j < d; ++j) dot = dot + q[j] * l[j];
            int n_g = team_ptr[g + 1] - team_ptr[g];
            ph[g] = log((double)n_g) + scale * dot;
            yy[g] = ph[g] + oracle_team_gumbel(seed, step, b, h, (uint64_t)g);
            rk[g].y = yy[g];
            rk[g].g = g;
        }
        qsort(rk, (size_t)M, sizeof(ranked_t), rank_cmp);
        tau = rk[Kp].y;
        for (int g = 0; g < M; ++g) { c[g] = 0.0; in_S[g] = 0; }
        for (int t = 0; t < Kp; ++t) {
            int g = rk[t].g;
            in_S[g] = 1;
            c[g] = -expm1(-exp(ph[g] - tau));
        }
    }

    /* common shift: the largest raw score among all rows that are read */
    double m = ref_shift;
    if (isnan(m)) {
        m = -INFINITY;
        for (int g = 0; g < M; ++g) {
            if (!in_S[g]) continue;
            for (int t = team_ptr[g]; t < team_ptr[g + 1]; ++t) {
                const double* k = K + (size_t)members[t] * d;
                double dot = 0.0;
                for (int j = 0; j < d; ++j) dot = dot + q[j] * k[j];
                double s = scale * dot;
                if (s > m) m = s;
            }
        }
        for (int i = 0; i < T; ++i) {
            const double* k = sK + (size_t)i * d;
            double dot = 0.0;
            for (int j = 0; j < d; ++j) dot = dot + q[j] * k[j];
            double s = scale * dot;
            if (s > m) m = s;
        }
    }

    double Zh = 0.0;
    for (int j = 0; j < d; ++j) U_hat[j] = 0.0;
    double* Ug = (double*)malloc(sizeof(double) * (size_t)d);
    if (!Ug) { free(c); free(in_S); free(ph); free(yy); free(rk); return -1; }
    /* exact suffix */
    for (int i = 0; i < T; ++i) {
        const double* k = sK + (size_t)i * d;
        const double* v = sV + (size_t)i * d;
        double dot = 0.0;
        for (int j = 0; j < d; ++j) dot = dot + q[j] * k[j];
        double a = exp(scale * dot - m);
        Zh = Zh + a;
        for (int j = 0; j < d; ++j) U_hat[j] = U_hat[j] + a * v[j];
    }
    /* selected teams, each divided by its correction */
    for (int g = 0; g < M; ++g) {
        if (!in_S[g]) continue;
        double Zg = 0.0;
        for (int j = 0; j < d; ++j) Ug[j] = 0.0;
        for (int t = team_ptr[g]; t < team_ptr[g + 1]; ++t) {
            const double* k = K + (size_t)members[t] * d;
            const double* v = V + (size_t)members[t] * d;
            double dot = 0.0;
            for (int j = 0; j < d; ++j) dot = dot + q[j] * k[j];
            double a = exp(scale * dot - m);
            Zg = Zg + a;
            for (int j = 0; j < d; ++j) Ug[j] = Ug[j] + a * v[j];
        }
        Zh = Zh + Zg / c[g];
        for (int j = 0; j < d; ++j) U_hat[j] = U_hat[j] + Ug[j] / c[g];
    }
    for (int j = 0; j < d; ++j) out[j] = U_hat[j] / Zh;
    *Z_hat = Zh;
    *shift_out = m;

    int ns = 0;
    for (int g = 0; g < M; ++g) {
        if (phi) phi[g] = ph[g];
        if (Y) Y[g] = yy[g];
        if (in_S[g]) {
            if (sel) sel[ns] = g;
            if (c_sel) c_sel[ns] = c[g];
            ++ns;
        }
    }
    if (tau_out) *tau_out = tau;
    free(Ug); free(c); free(in_S); free(ph); free(yy); free(rk);
    return ns;
}

/* ------------------------------------------------------------------------ */
/* eq. method-attention: dense softmax attention over the prompt rows K, V   */
/* [N, d] followed by the suffix rows sK, sV [T, d].  Same shift convention  */
/* as oracle_decode_head.  Returns 0, or -1 on bad arguments.                */
/* ------------------------------------------------------------------------ */
int oracle_dense_head(const double* q, int d, const double* K, const double* V, int N,
                      const double* sK, const double* sV, int T, double scale,
                      double* out, double* U, double* Z, double* shift_out)
{
    if (d < 1 || N < 0 || T < 0 || N + T < 1) return -1;
    double* s = (double*)malloc(sizeof(double) * (size_t)(N + T));
    if (!s) return -1;
    double m = -INFINITY;
    for (int i = 0; i < N + T; ++i) {
        const double* k = (i < N) ? K + (size_t)i * d : sK + (size_t)(i - N) * d;
        double dot = 0.0;
        for (int j = 0; j < d; ++j) dot = dot + q[j] * k[j];
        s[i] = scale * dot;
        if (s[i] > m) m = s[i];
    }
    double z = 0.0;
    for (int j = 0; j < d; ++j) U[j] = 0.0;
    for (int i = 0; i < N + T; ++i) {
        const double* v = (i < N) ? V + (size_t)i * d : sV + (size_t)(i - N) * d;
        double a = exp(s[i] - m);
        z = z + a;
        for (int j = 0; j < d; ++j) U[j] = U[j] + a * v[j];
    }
    for (int j = 0; j < d; ++j) out[j] = U[j] / z;
    *Z = z;
    *shift_out = m;
    free(s);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Team means (the routing keys of the centroid-guided variant, section      */
/* "Attention-distribution diagnostic": the arithmetic mean of the group's  */
/* keys).  Per team and dimension the members' values are summed in team    */
/* order (ascending token index) and divided by n_g.  out: [M, d].          */
/* ------------------------------------------------------------------------ */
int oracle_team_means(const double* K, int d, const int* members, const int* team_ptr, int M,
                      double* out)
{
    if (d < 1 || M < 1) return -1;
    for (int g = 0; g < M; ++g) {
        int n = team_ptr[g + 1] - team_ptr[g];
        if (n < 1) return -1;
        for (int j = 0; j < d; ++j) {
            double s = 0.0;
            for (int t = team_ptr[g]; t < team_ptr[g + 1]; ++t) s = s + K[(size_t)members[t] * d + j];
            out[(size_t)g * d + j] = s / (double)n;
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Alg. "Global minibatch k-means parent partition" for one (sequence, KV    */
/* head), with the settings theta stated after the algorithm: greedy         */
/* k-means++ seeding on a sample, minibatches drawn with replacement,        */
/* cumulative-count center updates, small-center reassignment and a          */
/* no-improvement stopping rule.  The paper fixes these through a library's  */
/* defaults; the steps below are this implementation's reading of them.     */
/*                                                                           */
/* Random words: Philox4x64-10, key (seed, 1), counter (a / 4, tag, s, 0),    */
/* output word a mod 4.  An index in [0, n) is floor(w n / 2^64); a uniform  */
/* in [0, 1) is (w >> 11) 2^-53.  The draws do not depend on the head.       */
/*   tag 0  init sample: s0 token indices (a = position in the sample)        */
/*   tag 1  first center: a sample position (a = 0)                           */
/*   tag 2  k-means++ trial a of center s                                     */
/*   tag 3  minibatch step s: token index of batch position a                 */
/*   tag 4  minibatch step s: batch position of the a-th reassigned center    */
/*                                                                           */
/* Seeding (greedy k-means++): s0 = init_size, or 3 * batch when 0, raised   */
/* to 3M when below M, capped at N.  Center 0 is a uniform sample point;     */
/* each later center draws L = 2 + floor(ln M) candidates, candidate t being  */
/* the first sample position whose running sum of D^2 (index order) exceeds  */
/* u_t times the total (the last position if none), and keeps the candidate  */
/* whose potential sum_j min(D^2_j, |x_j - cand|^2) is smallest (ties: the    */
/* earlier trial).  D^2_j is the squared distance to the nearest center.     */
/*                                                                           */
/* Steps: S = floor(max_iter N / batch).  Step s assigns every batch point to */
/* its nearest center (ties: lowest index; e = that distance) and updates     */
/* each center u that got n_u > 0 points:                                    */
/*   mu_u <- (mu_u w_u + sum of its points in batch order) / (w_u + n_u),    */
/*   w_u <- w_u + n_u   (w starts at 0).                                     */
/* Reassignment (ratio > 0): the centers with w_u < ratio * max w, at most   */
/* floor(batch / 2) of them in index order, each move to a batch point drawn */
/* uniformly (tag 4) and get w_u = the smallest w of the centers kept.       */
/* Stopping: I_s = mean e over the batch; the smoothed inertia is I_0, then  */
/* ewa (1 - alpha) + I_s alpha with alpha = min(1, 2 batch / (N + 1)); after */
/* max_no_improvement consecutive steps without a new minimum of it the loop */
/* ends (0: never).                                                          */
/* Final labels: nearest center of every token (ties: lowest index).         */
/*                                                                           */
/* X: [N, d].  Outputs: centers[M * d], labels[N], *steps_out = steps run,   */
/* init_centers[M * d] (NULL to skip) = the seeding result.  Returns 0 or -1. */
/* ------------------------------------------------------------------------ */
static uint64_t km_word(uint64_t seed, uint64_t a, uint64_t tag, uint64_t s)
{
    uint64_t ctr[4] = { a >> 2, tag, s, 0 };
    uint64_t key[2] = { seed, 1 };
    uint64_t out[4];
    philox4x64_10(ctr, key, out);
    return out[a & 3];
}

static uint64_t draw_index(uint64_t w, uint64_t n)
{
    return (uint64_t)(((unsigned __int128)w * n) >> 64);
}

static double draw_unit(uint64_t w)
{
    return (double)(w >> 11) * 0x1.0p-53;
}

static int nearest_center(const double* x, const double* C, int M, int d, double* dist)
{
    int best = 0;
    double bd = sqdist(x, C, d);
    for (int u = 1; u < M; ++u) {
        double t = sqdist(x, C + (size_t)u * d, d);
        if (t < bd) { bd = t; best = u; }
    }
    *dist = bd;
    return best;
}

int oracle_kmeans(const double* X, int N, int d, int M, int batch, int max_iter,
                  int max_no_improvement, double ratio, int init_size, uint64_t seed,
                  double* centers, int* labels, int* steps_out, double* init_centers)
{
    if (N < 1 || d < 1 || M < 1 || M > N || batch < 1 || max_iter < 0 || max_no_improvement < 0 ||
        !(ratio >= 0.0 && ratio < 1.0) || init_size < 0)
        return -1;
    int s0 = init_size > 0 ? init_size : 3 * batch;
    if (s0 < M) s0 = 3 * M;
    if (s0 > N) s0 = N;
    const int L = 2 + (int)floor(log((double)M));
    int* samp = (int*)malloc(sizeof(int) * (size_t)s0);
    double* D = (double*)malloc(sizeof(double) * (size_t)s0);
    double* cum = (double*)malloc(sizeof(double) * (size_t)s0);
    double* Dt = (double*)malloc(sizeof(double) * (size_t)L * (size_t)s0);
    double* w = (double*)malloc(sizeof(double) * (size_t)M);
    double* S = (double*)malloc(sizeof(double) * (size_t)M * (size_t)d);
    int* n = (int*)malloc(sizeof(int) * (size_t)M);
    int* mark = (int*)malloc(sizeof(int) * (size_t)M);
    int* idx = (int*)malloc(sizeof(int) * (size_t)batch);
    int* a = (int*)malloc(sizeof(int) * (size_t)batch);
    if (!samp || !D || !cum || !Dt || !w || !S || !n || !mark || !idx || !a) {
        free(samp); free(D); free(cum); free(Dt); free(w); free(S); free(n); free(mark); free(idx); free(a);
        return -1;
    }
#define XR(i) (X + (size_t)(i) * d)

    /* greedy k-means++ on the sample */
    for (int j = 0; j < s0; ++j) samp[j] = (int)draw_index(km_word(seed, j, 0, 0), (uint64_t)N);
    int c0 = samp[draw_index(km_word(seed, 0, 1, 0), (uint64_t)s0)];
    memcpy(centers, XR(c0), sizeof(double) * (size_t)d);
    for (int j = 0; j < s0; ++j) D[j] = sqdist(XR(samp[j]), centers, d);
    for (int c = 1; c < M; ++c) {
        double run = 0.0;
        for (int j = 0; j < s0; ++j) {
            run = run + D[j];
            cum[j] = run;
        }
        int best_t = -1, best_cand = 0;
        double best_pot = 0.0;
        for (int t = 0; t < L; ++t) {
            double target = draw_unit(km_word(seed, t, 2, c)) * run;
            int cand = s0 - 1;
            for (int j = 0; j < s0; ++j)
                if (cum[j] > target) { cand = j; break; }
            double pot = 0.0;
            for (int j = 0; j < s0; ++j) {
                double e = sqdist(XR(samp[j]), XR(samp[cand]), d);
                double m = e < D[j] ? e : D[j];
                Dt[(size_t)t * s0 + j] = m;
                pot = pot + m;
            }
            if (best_t < 0 || pot < best_pot) { best_t = t; best_pot = pot; best_cand = cand; }
        }
        memcpy(centers + (size_t)c * d, XR(samp[best_cand]), sizeof(double) * (size_t)d);
        memcpy(D, Dt + (size_t)best_t * s0, sizeof(double) * (size_t)s0);
    }
    if (init_centers) memcpy(init_centers, centers, sizeof(double) * (size_t)M * d);

    /* minibatch steps */
    long long steps = (long long)max_iter * N / batch;
    double alpha = 2.0 * batch / ((double)N + 1.0);
    if (alpha > 1.0) alpha = 1.0;
    double ewa = 0.0, ewa_min = INFINITY;
    int no_imp = 0, run_steps = 0;
    for (int u = 0; u < M; ++u) w[u] = 0.0;
    for (long long s = 0; s < steps; ++s) {
        double inert = 0.0;
        for (int j = 0; j < batch; ++j) {
            double e;
            idx[j] = (int)draw_index(km_word(seed, j, 3, (uint64_t)s), (uint64_t)N);
            a[j] = nearest_center(XR(idx[j]), centers, M, d, &e);
            inert = inert + e;
        }
        inert = inert / (double)batch;

        /* cumulative-count update */
        for (int u = 0; u < M; ++u) n[u] = 0;
        for (size_t k = 0; k < (size_t)M * d; ++k) S[k] = 0.0;
        for (int j = 0; j < batch; ++j) {
            n[a[j]] += 1;
            for (int k = 0; k < d; ++k) S[(size_t)a[j] * d + k] = S[(size_t)a[j] * d + k] + XR(idx[j])[k];
        }
        for (int u = 0; u < M; ++u) {
            if (n[u] == 0) continue;
            for (int k = 0; k < d; ++k) {
                double* m = centers + (size_t)u * d + k;
                *m = (*m * w[u] + S[(size_t)u * d + k]) / (w[u] + (double)n[u]);
            }
            w[u] = w[u] + (double)n[u];
        }

        /* reassignment of centers with too few points */
        if (ratio > 0.0) {
            double wmax = w[0];
            for (int u = 1; u < M; ++u)
                if (w[u] > wmax) wmax = w[u];
            double thr = ratio * wmax;
            int count = 0;
            for (int u = 0; u < M; ++u) {
                mark[u] = (w[u] < thr && count < batch / 2) ? 1 : 0;
                count += mark[u];
            }
            if (count > 0) {
                double wkeep = INFINITY;
                for (int u = 0; u < M; ++u)
                    if (!mark[u] && w[u] < wkeep) wkeep = w[u];
                int r = 0;
                for (int u = 0; u < M; ++u) {
                    if (!mark[u]) continue;
                    int j = (int)draw_index(km_word(seed, r, 4, (uint64_t)s), (uint64_t)batch);
                    memcpy(centers + (size_t)u * d, XR(idx[j]), sizeof(double) * (size_t)d);
                    w[u] = wkeep;
                    ++r;
                }
            }
        }
        run_steps = (int)(s + 1);

        /* smoothed minibatch inertia and the stopping rule */
        ewa = (s == 0) ? inert : ewa * (1.0 - alpha) + inert * alpha;
        if (ewa < ewa_min) {
            ewa_min = ewa;
            no_imp = 0;
        } else {
            ++no_imp;
        }
        if (max_no_improvement > 0 && no_imp >= max_no_improvement) break;
    }
    for (int i = 0; i < N; ++i) {
        double e;
        labels[i] = nearest_center(XR(i), centers, M, d, &e);
    }
    *steps_out = run_steps;
#undef XR
    free(samp); free(D); free(cum); free(Dt); free(w); free(S); free(n); free(mark); free(idx); free(a);
    return 0;
}
