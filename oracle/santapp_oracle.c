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
/* Team construction for one (sequence, KV head).                            */
/*                                                                           */
/* Parents: contiguous spans C_u = [uP, min((u+1)P, N)) (0-indexed).         */
/* Per parent C (members in ascending token order):                          */
/*   r = min(R, |C|), mu = mean of the member keys,                           */
/*   j_1 = argmin_i |k_i - mu|^2,                                            */
/*   j_u = argmax over non-representatives of min_{j in L} |k_i - k_j|^2,    */
/*   b_i = argmin_u |k_i - k_{j_u}|^2, then b_{j_u} = u (self-ownership),     */
/*   teams appended in representative order u = 1..r.                        */
/* Ties: representative choice by lowest token index, assignment by          */
/* representative-selection order.                                           */
/*                                                                           */
/* K: [N, d] row-major.  Outputs, in team order: members[N] (the token       */
/* indices of team 0 ascending, then team 1, ...), team_ptr[M+1] (CSR        */
/* offsets into members) and rep_token[M].  The caller sizes team_ptr and    */
/* rep_token for at most N teams.  Returns M, or -1 on bad arguments.        */
/* ------------------------------------------------------------------------ */
int oracle_build_teams(const double* K, int N, int d, int P, int R,
                       int* members, int* team_ptr, int* rep_token)
{
    if (N < 1 || d < 1 || P < 1 || R < 1) return -1;
    double* mu = (double*)malloc(sizeof(double) * (size_t)d);
    int* reps = (int*)malloc(sizeof(int) * (size_t)R);
    int* is_rep = (int*)malloc(sizeof(int) * (size_t)P);
    int* owner = (int*)malloc(sizeof(int) * (size_t)P);
    /* D[u * P + i] = |k_i - k_{j_u}|^2 for member i of the current parent */
    double* D = (double*)malloc(sizeof(double) * (size_t)R * (size_t)P);
    if (!mu || !reps || !is_rep || !owner || !D) {
        free(mu); free(reps); free(is_rep); free(owner); free(D);
        return -1;
    }
    int M = 0, filled = 0;
    team_ptr[0] = 0;
    int n_parents = (N + P - 1) / P;
    for (int p = 0; p < n_parents; ++p) {
        int start = p * P;
        int n = (start + P <= N) ? P : N - start;
        int r = R < n ? R : n;
        const double* Kc = K + (size_t)start * d;

        for (int j = 0; j < d; ++j) {
            double s = 0.0;
            for (int i = 0; i < n; ++i) s = s + Kc[(size_t)i * d + j];
            mu[j] = s / (double)n;
        }
        for (int i = 0; i < n; ++i) is_rep[i] = 0;

        /* first representative: the member nearest the parent mean */
        int best = 0;
        double best_d = sqdist(Kc, mu, d);
        for (int i = 1; i < n; ++i) {
            double t = sqdist(Kc + (size_t)i * d, mu, d);
            if (t < best_d) { best_d = t; best = i; }
        }
        reps[0] = best;
        is_rep[best] = 1;
        for (int i = 0; i < n; ++i)
            D[i] = sqdist(Kc + (size_t)i * d, Kc + (size_t)best * d, d);

        /* farthest-first: maximise the distance to the nearest chosen rep */
        for (int u = 1; u < r; ++u) {
            int pick = -1;
            double pick_d = -1.0;
            for (int i = 0; i < n; ++i) {
                if (is_rep[i]) continue;
                double m = D[i];
                for (int v = 1; v < u; ++v)
                    if (D[(size_t)v * P + i] < m) m = D[(size_t)v * P + i];
                if (pick < 0 || m > pick_d) { pick = i; pick_d = m; }
            }
            reps[u] = pick;
            is_rep[pick] = 1;
            for (int i = 0; i < n; ++i)
                D[(size_t)u * P + i] = sqdist(Kc + (size_t)i * d, Kc + (size_t)pick * d, d);
        }

        /* nearest-representative assignment, then representative self-ownership */
        for (int i = 0; i < n; ++i) {
            int bu = 0;
            double bd = D[i];
            for (int u = 1; u < r; ++u)
                if (D[(size_t)u * P + i] < bd) { bd = D[(size_t)u * P + i]; bu = u; }
            owner[i] = bu;
        }
        for (int u = 0; u < r; ++u) owner[reps[u]] = u;

        /* emit teams in representative order, members ascending */
        for (int u = 0; u < r; ++u) {
            for (int i = 0; i < n; ++i)
                if (owner[i] == u) members[filled++] = start + i;
            rep_token[M] = start + reps[u];
            team_ptr[M + 1] = filled;
            ++M;
        }
    }
    free(mu); free(reps); free(is_rep); free(owner); free(D);
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
