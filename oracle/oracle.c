/*
 * CPU float64 oracle for tree-structured WY verification of the gated delta rule.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file: only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header or constant with the
 * HIP library; both sides only read the same seeded inputs.
 *
 * What it computes is the plain definition, not the paper's closed form.
 * Per (sequence, head) unit, with S_{-1} := S0 and the draft nodes visited in
 * index order (parents precede children, Method: "Verifying a draft"):
 *
 *   P        = state of parent(t)                        (S0 when parent(t) == -1)
 *   vt_t     = beta_t (v_t - alpha_t P k_t)                (Method: "Key rewrite")
 *   S_t      = alpha_t P (I - beta_t k_t k_t^T) + beta_t v_t k_t^T      (eq. 1)
 *   o_t      = S_t q_t                                                  (eq. 1)
 *
 * which is the gated delta rule run along every root-to-node path, each parent
 * state computed once.  The matrix product P (I - beta k k^T) is written out
 * entry by entry as P - beta (P k) k^T; nothing else is rearranged.  Commit
 * (eq. 3's left-hand side) is the state reached by running eq. 1 along the
 * accepted root-to-node path from S0; an empty path leaves S0.
 *
 * States are d_v x d_k, row-major (Background: S in R^{d_v x d_k}, o = S q).
 * All arithmetic is float64.  Units are independent, so they are spread over
 * OpenMP threads; nothing inside a unit is blocked or reordered.
 *
 * Every function returns 0 on success, or a negative code:
 *   -1  a parent index outside [-1, t-1]
 *   -2  a path that is not a root-to-node path of the tree
 *   -3  bad sizes, or out of memory
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* One step of eq. 1 from state P (d_v x d_k) with token (k, v, alpha, beta).
 * Writes the new state to S (may not alias P), the pseudo-value to vt
 * (nullable) and, when q is given, o = S q to o. */
static void gdn_step(const double *P, const double *q, const double *k, const double *v,
                     double alpha, double beta, int dk, int dv,
                     double *S, double *vt, double *o) {
    for (int r = 0; r < dv; ++r) {
        const double *Pr = P + (size_t)r * dk;
        double *Sr = S + (size_t)r * dk;
        double Pk = 0.0;                                   /* (P k)_r */
        for (int c = 0; c < dk; ++c) Pk += Pr[c] * k[c];
        if (vt) vt[r] = beta * (v[r] - alpha * Pk);        /* key rewrite */
        for (int c = 0; c < dk; ++c)                       /* eq. 1, row r */
            Sr[c] = alpha * (Pr[c] - beta * Pk * k[c]) + beta * v[r] * k[c];
        if (o) {
            double acc = 0.0;                              /* o = S_t q_t */
            for (int c = 0; c < dk; ++c) acc += Sr[c] * q[c];
            o[r] = acc;
        }
    }
}

/* Verify: every node's output o_t and pseudo-value vt_t, optionally every
 * node's state.
 *   S0      [U, dv, dk]     q, k [U, N, dk]    v [U, N, dv]
 *   alpha, beta [U, N]      parent [U, N] (per unit; -1 = child of S0)
 *   o, vt   [U, N, dv]      states [U, N, dv, dk] or NULL                  */
int oracle_gdn_tree(int U, int N, int dk, int dv, const double *S0, const double *q,
                    const double *k, const double *v, const double *alpha, const double *beta,
                    const int32_t *parent, double *o, double *vt, double *states) {
    if (U < 0 || N < 1 || dk < 1 || dv < 1) return -3;
    for (int u = 0; u < U; ++u)
        for (int t = 0; t < N; ++t) {
            int p = parent[(size_t)u * N + t];
            if (p < -1 || p >= t) return -1;
        }
    const size_t SS = (size_t)dv * dk;
    int status = 0;
#pragma omp parallel
    {
        double *scratch = states ? NULL : (double *)malloc(sizeof(double) * SS * (size_t)N);
        if (!states && !scratch) {
#pragma omp atomic write
            status = -3;
        }
#pragma omp for schedule(dynamic)
        for (int u = 0; u < U; ++u) {
            if (!states && !scratch) continue;
            double *St = states ? states + (size_t)u * N * SS : scratch;
            const double *S0u = S0 + (size_t)u * SS;
            for (int t = 0; t < N; ++t) {
                size_t ut = (size_t)u * N + t;
                int p = parent[ut];
                const double *P = (p < 0) ? S0u : St + (size_t)p * SS;
                gdn_step(P, q + ut * dk, k + ut * dk, v + ut * dv, alpha[ut], beta[ut], dk, dv,
                         St + (size_t)t * SS, vt + ut * dv, o + ut * dv);
            }
        }
        free(scratch);
    }
    return status;
}

/* Warm-up: run eq. 1 in place over a chain of T tokens, state only.
 *   S [U, dv, dk] in/out    k [U, T, dk]   v [U, T, dv]   alpha, beta [U, T] */
int oracle_gdn_chain(int U, int T, int dk, int dv, double *S, const double *k, const double *v,
                     const double *alpha, const double *beta) {
    if (U < 0 || T < 0 || dk < 1 || dv < 1) return -3;
    const size_t SS = (size_t)dv * dk;
    int status = 0;
#pragma omp parallel
    {
        double *tmp = (double *)malloc(sizeof(double) * SS);
        if (!tmp) {
#pragma omp atomic write
            status = -3;
        }
#pragma omp for schedule(dynamic)
        for (int u = 0; u < U; ++u) {
            if (!tmp) continue;
            double *Su = S + (size_t)u * SS;
            for (int t = 0; t < T; ++t) {
                size_t ut = (size_t)u * T + t;
                gdn_step(Su, NULL, k + ut * dk, v + ut * dv, alpha[ut], beta[ut], dk, dv, tmp, NULL, NULL);
                memcpy(Su, tmp, sizeof(double) * SS);
            }
        }
        free(tmp);
    }
    return status;
}

/* Commit: the state of the accepted node, by running eq. 1 along the
 * root-to-node path from S0 (eq. 3's left-hand side).
 *   path [U, L_max] (root first), path_len [U] (0 = keep S0),
 *   parent [U, N] checks that the path really is a root-to-node path.
 *   S_out [U, dv, dk]                                                      */
int oracle_commit(int U, int N, int dk, int dv, int L_max, const double *S0, const double *k,
                  const double *v, const double *alpha, const double *beta, const int32_t *parent,
                  const int32_t *path, const int32_t *path_len, double *S_out) {
    if (U < 0 || N < 1 || dk < 1 || dv < 1 || L_max < 0) return -3;
    for (int u = 0; u < U; ++u) {
        int L = path_len[u];
        if (L < 0 || L > L_max) return -2;
        int prev = -1;
        for (int l = 0; l < L; ++l) {
            int a = path[(size_t)u * L_max + l];
            if (a < 0 || a >= N || parent[(size_t)u * N + a] != prev) return -2;
            prev = a;
        }
    }
    const size_t SS = (size_t)dv * dk;
    int status = 0;
#pragma omp parallel
    {
        double *tmp = (double *)malloc(sizeof(double) * SS);
        if (!tmp) {
#pragma omp atomic write
            status = -3;
        }
#pragma omp for schedule(dynamic)
        for (int u = 0; u < U; ++u) {
            if (!tmp) continue;
            double *Su = S_out + (size_t)u * SS;
            memcpy(Su, S0 + (size_t)u * SS, sizeof(double) * SS);
            for (int l = 0; l < path_len[u]; ++l) {
                size_t ua = (size_t)u * N + path[(size_t)u * L_max + l];
                gdn_step(Su, NULL, k + ua * dk, v + ua * dv, alpha[ua], beta[ua], dk, dv, tmp, NULL, NULL);
                memcpy(Su, tmp, sizeof(double) * SS);
            }
        }
        free(tmp);
    }
    return status;
}
