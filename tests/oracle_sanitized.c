/*
 * Request/response driver around the oracle, for running the oracle's pins
 * with AddressSanitizer and UndefinedBehaviorSanitizer (test-only).
 *
 * Built together with oracle/oracle.c by tests/test_oracle_sanitized.py as a
 * standalone executable, so the sanitizer runtimes come first in its own
 * library list.  Every array of a request is copied into a heap buffer of
 * exactly its size, so a read or write one element past any array lands in
 * a redzone and stops the process with a report.
 *
 * Protocol on stdin / stdout, native byte order:
 *   request  = int32 op, int32 sizes[...], then the input arrays
 *   response = int32 status, then the output arrays (only when status == 0)
 *   op 0 quit; op 1 threads -> int32; op 2 tree (U, N, dk, dv, with_states);
 *   op 3 chain (U, T, dk, dv); op 4 commit (U, N, dk, dv, L_max).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_threads(void);
int oracle_gdn_tree(int U, int N, int dk, int dv, const double *S0, const double *q, const double *k,
                    const double *v, const double *alpha, const double *beta, const int32_t *parent,
                    double *o, double *vt, double *states);
int oracle_gdn_chain(int U, int T, int dk, int dv, double *S, const double *k, const double *v,
                     const double *alpha, const double *beta);
int oracle_commit(int U, int N, int dk, int dv, int L_max, const double *S0, const double *k, const double *v,
                  const double *alpha, const double *beta, const int32_t *parent, const int32_t *path,
                  const int32_t *path_len, double *S_out);

static void die(const char *what) {
    fprintf(stderr, "oracle_sanitized: %s\n", what);
    exit(2);
}

static void *take(size_t count, size_t elem) {
    void *p = malloc(count ? count * elem : 1);
    if (!p) die("out of memory");
    if (count && fread(p, elem, count, stdin) != count) die("short read");
    return p;
}

static void *space(size_t count, size_t elem) {
    void *p = malloc(count ? count * elem : 1);
    if (!p) die("out of memory");
    return p;
}

static void give(const void *p, size_t count, size_t elem) {
    if (count && fwrite(p, elem, count, stdout) != count) die("short write");
}

static void give_status(int32_t s) { give(&s, 1, sizeof s); }

static int32_t get_int(void) {
    int32_t x;
    if (fread(&x, sizeof x, 1, stdin) != 1) die("short read");
    return x;
}

int main(void) {
    for (;;) {
        const int32_t op = get_int();
        if (op == 0) return 0;
        if (op == 1) {
            give_status(0);
            give_status(oracle_threads());
        } else if (op == 2) {
            const int U = get_int(), N = get_int(), dk = get_int(), dv = get_int(), with_states = get_int();
            if (U < 0 || N < 0 || dk < 0 || dv < 0) die("bad sizes");
            const size_t un = (size_t)U * N;
            double *S0 = take((size_t)U * dv * dk, 8), *q = take(un * dk, 8), *k = take(un * dk, 8);
            double *v = take(un * dv, 8), *alpha = take(un, 8), *beta = take(un, 8);
            int32_t *parent = take(un, 4);
            double *o = space(un * dv, 8), *vt = space(un * dv, 8);
            double *st = with_states ? space(un * dv * dk, 8) : NULL;
            const int32_t rc = oracle_gdn_tree(U, N, dk, dv, S0, q, k, v, alpha, beta, parent, o, vt, st);
            give_status(rc);
            if (rc == 0) {
                give(o, un * dv, 8);
                give(vt, un * dv, 8);
                if (st) give(st, un * dv * dk, 8);
            }
            free(S0), free(q), free(k), free(v), free(alpha), free(beta), free(parent), free(o), free(vt), free(st);
        } else if (op == 3) {
            const int U = get_int(), T = get_int(), dk = get_int(), dv = get_int();
            if (U < 0 || T < 0 || dk < 0 || dv < 0) die("bad sizes");
            const size_t ut = (size_t)U * T;
            double *S = take((size_t)U * dv * dk, 8), *k = take(ut * dk, 8), *v = take(ut * dv, 8);
            double *alpha = take(ut, 8), *beta = take(ut, 8);
            const int32_t rc = oracle_gdn_chain(U, T, dk, dv, S, k, v, alpha, beta);
            give_status(rc);
            if (rc == 0) give(S, (size_t)U * dv * dk, 8);
            free(S), free(k), free(v), free(alpha), free(beta);
        } else if (op == 4) {
            const int U = get_int(), N = get_int(), dk = get_int(), dv = get_int(), L_max = get_int();
            if (U < 0 || N < 0 || dk < 0 || dv < 0 || L_max < 0) die("bad sizes");
            const size_t un = (size_t)U * N;
            double *S0 = take((size_t)U * dv * dk, 8), *k = take(un * dk, 8), *v = take(un * dv, 8);
            double *alpha = take(un, 8), *beta = take(un, 8);
            int32_t *parent = take(un, 4), *path = take((size_t)U * L_max, 4), *path_len = take(U, 4);
            double *out = space((size_t)U * dv * dk, 8);
            const int32_t rc = oracle_commit(U, N, dk, dv, L_max, S0, k, v, alpha, beta, parent, path, path_len, out);
            give_status(rc);
            if (rc == 0) give(out, (size_t)U * dv * dk, 8);
            free(S0), free(k), free(v), free(alpha), free(beta), free(parent), free(path), free(path_len), free(out);
        } else {
            die("unknown op");
        }
        if (fflush(stdout) != 0) die("flush");
    }
}
