/*
 * Drives every entry point of the CPU oracle over seeded random small cases
 * and over invalid arguments, so that a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer can check its memory accesses and arithmetic.
 * Built by tests/test_oracle_sanitizers.py (gcc, host code only); prints
 * "ok" and exits 0 when every call returned and no sanitizer fired.
 */
#include <stdio.h>
#include <stdlib.h>

#include "../oracle/orloj_oracle.c"

static uint64_t state = 0x2209001590ull;

static uint64_t next_u64(void) {
    uint64_t z = (state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

static int below(int n) { return (int)(next_u64() % (uint64_t)n); }
static double unit(void) { return (double)(next_u64() >> 11) * 0x1.0p-53; }

static int cmp_double(const void *a, const void *b) {
    double x = *(const double *)a, y = *(const double *)b;
    return (x > y) - (x < y);
}

static void *xmalloc(size_t n) {
    void *p = malloc(n ? n : 1);
    if (!p) {
        fprintf(stderr, "out of memory\n");
        exit(2);
    }
    return p;
}

static int one_case(int it) {
    const int C = 1 + below(4), K = 1 + below(40), B = 1 + below(4);
    int32_t bs[4];
    int s = 0;
    for (int i = 0; i < B; ++i) bs[i] = (s += 1 + below(5));
    const int64_t N = below(14);
    const double w = 0.25 + 2.0 * unit(), now = 500.0, b = it % 3 == 0 ? 1e-4 : 0.05;
    uint32_t *counts = xmalloc(sizeof(uint32_t) * (size_t)B * C * K);
    for (int r = 0; r < B * C; ++r) {
        uint64_t tot = 0;
        for (int k = 0; k < K; ++k) {
            counts[(size_t)r * K + k] = below(3) == 0 ? 0u : (uint32_t)below(50);
            tot += counts[(size_t)r * K + k];
        }
        if (tot == 0) counts[(size_t)r * K + K - 1] = 1;
    }
    int32_t *cls = xmalloc(sizeof(int32_t) * (size_t)N);
    double *dl = xmalloc(sizeof(double) * (size_t)N), *cost = xmalloc(sizeof(double) * (size_t)N);
    for (int64_t i = 0; i < N; ++i) {
        cls[i] = below(C);
        dl[i] = now - 5.0 + 80.0 * unit();
        cost[i] = 3.0 * unit();
    }
    qsort(dl, (size_t)N, sizeof(double), cmp_double);
    for (int mode = 0; mode < 2; ++mode) {
        int64_t nc = 0, np = 0;
        for (int i = 0; i < B; ++i) {
            const int64_t c = mode ? N : (N < bs[i] ? N : bs[i]);
            nc += c;
            np += c * (c + 1) / 2;
        }
        double *P = xmalloc(sizeof(double) * (size_t)np), *pr = xmalloc(sizeof(double) * (size_t)np);
        double *E = xmalloc(sizeof(double) * (size_t)nc), *EL = xmalloc(sizeof(double) * (size_t)nc);
        double *S = xmalloc(sizeof(double) * (size_t)nc);
        int32_t sn, sb;
        double ss;
        if (orloj_oracle_score_model(C, K, B, bs, w, counts, N, cls, dl, it % 2 ? cost : NULL, now,
                                     b, mode, P, pr, E, EL, S, &sn, &sb, &ss))
            return 1;
        if (orloj_oracle_score_model_affine(C, K, B, bs, w, counts, 0.5 * unit(), 0.1 + unit(), N,
                                            cls, dl, it % 2 ? cost : NULL, now, b, mode, P, pr, E,
                                            EL, S, &sn, &sb, &ss))
            return 1;
        free(P); free(pr); free(E); free(EL); free(S);
    }
    {
        int32_t *tout = xmalloc(sizeof(int32_t) * (size_t)N), *batch = xmalloc(sizeof(int32_t) * (size_t)bs[B - 1]);
        double *score = xmalloc(sizeof(double) * (size_t)N);
        int32_t cand = 0, bn = 0;
        double *wts = xmalloc(sizeof(double) * (size_t)C);
        for (int c = 0; c < C; ++c) wts[c] = 0.1 + unit();
        int64_t *soff = xmalloc(sizeof(int64_t) * (size_t)(N + 1));
        double *sdl = xmalloc(sizeof(double) * (size_t)(2 * N)), *scost = xmalloc(sizeof(double) * (size_t)(2 * N));
        soff[0] = 0;
        for (int64_t i = 0; i < N; ++i) {
            const int k = 1 + below(2);
            soff[i + 1] = soff[i] + k;
            for (int j = 0; j < k; ++j) {
                sdl[soff[i] + j] = dl[i] + 10.0 * j;
                scost[soff[i] + j] = 1.0 + j;
            }
        }
        if (orloj_oracle_iterate_model(C, K, B, bs, w, counts, it % 2 ? wts : NULL, N, cls, dl,
                                       it % 2 ? cost : NULL, it % 3 ? soff : NULL,
                                       it % 3 ? sdl : NULL, it % 3 ? scost : NULL, now, b, tout,
                                       score, &cand, batch, &bn))
            return 1;
        free(tout); free(batch); free(score); free(wts); free(soff); free(sdl); free(scost);
    }
    {
        const int64_t ns = 50;
        int32_t *mo = xmalloc(sizeof(int32_t) * ns), *bi = xmalloc(sizeof(int32_t) * ns),
                *cl = xmalloc(sizeof(int32_t) * ns);
        double *lat = xmalloc(sizeof(double) * ns);
        for (int64_t i = 0; i < ns; ++i) {
            mo[i] = below(2) - (i == 7);          /* some out of range */
            bi[i] = below(B);
            cl[i] = below(C + 1);                 /* some out of range */
            lat[i] = i == 3 ? -1.0 : 100.0 * unit();
        }
        uint32_t *acc = xmalloc(sizeof(uint32_t) * (size_t)B * C * K);
        for (size_t r = 0; r < (size_t)B * C * K; ++r) acc[r] = counts[r];
        double wm = w;
        int64_t rej = 0;
        if (orloj_oracle_accumulate(1, B, C, K, &wm, ns, mo, bi, cl, lat, acc, &rej)) return 1;
        free(mo); free(bi); free(cl); free(lat); free(acc);
    }
    free(counts); free(cls); free(dl); free(cost);
    return 0;
}

int main(void) {
    for (int it = 0; it < 3000; ++it)
        if (one_case(it)) {
            fprintf(stderr, "case %d: an oracle call failed\n", it);
            return 1;
        }
    /* invalid arguments are rejected, not dereferenced */
    int32_t bs[2] = {2, 1}, sn, sb;
    double ss;
    uint32_t cnt[4] = {1, 2, 3, 4};
    if (orloj_oracle_cdf(0, cnt, NULL) != ORACLE_E_INVALID) return 1;
    if (orloj_oracle_score_model(1, 4, 2, bs, 1.0, cnt, 0, NULL, NULL, NULL, 0.0, 1e-4, 0, NULL,
                                 NULL, NULL, NULL, NULL, &sn, &sb, &ss) != ORACLE_E_INVALID)
        return 1;
    uint32_t zero[4] = {0, 0, 0, 0};
    double G[5];
    if (orloj_oracle_batch_cdf(4, 1, zero, G) != ORACLE_E_DATA) return 1;
    printf("ok\n");
    return 0;
}
