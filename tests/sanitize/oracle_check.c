/*
 * Runs every entry point of the C oracle (oracle/tl_oracle.c, compiled into
 * this program) on seeded random and edge-case inputs, meant to run under
 * AddressSanitizer and UndefinedBehaviorSanitizer: empty and ragged
 * scenarios, malformed entries, queued and arriving requests under a batch
 * cap and a binding KV capacity, lost requests, the size guard, horizon 1,
 * large blocks; feature rows with 3 and 4 features; forests of depth 0 to 12
 * with NaN and infinite thresholds and NaN rows; selection with IPS 0,
 * negative, NaN, infinite and tiny, and the binary search.  Prints a checksum
 * of all outputs; a sanitizer report or a nonzero return code fails it.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int tlo_project(int64_t S, int32_t H, int32_t N, const int64_t* req_offset, const int32_t* prompt,
                const int32_t* generated, const int32_t* remaining, const int32_t* arrival,
                const uint64_t* deadline_ns, const uint8_t* lost, const int32_t* kv_capacity,
                const int32_t* batch_cap, int32_t* batch, int32_t* kv, uint64_t* deadline_at, int32_t* n_iters,
                uint32_t* flags, int32_t* admit_iter);
int tlo_rows(int64_t S, int32_t F, int32_t H, int32_t n_features, const float* freqs, const int32_t* batch,
             const int32_t* kv, const float* engine, float* rows);
int tlo_forest_predict(int32_t n_trees, int32_t depth, int32_t n_features, float base_score, const uint8_t* feature,
                       const float* threshold, const float* leaf, const float* rows, int64_t n_rows, float* out);
uint64_t tlo_latency_ns(float ips);
int tlo_select(int64_t S, int32_t F, int32_t H, const float* ips, const uint64_t* deadline_at,
               const int32_t* n_iters, const uint64_t* tbt_slo_ns, const uint32_t* proj_flags, int32_t* freq_idx,
               uint32_t* status);
int tlo_select_binary(int64_t S, int32_t F, int32_t H, const float* ips, const uint64_t* deadline_at,
                      const int32_t* n_iters, const uint64_t* tbt_slo_ns, const uint32_t* proj_flags,
                      int32_t* freq_idx, uint32_t* status);

static uint64_t st = 0x243f6a8885a308d3ull;
static uint64_t next_u64(void) {   /* splitmix64 */
    uint64_t z = (st += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}
static double uni(void) { return (double)(next_u64() >> 11) * (1.0 / 9007199254740992.0); }
static int32_t irange(int32_t a, int32_t b) { return a + (int32_t)(uni() * (double)(b - a + 1)); }

static uint64_t h = 1469598103934665603ull;
static void mix(const void* p, size_t n) {
    const unsigned char* b = (const unsigned char*)p;
    for (size_t i = 0; i < n; ++i) h = (h ^ b[i]) * 1099511628211ull;
}

static void* xalloc(size_t n) {
    void* p = calloc(n ? n : 1, 1);
    if (!p) { fprintf(stderr, "out of memory\n"); exit(2); }
    return p;
}

static int projection_cases(void) {
    for (int trial = 0; trial < 400; ++trial) {
        const int64_t S = trial % 50 == 0 ? 0 : irange(1, 5);
        const int32_t H = trial % 13 == 0 ? 1 : irange(1, 40);
        const int32_t N = trial % 17 == 0 ? 65536 : irange(1, 8);
        int64_t* off = xalloc(sizeof(int64_t) * (size_t)(S + 1));
        for (int64_t s = 0; s < S; ++s) off[s + 1] = off[s] + (trial % 7 == 0 && s == 0 ? 0 : irange(0, 14));
        const int64_t R = off[S];
        int32_t *p = xalloc(4 * (size_t)R), *g = xalloc(4 * (size_t)R), *r = xalloc(4 * (size_t)R),
                *a = xalloc(4 * (size_t)R);
        uint64_t* dl = xalloc(8 * (size_t)R);
        uint8_t* lost = xalloc((size_t)R);
        for (int64_t i = 0; i < R; ++i) {
            p[i] = irange(0, 60);
            g[i] = irange(0, 20);
            r[i] = irange(1, H + 8);
            a[i] = uni() < 0.3 ? irange(0, H - 1) : -1;
            if (a[i] >= 0) g[i] = 0;
            dl[i] = uni() < 0.2 ? UINT64_MAX : (uint64_t)irange(1, 400000000);
            lost[i] = uni() < 0.05;
            const double u = uni();
            if (u < 0.03) r[i] = 0;                       /* malformed entries */
            else if (u < 0.05) p[i] = -3;
            else if (u < 0.06) a[i] = -7;
            else if (u < 0.07) { p[i] = 1 << 30; g[i] = 5; }
            else if (u < 0.075) { p[i] = 2000000000; g[i] = 0; }   /* prompt beyond 2^30 */
            else if (u < 0.10) { p[i] = (1 << 30) - 10; g[i] = 0; }  /* valid, but a few overflow the size guard */
        }
        int32_t *cap = xalloc(4 * (size_t)S), *bcap = xalloc(4 * (size_t)S);
        for (int64_t s = 0; s < S; ++s) {
            cap[s] = irange(0, 120);
            bcap[s] = irange(0, 10);
        }
        const int use_bcap = trial % 3 == 0;
        int32_t *B = xalloc(4 * (size_t)(S * H)), *KV = xalloc(4 * (size_t)(S * H)), *n = xalloc(4 * (size_t)S),
                *adm = xalloc(4 * (size_t)R);
        uint64_t* dla = xalloc(8 * (size_t)(S * H));
        uint32_t* fl = xalloc(4 * (size_t)S);
        if (tlo_project(S, H, N, off, p, g, r, a, trial % 5 ? dl : NULL, trial % 4 ? lost : NULL, cap,
                        use_bcap ? bcap : NULL, B, KV, dla, n, fl, trial % 2 ? adm : NULL)) return 1;
        mix(B, 4 * (size_t)(S * H)); mix(KV, 4 * (size_t)(S * H)); mix(dla, 8 * (size_t)(S * H));
        mix(n, 4 * (size_t)S); mix(fl, 4 * (size_t)S);
        if (trial % 2) mix(adm, 4 * (size_t)R);
        /* rows of the projection, 3 and 4 features */
        const int32_t F = irange(1, 5), nf = 3 + trial % 2;
        float* freqs = xalloc(4 * (size_t)F);
        float* eng = xalloc(4 * (size_t)S);
        for (int32_t f = 0; f < F; ++f) freqs[f] = 1000.0f + 250.0f * (float)f;
        for (int64_t s = 0; s < S; ++s) eng[s] = (float)(1 << irange(0, 3));
        float* rows = xalloc(4 * (size_t)(S * F * H * nf));
        if (tlo_rows(S, F, H, nf, freqs, B, KV, eng, rows)) return 1;
        mix(rows, 4 * (size_t)(S * F * H * nf));
        free(off); free(p); free(g); free(r); free(a); free(dl); free(lost); free(cap); free(bcap);
        free(B); free(KV); free(n); free(adm); free(dla); free(fl); free(freqs); free(eng); free(rows);
    }
    return 0;
}

static int forest_cases(void) {
    for (int trial = 0; trial < 60; ++trial) {
        const int32_t depth = trial % 13, T = irange(0, 6), nf = irange(1, 4);
        const int64_t n_int = ((int64_t)1 << depth) - 1, n_leaf = (int64_t)1 << depth;
        uint8_t* ft = xalloc((size_t)(T * n_int));
        float *th = xalloc(4 * (size_t)(T * n_int)), *lf = xalloc(4 * (size_t)(T * n_leaf));
        for (int64_t i = 0; i < T * n_int; ++i) {
            ft[i] = (uint8_t)irange(0, nf - 1);
            const double u = uni();
            th[i] = u < 0.05 ? NAN : u < 0.1 ? INFINITY : u < 0.15 ? -INFINITY : (float)(uni() * 100.0);
        }
        for (int64_t i = 0; i < T * n_leaf; ++i) lf[i] = (float)(uni() - 0.5);
        const int64_t n_rows = irange(0, 50);
        float *x = xalloc(4 * (size_t)(n_rows * nf)), *out = xalloc(4 * (size_t)n_rows);
        for (int64_t i = 0; i < n_rows * nf; ++i) x[i] = uni() < 0.05 ? NAN : (float)(uni() * 100.0);
        if (tlo_forest_predict(T, depth, nf, 40.0f, ft, th, lf, x, n_rows, out)) return 1;
        mix(out, 4 * (size_t)n_rows);
        free(ft); free(th); free(lf); free(x); free(out);
    }
    /* a feature index out of range is refused */
    uint8_t bad = 3;
    float thr = 1.0f, leaves[2] = {1.0f, 2.0f}, row[2] = {0, 0}, o;
    if (tlo_forest_predict(1, 1, 2, 0.0f, &bad, &thr, leaves, row, 1, &o) == 0) return 1;
    return 0;
}

static int selection_cases(void) {
    const float special[] = {0.0f, -3.0f, NAN, INFINITY, 1e-30f, 1e30f, 3.4e38f, 1e-45f};
    for (size_t i = 0; i < sizeof special / sizeof special[0]; ++i) {
        const uint64_t v = tlo_latency_ns(special[i]);
        mix(&v, 8);
    }
    for (int trial = 0; trial < 200; ++trial) {
        const int64_t S = irange(0, 6);
        const int32_t F = irange(1, 9), H = irange(1, 30);
        float* ips = xalloc(4 * (size_t)(S * F * H));
        for (int64_t i = 0; i < S * F * H; ++i) {
            const double u = uni();
            ips[i] = u < 0.08 ? special[irange(0, 7)] : (float)(5.0 + 120.0 * uni());
        }
        uint64_t* dla = xalloc(8 * (size_t)(S * H));
        for (int64_t i = 0; i < S * H; ++i) dla[i] = uni() < 0.7 ? UINT64_MAX : (uint64_t)irange(1, 2000000000);
        int32_t* n = xalloc(4 * (size_t)S);
        uint64_t* slo = xalloc(8 * (size_t)S);
        uint32_t* fl = xalloc(4 * (size_t)S);
        for (int64_t s = 0; s < S; ++s) {
            n[s] = irange(-2, H + 3);
            slo[s] = uni() < 0.05 ? UINT64_MAX : (uint64_t)irange(1, 60000000);
            fl[s] = uni() < 0.1 ? 2u : uni() < 0.05 ? 8u : 0u;
        }
        int32_t* idx = xalloc(4 * (size_t)S);
        uint32_t* stt = xalloc(4 * (size_t)S);
        if (tlo_select(S, F, H, ips, dla, n, slo, trial % 2 ? fl : NULL, idx, stt)) return 1;
        mix(idx, 4 * (size_t)S); mix(stt, 4 * (size_t)S);
        if (tlo_select_binary(S, F, H, ips, dla, n, slo, trial % 2 ? fl : NULL, idx, stt)) return 1;
        mix(idx, 4 * (size_t)S); mix(stt, 4 * (size_t)S);
        free(ips); free(dla); free(n); free(slo); free(fl); free(idx); free(stt);
    }
    return 0;
}

int main(void) {
    if (projection_cases()) { fprintf(stderr, "FAIL: projection\n"); return 1; }
    if (forest_cases()) { fprintf(stderr, "FAIL: forest\n"); return 1; }
    if (selection_cases()) { fprintf(stderr, "FAIL: selection\n"); return 1; }
    printf("oracle ok checksum=%016llx\n", (unsigned long long)h);
    return 0;
}
