/*
 * tl_oracle.c -- plain, slow, single-threaded CPU oracle for the batched
 * frequency-controller hot path of throttLL'eM (arXiv 2408.05235).
 *
 * TEST INFRASTRUCTURE.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  It shares no code, header,
 * table or helper with the HIP library; both implement the same definitions,
 * written down independently.
 *
 * What it computes, per what-if scenario (a scoreboard plus its limits):
 *   1. projection   Sec. 4.2, Eq. 1 and Eq. 2, with admission check 1 and the
 *                   batch cap of Sec. 4.3.2 for queued / arriving requests;
 *   2. prediction   Sec. 4.3.1: a gradient-boosted tree ensemble evaluated on
 *                   every (frequency, KV, batch[, engine size]) feature row;
 *   3. selection    Sec. 4.3.2 checks 2 and 3 (mean TBT, Eq. 3 cumulative
 *                   time, Eq. 4 deadlines) inside the throttling controller of
 *                   Sec. 4.5: the lowest frequency that passes both checks.
 *
 * Precision: projection and selection are integer arithmetic (times are
 * integer nanoseconds); the only floating-point steps are the fp32 threshold
 * comparisons of the trees, the ensemble sum (an fp32 running sum in tree
 * order) and the per-iteration time 1e9 / IPS (one IEEE fp64 division,
 * rounded up to whole nanoseconds).
 *
 * Where the paper leaves a point open, the comment at each function states
 * the reading it follows (relative iterations, the token produced in an
 * iteration not yet cached, strict E2E deadlines, exhaustive minimum, ...).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* per-scenario flags (same numeric values as the library's ABI) */
#define O_FLAG_BAD_REQUEST 1u  /* some entries were malformed and ignored        */
#define O_FLAG_LOST        2u  /* a "lost" request is in the current batch       */
#define O_FLAG_OVERCOMMIT  4u  /* the in-flight batch alone exceeds a limit      */
#define O_FLAG_OVERFLOW    8u  /* scenario not projected (count / size bound)    */
#define O_FLAG_UNSORTED   16u  /* queue entries not in non-decreasing arrival    */

/* selection status */
#define O_STATUS_OK         0u
#define O_STATUS_INFEASIBLE 1u
#define O_STATUS_LOST       2u
#define O_STATUS_INVALID    3u

#define O_NONE UINT64_MAX               /* "no deadline" */
#define O_LAT_SATURATED (1ull << 40)    /* per-iteration time for IPS <= 0, NaN, huge */

/* ceil(x / n) for x >= 0, n >= 1, written as plain integer division */
static int64_t ceil_div(int64_t x, int64_t n) { return (x + n - 1) / n; }

/* A scoreboard entry is usable if its lengths make sense. */
static int entry_ok(int32_t p, int32_t g, int32_t r, int32_t arr) {
    if (p < 0 || g < 0 || r < 1 || arr < -1) return 0;
    if ((int64_t)p + (int64_t)g > (1ll << 30)) return 0;
    return 1;
}

/*
 * Stage 1 for one scenario.  Arrays are the scenario's own slices.
 *
 * Timeline.  An in-flight request (arrival == -1) was scheduled g_i
 * iterations ago (s_i = k - g_i in Table 1's terms) and occupies the batch at
 * relative iterations j in [0, r_i) (Sec. 4.2: it completes at s_i + r^_i).
 * Queued requests form one FIFO in array order; the head may join at
 * iteration j >= its arrival iteration if
 *   - the batch (requests active at j) is below the batch cap, and
 *   - no projected KV value from j on exceeds the capacity once the head is
 *     virtually appended with s_a = j (Sec. 4.2 "Projections for new
 *     queries", Sec. 4.3.2 check 1).
 * Several requests may join in the same iteration; a blocked head blocks the
 * queue (strict FIFO).  Only the KV check is used for admission here; SLO
 * checks at admission time belong to the scheduler, not to the projection.
 *
 * Curves.  B[j] counts requests with a_i <= j < e_i.  KV[j] sums Eq. 1 over
 * them: the request holds its c_i = |q_i| + g_i cached tokens plus the
 * (j - a_i) tokens generated since a_i, in blocks of N tokens (Eq. 2).
 */
static void project_one(int32_t H, int32_t N, int64_t R,
                        const int32_t* prompt, const int32_t* gen, const int32_t* rem,
                        const int32_t* arrival, const uint64_t* deadline, const uint8_t* lost,
                        int32_t kv_cap, int32_t batch_cap, int has_batch_cap,
                        int32_t* B, int32_t* KV, uint64_t* dl_at, int32_t* n_iters,
                        uint32_t* flags_out, int32_t* admit_out)
{
    uint32_t flags = 0;
    for (int32_t j = 0; j < H; ++j) { B[j] = 0; KV[j] = 0; dl_at[j] = O_NONE; }
    *n_iters = 0;
    if (R < 0 || R > INT32_MAX) { *flags_out = O_FLAG_OVERFLOW; return; }

    int64_t* a = (int64_t*)malloc(sizeof(int64_t) * (size_t)(R > 0 ? R : 1));
    int64_t* e = (int64_t*)malloc(sizeof(int64_t) * (size_t)(R > 0 ? R : 1));
    int64_t* kvp = (int64_t*)calloc((size_t)(H > 0 ? H : 1), sizeof(int64_t));

    /* size guard: the sum of every valid entry's largest possible block count
     * must fit a signed 32-bit curve value */
    uint64_t bound = 0;
    for (int64_t i = 0; i < R; ++i) {
        a[i] = -1; e[i] = -1;
        if (admit_out) admit_out[i] = -1;
        if (!entry_ok(prompt[i], gen[i], rem[i], arrival[i])) { flags |= O_FLAG_BAD_REQUEST; continue; }
        bound += (uint64_t)ceil_div((int64_t)prompt[i] + gen[i] + H, N);
    }
    if (bound > (uint64_t)INT32_MAX) {
        *flags_out = (flags & O_FLAG_BAD_REQUEST) | O_FLAG_OVERFLOW;
        free(a); free(e); free(kvp);
        return;
    }

    /* in-flight requests: active from iteration 0 for r_i iterations */
    for (int64_t i = 0; i < R; ++i) {
        if (!entry_ok(prompt[i], gen[i], rem[i], arrival[i]) || arrival[i] != -1) continue;
        a[i] = 0;
        e[i] = rem[i];
        if (lost && lost[i]) flags |= O_FLAG_LOST;
        int64_t c = (int64_t)prompt[i] + gen[i];
        for (int64_t t = 0; t < e[i] && t < H; ++t) kvp[t] += ceil_div(c + t, N);
    }
    /* the in-flight batch on its own: last iteration where it exceeds the KV
     * capacity (no admission can happen at or before it), batch-cap excess */
    int64_t last_over = -1;
    for (int32_t t = 0; t < H; ++t)
        if (kvp[t] > kv_cap) last_over = t;
    int64_t inflight_now = 0;
    for (int64_t i = 0; i < R; ++i)
        if (a[i] == 0) ++inflight_now;
    if (last_over >= 0) flags |= O_FLAG_OVERCOMMIT;
    if (has_batch_cap && H > 0 && inflight_now > batch_cap) flags |= O_FLAG_OVERCOMMIT;

    /* queue order check (informational) */
    int32_t prev_arr = -1;
    for (int64_t i = 0; i < R; ++i) {
        if (!entry_ok(prompt[i], gen[i], rem[i], arrival[i]) || arrival[i] < 0) continue;
        if (arrival[i] < prev_arr) flags |= O_FLAG_UNSORTED;
        prev_arr = arrival[i];
    }

    /* FIFO admission, iteration by iteration */
    int64_t head = 0;
    for (int32_t j = 0; j < H; ++j) {
        while (head < R && (!entry_ok(prompt[head], gen[head], rem[head], arrival[head]) || arrival[head] < 0))
            ++head;
        if (head >= R) break;
        int64_t active = 0;   /* batch at iteration j */
        for (int64_t i = 0; i < R; ++i)
            if (a[i] >= 0 && a[i] <= j && j < e[i]) ++active;
        for (;;) {
            while (head < R && (!entry_ok(prompt[head], gen[head], rem[head], arrival[head]) || arrival[head] < 0))
                ++head;
            if (head >= R) break;
            if (arrival[head] > j) break;                       /* not arrived yet */
            if (j <= last_over) break;                          /* KV already above capacity */
            if (has_batch_cap && active >= batch_cap) break;    /* batch full */
            int64_t c = (int64_t)prompt[head] + gen[head];
            int64_t L = rem[head];
            int ok = 1;
            for (int64_t t = j; t < j + L && t < H; ++t)
                if (kvp[t] + ceil_div(c + (t - j), N) > kv_cap) { ok = 0; break; }
            if (!ok) break;
            a[head] = j;
            e[head] = (int64_t)j + L;
            for (int64_t t = j; t < j + L && t < H; ++t) kvp[t] += ceil_div(c + (t - j), N);
            ++active;
            ++head;
        }
    }

    /* curves by direct evaluation of Eq. 1 / Eq. 2 over the admitted set */
    int64_t n = 0;
    for (int32_t j = 0; j < H; ++j) {
        int64_t b = 0, kv = 0;
        for (int64_t i = 0; i < R; ++i) {
            if (a[i] < 0 || j < a[i] || j >= e[i]) continue;
            int64_t c = (int64_t)prompt[i] + gen[i];
            b += 1;
            kv += ceil_div(c + (j - a[i]), N);
        }
        B[j] = (int32_t)b;
        KV[j] = (int32_t)kv;
    }
    /* checkpoints: a request that completes inside the horizon must do so
     * before its deadline (Eq. 4); its last iteration in the batch is e_i - 1.
     * "lost" requests are ignored by the SLO checks (Sec. 4.3.2). */
    for (int64_t i = 0; i < R; ++i) {
        if (a[i] < 0) continue;
        int64_t end = e[i] < H ? e[i] : H;
        if (end > n) n = end;
        if (e[i] > H) continue;
        if (lost && lost[i]) continue;
        uint64_t d = deadline ? deadline[i] : O_NONE;
        if (d == O_NONE) continue;
        if (d < dl_at[e[i] - 1]) dl_at[e[i] - 1] = d;
    }
    *n_iters = (int32_t)n;
    *flags_out = flags;
    if (admit_out)
        for (int64_t i = 0; i < R; ++i) admit_out[i] = (int32_t)a[i];
    free(a); free(e); free(kvp);
}

int tlo_project(int64_t S, int32_t H, int32_t N,
                const int64_t* req_offset, const int32_t* prompt, const int32_t* generated,
                const int32_t* remaining, const int32_t* arrival, const uint64_t* deadline_ns,
                const uint8_t* lost, const int32_t* kv_capacity, const int32_t* batch_cap,
                int32_t* batch, int32_t* kv, uint64_t* deadline_at, int32_t* n_iters,
                uint32_t* flags, int32_t* admit_iter)
{
    if (S < 0 || H < 1 || N < 1) return 1;
    for (int64_t s = 0; s < S; ++s) {
        int64_t lo = req_offset[s], hi = req_offset[s + 1];
        int64_t R = hi - lo;
        if (R < 0 || R > INT32_MAX) {
            for (int32_t j = 0; j < H; ++j) {
                batch[s * H + j] = 0; kv[s * H + j] = 0; deadline_at[s * H + j] = O_NONE;
            }
            n_iters[s] = 0; flags[s] = O_FLAG_OVERFLOW;
            continue;
        }
        project_one(H, N, R, prompt + lo, generated + lo, remaining + lo, arrival + lo,
                    deadline_ns ? deadline_ns + lo : NULL, lost ? lost + lo : NULL,
                    kv_capacity[s], batch_cap ? batch_cap[s] : 0, batch_cap != NULL,
                    batch + s * H, kv + s * H, deadline_at + s * H, n_iters + s, flags + s,
                    admit_iter ? admit_iter + lo : NULL);
    }
    return 0;
}

/*
 * Feature rows (Sec. 4.3.2 check 2 queries the model with the engine size,
 * the projected batch sizes, the projected KV usage and a frequency).
 * Row (s, f, j) at index (s*F + f)*H + j holds, as fp32:
 *   [0] frequency f in MHz, [1] KV[s][j] blocks, [2] B[s][j], [3] E_s.
 */
int tlo_rows(int64_t S, int32_t F, int32_t H, int32_t n_features,
             const float* freqs, const int32_t* batch, const int32_t* kv,
             const float* engine, float* rows)
{
    if (n_features != 3 && n_features != 4) return 1;
    if (n_features == 4 && !engine) return 1;
    for (int64_t s = 0; s < S; ++s)
        for (int32_t f = 0; f < F; ++f)
            for (int32_t j = 0; j < H; ++j) {
                float* row = rows + (((s * F + f) * (int64_t)H) + j) * n_features;
                row[0] = freqs[f];
                row[1] = (float)kv[s * H + j];
                row[2] = (float)batch[s * H + j];
                if (n_features == 4) row[3] = engine[s];
            }
    return 0;
}

/*
 * The performance model M (Sec. 4.3.1): a gradient-boosted decision tree
 * ensemble.  Each tree is complete of depth d, stored in heap order: internal
 * node k tests x[feature_k] < threshold_k and continues at 2k+1 if true, at
 * 2k+2 otherwise; after d tests the node index minus (2^d - 1) names the leaf.
 * The prediction is base_score plus the leaf of every tree as a running
 * fp32 sum in tree order: acc = base_score, then acc = acc + leaf_t for
 * t = 0 .. T-1, every add rounded to nearest even (no reassociation, nothing
 * fused).  The paper does not state the sum's precision; single precision
 * in tree order is how a gradient-boosted ensemble that keeps its
 * predictions in fp32 (the XGBoost model of Sec. 4.3.1) adds its trees.
 */
int tlo_forest_predict(int32_t n_trees, int32_t depth, int32_t n_features, float base_score,
                       const uint8_t* feature, const float* threshold, const float* leaf,
                       const float* rows, int64_t n_rows, float* out)
{
    if (n_trees < 0 || depth < 0 || depth > 20 || n_features < 1) return 1;
    int64_t n_int = ((int64_t)1 << depth) - 1;
    int64_t n_leaf = (int64_t)1 << depth;
    for (int64_t i = 0; i < (int64_t)n_trees * n_int; ++i)
        if (feature[i] >= n_features) return 1;
    for (int64_t r = 0; r < n_rows; ++r) {
        const float* x = rows + r * n_features;
        float acc = base_score;
        for (int32_t t = 0; t < n_trees; ++t) {
            const uint8_t* ft = feature + (int64_t)t * n_int;
            const float* th = threshold + (int64_t)t * n_int;
            int64_t k = 0;
            for (int32_t level = 0; level < depth; ++level) {
                if (x[ft[k]] < th[k]) k = 2 * k + 1;
                else k = 2 * k + 2;
            }
            acc += leaf[(int64_t)t * n_leaf + (k - n_int)];
        }
        out[r] = acc;
    }
    return 0;
}

/* T'_j = 1 / T_j (Sec. 4.3.2 check 2) in whole nanoseconds, rounded up */
uint64_t tlo_latency_ns(float ips)
{
    if (!(ips > 0.0f)) return O_LAT_SATURATED;
    double q = 1e9 / (double)ips;
    if (!(q < (double)O_LAT_SATURATED)) return O_LAT_SATURATED;
    return (uint64_t)ceil(q);
}

/* Checks 2 and 3 of Sec. 4.3.2 for one scenario at one frequency. */
static int feasible_at(const float* ips_sf, int32_t H, const uint64_t* dl_at, int32_t n_iters,
                       uint64_t tbt_slo_ns)
{
    int64_t n = n_iters < 0 ? 0 : (n_iters > H ? H : n_iters);
    if (n == 0) return 1;
    uint64_t t_r = 0;   /* Eq. 3: estimated time to reach the end of iteration j */
    for (int64_t j = 0; j < n; ++j) {
        t_r += tlo_latency_ns(ips_sf[j]);
        if (dl_at[j] != O_NONE && !(t_r < dl_at[j])) return 0;   /* Eq. 4, t_cur = 0 */
    }
    /* mean TBT over the n projected iterations must not exceed the SLO */
    uint64_t budget = (tbt_slo_ns > UINT64_MAX / (uint64_t)n) ? UINT64_MAX : tbt_slo_ns * (uint64_t)n;
    return t_r <= budget;
}

/*
 * Throttling controller (Sec. 4.5).  The lowest frequency index whose
 * predicted times pass the TBT and E2E checks.  The search is exhaustive, so
 * it does not depend on feasibility being monotone in the frequency.  A lost
 * request in the batch bypasses the search and picks the highest frequency.
 * ips is laid out [S][F][H].
 */
int tlo_select(int64_t S, int32_t F, int32_t H, const float* ips, const uint64_t* deadline_at,
               const int32_t* n_iters, const uint64_t* tbt_slo_ns, const uint32_t* proj_flags,
               int32_t* freq_idx, uint32_t* status)
{
    if (S < 0 || F < 1 || H < 1) return 1;
    for (int64_t s = 0; s < S; ++s) {
        uint32_t fl = proj_flags ? proj_flags[s] : 0;
        if (fl & O_FLAG_OVERFLOW) { freq_idx[s] = F - 1; status[s] = O_STATUS_INVALID; continue; }
        if (fl & O_FLAG_LOST) { freq_idx[s] = F - 1; status[s] = O_STATUS_LOST; continue; }
        freq_idx[s] = F - 1;
        status[s] = O_STATUS_INFEASIBLE;
        for (int32_t f = 0; f < F; ++f) {
            if (feasible_at(ips + ((s * F + f) * (int64_t)H), H, deadline_at + s * H, n_iters[s],
                            tbt_slo_ns[s])) {
                freq_idx[s] = f;
                status[s] = O_STATUS_OK;
                break;
            }
        }
    }
    return 0;
}

/*
 * The paper's own search (Sec. 4.5): binary search over the frequency range
 * for the lowest frequency that passes the checks.  It agrees with the
 * exhaustive search whenever feasibility is monotone in the frequency.
 */
int tlo_select_binary(int64_t S, int32_t F, int32_t H, const float* ips, const uint64_t* deadline_at,
                      const int32_t* n_iters, const uint64_t* tbt_slo_ns, const uint32_t* proj_flags,
                      int32_t* freq_idx, uint32_t* status)
{
    if (S < 0 || F < 1 || H < 1) return 1;
    for (int64_t s = 0; s < S; ++s) {
        uint32_t fl = proj_flags ? proj_flags[s] : 0;
        if (fl & O_FLAG_OVERFLOW) { freq_idx[s] = F - 1; status[s] = O_STATUS_INVALID; continue; }
        if (fl & O_FLAG_LOST) { freq_idx[s] = F - 1; status[s] = O_STATUS_LOST; continue; }
        int32_t lo = 0, hi = F - 1;
        while (lo < hi) {
            int32_t mid = lo + (hi - lo) / 2;
            if (feasible_at(ips + ((s * F + mid) * (int64_t)H), H, deadline_at + s * H, n_iters[s], tbt_slo_ns[s]))
                hi = mid;
            else
                lo = mid + 1;
        }
        int ok = feasible_at(ips + ((s * F + lo) * (int64_t)H), H, deadline_at + s * H, n_iters[s], tbt_slo_ns[s]);
        freq_idx[s] = ok ? lo : F - 1;
        status[s] = ok ? O_STATUS_OK : O_STATUS_INFEASIBLE;
    }
    return 0;
}
