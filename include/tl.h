/*
 * tl.h -- C ABI of the MI355X (gfx950) library for the batched hot path of
 * throttLL'eM's per-iteration GPU-frequency controller (arXiv 2408.05235).
 *
 * For many independent what-if scenarios the library runs three stages, each
 * a HIP kernel on one device:
 *   tl_project        projected batch size and KV-cache blocks per future
 *                     iteration (Sec. 4.2, Eq. 1-2), with FIFO admission of
 *                     queued requests under the KV check of Sec. 4.3.2;
 *                     optionally the feature rows of the performance model;
 *   tl_forest_predict the performance model M, a gradient-boosted tree
 *                     ensemble predicting iterations per second (Sec. 4.3.1);
 *   tl_select_freq    the throttling controller (Sec. 4.5): per scenario the
 *                     lowest frequency whose predicted per-iteration times
 *                     pass the TBT check and the E2E deadlines (Sec. 4.3.2,
 *                     checks 2 and 3, Eq. 3-4).
 * and, from the same stages, tl_select_freq_binary (the controller's binary
 * search as the paper states it, querying the model only at probed
 * frequencies) and tl_admit (the admission control of Sec. 4.3.2 for one new
 * query per scenario).
 *
 * Conventions shared by every entry point
 *   - Pointers are DEVICE pointers (memory of the device that is current on
 *     the calling thread) owned by the caller, unless the comment says host.
 *     The library never frees or retains caller memory.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  Calls
 *     only enqueue work; none synchronizes.  Outputs are valid once the
 *     stream reaches that point.
 *   - Argument errors (sizes, NULL pointers, unsupported shapes) are detected
 *     on the host before anything is enqueued and return TL_EINVAL; nothing
 *     is written.  A failed HIP call returns TL_EDEVICE.  tl_last_error()
 *     then describes the failure (thread-local, valid until the next call).
 *   - Data-dependent anomalies never fail a call: they are reported per
 *     scenario through TL_FLAG_* bits and TL_STATUS_* values.
 *   - Results are deterministic: bit-identical across runs and launches.
 */
#ifndef TL_H
#define TL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TL_ABI_VERSION 1

typedef enum tl_status {
    TL_OK = 0,
    TL_EINVAL = 1,          /* invalid argument; nothing was enqueued          */
    TL_ENOMEM = 2,          /* device allocation failed                        */
    TL_EDEVICE = 3,         /* a HIP runtime call or kernel launch failed      */
    TL_EUNSUPPORTED = 4     /* valid but beyond the library's limits          */
} tl_status;

/* Limits of the library. */
#define TL_MAX_HORIZON 8192         /* H: future iterations per scenario      */
#define TL_MAX_BLOCK_TOKENS 65536   /* N: tokens per KV block                 */
#define TL_MAX_FREQS 4096           /* F: candidate frequencies               */
#define TL_MAX_FEATURES 4           /* model inputs (Sec. 4.3.1 lists four)   */
#define TL_MAX_DEPTH 14             /* tree depth                             */

/* Per-scenario flags written by tl_project (bitwise OR). */
#define TL_FLAG_BAD_REQUEST 1u  /* some scoreboard entries were malformed and ignored:
                                   prompt < 0, generated < 0, remaining < 1,
                                   arrival < -1, or prompt + generated > 2^30 */
#define TL_FLAG_LOST        2u  /* an in-flight request is marked lost (Sec. 4.3.2)   */
#define TL_FLAG_OVERCOMMIT  4u  /* the in-flight batch alone exceeds the KV capacity
                                   at some iteration, or exceeds the batch cap now    */
#define TL_FLAG_OVERFLOW    8u  /* scenario not projected: its request range is
                                   invalid, or sum over valid entries of
                                   ceil((prompt+generated+H)/N) > 2^31-1, so curves
                                   could overflow; outputs are zero / no deadline  */
#define TL_FLAG_UNSORTED   16u  /* queued entries are not in non-decreasing arrival
                                   order; the queue is still served in array order */
#define TL_FLAG_BAD_CANDIDATE 32u /* tl_admit only: the new query is malformed
                                   (prompt < 0 or > 2^30, length < 1) and was left
                                   out of the projection */

/* Per-scenario status written by tl_select_freq. */
#define TL_STATUS_OK         0u  /* freq_idx is the lowest feasible index           */
#define TL_STATUS_INFEASIBLE 1u  /* no frequency passes; freq_idx = F-1            */
#define TL_STATUS_LOST       2u  /* a lost request forces the maximum; freq_idx = F-1 */
#define TL_STATUS_INVALID    3u  /* scenario flagged TL_FLAG_OVERFLOW; freq_idx = F-1 */

/* Per-scenario decision written by tl_admit (Sec. 4.3.2). */
#define TL_ADMIT_OK             0u  /* checks 1-3 pass: schedule the query            */
#define TL_ADMIT_LOST           1u  /* only its own deadline fails: schedule it and
                                       mark it lost                                   */
#define TL_ADMIT_QUEUE_CAPACITY 2u  /* check 1: a projected KV value exceeds the
                                       capacity, or the batch running now exceeds
                                       the batch cap -> queue                         */
#define TL_ADMIT_QUEUE_TBT      3u  /* check 2: mean TBT at the maximum frequency
                                       exceeds the SLO -> queue                       */
#define TL_ADMIT_QUEUE_E2E      4u  /* check 3: a scheduled request would miss its
                                       deadline (Eq. 4) -> queue                      */
#define TL_ADMIT_INVALID        5u  /* malformed query or scenario not projected     */

/* Per-iteration time that stands for "no progress" (IPS <= 0, NaN, or
 * 1e9/IPS >= 2^40 ns). */
#define TL_LAT_SATURATED_NS (1ull << 40)
#define TL_NO_DEADLINE UINT64_MAX

int32_t tl_abi_version(void);        /* returns TL_ABI_VERSION */
const char* tl_last_error(void);     /* message for the last non-OK status on this thread */

/* ------------------------------------------------------------------------
 * The performance model M (Sec. 4.3.1): a gradient-boosted decision-tree
 * ensemble over the inputs the paper names (engine size, batch size, KV-cache
 * usage, GPU frequency) that predicts iterations per second.
 *
 * Trees are complete, of depth `depth`, in heap order: internal node k
 * (0 <= k < 2^depth - 1) compares x[feature[k]] < threshold[k] in fp32 and
 * continues at 2k+1 when true, 2k+2 otherwise (a NaN input goes to 2k+2);
 * after `depth` comparisons the node index minus (2^depth - 1) selects one of
 * the 2^depth leaves.  A shallower tree is expressed by padding with
 * threshold +inf (always 2k+1).  The prediction of a row is base_score plus
 * the selected leaf of every tree as an fp32 running sum in tree order
 * (acc = base_score, then acc += leaf_t for t = 0 .. n_trees-1, each add
 * rounded to nearest even): the paper does not state the sum's precision,
 * and this is how an ensemble that keeps its predictions in fp32 adds them.
 *
 * feature   host, uint8 [n_trees][2^depth - 1], each < n_features
 * threshold host, fp32  [n_trees][2^depth - 1]
 * leaf      host, fp32  [n_trees][2^depth]
 * The arrays are copied to the current device; the handle owns that copy and
 * must be used with the same device.  n_trees >= 0 (0 gives base_score),
 * 0 <= depth <= TL_MAX_DEPTH, 1 <= n_features <= TL_MAX_FEATURES.
 * Errors: TL_EINVAL (bad sizes, NULL, feature index out of range),
 * TL_ENOMEM, TL_EDEVICE.  On error *out is set to NULL.
 * ---------------------------------------------------------------------- */
typedef struct tl_forest tl_forest;

tl_status tl_forest_create(int32_t n_trees, int32_t depth, int32_t n_features, float base_score,
                           const uint8_t* feature, const float* threshold, const float* leaf,
                           tl_forest** out);
void tl_forest_destroy(tl_forest* forest);   /* NULL is ignored; synchronizes the device */

/* ------------------------------------------------------------------------
 * Scoreboard lengths under generation-length errors (Sec. 4.6): the
 * remaining-token counts tl_project takes, from the predictor's total
 * generation lengths.  Per request i of scenario s (CSR req_offset as in
 * tl_project):
 *   len = ceil(pred_len[i] * scale_num[s] / scale_den[s])   (scale_den 0: pred_len)
 *   len = min(len, max_tokens[s]);  if generated[i] >= len: len = max_tokens[s]
 *                                                   (both only when max_tokens[s] >= 1)
 *   remaining_out[i] = max(len - generated[i], 1)
 * Entries with generated < 0 or pred_len < 1 get 0, which tl_project ignores
 * as malformed.  Scenarios whose request range is invalid are not written.
 * remaining_out may alias neither input.
 * ---------------------------------------------------------------------- */
tl_status tl_adjust_lengths(int64_t n_scenarios, int64_t n_requests, const int64_t* req_offset,
                            const int32_t* generated, const int32_t* pred_len, const uint32_t* scale_num,
                            const uint32_t* scale_den, const int32_t* max_tokens, int32_t* remaining_out,
                            void* stream);

/* ------------------------------------------------------------------------
 * Stage 1 -- KV usage and batch-size projection (Sec. 4.2, Eq. 1-2).
 *
 * Scenario s owns requests req_offset[s] .. req_offset[s+1]-1 (a scoreboard,
 * Table 1).  Iterations are relative: j = 0 is the current iteration k.
 * Request i has prompt length |q_i| = prompt_len[i], has generated
 * generated[i] tokens and is projected to need remaining[i] more iterations.
 *   arrival_iter[i] == -1 : in the batch now (scheduled g_i iterations ago);
 *                           it occupies iterations [0, remaining[i]).
 *   arrival_iter[i] >= 0  : queued; it becomes eligible at that iteration.
 * Queued entries form one FIFO in array order.  At iteration j, after the
 * requests ending at j leave, the head joins (s_a = j, its lifetime is
 * [j, j + remaining)) iff it has arrived, the batch at j is below
 * batch_cap[s], and appending it keeps every projected KV value from j to
 * H-1 at or below kv_capacity[s] (Sec. 4.3.2 check 1); several may join at the
 * same j; a head that cannot join blocks the queue.
 *
 * Outputs ([s][j] row-major, j < H):
 *   batch[s][j]       number of requests in the batch at iteration j
 *   kv[s][j]          KV blocks in use: sum of ceil((prompt + generated +
 *                     (j - start)) / N) over those requests (Eq. 1-2)
 *   deadline_at[s][j] minimum deadline_ns over non-lost requests whose last
 *                     iteration in the batch is j (finishing inside the
 *                     horizon), TL_NO_DEADLINE if none (Eq. 4 checkpoints)
 *   n_iters[s]        number of projected iterations: min(H, last finish)
 *   flags[s]          TL_FLAG_* bits
 * Optional feature rows (rows != NULL), [s][f][j][n_features] fp32:
 *   (freqs_mhz[f], kv[s][j], batch[s][j] [, engine_size[s]])
 * the query vector of Sec. 4.3.2 check 2 for every candidate frequency.
 * freqs_mhz must be ascending; index F-1 is the maximum frequency.
 *
 * Scoreboards with long FIFO loops (no batch_cap and on average 1024 or more
 * requests per scenario) are projected heaviest first (results do not depend
 * on the order).  The order takes 4 bytes per scenario of device scratch
 * that the library owns, one per device: allocated on the first such call,
 * kept, and replaced only when more scenarios come.  If that allocation
 * fails the scenarios run in their own order (same results), as they do
 * while the stream is being captured into a graph.  Calls share it: a call
 * on another stream than the previous one first waits (on the device) for
 * the previous projection.
 * ---------------------------------------------------------------------- */
typedef struct tl_project_args {
    uint32_t struct_size;          /* sizeof(tl_project_args) */
    int32_t horizon;               /* H, 1 .. TL_MAX_HORIZON */
    int64_t n_scenarios;           /* S >= 0 */
    int64_t n_requests;            /* total entries; req_offset[S] must equal it */
    int32_t block_tokens;          /* N, 1 .. TL_MAX_BLOCK_TOKENS */
    int32_t n_freqs;               /* F (rows only), 1 .. TL_MAX_FREQS */
    int32_t n_features;            /* 3 or 4 (rows only) */
    int32_t reserved;
    const int64_t* req_offset;     /* [S+1] */
    const int32_t* prompt_len;     /* [n_requests] */
    const int32_t* generated;      /* [n_requests] */
    const int32_t* remaining;      /* [n_requests] */
    const int32_t* arrival_iter;   /* [n_requests] */
    const uint64_t* deadline_ns;   /* [n_requests], t_dead - t_cur in ns; NULL = none */
    const uint8_t* lost;           /* [n_requests], nonzero = lost; NULL = none */
    const int32_t* kv_capacity;    /* [S] blocks */
    const int32_t* batch_cap;      /* [S]; NULL = unlimited */
    int32_t* batch;                /* out [S][H] */
    int32_t* kv;                   /* out [S][H] */
    uint64_t* deadline_at;         /* out [S][H] */
    int32_t* n_iters;              /* out [S] */
    uint32_t* flags;               /* out [S] */
    const float* freqs_mhz;        /* [F] (rows only) */
    const float* engine_size;      /* [S] (rows with n_features == 4) */
    float* rows;                   /* out [S][F][H][n_features]; NULL = no rows */
} tl_project_args;

tl_status tl_project(const tl_project_args* args, void* stream);

/* ------------------------------------------------------------------------
 * Stage 2 -- the model M on arbitrary feature rows (Sec. 4.3.1).
 * rows [n_rows][n_features of the forest] fp32 row-major; out [n_rows] fp32.
 * ---------------------------------------------------------------------- */
tl_status tl_forest_predict(const tl_forest* forest, const float* rows, int64_t n_rows,
                            float* out, void* stream);

/* ------------------------------------------------------------------------
 * Stage 2 on the projection grid, fused with the row expansion: the same
 * values tl_forest_predict gives for the rows tl_project would write, without
 * materializing them (Sec. 4.3.2 check 2 and Sec. 4.5 query M for every
 * projected iteration at every candidate frequency).
 *   out[s][f][j] = M(freqs_mhz[f], kv[s][j], batch[s][j] [, engine_size[s]])
 * freqs_mhz [F]; kv, batch [S][H] int32 as written by tl_project (converted
 * to fp32); engine_size [S], required when the forest has 4 features and
 * ignored otherwise; out [S][F][H] fp32.  The forest must have 3 or 4
 * features in the order (frequency, KV, batch[, engine size]).
 * 1 <= F <= TL_MAX_FREQS, 1 <= H <= TL_MAX_HORIZON.
 * Work is ordered by an estimate of its cost (results do not depend on the
 * order).  The ordering needs 16 bytes per (scenario, 64-iteration chunk)
 * plus a radix sort's temporary storage of device scratch, which the forest
 * handle owns: it is allocated
 * on the first call, kept, and replaced only when a larger grid comes, so
 * repeated calls of one size allocate nothing.  If that allocation fails, or
 * the stream is being captured into a graph, the call runs without the
 * ordering (same results; tl_forest_predict_grid_noalloc keeps it under
 * capture).  Calls with one forest
 * share its scratch: a call on another stream than the previous one first
 * waits (on the device) for the previous call's work.  The forest's device
 * must be the current device.
 * ---------------------------------------------------------------------- */
tl_status tl_forest_predict_grid(const tl_forest* forest, int64_t n_scenarios, int32_t n_freqs,
                                 int32_t horizon, const float* freqs_mhz, const int32_t* kv,
                                 const int32_t* batch, const float* engine_size, float* out,
                                 void* stream);

/* ------------------------------------------------------------------------
 * tl_forest_predict_grid for callers that cannot allocate device memory
 * (code under stream capture, tight serving loops, hosts that forbid
 * allocation): same arguments, same results, no allocation of any kind.
 * The work order's scratch is a fixed 32 MiB array of the library on each
 * device (taken when the library is loaded): 16 bytes per (scenario,
 * 64-iteration chunk) pair plus the sort's temporary storage must fit, as
 * they do for 16384 scenarios x 2048 iterations (524,288 pairs) but not for
 * 65536 x 2048.  A grid whose order needs more returns TL_EUNSUPPORTED and
 * enqueues nothing.  Every call on one device shares that array: calls that
 * overlap on one device (concurrent streams, other threads) race and must
 * be serialized by the caller; tl_forest_predict_grid does not use it.
 * ---------------------------------------------------------------------- */
tl_status tl_forest_predict_grid_noalloc(const tl_forest* forest, int64_t n_scenarios, int32_t n_freqs,
                                         int32_t horizon, const float* freqs_mhz, const int32_t* kv,
                                         const int32_t* batch, const float* engine_size, float* out,
                                         void* stream);

/* ------------------------------------------------------------------------
 * Stage 2 through a table: the model compiled to its discrete input lattice.
 * The controller queries M only at a fixed list of frequencies, a few engine
 * sizes, integer batch sizes and integer KV blocks (Sec. 4.3.1 notes that
 * all inputs are bounded), so M can be evaluated once at every lattice point
 * and prediction becomes a table lookup:
 *   tl_lattice_create evaluates M (with tl_forest_predict_grid's kernels, so
 *   every value is the fp32 tree-order sum a walk gives) at every
 *   (engine size, batch 0..batch_max, frequency, KV 0..kv_max); the table
 *   takes n_engines x (batch_max + 1) x n_freqs x 4096 x ceil((kv_max + 1) /
 *   4096) x 4 bytes (tl_lattice_bytes), at most 256 GiB.
 *   tl_lattice_predict_grid gives out[s][f][j] exactly as
 *   tl_forest_predict_grid with the lattice's frequencies: lattice points are
 *   read from the table, other rows (KV or batch outside [0, max], an engine
 *   size not in the list) are walked.
 * freqs_mhz: device [n_freqs], copied.  engine_values: host
 * [n_engines <= 16], required for 4-feature forests (ignored otherwise).
 * The build is enqueued on `stream`, which the call synchronizes once (to
 * keep a host copy of the frequency list); the forest must outlive the
 * lattice.
 * Errors: TL_EINVAL, TL_EUNSUPPORTED (table too large), TL_ENOMEM,
 * TL_EDEVICE.
 * ---------------------------------------------------------------------- */
typedef struct tl_lattice tl_lattice;

tl_status tl_lattice_create(const tl_forest* forest, int32_t n_freqs, const float* freqs_mhz, int32_t n_engines,
                            const float* engine_values, int32_t kv_max, int32_t batch_max, void* stream,
                            tl_lattice** out);
void tl_lattice_destroy(tl_lattice* lattice);   /* NULL is ignored; synchronizes the device */
uint64_t tl_lattice_bytes(const tl_lattice* lattice);
tl_status tl_lattice_predict_grid(const tl_lattice* lattice, int64_t n_scenarios, int32_t horizon,
                                  const int32_t* kv, const int32_t* batch, const float* engine_size, float* out,
                                  void* stream);

/* ------------------------------------------------------------------------
 * Stage 3 -- frequency selection (Sec. 4.5 with Sec. 4.3.2 checks 2-3).
 *
 * ips [S][F][H] fp32: predicted iterations/s of scenario s at frequency f in
 * iteration j.  With n = clamp(n_iters[s], 0, H) and per-iteration times
 * lat = ceil(1e9 / ips) ns (one IEEE fp64 division; TL_LAT_SATURATED_NS for
 * ips <= 0, NaN or 1e9/ips >= 2^40), and T_R[l] = lat[0] + ... + lat[l-1]
 * (Eq. 3), frequency f is feasible iff n == 0, or
 *   T_R[n] <= tbt_slo_ns[s] * n            (mean TBT, check 2), and
 *   T_R[j+1] < deadline_at[s][j] for every j < n with a deadline (Eq. 4).
 * freq_idx[s] = lowest feasible f (status OK), else F-1 (INFEASIBLE).  If
 * proj_flags[s] has TL_FLAG_OVERFLOW: F-1, INVALID; else if it has
 * TL_FLAG_LOST: F-1, LOST (the search is bypassed).  proj_flags may be NULL.
 * ---------------------------------------------------------------------- */
tl_status tl_select_freq(const float* ips, int64_t n_scenarios, int32_t n_freqs, int32_t horizon,
                         const uint64_t* deadline_at, const int32_t* n_iters,
                         const uint64_t* tbt_slo_ns, const uint32_t* proj_flags,
                         int32_t* freq_idx, uint32_t* status, void* stream);

/* ------------------------------------------------------------------------
 * The paper's throttling controller as it states it (Sec. 4.5): a binary
 * search over the candidate frequencies that queries the model only at the
 * frequency each scenario probes.  Per scenario, with lo = 0, hi = F-1:
 * while lo < hi, mid = lo + (hi - lo) / 2, M on every projected iteration at
 * freqs_mhz[mid], feasible as in tl_select_freq -> hi = mid, else lo =
 * mid + 1; finally lo is checked: feasible -> freq_idx = lo (OK), else F-1
 * (INFEASIBLE).  Flags as in tl_select_freq (OVERFLOW -> INVALID, LOST ->
 * F-1 without a search).  It equals tl_select_freq whenever feasibility is
 * monotone in the frequency, and evaluates M on at most ceil(log2 F) + 1
 * rows per (scenario, iteration) instead of F: the check of lo evaluates
 * nothing new when hi has moved below F-1, since hi only moves to a probe
 * found feasible and then lo == hi.
 * kv, batch, deadline_at, n_iters, proj_flags: as written by tl_project;
 * freqs_mhz [F] ascending; engine_size [S] for 4-feature forests.
 * Work arrays of the caller: ips_work [S][H] fp32 (left holding, per
 * scenario, M at the last frequency it evaluated; rows of scenarios flagged
 * lost or overflow are not written) and search_work [3][S] int32.
 * On grids that give every CU at least two workgroups of the model's kernel
 * (16 wavefronts of 64 lanes x 16, else 8, consecutive iterations of one
 * scenario), the wavefronts' work is ordered by an estimate of its cost,
 * computed once per call, and the check of lo runs only the wavefronts of
 * scenarios that need an evaluation, compacted (results depend on neither).
 * Scratch: 20 bytes per wavefront plus a radix sort's temporary storage, in
 * the forest's device scratch, as for tl_forest_predict_grid (the larger of
 * the two needs is kept; neither ordering nor compaction under stream
 * capture or without the scratch).  Nothing else is allocated.
 * lattice (nullable): a table of the same forest and frequency count
 * (tl_lattice_create; TL_EINVAL otherwise); M at the probes is then read
 * from it, at the lattice's own frequencies (the same values when it was
 * built for freqs_mhz, which is the caller's to ensure: the list itself is
 * not compared).
 * ---------------------------------------------------------------------- */
tl_status tl_select_freq_binary(const tl_forest* forest, int64_t n_scenarios, int32_t n_freqs, int32_t horizon,
                                const float* freqs_mhz, const int32_t* kv, const int32_t* batch,
                                const float* engine_size, const uint64_t* deadline_at, const int32_t* n_iters,
                                const uint64_t* tbt_slo_ns, const uint32_t* proj_flags, float* ips_work,
                                int32_t* search_work, int32_t* freq_idx, uint32_t* status,
                                const tl_lattice* lattice, void* stream);

/* ------------------------------------------------------------------------
 * Admission control (Sec. 4.3.2) for one new query per scenario, as a batch
 * of what-ifs: the projection of tl_project on the scenario's scoreboard with
 * the query appended as a request that starts now (prompt cand_prompt[s],
 * nothing generated, active for the cand_len[s] iterations [0, L); queued and
 * arriving entries keep their FIFO admission behind it), the model at
 * max_freq_mhz on every projected iteration, and the paper's three checks in
 * order (the first failure decides):
 *   1. some projected KV value exceeds kv_capacity, or the batch running now
 *      exceeds batch_cap                         -> TL_ADMIT_QUEUE_CAPACITY
 *   2. with n = n_iters[s] and T_R as in tl_select_freq (Eq. 3),
 *      T_R[n] > tbt_slo_ns[s] * n (mean TBT)     -> TL_ADMIT_QUEUE_TBT
 *   3. T_R[e] < deadline fails for a scheduled, non-lost request ending at
 *      e <= H (Eq. 4)                            -> TL_ADMIT_QUEUE_E2E
 *      else, when L <= H and cand_deadline_ns[s] is set, T_R[L] <
 *      cand_deadline_ns[s] fails                 -> TL_ADMIT_LOST
 *   otherwise                                    -> TL_ADMIT_OK
 * A malformed query (flag TL_FLAG_BAD_CANDIDATE) or a scenario flagged
 * TL_FLAG_OVERFLOW gives TL_ADMIT_INVALID.
 *
 * `proj` describes the scoreboards and receives the projection with the query
 * (batch, kv, deadline_at without the query's deadline, n_iters, flags);
 * its rows, n_freqs, freqs_mhz and n_features are ignored.  engine_size [S]
 * is read for 4-feature forests.  ips [S][H] receives M at max_freq_mhz (rows
 * of scenarios flagged TL_FLAG_OVERFLOW hold M on the zero curves).  All
 * arrays are device arrays of the caller; the only scratch is the
 * projection's scenario order, as for tl_project, and the model kernel's
 * work order, as for tl_select_freq_binary.
 * Errors as for tl_project, plus a NULL forest, ips, decision, tbt_slo_ns,
 * cand_prompt or cand_len, or a forest without 3 or 4 features: TL_EINVAL.
 * ---------------------------------------------------------------------- */
typedef struct tl_admit_args {
    uint32_t struct_size;              /* sizeof(tl_admit_args) */
    uint32_t reserved;
    tl_project_args proj;              /* scoreboards; projection outputs */
    const tl_forest* forest;
    float max_freq_mhz;                /* the maximum available frequency */
    const float* engine_size;          /* [S], 4-feature forests */
    const uint64_t* tbt_slo_ns;        /* [S] */
    const int32_t* cand_prompt;        /* [S] prompt tokens of the new query */
    const int32_t* cand_len;           /* [S] its predicted length, >= 1 */
    const uint64_t* cand_deadline_ns;  /* [S] t_dead - t_cur; NULL or TL_NO_DEADLINE = none */
    float* ips;                        /* out [S][H] */
    uint32_t* decision;                /* out [S], TL_ADMIT_* */
    const tl_lattice* lattice;         /* nullable: a table of the same forest; used
                                          when max_freq_mhz is one of its frequencies */
} tl_admit_args;

tl_status tl_admit(const tl_admit_args* args, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TL_H */
