// Internal interface between the host API (api.cpp) and the kernel sources.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tl.h"
#include "record_format.h"

namespace tl {

struct ProjectParams {
    int64_t n_scenarios;
    int64_t n_requests;
    int32_t H;
    int32_t N;
    uint32_t div_m, div_l;          // invariant-divisor constants for N
    const int64_t* off;
    const int32_t* prompt;
    const int32_t* gen;
    const int32_t* rem;
    const int32_t* arr;
    const uint64_t* deadline;       // nullable
    const uint8_t* lost;            // nullable
    const int32_t* kv_cap;
    const int32_t* batch_cap;       // nullable
    int32_t* batch;
    int32_t* kv;
    uint64_t* deadline_at;
    int32_t* n_iters;
    uint32_t* flags;
    int32_t F;
    int32_t nf;
    const float* freqs;
    const float* engine;
    float* rows;                    // nullable
    // a new query appended to every scenario as a request that starts now
    // (admission control); both nullable together
    const int32_t* cand_prompt;     // [S]
    const int32_t* cand_len;        // [S]
    // nullable: workspace of project_order_bytes() bytes; with it the
    // scenarios are projected heaviest first (same results, shorter tail)
    void* order_ws;
};

// The model at one frequency per scenario on the projection grid:
// out[s][j] = M(f_s, kv[s][j], batch[s][j] [, engine[s]]), f_s = freqs[fidx[s]]
// or `freq` when fidx is null; scenarios with fidx[s] < 0 are left alone.
struct ColumnParams {
    int64_t S;
    int32_t H;
    const int32_t* kv;
    const int32_t* batch;
    float freq;
    const float* freqs;             // with fidx
    const int32_t* fidx;            // nullable
    const float* engine;            // 4-feature forests
    float* out;
    // optional work order of the leaf-reuse kernel: entry i is the
    // (scenario, column) pair s * n_cols + col that item i takes, where a
    // column is 64 x RPL consecutive iterations
    const uint32_t* order;
    // optional, with order: a device count of the entries of `order` to
    // take; items from it on are skipped, and workgroups wholly past it
    // return at once
    const int32_t* n_live;
    // rows mode (rows != NULL): out[i] = M(rows[i][0 .. n_features - 1]) for
    // i < n_rows; the fields above except `out` are not used
    const float* rows;
    int64_t n_rows;
};

// Admission decision from the IPS at the maximum frequency.
struct AdmitParams {
    const float* ips;               // [S][H]
    int64_t S;
    int32_t H;
    const uint64_t* deadline_at;
    const int32_t* n_iters;
    const uint64_t* tbt_slo_ns;
    const uint32_t* proj_flags;
    const int32_t* cand_len;
    const uint64_t* cand_deadline;  // nullable
    uint32_t* decision;
};

// State and inputs of the binary search over frequencies: work holds lo[S],
// hi[S] and probe[S] (the index M is evaluated at next, -1 = none); ips
// [S][H] holds M at each scenario's probe.
struct SearchParams {
    const float* ips;
    int64_t S;
    int32_t F;
    int32_t H;
    const uint64_t* deadline_at;
    const int32_t* n_iters;
    const uint64_t* tbt_slo_ns;
    const uint32_t* proj_flags;     // nullable
    int32_t* work;                  // [3][S]
    int32_t* freq_idx;
    uint32_t* status;
};

// Scoreboard lengths from predicted lengths (Sec. 4.6).
struct AdjustParams {
    int64_t S;
    int64_t n_requests;
    const int64_t* off;
    const int32_t* gen;
    const int32_t* pred;
    const uint32_t* num;
    const uint32_t* den;
    const int32_t* max_tokens;
    int32_t* out;
};

struct SelectParams {
    const float* ips;
    int64_t S;
    int32_t F;
    int32_t H;
    const uint64_t* deadline_at;
    const int32_t* n_iters;
    const uint64_t* tbt_slo_ns;
    const uint32_t* proj_flags;     // nullable
    int32_t* freq_idx;
    uint32_t* status;
};

// Device copy of a tree ensemble.  Arrays are padded by at least 64 bytes.
struct ForestDev {
    int32_t n_trees, depth, n_features;
    float base_score;
    const uint2* nodes;     // [T][2^d]: .x = threshold bits, .y = feature (entry 2^d - 1 unused)
    const float* leaves;    // [T][2^d]
    // Per leaf, the KV (feature 1) and batch (feature 2) constraints of its
    // root-to-leaf path as half-open intervals (kv_lo, kv_hi, batch_lo,
    // batch_hi): a row with lo <= x < hi in both features, and with the
    // frequency and engine size of a row known to reach the leaf, reaches the
    // same leaf.  Empty (lo = +inf) for leaves no row can reach.  Present when
    // n_features >= 3, else NULL.
    const float4* kvb_box;  // [T][2^d]
    // Tree records of the LDS-staged grid kernel, one per tree, back to back
    // (layout: record_layout).  Present when n_features >= 3 and the depth
    // is at most kMaxRecordDepth, else NULL.
    const uint4* records;
    // Quantiles of the forest's KV (feature 1) and batch (feature 2)
    // thresholds, ascending, at most kMaxCuts each (NULL / 0 when
    // n_features < 3).  Between two rows, the number of cuts crossed by KV
    // and batch estimates how many tree decisions change: the cost model
    // for ordering the grid kernel's work.
    const float* cuts_kv;
    const float* cuts_bs;
    int32_t n_cuts_kv, n_cuts_bs;
};

struct GridParams {
    int64_t S;
    int32_t F;
    int32_t H;
    const float* freqs;     // [F]
    const int32_t* kv;      // [S][H]
    const int32_t* batch;   // [S][H]
    const float* engine;    // [S] (4 features) or NULL
    float* out;             // [S][F][H]
    // optional work order: entry i is the (scenario, chunk) pair s * n_chunks
    // + chunk that the i-th item (of each frequency group) evaluates
    const uint32_t* order;
};

// The model compiled to its input lattice (engine sizes x batch 0..batch_max
// x frequencies x KV 0..kv_max, KV in chunks of kLatticeChunk).
constexpr int32_t kLatticeChunk = 4096;
constexpr int32_t kMaxLatticeEngines = 16;
struct LatticeDev {
    int32_t nf;                     // forest features (3 or 4)
    int32_t F, nE, nB, nC;          // frequencies, engine sizes, batch_max + 1, KV chunks
    int32_t kv_max, batch_max;
    float engines[kMaxLatticeEngines];
    const float* freqs;             // [F]
    const float* table;             // [nE][nB][nC * kLatticeChunk][F]
};

struct GatherParams {
    int64_t S;
    int32_t H;
    const int32_t* kv;              // [S][H]
    const int32_t* batch;           // [S][H]
    const float* engine;            // [S] (4 features)
    float* out;                     // [S][F][H]
};

hipError_t launch_lattice_inputs(const LatticeDev& L, int64_t s0, int64_t count, int32_t* kv, int32_t* batch,
                                 float* engine, hipStream_t stream);
hipError_t launch_lattice_transpose(const float* src, float* table, int64_t s0, int64_t count, int32_t F,
                                    hipStream_t stream);
hipError_t launch_lattice_gather(const ForestDev& f, const LatticeDev& L, const GatherParams& p, hipStream_t stream);
// M at one frequency per scenario from the table: out [S][H]
hipError_t launch_lattice_column(const ForestDev& f, const LatticeDev& L, const GatherParams& p,
                                 const int32_t* fidx, int32_t f_all, hipStream_t stream);

// A launch of `blocks` workgroups fits the grid (at most 2^31 - 1 in x).
inline bool grid_fits(int64_t blocks) { return blocks >= 0 && blocks <= 0x7fffffffll; }

hipError_t launch_project(const ProjectParams& p, hipStream_t stream);
// Workspace bytes for ordering the scenarios of a projection heaviest first;
// 0 when the ordering does not pay (short FIFO loops).
size_t project_order_bytes(const ProjectParams& p);
hipError_t launch_adjust(const AdjustParams& p, hipStream_t stream);
hipError_t launch_forest_rows(const ForestDev& f, const float* rows, int64_t n_rows, float* out,
                              hipStream_t stream);
// Scratch bytes the grid kernel's work order needs for this grid (0 when no
// order applies: small grids, deep trees, forests without cuts).
hipError_t grid_order_bytes(const ForestDev& f, const GridParams& g, size_t* bytes);
// ws (nullable): device workspace of ws_bytes for the work order; the order
// is computed when ws_bytes >= grid_order_bytes, otherwise items keep their
// natural numbering (same results).  Nothing is allocated.
hipError_t launch_forest_grid(const ForestDev& f, const GridParams& g, void* ws, size_t ws_bytes,
                              hipStream_t stream);
// The fixed work-order workspace of tl_forest_predict_grid_noalloc on the
// current device (a device address; looked up once per device).
constexpr size_t kNoAllocScratchBytes = (size_t)32 << 20;
hipError_t noalloc_scratch(void** ptr);
hipError_t launch_select(const SelectParams& p, hipStream_t stream);
hipError_t launch_forest_column(const ForestDev& f, const ColumnParams& c, hipStream_t stream);
// Scratch bytes a work order for launch_forest_column needs (0 when none
// applies: the leaf-reuse kernel is not used, or no cuts); the order depends
// only on the rows (KV, batch), not on the frequencies.
hipError_t column_order_bytes(const ForestDev& f, const ColumnParams& c, size_t* bytes);
// Enqueues the order into ws (at least column_order_bytes) and points
// c.order at it; later launches with the same rows may reuse it.
hipError_t order_forest_column(const ForestDev& f, ColumnParams& c, void* ws, hipStream_t stream);
// launch_forest_column for c.fidx-selected scenarios, with the leaf-reuse
// kernel's items of skipped scenarios (fidx < 0) compacted out first (in
// c.order's order when it has one), so that the launch's work follows the
// live scenarios only; scratch column_live_bytes in ws.  Without the
// leaf-reuse kernel, fidx or ws, a plain launch_forest_column.
hipError_t column_live_bytes(const ForestDev& f, const ColumnParams& c, size_t* bytes);
hipError_t launch_forest_column_live(const ForestDev& f, const ColumnParams& c, void* ws, hipStream_t stream);
// A work order: n pairs sorted by an estimated cost, most expensive first.
// Its workspace holds four arrays of one 32-bit word per pair (cost, code,
// and their sorted copies) and the sort's temporary storage.  The caller
// fills pair_order_cost / pair_order_code (pair i's cost and its code),
// then pair_order_sort points *order at the codes sorted by cost.
// pair_order_plan gives n = 0 (no order) when the forest has no cuts to
// estimate costs with, or n < min_pairs.
struct PairOrderPlan {
    int64_t n;          // pairs; 0 = no order
    size_t arr;         // bytes per array, 256-aligned
    size_t temp;        // sort temporary storage
    size_t bytes;       // 4 * arr + temp
};
hipError_t pair_order_plan(const ForestDev& f, int64_t n, int64_t min_pairs, PairOrderPlan* p);
inline uint32_t* pair_order_cost(const PairOrderPlan&, void* ws) { return (uint32_t*)ws; }
inline uint32_t* pair_order_code(const PairOrderPlan& p, void* ws) { return (uint32_t*)((unsigned char*)ws + p.arr); }
hipError_t pair_order_sort(const PairOrderPlan& p, void* ws, const uint32_t** order, hipStream_t stream);
// The same kernel on arbitrary rows [n_rows][n_features] (3 or 4 features,
// LDS records present); hipErrorNotSupported when the forest has no records.
hipError_t launch_forest_rows_lds(const ForestDev& f, const float* rows, int64_t n_rows, float* out,
                                  hipStream_t stream);
hipError_t launch_admit(const AdmitParams& p, hipStream_t stream);
// mode 0: init, 1: one search step, 3: probe lo, 2: final check
hipError_t launch_search_step(const SearchParams& p, int mode, hipStream_t stream);

}  // namespace tl
