// Host side of the C ABI: argument validation (before anything is enqueued),
// forest upload, kernel dispatch and error reporting.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "device_util.h"
#include "host_forest.h"
#include "tl.h"
#include "tl_internal.h"

struct tl_forest {
    int device;
    tl::ForestDev dev;
    void* nodes_mem;
    void* leaves_mem;
    void* box_mem;
    void* records_mem;
    void* cuts_mem;   // [kMaxCuts] KV cuts, then [kMaxCuts] batch cuts
    // Work-order scratch of the grid and column kernels, on the forest's
    // device: kept from call to call and only replaced by a larger one when a
    // larger grid comes.  ws_done is recorded on the stream of the last call that used
    // it; a call on another stream waits for it first.
    mutable std::mutex ws_mutex;
    mutable void* ws = nullptr;
    mutable size_t ws_bytes = 0;
    mutable hipEvent_t ws_done = nullptr;
    mutable hipStream_t ws_stream = nullptr;
    mutable bool ws_used = false;
};

struct tl_lattice {
    int device;
    const tl_forest* forest;
    tl::LatticeDev dev;
    void* mem;        // [F] frequencies (padded to 256 bytes), then the table
    uint64_t bytes;
    std::vector<float> host_freqs;
};

namespace {

thread_local char g_err[512] = "";

tl_status fail(tl_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

tl_status ok() {
    g_err[0] = '\0';
    return TL_OK;
}

tl_status from_hip(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(e == hipErrorOutOfMemory ? TL_ENOMEM : TL_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

extern "C" {

int32_t tl_abi_version(void) { return TL_ABI_VERSION; }

const char* tl_last_error(void) { return g_err; }

tl_status tl_forest_create(int32_t n_trees, int32_t depth, int32_t n_features, float base_score,
                           const uint8_t* feature, const float* threshold, const float* leaf,
                           tl_forest** out) {
    if (!out) return fail(TL_EINVAL, "tl_forest_create: out is NULL");
    *out = nullptr;
    if (n_trees < 0) return fail(TL_EINVAL, "tl_forest_create: n_trees %d < 0", n_trees);
    if (depth < 0 || depth > TL_MAX_DEPTH)
        return fail(TL_EINVAL, "tl_forest_create: depth %d outside [0, %d]", depth, TL_MAX_DEPTH);
    if (n_features < 1 || n_features > TL_MAX_FEATURES)
        return fail(TL_EINVAL, "tl_forest_create: n_features %d outside [1, %d]", n_features, TL_MAX_FEATURES);
    const int64_t n_int = (1ll << depth) - 1;
    const int64_t n_leaf = 1ll << depth;
    if (n_trees > 0 && (!leaf || (n_int > 0 && (!feature || !threshold))))
        return fail(TL_EINVAL, "tl_forest_create: NULL tree array");
    // device arrays use a per-tree stride of 2^d entries and 64 bytes of tail
    // padding, so staged blocks are whole, aligned 16-byte words
    const size_t cells = (size_t)n_trees * n_leaf;
    std::vector<uint2> nodes(cells + 8, make_uint2(0, 0));
    std::vector<float> leaves(cells + 16, 0.0f);
    for (int64_t t = 0; t < n_trees; ++t)
        for (int64_t k = 0; k < n_int; ++k) {
            const int64_t i = t * n_int + k;
            if (feature[i] >= n_features)
                return fail(TL_EINVAL, "tl_forest_create: node %lld uses feature %d >= n_features %d",
                            (long long)i, (int)feature[i], n_features);
            uint32_t bits;
            std::memcpy(&bits, &threshold[i], 4);
            nodes[(size_t)(t * n_leaf + k)] = make_uint2(bits, feature[i]);
        }
    for (size_t i = 0; i < cells; ++i) leaves[i] = leaf[i];
    std::vector<tl::host::Box> leaf_box;
    std::vector<float4> boxes;
    std::vector<unsigned char> records;
    if (n_features >= 3) {
        tl::host::leaf_boxes(n_trees, depth, feature, threshold, leaf_box);
        if (depth <= tl::kMaxRecordDepth) tl::host::build_records(n_trees, depth, feature, threshold, leaf, leaf_box, records);
        boxes.assign(cells + 4, make_float4(0, 0, 0, 0));
        for (size_t i = 0; i < leaf_box.size(); ++i)
            boxes[i] = make_float4(leaf_box[i].kv_lo, leaf_box[i].kv_hi, leaf_box[i].batch_lo, leaf_box[i].batch_hi);
    }
    std::vector<float> cuts_kv, cuts_bs;
    if (n_features >= 3 && n_int > 0) {
        cuts_kv = tl::host::threshold_cuts(n_trees * n_int, feature, threshold, 1);
        cuts_bs = tl::host::threshold_cuts(n_trees * n_int, feature, threshold, 2);
    }

    tl_forest* f = new (std::nothrow) tl_forest();
    if (!f) return fail(TL_ENOMEM, "tl_forest_create: host allocation failed");
    hipError_t e = hipGetDevice(&f->device);
    if (e != hipSuccess) { delete f; return from_hip(e, "tl_forest_create: hipGetDevice"); }
    e = hipEventCreateWithFlags(&f->ws_done, hipEventDisableTiming);
    if (e != hipSuccess) { delete f; return from_hip(e, "tl_forest_create: hipEventCreate"); }
    e = hipMalloc(&f->nodes_mem, nodes.size() * sizeof(uint2));
    if (e != hipSuccess) { (void)hipEventDestroy(f->ws_done); delete f; return from_hip(e, "tl_forest_create: hipMalloc(nodes)"); }
    e = hipMalloc(&f->leaves_mem, leaves.size() * sizeof(float));
    if (e != hipSuccess) { (void)hipFree(f->nodes_mem); (void)hipEventDestroy(f->ws_done); delete f; return from_hip(e, "tl_forest_create: hipMalloc(leaves)"); }
    f->box_mem = nullptr;
    f->records_mem = nullptr;
    f->cuts_mem = nullptr;
    const size_t cut_bytes = 2 * (size_t)tl::kMaxCuts * sizeof(float);
    if (!boxes.empty()) e = hipMalloc(&f->box_mem, boxes.size() * sizeof(float4));
    if (e == hipSuccess && !records.empty()) e = hipMalloc(&f->records_mem, records.size());
    if (e == hipSuccess && !cuts_kv.empty() && !cuts_bs.empty()) e = hipMalloc(&f->cuts_mem, cut_bytes);
    if (e != hipSuccess) {
        (void)hipFree(f->nodes_mem);
        (void)hipFree(f->leaves_mem);
        if (f->box_mem) (void)hipFree(f->box_mem);
        if (f->records_mem) (void)hipFree(f->records_mem);
        if (f->cuts_mem) (void)hipFree(f->cuts_mem);
        (void)hipEventDestroy(f->ws_done);
        delete f;
        return from_hip(e, "tl_forest_create: hipMalloc");
    }
    e = hipMemcpy(f->nodes_mem, nodes.data(), nodes.size() * sizeof(uint2), hipMemcpyHostToDevice);
    if (e == hipSuccess)
        e = hipMemcpy(f->leaves_mem, leaves.data(), leaves.size() * sizeof(float), hipMemcpyHostToDevice);
    if (e == hipSuccess && f->box_mem)
        e = hipMemcpy(f->box_mem, boxes.data(), boxes.size() * sizeof(float4), hipMemcpyHostToDevice);
    if (e == hipSuccess && f->records_mem)
        e = hipMemcpy(f->records_mem, records.data(), records.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess && f->cuts_mem) {
        std::vector<float> cuts(2 * (size_t)tl::kMaxCuts, 0.0f);
        std::copy(cuts_kv.begin(), cuts_kv.end(), cuts.begin());
        std::copy(cuts_bs.begin(), cuts_bs.end(), cuts.begin() + tl::kMaxCuts);
        e = hipMemcpy(f->cuts_mem, cuts.data(), cut_bytes, hipMemcpyHostToDevice);
    }
    if (e != hipSuccess) {
        (void)hipFree(f->nodes_mem);
        (void)hipFree(f->leaves_mem);
        if (f->box_mem) (void)hipFree(f->box_mem);
        if (f->records_mem) (void)hipFree(f->records_mem);
        if (f->cuts_mem) (void)hipFree(f->cuts_mem);
        (void)hipEventDestroy(f->ws_done);
        delete f;
        return from_hip(e, "tl_forest_create: hipMemcpy");
    }
    f->dev.n_trees = n_trees;
    f->dev.depth = depth;
    f->dev.n_features = n_features;
    f->dev.base_score = base_score;
    f->dev.nodes = (const uint2*)f->nodes_mem;
    f->dev.leaves = (const float*)f->leaves_mem;
    f->dev.kvb_box = (const float4*)f->box_mem;
    f->dev.records = (const uint4*)f->records_mem;
    f->dev.cuts_kv = f->cuts_mem ? (const float*)f->cuts_mem : nullptr;
    f->dev.cuts_bs = f->cuts_mem ? (const float*)f->cuts_mem + tl::kMaxCuts : nullptr;
    f->dev.n_cuts_kv = f->cuts_mem ? (int32_t)cuts_kv.size() : 0;
    f->dev.n_cuts_bs = f->cuts_mem ? (int32_t)cuts_bs.size() : 0;
    *out = f;
    return ok();
}

void tl_forest_destroy(tl_forest* f) {
    if (!f) return;
    int cur = 0;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(f->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(f->nodes_mem);
    (void)hipFree(f->leaves_mem);
    if (f->box_mem) (void)hipFree(f->box_mem);
    if (f->records_mem) (void)hipFree(f->records_mem);
    if (f->cuts_mem) (void)hipFree(f->cuts_mem);
    if (f->ws) (void)hipFree(f->ws);
    (void)hipEventDestroy(f->ws_done);
    (void)hipSetDevice(cur);
    delete f;
}

}  // extern "C"

namespace {

// Whether `st` is being captured into a graph.  The optional workspaces are
// then left out: growing them allocates, and handing them between streams
// waits on events recorded outside the capture.  (A failed query counts as
// capturing: leaving the workspace out only costs speed.)
bool capturing(hipStream_t st) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &cs) != hipSuccess) {
        (void)hipGetLastError();
        return true;
    }
    return cs != hipStreamCaptureStatusNone;
}

// Runs launch(ws, ws_bytes) with the forest's cached work-order workspace
// of at least `need` bytes, all of its launches on st.  In the steady state
// nothing is allocated; a larger need than any before replaces the
// workspace (after the last call that used it is done).  Without a
// workspace (need 0, allocation failed, or the stream is being captured)
// launch gets (nullptr, 0) and runs without the order, which changes only
// its speed.
template <class Launch>
hipError_t with_workspace(const tl_forest* f, size_t need, hipStream_t st, Launch&& launch) {
    if (need == 0 || capturing(st)) return launch(nullptr, (size_t)0);
    std::lock_guard<std::mutex> lock(f->ws_mutex);
    hipError_t e;
    if (need > f->ws_bytes) {
        if (f->ws) {
            if (f->ws_used) {
                e = hipEventSynchronize(f->ws_done);
                if (e != hipSuccess) return e;
            }
            (void)hipFree(f->ws);
            f->ws = nullptr;
            f->ws_bytes = 0;
            f->ws_used = false;
        }
        if (hipMalloc(&f->ws, need) == hipSuccess) {
            f->ws_bytes = need;
        } else {
            f->ws = nullptr;
            (void)hipGetLastError();   // clear the allocation error before the launches check theirs
        }
    }
    if (!f->ws) return launch(nullptr, (size_t)0);
    if (f->ws_used && f->ws_stream != st) {
        e = hipStreamWaitEvent(st, f->ws_done, 0);
        if (e != hipSuccess) return e;
    }
    const hipError_t el = launch(f->ws, f->ws_bytes);
    // recorded also after a failed launch, whose earlier kernels may have
    // been enqueued on st and use the workspace
    e = hipEventRecord(f->ws_done, st);
    if (e == hipSuccess) {
        f->ws_stream = st;
        f->ws_used = true;
    }
    return el != hipSuccess ? el : e;
}

hipError_t grid_with_workspace(const tl_forest* f, const tl::GridParams& g, hipStream_t st) {
    size_t need = 0;
    const hipError_t e = tl::grid_order_bytes(f->dev, g, &need);
    if (e != hipSuccess) return e;
    return with_workspace(f, need, st,
                          [&](void* ws, size_t bytes) { return tl::launch_forest_grid(f->dev, g, ws, bytes, st); });
}

// `run` (launches of the column kernel on c's rows, and whatever goes
// between them) with c.order set from the forest's workspace when there is
// one: the order is computed once, before run, and serves every launch.
template <class Run>
hipError_t column_with_order(const tl_forest* f, tl::ColumnParams& c, hipStream_t st, Run&& run) {
    size_t need = 0;
    const hipError_t e = tl::column_order_bytes(f->dev, c, &need);
    if (e != hipSuccess) return e;
    return with_workspace(f, need, st, [&](void* ws, size_t) {
        c.order = nullptr;
        if (ws) {
            const hipError_t eo = tl::order_forest_column(f->dev, c, ws, st);
            if (eo != hipSuccess) return eo;
        }
        return run();
    });
}

// Host checks of a projection request and its translation to kernel
// parameters; `who` prefixes messages.  Rows are only looked at when
// `with_rows` (tl_admit ignores them).
tl_status project_params(const tl_project_args* a, const char* who, bool with_rows, tl::ProjectParams* p) {
    if (a->struct_size < sizeof(tl_project_args))
        return fail(TL_EINVAL, "%s: struct_size %u < %zu", who, a->struct_size, sizeof(tl_project_args));
    if (a->n_scenarios < 0 || a->n_scenarios > 0x7fffffffll)
        return fail(TL_EINVAL, "%s: n_scenarios %lld outside [0, 2^31-1]", who, (long long)a->n_scenarios);
    if (a->horizon < 1 || a->horizon > TL_MAX_HORIZON)
        return fail(TL_EINVAL, "%s: horizon %d outside [1, %d]", who, a->horizon, TL_MAX_HORIZON);
    if (a->block_tokens < 1 || a->block_tokens > TL_MAX_BLOCK_TOKENS)
        return fail(TL_EINVAL, "%s: block_tokens %d outside [1, %d]", who, a->block_tokens, TL_MAX_BLOCK_TOKENS);
    if (a->n_requests < 0) return fail(TL_EINVAL, "%s: n_requests < 0", who);
    if (!a->req_offset || !a->kv_capacity || !a->batch || !a->kv || !a->deadline_at || !a->n_iters || !a->flags)
        return fail(TL_EINVAL, "%s: NULL required pointer", who);
    if (a->n_requests > 0 && (!a->prompt_len || !a->generated || !a->remaining || !a->arrival_iter))
        return fail(TL_EINVAL, "%s: NULL request array", who);
    const bool rows = with_rows && a->rows;
    if (rows) {
        if (a->n_freqs < 1 || a->n_freqs > TL_MAX_FREQS)
            return fail(TL_EINVAL, "%s: n_freqs %d outside [1, %d]", who, a->n_freqs, TL_MAX_FREQS);
        if (a->n_features != 3 && a->n_features != 4)
            return fail(TL_EINVAL, "%s: n_features %d is not 3 or 4", who, a->n_features);
        if (!a->freqs_mhz) return fail(TL_EINVAL, "%s: rows requested without freqs_mhz", who);
        if (a->n_features == 4 && !a->engine_size) return fail(TL_EINVAL, "%s: 4 features need engine_size", who);
        if (a->n_features == 4 && ((uintptr_t)a->rows & 15u))
            return fail(TL_EINVAL, "%s: rows must be 16-byte aligned for 4 features", who);
    }
    *p = tl::ProjectParams{};
    p->n_scenarios = a->n_scenarios;
    p->n_requests = a->n_requests;
    p->H = a->horizon;
    p->N = a->block_tokens;
    const tl::DivU32 dv = tl::make_divu32((uint32_t)a->block_tokens);
    p->div_m = dv.m;
    p->div_l = dv.l;
    p->off = a->req_offset;
    p->prompt = a->prompt_len;
    p->gen = a->generated;
    p->rem = a->remaining;
    p->arr = a->arrival_iter;
    p->deadline = a->deadline_ns;
    p->lost = a->lost;
    p->kv_cap = a->kv_capacity;
    p->batch_cap = a->batch_cap;
    p->batch = a->batch;
    p->kv = a->kv;
    p->deadline_at = a->deadline_at;
    p->n_iters = a->n_iters;
    p->flags = a->flags;
    p->rows = rows ? a->rows : nullptr;
    p->F = rows ? a->n_freqs : 0;
    p->nf = rows ? a->n_features : 0;
    p->freqs = rows ? a->freqs_mhz : nullptr;
    p->engine = rows ? a->engine_size : nullptr;
    p->cand_prompt = nullptr;
    p->cand_len = nullptr;
    p->order_ws = nullptr;
    return TL_OK;
}

// The projection's scenario order (heaviest first, for long FIFO loops) needs
// a workspace of one word per scenario: owned by the library, one per device,
// allocated on first use and replaced only by a larger one.  A call on
// another stream than the previous user first waits (on the device) for that
// user's projection.  Without the workspace (allocation failure, device
// number out of range, a stream being captured) the scenarios run in their
// own order: same results.
constexpr int kOrderDevices = 64;
struct OrderWorkspace {
    std::mutex m;
    void* ptr = nullptr;
    size_t bytes = 0;
    hipEvent_t done = nullptr;
    hipStream_t stream = nullptr;
    bool used = false;
};
OrderWorkspace g_order_ws[kOrderDevices];

hipError_t project_launch(tl::ProjectParams p, hipStream_t st) {
    const size_t need = tl::project_order_bytes(p);
    int dev = -1;
    if (need == 0 || capturing(st) || hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kOrderDevices)
        return tl::launch_project(p, st);
    OrderWorkspace& w = g_order_ws[dev];
    std::lock_guard<std::mutex> lock(w.m);
    hipError_t e = hipSuccess;
    if (!w.done && hipEventCreateWithFlags(&w.done, hipEventDisableTiming) != hipSuccess) {
        w.done = nullptr;
        (void)hipGetLastError();
        return tl::launch_project(p, st);
    }
    if (need > w.bytes) {
        if (w.ptr) {
            if (w.used) {
                e = hipEventSynchronize(w.done);
                if (e != hipSuccess) return e;
            }
            (void)hipFree(w.ptr);
            w.ptr = nullptr;
            w.bytes = 0;
            w.used = false;
        }
        if (hipMalloc(&w.ptr, need) == hipSuccess) {
            w.bytes = need;
        } else {
            w.ptr = nullptr;
            (void)hipGetLastError();   // clear the allocation error before the launches check theirs
        }
    }
    if (!w.ptr) return tl::launch_project(p, st);
    if (w.used && w.stream != st) {
        e = hipStreamWaitEvent(st, w.done, 0);
        if (e != hipSuccess) return e;
    }
    p.order_ws = w.ptr;
    const hipError_t el = tl::launch_project(p, st);
    // recorded also after a failed launch, whose order kernels may have been
    // enqueued on st and use the workspace
    e = hipEventRecord(w.done, st);
    if (e == hipSuccess) {
        w.stream = st;
        w.used = true;
    }
    return el != hipSuccess ? el : e;
}

}  // namespace

extern "C" {

tl_status tl_project(const tl_project_args* a, void* stream) {
    if (!a) return fail(TL_EINVAL, "tl_project: args is NULL");
    tl::ProjectParams p;
    const tl_status st = project_params(a, "tl_project", true, &p);
    if (st != TL_OK) return st;
    if (a->n_scenarios == 0) return ok();
    return from_hip(project_launch(p, (hipStream_t)stream), "tl_project: launch");
}

tl_status tl_admit(const tl_admit_args* a, void* stream) {
    if (!a) return fail(TL_EINVAL, "tl_admit: args is NULL");
    if (a->struct_size < sizeof(tl_admit_args))
        return fail(TL_EINVAL, "tl_admit: struct_size %u < %zu", a->struct_size, sizeof(tl_admit_args));
    tl::ProjectParams p;
    const tl_status st = project_params(&a->proj, "tl_admit", false, &p);
    if (st != TL_OK) return st;
    const tl_forest* f = a->forest;
    if (!f) return fail(TL_EINVAL, "tl_admit: forest is NULL");
    if (!a->tbt_slo_ns || !a->cand_prompt || !a->cand_len || !a->ips || !a->decision)
        return fail(TL_EINVAL, "tl_admit: NULL required pointer");
    if (f->dev.n_features != 3 && f->dev.n_features != 4)
        return fail(TL_EINVAL, "tl_admit: the forest has %d features, admission needs 3 or 4", f->dev.n_features);
    if (f->dev.n_features == 4 && !a->engine_size) return fail(TL_EINVAL, "tl_admit: 4 features need engine_size");
    if (a->lattice && a->lattice->forest != f)
        return fail(TL_EINVAL, "tl_admit: the lattice was built from another forest");
    const int64_t S = a->proj.n_scenarios;
    if (S == 0) return ok();
    const hipStream_t st_h = (hipStream_t)stream;
    p.cand_prompt = a->cand_prompt;
    p.cand_len = a->cand_len;
    hipError_t e = project_launch(p, st_h);
    if (e != hipSuccess) return from_hip(e, "tl_admit: projection launch");
    tl::ColumnParams c{};
    c.S = S;
    c.H = a->proj.horizon;
    c.kv = a->proj.kv;
    c.batch = a->proj.batch;
    c.freq = a->max_freq_mhz;
    c.engine = a->engine_size;
    c.out = a->ips;
    int32_t lat_f = -1;
    if (a->lattice) {
        const std::vector<float>& hf = a->lattice->host_freqs;
        for (size_t q = 0; q < hf.size(); ++q)
            if (hf[q] == a->max_freq_mhz) { lat_f = (int32_t)q; break; }
    }
    if (lat_f >= 0) {
        // the maximum frequency is on the lattice: one table read per row
        tl::GatherParams gp{};
        gp.S = S;
        gp.H = a->proj.horizon;
        gp.kv = a->proj.kv;
        gp.batch = a->proj.batch;
        gp.engine = f->dev.n_features == 4 ? a->engine_size : nullptr;
        gp.out = a->ips;
        e = tl::launch_lattice_column(f->dev, a->lattice->dev, gp, nullptr, lat_f, st_h);
    } else {
        e = column_with_order(f, c, st_h, [&]() { return tl::launch_forest_column(f->dev, c, st_h); });
    }
    if (e != hipSuccess) return from_hip(e, "tl_admit: model launch");
    tl::AdmitParams d{};
    d.ips = a->ips;
    d.S = S;
    d.H = a->proj.horizon;
    d.deadline_at = a->proj.deadline_at;
    d.n_iters = a->proj.n_iters;
    d.tbt_slo_ns = a->tbt_slo_ns;
    d.proj_flags = a->proj.flags;
    d.cand_len = a->cand_len;
    d.cand_deadline = a->cand_deadline_ns;
    d.decision = a->decision;
    return from_hip(tl::launch_admit(d, st_h), "tl_admit: decision launch");
}

tl_status tl_forest_predict(const tl_forest* f, const float* rows, int64_t n_rows, float* out, void* stream) {
    if (!f) return fail(TL_EINVAL, "tl_forest_predict: forest is NULL");
    if (n_rows < 0) return fail(TL_EINVAL, "tl_forest_predict: n_rows < 0");
    if (n_rows > 0 && (!rows || !out)) return fail(TL_EINVAL, "tl_forest_predict: NULL rows or out");
    if (n_rows > (int64_t)0x7fffffff * 256 * 4)
        return fail(TL_EUNSUPPORTED, "tl_forest_predict: n_rows %lld too large", (long long)n_rows);
    if (n_rows == 0) return ok();
    return from_hip(tl::launch_forest_rows(f->dev, rows, n_rows, out, (hipStream_t)stream),
                    "tl_forest_predict: launch");
}

}  // extern "C"

namespace {

// Host checks of a grid prediction and its kernel parameters; TL_OK with
// g->S == 0 means there is nothing to do.
tl_status grid_params(const char* who, const tl_forest* f, int64_t n_scenarios, int32_t n_freqs, int32_t horizon,
                      const float* freqs_mhz, const int32_t* kv, const int32_t* batch, const float* engine_size,
                      float* out, tl::GridParams* g) {
    *g = tl::GridParams{};
    if (!f) return fail(TL_EINVAL, "%s: forest is NULL", who);
    if (f->dev.n_features != 3 && f->dev.n_features != 4)
        return fail(TL_EINVAL, "%s: the forest has %d features, the grid needs 3 or 4", who, f->dev.n_features);
    if (n_scenarios < 0 || n_scenarios > 0x7fffffffll)
        return fail(TL_EINVAL, "%s: n_scenarios %lld outside [0, 2^31-1]", who, (long long)n_scenarios);
    if (n_freqs < 1 || n_freqs > TL_MAX_FREQS)
        return fail(TL_EINVAL, "%s: n_freqs %d outside [1, %d]", who, n_freqs, TL_MAX_FREQS);
    if (horizon < 1 || horizon > TL_MAX_HORIZON)
        return fail(TL_EINVAL, "%s: horizon %d outside [1, %d]", who, horizon, TL_MAX_HORIZON);
    if (n_scenarios > 0 && (!freqs_mhz || !kv || !batch || !out))
        return fail(TL_EINVAL, "%s: NULL required pointer", who);
    if (n_scenarios > 0 && f->dev.n_features == 4 && !engine_size)
        return fail(TL_EINVAL, "%s: a 4-feature forest needs engine_size", who);
    if (n_scenarios == 0) return ok();
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess || cur != f->device)
        return fail(TL_EINVAL, "%s: the forest lives on device %d, the current device is %d", who, f->device, cur);
    g->S = n_scenarios;
    g->F = n_freqs;
    g->H = horizon;
    g->freqs = freqs_mhz;
    g->kv = kv;
    g->batch = batch;
    g->engine = f->dev.n_features == 4 ? engine_size : nullptr;
    g->out = out;
    return ok();
}

}  // namespace

extern "C" {

tl_status tl_forest_predict_grid(const tl_forest* f, int64_t n_scenarios, int32_t n_freqs, int32_t horizon,
                                 const float* freqs_mhz, const int32_t* kv, const int32_t* batch,
                                 const float* engine_size, float* out, void* stream) {
    tl::GridParams g;
    const tl_status st = grid_params("tl_forest_predict_grid", f, n_scenarios, n_freqs, horizon, freqs_mhz, kv,
                                     batch, engine_size, out, &g);
    if (st != TL_OK || g.S == 0) return st;
    return from_hip(grid_with_workspace(f, g, (hipStream_t)stream), "tl_forest_predict_grid: launch");
}

tl_status tl_forest_predict_grid_noalloc(const tl_forest* f, int64_t n_scenarios, int32_t n_freqs,
                                         int32_t horizon, const float* freqs_mhz, const int32_t* kv,
                                         const int32_t* batch, const float* engine_size, float* out,
                                         void* stream) {
    const char* who = "tl_forest_predict_grid_noalloc";
    tl::GridParams g;
    const tl_status st = grid_params(who, f, n_scenarios, n_freqs, horizon, freqs_mhz, kv, batch, engine_size, out,
                                     &g);
    if (st != TL_OK || g.S == 0) return st;
    size_t need = 0;
    hipError_t e = tl::grid_order_bytes(f->dev, g, &need);
    if (e != hipSuccess) return from_hip(e, "tl_forest_predict_grid_noalloc: sizing the work order");
    if (need > tl::kNoAllocScratchBytes)
        return fail(TL_EUNSUPPORTED,
                    "%s: the work order of %lld scenarios x %d iterations needs %zu bytes of scratch, more than the "
                    "fixed %zu (use tl_forest_predict_grid)",
                    who, (long long)n_scenarios, horizon, need, tl::kNoAllocScratchBytes);
    void* ws = nullptr;
    if (need > 0) {
        e = tl::noalloc_scratch(&ws);
        if (e != hipSuccess) return from_hip(e, "tl_forest_predict_grid_noalloc: scratch address");
    }
    return from_hip(tl::launch_forest_grid(f->dev, g, ws, need > 0 ? tl::kNoAllocScratchBytes : 0,
                                           (hipStream_t)stream),
                    "tl_forest_predict_grid_noalloc: launch");
}

tl_status tl_select_freq(const float* ips, int64_t n_scenarios, int32_t n_freqs, int32_t horizon,
                         const uint64_t* deadline_at, const int32_t* n_iters, const uint64_t* tbt_slo_ns,
                         const uint32_t* proj_flags, int32_t* freq_idx, uint32_t* status, void* stream) {
    if (n_scenarios < 0 || n_scenarios > 0x7fffffffll)
        return fail(TL_EINVAL, "tl_select_freq: n_scenarios %lld outside [0, 2^31-1]", (long long)n_scenarios);
    if (n_freqs < 1 || n_freqs > TL_MAX_FREQS)
        return fail(TL_EINVAL, "tl_select_freq: n_freqs %d outside [1, %d]", n_freqs, TL_MAX_FREQS);
    if (horizon < 1) return fail(TL_EINVAL, "tl_select_freq: horizon %d < 1", horizon);
    if (n_scenarios > 0 && (!ips || !deadline_at || !n_iters || !tbt_slo_ns || !freq_idx || !status))
        return fail(TL_EINVAL, "tl_select_freq: NULL required pointer");
    if (n_scenarios == 0) return ok();
    tl::SelectParams p{};
    p.ips = ips;
    p.S = n_scenarios;
    p.F = n_freqs;
    p.H = horizon;
    p.deadline_at = deadline_at;
    p.n_iters = n_iters;
    p.tbt_slo_ns = tbt_slo_ns;
    p.proj_flags = proj_flags;
    p.freq_idx = freq_idx;
    p.status = status;
    return from_hip(tl::launch_select(p, (hipStream_t)stream), "tl_select_freq: launch");
}

tl_status tl_lattice_create(const tl_forest* f, int32_t n_freqs, const float* freqs_mhz, int32_t n_engines,
                            const float* engine_values, int32_t kv_max, int32_t batch_max, void* stream,
                            tl_lattice** out) {
    if (!out) return fail(TL_EINVAL, "tl_lattice_create: out is NULL");
    *out = nullptr;
    if (!f) return fail(TL_EINVAL, "tl_lattice_create: forest is NULL");
    const int32_t nf = f->dev.n_features;
    if (nf != 3 && nf != 4)
        return fail(TL_EINVAL, "tl_lattice_create: the forest has %d features, the lattice needs 3 or 4", nf);
    if (n_freqs < 1 || n_freqs > TL_MAX_FREQS)
        return fail(TL_EINVAL, "tl_lattice_create: n_freqs %d outside [1, %d]", n_freqs, TL_MAX_FREQS);
    if (!freqs_mhz) return fail(TL_EINVAL, "tl_lattice_create: freqs_mhz is NULL");
    if (nf == 4 && (n_engines < 1 || n_engines > tl::kMaxLatticeEngines || !engine_values))
        return fail(TL_EINVAL, "tl_lattice_create: a 4-feature forest needs 1..%d engine sizes",
                    tl::kMaxLatticeEngines);
    if (kv_max < 0 || batch_max < 0 || batch_max >= (1 << 20))
        return fail(TL_EINVAL, "tl_lattice_create: kv_max %d / batch_max %d outside range", kv_max, batch_max);
    tl::LatticeDev L{};
    L.nf = nf;
    L.F = n_freqs;
    L.nE = nf == 4 ? n_engines : 1;
    L.nB = batch_max + 1;
    L.nC = kv_max / tl::kLatticeChunk + 1;
    L.kv_max = kv_max;
    L.batch_max = batch_max;
    for (int32_t q = 0; q < tl::kMaxLatticeEngines; ++q) L.engines[q] = (nf == 4 && q < n_engines) ? engine_values[q] : 0.0f;
    const uint64_t n_scen = (uint64_t)L.nE * L.nB * L.nC;
    const uint64_t entries = n_scen * (uint64_t)L.F * tl::kLatticeChunk;
    const uint64_t bytes = entries * 4u;
    if (n_scen > 0x7fffffffull || bytes > (256ull << 30))
        return fail(TL_EUNSUPPORTED, "tl_lattice_create: the table would take %llu bytes (limit 256 GiB)",
                    (unsigned long long)bytes);
    const uint64_t freq_bytes = ((uint64_t)n_freqs * 4u + 255u) & ~255ull;
    tl_lattice* lat = new (std::nothrow) tl_lattice{};
    if (!lat) return fail(TL_ENOMEM, "tl_lattice_create: host allocation failed");
    lat->forest = f;
    lat->bytes = bytes;
    const hipStream_t st = (hipStream_t)stream;
    hipError_t e = hipGetDevice(&lat->device);
    if (e == hipSuccess) e = hipMalloc(&lat->mem, freq_bytes + bytes);
    if (e != hipSuccess) {
        delete lat;
        return from_hip(e, "tl_lattice_create: device allocation");
    }
    float* freqs = (float*)lat->mem;
    L.freqs = freqs;
    L.table = (const float*)((unsigned char*)lat->mem + freq_bytes);
    lat->dev = L;
    // build: one grid scenario per (engine size, batch, KV chunk), in batches
    // of scenarios through a temporary of at most ~512 MB, each transposed
    // into the table
    void* work = nullptr;
    const uint64_t per_scen = (uint64_t)n_freqs * tl::kLatticeChunk * 4u;
    const uint64_t batch_n = std::max<uint64_t>(1, std::min<uint64_t>(n_scen, (512ull << 20) / per_scen));
    lat->host_freqs.assign((size_t)n_freqs, 0.0f);
    e = hipMemcpyAsync(freqs, freqs_mhz, (size_t)n_freqs * 4u, hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess)
        e = hipMemcpyAsync(lat->host_freqs.data(), freqs_mhz, (size_t)n_freqs * 4u, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e == hipSuccess)
        e = hipMallocAsync(&work, batch_n * (per_scen + tl::kLatticeChunk * 8u + 4u) + 256u, st);
    if (e == hipSuccess) {
        float* grid_out = (float*)work;
        int32_t* kv = (int32_t*)(grid_out + batch_n * n_freqs * tl::kLatticeChunk);
        int32_t* batch = kv + batch_n * tl::kLatticeChunk;
        float* eng = (float*)(batch + batch_n * tl::kLatticeChunk);
        for (uint64_t s0 = 0; s0 < n_scen && e == hipSuccess; s0 += batch_n) {
            const int64_t cnt = (int64_t)std::min<uint64_t>(batch_n, n_scen - s0);
            e = tl::launch_lattice_inputs(L, (int64_t)s0, cnt, kv, batch, eng, st);
            if (e == hipSuccess) {
                tl::GridParams g{};
                g.S = cnt;
                g.F = n_freqs;
                g.H = tl::kLatticeChunk;
                g.freqs = freqs;
                g.kv = kv;
                g.batch = batch;
                g.engine = nf == 4 ? eng : nullptr;
                g.out = grid_out;
                e = grid_with_workspace(f, g, st);
            }
            if (e == hipSuccess)
                e = tl::launch_lattice_transpose(grid_out, (float*)L.table, (int64_t)s0, cnt, n_freqs, st);
        }
        const hipError_t e2 = hipFreeAsync(work, st);
        if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) {
        (void)hipStreamSynchronize(st);
        (void)hipFree(lat->mem);
        delete lat;
        return from_hip(e, "tl_lattice_create: build");
    }
    *out = lat;
    return ok();
}

void tl_lattice_destroy(tl_lattice* lat) {
    if (!lat) return;
    int cur = 0;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(lat->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(lat->mem);
    (void)hipSetDevice(cur);
    delete lat;
}

uint64_t tl_lattice_bytes(const tl_lattice* lat) { return lat ? lat->bytes : 0; }

tl_status tl_lattice_predict_grid(const tl_lattice* lat, int64_t n_scenarios, int32_t horizon, const int32_t* kv,
                                  const int32_t* batch, const float* engine_size, float* out, void* stream) {
    if (!lat) return fail(TL_EINVAL, "tl_lattice_predict_grid: lattice is NULL");
    if (n_scenarios < 0 || n_scenarios > 0x7fffffffll)
        return fail(TL_EINVAL, "tl_lattice_predict_grid: n_scenarios %lld outside [0, 2^31-1]", (long long)n_scenarios);
    if (horizon < 1 || horizon > TL_MAX_HORIZON)
        return fail(TL_EINVAL, "tl_lattice_predict_grid: horizon %d outside [1, %d]", horizon, TL_MAX_HORIZON);
    if (n_scenarios == 0) return ok();
    if (!kv || !batch || !out) return fail(TL_EINVAL, "tl_lattice_predict_grid: NULL required pointer");
    if (lat->dev.nf == 4 && !engine_size)
        return fail(TL_EINVAL, "tl_lattice_predict_grid: a 4-feature forest needs engine_size");
    tl::GatherParams p{};
    p.S = n_scenarios;
    p.H = horizon;
    p.kv = kv;
    p.batch = batch;
    p.engine = lat->dev.nf == 4 ? engine_size : nullptr;
    p.out = out;
    return from_hip(tl::launch_lattice_gather(lat->forest->dev, lat->dev, p, (hipStream_t)stream),
                    "tl_lattice_predict_grid: launch");
}

tl_status tl_adjust_lengths(int64_t n_scenarios, int64_t n_requests, const int64_t* req_offset,
                            const int32_t* generated, const int32_t* pred_len, const uint32_t* scale_num,
                            const uint32_t* scale_den, const int32_t* max_tokens, int32_t* remaining_out,
                            void* stream) {
    if (n_scenarios < 0 || n_scenarios > 0x7fffffffll)
        return fail(TL_EINVAL, "tl_adjust_lengths: n_scenarios %lld outside [0, 2^31-1]", (long long)n_scenarios);
    if (n_requests < 0) return fail(TL_EINVAL, "tl_adjust_lengths: n_requests < 0");
    if (n_scenarios == 0) return ok();
    if (!req_offset || !scale_num || !scale_den || !max_tokens)
        return fail(TL_EINVAL, "tl_adjust_lengths: NULL required pointer");
    if (n_requests > 0 && (!generated || !pred_len || !remaining_out))
        return fail(TL_EINVAL, "tl_adjust_lengths: NULL request array");
    tl::AdjustParams p{};
    p.S = n_scenarios;
    p.n_requests = n_requests;
    p.off = req_offset;
    p.gen = generated;
    p.pred = pred_len;
    p.num = scale_num;
    p.den = scale_den;
    p.max_tokens = max_tokens;
    p.out = remaining_out;
    return from_hip(tl::launch_adjust(p, (hipStream_t)stream), "tl_adjust_lengths: launch");
}

tl_status tl_select_freq_binary(const tl_forest* f, int64_t n_scenarios, int32_t n_freqs, int32_t horizon,
                                const float* freqs_mhz, const int32_t* kv, const int32_t* batch,
                                const float* engine_size, const uint64_t* deadline_at, const int32_t* n_iters,
                                const uint64_t* tbt_slo_ns, const uint32_t* proj_flags, float* ips_work,
                                int32_t* search_work, int32_t* freq_idx, uint32_t* status,
                                const tl_lattice* lattice, void* stream) {
    if (!f) return fail(TL_EINVAL, "tl_select_freq_binary: forest is NULL");
    if (lattice && (lattice->forest != f || lattice->dev.F != n_freqs))
        return fail(TL_EINVAL, "tl_select_freq_binary: the lattice was built from another forest or frequency count");
    if (n_scenarios < 0 || n_scenarios > 0x7fffffffll)
        return fail(TL_EINVAL, "tl_select_freq_binary: n_scenarios %lld outside [0, 2^31-1]", (long long)n_scenarios);
    if (n_freqs < 1 || n_freqs > TL_MAX_FREQS)
        return fail(TL_EINVAL, "tl_select_freq_binary: n_freqs %d outside [1, %d]", n_freqs, TL_MAX_FREQS);
    if (horizon < 1 || horizon > TL_MAX_HORIZON)
        return fail(TL_EINVAL, "tl_select_freq_binary: horizon %d outside [1, %d]", horizon, TL_MAX_HORIZON);
    if (n_scenarios == 0) return ok();
    if (!freqs_mhz || !kv || !batch || !deadline_at || !n_iters || !tbt_slo_ns || !ips_work || !search_work ||
        !freq_idx || !status)
        return fail(TL_EINVAL, "tl_select_freq_binary: NULL required pointer");
    if (f->dev.n_features != 3 && f->dev.n_features != 4)
        return fail(TL_EINVAL, "tl_select_freq_binary: the forest has %d features, the search needs 3 or 4",
                    f->dev.n_features);
    if (f->dev.n_features == 4 && !engine_size)
        return fail(TL_EINVAL, "tl_select_freq_binary: 4 features need engine_size");
    const hipStream_t st = (hipStream_t)stream;
    tl::SearchParams sp{};
    sp.ips = ips_work;
    sp.S = n_scenarios;
    sp.F = n_freqs;
    sp.H = horizon;
    sp.deadline_at = deadline_at;
    sp.n_iters = n_iters;
    sp.tbt_slo_ns = tbt_slo_ns;
    sp.proj_flags = proj_flags;
    sp.work = search_work;
    sp.freq_idx = freq_idx;
    sp.status = status;
    tl::ColumnParams c{};
    c.S = n_scenarios;
    c.H = horizon;
    c.kv = kv;
    c.batch = batch;
    c.freqs = freqs_mhz;
    c.fidx = search_work + 2 * n_scenarios;
    c.engine = engine_size;
    c.out = ips_work;
    tl::GatherParams gp{};
    gp.S = n_scenarios;
    gp.H = horizon;
    gp.kv = kv;
    gp.batch = batch;
    gp.engine = f->dev.n_features == 4 ? engine_size : nullptr;
    gp.out = ips_work;
    // M at every scenario's probe: a table read per row with a lattice, walks otherwise
    auto model = [&]() {
        return lattice ? tl::launch_lattice_column(f->dev, lattice->dev, gp, c.fidx, 0, st)
                       : tl::launch_forest_column(f->dev, c, st);
    };
    int32_t rounds = 0;
    while ((int64_t)1 << rounds < n_freqs) ++rounds;
    // live (nullable): scratch for compacting the final probe's work to the
    // scenarios that still probe
    auto search = [&](void* live) {
        hipError_t e = tl::launch_search_step(sp, 0, st);
        for (int32_t r = 0; r < rounds && e == hipSuccess; ++r) {
            e = model();
            if (e == hipSuccess) e = tl::launch_search_step(sp, 1, st);
        }
        if (e == hipSuccess) e = tl::launch_search_step(sp, 3, st);
        if (e == hipSuccess) e = live ? tl::launch_forest_column_live(f->dev, c, live, st) : model();
        if (e == hipSuccess) e = tl::launch_search_step(sp, 2, st);
        return e;
    };
    if (lattice) return from_hip(search(nullptr), "tl_select_freq_binary: launch");
    // The probes walk the same rows every round: one work order serves them
    // all.  Scratch: the order, then the final probe's live items.
    size_t need_order = 0, need_live = 0;
    hipError_t e = tl::column_order_bytes(f->dev, c, &need_order);
    if (e == hipSuccess) e = tl::column_live_bytes(f->dev, c, &need_live);
    if (e != hipSuccess) return from_hip(e, "tl_select_freq_binary: launch");
    need_order = (need_order + 255) & ~(size_t)255;
    e = with_workspace(f, need_order + need_live, st, [&](void* ws, size_t) {
        c.order = nullptr;
        if (!ws) return search(nullptr);
        if (need_order > 0) {
            const hipError_t eo = tl::order_forest_column(f->dev, c, ws, st);
            if (eo != hipSuccess) return eo;
        }
        return search(need_live > 0 ? (unsigned char*)ws + need_order : nullptr);
    });
    return from_hip(e, "tl_select_freq_binary: launch");
}

}  // extern "C"
