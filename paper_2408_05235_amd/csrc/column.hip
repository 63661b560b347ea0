// The model M (Sec. 4.3.1) at one frequency per scenario on the projection
// grid: out[s][j] = M(f_s, KV[s][j], B[s][j] [, E_s]), f_s = freqs[fidx[s]]
// (scenarios with fidx[s] < 0 are skipped) or one frequency for all.  This is the query of
// the admission checks (Sec. 4.3.2 check 2 asks M at the maximum frequency
// for every projected iteration) and of one probe of a search over
// frequencies (Sec. 4.5).
//
// A wavefront takes RPL stripes of 64 consecutive iterations of one scenario,
// RPL rows per lane; the rows differ, so every lane walks every tree (the grid
// kernel's leaf reuse needs many frequencies on the same row sequence).
// Sixteen wavefronts of a workgroup share two LDS buffers of tree-record
// blocks, copied straight from global memory and handed over without block
// barriers (stage_acquire / stage_release, which also set the wavefronts'
// issue priorities).  A lane walks its RPL rows through up to four trees at
// once, so RPL x trees chains of dependent LDS reads overlap (deep trees leave
// room for only two trees per block).  Leaves are added as an fp32 running sum
// in tree order, as everywhere in the library.
//
// On horizons of at least 64 x RPL iterations and grids of at least one
// workgroup per CU, forest_column_reuse_kernel gives each lane RPL (16, else
// 8) consecutive iterations instead and reuses leaves along them: every lane
// walks its first and last row, and the rows in between take those leaves
// where their boxes hold them (the grid kernel's box test, per lane).
//
// Forests too deep for LDS records are walked from global memory.
//
// Rows mode (P.rows): the same kernel on arbitrary feature rows, lane l of
// item i taking rows i*64*RPL + l + 64 r; every row carries its own
// frequency and engine size.  tl_forest_predict uses it for 3- and
// 4-feature forests with LDS records.
#include <algorithm>

#include "device_util.h"
#include "tl_internal.h"
#include "forest_walk.h"

namespace tl {
namespace {

constexpr int kColWaves = 16;
constexpr int kColThreads = kColWaves * kWave;
constexpr size_t kColLdsBudget = 152 * 1024;

template <int RPL>
struct ColumnItem {
    int64_t s;
    int32_t j[RPL];     // this lane's iterations (clamped into the horizon)
    bool row[RPL];      // ... and whether each is inside it
    bool valid;         // the wavefront has a scenario
};

template <int RPL>
__device__ __forceinline__ ColumnItem<RPL> column_item(const ColumnParams& P, int64_t item) {
    const int32_t span = kWave * RPL;
    const int32_t n_cols = (P.H + span - 1) / span;
    ColumnItem<RPL> c;
    c.valid = item < P.S * n_cols;
    c.s = c.valid ? item / n_cols : 0;
    // a scenario without a frequency to evaluate (index < 0) is skipped
    if (P.fidx && P.fidx[c.s] < 0) c.valid = false;
    const int32_t j0 = (int32_t)(item % n_cols) * span + lane_id();
#pragma unroll
    for (int r = 0; r < RPL; ++r) {
        const int32_t j = j0 + r * kWave;
        c.row[r] = c.valid && j < P.H;
        c.j[r] = min(j, P.H - 1);
    }
    return c;
}

__device__ __forceinline__ float column_freq(const ColumnParams& P, int64_t s) {
    return P.fidx ? P.freqs[max(P.fidx[s], 0)] : P.freq;
}

// The leaves lf[r][t] that NR rows (each with its own features) reach in NT
// consecutive staged trees (records R.bytes apart, the first at LDS byte
// address `tree`), all NR x NT chains of dependent LDS reads interleaved:
// every chain's node reads issue back to back, then the compares.
template <int NF, int NT, int NR>
__device__ __forceinline__ void walk_rows(uint32_t tree, const RecordLayout& R, int32_t depth, const float (&xf)[NR],
                                          const float (&kv)[NR], const float (&bs)[NR], const float (&xe)[NR],
                                          LeafAt (&lf)[NR][NT]) {
    const uint32_t rec_bytes = R.bytes;
    uint32_t a[NR][NT], cl[NT], cr[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const uint32_t root = tree + t * rec_bytes;
        cl[t] = 16u - root;
        cr[t] = 32u - root;
        asm volatile("" : "+v"(cl[t]), "+v"(cr[t]));
#pragma unroll
        for (int r = 0; r < NR; ++r) a[r][t] = root;
    }
    for (int32_t level = 0; level < depth; ++level) {
        uint4 w[NR][NT];
#pragma unroll
        for (int r = 0; r < NR; ++r)
#pragma unroll
            for (int t = 0; t < NT; ++t) w[r][t] = read_node(a[r][t]);
#pragma unroll
        for (int r = 0; r < NR; ++r)
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const bool left = node_feature<NF>(w[r][t], xf[r], kv[r], bs[r], xe[r]) < __uint_as_float(w[r][t].x);
                a[r][t] = 2u * a[r][t] + (left ? cl[t] : cr[t]);
            }
    }
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int t = 0; t < NT; ++t) lf[r][t] = leaf_at(a[r][t], tree + t * rec_bytes, R, depth);
}

// Walks NT consecutive staged trees for the RPL rows of a lane and adds the
// leaves to each row's sum in tree order.
template <int NF, int NT, int RPL>
__device__ __forceinline__ void add_leaves(uint32_t tree, const RecordLayout& R, int32_t depth,
                                           const float (&xf)[RPL], const float (&kv)[RPL], const float (&bs)[RPL],
                                           const float (&xe)[RPL], float (&acc)[RPL]) {
    LeafAt k[RPL][NT];
    walk_rows<NF, NT, RPL>(tree, R, depth, xf, kv, bs, xe, k);
#pragma unroll
    for (int r = 0; r < RPL; ++r)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[r] += leaf_value(k[r][t]);
}

template <int NF, int RPL, bool ROWS>
__global__ __launch_bounds__(kColThreads) void forest_column_lds_kernel(const uint4* __restrict__ records,
                                                                       int32_t n_trees, int32_t depth, int32_t tb,
                                                                       float base, ColumnParams P) {
    extern __shared__ __align__(16) unsigned char smem[];
    const RecordLayout R = record_layout(depth);
    const uint32_t rec_words = R.bytes / 16u;
    const uint32_t buf_bytes = stage_buffer_bytes(tb, R);
    const int wave = threadIdx.x / kWave;
    const int64_t item = __builtin_amdgcn_readfirstlane((int64_t)blockIdx.x * kColWaves + wave);
    float xf[RPL], kv[RPL], bs[RPL], xe[RPL];
    float acc[RPL];
    int64_t o[RPL];     // output index of each row, < 0: none
    bool valid;         // the wavefront has rows (uniform)
    if (ROWS) {
        const int64_t first = item * (kWave * RPL);
        valid = first < P.n_rows;
#pragma unroll
        for (int r = 0; r < RPL; ++r) {
            const int64_t i = first + lane_id() + r * kWave;
            o[r] = i < P.n_rows ? i : -1;
            const float* x = P.rows + (valid ? min(i, P.n_rows - 1) : 0) * NF;
            xf[r] = x[0];
            kv[r] = x[1];
            bs[r] = x[2];
            xe[r] = NF == 4 ? x[3] : 0.0f;
        }
    } else {
        const ColumnItem<RPL> c = column_item<RPL>(P, item);
        valid = c.valid;
        const float f_s = column_freq(P, c.s);
        const float e_s = NF == 4 ? P.engine[c.s] : 0.0f;
#pragma unroll
        for (int r = 0; r < RPL; ++r) {
            xf[r] = f_s;
            xe[r] = e_s;
            kv[r] = (float)P.kv[c.s * P.H + c.j[r]];
            bs[r] = (float)P.batch[c.s * P.H + c.j[r]];
            o[r] = c.row[r] ? c.s * P.H + c.j[r] : -1;
        }
    }
#pragma unroll
    for (int r = 0; r < RPL; ++r) {
        acc[r] = base;
        // the rows are complete before any staging load is in flight
        asm volatile("" ::"v"(xf[r]), "v"(kv[r]), "v"(bs[r]), "v"(xe[r]));
    }

    const int32_t n_blocks = (n_trees + tb - 1) / tb;
    StageSync* sync = (StageSync*)(smem + 2 * buf_bytes);
    if (threadIdx.x == 0) stage_sync_init(sync);
    if (n_blocks > 0) stage_block(records, n_trees, tb, rec_words, 0, lds_addr(smem), wave, kColWaves);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    bool sync_ok = true;
    for (int32_t b = 0; b < n_blocks; ++b) {
        const int cur = b & 1;
        if (b > 0)
            sync_ok &= stage_acquire(sync, b, kColWaves, records, n_trees, tb, rec_words,
                                     lds_addr(smem) + cur * buf_bytes);
        if (valid) {
            const int32_t cnt = min(tb, n_trees - b * tb);
            const uint32_t first = lds_addr(smem) + cur * buf_bytes;
            int32_t t = 0;
            if (RPL == 1)
                for (; t + 4 <= cnt; t += 4)
                    add_leaves<NF, 4, RPL>(first + t * R.bytes, R, depth, xf, kv, bs, xe, acc);
            for (; t + 2 <= cnt; t += 2)
                add_leaves<NF, 2, RPL>(first + t * R.bytes, R, depth, xf, kv, bs, xe, acc);
            if (t < cnt) add_leaves<NF, 1, RPL>(first + t * R.bytes, R, depth, xf, kv, bs, xe, acc);
        }
        stage_release(sync, b, kColWaves);
    }
#pragma unroll
    for (int r = 0; r < RPL; ++r)
        if (o[r] >= 0) P.out[o[r]] = sync_ok ? acc[r] : __builtin_nanf("");
}

// Leaf reuse along a lane's RPL consecutive rows with two anchors: every lane
// walks its first and last row through NT (1 or 2) consecutive staged trees in
// one interleaved pass (full wavefronts), keeps those leaves' values and KV /
// batch boxes, and gives every row in between the value of an anchor leaf
// whose box holds it (the frequency and engine size are the scenario's, so a
// row inside a leaf's box reaches that leaf), or of the leaf of the lane's
// last walk in between.  Only rows in none of these boxes walk, the trees
// they need, both in one pass when the wavefront needs both.
template <int NF, int NT, int RPL>
__device__ __forceinline__ void add_leaves_anchored(uint32_t tree, const RecordLayout& R, int32_t depth, float xf,
                                                    const float (&kv)[RPL], const float (&bs)[RPL], float xe,
                                                    float (&acc)[RPL]) {
    float va[2][NT];
    float4 ba[2][NT];
    {
        const float xfa[2] = {xf, xf}, kva[2] = {kv[0], kv[RPL - 1]}, bsa[2] = {bs[0], bs[RPL - 1]},
                    xea[2] = {xe, xe};
        LeafAt ka[2][NT];
        walk_rows<NF, NT, 2>(tree, R, depth, xfa, kva, bsa, xea, ka);
#pragma unroll
        for (int e = 0; e < 2; ++e)
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                va[e][t] = leaf_value(ka[e][t]);
                ba[e][t] = leaf_box(ka[e][t]);
            }
    }
    float vl[NT];
    float4 bl[NT];   // the last walk's leaf (none yet: empty box)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        vl[t] = 0.0f;
        bl[t] = make_float4(INFINITY, -INFINITY, INFINITY, -INFINITY);
    }
#pragma unroll
    for (int r = 0; r < RPL; ++r) {
        float v[NT];
        if (r == 0 || r == RPL - 1) {
#pragma unroll
            for (int t = 0; t < NT; ++t) v[t] = va[r == 0 ? 0 : 1][t];
        } else {
            bool need[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const bool in0 = in_box(ba[0][t], kv[r], bs[r]);
                const bool in1 = in_box(ba[1][t], kv[r], bs[r]);
                need[t] = !in0 && !in1 && !in_box(bl[t], kv[r], bs[r]);
                v[t] = in0 ? va[0][t] : (in1 ? va[1][t] : vl[t]);
            }
            if (NT == 2 && __builtin_amdgcn_ballot_w64(need[0]) != 0 &&
                __builtin_amdgcn_ballot_w64(need[NT - 1]) != 0) {
                LeafAt k[NT];
                walk<NF, NT>(tree, R, depth, xf, kv[r], bs[r], xe, k);
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    if (need[t]) {
                        v[t] = vl[t] = leaf_value(k[t]);
                        bl[t] = leaf_box(k[t]);
                    }
            } else {
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    if (need[t]) {
                        LeafAt k[1];
                        walk<NF, 1>(tree + t * R.bytes, R, depth, xf, kv[r], bs[r], xe, k);
                        v[t] = vl[t] = leaf_value(k[0]);
                        bl[t] = leaf_box(k[0]);
                    }
            }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[r] += v[t];
        asm volatile("" ::"v"(acc[r]));
    }
}

// M at one frequency per scenario with leaf reuse along each lane's RPL
// consecutive iterations (a wavefront takes 64 x RPL consecutive
// iterations of one scenario); staging as in forest_column_lds_kernel.
// LIVE: the items are the first *P.n_live entries of P.order.
template <int NF, int RPL, bool LIVE>
__global__ __launch_bounds__(kColThreads) void forest_column_reuse_kernel(const uint4* __restrict__ records,
                                                                         int32_t n_trees, int32_t depth,
                                                                         int32_t tb, float base, ColumnParams P) {
    extern __shared__ __align__(16) unsigned char smem[];
    const RecordLayout R = record_layout(depth);
    const uint32_t rec_words = R.bytes / 16u;
    const uint32_t buf_bytes = stage_buffer_bytes(tb, R);
    const int wave = threadIdx.x / kWave;
    const int64_t item = __builtin_amdgcn_readfirstlane((int64_t)blockIdx.x * kColWaves + wave);
    const int32_t span = kWave * RPL;
    const int32_t n_cols = (P.H + span - 1) / span;
    const int64_t n_items = LIVE ? (int64_t)*P.n_live : P.S * n_cols;
    // a workgroup wholly past the live items has nothing to stage for
    if (LIVE && (int64_t)blockIdx.x * kColWaves >= n_items) return;
    bool valid = item < n_items;
    // the (scenario, column) pair: item itself, or its entry of the work order
    const int64_t code = !valid ? 0 : P.order ? (int64_t)P.order[item] : item;
    const int64_t s = code / n_cols;
    if (P.fidx && P.fidx[s] < 0) valid = false;
    const int32_t j0 = (int32_t)(code % n_cols) * span + lane_id() * RPL;
    const float xf = column_freq(P, s);
    const float xe = NF == 4 ? P.engine[s] : 0.0f;
    float kv[RPL], bs[RPL];
    float acc[RPL];
#pragma unroll
    for (int r = 0; r < RPL; ++r) {
        const int32_t j = min(j0 + r, P.H - 1);
        kv[r] = (float)P.kv[s * P.H + j];
        bs[r] = (float)P.batch[s * P.H + j];
        acc[r] = base;
        asm volatile("" ::"v"(kv[r]), "v"(bs[r]));
    }
    asm volatile("" ::"v"(xf), "v"(xe));
    const int32_t n_blocks = (n_trees + tb - 1) / tb;
    StageSync* sync = (StageSync*)(smem + 2 * buf_bytes);
    if (threadIdx.x == 0) stage_sync_init(sync);
    if (n_blocks > 0) stage_block(records, n_trees, tb, rec_words, 0, lds_addr(smem), wave, kColWaves);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    bool sync_ok = true;
    for (int32_t b = 0; b < n_blocks; ++b) {
        const int cur = b & 1;
        if (b > 0)
            sync_ok &= stage_acquire(sync, b, kColWaves, records, n_trees, tb, rec_words,
                                     lds_addr(smem) + cur * buf_bytes);
        if (valid) {
            const int32_t cnt = min(tb, n_trees - b * tb);
            const uint32_t first = lds_addr(smem) + cur * buf_bytes;
            int32_t t = 0;
            for (; t + 2 <= cnt; t += 2)
                add_leaves_anchored<NF, 2, RPL>(first + t * R.bytes, R, depth, xf, kv, bs, xe, acc);
            if (t < cnt) add_leaves_anchored<NF, 1, RPL>(first + t * R.bytes, R, depth, xf, kv, bs, xe, acc);
        }
        stage_release(sync, b, kColWaves);
    }
    if (valid) {
#pragma unroll
        for (int r = 0; r < RPL; ++r)
            if (j0 + r < P.H) P.out[s * P.H + j0 + r] = sync_ok ? acc[r] : __builtin_nanf("");
    }
}

// Global-memory walks for forests without LDS records.
template <int NF>
__global__ __launch_bounds__(256) void forest_column_global_kernel(const uint2* __restrict__ nodes,
                                                                  const float* __restrict__ leaves,
                                                                  int32_t n_trees, int32_t depth, float base,
                                                                  ColumnParams P) {
    const int64_t item = (int64_t)blockIdx.x * (256 / kWave) + threadIdx.x / kWave;
    const ColumnItem<1> c = column_item<1>(P, item);
    if (!c.row[0]) return;
    float x[4];
    x[0] = column_freq(P, c.s);
    x[1] = (float)P.kv[c.s * P.H + c.j[0]];
    x[2] = (float)P.batch[c.s * P.H + c.j[0]];
    x[3] = NF == 4 ? P.engine[c.s] : 0.0f;
    const int64_t stride = (int64_t)1 << depth;
    const int32_t n_int = (1 << depth) - 1;
    float acc = base;
    for (int32_t t = 0; t < n_trees; ++t) {
        const uint2* nd = nodes + t * stride;
        int32_t k = 0;
        for (int32_t level = 0; level < depth; ++level) {
            const uint2 w = nd[k];
            const float v = x[w.y & 3u];
            k = 2 * k + (v < __uint_as_float(w.x) ? 1 : 2);
        }
        acc += leaves[t * stride + (k - n_int)];
    }
    P.out[c.s * P.H + c.j[0]] = acc;
}

// Trees per staged block: double buffers within the LDS budget.
int32_t column_trees_per_block(const ForestDev& f, size_t* lds) {
    if (!f.records || f.n_trees == 0) return 0;
    const RecordLayout R = record_layout(f.depth);
    // two tree buffers and their hand-over counters
    auto bytes = [&](int32_t n) { return 2 * (size_t)stage_buffer_bytes(n, R) + sizeof(StageSync); };
    int32_t tb = std::min<int32_t>(f.n_trees, 64);
    while (tb > 1 && bytes(tb) > kColLdsBudget) --tb;
    if (bytes(tb) > kColLdsBudget) return 0;
    *lds = bytes(tb);
    return tb;
}

template <int NF, int RPL, bool ROWS = false>
hipError_t launch_column_lds(const ForestDev& f, const ColumnParams& c, int32_t tb, size_t lds, hipStream_t stream) {
    const int64_t span = kWave * RPL;
    const int64_t items = ROWS ? (c.n_rows + span - 1) / span : c.S * ((c.H + span - 1) / span);
    if (!grid_fits((items + kColWaves - 1) / kColWaves)) return hipErrorInvalidConfiguration;
    const auto kern = forest_column_lds_kernel<NF, RPL, ROWS>;
    const hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)((items + kColWaves - 1) / kColWaves)), dim3(kColThreads), lds, stream,
                       f.records, f.n_trees, f.depth, tb, f.base_score, c);
    return hipGetLastError();
}

// Estimated cost of each (scenario, column) pair of the leaf-reuse kernel,
// for its work order.  A row is taken to need a walk when its cell of the
// KV / batch cut grid (the forest's threshold cuts) differs from the cells of
// its lane's two anchors and of the lane's last walked row; the kernel pays
// one walk time per row position at which any lane of the wavefront walks.
// cost = (those positions << 10) | (walks over all lanes, at most 64 x 14);
// with many trees nearly every position has a walk, and the second term,
// how fast the column's rows change, decides the order.
// One wavefront per pair; the cuts sit in LDS.  Writes cost[i] and the pair
// code i = s * n_cols + col.
constexpr int kColCostWaves = 4;

__global__ __launch_bounds__(kColCostWaves* kWave) void column_cost_kernel(
    const float* __restrict__ cuts_kv, int32_t n_kv, const float* __restrict__ cuts_bs, int32_t n_bs,
    const int32_t* __restrict__ kv, const int32_t* __restrict__ batch, int64_t S, int32_t H, int32_t rpl,
    uint32_t* __restrict__ cost, uint32_t* __restrict__ code) {
    __shared__ float ck[kMaxCuts], cb[kMaxCuts];
    for (int32_t i = threadIdx.x; i < n_kv; i += kColCostWaves * kWave) ck[i] = cuts_kv[i];
    for (int32_t i = threadIdx.x; i < n_bs; i += kColCostWaves * kWave) cb[i] = cuts_bs[i];
    __syncthreads();
    const int32_t span = kWave * rpl;
    const int32_t n_cols = (H + span - 1) / span;
    const int64_t pair = (int64_t)blockIdx.x * kColCostWaves + threadIdx.x / kWave;
    if (pair >= S * n_cols) return;
    const int64_t s = pair / n_cols;
    const int32_t j0 = (int32_t)(pair % n_cols) * span + lane_id() * rpl;
    // number of cuts <= x
    auto rank = [](const float* c, int32_t n, float x) {
        int32_t lo = 0, hi = n;
        while (lo < hi) {
            const int32_t mid = (lo + hi) >> 1;
            if (c[mid] <= x) lo = mid + 1;
            else hi = mid;
        }
        return (uint32_t)lo;
    };
    // the cell of the lane's row r (rows past the horizon repeat the last, as
    // in the kernel)
    auto cell = [&](int32_t r) {
        const int64_t i = s * H + min(j0 + r, H - 1);
        return rank(ck, n_kv, (float)kv[i]) << 16 | rank(cb, n_bs, (float)batch[i]);
    };
    const uint32_t a0 = cell(0), a1 = cell(rpl - 1);
    uint32_t last = a0, positions = 0, walks = 0;
    for (int32_t r = 1; r < rpl - 1; ++r) {
        const uint32_t c = cell(r);
        const bool need = c != a0 && c != a1 && c != last;
        if (need) last = c;
        const uint64_t lanes = __builtin_amdgcn_ballot_w64(need);
        positions += lanes != 0;
        walks += (uint32_t)__builtin_popcountll(lanes);
    }
    if (lane_id() == 0) {
        cost[pair] = positions << 10 | walks;
        code[pair] = (uint32_t)pair;
    }
}

// Rows per lane of the leaf-reuse kernel for these rows: 16 (else 8) where
// the horizon fills a wavefront's 64 x RPL rows and the grid still gives
// every CU a workgroup; 0 when the kernel does not apply.  *cus: the
// device's CUs.
hipError_t reuse_rows_per_lane(const ForestDev& f, const ColumnParams& c, int* rpl, int* cus) {
    *rpl = 0;
    size_t lds = 0;
    if (c.rows || column_trees_per_block(f, &lds) <= 0) return hipSuccess;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    for (int r : {16, 8}) {
        const int64_t items = c.S * ((c.H + kWave * r - 1) / (kWave * r));
        if (c.H >= kWave * r && items >= (int64_t)kColWaves * *cus) {
            *rpl = r;
            break;
        }
    }
    return hipSuccess;
}

template <int NF, int RPL>
hipError_t launch_column_reuse(const ForestDev& f, const ColumnParams& c, int32_t tb, size_t lds,
                               hipStream_t stream) {
    const int64_t items = c.S * ((c.H + kWave * RPL - 1) / (kWave * RPL));
    if (!grid_fits((items + kColWaves - 1) / kColWaves)) return hipErrorInvalidConfiguration;
    const auto kern =
        c.n_live ? forest_column_reuse_kernel<NF, RPL, true> : forest_column_reuse_kernel<NF, RPL, false>;
    const hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)((items + kColWaves - 1) / kColWaves)), dim3(kColThreads), lds, stream,
                       f.records, f.n_trees, f.depth, tb, f.base_score, c);
    return hipGetLastError();
}

template <int NF>
hipError_t launch_column(const ForestDev& f, const ColumnParams& c, hipStream_t stream) {
    size_t lds = 0;
    const int32_t tb = column_trees_per_block(f, &lds);
    if (tb > 0) {
        int rpl = 0, cus = 0;
        const hipError_t e = reuse_rows_per_lane(f, c, &rpl, &cus);
        if (e != hipSuccess) return e;
        if (rpl == 16) return launch_column_reuse<NF, 16>(f, c, tb, lds, stream);
        if (rpl == 8) return launch_column_reuse<NF, 8>(f, c, tb, lds, stream);
    }
    if (tb > 0) {
        // rows per lane: enough chains to overlap, without idle stripes on
        // short horizons
        if (c.H > 2 * kWave) return launch_column_lds<NF, 4>(f, c, tb, lds, stream);
        if (c.H > kWave) return launch_column_lds<NF, 2>(f, c, tb, lds, stream);
        return launch_column_lds<NF, 1>(f, c, tb, lds, stream);
    }
    const int64_t items = c.S * ((c.H + kWave - 1) / kWave);
    if (!grid_fits((items + 3) / 4)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(forest_column_global_kernel<NF>, dim3((unsigned)((items + 3) / 4)), dim3(256), 0, stream,
                       f.nodes, f.leaves, f.n_trees, f.depth, f.base_score, c);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_forest_column(const ForestDev& f, const ColumnParams& c, hipStream_t stream) {
    if (c.S == 0) return hipSuccess;
    return f.n_features == 4 ? launch_column<4>(f, c, stream) : launch_column<3>(f, c, stream);
}

namespace {

__global__ void column_live_clear_kernel(int32_t* n_live) { *n_live = 0; }

// The live items of the leaf-reuse kernel: entry i of the work order (or
// item i) is kept when its scenario is selected (fidx >= 0); a wavefront's
// kept entries stay in order and take consecutive slots from one atomic add.
__global__ __launch_bounds__(256) void column_live_kernel(const uint32_t* __restrict__ order,
                                                          const int32_t* __restrict__ fidx, int64_t n_items,
                                                          int32_t n_cols, uint32_t* __restrict__ live,
                                                          int32_t* __restrict__ n_live) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    uint32_t code = 0;
    bool keep = false;
    if (i < n_items) {
        code = order ? order[i] : (uint32_t)i;
        keep = fidx[code / (uint32_t)n_cols] >= 0;
    }
    const uint64_t m = __builtin_amdgcn_ballot_w64(keep);
    if (m == 0) return;
    int32_t base = 0;
    if (lane_id() == 0) base = atomicAdd(n_live, (int32_t)__builtin_popcountll(m));
    base = __shfl(base, 0);
    const uint32_t below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    if (keep) live[base + (int32_t)below] = code;
}

// The leaf-reuse kernel's work order for c's rows (p.n = 0: none).  It is
// only planned for grids of at least two workgroups per CU: with one, the
// kernel takes as long as its slowest wavefront whatever the order.
hipError_t plan_column_order(const ForestDev& f, const ColumnParams& c, int* rpl, PairOrderPlan* p) {
    *p = PairOrderPlan{0, 0, 0, 0};
    if (c.S == 0) return hipSuccess;
    int cus = 0;
    const hipError_t e = reuse_rows_per_lane(f, c, rpl, &cus);
    if (e != hipSuccess || *rpl == 0) return e;
    const int64_t span = kWave * *rpl;
    const int64_t items = c.S * ((c.H + span - 1) / span);
    return pair_order_plan(f, items, 2 * (int64_t)kColWaves * cus, p);
}

}  // namespace

hipError_t column_order_bytes(const ForestDev& f, const ColumnParams& c, size_t* bytes) {
    int rpl = 0;
    PairOrderPlan p;
    const hipError_t e = plan_column_order(f, c, &rpl, &p);
    *bytes = e == hipSuccess ? p.bytes : 0;
    return e;
}

hipError_t order_forest_column(const ForestDev& f, ColumnParams& c, void* ws, hipStream_t stream) {
    int rpl = 0;
    PairOrderPlan p;
    hipError_t e = plan_column_order(f, c, &rpl, &p);
    if (e != hipSuccess || p.n == 0) return e;
    hipLaunchKernelGGL(column_cost_kernel, dim3((unsigned)((p.n + kColCostWaves - 1) / kColCostWaves)),
                       dim3(kColCostWaves * kWave), 0, stream, f.cuts_kv, f.n_cuts_kv, f.cuts_bs, f.n_cuts_bs, c.kv,
                       c.batch, c.S, c.H, rpl, pair_order_cost(p, ws), pair_order_code(p, ws));
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return pair_order_sort(p, ws, &c.order, stream);
}

hipError_t column_live_bytes(const ForestDev& f, const ColumnParams& c, size_t* bytes) {
    *bytes = 0;
    int rpl = 0, cus = 0;
    if (c.S == 0 || !c.fidx) return hipSuccess;
    const hipError_t e = reuse_rows_per_lane(f, c, &rpl, &cus);
    if (e != hipSuccess || rpl == 0) return e;
    const int64_t span = kWave * rpl;
    const int64_t items = c.S * ((c.H + span - 1) / span);
    // as for the work order: with one workgroup per CU the launch lasts as
    // long as its slowest workgroup, compacted or not
    if (items < 2 * (int64_t)kColWaves * cus) return hipSuccess;
    *bytes = (((size_t)items * sizeof(uint32_t) + 255) & ~(size_t)255) + 256;
    return hipSuccess;
}

hipError_t launch_forest_column_live(const ForestDev& f, const ColumnParams& c, void* ws, hipStream_t stream) {
    int rpl = 0, cus = 0;
    hipError_t e = hipSuccess;
    if (ws && c.fidx && c.S > 0) e = reuse_rows_per_lane(f, c, &rpl, &cus);
    if (e != hipSuccess) return e;
    if (rpl == 0) return launch_forest_column(f, c, stream);
    const int32_t span = kWave * rpl;
    const int32_t n_cols = (c.H + span - 1) / span;
    const int64_t items = c.S * n_cols;
    uint32_t* live = (uint32_t*)ws;
    int32_t* n_live = (int32_t*)((unsigned char*)ws + (((size_t)items * sizeof(uint32_t) + 255) & ~(size_t)255));
    hipLaunchKernelGGL(column_live_clear_kernel, dim3(1), dim3(1), 0, stream, n_live);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (!grid_fits((items + 255) / 256)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(column_live_kernel, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, stream, c.order,
                       c.fidx, items, n_cols, live, n_live);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    ColumnParams d = c;
    d.order = live;
    d.n_live = n_live;
    return launch_forest_column(f, d, stream);
}

hipError_t launch_forest_rows_lds(const ForestDev& f, const float* rows, int64_t n_rows, float* out,
                                  hipStream_t stream) {
    size_t lds = 0;
    const int32_t tb = (f.n_features == 3 || f.n_features == 4) ? column_trees_per_block(f, &lds) : 0;
    if (tb <= 0) return hipErrorNotSupported;
    if (n_rows == 0) return hipSuccess;
    ColumnParams c{};
    c.rows = rows;
    c.n_rows = n_rows;
    c.out = out;
    return f.n_features == 4 ? launch_column_lds<4, 4, true>(f, c, tb, lds, stream)
                             : launch_column_lds<3, 4, true>(f, c, tb, lds, stream);
}

}  // namespace tl
