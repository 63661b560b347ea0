// Stage 2: the performance model M (Sec. 4.3.1), a gradient-boosted tree
// ensemble, evaluated on fp32 feature rows.  Every kernel here computes, for
// each row, base + the leaf of every tree as an fp32 running sum in tree
// order (every add rounded to nearest even).
//
// Grid kernels evaluate the rows of the projection grid without
// materializing them: row (s, f, j) = (freq[f], kv[s][j], batch[s][j]
// [, engine[s]]).  One wavefront takes one scenario and J consecutive future
// iterations; its lanes are the candidate frequencies, so every lane sees the
// same (KV, batch) sequence.  For each tree (in order) a lane keeps the leaf
// reached by its previous row together with the KV / batch box of that leaf
// (the bounds its root-to-leaf path puts on those two features); the next row
// reuses the leaf while its (KV, batch) stays inside the box.  This is exact:
// frequency and engine size are fixed for the lane, so a row inside the box
// takes every decision of the path the same way.  Between consecutive future
// iterations KV and batch move little, so most rows cost a box test and one
// fp32 add per tree; a walk happens on roughly one row in twenty.
//
//   forest_grid_lds_kernel     (depth <= 11) A 1024-thread workgroup (16
//       wavefronts, 16 x 64 x 64 rows) walks the ensemble in blocks of trees
//       staged in three LDS buffers.  A tree is one record (nodes, leaf values,
//       leaf boxes), so a block is one contiguous copy, made straight from
//       global memory into LDS and handed from wavefront to wavefront without
//       block barriers (stage_acquire / stage_release).  Tree walks read LDS
//       only.  A node step picks the tested feature with byte permutes and
//       compares once, all in vector registers (no lane-mask round trip).
//       Trees are taken in pairs that share one box test (a row that leaves
//       it walks only the tree whose own box it left), and rows in groups of
//       eight whose (KV, batch) hull is tested before any single row.  The
//       (scenario, chunk) items are ordered by an estimate of their walks,
//       so a workgroup's wavefronts do similar work.
//   forest_grid_global_kernel  (deeper trees) The same per-lane scheme with
//       nodes, leaves and boxes read from global memory, one row at a time.
//
// Device layout (built by tl_forest_create): nodes [T][2^d] (8 bytes:
// threshold bits, feature; the last entry of each tree is padding), leaves
// [T][2^d] fp32, and for 3-4 features the leaf boxes [T][2^d] (kv_lo, kv_hi,
// batch_lo, batch_hi) and, up to depth 11, the tree records of the LDS
// kernel.
//
// forest_rows_kernel evaluates arbitrary rows: each thread walks RPT
// consecutive rows through every tree (forests without LDS records; the
// others take the column kernel's staged walks).
#include <hipcub/hipcub.hpp>

#include <mutex>

#include "device_util.h"
#include "tl_internal.h"
#include "forest_walk.h"

namespace tl {
namespace {

template <int NF>
__device__ __forceinline__ float pick(const float (&x)[4], uint32_t f) {
    if (NF == 1) return x[0];
    if (NF == 2) return f == 0 ? x[0] : x[1];
    if (NF == 3) return f == 0 ? x[0] : (f == 1 ? x[1] : x[2]);
    return f == 0 ? x[0] : (f == 1 ? x[1] : (f == 2 ? x[2] : x[3]));
}

// grid row features: 0 frequency, 1 KV, 2 batch, 3 engine size
template <int NF>
__device__ __forceinline__ float pick_grid(uint32_t ft, float xf, float kv, float bs, float xe) {
    if (NF == 3) return ft == 0 ? xf : (ft == 1 ? kv : bs);
    return ft == 0 ? xf : (ft == 1 ? kv : (ft == 2 ? bs : xe));
}

template <int NF, int RPT>
__global__ __launch_bounds__(256) void forest_rows_kernel(const uint2* __restrict__ nodes,
                                                          const float* __restrict__ leaves,
                                                          int32_t n_trees, int32_t depth, float base,
                                                          const float* __restrict__ rows, int64_t n_rows,
                                                          float* __restrict__ out) {
    const int64_t r0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * RPT;
    if (r0 >= n_rows) return;
    const int nr = (int)min((int64_t)RPT, n_rows - r0);
    float x[RPT][4];
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
#pragma unroll
        for (int c = 0; c < 4; ++c) x[r][c] = 0.0f;
        if (r < nr) {
#pragma unroll
            for (int c = 0; c < NF; ++c) x[r][c] = rows[(r0 + r) * NF + c];
        }
    }
    float acc[RPT];
#pragma unroll
    for (int r = 0; r < RPT; ++r) acc[r] = base;
    const int32_t n_int = (1 << depth) - 1;
    const int32_t n_leaf = 1 << depth;
    for (int32_t t = 0; t < n_trees; ++t) {
        const uint2* nt = nodes + (int64_t)t * n_leaf;
        const float* lt = leaves + (int64_t)t * n_leaf;
        int32_t k[RPT];
#pragma unroll
        for (int r = 0; r < RPT; ++r) k[r] = 0;
        for (int32_t level = 0; level < depth; ++level) {
#pragma unroll
            for (int r = 0; r < RPT; ++r) {
                const uint2 nd = nt[k[r]];
                const float v = pick<NF>(x[r], nd.y);
                k[r] = 2 * k[r] + ((v < __uint_as_float(nd.x)) ? 1 : 2);
            }
        }
#pragma unroll
        for (int r = 0; r < RPT; ++r) acc[r] += lt[k[r] - n_int];
    }
#pragma unroll
    for (int r = 0; r < RPT; ++r)
        if (r < nr) out[r0 + r] = acc[r];
}

#ifndef TL_LDS_J
#define TL_LDS_J 64
#endif
#ifndef TL_LDS_WAVES
#define TL_LDS_WAVES 16
#endif
#ifndef TL_LDS_BUDGET_KIB
#define TL_LDS_BUDGET_KIB 160
#endif
// Tree buffers: three blocks of 2 trees at depth 10 (against two of 3) let a
// wavefront run two blocks ahead of the slowest and pair every tree.
constexpr int kLdsBuffers = 3;
#ifndef TL_LDS_WAVES_PER_SIMD
#define TL_LDS_WAVES_PER_SIMD 4
#endif
constexpr int kLdsJ = TL_LDS_J;          // future iterations per wavefront (LDS kernel)
constexpr int kGlobalJ = 32;             // future iterations per wavefront (global kernel)

// Which (scenario, frequency group, iteration chunk) a wavefront evaluates.
struct GridItem {
    bool valid;
    int64_t s;
    int32_t f, j0, nj;
};

// Items are numbered scenario-fastest: the wavefronts of one workgroup take
// the same iteration chunk (and frequency group) of consecutive scenarios.
// How many walks a chunk needs follows how fast KV and batch change there;
// workgroups whose wavefronts do similar work lose less time waiting for
// their slowest wavefront to release a tree buffer.  With a work order
// (P.order), item i of a frequency group takes
// the (scenario, chunk) pair order[i] instead: pairs sorted by estimated
// cost, most expensive first.
__device__ __forceinline__ GridItem grid_item(const GridParams& P, int64_t item, int J) {
    const int32_t n_chunks = (P.H + J - 1) / J;
    const int32_t n_fg = (P.F + kWave - 1) / kWave;
    GridItem g;
    g.valid = item < P.S * n_fg * n_chunks;
    const int64_t it = g.valid ? item : 0;
    const int64_t n_pairs = P.S * n_chunks;
    int32_t chunk;
    if (P.order) {
        const uint32_t code = P.order[it % n_pairs];
        g.s = code / (uint32_t)n_chunks;
        chunk = (int32_t)(code % (uint32_t)n_chunks);
        g.f = (int32_t)(it / n_pairs) * kWave + lane_id();
    } else {
        g.s = it % P.S;
        const int64_t rest = it / P.S;
        g.f = (int32_t)(rest % n_fg) * kWave + lane_id();
        chunk = (int32_t)(rest / n_fg);
    }
    g.j0 = chunk * J;
    g.nj = min(J, P.H - g.j0);
    return g;
}

// Estimated cost of each (scenario, chunk) pair of the grid: how many KV and
// batch threshold cuts its rows cross from one row to the next (each crossing
// may change a leaf, i.e. cost a walk).  One thread per pair; the cuts sit in
// LDS.  Writes cost[i] and the pair code i = s * n_chunks + chunk.
constexpr int kCostThreads = 256;

__global__ __launch_bounds__(kCostThreads) void grid_cost_kernel(const float* __restrict__ cuts_kv, int32_t n_kv,
                                                                 const float* __restrict__ cuts_bs, int32_t n_bs,
                                                                 const int32_t* __restrict__ kv,
                                                                 const int32_t* __restrict__ batch, int64_t S,
                                                                 int32_t H, int32_t J, uint32_t* __restrict__ cost,
                                                                 uint32_t* __restrict__ code) {
    __shared__ float ck[kMaxCuts], cb[kMaxCuts];
    for (int32_t i = threadIdx.x; i < n_kv; i += kCostThreads) ck[i] = cuts_kv[i];
    for (int32_t i = threadIdx.x; i < n_bs; i += kCostThreads) cb[i] = cuts_bs[i];
    __syncthreads();
    const int32_t n_chunks = (H + J - 1) / J;
    const int64_t i = (int64_t)blockIdx.x * kCostThreads + threadIdx.x;
    if (i >= S * n_chunks) return;
    const int64_t s = i / n_chunks;
    const int32_t j0 = (int32_t)(i % n_chunks) * J, j1 = min(j0 + J, H);
    // number of cuts <= x
    auto rank = [](const float* c, int32_t n, float x) {
        int32_t lo = 0, hi = n;
        while (lo < hi) {
            const int32_t mid = (lo + hi) >> 1;
            if (c[mid] <= x) lo = mid + 1;
            else hi = mid;
        }
        return lo;
    };
    int32_t rk = rank(ck, n_kv, (float)kv[s * H + j0]), rb = rank(cb, n_bs, (float)batch[s * H + j0]);
    uint32_t c = 0;
    for (int32_t j = j0 + 1; j < j1; ++j) {
        const int32_t nk = rank(ck, n_kv, (float)kv[s * H + j]), nb = rank(cb, n_bs, (float)batch[s * H + j]);
        c += (uint32_t)(abs(nk - rk) + abs(nb - rb));
        rk = nk;
        rb = nb;
    }
    cost[i] = c;
    code[i] = (uint32_t)i;
}

// ---------------------------------------------------------------- LDS-staged

constexpr int kLdsWaves = TL_LDS_WAVES;  // wavefronts per workgroup
constexpr int kLdsThreads = kLdsWaves * kWave;
// A wavefront-uniform value read into a scalar register: the compiler's lane
// read, with the empty asm statements hiding how x was computed and pinning
// the result to the scalar register file (the compiler would otherwise
// rematerialize it in vector registers).
__device__ __forceinline__ float to_sgpr(float x) {
    asm volatile("" : "+v"(x));
    int32_t r = __builtin_amdgcn_readfirstlane(__float_as_int(x));
    asm volatile("" : "+s"(r));
    return __int_as_float(r);
}

#ifndef TL_ROW_GROUP
#define TL_ROW_GROUP 8
#endif
constexpr int kRowGroup = TL_ROW_GROUP;   // rows whose (KV, batch) hull is tested as one

// Adds the leaves of NT (1 or 2) consecutive staged trees (records R.bytes
// apart, the first at `tree`) to the J row sums of a wavefront, in tree
// order.  hull[g] = (min KV, max KV, min batch, max batch) over the rows of
// group g; kv4 holds the rows' (KV, batch) pairs, two per 16 bytes.  A lane
// keeps the values of the leaves its walks reached, their boxes and the
// intersection of the boxes.  A group whose hull lies inside that
// intersection on every lane needs only its adds; other groups test row by
// row.  A lane whose row leaves the intersection walks only the trees whose
// own box it left (both in one pass when the wavefront needs both) and reads
// the new leaves' values and boxes.
template <int NF, int J, int NT>
__device__ __forceinline__ void eval_trees(const unsigned char* lds, uint32_t tree_off, const RecordLayout& R,
                                           int32_t depth,
                                           const float4* kv4, const float (&hull)[J / kRowGroup][4], float xf,
                                           float xe, float (&acc)[J]) {
    static_assert(J % kRowGroup == 0, "whole row groups");
    static_assert(NT == 1 || NT == 2, "one tree or a pair");
    // the pairs are re-read from LDS for each group that needs them rather
    // than held in registers across the tree loop
    asm volatile("" ::: "memory");
    const unsigned char* tree = lds + tree_off;
    const uint32_t tree_addr = lds_addr(tree);
    const uint32_t tree1 = tree_addr + R.bytes;
    // a pair's own leaf boxes, decoded, beside their intersection: after a
    // walk only the walked tree's box is read again
    float4 box, b0, b1 = make_float4(INFINITY, -INFINITY, INFINITY, -INFINITY);
    float v[NT];
    {
        // the chunk's first row walks every tree on every lane, outside the
        // group loop so that the loop's walks carry no first-row case
        const float4 q0 = kv4[0];
        LeafAt k[NT];
        walk<NF, NT>(tree_addr, R, depth, xf, q0.x, q0.y, xe, k);
        v[0] = leaf_value(k[0]);
        b0 = leaf_box(k[0]);
        box = b0;
        if (NT == 2) {
            v[NT - 1] = leaf_value(k[NT - 1]);
            b1 = leaf_box(k[NT - 1]);
            box = box_meet(b0, b1);
        }
    }
#pragma unroll
    for (int gi = 0; gi < J / kRowGroup; ++gi) {
        const uint64_t inside = __builtin_amdgcn_fcmpf(hull[gi][0], box.x, 3) &   // min KV >= kv_lo
                                __builtin_amdgcn_fcmpf(hull[gi][1], box.y, 4) &   // max KV < kv_hi
                                __builtin_amdgcn_fcmpf(hull[gi][2], box.z, 3) &
                                __builtin_amdgcn_fcmpf(hull[gi][3], box.w, 4);
        const bool test_rows = inside != __builtin_amdgcn_read_exec();   // wavefront-uniform
        float4 q = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
        for (int i = 0; i < kRowGroup; ++i) {
            if (test_rows) {
                if ((i & 1) == 0) {
                    // two rows per read; the barrier keeps the compiler from
                    // hoisting all reads of the group (registers)
                    asm volatile("" ::: "memory");
                    q = kv4[gi * (kRowGroup / 2) + i / 2];
                }
                const float kv = (i & 1) ? q.z : q.x;
                const float bs = (i & 1) ? q.w : q.y;
                if (!in_box(box, kv, bs)) {
                    if (NT == 1) {
                        LeafAt k[1];
                        walk<NF, 1>(tree_addr, R, depth, xf, kv, bs, xe, k);
                        v[0] = leaf_value(k[0]);
                        box = leaf_box(k[0]);
                    } else {
                        const bool n0 = !in_box(b0, kv, bs);
                        const bool n1 = !in_box(b1, kv, bs);
                        if (__builtin_amdgcn_ballot_w64(n0) != 0 && __builtin_amdgcn_ballot_w64(n1) != 0) {
                            LeafAt k[2];
                            walk<NF, 2>(tree_addr, R, depth, xf, kv, bs, xe, k);
                            if (n0) {
                                v[0] = leaf_value(k[0]);
                                b0 = leaf_box(k[0]);
                            }
                            if (n1) {
                                v[NT - 1] = leaf_value(k[1]);
                                b1 = leaf_box(k[1]);
                            }
                        } else {
                            if (n0) {
                                LeafAt k[1];
                                walk<NF, 1>(tree_addr, R, depth, xf, kv, bs, xe, k);
                                v[0] = leaf_value(k[0]);
                                b0 = leaf_box(k[0]);
                            }
                            if (n1) {
                                LeafAt k[1];
                                walk<NF, 1>(tree1, R, depth, xf, kv, bs, xe, k);
                                v[NT - 1] = leaf_value(k[0]);
                                b1 = leaf_box(k[0]);
                            }
                        }
                        box = box_meet(b0, b1);
                    }
                }
            }
            float& a = acc[gi * kRowGroup + i];
#pragma unroll
            for (int t = 0; t < NT; ++t) a += v[t];
            // consume the sum here so the adds are not sunk past later walks
            // (that would keep leaf values live)
            asm volatile("" ::"v"(a));
        }
    }
}

template <int NF, int J>
__global__ __launch_bounds__(kLdsThreads, TL_LDS_WAVES_PER_SIMD) void forest_grid_lds_kernel(const uint4* __restrict__ records,
                                                                      int32_t n_trees, int32_t depth,
                                                                      int32_t tb, float base, GridParams P) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int32_t n_leaf = 1 << depth;
    const RecordLayout R = record_layout(depth);
    const uint32_t rec_words = R.bytes / 16u;
    const uint32_t buf_bytes = stage_buffer_bytes(tb, R);

    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int64_t item = __builtin_amdgcn_readfirstlane((int64_t)blockIdx.x * kLdsWaves + wave);
    const GridItem g = grid_item(P, item, J);
    const int32_t F = P.F, H = P.H;
    const bool active = g.valid && g.f < F;
    // (a NaN frequency or engine size fails every "x < threshold" test and
    // takes every right turn, as in a plain walk)
    const float xf = P.freqs[g.f < F ? g.f : F - 1];
    const float xe = (NF == 4) ? P.engine[g.s] : 0.0f;
    // the J (KV, batch) pairs of this wavefront are the same for every lane;
    // they sit in LDS after the two tree buffers and are read as broadcasts
    float2* kvb = (float2*)(smem + kLdsBuffers * buf_bytes) + wave * J;
    StageSync* sync = (StageSync*)(smem + kLdsBuffers * buf_bytes + (size_t)kLdsWaves * J * sizeof(float2));
    if (threadIdx.x == 0) stage_sync_init<kLdsBuffers>(sync);
    for (int r = lane; r < J; r += kWave) {
        const int32_t j = g.j0 + min(r, g.nj - 1);
        kvb[r] = make_float2((float)P.kv[g.s * H + j], (float)P.batch[g.s * H + j]);
    }

    // staging: block 0 by every wavefront before the barrier, the others
    // handed over without barriers (stage_acquire / stage_release)
    const int32_t n_blocks = (n_trees + tb - 1) / tb;
    float acc[J];
#pragma unroll
    for (int jj = 0; jj < J; ++jj) acc[jj] = base;

    // Make the lane's frequency / engine size complete here, before any
    // staging copy is in flight: otherwise the walks inside the loop would
    // each wait for all outstanding copies.
    asm volatile("" ::"v"(xf), "v"(xe));
    if (n_blocks > 0) stage_block(records, n_trees, tb, rec_words, 0, lds_addr(smem), wave, kLdsWaves);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    // per row group, the (KV, batch) hull of its rows (wavefront-uniform)
    const float4* kvb4 = (const float4*)kvb;
    float hull[J / kRowGroup][4];
#pragma unroll
    for (int gi = 0; gi < J / kRowGroup; ++gi) {
        float klo = INFINITY, khi = -INFINITY, blo = INFINITY, bhi = -INFINITY;
#pragma unroll
        for (int i = 0; i < kRowGroup; ++i) {
            const float2 p = kvb[gi * kRowGroup + i];
            klo = fminf(klo, p.x);
            khi = fmaxf(khi, p.x);
            blo = fminf(blo, p.y);
            bhi = fmaxf(bhi, p.y);
        }
        hull[gi][0] = to_sgpr(klo);
        hull[gi][1] = to_sgpr(khi);
        hull[gi][2] = to_sgpr(blo);
        hull[gi][3] = to_sgpr(bhi);
    }
    bool sync_ok = true;
    for (int32_t b = 0; b < n_blocks; ++b) {
        const int cur = b % kLdsBuffers;
        if (b > 0)
            sync_ok &= stage_acquire<kLdsBuffers>(sync, b, kLdsWaves, records, n_trees, tb, rec_words,
                                                  lds_addr(smem + cur * buf_bytes));
        if (g.valid) {
            const int32_t cnt = min(tb, n_trees - b * tb);
            const uint32_t bp = cur * buf_bytes;
            // Trees are taken two at a time and a lane keeps the intersection
            // of the two leaf boxes: a row inside it reaches both leaves
            // again.  When a row leaves it, both trees are walked in one pass,
            // so the two chains of dependent LDS reads overlap.
            int32_t tt = 0;
            for (; tt + 1 < cnt; tt += 2)
                eval_trees<NF, J, 2>(smem, bp + tt * R.bytes, R, depth, kvb4, hull, xf, xe, acc);
            if (tt < cnt) eval_trees<NF, J, 1>(smem, bp + tt * R.bytes, R, depth, kvb4, hull, xf, xe, acc);
        }
        stage_release<kLdsBuffers>(sync, b, kLdsWaves);
    }
    if (active) {
        float* o = P.out + ((int64_t)g.s * F + g.f) * H + g.j0;
#pragma unroll
        for (int jj = 0; jj < J; ++jj)
            if (jj < g.nj) o[jj] = sync_ok ? acc[jj] : __builtin_nanf("");
    }
}

// ------------------------------------------------------------ global memory

constexpr int kGlobalWaves = 4;

template <int NF, int J>
__global__ __launch_bounds__(256) void forest_grid_global_kernel(const uint2* __restrict__ nodes,
                                                                 const float* __restrict__ leaves,
                                                                 const float4* __restrict__ boxes,
                                                                 int32_t n_trees, int32_t depth, float base,
                                                                 GridParams P) {
    __shared__ float2 kvb[kGlobalWaves][J];
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int64_t item = __builtin_amdgcn_readfirstlane((int64_t)blockIdx.x * kGlobalWaves + wave);
    const GridItem g = grid_item(P, item, J);
    const int32_t F = P.F, H = P.H;
    const bool active = g.valid && g.f < F;
    const float xf = P.freqs[g.f < F ? g.f : F - 1];
    const float xe = (NF == 4) ? P.engine[g.s] : 0.0f;
    if (lane < J) {
        const int32_t j = g.j0 + min(lane, g.nj - 1);
        kvb[wave][lane] = make_float2((float)P.kv[g.s * H + j], (float)P.batch[g.s * H + j]);
    }
    __syncthreads();
    if (!g.valid) return;

    float acc[J];
#pragma unroll
    for (int jj = 0; jj < J; ++jj) acc[jj] = base;
    const int32_t n_int = (1 << depth) - 1;
    const int32_t n_leaf = 1 << depth;
    for (int32_t t = 0; t < n_trees; ++t) {
        const uint2* nt = nodes + (int64_t)t * n_leaf;
        const float* lv = leaves + (int64_t)t * n_leaf;
        const float4* bx = boxes + (int64_t)t * n_leaf;
        float lo_k = INFINITY, hi_k = -INFINITY, lo_b = INFINITY, hi_b = -INFINITY;
        float val = 0.0f;
#pragma unroll
        for (int jj = 0; jj < J; ++jj) {
            const float2 v2 = kvb[wave][jj];
            const bool hit = (v2.x >= lo_k) & (v2.x < hi_k) & (v2.y >= lo_b) & (v2.y < hi_b);
            if (!hit) {
                int32_t k = 0;
                for (int32_t level = 0; level < depth; ++level) {
                    const uint2 nd = nt[k];
                    const float x = pick_grid<NF>(nd.y, xf, v2.x, v2.y, xe);
                    k = 2 * k + ((x < __uint_as_float(nd.x)) ? 1 : 2);
                }
                const int32_t leaf = k - n_int;
                val = lv[leaf];
                const float4 b = bx[leaf];
                lo_k = b.x;
                hi_k = b.y;
                lo_b = b.z;
                hi_b = b.w;
            }
            acc[jj] += val;
        }
    }
    if (active) {
        float* o = P.out + ((int64_t)g.s * F + g.f) * H + g.j0;
#pragma unroll
        for (int jj = 0; jj < J; ++jj)
            if (jj < g.nj) o[jj] = acc[jj];
    }
}

template <int NF>
hipError_t launch_nf(const ForestDev& f, const float* rows, int64_t n_rows, float* out, hipStream_t stream) {
    constexpr int RPT = 4;
    constexpr int TPB = 256;
    const int64_t threads = (n_rows + RPT - 1) / RPT;
    const int64_t blocks = (threads + TPB - 1) / TPB;
    if (!grid_fits(blocks)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((forest_rows_kernel<NF, RPT>), dim3((unsigned)blocks), dim3(TPB), 0, stream,
                       f.nodes, f.leaves, f.n_trees, f.depth, f.base_score, rows, n_rows, out);
    return hipGetLastError();
}

// Trees per staged block for the LDS kernel: two blocks and the wavefronts'
// (KV, batch) pairs must fit the LDS budget, and one block the staging
// registers.  0 = the LDS kernel cannot run.
int32_t lds_trees_per_block(const ForestDev& f, size_t* lds_bytes) {
    if (!f.records || f.depth > kMaxRecordDepth) return 0;
    const RecordLayout R = record_layout(f.depth);
    const size_t head = (size_t)kLdsWaves * kLdsJ * sizeof(float2) + sizeof(StageSync);
    const size_t budget = (size_t)TL_LDS_BUDGET_KIB * 1024;
    auto fits = [&](int32_t tb) { return kLdsBuffers * (size_t)stage_buffer_bytes(tb, R) + head <= budget; };
    int32_t tb = 64;
    while (tb > 1 && !fits(tb)) --tb;
    if (!fits(tb)) return 0;
    *lds_bytes = kLdsBuffers * (size_t)stage_buffer_bytes(tb, R) + head;
    return tb;
}

template <int NF>
hipError_t launch_grid_lds(const ForestDev& f, const GridParams& g, int32_t tb, size_t lds, hipStream_t stream) {
    const auto kern = forest_grid_lds_kernel<NF, kLdsJ>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    const int64_t n_chunks = (g.H + kLdsJ - 1) / kLdsJ;
    const int64_t n_fg = (g.F + kWave - 1) / kWave;
    const int64_t items = g.S * n_fg * n_chunks;
    const int64_t blocks = (items + kLdsWaves - 1) / kLdsWaves;
    if (!grid_fits(blocks)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kLdsThreads), lds, stream, f.records, f.n_trees,
                       f.depth, tb, f.base_score, g);
    return hipGetLastError();
}

template <int NF>
hipError_t launch_grid_global(const ForestDev& f, const GridParams& g, hipStream_t stream) {
    const int64_t n_chunks = (g.H + kGlobalJ - 1) / kGlobalJ;
    const int64_t n_fg = (g.F + kWave - 1) / kWave;
    const int64_t items = g.S * n_fg * n_chunks;
    const int64_t blocks = (items + kGlobalWaves - 1) / kGlobalWaves;
    if (!grid_fits(blocks)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((forest_grid_global_kernel<NF, kGlobalJ>), dim3((unsigned)blocks), dim3(kGlobalWaves * kWave),
                       0, stream, f.nodes, f.leaves, f.kvb_box, f.n_trees, f.depth, f.base_score, g);
    return hipGetLastError();
}

}  // namespace


hipError_t pair_order_plan(const ForestDev& f, int64_t n, int64_t min_pairs, PairOrderPlan* p) {
    *p = PairOrderPlan{0, 0, 0, 0};
    if (!f.cuts_kv || !f.cuts_bs || n < min_pairs || n >= (int64_t)1 << 31) return hipSuccess;
    size_t temp = 0;
    const hipError_t e = hipcub::DeviceRadixSort::SortPairsDescending(
        nullptr, temp, (const uint32_t*)nullptr, (uint32_t*)nullptr, (const uint32_t*)nullptr, (uint32_t*)nullptr,
        (int)n, 0, 32, (hipStream_t)0);
    if (e != hipSuccess) return e;
    p->n = n;
    p->arr = ((size_t)n * sizeof(uint32_t) + 255) & ~(size_t)255;
    p->temp = temp;
    p->bytes = 4 * p->arr + temp;
    return hipSuccess;
}

hipError_t pair_order_sort(const PairOrderPlan& p, void* ws, const uint32_t** order, hipStream_t stream) {
    unsigned char* base = (unsigned char*)ws;
    uint32_t* cost_sorted = (uint32_t*)(base + 2 * p.arr);
    uint32_t* sorted = (uint32_t*)(base + 3 * p.arr);
    size_t temp = p.temp;
    const hipError_t e = hipcub::DeviceRadixSort::SortPairsDescending(
        base + 4 * p.arr, temp, pair_order_cost(p, ws), cost_sorted, pair_order_code(p, ws), sorted, (int)p.n, 0, 32,
        stream);
    if (e != hipSuccess) return e;
    *order = sorted;
    return hipSuccess;
}

// Work order for the LDS grid kernel: (scenario, chunk) pairs by estimated
// cost, most expensive first, so a workgroup's wavefronts do similar work
// and the longest ones start first.
namespace {

hipError_t plan_order(const ForestDev& f, const GridParams& g, PairOrderPlan* p) {
    *p = PairOrderPlan{0, 0, 0, 0};
    size_t lds = 0;
    if (lds_trees_per_block(f, &lds) <= 0) return hipSuccess;   // the global kernel takes no order
    return pair_order_plan(f, g.S * ((g.H + kLdsJ - 1) / kLdsJ), 2 * kLdsWaves, p);
}

}  // namespace

hipError_t grid_order_bytes(const ForestDev& f, const GridParams& g, size_t* bytes) {
    PairOrderPlan p;
    const hipError_t e = plan_order(f, g, &p);
    *bytes = e == hipSuccess ? p.bytes : 0;
    return e;
}

hipError_t launch_forest_grid(const ForestDev& f, const GridParams& g_in, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
    GridParams g = g_in;
    g.order = nullptr;
    size_t lds = 0;
    const int32_t tb = lds_trees_per_block(f, &lds);
    if (tb <= 0) return f.n_features == 4 ? launch_grid_global<4>(f, g, stream) : launch_grid_global<3>(f, g, stream);
    PairOrderPlan p;
    hipError_t e = plan_order(f, g, &p);
    if (e != hipSuccess) return e;
    // the order only speeds the kernel up: without room for it the items
    // keep their natural numbering
    if (p.n > 0 && ws && ws_bytes >= p.bytes) {
        hipLaunchKernelGGL(grid_cost_kernel, dim3((unsigned)((p.n + kCostThreads - 1) / kCostThreads)),
                           dim3(kCostThreads), 0, stream, f.cuts_kv, f.n_cuts_kv, f.cuts_bs, f.n_cuts_bs, g.kv,
                           g.batch, g.S, g.H, kLdsJ, pair_order_cost(p, ws), pair_order_code(p, ws));
        e = hipGetLastError();
        if (e == hipSuccess) e = pair_order_sort(p, ws, &g.order, stream);
        if (e != hipSuccess) return e;
    }
    return f.n_features == 4 ? launch_grid_lds<4>(f, g, tb, lds, stream) : launch_grid_lds<3>(f, g, tb, lds, stream);
}

// Workspace of the grid kernel's work order for callers that cannot
// allocate (tl_forest_predict_grid_noalloc): one fixed array per device,
// shared by every such call on that device.  In host code `scratch` only
// names the symbol; its device address comes from hipGetSymbolAddress, once
// per device, and is kept in noalloc_ptr.
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex noalloc_mutex;
void* noalloc_ptr[kMaxDevices];
}  // namespace

hipError_t noalloc_scratch(void** ptr) {
    *ptr = nullptr;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(noalloc_mutex);
    if (!noalloc_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        noalloc_ptr[dev] = p;
    }
    *ptr = noalloc_ptr[dev];
    return hipSuccess;
}

hipError_t launch_forest_rows(const ForestDev& f, const float* rows, int64_t n_rows, float* out,
                              hipStream_t stream) {
    // 3- and 4-feature forests with LDS records: the staged walks of the
    // column kernel; otherwise walks from global memory
    const hipError_t e = launch_forest_rows_lds(f, rows, n_rows, out, stream);
    if (e != hipErrorNotSupported) return e;
    switch (f.n_features) {
        case 1: return launch_nf<1>(f, rows, n_rows, out, stream);
        case 2: return launch_nf<2>(f, rows, n_rows, out, stream);
        case 3: return launch_nf<3>(f, rows, n_rows, out, stream);
        default: return launch_nf<4>(f, rows, n_rows, out, stream);
    }
}

}  // namespace tl
