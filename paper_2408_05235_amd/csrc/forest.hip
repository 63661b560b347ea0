// Stage 2: the performance model M (Sec. 4.3.1), a gradient-boosted tree
// ensemble, evaluated on fp32 feature rows.  Every kernel here computes, for
// each row, base + the leaf of every tree, accumulated in fp64 in tree order
// and rounded once to fp32.
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
// fp64 add per tree; a walk happens on roughly one row in twenty.
//
//   forest_grid_lds_kernel     (depth <= 11) A 1024-thread workgroup (16
//       wavefronts, 16 x 32 x 64 rows) walks the ensemble in blocks of trees
//       that are staged in LDS, double-buffered: the next block is fetched
//       into registers while the current one is evaluated: nodes, leaf
//       values and leaf boxes.  Tree walks read LDS only.  Nodes hold one
//       threshold per feature (NaN for the features they do not test) so a
//       step is four compares and no feature selection.  Trees are walked in
//       pairs so that two chains of dependent LDS reads overlap.  The wavefront's
//       (KV, batch) pairs are uniform and live in scalar registers.
//   forest_grid_global_kernel  (deeper trees) The same per-lane scheme with
//       nodes, leaves and boxes read from global memory.
//
// Device layout (built by tl_forest_create): nodes [T][2^d] (8 bytes:
// threshold bits, feature; the last entry of each tree is padding), leaves
// [T][2^d] fp32, and for 3-4 features the leaf boxes [T][2^d] (kv_lo, kv_hi,
// batch_lo, batch_hi) and the 16-byte nodes of the LDS kernel [T][2^d].
//
// forest_rows_kernel evaluates arbitrary rows: each thread walks RPT
// consecutive rows through every tree.
#include "device_util.h"
#include "tl_internal.h"

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
    double acc[RPT];
#pragma unroll
    for (int r = 0; r < RPT; ++r) acc[r] = (double)base;
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
        for (int r = 0; r < RPT; ++r) acc[r] += (double)lt[k[r] - n_int];
    }
#pragma unroll
    for (int r = 0; r < RPT; ++r)
        if (r < nr) out[r0 + r] = (float)acc[r];
}

#ifndef TL_LDS_J
#define TL_LDS_J 32
#endif
#ifndef TL_LDS_WAVES
#define TL_LDS_WAVES 16
#endif
#ifndef TL_LDS_BUDGET_KIB
#define TL_LDS_BUDGET_KIB 152
#endif
constexpr int kLdsJ = TL_LDS_J;          // future iterations per wavefront (LDS kernel)
constexpr int kGlobalJ = 32;             // future iterations per wavefront (global kernel)

// Which (scenario, frequency group, iteration chunk) a wavefront evaluates.
struct GridItem {
    bool valid;
    int64_t s;
    int32_t f, j0, nj;
};

__device__ __forceinline__ GridItem grid_item(const GridParams& P, int64_t item, int J) {
    const int32_t n_chunks = (P.H + J - 1) / J;
    const int32_t n_fg = (P.F + kWave - 1) / kWave;
    GridItem g;
    g.valid = item < P.S * n_fg * n_chunks;
    const int64_t it = g.valid ? item : 0;
    const int32_t chunk = (int32_t)(it % n_chunks);
    const int64_t rest = it / n_chunks;
    g.f = (int32_t)(rest % n_fg) * kWave + lane_id();
    g.s = rest / n_fg;
    g.j0 = chunk * J;
    g.nj = min(J, P.H - g.j0);
    return g;
}

// ---------------------------------------------------------------- LDS-staged

// Whether (kv, batch) lies in a leaf box (kv_lo, kv_hi, batch_lo, batch_hi).
__device__ __forceinline__ bool in_box(const float4& b, float kv, float bs) {
    return (kv >= b.x) & (kv < b.y) & (bs >= b.z) & (bs < b.w);
}

// Lane mask of the lanes that go to 2k+1 at a node holding one threshold per
// feature: the node's own feature carries its threshold, the others NaN,
// which no "not >=" test (compare predicate 12: unordered or less than) can
// fail.  The tests run as wavefront lane masks.
template <int NF>
__device__ __forceinline__ uint64_t go_left(const float4& nd, float xf, float kv, float bs, float xe) {
    uint64_t m = __builtin_amdgcn_fcmpf(xf, nd.x, 12) & __builtin_amdgcn_fcmpf(kv, nd.y, 12) &
                 __builtin_amdgcn_fcmpf(bs, nd.z, 12);
    if (NF == 4) m &= __builtin_amdgcn_fcmpf(xe, nd.w, 12);
    return m;
}

// 1 for lanes whose bit is set in the wavefront lane mask m (go to 2k+1),
// 2 otherwise: one v_cndmask on the mask instead of extracting the lane's bit.
__device__ __forceinline__ int32_t child_step(uint64_t m) {
    int32_t step;
    asm("v_cndmask_b32_e64 %0, 2, 1, %1" : "=v"(step) : "s"(m));
    return step;
}

constexpr int kLdsWaves = TL_LDS_WAVES;  // wavefronts per workgroup
constexpr int kLdsThreads = kLdsWaves * kWave;
constexpr int kStageRegs = 4 * 16 / TL_LDS_WAVES;  // staged 16-byte words per thread per block
constexpr int kMaxLdsDepth = 11;

// Per staged tree: 2^d nodes (16 bytes, the last one padding), 2^d leaf
// values (4 bytes) and 2^d leaf boxes (16 bytes), each segment contiguous
// over the trees of a block.
struct StageLayout {
    uint32_t nodes, vals, boxes, stride;   // byte offsets inside a buffer, buffer size
};

__host__ __device__ inline StageLayout stage_layout(int32_t tb, int32_t n_leaf) {
    StageLayout L;
    L.nodes = 0;
    L.vals = (uint32_t)tb * n_leaf * 16u;
    L.boxes = L.vals + (((uint32_t)tb * n_leaf * 4u + 15u) & ~15u);
    L.stride = L.boxes + (uint32_t)tb * n_leaf * 16u;
    return L;
}

template <int NF, int J>
__global__ __launch_bounds__(kLdsThreads, 4) void forest_grid_lds_kernel(const uint4* __restrict__ nodes4,
                                                                      const float* __restrict__ leaves,
                                                                      const float4* __restrict__ boxes,
                                                                      int32_t n_trees, int32_t depth,
                                                                      int32_t tb, float base, GridParams P) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int32_t n_int = (1 << depth) - 1;
    const int32_t n_leaf = 1 << depth;
    const StageLayout L = stage_layout(tb, n_leaf);

    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int64_t item = __builtin_amdgcn_readfirstlane((int64_t)blockIdx.x * kLdsWaves + wave);
    const GridItem g = grid_item(P, item, J);
    const int32_t F = P.F, H = P.H;
    const bool active = g.valid && g.f < F;
    // A NaN input takes every right turn at its own nodes, as +inf does; +inf
    // also passes the "not >=" tests of the other features' NaN thresholds.
    float xf = P.freqs[g.f < F ? g.f : F - 1];
    float xe = (NF == 4) ? P.engine[g.s] : 0.0f;
    xf = (xf == xf) ? xf : INFINITY;
    xe = (xe == xe) ? xe : INFINITY;
    // the J (KV, batch) pairs of this wavefront are the same for every lane:
    // keep them in scalar registers
    float skv[J], sbs[J];
    {
        const int32_t j = g.j0 + min(lane % J, g.nj - 1);
        const float kvl = (float)P.kv[g.s * H + j], bsl = (float)P.batch[g.s * H + j];
#pragma unroll
        for (int jj = 0; jj < J; ++jj) {
            skv[jj] = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(kvl), jj));
            sbs[jj] = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(bsl), jj));
        }
    }

    // staging: block b holds trees [b*tb, b*tb + cnt), copied as 16-byte words
    // from the three global arrays (the host pads them so whole words exist).
    // Each thread moves up to kStageRegs words: one load per word straight
    // into its own register, so the loads stay in flight while the current
    // block is evaluated.
    const int32_t n_blocks = (n_trees + tb - 1) / tb;
    static_assert(kStageRegs == 4 || kStageRegs == 8, "staging code below moves four or eight words");
    uint4 rw0 = make_uint4(0, 0, 0, 0), rw1 = rw0, rw2 = rw0, rw3 = rw0;
    uint4 rw4 = rw0, rw5 = rw0, rw6 = rw0, rw7 = rw0;
    double acc[J];
#pragma unroll
    for (int jj = 0; jj < J; ++jj) acc[jj] = (double)base;

#define TL_STAGE_WORDS(b)                                                      \
    const int32_t cnt_ = min(tb, n_trees - (b) * tb);                          \
    const int32_t wn = cnt_ * n_leaf;                                          \
    const int32_t wv = (cnt_ * n_leaf * 4 + 15) / 16;                          \
    const int32_t wt = wn + wv + cnt_ * n_leaf;
#define TL_FETCH_WORD(r, reg)                                                  \
    {                                                                          \
        /* unconditional (threads past the block re-read word 0), so the   */ \
        /* four loads issue back to back without waits between them        */ \
        const int32_t i0 = (int32_t)threadIdx.x + (r) * kLdsThreads;           \
        const int32_t i = i0 < wt ? i0 : 0;                                    \
        const uint4* src = i < wn ? sn : (i < wn + wv ? sv : sb);              \
        reg = src[i];                                                          \
    }
#define TL_FETCH(b)                                                            \
    {                                                                          \
        TL_STAGE_WORDS(b)                                                      \
        const int64_t t0 = (int64_t)(b) * tb;                                  \
        const uint4* sn = nodes4 + t0 * n_leaf;                                \
        const uint4* sv = (const uint4*)(leaves + t0 * n_leaf) - wn;           \
        const uint4* sb = (const uint4*)(boxes + t0 * n_leaf) - (wn + wv);     \
        TL_FETCH_WORD(0, rw0) TL_FETCH_WORD(1, rw1)                            \
        TL_FETCH_WORD(2, rw2) TL_FETCH_WORD(3, rw3)                            \
        if (kStageRegs == 8) {                                                 \
            TL_FETCH_WORD(4, rw4) TL_FETCH_WORD(5, rw5)                        \
            TL_FETCH_WORD(6, rw6) TL_FETCH_WORD(7, rw7)                        \
        }                                                                      \
    }
#define TL_STORE_WORD(r, reg)                                                  \
    {                                                                          \
        const int32_t i = (int32_t)threadIdx.x + (r) * kLdsThreads;            \
        uint4* dst = i < wn ? dn : (i < wn + wv ? dv : db);                    \
        if (i < wt) dst[i] = reg;                                              \
    }
#define TL_STORE(b, buf)                                                       \
    {                                                                          \
        TL_STAGE_WORDS(b)                                                      \
        unsigned char* bp = smem + (buf) * L.stride;                           \
        uint4* dn = (uint4*)(bp + L.nodes);                                    \
        uint4* dv = (uint4*)(bp + L.vals) - wn;                                \
        uint4* db = (uint4*)(bp + L.boxes) - (wn + wv);                        \
        TL_STORE_WORD(0, rw0) TL_STORE_WORD(1, rw1)                            \
        TL_STORE_WORD(2, rw2) TL_STORE_WORD(3, rw3)                            \
        if (kStageRegs == 8) {                                                 \
            TL_STORE_WORD(4, rw4) TL_STORE_WORD(5, rw5)                        \
            TL_STORE_WORD(6, rw6) TL_STORE_WORD(7, rw7)                        \
        }                                                                      \
    }

    // Make the lane's frequency / engine size complete here, before any
    // staging load is in flight: otherwise the walks inside the loop would
    // each wait for all outstanding loads, including the prefetch.
    asm volatile("" ::"v"(xf), "v"(xe));
    if (n_blocks > 0) {
        TL_FETCH(0)
        TL_STORE(0, 0)
    }
    __syncthreads();
    for (int32_t b = 0; b < n_blocks; ++b) {
        const int cur = b & 1;
        if (b + 1 < n_blocks) TL_FETCH(b + 1)
        if (g.valid) {
            const int32_t cnt = min(tb, n_trees - b * tb);
            const unsigned char* bp = smem + cur * L.stride;
            const float4* nb = (const float4*)(bp + L.nodes);
            const float* vb = (const float*)(bp + L.vals);
            const float4* bb = (const float4*)(bp + L.boxes);
            // Trees are taken two at a time: when either tree's leaf must be
            // found again, both are walked in one pass, so the two chains of
            // dependent LDS reads overlap.  A lane still inside its box walks
            // back to the same leaf, so no per-tree selection is needed.
            int32_t tt = 0;
            for (; tt + 1 < cnt; tt += 2) {
                const float4* na = nb + tt * n_leaf;
                const float4* nc = na + n_leaf;
                float4 ba = make_float4(INFINITY, -INFINITY, INFINITY, -INFINITY), bc = ba;
                double va = 0.0, vc = 0.0;
#pragma unroll
                for (int jj = 0; jj < J; ++jj) {
                    const float kvj = skv[jj], bsj = sbs[jj];
                    const bool hit = in_box(ba, kvj, bsj) & in_box(bc, kvj, bsj);
                    if (!hit) {
                        int32_t ka = 0, kc = 0;
                        for (int32_t level = 0; level < depth; ++level) {
                            const float4 da = na[ka], dc = nc[kc];
                            ka = 2 * ka + child_step(go_left<NF>(da, xf, kvj, bsj, xe));
                            kc = 2 * kc + child_step(go_left<NF>(dc, xf, kvj, bsj, xe));
                        }
                        const int32_t la = tt * n_leaf + ka - n_int, lc = la + n_leaf + kc - ka;
                        va = (double)vb[la];
                        vc = (double)vb[lc];
                        ba = bb[la];
                        bc = bb[lc];
                    }
                    acc[jj] += va;
                    acc[jj] += vc;
                    // consume the sum here so the adds are not sunk to the end
                    // of the loop (that would keep J leaf-value pairs live)
                    asm volatile("" ::"v"(acc[jj]));
                }
            }
            for (; tt < cnt; ++tt) {
                const float4* na = nb + tt * n_leaf;
                float4 ba = make_float4(INFINITY, -INFINITY, INFINITY, -INFINITY);
                double va = 0.0;
#pragma unroll
                for (int jj = 0; jj < J; ++jj) {
                    const float kvj = skv[jj], bsj = sbs[jj];
                    if (!in_box(ba, kvj, bsj)) {
                        int32_t ka = 0;
                        for (int32_t level = 0; level < depth; ++level)
                            ka = 2 * ka + child_step(go_left<NF>(na[ka], xf, kvj, bsj, xe));
                        const int32_t la = tt * n_leaf + ka - n_int;
                        va = (double)vb[la];
                        ba = bb[la];
                    }
                    acc[jj] += va;
                    asm volatile("" ::"v"(acc[jj]));
                }
            }
        }
        if (b + 1 < n_blocks) TL_STORE(b + 1, cur ^ 1)
        __syncthreads();
    }
#undef TL_STORE
#undef TL_STORE_WORD
#undef TL_FETCH
#undef TL_FETCH_WORD
#undef TL_STAGE_WORDS
    if (active) {
        float* o = P.out + ((int64_t)g.s * F + g.f) * H + g.j0;
#pragma unroll
        for (int jj = 0; jj < J; ++jj)
            if (jj < g.nj) o[jj] = (float)acc[jj];
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

    double acc[J];
#pragma unroll
    for (int jj = 0; jj < J; ++jj) acc[jj] = (double)base;
    const int32_t n_int = (1 << depth) - 1;
    const int32_t n_leaf = 1 << depth;
    for (int32_t t = 0; t < n_trees; ++t) {
        const uint2* nt = nodes + (int64_t)t * n_leaf;
        const float* lv = leaves + (int64_t)t * n_leaf;
        const float4* bx = boxes + (int64_t)t * n_leaf;
        float lo_k = INFINITY, hi_k = -INFINITY, lo_b = INFINITY, hi_b = -INFINITY;
        double val = 0.0;
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
                val = (double)lv[leaf];
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
            if (jj < g.nj) o[jj] = (float)acc[jj];
    }
}

template <int NF>
hipError_t launch_nf(const ForestDev& f, const float* rows, int64_t n_rows, float* out, hipStream_t stream) {
    constexpr int RPT = 4;
    constexpr int TPB = 256;
    const int64_t threads = (n_rows + RPT - 1) / RPT;
    const int64_t blocks = (threads + TPB - 1) / TPB;
    hipLaunchKernelGGL((forest_rows_kernel<NF, RPT>), dim3((unsigned)blocks), dim3(TPB), 0, stream,
                       f.nodes, f.leaves, f.n_trees, f.depth, f.base_score, rows, n_rows, out);
    return hipGetLastError();
}

// Trees per staged block for the LDS kernel: two blocks must fit the LDS
// budget and one block the staging registers; the value segments of a block
// must be whole 16-byte words.  0 = the LDS kernel cannot run.
int32_t lds_trees_per_block(const ForestDev& f, size_t* lds_bytes) {
    if (f.depth > kMaxLdsDepth || !f.kvb_box || !f.nodes4) return 0;
    const int32_t n_leaf = 1 << f.depth;
    const size_t budget = (size_t)TL_LDS_BUDGET_KIB * 1024;
    auto fits = [&](int32_t tb) {
        const StageLayout L = stage_layout(tb, n_leaf);
        const size_t words = (size_t)tb * n_leaf * 36 / 16 + 2;
        return 2 * (size_t)L.stride <= budget && words <= (size_t)kStageRegs * kLdsThreads;
    };
    const int32_t step = n_leaf >= 4 ? 1 : 4 / n_leaf;   // whole 16-byte words per block
    int32_t tb = 64;
    while (tb > step && !fits(tb)) tb -= step;
    if (!fits(tb)) return 0;
    *lds_bytes = 2 * (size_t)stage_layout(tb, n_leaf).stride;
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
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kLdsThreads), lds, stream, f.nodes4, f.leaves,
                       f.kvb_box, f.n_trees, f.depth, tb, f.base_score, g);
    return hipGetLastError();
}

template <int NF>
hipError_t launch_grid_global(const ForestDev& f, const GridParams& g, hipStream_t stream) {
    const int64_t n_chunks = (g.H + kGlobalJ - 1) / kGlobalJ;
    const int64_t n_fg = (g.F + kWave - 1) / kWave;
    const int64_t items = g.S * n_fg * n_chunks;
    const int64_t blocks = (items + kGlobalWaves - 1) / kGlobalWaves;
    hipLaunchKernelGGL((forest_grid_global_kernel<NF, kGlobalJ>), dim3((unsigned)blocks), dim3(kGlobalWaves * kWave),
                       0, stream, f.nodes, f.leaves, f.kvb_box, f.n_trees, f.depth, f.base_score, g);
    return hipGetLastError();
}

}  // namespace


hipError_t launch_forest_grid(const ForestDev& f, const GridParams& g, hipStream_t stream) {
    size_t lds = 0;
    const int32_t tb = lds_trees_per_block(f, &lds);
    if (tb > 0)
        return f.n_features == 4 ? launch_grid_lds<4>(f, g, tb, lds, stream) : launch_grid_lds<3>(f, g, tb, lds, stream);
    return f.n_features == 4 ? launch_grid_global<4>(f, g, stream) : launch_grid_global<3>(f, g, stream);
}

hipError_t launch_forest_rows(const ForestDev& f, const float* rows, int64_t n_rows, float* out,
                              hipStream_t stream) {
    switch (f.n_features) {
        case 1: return launch_nf<1>(f, rows, n_rows, out, stream);
        case 2: return launch_nf<2>(f, rows, n_rows, out, stream);
        case 3: return launch_nf<3>(f, rows, n_rows, out, stream);
        default: return launch_nf<4>(f, rows, n_rows, out, stream);
    }
}

}  // namespace tl
