// Stage 2: the performance model M (Sec. 4.3.1), a gradient-boosted tree
// ensemble, evaluated on fp32 feature rows.
//
// Two kernels compute the same function.
//
// forest_grid_kernel evaluates the rows of the projection grid without
// materializing them: row (s, f, j) = (freq[f], kv[s][j], batch[s][j]
// [, engine[s]]).  One wavefront takes one scenario and J consecutive future
// iterations; its lanes are the candidate frequencies, so every lane sees the
// same (KV, batch) sequence.  For each tree (in order) a lane keeps the leaf
// reached by its previous row together with that leaf's KV / batch box; the
// next row reuses the leaf while its (KV, batch) stays inside the box, which
// is exact because frequency and engine size are fixed for the lane.  Only
// rows that leave the box walk the tree again.  Between consecutive future
// iterations KV and batch move little, so most rows cost a box test and one
// fp64 add per tree instead of a depth-long walk.
//
// forest_rows_kernel evaluates arbitrary rows.  Each thread evaluates RPT
// consecutive rows.  Rows produced by the projection
// are ordered [scenario][frequency][iteration], so a thread's rows -- and the
// 64 x RPT rows of a wavefront -- are consecutive future iterations at one
// frequency.  Their (KV, batch) values change slowly, so lanes of a wave walk
// the same nodes most of the time and node loads are mostly broadcasts.
// Trees are visited in order and the leaf values are accumulated in fp64 in
// that order, then rounded once to fp32.
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

template <int NF, int RPT>
__global__ __launch_bounds__(256) void forest_rows_kernel(const uint2* __restrict__ nodes,
                                                          const double* __restrict__ leaves,
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
        const uint2* nt = nodes + (int64_t)t * n_int;
        const double* lt = leaves + (int64_t)t * n_leaf;
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
        if (r < nr) out[r0 + r] = (float)acc[r];
}

constexpr int kGridJ = 32;            // iterations per wavefront
constexpr int kGridWaves = 4;         // wavefronts per workgroup

template <int NF, int J>
__global__ __launch_bounds__(256) void forest_grid_kernel(const uint2* __restrict__ nodes,
                                                          const double* __restrict__ leaves,
                                                          const float4* __restrict__ boxes,
                                                          int32_t n_trees, int32_t depth, float base,
                                                          GridParams P) {
    __shared__ float2 kvb[kGridWaves][J];
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int32_t H = P.H, F = P.F;
    const int32_t n_chunks = (H + J - 1) / J;
    const int32_t n_fg = (F + kWave - 1) / kWave;
    const int64_t item = __builtin_amdgcn_readfirstlane((int64_t)blockIdx.x * kGridWaves + wave);
    const bool valid = item < P.S * n_fg * n_chunks;   // uniform per wave
    const int64_t it = valid ? item : 0;
    const int32_t chunk = (int32_t)(it % n_chunks);
    const int64_t rest = it / n_chunks;
    const int32_t fg = (int32_t)(rest % n_fg);
    const int64_t s = rest / n_fg;
    const int32_t f = fg * kWave + lane;
    const bool active = valid && f < F;
    const float xf = P.freqs[f < F ? f : F - 1];
    const float xe = (NF == 4) ? P.engine[s] : 0.0f;
    const int32_t j0 = chunk * J;
    const int32_t nj = min(J, H - j0);
    if (lane < J) {
        const int32_t j = j0 + min(lane, nj - 1);
        kvb[wave][lane] = make_float2((float)P.kv[s * H + j], (float)P.batch[s * H + j]);
    }
    __syncthreads();
    if (!valid) return;

    double acc[J];
#pragma unroll
    for (int jj = 0; jj < J; ++jj) acc[jj] = (double)base;
    const int32_t n_int = (1 << depth) - 1;
    const int32_t n_leaf = 1 << depth;
    for (int32_t t = 0; t < n_trees; ++t) {
        const uint2* nt = nodes + (int64_t)t * n_int;
        const double* lv = leaves + (int64_t)t * n_leaf;
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
                    const uint32_t ft = nd.y;
                    const float x = ft == 0 ? xf : (ft == 1 ? v2.x : (ft == 2 ? v2.y : xe));
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
        float* o = P.out + ((int64_t)s * F + f) * H + j0;
#pragma unroll
        for (int jj = 0; jj < J; ++jj)
            if (jj < nj) o[jj] = (float)acc[jj];
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

}  // namespace

hipError_t launch_forest_grid(const ForestDev& f, const GridParams& g, hipStream_t stream) {
    const int64_t n_chunks = (g.H + kGridJ - 1) / kGridJ;
    const int64_t n_fg = (g.F + kWave - 1) / kWave;
    const int64_t items = g.S * n_fg * n_chunks;
    const int64_t blocks = (items + kGridWaves - 1) / kGridWaves;
    if (f.n_features == 4)
        hipLaunchKernelGGL((forest_grid_kernel<4, kGridJ>), dim3((unsigned)blocks), dim3(kGridWaves * kWave), 0,
                           stream, f.nodes, f.leaves, f.kvb_box, f.n_trees, f.depth, f.base_score, g);
    else
        hipLaunchKernelGGL((forest_grid_kernel<3, kGridJ>), dim3((unsigned)blocks), dim3(kGridWaves * kWave), 0,
                           stream, f.nodes, f.leaves, f.kvb_box, f.n_trees, f.depth, f.base_score, g);
    return hipGetLastError();
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
