// Stage 2: the performance model M (Sec. 4.3.1), a gradient-boosted tree
// ensemble, evaluated on fp32 feature rows.
//
// Each thread evaluates RPT consecutive rows.  Rows produced by the projection
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
