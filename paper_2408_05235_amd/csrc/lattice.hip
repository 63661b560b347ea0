// The model M (Sec. 4.3.1) compiled to a table over its discrete input
// lattice.  The inputs the controller queries are bounded and discrete: a
// fixed list of candidate frequencies, a few engine sizes, integer batch
// sizes and integer KV-cache blocks.  Every lattice point's value is the
// ensemble's output computed by the grid kernel (the same tree walks and the
// same fp32 running sums in tree order), so a lookup returns exactly what a
// walk would.
//
// Layout: value(e, b, kv, f) at (((e * nB + b) * nC * kHc + kv) * F + f): the
// F frequencies of one lattice point are contiguous, so a row of the
// projection reads one run of F values.  The build evaluates one grid
// "scenario" s' = (e * nB + b) * nC + c per (e, b, KV chunk c) whose KV curve
// is c*kHc + 0 .. kHc-1 and whose batch curve is b; the grid kernel writes it
// as [s'][f][r], which a tiled transpose turns into [s'][r][f] = the layout
// above.  Scenarios are built in batches through a bounded temporary.
//
// Prediction on the projection grid is then a gather: out[s][f][j] =
// value(E_s, B[s][j], KV[s][j], f), 4 bytes written and 4 read per row.
// Rows outside the lattice (KV or batch beyond its bounds or negative, an
// engine size not in its list) are walked tree by tree from global memory.
#include <algorithm>

#include "device_util.h"
#include "tl_internal.h"

namespace tl {
namespace {

__global__ __launch_bounds__(256) void lattice_inputs_kernel(LatticeDev L, int64_t s0, int64_t count, int32_t* kv,
                                                             int32_t* batch, float* engine) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= count * kLatticeChunk) return;
    const int64_t s = s0 + i / kLatticeChunk;
    const int32_t r = (int32_t)(i % kLatticeChunk);
    const int32_t c = (int32_t)(s % L.nC);
    const int32_t b = (int32_t)((s / L.nC) % L.nB);
    const int32_t e = (int32_t)(s / ((int64_t)L.nC * L.nB));
    // points past kv_max are never looked up; keep them inside the domain
    kv[i] = min(c * kLatticeChunk + r, L.kv_max);
    batch[i] = b;
    if (r == 0) engine[i / kLatticeChunk] = L.engines[e];
}

// [count][F][kHc] (grid output of scenarios s0 ..) -> table [s][kHc][F],
// 64 x 64 tiles through LDS
constexpr int kTile = 64;

__global__ __launch_bounds__(256) void lattice_transpose_kernel(const float* __restrict__ src, float* __restrict__ table,
                                                                int64_t s0, int32_t F) {
    __shared__ float tile[kTile][kTile + 1];
    const int32_t n_ft = (F + kTile - 1) / kTile;
    const int32_t n_rt = kLatticeChunk / kTile;
    const int64_t bid = blockIdx.x;
    const int64_t sl = bid / ((int64_t)n_ft * n_rt);
    const int32_t ft = (int32_t)((bid / n_rt) % n_ft);
    const int32_t rt = (int32_t)(bid % n_rt);
    const float* in = src + sl * (int64_t)F * kLatticeChunk;
    float* out = table + (s0 + sl) * (int64_t)kLatticeChunk * F;
    const int tx = threadIdx.x % kTile, ty = threadIdx.x / kTile;   // 64 x 4
    for (int k = ty; k < kTile; k += 256 / kTile) {
        const int32_t f = ft * kTile + k, r = rt * kTile + tx;
        if (f < F) tile[k][tx] = in[(int64_t)f * kLatticeChunk + r];
    }
    __syncthreads();
    for (int k = ty; k < kTile; k += 256 / kTile) {
        const int32_t r = rt * kTile + k, f = ft * kTile + tx;
        if (f < F) out[(int64_t)r * F + f] = tile[tx][k];
    }
}

// fp32 running sum in tree order over heap-ordered trees in global memory
__device__ __forceinline__ float walk_global(const ForestDev& f, const float (&x)[4]) {
    const int64_t stride = (int64_t)1 << f.depth;
    const int32_t n_int = (1 << f.depth) - 1;
    float acc = f.base_score;
    for (int32_t t = 0; t < f.n_trees; ++t) {
        const uint2* nd = f.nodes + t * stride;
        int32_t k = 0;
        for (int32_t level = 0; level < f.depth; ++level) {
            const uint2 w = nd[k];
            k = 2 * k + (x[w.y & 3u] < __uint_as_float(w.x) ? 1 : 2);
        }
        acc += f.leaves[t * stride + (k - n_int)];
    }
    return acc;
}

constexpr int kGatherThreads = 256;

// One thread per (scenario, iteration): it reads KV and batch once, then the
// contiguous run of the lattice point's F values, and writes them to the F
// outputs of the row (consecutive iterations of a workgroup write
// consecutive addresses for each frequency).
__global__ __launch_bounds__(kGatherThreads) void lattice_gather_kernel(ForestDev f, LatticeDev L, GatherParams P,
                                                                         int32_t n_jb) {
    const int64_t s = blockIdx.x / (uint32_t)n_jb;
    const int32_t j = (int32_t)(blockIdx.x % (uint32_t)n_jb) * kGatherThreads + threadIdx.x;
    if (j >= P.H) return;
    const int32_t kv = P.kv[s * P.H + j];
    const int32_t b = P.batch[s * P.H + j];
    const float xe = P.engine ? P.engine[s] : 0.0f;
    int32_t e = 0;
    if (L.nf == 4) {
        e = -1;
        for (int32_t q = 0; q < L.nE; ++q)
            if (L.engines[q] == xe) { e = q; break; }
    }
    const int32_t F = L.F;
    float* out = P.out + s * (int64_t)F * P.H + j;
    if (e >= 0 && kv >= 0 && kv <= L.kv_max && b >= 0 && b <= L.batch_max) {
        const float* t = L.table + ((((int64_t)e * L.nB + b) * L.nC) * kLatticeChunk + kv) * F;
        int32_t fi = 0;
        if ((F & 3) == 0) {
            // runs of 4k floats start 16-byte aligned: 64 values at a time,
            // all loads in flight before the (streaming) stores
            for (; fi + 64 <= F; fi += 64) {
                float4 v[16];
#pragma unroll
                for (int k = 0; k < 16; ++k) v[k] = *(const float4*)(t + fi + 4 * k);
#pragma unroll
                for (int k = 0; k < 16; ++k) {
                    float* o = out + (int64_t)(fi + 4 * k) * P.H;
                    __builtin_nontemporal_store(v[k].x, o);
                    __builtin_nontemporal_store(v[k].y, o + P.H);
                    __builtin_nontemporal_store(v[k].z, o + 2 * (int64_t)P.H);
                    __builtin_nontemporal_store(v[k].w, o + 3 * (int64_t)P.H);
                }
            }
            for (; fi < F; fi += 4) {
                const float4 v = *(const float4*)(t + fi);
                out[(int64_t)fi * P.H] = v.x;
                out[(int64_t)(fi + 1) * P.H] = v.y;
                out[(int64_t)(fi + 2) * P.H] = v.z;
                out[(int64_t)(fi + 3) * P.H] = v.w;
            }
        }
        for (; fi < F; ++fi) out[(int64_t)fi * P.H] = t[fi];
    } else {
        for (int32_t fi = 0; fi < F; ++fi) {
            const float x[4] = {L.freqs[fi], (float)kv, (float)b, xe};
            out[(int64_t)fi * P.H] = walk_global(f, x);
        }
    }
}

// M at one frequency per scenario (index fidx[s], or f_all; scenarios with
// an index < 0 are skipped): one thread per (scenario, iteration), one table
// read.
__global__ __launch_bounds__(kGatherThreads) void lattice_column_kernel(ForestDev f, LatticeDev L, GatherParams P,
                                                                         const int32_t* fidx, int32_t f_all,
                                                                         int32_t n_jb) {
    const int64_t s = blockIdx.x / (uint32_t)n_jb;
    const int32_t j = (int32_t)(blockIdx.x % (uint32_t)n_jb) * kGatherThreads + threadIdx.x;
    if (j >= P.H) return;
    const int32_t fi = fidx ? fidx[s] : f_all;
    if (fi < 0 || fi >= L.F) return;
    const int32_t kv = P.kv[s * P.H + j];
    const int32_t b = P.batch[s * P.H + j];
    const float xe = P.engine ? P.engine[s] : 0.0f;
    int32_t e = 0;
    if (L.nf == 4) {
        e = -1;
        for (int32_t q = 0; q < L.nE; ++q)
            if (L.engines[q] == xe) { e = q; break; }
    }
    float v;
    if (e >= 0 && kv >= 0 && kv <= L.kv_max && b >= 0 && b <= L.batch_max) {
        v = L.table[((((int64_t)e * L.nB + b) * L.nC) * kLatticeChunk + kv) * L.F + fi];
    } else {
        const float x[4] = {L.freqs[fi], (float)kv, (float)b, xe};
        v = walk_global(f, x);
    }
    P.out[s * P.H + j] = v;
}

}  // namespace

hipError_t launch_lattice_column(const ForestDev& f, const LatticeDev& L, const GatherParams& p,
                                 const int32_t* fidx, int32_t f_all, hipStream_t stream) {
    if (p.S == 0) return hipSuccess;
    const int32_t n_jb = (p.H + kGatherThreads - 1) / kGatherThreads;
    const int64_t blocks = p.S * n_jb;
    if (!grid_fits(blocks)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(lattice_column_kernel, dim3((unsigned)blocks), dim3(kGatherThreads), 0, stream, f, L, p, fidx,
                       f_all, n_jb);
    return hipGetLastError();
}

hipError_t launch_lattice_inputs(const LatticeDev& L, int64_t s0, int64_t count, int32_t* kv, int32_t* batch,
                                 float* engine, hipStream_t stream) {
    const int64_t n = count * kLatticeChunk;
    if (!grid_fits((n + 255) / 256)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(lattice_inputs_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, L, s0, count,
                       kv, batch, engine);
    return hipGetLastError();
}

hipError_t launch_lattice_transpose(const float* src, float* table, int64_t s0, int64_t count, int32_t F,
                                    hipStream_t stream) {
    const int64_t blocks = count * ((F + kTile - 1) / kTile) * (kLatticeChunk / kTile);
    if (!grid_fits(blocks)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(lattice_transpose_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, src, table, s0, F);
    return hipGetLastError();
}

hipError_t launch_lattice_gather(const ForestDev& f, const LatticeDev& L, const GatherParams& p, hipStream_t stream) {
    if (p.S == 0) return hipSuccess;
    const int32_t n_jb = (p.H + kGatherThreads - 1) / kGatherThreads;
    const int64_t blocks = p.S * n_jb;
    if (!grid_fits(blocks)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(lattice_gather_kernel, dim3((unsigned)blocks), dim3(kGatherThreads), 0, stream, f, L, p, n_jb);
    return hipGetLastError();
}

}  // namespace tl
