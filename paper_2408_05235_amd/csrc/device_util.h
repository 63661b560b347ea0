// Device helpers for the gfx950 kernels: 64-lane wavefront scans and
// reductions, and division by a run-time invariant divisor.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tl {

constexpr int kWave = 64;

// Unsigned division by an invariant divisor d >= 1 for dividends x < 2^31
// (Granlund & Montgomery, "Division by invariant integers using
// multiplication", 1994): with l = ceil(log2 d) and
// m = floor(2^32 (2^l - d) / d) + 1, x / d = (mulhi(m, x) + x) >> l.
// mulhi(m, x) <= x keeps the 32-bit sum from wrapping while x < 2^31.
struct DivU32 {
    uint32_t d, m, l;
};

__host__ inline DivU32 make_divu32(uint32_t d) {
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;
    uint64_t m = (((1ull << l) - d) << 32) / d + 1;
    return DivU32{d, (uint32_t)m, l};
}

__device__ __forceinline__ uint32_t div_u32(uint32_t x, DivU32 q) {
    uint32_t hi = __umulhi(q.m, x);
    return (hi + x) >> q.l;
}

__device__ __forceinline__ uint32_t ceil_div_u32(uint32_t x, DivU32 q) {
    return div_u32(x + q.d - 1, q);   // caller keeps x + d - 1 < 2^31
}

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

__device__ __forceinline__ int32_t wave_incl_scan(int32_t v) {
    const int lane = lane_id();
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        int32_t u = __shfl_up(v, d);
        if (lane >= d) v += u;
    }
    return v;
}

__device__ __forceinline__ uint64_t wave_incl_scan_u64(uint64_t v) {
    const int lane = lane_id();
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        uint64_t u = __shfl_up(v, d);
        if (lane >= d) v += u;
    }
    return v;
}

__device__ __forceinline__ int32_t wave_incl_max(int32_t v) {
    const int lane = lane_id();
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        int32_t u = __shfl_up(v, d);
        if (lane >= d) v = max(v, u);
    }
    return v;
}

// Butterfly reductions: every lane ends with the same value, which is
// returned through a lane read so the compiler treats it as wave-uniform.
__device__ __forceinline__ int32_t wave_max(int32_t v) {
#pragma unroll
    for (int d = kWave / 2; d >= 1; d >>= 1) v = max(v, __shfl_xor(v, d));
    return __builtin_amdgcn_readfirstlane(v);
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
    for (int d = kWave / 2; d >= 1; d >>= 1) v += __shfl_xor(v, d);
    return ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int32_t)(v >> 32)) << 32) |
           (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)(uint32_t)v);
}

__device__ __forceinline__ int32_t wave_sum(int32_t v) {
#pragma unroll
    for (int d = kWave / 2; d >= 1; d >>= 1) v += __shfl_xor(v, d);
    return __builtin_amdgcn_readfirstlane(v);
}

__device__ __forceinline__ uint32_t wave_or(uint32_t v) {
#pragma unroll
    for (int d = kWave / 2; d >= 1; d >>= 1) v |= __shfl_xor(v, d);
    return (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)v);
}

}  // namespace tl
