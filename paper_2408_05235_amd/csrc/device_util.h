// Device helpers for the gfx950 kernels: 64-lane wavefront scans and
// reductions, and division by a run-time invariant divisor.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <limits.h>

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

// Wavefront scans by DPP (data movement inside the VALU, no LDS round
// trips): shifts by 1, 2, 4 and 8 lanes within each row of 16 lanes, then
// the last lane of row 0 into row 1 and of row 2 into row 3 (row_bcast:15),
// then lane 31 into rows 2 and 3 (row_bcast:31).  A lane whose source is
// outside its row, or whose row the step leaves out, takes the operation's
// identity.  The whole wavefront must be active.
namespace dpp {
constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
constexpr int kRowBcast15 = 0x142, kRowBcast31 = 0x143;
constexpr int kWaveShr1 = 0x138;   // every lane from the lane below (lane 0: identity)

template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ int32_t move(int32_t v, int32_t identity) {
    return __builtin_amdgcn_update_dpp(identity, v, CTRL, ROW_MASK, 0xf, false);
}

template <class Op>
__device__ __forceinline__ int32_t scan(int32_t v, int32_t identity, Op op) {
    v = op(v, move<kRowShr1>(v, identity));
    v = op(v, move<kRowShr2>(v, identity));
    v = op(v, move<kRowShr4>(v, identity));
    v = op(v, move<kRowShr8>(v, identity));
    v = op(v, move<kRowBcast15, 0xa>(v, identity));
    v = op(v, move<kRowBcast31, 0xc>(v, identity));
    return v;
}

template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ uint64_t move_u64(uint64_t v) {
    const uint32_t lo = (uint32_t)move<CTRL, ROW_MASK>((int32_t)(uint32_t)v, 0);
    const uint32_t hi = (uint32_t)move<CTRL, ROW_MASK>((int32_t)(uint32_t)(v >> 32), 0);
    return ((uint64_t)hi << 32) | lo;
}
}  // namespace dpp

__device__ __forceinline__ int32_t wave_incl_scan(int32_t v) {
    return dpp::scan(v, 0, [](int32_t a, int32_t b) { return a + b; });
}

__device__ __forceinline__ uint64_t wave_incl_scan_u64(uint64_t v) {
    v += dpp::move_u64<dpp::kRowShr1>(v);
    v += dpp::move_u64<dpp::kRowShr2>(v);
    v += dpp::move_u64<dpp::kRowShr4>(v);
    v += dpp::move_u64<dpp::kRowShr8>(v);
    v += dpp::move_u64<dpp::kRowBcast15, 0xa>(v);
    v += dpp::move_u64<dpp::kRowBcast31, 0xc>(v);
    return v;
}

__device__ __forceinline__ int32_t wave_incl_max(int32_t v) {
    return dpp::scan(v, INT32_MIN, [](int32_t a, int32_t b) { return a > b ? a : b; });
}

// The value of the lane below (lane 0: `identity`).
__device__ __forceinline__ int32_t wave_shift_up1(int32_t v, int32_t identity) {
    return dpp::move<dpp::kWaveShr1>(v, identity);
}

// Reductions: the scan's last lane, read into a scalar register (every lane
// gets the same, wave-uniform value).
__device__ __forceinline__ int32_t lane63(int32_t v) { return __builtin_amdgcn_readlane(v, kWave - 1); }

__device__ __forceinline__ uint64_t lane63_u64(uint64_t v) {
    return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int32_t)(v >> 32), kWave - 1) << 32) |
           (uint32_t)__builtin_amdgcn_readlane((int32_t)(uint32_t)v, kWave - 1);
}

__device__ __forceinline__ int32_t wave_max(int32_t v) { return lane63(wave_incl_max(v)); }

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) { return lane63_u64(wave_incl_scan_u64(v)); }

__device__ __forceinline__ int32_t wave_sum(int32_t v) { return lane63(wave_incl_scan(v)); }

__device__ __forceinline__ uint32_t wave_or(uint32_t v) {
    return (uint32_t)lane63(dpp::scan((int32_t)v, 0, [](int32_t a, int32_t b) { return a | b; }));
}

}  // namespace tl
