// Formats of the forest data the host builds and the kernels read: the
// LDS-staged tree records and the threshold cuts.  No HIP headers, so the
// host-side builders (host_forest.cpp) also compile as plain C++.
#pragma once

#include <stdint.h>

#if defined(__HIP__) || defined(__HIPCC__)
#define TL_HOST_DEVICE __host__ __device__
#else
#define TL_HOST_DEVICE
#endif

namespace tl {

constexpr int32_t kMaxCuts = 4096;

constexpr int kMaxRecordDepth = 11;

// One tree as the LDS-staged kernels read it (byte ranges, each starting on
// a 16-byte boundary):
//   [0, boxes)      2^d node slots of 16 bytes, slot k = (threshold,
//                   sel_lo, sel_hi, value of leaf k).  The selectors are
//                   byte-permute selectors that pick the tested feature c
//                   out of (frequency, KV, batch, engine size): sel_lo picks
//                   between frequency and KV and, with the same selector,
//                   between batch and engine size (bit 0 of c), sel_hi
//                   between the two picks (bit 1 of c).  A row goes to 2k+1
//                   iff x_c < threshold.  Slot 2^d - 1 holds no node, only
//                   the last leaf's value.
//   [boxes, bytes)  leaf boxes, 8 bytes per leaf: the leaf's KV / batch box
//                   (kvb_box) as integer bounds, word 0 = kv_lo | batch_lo
//                   << 20, word 1 = kv_hi | batch_hi << 20, meaning kv_lo <=
//                   KV < kv_hi and batch_lo <= batch < batch_hi for integer
//                   KV and batch.  The bounds are rounded up to integers and
//                   clamped to [0, 2^20 - 1] (KV) and [0, 2^12 - 1] (batch);
//                   a clamped box is a subset of the leaf's own, so a row
//                   inside it still reaches the leaf, and a row outside it
//                   only walks the tree again.
// A block of consecutive trees is one contiguous byte range, staged as is.
constexpr uint32_t kBoxKvMax = (1u << 20) - 1;
constexpr uint32_t kBoxBatchMax = (1u << 12) - 1;

struct RecordLayout {
    uint32_t boxes, bytes;
};

TL_HOST_DEVICE inline RecordLayout record_layout(int32_t depth) {
    const uint32_t n_leaf = 1u << depth;
    RecordLayout r;
    r.boxes = 16u * n_leaf;
    r.bytes = r.boxes + ((8u * n_leaf + 15u) & ~15u);
    return r;
}

}  // namespace tl
