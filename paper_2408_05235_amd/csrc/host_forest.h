// Host-side preparation of a tree ensemble for the kernels (plain C++, no
// HIP): the KV / batch box of every leaf, the LDS tree records and the
// threshold cuts of the work-order cost model.  Trees are complete, depth d,
// heap order: internal node k tests x[feature] < threshold and continues at
// 2k+1 if true, at 2k+2 otherwise (Sec. 4.3.1 model M).
#pragma once

#include <stdint.h>

#include <vector>

#include "record_format.h"

namespace tl {
namespace host {

// The bounds a leaf's root-to-leaf path puts on features 1 (KV) and 2
// (batch) as half-open intervals: a row with kv_lo <= KV < kv_hi and
// batch_lo <= batch < batch_hi reaches the leaf whenever a row with the same
// frequency and engine size does.  Empty (lo = +inf, hi = -inf) for leaves
// no row can reach.
struct Box {
    float kv_lo, kv_hi, batch_lo, batch_hi;
};

// boxes of every leaf of every tree, [n_trees][2^depth]
void leaf_boxes(int32_t n_trees, int32_t depth, const uint8_t* feature, const float* threshold,
                std::vector<Box>& out);

// One bound of a leaf box as stored in the records: ceil(x) clamped to
// [0, maxv] (for integer inputs, x >= lo iff x >= ceil(lo) and x < hi iff
// x < ceil(hi); clamping can only shrink the box).
uint32_t box_bound(float x, uint32_t maxv);

// The records of all trees (record_layout(depth).bytes each, back to back,
// plus 64 bytes of padding) from the node arrays [n_trees][2^depth - 1], the
// leaves [n_trees][2^depth] and the leaf boxes.  depth <= kMaxRecordDepth.
void build_records(int32_t n_trees, int32_t depth, const uint8_t* feature, const float* threshold, const float* leaf,
                   const std::vector<Box>& boxes, std::vector<unsigned char>& out);

// Up to kMaxCuts quantiles of the finite thresholds of feature fi over
// n_nodes nodes, ascending.
std::vector<float> threshold_cuts(int64_t n_nodes, const uint8_t* feature, const float* threshold, int fi);

}  // namespace host
}  // namespace tl
