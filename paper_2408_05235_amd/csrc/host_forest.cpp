// Host-side preparation of a tree ensemble (see host_forest.h).
#include "host_forest.h"

#include <algorithm>
#include <cmath>
#include <cstring>

namespace tl {
namespace host {

// Going to 2k+1 means x < thr (an upper bound); going to 2k+2 means
// !(x < thr), i.e. x >= thr for non-NaN x (a lower bound).  A NaN threshold
// sends every row to 2k+2: no constraint there, and nothing reaches the 2k+1
// side, whose leaves get an empty box.
void leaf_boxes(int32_t n_trees, int32_t depth, const uint8_t* feature, const float* threshold,
                std::vector<Box>& out) {
    const int64_t n_int = (1ll << depth) - 1;
    const int64_t n_leaf = 1ll << depth;
    out.assign((size_t)(n_trees * n_leaf), Box{0, 0, 0, 0});
    for (int64_t t = 0; t < n_trees; ++t) {
        const uint8_t* ft = feature + t * n_int;
        const float* th = threshold + t * n_int;
        for (int64_t L = 0; L < n_leaf; ++L) {
            float lo[2] = {-INFINITY, -INFINITY}, hi[2] = {INFINITY, INFINITY};
            bool empty = false;
            int64_t k = 0;
            for (int32_t l = 0; l < depth; ++l) {
                const int bit = (int)((L >> (depth - 1 - l)) & 1);   // 0: to 2k+1, 1: to 2k+2
                const float thr = th[k];
                const int f = ft[k];
                if (bit == 0) {
                    if (std::isnan(thr)) empty = true;
                    else if (f == 1 || f == 2) hi[f - 1] = std::fmin(hi[f - 1], thr);
                } else if (!std::isnan(thr) && (f == 1 || f == 2)) {
                    lo[f - 1] = std::fmax(lo[f - 1], thr);
                }
                k = 2 * k + 1 + bit;
            }
            out[(size_t)(t * n_leaf + L)] = empty ? Box{INFINITY, -INFINITY, INFINITY, -INFINITY}
                                                  : Box{lo[0], hi[0], lo[1], hi[1]};
        }
    }
}

uint32_t box_bound(float x, uint32_t maxv) {
    const double c = std::ceil((double)x);
    if (!(c > 0.0)) return 0;
    if (c >= (double)maxv) return maxv;
    return (uint32_t)c;
}

void build_records(int32_t n_trees, int32_t depth, const uint8_t* feature, const float* threshold, const float* leaf,
                   const std::vector<Box>& boxes, std::vector<unsigned char>& out) {
    // node slots (threshold, sel_lo, sel_hi, leaf value; sel_lo picks
    // frequency / KV and batch / engine size by bit 0 of the feature, sel_hi
    // between the two by bit 1), then the leaf boxes as packed integer bounds
    constexpr uint32_t kLow = 0x03020100u, kHigh = 0x07060504u;
    const int64_t n_int = (1ll << depth) - 1;
    const int64_t n_leaf = 1ll << depth;
    const RecordLayout R = record_layout(depth);
    out.assign((size_t)n_trees * R.bytes + 64, 0);
    for (int64_t t = 0; t < n_trees; ++t) {
        unsigned char* rec = out.data() + (size_t)t * R.bytes;
        uint32_t slot[4];
        for (int64_t k = 0; k < n_leaf; ++k) {
            slot[0] = slot[1] = slot[2] = 0;
            if (k < n_int) {
                const int64_t i = t * n_int + k;
                const int fi = feature[i];
                std::memcpy(&slot[0], &threshold[i], 4);
                slot[1] = (fi & 1) ? kHigh : kLow;
                slot[2] = (fi & 2) ? kHigh : kLow;
            }
            std::memcpy(&slot[3], &leaf[t * n_leaf + k], 4);
            std::memcpy(rec + 16 * k, slot, 16);
            const Box& b = boxes[(size_t)(t * n_leaf + k)];
            const uint32_t w[2] = {box_bound(b.kv_lo, kBoxKvMax) | box_bound(b.batch_lo, kBoxBatchMax) << 20,
                                   box_bound(b.kv_hi, kBoxKvMax) | box_bound(b.batch_hi, kBoxBatchMax) << 20};
            std::memcpy(rec + R.boxes + 8 * k, w, 8);
        }
    }
}

std::vector<float> threshold_cuts(int64_t n_nodes, const uint8_t* feature, const float* threshold, int fi) {
    std::vector<float> t;
    for (int64_t i = 0; i < n_nodes; ++i)
        if (feature[i] == fi && std::isfinite(threshold[i])) t.push_back(threshold[i]);
    std::sort(t.begin(), t.end());
    if ((int64_t)t.size() <= kMaxCuts) return t;
    std::vector<float> c(kMaxCuts);
    for (int64_t i = 0; i < kMaxCuts; ++i) c[(size_t)i] = t[(size_t)(i * (int64_t)t.size() / kMaxCuts)];
    return c;
}

}  // namespace host
}  // namespace tl
