// Checks of the host-side forest preparation (host_forest.cpp) on random
// ensembles with odd depths and NaN / +-inf / integer thresholds, meant to
// run under AddressSanitizer and UndefinedBehaviorSanitizer:
//   - every record holds the tree's thresholds, selectors and leaf values
//     where the record format puts them;
//   - a row reaches a leaf only from inside that leaf's box, and every row
//     inside a leaf's box (the float box, and the packed integer box decoded
//     as the kernels decode it) with the same frequency and engine size
//     reaches the same leaf, checked with a plain tree walk;
//   - the cuts are finite thresholds of their feature, ascending, at most
//     kMaxCuts.
// Prints a checksum of everything built; exits 1 on the first failure.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "host_forest.h"

namespace {

uint64_t g_state = 0x9e3779b97f4a7c15ull;
uint64_t next_u64() {   // splitmix64
    uint64_t z = (g_state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}
double uniform() { return (double)(next_u64() >> 11) * (1.0 / 9007199254740992.0); }
int64_t below(int64_t n) { return (int64_t)(uniform() * (double)n); }

uint64_t g_hash = 1469598103934665603ull;
void mix(const void* p, size_t n) {
    const unsigned char* b = (const unsigned char*)p;
    for (size_t i = 0; i < n; ++i) g_hash = (g_hash ^ b[i]) * 1099511628211ull;
}

int fail(const char* what, int tree, long long where) {
    std::fprintf(stderr, "FAIL: %s (tree %d, at %lld)\n", what, tree, where);
    return 1;
}

// plain walk: leaf index reached by row x
int64_t walk(const uint8_t* ft, const float* th, int depth, const float* x) {
    int64_t k = 0;
    for (int l = 0; l < depth; ++l) k = (x[ft[k]] < th[k]) ? 2 * k + 1 : 2 * k + 2;
    return k - ((1ll << depth) - 1);
}

bool in_float_box(const tl::host::Box& b, float kv, float bs) {
    return kv >= b.kv_lo && kv < b.kv_hi && bs >= b.batch_lo && bs < b.batch_hi;
}

}  // namespace

int main() {
    const uint32_t kLow = 0x03020100u, kHigh = 0x07060504u;
    long long rows_checked = 0, inside_checked = 0;
    for (int trial = 0; trial < 60; ++trial) {
        const int depth = (int)below(tl::kMaxRecordDepth + 1);            // 0 .. 11
        const int nf = 3 + (int)below(2);
        const int n_trees = 1 + (int)below(depth >= 9 ? 3 : 12);
        const int64_t n_int = (1ll << depth) - 1, n_leaf = 1ll << depth;
        std::vector<uint8_t> feature((size_t)(n_trees * n_int));
        std::vector<float> threshold(feature.size()), leaf((size_t)(n_trees * n_leaf));
        const float lo[4] = {1000.f, 0.f, 0.f, 1.f}, hi[4] = {2000.f, 70000.f, 300.f, 8.f};
        for (size_t i = 0; i < feature.size(); ++i) {
            const int f = (int)below(nf);
            feature[i] = (uint8_t)f;
            const double u = uniform();
            float t = (float)(lo[f] + (hi[f] - lo[f]) * uniform());
            if (u < 0.04) t = NAN;
            else if (u < 0.07) t = INFINITY;
            else if (u < 0.10) t = -INFINITY;
            else if (u < 0.25) t = std::floor(t);                          // ties with integer inputs
            else if (u < 0.28) t = (float)(2000000 + below(100));          // beyond the packed KV range
            threshold[i] = t;
        }
        for (auto& v : leaf) v = (float)(uniform() - 0.5);
        std::vector<tl::host::Box> boxes;
        tl::host::leaf_boxes(n_trees, depth, feature.data(), threshold.data(), boxes);
        std::vector<unsigned char> rec;
        tl::host::build_records(n_trees, depth, feature.data(), threshold.data(), leaf.data(), boxes, rec);
        const tl::RecordLayout R = tl::record_layout(depth);
        if (rec.size() != (size_t)n_trees * R.bytes + 64) return fail("record size", -1, (long long)rec.size());
        mix(rec.data(), rec.size());
        for (int t = 0; t < n_trees; ++t) {
            const unsigned char* r = rec.data() + (size_t)t * R.bytes;
            const uint8_t* ft = feature.data() + t * n_int;
            const float* th = threshold.data() + t * n_int;
            for (int64_t k = 0; k < n_leaf; ++k) {
                uint32_t w[4];
                std::memcpy(w, r + 16 * k, 16);
                uint32_t lb;
                std::memcpy(&lb, &leaf[(size_t)(t * n_leaf + k)], 4);
                if (w[3] != lb) return fail("leaf value in node slot", t, k);
                if (k < n_int) {
                    uint32_t tb;
                    std::memcpy(&tb, &th[k], 4);
                    if (w[0] != tb) return fail("threshold", t, k);
                    if (w[1] != ((ft[k] & 1) ? kHigh : kLow) || w[2] != ((ft[k] & 2) ? kHigh : kLow))
                        return fail("selectors", t, k);
                } else if (w[0] | w[1] | w[2]) {
                    return fail("padding slot", t, k);
                }
            }
            // box semantics against plain walks
            for (int q = 0; q < 200; ++q) {
                float x[4] = {(float)(1000 + below(1001)), (float)below(70001), (float)below(301), (float)(1 + below(8))};
                if (q % 7 == 0) x[0] = (float)(lo[0] + (hi[0] - lo[0]) * uniform());
                const int64_t L = walk(ft, th, depth, x);
                const tl::host::Box& b = boxes[(size_t)(t * n_leaf + L)];
                if (!in_float_box(b, x[1], x[2])) return fail("walked row outside its leaf's box", t, L);
                ++rows_checked;
                uint32_t bw[2];
                std::memcpy(bw, r + R.boxes + 8 * L, 8);
                const uint32_t klo = bw[0] & tl::kBoxKvMax, khi = bw[1] & tl::kBoxKvMax;
                const uint32_t blo = bw[0] >> 20, bhi = bw[1] >> 20;
                for (int m = 0; m < 8; ++m) {
                    float y[4] = {x[0], x[1], x[2], x[3]};
                    if (m & 1) {   // a row inside the packed box, as the kernels decode it
                        if (klo >= khi || blo >= bhi) break;
                        y[1] = (float)(klo + (uint32_t)below((int64_t)(khi - klo)));
                        y[2] = (float)(blo + (uint32_t)below((int64_t)(bhi - blo)));
                        if (!(y[1] >= (float)klo && y[1] < (float)khi)) return fail("packed box decode", t, L);
                    } else {       // a row inside the float box
                        const double a = std::isfinite(b.kv_lo) ? b.kv_lo : -5.0;
                        const double c = std::isfinite(b.kv_hi) ? b.kv_hi : 80000.0;
                        const double d = std::isfinite(b.batch_lo) ? b.batch_lo : -5.0;
                        const double e = std::isfinite(b.batch_hi) ? b.batch_hi : 400.0;
                        y[1] = (float)std::ceil(a + (c - a) * uniform());
                        y[2] = (float)std::ceil(d + (e - d) * uniform());
                        if (!in_float_box(b, y[1], y[2])) continue;
                    }
                    if (walk(ft, th, depth, y) != L) return fail("row inside the box reaches another leaf", t, L);
                    ++inside_checked;
                }
            }
        }
        for (int fi = 1; fi <= 2; ++fi) {
            const std::vector<float> c = tl::host::threshold_cuts(n_trees * n_int, feature.data(), threshold.data(), fi);
            if ((int64_t)c.size() > tl::kMaxCuts) return fail("too many cuts", fi, (long long)c.size());
            for (size_t i = 0; i < c.size(); ++i) {
                if (!std::isfinite(c[i])) return fail("cut not finite", fi, (long long)i);
                if (i && c[i] < c[i - 1]) return fail("cuts not ascending", fi, (long long)i);
            }
            if (!c.empty()) mix(c.data(), c.size() * sizeof(float));
        }
    }
    // box_bound at the edges
    const float probes[] = {-INFINITY, -1.5f, -0.f, 0.f, 0.5f, 1.f, 1048574.5f, 1048575.f, 2e9f, INFINITY};
    for (float p : probes) {
        const uint32_t v = tl::host::box_bound(p, tl::kBoxKvMax);
        mix(&v, 4);
        if (v > tl::kBoxKvMax) return fail("box_bound above its maximum", -1, (long long)v);
    }
    std::printf("host_forest ok rows=%lld inside=%lld checksum=%016llx\n", rows_checked, inside_checked,
                (unsigned long long)g_hash);
    return 0;
}
