// Node walks over tree records staged in LDS and leaf-box tests, shared by
// the forest kernels.
// A record node is (threshold, sel1, sel2, sel3): the byte-permute selectors
// that pick the tested feature out of the row (see node_feature); internal
// nodes sit in heap order 16 bytes apart from the record's start.
#pragma once

#include "device_util.h"
#include "tl_internal.h"

namespace tl {
namespace {

// The value of the feature a record node tests, picked with byte permutes:
// node = (threshold, sel_lo, sel_hi, leaf value); sel_lo picks frequency or
// KV and, with the same selector, batch or engine size; sel_hi picks between
// the two (v_perm_b32: selector 0x03020100 keeps the second operand,
// 0x07060504 takes the first).
template <int NF>
__device__ __forceinline__ float node_feature(const uint4& nd, float xf, float kv, float bs, float xe) {
    const uint32_t x01 = __builtin_amdgcn_perm(__float_as_uint(kv), __float_as_uint(xf), nd.y);
    const uint32_t x23 = NF == 4 ? __builtin_amdgcn_perm(__float_as_uint(xe), __float_as_uint(bs), nd.y)
                                 : __float_as_uint(bs);
    return __uint_as_float(__builtin_amdgcn_perm(x23, x01, nd.z));
}

// Whether (kv, batch) lies in a leaf box (kv_lo, kv_hi, batch_lo, batch_hi).
__device__ __forceinline__ bool in_box(const float4& b, float kv, float bs) {
    return (kv >= b.x) & (kv < b.y) & (bs >= b.z) & (bs < b.w);
}

// The intersection of two decoded leaf boxes.  Their bounds are
// non-negative integers as floats, whose bit patterns order like the values,
// so an integer max / min (one instruction each; fmaxf / fminf would first
// canonicalize both operands) gives the float max / min exactly.
__device__ __forceinline__ float bound_max(float a, float b) {
    return __int_as_float(max(__float_as_int(a), __float_as_int(b)));
}
__device__ __forceinline__ float bound_min(float a, float b) {
    return __int_as_float(min(__float_as_int(a), __float_as_int(b)));
}
__device__ __forceinline__ float4 box_meet(const float4& a, const float4& b) {
    return make_float4(bound_max(a.x, b.x), bound_min(a.y, b.y), bound_max(a.z, b.z), bound_min(a.w, b.w));
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) const u32x4 lds_u32x4;
typedef __attribute__((address_space(3))) const u32x2 lds_u32x2;
typedef __attribute__((address_space(3))) const float lds_f32;

// LDS byte address of a location in the kernel's dynamic LDS.
__device__ __forceinline__ uint32_t lds_addr(const unsigned char* p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const unsigned char*)p;
}

// The node slot at LDS byte address `a`, (threshold, sel_lo, sel_hi, leaf
// value), read whole (a 12-byte read of the node alone measured slower).
__device__ __forceinline__ uint4 read_node(uint32_t a) {
    const u32x4 w = *(lds_u32x4*)(uintptr_t)a;
    return make_uint4(w.x, w.y, w.z, w.w);
}

// A leaf reached by a walk, as the LDS byte addresses of its value and of
// its box.
struct LeafAt {
    uint32_t value, box;
};

// The leaf at which a walk of the staged tree whose record starts at LDS
// byte address `tree` ended, from the walk's final address a = tree +
// 16 (n_int + L) (heap slot n_int + L, leaf L): its value is word 3 of node
// slot L, i.e. at a - 16 n_int + 12, and its box at tree + boxes + 8 L =
// a / 2 + (tree / 2 + boxes - 8 n_int) (tree and a are multiples of 16).
__device__ __forceinline__ LeafAt leaf_at(uint32_t a, uint32_t tree, const RecordLayout& R, int32_t depth) {
    const uint32_t n_int16 = 16u * ((1u << depth) - 1u);
    return LeafAt{a - (n_int16 - 12u), (a >> 1) + ((tree >> 1) + R.boxes - n_int16 / 2u)};
}

// The value of a leaf.
__device__ __forceinline__ float leaf_value(const LeafAt& l) {
    return *(lds_f32*)(uintptr_t)l.value;
}

// The KV / batch box of a leaf, decoded from its packed integer bounds into
// (kv_lo, kv_hi, batch_lo, batch_hi) as floats (exact: all bounds are below
// 2^24).
__device__ __forceinline__ float4 leaf_box(const LeafAt& l) {
    const u32x2 w = *(lds_u32x2*)(uintptr_t)l.box;
    return make_float4((float)(w.x & kBoxKvMax), (float)(w.y & kBoxKvMax), (float)(w.x >> 20),
                       (float)(w.y >> 20));
}

// Staging of tree blocks: block b is trees [b*tb, b*tb + cnt), one
// contiguous range of 16-byte words in global memory and in LDS.  It is
// copied in pieces of 64 lanes x 16 bytes straight from global memory into
// LDS (global_load_lds_dwordx4, no registers), wavefront w of n taking
// pieces w, w + n, ... (n = 1: one wavefront copies it all).  Lanes past the
// block's last word copy its first word into the buffer's padding (buffers
// are whole pieces), so no lane writes outside its buffer.
constexpr uint32_t kStagePiece = kWave * 16;

__host__ __device__ inline uint32_t stage_buffer_bytes(int32_t tb, const RecordLayout& R) {
    return ((uint32_t)tb * R.bytes + kStagePiece - 1) / kStagePiece * kStagePiece;
}

// One piece: lane l copies the 16 bytes at its `src` to LDS byte address
// lds + 16 l (lds the same in every lane).  Issued as an instruction the
// compiler does not track, so it does not make the evaluation's LDS reads
// wait for the copy (they read other buffers); a kernel waits for its copies
// (vmcnt) before it hands the buffer over (a workgroup barrier, or
// publishing `ready` in stage_acquire), and has no other vector-memory load
// in flight inside its block loop.
__device__ __forceinline__ void stage_piece(const uint4* src, uint32_t lds) {
    const uint32_t base = __builtin_amdgcn_readfirstlane(lds);   // wavefront-uniform by construction
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(base), "v"(src) : "memory", "m0");
}

// Enqueues this wavefront's pieces of block b (rec_words 16-byte words per
// tree) into the LDS buffer at byte address dst.
__device__ __forceinline__ void stage_block(const uint4* records, int32_t n_trees, int32_t tb, uint32_t rec_words,
                                            int32_t b, uint32_t dst, int wave, int n_waves) {
    const uint32_t words = (uint32_t)min(tb, n_trees - b * tb) * rec_words;
    const uint4* src = records + (int64_t)b * tb * rec_words;
    const uint32_t n_pieces = (words + kWave - 1) / kWave;
    for (uint32_t pc = (uint32_t)wave; pc < n_pieces; pc += (uint32_t)n_waves) {
        const uint32_t i = pc * kWave + lane_id();
        stage_piece(src + (i < words ? i : 0u), dst + pc * kStagePiece);
    }
}

// Hand-over of NB LDS buffers of tree blocks between the wavefronts of a
// workgroup without block barriers.  Block b lives in buffer b % NB; block 0
// is copied by every wavefront before the workgroup's one barrier.  Per
// buffer: `claimed` = the last block a wavefront took on to copy into it,
// `ready` = the last block whose copy is complete, `done` = how many
// (wavefront, block) pairs have finished with it.  The first wavefront that
// needs block b and finds it unclaimed claims it, waits until every
// wavefront has finished block b - NB (the buffer's previous occupant),
// copies the whole block, waits for its copy and publishes `ready`; the others
// wait for `ready`.  A wavefront can thus run up to NB - 1 blocks ahead of the
// slowest one instead of meeting it at every block.  Issue priority follows
// the order in which wavefronts finish a block: the later a wavefront leaves
// block b among its workgroup's, the higher its priority (s_setprio) while it
// evaluates block b + 1, and a wavefront that arrives at a block before its
// copy is there drops to the lowest; the oldest wavefronts of a SIMD would
// otherwise keep winning issue and the youngest set the pace.  Every wait is
// bounded (kSyncSpins sleeps); one that runs out makes stage_acquire return
// false, and the caller marks its results invalid, so every wavefront ends.
constexpr int kMaxStageBuffers = 3;
struct StageSync {
    int32_t claimed[kMaxStageBuffers];
    int32_t ready[kMaxStageBuffers];
    int32_t done[kMaxStageBuffers];
};
constexpr int32_t kSyncSpins = 1 << 20;

template <int NB = 2>
__device__ __forceinline__ void stage_sync_init(StageSync* sync) {
    sync->claimed[0] = 0;   // block 0: copied by every wavefront
    sync->ready[0] = 0;
    sync->done[0] = 0;
    for (int i = 1; i < NB; ++i) {
        sync->claimed[i] = i - NB;   // block i claims buffer i from "block i - NB"
        sync->ready[i] = -1;
        sync->done[i] = 0;
    }
}

__device__ __forceinline__ int32_t sync_load(const int32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Makes block b >= 1 (trees [b*tb, ...), rec_words 16-byte words per tree)
// available in its buffer at LDS byte address buf; n_waves wavefronts share
// the buffers.
template <int NB = 2>
__device__ __forceinline__ bool stage_acquire(StageSync* sync, int32_t b, int n_waves, const uint4* records,
                                              int32_t n_trees, int32_t tb, uint32_t rec_words, uint32_t buf) {
    const int cur = b % NB;
    const int32_t need_done = n_waves * (b / NB);
    int32_t spins = 0;
    if (sync_load(&sync->ready[cur]) != b) __builtin_amdgcn_s_setprio(0);   // ahead of the others
    while (sync_load(&sync->ready[cur]) != b && spins < kSyncSpins) {
        int32_t won = 0;
        if (sync_load(&sync->claimed[cur]) == b - NB) {
            if (lane_id() == 0) {
                int32_t expect = b - NB;
                won = __hip_atomic_compare_exchange_strong(&sync->claimed[cur], &expect, b, __ATOMIC_ACQ_REL,
                                                           __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
            }
            won = __builtin_amdgcn_readfirstlane(won);
        }
        if (won) {
            while (sync_load(&sync->done[cur]) < need_done && spins < kSyncSpins) {
                __builtin_amdgcn_s_sleep(1);
                ++spins;
            }
            stage_block(records, n_trees, tb, rec_words, b, buf, 0, 1);
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            if (lane_id() == 0) __hip_atomic_store(&sync->ready[cur], b, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
            break;
        }
        __builtin_amdgcn_s_sleep(1);
        ++spins;
    }
    return spins < kSyncSpins;
}

// This wavefront has finished with block b (its reads have all returned);
// n_waves share the buffers.
template <int NB = 2>
__device__ __forceinline__ void stage_release(StageSync* sync, int32_t b, int n_waves) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    int32_t before = 0;
    if (lane_id() == 0)
        before = __hip_atomic_fetch_add(&sync->done[b % NB], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    // how many wavefronts left block b before this one, in quarters
    const int32_t quarter = 4 * (__builtin_amdgcn_readfirstlane(before) % n_waves) / n_waves;
    if (quarter == 3) __builtin_amdgcn_s_setprio(3);
    else if (quarter == 2) __builtin_amdgcn_s_setprio(2);
    else if (quarter == 1) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(0);
}

// Walks NT consecutive staged trees (records R.bytes apart, the first at
// LDS byte address `tree`) from the root for one row; lf[t] = the leaf
// reached in tree t.  The walks of two trees interleave, so their chains of
// dependent LDS reads overlap.
template <int NF, int NT>
__device__ __forceinline__ void walk(uint32_t tree, const RecordLayout& R, int32_t depth, float xf, float kv, float bs,
                                     float xe, LeafAt (&lf)[NT]) {
    const uint32_t rec_bytes = R.bytes;
    // the loop carries node byte addresses: child 2k+1 of the node at
    // a = root + 16 k sits at 2 a + (16 - root), child 2k+2 16 bytes later
    uint32_t a[NT], cl[NT], cr[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        a[t] = tree + t * rec_bytes;
        cl[t] = 16u - a[t];
        cr[t] = 32u - a[t];
        // opaque to the optimizer, which would otherwise rewrite the select
        // of the two offsets as an add after the compare
        asm volatile("" : "+v"(cl[t]), "+v"(cr[t]));
    }
    for (int32_t level = 0; level < depth; ++level) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const uint4 nd = read_node(a[t]);
            const bool left = node_feature<NF>(nd, xf, kv, bs, xe) < __uint_as_float(nd.x);
            a[t] = 2u * a[t] + (left ? cl[t] : cr[t]);
        }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) lf[t] = leaf_at(a[t], tree + t * rec_bytes, R, depth);
}

}  // namespace
}  // namespace tl
