// Stage 1: KV usage and batch-size projection (Sec. 4.2, Eq. 1-2) with FIFO
// admission of queued requests under the KV check of Sec. 4.3.2.
//
// One 64-lane wavefront per scenario; the per-iteration curves live in LDS.
//
// In-flight requests are turned into O(1) events each instead of O(r) curve
// updates.  For a request with c cached tokens active on [0, e):
//   KV_i[j] = ceil((c + j) / N)   (Eq. 1 with j - s_i = g_i + j)
// starts at ceil(c / N), grows by one block at every j >= 1 with
// c + j == 1 (mod N) -- a comb of period N beginning at j0 -- and drops to 0
// at e.  So KV = prefix-sum over j of
//   (jumps at 0 and e)  +  C[j],  C[j] = C[j - N] + comb_diff[j],
// where comb_diff gets +1 at j0 and -1 at the first comb point >= e.  The
// batch curve is the prefix sum of +1 at 0 / -1 at e.  One LDS array holds
// the comb differences, then (scanned in place) C, then C plus the jumps,
// then KV: two H-long int32 arrays per scenario in all, so more scenarios'
// wavefronts share a compute unit.
//
// For admission control a new query can be appended to every scenario as a
// request that starts now (Sec. 4.3.2, the "virtual" scoreboard); it adds
// in-flight events like the others.
//
// Queued requests are admitted in FIFO order by the same wave, each at the
// first iteration from its arrival (and from the previous admission) where
// its KV contribution over its in-horizon lifetime fits under the capacity.
// Admissions only happen after the last iteration at which the in-flight
// batch alone exceeds the capacity, which makes the lifetime check equal to
// checking the whole projected vector from the current iteration on.
// Without a batch cap, up to 64 requests are tried at once at their FIFO
// targets with one check of their summed contribution; when that fails the
// batch shrinks, and below 8 requests a growing number of them are admitted
// one at a time before batching again.
#include "device_util.h"
#include "tl_internal.h"

namespace tl {
namespace {

constexpr uint64_t kNoDeadline = ~0ull;

__device__ __forceinline__ bool entry_ok(int32_t p, int32_t g, int32_t r, int32_t a) {
    return p >= 0 && g >= 0 && r >= 1 && a >= -1 && (int64_t)p + (int64_t)g <= (1ll << 30);
}

// sum of DA[t] for t in (j, j2], j2 < H; every lane returns the same value
__device__ __forceinline__ int32_t sum_range(const int32_t* DA, int32_t j, int32_t j2) {
    if (j2 == j + 1) return __builtin_amdgcn_readfirstlane(DA[j2]);
    int32_t acc = 0;
    for (int32_t t0 = j + 1; t0 <= j2; t0 += kWave) {
        int32_t t = t0 + lane_id();
        acc += (t <= j2) ? DA[t] : 0;
    }
    return wave_sum(acc);
}

// Events of one request that holds c cached tokens now and stays in the batch
// on [0, e), in two parts.  The block comb: +1 at its first new-block
// iteration j0 and -1 at the first comb point at or past e (a stride-N prefix
// scan turns these into the per-iteration increments).  The jumps: batch +1
// at 0 / -1 at e, KV +ceil(c/N) at 0 (counted in kv0) and -KV_i[e-1] at e;
// the request is counted in n_in and n_end.
__device__ __forceinline__ void inflight_comb(int32_t c, int32_t e, int32_t H, int32_t N, const DivU32& divN,
                                              int32_t* X) {
    const int32_t lim = min(e, H);
    const int32_t rc = (int32_t)((uint32_t)c - div_u32((uint32_t)c, divN) * (uint32_t)N);
    const int32_t j0 = (rc == 0) ? 1 : (N + 1 - rc);
    if (j0 < lim) {
        atomicAdd(&X[j0], 1);
        if (e < H) {
            const int32_t jend = j0 + N * (int32_t)ceil_div_u32((uint32_t)(e - j0), divN);
            if (jend < H) atomicAdd(&X[jend], -1);
        }
    }
}

__device__ __forceinline__ void inflight_jumps(int32_t c, int32_t e, int32_t H, const DivU32& divN, int32_t* BI,
                                               int32_t* X, int32_t& n_in, int32_t& kv0, int32_t& n_end) {
    ++n_in;
    kv0 += (int32_t)ceil_div_u32((uint32_t)c, divN);
    n_end = max(n_end, min(e, H));
    if (e < H) {
        atomicAdd(&BI[e], -1);
        atomicAdd(&X[e], -(int32_t)ceil_div_u32((uint32_t)(c + e - 1), divN));
    }
}

// Adds (or, NEG, takes away) the KV blocks ceil((c + t - a) / N) of a request
// with c cached tokens that starts at iteration a (Eq. 1) to KV[t] for every
// t in [a, lim), a <= lim <= H, 64 iterations per step, by LDS adds that
// return nothing.  POW2: N is a power of two no larger than 64 (log2 N =
// divN.l), so the division is a shift and the value grows by exactly 64 / N
// from one step to the next; the whole steps go 2 * UNROLL per loop trip.
// Otherwise every step divides, UNROLL steps per trip.
template <bool NEG, bool POW2, int UNROLL>
__device__ __forceinline__ void add_request(int32_t* KV, int32_t c, int32_t a, int32_t lim, const DivU32& divN) {
    const int lane = lane_id();
    if (POW2) {
        int32_t v = (int32_t)(((uint32_t)c + divN.d - 1u + (uint32_t)lane) >> divN.l);
        if (NEG) v = -v;
        const int32_t step = NEG ? -(kWave >> divN.l) : (kWave >> divN.l);
        int32_t* q = KV + a + lane;
        int32_t n = (int32_t)((uint32_t)(lim - a) / kWave);   // whole steps
        for (; n >= 2 * UNROLL; n -= 2 * UNROLL) {
#pragma unroll
            for (int u = 0; u < 2 * UNROLL; ++u) atomicAdd(q + u * kWave, v + u * step);
            q += 2 * UNROLL * kWave;
            v += 2 * UNROLL * step;
        }
        for (; n > 0; --n) {
            atomicAdd(q, v);
            q += kWave;
            v += step;
        }
        if (lane < ((lim - a) & (kWave - 1))) atomicAdd(q, v);
    } else {
#pragma unroll UNROLL
        for (int32_t t0 = a; t0 < lim; t0 += kWave) {
            const int32_t t = t0 + lane;
            if (t < lim) {
                const int32_t v = (int32_t)ceil_div_u32((uint32_t)(c + t - a), divN);
                atomicAdd(&KV[t], NEG ? -v : v);
            }
        }
    }
}

// Scenario order for long FIFO loops: one wavefront per scenario, whose time
// grows with its number of requests; launched heaviest first, the last
// wavefronts of the grid are short ones instead of whichever came last.  A
// counting sort over kOrderBuckets classes of the request count (six per
// doubling), heaviest class first; the order inside a class is whatever the
// atomics give (each scenario's results do not depend on it).  Workspace:
// the counters, then the order [S].
constexpr int kOrderBuckets = 128;

__device__ __forceinline__ int order_bucket(const int64_t* off, int64_t s) {
    const int64_t n = off[s + 1] - off[s];
    const float c = n > 0 ? (float)n : 0.0f;   // malformed offsets: lightest class
    return kOrderBuckets - 1 - min(kOrderBuckets - 1, (int)(log2f(c + 1.0f) * 6.0f));
}

__global__ __launch_bounds__(kOrderBuckets) void order_clear_kernel(uint32_t* counts) {
    counts[threadIdx.x] = 0;
}

__global__ __launch_bounds__(256) void order_count_kernel(const int64_t* off, int64_t S, uint32_t* counts) {
    const int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (s < S) atomicAdd(&counts[order_bucket(off, s)], 1u);
}

// exclusive prefix of the class counts, in place: each becomes its class's
// first position
__global__ __launch_bounds__(kWave) void order_start_kernel(uint32_t* counts) {
    uint32_t carry = 0;
    for (int i0 = 0; i0 < kOrderBuckets; i0 += kWave) {
        const uint32_t c = counts[i0 + lane_id()];
        const uint32_t incl = (uint32_t)wave_incl_scan((int32_t)c) + carry;
        counts[i0 + lane_id()] = incl - c;
        carry = (uint32_t)__builtin_amdgcn_readlane((int32_t)incl, kWave - 1);
    }
}

__global__ __launch_bounds__(256) void order_place_kernel(const int64_t* off, int64_t S, uint32_t* counts,
                                                          int32_t* order) {
    const int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (s < S) order[atomicAdd(&counts[order_bucket(off, s)], 1u)] = (int32_t)s;
}

// Smallest batch of queued requests tried at once (no batch cap): below it the
// admission loop takes requests one at a time.
constexpr int32_t kMinBatch = 8;

// BD_LDS: the batch difference array lives in LDS beside the KV curve, as a
// batch cap needs (the admission loop reads its running sums).  Without a
// cap it is only added to and finally prefix-summed, so it accumulates with
// atomics in the scenario's own batch output row instead: half the LDS, twice
// the scenario wavefronts per CU.
template <bool BD_LDS, bool POW2>
__global__ __launch_bounds__(64) void project_kernel(ProjectParams P) {
    extern __shared__ int32_t lds[];
    const int32_t H = P.H;
    const int32_t N = P.N;
    const DivU32 divN{(uint32_t)N, P.div_m, P.div_l};
    const int lane = lane_id();
    const int64_t s = P.order_ws ? (int64_t)((const int32_t*)P.order_ws + kOrderBuckets)[blockIdx.x] : blockIdx.x;
    int32_t* outB = P.batch + s * H;
    int32_t* KV = lds;                      // comb diff, comb prefix, + jumps, then KV values
    int32_t* BI = BD_LDS ? lds + H : outB;  // batch difference array
    int32_t* outKV = P.kv + s * H;
    uint64_t* outDL = P.deadline_at + s * H;

    for (int32_t t = lane; t < H; t += kWave) {
        KV[t] = 0;
        BI[t] = 0;
        outDL[t] = kNoDeadline;
    }
    __threadfence();
    __syncthreads();

    const int64_t lo = P.off[s];
    const int64_t hi = P.off[s + 1];
    const bool bad_range = lo < 0 || hi < lo || hi > P.n_requests || hi - lo > 0x7fffffffll;

    // pass A: validity, size guard, lost / queue information
    uint64_t bound = 0;
    uint32_t fl = 0;
    int32_t has_queue = 0;
    if (!bad_range) {
        int32_t arr_carry = -1;
        for (int64_t base = lo; base < hi; base += kWave) {
            const int64_t i = base + lane;
            const bool in = i < hi;
            int32_t p = 0, g = 0, r = 0, a = -1;
            if (in) { p = P.prompt[i]; g = P.gen[i]; r = P.rem[i]; a = P.arr[i]; }
            const bool ok = in && entry_ok(p, g, r, a);
            if (in && !ok) fl |= TL_FLAG_BAD_REQUEST;
            if (ok) bound += ceil_div_u32((uint32_t)(p + g + H), divN);
            if (ok && a == -1 && P.lost && P.lost[i]) fl |= TL_FLAG_LOST;
            const bool queued = ok && a >= 0;
            if (queued && a < H) has_queue = 1;
            // queue order: each queued arrival must be >= every earlier one
            const int32_t v = queued ? a : -1;
            const int32_t incl = wave_incl_max(v);
            const int32_t excl = max(wave_shift_up1(incl, -1), arr_carry);
            if (queued && a < excl) fl |= TL_FLAG_UNSORTED;
            arr_carry = max(arr_carry, lane63(incl));
        }
    }
    // the appended query (admission control): one more request that starts
    // now; a malformed one is left out and flagged
    int32_t cand_p = 0, cand_l = 0;
    bool cand = false;
    if (P.cand_len && !bad_range) {
        cand_p = P.cand_prompt[s];
        cand_l = P.cand_len[s];
        cand = entry_ok(cand_p, 0, cand_l, -1);
        if (!cand) fl |= TL_FLAG_BAD_CANDIDATE;
        else if (lane == 0) bound += ceil_div_u32((uint32_t)(cand_p + H), divN);
    }
    bound = wave_sum_u64(bound);
    fl = wave_or(fl);
    has_queue = wave_max(has_queue);

    if (bad_range || bound > 0x7fffffffull) {
        for (int32_t t = lane; t < H; t += kWave) { outB[t] = 0; outKV[t] = 0; }
        if (lane == 0) {
            P.n_iters[s] = 0;
            P.flags[s] = bad_range ? TL_FLAG_OVERFLOW : ((fl & TL_FLAG_BAD_REQUEST) | TL_FLAG_OVERFLOW);
        }
        return;
    }

    // pass B1: the in-flight requests' block combs, then their stride-N
    // prefix in place (every later write adds to it)
    for (int64_t base = lo; base < hi; base += kWave) {
        const int64_t i = base + lane;
        if (i >= hi) continue;
        const int32_t p = P.prompt[i], g = P.gen[i], r = P.rem[i], a = P.arr[i];
        if (!entry_ok(p, g, r, a) || a != -1) continue;
        inflight_comb(p + g, r, H, N, divN, KV);
    }
    if (cand && lane == 0) inflight_comb(cand_p, cand_l, H, N, divN, KV);
    __syncthreads();
    {
        const int32_t lane_mod = lane % N;
        for (int32_t t0 = 0; t0 < H; t0 += kWave) {
            const int32_t t = t0 + lane;
            const bool in = t < H;
            int32_t c = in ? KV[t] : 0;
            for (int32_t d = N; d < kWave; d <<= 1) {
                const int32_t u = __shfl_up(c, d);
                if (lane >= d) c += u;
            }
            const int32_t prev = t0 + lane_mod - N;
            if (prev >= 0 && in) c += KV[prev];
            if (in) KV[t] = c;
        }
    }
    __syncthreads();

    // pass B2: jumps, batch events, deadline checkpoints
    int32_t n_end = 0, n_in = 0, kv0 = 0;
    for (int64_t base = lo; base < hi; base += kWave) {
        const int64_t i = base + lane;
        if (i >= hi) continue;
        const int32_t p = P.prompt[i], g = P.gen[i], r = P.rem[i], a = P.arr[i];
        if (!entry_ok(p, g, r, a) || a != -1) continue;
        const int32_t e = r;
        inflight_jumps(p + g, e, H, divN, BI, KV, n_in, kv0, n_end);
        const bool is_lost = P.lost && P.lost[i];
        const uint64_t d = P.deadline ? P.deadline[i] : kNoDeadline;
        if (e <= H && !is_lost && d != kNoDeadline) atomicMin((unsigned long long*)&outDL[e - 1], (unsigned long long)d);
    }
    if (cand && lane == 0) inflight_jumps(cand_p, cand_l, H, divN, BI, KV, n_in, kv0, n_end);
    n_in = wave_sum(n_in);
    kv0 = wave_sum(kv0);
    n_end = wave_max(n_end);
    if (lane == 0) {
        if (BD_LDS) BI[0] += n_in;
        else atomicAdd(&BI[0], n_in);
        KV[0] += kv0;
    }
    __syncthreads();

    // the KV prefix sum; last over-capacity iteration.  The batch curve stays
    // a difference array: admissions add their +1 / -1 to it and the output
    // takes its prefix sum.
    const int32_t cap = P.kv_cap[s];
    // bound (pass A) is at least the KV of every iteration: when it fits the
    // capacity, no admission check can fail and the checks are skipped
    const bool kv_fits = cap >= 0 && bound <= (uint64_t)cap;
    int32_t last_over = -1;
    {
        int32_t carry_kv = 0;
        for (int32_t t0 = 0; t0 < H; t0 += kWave) {
            const int32_t t = t0 + lane;
            const bool in = t < H;
            const int32_t y = wave_incl_scan(in ? KV[t] : 0) + carry_kv;
            carry_kv = __builtin_amdgcn_readlane(y, kWave - 1);
            if (in) {
                KV[t] = y;
                if (y > cap) last_over = t;
            }
        }
    }
    last_over = wave_max(last_over);
    const bool has_bcap = BD_LDS && P.batch_cap != nullptr;   // (the host takes BD_LDS with a cap)
    const int32_t bcap = has_bcap ? P.batch_cap[s] : 0;
    if (last_over >= 0 || (has_bcap && n_in > bcap)) fl |= TL_FLAG_OVERCOMMIT;

    // FIFO admission of queued requests.  One wave does it; every value the
    // loop carries (iteration j, batch size, the head's fields, check
    // outcomes) is wave-uniform and kept in scalar registers.  LDS accesses
    // of one wave are processed in order, so one lane's updates are seen by
    // the later reads of every lane.
    int32_t* BD = BI;   // batch differences: in-flight requests, then admitted ones
    if (has_queue) {
        __syncthreads();
        int32_t j = 0;
        int32_t run = 0;    // batch size at j (prefix of BD; kept only under a batch cap)
        if (has_bcap) run = __builtin_amdgcn_readfirstlane(BD[0]);
        int32_t bsz = kWave;   // requests tried as one batch (no batch cap)
        int32_t seq_left = 0;  // one-at-a-time admissions before the next batch try
        int32_t backoff = 1;   // ... after the next run of failed batches
        int64_t cb = lo - kWave;
        int32_t q_arr = 0, q_c = 0, q_len = 0, q_lost = 0;
        uint64_t q_dl = kNoDeadline;
        uint64_t mask = 0;
        for (;;) {
            while (mask == 0) {
                cb += kWave;
                if (cb >= hi) break;
                const int64_t i = cb + lane;
                bool q = false;
                if (i < hi) {
                    q_arr = P.arr[i];
                    const int32_t p = P.prompt[i], g = P.gen[i];
                    q_len = P.rem[i];
                    q = entry_ok(p, g, q_len, q_arr) && q_arr >= 0;
                    q_c = p + g;
                    q_lost = P.lost ? P.lost[i] : 0;
                    q_dl = P.deadline ? P.deadline[i] : kNoDeadline;
                }
                mask = __ballot(q);
            }
            if (mask == 0) break;

            if (!has_bcap && bsz > 1 && seq_left == 0) {
                // Batched admission of the next bsz queued requests, each at
                // its FIFO target: the running maximum of the arrivals, from
                // max(j, last_over + 1).  Their summed contribution is added
                // to the KV curve and checked once.  If the sum fits
                // everywhere, so does every request's own check at its target
                // (each sees the KV of the requests before it, which is no
                // more than the sum): these are exactly the admissions the
                // one-at-a-time loop makes.  Otherwise the contributions are
                // taken out again and fewer are tried.
                const int32_t lo_j = max(j, last_over + 1);
                const uint32_t below = __builtin_amdgcn_mbcnt_hi(
                    (uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                const bool mem = ((mask >> lane) & 1) && (int32_t)below < bsz;
                const int32_t a = wave_incl_max(mem ? max(q_arr, lo_j) : -1);
                const uint64_t memm = __ballot(mem);
                const uint64_t over = __ballot(mem && a >= H);
                const uint64_t take = over ? (memm & ((over & (~over + 1)) - 1)) : memm;
                if (take == 0) break;   // the head cannot start within the horizon
                // each member's in-horizon end, on its own lane
                const int32_t lim_l = q_len >= H - a ? H : a + q_len;
                const int32_t r_end = wave_max(((take >> lane) & 1) ? lim_l : 0);
                for (uint64_t mm = take; mm; mm &= mm - 1) {
                    const int m = __ffsll((unsigned long long)mm) - 1;
                    const int32_t am = __builtin_amdgcn_readlane(a, m);
                    const int32_t cm = __builtin_amdgcn_readlane(q_c, m);
                    const int32_t lim = __builtin_amdgcn_readlane(lim_l, m);
                    // LDS adds without a returned value: no wait per chunk
                    add_request<false, POW2, 1>(KV, cm, am, lim, divN);
                }
                const int32_t a_first = __builtin_amdgcn_readlane(a, __ffsll((unsigned long long)take) - 1);
                bool bad = false;
                if (!kv_fits) {
                    int32_t t0 = a_first;
#pragma unroll 4
                    for (; t0 + kWave <= r_end; t0 += kWave) bad |= KV[t0 + lane] > cap;
                    if (t0 + lane < r_end) bad |= KV[t0 + lane] > cap;
                }
                const bool fits = __ballot(bad) == 0;
                if (!fits) {
                    // take the batch's contributions out again
                    for (uint64_t mm = take; mm; mm &= mm - 1) {
                        const int m = __ffsll((unsigned long long)mm) - 1;
                        const int32_t am = __builtin_amdgcn_readlane(a, m);
                        const int32_t cm = __builtin_amdgcn_readlane(q_c, m);
                        const int32_t lim = __builtin_amdgcn_readlane(lim_l, m);
                        add_request<true, POW2, 1>(KV, cm, am, lim, divN);
                    }
                    // shrink the batch; once down to single requests, admit
                    // a growing number of them one at a time before batching
                    // again (the capacity binds)
                    bsz >>= 2;
                    if (bsz < kMinBatch) {
                        bsz = kMinBatch;
                        seq_left = backoff;
                        backoff = min(2 * backoff, 256);
                    }
                    continue;
                }
                if ((take >> lane) & 1) {
                    const int64_t e = (int64_t)a + q_len;
                    atomicAdd(&BD[a], 1);
                    if (e < H) atomicAdd(&BD[e], -1);
                    if (e <= H && !q_lost && q_dl != kNoDeadline)
                        atomicMin((unsigned long long*)&outDL[e - 1], (unsigned long long)q_dl);
                }
                n_end = max(n_end, r_end);
                j = __builtin_amdgcn_readlane(a, 63 - __clzll((long long)take));
                mask &= ~take;
                bsz = min(kWave, 2 * bsz);
                backoff = 1;
                if (over) break;
                continue;
            }

            // One request at a time (under a batch cap, or after batches
            // failed).  The head of the queue: uniform lane, lane reads.
            const int hl = __ffsll((unsigned long long)mask) - 1;
            const int32_t h_arr = __builtin_amdgcn_readlane(q_arr, hl);
            const int32_t h_c = __builtin_amdgcn_readlane(q_c, hl);
            const int32_t h_len = __builtin_amdgcn_readlane(q_len, hl);
            const int32_t h_lost = __builtin_amdgcn_readlane(q_lost, hl);
            const uint64_t h_dl =
                ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int32_t)(q_dl >> 32), hl) << 32) |
                (uint32_t)__builtin_amdgcn_readlane((int32_t)(uint32_t)q_dl, hl);
            const int32_t target = max(max(h_arr, j), last_over + 1);
            if (h_arr >= H || target >= H) break;
            if (has_bcap && target > j) run += sum_range(BD, j, target);
            j = target;
            bool admitted = false;
            for (;;) {
                bool ok = !has_bcap || run < bcap;
                int32_t t_bad = -1;
                if (ok) {
                    // 4 x 64 iterations per round (their LDS reads in flight
                    // together); the earliest overflowing iteration wins
                    const int32_t lim = kv_fits ? j : (int32_t)min((int64_t)j + h_len, (int64_t)H);
                    for (int32_t t0 = j; t0 < lim && t_bad < 0; t0 += 4 * kWave) {
                        uint64_t m[4];
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            const int32_t t = t0 + k * kWave + lane;
                            bool badt = false;
                            if (t < lim)
                                badt = KV[t] + (int32_t)(POW2 ? ((uint32_t)(h_c + t - j) + divN.d - 1u) >> divN.l
                                                              : ceil_div_u32((uint32_t)(h_c + t - j), divN)) > cap;
                            m[k] = __ballot(badt);
                        }
#pragma unroll
                        for (int k = 3; k >= 0; --k)
                            if (m[k]) t_bad = t0 + k * kWave + __ffsll((unsigned long long)m[k]) - 1;
                    }
                    ok = t_bad < 0;
                }
                if (ok) { admitted = true; break; }
                if (has_bcap && run >= bcap) {
                    // The batch is full: the next start to try is the first
                    // later iteration with a free slot, found 64 iterations
                    // at a time from the batch differences (what stepping
                    // one iteration at a time reaches).
                    int32_t base = j, r = run, found = -1;
                    while (base + 1 < H) {
                        const int32_t t = base + 1 + lane;
                        const int32_t pre = wave_incl_scan(t < H ? BD[t] : 0) + r;   // batch size at t
                        const uint64_t m = __ballot(t < H && pre < bcap);
                        if (m) {
                            const int l = __ffsll((unsigned long long)m) - 1;
                            found = base + 1 + l;
                            r = __builtin_amdgcn_readlane(pre, l);
                            break;
                        }
                        r = __builtin_amdgcn_readlane(pre, kWave - 1);
                        base += kWave;
                    }
                    if (found < 0) break;
                    run = r;
                    j = found;
                    continue;
                }
                // Next start to try.  If iteration t_bad overflowed, every
                // start j2 in (j, t_bad] whose own contribution there,
                // ceil((c + t_bad - j2) / N), exceeds room = cap - KV[t_bad]
                // fails the same way: j2 < c + t_bad - N * room (all of
                // them when room < 0).  Skipping those gives the same
                // admission iteration.
                int32_t nj = j + 1;
                if (t_bad >= 0) {
                    const int32_t room = cap - __builtin_amdgcn_readfirstlane(KV[t_bad]);
                    int64_t first = (int64_t)t_bad + 1;
                    if (room >= 0) first = min(first, (int64_t)h_c + t_bad - (int64_t)N * room);
                    nj = (int32_t)max((int64_t)nj, first);
                }
                if (nj >= H) break;
                if (has_bcap) run += sum_range(BD, j, nj);
                j = nj;
            }
            if (!admitted) break;
            const int64_t e = (int64_t)j + h_len;
            const int32_t lim = (int32_t)min(e, (int64_t)H);
            add_request<false, POW2, 4>(KV, h_c, j, lim, divN);
            if (lane == 0) {
                if (BD_LDS) {
                    BD[j] += 1;
                    if (e < H) BD[e] -= 1;
                } else {
                    atomicAdd(&BD[j], 1);
                    if (e < H) atomicAdd(&BD[e], -1);
                }
                if (e <= H && !h_lost && h_dl != kNoDeadline)
                    atomicMin((unsigned long long*)&outDL[e - 1], (unsigned long long)h_dl);
            }
            run += 1;
            n_end = max(n_end, lim);
            mask &= mask - 1;
            if (seq_left > 0) --seq_left;
        }
    }
    __syncthreads();

    // outputs: curves (batch = prefix sum of BD), scalars
    if (BD_LDS) {
        int32_t carry_b = 0;
        for (int32_t t0 = 0; t0 < H; t0 += kWave) {
            const int32_t t = t0 + lane;
            const bool in = t < H;
            const int32_t b = wave_incl_scan(in ? BD[t] : 0) + carry_b;
            carry_b = __builtin_amdgcn_readlane(b, kWave - 1);
            if (!in) continue;
            const int32_t k = KV[t];
            outB[t] = b;
            outKV[t] = k;
        }
    } else {
        // the differences were added at L2 by atomics: read them there,
        // eight 64-iteration chunks in flight at a time, then scan
        constexpr int kChunks = 8;
        int32_t carry_b = 0;
        for (int32_t g0 = 0; g0 < H; g0 += kChunks * kWave) {
            int32_t d[kChunks];
#pragma unroll
            for (int c = 0; c < kChunks; ++c) {
                const int32_t t = g0 + c * kWave + lane;
                d[c] = t < H ? __hip_atomic_load(&BD[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
            }
#pragma unroll
            for (int c = 0; c < kChunks; ++c) {
                const int32_t t = g0 + c * kWave + lane;
                const int32_t b = wave_incl_scan(d[c]) + carry_b;
                carry_b = __builtin_amdgcn_readlane(b, kWave - 1);
                if (t < H) {
                    outB[t] = b;
                    outKV[t] = KV[t];
                }
            }
        }
    }
    if (lane == 0) {
        P.n_iters[s] = n_end;
        P.flags[s] = fl;
    }
}

// Feature rows of the grid, written out when requested: row (s, f, j) =
// (freq[f], KV[s][j], B[s][j] [, engine[s]]) from the curves project_kernel
// wrote.  One thread per (s, j) writes its F rows with one 16- or 12-byte
// store each; consecutive threads write consecutive rows of one frequency.
constexpr int kRowsThreads = 256;

template <int NF>
__global__ __launch_bounds__(kRowsThreads) void expand_rows_kernel(ProjectParams P) {
    const int32_t H = P.H;
    const int32_t n_jb = (H + kRowsThreads - 1) / kRowsThreads;
    const int64_t s = blockIdx.x / (uint32_t)n_jb;
    const int32_t t = (int32_t)(blockIdx.x % (uint32_t)n_jb) * kRowsThreads + threadIdx.x;
    if (t >= H) return;
    const float kf = (float)P.kv[s * H + t], bf = (float)P.batch[s * H + t];
    const float eng = NF == 4 ? P.engine[s] : 0.0f;
    float* row = P.rows + ((int64_t)s * P.F * H + t) * NF;
    const int64_t f_stride = (int64_t)H * NF;
#pragma unroll 4
    for (int32_t f = 0; f < P.F; ++f) {
        if (NF == 4)
            *(float4*)(row + f * f_stride) = make_float4(P.freqs[f], kf, bf, eng);
        else
            *(float3*)(row + f * f_stride) = make_float3(P.freqs[f], kf, bf);
    }
}

// Remaining-token counts from the predictor's total lengths (Sec. 4.6):
// inflate by num/den (rounded up; den = 0: none), limit to max_tokens, reset
// to max_tokens past an outrun prediction, remaining = max(length - gen, 1);
// malformed entries get 0.  One wavefront per scenario, 64 entries a step.
constexpr int kAdjustWaves = 4;

__global__ __launch_bounds__(kAdjustWaves * kWave) void adjust_kernel(AdjustParams P) {
    const int64_t s = (int64_t)blockIdx.x * kAdjustWaves + threadIdx.x / kWave;
    if (s >= P.S) return;
    const int64_t lo = P.off[s], hi = P.off[s + 1];
    if (lo < 0 || hi < lo || hi > P.n_requests) return;
    const uint32_t num = P.num[s], den = P.den[s];
    const int32_t mt = P.max_tokens[s];
    for (int64_t i = lo + lane_id(); i < hi; i += kWave) {
        const int32_t g = P.gen[i], r = P.pred[i];
        int32_t out = 0;
        if (g >= 0 && r >= 1) {
            int64_t len = r;
            if (den > 0) {
                const uint64_t x = (uint64_t)r * num;
                len = (int64_t)min((x + den - 1) / den, (uint64_t)0x7fffffff);
            }
            if (mt >= 1) {
                len = min(len, (int64_t)mt);
                if (g >= len) len = mt;
            }
            out = (int32_t)max(len - g, (int64_t)1);
        }
        P.out[i] = out;
    }
}

}  // namespace

hipError_t launch_adjust(const AdjustParams& p, hipStream_t stream) {
    if (p.S == 0) return hipSuccess;
    hipLaunchKernelGGL(adjust_kernel, dim3((unsigned)((p.S + kAdjustWaves - 1) / kAdjustWaves)),
                       dim3(kAdjustWaves * kWave), 0, stream, p);
    return hipGetLastError();
}

// Long FIFO loops: no batch cap and on average 1024 or more requests per
// scenario.
bool long_fifo_loops(const ProjectParams& p) {
    return p.batch_cap == nullptr && p.n_requests >= (int64_t)1024 * p.n_scenarios;
}

size_t project_order_bytes(const ProjectParams& p) {
    if (!long_fifo_loops(p) || p.n_scenarios < 2 || p.n_scenarios > 0x7fffffffll) return 0;
    return (size_t)(kOrderBuckets + p.n_scenarios) * sizeof(int32_t);
}

hipError_t launch_project(const ProjectParams& p, hipStream_t stream) {
    // The batch differences go to global memory where occupancy pays (long
    // FIFO loops); otherwise the LDS array is faster.
    const bool bd_lds = !long_fifo_loops(p);
    const size_t lds = (size_t)(bd_lds ? 2 : 1) * p.H * sizeof(int32_t);
    // block sizes that are powers of two up to 64 take shifts instead of
    // divisions in the admission loops
    const bool pow2 = p.N <= kWave && (p.N & (p.N - 1)) == 0;
    void (*const kern)(ProjectParams) = bd_lds ? (pow2 ? project_kernel<true, true> : project_kernel<true, false>)
                                               : (pow2 ? project_kernel<false, true> : project_kernel<false, false>);
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    if (p.order_ws) {
        uint32_t* counts = (uint32_t*)p.order_ws;
        const unsigned nb = (unsigned)((p.n_scenarios + 255) / 256);
        hipLaunchKernelGGL(order_clear_kernel, dim3(1), dim3(kOrderBuckets), 0, stream, counts);
        hipLaunchKernelGGL(order_count_kernel, dim3(nb), dim3(256), 0, stream, p.off, p.n_scenarios, counts);
        hipLaunchKernelGGL(order_start_kernel, dim3(1), dim3(kWave), 0, stream, counts);
        hipLaunchKernelGGL(order_place_kernel, dim3(nb), dim3(256), 0, stream, p.off, p.n_scenarios, counts,
                           (int32_t*)p.order_ws + kOrderBuckets);
        const hipError_t e0 = hipGetLastError();
        if (e0 != hipSuccess) return e0;
    }
    hipLaunchKernelGGL(kern, dim3((unsigned)p.n_scenarios), dim3(64), lds, stream, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !p.rows) return e;
    const int64_t blocks = p.n_scenarios * ((p.H + kRowsThreads - 1) / kRowsThreads);
    if (!grid_fits(blocks)) return hipErrorInvalidConfiguration;
    if (p.nf == 4)
        hipLaunchKernelGGL(expand_rows_kernel<4>, dim3((unsigned)blocks), dim3(kRowsThreads), 0, stream, p);
    else
        hipLaunchKernelGGL(expand_rows_kernel<3>, dim3((unsigned)blocks), dim3(kRowsThreads), 0, stream, p);
    return hipGetLastError();
}

}  // namespace tl
