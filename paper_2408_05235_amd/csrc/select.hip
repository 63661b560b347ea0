// Stage 3: the throttling controller (Sec. 4.5) with the TBT and E2E checks of
// Sec. 4.3.2 (checks 2 and 3, Eq. 3-4).
//
// One 256-thread workgroup per scenario; its four wavefronts take the
// candidate frequencies in rounds of four, lowest first, and the first round
// with a feasible frequency ends the search.  For one frequency a wave walks
// the projected iterations 256 at a time, four consecutive ones per lane:
// per-iteration time in integer ns, the lane's running sum plus an exclusive
// wave scan of lane totals and the carry gives Eq. 3's cumulative time
// T_R[j+1], which is compared with the deadline of requests ending at j.  The
// walk stops at the first violated deadline.
//
// The admission decision of Sec. 4.3.2 and the steps of the paper's binary
// search over frequencies use the same arithmetic at one frequency per
// scenario.
#include "device_util.h"
#include "tl_internal.h"

namespace tl {
namespace {

constexpr uint64_t kNoDeadline = ~0ull;
constexpr uint64_t kSat = 1ull << 40;

// T'_j = 1 / T_j in whole ns, rounded up; IEEE fp64 division
__device__ __forceinline__ uint64_t latency_ns(float ips) {
    if (!(ips > 0.0f)) return kSat;
    const double q = 1e9 / (double)ips;
    if (!(q < 1099511627776.0)) return kSat;
    return (uint64_t)ceil(q);
}

constexpr int kWavesPerBlock = 4;
constexpr int kPerLane = 4;                   // consecutive iterations per lane
constexpr int kStep = kWave * kPerLane;       // iterations per wavefront step

// Eq. 3-4 for one frequency, by one wavefront: per-iteration times of `ips`
// over the n projected iterations, T_R[j+1] < dl[j] for every deadline and
// T_R[n] <= budget.  A lane takes four consecutive iterations: their running
// sum, then one wave scan of the lane totals per 256 iterations.  Stops at
// the first missed deadline.  Every lane returns the same value.
__device__ __forceinline__ bool feasible_wave(const float* ips, const uint64_t* dl, int32_t n, uint64_t budget) {
    const int lane = lane_id();
    uint64_t carry = 0;
    for (int32_t j0 = 0; j0 < n; j0 += kStep) {
        const int32_t jb = j0 + kPerLane * lane;
        uint64_t p[kPerLane];
        uint64_t run = 0;
#pragma unroll
        for (int k = 0; k < kPerLane; ++k) {
            run += (jb + k < n) ? latency_ns(ips[jb + k]) : 0ull;
            p[k] = run;
        }
        const uint64_t before = wave_incl_scan_u64(run) - run + carry;   // T_R[jb]
        bool bad = false;
#pragma unroll
        for (int k = 0; k < kPerLane; ++k) {
            if (jb + k < n) {
                const uint64_t d = dl[jb + k];
                bad |= d != kNoDeadline && !(before + p[k] < d);
            }
        }
        carry = lane63_u64(before + run);
        if (__ballot(bad)) return false;
    }
    return carry <= budget;
}

// The lowest feasible frequency of one scenario.  The four wavefronts of the
// workgroup take frequencies in rounds of four, lowest first; the first
// round with a feasible frequency ends the search (no higher frequency can
// be the minimum).
__global__ __launch_bounds__(256) void select_kernel(SelectParams P) {
    __shared__ uint32_t round_ok;
    const int64_t s = blockIdx.x;
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int32_t F = P.F, H = P.H;
    const uint32_t fl = P.proj_flags ? P.proj_flags[s] : 0u;
    if (fl & (TL_FLAG_OVERFLOW | TL_FLAG_LOST)) {
        if (threadIdx.x == 0) {
            P.freq_idx[s] = F - 1;
            P.status[s] = (fl & TL_FLAG_OVERFLOW) ? TL_STATUS_INVALID : TL_STATUS_LOST;
        }
        return;
    }
    const int32_t n = min(max(P.n_iters[s], 0), H);
    if (n == 0) {
        if (threadIdx.x == 0) {
            P.freq_idx[s] = 0;
            P.status[s] = TL_STATUS_OK;
        }
        return;
    }
    if (threadIdx.x == 0) round_ok = 0;
    __syncthreads();
    const uint64_t slo = P.tbt_slo_ns[s];
    const uint64_t budget = (slo > ~0ull / (uint64_t)n) ? ~0ull : slo * (uint64_t)n;
    const uint64_t* dl = P.deadline_at + s * H;
    int32_t best = -1;
    for (int32_t f0 = 0; f0 < F; f0 += kWavesPerBlock) {
        const int32_t f = f0 + wave;
        const bool ok = f < F && feasible_wave(P.ips + ((int64_t)s * F + f) * H, dl, n, budget);
        if (ok && lane == 0) atomicOr(&round_ok, 1u << wave);
        __syncthreads();
        const uint32_t m = round_ok;
        // every thread has read this round's mask before the next round writes
        __syncthreads();
        if (m) {
            best = f0 + __ffs(m) - 1;
            break;
        }
    }
    if (threadIdx.x == 0) {
        P.freq_idx[s] = best >= 0 ? best : F - 1;
        P.status[s] = best >= 0 ? TL_STATUS_OK : TL_STATUS_INFEASIBLE;
    }
}

// Eq. 3-4 at one frequency for one scenario, by one wavefront: with
// per-iteration times of `ips` over the n projected iterations, returns
// T_R[n] and whether some deadline of `dl` (T_R[j+1] < dl[j]) is missed;
// *miss_own tells whether T_R[own_at + 1] < d_own fails (own_at < 0: none).
// Every lane returns the same values.
__device__ __forceinline__ uint64_t wave_times(const float* ips, const uint64_t* dl, int32_t n, int32_t own_at,
                                               uint64_t d_own, bool* miss, bool* miss_own) {
    const int lane = lane_id();
    uint64_t carry = 0;
    bool m = false, mo = false;
    for (int32_t j0 = 0; j0 < n; j0 += kWave) {
        const int32_t j = j0 + lane;
        const bool in = j < n;
        const uint64_t lat = in ? latency_ns(ips[j]) : 0ull;
        const uint64_t tr = wave_incl_scan_u64(lat) + carry;
        const uint64_t d = in ? dl[j] : kNoDeadline;
        m |= in && d != kNoDeadline && !(tr < d);
        mo |= in && j == own_at && !(tr < d_own);
        carry = lane63_u64(tr);
    }
    *miss = __ballot(m) != 0;
    *miss_own = __ballot(mo) != 0;
    return carry;
}

__device__ __forceinline__ bool within_tbt(uint64_t t_r_n, uint64_t slo, int32_t n) {
    const uint64_t budget = n == 0 ? ~0ull : (slo > ~0ull / (uint64_t)n) ? ~0ull : slo * (uint64_t)n;
    return t_r_n <= budget;
}

// Admission decision (Sec. 4.3.2 checks 1-3) of one new query per scenario
// from the projection with it and M at the maximum frequency: one wavefront
// per scenario; the deadline of the query itself (ending at cand_len, when
// inside the horizon) is checked apart from the scheduled requests'
// deadlines in deadline_at.
constexpr int kAdmitWaves = 4;

__global__ __launch_bounds__(kAdmitWaves * kWave) void admit_kernel(AdmitParams P) {
    const int64_t s = (int64_t)blockIdx.x * kAdmitWaves + threadIdx.x / kWave;
    if (s >= P.S) return;
    const int32_t H = P.H;
    const uint32_t fl = P.proj_flags[s];
    uint32_t dec;
    if (fl & (TL_FLAG_OVERFLOW | TL_FLAG_BAD_CANDIDATE)) {
        dec = TL_ADMIT_INVALID;
    } else if (fl & TL_FLAG_OVERCOMMIT) {
        // the requests running now (the query among them) exceed the KV
        // capacity at some iteration or the batch cap: every value of the
        // projected KV vector is within the capacity otherwise, since queued
        // requests are only admitted where they fit
        dec = TL_ADMIT_QUEUE_CAPACITY;
    } else {
        const int32_t n = min(max(P.n_iters[s], 0), H);
        const int32_t L = P.cand_len[s];
        const uint64_t d_own = P.cand_deadline ? P.cand_deadline[s] : kNoDeadline;
        const int32_t own_at = (d_own != kNoDeadline && L <= H) ? L - 1 : -1;   // T_R[L] = T_R[own_at + 1]
        bool miss, miss_own;
        const uint64_t t_r = wave_times(P.ips + s * H, P.deadline_at + s * H, n, own_at, d_own, &miss, &miss_own);
        if (!within_tbt(t_r, P.tbt_slo_ns[s], n)) dec = TL_ADMIT_QUEUE_TBT;
        else if (miss) dec = TL_ADMIT_QUEUE_E2E;
        else if (miss_own) dec = TL_ADMIT_LOST;
        else dec = TL_ADMIT_OK;
    }
    if (lane_id() == 0) P.decision[s] = dec;
}

// Binary search over the candidate frequencies (Sec. 4.5), one step per
// launch for every scenario.  State per scenario: lo, hi (the search
// interval) and probe (the frequency index M was evaluated at, -1 = none).
// Step: feasible at the probe -> hi = probe, else lo = probe + 1; then the
// next probe is the midpoint while lo < hi.  The last step (final = true)
// checks lo itself and writes the result.  Scenarios flagged overflow / lost
// are settled by the first step (mode init) without probes.
constexpr int kSearchWaves = 4;

__global__ __launch_bounds__(kSearchWaves * kWave) void search_kernel(SearchParams P, int mode) {
    const int64_t s = (int64_t)blockIdx.x * kSearchWaves + threadIdx.x / kWave;
    if (s >= P.S) return;
    const int lane = lane_id();
    int32_t* lo = P.work;
    int32_t* hi = P.work + P.S;
    int32_t* probe = P.work + 2 * P.S;
    const int32_t F = P.F, H = P.H;
    if (mode == 0) {   // init
        const uint32_t fl = P.proj_flags ? P.proj_flags[s] : 0u;
        const bool settled = (fl & (TL_FLAG_OVERFLOW | TL_FLAG_LOST)) != 0;
        if (lane == 0) {
            lo[s] = settled ? -1 : 0;
            hi[s] = settled ? -1 : F - 1;
            probe[s] = (settled || F == 1) ? -1 : (F - 1) / 2;
            if (settled) {
                P.freq_idx[s] = F - 1;
                P.status[s] = (fl & TL_FLAG_OVERFLOW) ? TL_STATUS_INVALID : TL_STATUS_LOST;
            }
        }
        return;
    }
    const int32_t p = probe[s];
    if (p < 0) return;
    const int32_t n = min(max(P.n_iters[s], 0), H);
    bool miss, miss_own;
    const uint64_t t_r = wave_times(P.ips + s * H, P.deadline_at + s * H, n, -1, kNoDeadline, &miss, &miss_own);
    const bool ok = !miss && within_tbt(t_r, P.tbt_slo_ns[s], n);
    if (lane != 0) return;
    if (mode == 2) {   // final check of lo
        P.freq_idx[s] = ok ? p : F - 1;
        P.status[s] = ok ? TL_STATUS_OK : TL_STATUS_INFEASIBLE;
        probe[s] = -1;
        return;
    }
    int32_t l = lo[s], h = hi[s];
    if (ok) h = p;
    else l = p + 1;
    lo[s] = l;
    hi[s] = h;
    probe[s] = l < h ? l + (h - l) / 2 : -1;
}

// Before the final check, lo == hi for every unsettled scenario.  hi only
// moves to a probe found feasible, and no probe is ever F-1 (the midpoint of
// lo < hi lies below hi), so hi < F-1 means lo was probed and found
// feasible: the scenario is settled here with lo (OK), as the final check of
// lo would settle it.  The others (hi still F-1) probe lo.
__global__ __launch_bounds__(256) void search_final_probe_kernel(SearchParams P) {
    const int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (s >= P.S) return;
    const int32_t l = P.work[s], h = P.work[P.S + s];
    const bool known = l >= 0 && l == h && h < P.F - 1;
    if (known) {
        P.freq_idx[s] = l;
        P.status[s] = TL_STATUS_OK;
    }
    P.work[2 * P.S + s] = known ? -1 : l;   // -1 stays -1 (settled)
}

}  // namespace

hipError_t launch_admit(const AdmitParams& p, hipStream_t stream) {
    if (p.S == 0) return hipSuccess;
    hipLaunchKernelGGL(admit_kernel, dim3((unsigned)((p.S + kAdmitWaves - 1) / kAdmitWaves)),
                       dim3(kAdmitWaves * kWave), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_search_step(const SearchParams& p, int mode, hipStream_t stream) {
    if (p.S == 0) return hipSuccess;
    if (mode == 3) {
        hipLaunchKernelGGL(search_final_probe_kernel, dim3((unsigned)((p.S + 255) / 256)), dim3(256), 0, stream, p);
    } else {
        hipLaunchKernelGGL(search_kernel, dim3((unsigned)((p.S + kSearchWaves - 1) / kSearchWaves)),
                           dim3(kSearchWaves * kWave), 0, stream, p, mode);
    }
    return hipGetLastError();
}

hipError_t launch_select(const SelectParams& p, hipStream_t stream) {
    hipLaunchKernelGGL(select_kernel, dim3((unsigned)p.S), dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace tl
