"""Seeded random sweeps against the oracle, through the C ABI.

Projection and admission: random scoreboards (1-119 scenarios, H up to
3000, block sizes 1-100, 0-3000 requests per scenario, any queued
fraction, sorted or unsorted arrivals, binding, loose or unreachable KV
caps, batch caps or none, malformed and lost entries), every third case as
an admission what-if with a small random forest; curves, checkpoints, flags
and decisions bit-exact.

Selection: random IPS (scaled per case, special values, increasing in the
frequency on half of the scenarios), deadlines, SLO budgets and flags over
random shapes; index and status bit-exact.

Models: the grid kernel (random S, F up to 129, H up to 700), the LDS-staged
row walks (up to 20 000 rows, NaN features) and the column query at one
frequency per scenario (the binary search's final probe; half of the cases
at the sizes that take the leaf-reuse column kernel, half of the scenarios
with a batch that changes at every iteration).  Forests of 0-39 trees,
depth 0-11, 3 or 4 features.  Every output is compared bit for bit."""
import numpy as np
import pytest

import oracle
from paper_2408_05235_amd import synth
from test_gpu_admit import check_admit, random_candidates
from test_gpu_parity import (assert_projection_equal, gpu_project, gpu_select, random_boards, random_curves,
                             random_forest, random_rows, random_selection)

pytestmark = pytest.mark.gpu

N_CASES = 600


def _case(seed):
    import torch
    from paper_2408_05235_amd import api
    rng = np.random.default_rng(10_000 + seed)
    nf = int(rng.choice([3, 4]))
    d = int(rng.integers(0, 12))
    T = int(rng.integers(0, 40))
    kind = seed % 3
    if kind == 2 and rng.random() < 0.5:
        big = True
        T = min(T, 12)
    else:
        big = False
    fd = random_forest(rng, T, d, nf, kvmax=4000, bmax=250)
    f = api.Forest.from_dict(fd)
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a, dt)).cuda()
    try:
        if kind == 0:
            S, F, H = int(rng.integers(1, 9)), int(rng.integers(1, 130)), int(rng.integers(1, 700))
            kv, bs = random_curves(rng, S, H, kvmax=4000, bmax=250)
            freqs = synth.frequency_grid(F)
            eng = rng.choice([1.0, 2.0, 4.0, 8.0], S).astype(np.float32) if nf == 4 else None
            got = f.tl_forest_predict_grid(t(freqs, np.float32), t(kv, np.int32), t(bs, np.int32),
                                           None if eng is None else t(eng, np.float32))
            exp = oracle.forest_predict(fd, oracle.rows(freqs, bs, kv, eng, nf)).reshape(S, F, H)
            what = f"grid S={S} F={F} H={H}"
        elif kind == 1:
            n = int(rng.integers(1, 20000))
            x = random_rows(rng, n, nf)
            got = f.tl_forest_predict(torch.from_numpy(x).cuda())
            exp = oracle.forest_predict(fd, x)
            what = f"rows n={n}"
        else:
            S = int(rng.integers(2048, 4097)) if big else int(rng.integers(1, 60))
            H = int(rng.integers(512, 1100)) if big else int(rng.integers(1, 2100))
            kv, bs = random_curves(rng, S, H, kvmax=4000, bmax=250)
            fast = rng.random(S) < 0.5
            nfast = int(fast.sum())
            bs[fast] = np.clip(rng.integers(20, 200, (nfast, 1)) + np.cumsum(rng.choice([-1, 1], (nfast, H)), axis=1),
                               0, None)
            freqs = synth.frequency_grid(8)[int(rng.integers(0, 8)):][:1]
            eng = rng.choice([1.0, 2.0, 4.0, 8.0], S).astype(np.float32) if nf == 4 else None
            # one frequency: the search's final probe evaluates M there on every row
            out = {"ips_work": torch.full((S, H), -1.0, dtype=torch.float32, device="cuda")}
            api.tl_select_freq_binary(f, t(freqs, np.float32), t(kv, np.int32), t(bs, np.int32),
                                      torch.full((S, H), -1, dtype=torch.int64, device="cuda"),
                                      torch.full((S,), H, dtype=torch.int32, device="cuda"),
                                      torch.full((S,), 10 ** 12, dtype=torch.int64, device="cuda"), None,
                                      None if eng is None else t(eng, np.float32), out)
            got = out["ips_work"]
            exp = oracle.forest_predict(fd, oracle.rows(freqs, bs, kv, eng, nf)).reshape(S, H)
            what = f"column S={S} H={H}"
        torch.cuda.synchronize()
        g = got.cpu().numpy().astype(np.float32)
        e = np.asarray(exp, np.float32)
        bad = np.nonzero(g.reshape(-1).view(np.uint32) != e.reshape(-1).view(np.uint32))[0]
        return what, bad
    finally:
        f.close()


def test_random_sweep(gpu):
    for seed in range(N_CASES):
        what, bad = _case(seed)
        assert bad.size == 0, f"seed {seed} ({what}): {bad.size} outputs differ, first at {bad[:5].tolist()}"


N_BOARD_CASES = 300


def test_random_projection_and_admission_sweep(gpu):
    for seed in range(N_BOARD_CASES):
        rng = np.random.default_rng(50_000 + seed)
        S, H = int(rng.integers(1, 120)), int(rng.integers(1, 3000))
        N = int(rng.choice([1, 3, 7, 16, 64, 100]))
        rmax = int(rng.choice([0, 5, 40, 300, 1000, 3000]))   # 3000: the projection's global-memory batch array
        qfrac = float(rng.random())
        u = rng.random()
        tight = u < 0.4
        cap = (rng.integers(max(1, N), N * 10 + 50, S).astype(np.int32) if tight
               else np.full(S, 1 << 30, np.int32) if u > 0.75 else None)   # binding, never binding, generated
        inp = random_boards(rng, S, H, N, rmax=rmax, qfrac=qfrac, unsorted=bool(rng.random() < 0.3), cap=cap)
        where = f"seed {seed} S={S} H={H} N={N} rmax={rmax} q={qfrac:.2f} tight={tight}"
        if seed % 3 == 2:
            nf = int(rng.choice([3, 4]))
            inp["tbt_slo_ns"] = rng.integers(5_000_000, 60_000_000, S).astype(np.uint64)
            if nf == 4:
                inp["engine_size"] = rng.choice([1.0, 2.0, 4.0, 8.0], S).astype(np.float32)
            fd = random_forest(rng, int(rng.integers(0, 20)), int(rng.integers(0, 9)), nf, kvmax=4000, bmax=300)
            fd["base_score"] = np.float32(60.0)
            check_admit(inp, fd, 2000.0, random_candidates(rng, inp), "admission " + where)
        else:
            assert_projection_equal(gpu_project(inp), oracle.project(inp), where)


N_SELECT_CASES = 300


def test_random_selection_sweep(gpu):
    for seed in range(N_SELECT_CASES):
        rng = np.random.default_rng(90_000 + seed)
        S, F, H = int(rng.integers(1, 80)), int(rng.integers(1, 130)), int(rng.integers(1, 1500))
        ips, dl, n, tbt, flags = random_selection(rng, S, F, H)
        ips *= np.float32(rng.uniform(0.2, 5.0))
        mono = rng.random(S) < 0.5
        ips[mono] = np.sort(ips[mono], axis=1)
        fl = flags if rng.random() < 0.7 else None
        gi, gs = gpu_select(ips, dl, n, tbt, fl)
        oi, os_ = oracle.select(ips, dl, n, tbt, fl)
        assert np.array_equal(gi, oi) and np.array_equal(gs.view(np.uint32), os_), \
            f"seed {seed} S={S} F={F} H={H}: scenarios {np.nonzero((gi != oi) | (gs.view(np.uint32) != os_))[0][:5]}"
