"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Projections, selected frequencies and statuses must match bit for bit; the
ensemble outputs must match within 1e-5 relative (they are expected to be
bit-identical, and the tests also count exact matches).  Inputs come only
from the seeded generator or are written here; expected values come only
from the oracle or the hand-computed fixtures.
"""
import numpy as np
import pytest

import goldens
import oracle
from paper_2408_05235_amd import configs, synth

pytestmark = pytest.mark.gpu

NONE = np.uint64(0xFFFFFFFFFFFFFFFF)
RTOL = 1e-5


def _api():
    from paper_2408_05235_amd import api
    return api


def _np(t, dtype=None):
    a = t.detach().cpu().numpy()
    if dtype is not None:
        a = a.view(dtype)
    return a


def gpu_project(inp, rows=False, freqs=None, engine=None, n_features=3):
    import torch
    api = _api()
    d = api.upload(dict(inp, tbt_slo_ns=np.zeros(inp["n_scenarios"], np.uint64),
                        freqs_mhz=np.zeros(1, np.float32) if freqs is None else freqs,
                        engine_size=engine, n_features=n_features))
    out = api.tl_project(d["req_offset"], d["prompt"], d["generated"], d["remaining"], d["arrival"],
                         d["kv_capacity"], d["horizon"], d["block_tokens"], d["deadline_ns"], d["lost"],
                         d["batch_cap"], d["freqs_mhz"] if rows else None, d["engine_size"], n_features, rows)
    torch.cuda.synchronize()
    res = dict(batch=_np(out["batch"]), kv=_np(out["kv"]), deadline_at=_np(out["deadline_at"], np.uint64),
               n_iters=_np(out["n_iters"]), flags=_np(out["flags"], np.uint32))
    if rows:
        res["rows"] = _np(out["rows"])
    return res


def assert_projection_equal(g, o, where=""):
    for k in ("batch", "kv", "deadline_at", "n_iters", "flags"):
        a, b = np.asarray(g[k]), np.asarray(o[k])
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)
            raise AssertionError(f"{where} {k} differs at {bad[:5].tolist()}: gpu {a[tuple(bad[0])]} oracle {b[tuple(bad[0])]}")


def assert_ips_close(g, o, where=""):
    g = np.asarray(g, np.float32)
    o = np.asarray(o, np.float32)
    assert g.shape == o.shape
    both_nan = np.isnan(g) & np.isnan(o)
    ok = both_nan | (g == o) | (np.abs(g.astype(np.float64) - o) <= RTOL * np.abs(o.astype(np.float64)))
    assert ok.all(), f"{where} ips mismatch at {np.argwhere(~ok)[:5].tolist()}"
    return int(((g == o) | both_nan).sum())


# --------------------------------------------------------------- fixtures

@pytest.mark.parametrize("name", ["proj_inflight_eq1_eq2.json", "proj_batchcap_fifo.json",
                                  "proj_kv_blocked_fifo.json", "proj_overcommit_blocks_queue.json"])
def test_golden_projection_gpu(gpu, name):
    g = goldens.load(name)
    out = gpu_project(goldens.scoreboard(g))
    ex = g["expect"]
    assert out["batch"][0].tolist() == ex["batch"]
    assert out["kv"][0].tolist() == ex["kv"]
    assert np.array_equal(out["deadline_at"][0], goldens.deadline_map(ex["deadline_at"]))
    assert int(out["n_iters"][0]) == ex["n_iters"]
    assert int(out["flags"][0]) == ex["flags"]


def test_golden_selection_gpu(gpu):
    import torch
    api = _api()
    g = goldens.load("select_two_stumps.json")
    forest = api.Forest.from_dict(goldens.forest(g))
    freqs = np.array(g["freqs_mhz"], np.float32)
    for case in g["cases"]:
        sigma = case["sigma_ns"]
        inp = goldens.scoreboard(g, deadline_ns=[sigma * r for r in g["remaining"]], lost=case["lost"])
        inp.update(tbt_slo_ns=np.array([sigma], np.uint64), freqs_mhz=freqs, engine_size=None, n_features=3)
        d = api.upload(inp)
        ctl = api.Controller(d, forest)
        idx, st = ctl.step()
        torch.cuda.synchronize()
        assert _np(ctl.ips)[0].tolist() == g["expect_ips"]
        assert (int(idx[0]), int(st[0])) == (case["freq_idx"], case["status"]), case


# -------------------------------------------------- projection, random boards

def random_boards(rng, S, H, N, rmax=40, qfrac=0.3, bad=0.03, lost=0.02, unsorted=False, cap=None):
    counts = rng.integers(0, rmax + 1, S)
    counts[rng.random(S) < 0.05] = 0                     # empty scenarios
    off = np.zeros(S + 1, np.int64)
    np.cumsum(counts, out=off[1:])
    R = int(off[-1])
    prompt = rng.integers(0, 3 * N * 8 + 50, R).astype(np.int32)
    gen = rng.integers(0, 30, R).astype(np.int32)
    rem = rng.integers(1, 2 * H + 2, R).astype(np.int32)
    arr = np.full(R, -1, np.int32)
    for s in range(S):
        lo, hi = off[s], off[s + 1]
        nq = int(rng.binomial(hi - lo, qfrac))
        if nq:
            a = np.sort(rng.integers(0, H + 5, nq)).astype(np.int32)
            if unsorted and nq > 1 and rng.random() < 0.5:
                rng.shuffle(a)
            arr[hi - nq:hi] = a
            gen[hi - nq:hi] = 0
    m = rng.random(R) < bad
    prompt[m & (rng.random(R) < 0.5)] = -3
    rem[m & (rng.random(R) < 0.5)] = 0
    dl = (rng.integers(1, 10 ** 9, R)).astype(np.uint64)
    dl[rng.random(R) < 0.2] = NONE
    if cap is None:
        cap = rng.integers(N * 4, N * 40 + 200, S).astype(np.int32)
    return dict(n_scenarios=S, horizon=H, block_tokens=N, req_offset=off, prompt=prompt, generated=gen,
                remaining=rem, arrival=arr, deadline_ns=dl,
                lost=(rng.random(R) < lost).astype(np.uint8),
                kv_capacity=np.asarray(cap, np.int32),
                batch_cap=rng.integers(1, 30, S).astype(np.int32) if rng.random() < 0.5 else None)


@pytest.mark.parametrize("H,N,seed,rmax,qfrac", [(2048, 16, 20, 4000, 0.7), (700, 5, 21, 2500, 0.95),
                                                 (4096, 64, 22, 3000, 0.5)])
def test_project_many_requests(gpu, H, N, seed, rmax, qfrac):
    """Boards with thousands of requests per scenario and no batch cap: the
    projection keeps its batch differences in global memory (long FIFO
    loops); everything still equals the oracle."""
    rng = np.random.default_rng(seed)
    inp = random_boards(rng, 40, H, N, rmax=rmax, qfrac=qfrac, unsorted=(seed % 2 == 1))
    inp["batch_cap"] = None
    assert int(inp["req_offset"][-1]) >= 1024 * 40
    assert_projection_equal(gpu_project(inp), oracle.project(inp), f"H={H} N={N} rmax={rmax}")


def test_project_order_workspace_grows_and_changes_stream(gpu):
    """Long-FIFO boards are projected in an order kept in a per-device
    workspace of the library: a larger board replaces it, and calls from
    another stream wait for the previous user.  Every call equals the oracle."""
    import torch
    boards = []
    for i, S in enumerate((40, 96, 40)):
        inp = random_boards(np.random.default_rng(30 + i), S, 1024, 16, rmax=3000, qfrac=0.6)
        inp["batch_cap"] = None
        assert int(inp["req_offset"][-1]) >= 1024 * S
        boards.append(inp)
    side = torch.cuda.Stream()
    for i, inp in enumerate(boards):
        if i == 1:
            with torch.cuda.stream(side):
                g = gpu_project(inp)
        else:
            g = gpu_project(inp)
        assert_projection_equal(g, oracle.project(inp), f"board {i} S={inp['n_scenarios']}")


@pytest.mark.parametrize("H,N,seed", [(1, 16, 0), (7, 1, 1), (64, 16, 2), (100, 3, 3), (513, 16, 4),
                                      (1000, 64, 5), (257, 100, 6), (2048, 16, 7), (130, 7, 8),
                                      (600, 128, 9)])
def test_project_random_boards(gpu, H, N, seed):
    rng = np.random.default_rng(seed)
    inp = random_boards(rng, 300, H, N, unsorted=(seed % 2 == 1))
    g = gpu_project(inp)
    o = oracle.project(inp)
    assert_projection_equal(g, o, f"H={H} N={N}")
    # the cases that matter were exercised
    fl = o["flags"]
    assert (fl & oracle.FLAG_BAD_REQUEST).any() and (fl & oracle.FLAG_LOST).any()


def test_project_max_horizon_and_long_lifetimes(gpu):
    rng = np.random.default_rng(42)
    inp = random_boards(rng, 24, 8192, 16, rmax=60, qfrac=0.5)
    inp["remaining"] = rng.integers(1, 9000, inp["prompt"].size).astype(np.int32)
    assert_projection_equal(gpu_project(inp), oracle.project(inp), "H=8192")


def test_project_overcommit_and_caps(gpu):
    rng = np.random.default_rng(9)
    inp = random_boards(rng, 400, 300, 4, rmax=50, qfrac=0.5, cap=rng.integers(0, 120, 400))
    o = oracle.project(inp)
    assert (o["flags"] & oracle.FLAG_OVERCOMMIT).any()
    assert_projection_equal(gpu_project(inp), o, "overcommit")


@pytest.mark.parametrize("bcap,seed", [(False, 11), (True, 12), (False, 13)])
def test_project_long_queues(gpu, bcap, seed):
    """Hundreds of queued requests per scenario (several 64-request windows),
    capacities from slack to binding, some arrival orders unsorted: the
    batched and the one-at-a-time admission paths both run and must give the
    oracle's admissions."""
    rng = np.random.default_rng(seed)
    S, H, N = 48, 600, 16
    counts = rng.integers(150, 400, S)
    off = np.zeros(S + 1, np.int64)
    np.cumsum(counts, out=off[1:])
    R = int(off[-1])
    prompt = rng.integers(16, 2000, R).astype(np.int32)
    gen = np.zeros(R, np.int32)
    rem = np.clip(rng.lognormal(4.0, 1.0, R), 1, 3 * H).astype(np.int32)
    arr = np.full(R, -1, np.int32)
    for s in range(S):
        lo, hi = off[s], off[s + 1]
        nin = int(rng.integers(0, 30))
        gen[lo:lo + nin] = rng.integers(0, 200, nin)
        a = np.sort(rng.integers(0, H + 20, hi - lo - nin)).astype(np.int32)
        if s % 7 == 3:
            rng.shuffle(a)
        arr[lo + nin:hi] = a
    cap = rng.integers(300, 6000, S).astype(np.int32)
    inp = dict(n_scenarios=S, horizon=H, block_tokens=N, req_offset=off, prompt=prompt, generated=gen,
               remaining=rem, arrival=arr, deadline_ns=rng.integers(1, 10 ** 9, R).astype(np.uint64),
               lost=(rng.random(R) < 0.01).astype(np.uint8), kv_capacity=cap,
               batch_cap=rng.integers(5, 60, S).astype(np.int32) if bcap else None)
    o = oracle.project(inp, return_admit=True)
    adm = o["admit_iter"]
    late = (adm > arr) & (arr >= 0)
    assert late.sum() > 100 and ((adm >= 0) & (adm == arr)).sum() > 1000   # both regimes occur
    assert_projection_equal(gpu_project(inp), o, f"long queues bcap={bcap}")


def test_project_size_guard(gpu):
    H, N = 16, 1
    big = 1 << 30
    inp = dict(n_scenarios=3, horizon=H, block_tokens=N, req_offset=np.array([0, 1, 4, 4], np.int64),
               prompt=np.array([big, big, big, big], np.int32), generated=np.zeros(4, np.int32),
               remaining=np.array([4, 4, 4, 4], np.int32), arrival=np.full(4, -1, np.int32),
               deadline_ns=None, lost=None, kv_capacity=np.array([2 ** 31 - 1] * 3, np.int32), batch_cap=None)
    g = gpu_project(inp)
    assert_projection_equal(g, oracle.project(inp), "guard")
    assert g["flags"].tolist() == [0, oracle.FLAG_OVERFLOW, 0]


def test_project_rejects_bad_request_ranges_on_device(gpu):
    """Offsets outside [0, n_requests] are flagged, not read."""
    inp = dict(n_scenarios=3, horizon=8, block_tokens=4, req_offset=np.array([0, 2, 1, 3], np.int64),
               prompt=np.array([4, 4, 4], np.int32), generated=np.zeros(3, np.int32),
               remaining=np.array([3, 3, 3], np.int32), arrival=np.full(3, -1, np.int32),
               deadline_ns=None, lost=None, kv_capacity=np.array([100] * 3, np.int32), batch_cap=None)
    g = gpu_project(inp)
    assert g["flags"].tolist() == [0, oracle.FLAG_OVERFLOW, 0]
    assert g["batch"][1].sum() == 0


def test_project_rows(gpu):
    rng = np.random.default_rng(3)
    inp = random_boards(rng, 50, 200, 16)
    freqs = synth.frequency_grid(17)
    for nf in (3, 4):
        engine = rng.choice([1.0, 2.0, 4.0, 8.0], 50).astype(np.float32) if nf == 4 else None
        g = gpu_project(inp, rows=True, freqs=freqs, engine=engine, n_features=nf)
        o = oracle.project(inp)
        assert_projection_equal(g, o, "rows")
        x = oracle.rows(freqs, o["batch"], o["kv"], engine, nf)
        assert np.array_equal(g["rows"], x)


# ------------------------------------------------------------------ forest

def random_forest(rng, T, d, nf, kvmax=5000, bmax=300):
    n_int = (1 << d) - 1
    feat = rng.integers(0, nf, (T, n_int)).astype(np.uint8)
    hi = np.array([2000.0, kvmax, bmax, 8.0][:nf])
    lo = np.array([1000.0, 0.0, 0.0, 1.0][:nf])
    thr = (lo[feat] + (hi[feat] - lo[feat]) * rng.random((T, n_int))).astype(np.float32)
    snap = rng.random((T, n_int)) < 0.2
    thr[snap] = np.rint(thr[snap])
    thr[rng.random((T, n_int)) < 0.01] = np.inf
    thr[rng.random((T, n_int)) < 0.01] = -np.inf
    leaf = rng.normal(0, 1, (T, 1 << d)).astype(np.float32)
    return dict(n_trees=T, depth=d, n_features=nf, base_score=np.float32(rng.normal(40, 5)),
                feature=feat, threshold=thr, leaf=leaf)


def random_rows(rng, n, nf, kvmax=5000, bmax=300):
    cols = [rng.choice(synth.frequency_grid(64), n), rng.integers(0, kvmax, n), rng.integers(0, bmax, n),
            rng.choice([1.0, 2.0, 4.0, 8.0], n)]
    x = np.stack(cols[:nf], axis=1).astype(np.float32)
    x[rng.random(x.shape) < 0.001] = np.nan
    return x


# 3- and 4-feature forests up to depth 11 take the LDS-staged row walks
# (odd tree counts end on a single tree), the others the global-memory walks
@pytest.mark.parametrize("T,d,nf,n", [(0, 3, 3, 100), (1, 0, 3, 77), (5, 1, 1, 1000), (50, 6, 3, 12345),
                                      (20, 10, 4, 4099), (7, 14, 2, 513), (300, 8, 3, 65537),
                                      (33, 11, 4, 3001), (9, 9, 4, 100003), (3, 12, 3, 999)])
def test_forest_random(gpu, T, d, nf, n):
    import torch
    api = _api()
    rng = np.random.default_rng(T * 31 + d)
    fd = random_forest(rng, T, d, nf)
    x = random_rows(rng, n, nf)
    f = api.Forest.from_dict(fd)
    got = _np(f.tl_forest_predict(torch.from_numpy(x).cuda()))
    torch.cuda.synchronize()
    exp = oracle.forest_predict(fd, x)
    exact = assert_ips_close(got, exp, f"T={T} d={d}")
    assert exact == n      # fp32 running sums in tree order on both sides


def test_forest_rows_at_an_offset(gpu):
    """4-feature rows that start 4 bytes into their buffer (not 16-byte
    aligned) through the LDS-staged row walks."""
    import torch
    api = _api()
    rng = np.random.default_rng(4343)
    fd = random_forest(rng, 37, 8, 4)
    n = 3001
    x = random_rows(rng, n, 4)
    buf = torch.zeros(n * 4 + 1, dtype=torch.float32)
    buf[1:] = torch.from_numpy(x.reshape(-1))
    dev = buf.cuda()[1:].view(n, 4)
    assert dev.data_ptr() % 16 == 4
    f = api.Forest.from_dict(fd)
    got = _np(f.tl_forest_predict(dev))
    torch.cuda.synchronize()
    exp = oracle.forest_predict(fd, x)
    assert assert_ips_close(got, exp, "offset rows") == n


def random_curves(rng, S, H, kvmax=5000, bmax=300):
    """Slowly varying KV / batch curves with jumps, like projections."""
    kv = np.clip(rng.integers(0, kvmax, (S, 1)) + np.cumsum(rng.integers(-12, 10, (S, H)), axis=1), 0, None)
    bs = np.clip(rng.integers(0, bmax, (S, 1)) + np.cumsum(rng.integers(-1, 1, (S, H)) * (rng.random((S, H)) < 0.2), axis=1), 0, None)
    jump = rng.random((S, H)) < 0.01
    kv = np.where(jump, rng.integers(0, kvmax, (S, H)), kv)
    return kv.astype(np.int32), bs.astype(np.int32)


@pytest.mark.parametrize("S,F,H,T,d,nf", [(3, 64, 1024, 40, 10, 4), (5, 17, 100, 30, 6, 3), (2, 130, 70, 20, 8, 3),
                                          (4, 48, 33, 25, 8, 3), (1, 1, 1, 3, 2, 4), (2, 64, 64, 0, 4, 3),
                                          (3, 32, 95, 10, 0, 3), (2, 20, 40, 150, 3, 3), (3, 64, 50, 7, 12, 4),
                                          (2, 40, 77, 5, 13, 3), (1, 64, 37, 3, 14, 4),
                                          # several 64-iteration chunks with ragged tails of 8 and 1 rows
                                          (3, 64, 200, 40, 10, 3), (2, 70, 129, 33, 8, 4), (4, 64, 65, 21, 9, 3),
                                          # depth 11: one tree per staged block (every tree a single)
                                          (2, 64, 130, 7, 11, 3),
                                          # depth 10 (two-tree blocks in three buffers): one tree, one
                                          # pair, an odd count whose last block holds a single tree
                                          (2, 33, 70, 1, 10, 4), (3, 64, 100, 2, 10, 3), (2, 64, 150, 5, 10, 4)])
def test_forest_grid(gpu, S, F, H, T, d, nf):
    """The fused grid kernel equals the oracle on the rows it stands for."""
    import torch
    api = _api()
    rng = np.random.default_rng(S * 1000 + F + H + T)
    fd = random_forest(rng, T, d, nf)
    kv, bs = random_curves(rng, S, H)
    freqs = synth.frequency_grid(F)
    eng = rng.choice([1.0, 2.0, 4.0, 8.0], S).astype(np.float32) if nf == 4 else None
    f = api.Forest.from_dict(fd)
    t = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    got = _np(f.tl_forest_predict_grid(t(freqs), t(kv), t(bs), t(eng)))
    torch.cuda.synchronize()
    exp = oracle.forest_predict(fd, oracle.rows(freqs, bs, kv, eng, nf))
    assert assert_ips_close(got, exp, "grid") == exp.size


def _order_sensitive_forest(rng, T, d, nf):
    """Random trees whose leaves make the fp32 running sum depend on its
    order: trees 3k add +2^24, trees 3k+1 a random value in (-4, 4) with a
    fraction, trees 3k+2 subtract 2^24, so every middle value is rounded to
    the 2-unit spacing at 2^24 before it is taken out again."""
    fd = random_forest(rng, T, d, nf)
    leaf = fd["leaf"]
    leaf[0::3] = np.float32(2.0 ** 24)
    leaf[1::3] = (rng.uniform(-4, 4, leaf[1::3].shape) + 0.25).astype(np.float32)
    leaf[2::3] = np.float32(-(2.0 ** 24))
    fd["base_score"] = np.float32(0.75)
    return fd


@pytest.mark.parametrize("T,d,nf", [(61, 8, 3), (31, 10, 4)])
def test_forest_sum_order_is_tree_order(gpu, T, d, nf):
    """fp32 running sums in tree order on every forest path: a forest whose
    result changes with the order of the adds gives the oracle's values on
    the row walks and on the grid kernel (both wide and with a short tail)."""
    import torch
    api = _api()
    rng = np.random.default_rng(T + d)
    fd = _order_sensitive_forest(rng, T, d, nf)
    x = random_rows(rng, 4099, nf)
    x[np.isnan(x)] = 1500.0
    exp_rows = oracle.forest_predict(fd, x)
    # the test can tell orders apart: an fp64 sum differs on most rows
    f64 = np.full(x.shape[0], np.float64(fd["base_score"]))
    for t in range(T):
        sub = dict(fd, n_trees=1, feature=fd["feature"][t:t + 1], threshold=fd["threshold"][t:t + 1],
                   leaf=fd["leaf"][t:t + 1], base_score=np.float32(0))
        f64 += oracle.forest_predict(sub, x).astype(np.float64)
    assert np.mean(f64.astype(np.float32) != exp_rows) > 0.5
    f = api.Forest.from_dict(fd)
    got = _np(f.tl_forest_predict(torch.from_numpy(x).cuda()))
    torch.cuda.synchronize()
    assert np.array_equal(got, exp_rows)
    S, F, H = 3, 64, 131
    kv, bs = random_curves(rng, S, H)
    freqs = synth.frequency_grid(F)
    eng = rng.choice([1.0, 2.0, 4.0, 8.0], S).astype(np.float32) if nf == 4 else None
    t = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    grid = _np(f.tl_forest_predict_grid(t(freqs), t(kv), t(bs), t(eng)))
    torch.cuda.synchronize()
    assert np.array_equal(grid, oracle.forest_predict(fd, oracle.rows(freqs, bs, kv, eng, nf)))
    f.close()


def test_forest_grid_nan_and_infinite_thresholds(gpu):
    """Leaves behind NaN thresholds are unreachable; +-inf thresholds bound
    nothing.  The box reuse must still give the tree-walk result."""
    import torch
    api = _api()
    rng = np.random.default_rng(5)
    fd = random_forest(rng, 30, 7, 3)
    thr = fd["threshold"]
    m = rng.random(thr.shape)
    thr[m < 0.05] = np.nan
    thr[(m >= 0.05) & (m < 0.1)] = np.inf
    thr[(m >= 0.1) & (m < 0.15)] = -np.inf
    kv, bs = random_curves(rng, 4, 300)
    freqs = synth.frequency_grid(40)
    f = api.Forest.from_dict(fd)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    got = _np(f.tl_forest_predict_grid(t(freqs), t(kv), t(bs)))
    torch.cuda.synchronize()
    exp = oracle.forest_predict(fd, oracle.rows(freqs, bs, kv, None, 3))
    assert assert_ips_close(got, exp, "grid-nan") == exp.size


# --------------------------------------------------------------- selection

def random_selection(rng, S, F, H):
    ips = rng.uniform(5, 120, (S, F, H)).astype(np.float32)
    special = rng.random((S, F, H))
    ips[special < 0.002] = 0.0
    ips[(special >= 0.002) & (special < 0.003)] = np.nan
    ips[(special >= 0.003) & (special < 0.004)] = -1.0
    ips[(special >= 0.004) & (special < 0.005)] = np.inf
    ips[(special >= 0.005) & (special < 0.006)] = 1e-9
    n = rng.integers(-2, H + 3, S).astype(np.int32)
    dl = np.full((S, H), NONE, np.uint64)
    nd = rng.integers(0, 6, S)
    for s in range(S):
        js = rng.integers(0, H, nd[s])
        dl[s, js] = (rng.uniform(0.5, 1.5, js.size) * 30e6 * (js + 1)).astype(np.uint64)
    tbt = rng.integers(5_000_000, 60_000_000, S).astype(np.uint64)
    tbt[rng.random(S) < 0.01] = NONE          # saturating SLO budget
    flags = np.zeros(S, np.uint32)
    flags[rng.random(S) < 0.03] = oracle.FLAG_LOST
    flags[rng.random(S) < 0.01] |= oracle.FLAG_OVERFLOW
    flags[rng.random(S) < 0.05] |= oracle.FLAG_OVERCOMMIT
    return ips, dl, n, tbt, flags


def gpu_select(ips, dl, n, tbt, flags):
    import torch
    api = _api()
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    idx, st = api.tl_select_freq(t(ips), t(dl.view(np.int64)), t(n), t(tbt.view(np.int64)),
                                 None if flags is None else t(flags.view(np.int32)))
    torch.cuda.synchronize()
    return _np(idx), _np(st)


@pytest.mark.parametrize("S,F,H,seed", [(1, 1, 1, 0), (50, 17, 512, 1), (200, 64, 100, 2), (40, 100, 300, 3),
                                        (300, 5, 65, 4), (10, 4096, 8, 5)])
def test_select_random(gpu, S, F, H, seed):
    rng = np.random.default_rng(seed)
    ips, dl, n, tbt, flags = random_selection(rng, S, F, H)
    gi, gs = gpu_select(ips, dl, n, tbt, flags)
    oi, os_ = oracle.select(ips, dl, n, tbt, flags)
    assert np.array_equal(gi, oi) and np.array_equal(gs.view(np.uint32), os_)
    gi, gs = gpu_select(ips, dl, n, tbt, None)
    oi, os_ = oracle.select(ips, dl, n, tbt, None)
    assert np.array_equal(gi, oi) and np.array_equal(gs.view(np.uint32), os_)


def test_select_full_shape_generated_ips(gpu):
    """Selection alone at the forest-bound workload's shape (S=4096, F=64,
    H=1024) on generated predictions, every scenario compared."""
    rng = np.random.default_rng(77)
    S, F, H = 4096, 64, 1024
    ips = rng.normal(40, 6, (S, F, H)).astype(np.float32)
    n = rng.integers(0, H + 1, S).astype(np.int32)
    dl = np.full((S, H), NONE, np.uint64)
    js = rng.integers(0, H, (S, 8))
    for k in range(8):
        dl[np.arange(S), js[:, k]] = (rng.uniform(0.8, 1.6, S) * 25e6 * (js[:, k] + 1)).astype(np.uint64)
    tbt = rng.integers(10_000_000, 50_000_001, S).astype(np.uint64)
    flags = np.zeros(S, np.uint32)
    gi, gs = gpu_select(ips, dl, n, tbt, flags)
    oi, os_ = oracle.select(ips, dl, n, tbt, flags)
    assert np.array_equal(gi, oi) and np.array_equal(gs.view(np.uint32), os_)
    assert len(np.unique(oi)) > 10


# ---------------------------------------------------------- whole pipeline

SCALED = [
    (0, dict()),
    (1, dict(n_scenarios=12)),
    (2, dict(n_scenarios=6)),
    (3, dict(n_scenarios=3, forest_n_trees=300)),
    (4, dict(n_scenarios=6)),
]


@pytest.mark.parametrize("ci,over", SCALED, ids=[c["name"] for c in configs.CONFIGS])
def test_pipeline_scaled_configs(gpu, ci, over):
    import torch
    api = _api()
    cfg = synth.scaled(configs.get_config(ci), **over)
    inp = synth.make_inputs(cfg)
    ctl = api.Controller(api.upload(inp), api.Forest.from_dict(inp["forest"]),
                         materialize_rows=(ci % 2 == 1))
    idx, st = ctl.step()
    torch.cuda.synchronize()
    o = oracle.end_to_end(inp)
    g = dict(batch=_np(ctl.buf["batch"]), kv=_np(ctl.buf["kv"]),
             deadline_at=_np(ctl.buf["deadline_at"], np.uint64), n_iters=_np(ctl.buf["n_iters"]),
             flags=_np(ctl.buf["flags"], np.uint32))
    assert_projection_equal(g, o, cfg["name"])
    exact = assert_ips_close(_np(ctl.ips), o["ips"], cfg["name"])
    assert exact == o["ips"].size
    assert np.array_equal(_np(idx), o["freq_idx"]) and np.array_equal(_np(st).view(np.uint32), o["status"])


def test_determinism(gpu):
    import torch
    api = _api()
    cfg = synth.scaled(configs.get_config(1), n_scenarios=20)
    inp = synth.make_inputs(cfg)
    ctl = api.Controller(api.upload(inp), api.Forest.from_dict(inp["forest"]))
    ctl.step()
    torch.cuda.synchronize()
    a = [_np(ctl.ips).copy(), _np(ctl.buf["kv"]).copy(), _np(ctl.sel["freq_idx"]).copy()]
    ctl.step()
    torch.cuda.synchronize()
    b = [_np(ctl.ips), _np(ctl.buf["kv"]), _np(ctl.sel["freq_idx"])]
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    # the materialized rows through the generic kernel, at an offset (a
    # different launch grid), give the same values as the fused grid kernel
    ctl2 = api.Controller(ctl.d, ctl.forest, materialize_rows=True)
    ctl2.project()
    rows = ctl2.buf["rows"].reshape(-1, 3)
    part = ctl.forest.tl_forest_predict(rows[1001:].contiguous())
    torch.cuda.synchronize()
    assert np.array_equal(_np(part), _np(ctl.ips).reshape(-1)[1001:])


def test_maximum_frequencies_and_horizon(gpu):
    """F = TL_MAX_FREQS and H = TL_MAX_HORIZON through the grid kernel and
    the selection (one scenario, 33.5 M rows, a small forest)."""
    import torch
    api = _api()
    rng = np.random.default_rng(4242)
    F, H = 4096, 8192
    fd = random_forest(rng, 3, 4, 4, kvmax=6000, bmax=300)
    fd["base_score"] = np.float32(60.0)
    kv, bs = random_curves(rng, 1, H, kvmax=6000, bmax=300)
    eng = np.array([4.0], np.float32)
    freqs = synth.frequency_grid(F)
    f = api.Forest.from_dict(fd)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    ips = f.tl_forest_predict_grid(t(freqs), t(kv), t(bs), t(eng))
    dl = np.full((1, H), NONE, np.uint64)
    dl[0, [10, 4000, 8191]] = [400_000_000, 80_000_000_000, 150_000_000_000]
    n = np.array([H], np.int32)
    tbt = np.array([16_500_000], np.uint64)        # the lowest passing index is 3760
    idx, st = api.tl_select_freq(ips, t(dl.view(np.int64)), t(n), t(tbt.view(np.int64)), None)
    torch.cuda.synchronize()
    got = _np(ips)
    exp = oracle.forest_predict(fd, oracle.rows(freqs, bs, kv, eng, 4))
    assert np.array_equal(got, exp)
    oi, os_ = oracle.select(exp, dl, n, tbt)
    assert (int(_np(idx)[0]), int(_np(st)[0])) == (int(oi[0]), int(os_[0]))
    assert int(oi[0]) > 1000          # deep into the rounds of four
    f.close()
