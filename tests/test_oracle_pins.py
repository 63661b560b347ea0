"""Pins of the CPU oracle against things other than itself.

Each test fixes part of the oracle by a route independent of its code:
hand-computed examples (tests/golden/, each with its citation), an engine
simulation that allocates KV blocks token by token, the textbook FIFO list
schedule, a brute-force check of the admission rule as the paper states it,
scikit-learn's own tree traversal, exact rational arithmetic, closed forms and
invariants.  None of them needs a GPU.
"""
import heapq
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st, HealthCheck

import goldens
import oracle

NONE = np.uint64(0xFFFFFFFFFFFFFFFF)


# ---------------------------------------------------------------- golden files

@pytest.mark.parametrize("name", ["proj_inflight_eq1_eq2.json", "proj_batchcap_fifo.json",
                                  "proj_kv_blocked_fifo.json", "proj_overcommit_blocks_queue.json"])
def test_golden_projection(name):
    g = goldens.load(name)
    out = oracle.project(goldens.scoreboard(g), return_admit=True)
    ex = g["expect"]
    assert out["batch"][0].tolist() == ex["batch"]
    assert out["kv"][0].tolist() == ex["kv"]
    assert np.array_equal(out["deadline_at"][0], goldens.deadline_map(ex["deadline_at"]))
    assert int(out["n_iters"][0]) == ex["n_iters"]
    assert int(out["flags"][0]) == ex["flags"]
    assert out["admit_iter"].tolist() == ex["admit_iter"]


def test_golden_selection():
    g = goldens.load("select_two_stumps.json")
    forest = goldens.forest(g)
    freqs = np.array(g["freqs_mhz"], np.float32)
    for case in g["cases"]:
        sigma = case["sigma_ns"]
        dl = [sigma * r for r in g["remaining"]]
        proj = oracle.project(goldens.scoreboard(g, deadline_ns=dl, lost=case["lost"]))
        x = oracle.rows(freqs, proj["batch"], proj["kv"], None, 3)
        ips = oracle.forest_predict(forest, x)
        assert ips[0].tolist() == g["expect_ips"]
        idx, stt = oracle.select(ips, proj["deadline_at"], proj["n_iters"],
                                 np.array([sigma], np.uint64), proj["flags"])
        assert (int(idx[0]), int(stt[0])) == (case["freq_idx"], case["status"]), case


def test_golden_engine_size_two_scenarios():
    """Four-feature rows of several scenarios: the row (s, f, j) must carry
    scenario s's own curves and engine size at frequency f, in [S][F][H]
    order, through prediction and selection (hand-computed)."""
    g = goldens.load("e2e_engine_size_two_scenarios.json")
    forest = goldens.forest(g)
    freqs = np.array(g["freqs_mhz"], np.float32)
    for case in g["cases"]:
        inp = goldens.scoreboard_multi(g, case["sigma_ns"], lost=case["lost"])
        proj = oracle.project(inp)
        assert proj["batch"].tolist() == g["expect_batch"]
        assert proj["kv"].tolist() == g["expect_kv"]
        assert proj["n_iters"].tolist() == g["expect_n_iters"]
        x = oracle.rows(freqs, proj["batch"], proj["kv"], inp["engine_size"], 4)
        assert x.tolist() == g["expect_rows"]
        ips = oracle.forest_predict(forest, x)
        assert ips.tolist() == g["expect_ips"]
        idx, stt = oracle.select(ips, proj["deadline_at"], proj["n_iters"], inp["tbt_slo_ns"],
                                 proj["flags"])
        assert idx.tolist() == case["freq_idx"] and stt.tolist() == case["status"], case["note"]
        full = oracle.end_to_end(dict(inp, freqs_mhz=freqs, n_features=4, forest=forest))
        assert full["ips"].tolist() == g["expect_ips"]
        assert full["freq_idx"].tolist() == case["freq_idx"], case["note"]


def test_rows_three_features_several_scenarios():
    """Without the engine-size column the rows keep the same [S][F][H]
    order (the same hand-computed curves as the four-feature fixture)."""
    g = goldens.load("e2e_engine_size_two_scenarios.json")
    proj = oracle.project(goldens.scoreboard_multi(g, [1, 1]))
    x = oracle.rows(np.array(g["freqs_mhz"], np.float32), proj["batch"], proj["kv"], None, 3)
    assert x.tolist() == [[[r[:3] for r in rf] for rf in rs] for rs in g["expect_rows"]]


# ------------------------------------------------ engine simulation (Eq. 1, 2)

def simulate_engine(H, N, reqs):
    """Token-level simulation of a paged KV cache.

    ``reqs`` is a list of (cached_tokens, join_iter, n_iters).  Each request
    allocates blocks of N tokens as its cache grows; at every iteration it
    holds its cache, then generates one token; after its last iteration its
    blocks are freed.  Returns the per-iteration batch size and block count.
    """
    B = np.zeros(H, np.int64)
    KV = np.zeros(H, np.int64)
    state = []
    pending = sorted(range(len(reqs)), key=lambda i: reqs[i][1])
    pi = 0
    for j in range(H):
        while pi < len(pending) and reqs[pending[pi]][1] == j:
            c, _, L = reqs[pending[pi]]
            blocks = 0
            while blocks * N < c:
                blocks += 1
            state.append([c, blocks, L])
            pi += 1
        B[j] = len(state)
        KV[j] = sum(s[1] for s in state)
        nxt = []
        for s in state:
            s[0] += 1
            s[2] -= 1
            if s[2] == 0:
                continue          # struck from the scoreboard, blocks freed
            while s[1] * N < s[0]:
                s[1] += 1         # the new token needs a fresh block
            nxt.append(s)
        state = nxt
    return B, KV


def _inflight_board(rng, R, H, N, pmax=60, gmax=20, rmax=None):
    rmax = rmax or 2 * H
    return dict(
        n_scenarios=1, horizon=H, block_tokens=N,
        req_offset=np.array([0, R], np.int64),
        prompt=rng.integers(0, pmax, R).astype(np.int32),
        generated=rng.integers(0, gmax, R).astype(np.int32),
        remaining=rng.integers(1, rmax, R).astype(np.int32),
        arrival=np.full(R, -1, np.int32),
        deadline_ns=None, lost=None,
        kv_capacity=np.array([1 << 30], np.int32), batch_cap=None)


@pytest.mark.parametrize("seed", range(12))
def test_projection_matches_engine_simulation(seed):
    rng = np.random.default_rng(seed)
    H = int(rng.integers(1, 80))
    N = int(rng.integers(1, 20))
    R = int(rng.integers(0, 30))
    inp = _inflight_board(rng, R, H, N)
    out = oracle.project(inp)
    reqs = [(int(p) + int(g), 0, int(r)) for p, g, r in
            zip(inp["prompt"], inp["generated"], inp["remaining"])]
    B, KV = simulate_engine(H, N, reqs)
    assert out["batch"][0].tolist() == B.tolist()
    assert out["kv"][0].tolist() == KV.tolist()
    e = [min(int(r), H) for r in inp["remaining"]]
    assert int(out["n_iters"][0]) == (max(e) if e else 0)


# ------------------------------------------- FIFO list schedule (batch cap)

@pytest.mark.parametrize("seed", range(10))
def test_batch_cap_admission_is_fifo_list_schedule(seed):
    """With unlimited KV capacity and every queued request present at
    iteration 0, admission is the textbook FIFO schedule on `cap` servers:
    each request starts when the earliest server frees up."""
    rng = np.random.default_rng(100 + seed)
    H = int(rng.integers(20, 200))
    cap = int(rng.integers(1, 8))
    n_in = int(rng.integers(0, cap + 1))
    n_q = int(rng.integers(0, 25))
    R = n_in + n_q
    inp = _inflight_board(rng, R, H, 4, rmax=H // 2 + 2)
    inp["arrival"][n_in:] = 0
    inp["generated"][n_in:] = 0
    inp["batch_cap"] = np.array([cap], np.int32)
    out = oracle.project(inp, return_admit=True)
    servers = [int(r) for r in inp["remaining"][:n_in]] + [0] * (cap - n_in)
    heapq.heapify(servers)
    expect = [0] * n_in
    for k in range(n_in, R):
        t = heapq.heappop(servers)
        if t >= H:
            expect.append(-1)
            heapq.heappush(servers, t)
            continue
        expect.append(t)
        heapq.heappush(servers, t + int(inp["remaining"][k]))
    # once one request misses the horizon, all later ones do too
    seen_miss = False
    for k in range(n_in, R):
        seen_miss = seen_miss or expect[k] == -1
        if seen_miss:
            expect[k] = -1
    assert out["admit_iter"].tolist() == expect


# ------------------------------ admission: the paper's rule, checked by brute force

def _check_rule(H, N, cap_kv, cap_b, admitted, cand, j):
    """Would `cand` = (c, L) pass Sec. 4.3.2 check 1 and the batch cap at j,
    given the `admitted` list of (c, a, L)?  Literal form: append it with
    s_a = j and require every projected KV value from j on to be <= capacity."""
    B0, KV0 = simulate_engine(H, N, [(c, a, L) for c, a, L in admitted])
    if cap_b is not None and B0[j] >= cap_b:
        return False
    B1, KV1 = simulate_engine(H, N, [(c, a, L) for c, a, L in admitted] + [(cand[0], j, cand[1])])
    return bool(np.all(KV1[j:] <= cap_kv))


@pytest.mark.parametrize("seed", range(25))
def test_admission_is_earliest_feasible_fifo(seed):
    rng = np.random.default_rng(500 + seed)
    H = int(rng.integers(5, 40))
    N = int(rng.integers(1, 6))
    n_in = int(rng.integers(0, 5))
    n_q = int(rng.integers(1, 8))
    R = n_in + n_q
    inp = _inflight_board(rng, R, H, N, pmax=20, gmax=5, rmax=H)
    arr = np.sort(rng.integers(0, H + 3, n_q)).astype(np.int32)
    inp["arrival"][n_in:] = arr
    inp["generated"][n_in:] = 0
    cap_kv = int(rng.integers(5, 60))
    inp["kv_capacity"] = np.array([cap_kv], np.int32)
    cap_b = int(rng.integers(1, 6)) if rng.random() < 0.5 else None
    inp["batch_cap"] = None if cap_b is None else np.array([cap_b], np.int32)
    out = oracle.project(inp, return_admit=True)
    a = out["admit_iter"].tolist()
    admitted = [(int(inp["prompt"][i]) + int(inp["generated"][i]), 0, int(inp["remaining"][i]))
                for i in range(n_in)]
    prev = 0
    for k in range(n_in, R):
        c, L, arrk = int(inp["prompt"][k]), int(inp["remaining"][k]), int(arr[k - n_in])
        start = max(prev, arrk)
        if a[k] == -1:
            for j in range(start, H):
                assert not _check_rule(H, N, cap_kv, cap_b, admitted, (c, L), j)
            assert all(x == -1 for x in a[k:])
            break
        assert a[k] >= start
        for j in range(start, a[k]):
            assert not _check_rule(H, N, cap_kv, cap_b, admitted, (c, L), j), (k, j)
        assert _check_rule(H, N, cap_kv, cap_b, admitted, (c, L), a[k])
        admitted.append((c, a[k], L))
        prev = a[k]
    B, KV = simulate_engine(H, N, admitted)
    assert out["batch"][0].tolist() == B.tolist()
    assert out["kv"][0].tolist() == KV.tolist()


# ----------------------------------------------------------------- invariants

@st.composite
def boards(draw):
    H = draw(st.integers(1, 40))
    N = draw(st.integers(1, 8))
    R = draw(st.integers(0, 14))
    p = draw(st.lists(st.integers(0, 40), min_size=R, max_size=R))
    g = draw(st.lists(st.integers(0, 10), min_size=R, max_size=R))
    r = draw(st.lists(st.integers(1, 50), min_size=R, max_size=R))
    n_q = draw(st.integers(0, R))
    arr = sorted(draw(st.lists(st.integers(0, H + 3), min_size=n_q, max_size=n_q)))
    arrival = [-1] * (R - n_q) + arr
    cap = draw(st.integers(0, 150))
    bcap = draw(st.one_of(st.none(), st.integers(1, 8)))
    return dict(n_scenarios=1, horizon=H, block_tokens=N, req_offset=np.array([0, R], np.int64),
                prompt=np.array(p, np.int32), generated=np.array(g, np.int32),
                remaining=np.array(r, np.int32), arrival=np.array(arrival, np.int32),
                deadline_ns=None, lost=None, kv_capacity=np.array([cap], np.int32),
                batch_cap=None if bcap is None else np.array([bcap], np.int32))


@settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(boards())
def test_projection_invariants(inp):
    out = oracle.project(inp, return_admit=True)
    B, KV, a = out["batch"][0], out["kv"][0], out["admit_iter"]
    H = inp["horizon"]
    fl = int(out["flags"][0])
    queued = inp["arrival"] >= 0
    if not fl & oracle.FLAG_OVERCOMMIT:
        assert np.all(KV <= inp["kv_capacity"][0])
        if inp["batch_cap"] is not None:
            assert np.all(B <= inp["batch_cap"][0])
    if not queued.any():
        assert np.all(np.diff(B) <= 0), "batch must not grow without arrivals"
    c = inp["prompt"].astype(np.int64) + inp["generated"]
    if np.all(c >= 1):
        assert np.all(KV >= B)
    e = np.where(a >= 0, a + inp["remaining"].astype(np.int64), -1)
    occupied = sum(min(int(e[i]), H) - int(a[i]) for i in range(a.size) if a[i] >= 0)
    assert int(B.sum()) == occupied
    aq = a[queued]
    adm = aq[aq >= 0]
    assert np.all(np.diff(adm) >= 0), "FIFO: admission times follow queue order"
    if (aq == -1).any():
        assert np.all(aq[np.argmax(aq == -1):] == -1), "a blocked head blocks the queue"
    assert np.all(a[queued & (a >= 0)] >= inp["arrival"][queued & (a >= 0)])
    n = int(out["n_iters"][0])
    assert n == (max([min(int(x), H) for x in e[a >= 0]]) if (a >= 0).any() else 0)


def test_deadline_map_and_lost():
    """Deadlines land on the last in-batch iteration of requests finishing in
    the horizon; lost requests are ignored and flag the scenario (Sec. 4.3.2,
    Sec. 4.5); the minimum wins when two requests finish together."""
    inp = dict(n_scenarios=1, horizon=6, block_tokens=4, req_offset=np.array([0, 4], np.int64),
               prompt=np.array([1, 1, 1, 1], np.int32), generated=np.zeros(4, np.int32),
               remaining=np.array([3, 3, 9, 2], np.int32), arrival=np.full(4, -1, np.int32),
               deadline_ns=np.array([70, 50, 10, 5], np.uint64), lost=np.array([0, 0, 0, 1], np.uint8),
               kv_capacity=np.array([100], np.int32), batch_cap=None)
    out = oracle.project(inp)
    assert out["deadline_at"][0].tolist() == [int(NONE), int(NONE), 50, int(NONE), int(NONE), int(NONE)]
    assert int(out["flags"][0]) == oracle.FLAG_LOST
    assert int(out["n_iters"][0]) == 6


def test_size_guard_and_bad_entries():
    H, N = 16, 1
    big = 1 << 30
    one = dict(n_scenarios=2, horizon=H, block_tokens=N, req_offset=np.array([0, 1, 4], np.int64),
               prompt=np.array([big, big, big, big], np.int32), generated=np.zeros(4, np.int32),
               remaining=np.array([4, 4, 4, 4], np.int32), arrival=np.full(4, -1, np.int32),
               deadline_ns=None, lost=None, kv_capacity=np.array([2**31 - 1] * 2, np.int32),
               batch_cap=None)
    out = oracle.project(one)
    assert int(out["flags"][0]) == 0 and out["kv"][0, 0] == big
    assert int(out["flags"][1]) == oracle.FLAG_OVERFLOW
    assert out["kv"][1].sum() == 0 and out["n_iters"][1] == 0
    bad = dict(one, n_scenarios=1, req_offset=np.array([0, 4], np.int64),
               prompt=np.array([-1, 5, 5, big + 1], np.int32), remaining=np.array([3, 0, 2, 1], np.int32),
               kv_capacity=np.array([1000], np.int32))
    out = oracle.project(bad)
    assert int(out["flags"][0]) == oracle.FLAG_BAD_REQUEST
    assert out["batch"][0].tolist()[:3] == [1, 1, 0]


def test_unsorted_queue_flag():
    inp = dict(n_scenarios=1, horizon=10, block_tokens=4, req_offset=np.array([0, 2], np.int64),
               prompt=np.array([4, 4], np.int32), generated=np.zeros(2, np.int32),
               remaining=np.array([2, 2], np.int32), arrival=np.array([5, 3], np.int32),
               deadline_ns=None, lost=None, kv_capacity=np.array([100], np.int32), batch_cap=None)
    out = oracle.project(inp, return_admit=True)
    assert int(out["flags"][0]) & oracle.FLAG_UNSORTED
    # FIFO in array order: the head (arrival 5) blocks the entry behind it
    assert out["admit_iter"].tolist() == [5, 5]


# -------------------------------------------------------------------- forest

def _f32_down(t):
    c = np.float32(t)
    if float(c) > t:
        c = np.nextafter(c, np.float32(-np.inf))
    return c


def _complete_from_sklearn(tree, depth, values):
    """Heap-ordered complete tree equivalent to a fitted sklearn tree.
    sklearn goes left iff x <= t (fp32 x, fp64 t); that equals
    x < nextup(largest fp32 <= t).  Shallow leaves are pushed down through
    always-left nodes (threshold +inf)."""
    n_int = (1 << depth) - 1
    feat = np.zeros(n_int, np.uint8)
    thr = np.zeros(n_int, np.float32)
    leaf = np.zeros(1 << depth, np.float32)
    tl, tr = tree.children_left, tree.children_right

    def rec(node, k, level):
        if level == depth:
            leaf[k - n_int] = values[node]
            return
        if tl[node] == -1:
            feat[k] = 0
            thr[k] = np.float32(np.inf)
            rec(node, 2 * k + 1, level + 1)
            fill(2 * k + 2, level + 1)
            return
        feat[k] = tree.feature[node]
        thr[k] = np.nextafter(_f32_down(float(tree.threshold[node])), np.float32(np.inf))
        rec(tl[node], 2 * k + 1, level + 1)
        rec(tr[node], 2 * k + 2, level + 1)

    def fill(k, level):
        if level == depth:
            leaf[k - n_int] = 0.0
            return
        feat[k] = 0
        thr[k] = np.float32(np.inf)
        fill(2 * k + 1, level + 1)
        fill(2 * k + 2, level + 1)

    rec(0, 0, 0)
    return feat, thr, leaf


def _feature_rows(rng, n, nf):
    cols = [rng.choice(np.arange(1000, 2001, 25), n).astype(np.float32),
            rng.integers(0, 4000, n).astype(np.float32),
            rng.integers(0, 64, n).astype(np.float32),
            rng.choice([1.0, 2.0, 4.0, 8.0], n).astype(np.float32)]
    return np.stack(cols[:nf], axis=1)


@pytest.mark.parametrize("nf,depth", [(3, 4), (4, 6), (3, 8)])
def test_forest_matches_sklearn_traversal(nf, depth):
    from sklearn.tree import DecisionTreeRegressor
    rng = np.random.default_rng(7 + depth)
    X = _feature_rows(rng, 3000, nf)
    T = 12
    feats, thrs, leaves = [], [], []
    base = np.float32(40.0)
    Xq = _feature_rows(rng, 2500, nf)
    # include exact ties with training values so thresholds are hit from both sides
    Xq[:500] = X[:500]
    expect = np.zeros(Xq.shape[0])
    for t in range(T):
        y = rng.normal(size=X.shape[0])
        md = depth if t % 3 else max(1, depth - 2)   # some shallower trees
        skt = DecisionTreeRegressor(max_depth=md, random_state=t).fit(X, y).tree_
        values = (rng.integers(-1000, 1000, skt.node_count) / 64.0).astype(np.float32)
        f, th, lf = _complete_from_sklearn(skt, depth, values)
        feats.append(f); thrs.append(th); leaves.append(lf)
        expect += values[skt.apply(Xq)].astype(np.float64)
    forest = dict(n_trees=T, depth=depth, n_features=nf, base_score=base,
                  feature=np.stack(feats), threshold=np.stack(thrs), leaf=np.stack(leaves))
    got = oracle.forest_predict(forest, Xq)
    assert np.array_equal(got, (expect + 40.0).astype(np.float32))


def _forest(T, d, nf, feat, thr, leaf, base=0.0):
    return dict(n_trees=T, depth=d, n_features=nf, base_score=np.float32(base),
                feature=np.broadcast_to(np.asarray(feat, np.uint8), (T, (1 << d) - 1)).copy(),
                threshold=np.broadcast_to(np.asarray(thr, np.float32), (T, (1 << d) - 1)).copy(),
                leaf=np.broadcast_to(np.asarray(leaf, np.float32), (T, 1 << d)).copy())


def test_forest_closed_forms():
    rng = np.random.default_rng(3)
    X = _feature_rows(rng, 100, 3)
    d = 5
    leaf = rng.normal(size=(7, 1 << d)).astype(np.float32)
    f_in = _forest(7, d, 3, 1, np.inf, 0, base=1.5)
    f_in["leaf"] = leaf
    # every row reaches leaf 0 (all thresholds +inf: always left) or the last
    # leaf (-inf: always right) of every tree; the sum runs in fp32, tree order
    def running_sum(base, vals):
        acc = np.float32(base)
        for v in vals:
            acc = np.float32(acc + v)
        return acc
    assert np.array_equal(oracle.forest_predict(f_in, X), np.full(100, running_sum(1.5, leaf[:, 0])))
    f_in["threshold"][:] = -np.inf
    assert np.array_equal(oracle.forest_predict(f_in, X), np.full(100, running_sum(1.5, leaf[:, -1])))
    same = _forest(300, 3, 3, 2, 10.0, 0.5, base=2.0)
    assert np.all(oracle.forest_predict(same, X) == np.float32(2.0 + 0.5 * 300))
    # depth-1 stump on the frequency: closed form
    stump = _forest(1, 1, 3, 0, 1500.0, [3.0, 7.0])
    got = oracle.forest_predict(stump, X)
    assert np.array_equal(got, np.where(X[:, 0] < 1500.0, 3.0, 7.0).astype(np.float32))


def test_forest_tie_nan_depth0_and_fp32_running_sum():
    stump = _forest(1, 1, 3, 1, 100.0, [1.0, 2.0])
    x = np.array([[1000, 100, 0], [1000, 99.99999, 0], [1000, np.nan, 0]], np.float32)
    assert oracle.forest_predict(stump, x).tolist() == [2.0, 1.0, 2.0]   # x == thr and NaN go right
    d0 = dict(n_trees=3, depth=0, n_features=3, base_score=np.float32(1.0),
              feature=np.zeros((3, 0), np.uint8), threshold=np.zeros((3, 0), np.float32),
              leaf=np.array([[0.25], [0.5], [1.0]], np.float32))
    assert oracle.forest_predict(d0, x).tolist() == [2.75] * 3
    # an fp32 running sum from the base: each 2^-25 is below half an ulp of
    # 1.0 and is lost (fp64 accumulation would give 1 + 3*2^-25 -> 1 + 2^-23)
    tiny = _forest(3, 1, 3, 0, 0.0, [2.0 ** -25, 2.0 ** -25], base=1.0)
    assert oracle.forest_predict(tiny, x[:1])[0] == np.float32(1.0)
    # 1 + 2^-24 is a tie that rounds to even (1.0), twice; the two leaves
    # added first would give 1 + 2^-23 exactly: the base comes first and the
    # trees follow in order
    tie = _forest(2, 1, 3, 0, 0.0, [2.0 ** -24, 2.0 ** -24], base=1.0)
    assert oracle.forest_predict(tie, x[:1])[0] == np.float32(1.0)
    # tree order: 2^24 + 1 - 2^24 is 0 in fp32 (2^24 + 1 rounds to 2^24),
    # the reverse order 1 - 2^24 + 2^24 is 1
    fwd = _forest(3, 1, 3, 0, 0.0, [0.0, 0.0])
    fwd["leaf"] = np.array([[2.0 ** 24] * 2, [1.0] * 2, [-(2.0 ** 24)] * 2], np.float32)
    assert oracle.forest_predict(fwd, x[:1])[0] == np.float32(0.0)
    rev = dict(fwd, leaf=fwd["leaf"][::-1].copy())
    assert oracle.forest_predict(rev, x[:1])[0] == np.float32(1.0)
    # a running sum that crosses 2^24: (2^24 - 1) + 1 + 1 + 1 is exactly
    # 2^24 + 2 (representable), but after the first add every 2^24 + 1 rounds
    # back to 2^24 (even)
    cross = _forest(3, 1, 3, 0, 0.0, [1.0, 1.0], base=2.0 ** 24 - 1)
    assert oracle.forest_predict(cross, x[:1])[0] == np.float32(2.0 ** 24)


def test_forest_rejects_bad_feature():
    bad = _forest(1, 1, 3, 3, 0.0, [0.0, 0.0])
    with pytest.raises(ValueError):
        oracle.forest_predict(bad, np.zeros((1, 3), np.float32))


# ------------------------------------------------------- latency (T' = 1/T)

def test_latency_exact_values():
    L = oracle.latency_ns
    assert L(50.0) == 20_000_000
    assert L(75.0) == 13_333_334
    assert L(3.0) == 333_333_334
    assert L(1e9) == 1
    assert L(1e30) == 1
    assert L(float("inf")) == 0
    for bad in (0.0, -0.0, -5.0, float("nan"), float("-inf"), 1e-3 * 2.0 ** -20):
        assert L(bad) == oracle.LAT_SATURATED


def test_latency_against_exact_rationals():
    """ceil(1e9/x) computed in exact rationals; the fp64 route may only differ
    where the exact quotient lies within one fp64 ulp above an integer."""
    rng = np.random.default_rng(11)
    xs = np.concatenate([rng.uniform(1, 200, 20000), rng.uniform(1e-2, 1e6, 5000)]).astype(np.float32)
    xs = np.concatenate([xs, np.float32([1, 2, 4, 5, 8, 10, 16, 20, 25, 40, 64, 80, 125, 128])])
    mism = 0
    for x in xs:
        q = Fraction(10 ** 9) / Fraction(float(x))
        exact = -((-q.numerator) // q.denominator)
        got = oracle.latency_ns(float(x))
        if got != exact:
            mism += 1
            assert got == exact - 1 and q - (exact - 1) < Fraction(1, 2 ** 20)
    assert mism <= 3


# ---------------------------------------------------------------- selection

def _sel_inputs(rng, S, F, H):
    ips = rng.uniform(10, 100, (S, F, H)).astype(np.float32)
    n = rng.integers(0, H + 1, S).astype(np.int32)
    dl = np.full((S, H), NONE, np.uint64)
    for s in range(S):
        for j in rng.choice(max(int(n[s]), 1), size=min(3, max(int(n[s]), 1)), replace=False):
            if j < n[s]:
                dl[s, j] = np.uint64(rng.integers(1, 60_000_000) * (j + 1))
    tbt = rng.integers(8_000_000, 60_000_000, S).astype(np.uint64)
    return ips, dl, n, tbt


def test_binary_search_equals_sweep_when_monotone():
    rng = np.random.default_rng(5)
    S, F, H = 200, 16, 40
    ips, dl, n, tbt = _sel_inputs(rng, S, F, H)
    ips = np.sort(ips, axis=1)          # faster at every higher frequency
    a = oracle.select(ips, dl, n, tbt)
    b = oracle.select_binary(ips, dl, n, tbt)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert (a[1] == 0).sum() > 20 and (a[1] == 1).sum() > 5


def test_binary_search_check_of_lo_is_known_when_hi_moved():
    """Sec. 4.5's search as the oracle runs it, replayed over the oracle's
    own feasibility at every frequency (unsorted IPS: feasibility far from
    monotone).  hi moves only to a probe found feasible and no probe is F-1
    (the midpoint of lo < hi lies below hi), so whenever hi ends below F-1,
    lo == hi was probed and found feasible: the final check of lo then
    decides nothing new, and answering lo (OK) without it gives the oracle's
    answer.  Only searches whose hi stayed at F-1 need that evaluation."""
    rng = np.random.default_rng(12)
    for F in (1, 2, 3, 5, 16, 48, 64, 100):
        S, H = 120, 30
        ips, dl, n, tbt = _sel_inputs(rng, S, F, H)
        feas = np.stack([oracle.select(np.ascontiguousarray(ips[:, f:f + 1]), dl, n, tbt)[1] == 0
                         for f in range(F)], axis=1)
        idx, st = oracle.select_binary(ips, dl, n, tbt)
        need_eval = 0
        for s_ in range(S):
            lo, hi, probed = 0, F - 1, {}
            while lo < hi:
                mid = lo + (hi - lo) // 2
                assert mid < F - 1
                probed[mid] = bool(feas[s_, mid])
                if probed[mid]:
                    hi = mid
                else:
                    lo = mid + 1
            assert lo == hi
            if hi < F - 1:
                assert probed.get(lo) is True
                assert (idx[s_], st[s_]) == (lo, 0)
            else:
                need_eval += 1
                assert (idx[s_], st[s_]) == ((lo, 0) if feas[s_, lo] else (F - 1, 1))
        assert 0 < need_eval <= S and (F == 1 or need_eval < S)


def test_selection_monotone_in_slo_and_ips():
    rng = np.random.default_rng(6)
    S, F, H = 150, 12, 30
    ips, dl, n, tbt = _sel_inputs(rng, S, F, H)
    idx0, st0 = oracle.select(ips, dl, n, tbt)
    idx1, st1 = oracle.select(ips, dl, n, tbt + np.uint64(5_000_000))
    # a looser TBT SLO never raises the frequency (deadlines unchanged)
    assert np.all(idx1 <= idx0)
    idx2, _ = oracle.select(ips * np.float32(1.3), dl, n, tbt)
    assert np.all(idx2 <= idx0)


def test_selection_chooses_lowest_feasible():
    """The chosen f passes both checks and every lower one fails: verified
    with per-iteration times from exact rationals and Python integers."""
    rng = np.random.default_rng(9)
    S, F, H = 40, 8, 25
    ips, dl, n, tbt = _sel_inputs(rng, S, F, H)
    idx, stt = oracle.select(ips, dl, n, tbt)

    def ok(s, f):
        if n[s] == 0:
            return True
        acc = 0
        for j in range(int(n[s])):
            q = Fraction(10 ** 9) / Fraction(float(ips[s, f, j]))
            acc += -((-q.numerator) // q.denominator)
            if dl[s, j] != NONE and not acc < int(dl[s, j]):
                return False
        return acc <= int(tbt[s]) * int(n[s])

    for s in range(S):
        feas = [ok(s, f) for f in range(F)]
        if any(feas):
            assert stt[s] == 0 and idx[s] == feas.index(True)
        else:
            assert stt[s] == 1 and idx[s] == F - 1


def test_selection_special_cases():
    S, F, H = 4, 5, 10
    ips = np.full((S, F, H), 1e30, np.float32)
    dl = np.full((S, H), NONE, np.uint64)
    dl[:, 3] = 5                                   # 4 iterations at 1 ns each: 4 < 5
    n = np.array([10, 0, 10, 10], np.int32)
    tbt = np.array([1, 1, 1, 1], np.uint64)
    flags = np.array([0, 0, oracle.FLAG_LOST, oracle.FLAG_OVERFLOW | oracle.FLAG_LOST], np.uint32)
    idx, stt = oracle.select(ips, dl, n, tbt, flags)
    assert idx.tolist() == [0, 0, F - 1, F - 1]
    assert stt.tolist() == [0, 0, oracle.STATUS_LOST, oracle.STATUS_INVALID]
    ips[:] = 0.0
    idx, stt = oracle.select(ips, dl, n, tbt, np.zeros(S, np.uint32))
    assert idx.tolist() == [F - 1, 0, F - 1, F - 1]
    assert stt.tolist() == [1, 0, 1, 1]
    # deadlines are strict (Eq. 4): time exactly at the deadline fails
    ips[:] = 1e30
    dl[:, 3] = 4
    idx, stt = oracle.select(ips, dl, n, tbt, np.zeros(S, np.uint32))
    assert stt.tolist() == [1, 0, 1, 1]


# ------------------------------------------ admission control (Sec. 4.3.2)

def _admit_board(g, case):
    sigma = case["sigma_ns"]
    inp = goldens.scoreboard(g, deadline_ns=[sigma * r for r in g["remaining"]], lost=case.get("lost"))
    if "kv_capacity" in case:
        inp["kv_capacity"] = np.array([case["kv_capacity"]], np.int32)
    if "batch_cap" in case:
        inp["batch_cap"] = np.array([case["batch_cap"]], np.int32)
    inp["tbt_slo_ns"] = np.array([sigma], np.uint64)
    return inp


def test_golden_admission():
    g = goldens.load("admit_two_stumps.json")
    forest = goldens.forest(g)
    for case in g["cases"]:
        inp = _admit_board(g, case)
        d = case["cand_deadline"]
        out = oracle.admit(inp, [case["cand_prompt"]], [case["cand_len"]],
                           None if d is None else np.array([d], np.uint64), g["max_freq_mhz"], forest)
        assert int(out["decision"][0]) == case["decision"], case["note"]
        ex = g["expect_by_len"].get(str(case["cand_len"]))
        if ex is not None and case["decision"] != oracle.QUEUE_CAPACITY:
            assert out["kv"][0].tolist() == ex["kv"]
            assert out["batch"][0].tolist() == ex["batch"]
            assert out["ips"][0].tolist() == ex["ips"]


def test_golden_admission_engine_size_two_scenarios():
    """Admission on several scenarios with a four-feature model: check 2
    queries M with each scenario's own engine size (hand-computed)."""
    g = goldens.load("admit_engine_size_two_scenarios.json")
    forest = goldens.forest(g)
    for case in g["cases"]:
        inp = goldens.scoreboard_multi(dict(g, kv_capacity=case["kv_capacity"]), case["sigma_ns"])
        inp["forest"] = forest
        d = case["cand_deadline"]
        out = oracle.admit(inp, g["cand_prompt"], g["cand_len"],
                           None if d is None else np.array(d, np.uint64), g["max_freq_mhz"])
        assert out["decision"].tolist() == case["decision"], case["note"]
        for s, dec in enumerate(case["decision"]):
            assert out["batch"][s].tolist() == g["expect_batch"][s]
            assert out["kv"][s].tolist() == g["expect_kv"][s]
            if dec != oracle.QUEUE_CAPACITY:
                assert out["ips"][s].tolist() == g["expect_ips"][s]


def _random_admission(rng, queued):
    H = int(rng.integers(4, 40))
    N = int(rng.integers(1, 9))
    R = int(rng.integers(0, 12))
    inp = _inflight_board(rng, R, H, N, pmax=40, gmax=10, rmax=H + 6)
    if queued and R:
        q = rng.random(R) < 0.3
        inp["arrival"] = np.where(q, np.sort(rng.integers(0, H, R)), -1).astype(np.int32)
        inp["generated"] = np.where(q, 0, inp["generated"]).astype(np.int32)
    p = int(rng.integers(0, 40))
    L = int(rng.integers(1, H + 8))
    sigma = int(rng.integers(5_000_000, 40_000_000))
    inp["deadline_ns"] = (inp["remaining"] * sigma * rng.uniform(0.6, 1.6, R)).astype(np.uint64) + np.uint64(1)
    inp["lost"] = (rng.random(R) < 0.1).astype(np.uint8)
    kvmax = int(oracle.project(inp)["kv"].max()) if H else 0
    margin = (p + L) // N + 2 if rng.random() < 0.75 else 0
    inp["kv_capacity"] = np.array([kvmax + margin + int(rng.integers(-2, 4))], np.int32)
    if rng.random() < 0.3:
        inp["batch_cap"] = np.array([R + int(rng.integers(0, 3))], np.int32)
    inp["tbt_slo_ns"] = np.array([sigma], np.uint64)
    T, d = int(rng.integers(1, 5)), int(rng.integers(1, 4))
    forest = dict(n_trees=T, depth=d, n_features=3, base_score=np.float32(30.0),
                  feature=rng.integers(0, 3, (T, (1 << d) - 1)).astype(np.uint8),
                  threshold=np.stack([rng.choice([1100.0, 1500.0, 1900.0, 50.0, 200.0, 2.0, 5.0, 9.0],
                                                 (1 << d) - 1) for _ in range(T)]).astype(np.float32),
                  leaf=rng.uniform(-20, 40, (T, 1 << d)).astype(np.float32))
    dc = np.uint64(1 + sigma * L * rng.uniform(0.6, 1.6)) if rng.random() < 0.8 else NONE
    return inp, forest, p, L, dc


def _controller_feasible(inp, forest, p, L, dc, fmax):
    """Check 2 and 3 by the controller's own selection (Sec. 4.5) on the board
    with the query appended, at the single frequency fmax."""
    R = int(inp["req_offset"][-1])
    b = dict(inp)
    b["req_offset"] = np.array([0, R + 1], np.int64)
    for k, v in (("prompt", p), ("generated", 0), ("remaining", L), ("arrival", -1)):
        b[k] = np.append(inp[k], np.int32(v)).astype(np.int32)
    b["deadline_ns"] = np.append(inp["deadline_ns"], np.uint64(dc)).astype(np.uint64)
    b["lost"] = np.append(inp["lost"], np.uint8(0)).astype(np.uint8)
    proj = oracle.project(b)
    x = oracle.rows(np.array([fmax], np.float32), proj["batch"], proj["kv"], None, 3)
    ips = oracle.forest_predict(forest, x)
    _, stt = oracle.select(ips, proj["deadline_at"], proj["n_iters"], inp["tbt_slo_ns"], None)
    return int(stt[0]) == oracle.STATUS_OK, proj


@pytest.mark.parametrize("queued", [False, True])
def test_admission_agrees_with_controller_and_brute_force(queued):
    """Checks 2-3 of the admission decision equal the controller's
    feasibility at the maximum frequency (with and without the query's own
    deadline); check 1 equals a brute-force maximum of Eq. 1 over the
    requests running now."""
    rng = np.random.default_rng(40 + queued)
    seen = set()
    fmax = 2000.0
    for _ in range(150):
        inp, forest, p, L, dc = _random_admission(rng, queued)
        dec = int(oracle.admit(inp, [p], [L], np.array([dc], np.uint64), fmax, forest)["decision"][0])
        seen.add(dec)
        with_own, proj = _controller_feasible(inp, forest, p, L, dc, fmax)
        without_own, _ = _controller_feasible(inp, forest, p, L, NONE, fmax)
        H, N = int(inp["horizon"]), int(inp["block_tokens"])
        running = [(int(a) + int(g), int(r)) for a, g, r, ar in
                   zip(inp["prompt"], inp["generated"], inp["remaining"], inp["arrival"]) if ar == -1]
        running.append((p, L))
        kv_now = [sum(-(-(c + j) // N) for c, r in running if j < r) for j in range(H)]
        over = max(kv_now) > int(inp["kv_capacity"][0])
        bcap = inp.get("batch_cap")
        over_b = bcap is not None and len(running) > int(bcap[0])
        if dec == oracle.QUEUE_CAPACITY:
            assert over or over_b
            continue
        assert not over and not over_b
        if dec == oracle.ADMIT_OK:
            assert with_own and without_own
        elif dec == oracle.ADMIT_LOST:
            assert without_own and not with_own and L <= H
        else:
            assert dec in (oracle.QUEUE_TBT, oracle.QUEUE_E2E) and not without_own
    assert {oracle.ADMIT_OK, oracle.QUEUE_CAPACITY} <= seen and len(seen) >= 4, seen


def test_admission_monotone_in_slo_and_own_deadline():
    rng = np.random.default_rng(77)
    fmax = 2000.0
    changed = 0
    for _ in range(120):
        inp, forest, p, L, dc = _random_admission(rng, False)
        d0 = int(oracle.admit(inp, [p], [L], np.array([dc], np.uint64), fmax, forest)["decision"][0])
        loose = dict(inp, tbt_slo_ns=inp["tbt_slo_ns"] * np.uint64(2))
        d1 = int(oracle.admit(loose, [p], [L], np.array([dc], np.uint64), fmax, forest)["decision"][0])
        # a looser TBT SLO (deadlines unchanged) only lifts a TBT queueing
        assert d1 == d0 or d0 == oracle.QUEUE_TBT
        changed += d1 != d0
        later = NONE if dc == NONE else np.uint64(int(dc) + 50_000_000)
        d2 = int(oracle.admit(inp, [p], [L], np.array([later], np.uint64), fmax, forest)["decision"][0])
        assert d2 == d0 or (d0 == oracle.ADMIT_LOST and d2 == oracle.ADMIT_OK)


# ------------------------------------ generation-length errors (Sec. 4.6)

def test_adjust_lengths_hand_values():
    """Hand-computed entries: inflation rounded up, the max_tokens limit, the
    overrun reset to max_tokens, and malformed entries."""
    # scenario 0: factor 3/2, max 100; scenario 1: factor 1, max 64;
    # scenario 2: factor 2, max 150; scenario 3: no inflation (den 0), no limit
    off = [0, 3, 6, 8, 11]
    gen = [10, 0, 5,    30, 70, 3,    0, 149,    4, -1, 2]
    pred = [15, 1, 7,   20, 20, 60,   100, 90,   9, 5, 0]
    num, den, mt = [3, 1, 2, 7], [2, 1, 1, 0], [100, 64, 150, 0]
    want = [
        13,   # ceil(15 * 1.5) = 23 tokens, 10 generated
        2,    # ceil(1.5) = 2
        6,    # ceil(10.5) = 11, 5 generated
        34,   # 20 tokens but 30 generated: overrun -> 64 - 30
        1,    # overrun -> 64, already past it: ends now
        57,   # 60 - 3, no inflation at factor 1
        150,  # 200 limited to 150
        1,    # 180 -> 150, 149 generated
        5,    # den 0: 9 - 4
        0,    # negative generated count: malformed
        0,    # predicted length 0: malformed
    ]
    got = oracle.adjust_lengths(off, gen, pred, num, den, mt)
    assert got.tolist() == want


def test_adjust_lengths_identity_and_monotone():
    rng = np.random.default_rng(3)
    n = 500
    gen = rng.integers(0, 300, n)
    pred = gen + rng.integers(1, 300, n)
    off = [0, n]
    # factor 1 without a limit leaves the scoreboard's remaining counts
    assert oracle.adjust_lengths(off, gen, pred, [5], [5], [0]).tolist() == (pred - gen).tolist()
    base = oracle.adjust_lengths(off, gen, pred, [11], [10], [1 << 20])
    more = oracle.adjust_lengths(off, gen, pred, [13], [10], [1 << 20])
    assert np.all(more >= base) and np.all(base >= pred - gen) and np.all(base >= 1)
