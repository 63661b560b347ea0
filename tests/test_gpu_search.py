"""Parity of tl_select_freq_binary (the controller's binary search over
frequencies, Sec. 4.5, with the model evaluated only at probed frequencies)
with the oracle's binary search on the model at every frequency.  Indices
and statuses must match bit for bit.  Inputs come from the seeded generators
or are written here; expected values come only from the oracle."""
import numpy as np
import pytest

import oracle
from paper_2408_05235_amd import configs, synth
from test_gpu_parity import random_curves, random_forest

pytestmark = pytest.mark.gpu

NONE = np.uint64(0xFFFFFFFFFFFFFFFF)


def _np(t):
    return t.detach().cpu().numpy()


def gpu_binary(fd, freqs, kv, bs, dl, n, tbt, flags, eng, want_ips=False):
    """(freq_idx, status) of tl_select_freq_binary, and with want_ips its
    ips_work (filled with NaN before the call)."""
    import torch
    from paper_2408_05235_amd import api
    t = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    f = api.Forest.from_dict(fd)
    work = {"ips_work": torch.full(kv.shape, float("nan"), dtype=torch.float32, device="cuda")}
    idx, st = api.tl_select_freq_binary(f, t(freqs), t(kv), t(bs), t(dl.view(np.int64)), t(n),
                                        t(tbt.view(np.int64)), None if flags is None else t(flags.view(np.int32)),
                                        t(eng), work)
    torch.cuda.synchronize()
    out = _np(idx), _np(st).view(np.uint32)
    if want_ips:
        out = out + (work["ips_work"].cpu().numpy(),)
    f.close()
    return out


def last_probes(ips, dl, n, tbt, flags):
    """The frequency each scenario's binary search evaluated M at last, from
    the oracle's feasibility at every frequency: the probes lo + (hi - lo) / 2
    while lo < hi, then lo itself unless hi moved below F-1 (a feasible probe
    at hi = lo, whose check needs no new evaluation); -1 for scenarios
    flagged lost or overflow, which probe nothing."""
    S, F = ips.shape[:2]
    feas = np.stack([oracle.select(np.ascontiguousarray(ips[:, f:f + 1]), dl, n, tbt, None)[1] == oracle.STATUS_OK
                     for f in range(F)], axis=1)
    out = np.full(S, -1, np.int64)
    for s in range(S):
        if flags is not None and flags[s] & (oracle.FLAG_LOST | oracle.FLAG_OVERFLOW):
            continue
        lo, hi, last = 0, F - 1, -1
        while lo < hi:
            mid = lo + (hi - lo) // 2
            last = mid
            if feas[s, mid]:
                hi = mid
            else:
                lo = mid + 1
        out[s] = lo if hi == F - 1 else last
    return out


def assert_last_probe_ips(got, ips, last):
    """ips_work: M at each scenario's last probe; untouched (NaN) rows for
    scenarios that probe nothing."""
    for s in range(got.shape[0]):
        if last[s] < 0:
            assert np.all(np.isnan(got[s])), s
        else:
            assert np.array_equal(got[s].view(np.uint32), ips[s, last[s]].astype(np.float32).view(np.uint32)), \
                (s, int(last[s]))


def random_checks(rng, S, H, kv):
    n = rng.integers(-2, H + 3, S).astype(np.int32)
    dl = np.full((S, H), NONE, np.uint64)
    for s in range(S):
        js = rng.integers(0, H, rng.integers(0, 6))
        dl[s, js] = (rng.uniform(0.5, 1.5, js.size) * 25e6 * (js + 1)).astype(np.uint64)
    tbt = rng.integers(8_000_000, 40_000_000, S).astype(np.uint64)
    flags = np.zeros(S, np.uint32)
    flags[rng.random(S) < 0.04] = oracle.FLAG_LOST
    flags[rng.random(S) < 0.02] |= oracle.FLAG_OVERFLOW
    return dl, n, tbt, flags


def monotone_forest(rng, T, d, nf):
    """Leaf value proportional to the lower frequency bound of the leaf's
    path.  Two frequencies f1 < f2 on one row part at a frequency node with
    threshold f1 < thr <= f2, so f2's leaf has a bound >= thr > f1 >= f1's
    bound: every tree, hence the ensemble, is non-decreasing in the frequency
    on every row, and feasibility is monotone."""
    fd = random_forest(rng, T, d, nf, kvmax=3000, bmax=200)
    n_int = (1 << d) - 1
    for t in range(T):
        for leaf in range(1 << d):
            k, lo = leaf + n_int, 1000.0
            while k > 0:
                parent = (k - 1) // 2
                thr = float(fd["threshold"][t, parent])
                if fd["feature"][t, parent] == 0 and k == 2 * parent + 2 and np.isfinite(thr):
                    lo = max(lo, thr)
                k = parent
            fd["leaf"][t, leaf] = np.float32(lo / 1000.0 * 60.0 / max(T, 1))
    fd["base_score"] = np.float32(0.0)
    return fd


@pytest.mark.parametrize("S,F,H,T,d,nf,mono,seed", [
    (40, 64, 256, 30, 6, 3, True, 0), (40, 64, 256, 30, 6, 3, False, 1), (25, 17, 100, 20, 8, 4, False, 2),
    (30, 1, 64, 10, 4, 3, False, 3), (30, 2, 70, 10, 4, 3, True, 4), (20, 100, 33, 12, 10, 4, False, 5),
    (16, 48, 513, 8, 12, 3, False, 6), (10, 3, 1, 5, 3, 3, False, 7), (12, 64, 1024, 0, 4, 3, False, 8)])
def test_binary_search_random(gpu, S, F, H, T, d, nf, mono, seed):
    rng = np.random.default_rng(700 + seed)
    fd = monotone_forest(rng, T, d, nf) if mono else random_forest(rng, T, d, nf, kvmax=3000, bmax=200)
    if not mono:
        fd["base_score"] = np.float32(45.0)
    kv, bs = random_curves(rng, S, H, kvmax=3000, bmax=200)
    freqs = synth.frequency_grid(F)
    eng = rng.choice([1.0, 2.0, 4.0, 8.0], S).astype(np.float32) if nf == 4 else None
    dl, n, tbt, flags = random_checks(rng, S, H, kv)
    idx, st, work = gpu_binary(fd, freqs, kv, bs, dl, n, tbt, flags, eng, want_ips=True)
    ips = oracle.forest_predict(fd, oracle.rows(freqs, bs, kv, eng, nf))
    oi, os_ = oracle.select_binary(ips, dl, n, tbt, flags)
    assert np.array_equal(idx, oi) and np.array_equal(st, os_), np.nonzero((idx != oi) | (st != os_))[0][:5]
    assert_last_probe_ips(work, ips, last_probes(ips, dl, n, tbt, flags))
    ei, es = oracle.select(ips, dl, n, tbt, flags)
    if mono:
        assert np.array_equal(idx, ei) and np.array_equal(st, es)
    assert len(set(st.tolist())) >= 2


@pytest.mark.parametrize("S,H", [(4096, 512), (2048, 1000), (4096, 1100), (8192, 1024)])
def test_binary_search_at_reuse_sizes(gpu, S, H):
    """Grids large enough for the column kernel with leaf reuse along each
    lane's rows: 8 rows a lane (a whole and a ragged last wavefront of
    iterations) and 16 rows a lane (ragged; and on 256 CUs at 8192 x 1024,
    two workgroups per CU, where the items follow the estimated-cost work
    order, the odd scenarios' columns first).  Half of the scenarios have a
    batch that changes at every iteration, so many rows lie outside both
    anchor leaves' boxes and walk.  Indices and statuses equal the
    oracle's."""
    rng = np.random.default_rng(777 + H)
    F, T, d, nf = 5, 20, 6, 4
    fd = random_forest(rng, T, d, nf, kvmax=3000, bmax=200)
    fd["base_score"] = np.float32(45.0)
    kv, bs = random_curves(rng, S, H, kvmax=3000, bmax=200)
    fast = np.arange(S) % 2 == 1
    nfast = int(fast.sum())
    bs[fast] = np.clip(rng.integers(20, 180, (nfast, 1)) + np.cumsum(rng.choice([-1, 1], (nfast, H)), axis=1),
                       0, None).astype(np.int32)
    freqs = synth.frequency_grid(F)
    eng = rng.choice([1.0, 2.0, 4.0, 8.0], S).astype(np.float32)
    dl, n, tbt, flags = random_checks(rng, S, H, kv)
    idx, st, work = gpu_binary(fd, freqs, kv, bs, dl, n, tbt, flags, eng, want_ips=True)
    ips = oracle.forest_predict(fd, oracle.rows(freqs, bs, kv, eng, nf))
    oi, os_ = oracle.select_binary(ips, dl, n, tbt, flags)
    assert np.array_equal(idx, oi) and np.array_equal(st, os_), np.nonzero((idx != oi) | (st != os_))[0][:5]
    assert len(set(st.tolist())) >= 2
    last = last_probes(ips, dl, n, tbt, flags)
    # some scenarios settle without a final evaluation, others need one
    assert np.any((last >= 0) & (last < F - 1)) and np.any(last == F - 1)
    assert_last_probe_ips(work, ips, last)


SCALED = [
    (0, dict()),
    (1, dict(n_scenarios=10)),
    (2, dict(n_scenarios=6)),
    (3, dict(n_scenarios=4, forest_n_trees=300)),
    (4, dict(n_scenarios=5)),
]


@pytest.mark.parametrize("ci,over", SCALED, ids=[c["name"] for c in configs.CONFIGS])
def test_binary_search_scaled_configs(gpu, ci, over):
    import torch
    from paper_2408_05235_amd import api
    cfg = synth.scaled(configs.get_config(ci), **over)
    inp = synth.make_inputs(cfg)
    ctl = api.Controller(api.upload(inp), api.Forest.from_dict(inp["forest"]))
    ctl.project()
    idx, st = ctl.select_binary()
    torch.cuda.synchronize()
    o = oracle.end_to_end(inp)
    oi, os_ = oracle.select_binary(o["ips"], o["deadline_at"], o["n_iters"], inp["tbt_slo_ns"], o["flags"])
    assert np.array_equal(_np(idx), oi) and np.array_equal(_np(st).view(np.uint32), os_)


# (config, scenarios compared with the oracle at full size)
PLAN_FULL = {1: [0, 1023], 3: [0, 1, 4095], 4: [0, 16383]}


@pytest.mark.parametrize("ci", sorted(PLAN_FULL), ids=[configs.CONFIGS[c]["name"] for c in sorted(PLAN_FULL)])
def test_binary_search_full_size(gpu, ci):
    """The binary search at a workload's full size, in the configuration the
    benchmark times (the column kernel with leaf reuse at every probe):
    sampled scenarios' indices and statuses equal the oracle's binary search
    over its model at every frequency.  The oracle runs in threads (its C
    calls release the interpreter lock)."""
    import os
    from concurrent.futures import ThreadPoolExecutor
    import torch
    from paper_2408_05235_amd import api
    cfg = configs.get_config(ci)
    inp = synth.make_inputs(cfg)
    ctl = api.Controller(api.upload(inp), api.Forest.from_dict(inp["forest"]))
    ctl.project()
    idx, st = ctl.select_binary()
    torch.cuda.synchronize()
    idx, st = _np(idx), _np(st).view(np.uint32)

    def run(s):
        sub = synth.subset(inp, [s])
        o = oracle.end_to_end(sub)
        return s, oracle.select_binary(o["ips"], o["deadline_at"], o["n_iters"], sub["tbt_slo_ns"], o["flags"])
    with ThreadPoolExecutor(max(1, min(16, len(os.sched_getaffinity(0))))) as ex:
        for s, (oi, os_) in ex.map(run, PLAN_FULL[ci]):
            assert int(idx[s]) == int(oi[0]) and int(st[s]) == int(os_[0]), (cfg["name"], s, idx[s], st[s], oi, os_)
