"""Parity at the five workloads' full sizes, in the configuration bench.py
times (fused grid prediction): the projection of every scenario (c4: two
blocks of 512 scenarios), whole scenarios end to end, the selection stage
on every scenario (c4: four blocks of 2048; the oracle's selection on the
GPU's IPS), a million random forest rows, and properties over every
scenario.  The oracle runs in threads (its C calls release the interpreter
lock), each on its own scenarios."""
import os
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from paper_2408_05235_amd import configs, synth

pytestmark = pytest.mark.gpu

RTOL = 1e-5
WORKERS = max(1, min(16, len(os.sched_getaffinity(0))))


def _np(t, dtype=None):
    a = t.detach().cpu().numpy()
    return a.view(dtype) if dtype is not None else a


# (config, scenarios checked end to end, scenario ranges whose projection is
# compared: None = all of them in one oracle call)
PLAN = {0: ([0], None), 1: ([0, 1023], None), 2: ([0, 255], None),
        3: ([0, 1, 2047, 4095], None), 4: ([0, 16383], [(0, 512), (15872, 16384)])}
# c4's selection: blocks of 2048 scenarios (its IPS takes 805 MB per block)
SELECT_BLOCKS = {4: [0, 4096, 8192, 14336]}


def _project_ranges(inp, ranges):
    """Oracle projection of scenario ranges, 64 scenarios per task."""
    tasks = [(a, min(a + 64, hi)) for lo, hi in ranges for a in range(lo, hi, 64)]

    def run(ab):
        a, b = ab
        return a, oracle.project(synth.subset(inp, list(range(a, b))))
    with ThreadPoolExecutor(WORKERS) as ex:
        return list(ex.map(run, tasks))


def _check_projection(got, o, s0, where):
    n = o["kv"].shape[0]
    for k in ("batch", "kv", "deadline_at", "n_iters", "flags"):
        a, b = got[k][s0:s0 + n], o[k]
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)[0]
            raise AssertionError(f"{where}: {k} differs at scenario {s0 + bad[0]} {bad[1:].tolist()}")


@pytest.mark.parametrize("ci", range(5), ids=[c["name"] for c in configs.CONFIGS])
def test_full_size(gpu, ci):
    import torch
    from paper_2408_05235_amd import api

    cfg = configs.get_config(ci)
    t0 = time.time()
    inp = synth.make_inputs(cfg)
    print(f"{cfg['name']}: inputs {time.time() - t0:.1f}s", flush=True)
    forest = api.Forest.from_dict(inp["forest"])
    ctl = api.Controller(api.upload(inp), forest)
    idx, st = ctl.step()
    torch.cuda.synchronize()
    print(f"{cfg['name']}: gpu step done {time.time() - t0:.1f}s", flush=True)
    S, H, F = inp["n_scenarios"], inp["horizon"], inp["n_freqs"]
    kv, batch = _np(ctl.buf["kv"]), _np(ctl.buf["batch"])
    dl, n_iters = _np(ctl.buf["deadline_at"], np.uint64), _np(ctl.buf["n_iters"])
    flags = _np(ctl.buf["flags"], np.uint32)
    idx, st = _np(idx), _np(st).view(np.uint32)
    got = dict(batch=batch, kv=kv, deadline_at=dl, n_iters=n_iters, flags=flags)

    # projection: every scenario in one oracle call ([S][H] layout), or c4's
    # two blocks of 1024 scenarios
    full, ranges = PLAN[ci]
    if ranges is None:
        _check_projection(got, oracle.project(inp), 0, cfg["name"])
        n_proj = S
    else:
        n_proj = 0
        for s0, o in _project_ranges(inp, ranges):
            _check_projection(got, o, s0, cfg["name"])
            n_proj += o["kv"].shape[0]
    print(f"{cfg['name']}: projection of {n_proj} scenarios ok {time.time() - t0:.1f}s", flush=True)

    # whole scenarios end to end (rows, forest, selection by the oracle)
    def e2e(s):
        return s, oracle.end_to_end(synth.subset(inp, [s]))
    with ThreadPoolExecutor(min(WORKERS, len(full))) as ex:
        for s, o in ex.map(e2e, full):
            g = _np(ctl.ips[s])
            exact = int((g == o["ips"][0]).sum())
            assert np.allclose(g, o["ips"][0], rtol=RTOL, atol=0) and exact == g.size, (s, exact)
            assert (idx[s], st[s]) == (o["freq_idx"][0], o["status"][0]), s
    print(f"{cfg['name']}: {len(full)} scenarios end to end ok {time.time() - t0:.1f}s", flush=True)

    # the selection stage: the oracle's selection on the GPU's own
    # projections and IPS, every scenario (c4: four blocks of 2048)
    n_sel = 0
    for b0 in SELECT_BLOCKS.get(ci, [0]):
        blk = slice(b0, min(S, b0 + (2048 if ci in SELECT_BLOCKS else S)))
        ips_blk = _np(ctl.ips[blk])
        oi, os_ = oracle.select(ips_blk, dl[blk], n_iters[blk], inp["tbt_slo_ns"][blk], flags[blk])
        assert np.array_equal(idx[blk], oi) and np.array_equal(st[blk], os_), \
            (b0, np.nonzero((idx[blk] != oi) | (st[blk] != os_))[0][:5])
        n_sel += ips_blk.shape[0]
        del ips_blk
    print(f"{cfg['name']}: selection on {n_sel} scenarios ok {time.time() - t0:.1f}s", flush=True)

    rng = np.random.default_rng(ci)
    # the forest stage on random (scenario, frequency, iteration) rows built
    # from the GPU's own curves (c3, 2000 trees of depth 10: 400 000 rows)
    n_rows = min(S * F * H, 1_000_000)
    rs = rng.integers(0, S, n_rows)
    rf = rng.integers(0, F, n_rows)
    rj = rng.integers(0, H, n_rows)
    cols = [inp["freqs_mhz"][rf], kv[rs, rj].astype(np.float32), batch[rs, rj].astype(np.float32)]
    if inp["n_features"] == 4:
        cols.append(inp["engine_size"][rs])
    x = np.stack(cols, axis=1).astype(np.float32)
    with ThreadPoolExecutor(WORKERS) as ex:
        want = np.concatenate(list(ex.map(lambda c: oracle.forest_predict(inp["forest"], c),
                                          np.array_split(x, WORKERS))))
    import torch
    flat = ctl.ips.reshape(-1)
    pos = torch.from_numpy((rs * F + rf) * H + rj).cuda()
    got = _np(flat[pos])
    assert np.array_equal(got, want), int((got != want).sum())
    print(f"{cfg['name']}: {n_rows} random rows ok {time.time() - t0:.1f}s", flush=True)

    # properties over every scenario
    assert np.all((st == oracle.STATUS_LOST) == ((flags & oracle.FLAG_LOST) != 0))
    assert np.all(idx[st != oracle.STATUS_OK] == F - 1)
    assert np.all((idx >= 0) & (idx < F))
    # KV within capacity in every scenario whose in-flight batch was not
    # already over it
    ok_s = (flags & oracle.FLAG_OVERCOMMIT) == 0
    assert np.all(kv[ok_s] <= inp["kv_capacity"][ok_s, None])
    if inp.get("batch_cap") is not None:
        assert np.all(batch <= inp["batch_cap"][:, None])
    off = inp["req_offset"]
    per = np.diff(off)
    if not np.any(inp["arrival"] >= 0):
        assert np.all(np.diff(batch, axis=1) <= 0)
        assert np.array_equal(batch[:, 0], per)
        last = np.maximum.reduceat(inp["remaining"], off[:-1]) if per.min() > 0 else None
        if last is not None:
            assert np.array_equal(n_iters, np.minimum(last, H))
    forest.close()
