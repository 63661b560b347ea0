"""Parity at the five workloads' full sizes, in the configuration bench.py
times (fused grid prediction), on outputs the oracle can afford: a few whole
scenarios end to end, the selection stage on every scenario (the oracle's
selection on the GPU's IPS), a million random forest rows (400 000 on the
2000-tree workload), and properties over every scenario."""
import time

import numpy as np
import pytest

import oracle
from paper_2408_05235_amd import configs, synth

pytestmark = pytest.mark.gpu

RTOL = 1e-5


def _np(t, dtype=None):
    a = t.detach().cpu().numpy()
    return a.view(dtype) if dtype is not None else a


# (config, scenarios checked end to end, scenarios checked for projection + rows)
PLAN = {0: ([0], []), 1: ([0, 1023], [1, 517]), 2: ([0, 255], [3, 128]),
        3: ([4095], [0, 2048]), 4: ([0, 16383], [5, 9000])}


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

    full, proj_only = PLAN[ci]
    rng = np.random.default_rng(ci)
    for s in full + proj_only:
        sub = synth.subset(inp, [s])
        o = oracle.project(sub)
        assert np.array_equal(kv[s], o["kv"][0]), (s, "kv")
        assert np.array_equal(batch[s], o["batch"][0]), (s, "batch")
        assert np.array_equal(dl[s], o["deadline_at"][0]), (s, "deadline_at")
        assert n_iters[s] == o["n_iters"][0] and flags[s] == o["flags"][0], s
        # sampled rows of this scenario
        fj = rng.integers(0, F, 2000), rng.integers(0, H, 2000)
        x = oracle.rows(inp["freqs_mhz"], o["batch"], o["kv"],
                        None if sub.get("engine_size") is None else sub["engine_size"], inp["n_features"])[0]
        want = oracle.forest_predict(inp["forest"], x[fj[0], fj[1]])
        got = _np(ctl.ips[s])[fj[0], fj[1]]
        assert np.array_equal(got, want), (s, "ips", int((got != want).sum()))
    print(f"{cfg['name']}: sampled projection/rows ok {time.time() - t0:.1f}s", flush=True)
    for s in full:
        o = oracle.end_to_end(synth.subset(inp, [s]))
        got = _np(ctl.ips[s])
        exact = int((got == o["ips"][0]).sum())
        assert np.allclose(got, o["ips"][0], rtol=RTOL, atol=0) and exact == got.size, (s, exact)
        assert (idx[s], st[s]) == (o["freq_idx"][0], o["status"][0]), s
    print(f"{cfg['name']}: end-to-end scenarios ok {time.time() - t0:.1f}s", flush=True)

    # the selection stage on every scenario (c4: a block of 2048 scenarios):
    # the oracle's selection on the GPU's own projections and IPS
    blk = slice(0, S) if S * F * H <= 300_000_000 else slice(4096, 4096 + 2048)
    ips_all = _np(ctl.ips[blk])
    oi, os_ = oracle.select(ips_all, dl[blk], n_iters[blk], inp["tbt_slo_ns"][blk], flags[blk])
    assert np.array_equal(idx[blk], oi) and np.array_equal(st[blk], os_), \
        np.nonzero((idx[blk] != oi) | (st[blk] != os_))[0][:5]
    print(f"{cfg['name']}: selection on {ips_all.shape[0]} scenarios ok {time.time() - t0:.1f}s", flush=True)
    del ips_all

    # the forest stage on random (scenario, frequency, iteration) rows built
    # from the GPU's own curves (c3, 2000 trees of depth 10: 400 000 rows)
    n_rows = min(S * F * H, 400_000 if ci == 3 else 1_000_000)
    rs = rng.integers(0, S, n_rows)
    rf = rng.integers(0, F, n_rows)
    rj = rng.integers(0, H, n_rows)
    cols = [inp["freqs_mhz"][rf], kv[rs, rj].astype(np.float32), batch[rs, rj].astype(np.float32)]
    if inp["n_features"] == 4:
        cols.append(inp["engine_size"][rs])
    want = oracle.forest_predict(inp["forest"], np.stack(cols, axis=1).astype(np.float32))
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
    assert np.all(kv <= inp["kv_capacity"][:, None]) or np.any(flags & oracle.FLAG_OVERCOMMIT)
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
