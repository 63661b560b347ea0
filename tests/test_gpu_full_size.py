"""Parity at the five workloads' full sizes, in the configuration bench.py
times (fused grid prediction), on outputs the oracle can afford: a few whole
scenarios end to end, sampled rows, and properties over every scenario."""
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
