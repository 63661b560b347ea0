"""Parity of tl_adjust_lengths (generation-length errors, Sec. 4.6) with the
oracle, alone and feeding the projection and the controller.  Integer
outputs must match bit for bit."""
import numpy as np
import pytest

import oracle
from paper_2408_05235_amd import configs, synth

pytestmark = pytest.mark.gpu


def _t(a, dt):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dt).view(np.int32 if dt == np.uint32 else dt)).cuda()


def gpu_adjust(off, gen, pred, num, den, mt):
    import torch
    from paper_2408_05235_amd import api
    out = api.tl_adjust_lengths(_t(off, np.int64), _t(gen, np.int32), _t(pred, np.int32), _t(num, np.uint32),
                                _t(den, np.uint32), _t(mt, np.int32))
    torch.cuda.synchronize()
    return out.cpu().numpy()


def random_lengths(rng, S, rmax):
    counts = rng.integers(0, rmax + 1, S)
    off = np.zeros(S + 1, np.int64)
    np.cumsum(counts, out=off[1:])
    R = int(off[-1])
    gen = rng.integers(0, 3000, R).astype(np.int32)
    pred = rng.integers(1, 3000, R).astype(np.int32)
    pred[rng.random(R) < 0.01] = 0
    gen[rng.random(R) < 0.01] = -4
    big = rng.random(R) < 0.01
    pred[big] = rng.integers(2 ** 30, 2 ** 31 - 1, int(big.sum()))
    num = rng.integers(1, 40, S).astype(np.uint32)
    den = rng.integers(1, 30, S).astype(np.uint32)
    den[rng.random(S) < 0.1] = 0
    num[rng.random(S) < 0.05] = 4_000_000_000           # huge factors: clamped at 2^31 - 1
    mt = rng.integers(1, 4096, S).astype(np.int32)
    mt[rng.random(S) < 0.1] = 0
    mt[rng.random(S) < 0.05] = -7
    return off, gen, pred, num, den, mt


@pytest.mark.parametrize("S,rmax,seed", [(1, 0, 0), (1, 1, 1), (50, 300, 2), (257, 70, 3), (4, 5000, 4)])
def test_adjust_lengths_random(gpu, S, rmax, seed):
    rng = np.random.default_rng(900 + seed)
    args = random_lengths(rng, S, rmax)
    got = gpu_adjust(*args)
    want = oracle.adjust_lengths(*args)
    assert np.array_equal(got, want), np.nonzero(got != want)[0][:5]


def test_adjust_lengths_full_size(gpu):
    """The c4 workload's 143 M entries (predicted total = generated +
    remaining), factor 11/10 and a 4096-token limit; sampled scenarios against
    the oracle, properties over all."""
    cfg = configs.get_config(4)
    inp = synth.make_inputs(cfg)
    S = inp["n_scenarios"]
    pred = (inp["generated"].astype(np.int64) + inp["remaining"]).astype(np.int32)
    num, den, mt = np.full(S, 11, np.uint32), np.full(S, 10, np.uint32), np.full(S, 4096, np.int32)
    got = gpu_adjust(inp["req_offset"], inp["generated"], pred, num, den, mt)
    assert np.all(got >= 1) and np.all(got <= 4096)
    assert np.all(got >= np.minimum(inp["remaining"], 4096 - inp["generated"]))
    off = inp["req_offset"]
    for s in (0, 7777, S - 1):
        lo, hi = int(off[s]), int(off[s + 1])
        want = oracle.adjust_lengths([0, hi - lo], inp["generated"][lo:hi], pred[lo:hi], num[:1], den[:1], mt[:1])
        assert np.array_equal(got[lo:hi], want), s


@pytest.mark.parametrize("ci,over", [(1, dict(n_scenarios=8)), (2, dict(n_scenarios=4)), (4, dict(n_scenarios=3))])
def test_adjusted_lengths_through_the_controller(gpu, ci, over):
    """Adjusted scoreboards (factor 5/4, limit 2048) projected and controlled
    on the GPU equal the oracle's adjust -> project -> predict -> select."""
    import torch
    from paper_2408_05235_amd import api
    cfg = synth.scaled(configs.get_config(ci), **over)
    inp = synth.make_inputs(cfg)
    S = inp["n_scenarios"]
    pred = (inp["generated"].astype(np.int64) + inp["remaining"]).astype(np.int32)
    num, den, mt = np.full(S, 5, np.uint32), np.full(S, 4, np.uint32), np.full(S, 2048, np.int32)
    d = api.upload(inp)
    rem = api.tl_adjust_lengths(d["req_offset"], d["generated"], _t(pred, np.int32), _t(num, np.uint32),
                                _t(den, np.uint32), _t(mt, np.int32))
    d["remaining"] = rem
    ctl = api.Controller(d, api.Forest.from_dict(inp["forest"]))
    idx, st = ctl.step()
    torch.cuda.synchronize()
    adj = dict(inp, remaining=oracle.adjust_lengths(inp["req_offset"], inp["generated"], pred, num, den, mt))
    assert np.array_equal(rem.cpu().numpy(), adj["remaining"])
    o = oracle.end_to_end(adj)
    assert np.array_equal(ctl.buf["kv"].cpu().numpy(), o["kv"])
    assert np.array_equal(ctl.buf["batch"].cpu().numpy(), o["batch"])
    assert np.array_equal(idx.cpu().numpy(), o["freq_idx"])
    assert np.array_equal(st.cpu().numpy().view(np.uint32), o["status"])
