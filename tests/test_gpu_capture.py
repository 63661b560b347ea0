"""The projection and the grid prediction captured into a graph.

While a stream is being captured, tl_project and tl_forest_predict_grid
leave their optional library-owned workspaces out (the projection's scenario
order, the grid's work order): growing them would allocate and handing them
between streams would wait on events recorded outside the capture.  The
captured calls must give the eager results, replay after replay, with eager
calls (which do use the workspaces) and synchronizations in between.
"""
import numpy as np
import pytest

import oracle
from paper_2408_05235_amd import synth
from test_gpu_parity import assert_projection_equal, random_boards, random_curves, random_forest

pytestmark = pytest.mark.gpu


def _project(api, d, S):
    return api.tl_project(d["req_offset"], d["prompt"], d["generated"], d["remaining"], d["arrival"],
                          d["kv_capacity"], d["horizon"], d["block_tokens"], d["deadline_ns"], d["lost"],
                          d["batch_cap"], None, None, 3, False)


def _host(res):
    return dict(batch=res["batch"].cpu().numpy(), kv=res["kv"].cpu().numpy(),
                deadline_at=res["deadline_at"].cpu().numpy().view(np.uint64),
                n_iters=res["n_iters"].cpu().numpy(), flags=res["flags"].cpu().numpy().view(np.uint32))


def test_captured_projection_and_grid_replays(gpu):
    import torch
    from paper_2408_05235_amd import api
    rng = np.random.default_rng(45)
    # long FIFO loops without a batch cap: the ordered projection when eager
    S = 40
    inp = random_boards(rng, S, 512, 16, rmax=3000, qfrac=0.6)
    inp["batch_cap"] = None
    assert int(inp["req_offset"][-1]) >= 1024 * S
    d = api.upload(dict(inp, tbt_slo_ns=np.zeros(S, np.uint64), freqs_mhz=np.zeros(1, np.float32),
                        engine_size=None, n_features=3))
    exp_proj = oracle.project(inp)
    eager = _host(_project(api, d, S))
    torch.cuda.synchronize()
    assert_projection_equal(eager, exp_proj, "eager")

    fd = random_forest(rng, 30, 8, 3)
    forest = api.Forest.from_dict(fd)
    kv, bs = random_curves(rng, 6, 300)
    freqs = synth.frequency_grid(64)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    dkv, dbs, dfr = t(kv), t(bs), t(freqs)
    exp_grid = oracle.forest_predict(fd, oracle.rows(freqs, bs, kv, None, 3))
    eager_grid = forest.tl_forest_predict_grid(dfr, dkv, dbs).cpu().numpy()
    assert np.array_equal(eager_grid, exp_grid)

    # warm up on a side stream, then capture both calls
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _project(api, d, S)
        forest.tl_forest_predict_grid(dfr, dkv, dbs)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    grid_out = torch.full((6, 64, 300), -1.0, dtype=torch.float32, device="cuda")
    with torch.cuda.graph(graph):
        cap = _project(api, d, S)
        forest.tl_forest_predict_grid(dfr, dkv, dbs, out=grid_out)
    for rep in range(3):
        graph.replay()
        torch.cuda.synchronize()
        assert_projection_equal(_host(cap), exp_proj, f"replay {rep}")
        assert np.array_equal(grid_out.cpu().numpy(), exp_grid), f"replay {rep}"
        # eager calls between the replays, through the workspaces
        assert_projection_equal(_host(_project(api, d, S)), exp_proj, f"eager after replay {rep}")
        assert np.array_equal(forest.tl_forest_predict_grid(dfr, dkv, dbs).cpu().numpy(), exp_grid)
        torch.cuda.synchronize()
    forest.close()


def test_captured_binary_search_replays(gpu):
    """The binary search at a size where eager calls order the column
    kernel's work by estimated cost (8192 x 1024 iterations on 256 CUs: two
    workgroups per CU), captured into a graph, where the order is left out:
    every replay gives the eager call's indices, statuses and final-probe
    model values, with eager calls (through the forest's scratch) between
    the replays; sampled scenarios equal the oracle's search."""
    import torch
    from paper_2408_05235_amd import api
    from test_gpu_search import random_checks
    rng = np.random.default_rng(46)
    S, H, F, nf = 8192, 1024, 5, 4
    fd = random_forest(rng, 20, 6, nf, kvmax=3000, bmax=200)
    fd["base_score"] = np.float32(45.0)
    kv, bs = random_curves(rng, S, H, kvmax=3000, bmax=200)
    # odd scenarios: a batch that changes at every iteration (costly columns)
    fast = np.arange(S) % 2 == 1
    nfast = int(fast.sum())
    bs[fast] = np.clip(rng.integers(20, 180, (nfast, 1)) + np.cumsum(rng.choice([-1, 1], (nfast, H)), axis=1),
                       0, None).astype(np.int32)
    freqs = synth.frequency_grid(F)
    eng = rng.choice([1.0, 2.0, 4.0, 8.0], S).astype(np.float32)
    dl, n, tbt, flags = random_checks(rng, S, H, kv)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    args = (t(freqs), t(kv), t(bs), t(dl.view(np.int64)), t(n), t(tbt.view(np.int64)), t(flags.view(np.int32)))
    deng = t(eng)
    forest = api.Forest.from_dict(fd)

    def bufs():
        return dict(ips_work=torch.full((S, H), -1.0, dtype=torch.float32, device="cuda"),
                    search_work=torch.zeros((3, S), dtype=torch.int32, device="cuda"),
                    freq_idx=torch.full((S,), -1, dtype=torch.int32, device="cuda"),
                    status=torch.full((S,), -1, dtype=torch.int32, device="cuda"))

    def call(out):
        return api.tl_select_freq_binary(forest, *args, engine_size=deng, out=out)

    def host(out):
        return {k: out[k].cpu().numpy() for k in ("ips_work", "freq_idx", "status")}

    ref = bufs()
    call(ref)
    torch.cuda.synchronize()
    eager = host(ref)
    sample = np.array([0, 1, S // 2 + 1, S - 1])
    ips = oracle.forest_predict(fd, oracle.rows(freqs, bs[sample], kv[sample], eng[sample], nf))
    oi, os_ = oracle.select_binary(ips, dl[sample], n[sample], tbt[sample], flags[sample])
    assert np.array_equal(eager["freq_idx"][sample], oi)
    assert np.array_equal(eager["status"][sample].view(np.uint32), os_)

    cap = bufs()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(cap)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(cap)
    for rep in range(3):
        for v in cap.values():
            v.fill_(-1)
        graph.replay()
        torch.cuda.synchronize()
        got = host(cap)
        for k in eager:
            assert np.array_equal(got[k], eager[k]), (k, rep)
        again = bufs()
        call(again)
        torch.cuda.synchronize()
        got = host(again)
        for k in eager:
            assert np.array_equal(got[k], eager[k]), (k, "eager after replay", rep)
    forest.close()
