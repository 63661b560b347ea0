"""tl_forest_predict_grid_noalloc (the grid prediction for callers that
cannot allocate) against tl_forest_predict_grid, through the C ABI: two
calls in a row, the second on a smaller grid, bit for bit; a grid beyond
its fixed scratch is refused before anything is enqueued."""
import numpy as np
import pytest

import oracle
from paper_2408_05235_amd import configs, synth

pytestmark = pytest.mark.gpu


def _grid_inputs(n_scenarios, trees):
    cfg = synth.scaled(configs.get_config(3), n_scenarios=n_scenarios, forest_n_trees=trees)
    inp = synth.make_inputs(cfg)
    proj = oracle.project(inp)
    return inp, proj


def test_noalloc_equals_allocating_entry_point(gpu):
    import torch
    from paper_2408_05235_amd import api, _lib
    inp, proj = _grid_inputs(256, 60)
    f = api.Forest.from_dict(inp["forest"])
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    freqs = t(inp["freqs_mhz"])
    eng = t(inp["engine_size"])
    sizes = [(256, 1024), (40, 600)]       # second call smaller: fewer scenarios, shorter horizon
    for S, H in sizes:
        kv = t(proj["kv"][:S, :H])
        bs = t(proj["batch"][:S, :H])
        print(f"noalloc grid S={S} F={freqs.numel()} H={H}", flush=True)
        ref = f.tl_forest_predict_grid(freqs, kv, bs, eng[:S])
        out = torch.full_like(ref, float("nan"))
        f.tl_forest_predict_grid(freqs, kv, bs, eng[:S], out=out, noalloc=True)
        torch.cuda.synchronize()
        a, b = ref.cpu().numpy(), out.cpu().numpy()
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), f"S={S} H={H}: outputs differ"
        # and the first scenario against the oracle
        x = oracle.rows(inp["freqs_mhz"], proj["batch"][:1, :H], proj["kv"][:1, :H], inp["engine_size"][:1], 4)
        exp = oracle.forest_predict(inp["forest"], x)
        assert np.array_equal(b[:1].view(np.uint32), exp.view(np.uint32))
    # a grid without a work order (too few chunks) takes no scratch
    kv = t(proj["kv"][:1, :64])
    bs = t(proj["batch"][:1, :64])
    ref = f.tl_forest_predict_grid(freqs, kv, bs, eng[:1])
    out = f.tl_forest_predict_grid(freqs, kv, bs, eng[:1], out=torch.empty_like(ref), noalloc=True)
    torch.cuda.synchronize()
    assert np.array_equal(ref.cpu().numpy(), out.cpu().numpy())
    f.close()
    assert _lib.lib().tl_abi_version() == 1


def test_noalloc_refuses_grids_beyond_its_scratch(gpu):
    import torch
    from paper_2408_05235_amd import api, _lib
    rng = np.random.default_rng(3)
    fd = synth.make_forest(rng, 4, 10, 3, "profile", 40.0, 65536, 128, synth.frequency_grid(8))
    f = api.Forest.from_dict(fd)
    S, H = 65536, 2048                      # 2^21 (scenario, chunk) pairs: 32 MiB for the arrays alone
    kv = torch.zeros((S, H), dtype=torch.int32, device="cuda")
    bs = torch.zeros((S, H), dtype=torch.int32, device="cuda")
    freqs = torch.tensor([1500.0], dtype=torch.float32, device="cuda")
    out = torch.full((S, 1, H), -1.0, dtype=torch.float32, device="cuda")
    with pytest.raises(_lib.TLError) as ei:
        f.tl_forest_predict_grid(freqs, kv, bs, None, out=out, noalloc=True)
    assert ei.value.status == _lib.TL_EUNSUPPORTED and "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((out == -1.0).all())        # nothing was enqueued
    f.close()
