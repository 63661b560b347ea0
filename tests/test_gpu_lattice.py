"""The model compiled to its input lattice (tl_lattice_create /
tl_lattice_predict_grid) gives the same values as the oracle and as the
fused grid kernel, on lattice points and off them (rows outside the bounds,
engine sizes not in the list).  Float outputs must be bit-identical."""
import numpy as np
import pytest

import oracle
from paper_2408_05235_amd import configs, synth
from test_gpu_parity import random_curves, random_forest

pytestmark = pytest.mark.gpu


def _t(a):
    import torch
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("F,T,d,nf,kv_max,b_max,seed", [
    (17, 30, 6, 3, 5000, 120, 0), (64, 25, 8, 4, 4095, 60, 1), (5, 12, 12, 4, 8191, 30, 2),
    (1, 8, 3, 3, 0, 0, 3), (48, 0, 4, 3, 100, 10, 4)])
def test_lattice_random(gpu, F, T, d, nf, kv_max, b_max, seed):
    import torch
    from paper_2408_05235_amd import api
    rng = np.random.default_rng(1100 + seed)
    fd = random_forest(rng, T, d, nf, kvmax=kv_max + 50, bmax=b_max + 5)
    S, H = 9, 300
    kv, bs = random_curves(rng, S, H, kvmax=int(max(kv_max, 1) * 1.1 + 20), bmax=b_max + 3)
    kv[0, :5] = [0, kv_max, kv_max + 1, 4095, 4096]      # edges and chunk boundary
    bs[1, :3] = [0, b_max, b_max + 1]
    freqs = synth.frequency_grid(F)
    engines = [1.0, 2.0, 4.0, 8.0]
    eng = None
    if nf == 4:
        eng = rng.choice([1.0, 2.0, 4.0, 8.0, 3.0], S).astype(np.float32)   # 3.0: not in the lattice
        eng[0] = 3.0
    f = api.Forest.from_dict(fd)
    lat = api.Lattice(f, _t(freqs), kv_max, b_max, engines if nf == 4 else None)
    got = lat.tl_lattice_predict_grid(_t(kv), _t(bs), _t(eng)).cpu().numpy()
    grid = f.tl_forest_predict_grid(_t(freqs), _t(kv), _t(bs), _t(eng)).cpu().numpy()
    torch.cuda.synchronize()
    want = oracle.forest_predict(fd, oracle.rows(freqs, bs, kv, eng, nf))
    assert np.array_equal(got, grid)
    assert np.array_equal(got, want)
    assert lat.nbytes == (4 if nf == 4 else 1) * (b_max + 1) * F * 4096 * (kv_max // 4096 + 1) * 4
    lat.close()


def test_lattice_scaled_c3(gpu):
    """c3's forest (300 of its trees) over the lattice the workload spans,
    in the controller: the same IPS and selection as the grid kernel."""
    import torch
    from paper_2408_05235_amd import api
    cfg = synth.scaled(configs.get_config(3), n_scenarios=24, forest_n_trees=300)
    inp = synth.make_inputs(cfg)
    ctl = api.Controller(api.upload(inp), api.Forest.from_dict(inp["forest"]))
    ctl.step()
    kvmax = int(ctl.buf["kv"].max().item())
    bmax = int(ctl.buf["batch"].max().item())
    lat = api.Lattice(ctl.forest, ctl.d["freqs_mhz"], kvmax - 7, bmax, [1.0, 2.0, 4.0, 8.0])
    got = lat.tl_lattice_predict_grid(ctl.buf["kv"], ctl.buf["batch"], ctl.d["engine_size"])
    torch.cuda.synchronize()
    assert torch.equal(got, ctl.ips)
    lat.close()


@pytest.mark.parametrize("ci,over", [(1, dict(n_scenarios=12)), (3, dict(n_scenarios=8, forest_n_trees=200))])
def test_lattice_in_admission_and_binary_search(gpu, ci, over):
    """Admission what-ifs and the binary search read M from a lattice with
    the same decisions, indices and IPS as with walks; a lattice of another
    forest is refused."""
    import torch
    from paper_2408_05235_amd import api, _lib
    cfg = synth.scaled(configs.get_config(ci), **over)
    inp = synth.make_inputs(cfg)
    d = api.upload(inp)
    ctl = api.Controller(d, api.Forest.from_dict(inp["forest"]))
    ctl.project()
    engines = [1.0, 2.0, 4.0, 8.0] if inp["n_features"] == 4 else None
    # bounds smaller than the workload: rows past them are walked, also exactly
    lat = api.Lattice(ctl.forest, d["freqs_mhz"], 20000, 140, engines)
    i0, s0 = [x.clone() for x in ctl.select_binary()]
    i1, s1 = ctl.select_binary(lat)
    torch.cuda.synchronize()
    assert torch.equal(i0, i1) and torch.equal(s0, s1)
    cand = synth.make_candidates(cfg, inp)
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a, dt).view(np.int64 if dt == np.uint64 else dt)).cuda()
    fmax = float(inp["freqs_mhz"][-1])
    args = (ctl.forest, fmax, d["tbt_slo_ns"], t(cand["cand_prompt"], np.int32), t(cand["cand_len"], np.int32),
            d["req_offset"], d["prompt"], d["generated"], d["remaining"], d["arrival"], d["kv_capacity"],
            d["horizon"], d["block_tokens"], d["deadline_ns"], d["lost"], d["batch_cap"], d["engine_size"],
            t(cand["cand_deadline_ns"], np.uint64))
    a0 = api.tl_admit(*args)
    a0 = {k: v.clone() for k, v in a0.items()}
    a1 = api.tl_admit(*args, lattice=lat)
    torch.cuda.synchronize()
    for k in ("decision", "ips", "kv", "batch", "flags"):
        assert torch.equal(a0[k], a1[k]), k
    other = api.Forest.from_dict(random_forest(np.random.default_rng(5), 4, 3, inp["n_features"]))
    # refused on the host before anything is enqueued: the outputs keep
    # what they held
    sentinel = {k: v.clone().fill_(-7) for k, v in a1.items()}
    out = {k: v.clone() for k, v in sentinel.items()}
    with pytest.raises(_lib.TLError):
        api.tl_admit(other, *args[1:], out=out, lattice=lat)
    torch.cuda.synchronize()
    for k in sentinel:
        assert torch.equal(out[k], sentinel[k]), k
    lat.close()
    other.close()
