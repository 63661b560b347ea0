"""Seeded synthetic inputs for the frequency-controller hot path.

This module only draws inputs: scoreboards, capacities, SLOs, candidate
frequencies and a synthetic tree ensemble.  It holds none of the method's
arithmetic (no projection, no tree evaluation, no selection), so both the HIP
path and the CPU oracle can consume its output.

The scoreboard of a scenario (Sec. 4.2, Table 1) is stored CSR-style:
``req_offset[s]:req_offset[s+1]`` are the requests of scenario ``s``, each
with a prompt length |q_i|, the tokens it has generated so far, its projected
remaining tokens, the iteration at which it joins the queue (``-1`` = already
in the batch), its E2E deadline relative to now (t_dead - t_cur of Eq. 4, in
ns) and a "lost" mark (Sec. 4.3.2, last paragraph).

The paper measures on a production LLM trace that is not available here; the
distributions below only mimic its ranges (Sec. 3.4): prompts mostly below a
few thousand tokens, generation lengths of tens to hundreds of tokens with a
long tail, per-token latencies of tens of ms.
"""
from __future__ import annotations

import numpy as np

UINT64_MAX = np.uint64(0xFFFFFFFFFFFFFFFF)

# Column order of a feature row (Sec. 4.3.1 lists engine size, batch size,
# KV usage and GPU frequency as the model's inputs).
FEAT_FREQ, FEAT_KV, FEAT_BATCH, FEAT_ENGINE = 0, 1, 2, 3


def _rng(seed_seq):
    return np.random.Generator(np.random.PCG64(seed_seq))


def _draw(rng, spec, size):
    """Draw integers from ``("uniform", lo, hi)`` (inclusive) or
    ``("lognormal", mu, sigma, lo, hi)`` (rounded to nearest, clipped)."""
    kind = spec[0]
    if kind == "uniform":
        return rng.integers(spec[1], spec[2], size=size, endpoint=True, dtype=np.int64).astype(np.int32)
    if kind == "lognormal":
        x = np.rint(rng.lognormal(spec[1], spec[2], size=size))
        return np.clip(x, spec[3], spec[4]).astype(np.int32)
    raise ValueError(spec)


def frequency_grid(n_freqs, lo_mhz=1000, hi_mhz=2000):
    """Candidate frequencies, ascending integer MHz spanning [lo, hi]."""
    if n_freqs == 1:
        return np.array([hi_mhz], dtype=np.float32)
    k = np.arange(n_freqs, dtype=np.int64)
    return (lo_mhz + (k * (hi_mhz - lo_mhz)) // (n_freqs - 1)).astype(np.float32)


def make_forest(rng, n_trees, depth, n_features, leaves, base_score, kv_max,
                batch_max, freqs, leaf_sigma=0.1, snap_prob=0.1):
    """A seeded complete-tree ensemble in heap order.

    Internal node k has children 2k+1 (taken when x[feature] < threshold) and
    2k+2; there are 2**depth - 1 internal nodes and 2**depth leaves per tree.
    Each node splits a uniformly chosen feature at a uniform point inside the
    node's current box; a fraction of thresholds is snapped onto values the
    inputs actually take (integers, grid frequencies) so that x == threshold
    ties occur.  ``leaves="profile"`` gives leaf values that make the ensemble
    approximate a smooth IPS surface (slower at low frequency, high batch and
    high KV use); ``"normal"`` draws N(0, leaf_sigma).
    """
    n_int = (1 << depth) - 1
    lo_all = np.array([1000.0, 0.0, 0.0, 1.0][:n_features])
    hi_all = np.array([2000.0, float(kv_max), float(batch_max), 8.0][:n_features])
    feature = np.zeros((n_trees, n_int), dtype=np.uint8)
    threshold = np.zeros((n_trees, n_int), dtype=np.float32)
    lo = np.broadcast_to(lo_all, (n_trees, 1, n_features)).copy()
    hi = np.broadcast_to(hi_all, (n_trees, 1, n_features)).copy()
    freqs64 = np.asarray(freqs, dtype=np.float64)
    for level in range(depth):
        width = 1 << level
        first = width - 1
        feat = rng.integers(0, n_features, size=(n_trees, width))
        flo = np.take_along_axis(lo, feat[..., None], axis=2)[..., 0]
        fhi = np.take_along_axis(hi, feat[..., None], axis=2)[..., 0]
        thr = flo + (fhi - flo) * rng.random((n_trees, width))
        snap = rng.random((n_trees, width)) < snap_prob
        is_freq = feat == FEAT_FREQ
        nearest = freqs64[np.abs(thr[..., None] - freqs64).argmin(axis=-1)]
        thr = np.where(snap & is_freq, nearest, thr)
        thr = np.where(snap & ~is_freq, np.rint(thr), thr)
        thr32 = thr.astype(np.float32)
        feature[:, first:first + width] = feat
        threshold[:, first:first + width] = thr32
        # child boxes: left child keeps values < thr, right child >= thr
        lo_c = np.repeat(lo, 2, axis=1)
        hi_c = np.repeat(hi, 2, axis=1)
        t64 = thr32.astype(np.float64)
        idx = np.arange(width)
        for side in (0, 1):
            sel = 2 * idx + side
            box = hi_c if side == 0 else lo_c
            cur = box[:, sel, :]
            np.put_along_axis(cur, feat[..., None], t64[..., None], axis=2)
            box[:, sel, :] = cur
        lo, hi = lo_c, hi_c
    n_leaf = 1 << depth
    if leaves == "normal":
        leaf = rng.normal(0.0, leaf_sigma, size=(n_trees, n_leaf)).astype(np.float32)
    elif leaves == "profile":
        centre = 0.5 * (lo + hi)
        f = centre[..., FEAT_FREQ]
        kv = centre[..., FEAT_KV]
        bs = centre[..., FEAT_BATCH]
        tbt_ms = 12.0 * (2000.0 / f) ** 0.8 * (1.0 + 0.5 * bs / batch_max + 0.5 * kv / kv_max)
        target = 1000.0 / tbt_ms
        leaf = ((target - base_score) / n_trees
                + rng.normal(0.0, 0.01, size=(n_trees, n_leaf))).astype(np.float32)
    else:
        raise ValueError(leaves)
    return dict(n_trees=n_trees, depth=depth, n_features=n_features,
                base_score=np.float32(base_score),
                feature=feature, threshold=threshold, leaf=leaf)


def make_inputs(cfg, seed=None):
    """Draw every input of one workload.  Deterministic in (cfg, seed)."""
    seed = cfg["seed"] if seed is None else seed
    ss = np.random.SeedSequence(seed)
    s_req, s_arr, s_slo, s_forest, s_lost, s_eng = ss.spawn(6)
    r_req, r_arr, r_slo, r_forest, r_lost, r_eng = map(
        _rng, (s_req, s_arr, s_slo, s_forest, s_lost, s_eng))

    S = int(cfg["n_scenarios"])
    H = int(cfg["horizon"])
    R_in = int(cfg["n_inflight"])
    Q = int(cfg.get("queued", 0))

    # in-flight requests [S, R_in]
    p_in = _draw(r_req, cfg["prompt"], (S, R_in))
    g_in = _draw(r_req, cfg["generated"], (S, R_in))
    r_in = _draw(r_req, cfg["remaining"], (S, R_in))
    # requests already queued at iteration 0 [S, Q]
    if Q:
        p_q = _draw(r_req, cfg["prompt"], (S, Q))
        r_q = _draw(r_req, cfg["remaining"], (S, Q))
    # Poisson arrivals at iterations 0..H-1
    arr = cfg.get("arrivals")
    if arr:
        rate = r_arr.uniform(arr["rate"][0], arr["rate"][1], size=S)
        counts = r_arr.poisson(rate[:, None], size=(S, H)).astype(np.int64)
        n_arr = counts.sum(axis=1)
    else:
        n_arr = np.zeros(S, dtype=np.int64)

    per = R_in + Q + n_arr
    req_offset = np.zeros(S + 1, dtype=np.int64)
    np.cumsum(per, out=req_offset[1:])
    total = int(req_offset[-1])
    prompt = np.empty(total, dtype=np.int32)
    generated = np.zeros(total, dtype=np.int32)
    remaining = np.empty(total, dtype=np.int32)
    arrival = np.empty(total, dtype=np.int32)

    base = req_offset[:-1]
    idx_in = (base[:, None] + np.arange(R_in)[None, :]).ravel()
    prompt[idx_in] = p_in.ravel()
    generated[idx_in] = g_in.ravel()
    remaining[idx_in] = r_in.ravel()
    arrival[idx_in] = -1
    if Q:
        idx_q = (base[:, None] + R_in + np.arange(Q)[None, :]).ravel()
        prompt[idx_q] = p_q.ravel()
        remaining[idx_q] = r_q.ravel()
        arrival[idx_q] = 0
    if arr:
        n_tot = int(n_arr.sum())
        start = np.repeat(base + R_in + Q, n_arr)
        first = np.repeat(np.cumsum(n_arr) - n_arr, n_arr)
        idx_a = start + (np.arange(n_tot) - first)
        iters = np.tile(np.arange(H, dtype=np.int32), S)
        arrival[idx_a] = np.repeat(iters, counts.ravel())
        prompt[idx_a] = _draw(r_arr, arr["prompt"], n_tot)
        remaining[idx_a] = _draw(r_arr, arr["length"], n_tot)

    # per-token SLO sigma_s in ns (Sec. 5.1 states SLOs per engine)
    kind = cfg["slo_ms"][0]
    if kind == "fixed":
        slo = np.full(S, int(round(cfg["slo_ms"][1] * 1e6)), dtype=np.uint64)
    else:
        lo_us, hi_us = int(cfg["slo_ms"][1] * 1000), int(cfg["slo_ms"][2] * 1000)
        slo = (r_slo.integers(lo_us, hi_us, size=S, endpoint=True).astype(np.uint64)
               * np.uint64(1000))

    # E2E deadlines relative to now: in-flight requests must finish their
    # remaining tokens at sigma_s per token; queued and arriving requests carry
    # no deadline yet.
    deadline = np.full(total, UINT64_MAX, dtype=np.uint64)
    deadline[idx_in] = (np.repeat(slo, R_in) * r_in.ravel().astype(np.uint64))

    # a small fraction of scenarios holds one "lost" in-flight request
    lost = np.zeros(total, dtype=np.uint8)
    p_lost = float(cfg.get("lost_scenario_prob", 0.0))
    if p_lost > 0 and R_in > 0:
        which = np.nonzero(r_lost.random(S) < p_lost)[0]
        pick = r_lost.integers(0, R_in, size=which.size)
        lost[base[which] + pick] = 1

    fc = cfg["forest"]
    n_feat = int(fc["n_features"])
    engine = None
    if n_feat == 4:
        engine = r_eng.choice(np.array([1.0, 2.0, 4.0, 8.0], dtype=np.float32), size=S)
    freqs = frequency_grid(int(cfg["n_freqs"]))
    forest = make_forest(r_forest, int(fc["n_trees"]), int(fc["depth"]), n_feat,
                         fc["leaves"], float(fc["base_score"]), int(cfg["kv_capacity"]),
                         int(fc["batch_max"]), freqs, leaf_sigma=float(fc.get("leaf_sigma", 0.1)))

    batch_cap = None
    if cfg.get("batch_cap") is not None:
        batch_cap = np.full(S, int(cfg["batch_cap"]), dtype=np.int32)

    return dict(
        n_scenarios=S, horizon=H, block_tokens=int(cfg["block_tokens"]),
        n_freqs=int(cfg["n_freqs"]), n_features=n_feat,
        req_offset=req_offset, prompt=prompt, generated=generated,
        remaining=remaining, arrival=arrival, deadline_ns=deadline, lost=lost,
        kv_capacity=np.full(S, int(cfg["kv_capacity"]), dtype=np.int32),
        batch_cap=batch_cap, tbt_slo_ns=slo, freqs_mhz=freqs,
        engine_size=engine, forest=forest,
    )


def make_candidates(cfg, inp, seed=None):
    """One new query per scenario for admission control (Sec. 4.3.2): its
    prompt and predicted length drawn like the workload's requests (arrival
    distributions where the workload has arrivals), and an E2E deadline of
    sigma_s per predicted token, the rule of the in-flight deadlines.
    Deterministic in (cfg, seed)."""
    seed = (cfg["seed"] if seed is None else seed) + 7919
    rng = _rng(np.random.SeedSequence(seed))
    S = int(inp["n_scenarios"])
    arr = cfg.get("arrivals")
    prompt = _draw(rng, arr["prompt"] if arr else cfg["prompt"], S)
    length = _draw(rng, arr["length"] if arr else cfg["remaining"], S)
    deadline = np.asarray(inp["tbt_slo_ns"], np.uint64) * length.astype(np.uint64)
    return dict(cand_prompt=prompt, cand_len=length, cand_deadline_ns=deadline)


def scaled(cfg, **overrides):
    """A copy of a workload with some sizes replaced (same distributions)."""
    out = dict(cfg)
    forest = dict(out["forest"])
    for k, v in overrides.items():
        if k.startswith("forest_"):
            forest[k[len("forest_"):]] = v
        else:
            out[k] = v
    out["forest"] = forest
    return out


def subset(inp, scenarios):
    """The inputs restricted to a list of scenarios (CSR re-based)."""
    scenarios = np.asarray(scenarios, dtype=np.int64)
    off = inp["req_offset"]
    counts = off[scenarios + 1] - off[scenarios]
    new_off = np.zeros(scenarios.size + 1, dtype=np.int64)
    np.cumsum(counts, out=new_off[1:])
    idx = np.concatenate([np.arange(off[s], off[s + 1]) for s in scenarios]) if scenarios.size else np.zeros(0, np.int64)
    out = dict(inp)
    out["n_scenarios"] = int(scenarios.size)
    out["req_offset"] = new_off
    for k in ("prompt", "generated", "remaining", "arrival", "deadline_ns", "lost"):
        out[k] = inp[k][idx]
    for k in ("kv_capacity", "batch_cap", "tbt_slo_ns", "engine_size"):
        if inp.get(k) is not None:
            out[k] = inp[k][scenarios]
    return out
