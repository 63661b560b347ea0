"""CPU oracle for the frequency-controller hot path (test infrastructure).

Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It wraps ``tl_oracle.c`` (plain,
single-threaded C compiled with gcc) through ctypes and numpy; it shares no
code with the HIP library and never imports it.

Functions follow the paper: ``project`` (Sec. 4.2, Eq. 1-2, admission check 1
of Sec. 4.3.2), ``rows`` and ``forest_predict`` (Sec. 4.3.1), ``select`` and
``select_binary`` (Sec. 4.3.2 checks 2-3, Eq. 3-4, Sec. 4.5), ``latency_ns``
(T' = 1/T in ns), ``end_to_end`` (all three stages), ``admit`` (the
admission control of Sec. 4.3.2 for one new query per scenario) and
``adjust_lengths`` (the generation-length error handling of Sec. 4.6).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tl_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libtl_oracle.so")

FLAG_BAD_REQUEST, FLAG_LOST, FLAG_OVERCOMMIT, FLAG_OVERFLOW, FLAG_UNSORTED = 1, 2, 4, 8, 16
STATUS_OK, STATUS_INFEASIBLE, STATUS_LOST, STATUS_INVALID = 0, 1, 2, 3
ADMIT_OK, ADMIT_LOST, QUEUE_CAPACITY, QUEUE_TBT, QUEUE_E2E, ADMIT_INVALID = 0, 1, 2, 3, 4, 5
NO_DEADLINE = np.uint64(0xFFFFFFFFFFFFFFFF)
LAT_SATURATED = 1 << 40


def build():
    """Compile the oracle with gcc: -O2, no fast-math, no FMA contraction."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
           "-fno-fast-math", "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i64, i32, f32 = ctypes.c_int64, ctypes.c_int32, ctypes.c_float
    lib.tlo_project.argtypes = [i64, i32, i32] + [P] * 15
    lib.tlo_project.restype = ctypes.c_int
    lib.tlo_rows.argtypes = [i64, i32, i32, i32, P, P, P, P, P]
    lib.tlo_rows.restype = ctypes.c_int
    lib.tlo_forest_predict.argtypes = [i32, i32, i32, f32, P, P, P, P, i64, P]
    lib.tlo_forest_predict.restype = ctypes.c_int
    lib.tlo_latency_ns.argtypes = [f32]
    lib.tlo_latency_ns.restype = ctypes.c_uint64
    for name in ("tlo_select", "tlo_select_binary"):
        fn = getattr(lib, name)
        fn.argtypes = [i64, i32, i32] + [P] * 7
        fn.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def project(inp, return_admit=False):
    """Stage 1 on every scenario of ``inp`` (a dict from ``synth.make_inputs``)."""
    lib = _load()
    S, H, N = int(inp["n_scenarios"]), int(inp["horizon"]), int(inp["block_tokens"])
    off = _c(inp["req_offset"], np.int64)
    args = [_c(inp[k], t) for k, t in (("prompt", np.int32), ("generated", np.int32),
                                        ("remaining", np.int32), ("arrival", np.int32))]
    deadline = _c(inp.get("deadline_ns"), np.uint64)
    lost = _c(inp.get("lost"), np.uint8)
    cap = _c(inp["kv_capacity"], np.int32)
    bcap = _c(inp.get("batch_cap"), np.int32)
    batch = np.zeros((S, H), np.int32)
    kv = np.zeros((S, H), np.int32)
    dl = np.zeros((S, H), np.uint64)
    n_iters = np.zeros(S, np.int32)
    flags = np.zeros(S, np.uint32)
    admit = np.zeros(int(off[-1]) if S else 0, np.int32) if return_admit else None
    rc = lib.tlo_project(S, H, N, _ptr(off), *[_ptr(a) for a in args], _ptr(deadline), _ptr(lost),
                         _ptr(cap), _ptr(bcap), _ptr(batch), _ptr(kv), _ptr(dl), _ptr(n_iters),
                         _ptr(flags), _ptr(admit))
    if rc:
        raise ValueError("tlo_project rejected its arguments")
    out = dict(batch=batch, kv=kv, deadline_at=dl, n_iters=n_iters, flags=flags)
    if return_admit:
        out["admit_iter"] = admit
    return out


def rows(freqs, batch, kv, engine=None, n_features=3):
    """Feature rows [S][F][H][n_features] from projected curves."""
    lib = _load()
    batch = _c(batch, np.int32)
    kv = _c(kv, np.int32)
    S, H = batch.shape
    freqs = _c(freqs, np.float32)
    F = freqs.size
    engine = _c(engine, np.float32)
    out = np.zeros((S, F, H, n_features), np.float32)
    rc = lib.tlo_rows(S, F, H, n_features, _ptr(freqs), _ptr(batch), _ptr(kv), _ptr(engine), _ptr(out))
    if rc:
        raise ValueError("tlo_rows rejected its arguments")
    return out


def forest_predict(forest, x):
    """Ensemble output for every row of ``x`` ([..., n_features] fp32):
    base_score plus every tree's leaf, an fp32 running sum in tree order."""
    lib = _load()
    nf = int(forest["n_features"])
    x = _c(x, np.float32)
    shape = x.shape[:-1]
    assert x.shape[-1] == nf
    n_rows = int(np.prod(shape)) if shape else 1
    out = np.zeros(n_rows, np.float32)
    feat = _c(forest["feature"], np.uint8)
    thr = _c(forest["threshold"], np.float32)
    leaf = _c(forest["leaf"], np.float32)
    rc = lib.tlo_forest_predict(int(forest["n_trees"]), int(forest["depth"]), nf,
                                float(forest["base_score"]), _ptr(feat), _ptr(thr), _ptr(leaf),
                                _ptr(x), n_rows, _ptr(out))
    if rc:
        raise ValueError("tlo_forest_predict rejected its arguments")
    return out.reshape(shape)


def latency_ns(ips):
    lib = _load()
    return int(lib.tlo_latency_ns(float(np.float32(ips))))


def _select(fn_name, ips, deadline_at, n_iters, tbt_slo_ns, proj_flags):
    lib = _load()
    ips = _c(ips, np.float32)
    S, F, H = ips.shape
    dl = _c(deadline_at, np.uint64)
    n_iters = _c(n_iters, np.int32)
    tbt = _c(tbt_slo_ns, np.uint64)
    fl = _c(proj_flags, np.uint32)
    idx = np.zeros(S, np.int32)
    st = np.zeros(S, np.uint32)
    rc = getattr(lib, fn_name)(S, F, H, _ptr(ips), _ptr(dl), _ptr(n_iters), _ptr(tbt), _ptr(fl),
                               _ptr(idx), _ptr(st))
    if rc:
        raise ValueError(fn_name + " rejected its arguments")
    return idx, st


def select(ips, deadline_at, n_iters, tbt_slo_ns, proj_flags=None):
    """Lowest SLO-feasible frequency index per scenario (exhaustive)."""
    return _select("tlo_select", ips, deadline_at, n_iters, tbt_slo_ns, proj_flags)


def select_binary(ips, deadline_at, n_iters, tbt_slo_ns, proj_flags=None):
    """The paper's binary search over frequencies."""
    return _select("tlo_select_binary", ips, deadline_at, n_iters, tbt_slo_ns, proj_flags)


def end_to_end(inp):
    """All three stages; returns the projection, the IPS tensor and the choice."""
    proj = project(inp)
    x = rows(inp["freqs_mhz"], proj["batch"], proj["kv"], inp.get("engine_size"),
             int(inp["n_features"]))
    ips = forest_predict(inp["forest"], x)
    idx, st = select(ips, proj["deadline_at"], proj["n_iters"], inp["tbt_slo_ns"], proj["flags"])
    return dict(proj, ips=ips, freq_idx=idx, status=st)


def _append_candidate(inp, s, p, L):
    """Scenario s of ``inp`` with the new query appended as a request that
    starts now: prompt p, nothing generated, L iterations, no deadline (its
    own deadline is checked apart), not lost."""
    lo, hi = int(inp["req_offset"][s]), int(inp["req_offset"][s + 1])
    out = dict(n_scenarios=1, horizon=inp["horizon"], block_tokens=inp["block_tokens"],
               req_offset=np.array([0, hi - lo + 1], np.int64))
    for k, v, t in (("prompt", p, np.int32), ("generated", 0, np.int32), ("remaining", L, np.int32),
                    ("arrival", -1, np.int32)):
        out[k] = np.append(np.asarray(inp[k][lo:hi], t), t(v))
    if inp.get("deadline_ns") is not None:
        out["deadline_ns"] = np.append(np.asarray(inp["deadline_ns"][lo:hi], np.uint64), NO_DEADLINE)
    if inp.get("lost") is not None:
        out["lost"] = np.append(np.asarray(inp["lost"][lo:hi], np.uint8), np.uint8(0))
    out["kv_capacity"] = np.asarray(inp["kv_capacity"][s:s + 1], np.int32)
    if inp.get("batch_cap") is not None:
        out["batch_cap"] = np.asarray(inp["batch_cap"][s:s + 1], np.int32)
    return out


def admit(inp, cand_prompt, cand_len, cand_deadline_ns, max_freq_mhz, forest=None):
    """Admission control for one new query per scenario (Sec. 4.3.2).

    The query joins the scenario's virtual scoreboard as a request that starts
    now (prompt ``cand_prompt[s]``, nothing generated, active for the
    ``cand_len[s]`` iterations [0, L)).  On the projection with it (Eq. 1-2):
      1. KV: some projected KV value exceeds the capacity, or the batch that
         runs now exceeds the batch cap -> QUEUE_CAPACITY;
      2. TBT: with M queried at the maximum frequency, T' = 1/T per iteration
         (``latency_ns``) and T_R[l] = T'[0] + ... + T'[l-1] (Eq. 3), the mean
         T' over the n projected iterations exceeds the SLO, T_R[n] > sigma*n
         -> QUEUE_TBT;
      3. E2E (Eq. 4): a scheduled request that is not lost and ends inside the
         horizon at e misses T_R[e] < deadline -> QUEUE_E2E; if only the new
         query's own deadline fails (checked when L <= H) -> ADMIT_LOST
         (scheduled, marked lost);
    otherwise ADMIT_OK.  A malformed query (prompt < 0 or > 2^30, L < 1) or a
    scenario the projection cannot size -> ADMIT_INVALID.
    Returns decision[S], ips[S][H] at the maximum frequency (zeros where not
    evaluated) and the projection with the query."""
    forest = inp["forest"] if forest is None else forest
    S, H = int(inp["n_scenarios"]), int(inp["horizon"])
    nf = int(forest["n_features"])
    dec = np.zeros(S, np.uint32)
    ips_all = np.zeros((S, H), np.float32)
    proj_all = dict(batch=np.zeros((S, H), np.int32), kv=np.zeros((S, H), np.int32),
                    deadline_at=np.full((S, H), NO_DEADLINE, np.uint64),
                    n_iters=np.zeros(S, np.int32), flags=np.zeros(S, np.uint32))
    for s in range(S):
        p, L = int(cand_prompt[s]), int(cand_len[s])
        d_own = np.uint64(cand_deadline_ns[s]) if cand_deadline_ns is not None else NO_DEADLINE
        if p < 0 or p > (1 << 30) or L < 1:
            dec[s] = ADMIT_INVALID
            continue
        board = _append_candidate(inp, s, p, L)
        proj = project(board)
        for k in proj_all:
            proj_all[k][s] = proj[k][0]
        if proj["flags"][0] & FLAG_OVERFLOW:
            dec[s] = ADMIT_INVALID
            continue
        # check 1: the projected KV vector against the capacity
        kv = proj["kv"][0]
        bcap = board.get("batch_cap")
        if int(kv.max()) > int(board["kv_capacity"][0]) or (bcap is not None and
                                                          int(proj["batch"][0][0]) > int(bcap[0])):
            dec[s] = QUEUE_CAPACITY
            continue
        # check 2: M at the maximum frequency on every projected iteration
        eng = None if nf == 3 else np.asarray(inp["engine_size"][s:s + 1], np.float32)
        x = rows(np.array([max_freq_mhz], np.float32), proj["batch"], proj["kv"], eng, nf)
        ips = forest_predict(forest, x)[0, 0]
        ips_all[s] = ips
        n = int(proj["n_iters"][0])
        t_r = [0]
        for j in range(n):
            t_r.append(t_r[-1] + latency_ns(ips[j]))
        sigma = int(inp["tbt_slo_ns"][s])
        if n > 0 and t_r[n] > sigma * n:
            dec[s] = QUEUE_TBT
            continue
        # check 3: Eq. 4 for the scheduled requests, then the new one
        dl = proj["deadline_at"][0]
        if any(dl[j] != NO_DEADLINE and not t_r[j + 1] < int(dl[j]) for j in range(n)):
            dec[s] = QUEUE_E2E
            continue
        if d_own != NO_DEADLINE and L <= H and not t_r[L] < int(d_own):
            dec[s] = ADMIT_LOST
            continue
        dec[s] = ADMIT_OK
    return dict(proj_all, decision=dec, ips=ips_all)


def adjust_lengths(req_offset, generated, pred_len, scale_num, scale_den, max_tokens):
    """Remaining-token counts of the scoreboard from the predictor's total
    generation lengths (Sec. 4.6): the prediction is inflated by the
    scenario's factor num/den (rounded up; den = 0 means no inflation) and
    limited to max_tokens; a request that has already generated at least that
    many tokens is updated to max_tokens.  remaining = max(length - generated,
    1).  max_tokens < 1 means no limit.  Entries with generated < 0 or a
    predicted length < 1 get 0 (the projection ignores them as malformed)."""
    off = np.asarray(req_offset, np.int64)
    out = np.zeros(int(off[-1]) if off.size else 0, np.int32)
    for s in range(off.size - 1):
        num, den, mt = int(scale_num[s]), int(scale_den[s]), int(max_tokens[s])
        for i in range(int(off[s]), int(off[s + 1])):
            g, r = int(generated[i]), int(pred_len[i])
            if g < 0 or r < 1:
                out[i] = 0
                continue
            length = -(-(r * num) // den) if den > 0 else r
            length = min(length, 2 ** 31 - 1)
            if mt >= 1:
                length = min(length, mt)
                if g >= length:
                    length = mt
            out[i] = max(length - g, 1)
    return out
