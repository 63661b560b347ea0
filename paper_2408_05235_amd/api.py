"""Python entry points with the names of the C ABI; argument marshalling only.

Every computation runs in the HIP kernels of libtl.so.  Tensors must live on
the current CUDA(HIP) device; work is enqueued on torch's current stream.
Unsigned 64-bit quantities (deadlines, SLOs) travel as ``torch.int64``
tensors holding the same bits; 32-bit flag words as ``torch.int32``.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import _lib
from ._lib import check, lib


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _need(t, dtype, name, shape=None):
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t


def _opt(t, dtype, name, shape=None):
    return None if t is None else _need(t, dtype, name, shape)


def _project_args(req_offset, prompt_len, generated, remaining, arrival_iter, kv_capacity,
                  horizon, block_tokens, deadline_ns, lost, batch_cap, out):
    """Checked tl_project_args for the scoreboards, with the curve outputs
    (taken from ``out`` or allocated).  Returns (args, outputs)."""
    _need(req_offset, torch.int64, "req_offset")
    S = req_offset.numel() - 1
    R = prompt_len.numel()
    for name, t in (("prompt_len", prompt_len), ("generated", generated),
                    ("remaining", remaining), ("arrival_iter", arrival_iter)):
        _need(t, torch.int32, name, (R,))
    _need(kv_capacity, torch.int32, "kv_capacity", (S,))
    _opt(deadline_ns, torch.int64, "deadline_ns", (R,))
    _opt(lost, torch.uint8, "lost", (R,))
    _opt(batch_cap, torch.int32, "batch_cap", (S,))
    H = int(horizon)
    dev = req_offset.device
    o = out or {}

    def buf(name, shape, dtype):
        t = o.get(name) if o.get(name) is not None else torch.empty(shape, dtype=dtype, device=dev)
        return _need(t, dtype, name, shape)

    res = dict(batch=buf("batch", (S, H), torch.int32), kv=buf("kv", (S, H), torch.int32),
               deadline_at=buf("deadline_at", (S, H), torch.int64), n_iters=buf("n_iters", (S,), torch.int32),
               flags=buf("flags", (S,), torch.int32))
    a = _lib.ProjectArgs()
    a.struct_size = ctypes.sizeof(_lib.ProjectArgs)
    a.horizon = H
    a.n_scenarios = S
    a.n_requests = R
    a.block_tokens = int(block_tokens)
    a.req_offset = _p(req_offset)
    a.prompt_len = _p(prompt_len)
    a.generated = _p(generated)
    a.remaining = _p(remaining)
    a.arrival_iter = _p(arrival_iter)
    a.deadline_ns = _p(deadline_ns)
    a.lost = _p(lost)
    a.kv_capacity = _p(kv_capacity)
    a.batch_cap = _p(batch_cap)
    a.batch, a.kv, a.deadline_at = _p(res["batch"]), _p(res["kv"]), _p(res["deadline_at"])
    a.n_iters, a.flags = _p(res["n_iters"]), _p(res["flags"])
    return a, res


def tl_project(req_offset, prompt_len, generated, remaining, arrival_iter, kv_capacity,
               horizon, block_tokens, deadline_ns=None, lost=None, batch_cap=None,
               freqs_mhz=None, engine_size=None, n_features=3, want_rows=True, out=None):
    """Stage 1 (tl_project).  Returns a dict of device tensors:
    batch, kv [S,H] int32; deadline_at [S,H] int64 (uint64 bits); n_iters [S]
    int32; flags [S] int32 (uint32 bits); rows [S,F,H,n_features] fp32 when
    ``want_rows`` and ``freqs_mhz`` is given."""
    a, res = _project_args(req_offset, prompt_len, generated, remaining, arrival_iter, kv_capacity,
                           horizon, block_tokens, deadline_ns, lost, batch_cap, out)
    S, H = int(a.n_scenarios), int(a.horizon)
    rows_on = bool(want_rows and freqs_mhz is not None)
    if rows_on:
        F = int(freqs_mhz.numel())
        _need(freqs_mhz, torch.float32, "freqs_mhz", (F,))
        if n_features == 4:
            _need(engine_size, torch.float32, "engine_size", (S,))
        o = out or {}
        rows = o.get("rows")
        if rows is None:
            rows = torch.empty((S, F, H, n_features), dtype=torch.float32, device=req_offset.device)
        _need(rows, torch.float32, "rows", (S, F, H, n_features))
        a.n_freqs, a.n_features = F, int(n_features)
        a.freqs_mhz, a.engine_size, a.rows = _p(freqs_mhz), _p(engine_size), _p(rows)
        res["rows"] = rows
    check(lib().tl_project(ctypes.byref(a), _stream()))
    return res


def tl_admit(forest, max_freq_mhz, tbt_slo_ns, cand_prompt, cand_len, req_offset, prompt_len, generated,
             remaining, arrival_iter, kv_capacity, horizon, block_tokens, deadline_ns=None, lost=None,
             batch_cap=None, engine_size=None, cand_deadline_ns=None, out=None, lattice=None):
    """Admission control (tl_admit) for one new query per scenario.  Returns
    the projection with the query (batch, kv, deadline_at, n_iters, flags as
    in tl_project), ips [S,H] fp32 at max_freq_mhz and decision [S] int32
    (TL_ADMIT_* codes)."""
    a, res = _project_args(req_offset, prompt_len, generated, remaining, arrival_iter, kv_capacity,
                           horizon, block_tokens, deadline_ns, lost, batch_cap, out)
    S, H = int(a.n_scenarios), int(a.horizon)
    dev = req_offset.device
    _need(tbt_slo_ns, torch.int64, "tbt_slo_ns", (S,))
    _need(cand_prompt, torch.int32, "cand_prompt", (S,))
    _need(cand_len, torch.int32, "cand_len", (S,))
    _opt(cand_deadline_ns, torch.int64, "cand_deadline_ns", (S,))
    if forest.n_features == 4:
        _need(engine_size, torch.float32, "engine_size", (S,))
    o = out or {}
    ips = o.get("ips") if o.get("ips") is not None else torch.empty((S, H), dtype=torch.float32, device=dev)
    dec = o.get("decision") if o.get("decision") is not None else torch.empty(S, dtype=torch.int32, device=dev)
    _need(ips, torch.float32, "ips", (S, H))
    _need(dec, torch.int32, "decision", (S,))
    b = _lib.AdmitArgs()
    b.struct_size = ctypes.sizeof(_lib.AdmitArgs)
    b.proj = a
    b.forest = forest._h
    b.max_freq_mhz = float(max_freq_mhz)
    b.engine_size = _p(engine_size) if forest.n_features == 4 else None
    b.tbt_slo_ns = _p(tbt_slo_ns)
    b.cand_prompt, b.cand_len, b.cand_deadline_ns = _p(cand_prompt), _p(cand_len), _p(cand_deadline_ns)
    b.ips, b.decision = _p(ips), _p(dec)
    b.lattice = None if lattice is None else lattice._h
    check(lib().tl_admit(ctypes.byref(b), _stream()))
    res.update(ips=ips, decision=dec)
    return res


class Forest:
    """Device copy of a tree ensemble (tl_forest_create / tl_forest_destroy)."""

    def __init__(self, n_trees, depth, n_features, base_score, feature, threshold, leaf):
        feature = np.ascontiguousarray(feature, dtype=np.uint8)
        threshold = np.ascontiguousarray(threshold, dtype=np.float32)
        leaf = np.ascontiguousarray(leaf, dtype=np.float32)
        n_int = (1 << int(depth)) - 1
        if feature.size != n_trees * n_int or threshold.size != n_trees * n_int or leaf.size != n_trees * (n_int + 1):
            raise ValueError("tree array sizes do not match n_trees and depth")
        self.n_trees, self.depth, self.n_features = int(n_trees), int(depth), int(n_features)
        self.base_score = float(np.float32(base_score))
        h = ctypes.c_void_p()
        check(lib().tl_forest_create(self.n_trees, self.depth, self.n_features, self.base_score,
                                     feature.ctypes.data_as(ctypes.c_void_p),
                                     threshold.ctypes.data_as(ctypes.c_void_p),
                                     leaf.ctypes.data_as(ctypes.c_void_p), ctypes.byref(h)))
        self._h = h

    @classmethod
    def from_dict(cls, d):
        return cls(d["n_trees"], d["depth"], d["n_features"], d["base_score"],
                   d["feature"], d["threshold"], d["leaf"])

    def tl_forest_predict(self, rows, out=None):
        """IPS for every row of ``rows`` ([..., n_features] fp32 device tensor)."""
        _need(rows, torch.float32, "rows")
        if rows.shape[-1] != self.n_features:
            raise ValueError(f"rows have {rows.shape[-1]} features, forest has {self.n_features}")
        n = rows.numel() // self.n_features
        if out is None:
            out = torch.empty(rows.shape[:-1], dtype=torch.float32, device=rows.device)
        _need(out, torch.float32, "out")
        if out.numel() != n:
            raise ValueError("out has the wrong number of elements")
        check(lib().tl_forest_predict(self._h, _p(rows), n, _p(out), _stream()))
        return out

    predict = tl_forest_predict

    def tl_forest_predict_grid(self, freqs_mhz, kv, batch, engine_size=None, out=None, noalloc=False):
        """IPS on the projection grid: out[s, f, j] = M(freqs[f], kv[s, j],
        batch[s, j] [, engine[s]]) without materializing the rows.  With
        ``noalloc`` (and ``out`` given) the call goes to
        tl_forest_predict_grid_noalloc, which allocates nothing."""
        _need(kv, torch.int32, "kv")
        if kv.dim() != 2:
            raise ValueError("kv must be [S, H]")
        S, H = kv.shape
        F = freqs_mhz.numel()
        _need(freqs_mhz, torch.float32, "freqs_mhz", (F,))
        _need(batch, torch.int32, "batch", (S, H))
        if self.n_features == 4:
            _need(engine_size, torch.float32, "engine_size", (S,))
        else:
            engine_size = None
        if out is None:
            out = torch.empty((S, F, H), dtype=torch.float32, device=kv.device)
        _need(out, torch.float32, "out", (S, F, H))
        fn = lib().tl_forest_predict_grid_noalloc if noalloc else lib().tl_forest_predict_grid
        check(fn(self._h, S, F, H, _p(freqs_mhz), _p(kv), _p(batch), _p(engine_size), _p(out), _stream()))
        return out

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().tl_forest_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Lattice:
    """The model compiled to its input lattice (tl_lattice_create): every
    (engine size, batch 0..batch_max, frequency, KV 0..kv_max) evaluated once;
    prediction on the projection grid is then a table lookup with the same
    values (tl_lattice_predict_grid).  Keeps the forest alive."""

    def __init__(self, forest, freqs_mhz, kv_max, batch_max, engine_values=None):
        _need(freqs_mhz, torch.float32, "freqs_mhz")
        self.forest = forest
        self.n_freqs = int(freqs_mhz.numel())
        ev = np.ascontiguousarray(engine_values if engine_values is not None else [], dtype=np.float32)
        h = ctypes.c_void_p()
        check(lib().tl_lattice_create(forest._h, self.n_freqs, _p(freqs_mhz), int(ev.size),
                                      ev.ctypes.data_as(ctypes.c_void_p) if ev.size else None, int(kv_max),
                                      int(batch_max), _stream(), ctypes.byref(h)))
        self._h = h
        self.nbytes = int(lib().tl_lattice_bytes(h))

    def tl_lattice_predict_grid(self, kv, batch, engine_size=None, out=None):
        """IPS [S, F, H] for the projection curves kv, batch [S, H] int32."""
        _need(kv, torch.int32, "kv")
        if kv.dim() != 2:
            raise ValueError("kv must be [S, H]")
        S, H = kv.shape
        _need(batch, torch.int32, "batch", (S, H))
        if self.forest.n_features == 4:
            _need(engine_size, torch.float32, "engine_size", (S,))
        if out is None:
            out = torch.empty((S, self.n_freqs, H), dtype=torch.float32, device=kv.device)
        _need(out, torch.float32, "out", (S, self.n_freqs, H))
        check(lib().tl_lattice_predict_grid(self._h, S, H, _p(kv), _p(batch),
                                            _p(engine_size) if self.forest.n_features == 4 else None, _p(out),
                                            _stream()))
        return out

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().tl_lattice_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def tl_select_freq(ips, deadline_at, n_iters, tbt_slo_ns, proj_flags=None, out=None):
    """Stage 3 (tl_select_freq).  ips [S,F,H] fp32.  Returns (freq_idx int32
    [S], status int32 [S])."""
    _need(ips, torch.float32, "ips")
    if ips.dim() != 3:
        raise ValueError("ips must be [S, F, H]")
    S, F, H = ips.shape
    _need(deadline_at, torch.int64, "deadline_at", (S, H))
    _need(n_iters, torch.int32, "n_iters", (S,))
    _need(tbt_slo_ns, torch.int64, "tbt_slo_ns", (S,))
    _opt(proj_flags, torch.int32, "proj_flags", (S,))
    o = out or {}
    idx = o.get("freq_idx") if o.get("freq_idx") is not None else torch.empty(S, dtype=torch.int32, device=ips.device)
    st = o.get("status") if o.get("status") is not None else torch.empty(S, dtype=torch.int32, device=ips.device)
    _need(idx, torch.int32, "freq_idx", (S,))
    _need(st, torch.int32, "status", (S,))
    check(lib().tl_select_freq(_p(ips), S, F, H, _p(deadline_at), _p(n_iters), _p(tbt_slo_ns),
                               _p(proj_flags), _p(idx), _p(st), _stream()))
    return idx, st


def tl_select_freq_binary(forest, freqs_mhz, kv, batch, deadline_at, n_iters, tbt_slo_ns, proj_flags=None,
                          engine_size=None, out=None, lattice=None):
    """The controller's binary search over frequencies (tl_select_freq_binary),
    querying the model only at probed frequencies (read from ``lattice``, a
    Lattice of the same forest built for freqs_mhz, when given).  kv, batch
    [S,H] int32 as written by tl_project.  Returns (freq_idx int32 [S],
    status int32 [S])."""
    _need(kv, torch.int32, "kv")
    if kv.dim() != 2:
        raise ValueError("kv must be [S, H]")
    S, H = kv.shape
    F = int(freqs_mhz.numel())
    _need(freqs_mhz, torch.float32, "freqs_mhz", (F,))
    _need(batch, torch.int32, "batch", (S, H))
    _need(deadline_at, torch.int64, "deadline_at", (S, H))
    _need(n_iters, torch.int32, "n_iters", (S,))
    _need(tbt_slo_ns, torch.int64, "tbt_slo_ns", (S,))
    _opt(proj_flags, torch.int32, "proj_flags", (S,))
    if forest.n_features == 4:
        _need(engine_size, torch.float32, "engine_size", (S,))
    o = out or {}
    dev = kv.device

    def buf(name, shape, dtype):
        t = o.get(name) if o.get(name) is not None else torch.empty(shape, dtype=dtype, device=dev)
        return _need(t, dtype, name, shape)

    ips = buf("ips_work", (S, H), torch.float32)
    work = buf("search_work", (3, S), torch.int32)
    idx = buf("freq_idx", (S,), torch.int32)
    st = buf("status", (S,), torch.int32)
    check(lib().tl_select_freq_binary(forest._h, S, F, H, _p(freqs_mhz), _p(kv), _p(batch),
                                      _p(engine_size) if forest.n_features == 4 else None, _p(deadline_at),
                                      _p(n_iters), _p(tbt_slo_ns), _p(proj_flags), _p(ips), _p(work), _p(idx),
                                      _p(st), None if lattice is None else lattice._h, _stream()))
    return idx, st


def tl_adjust_lengths(req_offset, generated, pred_len, scale_num, scale_den, max_tokens, out=None):
    """Scoreboard remaining-token counts from predicted total lengths under
    generation-length errors (tl_adjust_lengths).  Per-scenario scale_num,
    scale_den (int32 tensors holding uint32 bits) and max_tokens.  Returns
    remaining [R] int32."""
    _need(req_offset, torch.int64, "req_offset")
    S = req_offset.numel() - 1
    R = generated.numel()
    _need(generated, torch.int32, "generated", (R,))
    _need(pred_len, torch.int32, "pred_len", (R,))
    for name, t in (("scale_num", scale_num), ("scale_den", scale_den), ("max_tokens", max_tokens)):
        _need(t, torch.int32, name, (S,))
    rem = out if out is not None else torch.empty(R, dtype=torch.int32, device=req_offset.device)
    _need(rem, torch.int32, "out", (R,))
    check(lib().tl_adjust_lengths(S, R, _p(req_offset), _p(generated), _p(pred_len), _p(scale_num),
                                  _p(scale_den), _p(max_tokens), _p(rem), _stream()))
    return rem


# short names
project = tl_project
select_freq = tl_select_freq
select_freq_binary = tl_select_freq_binary
admit = tl_admit
adjust_lengths = tl_adjust_lengths


def upload(inp, device="cuda"):
    """Copy a numpy input dict (``synth.make_inputs``) to device tensors."""
    def t(a, dtype=None):
        if a is None:
            return None
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint64:
            a = a.view(np.int64)
        if a.dtype == np.uint32:
            a = a.view(np.int32)
        return torch.from_numpy(a).to(device)

    return dict(
        n_scenarios=int(inp["n_scenarios"]), horizon=int(inp["horizon"]),
        block_tokens=int(inp["block_tokens"]), n_features=int(inp["n_features"]),
        req_offset=t(inp["req_offset"]), prompt=t(inp["prompt"]), generated=t(inp["generated"]),
        remaining=t(inp["remaining"]), arrival=t(inp["arrival"]), deadline_ns=t(inp.get("deadline_ns")),
        lost=t(inp.get("lost")), kv_capacity=t(inp["kv_capacity"]), batch_cap=t(inp.get("batch_cap")),
        tbt_slo_ns=t(inp["tbt_slo_ns"]), freqs_mhz=t(inp["freqs_mhz"]),
        engine_size=t(inp.get("engine_size")),
    )


class Controller:
    """The whole hot path for one batch of scenarios: project -> predict ->
    select, enqueued back to back on the current stream with preallocated
    buffers (no host round trip between stages).

    By default the feature rows are formed inside the forest kernel
    (tl_forest_predict_grid); with ``materialize_rows=True`` tl_project writes
    them and tl_forest_predict reads them back (same results)."""

    def __init__(self, dev_inputs, forest, materialize_rows=False):
        self.d = dev_inputs
        self.forest = forest
        self.materialize_rows = materialize_rows
        d = dev_inputs
        S, H = d["n_scenarios"], d["horizon"]
        F, nf = d["freqs_mhz"].numel(), d["n_features"]
        dev = d["req_offset"].device
        self.buf = dict(
            batch=torch.empty((S, H), dtype=torch.int32, device=dev),
            kv=torch.empty((S, H), dtype=torch.int32, device=dev),
            deadline_at=torch.empty((S, H), dtype=torch.int64, device=dev),
            n_iters=torch.empty(S, dtype=torch.int32, device=dev),
            flags=torch.empty(S, dtype=torch.int32, device=dev),
        )
        if materialize_rows:
            self.buf["rows"] = torch.empty((S, F, H, nf), dtype=torch.float32, device=dev)
        self.ips = torch.empty((S, F, H), dtype=torch.float32, device=dev)
        self.sel = dict(freq_idx=torch.empty(S, dtype=torch.int32, device=dev),
                        status=torch.empty(S, dtype=torch.int32, device=dev))

    def project(self):
        d = self.d
        return tl_project(d["req_offset"], d["prompt"], d["generated"], d["remaining"], d["arrival"],
                          d["kv_capacity"], d["horizon"], d["block_tokens"], d["deadline_ns"],
                          d["lost"], d["batch_cap"], d["freqs_mhz"], d["engine_size"],
                          d["n_features"], self.materialize_rows, self.buf)

    def predict(self):
        if self.materialize_rows:
            return self.forest.tl_forest_predict(self.buf["rows"], self.ips)
        return self.forest.tl_forest_predict_grid(self.d["freqs_mhz"], self.buf["kv"], self.buf["batch"],
                                                  self.d["engine_size"], self.ips)

    def select(self):
        return tl_select_freq(self.ips, self.buf["deadline_at"], self.buf["n_iters"],
                              self.d["tbt_slo_ns"], self.buf["flags"], self.sel)

    def step(self):
        self.project()
        self.predict()
        return self.select()

    def select_binary(self, lattice=None):
        """The paper's binary search over the frequencies on the projection
        (tl_select_freq_binary): the model only at probed frequencies, read
        from ``lattice`` when given."""
        d, b = self.d, self.buf
        if "search" not in self.__dict__:
            S, H = d["n_scenarios"], d["horizon"]
            dev = d["req_offset"].device
            self.search = dict(ips_work=torch.empty((S, H), dtype=torch.float32, device=dev),
                               search_work=torch.empty((3, S), dtype=torch.int32, device=dev),
                               freq_idx=torch.empty(S, dtype=torch.int32, device=dev),
                               status=torch.empty(S, dtype=torch.int32, device=dev))
        return tl_select_freq_binary(self.forest, d["freqs_mhz"], b["kv"], b["batch"], b["deadline_at"],
                                     b["n_iters"], d["tbt_slo_ns"], b["flags"], d["engine_size"], self.search,
                                     lattice)
