"""The C-ABI library without a GPU: it loads, exports every symbol the header
declares, and rejects bad arguments on the host before enqueueing anything."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2408_05235_amd import _lib, build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "tl.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tl_[a-z_]+)\s*\(", text)))


def test_header_declares_the_abi():
    assert header_functions() == sorted(_lib.EXPORTED)


def test_library_exports_every_symbol():
    L = _lib.lib()
    out = subprocess.run(["nm", "-D", "--defined-only", build.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (tl_\w+)", out))
    for name in header_functions():
        assert name in exported, name
        assert hasattr(L, name)
    assert L.tl_abi_version() == 1
    assert L.tl_last_error() is not None


def _args(**kw):
    a = _lib.ProjectArgs()
    a.struct_size = ctypes.sizeof(_lib.ProjectArgs)
    a.horizon, a.n_scenarios, a.n_requests, a.block_tokens = 8, 1, 0, 16
    dummy = ctypes.c_void_p(16)   # never dereferenced: validation fails first
    for f in ("req_offset", "kv_capacity", "batch", "kv", "deadline_at", "n_iters", "flags"):
        setattr(a, f, dummy)
    for k, v in kw.items():
        setattr(a, k, v)
    return a


@pytest.mark.parametrize("kw,needle", [
    (dict(struct_size=8), "struct_size"),
    (dict(horizon=0), "horizon"),
    (dict(horizon=8193), "horizon"),
    (dict(block_tokens=0), "block_tokens"),
    (dict(n_scenarios=-1), "n_scenarios"),
    (dict(n_requests=-5), "n_requests"),
    (dict(req_offset=None), "NULL"),
    (dict(n_requests=3), "NULL request array"),
    (dict(rows=ctypes.c_void_p(16), n_freqs=0, n_features=3), "n_freqs"),
    (dict(rows=ctypes.c_void_p(16), n_freqs=4, n_features=5), "n_features"),
    (dict(rows=ctypes.c_void_p(16), n_freqs=4, n_features=3), "freqs_mhz"),
    (dict(rows=ctypes.c_void_p(16), n_freqs=4, n_features=4, freqs_mhz=ctypes.c_void_p(16)), "engine_size"),
    (dict(rows=ctypes.c_void_p(20), n_freqs=4, n_features=4, freqs_mhz=ctypes.c_void_p(16),
          engine_size=ctypes.c_void_p(16)), "aligned"),
])
def test_project_rejects_bad_arguments(kw, needle):
    L = _lib.lib()
    a = _args(**kw)
    assert L.tl_project(ctypes.byref(a), None) == _lib.TL_EINVAL
    assert needle in L.tl_last_error().decode()
    assert L.tl_project(None, None) == _lib.TL_EINVAL


def test_project_with_no_scenarios_is_a_no_op():
    L = _lib.lib()
    assert L.tl_project(ctypes.byref(_args(n_scenarios=0)), None) == _lib.TL_OK


def test_select_and_predict_reject_bad_arguments():
    L = _lib.lib()
    d = ctypes.c_void_p(16)
    assert L.tl_select_freq(d, -1, 4, 8, d, d, d, None, d, d, None) == _lib.TL_EINVAL
    assert L.tl_select_freq(d, 1, 0, 8, d, d, d, None, d, d, None) == _lib.TL_EINVAL
    assert L.tl_select_freq(d, 1, 4097, 8, d, d, d, None, d, d, None) == _lib.TL_EINVAL
    assert L.tl_select_freq(d, 1, 4, 0, d, d, d, None, d, d, None) == _lib.TL_EINVAL
    assert L.tl_select_freq(None, 1, 4, 8, d, d, d, None, d, d, None) == _lib.TL_EINVAL
    assert L.tl_select_freq(None, 0, 4, 8, None, None, None, None, None, None, None) == _lib.TL_OK
    assert L.tl_forest_predict(None, d, 1, d, None) == _lib.TL_EINVAL


def _admit_args(**kw):
    b = _lib.AdmitArgs()
    b.struct_size = ctypes.sizeof(_lib.AdmitArgs)
    b.proj = _args()
    dummy = ctypes.c_void_p(16)   # never dereferenced: validation fails first
    for f in ("forest", "tbt_slo_ns", "cand_prompt", "cand_len", "ips", "decision"):
        setattr(b, f, dummy)
    b.max_freq_mhz = 2000.0
    for k, v in kw.items():
        if k.startswith("proj_"):
            setattr(b.proj, k[5:], v)
        else:
            setattr(b, k, v)
    return b


@pytest.mark.parametrize("kw,needle", [
    (dict(struct_size=16), "struct_size"),
    (dict(proj_struct_size=8), "struct_size"),
    (dict(proj_horizon=0), "horizon"),
    (dict(proj_block_tokens=0), "block_tokens"),
    (dict(proj_req_offset=None), "NULL"),
    (dict(forest=None), "forest is NULL"),
    (dict(cand_len=None), "NULL required pointer"),
    (dict(decision=None), "NULL required pointer"),
])
def test_admit_rejects_bad_arguments(kw, needle):
    L = _lib.lib()
    b = _admit_args(**kw)
    assert L.tl_admit(ctypes.byref(b), None) == _lib.TL_EINVAL
    assert needle in L.tl_last_error().decode()
    assert L.tl_admit(None, None) == _lib.TL_EINVAL


def test_adjust_lengths_rejects_bad_arguments():
    L = _lib.lib()
    d = ctypes.c_void_p(16)
    assert L.tl_adjust_lengths(-1, 0, d, d, d, d, d, d, d, None) == _lib.TL_EINVAL
    assert L.tl_adjust_lengths(1, -1, d, d, d, d, d, d, d, None) == _lib.TL_EINVAL
    assert L.tl_adjust_lengths(1, 5, None, d, d, d, d, d, d, None) == _lib.TL_EINVAL
    assert L.tl_adjust_lengths(1, 5, d, None, d, d, d, d, d, None) == _lib.TL_EINVAL
    assert "NULL request array" in L.tl_last_error().decode()
    assert L.tl_adjust_lengths(0, 0, None, None, None, None, None, None, None, None) == _lib.TL_OK


def test_binary_search_rejects_bad_arguments():
    L = _lib.lib()
    d = ctypes.c_void_p(16)
    args = [d, 1, 4, 8] + [d] * 12 + [None, None]
    for pos, bad, needle in ((0, None, "forest is NULL"), (1, -1, "n_scenarios"), (2, 0, "n_freqs"),
                             (2, 4097, "n_freqs"), (3, 0, "horizon"), (4, None, "NULL required pointer")):
        a = list(args)
        a[pos] = bad
        assert L.tl_select_freq_binary(*a) == _lib.TL_EINVAL
        assert needle in L.tl_last_error().decode()


def test_lattice_rejects_bad_arguments():
    L = _lib.lib()
    d = ctypes.c_void_p(16)
    h = ctypes.c_void_p(99)
    assert L.tl_lattice_create(None, 4, d, 0, None, 10, 10, None, ctypes.byref(h)) == _lib.TL_EINVAL
    assert h.value is None
    assert L.tl_lattice_create(d, 4, d, 0, None, 10, 10, None, None) == _lib.TL_EINVAL
    assert L.tl_lattice_predict_grid(None, 1, 8, d, d, None, d, None) == _lib.TL_EINVAL
    assert L.tl_lattice_bytes(None) == 0
    L.tl_lattice_destroy(None)


def test_forest_create_rejects_bad_trees():
    L = _lib.lib()
    h = ctypes.c_void_p(123)
    feat = np.array([0, 3, 1], np.uint8)       # feature 3 with 3 features: invalid
    thr = np.zeros(3, np.float32)
    leaf = np.zeros(4, np.float32)
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    assert L.tl_forest_create(1, 2, 3, 0.0, P(feat), P(thr), P(leaf), ctypes.byref(h)) == _lib.TL_EINVAL
    assert h.value is None
    assert "feature" in L.tl_last_error().decode()
    assert L.tl_forest_create(1, 15, 3, 0.0, P(feat), P(thr), P(leaf), ctypes.byref(h)) == _lib.TL_EINVAL
    assert L.tl_forest_create(1, 2, 5, 0.0, P(feat), P(thr), P(leaf), ctypes.byref(h)) == _lib.TL_EINVAL
    assert L.tl_forest_create(-1, 2, 3, 0.0, P(feat), P(thr), P(leaf), ctypes.byref(h)) == _lib.TL_EINVAL
    assert L.tl_forest_create(1, 2, 3, 0.0, None, P(thr), P(leaf), ctypes.byref(h)) == _lib.TL_EINVAL
    assert L.tl_forest_create(1, 2, 3, 0.0, P(feat), P(thr), P(leaf), None) == _lib.TL_EINVAL
    L.tl_forest_destroy(None)


DIV_TEST = r"""
#include <cstdio>
#include <cstdint>
#include "device_util.h"
// host model of the device routine (mulhi is the high half of the 64-bit product)
static uint32_t host_div(uint32_t x, tl::DivU32 q) {
    uint32_t hi = (uint32_t)(((uint64_t)q.m * x) >> 32);
    return (hi + x) >> q.l;
}
int main() {
    uint64_t bad = 0;
    for (uint32_t d = 1; d <= 65536; ++d) {
        tl::DivU32 q = tl::make_divu32(d);
        uint32_t xs[] = {0u, 1u, d - 1, d, d + 1, 2 * d - 1, 2 * d, 1u << 20, (1u << 30) + 12345u,
                         0x7fffffffu - d, 0x7fffffffu, 0x7ffffffeu, 123456789u};
        for (uint32_t x : xs) if (host_div(x, q) != x / d) ++bad;
        for (uint32_t x = 0; x < 4096; ++x) if (host_div(x * 7919u, q) != (x * 7919u) / d) ++bad;
    }
    printf("%llu\n", (unsigned long long)bad);
    return bad != 0;
}
"""


def test_invariant_divisor_constants(tmp_path):
    src = tmp_path / "t.cpp"
    src.write_text(DIV_TEST)
    exe = tmp_path / "t"
    subprocess.run([build.hipcc(), "-O2", "-std=c++17", "-x", "hip", "--offload-arch=gfx950",
                    "-I", build.CSRC, "-I", build.INCLUDE, str(src), "-o", str(exe)],
                   check=True, capture_output=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0 and out.stdout.strip() == "0", out.stdout + out.stderr
