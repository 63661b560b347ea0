"""Load the hand-computed fixtures under tests/golden/ as input dicts."""
import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
NONE = np.uint64(0xFFFFFFFFFFFFFFFF)


def load(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return json.load(fh)


def scoreboard(g, deadline_ns=None, lost=None):
    n = len(g["prompt"])
    dl = deadline_ns if deadline_ns is not None else g.get("deadline_ns")
    return dict(
        n_scenarios=1, horizon=g["horizon"], block_tokens=g["block_tokens"],
        req_offset=np.array([0, n], np.int64),
        prompt=np.array(g["prompt"], np.int32), generated=np.array(g["generated"], np.int32),
        remaining=np.array(g["remaining"], np.int32), arrival=np.array(g["arrival"], np.int32),
        deadline_ns=None if dl is None else np.array(dl, np.uint64),
        lost=None if lost is None else np.array(lost, np.uint8),
        kv_capacity=np.array([g["kv_capacity"]], np.int32),
        batch_cap=None if g.get("batch_cap") is None else np.array([g["batch_cap"]], np.int32),
    )


def deadline_map(lst):
    return np.array([NONE if v is None else np.uint64(v) for v in lst], np.uint64)


def forest(g):
    f = g["forest"]
    return dict(n_trees=f["n_trees"], depth=f["depth"], n_features=f["n_features"],
                base_score=np.float32(f["base_score"]),
                feature=np.array(f["feature"], np.uint8).reshape(f["n_trees"], -1),
                threshold=np.array(f["threshold"], np.float32).reshape(f["n_trees"], -1),
                leaf=np.array(f["leaf"], np.float32).reshape(f["n_trees"], -1))


def scoreboard_multi(g, sigma_ns, lost=None):
    """Several scenarios from one fixture: CSR offsets, per-scenario
    capacities and engine sizes; deadlines sigma_s * r_i per request."""
    off = np.array(g["req_offset"], np.int64)
    S = off.size - 1
    rem = np.array(g["remaining"], np.int64)
    sig = np.repeat(np.array(sigma_ns, np.uint64), np.diff(off))
    return dict(
        n_scenarios=S, horizon=g["horizon"], block_tokens=g["block_tokens"], req_offset=off,
        prompt=np.array(g["prompt"], np.int32), generated=np.array(g["generated"], np.int32),
        remaining=rem.astype(np.int32), arrival=np.array(g["arrival"], np.int32),
        deadline_ns=(rem.astype(np.uint64) * sig).astype(np.uint64),
        lost=None if lost is None else np.array(lost, np.uint8),
        kv_capacity=np.array(g.get("kv_capacity", [1 << 30] * S), np.int32),
        batch_cap=None,
        engine_size=np.array(g["engine_size"], np.float32),
        tbt_slo_ns=np.array(sigma_ns, np.uint64),
    )
