"""The grid kernel's barrier-free hand-over of its two LDS tree buffers
(stage_acquire / stage_release in forest_walk.h), as a model run on the CPU.

Wavefronts advance one step at a time in a seeded random order: a step is an
atomic operation on the shared counters (a compare-and-swap, an add, a load),
part of a block's evaluation or part of a copy.  Over many schedules, worker
counts and block counts, the checks are that every wavefront finishes, that a
wavefront evaluates block b only while buffer b & 1 holds block b completely
copied, and that no copy into a buffer starts while any wavefront still
evaluates the block that buffer held before.
"""
import random

import pytest


def run_schedule(n_waves, n_blocks, seed):
    rnd = random.Random(seed)
    claimed, ready, done = [0, -1], [0, -1], [0, 0]
    held = [0, None]                 # block a buffer holds, ("copy", b) while it is copied
    users = [set(range(n_waves)), set()]
    st = [{"b": 0, "phase": "eval"} for _ in range(n_waves)]
    steps = 0
    while any(s["phase"] != "end" for s in st):
        steps += 1
        assert steps < 10 ** 7, "no progress"
        w = rnd.randrange(n_waves)
        s = st[w]
        b = s["b"]
        cur = b & 1
        if s["phase"] == "end":
            continue
        if s["phase"] == "eval":
            assert held[cur] == b, (w, b, held)
            if rnd.random() < 0.3:      # the evaluation takes a random number of steps
                continue
            users[cur].discard(w)
            done[cur] += 1             # stage_release
            if b + 1 == n_blocks:
                s["phase"] = "end"
            else:
                s["b"], s["phase"] = b + 1, "acquire"
        elif s["phase"] == "acquire":  # stage_acquire: wait for ready, or claim
            if ready[cur] == b:
                s["phase"] = "eval"
                users[cur].add(w)
            elif claimed[cur] == b - 2:
                claimed[cur] = b       # the compare-and-swap this wavefront won
                s["phase"] = "wait_done"
        elif s["phase"] == "wait_done":
            if done[cur] >= n_waves * (b >> 1):
                assert not users[cur], ("copy over a buffer in use", w, b, users[cur])
                held[cur] = ("copy", b)
                s["phase"] = "copying"
        elif s["phase"] == "copying":
            if rnd.random() < 0.5:
                continue
            held[cur] = b
            ready[cur] = b
            s["phase"] = "eval"
            users[cur].add(w)
    return steps


@pytest.mark.parametrize("n_waves", [1, 2, 3, 16])
def test_stage_hand_over_model(n_waves):
    for seed in range(300):
        rnd = random.Random(1000 * n_waves + seed)
        run_schedule(n_waves, rnd.randint(1, 30), 1000 * n_waves + seed)
