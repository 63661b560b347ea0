"""The barrier-free hand-over of the LDS tree buffers (stage_acquire /
stage_release in forest_walk.h; three buffers in the grid kernel, two in the
column kernels), as a model run on the CPU.

Wavefronts advance one step at a time in a seeded random order: a step is an
atomic operation on the shared counters (a compare-and-swap, an add, a load),
part of a block's evaluation or part of a copy.  Over many schedules, worker
counts, block counts and buffer counts NB, the checks are that every
wavefront finishes, that a wavefront evaluates block b only while buffer
b % NB holds block b completely copied, that no copy into a buffer starts
while any wavefront still evaluates the block that buffer held before, and
that a wavefront waiting for block b is never more than NB blocks ahead of
the slowest (it evaluates at most NB - 1 ahead).
"""
import random

import pytest


def run_schedule(n_waves, n_blocks, seed, nb=2):
    rnd = random.Random(seed)
    # stage_sync_init: buffer 0 holds block 0; buffer i waits for block i,
    # claimed from "block i - nb"
    claimed = [0] + [i - nb for i in range(1, nb)]
    ready = [0] + [-1] * (nb - 1)
    done = [0] * nb
    held = [0] + [None] * (nb - 1)   # block a buffer holds, ("copy", b) while it is copied
    users = [set(range(n_waves))] + [set() for _ in range(nb - 1)]
    st = [{"b": 0, "phase": "eval"} for _ in range(n_waves)]
    steps = 0
    while any(s["phase"] != "end" for s in st):
        steps += 1
        assert steps < 10 ** 7, "no progress"
        w = rnd.randrange(n_waves)
        s = st[w]
        b = s["b"]
        cur = b % nb
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
            elif claimed[cur] == b - nb:
                claimed[cur] = b       # the compare-and-swap this wavefront won
                s["phase"] = "wait_done"
        elif s["phase"] == "wait_done":
            if done[cur] >= n_waves * (b // nb):
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
        live = [x["b"] for x in st if x["phase"] != "end"]
        assert not live or max(live) - min(live) <= nb, ("too far ahead", live)
    return steps


@pytest.mark.parametrize("nb", [2, 3])
@pytest.mark.parametrize("n_waves", [1, 2, 3, 16])
def test_stage_hand_over_model(n_waves, nb):
    for seed in range(300):
        rnd = random.Random(1000 * n_waves + seed)
        run_schedule(n_waves, rnd.randint(1, 30), 1000 * n_waves + seed, nb)
