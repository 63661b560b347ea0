"""The benchmark's count of model evaluations per binary search, derived
from the search's results, against a direct replay of the search (Sec. 4.5)
over random feasibility tables: probes while lo < hi, plus the check of lo
only when hi stayed at F-1."""
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def _replay(feas):
    F = len(feas)
    lo, hi, n = 0, F - 1, 0
    while lo < hi:
        mid = lo + (hi - lo) // 2
        n += 1
        if feas[mid]:
            hi = mid
        else:
            lo = mid + 1
    if hi < F - 1:
        return lo, 0, n
    return (lo, 0, n + 1) if feas[lo] else (F - 1, 1, n + 1)


def test_search_evaluations_match_replay():
    rng = np.random.default_rng(3)
    for F in (1, 2, 3, 5, 16, 48, 64, 100):
        idx, st, want = [], [], []
        for _ in range(200):
            i, s, n = _replay(rng.random(F) < rng.uniform(0.05, 0.95))
            idx.append(i)
            st.append(s)
            want.append(n)
        # scenarios settled by their flags (lost 2, invalid 3) evaluate nothing
        idx += [F - 1, F - 1]
        st += [2, 3]
        want += [0, 0]
        assert bench.search_evaluations(idx, st, F).tolist() == want
