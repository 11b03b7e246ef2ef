"""Host-side helpers of bench.py (no GPU)."""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import bench  # noqa: E402


def test_spread_nearest_rank_p90():
    v = [float(x) for x in range(20, 0, -1)]      # 20 .. 1, unsorted input
    assert bench.spread(v) == {"median": 10.5, "min": 1.0, "p90": 18.0}
    assert bench.spread([3.0, 1.0, 2.0, 10.0, 4.0]) == {"median": 3.0, "min": 1.0, "p90": 10.0}
    assert bench.spread([float(x) for x in range(1, 11)])["p90"] == 9.0
    assert bench.spread([2.5]) == {"median": 2.5, "min": 2.5, "p90": 2.5}
