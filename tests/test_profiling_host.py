"""Host logic of the profile summaries: dispatches of a counter profile are
attributed to the stages of the traced layer calls between the library's
stage markers (k_stage_begin opens a call, k_stage_mark closes each stage),
in the order bench.py's schedule lists the calls."""
import pytest

from paper_2009_00804_amd import profiling as P


def test_dispatches_attributed_between_stage_markers():
    sched = [{"workload": "w", "layers": [["a", "b"], ["c"]], "calls": 2}]
    disp = [("before", 1.0),
            ("k_stage_begin", 0), ("g1", 2.0), ("k_stage_mark", 0), ("g2", 3.0), ("k_stage_mark", 0),
            ("between", 9.0),
            ("k_stage_begin", 0), ("g3", 4.0), ("k_stage_mark", 0),
            ("k_stage_begin", 0), ("g1", 2.0), ("k_stage_mark", 0), ("g2", 3.0), ("g2b", 1.0),
            ("k_stage_mark", 0),
            ("k_stage_begin", 0), ("g3", 4.0), ("k_stage_mark", 0), ("after", 7.0)]
    acc, kern = P.attribute(disp, sched)
    assert acc == {("w", 1, "a"): 4.0, ("w", 1, "b"): 7.0, ("w", 2, "c"): 8.0}
    assert kern[("w", 1, "b")] == {"g2", "g2b"}


def test_attribution_refuses_a_profile_that_disagrees_with_the_schedule():
    sched = [{"workload": "w", "layers": [["a"]], "calls": 2}]
    one_call = [("k_stage_begin", 0), ("g", 1.0), ("k_stage_mark", 0)]
    with pytest.raises(ValueError):
        P.attribute(one_call, sched)
    with pytest.raises(ValueError):
        P.attribute(one_call * 3, sched)
