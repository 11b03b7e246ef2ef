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


def test_counter_summary_sums_a_stages_dispatches_by_slot(tmp_path):
    """Counter mode: gather1 (fp32) is dispatches 0-3 of every five of the
    sliced-sum kernel plus the first of every three combines; its derived
    figures come from the per-launch sums."""
    import csv
    import types
    names = (["k_gather_sum<float, 8, 1, 4, 4, true>(saga::GatherArgs, int, int)"] * 5
             + ["k_combine<float>(saga::GatherArgs)"] * 3)
    rows, did = [], 0
    for _ in range(2):
        for i, n in enumerate(names):
            did += 1
            hit = 30.0 if i < 4 else (5.0 if n.startswith("k_gather") else 1.0)
            for c, v in (("TCC_HIT_sum", hit), ("TCC_MISS_sum", 10.0), ("GRBM_GUI_ACTIVE", 1000.0),
                         ("TCP_TCC_READ_REQ_sum", 100.0), ("TCP_TCC_READ_REQ_LATENCY_sum", 54500.0)):
                rows.append({"Dispatch_Id": did, "Kernel_Name": n, "Counter_Name": c,
                             "Counter_Value": v})
    d = tmp_path / "p1"
    d.mkdir()
    with open(d / "run_counter_collection.csv", "w") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)
    a = types.SimpleNamespace(counters=str(d), dtype="f32", command="cmd", passes="p", out=str(tmp_path),
                              tag="t")
    P.counters_main(a)
    text = (tmp_path / "counters_t_f32.txt").read_text()
    g1 = text.split("## gather1")[1].split("##")[0]
    # four sliced passes at 30 hits + one combine at 1 hit; five dispatches of misses
    assert "TCC_HIT_sum" in g1 and " 121\n" in g1
    assert "= L2 hit rate: %.4g" % (121 / 171) in g1
    assert "= L1->L2 read latency, cycles per request: 545" in g1
    assert "= L1->L2 reads in flight per CU: %.4g" % (8 * 5 * 54500 / (5 * 1000 * 256)) in g1
    # gather2 takes the fifth sliced pass (5 hits) and combines 1 and 2, but
    # its 9-column kernel is absent from this profile: no gather2 section
    assert "## gather2" not in text


def test_short_names_drop_namespaces_and_arguments():
    """The library's stage markers live in an anonymous namespace of their
    own (not saga's): their short names must still be the bare kernel names
    the attribution looks for."""
    assert P._short("(anonymous namespace)::k_stage_begin()") == "k_stage_begin()"
    assert P._short("saga::(anonymous namespace)::k_stage_mark()").startswith("k_stage_mark")
    assert P._short("void saga::(anonymous namespace)::k_combine<float>(saga::GatherArgs)") == \
        "k_combine<float>"


def test_marker_ranges_attributed_to_layer_calls_and_stages():
    """roctx ranges of a marker trace: each "saga_layer" range holds its
    stages' "saga stage k" ranges in order; host times are attributed to
    (workload, layer, stage) in the schedule's call order."""
    sched = [{"workload": "w", "layers": [["a", "b"], ["c"]], "calls": 2}]
    rng = []
    t = 0
    for _ in range(2):
        rng.append(("saga_layer", t, t + 100))
        rng += [("saga stage 0", t + 5, t + 40), ("saga stage 1", t + 45, t + 95)]
        rng.append(("saga_layer", t + 200, t + 260))
        rng.append(("saga stage 0", t + 210, t + 250))
        t += 1000
    lay, acc = P.attribute_ranges(sorted(rng, key=lambda x: (x[1], -x[2])), sched)
    assert lay == {("w", 1): [100, 100], ("w", 2): [60, 60]}
    assert acc == {("w", 1, "a"): [35, 35], ("w", 1, "b"): [50, 50], ("w", 2, "c"): [40, 40]}
    bad = [r if r[1] != 45 else ("saga stage 1", 45, 150) for r in rng]  # stage outside its call
    with pytest.raises(ValueError):
        P.attribute_ranges(sorted(bad, key=lambda x: (x[1], -x[2])), sched)
    with pytest.raises(ValueError):
        P.attribute_ranges(sorted(rng, key=lambda x: (x[1], -x[2]))[:-2], sched)
