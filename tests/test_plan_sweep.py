"""Host side of the planner-regret tool (no GPU): its step set and the
forced key splits and unit sizes it tries."""
from paper_2607_02043_amd import plan_sweep as P


def test_steps_are_distinct_and_cover_the_benchmark():
    s = P.steps()
    names = [x[0] for x in s]
    assert len(names) == len(set(names)) == 79
    assert {"workload 2", "workload 3", "workload 5", "workload 4 C=4096"} <= set(names)
    for _, prefix, q, page in s:
        assert len(prefix) == len(q) and page == 64 and all(c >= 1 for c in q)


def test_forced_values_stay_inside_the_step():
    prefix, q = [998] * 4 + [372], [1] * 4 + [124]
    assert P.key_splits(prefix, q) == [64, 128, 256, 16320]  # below the chunk's 496 keys, and unsplit
    u = P.unit_sizes(prefix, q)
    assert u[0] == 1 and max(u) <= 4 * 32 and len(u) == len(set(u))
    assert P.unit_sizes([0, 500], [300, 200]) == [0]  # no decode rows
    assert P.key_splits([5, 6], [1, 1]) == [16320]  # no chunk
