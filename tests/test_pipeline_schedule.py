"""The 1F1B schedule the first-stage measurement replays (Sec. 3.2.2): pinned
by its defining properties, checked for every small (stages, stage, micro-batches)."""
import pytest

from paper_2411_06465_amd.pipeline import one_f_one_b


def in_flight_peak(ops):
    live, peak = 0, 0
    for op, _ in ops:
        live += 1 if op == "F" else -1
        peak = max(peak, live)
    return peak


@pytest.mark.parametrize("stages", [1, 2, 3, 4, 8])
@pytest.mark.parametrize("m", [1, 2, 3, 5, 8, 13])
def test_schedule_properties(stages, m):
    for stage in range(stages):
        ops = one_f_one_b(stage, stages, m)
        assert sorted(ops) == sorted([("F", i) for i in range(m)] + [("B", i) for i in range(m)])
        pos = {op: k for k, op in enumerate(ops)}
        for i in range(m):
            assert pos[("F", i)] < pos[("B", i)]
            if i:
                assert pos[("F", i - 1)] < pos[("F", i)] and pos[("B", i - 1)] < pos[("B", i)]
        # stage s holds at most p - s micro-batches: the first stage p, the last one
        assert in_flight_peak(ops) == min(stages - stage, m)
        # after the warm-up, forwards and backwards alternate
        warm = min(stages - stage - 1, m)
        steady = ops[warm:warm + 2 * (m - warm)]
        assert [op for op, _ in steady] == ["F", "B"] * (m - warm)


def test_first_stage_of_the_70b_layout():
    # (t, c, p) = (8, 1, 8), 80 layers: stage 0 runs 7 warm-up forwards, then
    # holds 8 micro-batches of its 10 layers: 80 layer stashes
    ops = one_f_one_b(0, 8, 8)
    assert ops[:8] == [("F", i) for i in range(8)] and ops[8] == ("B", 0)
    assert in_flight_peak(ops) * (80 // 8) == 80


def test_bad_arguments():
    for args in [(2, 2, 4), (-1, 2, 4), (0, 2, 0)]:
        with pytest.raises(ValueError):
            one_f_one_b(*args)
