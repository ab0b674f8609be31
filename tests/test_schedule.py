"""Host-side schedules (CPU): when SET runs and the auxiliary loss weight."""
import pytest

from paper_2411_03171_amd import schedule


def test_set_due_stops_at_two_thirds():
    # 1000 steps, SET every 100: after steps 100..600 (660 is the last step allowed)
    due = [t for t in range(1, 1001) if schedule.set_due(t, 100, 1000)]
    assert due == [100, 200, 300, 400, 500, 600]
    # the stop is inclusive: 66 of 100 steps, interval 33 -> steps 33 and 66
    assert [t for t in range(1, 101) if schedule.set_due(t, 33, 100)] == [33, 66]
    assert not schedule.set_due(0, 10, 100)
    assert not schedule.set_due(10, 0, 100)
    # a different stop fraction
    assert [t for t in range(1, 101) if schedule.set_due(t, 20, 100, stop_frac=1.0)] == [20, 40, 60, 80, 100]


def test_set_round_counts_updates():
    assert [schedule.set_round(t, 20) for t in (20, 40, 60)] == [1, 2, 3]


@pytest.mark.parametrize("epoch,expected", [(0, 1.0), (2, 0.75), (4, 0.5), (7.2, 0.1), (8, 0.0), (30, 0.0)])
def test_aux_weight_linear_decay(epoch, expected):
    assert schedule.aux_weight(epoch, 1.0, 8) == pytest.approx(expected, abs=1e-12)


def test_aux_weight_special_cutoffs():
    assert schedule.aux_weight(100, 0.5, None) == 0.5        # no cut-off: full training
    assert schedule.aux_weight(0, 0.5, 0) == 0.0             # cut-off 0: no auxiliary loss
    assert schedule.aux_weight(-1, 2.0, 10) == 2.0           # before the first epoch
    ws = [schedule.aux_weight(e / 10, 1.0, 15) for e in range(200)]
    assert all(a >= b for a, b in zip(ws, ws[1:]))           # never increases
