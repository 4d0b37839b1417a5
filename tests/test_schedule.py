"""Host logic of the Monte Carlo schedule (Sec. IV-B with the constants of
Sec. IV-D).  CPU only."""
import pytest

from paper_2210_10108_amd.driver import MCSchedule, PAPER_SCHEDULE


def test_paper_schedule_constants():
    s = PAPER_SCHEDULE
    assert (s.n_hypotheses, s.s1, s.s2, s.rounds, s.keep_frac) == (64, 512, 512, 4, 0.25)
    assert s.total_steps == 2560                      # s1 + S s2
    rounds = {k: s.resample_round(k) for k in range(s.total_steps + 1) if s.resample_round(k)}
    assert rounds == {512: 1, 1024: 2, 1536: 3, 2048: 4}
    # r = 0.25 halved every round: 16, 8, 4 and 2 of the 64 hypotheses survive
    assert [s.keep_fraction(j) for j in (1, 2, 3, 4)] == [0.25, 0.125, 0.0625, 0.03125]
    assert [s.n_keep(j) for j in (1, 2, 3, 4)] == [16, 8, 4, 2]


def test_schedule_edges():
    s = MCSchedule(n_hypotheses=5, s1=3, s2=2, rounds=3, keep_frac=0.5)
    assert s.total_steps == 9
    assert [s.resample_round(k) for k in range(11)] == [0, 0, 0, 1, 0, 2, 0, 3, 0, 0, 0]
    assert [s.n_keep(j) for j in (1, 2, 3)] == [2, 1, 1]   # never below one
    assert MCSchedule(rounds=0).total_steps == 512
    assert all(MCSchedule(rounds=0).resample_round(k) == 0 for k in range(600))
    for bad in (dict(s1=0), dict(s2=0), dict(n_hypotheses=0), dict(keep_frac=1.5),
                dict(rounds=-1)):
        with pytest.raises(ValueError):
            MCSchedule(**bad)
