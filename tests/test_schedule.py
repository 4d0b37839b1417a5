"""Host logic of the Monte Carlo schedule (Sec. IV-B with the constants of
Sec. IV-D).  CPU only."""
import pytest

from paper_2210_10108_amd.driver import MCSchedule, PAPER_SCHEDULE


def golden():
    """tests/golden/schedule_sec4d.txt: name -> values."""
    import os
    out = {}
    path = os.path.join(os.path.dirname(__file__), "golden", "schedule_sec4d.txt")
    for line in open(path):
        if line.strip() and not line.startswith("#"):
            name, *vals = line.split()
            out[name] = [float(v) for v in vals]
    return out


def test_paper_schedule_constants():
    g = golden()
    s = PAPER_SCHEDULE
    assert (s.n_hypotheses, s.s1, s.s2, s.rounds, s.keep_frac) == (
        g["hypotheses"][0], g["first_stage_steps"][0], g["stage_steps"][0],
        g["resampling_rounds"][0], g["keep_fraction"][0])
    assert s.total_steps == g["total_steps"][0]      # s1 + S s2
    rounds = {k: s.resample_round(k) for k in range(s.total_steps + 1) if s.resample_round(k)}
    assert sorted(rounds) == g["round_after_step"] and list(rounds.values()) == [1, 2, 3, 4]
    # r halved every round: the kept counts of the fixture
    assert [s.keep_fraction(j) for j in (1, 2, 3, 4)] == [0.25, 0.125, 0.0625, 0.03125]
    assert [s.n_keep(j) for j in (1, 2, 3, 4)] == g["kept"]


def test_paper_learning_rates():
    from paper_2210_10108_amd.pnerf import AdamParams
    g = golden()
    a = AdamParams()
    assert a.lr_rot == pytest.approx(g["lr_rotation"][0])
    assert a.lr_trans == pytest.approx(g["lr_translation"][0])
    assert a.decay_base == pytest.approx(g["lr_decay_base"][0])
    assert a.decay_steps == g["lr_decay_steps"][0]


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
