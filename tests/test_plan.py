"""Eq. 2 against hand-worked values, and microbatch planning."""
import os

import pytest

from paper_2608_01891_amd import plan

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "eq2_layer_time.txt")


def _rows():
    with open(GOLDEN) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                ta, tf, tc, m, t = line.split()
                yield float(ta), float(tf), float(tc), int(m), float(t)


@pytest.mark.parametrize("ta,tf,tc,M,t", list(_rows()))
def test_eq2_golden(ta, tf, tc, M, t):
    assert plan.eq2_layer_time(ta, tf, tc, M) == pytest.approx(t, abs=1e-12)


def test_eq2_rejects_zero_depth():
    with pytest.raises(ValueError):
        plan.eq2_layer_time(1, 1, 1, 0)


def test_equal_microbatches():
    assert plan.equal_microbatches(256, 4) == [64, 64, 64, 64]
    assert plan.equal_microbatches(10, 3) == [4, 3, 3]
    with pytest.raises(ValueError):
        plan.equal_microbatches(2, 3)


def test_candidate_splits_are_partitions():
    c = plan.candidate_splits(384)
    assert [384] in c and [192, 192] in c and [96, 96, 96, 96] in c
    assert [128, 256] in c and [256, 128] in c  # the paper's adaptive 128+256 example
    for s in c:
        assert sum(s) == 384 and all(n >= 1 for n in s)
    assert len({tuple(s) for s in c}) == len(c)
    assert plan.candidate_splits(2, depths=(1, 2, 4)) == [[2], [1, 1]]


def test_eq2_predict_reduces_to_eq2():
    t_a = lambda n: 0.01 * n
    t_f = lambda n: 2.0 + 0.005 * n
    assert plan.eq2_predict([100], t_a, t_f, 0.5) == pytest.approx(1.0 + 2.5 + 0.5)
    # M = 2: max(sum t_A, sum t_F) + t_comm / 2
    assert plan.eq2_predict([50, 50], t_a, t_f, 0.5) == pytest.approx(max(1.0, 4.5) + 0.25)


def test_choose_split_picks_the_minimum():
    t_a = lambda n: 0.5 + 0.02 * n    # attention: launch cost plus KV bytes of n sequences
    t_f = lambda n: 1.5 + 0.002 * n   # FFN dominated by streaming the weights once per microbatch
    c = plan.candidate_splits(384)
    best, cost = plan.choose_split(c, lambda s: plan.eq2_predict(s, t_a, t_f))
    assert cost == min(plan.eq2_predict(s, t_a, t_f) for s in c)
    # M=1 pays t_A + t_F, M=4 pays four attention launches: M=2 wins strictly
    assert len(best) == 2
    assert cost < plan.eq2_predict([384], t_a, t_f) and cost < plan.eq2_predict([96] * 4, t_a, t_f)
