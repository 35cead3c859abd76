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
