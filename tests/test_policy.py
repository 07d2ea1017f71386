"""Timestep policy (first 20 % of the denoising steps dense, Sec. 4 setup): host logic."""
import pytest

from paper_2609_37001_amd.policy import TimestepPolicy


@pytest.mark.parametrize("total,frac,dense", [(50, 0.2, 10), (30, 0.2, 6), (33, 0.2, 7), (1, 0.2, 1),
                                               (50, 0.0, 0), (50, 1.0, 50), (10, 0.25, 3)])
def test_dense_step_counts(total, frac, dense):
    p = TimestepPolicy(total, frac)
    assert p.dense_steps == dense
    assert [p.is_dense(s) for s in range(total)] == [True] * dense + [False] * (total - dense)


def test_invalid_arguments():
    with pytest.raises(ValueError):
        TimestepPolicy(0)
    with pytest.raises(ValueError):
        TimestepPolicy(10, 1.5)
    with pytest.raises(ValueError):
        TimestepPolicy(10).is_dense(10)
