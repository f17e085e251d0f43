"""Budget schedules (host logic, no GPU)."""
import pytest

from paper_2606_14782_amd import budgets


@pytest.mark.parametrize("mean,L,ratio", [(256, 32, 0.25), (64, 28, 0.1), (128, 32, 1.0),
                                          (3, 40, 0.05), (1, 5, 0.5), (100, 1, 0.25)])
def test_pyramid_schedule(mean, L, ratio):
    k = budgets.pyramid(mean, L, ratio)
    assert len(k) == L
    assert sum(k) == mean * L                      # same total as the uniform budget
    assert min(k) >= 1
    assert all(a >= b for a, b in zip(k, k[1:]))   # shrinks with depth
    if ratio == 1.0:
        assert k == budgets.uniform(mean, L)
    elif L > 1 and mean >= 16:
        assert abs(k[-1] / k[0] - ratio) < 0.05 + 2.0 / k[0]


def test_schedule_arguments():
    with pytest.raises(ValueError):
        budgets.pyramid(0, 4)
    with pytest.raises(ValueError):
        budgets.pyramid(10, 4, ratio=0.0)
    with pytest.raises(ValueError):
        budgets.uniform(5, 0)
