"""Pins of the cost-model oracle (Eq. 9-10) (no GPU)."""
import pytest

from oracle import cost


def test_window_is_clamped_at_zero():
    assert cost.window_us(100.0, 120.0) == 0.0
    assert cost.window_us(36800.0, 800.0) == 36000.0
    assert cost.swap_budget(100.0, 120.0, 5.0, 100.0, 10) == 0


def test_swap_cost_counts_both_experts():
    # moving 9 MB each way over a 153 GB/s link (153000 bytes/us) plus 10 us of launch overhead
    c = cost.swap_cost_us(10.0, 153000.0, 9_000_000, 9_000_000)
    assert c == pytest.approx(10.0 + 18_000_000 / 153000.0)
    assert cost.swap_cost_us(10.0, 153000.0, 9_000_000, 0) == pytest.approx(10.0 + 9_000_000 / 153000.0)


def test_budget_counts_whole_swaps():
    # window 1000 us, each swap 10 + 2*450/1 = 910 us -> exactly one swap; 1820 us -> two
    assert cost.swap_budget(1000.0, 0.0, 10.0, 1.0, 450) == 1
    assert cost.swap_budget(1830.0, 10.0, 10.0, 1.0, 450) == 2
    assert cost.swap_budget(1829.0, 10.0, 10.0, 1.0, 450) == 1


def test_budget_monotone():
    prev = -1
    for t in range(0, 40000, 500):
        b = cost.swap_budget(float(t), 300.0, 20.0, 100000.0, 9_000_000)
        assert b >= prev
        prev = b


def test_invalid_parameters():
    with pytest.raises(ValueError):
        cost.swap_cost_us(1.0, 0.0, 1, 1)
    with pytest.raises(ValueError):
        cost.swap_budget(10.0, 0.0, 0.0, 1.0, 0)
