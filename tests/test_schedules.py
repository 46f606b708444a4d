"""Schedules of the paper: values the appendix and the training protocol fix."""
import pytest

from paper_2608_05088_amd.schedules import geometric, lambda_lr, linear_warmup, wsd


def test_wsd_appendix_schedule():
    # Appendix B: warm up to eta_max over 500 iterations, hold for 3500, decay to 0 over 1000.
    f = wsd(500, 3500, 1000)
    eta = [1e-3 * f(t) for t in range(1, 5001)]
    assert eta[0] == pytest.approx(1e-3 / 500)
    assert eta[499] == pytest.approx(1e-3)              # t = 500: peak reached
    assert all(e == 1e-3 for e in eta[500:4000])        # t = 501 .. 4000: stable
    assert eta[4499] == pytest.approx(0.5e-3)           # half-way down the decay
    assert eta[4999] == 0.0                             # t = 5000: eta_min
    assert all(a <= b for a, b in zip(eta[:500], eta[1:501]))
    assert all(a >= b for a, b in zip(eta[4000:-1], eta[4001:]))
    # Area under the trapezoid: 500/2 + 3500 + 1000/2 iterations at eta_max (sums of arithmetic series).
    assert sum(f(t) for t in range(1, 5001)) == pytest.approx(250.5 + 3500 + 499.5)


def test_linear_warmup_first_ten_percent():
    f = linear_warmup(10_000)
    assert f(1) == pytest.approx(1e-3)
    assert f(1000) == 1.0 and f(1001) == 1.0 and f(10_000) == 1.0
    assert f(500) == pytest.approx(0.5)


def test_geometric_staircase():
    f = geometric(50, 0.5)
    assert [f(t) for t in (1, 50, 51, 100, 101, 151)] == [1.0, 1.0, 0.5, 0.5, 0.25, 0.125]


def test_invalid_arguments():
    with pytest.raises(ValueError):
        wsd(-1, 1, 1)
    with pytest.raises(ValueError):
        geometric(0, 0.5)
    with pytest.raises(ValueError):
        linear_warmup(0)
    with pytest.raises(ValueError):
        wsd(1, 1, 1)(0)


def test_lambda_lr_drives_the_adapter_rates():
    import torch
    from paper_2608_05088_amd.optim import MALT
    w = torch.zeros(4, 4, requires_grad=True)
    b = torch.zeros(4, requires_grad=True)
    opt = MALT([w, b], lr=1e-3, adamw_lr=4e-4)
    sched = lambda_lr(opt, wsd(2, 1, 2))
    seen = []
    for _ in range(6):
        seen.append(opt.param_groups[0]["lr"])
        sched.step()
    assert seen == pytest.approx([5e-4, 1e-3, 1e-3, 5e-4, 0.0, 0.0])
