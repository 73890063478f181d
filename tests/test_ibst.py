"""Host tests of the online threshold controller (iterative binary search
for the truncation threshold).  The pins are properties of bisection on a
monotone curve, with the band's threshold interval from a closed form:
for s(theta) = 1 - exp(-theta / tau) the band [T - eps, T + eps] is
theta in [-tau ln(1 - T + eps), -tau ln(1 - T - eps)]."""

import math

import numpy as np
import pytest

from paper_2410_20790_amd.ibst import (IBST, nonlinear_tensors,
                                       sparsity_from_counts)
from workloads import (crnn_vgg_net, efficientnet_mini_net, resnet_mini_net,
                       toy_net)

T, EPS, TMAX = 0.9, 0.025, 1.0


def exp_curve(tau):
    return lambda th: 1.0 - math.exp(-th / tau)


def exp_band(tau, t=T, eps=EPS):
    return (-tau * math.log(1.0 - t + eps), -tau * math.log(1.0 - t - eps))


def logistic_curve(mid, k):
    return lambda th: 1.0 / (1.0 + math.exp(-(th - mid) * k))


def logistic_band(mid, k, t=T, eps=EPS):
    inv = lambda s: mid + math.log(s / (1.0 - s)) / k  # noqa: E731
    return inv(t - eps), inv(t + eps)


def run_cycle(c, curve, frames, tensor=1, n=3):
    """Frames of one cycle on one controlled tensor; returns the
    thresholds each frame ran with."""
    used = []
    for _ in range(frames):
        th = c.thresholds()[tensor]
        used.append(th)
        s = np.zeros(n)
        s[tensor] = curve(th)
        c.update(s)
    return used


CURVES = [
    ("exp tau=0.05", exp_curve(0.05), exp_band(0.05)),
    ("exp tau=0.3", exp_curve(0.3), exp_band(0.3)),
    ("exp tau=0.02", exp_curve(0.02), exp_band(0.02)),
    ("logistic steep", logistic_curve(0.7, 60.0), logistic_band(0.7, 60.0)),
    ("logistic low", logistic_curve(0.013, 900.0),
     logistic_band(0.013, 900.0)),
]


@pytest.mark.parametrize("name,curve,band", CURVES, ids=[c[0] for c in CURVES])
def test_converges_within_bisection_bound(name, curve, band):
    a, b = band
    assert 0.0 < a < b < TMAX
    bound = math.ceil(math.log2(TMAX / (b - a))) + 1
    c = IBST(3, [1], T, EPS, TMAX)
    used = run_cycle(c, curve, bound + 10)
    first = next(i for i, th in enumerate(used) if a <= th <= b)
    assert first + 1 <= bound, (first, bound)
    # once inside the band the threshold no longer moves
    assert all(th == used[first] for th in used[first:])
    assert T - EPS <= curve(used[first]) <= T + EPS


@pytest.mark.parametrize("name,curve,band", CURVES, ids=[c[0] for c in CURVES])
def test_bracket_keeps_the_band(name, curve, band):
    a, b = band
    c = IBST(3, [1], T, EPS, TMAX)
    for _ in range(30):
        assert c.lo[1] <= a and b <= c.hi[1]
        assert c.lo[1] <= c.theta[1] <= c.hi[1]
        s = np.zeros(3)
        s[1] = curve(c.theta[1])
        c.update(s)


def test_bisection_points_are_dyadic():
    """Each out-of-band step halves the bracket: after k steps from
    theta_max / 2 the threshold is an odd multiple of theta_max / 2^(k+1)."""
    curve = exp_curve(0.004)  # band far below theta_max / 2
    c = IBST(3, [1], T, EPS, TMAX)
    used = run_cycle(c, curve, 6)
    for k, th in enumerate(used):
        m = th * 2 ** (k + 1) / TMAX
        assert m == int(m) and int(m) % 2 == 1, (k, th)
    assert used == sorted(used, reverse=True)  # too sparse: always lower


def test_cycles_follow_a_moving_curve():
    """Between chunks the sparsity curve moves (other content).  A restarted
    bracket finds the new band within the bound; one search that is never
    restarted has collapsed its bracket and cannot."""
    first, second = exp_curve(0.02), exp_curve(0.25)
    a2, b2 = exp_band(0.25)
    bound = math.ceil(math.log2(TMAX / (b2 - a2))) + 1

    ibst = IBST(3, [1], T, EPS, TMAX)
    run_cycle(ibst, first, 12)
    ibst.start_cycle()
    used = run_cycle(ibst, second, bound)
    assert any(a2 <= th <= b2 for th in used)

    bst = IBST(3, [1], T, EPS, TMAX)
    run_cycle(bst, first, 12)
    used = run_cycle(bst, second, 12)
    assert not any(a2 <= th <= b2 for th in used)


def test_uncontrolled_tensors_keep_their_threshold():
    c = IBST(4, [0, 2], fixed=0.01)
    assert c.thresholds() == [0.5, 0.01, 0.5, 0.01]
    c.update([0.0, 0.0, 1.0, 1.0])
    assert c.thresholds() == [0.75, 0.01, 0.25, 0.01]
    c.update([0.9, 0.9, 0.9, 0.9])  # in band: unchanged
    assert c.thresholds() == [0.75, 0.01, 0.25, 0.01]


def test_argument_checks():
    with pytest.raises(ValueError):
        IBST(3, [3])
    with pytest.raises(ValueError):
        IBST(3, [1], target=1.5)
    c = IBST(3, [1])
    with pytest.raises(ValueError):
        c.update([0.5, 0.5])


def test_sparsity_from_counts():
    s = sparsity_from_counts([10, 0, 64], [100, 50, 64])
    np.testing.assert_array_equal(s, [0.9, 1.0, 0.0])


def test_nonlinear_tensors():
    # toy: conv+ReLU, conv (linear output)
    assert nonlinear_tensors(toy_net().layers) == [0, 1]
    assert nonlinear_tensors(toy_net().layers, include_input=False) == [1]
    # every CRNN conv has ReLU
    crnn = crnn_vgg_net()
    assert nonlinear_tensors(crnn.layers) == list(range(len(crnn.layers) + 1))
    # ResNet: the downsample 1x1 and the last conv of a branch are linear
    # before the add only when they carry no activation
    res = resnet_mini_net()
    exp = [0] + [j + 1 for j, L in enumerate(res.layers) if L.act != 0]
    assert nonlinear_tensors(res.layers) == exp
    # EfficientNet: linear projections are left out, SE layers are in
    eff = efficientnet_mini_net()
    got = nonlinear_tensors(eff.layers)
    for j, L in enumerate(eff.layers):
        assert ((j + 1) in got) == (L.act != 0 or L.se_mid > 0)
