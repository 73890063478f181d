"""Pins of the oracle's residual-carry mode (carry=True): every emitted
tensor keeps the consumers' view Y_hat (the sum of the deltas they
received); candidate rows emit e - Y_hat and truncated rows carry their
residual.  What fixes it, independently of its code:

* threshold 0: the same result as the drop semantics and as the dense
  forward (Eq. 2), up to f32 rounding (the carry forms each delta against
  the accumulated view, the drop semantics against the previous state);
* the carry bound: after every frame, at every site of every tensor,
  |e - Y_hat| <= threshold (a kept row leaves only the storage rounding of
  its delta, a truncated row's residual is what the threshold truncated,
  a site that is not a candidate has not moved);
* the drop semantics break that bound on the same video (the consumers'
  view, tracked from its kept rows, drifts away from e), so the bound
  is not met by accident;
* linearity of what the consumers see: every layer's state equals the
  dense convolution of its source's Y_hat (plus bias and the residual
  source's Y_hat), the committed input X_hat for the frame delta;
* a planted mistake (carry without the commit of kept deltas) fails."""

import numpy as np
import pytest

import oracle
from workloads import (crnn_vgg_net, depthwise_test_net,
                       efficientnet_mini_net, random_sparse_video,
                       resnet_mini_net, textline_video, toy_net, toy_video)


def cases():
    return [
        ("toy", toy_net(), toy_video(seed=5, n_frames=8)),
        ("resnet_mini", resnet_mini_net(),
         random_sparse_video(16, 8, 1, 32, 48, 3, 0.08)),
        ("dw", depthwise_test_net(),
         random_sparse_video(17, 7, 1, 24, 40, 16, 0.1)),
        ("crnn_small", crnn_vgg_net(H=16, W=32),
         textline_video(seed=2, n_frames=7, H=16, W=32, band=3)),
        ("effnet_mini", efficientnet_mini_net(),
         random_sparse_video(18, 6, 1, 32, 40, 3, 0.08)),
    ]


IDS = [c[0] for c in cases()]


def make(net, carry):
    return oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C,
                            net.dtype, carry=carry)


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-30))


@pytest.mark.parametrize("name,net,frames", cases(), ids=IDS)
def test_carry_at_threshold_zero(name, net, frames):
    r1, r2 = make(net, False), make(net, True)
    r1.encode_reference(frames[0])
    r2.encode_reference(frames[0])
    thr = [0.0] * (len(net.layers) + 1)
    for t in range(1, len(frames)):
        o1 = r1.encode_diff(frames[t], thr)
        o2 = r2.encode_diff(frames[t], thr)
        assert rel(o2, o1) < 1e-5, (name, t)
        dense, _, _ = oracle.dense_forward(net.layers, frames[t], net.dtype)
        assert rel(o2, dense) < 1e-5, (name, t)


def carry_gap(o, i):
    return float(np.abs(o.emitted(i).astype(np.float64)
                        - o.Y[i].astype(np.float64)).max())


@pytest.mark.parametrize("name,net,frames", cases(), ids=IDS)
def test_carry_bound(name, net, frames):
    thr_v = 0.05
    o = make(net, True)
    o.encode_reference(frames[0])
    thr = [thr_v] * (len(net.layers) + 1)
    for t in range(1, len(frames)):
        o.encode_diff(frames[t], thr)
        for i in range(len(net.layers)):
            scale = max(float(np.abs(o.emitted(i)).max()), 1.0)
            assert carry_gap(o, i) <= thr_v + 1e-6 * scale, (name, t, i)


def test_drop_semantics_break_the_bound():
    """The consumers' view under the drop semantics (reference activation
    plus every kept delta) drifts beyond the threshold on a longer video."""
    net = resnet_mini_net()
    frames = random_sparse_video(16, 8, 1, 32, 48, 3, 0.08)
    thr_v = 0.05
    o = make(net, False)
    o.encode_reference(frames[0])
    _, _, acts = oracle.dense_forward(net.layers, frames[0], "f32")
    view = {i: acts[i].reshape(-1, L.c_out).copy()
            for i, L in enumerate(net.layers)}
    worst = 0.0
    for t in range(1, len(frames)):
        o.encode_diff(frames[t], [thr_v] * (len(net.layers) + 1))
        for i, L in enumerate(net.layers):
            T = o.last["tensors"][i + 1]
            view[i][T["pix"]] += T["rows"]
            if o.stateful[i]:
                e = oracle.sparsetem_oracle.activation(o.P[i], L.act)
                if L.pool_k[0] > 0:
                    e = oracle.maxpool_nhwc(np.asarray(e, np.float64),
                                            L.pool_k, L.pool_s, L.pool_p)
                gap = np.abs(np.asarray(e, np.float64).reshape(-1, L.c_out)
                             - view[i]).max()
                worst = max(worst, float(gap))
    assert worst > 2 * thr_v, worst


def dense_state_from_views(o, i):
    """f32 dense convolution of what layer i's consumers-side inputs are:
    its source's Y_hat (X_hat for the input), plus bias, plus the residual
    source's Y_hat."""
    L = o.layers[i]
    shape = o.shapes[L.src]
    x = (o.xhat if L.src == -1 else o.Y[L.src]).reshape(shape)
    a = oracle.conv2d_nhwc(np.asarray(x, np.float64), L.weight, L.bias, L.s,
                           L.p, L.groups)
    if L.residual_src != -2:
        a = a + o.Y[L.residual_src].reshape(a.shape)
    return a


@pytest.mark.parametrize("name,net,frames", cases(), ids=IDS)
def test_state_is_dense_conv_of_consumers_view(name, net, frames):
    o = make(net, True)
    o.encode_reference(frames[0])
    for t in range(1, len(frames)):
        o.encode_diff(frames[t], [0.05] * (len(net.layers) + 1))
        for i in range(len(net.layers)):
            P = o.P[i].reshape(-1)
            D = dense_state_from_views(o, i).reshape(-1)
            assert rel(P, D) < 1e-5, (name, t, i, rel(P, D))


def test_planted_mistake_no_commit_is_caught():
    """Carry without adding the kept deltas to Y_hat (planted by restoring
    the view from before a frame): the consumers' view no longer matches
    what the state was built from, and the linearity pin fails."""
    net = resnet_mini_net()
    frames = random_sparse_video(16, 4, 1, 32, 48, 3, 0.08)
    o = make(net, True)
    o.encode_reference(frames[0])
    before = {i: y.copy() for i, y in o.Y.items()}
    o.encode_diff(frames[1], [0.05] * (len(net.layers) + 1))
    o.Y = before
    bad = max(rel(o.P[i].reshape(-1), dense_state_from_views(o, i)
                  .reshape(-1)) for i in range(1, len(net.layers)))
    assert bad > 1e-3, bad
