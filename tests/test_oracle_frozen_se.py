"""Pins of the oracle's frozen squeeze-excitation mode (an approximation,
flagged as inexact): the reference frame's gates are kept for the chunk's
diff frames.  What fixes it:

* threshold 0: the output equals a dense forward of the frame whose
  squeeze-excitation layers apply the reference frame's gates (Eq. 2 with
  a fixed per-channel scale);
* a net without squeeze-excitation encodes exactly as without the flag;
* it is an approximation: away from the reference frame the output leaves
  the exact dense forward (whose gates follow every frame)."""

import numpy as np

import oracle
from oracle import sparsetem_oracle as so
from workloads import (efficientnet_mini_net, random_sparse_video,
                       resnet_mini_net)


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-30))


def dense_with_gates(layers, frame, dtype, gates):
    """Dense forward of one frame with the squeeze-excitation gates fixed
    to `gates[i]` (written from the layer definitions, as dense_forward)."""
    acts = {-1: so.round_storage(frame, dtype)}
    out = None
    for i, L in enumerate(layers):
        a = so.conv2d_nhwc(acts[L.src], L.weight, L.bias, L.s, L.p, L.groups)
        if L.residual_src != -2:
            a = a + acts[L.residual_src]
        p32 = so.f32(a)
        stateful = (L.act != so.ACT_NONE or L.pool_k[0] > 0 or L.se_mid
                    or i == len(layers) - 1)
        e32 = p32
        if stateful:
            e32 = so.f32(so.activation(p32, L.act).astype(np.float64))
            if L.pool_k[0] > 0:
                e32 = so.f32(so.maxpool_nhwc(e32, L.pool_k, L.pool_s,
                                             L.pool_p))
            if L.se_mid:
                e32 = so.se_apply(e32, gates[i])
        acts[i] = so.round_storage(e32, dtype)
        if i == len(layers) - 1:
            out = e32
    return out


def test_frozen_se_at_threshold_zero():
    net = efficientnet_mini_net()
    frames = random_sparse_video(21, 5, 1, 32, 40, 3, 0.08)
    o = oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C,
                         net.dtype, frozen_se=True)
    o.encode_reference(frames[0])
    gates = {i: g.copy() for i, g in o.S.items()}
    assert gates, "the net has squeeze-excitation layers"
    thr = [0.0] * (len(net.layers) + 1)
    for t in range(1, len(frames)):
        out = o.encode_diff(frames[t], thr)
        ref = dense_with_gates(net.layers, frames[t], net.dtype, gates)
        assert rel(out, ref) < 1e-5, (t, rel(out, ref))
        for i in gates:
            np.testing.assert_array_equal(o.S[i], gates[i])


def test_frozen_se_without_se_is_exact():
    net = resnet_mini_net()
    frames = random_sparse_video(22, 4, 1, 32, 48, 3, 0.08)
    a = oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C, "f32")
    b = oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C, "f32",
                         frozen_se=True)
    a.encode_reference(frames[0])
    b.encode_reference(frames[0])
    thr = [0.05] * (len(net.layers) + 1)
    for t in range(1, len(frames)):
        np.testing.assert_array_equal(a.encode_diff(frames[t], thr),
                                      b.encode_diff(frames[t], thr))


def test_frozen_se_is_an_approximation():
    net = efficientnet_mini_net()
    frames = random_sparse_video(23, 5, 1, 32, 40, 3, 0.15)
    o = oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C,
                         net.dtype, frozen_se=True)
    o.encode_reference(frames[0])
    thr = [0.0] * (len(net.layers) + 1)
    worst = 0.0
    for t in range(1, len(frames)):
        out = o.encode_diff(frames[t], thr)
        dense, _, _ = oracle.dense_forward(net.layers, frames[t], net.dtype)
        worst = max(worst, rel(out, dense))
    assert worst > 1e-4, worst
