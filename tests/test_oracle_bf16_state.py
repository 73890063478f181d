"""Pins of the oracle's bf16-state mode (an approximation: every stored
pre-activation is rounded to bf16, nearest with ties to even, before the
activation sees it).  What fixes it, independently of the oracle's own
arithmetic:

* every stored state value is a bf16 value (the low 16 bits of its f32
  pattern are zero);
* a frame equal to the previous one changes nothing, bit for bit;
* against the plain definition: the first layer's state after t diff frames
  at threshold 0 is the dense pre-activation of frame t (torch's conv2d)
  up to one bf16 rounding per update (relative 2^-8 of the magnitude each);
* the consumers' sum of a layer's emitted deltas over the frames equals f
  of the stored final state minus f of the stored reference state (the
  deltas are formed from the stored, rounded values), within f32 rounding
  of each delta;
* max-pooled nets and residual carry are refused."""

import numpy as np
import pytest
import torch

import oracle
from oracle import sparsetem_oracle as so
from workloads import (efficientnet_mini_net, random_sparse_video,
                       resnet_mini_net, toy_net, toy_video)


def is_bf16(x):
    u = np.ascontiguousarray(np.asarray(x, np.float32)).view(np.uint32)
    return bool(np.all((u & 0xFFFF) == 0))


def test_state_is_bf16_representable():
    net = efficientnet_mini_net()
    o = oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C, "f32",
                         state_bf16=True)
    frames = random_sparse_video(31, 4, 1, net.H, net.W, net.C, 0.1)
    o.encode_reference(frames[0])
    for i in o.P:
        assert is_bf16(o.P[i]), f"reference state {i}"
    for f in frames[1:]:
        o.encode_diff(f, [0.0] * (len(net.layers) + 1))
        for i in o.P:
            assert is_bf16(o.P[i]), f"state {i}"
    # and the exact mode's state is not (the rounding is what differs)
    e = oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C, "f32")
    e.encode_reference(frames[0])
    assert not all(is_bf16(p) for p in e.P.values())


def test_zero_delta_changes_nothing():
    net = toy_net()
    frames = toy_video(seed=5, n_frames=2)
    o = oracle.OracleNet(net.layers, 1, 64, 64, 16, "f32", state_bf16=True)
    o.encode_reference(frames[0])
    o.encode_diff(frames[1], [0.0] * 3)
    P = {i: p.copy() for i, p in o.P.items()}
    out0 = o.last["out"].copy()
    out = o.encode_diff(frames[1], [0.0] * 3)
    for i in P:
        assert np.array_equal(P[i].view(np.uint32), o.P[i].view(np.uint32))
    assert np.array_equal(np.asarray(out, np.float32).view(np.uint32),
                          np.asarray(out0, np.float32).view(np.uint32))
    assert all(len(T["pix"]) == 0 for T in o.last["tensors"])


def torch_preact(frame, L):
    """Dense pre-activation of one conv layer on an NHWC frame, from
    torch's conv2d in float64."""
    x = torch.from_numpy(np.asarray(frame, np.float64)).permute(0, 3, 1, 2)
    w = torch.from_numpy(np.asarray(L.weight, np.float64))
    b = torch.from_numpy(np.asarray(L.bias, np.float64))
    y = torch.nn.functional.conv2d(x, w, b, stride=L.s, padding=L.p,
                                   groups=L.groups)
    return y.permute(0, 2, 3, 1).numpy()


def test_first_layer_within_one_rounding_per_update():
    net = toy_net()
    frames = toy_video(seed=6, n_frames=6)
    o = oracle.OracleNet(net.layers, 1, 64, 64, 16, "f32", state_bf16=True)
    o.encode_reference(frames[0])
    L = net.layers[0]
    worst = 0.0
    for t in range(1, len(frames)):
        o.encode_diff(frames[t], [0.0] * 3)
        exact = torch_preact(frames[t], L)
        got = o.P[0].reshape(exact.shape).astype(np.float64)
        scale = np.abs(exact).max()
        err = np.abs(got - exact).max()
        assert err <= (t + 1) * 2.0 ** -8 * scale + 1e-5 * scale, (t, err)
        worst = max(worst, err / scale)
    # the rounding is visible: bf16-sized, not f32-sized, deviations
    assert worst > 1e-4


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_emitted_deltas_telescope_to_stored_state(dtype):
    """Layer 0 of the toy net (ReLU, 16 channels): reference activation
    plus every frame's emitted delta rows equals f of the stored state."""
    net = toy_net(dtype=dtype)
    frames = toy_video(seed=7, n_frames=6)
    o = oracle.OracleNet(net.layers, 1, 64, 64, 16, dtype, state_bf16=True)
    o.encode_reference(frames[0])
    view = so.round_storage(np.maximum(o.P[0].astype(np.float64), 0.0),
                            dtype).reshape(-1, 16)
    n_rows = 0
    for f in frames[1:]:
        o.encode_diff(f, [0.0] * 3)
        T = o.last["tensors"][1]
        view[T["pix"]] += T["rows"]
        n_rows += len(T["pix"])
    assert n_rows > 0
    final = np.maximum(o.P[0].astype(np.float64), 0.0).reshape(-1, 16)
    scale = np.abs(final).max()
    # each delta is rounded once to the storage dtype (f32: 2^-24, bf16:
    # 2^-9 relative); five frames
    eps = 2.0 ** -24 if dtype == "f32" else 2.0 ** -9
    assert np.abs(view - final).max() <= 6 * eps * 2 * scale + 1e-7 * scale


def test_refused_with_pools_or_carry():
    net = resnet_mini_net()          # 3x3/2 max-pool after the stem
    with pytest.raises(ValueError):
        oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C, "f32",
                         state_bf16=True)
    t = toy_net()
    with pytest.raises(ValueError):
        oracle.OracleNet(t.layers, 1, 64, 64, 16, "f32", carry=True,
                         state_bf16=True)
