"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test ties the oracle to something other than itself: a library routine
(PyTorch conv2d / max_pool2d / dtype conversion), the paper's worked
example of dense amplification, closed forms, brute-force enumeration,
the linearity invariant of Eq. 2 (threshold 0 reproduces the dense forward),
the zero-delta invariant, an independent dense-tensor simulation of the
truncation semantics, and an error bound for the first layer.  A planted
mistake in the oracle (last tests) must make a pin fail.
"""

import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import sparsetem_oracle as so
from workloads import (ACT_NONE, ACT_RELU, ACT_SILU, LayerSpec, crnn_vgg_net,
                       depthwise_test_net, efficientnet_mini_net,
                       random_sparse_video, resnet_mini_net, textline_video,
                       toy_net, toy_video)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rel_err(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-30))


def torch_conv_nhwc(x, w, b, s, p, g):
    xt = torch.from_numpy(np.asarray(x, np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(np.asarray(w, np.float64))
    bt = None if b is None else torch.from_numpy(np.asarray(b, np.float64))
    return F.conv2d(xt, wt, bt, stride=s, padding=p,
                    groups=g).permute(0, 2, 3, 1).numpy()


# ------------------------------------------------------ library routines

@pytest.mark.parametrize("cfg", [
    # N, H, W, Cin, Cout, k, s, p, groups
    (1, 9, 11, 3, 5, (3, 3), (1, 1), (1, 1), 1),
    (2, 10, 7, 4, 6, (3, 3), (2, 2), (1, 1), 1),
    (1, 13, 17, 3, 8, (7, 7), (2, 2), (3, 3), 1),
    (1, 8, 8, 6, 6, (5, 5), (2, 2), (2, 2), 6),
    (1, 6, 9, 8, 8, (3, 3), (1, 1), (1, 1), 8),
    (1, 5, 6, 4, 8, (1, 1), (2, 2), (0, 0), 1),
    (1, 6, 6, 4, 6, (3, 3), (1, 1), (0, 0), 2),
    (1, 7, 5, 2, 3, (2, 3), (1, 2), (1, 0), 1),
])
def test_dense_conv_matches_torch(cfg):
    N, H, W, Cin, Cout, k, s, p, g = cfg
    rng = np.random.default_rng(1)
    x = rng.standard_normal((N, H, W, Cin))
    w = rng.standard_normal((Cout, Cin // g, *k))
    b = rng.standard_normal(Cout)
    ours = oracle.conv2d_nhwc(x, w, b, s, p, g)
    ref = torch_conv_nhwc(x, w, b, s, p, g)
    assert ours.shape == ref.shape
    np.testing.assert_allclose(ours, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("k,s,p", [((2, 2), (2, 2), (0, 0)),
                                   ((2, 1), (2, 1), (0, 0)),
                                   ((3, 3), (2, 2), (1, 1)),
                                   ((3, 2), (1, 2), (1, 0))])
def test_maxpool_matches_torch(k, s, p):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 9, 10, 3))
    ours = oracle.maxpool_nhwc(x, k, s, p)
    ref = F.max_pool2d(torch.from_numpy(x).permute(0, 3, 1, 2), k, s,
                       p).permute(0, 2, 3, 1).numpy()
    np.testing.assert_array_equal(ours, ref)


@pytest.mark.parametrize("dtype,tdt", [("bf16", torch.bfloat16),
                                       ("f16", torch.float16)])
def test_round_storage_matches_torch_conversion(dtype, tdt):
    rng = np.random.default_rng(3)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-3).astype(np.float32),
        # exact ties of the bf16 / f16 grids
        np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -11, 1 + 3 * 2 ** -11,
                  -1 - 2 ** -8, 0.0, -0.0], np.float32)])
    ours = oracle.round_storage(x, dtype)
    ref = torch.from_numpy(x).to(tdt).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)


def test_activation_matches_torch():
    x = np.linspace(-30, 30, 4001).astype(np.float32)
    xt = torch.from_numpy(x.astype(np.float64))
    np.testing.assert_array_equal(oracle.activation(x, ACT_RELU),
                                  F.relu(xt).numpy().astype(np.float32))
    np.testing.assert_allclose(oracle.activation(x, ACT_SILU),
                               F.silu(xt).numpy().astype(np.float32),
                               rtol=2e-7, atol=1e-30)
    np.testing.assert_array_equal(oracle.activation(x, ACT_NONE), x)


def test_se_gates_match_torch():
    """Squeeze-excitation gates against a torch formulation (adaptive average
    pool, two 1x1 convolutions, SiLU, sigmoid) in fp64."""
    net = efficientnet_mini_net()
    L = [l for l in net.layers if l.se_mid][1]
    rng = np.random.default_rng(11)
    a = rng.standard_normal((2, 5, 7, L.c_out)).astype(np.float32)
    ours = oracle.se_gates(a, L)
    at = torch.from_numpy(a.astype(np.float64)).permute(0, 3, 1, 2)
    m = F.adaptive_avg_pool2d(at, 1)
    z = F.silu(F.conv2d(m, torch.from_numpy(L.se_w1.astype(np.float64))
                        [:, :, None, None],
                        torch.from_numpy(L.se_b1.astype(np.float64))))
    e = F.conv2d(z, torch.from_numpy(L.se_w2.astype(np.float64))
                 [:, :, None, None], torch.from_numpy(L.se_b2.astype(
                     np.float64)))
    ref = torch.sigmoid(e)[:, :, 0, 0].numpy()
    np.testing.assert_allclose(ours, ref, rtol=2e-6, atol=1e-7)


# ------------------------------------------------------- rulebook pins

def test_single_pixel_amplification_golden():
    """Paper's worked example: one diff pixel -> nine after a 3x3 conv."""
    rows = [tuple(map(int, ln.split())) for ln in
            open(os.path.join(GOLDEN, "single_pixel_3x3.txt"))
            if ln.strip() and not ln.startswith("#")]
    H = W = 8
    pix = np.array([3 * W + 4])
    R = oracle.rulebook(pix, (H, W), (H, W), (3, 3), (1, 1), (1, 1))
    got = [(int(k), int(o) // W, int(o) % W) for k, i, o in R]
    assert len(got) == 9
    assert got == rows
    assert (R[:, 1] == pix[0]).all()


@pytest.mark.parametrize("k,s,p,H,W,site,expect", [
    ((3, 3), (1, 1), (1, 1), 8, 8, (3, 3), 9),     # interior
    ((3, 3), (1, 1), (1, 1), 8, 8, (0, 3), 6),     # edge
    ((3, 3), (1, 1), (1, 1), 8, 8, (0, 7), 4),     # corner
    ((3, 3), (1, 1), (0, 0), 8, 8, (0, 0), 1),     # valid conv corner
    ((5, 5), (1, 1), (2, 2), 9, 9, (4, 4), 25),
    ((5, 5), (1, 1), (2, 2), 9, 9, (0, 1), 12),
    ((3, 3), (2, 2), (1, 1), 9, 9, (4, 4), 1),     # even/even under s2
    ((3, 3), (2, 2), (1, 1), 9, 9, (3, 4), 2),
    ((3, 3), (2, 2), (1, 1), 9, 9, (3, 5), 4),
    ((7, 7), (2, 2), (3, 3), 16, 16, (7, 7), 16),  # odd/odd: 4 x 4
    ((7, 7), (2, 2), (3, 3), 16, 16, (8, 7), 12),
    ((7, 7), (2, 2), (3, 3), 16, 16, (8, 8), 9),
    ((1, 1), (1, 1), (0, 0), 5, 5, (2, 2), 1),
    ((1, 1), (2, 2), (0, 0), 6, 6, (3, 2), 0),     # dropped by stride
])
def test_single_pixel_closed_forms(k, s, p, H, W, site, expect):
    Ho = so.out_size(H, k[0], s[0], p[0])
    Wo = so.out_size(W, k[1], s[1], p[1])
    R = oracle.rulebook(np.array([site[0] * W + site[1]]), (H, W), (Ho, Wo),
                        k, s, p)
    assert len(R) == expect


def brute_rulebook(active, N, H, W, Ho, Wo, k, s, p):
    """Enumerate by definition: every (output, offset) whose input site is
    an active pixel."""
    act = set(int(a) for a in active)
    out = []
    for kk in range(k[0] * k[1]):
        ky, kx = divmod(kk, k[1])
        for n in range(N):
            for oy in range(Ho):
                for ox in range(Wo):
                    iy = oy * s[0] - p[0] + ky
                    ix = ox * s[1] - p[1] + kx
                    if 0 <= iy < H and 0 <= ix < W:
                        ip = (n * H + iy) * W + ix
                        if ip in act:
                            out.append((kk, ip, (n * Ho + oy) * Wo + ox))
    out.sort(key=lambda t: (t[0], t[1]))
    return out


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("geom", [((3, 3), (1, 1), (1, 1)),
                                  ((3, 3), (2, 2), (1, 1)),
                                  ((5, 5), (2, 2), (2, 2)),
                                  ((7, 7), (2, 2), (3, 3)),
                                  ((2, 3), (1, 2), (0, 1))])
def test_rulebook_bruteforce(seed, geom):
    k, s, p = geom
    rng = np.random.default_rng(seed)
    N, H, W = 2, int(rng.integers(3, 9)), int(rng.integers(3, 9))
    Ho, Wo = so.out_size(H, k[0], s[0], p[0]), so.out_size(W, k[1], s[1], p[1])
    if Ho <= 0 or Wo <= 0:
        pytest.skip("empty output")
    active = np.flatnonzero(rng.random(N * H * W) < rng.uniform(0.05, 0.6))
    R = oracle.rulebook(active, (H, W), (Ho, Wo), k, s, p)
    assert [tuple(map(int, r)) for r in R] == brute_rulebook(
        active, N, H, W, Ho, Wo, k, s, p)


# ------------------------------------------------ diff-chain invariants

def small_cases():
    """(net, frames) pairs at sizes the oracle finishes in about a second."""
    return [
        ("toy", toy_net(), toy_video(seed=0, n_frames=4)),
        ("toy_b2", toy_net(H=20, W=28, batch=2),
         random_sparse_video(5, 4, 2, 20, 28, 16, 0.1)),
        ("resnet_mini", resnet_mini_net(),
         random_sparse_video(6, 4, 1, 32, 48, 3, 0.08)),
        ("dw", depthwise_test_net(),
         random_sparse_video(7, 4, 1, 24, 40, 16, 0.1)),
        ("crnn_small", crnn_vgg_net(H=16, W=32),
         textline_video(seed=1, n_frames=4, H=16, W=32, band=3)),
        ("effnet_mini", efficientnet_mini_net(),
         random_sparse_video(3, 4, 1, 32, 40, 3, 0.08)),
    ]


def make_oracle(net):
    return oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C,
                            net.dtype)


@pytest.mark.parametrize("name,net,frames", small_cases(),
                         ids=[c[0] for c in small_cases()])
def test_threshold_zero_equals_dense(name, net, frames):
    """Eq. 2: at threshold 0 Diff Computation reproduces the dense forward
    of every diff frame (up to f32 rounding of the accumulated state)."""
    o = make_oracle(net)
    out0 = o.encode_reference(frames[0])
    ref_out, _, _ = oracle.dense_forward(net.layers, frames[0], net.dtype)
    np.testing.assert_array_equal(out0, ref_out)
    thr = [0.0] * (len(net.layers) + 1)
    for t in range(1, len(frames)):
        out = o.encode_diff(frames[t], thr)
        dense, P, _ = oracle.dense_forward(net.layers, frames[t], net.dtype)
        assert rel_err(out, dense) < 1e-5, (t, rel_err(out, dense))
        for i, p in P.items():
            assert rel_err(o.P[i], p) < 1e-5, (t, i)
        assert 0 < o.density(0) < 1


def test_threshold_zero_equals_dense_bf16():
    net = resnet_mini_net(dtype="bf16")
    frames = random_sparse_video(8, 4, 1, 32, 48, 3, 0.08, dtype="bf16")
    o = make_oracle(net)
    o.encode_reference(frames[0])
    for t in range(1, 4):
        out = o.encode_diff(frames[t], [0.0] * (len(net.layers) + 1))
        dense, _, _ = oracle.dense_forward(net.layers, frames[t], "bf16")
        assert rel_err(out, dense) < 2e-2


ZERO_CASES = [small_cases()[i] for i in (0, 1, 2, 5)]


@pytest.mark.parametrize("name,net,frames", ZERO_CASES,
                         ids=[c[0] for c in ZERO_CASES])
def test_zero_delta_is_identity(name, net, frames):
    """A frame equal to the committed input has no diff pixel at any layer
    and leaves output and state bitwise unchanged."""
    o = make_oracle(net)
    o.encode_reference(frames[0])
    o.encode_diff(frames[1], [0.0] * (len(net.layers) + 1))
    prev_out = o._dense_output().copy()
    prev_P = {i: p.copy() for i, p in o.P.items()}
    out = o.encode_diff(frames[1], [0.0] * (len(net.layers) + 1))
    for t in range(len(net.layers) + 1):
        assert o.density(t) == 0.0
    np.testing.assert_array_equal(out, prev_out)
    for i in prev_P:
        np.testing.assert_array_equal(o.P[i], prev_P[i])
    assert o.flops() == 0


def test_negative_threshold_keeps_everything():
    net = resnet_mini_net()
    frames = random_sparse_video(9, 2, 1, 32, 48, 3, 0.05)
    o = make_oracle(net)
    o.encode_reference(frames[0])
    o.encode_diff(frames[1], [-1.0] * (len(net.layers) + 1))
    for t in range(len(net.layers) + 1):
        assert o.density(t) == 1.0


def test_telescoping_sum_of_deltas():
    """At threshold 0, reference activation + sum of emitted deltas over
    the chunk equals the current activation f(P_t)."""
    net = toy_net()
    frames = toy_video(seed=3, n_frames=4)
    o = make_oracle(net)
    o.encode_reference(frames[0])
    _, _, acts0 = oracle.dense_forward(net.layers, frames[0], "f32")
    acc = acts0[0].reshape(-1, 16).copy()
    for t in range(1, 4):
        o.encode_diff(frames[t], [0.0] * 3)
        T = o.last["tensors"][1]
        acc[T["pix"]] += T["rows"]
    _, _, acts = oracle.dense_forward(net.layers, frames[3], "f32")
    assert rel_err(acc, acts[0].reshape(-1, 16)) < 1e-5


def test_first_layer_error_bound():
    """With a positive input threshold the first layer's state differs from
    the dense pre-activation by at most thr * sum |W| per output channel
    (every uncommitted input difference is at most thr in each channel)."""
    net = toy_net()
    frames = toy_video(seed=4, n_frames=4)
    # add small sub-threshold jitter everywhere on the diff frames
    rng = np.random.default_rng(0)
    thr0 = 0.05
    jit = [frames[0]] + [f + rng.uniform(-0.04, 0.04, f.shape).astype(
        np.float32) for f in frames[1:]]
    o = make_oracle(net)
    o.encode_reference(jit[0])
    bound = thr0 * np.abs(net.layers[0].weight).sum(axis=(1, 2, 3))
    for t in range(1, 4):
        o.encode_diff(jit[t], [thr0, 0.0, 0.0])
        _, P, _ = oracle.dense_forward(net.layers, jit[t], "f32")
        err = np.abs(o.P[0] - P[0]).reshape(-1, 16).max(axis=0)
        assert (err <= bound * (1 + 1e-5) + 1e-5).all()
        assert err.max() > 0  # the truncation really happened


def test_nonlinearity_cannot_take_deltas():
    """Eq. 3: applying the non-linearity to the delta instead of to the
    reconstructed pre-activation is wrong; the oracle's handling is right."""
    net = toy_net()
    frames = toy_video(seed=5, n_frames=2)
    o = make_oracle(net)
    o.encode_reference(frames[0])
    out = o.encode_diff(frames[1], [0.0] * 3)
    dense, P, acts = oracle.dense_forward(net.layers, frames[1], "f32")
    _, P0, acts0 = oracle.dense_forward(net.layers, frames[0], "f32")
    L0 = net.layers[0]
    dX = frames[1] - frames[0]
    naive_act0 = acts0[0] + np.maximum(
        oracle.conv2d_nhwc(dX, L0.weight, None, L0.s, L0.p), 0.0)
    assert rel_err(naive_act0, acts[0]) > 1e-2
    assert rel_err(out, dense) < 1e-5


# --------------------------------------- independent dense simulation

def dense_delta_sim(net, frames, thr):
    """Dense-tensor re-statement of the truncation semantics: every tensor
    is a full map that is zero on truncated pixels; convolutions go through
    torch conv2d.  Written independently of the oracle's sparse code."""
    layers = net.layers
    stateful = [L.act != ACT_NONE or L.pool_k[0] > 0 or L.se_mid > 0
                or i == len(layers) - 1 for i, L in enumerate(layers)]

    def gates(a, L):
        # squeeze-excitation re-stated with torch ops
        at = torch.from_numpy(a.astype(np.float64))
        m = at.mean(dim=(1, 2)).float().double()
        z = (m @ torch.from_numpy(L.se_w1.astype(np.float64)).T
             + torch.from_numpy(L.se_b1.astype(np.float64))).float().double()
        z = (z / (1 + torch.exp(-z))).float().double()
        e = (z @ torch.from_numpy(L.se_w2.astype(np.float64)).T
             + torch.from_numpy(L.se_b2.astype(np.float64))).float().double()
        return torch.sigmoid(e).float().numpy()

    def gate(a, g):
        return (a.astype(np.float64) * g[:, None, None, :].astype(
            np.float64)).astype(np.float32)

    def act(x, a):
        x64 = x.astype(np.float64)
        if a == ACT_RELU:
            y = np.maximum(x64, 0)
        elif a == ACT_SILU:
            y = x64 / (1 + np.exp(-x64))
        else:
            y = x64
        return y.astype(np.float32)

    def pool(x, L):
        if L.pool_k[0] == 0:
            return x
        return F.max_pool2d(torch.from_numpy(x.astype(np.float64)).permute(
            0, 3, 1, 2), L.pool_k, L.pool_s, L.pool_p).permute(
            0, 2, 3, 1).numpy().astype(np.float32)

    def mask(d, t):
        keep = np.abs(d).max(axis=-1) > t
        return d * keep[..., None]

    # reference
    acts = {-1: frames[0].astype(np.float64)}
    P, S = {}, {}
    for i, L in enumerate(layers):
        a = torch_conv_nhwc(acts[L.src], L.weight, L.bias, L.s, L.p, L.groups)
        if L.residual_src != -2:
            a = a + acts[L.residual_src]
        p32 = a.astype(np.float32)
        if stateful[i]:
            P[i] = p32
            e = pool(act(p32, L.act), L)
            if L.se_mid:
                S[i] = gates(e, L)
                e = gate(e, S[i])
            acts[i] = e.astype(np.float64)
        else:
            acts[i] = p32.astype(np.float64)
    xhat = frames[0].astype(np.float32).copy()
    outs, masks = [], []
    for f in frames[1:]:
        D = f.astype(np.float32) - xhat
        d = {-1: mask(D, thr[0]).astype(np.float64)}
        keep0 = np.abs(D).max(axis=-1) > thr[0]
        xhat[keep0] = f.astype(np.float32)[keep0]
        fm = [keep0]
        for i, L in enumerate(layers):
            dp = torch_conv_nhwc(d[L.src], L.weight, None, L.s, L.p, L.groups)
            if L.residual_src != -2:
                dp = dp + d[L.residual_src]
            dp32 = dp.astype(np.float32)
            if stateful[i]:
                Pn = (P[i].astype(np.float64) + dp32).astype(np.float32)
                en = pool(act(Pn, L.act), L)
                eo = pool(act(P[i], L.act), L)
                if L.se_mid:
                    sn = gates(en, L)
                    en, eo = gate(en, sn), gate(eo, S[i])
                    S[i] = sn
                e = (en.astype(np.float64) - eo.astype(np.float64))
                P[i] = Pn
                e = e.astype(np.float32)
            else:
                e = dp32
            fm.append(np.abs(e).max(axis=-1) > thr[i + 1])
            d[i] = mask(e, thr[i + 1]).astype(np.float64)
        last = pool(act(P[len(layers) - 1], layers[-1].act), layers[-1])
        if layers[-1].se_mid:
            last = gate(last, S[len(layers) - 1])
        outs.append(last)
        masks.append(fm)
    return outs, masks


SIM_CASES = [small_cases()[i] for i in (0, 1, 2, 3, 5)]


@pytest.mark.parametrize("name,net,frames", SIM_CASES,
                         ids=[c[0] for c in SIM_CASES])
@pytest.mark.parametrize("thr", [0.0, 0.05])
def test_matches_dense_delta_simulation(name, net, frames, thr):
    thrs = [thr] * (len(net.layers) + 1)
    sim_out, sim_masks = dense_delta_sim(net, frames, thrs)
    o = make_oracle(net)
    o.encode_reference(frames[0])
    for t in range(1, len(frames)):
        out = o.encode_diff(frames[t], thrs)
        for ti, T in enumerate(o.last["tensors"]):
            m = np.zeros(int(np.prod(T["grid"])), bool)
            m[T["pix"]] = True
            sm = sim_masks[t - 1][ti].reshape(-1)
            diff = np.flatnonzero(m != sm)
            # masks may only differ on rows within rounding of the threshold
            if len(diff):
                cm = dict(zip(T["cand"].tolist(), T["cand_max"].tolist()))
                for pxl in diff:
                    assert abs(cm.get(int(pxl), 0.0) - thrs[ti]) < 1e-6
        assert rel_err(out, sim_out[t - 1]) < 1e-5


# ------------------------------------------------ planted mistakes

def test_planted_mistake_no_commit_is_caught(monkeypatch):
    """Not committing kept pixels to the Subtraction buffer breaks Eq. 2 on
    the second diff frame; the threshold-0 pin must catch it."""
    net = toy_net()
    frames = toy_video(seed=0, n_frames=3)
    o = make_oracle(net)
    o.encode_reference(frames[0])
    saved = o.xhat.copy()
    o.encode_diff(frames[1], [0.0] * 3)
    o.xhat = saved                      # the planted mistake
    out = o.encode_diff(frames[2], [0.0] * 3)
    dense, _, _ = oracle.dense_forward(net.layers, frames[2], "f32")
    assert rel_err(out, dense) > 1e-3


def test_planted_mistake_bias_in_delta_is_caught(monkeypatch):
    net = toy_net()
    frames = toy_video(seed=0, n_frames=2)
    orig = so._apply_offset

    def with_bias(rows, w, ky, kx, groups):
        return orig(rows, w, ky, kx, groups) + 0.1   # planted mistake
    monkeypatch.setattr(so, "_apply_offset", with_bias)
    o = make_oracle(net)
    o.encode_reference(frames[0])
    out = o.encode_diff(frames[1], [0.0] * 3)
    dense, _, _ = oracle.dense_forward(net.layers, frames[1], "f32")
    assert rel_err(out, dense) > 1e-3


def test_planted_mistake_flipped_offset_is_caught(monkeypatch):
    orig = so.window_targets

    def flipped(pix, in_hw, out_hw, k, s, p):
        R = orig(pix, in_hw, out_hw, k, s, p)
        R = R.copy()
        R[:, 0] = k[0] * k[1] - 1 - R[:, 0]          # planted mistake
        return R
    monkeypatch.setattr(so, "window_targets", flipped)
    active = np.array([5, 17, 30])
    R = so.rulebook(active, (6, 7), (6, 7), (3, 3), (1, 1), (1, 1))
    assert [tuple(map(int, r)) for r in R] != brute_rulebook(
        active, 1, 6, 7, 6, 7, (3, 3), (1, 1), (1, 1))


def test_planted_mistake_frozen_se_gates_is_caught(monkeypatch):
    """Keeping the reference frame's squeeze-excitation gates in diff
    frames (instead of recomputing them from the dense activation) breaks
    Eq. 2 for a net with squeeze-excitation; the threshold-0 pin must catch
    it."""
    net = efficientnet_mini_net()
    frames = random_sparse_video(3, 2, 1, 32, 40, 3, 0.08)
    dense, _, _ = oracle.dense_forward(net.layers, frames[1], "f32")
    o = make_oracle(net)
    o.encode_reference(frames[0])
    frozen = {i: s.copy() for i, s in o.S.items()}
    monkeypatch.setattr(so, "se_gates",
                        lambda a, L: frozen[net.layers.index(L)])
    out = o.encode_diff(frames[1], [0.0] * (len(net.layers) + 1))
    assert rel_err(out, dense) > 1e-4


# ------------------------------------------------ algorithmic FLOP count

def _single_conv(cin, cout, groups, H, W, k=(3, 3), p=(1, 1)):
    rng = np.random.default_rng(11)
    L = LayerSpec(src=-1, c_in=cin, c_out=cout, k=k, s=(1, 1), p=p,
                  groups=groups, act=ACT_RELU)
    L.weight = rng.standard_normal((cout, cin // groups, *k)).astype(
        np.float32)
    L.bias = np.zeros(cout, np.float32)
    return L


@pytest.mark.parametrize("cin,cout,groups", [(4, 6, 1), (8, 8, 8)])
@pytest.mark.parametrize("y,x,taps", [(3, 4, 9),    # interior: 3x3 outputs
                                      (0, 0, 4),    # corner: 2x2
                                      (0, 4, 6)])   # edge: 2x3
def test_flops_single_pixel(cin, cout, groups, y, x, taps):
    """One changed pixel under a 3x3 / pad-1 convolution reaches `taps`
    outputs (the dense amplification example, clipped at borders), and each
    reached output costs one multiply-add per input channel of its group
    and output channel: 2 * taps * (Cin / groups) * Cout."""
    H, W = 8, 9
    L = _single_conv(cin, cout, groups, H, W)
    o = so.OracleNet([L], 1, H, W, cin, "f32")
    f0 = np.zeros((1, H, W, cin), np.float32)
    f1 = f0.copy()
    f1[0, y, x, :] = 1.0
    o.encode_reference(f0)
    o.encode_diff(f1, [0.0, 0.0])
    assert o.flops() == 2 * taps * (cin // groups) * cout


@pytest.mark.parametrize("cin,cout,groups", [(3, 5, 1), (6, 6, 6)])
def test_flops_everything_active(cin, cout, groups):
    """Negative threshold: every input pixel is active, so the pairs are all
    in-bounds (input, output) window pairs.  For a 3x3 / stride-1 / pad-1
    window on an H x W map offset (dy, dx) has (H - |dy|)(W - |dx|) of
    them, which sums to (3H - 2)(3W - 2)."""
    H, W = 6, 7
    L = _single_conv(cin, cout, groups, H, W)
    o = so.OracleNet([L], 1, H, W, cin, "f32")
    rng = np.random.default_rng(2)
    f0 = rng.random((1, H, W, cin), dtype=np.float32)
    o.encode_reference(f0)
    o.encode_diff(f0 + 1.0, [-1.0, -1.0])
    pairs = (3 * H - 2) * (3 * W - 2)
    assert o.last["layers"][0]["pairs"] == pairs
    assert o.flops() == 2 * pairs * (cin // groups) * cout
