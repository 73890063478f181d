"""GPU parity: the HIP path (called through the C ABI) against the CPU
oracle on identical seeded inputs, after every frame of a chunk.

Exact: frame-delta masks and rows, candidate lists, kept lists (outside the
rounding band), rulebooks and pair counts.  Within tolerance (1e-4 relative
for f32, 2e-2 for f16/bf16, per tensor against the oracle's largest
magnitude): emitted delta rows, pre-activation state, network output.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2410_20790_amd import SparseTemNet
from paper_2410_20790_amd import binding as B
from parity_util import (RTOL, compare_frame, make_pair, rel, run_chunk,
                         say, to_dev)
from workloads import (crnn_vgg_net, depthwise_test_net, driving_video,
                       efficientnet_mini_net, efficientnet_net,
                       object_video, random_sparse_video, resnet50_net,
                       resnet_mini_net, textline_video, toy_net, toy_video)

pytestmark = pytest.mark.gpu


# ----------------------------------------------------------- toy encoder

@pytest.mark.parametrize("thr", [0.0, 0.05])
def test_toy_chunk(thr):
    """One 3x3 conv + ReLU + 1x1 conv on a 4-frame 64x64x16 chunk with 10%
    of sites redrawn per frame in 8x8 patches."""
    run_chunk(toy_net(), toy_video(seed=0, n_frames=4), thr, f"toy thr={thr}")


def test_toy_ragged_batch():
    """Batch of 2 on a 20x28 map: tile tails and an image boundary."""
    net = toy_net(H=20, W=28, batch=2)
    run_chunk(net, random_sparse_video(5, 4, 2, 20, 28, 16, 0.1), 0.0,
              "toy ragged")


def test_toy_single_pixel_amplification():
    """One changed interior pixel reaches nine 3x3 outputs (dense
    amplification example); the 1x1 layer then sees those nine."""
    net = toy_net(H=16, W=16)
    f0 = np.random.default_rng(3).random((1, 16, 16, 16), dtype=np.float32)
    f1 = f0.copy()
    f1[0, 7, 9] += 0.5
    o, g = run_chunk(net, [f0, f1], 0.0, "toy one pixel")
    try:
        assert len(B.st_debug_active(g.handle, -1)) == 1
        pairs, act = B.st_debug_counters(g.handle, 2)
        assert pairs[0] == 9
        pix, _ = B.st_debug_candidates(g.handle, 0, 16)
        assert len(pix) == 9
    finally:
        g.close()


# --------------------------------------------------------- CRNN encoder

@pytest.mark.parametrize("thr", [0.0, 0.02])
def test_crnn_chunk(thr):
    """CRNN-style VGG encoder at 32x128 (seven 3x3 convs, 2x2 and 2x1
    pools) on a scrolling text line."""
    net = crnn_vgg_net()
    run_chunk(net, textline_video(seed=1, n_frames=5), thr, f"crnn thr={thr}",
              max_band=4 if thr else 0)


# ------------------------------------------------------- ResNet family

@pytest.mark.parametrize("thr", [0.0, 0.05])
def test_resnet_mini_f32(thr):
    """7x7/2 stem, overlapping 3x3/2 pool, bottlenecks with strided 3x3,
    downsample and identity shortcuts."""
    net = resnet_mini_net()
    run_chunk(net, random_sparse_video(6, 4, 1, 32, 48, 3, 0.08), thr,
              f"resnet_mini thr={thr}", max_band=4 if thr else 0)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_resnet_mini_half(dtype):
    net = resnet_mini_net(dtype=dtype, H=40, W=56)
    run_chunk(net, random_sparse_video(8, 4, 1, 40, 56, 3, 0.08, dtype=dtype),
              0.0, f"resnet_mini {dtype}")


def test_resnet50_small_bf16():
    """ResNet-50 (all 53 convs) at 64x128 in bf16, clustered changes."""
    net = resnet50_net(H=64, W=128)
    frames = driving_video(seed=2, n_frames=3, H=64, W=128, density=0.10,
                           side=(8, 32))
    run_chunk(net, frames, 0.0, "resnet50 64x128 bf16", max_band=8)


# ------------------------------------------------------------ depthwise

@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_depthwise(dtype):
    net = depthwise_test_net(dtype=dtype)
    run_chunk(net, random_sparse_video(7, 4, 1, 24, 40, 16, 0.1, dtype=dtype),
              0.0, f"depthwise {dtype}")


# ------------------------------------------------- EfficientNet family

@pytest.mark.parametrize("dtype,thr", [("f32", 0.0), ("f32", 0.05),
                                       ("f16", 0.0), ("bf16", 0.0)])
def test_efficientnet_mini(dtype, thr):
    """MBConv blocks: expand, depthwise 3x3 / 5x5 stride 2, exact
    squeeze-excitation, linear project with identity skip."""
    net = efficientnet_mini_net(dtype=dtype)
    run_chunk(net, random_sparse_video(3, 4, 1, 32, 40, 3, 0.08, dtype=dtype),
              thr, f"effnet_mini {dtype} thr={thr}",
              max_band=8 if (thr or dtype != "f32") else 0)


def test_efficientnet_b0_small_f16():
    """All 16 MBConv blocks of EfficientNet-B0 at 64x64, fp16, on the
    detection-like video (global translation plus moving objects)."""
    net = efficientnet_net(H=64, W=64)
    frames = object_video(seed=1, n_frames=3, H=64, W=64, obj=8)
    run_chunk(net, frames, 0.02, "effnet-b0 64x64 f16", max_band=64)


# ---------------------------------------- online threshold adjustment

@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_ibst_chunk(dtype):
    """Thresholds chosen per frame by the iterative binary search from the
    oracle's sparsities; the GPU encodes with the same thresholds, and a
    second controller fed from the GPU's own densities must choose the same
    thresholds."""
    from paper_2410_20790_amd.ibst import (IBST, nonlinear_tensors,
                                           sparsity_from_counts)
    net = efficientnet_mini_net(dtype=dtype)
    frames = object_video(seed=2, n_frames=7, H=32, W=40, obj=8,
                          obj_frac=0.1, dtype=dtype)
    L_n = len(net.layers)
    ctl = nonlinear_tensors(net.layers)
    c_o = IBST(L_n + 1, ctl, target=0.7, eps=0.05, theta_max=0.5)
    c_g = IBST(L_n + 1, ctl, target=0.7, eps=0.05, theta_max=0.5)
    o, g = make_pair(net)
    tag = f"ibst {dtype}"
    try:
        o.encode_reference(frames[0])
        g.encode_reference(to_dev(frames[0], dtype))
        grids = [int(np.prod(g.tensor_shape(k - 1)[:3]))
                 for k in range(L_n + 1)]
        n_band = 0
        for t in range(1, len(frames)):
            if t == 4:  # a new cycle restarts the brackets
                c_o.start_cycle()
                c_g.start_cycle()
            thr = c_o.thresholds()
            if n_band == 0:  # equal counts so far: equal decisions
                assert thr == c_g.thresholds(), f"{tag} f{t}"
            say(f"[gpu] {tag}: frame {t} thr[0:3]={thr[:3]}")
            o.encode_diff(frames[t], thr)
            out_g = g.encode_diff(to_dev(frames[t], dtype), thr)
            torch.cuda.synchronize()
            n_band += compare_frame(net, o, g, out_g, f"{tag} f{t}")
            c_o.update([1.0 - o.density(k) for k in range(L_n + 1)])
            _, act = B.st_debug_counters(g.handle, L_n)
            c_g.update(sparsity_from_counts(act, grids))
        assert n_band <= (0 if dtype == "f32" else 4)
        assert any(v > 0 for v in c_o.thresholds())
    finally:
        g.close()


# ----------------------------------------------------------- edge cases

def test_zero_delta_leaves_everything_unchanged():
    net = resnet_mini_net()
    frames = random_sparse_video(11, 2, 1, 32, 48, 3, 0.1)
    o, g = run_chunk(net, frames, 0.0, "zero delta warm-up")
    try:
        thr = [0.0] * (len(net.layers) + 1)
        x = to_dev(frames[1], "f32")
        out1 = g.encode_diff(x, thr)
        P1 = {i: B.st_debug_state(g.handle, i, o.P[i].shape) for i in o.P}
        say("[gpu] zero delta: repeat frame")
        out2 = g.encode_diff(x, thr)
        torch.cuda.synchronize()
        assert torch.equal(out1, out2)
        _, act = B.st_debug_counters(g.handle, len(net.layers))
        assert (act == 0).all()
        for i in o.P:
            np.testing.assert_array_equal(
                B.st_debug_state(g.handle, i, o.P[i].shape), P1[i])
    finally:
        g.close()


def test_negative_threshold_reproduces_dense():
    """thr < 0 keeps every site: the diff pass then touches every pixel and
    must agree with a dense reference pass on the same frame."""
    net = resnet_mini_net()
    frames = random_sparse_video(12, 2, 1, 32, 48, 3, 0.05)
    o, g = make_pair(net)
    g2 = SparseTemNet(net.layers, 1, 32, 48, 3, "f32")
    try:
        g.encode_reference(to_dev(frames[0], "f32"))
        out = g.encode_diff(to_dev(frames[1], "f32"),
                            [-1.0] * (len(net.layers) + 1))
        dense = g2.encode_reference(to_dev(frames[1], "f32"))
        torch.cuda.synchronize()
        for t in range(len(net.layers) + 1):
            assert g.density(t - 1) == 1.0
        assert rel(out.cpu().numpy(), dense.cpu().numpy()) < 1e-4
    finally:
        g.close()
        g2.close()


def test_threshold_zero_matches_dense_pass_over_chunk():
    """Linearity invariant on the GPU alone: at threshold 0 every diff
    output equals the dense pass of that frame."""
    net = crnn_vgg_net()
    frames = textline_video(seed=4, n_frames=6)
    g = SparseTemNet(net.layers, 1, 32, 128, 1, "f32")
    g2 = SparseTemNet(net.layers, 1, 32, 128, 1, "f32")
    try:
        g.encode_reference(to_dev(frames[0], "f32"))
        for t in range(1, 6):
            out = g.encode_diff(to_dev(frames[t], "f32"), [0.0] * 8)
            dense = g2.encode_reference(to_dev(frames[t], "f32"))
            torch.cuda.synchronize()
            assert rel(out.cpu().numpy(), dense.cpu().numpy()) < 1e-4
    finally:
        g.close()
        g2.close()


def test_repeat_runs_are_bitwise_identical():
    net = resnet_mini_net()
    frames = random_sparse_video(13, 4, 1, 32, 48, 3, 0.1)
    outs = []
    for rep in range(2):
        g = SparseTemNet(net.layers, 1, 32, 48, 3, "f32")
        try:
            g.encode_reference(to_dev(frames[0], "f32"))
            res = []
            for t in range(1, 4):
                res.append(g.encode_diff(to_dev(frames[t], "f32"),
                                         [0.01] * (len(net.layers) + 1)).cpu())
            outs.append(res)
        finally:
            g.close()
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_api_errors_on_gpu():
    net = toy_net()
    g = SparseTemNet(net.layers, 1, 64, 64, 16, "f32")
    try:
        x = to_dev(toy_video(n_frames=1)[0], "f32")
        with pytest.raises(B.StError) as e:
            g.encode_diff(x, [0.0] * 3)
        assert e.value.status == B.ST_ERR_STATE
        g.encode_reference(x)
        with pytest.raises(B.StError) as e:
            g.encode_diff(x, [0.0, float("nan"), 0.0])
        assert e.value.status == B.ST_ERR_INVALID_ARG
        with pytest.raises(B.StError):
            g.density(5)
        assert g.density(-1) == 1.0   # reference pass: every site active
    finally:
        g.close()


def test_per_image_density():
    net = toy_net(H=16, W=16, batch=3)
    frames = random_sparse_video(14, 2, 3, 16, 16, 16, 0.0)
    f1 = frames[0].copy()
    f1[1, :4] += 1.0        # image 1: 4 of 16 rows change
    g = SparseTemNet(net.layers, 3, 16, 16, 16, "f32")
    try:
        g.encode_reference(to_dev(frames[0], "f32"))
        g.encode_diff(to_dev(f1, "f32"), [0.0] * 3)
        assert g.density(-1, 0) == 0.0
        assert g.density(-1, 1) == 0.25
        assert g.density(-1, 2) == 0.0
        assert abs(g.density(-1) - 0.25 / 3) < 1e-7
    finally:
        g.close()


# ------------------------------------------------ full-size workloads

def test_resnet50_full_size_first_layer_exact():
    """ResNet-50 at 1024x2048 bf16 with 10% clustered change, in the launch
    configuration the benchmark times: the frame-delta mask and the stem's
    rulebook must equal the oracle's bit for bit, its state within the bf16
    tolerance; the oracle runs the stem alone (its output needs no deeper
    layer)."""
    net = resnet50_net()
    frames = driving_video(seed=0, n_frames=2, density=0.10)
    stem = [net.layers[0]]
    o = oracle.OracleNet(stem, 1, 1024, 2048, 3, "bf16")
    say("[gpu] resnet50 full: oracle stem")
    o.encode_reference(frames[0])
    o.encode_diff(frames[1], [0.0, 0.0])
    g = SparseTemNet(net.layers, 1, 1024, 2048, 3, "bf16")
    try:
        say("[gpu] resnet50 full: gpu")
        g.encode_reference(to_dev(frames[0], "bf16"))
        g.encode_diff(to_dev(frames[1], "bf16"),
                      [0.0] * (len(net.layers) + 1), write_out=False)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(B.st_debug_active(g.handle, -1),
                                      o.last["tensors"][0]["pix"])
        R = B.st_debug_rulebook(g.handle, 0)
        np.testing.assert_array_equal(R.astype(np.int64),
                                      o.last["layers"][0]["rulebook"])
        P0 = B.st_debug_state(g.handle, 0, o.P[0].shape)
        assert rel(P0, o.P[0]) < RTOL["bf16"]
        pix, _ = B.st_debug_candidates(g.handle, 0, 64)
        np.testing.assert_array_equal(pix, o.last["tensors"][1]["cand"])
        d0 = g.density(-1)
        assert 0.09 < d0 < 0.2
    finally:
        g.close()


def test_resnet50_full_size_linearity():
    """At threshold 0 the diff output of a full-size frame equals the dense
    pass of that frame (property that holds at any size)."""
    net = resnet50_net()
    frames = driving_video(seed=1, n_frames=3, density=0.10)
    g = SparseTemNet(net.layers, 1, 1024, 2048, 3, "bf16")
    g2 = SparseTemNet(net.layers, 1, 1024, 2048, 3, "bf16")
    try:
        say("[gpu] resnet50 full linearity")
        g.encode_reference(to_dev(frames[0], "bf16"))
        for t in (1, 2):
            out = g.encode_diff(to_dev(frames[t], "bf16"),
                                [0.0] * (len(net.layers) + 1))
        dense = g2.encode_reference(to_dev(frames[2], "bf16"))
        torch.cuda.synchronize()
        assert rel(out.cpu().numpy(), dense.cpu().numpy()) < 2e-2
    finally:
        g.close()
        g2.close()


# -------------------------------------------------------- graph replay

@pytest.mark.parametrize("which", ["toy", "crnn", "resnet_mini"])
def test_graph_replay_matches_eager(which):
    """A diff frame replayed as a HIP graph gives bitwise the eager result:
    two nets encode the same chunk, one eagerly and one by graph replay
    (each replay separated by eager work and a synchronisation); outputs
    and states are compared after every frame."""
    if which == "toy":
        net, frames, thr = toy_net(), toy_video(seed=4, n_frames=5), 0.0
    elif which == "crnn":
        net = crnn_vgg_net()
        frames, thr = textline_video(seed=4, n_frames=5), 0.02
    else:
        net = resnet_mini_net()
        frames = random_sparse_video(6, 5, 1, 32, 48, 3, 0.08)
        thr = 0.0
    thr_l = [thr] * (len(net.layers) + 1)
    ge = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, net.dtype)
    gg = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, net.dtype)
    try:
        say(f"[gpu] graph replay {which}")
        dev = [to_dev(f, net.dtype) for f in frames]
        ge.encode_reference(dev[0])
        out_g = gg.new_output()
        gg.encode_reference(dev[0], out=out_g)
        torch.cuda.synchronize()
        replay = gg.capture_diff(thr_l, out_g)
        for t in range(1, len(frames)):
            out_e = ge.encode_diff(dev[t], thr_l)
            torch.cuda.synchronize()
            replay(dev[t])
            torch.cuda.synchronize()
            np.testing.assert_array_equal(out_g.cpu().numpy(),
                                          out_e.cpu().numpy())
            for t2 in range(len(net.layers) + 1):
                np.testing.assert_array_equal(
                    B.st_debug_active(gg.handle, t2 - 1),
                    B.st_debug_active(ge.handle, t2 - 1))
                C = ge.tensor_shape(t2 - 1)[3]
                pg, rg = B.st_debug_candidates(gg.handle, t2 - 1, C)
                pe, re_ = B.st_debug_candidates(ge.handle, t2 - 1, C)
                np.testing.assert_array_equal(pg, pe)
                np.testing.assert_array_equal(rg, re_)
    finally:
        ge.close()
        gg.close()


@pytest.mark.parametrize("frozen", [False, True])
def test_graph_replay_squeeze_excitation_adaptive(frozen):
    """Graph replay of the adaptive entry on the mini EfficientNet (exact or
    frozen squeeze-excitation, device-adjusted thresholds): the gate slots
    are chosen by a parity word in device memory, so replays and a
    reference frame encoded directly between them follow the eager net bit
    for bit -- outputs, kept lists, states and thresholds after every
    frame, each replay separated by eager work and a synchronisation."""
    from paper_2410_20790_amd.ibst import nonlinear_tensors
    from workloads import efficientnet_mini_net, object_video
    net = efficientnet_mini_net()
    frames = object_video(seed=12, n_frames=9, H=32, W=40, obj=8,
                          obj_frac=0.1)
    L_n = len(net.layers)
    ctl = nonlinear_tensors(net.layers)
    kw = dict(frozen_se=frozen)
    ge = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, "f32", **kw)
    gg = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, "f32", **kw)
    try:
        say(f"[gpu] graph replay squeeze-excitation frozen={frozen}")
        for g in (ge, gg):
            g.set_threshold_control(ctl, [0.01] * (L_n + 1), 0.7, 0.05, 0.5)
        dev = [to_dev(f, "f32") for f in frames]
        out_g = gg.new_output()
        ge.encode_reference(dev[0])
        gg.encode_reference(dev[0], out=out_g)
        torch.cuda.synchronize()
        replay = gg.capture_diff(None, out_g)
        for t in range(1, len(frames)):
            if t == 5:  # a reference frame in the middle, encoded directly
                ge.encode_reference(dev[t])
                gg.encode_reference(dev[t], out=out_g)
                torch.cuda.synchronize()
                continue
            out_e = ge.encode_diff_adaptive(dev[t])
            torch.cuda.synchronize()
            replay(dev[t])
            torch.cuda.synchronize()
            np.testing.assert_array_equal(out_g.cpu().numpy(),
                                          out_e.cpu().numpy(),
                                          err_msg=f"frame {t}")
            np.testing.assert_array_equal(gg.thresholds(), ge.thresholds())
            for t2 in range(L_n + 1):
                np.testing.assert_array_equal(
                    B.st_debug_active(gg.handle, t2 - 1),
                    B.st_debug_active(ge.handle, t2 - 1))
            for i, L in enumerate(net.layers):
                shape = tuple(ge.tensor_shape(i)[:3]) + (L.c_out,)
                try:
                    Pe = B.st_debug_state(ge.handle, i, shape)
                except B.StError:
                    continue  # no state in this layer
                np.testing.assert_array_equal(
                    B.st_debug_state(gg.handle, i, shape), Pe)
    finally:
        ge.close()
        gg.close()
