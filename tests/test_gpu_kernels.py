"""Tight per-kernel parity: one- and two-layer nets, so both sides see
identical inputs and the only difference is summation order (f32 on the
GPU, fp64 in the oracle).  Pre-activation state within 1e-5 of its scale,
emitted deltas within one storage ulp (plus the state's rounding), masks and
rulebooks exact.  Geometries cover every path of the kernels: ragged row and
channel tiles, several reduction stages, small input channels packed across
kernel offsets, strides, 5x5 and 7x7 windows, 1x1 identity rulebooks,
depthwise, max-pool (disjoint and overlapping), linear layers, and deep
reductions split across work units."""

import numpy as np
import pytest
import torch

from paper_2410_20790_amd import binding as B
from parity_util import make_pair, say, to_dev
from workloads import (ACT_NONE, ACT_RELU, ACT_SILU, LayerSpec, NetSpec,
                       random_sparse_video, to_storage)

pytestmark = pytest.mark.gpu

ULP = {"f32": 2.0 ** -23, "f16": 2.0 ** -10, "bf16": 2.0 ** -7}

GEOMS = {
    # name: (Cin, Cout, k, s, p, groups, act, pool(k, s, p) or None)
    "3x3": (24, 40, (3, 3), (1, 1), (1, 1), 1, ACT_RELU, None),
    "3x3_wide": (256, 136, (3, 3), (1, 1), (1, 1), 1, ACT_RELU, None),
    "3x3_s2": (32, 64, (3, 3), (2, 2), (1, 1), 1, ACT_RELU, None),
    "5x5": (8, 16, (5, 5), (1, 1), (2, 2), 1, ACT_SILU, None),
    "7x7_s2_c3": (3, 64, (7, 7), (2, 2), (3, 3), 1, ACT_RELU, None),
    "3x3_c1": (1, 64, (3, 3), (1, 1), (1, 1), 1, ACT_RELU, None),
    "1x1": (64, 256, (1, 1), (1, 1), (0, 0), 1, ACT_RELU, None),
    "1x1_s2": (64, 128, (1, 1), (2, 2), (0, 0), 1, ACT_NONE, None),
    "2x3_asym": (16, 24, (2, 3), (1, 2), (1, 0), 1, ACT_SILU, None),
    "dw3": (48, 48, (3, 3), (1, 1), (1, 1), 48, ACT_SILU, None),
    "dw5_s2": (40, 40, (5, 5), (2, 2), (2, 2), 40, ACT_RELU, None),
    "pool2x2": (16, 64, (3, 3), (1, 1), (1, 1), 1, ACT_RELU,
                ((2, 2), (2, 2), (0, 0))),
    "pool3x3_s2": (8, 32, (3, 3), (1, 1), (1, 1), 1, ACT_RELU,
                   ((3, 3), (2, 2), (1, 1))),
    "pool2x1": (16, 32, (3, 3), (1, 1), (1, 1), 1, ACT_RELU,
                ((2, 1), (2, 1), (0, 0))),
    # deep reductions on few output tiles: the reduction is split across
    # work units and finished by the split epilogue (state, pooled-defer)
    "3x3_deep": (512, 512, (3, 3), (1, 1), (1, 1), 1, ACT_RELU, None),
    "1x1_deep": (1024, 256, (1, 1), (1, 1), (0, 0), 1, ACT_RELU, None),
    "pool_deep": (256, 64, (3, 3), (1, 1), (1, 1), 1, ACT_RELU,
                  ((2, 2), (2, 2), (0, 0))),
}


def one_layer(name, dtype, H=23, W=37, batch=2, seed=0):
    cin, cout, k, s, p, g, act, pool = GEOMS[name]
    rng = np.random.default_rng(seed)
    L = LayerSpec(src=-1, c_in=cin, c_out=cout, k=k, s=s, p=p, groups=g,
                  act=act, name=name)
    L.weight = to_storage(rng.normal(0, 1.0 / np.sqrt(cin // g * k[0] * k[1]),
                                     (cout, cin // g, *k)), dtype)
    L.bias = to_storage(rng.normal(0, 0.1, cout), dtype)
    if pool:
        L.pool_k, L.pool_s, L.pool_p = pool
    return NetSpec(name, [L], batch, H, W, cin, dtype)


def check(net, frames, thr):
    o, g = make_pair(net)
    try:
        dt = net.dtype
        o.encode_reference(frames[0])
        g.encode_reference(to_dev(frames[0], dt))
        for t in range(1, len(frames)):
            thr_l = [thr] * (len(net.layers) + 1)
            o.encode_diff(frames[t], thr_l)
            out = g.encode_diff(to_dev(frames[t], dt), thr_l)
            torch.cuda.synchronize()
            for i in o.P:
                Pg = B.st_debug_state(g.handle, i, o.P[i].shape)
                sc = np.abs(o.P[i]).max()
                assert np.abs(Pg - o.P[i]).max() <= 1e-5 * sc, f"state {i}"
            for ti in range(len(net.layers) + 1):
                T = o.last["tensors"][ti]
                np.testing.assert_array_equal(
                    B.st_debug_active(g.handle, ti - 1), T["pix"])
                if ti == 0:
                    continue
                pix, rows = B.st_debug_candidates(g.handle, ti - 1, T["C"])
                np.testing.assert_array_equal(pix, T["cand"])
                ref = T["cand_rows"]
                Pmax = max([np.abs(p).max() for p in o.P.values()] + [1.0])
                tol = ULP[dt] * np.abs(ref) + 1e-5 * Pmax
                bad = np.abs(rows - ref) > tol
                assert not bad.any(), (
                    f"tensor {ti}: {bad.sum()} elements beyond one ulp, worst "
                    f"{np.abs(rows - ref).max()}")
                R = B.st_debug_rulebook(g.handle, ti - 1)
                np.testing.assert_array_equal(
                    R.astype(np.int64), o.last["layers"][ti - 1]["rulebook"])
            oo = o.last["out"]
            assert np.abs(out.cpu().numpy() - oo).max() <= \
                1e-5 * np.abs(oo).max() + ULP["f32"]
    finally:
        g.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("name", list(GEOMS))
def test_single_layer(name, dtype):
    net = one_layer(name, dtype)
    say(f"[gpu] single layer {name} {dtype}")
    frames = random_sparse_video(21, 3, 2, 23, 37, net.C, 0.07, dtype=dtype)
    check(net, frames, 0.0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_linear_then_residual(dtype):
    """A linear (non-stateful) layer feeding a 3x3 conv whose residual input
    is the network input: exercises pass-through deltas, the union of
    convolution and residual rows, and the residual add in the epilogue."""
    rng = np.random.default_rng(4)
    C = 16
    l0 = LayerSpec(src=-1, c_in=C, c_out=24, k=(1, 1), s=(1, 1), p=(0, 0),
                   act=ACT_NONE, name="lin")
    l1 = LayerSpec(src=0, c_in=24, c_out=C, k=(3, 3), s=(1, 1), p=(1, 1),
                   act=ACT_RELU, residual_src=-1, name="res")
    for L in (l0, l1):
        L.weight = to_storage(rng.normal(0, 0.2, (L.c_out, L.c_in, *L.k)),
                              dtype)
        L.bias = to_storage(rng.normal(0, 0.1, L.c_out), dtype)
    net = NetSpec("lin_res", [l0, l1], 1, 19, 29, C, dtype)
    say(f"[gpu] linear+residual {dtype}")
    check(net, random_sparse_video(22, 4, 1, 19, 29, C, 0.06, dtype=dtype),
          0.0)


@pytest.mark.parametrize("thr", [0.1, -1.0])
def test_single_layer_thresholds(thr):
    net = one_layer("3x3", "f32")
    frames = random_sparse_video(23, 3, 2, 23, 37, 24, 0.2)
    say(f"[gpu] thresholds {thr}")
    check(net, frames, thr)


def test_empty_delta_frame():
    """A diff frame with no change: zero rows at every stage, no launch
    may read past an empty list."""
    net = one_layer("pool3x3_s2", "f32")
    f = random_sparse_video(24, 1, 2, 23, 37, 8, 0.0)[0]
    check(net, [f, f.copy(), f.copy()], 0.0)


def se_net(dtype, last_se):
    """1x1 expand (SiLU) -> depthwise 3x3 (SiLU) + squeeze-excitation
    [-> linear 1x1 project]: every path of the squeeze-excitation kernels,
    with the gated layer last (output gated) or feeding a 1x1 layer."""
    rng = np.random.default_rng(5)
    C, E, M = 8, 24, 4
    l0 = LayerSpec(src=-1, c_in=C, c_out=E, k=(1, 1), s=(1, 1), p=(0, 0),
                   act=ACT_SILU, name="expand")
    l1 = LayerSpec(src=0, c_in=E, c_out=E, k=(3, 3), s=(1, 1), p=(1, 1),
                   groups=E, act=ACT_SILU, se_mid=M, name="dw_se")
    layers = [l0, l1]
    if not last_se:
        layers.append(LayerSpec(src=1, c_in=E, c_out=C, k=(1, 1), s=(1, 1),
                                p=(0, 0), act=ACT_NONE, residual_src=-1,
                                name="project"))
    for L in layers:
        L.weight = to_storage(rng.normal(0, 0.3, (L.c_out, L.c_in // L.groups,
                                                  *L.k)), dtype)
        L.bias = to_storage(rng.normal(0, 0.1, L.c_out), dtype)
    l1.se_w1 = to_storage(rng.normal(0, 0.3, (M, E)), dtype)
    l1.se_b1 = to_storage(rng.normal(0, 0.1, M), dtype)
    l1.se_w2 = to_storage(rng.normal(0, 0.3, (E, M)), dtype)
    l1.se_b2 = to_storage(rng.normal(1, 0.2, E), dtype)
    return NetSpec("se", layers, 2, 19, 23, C, dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("last_se", [True, False])
def test_squeeze_excitation(dtype, last_se):
    net = se_net(dtype, last_se)
    say(f"[gpu] squeeze-excitation {dtype} last={last_se}")
    frames = random_sparse_video(25, 4, 2, 19, 23, 8, 0.08, dtype=dtype)
    o, g = make_pair(net)
    try:
        o.encode_reference(frames[0])
        out = g.encode_reference(to_dev(frames[0], dtype))
        torch.cuda.synchronize()
        tol = 1e-5 if dtype == "f32" else 2e-2
        assert np.abs(out.cpu().numpy() - o.last["out"]).max() <= \
            tol * np.abs(o.last["out"]).max()
        thr = [0.0] * (len(net.layers) + 1)
        for t in range(1, 4):
            o.encode_diff(frames[t], thr)
            out = g.encode_diff(to_dev(frames[t], dtype), thr)
            torch.cuda.synchronize()
            oo = o.last["out"]
            assert np.abs(out.cpu().numpy() - oo).max() <= \
                tol * np.abs(oo).max()
            for i in o.P:
                Pg = B.st_debug_state(g.handle, i, o.P[i].shape)
                assert np.abs(Pg - o.P[i]).max() <= \
                    tol * np.abs(o.P[i]).max(), f"state {i}"
            T = o.last["tensors"][2]
            pix, rows = B.st_debug_candidates(g.handle, 1, T["C"])
            np.testing.assert_array_equal(pix, T["cand"])  # every site
            sc = np.abs(T["cand_rows"]).max()
            assert np.abs(rows - T["cand_rows"]).max() <= tol * sc + \
                (2.0 ** -7 if dtype != "f32" else 0) * sc
    finally:
        g.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kind", ["conv", "dw"])
def test_large_grid(kind, dtype):
    """A large grid (one layer at 416x416, 173056 sites): hundreds of
    compaction tiles, per-64-row kept counts from the GEMM's last block per
    row tile or from the group-count kernel after a depthwise layer."""
    rng = np.random.default_rng(11)
    H = W = 416
    C = 8 if kind == "conv" else 16
    L = LayerSpec(src=-1, c_in=C, c_out=16, k=(3, 3), s=(1, 1), p=(1, 1),
                  groups=1 if kind == "conv" else 16, act=ACT_RELU, name=kind)
    L.weight = to_storage(rng.normal(0, 0.3, (L.c_out, L.c_in // L.groups,
                                              *L.k)), dtype)
    L.bias = to_storage(rng.normal(0, 0.1, L.c_out), dtype)
    net = NetSpec("large", [L], 1, H, W, C, dtype)
    say(f"[gpu] large tensor {kind} {dtype}")
    frames = random_sparse_video(31, 3, 1, H, W, C, 0.05, dtype=dtype)
    for thr in (0.0, 0.05):
        check(net, frames, thr)
