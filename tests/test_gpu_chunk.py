"""Chunk mode (st_encode_chunk: a chunk's diff frames encoded layer-major,
the SparseBatch schedule) against the oracle run frame by frame, and
against the library's own frame-by-frame path.  After every chunk: each
frame's output, each frame's kept list of every tensor (rows whose keep
decision rounds differently on the two sides -- their max |delta| within a
band around the threshold -- are counted and bounded) and each frame's
input density; after the chunk, the pre-activation state."""

import numpy as np
import pytest
import torch

import oracle
from paper_2410_20790_amd import SparseTemNet
from paper_2410_20790_amd import binding as B
from parity_util import RTOL, band, rel, say, to_dev
from workloads import (crnn_vgg_net, depthwise_test_net, random_sparse_video,
                       resnet_mini_net, textline_video, to_storage, toy_net,
                       toy_video)

pytestmark = pytest.mark.gpu


def run_chunks(net, frames, thr, F, tag, max_band=0, frozen_se=False):
    dt = net.dtype
    L_n = len(net.layers)
    thr_l = [thr] * (L_n + 1)
    o = oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C, dt,
                         frozen_se=frozen_se)
    g = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt,
                     max_frames=F, frozen_se=frozen_se)
    s = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt,
                     frozen_se=frozen_se)
    try:
        say(f"[gpu] chunk {tag}: reference frame")
        o.encode_reference(frames[0])
        g.encode_reference(to_dev(frames[0], dt))
        s.encode_reference(to_dev(frames[0], dt))
        t, n_band = 1, 0
        while t < len(frames):
            nf = min(F, len(frames) - t)
            say(f"[gpu] chunk {tag}: frames {t}..{t + nf - 1}")
            chunk = torch.stack([to_dev(f, dt) for f in frames[t:t + nf]])
            B.st_profile_begin(g.handle, 1 << 16, 2)
            outs = g.encode_chunk(chunk.contiguous(), thr_l)
            torch.cuda.synchronize()
            _, counts = B.st_profile_end(g.handle, L_n)
            aff_union = [set() for _ in range(L_n)]
            acts = [B.st_debug_active(g.handle, k - 1) for k in range(L_n + 1)]
            dens0 = [g.density(-1, j * net.batch) for j in range(nf)]
            for j in range(nf):
                o.encode_diff(frames[t + j], thr_l)
                out_s = s.encode_diff(to_dev(frames[t + j], dt), thr_l)
                torch.cuda.synchronize()
                oo = o.last["out"]
                e = rel(outs[j].cpu().numpy(), oo)
                assert e <= RTOL[dt], f"{tag} frame {t + j}: output {e}"
                es = rel(outs[j].cpu().numpy(), out_s.cpu().numpy())
                assert es <= (1e-5 if dt == "f32" else RTOL[dt]), \
                    f"{tag} frame {t + j}: chunk vs frame-by-frame {es}"
                for k in range(L_n):
                    aff_union[k] |= set(o.last["layers"][k]["O"].tolist())
                for k in range(L_n + 1):
                    T = o.last["tensors"][k]
                    npix = int(np.prod(T["grid"]))
                    a = acts[k]
                    mine = a[(a >= j * npix) & (a < (j + 1) * npix)] - j * npix
                    diff = set(mine.tolist()) ^ set(T["pix"].tolist())
                    if diff:
                        cm = dict(zip(T["cand"].tolist(),
                                      T["cand_max"].tolist()))
                        sc = max(np.abs(T["cand_max"]).max(), 1e-30)
                        bw = band(dt, max(thr, 0.0), sc)
                        for p in diff:
                            assert abs(cm.get(p, 0.0) - max(thr, 0.0)) <= bw, (
                                f"{tag} frame {t + j} tensor {k}: pixel {p} "
                                "kept on one side only")
                        n_band += len(diff)
                N, H, W = o.last["tensors"][0]["grid"]
                d0 = np.sum(o.last["tensors"][0]["pix"] < H * W) / float(H * W)
                assert abs(dens0[j] - d0) <= 1e-6 + n_band / (H * W)
            # sites whose state a fused epilogue (or a pooled layer's)
            # updated: the union of the layer's affected outputs over the
            # chunk's frames
            for j in range(L_n):
                if counts[0, j, 6] and max_band == 0:
                    assert counts[0, j, 6] == len(aff_union[j]), (
                        f"{tag} chunk at {t}: layer {j} sites")
            for i in o.P:
                Pg = B.st_debug_state(g.handle, i, o.P[i].shape)
                e = rel(Pg, o.P[i])
                assert e <= RTOL[dt], f"{tag} after frame {t + nf - 1}: " \
                    f"state {i} {e}"
            t += nf
        assert n_band <= max_band, f"{tag}: {n_band} band rows"
    finally:
        g.close()
        s.close()


@pytest.mark.parametrize("thr", [0.0, 0.05])
def test_chunk_toy(thr):
    run_chunks(toy_net(), toy_video(seed=3, n_frames=9), thr, 4,
               f"toy thr={thr}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_chunk_resnet_mini(dtype):
    """7x7/2 stem with an overlapping 3x3/2 max-pool (the chunk pool path),
    bottlenecks with downsample and identity shortcuts."""
    net = resnet_mini_net(dtype=dtype)
    run_chunks(net, random_sparse_video(12, 8, 1, 32, 48, 3, 0.08,
                                        dtype=dtype),
               0.0, 3, f"resnet_mini {dtype}",
               max_band=0 if dtype == "f32" else 8)


def test_chunk_crnn():
    """Four max-pools (2x2/2 and 2x1), thresholds above zero."""
    run_chunks(crnn_vgg_net(), textline_video(seed=5, n_frames=11), 0.02, 5,
               "crnn thr=0.02", max_band=4)


def test_chunk_depthwise():
    net = depthwise_test_net()
    run_chunks(net, random_sparse_video(13, 7, 1, 24, 40, 16, 0.1), 0.0, 6,
               "depthwise")


def pointwise_first_net(seed=1031):
    """1x1 stride-1 layers first: one fed by the frame delta, one fed by a
    layer's kept rows (the two ways a 1x1 layer's list is formed in a
    chunk), then a 3x3 layer and a 1x1 output layer."""
    from workloads.nets import ACT_NONE, ACT_RELU, LayerSpec, NetSpec
    rng = np.random.default_rng(seed)

    def conv(src, cin, cout, k, act):
        L = LayerSpec(src=src, c_in=cin, c_out=cout, k=(k, k), s=(1, 1),
                      p=(k // 2, k // 2), act=act)
        L.weight = rng.normal(0.0, 0.15, (cout, cin, k, k)).astype(np.float32)
        L.bias = rng.normal(0.0, 0.1, (cout,)).astype(np.float32)
        return L
    layers = [conv(-1, 16, 32, 1, ACT_RELU), conv(0, 32, 32, 1, ACT_RELU),
              conv(1, 32, 16, 3, ACT_RELU), conv(2, 16, 8, 1, ACT_NONE)]
    return NetSpec("pointwise_first", layers, 1, 64, 64, 16, "f32")


@pytest.mark.parametrize("thr", [0.0, 0.05])
def test_chunk_pointwise_layers(thr):
    """Row tiles of the fused 1x1 layers: cut by a pass of their own (fed
    by the frame delta) and by the producer's list compaction; chunks of
    4, 4 and 1 frames."""
    run_chunks(pointwise_first_net(), toy_video(seed=21, n_frames=10), thr,
               4, f"pointwise thr={thr}")


def test_chunk_single_frame_and_batch():
    """A batch of two images (items are frames x images), and a last chunk
    of one frame."""
    from dataclasses import replace
    net = replace(resnet_mini_net(), batch=2)
    frames = random_sparse_video(14, 4, 2, 32, 48, 3, 0.1)
    run_chunks(net, frames, 0.0, 2, "batch 2")


def test_chunk_frozen_se():
    """Squeeze-excitation with the reference frame's gates (an
    approximation) batches like any layer: the mini EfficientNet in chunks
    of 3, against the oracle's frozen mode and the frame-by-frame path."""
    from workloads import efficientnet_mini_net
    net = efficientnet_mini_net()
    run_chunks(net, random_sparse_video(24, 8, 1, 32, 40, 3, 0.08), 0.02, 3,
               "frozen se", max_band=2, frozen_se=True)


@pytest.mark.parametrize("dtype,thr", [("f32", 0.0), ("f32", 0.05),
                                       ("f16", 0.0)])
def test_chunk_exact_se(dtype, thr):
    """Exact squeeze-excitation inside a chunk: for each frame in turn the
    squeeze over the sites that frame updated, the excitation from the
    moved channel sums and the emission at every site, f(P_t) s_t -
    f(P_{t-1}) s_{t-1} (the mini EfficientNet in chunks of 3, against the
    oracle and the frame-by-frame path)."""
    from workloads import efficientnet_mini_net
    net = efficientnet_mini_net(dtype=dtype)
    run_chunks(net, random_sparse_video(25, 8, 1, 32, 40, 3, 0.08,
                                        dtype=dtype),
               thr, 3, f"exact se {dtype} thr={thr}",
               max_band=0 if (dtype == "f32" and thr == 0.0) else 8)


def test_chunk_b0_exact_se():
    """All 16 MBConv blocks of EfficientNet-B0 at 64x64 fp16 with exact
    squeeze-excitation, chunks of 4 and a ragged last chunk, on the
    detection-like video."""
    from workloads import efficientnet_net, object_video
    net = efficientnet_net(H=64, W=64)
    frames = object_video(seed=1, n_frames=7, H=64, W=64, obj=8)
    run_chunks(net, frames, 0.02, 4, "effnet-b0 64x64 f16 exact se",
               max_band=128)


def test_chunk_resnet50_full_size():
    """ResNet-50 at 1024x2048 bf16 with 10% clustered change in the launch
    configuration the benchmark times (a reference frame, then the chunk's
    9 diff frames in one call): every frame's input kept list equals the
    frame-by-frame path's bit for bit, every frame's output equals it within
    the bf16 tolerance, and the last frame's output equals the dense pass
    of that frame (threshold 0; properties that hold at any size)."""
    from workloads import driving_video, resnet50_net
    net = resnet50_net()
    frames = driving_video(seed=2, n_frames=10, density=0.10)
    thr = [0.0] * (len(net.layers) + 1)
    g = SparseTemNet(net.layers, 1, 1024, 2048, 3, "bf16", max_frames=9)
    s = SparseTemNet(net.layers, 1, 1024, 2048, 3, "bf16")
    d = SparseTemNet(net.layers, 1, 1024, 2048, 3, "bf16")
    try:
        say("[gpu] chunk resnet50 full: reference frame")
        g.encode_reference(to_dev(frames[0], "bf16"))
        s.encode_reference(to_dev(frames[0], "bf16"))
        chunk = torch.stack([to_dev(f, "bf16") for f in frames[1:]])
        say("[gpu] chunk resnet50 full: chunk of 9")
        outs = g.encode_chunk(chunk.contiguous(), thr)
        torch.cuda.synchronize()
        act_c = B.st_debug_active(g.handle, -1)
        npix = 1024 * 2048
        for j in range(9):
            out_s = s.encode_diff(to_dev(frames[1 + j], "bf16"), thr)
            torch.cuda.synchronize()
            mine = np.sort(act_c[(act_c >= j * npix) &
                                 (act_c < (j + 1) * npix)] - j * npix)
            np.testing.assert_array_equal(mine, B.st_debug_active(s.handle,
                                                                   -1))
            e = rel(outs[j].cpu().numpy(), out_s.cpu().numpy())
            assert e <= RTOL["bf16"], f"frame {j + 1}: chunk vs frames {e}"
        dense = d.encode_reference(to_dev(frames[9], "bf16"))
        torch.cuda.synchronize()
        e = rel(outs[8].cpu().numpy(), dense.cpu().numpy())
        assert e <= RTOL["bf16"], f"last frame vs dense pass {e}"
    finally:
        g.close()
        s.close()
        d.close()


def long_reduction_net(dtype, seed=1733):
    """Layers on the 128x128-tile gather-GEMM: a 3x3 256->256 layer and a
    1x1 2048->128 layer (long reductions, output channels a multiple of
    128) between ordinary ones, all half-precision."""
    from workloads.nets import ACT_NONE, ACT_RELU, LayerSpec, NetSpec
    rng = np.random.default_rng(seed)

    def conv(src, cin, cout, k, act, gain=1.0):
        L = LayerSpec(src=src, c_in=cin, c_out=cout, k=(k, k), s=(1, 1),
                      p=(k // 2, k // 2), act=act)
        std = gain * np.sqrt(2.0 / (cin * k * k))
        L.weight = to_storage(rng.normal(0.0, std, (cout, cin, k, k)), dtype)
        L.bias = to_storage(rng.normal(0.0, 0.05, (cout,)), dtype)
        return L
    layers = [conv(-1, 16, 256, 1, ACT_RELU), conv(0, 256, 256, 3, ACT_RELU),
              conv(1, 256, 2048, 1, ACT_RELU),
              conv(2, 2048, 128, 1, ACT_RELU),
              conv(3, 128, 64, 1, ACT_NONE, gain=0.5)]
    return NetSpec(f"long_reduction_{dtype}", layers, 1, 40, 56, 16, dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_chunk_long_reductions(dtype):
    """128x128 tiles: two run-aligned row tiles per GEMM tile, each
    finished by the chunk-state epilogue (ragged last tiles, chunks of 4 and
    a last chunk of 2), against the oracle frame by frame and the
    frame-by-frame path."""
    net = long_reduction_net(dtype)
    frames = random_sparse_video(31, 7, 1, 40, 56, 16, 0.1, dtype=dtype)
    run_chunks(net, frames, 0.0, 4, f"long reductions {dtype}", max_band=8)


def _conv_state_shape(g, net, i):
    """Shape of layer i's pre-activation state: its convolution's output
    grid (before any pooling) by its output channels."""
    L = net.layers[i]
    N, H, W, _ = g.tensor_shape(L.src)
    Ho = (H + 2 * L.p[0] - L.k[0]) // L.s[0] + 1
    Wo = (W + 2 * L.p[1] - L.k[1]) // L.s[1] + 1
    return (N, Ho, Wo, L.c_out)


@pytest.mark.parametrize("which", ["toy", "resnet_mini", "long_reductions"])
def test_graph_replay_chunk_matches_eager(which):
    """A chunk encode (st_encode_chunk) captured once as a HIP graph and
    replayed for consecutive chunks, and again after a reference frame
    encoded directly, gives bitwise the eager net's results: every frame's
    output, the kept and candidate lists of every tensor, and every
    layer's state after each chunk (each replay separated by eager work
    and a synchronisation).  The replays rerun the same compactions, whose
    look-back statuses alternate between two sets that each compaction
    clears for the next."""
    F = 4
    if which == "toy":
        net, frames, thr = toy_net(), toy_video(seed=21, n_frames=14), 0.0
    elif which == "resnet_mini":
        net = resnet_mini_net()
        frames = random_sparse_video(22, 14, 1, 32, 48, 3, 0.08)
        thr = 0.0
    else:
        net = long_reduction_net("bf16")
        frames = random_sparse_video(23, 14, 1, 40, 56, 16, 0.1,
                                     dtype="bf16")
        thr = 0.0
    dt = net.dtype
    L_n = len(net.layers)
    thr_l = [thr] * (L_n + 1)
    ge = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt,
                      max_frames=F)
    gg = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt,
                      max_frames=F)
    try:
        say(f"[gpu] chunk graph replay {which}")
        dev = [to_dev(f, dt) for f in frames]
        ge.encode_reference(dev[0])
        gg.encode_reference(dev[0])
        torch.cuda.synchronize()
        slot = torch.zeros((F,) + tuple(gg.in_shape), dtype=gg.tdtype,
                           device=gg.device)
        out_g = torch.empty((F,) + tuple(gg.out_shape), dtype=torch.float32,
                            device=gg.device)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            gg.encode_chunk(slot, thr_l, out=out_g)
        # chunks at frames 1 and 5 back to back, a reference frame at 9
        # encoded directly, a chunk at 10
        for t in (1, 5, 9, 10):
            if t == 9:
                ge.encode_reference(dev[t])
                gg.encode_reference(dev[t])
                torch.cuda.synchronize()
                continue
            chunk = torch.stack(dev[t:t + F]).contiguous()
            out_e = ge.encode_chunk(chunk, thr_l)
            torch.cuda.synchronize()
            slot.copy_(chunk)
            graph.replay()
            torch.cuda.synchronize()
            np.testing.assert_array_equal(out_g.cpu().numpy(),
                                          out_e.cpu().numpy(),
                                          err_msg=f"{which} chunk at {t}")
            for k in range(L_n + 1):
                np.testing.assert_array_equal(
                    B.st_debug_active(gg.handle, k - 1),
                    B.st_debug_active(ge.handle, k - 1),
                    err_msg=f"{which} chunk at {t}: kept list {k}")
                C = ge.tensor_shape(k - 1)[3]
                pg, rg = B.st_debug_candidates(gg.handle, k - 1, C)
                pe, re_ = B.st_debug_candidates(ge.handle, k - 1, C)
                np.testing.assert_array_equal(pg, pe)
                np.testing.assert_array_equal(rg, re_)
            n_state = 0
            for i in range(L_n):
                shape = _conv_state_shape(ge, net, i)
                try:
                    Pe = B.st_debug_state(ge.handle, i, shape)
                except B.StError:
                    continue  # a layer without state
                Pg = B.st_debug_state(gg.handle, i, shape)
                np.testing.assert_array_equal(
                    Pg, Pe, err_msg=f"{which} chunk at {t}: state {i}")
                n_state += 1
            assert n_state >= 1, f"{which}: no state compared"
    finally:
        ge.close()
        gg.close()
