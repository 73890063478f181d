"""Teacher-forced per-layer parity of deep half-precision chains.

End to end, a 53-layer bf16 chain drifts: both sides re-round every emitted
delta to 8 mantissa bits, so after a few layers they no longer see the same
inputs and only state and output are comparable (at 2e-2 relative).  Here
every layer is instead checked on exactly the inputs the GPU gave it: the
GPU's kept rows of the layer's input (and residual input), its cached
pre-activation before the frame (and, for squeeze-excitation, the gates
that state implies), fed to the oracle's single-layer step (Eq. 2 on the
kept pixels, Accumulation, the non-linear handling of Eq. 3).  What the two
sides then differ by is the summation order of one layer alone, so the bar
is the per-kernel one: affected and candidate sites exact, the updated state
within 1e-5 of the layer's state scale, every emitted delta within one
storage ulp plus that, and the kept rows exact apart from rows whose keep
decision lies within the rounding band of the threshold.

Both entries are covered: the frame-by-frame path (st_encode_diff) and the
SparseBatch chunk path (st_encode_chunk), whose frames are replayed through
the oracle's step one at a time on the GPU's per-frame kept rows, with the
state carried from frame to frame on the oracle side (the GPU exposes the
state after the chunk only).
"""

import numpy as np
import pytest
import torch

import oracle
from oracle import sparsetem_oracle as so
from paper_2410_20790_amd import SparseTemNet
from paper_2410_20790_amd import binding as B
from parity_util import band, say, to_dev
from workloads import (depthwise_test_net, driving_video,
                       efficientnet_mini_net, efficientnet_net, object_video,
                       random_sparse_video, resnet50_net, resnet_mini_net)

pytestmark = pytest.mark.gpu

ULP = {"f32": 2.0 ** -23, "f16": 2.0 ** -10, "bf16": 2.0 ** -7}


def gpu_tensors(g, o, nf=1):
    """Per frame j < nf of the last encode, per tensor (index 0 = frame
    delta): the kept sites, their delta rows and all candidates (sites,
    rows).  In a chunk the items are frame * grid + site, in site-major
    order; each tensor is copied from the device once."""
    L_n = len(o.layers)
    frames = [[None] * (L_n + 1) for _ in range(nf)]
    for t in range(L_n + 1):
        grid = int(np.prod(o.shapes[t - 1][:3]))
        kept_all = B.st_debug_active(g.handle, t - 1)
        cpix_all, crows_all = B.st_debug_candidates(g.handle, t - 1,
                                                    o.shapes[t - 1][3])
        for j in range(nf):
            cpix, crows, kept = cpix_all, crows_all, kept_all
            if nf > 1:
                sel = (cpix // grid) == j
                cpix, crows = cpix[sel] - j * grid, crows[sel]
                order = np.argsort(cpix, kind="stable")
                cpix, crows = cpix[order], crows[order]
                kept = kept[(kept // grid) == j] - j * grid
            kept = np.sort(kept)
            pos = np.searchsorted(cpix, kept)
            assert np.array_equal(cpix[pos], kept), "kept rows are candidates"
            frames[j][t] = dict(pix=kept.astype(np.int64),
                                rows=crows[pos].astype(np.float64),
                                cand=cpix.astype(np.int64), cand_rows=crows)
        del kept_all, cpix_all, crows_all
    return frames


def check_layer(o, net, i, st, P_after, T, thr, tag, slack=1.0):
    """One layer's step on the GPU's inputs (st, from the oracle) against
    what the GPU produced (its candidates / kept rows T and, for a stateful
    layer, the state after the step).  `slack` scales the summation-order
    allowance (a chunk's frame j sees states j steps away from the last
    state both sides share).  Returns the band rows."""
    L = net.layers[i]
    dt = net.dtype
    np.testing.assert_array_equal(T["cand"], st["cand"],
                                  err_msg=f"{tag}: candidates of layer {i}")
    if st["P"] is not None:
        scale = max(float(np.abs(st["P"]).max()), 1e-30)
        err = float(np.abs(P_after - st["P"]).max())
        assert err <= 1e-5 * scale, (f"{tag}: state of layer {i}: {err} > "
                                     f"1e-5 * {scale}")
    else:
        scale = max(float(np.abs(st["cand_rows"]).max()), 1e-30)
    ref = st["cand_rows"]
    tol = ULP[dt] * np.abs(ref) + slack * 1e-5 * scale
    bad = np.abs(T["cand_rows"] - ref) > tol
    assert not bad.any(), (
        f"{tag}: layer {i}: {int(bad.sum())} delta elements beyond one ulp, "
        f"worst {float(np.abs(T['cand_rows'] - ref).max())}")
    # keep decisions on the oracle's values of the same inputs
    cmax = np.abs(ref).max(axis=1) if len(ref) else np.zeros(0)
    mine = set(st["cand"][cmax > thr].tolist())
    diff = mine ^ set(T["pix"].tolist())
    if diff:
        cm = dict(zip(st["cand"].tolist(), cmax.tolist()))
        bw = band(dt, max(thr, 0.0), max(float(cmax.max()), 1e-30))
        for p in diff:
            assert abs(cm.get(p, 0.0) - max(thr, 0.0)) <= bw, (
                f"{tag}: layer {i} site {p} kept on one side only "
                f"(max {cm.get(p)}, thr {thr})")
    return len(diff)


def gates_of(net, i, P):
    """The squeeze-excitation gates a layer's cached pre-activation implies
    (what the GPU's gate state follows)."""
    L = net.layers[i]
    return so.se_gates(so.activation(P, L.act), L)


def forced_frame(o, net, T, P_before, thr, tag, j=0, P_after=None):
    """Replay one frame (frame j of a chunk) layer by layer through the
    oracle on the GPU's inputs T (gpu_tensors); returns (band rows, the
    oracle-side states after the frame)."""
    n_band = 0
    states = {}
    for i, L in enumerate(net.layers):
        src = T[L.src + 1]
        skip = T[L.residual_src + 1] if L.residual_src != -2 else None
        P_old = P_before.get(i)
        S_old = gates_of(net, i, P_old) if L.se_mid else None
        st = o.layer_step(i, src["pix"], src["rows"],
                          None if skip is None else skip["pix"],
                          None if skip is None else skip["rows"],
                          P_old, S_old)
        Pa = None
        if st["P"] is not None:
            states[i] = st["P"]
            Pa = P_after[i] if P_after is not None else st["P"]
        # frame j of a chunk: both states before it are j steps from the
        # shared one, each step within the allowance; the delta is a
        # difference of two such states
        n_band += check_layer(o, net, i, st, Pa, T[i + 1], thr[i + 1],
                              f"{tag} layer {i}", slack=2 * j + 1)
    return n_band, states


def gpu_states(net, o, g):
    return {i: B.st_debug_state(g.handle, i, o.shapes_conv[i])
            for i in range(len(net.layers)) if o.stateful[i]}


def prepare(net):
    o = oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C,
                         net.dtype)
    o.shapes_conv = {i: (net.batch, gg.Ho, gg.Wo, L.c_out)
                     for i, (gg, L) in enumerate(zip(o.geo, net.layers))}
    return o


def run_frames(net, frames, thr, tag, max_band):
    o = prepare(net)
    g = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, net.dtype)
    thr_l = [thr] * (len(net.layers) + 1)
    try:
        g.encode_reference(to_dev(frames[0], net.dtype))
        n_band = 0
        for t in range(1, len(frames)):
            say(f"[gpu] teacher-forced {tag}: frame {t}")
            P_before = gpu_states(net, o, g)
            g.encode_diff(to_dev(frames[t], net.dtype), thr_l)
            torch.cuda.synchronize()
            P_after = gpu_states(net, o, g)
            nb, _ = forced_frame(o, net, gpu_tensors(g, o)[0], P_before,
                                 thr_l, f"{tag} f{t}", P_after=P_after)
            n_band += nb
        assert n_band <= max_band, f"{tag}: {n_band} band rows"
    finally:
        g.close()


def run_chunk(net, frames, thr, tag, max_band, max_band_frac=0.0):
    """One reference frame, then frames[1:] as one st_encode_chunk call; the
    frames are replayed one by one, the oracle's states carried along, and
    the state after the chunk compared with the GPU's.  Band rows allowed:
    max_band, plus max_band_frac of the kept rows compared."""
    o = prepare(net)
    nf = len(frames) - 1
    g = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, net.dtype,
                     max_frames=nf)
    thr_l = [thr] * (len(net.layers) + 1)
    try:
        g.encode_reference(to_dev(frames[0], net.dtype))
        torch.cuda.synchronize()
        P = gpu_states(net, o, g)
        say(f"[gpu] teacher-forced {tag}: chunk of {nf}")
        chunk = torch.stack([to_dev(f, net.dtype) for f in frames[1:]])
        g.encode_chunk(chunk.contiguous(), thr_l)
        torch.cuda.synchronize()
        n_band = 0
        Ts = gpu_tensors(g, o, nf)
        n_rows = sum(len(T["pix"]) for Tj in Ts for T in Tj[1:])
        for j in range(nf):
            say(f"[gpu] teacher-forced {tag}: frame {j + 1}")
            nb, P = forced_frame(o, net, Ts[j], P, thr_l, f"{tag} f{j + 1}",
                                 j=j)
            Ts[j] = None
            n_band += nb
        P_gpu = gpu_states(net, o, g)
        for i in P:
            scale = max(float(np.abs(P[i]).max()), 1e-30)
            err = float(np.abs(P_gpu[i] - P[i]).max())
            # nf updates of the same state, each within 1e-5 of its scale
            assert err <= nf * 1e-5 * scale, (
                f"{tag}: state of layer {i} after the chunk: {err}")
        say(f"[gpu] teacher-forced {tag}: {n_band} band rows of {n_rows} "
            "kept rows")
        assert n_band <= max_band + max_band_frac * n_rows, \
            f"{tag}: {n_band} band rows"
    finally:
        g.close()


def test_resnet50_bf16_frames():
    """ResNet-50 (53 convolutions) at 64x128 in bf16, clustered changes,
    frame by frame."""
    net = resnet50_net(H=64, W=128)
    frames = driving_video(seed=2, n_frames=3, H=64, W=128, density=0.10,
                           side=(8, 32))
    run_frames(net, frames, 0.0, "resnet50 64x128 bf16", max_band=16)


@pytest.mark.parametrize("thr", [0.0, 0.02])
def test_resnet50_bf16_chunk(thr):
    """The same net in the SparseBatch schedule (the chunk-state GEMM
    epilogue, the deferred pooled stem, run-aligned tiles): a chunk of 4."""
    net = resnet50_net(H=64, W=128)
    frames = driving_video(seed=5, n_frames=5, H=64, W=128, density=0.10,
                           side=(8, 32))
    run_chunk(net, frames, thr, f"resnet50 64x128 bf16 chunk thr={thr}",
              max_band=32)


def test_efficientnet_b0_f16_frames():
    """EfficientNet-B0 at 64x64 in f16 (expand, depthwise 3x3 / 5x5,
    exact squeeze-excitation, linear projection with skip)."""
    net = efficientnet_net(H=64, W=64, dtype="f16")
    frames = object_video(seed=4, n_frames=3, H=64, W=64, dtype="f16")
    run_frames(net, frames, 0.0, "effnet_b0 64x64 f16", max_band=16)


MINI = {
    "resnet_mini": lambda dt: (resnet_mini_net(dtype=dt, H=40, W=56),
                               random_sparse_video(8, 3, 1, 40, 56, 3, 0.08,
                                                   dtype=dt)),
    "effnet_mini": lambda dt: (efficientnet_mini_net(dtype=dt),
                               random_sparse_video(3, 3, 1, 32, 40, 3, 0.08,
                                                   dtype=dt)),
    "depthwise": lambda dt: (depthwise_test_net(dtype=dt),
                             random_sparse_video(7, 3, 1, 24, 40, 16, 0.1,
                                                 dtype=dt)),
}


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("name", list(MINI))
def test_mini_half_frames(name, dtype):
    """The small half-precision nets of the end-to-end chain tests (ResNet
    layer kinds, MBConv blocks with exact squeeze-excitation, depthwise
    stacks), each layer on identical inputs."""
    net, frames = MINI[name](dtype)
    run_frames(net, frames, 0.0, f"{name} {dtype}", max_band=8)
