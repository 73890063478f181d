"""Online threshold adjustment on the device (st_set_threshold_control /
st_encode_diff_adaptive) against the host controller: the host controller
is fed the kept-row counters of a second net that encodes the same frames
with the host's thresholds.  Both take the same f64 bisection steps from
the same counts, so every frame's thresholds must be bit-equal, and with
equal thresholds the deterministic kernels give bit-equal outputs.  Cycles
restart at every reference frame on both sides."""

import numpy as np
import pytest
import torch

from paper_2410_20790_amd import SparseTemNet
from paper_2410_20790_amd import binding as B
from paper_2410_20790_amd.ibst import (IBST, nonlinear_tensors,
                                       sparsity_from_counts)
from parity_util import say, to_dev
from workloads import efficientnet_mini_net, efficientnet_net, object_video

pytestmark = pytest.mark.gpu


def run_pair(net, frames, chunk, tag, target=0.7, eps=0.05, theta_max=0.5,
             fixed=0.01):
    dt = net.dtype
    L_n = len(net.layers)
    ctl = nonlinear_tensors(net.layers)
    host = IBST(L_n + 1, ctl, target, eps, theta_max, fixed=fixed)
    d = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt)
    h = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt)
    try:
        d.set_threshold_control(ctl, [fixed] * (L_n + 1), target, eps,
                                theta_max)
        grids = [int(np.prod(h.tensor_shape(k - 1)[:3]))
                 for k in range(L_n + 1)]
        seen = set()
        for t, f in enumerate(frames):
            x = to_dev(f, dt)
            if t % chunk == 0:
                say(f"[gpu] {tag}: reference frame {t}")
                d.encode_reference(x)
                h.encode_reference(x)
                host.start_cycle()
                continue
            thr_h = np.array(host.thresholds(), dtype=np.float32)
            thr_d = d.thresholds()
            assert np.array_equal(thr_d, thr_h), f"{tag} frame {t}"
            seen.add(tuple(thr_h.tolist()))
            say(f"[gpu] {tag}: frame {t} thr[0:3]={thr_h[:3]}")
            out_d = d.encode_diff_adaptive(x)
            out_h = h.encode_diff(x, host.thresholds())
            torch.cuda.synchronize()
            assert torch.equal(out_d, out_h), f"{tag} frame {t}: output"
            _, act = B.st_debug_counters(h.handle, L_n)
            host.update(sparsity_from_counts(act, grids))
        # the search moved the thresholds, and the last frame's step is
        # visible too
        assert len(seen) > 2, f"{tag}: thresholds never moved"
        assert np.array_equal(d.thresholds(),
                              np.array(host.thresholds(), np.float32))
    finally:
        d.close()
        h.close()


@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_device_controller_matches_host(dtype):
    net = efficientnet_mini_net(dtype=dtype)
    frames = object_video(seed=4, n_frames=13, H=32, W=40, obj=8,
                          obj_frac=0.1, dtype=dtype)
    run_pair(net, frames, 6, f"device ibst {dtype}")


def test_device_controller_efficientnet_b0_full_size():
    """EfficientNet-B0 at 512x512 f16 on the detection-like video, the
    launch configuration the bench measures (target 0.9)."""
    net = efficientnet_net(H=512, W=512, dtype="f16")
    frames = object_video(seed=0, n_frames=9, H=512, W=512, dtype="f16")
    run_pair(net, frames, 8, "device ibst b0 512", target=0.9, eps=0.025,
             theta_max=1.0, fixed=0.0)


def run_chunk_pair(net, frames, F, cycle_refs, tag, target=0.7, eps=0.05,
                   theta_max=0.5, fixed=0.01, frozen_se=False):
    """Reference frame, then the next F frames as one chunk, repeated.  The
    device takes one step per chunk from the chunk's kept rows over
    sites x frames and restarts its search every cycle_refs reference
    frames; the host controller, fed a second net's counts (the same chunk
    with the host's thresholds), does the same."""
    dt = net.dtype
    L_n = len(net.layers)
    ctl = nonlinear_tensors(net.layers)
    host = IBST(L_n + 1, ctl, target, eps, theta_max, fixed=fixed)
    kw = dict(max_frames=F, frozen_se=frozen_se)
    d = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt, **kw)
    h = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt, **kw)
    try:
        d.set_threshold_control(ctl, [fixed] * (L_n + 1), target, eps,
                                theta_max, cycle_refs=cycle_refs)
        grids = [int(np.prod(h.tensor_shape(k - 1)[:3]))
                 for k in range(L_n + 1)]
        seen, t, n_ref = set(), 0, 0
        while t < len(frames):
            say(f"[gpu] {tag}: reference frame {t}")
            x = to_dev(frames[t], dt)
            d.encode_reference(x)
            h.encode_reference(x)
            if n_ref % cycle_refs == 0:
                host.start_cycle()
            n_ref += 1
            t += 1
            nf = min(F, len(frames) - t)
            if nf == 0:
                break
            thr_h = np.array(host.thresholds(), dtype=np.float32)
            assert np.array_equal(d.thresholds(), thr_h), f"{tag} frame {t}"
            seen.add(tuple(thr_h.tolist()))
            say(f"[gpu] {tag}: chunk {t}..{t + nf - 1} thr[0:3]={thr_h[:3]}")
            chunk = torch.stack([to_dev(f, dt) for f in frames[t:t + nf]])
            out_d = d.encode_chunk(chunk.contiguous(), None)
            out_h = h.encode_chunk(chunk.contiguous(), host.thresholds())
            torch.cuda.synchronize()
            assert torch.equal(out_d, out_h), f"{tag} chunk at {t}: output"
            _, act = B.st_debug_counters(h.handle, L_n)
            host.update(sparsity_from_counts(act, [g * nf for g in grids]))
            t += nf
        assert len(seen) > 2, f"{tag}: thresholds never moved"
        assert np.array_equal(d.thresholds(),
                              np.array(host.thresholds(), np.float32))
    finally:
        d.close()
        h.close()


@pytest.mark.parametrize("cycle_refs", [1, 3])
def test_device_controller_chunks(cycle_refs):
    """One step per chunk: a cycle of one reference frame takes a single
    step before its restart (brackets reset, theta carried on); a cycle of
    three takes three.  Frozen squeeze-excitation, so the mini EfficientNet
    batches; chunks of 4 with a ragged last one."""
    net = efficientnet_mini_net()
    frames = object_video(seed=6, n_frames=22, H=32, W=40, obj=8,
                          obj_frac=0.1)
    run_chunk_pair(net, frames, 4, cycle_refs,
                   f"chunk ibst cycle {cycle_refs}", frozen_se=True)
