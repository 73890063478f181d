"""Residual carry (ST_NET_RESIDUAL_CARRY) against the oracle's carry mode:
after every frame the output, every tensor's candidate rows and kept list
(band rows counted and bounded), every layer's state and, while no keep
decision has differed, every layer's consumers' view.  On the GPU's own
state the carry bound |e - view| <= threshold is checked too, for the
layers whose emitted value is the activated state itself."""

import numpy as np
import pytest
import torch

from paper_2410_20790_amd import binding as B
from parity_util import RTOL, run_chunk
from workloads import (crnn_vgg_net, depthwise_test_net,
                       efficientnet_mini_net, random_sparse_video,
                       resnet_mini_net, textline_video, toy_net, toy_video)

pytestmark = pytest.mark.gpu

ACT = {0: lambda x: x, 1: lambda x: np.maximum(x, 0.0),
       2: lambda x: x / (1.0 + np.exp(-x))}


def cases():
    return [
        ("toy", toy_net(), toy_video(seed=5, n_frames=6), 0.05, 0),
        ("resnet_mini f32", resnet_mini_net(),
         random_sparse_video(16, 6, 1, 32, 48, 3, 0.08), 0.05, 0),
        ("resnet_mini bf16", resnet_mini_net(dtype="bf16"),
         random_sparse_video(16, 6, 1, 32, 48, 3, 0.08, dtype="bf16"), 0.05,
         12),
        ("crnn", crnn_vgg_net(), textline_video(seed=5, n_frames=6), 0.02,
         4),
        ("dw", depthwise_test_net(),
         random_sparse_video(17, 6, 1, 24, 40, 16, 0.1), 0.05, 0),
        ("effnet_mini", efficientnet_mini_net(),
         random_sparse_video(18, 6, 1, 32, 40, 3, 0.08), 0.05, 2),
    ]


@pytest.mark.parametrize("name,net,frames,thr,max_band", cases(),
                         ids=[c[0] for c in cases()])
def test_residual_carry_matches_oracle(name, net, frames, thr, max_band):
    o, g = run_chunk(net, frames, thr, f"carry {name}", max_band=max_band,
                     carry=True)
    try:
        torch.cuda.synchronize()
        for i, L in enumerate(net.layers):
            if L.pool_k[0] > 0 or L.se_mid:
                continue
            P = B.st_debug_state(g.handle, i, o.P[i].shape).astype(np.float64)
            V = B.st_debug_carry(g.handle, i, o.Y[i].shape)
            e = ACT[L.act](P).reshape(V.shape)
            gap = float(np.abs(e - V).max())
            slack = RTOL[net.dtype] * max(float(np.abs(e).max()), 1.0)
            assert gap <= thr + slack, f"{name}: layer {i} gap {gap}"
    finally:
        g.close()


def chunk_cases():
    return [
        ("toy", toy_net(), toy_video(seed=7, n_frames=8), 0.05, 3),
        ("resnet_mini f32", resnet_mini_net(),
         random_sparse_video(17, 8, 1, 32, 48, 3, 0.08), 0.05, 3),
        ("crnn", crnn_vgg_net(), textline_video(seed=6, n_frames=9), 0.02, 4),
        ("resnet_mini bf16", resnet_mini_net(dtype="bf16"),
         random_sparse_video(18, 8, 1, 32, 48, 3, 0.08, dtype="bf16"), 0.05,
         3),
    ]


@pytest.mark.parametrize("name,net,frames,thr,F", chunk_cases(),
                         ids=[c[0] for c in chunk_cases()])
def test_residual_carry_in_chunks(name, net, frames, thr, F):
    """The chunk entry with residual carry takes every frame's keep
    decision before forming the site's next frame, so it equals
    frame-by-frame encoding with carry: per frame the kept lists (bit for
    bit) and outputs, after each chunk every state and every consumers'
    view; and the outputs against the oracle's carry mode."""
    import oracle
    from paper_2410_20790_amd import SparseTemNet
    from parity_util import rel, say, to_dev
    dt = net.dtype
    L_n = len(net.layers)
    thr_l = [thr] * (L_n + 1)
    o = oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C, dt,
                         carry=True)
    c = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt,
                     max_frames=F, carry=True)
    f = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt,
                     carry=True)
    tight = 1e-5 if dt == "f32" else RTOL[dt]
    try:
        say(f"[gpu] carry chunks {name}: reference frame")
        o.encode_reference(frames[0])
        c.encode_reference(to_dev(frames[0], dt))
        f.encode_reference(to_dev(frames[0], dt))
        t = 1
        while t < len(frames):
            nf = min(F, len(frames) - t)
            say(f"[gpu] carry chunks {name}: frames {t}..{t + nf - 1}")
            chunk = torch.stack([to_dev(x, dt) for x in frames[t:t + nf]])
            outs = c.encode_chunk(chunk.contiguous(), thr_l)
            torch.cuda.synchronize()
            acts = [B.st_debug_active(c.handle, k - 1)
                    for k in range(L_n + 1)]
            for j in range(nf):
                o.encode_diff(frames[t + j], thr_l)
                out_f = f.encode_diff(to_dev(frames[t + j], dt), thr_l)
                torch.cuda.synchronize()
                e = rel(outs[j].cpu().numpy(), out_f.cpu().numpy())
                assert e <= tight, f"{name} frame {t + j}: chunk vs frames {e}"
                e = rel(outs[j].cpu().numpy(), o.last["out"])
                assert e <= RTOL[dt], f"{name} frame {t + j}: vs oracle {e}"
                for k in range(L_n + 1):
                    npix = int(np.prod(f.tensor_shape(k - 1)[:3]))
                    a = acts[k]
                    mine = np.sort(a[(a >= j * npix) & (a < (j + 1) * npix)]
                                   - j * npix)
                    np.testing.assert_array_equal(
                        mine, B.st_debug_active(f.handle, k - 1),
                        err_msg=f"{name} frame {t + j} tensor {k}")
            for i, L in enumerate(net.layers):
                shape = tuple(f.tensor_shape(i)[:3]) + (L.c_out,)
                Vc = B.st_debug_carry(c.handle, i, shape)
                Vf = B.st_debug_carry(f.handle, i, shape)
                assert rel(Vc, Vf) <= tight, f"{name} view {i}"
            for i in o.P:
                Pc = B.st_debug_state(c.handle, i, o.P[i].shape)
                Pf = B.st_debug_state(f.handle, i, o.P[i].shape)
                assert rel(Pc, Pf) <= tight, f"{name} state {i}"
            t += nf
    finally:
        c.close()
        f.close()
