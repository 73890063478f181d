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
