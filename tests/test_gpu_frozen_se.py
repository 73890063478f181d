"""Frozen squeeze-excitation (ST_NET_FROZEN_SE, an approximation) against
the oracle's frozen mode, frame by frame: every artefact of every diff
frame (outputs, candidates, kept lists, states), on the mini EfficientNet
in f32 and f16 and on EfficientNet-B0 at 64x64 f16."""

import pytest

from parity_util import run_chunk
from workloads import (efficientnet_mini_net, efficientnet_net, object_video,
                       random_sparse_video)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,thr", [("f32", 0.0), ("f32", 0.05),
                                       ("f16", 0.05)])
def test_frozen_se_mini(dtype, thr):
    net = efficientnet_mini_net(dtype=dtype)
    frames = random_sparse_video(25, 6, 1, 32, 40, 3, 0.08, dtype=dtype)
    o, g = run_chunk(net, frames, thr, f"frozen se {dtype} thr={thr}",
                     max_band=0 if dtype == "f32" else 6, frozen_se=True)
    g.close()


def test_frozen_se_b0_small():
    net = efficientnet_net(H=64, W=64, dtype="f16")
    frames = object_video(seed=3, n_frames=4, H=64, W=64, obj=8,
                          obj_frac=0.05, dtype="f16")
    o, g = run_chunk(net, frames, 0.02, "frozen se b0 64", max_band=24,
                     frozen_se=True)
    g.close()
