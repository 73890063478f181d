"""The entry point that allocates nothing: st_bind_workspace_static binds a
net to the library's own per-device workspace (a static device array of
ST_STATIC_WORKSPACE_BYTES), for callers that cannot allocate device memory.
Its results must equal those of the same net bound to a caller's workspace
(st_bind_workspace): outputs, kept lists and states after a reference frame
and two diff frames, on two bindings in a row -- the second with a smaller
input, over what the first left in the array -- after which the first net,
whose binding was taken over, must refuse to run."""

import numpy as np
import pytest
import torch

from paper_2410_20790_amd import SparseTemNet
from paper_2410_20790_amd import binding as B
from parity_util import say, to_dev
from workloads import toy_net, toy_video

pytestmark = pytest.mark.gpu


def encode(g, net, frames, thr):
    outs = [g.encode_reference(to_dev(frames[0], net.dtype)).cpu().numpy()]
    lists, states = [], []
    for f in frames[1:]:
        outs.append(g.encode_diff(to_dev(f, net.dtype), thr).cpu().numpy())
        torch.cuda.synchronize()
        lists.append([B.st_debug_active(g.handle, t - 1)
                      for t in range(len(net.layers) + 1)])
        states.append(B.st_debug_state(
            g.handle, 1, (net.batch, net.H, net.W, net.layers[1].c_out)))
    return outs, lists, states


@pytest.mark.parametrize("thr", [0.0, 0.05])
def test_static_workspace_matches_caller_workspace(thr):
    first = None
    for k, (H, W) in enumerate(((64, 64), (32, 48))):
        net = toy_net(H=H, W=W)
        frames = toy_video(seed=3 + k, n_frames=3, H=H, W=W)
        thr_l = [thr] * (len(net.layers) + 1)
        say(f"[gpu] static workspace, binding {k + 1}: {H}x{W}")
        s = SparseTemNet(net.layers, 1, H, W, net.C, net.dtype,
                         static_workspace=True)
        assert s.ws_bytes <= B.STATIC_WORKSPACE_BYTES
        got = encode(s, net, frames, thr_l)
        c = SparseTemNet(net.layers, 1, H, W, net.C, net.dtype)
        want = encode(c, net, frames, thr_l)
        c.close()
        for a, b in zip(got[0], want[0]):
            # the same kernels on the same inputs: equal, well inside the
            # 1e-4 relative bar of f32 nets
            assert np.abs(a - b).max() <= 1e-4 * np.abs(b).max()
            np.testing.assert_array_equal(a, b)
        for la, lb in zip(got[1], want[1]):
            for x, y in zip(la, lb):
                np.testing.assert_array_equal(x, y)
        for x, y in zip(got[2], want[2]):
            np.testing.assert_array_equal(x, y)
        if first is not None:
            # the first net's binding was taken over
            with pytest.raises(B.StError) as e:
                first.encode_diff(to_dev(toy_video(seed=9, n_frames=1)[0],
                                         "f32"), [thr] * 3)
            assert e.value.status == B.ST_ERR_STATE
            first.close()
        first = s
    first.close()
