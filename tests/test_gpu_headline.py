"""The benchmark's headline configuration against the oracle.

ResNet-50 (53 convolutions) in bf16 on 1024x2048x3 frames, 10% of the sites
re-drawn per frame in clustered rectangles, chunks of 10 frames: a dense
reference frame, then the chunk's 9 diff frames in one st_encode_chunk call
on a net created for 9 frames per call -- the launch configuration bench.py
times.  Only this size reaches some paths: compactions whose tiles are cut
at site runs over millions of items, the run-tile pass for lists too long
for whole-site tiles, deep 1x1 layers with hundreds of thousands of rows
over nine frames.

The SparseBatch schedule only reorders the work of the frame-by-frame
definition (section "Design of SparseBatch"), so its result must equal the
oracle run one frame at a time (Eq. 2 on the diff pixels, Eq. 3 at every
non-linear layer).  At threshold 0, per frame: the network output (2e-2
relative), the
frame delta's kept pixels and rows (bit-exact), every tensor's candidate
sites (exact wherever the kept rows of the layer's inputs agree) and kept sites
(exact apart from rows whose keep decision lies within the rounding band of
the threshold, each one checked), the input density; after the chunk,
every cached pre-activation (2e-2 relative).  One frame through the
frame-by-frame entry at the same size is compared the same way.  At
threshold 0.02 every layer of the chunk is checked on the GPU's own inputs
(teacher forcing, as test_gpu_teacher.py does at 64x128).

The oracle's dense reference frame is computed once and copied for each
case.  Where a layer's inputs agree, every row whose keep decision differs
is checked to lie near the threshold; at threshold 0 those are rows whose
largest delta is a few millionths of the tensor's largest (zero on one
side, a rounding residue on the other, where the two sides' bf16 states sit
on either side of a ReLU's kink).  Downstream of such a row the inputs
differ by it and the rows that differ there are counted; all differing
rows together are bounded at 0.5% of the kept rows compared.  (The
teacher-forced tests check every layer of the same chain on identical
inputs at one storage ulp.)
"""

import copy

import numpy as np
import pytest
import torch

import oracle
from paper_2410_20790_amd import SparseTemNet
from paper_2410_20790_amd import binding as B
import test_gpu_teacher as teacher
from parity_util import RTOL, band, compare_frame, rel, say, to_dev
from workloads import driving_video, resnet50_net

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

H, W, CHUNK = 1024, 2048, 10


@pytest.fixture(scope="module")
def headline():
    net = resnet50_net(H=H, W=W)
    frames = driving_video(seed=0, n_frames=CHUNK, H=H, W=W, density=0.10)
    say("[gpu] headline: oracle reference frame (dense, 1024x2048)")
    o = oracle.OracleNet(net.layers, 1, H, W, 3, "bf16")
    o.encode_reference(frames[0])
    o.last = None   # the reference frame's dense activations (GBs) go
    return net, frames, o


def frame_items(a, j, npix):
    """Sites of frame j among chunk items (frame * npix + site), sorted."""
    m = (a >= j * npix) & (a < (j + 1) * npix)
    return np.sort(a[m].astype(np.int64) - j * npix)


def check_kept(mine, ref, T, thr, tag, validate=True):
    """Kept sites: exact, or differing rows near the threshold, each checked
    against the oracle's candidate maximum when `validate` (the layer's
    inputs agree): within 8 bf16 ulps of the threshold (or of the tensor's
    scale at threshold 0) -- the two sides' states drift apart by a few
    ulps over a chunk's frames, so the deltas near the threshold can too.
    Returns the number of differing rows."""
    diff = np.setxor1d(mine, ref)
    if len(diff) and validate:
        cand, cmax = T["cand"], T["cand_max"]
        if len(cand):
            pos = np.clip(np.searchsorted(cand, diff), 0, len(cand) - 1)
            m = np.where(cand[pos] == diff, cmax[pos], 0.0)
            sc = max(float(np.abs(cmax).max()), 1e-30)
        else:
            m, sc = np.zeros(len(diff)), 1e-30
        bw = 16 * band("bf16", max(thr, 0.0), sc)
        bad = np.abs(m - max(thr, 0.0)) > bw
        assert not bad.any(), (f"{tag}: {int(bad.sum())} sites kept on one "
                               f"side only outside the band, e.g. "
                               f"{diff[bad][:5]} (max {m[bad][:5]})")
    return len(diff)


def run_headline_chunk(net, frames, o, thr, n_oracle, max_band):
    """One st_encode_chunk of the 9 diff frames; the oracle follows frame by
    frame for the first n_oracle of them (all 9: the states after the chunk
    are compared too).  max_band: band rows allowed per kept row compared."""
    L_n = len(net.layers)
    thr_l = [thr] * (L_n + 1)
    nf = CHUNK - 1
    g = SparseTemNet(net.layers, 1, H, W, 3, "bf16", max_frames=nf)
    try:
        g.encode_reference(to_dev(frames[0], "bf16"))
        chunk = torch.stack([to_dev(f, "bf16") for f in frames[1:]])
        say(f"[gpu] headline chunk thr={thr}: st_encode_chunk of {nf}")
        outs = g.encode_chunk(chunk.contiguous(), thr_l)
        torch.cuda.synchronize()
        acts = [B.st_debug_active(g.handle, t - 1) for t in range(L_n + 1)]
        cands = [B.st_debug_candidates(g.handle, t - 1, 0, with_rows=False)[0]
                 for t in range(1, L_n + 1)]
        pix0, rows0 = B.st_debug_candidates(g.handle, -1, 3)
        dens0 = [g.density(-1, j) for j in range(nf)]
        n_band, n_casc, n_rows = 0, 0, 0
        for j in range(n_oracle):
            say(f"[gpu] headline chunk thr={thr}: oracle frame {j + 1}")
            out_o = o.encode_diff(frames[j + 1], thr_l)
            e = rel(outs[j].cpu().numpy(), out_o)
            assert e <= RTOL["bf16"], f"frame {j + 1}: output {e}"
            T0 = o.last["tensors"][0]
            npix0 = H * W
            # frame delta: kept pixels and rows bit-exact
            m = (pix0 >= j * npix0) & (pix0 < (j + 1) * npix0)
            p0, r0 = pix0[m].astype(np.int64) - j * npix0, rows0[m]
            order = np.argsort(p0)
            np.testing.assert_array_equal(p0[order], T0["pix"])
            np.testing.assert_array_equal(r0[order].astype(np.float64),
                                          T0["rows"])
            assert abs(dens0[j] - len(T0["pix"]) / npix0) <= 1e-6
            # a tensor's candidates follow from the kept rows of its layer's
            # inputs in the same frame: exact wherever those agree
            same = {0: True}
            fb, fc = 0, 0
            for t in range(1, L_n + 1):
                L = net.layers[t - 1]
                T = o.last["tensors"][t]
                npix = int(np.prod(T["grid"]))
                tag = f"thr={thr} frame {j + 1} tensor {t}"
                inputs_same = same[L.src + 1] and (
                    L.residual_src == -2 or same[L.residual_src + 1])
                if inputs_same:
                    np.testing.assert_array_equal(
                        frame_items(cands[t - 1], j, npix), T["cand"],
                        err_msg=f"{tag}: candidates")
                nb = check_kept(frame_items(acts[t], j, npix), T["pix"], T,
                                o.last["thr"][t], tag, validate=inputs_same)
                n_rows += len(T["pix"])
                same[t] = nb == 0
                if inputs_same:
                    fb += nb
                else:
                    fc += nb
            say(f"[gpu]   frame {j + 1}: {fb} rows kept on one side only "
                f"where the inputs agree, {fc} downstream of those")
            n_band += fb
            n_casc += fc
        if n_oracle == nf:
            for i in o.P:
                Pg = B.st_debug_state(g.handle, i, o.P[i].shape)
                e = rel(Pg, o.P[i])
                assert e <= RTOL["bf16"], f"state of layer {i}: {e}"
        say(f"[gpu] headline chunk thr={thr}: {n_band} band rows and "
            f"{n_casc} downstream of them, of {n_rows} kept rows")
        # every such row was checked one by one above; their number is
        # bounded relative to the rows compared
        assert n_band + n_casc <= max_band * n_rows, \
            f"{n_band} + {n_casc} band rows"
    finally:
        g.close()


def test_headline_chunk_exact(headline):
    """Threshold 0 (the headline's setting): all nine frames against the
    oracle, and the states after the chunk."""
    net, frames, o = headline
    run_headline_chunk(net, frames, copy.deepcopy(o), 0.0, CHUNK - 1,
                       max_band=5e-3)


def test_headline_chunk_teacher_forced():
    """Threshold 0.02 (the configuration's second setting), every layer of
    every frame of the chunk replayed through the oracle's single-layer step
    on the GPU's inputs (its kept rows of the layer's inputs, the state
    carried from the GPU's reference frame): candidates exact, deltas within
    one bf16 ulp, keep decisions exact apart from the rounding band, states
    after the chunk within nine steps' summation-order allowance.  End to
    end at this threshold the two sides' bf16 drift moves rows across the
    threshold in the deep layers; here each layer sees the same inputs."""
    net = resnet50_net(H=H, W=W)
    frames = driving_video(seed=0, n_frames=CHUNK, H=H, W=W, density=0.10)
    teacher.run_chunk(net, frames, 0.02, "headline 1024x2048 thr=0.02",
                      max_band=16, max_band_frac=1e-4)


def test_headline_frame_path(headline):
    """The frame-by-frame entry at the same size: one diff frame against the
    oracle (outputs, candidates, kept lists, states, pair counts)."""
    net, frames, o = headline
    o = copy.deepcopy(o)
    L_n = len(net.layers)
    g = SparseTemNet(net.layers, 1, H, W, 3, "bf16")
    try:
        g.encode_reference(to_dev(frames[0], "bf16"))
        thr_l = [0.0] * (L_n + 1)
        say("[gpu] headline frame path: diff frame 1")
        out_g = g.encode_diff(to_dev(frames[1], "bf16"), thr_l)
        torch.cuda.synchronize()
        o.encode_diff(frames[1], thr_l)
        n_band = compare_frame(net, o, g, out_g, "headline frame 1",
                               check_rulebook=False)
        pairs, _ = B.st_debug_counters(g.handle, L_n)
        if n_band == 0:
            for i in range(L_n):
                assert pairs[i] == o.last["layers"][i]["pairs"], f"layer {i}"
        n_rows = sum(len(o.last["tensors"][t]["pix"]) for t in range(L_n + 1))
        assert n_band <= 5e-3 * n_rows, f"{n_band} band rows of {n_rows}"
    finally:
        g.close()
