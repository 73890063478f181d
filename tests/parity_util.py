"""Comparison helpers for the GPU-vs-oracle parity tests.

Tolerances (per tensor, relative to the oracle's largest magnitude):
1e-4 for f32 nets, 2e-2 for f16/bf16 nets; half-precision deltas of stateful
layers are compared layer by layer on identical inputs instead (see
compare_frame and test_gpu_teacher.py).  Masks, active lists and
rulebooks are compared exactly; where a row's keep decision depends on
floating point that the two sides round differently (its max |delta| lies
within a band around the threshold) it is reported and allowed.
"""

import sys

import numpy as np
import torch

import oracle
from paper_2410_20790_amd import SparseTemNet
from paper_2410_20790_amd import binding as B

RTOL = {"f32": 1e-4, "f16": 2e-2, "bf16": 2e-2}
TORCH = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    if a.size == 0 and b.size == 0:
        return 0.0
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-30))


def band(dtype, thr, scale):
    base = max(thr, 1e-3 * scale, 1e-30)
    return (1e-5 if dtype == "f32" else 2.0 ** -7) * base


def to_dev(frame, dtype):
    return torch.from_numpy(np.ascontiguousarray(frame)).to(
        "cuda", TORCH[dtype]).contiguous()


def make_pair(net, carry=False, frozen_se=False, state_bf16=False):
    o = oracle.OracleNet(net.layers, net.batch, net.H, net.W, net.C,
                         net.dtype, carry=carry, frozen_se=frozen_se,
                         state_bf16=state_bf16)
    g = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, net.dtype,
                     carry=carry, frozen_se=frozen_se, bf16_state=state_bf16)
    return o, g


def check_views(net, o, g, tag):
    """Residual carry: every layer's consumers' view on the GPU against the
    oracle's (valid while no keep decision has differed)."""
    for i in range(len(net.layers)):
        V = B.st_debug_carry(g.handle, i, o.Y[i].shape)
        e = rel(V, o.Y[i])
        assert e <= RTOL[net.dtype], f"{tag}: view of layer {i}: {e}"


def compare_frame(net, o, g, out_g, tag, check_rulebook=True, tol_dtype=None):
    """Compare every artefact of the last diff frame.  Returns the number
    of band rows (keep decisions that legitimately differ).  tol_dtype:
    the precision the tolerances and bands are taken at (default: the
    net's storage dtype; "bf16" for a bf16 state, whose values the two
    sides may round to neighbouring bf16 values when their f32 sums differ
    in the last bit)."""
    dt = tol_dtype or net.dtype
    rtol = RTOL[dt]
    out_o = o.last["out"]
    e = rel(out_g.cpu().numpy(), out_o)
    assert e <= rtol, f"{tag}: output rel err {e}"
    n_band = 0
    exact_inputs = True
    L_n = len(net.layers)
    for t in range(L_n + 1):
        T = o.last["tensors"][t]
        layer = t - 1
        act_g = B.st_debug_active(g.handle, layer)
        pix_g, rows_g = B.st_debug_candidates(g.handle, layer, T["C"])
        thr = o.last["thr"][t]
        if t == 0:
            # frame delta: exact masks, exact values (same f32 arithmetic)
            np.testing.assert_array_equal(act_g, T["pix"], err_msg=tag)
            np.testing.assert_array_equal(rows_g.astype(np.float64),
                                          T["rows"], err_msg=tag)
            continue
        if exact_inputs:
            np.testing.assert_array_equal(
                pix_g, T["cand"], err_msg=f"{tag}: candidates of tensor {t}")
        # candidate delta values (before truncation), at the feature-map
        # tolerance relative to the tensor's largest delta.  Half-precision
        # deltas of stateful layers are the exception: a delta
        # f(P_new) - f(P_old) is small next to the state, and in a deep
        # half-precision chain the two sides' re-rounding of every emitted
        # activation moves their states apart by up to ~1% of the state's
        # scale, far more than the delta's own 2e-2.  Those deltas are
        # compared layer by layer on identical inputs instead
        # (test_gpu_teacher.py, at one storage ulp); here the state they are
        # differences of is compared at 2e-2.
        half_state = dt != "f32" and (t - 1) in o.P
        if exact_inputs and len(T["cand"]) and not half_state:
            err = float(np.abs(rows_g - T["cand_rows"]).max())
            bound = rtol * float(np.abs(T["cand_rows"]).max())
            assert err <= bound, (f"{tag}: delta rows of tensor {t}: "
                                  f"{err} > {bound}")
        # kept sets: exact except band rows
        a, b = set(act_g.tolist()), set(T["pix"].tolist())
        diff = a ^ b
        if diff:
            cm = dict(zip(T["cand"].tolist(), T["cand_max"].tolist()))
            scale = max(np.abs(T["cand_max"]).max(), 1e-30)
            bw = band(dt, max(thr, 0.0), scale)
            for p in diff:
                assert abs(cm.get(p, 0.0) - max(thr, 0.0)) <= bw, (
                    f"{tag}: tensor {t} pixel {p} kept on one side only "
                    f"(max {cm.get(p)}, thr {thr})")
            n_band += len(diff)
            exact_inputs = False
        # rulebook of layer t-1 (exact while its input list is exact)
    if check_rulebook:
        check_rulebooks(net, o, g, tag)
    for i, L in enumerate(net.layers):
        if i in o.P:
            Pg = B.st_debug_state(g.handle, i, o.P[i].shape)
            e = rel(Pg, o.P[i])
            assert e <= rtol, f"{tag}: state of layer {i}: {e}"
    return n_band


def check_rulebooks(net, o, g, tag):
    act_equal = [True]
    for t in range(len(net.layers) + 1):
        T = o.last["tensors"][t]
        act_equal.append(np.array_equal(B.st_debug_active(g.handle, t - 1),
                                        T["pix"]))
    for i, L in enumerate(net.layers):
        if not act_equal[L.src + 2]:
            continue
        if L.residual_src != -2 and not act_equal[L.residual_src + 2]:
            continue
        R = B.st_debug_rulebook(g.handle, i)
        np.testing.assert_array_equal(
            R.astype(np.int64), o.last["layers"][i]["rulebook"],
            err_msg=f"{tag}: rulebook of layer {i}")
        pairs, _ = B.st_debug_counters(g.handle, len(net.layers))
        assert pairs[i] == o.last["layers"][i]["pairs"]


def run_chunk(net, frames, thr, tag, max_band=0, carry=False,
              frozen_se=False, state_bf16=False):
    """Encode a chunk on both sides and compare after every frame (with
    carry, also the consumers' views while no keep decision differed)."""
    o, g = make_pair(net, carry, frozen_se, state_bf16)
    tdt = "bf16" if state_bf16 else net.dtype
    try:
        thr_l = [thr] * (len(net.layers) + 1) if np.isscalar(thr) else thr
        say(f"[gpu] {tag}: reference frame")
        out_o = o.encode_reference(frames[0])
        out_g = g.encode_reference(to_dev(frames[0], net.dtype))
        torch.cuda.synchronize()
        e = rel(out_g.cpu().numpy(), out_o)
        assert e <= RTOL[tdt], f"{tag}: reference output {e}"
        for i in o.P:
            Pg = B.st_debug_state(g.handle, i, o.P[i].shape)
            assert rel(Pg, o.P[i]) <= RTOL[tdt], f"{tag}: ref state {i}"
        total_band = 0
        for t in range(1, len(frames)):
            say(f"[gpu] {tag}: diff frame {t}")
            o.encode_diff(frames[t], thr_l)
            out_g = g.encode_diff(to_dev(frames[t], net.dtype), thr_l)
            torch.cuda.synchronize()
            total_band += compare_frame(net, o, g, out_g, f"{tag} f{t}",
                                        tol_dtype=tdt)
            if carry and total_band == 0:
                check_views(net, o, g, f"{tag} f{t}")
            for t2 in range(len(net.layers) + 1):
                dg = g.density(t2 - 1)
                do = o.density(t2)
                N, H, W = o.last["tensors"][t2]["grid"]
                assert abs(dg - do) <= (total_band + 0.5) / (N * H * W)
        assert total_band <= max_band, f"{tag}: {total_band} band rows"
        return o, g
    except BaseException:
        g.close()
        raise
