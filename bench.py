#!/usr/bin/env python3
"""Benchmark of the diff-computation encoder on one MI355X.

One step = one diff frame through the whole hot path (frame-delta mask and
compaction, and for every layer rulebook, gather-GEMM / depthwise conv with
the fused state update and delta emission, pool handling, truncation), plus
the dense network output, on synthetic temporally continuous video resident
in HBM.  Default workload: ResNet-50 encoder, bf16 storage, 1024x2048x3
frames, 10% of the sites re-drawn per frame in clustered rectangles,
threshold 0 (exact).

Prints one JSON line with diff-frames/s (value), algorithmic TFLOP/s,
speedup over dense convolution of the same net (MIOpen through PyTorch, and
the library's own dense pass), the roofline of the dominant kernel from HIP
events recorded around every launch in a second timed pass, and the CPU
oracle's rate on the host cores.
"""

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("diff-frames/sec + effective TFLOP/s at 10% change density; "
          "speedup vs dense")
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f16": 2500.0, "f32": 157.3}
ESIZE = {"f32": 4, "f16": 2, "bf16": 2}


def log(msg):
    """Progress of the run, on stderr (stdout ends with the one result
    line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def workload(name, density):
    """Network, synthetic video and run shape of a named workload.  `chunk`
    is the number of frames per reference frame (None: one reference, then
    diff frames only); `ibst` selects online threshold adjustment."""
    from workloads import (crnn_vgg_net, driving_video, efficientnet_net,
                           multistream_video, object_video, resnet50_net,
                           textline_video, toy_net, toy_video)
    if name == "resnet50":
        net = resnet50_net(H=1024, W=2048)
        return dict(
            net=net, desc=f"resnet50-bf16-1024x2048-density{density:g}",
            frames=lambda n, H=1024, W=2048: driving_video(
                seed=0, n_frames=n, H=H, W=W, density=density),
            crop=(256, 512), chunk=10, ibst=False)
    if name == "effnet_b0":
        net = efficientnet_net(H=512, W=512, dtype="f16")
        return dict(
            net=net, desc="efficientnet_b0-f16-512x512-objects-ibst0.9",
            frames=lambda n: object_video(seed=0, n_frames=n, H=512, W=512,
                                          dtype="f16"),
            crop=None, chunk=8, ibst=True)
    if name == "multistream":
        net = efficientnet_net(H=256, W=256, dtype="bf16", batch=32)
        wl = dict(net=net,
                  desc="efficientnet_b0x32-bf16-256x256-streams-ibst0.9",
                  crop=None, chunk=8, ibst=True)

        def frames(n):
            f, d = multistream_video(n_frames=n, N=32, H=256, W=256)
            wl["stream_density_targets"] = [float(v) for v in d]
            return f
        wl["frames"] = frames
        return wl
    if name == "crnn":
        net = crnn_vgg_net()
        return dict(net=net, desc="crnn_vgg-f32-32x128-band7",
                    frames=lambda n, H=32, W=128: textline_video(
                        seed=0, n_frames=n, H=H, W=W),
                    crop=None, chunk=16, ibst=False)
    if name == "toy":
        net = toy_net()
        return dict(net=net, desc="toy-f32-64x64x16-density0.1",
                    frames=lambda n, H=64, W=64: toy_video(
                        seed=0, n_frames=n, H=H, W=W), crop=None,
                    chunk=4, ibst=False)
    raise SystemExit(f"unknown workload {name}")


def dense_flops(net, shapes):
    tot = 0
    for i, L in enumerate(net.layers):
        N, Ho, Wo = shapes[i]
        tot += 2 * N * Ho * Wo * L.c_out * (L.c_in // L.groups) * \
            L.k[0] * L.k[1]
    return tot


def conv_launch_bytes(L, c, es, mode):
    """Algorithmic HBM bytes of one conv launch (gather-GEMM or depthwise)
    with fused epilogue, from the frame's counters
    c = (affected outputs, pairs, kept input rows, candidate rows, kept
    rows, kept residual rows, updated sites of a chunk): every kept input
    row and the weights read once, the neighbour table and output list read
    once, the f32 state read and written and the delta written once per
    affected output row (or the deferred f32 update written, for pooled
    layers; in a chunk's fused epilogue the delta written per row and the
    state read and written once per site; in a pooled layer's chunk
    epilogue the f32 state after each frame written per row and the state
    read once per site), the residual rows read once."""
    nO, pairs, n_in, _, _, n_skip = (int(v) for v in c[:6])
    sites = int(c[6]) if len(c) > 6 else 0
    K = L.k[0] * L.k[1]
    b = n_in * L.c_in * es + K * (L.c_in // L.groups) * L.c_out * es
    b += nO * (K + 1) * 4
    if mode == "state":
        b += nO * L.c_out * (4 + 4 + es)
    elif mode == "fused":
        b += nO * L.c_out * es + sites * L.c_out * (4 + 4)
    elif mode == "fused_pool":
        b += nO * L.c_out * 4 + sites * L.c_out * 4
    elif mode == "defer":
        b += nO * L.c_out * 4
    else:
        b += nO * L.c_out * es
    b += n_skip * L.c_out * es
    return b


def layer_mode(net, i):
    L = net.layers[i]
    if L.pool_k[0] > 0 or L.se_mid:
        return "defer"
    if L.act != 0 or i == len(net.layers) - 1:
        return "state"
    return "linear"


def torch_dense_model(net, dtype):
    import torch
    import torch.nn.functional as F
    tdt = {"f32": torch.float32, "f16": torch.float16,
           "bf16": torch.bfloat16}[dtype]
    Ws = [torch.as_tensor(L.weight).to("cuda", tdt).contiguous(
        memory_format=torch.channels_last) for L in net.layers]
    Bs = [torch.as_tensor(L.bias).to("cuda", tdt) for L in net.layers]
    SE = {i: [torch.as_tensor(getattr(L, k)).to("cuda", tdt)
              for k in ("se_w1", "se_b1", "se_w2", "se_b2")]
          for i, L in enumerate(net.layers) if L.se_mid}

    def fwd(x_nhwc):
        acts = {-1: x_nhwc.permute(0, 3, 1, 2)}
        for i, L in enumerate(net.layers):
            y = F.conv2d(acts[L.src], Ws[i], Bs[i], L.s, L.p, 1, L.groups)
            if L.residual_src != -2:
                y = y + acts[L.residual_src]
            if L.act == 1:
                y = F.relu(y)
            elif L.act == 2:
                y = F.silu(y)
            if L.pool_k[0] > 0:
                y = F.max_pool2d(y, L.pool_k, L.pool_s, L.pool_p)
            if L.se_mid:
                w1, b1, w2, b2 = SE[i]
                z = F.silu(F.linear(y.mean(dim=(2, 3)), w1, b1))
                y = y * torch.sigmoid(F.linear(z, w2, b2))[:, :, None, None]
            acts[i] = y
        return acts[len(net.layers) - 1]
    return fwd


def time_gpu(fn, reps, warm=2):
    import torch
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        torch.cuda.synchronize()
        ts.append(a.elapsed_time(b))
    return statistics.median(ts)


def cpu_baseline(wl, net, thr_val, n_diff=2, single_thread=True):
    """The oracle (numpy, fp64 accumulation) on the host cores, on a bounded
    sample of the same workload: a spatial crop of the same synthetic video
    (full frames when the workload is small), one untimed reference frame
    and `n_diff` timed diff frames; the rate is scaled to full frames by
    the pixel ratio.  Timed with the BLAS thread pool as it comes (every
    core the process may use) and, with single_thread, again with one
    thread.  `cores` is the number of threads the timed run used: the BLAS
    pool's (the oracle's products); its element-wise numpy steps run on
    one thread."""
    import oracle
    from threadpoolctl import threadpool_info, threadpool_limits
    crop = wl["crop"]
    frames = wl["frames"](n_diff + 1)
    H, W = net.H, net.W
    if crop:
        # the crop position whose change density over the diff frames is
        # closest to the full frame's (changes are clustered, so an
        # arbitrary corner can be far from representative)
        h, w = crop
        ch = [np.any(frames[t] != frames[t - 1], axis=-1)
              for t in range(1, n_diff + 1)]
        full = np.mean([c.mean() for c in ch])
        best = None
        for y in range(0, H - h + 1, h // 2):
            for x in range(0, W - w + 1, w // 2):
                dd = np.mean([c[:, y:y + h, x:x + w].mean() for c in ch])
                if best is None or abs(dd - full) < best[0]:
                    best = (abs(dd - full), y, x)
        _, y0, x0 = best
        frames = [np.ascontiguousarray(f[:, y0:y0 + h, x0:x0 + w, :])
                  for f in frames]
    else:
        h, w = H, W
    thr = [thr_val] * (len(net.layers) + 1)

    def timed():
        o = oracle.OracleNet(net.layers, net.batch, h, w, net.C, net.dtype)
        o.encode_reference(frames[0])
        dens = []
        t0 = time.perf_counter()
        for t in range(1, n_diff + 1):
            o.encode_diff(frames[t], thr)
            dens.append(o.density(0))
        return (time.perf_counter() - t0) / n_diff, float(np.mean(dens))

    dt, dens = timed()
    scale = (h * w) / float(H * W)
    threads = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    res = {"value": scale / dt, "unit": "diff-frames/s", "cores": threads,
           "kind": "oracle",
           "sample": (f"{n_diff} diff frames of a {h}x{w} "
                      + ("crop" if crop else "frame")
                      + f" (density {dens:.3f}) after an untimed reference, "
                      f"{dt:.2f} s/frame, scaled by {scale:g}"),
           "affinity_cores": len(os.sched_getaffinity(0)),
           "s_per_sample_frame": dt}
    if single_thread:
        with threadpool_limits(limits=1):
            dt1, _ = timed()
        res["single_thread"] = {"value": scale / dt1,
                                "s_per_sample_frame": dt1}
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                res["cpu_model"] = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return res


COPY_BYTES = 256 << 20


def copy_calibration():
    """A plain device-to-device copy of COPY_BYTES, launched 10 times: the
    reference whose FETCH_SIZE / WRITE_SIZE counters convert the conv
    kernel's counter readings into bytes."""
    import torch
    x = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(10):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "launches": 10}))


def measured_peaks():
    """The box's own ceilings beside the published ones: a STREAM-like
    device copy of 1 GiB (read + write bytes over the time of one copy,
    best of 10 HIP-event-timed copies) and a large bf16 matrix product
    (8192^3 on the library GEMM, the MFMA-bound ceiling a practical kernel
    reaches; best of 5)."""
    import torch
    n = (1 << 30) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    y.copy_(x)

    def best(fn, reps):
        t = []
        for _ in range(reps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            t.append(a.elapsed_time(b) * 1e-3)
        return min(t)

    copy_s = best(lambda: y.copy_(x), 10)
    del x, y
    m = 8192
    a = torch.randn(m, m, dtype=torch.bfloat16, device="cuda")
    b = torch.randn(m, m, dtype=torch.bfloat16, device="cuda")
    c = a @ b
    gemm_s = best(lambda: torch.matmul(a, b, out=c), 5)
    del a, b, c
    torch.cuda.empty_cache()
    return {"copy_GBps": 2.0 * (1 << 30) / copy_s / 1e9,
            "bf16_gemm_TFLOPs": 2.0 * m ** 3 / gemm_s / 1e12,
            "published": {"hbm_GBps": HBM_PEAK_GBS,
                          "bf16_mfma_TFLOPs": MFMA_PEAK_TFLOPS["bf16"]}}


def kernel_source_hash():
    import hashlib
    src = os.path.join(ROOT, "paper_2410_20790_amd", "csrc",
                       "st_kernels.hip")
    return hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]


def measured_traffic(workload_desc, kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary
    (profiles/hbm_traffic.json), or None when it is missing, was taken on
    another workload, or the kernel source changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    try:
        d = json.load(open(path))
    except (OSError, ValueError):
        return None
    e = d.get(workload_desc, {}).get(kernel)
    if not e or e.get("source_hash") != kernel_source_hash():
        return None
    return e.get("bytes_per_launch")


KCLASS = {"k_conv_gemm": "conv_gemm", "k_conv_gemm_big": "conv_gemm",
          "k_conv_dw": "conv_dw",
          "k_split_epi": "conv_split_epi", "k_pool_emit": "pool_emit",
          "k_commit": "commit", "k_output": "output",
          "k_se_squeeze": "se_squeeze", "k_se_emit": "se_emit",
          "k_chunk_update": "chunk_update",
          "k_chunk_pool_emit": "chunk_pool_emit",
          "k_chunk_commit": "chunk_commit"}


# the compactions by predicate (pool-site compactions share FlagPred with
# the rulebooks)
PCLASS = {"ScanPred": "scan_compact", "ChunkScanPred": "chunk_scan_compact",
          "FlagPred": "flag_compact", "ListPred": "list_compact"}


def demangle(name):
    """The readable name of a kernel symbol (the counter files name some
    kernels by their mangled symbol)."""
    if not name.startswith("_Z"):
        return name
    import subprocess
    try:
        r = subprocess.run(["c++filt", name], capture_output=True, text=True)
        out = r.stdout.strip()
    except OSError:
        out = ""
    if out and out != name:
        return out
    return demangle_st(name)


def demangle_st(name):
    """Enough of the Itanium mangling for this library's kernel templates
    (c++filt does not know _Float16's DF16_): st::<name><args>, the
    arguments being the storage types, predicate structs and bools/ints."""
    import re
    m = re.match(r"_ZN2st(\d+)", name)
    if not m:
        return name
    n = int(m.group(1))
    i = m.end()
    fn = name[i:i + n]
    rest = name[i + n:]
    if not rest.startswith("I"):
        return f"st::{fn}"
    types = {"DF16_": "_Float16", "f": "float", "NS_6bf16_tE": "st::bf16_t"}
    args, j = [], 1
    while j < len(rest) and rest[j] != "E":
        if rest.startswith("Lb", j):
            args.append("true" if rest[j + 2] == "1" else "false")
            j = rest.index("E", j) + 1
            continue
        if rest.startswith("Li", j):
            k = rest.index("E", j)
            args.append(rest[j + 2:k])
            j = k + 1
            continue
        for code, t in types.items():
            if rest.startswith(code, j):
                args.append(t)
                j += len(code)
                break
        else:
            mm = re.match(r"NS_(\d+)", rest[j:])
            if not mm:
                break
            ln = int(mm.group(1))
            k = j + mm.end()
            sname = "st::" + rest[k:k + ln]
            k += ln
            if rest.startswith("I", k):  # the struct's own type argument
                for code, t in types.items():
                    if rest.startswith(code, k + 1):
                        sname += f"<{t}>"
                        k += 1 + len(code)
                        break
                k = rest.index("E", k) + 1
            if rest.startswith("E", k):
                k += 1
            args.append(sname)
            j = k
    return f"st::{fn}<{', '.join(args)}>"


def kernel_class(kernel_name):
    """Kernel class of a traced kernel name, None for kernels outside the
    diff pass (reference-pass instantiations, library kernels)."""
    head = demangle(kernel_name).split("(")[0]
    if head.startswith("void "):
        head = head[5:]
    fn = head.split("<")[0].split("::")[-1]
    targs = (head.split("<", 1)[1].rstrip(">").split(", ")
             if "<" in head else [])
    if fn == "k_compact":
        return PCLASS.get(targs[0].split("<")[0].split("::")[-1])
    if fn == "k_chunk_scan_prep":
        return "chunk_scan_mask"
    if fn == "k_chunk_xhat_commit":
        return "chunk_xhat_commit"
    if fn not in KCLASS:
        return None
    if fn in ("k_conv_gemm", "k_conv_dw", "k_split_epi") and \
            targs[1:2] == ["true"]:
        return None  # reference-pass instantiations
    return KCLASS[fn]


def ingest_mfma(base, workload_name, density, schedule=None):
    """MFMA utilisation of the diff-pass gather-GEMM from one rocprofv3
    --pmc run (DIR/pmc_mfma): per dispatch, the cycles the MFMA units were
    busy summed over every SIMD over (GPU-active cycles x 1024 SIMDs), the
    MFMA work issued (MOPS x 512 FLOP) and its rate over the dispatch's
    duration; averaged over the dispatches of each kernel build.  Written to
    profiles/mfma_util.json with the kernel source hash."""
    import csv
    import collections
    path = os.path.join(base, "pmc_mfma", "run_counter_collection.csv")
    disp = collections.defaultdict(dict)
    names = {}
    for r in csv.DictReader(open(path)):
        raw = r["Kernel_Name"]
        if raw not in names:
            names[raw] = demangle(raw).split("(")[0].replace("void ", "")
        name = names[raw]
        if not name.startswith("st::k_conv_gemm"):
            continue
        d = disp[r["Dispatch_Id"]]
        d["name"] = name
        d["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + \
            float(r["Counter_Value"])
    per = collections.defaultdict(list)
    for d in disp.values():
        per[d["name"]].append(d)
    # GRBM_GUI_ACTIVE is summed over the 8 XCDs (each counts the
    # dispatch's active cycles); the MFMA busy cycles over all 1024 SIMDs
    simds, xcds = 256 * 4, 8
    out = {}
    for name, ds in sorted(per.items()):
        busy = sum(d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) for d in ds)
        act = sum(d.get("GRBM_GUI_ACTIVE", 0.0) for d in ds) / xcds
        mops = sum(d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) +
                   d.get("SQ_INSTS_VALU_MFMA_MOPS_F16", 0.0) for d in ds)
        ns = sum(d["ns"] for d in ds)
        out[name] = {"dispatches": len(ds),
                     "mfma_busy_frac": busy / max(act * simds, 1.0),
                     "mfma_gflop_per_dispatch": mops * 512 / len(ds) / 1e9,
                     "mfma_tflops": mops * 512 / max(ns, 1) / 1e3,
                     "avg_dispatch_us": ns / len(ds) / 1e3}
    wl = workload(workload_name, density)
    out_path = os.path.join(ROOT, "profiles", "mfma_util.json")
    try:
        dd = json.load(open(out_path))
    except (OSError, ValueError):
        dd = {}
    dd[f"{wl['desc']}-{default_schedule(wl, schedule)}"] = {
        "source_hash": kernel_source_hash(), "kernels": out}
    json.dump(dd, open(out_path, "w"), indent=1, sort_keys=True)
    for name, v in out.items():
        print(f"| `{name}` | {v['dispatches']} | {v['avg_dispatch_us']:.1f} "
              f"| {100 * v['mfma_busy_frac']:.1f}% | "
              f"{v['mfma_gflop_per_dispatch']:.2f} | {v['mfma_tflops']:.1f} |")


def ingest_counters(base, workload_name, density, schedule=None):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE (KiB) of the diff-pass kernels,
    scaled by what the same counters read for a plain copy of COPY_BYTES,
    averaged per launch; written to profiles/hbm_traffic.json with the
    kernel source hash."""
    import csv
    import collections

    def rows(name):
        path = os.path.join(base, name, "run_counter_collection.csv")
        return list(csv.DictReader(open(path)))

    scale = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        # the copy calibration of this run, else the one beside it
        cal = f"pmc_copy_{c}"
        if not os.path.isdir(os.path.join(base, cal)):
            cal = os.path.join("..", cal)
        v = [float(r["Counter_Value"]) for r in rows(cal)
             if "copyBuffer" in r["Kernel_Name"]]
        scale[c] = (COPY_BYTES / 1024.0) / (sum(v) / len(v))
    per = collections.defaultdict(lambda: collections.defaultdict(list))
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        for r in rows(f"pmc_bench_{c}"):
            k = kernel_class(r["Kernel_Name"])
            if k:
                per[k][c].append(float(r["Counter_Value"]))
    wl = workload(workload_name, density)
    out_path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    try:
        d = json.load(open(out_path))
    except (OSError, ValueError):
        d = {}
    entry = {}
    for k, v in per.items():
        f = sum(v["FETCH_SIZE"]) / max(len(v["FETCH_SIZE"]), 1)
        w = sum(v["WRITE_SIZE"]) / max(len(v["WRITE_SIZE"]), 1)
        entry[k] = {"bytes_per_launch": 1024.0 * (f * scale["FETCH_SIZE"] +
                                                  w * scale["WRITE_SIZE"]),
                    "fetch_kib_raw": f, "write_kib_raw": w,
                    "launches": len(v["FETCH_SIZE"]),
                    "scale": scale, "source_hash": kernel_source_hash()}
    d[f"{wl['desc']}-{default_schedule(wl, schedule)}"] = entry
    json.dump(d, open(out_path, "w"), indent=1, sort_keys=True)
    print(json.dumps(entry))


def density_sweep(net, thr, densities, steps, chunk, schedule):
    """diff-frames/s and algorithmic TFLOP/s at several change densities of
    the same video recipe, in the given schedule (each: a reference frame
    and one warm-up chunk, then `steps` timed diff frames in chunks of
    `chunk` frames, reference frames synchronised around and left out)."""
    import torch
    from paper_2410_20790_amd import SparseTemNet
    from paper_2410_20790_amd import binding as B
    from workloads import driving_video
    tdt = torch.bfloat16 if net.dtype == "bf16" else torch.float32
    batch = chunk - 1 if schedule == "chunk" else 1
    out = {}
    g = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, net.dtype,
                     max_frames=batch)
    o = torch.empty((batch,) + tuple(g.out_shape), dtype=torch.float32,
                    device="cuda")
    if batch == 1:
        o = o[0]
    L_n = len(net.layers)
    thr_l = [thr] * (L_n + 1)
    for d in densities:
        fr_np = driving_video(seed=7, n_frames=frames_needed(
            chunk, chunk - 1, steps, 0), H=net.H, W=net.W, density=d)
        fr = torch.empty((len(fr_np), net.batch, net.H, net.W, net.C),
                         dtype=tdt, device="cuda")
        for i, f in enumerate(fr_np):
            fr[i].copy_(torch.from_numpy(f))
        del fr_np
        feed = Feed(g, L_n, fr, chunk, thr_l, None, o, batch)
        run_diffs(feed, chunk - 1)
        wall, _ = run_diffs(feed, steps)
        ms = wall * 1000.0 / steps
        pairs, _ = B.st_debug_counters(g.handle, L_n)
        fl = sum(2 * int(pairs[j]) * (L.c_in // L.groups) * L.c_out
                 for j, L in enumerate(net.layers)) / feed.last_m
        out[f"{d:g}"] = {"ms_per_frame": ms, "diff_frames_per_s": 1000.0 / ms,
                         "input_density": g.density(-1),
                         "alg_gflop": fl / 1e9,
                         "effective_tflops": fl / (ms * 1e-3) / 1e12}
        del fr
    g.close()
    return out


class Feed:
    """Walks a synthetic video: a reference frame every `chunk` frames (only
    the first frame when chunk is None), diff frames in between.  With
    `batch` > 1 (the SparseBatch schedule) the diff frames of a chunk are
    encoded up to `batch` at a time by one st_encode_chunk call, else one
    st_encode_diff call per frame.  ctl = "device": the thresholds are
    adjusted on the device (st_encode_diff_adaptive, or
    st_encode_chunk_adaptive with one step per chunk; no host round trip);
    ctl = a host controller: each diff frame's thresholds come from it and
    its kept-row counters are fed back after the frame (one host round trip
    per frame, part of the timed work)."""

    def __init__(self, g, n_layers, frames, chunk, thr, ctl, out, batch=1):
        from paper_2410_20790_amd import binding as B
        self.B = B
        self.replay = None     # a captured diff-frame graph, when set
        self.g, self.frames, self.chunk = g, frames, chunk
        self.thr, self.ctl, self.out = thr, ctl, out
        self.batch = batch
        if batch > 1 and ctl not in (None, "device"):
            raise ValueError("the host controller adjusts thresholds per "
                             "frame")
        self.device_ctl = ctl == "device"
        if self.device_ctl:
            self.ctl = None
        self.pos = 0
        self.L_n = n_layers
        self.grids = [int(np.prod(g.tensor_shape(t - 1)[:3]))
                      for t in range(self.L_n + 1)]
        self.sparsity = []     # per diff frame, every tensor

    def next_is_ref(self):
        return self.pos == 0 or bool(self.chunk and self.pos % self.chunk == 0)

    def ref(self):
        if self.ctl:
            self.ctl.start_cycle()
        self.g.encode_reference(self.frames[self.pos],
                                out=self.out[0] if self.batch > 1
                                else self.out)
        self.pos += 1

    def diff(self, limit=1):
        """Encode up to `limit` diff frames (at most to the next reference
        frame); returns how many."""
        from paper_2410_20790_amd.ibst import sparsity_from_counts
        if self.batch > 1:
            m = min(limit, self.batch)
            if self.chunk:
                m = min(m, self.chunk - self.pos % self.chunk)
            self.g.encode_chunk(self.frames[self.pos:self.pos + m],
                                None if self.device_ctl else self.thr,
                                out=self.out[:m])
            self.pos += m
            self.last_m = m
            return m
        thr = self.ctl.thresholds() if self.ctl else self.thr
        if self.replay is not None:
            self.replay(self.frames[self.pos])
        elif self.device_ctl:
            self.g.encode_diff_adaptive(self.frames[self.pos], out=self.out)
        else:
            self.g.encode_diff(self.frames[self.pos], thr, out=self.out)
        self.pos += 1
        self.last_m = 1
        if self.ctl:
            _, act = self.B.st_debug_counters(self.g.handle, self.L_n)
            sp = sparsity_from_counts(act, self.grids)
            self.sparsity.append(sp)
            self.ctl.update(sp)
        return 1


def run_diffs(feed, n):
    """Encode frames until `n` diff frames are done.  Returns the wall
    seconds spent in diff frames (reference frames in between are
    synchronised around and left out) and the reference frames' ms."""
    import torch
    total, refs, done = 0.0, [], 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while done < n:
        if feed.next_is_ref():
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            total += t1 - t0
            feed.ref()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            refs.append((t0 - t1) * 1000.0)
        else:
            done += feed.diff(n - done)
    torch.cuda.synchronize()
    total += time.perf_counter() - t0
    return total, refs


def frames_needed(chunk, W, K, KP, KG=0, align=False):
    """Frames consumed by the warm-up (W; with align, continued to the end
    of its chunk), timed (K), profiled (KP) and graph-replay (KG) passes,
    reference frames included."""
    pos = 0

    def is_ref(p):
        return p == 0 or bool(chunk and p % chunk == 0)

    def diffs(n):
        nonlocal pos
        d = 0
        while d < n:
            d += 0 if is_ref(pos) else 1
            pos += 1
    diffs(W)
    if align and chunk:
        while not is_ref(pos):
            pos += 1
    diffs(K)
    if chunk:  # the profiled frames start with a reference frame
        while not is_ref(pos):
            pos += 1
        pos += 1
    pos += KP
    diffs(KG)
    return pos


def kernel_table(net, recs, counts, es, chunk_mode=False, nf=1):
    """Per kernel class: launches, time, algorithmic bytes / FLOPs from the
    frame's counters (see conv_launch_bytes).  In chunk mode a profiled
    "frame" is one chunk of nf frames (counters summed over its frames); a
    stateful layer whose GEMM epilogue applies the chunk's updates is
    charged its delta rows and one state read and write per updated site,
    the others write f32 update rows.

    The other kernels' bytes are their minimal traffic from the same
    counters: every item a compaction pass visits read once (a keep byte or
    a row maximum), every kept item's list, map and neighbour entries
    written once; the chunk update reads each updated site's state once and
    each update row once, writes each delta row (or, before a pool, each
    per-frame state) once and each updated site's state once, the output
    layer's update also every site's state and dense output per frame; the
    pool emission writes each pooled row once and reads the states of the
    conv sites its window adds over the previous pooled site (stride area)
    for both frame states; the commit reads each updated site's last state
    and writes it once."""
    from paper_2410_20790_amd import binding as B
    classes = {}
    n_in = net.batch * net.H * net.W
    seen = set()
    for r in recs:
        name = B.KERNEL_CLASSES[r["kernel"]]
        c = classes.setdefault(name, {"launches": 0, "ms": 0.0, "bytes": 0.0,
                                      "flops": 0.0})
        c["launches"] += 1
        c["ms"] += float(r["ms"])
        f, j = int(r["frame"]), int(r["layer"])
        if f >= len(counts):
            continue
        L = net.layers[j] if j >= 0 else None
        cnt = counts[f, j] if j >= 0 else None
        if name in ("conv_gemm", "conv_dw"):
            mode = layer_mode(net, j)
            if chunk_mode and mode == "state":
                mode = "fused" if counts[f, j, 6] > 0 else "defer"
            elif chunk_mode and L.pool_k[0] > 0 and counts[f, j, 6] > 0:
                mode = "fused_pool"
            c["bytes"] += conv_launch_bytes(L, cnt, es, mode)
            c["flops"] += 2.0 * cnt[1] * (L.c_in // L.groups) * L.c_out
        elif name in ("se_squeeze", "se_emit"):
            # squeeze: the site map, and f32 state and update rows of the
            # affected sites; emit: the state and map of every site, update
            # rows, the delta and row bookkeeping of every site written,
            # and the affected state rows written back
            npix = int(np.prod(net_conv_grid(net, j)))
            nO = int(cnt[0])
            if name == "se_squeeze":
                b = npix * 4 + nO * L.c_out * 8
            else:
                b = npix * (L.c_out * (4 + es) + 16) + nO * L.c_out * 8
            c["bytes"] += b
        elif name == "chunk_update":
            nO, sites = int(cnt[0]), int(cnt[7])
            npix = int(np.prod(net_conv_grid(net, j)))
            pool = L.pool_k[0] > 0
            b = nO * (4 + 4 * L.c_out)             # list + update rows read
            if sites:                              # walks the affected list
                b += sites * L.c_out * 4           # state read
                if pool:
                    b += nO * L.c_out * 4 + sites * 4   # P_t rows, frame bits
                else:
                    b += nO * (L.c_out * es + 4) + sites * L.c_out * 4
            else:                                  # every site (output)
                b += nf * npix * 4 + npix * L.c_out * 4      # maps, state
                b += nf * npix * L.c_out * 4                 # dense output
                b += nO * (L.c_out * es + 4) + min(nO, npix) * L.c_out * 4
            c["bytes"] += b
        elif name == "commit":
            if chunk_mode:
                sites = int(cnt[6]) + int(cnt[7])
                c["bytes"] += int(cnt[0]) * 4 + sites * (L.c_out * 8 + 4)
            else:
                c["bytes"] += int(cnt[0]) * (4 + L.c_out * 12)
        elif name == "pool_emit":
            nQ = int(cnt[3])
            area = L.pool_s[0] * L.pool_s[1]
            c["bytes"] += nQ * (4 + L.c_out * es + 4) + \
                nQ * area * 2 * L.c_out * 4
        elif name in ("rb_count", "pool_count"):
            npix = int(np.prod(net_conv_grid(net, j)))
            if name == "pool_count":
                g = net_out_grid(net, j)
                npix = int(np.prod(g))
            c["bytes"] += npix * nf                       # flag bytes
        elif name in ("rb_compact", "pool_compact"):
            npix = int(np.prod(net_conv_grid(net, j)))
            K = L.k[0] * L.k[1]
            if name == "pool_compact":
                npix = int(np.prod(net_out_grid(net, j)))
                kept, K = int(cnt[3]), 0
            else:
                kept = int(cnt[0])
            # flags read; per kept item list, map, row maximum written and
            # the flag cleared; neighbour entries written and input map read
            c["bytes"] += npix * nf + kept * (13 + 8 * K)
        elif name == "list_count":
            n = int(cnt[3])
            c["bytes"] += n * 4 + (n // 64 + 1) * 4
        elif name == "list_compact":
            n, kept = int(cnt[3]), int(cnt[4])
            # row maximum and row site read per candidate; kept list written
            # per kept row, the map cleared per dropped row; consumers'
            # affected-output marks or identity lists (12 bytes) per kept row
            c["bytes"] += n * 8 + kept * 16 + (n - kept) * 4
        elif name in ("scan_mask", "scan_compact") and (name, f) in seen:
            continue  # a chunk's second kernel of the class: charged once
        elif name == "scan_mask":
            # frames and X_hat read; keep bytes written (a chunk: also the
            # base-frame and last-frame bytes)
            C = net.C
            seen.add((name, f))
            c["bytes"] += n_in * ((2 * C * es + 1) if not chunk_mode else
                                  (nf * C * es + C * es + 2 * nf + 1))
        elif name == "scan_compact":
            seen.add((name, f))
            n0 = int(counts[f, 0, 2]) if net.layers[0].src == -1 else 0
            C, Cp = net.C, (net.C + 7) // 8 * 8
            if chunk_mode:
                # keep bytes read; per kept item its frame and reference
                # value read, the delta row and list, map entries written;
                # X_hat committed at the changed sites (bounded by the kept
                # items)
                c["bytes"] += n_in * nf + n0 * (2 * C * es + Cp * es + 12) \
                    + min(n0, n_in) * 2 * C * es
            else:
                # frame and X_hat read at every site (the mask); per kept
                # pixel the delta row and list, map entries written and
                # X_hat committed
                c["bytes"] += n_in * 2 * C * es + n0 * (Cp * es + 12 +
                                                        C * es)
    return classes


def net_out_grid(net, j):
    """(N, Hp, Wp) of layer j's emitted tensor (after its pool)."""
    N, Ho, Wo = net_conv_grid(net, j)
    L = net.layers[j]
    if L.pool_k[0] > 0:
        Ho = (Ho + 2 * L.pool_p[0] - L.pool_k[0]) // L.pool_s[0] + 1
        Wo = (Wo + 2 * L.pool_p[1] - L.pool_k[1]) // L.pool_s[1] + 1
    return (N, Ho, Wo)


_GRIDS = {}


def net_conv_grid(net, j):
    """(N, Ho, Wo) of layer j's convolution output."""
    key = (id(net), j)
    if key not in _GRIDS:
        shapes = {-1: (net.H, net.W)}
        for i, L in enumerate(net.layers):
            Hi, Wi = shapes[L.src]
            Ho = (Hi + 2 * L.p[0] - L.k[0]) // L.s[0] + 1
            Wo = (Wi + 2 * L.p[1] - L.k[1]) // L.s[1] + 1
            _GRIDS[(id(net), i)] = (net.batch, Ho, Wo)
            if L.pool_k[0] > 0:
                Ho = (Ho + 2 * L.pool_p[0] - L.pool_k[0]) // L.pool_s[0] + 1
                Wo = (Wo + 2 * L.pool_p[1] - L.pool_k[1]) // L.pool_s[1] + 1
            shapes[i] = (Ho, Wo)
    return _GRIDS[key]


def event_overhead_us(reps=50):
    """Median time an event pair reports around one minimal kernel when the
    host is ahead of the device (the stream is first kept busy for a few ms,
    as in the timed passes): the dispatch latency that every per-launch
    event pair also encloses, which a kernel trace does not count."""
    import torch
    x = torch.zeros(1, device="cuda")
    busy = torch.empty(64 << 20, device="cuda")
    for _ in range(20):
        busy.fill_(1.0)
    evs = []
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        x.add_(1.0)
        b.record()
        evs.append((a, b))
    torch.cuda.synchronize()
    del busy
    return statistics.median(a.elapsed_time(b) * 1000.0 for a, b in evs)


def roofline_of(classes, dt, desc):
    dom = max(classes, key=lambda k: classes[k]["ms"])
    dc = classes[dom]
    avg_s = dc["ms"] * 1e-3 / dc["launches"]
    if not (dc["bytes"] or dc["flops"]):
        return {"kernel": dom, "bound": None, "launches": dc["launches"],
                "avg_launch_us": avg_s * 1e6}
    ai = dc["flops"] / max(dc["bytes"], 1.0)
    ridge = MFMA_PEAK_TFLOPS[dt] * 1e12 / (HBM_PEAK_GBS * 1e9)
    if dc["flops"] and ai > ridge:
        ach = dc["flops"] / dc["launches"] / avg_s / 1e12
        roof = {"bound": "mfma", "achieved": ach,
                "peak": MFMA_PEAK_TFLOPS[dt], "unit": "TFLOP/s",
                "frac": ach / MFMA_PEAK_TFLOPS[dt], "traffic": None}
    else:
        ach = dc["bytes"] / dc["launches"] / avg_s / 1e9
        roof = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": ach / HBM_PEAK_GBS, "traffic": None}
    tb = measured_traffic(desc, dom)
    if tb is not None:
        roof["traffic"] = tb
    roof.update({"kernel": dom, "launches": dc["launches"],
                 "avg_launch_us": avg_s * 1e6,
                 "alg_bytes_per_launch": dc["bytes"] / dc["launches"],
                 "alg_flops_per_launch": dc["flops"] / dc["launches"],
                 "arith_intensity": ai})
    return roof


def measure(wl, K, W, KP, thr_val, dense=True, target=0.9, eps=0.025,
            schedule="frame", frozen_se=False, thr_list=None,
            ibst=None, bf16_state=False):
    """Time K diff frames of a workload (after W warm-up diff frames), then
    KP more with an event pair around every launch; dense comparators on
    the same net.  schedule "chunk" encodes each chunk's diff frames in one
    st_encode_chunk call (SparseBatch; KP becomes one whole chunk),
    "frame" one st_encode_diff call per frame."""
    import torch
    from paper_2410_20790_amd import SparseTemNet
    from paper_2410_20790_amd import binding as B
    from paper_2410_20790_amd.ibst import nonlinear_tensors
    net = wl["net"]
    dt = net.dtype
    es = ESIZE[dt]
    chunk = wl["chunk"]
    batch = chunk - 1 if schedule == "chunk" else 1
    if schedule == "chunk":
        KP = batch
    elif chunk:
        KP = min(KP, chunk - 1)
    # graph replay of the per-frame launch sequence (fixed or device-adjusted
    # thresholds, any layer kind)
    use_ibst = wl["ibst"] if ibst is None else ibst
    KG = K if schedule == "frame" else 0
    t_gen = time.perf_counter()
    frames_np = wl["frames"](frames_needed(chunk, W, K, KP, KG,
                                           align=schedule == "chunk"))
    t_gen = time.perf_counter() - t_gen
    tdt = {"f32": torch.float32, "f16": torch.float16,
           "bf16": torch.bfloat16}[dt]
    # one resident [n, N, H, W, C] tensor: frame i and chunk slices of it
    # are contiguous views
    frames = torch.empty((len(frames_np), net.batch, net.H, net.W, net.C),
                         dtype=tdt, device="cuda")
    for i, f in enumerate(frames_np):
        frames[i].copy_(torch.from_numpy(f))
    del frames_np
    g = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt,
                     max_frames=batch, frozen_se=frozen_se,
                     bf16_state=bf16_state)
    L_n = len(net.layers)
    thr = list(thr_list) if thr_list is not None else [thr_val] * (L_n + 1)
    if batch > 1:
        out = torch.empty((batch,) + tuple(g.out_shape),
                          dtype=torch.float32, device="cuda")
        out0 = out[0]
    else:
        out = out0 = g.new_output()
    ctl = None
    ctl_idx = nonlinear_tensors(net.layers)
    if use_ibst:
        # the online threshold adjustment runs on the device; a chunk is
        # one step, so a search spans chunk - 1 reference periods (as many
        # steps as frame by frame)
        g.set_threshold_control(ctl_idx, thr, target, eps, 1.0,
                                cycle_refs=batch)
        ctl = "device"
    feed = Feed(g, L_n, frames, chunk, thr, ctl, out, batch)
    dflops = dense_flops(net, [net_conv_grid(net, i) for i in range(L_n)])

    run_diffs(feed, W)  # reference frame + warm-up
    if schedule == "chunk":
        # the warm-up finishes its chunk, so that the timed frames start at
        # a chunk boundary (whole chunks, the last one possibly shorter)
        while not feed.next_is_ref():
            feed.diff(chunk)

    # ---- timed region: K diff frames (reference frames of later chunks
    # are synchronised around and excluded)
    s_ev = torch.cuda.Event(enable_timing=True)
    e_ev = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s_ev.record()
    wall, refs = run_diffs(feed, K)
    e_ev.record()
    torch.cuda.synchronize()
    ms_step = wall * 1000.0 / K
    ev_ms = s_ev.elapsed_time(e_ev) / K if not refs else None
    dens0 = g.density(-1)

    # ---- profiled diff frames: an event pair around every launch
    if chunk:
        while not feed.next_is_ref():
            feed.diff(chunk)
        feed.ref()
    B.st_profile_begin(g.handle, KP * 1024, KP + 1)
    torch.cuda.synchronize()
    tp = time.perf_counter()
    done = 0
    while done < KP:
        done += feed.diff(KP - done)
    torch.cuda.synchronize()
    prof_ms_step = (time.perf_counter() - tp) * 1000.0 / KP
    recs, counts = B.st_profile_end(g.handle, L_n)
    # per diff frame (a profiled record of the chunk schedule is a chunk)
    alg_flops = sum(
        2 * int(counts[f, j, 1]) * (L.c_in // L.groups) * L.c_out
        for f in range(len(counts))
        for j, L in enumerate(net.layers)) / KP
    classes = kernel_table(net, recs, counts, es,
                           chunk_mode=schedule == "chunk",
                           nf=batch if schedule == "chunk" else 1)
    total_ms = sum(c["ms"] for c in classes.values())
    kern = {}
    for name, c in sorted(classes.items(), key=lambda kv: -kv[1]["ms"]):
        e = {"launches": c["launches"],
             "avg_us": 1000.0 * c["ms"] / c["launches"],
             "share": c["ms"] / total_ms}
        if c["bytes"]:
            e["alg_GBps"] = c["bytes"] / (c["ms"] * 1e-3) / 1e9
            e["hbm_frac"] = e["alg_GBps"] / HBM_PEAK_GBS
        if c["flops"]:
            e["alg_TFLOPs"] = c["flops"] / (c["ms"] * 1e-3) / 1e12
            e["mfma_frac"] = e["alg_TFLOPs"] / MFMA_PEAK_TFLOPS[dt]
        kern[name] = e
    desc = f"{wl['desc']}-{schedule}"
    roof = roofline_of(classes, dt, desc)
    # online adjustment: sparsity of every tensor in the profiled frames
    # (their kept-row counters), thresholds after them
    ibst_sp = ibst_thr = None
    if ctl == "device":
        ibst_thr = g.thresholds()
        rows = []
        for f in range(len(counts)):
            kept = np.zeros(L_n + 1)
            for j, L in enumerate(net.layers):
                kept[j + 1] = counts[f, j, 4]
                if L.src == -1:
                    kept[0] = counts[f, j, 2]
            # a record of the chunk schedule covers `batch` frames
            rows.append(1.0 - kept / (batch * np.array(feed.grids,
                                                       dtype=np.float64)))
        ibst_sp = np.array(rows)
    roof["event_pair_overhead_us"] = event_overhead_us()

    # ---- graph replay: the same diff frames' launch sequence captured once
    # and replayed per frame (the frame is copied into the graph's input
    # slot first; that copy is timed too)
    graph = None
    if KG:
        if chunk and feed.next_is_ref():
            feed.ref()
        feed.replay = g.capture_diff(None if ctl == "device" else thr, out)
        gwall, grefs = run_diffs(feed, KG)
        feed.replay = None
        graph = {"diff_frames_per_s": KG / gwall,
                 "ms_per_step": gwall * 1000.0 / KG,
                 "steps": KG}
    stream_dens = ([round(g.density(-1, n), 5) for n in range(net.batch)]
                   if net.batch > 1 else None)

    # ---- dense comparators on the same GPU, net and dtype: the library's
    # own dense pass, and MIOpen through PyTorch both with its default
    # algorithm choice and with its benchmarking search (each convolution
    # shape timed over MIOpen's candidate solvers on first use, the fastest
    # kept)
    dense_ms = {}
    if dense:
        x = frames[0]
        dense_ms["own_dense_ms"] = time_gpu(
            lambda: g.encode_reference(x, out=out0), 5)
        fwd = torch_dense_model(net, dt)
        prev = torch.backends.cudnn.benchmark
        with torch.no_grad():
            torch.backends.cudnn.benchmark = False
            dense_ms["miopen_default_ms"] = time_gpu(lambda: fwd(x), 10,
                                                     warm=3)
            torch.backends.cudnn.benchmark = True
            t_find = time.perf_counter()
            fwd(x)
            torch.cuda.synchronize()
            dense_ms["miopen_find_s"] = time.perf_counter() - t_find
            dense_ms["miopen_ms"] = time_gpu(lambda: fwd(x), 10, warm=3)
            ref_t = fwd(x).permute(0, 2, 3, 1).float()
            torch.backends.cudnn.benchmark = prev
        g.encode_reference(x, out=out0)
        torch.cuda.synchronize()
        dense_ms["miopen_vs_own_rel_err"] = float(
            (ref_t - out0).abs().max() / out0.abs().max())
        dense_ms["miopen_tflops"] = dflops / (dense_ms["miopen_ms"] * 1e-3) \
            / 1e12
        dense_ms["own_dense_tflops"] = dflops / (
            dense_ms["own_dense_ms"] * 1e-3) / 1e12

    res = {
        "schedule": schedule,
        "workload": desc,
        "value": 1000.0 / ms_step,
        "ms_per_step": ms_step,
        "event_ms_per_step": ev_ms,
        "effective_tflops": alg_flops / (ms_step * 1e-3) / 1e12,
        "alg_gflop_per_frame": alg_flops / 1e9,
        "dense_gflop_per_frame": dflops / 1e9,
        "dense_equiv_tflops": dflops / (ms_step * 1e-3) / 1e12,
        "measured_input_density": dens0,
        "workspace_bytes": g.ws_bytes,
    }
    if chunk:
        ref_ms = float(np.median(refs)) if refs else None
        res["chunk"] = chunk
        res["ref_ms"] = ref_ms
        if ref_ms is not None:
            res["chunk_amortised_frames_per_s"] = 1000.0 * chunk / (
                ref_ms + (chunk - 1) * ms_step)
    if dense_ms:
        res["speedup_vs_dense"] = {
            "miopen": dense_ms["miopen_ms"] / ms_step,
            "miopen_default": dense_ms["miopen_default_ms"] / ms_step,
            "own_dense": dense_ms["own_dense_ms"] / ms_step}
        res["dense_ms"] = dense_ms
    if ibst_sp is not None and len(ibst_sp):
        s_c = ibst_sp[:, ctl_idx]
        th = ibst_thr[ctl_idx]
        res["ibst"] = {
            "where": "device (st_encode_chunk_adaptive, one step per "
                     f"chunk, a search over {batch} chunks)"
                     if schedule == "chunk" else
                     "device (st_encode_diff_adaptive)",
            "target": target, "eps": eps, "theta_max": 1.0,
            "controlled_tensors": len(ctl_idx),
            "sample": f"the {len(ibst_sp)} event-instrumented "
                      + ("chunk" if schedule == "chunk" else "diff frames"),
            "mean_sparsity_controlled": float(s_c.mean()),
            "in_band_frac_last_frame": float(np.mean(
                np.abs(s_c[-1] - target) <= eps)),
            "theta_last": {"min": float(th.min()),
                           "median": float(np.median(th)),
                           "max": float(th.max())},
            "mean_input_sparsity": float(ibst_sp[:, 0].mean())}
    if stream_dens:
        res["per_stream_input_density"] = stream_dens
        if "stream_density_targets" in wl:
            res["stream_change_targets"] = [
                round(v, 5) for v in wl["stream_density_targets"]]
    if graph:
        res["graph_replay"] = graph
    res["roofline"] = roof
    res["kernels"] = kern
    if ibst_thr is not None:
        res["_thresholds"] = ibst_thr
    res["profiled_ms_per_step"] = prof_ms_step
    res["frame_gen_s"] = t_gen
    g.close()
    del frames
    return res


def carry_comparison(name, thr_val, steps=18):
    """Drop (the paper's schedule) against residual carry on one workload
    at a threshold above zero, frame by frame over one chunk: every diff
    frame's output error against the dense forward of the same frame (the
    library's own dense pass), the diff-frames/s of both over `steps` timed
    frames of further chunks, frame by frame and in SparseBatch chunks (the
    chunk entry gives the frame-by-frame results), and the workspace of
    both."""
    import torch
    from paper_2410_20790_amd import SparseTemNet
    wl = workload(name, 0.10)
    net = wl["net"]
    dt = net.dtype
    chunk = wl["chunk"]
    tdt = {"f32": torch.float32, "f16": torch.float16,
           "bf16": torch.bfloat16}[dt]
    n = frames_needed(chunk, 0, chunk - 1 + steps, 0)
    frames = torch.empty((n, net.batch, net.H, net.W, net.C), dtype=tdt,
                         device="cuda")
    for i, f in enumerate(wl["frames"](n)):
        frames[i].copy_(torch.from_numpy(f))
    thr = [thr_val] * (len(net.layers) + 1)
    mk = lambda carry: SparseTemNet(net.layers, net.batch, net.H, net.W,  # noqa: E731
                                    net.C, dt, carry=carry)
    nets = {"drop": mk(False), "carry": mk(True)}
    dense = mk(False)
    res = {"workload": wl["desc"], "thr": thr_val, "chunk": chunk}
    try:
        errs = {k: [] for k in nets}
        for g in nets.values():
            g.encode_reference(frames[0])
        for t in range(1, chunk):
            ref = dense.encode_reference(frames[t])
            scale = float(ref.abs().max())
            for k, g in nets.items():
                out = g.encode_diff(frames[t], thr)
                errs[k].append(float((out - ref).abs().max()) / scale)
        torch.cuda.synchronize()
        for k, g in nets.items():
            feed = Feed(g, len(net.layers), frames, chunk, thr, None,
                        g.new_output())
            feed.pos = chunk
            wall, _ = run_diffs(feed, steps)
            res[k] = {"diff_frames_per_s": steps / wall,
                      "max_rel_err_vs_dense_per_frame":
                          [round(e, 6) for e in errs[k]],
                      "workspace_bytes": g.ws_bytes}
        # SparseBatch chunks (one st_encode_chunk call per chunk)
        for k, carry in (("drop", False), ("carry", True)):
            gc = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, dt,
                              max_frames=chunk - 1, carry=carry)
            try:
                oc = torch.empty((chunk - 1,) + tuple(gc.out_shape),
                                 dtype=torch.float32, device="cuda")
                feed = Feed(gc, len(net.layers), frames, chunk, thr, None,
                            oc, chunk - 1)
                run_diffs(feed, chunk - 1)
                wall, _ = run_diffs(feed, steps)
                res[k]["chunk_diff_frames_per_s"] = steps / wall
            finally:
                gc.close()
        res["extra_memory_bytes"] = (nets["carry"].ws_bytes -
                                     nets["drop"].ws_bytes)
    finally:
        for g in list(nets.values()) + [dense]:
            g.close()
        del frames
        torch.cuda.empty_cache()
    return res


def frozen_se_comparison(name, steps=14, warmup=7):
    """Squeeze-excitation with the reference frame's gates (an
    approximation) on an EfficientNet workload: frame by frame with the
    online threshold adjustment (as the exact line), then in SparseBatch
    chunks with the adjustment stepping once per chunk, and in chunks at
    the thresholds the frame run ended with; and the approximation alone --
    each diff frame's output at threshold 0 against the exact dense forward
    -- over one chunk."""
    import torch
    from paper_2410_20790_amd import SparseTemNet
    wl = workload(name, 0.0)
    net = wl["net"]
    keys = ("value", "ms_per_step", "effective_tflops", "ref_ms",
            "chunk_amortised_frames_per_s", "speedup_vs_dense", "ibst",
            "roofline", "graph_replay")
    fr = measure(wl, steps, warmup, 7, 0.0, frozen_se=True)
    out = {"frame_ibst": {k: fr[k] for k in keys if k in fr}}
    thr_end = [float(v) for v in fr.pop("_thresholds")]
    # warm-up over one whole search (chunk - 1 chunks), timed over two more
    nb = wl["chunk"] - 1
    ci = measure(wl, 2 * nb, nb * nb, 7, 0.0, dense=False, frozen_se=True,
                 schedule="chunk")
    ci.pop("_thresholds", None)
    out["chunk_ibst"] = {k: ci[k] for k in keys if k in ci}
    ch = measure(wl, steps, warmup, 7, 0.0, dense=False, frozen_se=True,
                 schedule="chunk", thr_list=thr_end, ibst=False)
    out["chunk_fixed_thr"] = {k: ch[k] for k in keys if k in ch}
    out["chunk_fixed_thr"]["thresholds"] = "the frame run's final ones"
    # the approximation alone
    chunk = wl["chunk"]
    frames = [torch.from_numpy(f).to("cuda") for f in wl["frames"](chunk)]
    tdt = {"f32": torch.float32, "f16": torch.float16,
           "bf16": torch.bfloat16}[net.dtype]
    frames = [f.to(tdt).contiguous() for f in frames]
    g = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, net.dtype,
                     frozen_se=True)
    d = SparseTemNet(net.layers, net.batch, net.H, net.W, net.C, net.dtype)
    try:
        g.encode_reference(frames[0])
        errs = []
        thr0 = [0.0] * (len(net.layers) + 1)
        for t in range(1, chunk):
            o = g.encode_diff(frames[t], thr0)
            ref = d.encode_reference(frames[t])
            errs.append(float((o - ref).abs().max() / ref.abs().max()))
        out["max_rel_err_vs_exact_dense_at_thr0"] = [round(e, 5)
                                                     for e in errs]
    finally:
        g.close()
        d.close()
        torch.cuda.empty_cache()
    return out


def bf16_state_comparison(name, steps=14, warmup=7):
    """bf16 pre-activation state (an approximation that halves the state)
    against the f32 state on an EfficientNet workload: diff-frames/s frame
    by frame with the device IBST (exact squeeze-excitation) and in
    SparseBatch chunks with frozen gates and one IBST step per chunk, the
    workspace of both, and the approximation alone -- each diff frame's
    output at threshold 0 (exact squeeze-excitation) against the exact
    dense forward -- over one chunk, for both states."""
    import torch
    from paper_2410_20790_amd import SparseTemNet
    wl = workload(name, 0.0)
    net = wl["net"]
    nb = wl["chunk"] - 1
    keys = ("value", "ms_per_step", "workspace_bytes")
    out = {}
    for label, b16 in (("f32_state", False), ("bf16_state", True)):
        fr = measure(wl, steps, warmup, 7, 0.0, dense=False,
                     bf16_state=b16)
        ch = measure(wl, 2 * nb, nb * nb, 7, 0.0, dense=False,
                     frozen_se=True, schedule="chunk", bf16_state=b16)
        out[label] = {"frame_ibst": {k: fr[k] for k in keys},
                      "chunk_frozen_se_ibst": {k: ch[k] for k in keys}}
    out["state_bytes_saved"] = (out["f32_state"]["frame_ibst"]
                                ["workspace_bytes"] -
                                out["bf16_state"]["frame_ibst"]
                                ["workspace_bytes"])
    tdt = {"f32": torch.float32, "f16": torch.float16,
           "bf16": torch.bfloat16}[net.dtype]
    frames = [torch.from_numpy(f).to("cuda").to(tdt).contiguous()
              for f in wl["frames"](wl["chunk"])]
    mk = lambda b16: SparseTemNet(net.layers, net.batch, net.H, net.W,  # noqa: E731
                                  net.C, net.dtype, bf16_state=b16)
    nets = {"f32_state": mk(False), "bf16_state": mk(True)}
    d = mk(False)
    try:
        errs = {k: [] for k in nets}
        thr0 = [0.0] * (len(net.layers) + 1)
        for g in nets.values():
            g.encode_reference(frames[0])
        for t in range(1, len(frames)):
            ref = d.encode_reference(frames[t])
            scale = float(ref.abs().max())
            for k, g in nets.items():
                o = g.encode_diff(frames[t], thr0)
                errs[k].append(round(float((o - ref).abs().max()) / scale,
                                     6))
        for k in nets:
            out[k]["max_rel_err_vs_exact_dense_at_thr0"] = errs[k]
    finally:
        for g in list(nets.values()) + [d]:
            g.close()
        torch.cuda.empty_cache()
    return out


def default_schedule(wl, requested=None):
    """SparseBatch (one st_encode_chunk call per chunk) for nets whose
    input has at most 16 channels and whose thresholds are fixed over a
    chunk; with the online threshold search (which steps after every frame
    of the frame-by-frame entry) one st_encode_diff call per frame."""
    net = wl["net"]
    ok = (wl["chunk"] and wl["chunk"] > 2 and not wl["ibst"] and
          net.C <= 16)
    if requested == "frame" or not ok:
        return "frame"
    return "chunk"


FRAME_KEYS = ("value", "ms_per_step", "event_ms_per_step", "effective_tflops",
              "ref_ms", "chunk_amortised_frames_per_s", "roofline",
              "graph_replay", "profiled_ms_per_step", "workload")


def extra_workload(name, steps, warmup, thr=0.0, cpu_chunk=False):
    """A secondary workload measured in the same run, summarised; in the
    SparseBatch schedule where it applies, with the frame-by-frame figure
    beside it.  cpu_chunk: the oracle's rate over one whole chunk of diff
    frames beside it (small workloads)."""
    import torch
    wl = workload(name, 0.0)
    net = wl["net"]
    sched = default_schedule(wl)
    log(f"workload {name}: {sched} schedule")
    r = measure(wl, steps, warmup, 7, thr, schedule=sched)
    r.pop("_thresholds", None)
    if sched == "chunk":
        f = measure(wl, steps, warmup, 7, thr, dense=False, schedule="frame")
        r["frame_by_frame"] = {k: f[k] for k in FRAME_KEYS if k in f}
    elif wl["ibst"] and wl["chunk"] and net.C <= 16:
        # SparseBatch chunks (exact squeeze-excitation per frame inside the
        # chunk) with the threshold search stepping once per chunk: warm-up
        # over one whole search (chunk - 1 chunks), timed over two more
        nb = wl["chunk"] - 1
        log(f"workload {name}: chunk schedule, one search step per chunk")
        c = measure(wl, 2 * nb, nb * nb, 7, thr, dense=False,
                    schedule="chunk")
        c.pop("_thresholds", None)
        r["chunk_ibst"] = {k: c[k] for k in
                           ("value", "ms_per_step", "effective_tflops",
                            "ref_ms", "chunk_amortised_frames_per_s", "ibst",
                            "roofline") if k in c}
    if cpu_chunk:
        r["cpu_baseline"] = cpu_baseline(wl, net, thr,
                                         n_diff=wl["chunk"] - 1)
    r["config"] = {"workload": wl["desc"], "batch": net.batch, "H": net.H,
                   "W": net.W, "C": net.C, "layers": len(net.layers),
                   "dtype": net.dtype, "chunk": wl["chunk"],
                   "thr": "ibst" if wl["ibst"] else thr}
    torch.cuda.empty_cache()
    return r


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=45,
                    help="timed diff frames (ResNet-50: five chunks of 9)")
    ap.add_argument("--warmup", type=int, default=9)
    ap.add_argument("--workload", default="resnet50",
                    choices=["resnet50", "effnet_b0", "multistream", "crnn",
                             "toy"])
    ap.add_argument("--schedule", choices=["chunk", "frame"], default=None,
                    help="chunk: the diff frames of a chunk in one "
                         "st_encode_chunk call (SparseBatch; the default "
                         "where the net allows it); frame: one "
                         "st_encode_diff call per frame")
    ap.add_argument("--density", type=float, default=0.10)
    ap.add_argument("--thr", type=float, default=0.0)
    ap.add_argument("--profile-steps", type=int, default=9)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-frame", action="store_true",
                    help="skip the frame-by-frame comparison pass")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the other workloads (EfficientNet-B0 512x512 "
                         "f16 and 32 streams of 256x256 bf16, both with "
                         "online threshold adjustment; CRNN-VGG text lines; "
                         "the toy net)")
    ap.add_argument("--sweep-steps", type=int, default=18)
    ap.add_argument("--full-out", default="gpurun_out/bench_full.json",
                    help="where the full result (every sub-measurement) is "
                         "written as JSON; stdout ends with one compact "
                         "headline line ('' to skip the file)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of a known size "
                         "(reference kernel for the HBM byte counters)")
    ap.add_argument("--ingest-counters", metavar="DIR",
                    help="turn rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs "
                         "(DIR/pmc_{bench,copy}_{FETCH,WRITE}_SIZE) into "
                         "profiles/hbm_traffic.json")
    ap.add_argument("--ingest-mfma", metavar="DIR",
                    help="turn a rocprofv3 --pmc run of the MFMA counters "
                         "(DIR/pmc_mfma) into profiles/mfma_util.json")
    args = ap.parse_args()
    if args.ingest_mfma:
        ingest_mfma(args.ingest_mfma, args.workload, args.density,
                    args.schedule)
        return
    if args.copy_calibration:
        copy_calibration()
        return
    if args.ingest_counters:
        ingest_counters(args.ingest_counters, args.workload, args.density,
                        args.schedule)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: there is no multi-GPU path "
              "(independent streams would shard by image, one net per GPU). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    wl = workload(args.workload, args.density)
    net = wl["net"]
    sched = default_schedule(wl, args.schedule)
    K, W, KP = args.steps, args.warmup, args.profile_steps
    log(f"headline: {wl['desc']}, {sched} schedule, {K} timed diff frames")
    r = measure(wl, K, W, KP, args.thr, dense=not args.no_dense,
                schedule=sched)
    r.pop("_thresholds", None)
    if not args.no_dense:
        r["roofline"]["measured_peaks"] = measured_peaks()
    res = {
        "metric": METRIC,
        "value": r.pop("value"),
        "unit": "diff-frames/s",
        "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": r.pop("ms_per_step"),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": net.dtype,
        "data": "synthetic (seeded temporally continuous video, "
                "random-init weights)",
        "config": {"workload": r.pop("workload"), "batch": net.batch,
                   "H": net.H, "W": net.W, "C": net.C,
                   "layers": len(net.layers), "chunk": wl["chunk"],
                   "schedule": sched,
                   "target_density": args.density,
                   "measured_input_density": r.pop("measured_input_density"),
                   "thr": "ibst" if wl["ibst"] else args.thr},
    }
    res.update(r)
    if sched == "chunk" and not args.no_frame:
        log("frame-by-frame schedule on the same video")
        f = measure(wl, K, W, KP, args.thr, dense=False, schedule="frame")
        res["frame_by_frame"] = {k: f[k] for k in FRAME_KEYS if k in f}
    res["kernel_source_hash"] = kernel_source_hash()
    if args.workload == "resnet50" and not args.no_sweep:
        log("density sweep")
        res["density_sweep"] = density_sweep(
            net, args.thr, [0.02, 0.05, 0.10, 0.20, 0.40], args.sweep_steps,
            wl["chunk"], sched)
    if args.workload == "resnet50" and not args.no_extra:
        res["other_workloads"] = {
            "effnet_b0": extra_workload("effnet_b0", 14, 7),
            "effnet_b0_frozen_se": frozen_se_comparison("effnet_b0"),
            "multistream": extra_workload("multistream", 14, 7),
            "multistream_frozen_se": frozen_se_comparison("multistream"),
            "effnet_b0_bf16_state": bf16_state_comparison("effnet_b0"),
            "multistream_bf16_state": bf16_state_comparison("multistream"),
            "crnn": extra_workload("crnn", 30, 15, thr=0.02,
                                   cpu_chunk=not args.no_cpu_baseline),
            "toy": extra_workload("toy", 30, 3,
                                  cpu_chunk=not args.no_cpu_baseline)}
    if args.workload == "resnet50" and not args.no_extra:
        log("residual carry against drop")
        res["residual_carry"] = {
            "resnet50": carry_comparison("resnet50", 0.02),
            "toy": carry_comparison("toy", 0.05, steps=30)}
    if not args.no_cpu_baseline:
        log("cpu baseline (the oracle on the host cores)")
        res["cpu_baseline"] = cpu_baseline(wl, net, args.thr)
    if "dense_ms" in res and "measured_peaks" in res["roofline"]:
        # the dense network at the box's measured library-GEMM ceiling: a
        # bound no dense implementation beats, not a measured comparator
        ceil = res["roofline"]["measured_peaks"]["bf16_gemm_TFLOPs"]
        res["dense_ms"]["at_gemm_ceiling_ms"] = (
            res["dense_gflop_per_frame"] / ceil)
        res["speedup_vs_dense"]["dense_at_gemm_ceiling"] = (
            res["dense_ms"]["at_gemm_ceiling_ms"] / res["ms_per_step"])
    full = args.full_out
    if full:
        d = os.path.dirname(full)
        if d:
            os.makedirs(d, exist_ok=True)
        with open(full, "w") as fh:
            json.dump(res, fh, indent=1)
        log(f"full result: {full}")
    print(json.dumps(headline(res, full)), flush=True)


def _r(x, nd=4):
    """x to nd significant digits (None passes)."""
    if x is None or isinstance(x, (bool, str)):
        return x
    if isinstance(x, int):
        return x
    return float(f"{x:.{nd}g}")


def headline(res, full_path):
    """The one result line: the contract's keys, the dominant kernel's
    roofline, the CPU baseline and the dense speedups, rounded; everything
    else stays in the full result file."""
    keys = ("metric", "value", "unit", "n_gpus", "steps", "warmup",
            "ms_per_step", "higher_is_better", "scaling", "vs_baseline",
            "dtype", "data")
    h = {k: _r(res[k]) for k in keys if k in res}
    c = res["config"]
    h["config"] = {"workload": c["workload"], "schedule": c["schedule"],
                   "chunk": c["chunk"], "thr": c["thr"],
                   "input_density": _r(c["measured_input_density"], 3)}
    for k in ("effective_tflops", "dense_equiv_tflops", "ref_ms",
              "chunk_amortised_frames_per_s"):
        if res.get(k) is not None:
            h[k] = _r(res[k])
    if "speedup_vs_dense" in res:
        h["speedup_vs_dense"] = {k: _r(v, 3) for k, v in
                                 res["speedup_vs_dense"].items()}
        h["dense_ms"] = {k: _r(res["dense_ms"][k]) for k in
                         ("miopen_ms", "miopen_default_ms", "own_dense_ms",
                          "at_gemm_ceiling_ms") if k in res["dense_ms"]}
    rf = res["roofline"]
    h["roofline"] = {k: _r(rf.get(k)) for k in
                     ("kernel", "bound", "achieved", "peak", "unit", "frac",
                      "traffic", "avg_launch_us", "launches")}
    mp = rf.get("measured_peaks")
    if mp:
        h["roofline"]["box_copy_GBps"] = _r(mp["copy_GBps"])
        h["roofline"]["box_bf16_gemm_TFLOPs"] = _r(mp["bf16_gemm_TFLOPs"])
    cb = res.get("cpu_baseline")
    if cb:
        h["cpu_baseline"] = {"value": _r(cb["value"]), "unit": cb["unit"],
                             "cores": cb["cores"], "kind": cb["kind"],
                             "sample": cb["sample"]}
        if "single_thread" in cb:
            h["cpu_baseline"]["single_thread_value"] = _r(
                cb["single_thread"]["value"])
    if full_path:
        h["full_result"] = full_path
    return h


if __name__ == "__main__":
    main()
