"""Host-only checks of the C ABI: the library loads, exports every entry
point the header declares, validates layer graphs and sizes the workspace
without touching a GPU."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2410_20790_amd import binding as B
from workloads import (crnn_vgg_net, depthwise_test_net, resnet50_net,
                       resnet_mini_net, toy_net)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparsetem.h")


def header_symbols():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(st_[a-z_]+)\s*\(", txt)))


def test_header_declares_the_binding_names():
    assert header_symbols() == sorted(B.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(B.LIB_PATH)
    for name in header_symbols():
        assert hasattr(lib, name), name


def descs(net, fake_ptr=0x1000):
    from paper_2410_20790_amd.net import layer_desc
    return [layer_desc(L, fake_ptr, fake_ptr) for L in net.layers]


def create(net, **over):
    d = descs(net)
    for i, kv in over.get("patch", {}).items():
        for k, v in kv.items():
            setattr(d[i], k, v)
    return B.st_create_net(d, over.get("batch", net.batch),
                           over.get("H", net.H), over.get("W", net.W),
                           over.get("C", net.C),
                           over.get("dtype", B.DTYPE_CODES[net.dtype]))


@pytest.mark.parametrize("mk", [toy_net, crnn_vgg_net, resnet_mini_net,
                                depthwise_test_net])
def test_create_valid_nets(mk):
    net = mk()
    h = create(net)
    try:
        assert B.st_workspace_bytes(h) > 0
        shp = B.st_tensor_shape(h, len(net.layers) - 1)
        assert shp[0] == net.batch and shp[3] == net.layers[-1].c_out
        assert B.st_tensor_shape(h, -1) == (net.batch, net.H, net.W, net.C)
    finally:
        B.st_destroy_net(h)


def test_output_shapes_match_geometry():
    net = crnn_vgg_net()
    h = create(net)
    try:
        assert B.st_tensor_shape(h, 0) == (1, 16, 64, 64)
        assert B.st_tensor_shape(h, 1) == (1, 8, 32, 128)
        assert B.st_tensor_shape(h, 3) == (1, 4, 32, 256)
        assert B.st_tensor_shape(h, 6) == (1, 2, 32, 512)
    finally:
        B.st_destroy_net(h)


def test_resnet50_workspace_fits_one_gpu():
    net_shape_only = resnet50_net.__wrapped__ if hasattr(
        resnet50_net, "__wrapped__") else None
    net = resnet50_net(H=1024, W=2048)
    h = create(net)
    try:
        shp = B.st_tensor_shape(h, len(net.layers) - 1)
        assert shp == (1, 32, 64, 2048)
        ws = B.st_workspace_bytes(h)
        # f32 pre-activation state alone is ~1.6 GB; everything < 8 GB
        assert 1.6e9 < ws < 8e9
    finally:
        B.st_destroy_net(h)


@pytest.mark.parametrize("patch,status", [
    ({0: {"src": 0}}, B.ST_ERR_INVALID_ARG),          # self reference
    ({1: {"src": 5}}, B.ST_ERR_INVALID_ARG),          # forward reference
    ({1: {"c_in": 7}}, B.ST_ERR_INVALID_ARG),         # channel mismatch
    ({0: {"k_h": 0}}, B.ST_ERR_INVALID_ARG),
    ({0: {"s_w": 0}}, B.ST_ERR_INVALID_ARG),
    ({0: {"p_h": -1}}, B.ST_ERR_INVALID_ARG),
    ({0: {"act": 9}}, B.ST_ERR_INVALID_ARG),
    ({0: {"groups": 4}}, B.ST_ERR_UNSUPPORTED),       # grouped, not depthwise
    ({0: {"se_mid": 4}}, B.ST_ERR_INVALID_ARG),       # no SE weights
    ({0: {"se_mid": -1}}, B.ST_ERR_INVALID_ARG),
    ({0: {"weight": None}}, B.ST_ERR_INVALID_ARG),
    ({1: {"residual_src": -1}}, B.ST_ERR_INVALID_ARG),  # 16 ch vs 32 out
    ({0: {"pool_k_h": 2, "pool_k_w": 2, "pool_s_h": 2, "pool_s_w": 2,
          "pool_p_h": 2, "pool_p_w": 0}}, B.ST_ERR_INVALID_ARG),
    ({0: {"k_h": 9, "k_w": 9, "p_h": 4, "p_w": 4}}, B.ST_ERR_UNSUPPORTED),
])
def test_invalid_descriptors(patch, status):
    with pytest.raises(B.StError) as e:
        create(toy_net(), patch=patch)
    assert e.value.status == status
    assert B.st_last_error()


@pytest.mark.parametrize("kw,status", [
    ({"batch": 0}, B.ST_ERR_INVALID_ARG),
    ({"H": 0}, B.ST_ERR_INVALID_ARG),
    ({"C": 3}, B.ST_ERR_INVALID_ARG),
    ({"dtype": 7}, B.ST_ERR_INVALID_ARG),
    ({"H": 1, "W": 1}, B.ST_ERR_INVALID_ARG),   # fine conv, but see below
])
def test_invalid_shapes(kw, status):
    if kw == {"H": 1, "W": 1}:
        # a 1x1 input is still a valid 3x3/pad-1 conv input
        h = create(toy_net(), **kw)
        B.st_destroy_net(h)
        return
    with pytest.raises(B.StError) as e:
        create(toy_net(), **kw)
    assert e.value.status == status


def test_empty_output_rejected():
    net = toy_net(H=2, W=2)
    with pytest.raises(B.StError) as e:
        create(net, patch={0: {"p_h": 0, "p_w": 0}})
    assert e.value.status == B.ST_ERR_INVALID_ARG


def test_null_arguments():
    lib = B.library()
    out = ctypes.c_void_p()
    assert lib.st_create_net(None, 1, 1, 4, 4, 16, 0,
                             ctypes.byref(out)) == B.ST_ERR_INVALID_ARG
    assert lib.st_workspace_bytes(None, None) == B.ST_ERR_INVALID_ARG
    h = create(toy_net())
    try:
        # unbound workspace: encodes report a state error, not a crash
        thr = (ctypes.c_float * 3)(0, 0, 0)
        assert lib.st_encode_reference(h, 0x1000, None, None) == B.ST_ERR_STATE
        assert lib.st_encode_diff(h, 0x1000, thr, None, None) == B.ST_ERR_STATE
        assert lib.st_bind_workspace(h, None, 1 << 20, None) == \
            B.ST_ERR_INVALID_ARG
        assert lib.st_bind_workspace(h, 0x1001, 1 << 40, None) == \
            B.ST_ERR_INVALID_ARG
        assert lib.st_bind_workspace(h, 0x1000, 16, None) == B.ST_ERR_WORKSPACE
        assert "small" in B.st_last_error(h)
    finally:
        B.st_destroy_net(h)


def test_workspace_scales_with_batch():
    a = create(toy_net(batch=1))
    b = create(toy_net(batch=4))
    try:
        wa, wb = B.st_workspace_bytes(a), B.st_workspace_bytes(b)
        assert 3.5 * wa < wb < 4.5 * wa
    finally:
        B.st_destroy_net(a)
        B.st_destroy_net(b)


def test_single_hip_runtime():
    """Importing the binding first must not load a second HIP runtime next
    to PyTorch's (two HSA runtimes in one process cannot share the GPU)."""
    import subprocess
    import sys
    code = ("from paper_2410_20790_amd import binding\n"
            "import torch\n"
            "libs = {l.split()[-1] for l in open('/proc/self/maps')\n"
            "        if 'libamdhip64' in l}\n"
            "print(len(libs))\n")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", code], cwd=root,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip().splitlines()[-1] == "1"


def test_chunked_create_and_workspace():
    """A chunk-capable net: item buffers grow with max_frames, the state
    does not; max_frames outside [1, 32] is rejected; a chunk encode on an
    unbound net is a state error (no HIP call is made)."""
    net = resnet_mini_net()
    d = descs(net)
    h1 = B.st_create_net(d, net.batch, net.H, net.W, net.C, B.ST_F32)
    h8 = B.st_create_net_chunked(d, net.batch, 8, net.H, net.W, net.C,
                                 B.ST_F32)
    try:
        w1, w8 = B.st_workspace_bytes(h1), B.st_workspace_bytes(h8)
        assert w1 < w8 < 8 * w1
        with pytest.raises(B.StError) as e:
            B.st_encode_chunk(h8, 0x1000, 2, [0.0] * (len(net.layers) + 1),
                              None)
        assert e.value.status == B.ST_ERR_STATE
    finally:
        B.st_destroy_net(h1)
        B.st_destroy_net(h8)
    for bad in (0, 33):
        with pytest.raises(B.StError) as e:
            B.st_create_net_chunked(d, net.batch, bad, net.H, net.W, net.C,
                                    B.ST_F32)
        assert e.value.status == B.ST_ERR_INVALID_ARG


def test_threshold_control_needs_a_bound_net():
    """The device threshold controller writes the workspace: on a net with
    none bound every entry point is a state error (no HIP call is made)."""
    net = toy_net()
    h = B.st_create_net(descs(net), net.batch, net.H, net.W, net.C, B.ST_F32)
    try:
        n = len(net.layers) + 1
        with pytest.raises(B.StError) as e:
            B.st_set_threshold_control(h, [1] * n, [0.0] * n)
        assert e.value.status == B.ST_ERR_STATE
        with pytest.raises(B.StError) as e:
            B.st_encode_diff_adaptive(h, 0x1000)
        assert e.value.status == B.ST_ERR_STATE
        with pytest.raises(B.StError) as e:
            B.st_get_thresholds(h, n)
        assert e.value.status == B.ST_ERR_STATE
        with pytest.raises(B.StError) as e:
            B.st_encode_chunk_adaptive(h, 0x1000, 2)
        assert e.value.status == B.ST_ERR_STATE
        with pytest.raises(ValueError):
            B.st_set_threshold_control(h, [1] * n, [0.0] * (n - 1))
    finally:
        B.st_destroy_net(h)


def test_residual_carry_flag():
    """ST_NET_RESIDUAL_CARRY adds one f32 view per layer output (and a state
    for layers without non-linearity), with or without chunk capacity;
    unknown flags are rejected."""
    net = resnet_mini_net()
    d = descs(net)
    h0 = B.st_create_net(d, net.batch, net.H, net.W, net.C, B.ST_F32)
    h1 = B.st_create_net_ex(d, net.batch, 1, net.H, net.W, net.C, B.ST_F32,
                            B.NET_RESIDUAL_CARRY)
    try:
        extra = B.st_workspace_bytes(h1) - B.st_workspace_bytes(h0)
        views = 0
        for L in net.layers:
            views += 4 * 8 * ((L.c_out + 7) // 8)   # lower bound per site
        assert extra >= views
        with pytest.raises(B.StError) as e:
            B.st_debug_carry(h0, 0, (1,))
        assert e.value.status == B.ST_ERR_STATE
    finally:
        B.st_destroy_net(h0)
        B.st_destroy_net(h1)
    # an unknown flag, and carry with frozen squeeze-excitation (exclusive)
    for flags, status in ((8, B.ST_ERR_INVALID_ARG),
                          (B.NET_RESIDUAL_CARRY | B.NET_FROZEN_SE,
                           B.ST_ERR_INVALID_ARG)):
        with pytest.raises(B.StError) as e:
            B.st_create_net_ex(d, net.batch, 1, net.H, net.W, net.C,
                               B.ST_F32, flags)
        assert e.value.status == status
    # with chunk capacity too
    h4 = B.st_create_net_ex(d, net.batch, 4, net.H, net.W, net.C, B.ST_F32,
                            B.NET_RESIDUAL_CARRY)
    B.st_destroy_net(h4)


def test_bf16_state_flag():
    """ST_NET_BF16_STATE halves every stateful layer's state (2 bytes per
    value instead of 4); it is refused for max-pooled nets and with
    residual carry."""
    from oracle import sparsetem_oracle as so
    net = toy_net()
    d = descs(net)
    h0 = B.st_create_net(d, net.batch, net.H, net.W, net.C, B.ST_F32)
    h1 = B.st_create_net_ex(d, net.batch, 1, net.H, net.W, net.C, B.ST_F32,
                            B.NET_BF16_STATE)
    try:
        saved = B.st_workspace_bytes(h0) - B.st_workspace_bytes(h1)
        want = 0
        for i, L in enumerate(net.layers):
            if so._is_stateful(net.layers, i):
                n, h, w, _ = B.st_tensor_shape(h0, i)
                want += 2 * n * h * w * ((L.c_out + 7) // 8 * 8)
        # each allocation is rounded up to the workspace alignment
        assert want <= saved + 256 * len(net.layers)
        assert saved <= want + 256 * len(net.layers)
    finally:
        B.st_destroy_net(h0)
        B.st_destroy_net(h1)
    pooled = resnet_mini_net()
    for n, flags in ((pooled, B.NET_BF16_STATE),
                     (net, B.NET_BF16_STATE | B.NET_RESIDUAL_CARRY)):
        with pytest.raises(B.StError) as e:
            B.st_create_net_ex(descs(n), n.batch, 1, n.H, n.W, n.C, B.ST_F32,
                               flags)
        assert e.value.status == B.ST_ERR_UNSUPPORTED


def test_static_workspace_rejects_a_net_too_large():
    """The no-allocation binding checks the net's workspace against the
    static one before any device call."""
    net = resnet50_net(H=1024, W=2048)
    h = create(net)
    try:
        assert B.st_workspace_bytes(h) > B.STATIC_WORKSPACE_BYTES
        with pytest.raises(B.StError) as e:
            B.st_bind_workspace_static(h)
        assert e.value.status == B.ST_ERR_WORKSPACE
    finally:
        B.st_destroy_net(h)
