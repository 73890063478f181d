"""ctypes binding of the C ABI declared in include/sparsetem.h.

Every function here has the name of the C entry point it wraps and only
marshals arguments: Python sequences become C arrays, integer device
addresses become pointers, a non-OK status becomes ``StError`` carrying
``st_last_error``.  All computation happens in the HIP library; importing
this module fails loudly if the library has not been built.
"""

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)),
                        "libsparsetem.so")

ST_OK, ST_ERR_INVALID_ARG, ST_ERR_UNSUPPORTED = 0, 1, 2
ST_ERR_STATE, ST_ERR_WORKSPACE, ST_ERR_HIP = 3, 4, 5
ST_F32, ST_F16, ST_BF16 = 0, 1, 2
DTYPE_CODES = {"f32": ST_F32, "f16": ST_F16, "bf16": ST_BF16}

KERNEL_CLASSES = [
    "scan_mask", "scan_compact", "rb_mark", "rb_count", "rb_compact",
    "rb_nbr", "rb_ident", "conv_gemm", "conv_dw", "pool_mark", "pool_count",
    "pool_compact", "pool_emit", "commit", "list_count", "list_compact",
    "output", "cleanup", "reset", "se_squeeze", "se_excite", "se_emit",
    "conv_split_epi", "chunk_update", "run_tiles", "carry_commit",
]

EXPORTED = [
    "st_create_net", "st_create_net_chunked", "st_workspace_bytes",
    "st_bind_workspace", "st_encode_reference", "st_encode_diff",
    "st_encode_chunk", "st_layer_density",
    "st_tensor_shape", "st_destroy_net", "st_last_error", "st_debug_active",
    "st_debug_candidates", "st_debug_rulebook", "st_debug_state",
    "st_debug_counters", "st_profile_begin", "st_profile_end",
    "st_set_threshold_control", "st_encode_diff_adaptive",
    "st_get_thresholds", "st_create_net_ex", "st_debug_carry",
    "st_encode_chunk_adaptive", "st_bind_workspace_static",
]


class StError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"status {status}: {msg}")
        self.status = status


class st_layer_desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "src", "residual_src", "c_in", "c_out", "groups", "k_h", "k_w",
        "s_h", "s_w", "p_h", "p_w", "act", "pool_k_h", "pool_k_w",
        "pool_s_h", "pool_s_w", "pool_p_h", "pool_p_w", "se_mid")] + [
        (n, ctypes.c_void_p) for n in (
            "weight", "bias", "se_w1", "se_b1", "se_w2", "se_b2")]


class st_launch_record(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int32), ("layer", ctypes.c_int32),
                ("frame", ctypes.c_int32), ("ms", ctypes.c_float)]


def _load():
    # The library must use the HIP runtime PyTorch ships (its device
    # pointers and streams come from there).  Loaded first, the library
    # would pull in the system runtime and PyTorch a second copy of it: two
    # HSA runtimes in one process, and the second to open the device finds
    # none.  Importing torch first makes the library bind to torch's copy.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with "
            "`python -m paper_2410_20790_amd.build` (no CPU fallback exists)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, U64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                        ctypes.c_uint64)
    sig = {
        "st_create_net": [ctypes.POINTER(st_layer_desc), I32, I32, I32, I32,
                          I32, I32, ctypes.POINTER(P)],
        "st_create_net_chunked": [ctypes.POINTER(st_layer_desc), I32, I32,
                                  I32, I32, I32, I32, I32,
                                  ctypes.POINTER(P)],
        "st_create_net_ex": [ctypes.POINTER(st_layer_desc), I32, I32, I32,
                             I32, I32, I32, I32, ctypes.c_uint32,
                             ctypes.POINTER(P)],
        "st_debug_carry": [P, I32, P, I64],
        "st_encode_chunk": [P, P, I32, ctypes.POINTER(ctypes.c_float), P, P],
        "st_workspace_bytes": [P, ctypes.POINTER(U64)],
        "st_bind_workspace": [P, P, U64, P],
        "st_bind_workspace_static": [P, P],
        "st_encode_reference": [P, P, P, P],
        "st_encode_diff": [P, P, ctypes.POINTER(ctypes.c_float), P, P],
        "st_layer_density": [P, I32, I32, ctypes.POINTER(ctypes.c_float)],
        "st_tensor_shape": [P, I32, ctypes.POINTER(I32)],
        "st_debug_active": [P, I32, P, I64, ctypes.POINTER(I64)],
        "st_debug_candidates": [P, I32, P, P, I64, ctypes.POINTER(I64)],
        "st_debug_rulebook": [P, I32, P, I64, ctypes.POINTER(I64)],
        "st_debug_state": [P, I32, P, I64],
        "st_debug_counters": [P, P, P],
        "st_profile_begin": [P, I32, I32],
        "st_profile_end": [P, P, I32, ctypes.POINTER(I32), P, I32,
                           ctypes.POINTER(I32)],
        "st_set_threshold_control": [P, ctypes.POINTER(ctypes.c_uint8),
                                     ctypes.POINTER(ctypes.c_float),
                                     ctypes.c_double, ctypes.c_double,
                                     ctypes.c_double, ctypes.c_double, I32,
                                     P],
        "st_encode_diff_adaptive": [P, P, P, P],
        "st_encode_chunk_adaptive": [P, P, I32, P, P],
        "st_get_thresholds": [P, ctypes.POINTER(ctypes.c_float)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = I32
    lib.st_destroy_net.argtypes = [P]
    lib.st_destroy_net.restype = None
    lib.st_last_error.argtypes = [P]
    lib.st_last_error.restype = ctypes.c_char_p
    return lib


_lib = _load()


def library():
    return _lib


def _check(status, net=None):
    if status != ST_OK:
        msg = _lib.st_last_error(net)
        raise StError(status, msg.decode() if msg else "")


def _ptr(x) -> Optional[int]:
    return None if x is None else int(x)


# ------------------------------------------------------------- lifecycle

def st_create_net(layers: Sequence[st_layer_desc], batch, in_h, in_w, in_c,
                  dtype) -> int:
    arr = (st_layer_desc * len(layers))(*layers)
    out = ctypes.c_void_p()
    _check(_lib.st_create_net(arr, len(layers), batch, in_h, in_w, in_c,
                              dtype, ctypes.byref(out)))
    return out.value


def st_create_net_chunked(layers: Sequence[st_layer_desc], batch,
                          max_frames, in_h, in_w, in_c, dtype) -> int:
    arr = (st_layer_desc * len(layers))(*layers)
    out = ctypes.c_void_p()
    _check(_lib.st_create_net_chunked(arr, len(layers), batch, max_frames,
                                      in_h, in_w, in_c, dtype,
                                      ctypes.byref(out)))
    return out.value


NET_RESIDUAL_CARRY = 1
NET_FROZEN_SE = 2
NET_BF16_STATE = 4


def st_create_net_ex(layers: Sequence[st_layer_desc], batch, max_frames,
                     in_h, in_w, in_c, dtype, flags) -> int:
    arr = (st_layer_desc * len(layers))(*layers)
    out = ctypes.c_void_p()
    _check(_lib.st_create_net_ex(arr, len(layers), batch, max_frames, in_h,
                                 in_w, in_c, dtype, flags,
                                 ctypes.byref(out)))
    return out.value


def st_workspace_bytes(net) -> int:
    b = ctypes.c_uint64()
    _check(_lib.st_workspace_bytes(net, ctypes.byref(b)), net)
    return b.value


def st_bind_workspace(net, dev_ptr, nbytes, stream=0):
    _check(_lib.st_bind_workspace(net, _ptr(dev_ptr), nbytes, _ptr(stream)),
           net)


def st_bind_workspace_static(net, stream=0):
    _check(_lib.st_bind_workspace_static(net, _ptr(stream)), net)


STATIC_WORKSPACE_BYTES = 64 << 20


def st_encode_reference(net, frame_ptr, out_ptr=None, stream=0):
    _check(_lib.st_encode_reference(net, _ptr(frame_ptr), _ptr(out_ptr),
                                    _ptr(stream)), net)


def st_encode_diff(net, frame_ptr, thr, out_ptr=None, stream=0):
    t = (ctypes.c_float * len(thr))(*[float(v) for v in thr])
    _check(_lib.st_encode_diff(net, _ptr(frame_ptr), t, _ptr(out_ptr),
                               _ptr(stream)), net)


def st_set_threshold_control(net, controlled, fixed_thr, target=0.9,
                             eps=0.025, theta_max=1.0, theta0=-1.0,
                             stream=0, cycle_refs=1):
    """controlled: n_layers + 1 flags; fixed_thr: n_layers + 1 thresholds
    (used by the tensors that are not controlled); a search cycle spans
    cycle_refs reference frames."""
    if len(controlled) != len(fixed_thr):
        raise ValueError("controlled and fixed_thr differ in length")
    c = (ctypes.c_uint8 * len(controlled))(*[1 if v else 0
                                             for v in controlled])
    f = (ctypes.c_float * len(fixed_thr))(*[float(v) for v in fixed_thr])
    _check(_lib.st_set_threshold_control(net, c, f, float(target), float(eps),
                                         float(theta_max), float(theta0),
                                         int(cycle_refs), _ptr(stream)), net)


def st_encode_diff_adaptive(net, frame_ptr, out_ptr=None, stream=0):
    _check(_lib.st_encode_diff_adaptive(net, _ptr(frame_ptr), _ptr(out_ptr),
                                        _ptr(stream)), net)


def st_encode_chunk_adaptive(net, frames_ptr, n_frames, out_ptr=None,
                             stream=0):
    _check(_lib.st_encode_chunk_adaptive(net, _ptr(frames_ptr), n_frames,
                                         _ptr(out_ptr), _ptr(stream)), net)


def st_get_thresholds(net, n_tensors):
    t = (ctypes.c_float * n_tensors)()
    _check(_lib.st_get_thresholds(net, t), net)
    return np.array(t[:], dtype=np.float32)


def st_encode_chunk(net, frames_ptr, n_frames, thr, out_ptr=None, stream=0):
    t = (ctypes.c_float * len(thr))(*[float(v) for v in thr])
    _check(_lib.st_encode_chunk(net, _ptr(frames_ptr), n_frames, t,
                                _ptr(out_ptr), _ptr(stream)), net)


def st_layer_density(net, layer, image=-1) -> float:
    d = ctypes.c_float()
    _check(_lib.st_layer_density(net, layer, image, ctypes.byref(d)), net)
    return d.value


def st_tensor_shape(net, layer):
    s = (ctypes.c_int32 * 4)()
    _check(_lib.st_tensor_shape(net, layer, s), net)
    return tuple(s)


def st_destroy_net(net):
    _lib.st_destroy_net(net)


def st_last_error(net=None) -> str:
    m = _lib.st_last_error(net)
    return m.decode() if m else ""


# ----------------------------------------------------------- introspection

def st_debug_active(net, layer) -> np.ndarray:
    n = ctypes.c_int64()
    _check(_lib.st_debug_active(net, layer, None, 0, ctypes.byref(n)), net)
    idx = np.zeros(n.value, np.int32)
    _check(_lib.st_debug_active(net, layer, idx.ctypes.data, n.value,
                                ctypes.byref(n)), net)
    return idx


def st_debug_candidates(net, layer, channels, with_rows=True):
    """(pixel ids, f32 rows) of the candidates; rows None when not asked."""
    n = ctypes.c_int64()
    _check(_lib.st_debug_candidates(net, layer, None, None, 0,
                                    ctypes.byref(n)), net)
    pix = np.zeros(n.value, np.int32)
    rows = np.zeros((n.value, channels), np.float32) if with_rows else None
    _check(_lib.st_debug_candidates(net, layer, pix.ctypes.data,
                                    rows.ctypes.data if with_rows else None,
                                    n.value, ctypes.byref(n)), net)
    return pix, rows


def st_debug_rulebook(net, layer) -> np.ndarray:
    n = ctypes.c_int64()
    _check(_lib.st_debug_rulebook(net, layer, None, 0, ctypes.byref(n)), net)
    kio = np.zeros((n.value, 3), np.int32)
    _check(_lib.st_debug_rulebook(net, layer, kio.ctypes.data, n.value,
                                  ctypes.byref(n)), net)
    return kio


def st_debug_state(net, layer, shape) -> np.ndarray:
    P = np.zeros(shape, np.float32)
    _check(_lib.st_debug_state(net, layer, P.ctypes.data, P.size), net)
    return P


def st_debug_carry(net, layer, shape) -> np.ndarray:
    """Consumers' view of layer `layer`'s emitted tensor (residual carry)."""
    V = np.zeros(shape, np.float32)
    _check(_lib.st_debug_carry(net, layer, V.ctypes.data, V.size), net)
    return V


def st_debug_counters(net, n_layers):
    pairs = np.zeros(n_layers, np.int64)
    act = np.zeros(n_layers + 1, np.int64)
    _check(_lib.st_debug_counters(net, pairs.ctypes.data, act.ctypes.data),
           net)
    return pairs, act


# ------------------------------------------------------------- measurement

def st_profile_begin(net, max_launches, max_frames):
    _check(_lib.st_profile_begin(net, max_launches, max_frames), net)


def st_profile_end(net, n_layers, cap=1 << 20, cap_frames=4096):
    recs = (st_launch_record * cap)()
    n = ctypes.c_int32()
    nf = ctypes.c_int32()
    counts = np.zeros((cap_frames, n_layers, 8), np.int64)
    _check(_lib.st_profile_end(net, recs, cap, ctypes.byref(n),
                               counts.ctypes.data, cap_frames,
                               ctypes.byref(nf)), net)
    out = np.array([(r.kernel, r.layer, r.frame, r.ms)
                    for r in recs[:min(n.value, cap)]],
                   dtype=[("kernel", "i4"), ("layer", "i4"), ("frame", "i4"),
                          ("ms", "f4")])
    return out, counts[:min(nf.value, cap_frames)]
