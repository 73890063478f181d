"""Torch-memory wrapper around the C ABI: owns the device weights and the
workspace as torch tensors and passes their addresses and the current HIP
stream to the library.  No computation happens here."""

from typing import Optional, Sequence

import numpy as np
import torch

from . import binding as B

TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16,
                "bf16": torch.bfloat16}


def layer_desc(L, w_ptr: int, b_ptr: Optional[int],
               se_ptrs=(None, None, None, None)) -> B.st_layer_desc:
    """Descriptor of one layer from an object with the LayerSpec fields
    (src, residual_src, c_in, c_out, groups, k, s, p, act, pool_k, pool_s,
    pool_p, se_mid); se_ptrs are the device addresses of the
    squeeze-excitation weights (w1, b1, w2, b2)."""
    return B.st_layer_desc(
        src=L.src, residual_src=L.residual_src, c_in=L.c_in, c_out=L.c_out,
        groups=L.groups, k_h=L.k[0], k_w=L.k[1], s_h=L.s[0], s_w=L.s[1],
        p_h=L.p[0], p_w=L.p[1], act=L.act, pool_k_h=L.pool_k[0],
        pool_k_w=L.pool_k[1], pool_s_h=L.pool_s[0], pool_s_w=L.pool_s[1],
        pool_p_h=L.pool_p[0], pool_p_w=L.pool_p[1], se_mid=L.se_mid,
        weight=w_ptr, bias=b_ptr, se_w1=se_ptrs[0], se_b1=se_ptrs[1],
        se_w2=se_ptrs[2], se_b2=se_ptrs[3])


class SparseTemNet:
    """One diff encoder: reference frame via ``encode_reference``, then
    diff frames via ``encode_diff``, or up to ``max_frames`` of them at once
    via ``encode_chunk`` (see include/sparsetem.h).  ``carry``: residual
    carry (ST_NET_RESIDUAL_CARRY); ``frozen_se``:
    squeeze-excitation gates kept from the reference frame
    (ST_NET_FROZEN_SE, an approximation); ``bf16_state``: pre-activation
    state stored in bf16 (ST_NET_BF16_STATE, an approximation);
    ``static_workspace``: bound to the library's own per-device workspace
    (st_bind_workspace_static) instead of a torch allocation."""

    def __init__(self, layers: Sequence, batch: int, H: int, W: int, C: int,
                 dtype: str = "f32", device="cuda", max_frames: int = 1,
                 carry: bool = False, frozen_se: bool = False,
                 bf16_state: bool = False, static_workspace: bool = False):
        self.dtype = dtype
        self.tdtype = TORCH_DTYPES[dtype]
        dev = torch.device(device)
        if dev.type == "cuda" and dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        self.n_layers = len(layers)
        self.has_se = any(getattr(L, "se_mid", 0) for L in layers)
        self.in_shape = (batch, H, W, C)
        self._w, self._b, descs = [], [], []
        for L in layers:
            w = torch.as_tensor(np.asarray(L.weight)).to(
                self.device, self.tdtype).contiguous()
            b = None
            if L.bias is not None:
                b = torch.as_tensor(np.asarray(L.bias)).to(
                    self.device, self.tdtype).contiguous()
            self._w.append(w)
            self._b.append(b)
            se = (None, None, None, None)
            if getattr(L, "se_mid", 0):
                t = [torch.as_tensor(np.asarray(x)).to(
                    self.device, self.tdtype).contiguous()
                    for x in (L.se_w1, L.se_b1, L.se_w2, L.se_b2)]
                self._w.extend(t)
                se = tuple(x.data_ptr() for x in t)
            descs.append(layer_desc(L, w.data_ptr(),
                                    None if b is None else b.data_ptr(), se))
        self.max_frames = max_frames
        self.carry = carry
        self.frozen_se = frozen_se
        self.bf16_state = bf16_state
        if carry or frozen_se or bf16_state:
            flags = ((B.NET_RESIDUAL_CARRY if carry else 0) |
                     (B.NET_FROZEN_SE if frozen_se else 0) |
                     (B.NET_BF16_STATE if bf16_state else 0))
            self.handle = B.st_create_net_ex(descs, batch, max_frames, H, W,
                                             C, B.DTYPE_CODES[dtype], flags)
        elif max_frames > 1:
            self.handle = B.st_create_net_chunked(descs, batch, max_frames,
                                                  H, W, C,
                                                  B.DTYPE_CODES[dtype])
        else:
            self.handle = B.st_create_net(descs, batch, H, W, C,
                                          B.DTYPE_CODES[dtype])
        self.ws_bytes = B.st_workspace_bytes(self.handle)
        if static_workspace:
            # the library's own per-device workspace: nothing allocated
            self.ws = None
            B.st_bind_workspace_static(self.handle, self._stream())
        else:
            self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8,
                                  device=self.device)
            B.st_bind_workspace(self.handle, self.ws.data_ptr(),
                                self.ws_bytes, self._stream())
        torch.cuda.current_stream(self.device).synchronize()
        self.out_shape = B.st_tensor_shape(self.handle, self.n_layers - 1)

    def _stream(self) -> int:
        return torch.cuda.current_stream(self.device).cuda_stream

    def _check_frame(self, frame):
        if (frame.device != self.device or frame.dtype != self.tdtype
                or tuple(frame.shape) != self.in_shape
                or not frame.is_contiguous()):
            raise ValueError("frame must be a contiguous NHWC device tensor "
                             f"{self.in_shape} of {self.tdtype}")

    def new_output(self):
        return torch.empty(self.out_shape, dtype=torch.float32,
                           device=self.device)

    def encode_reference(self, frame, out=None):
        self._check_frame(frame)
        out = self.new_output() if out is None else out
        B.st_encode_reference(self.handle, frame.data_ptr(), out.data_ptr(),
                              self._stream())
        return out

    def encode_diff(self, frame, thr, out=None, write_out=True):
        self._check_frame(frame)
        if len(thr) != self.n_layers + 1:
            raise ValueError("thr needs n_layers + 1 entries")
        if write_out and out is None:
            out = self.new_output()
        B.st_encode_diff(self.handle, frame.data_ptr(), thr,
                         out.data_ptr() if write_out else None,
                         self._stream())
        return out

    def set_threshold_control(self, controlled, fixed_thr, target=0.9,
                              eps=0.025, theta_max=1.0, theta0=None,
                              cycle_refs=1):
        """Online threshold adjustment on the device: `controlled` lists the
        indices (into thr) of the tensors whose threshold is searched;
        fixed_thr (n_layers + 1) holds the others'; a search cycle spans
        cycle_refs reference frames."""
        if len(fixed_thr) != self.n_layers + 1:
            raise ValueError("fixed_thr needs n_layers + 1 entries")
        flags = [0] * (self.n_layers + 1)
        for t in controlled:
            if not 0 <= t <= self.n_layers:
                raise ValueError("controlled tensor index out of range")
            flags[t] = 1
        B.st_set_threshold_control(self.handle, flags, fixed_thr, target, eps,
                                   theta_max,
                                   -1.0 if theta0 is None else theta0,
                                   self._stream(), cycle_refs)

    def encode_diff_adaptive(self, frame, out=None, write_out=True):
        """A diff frame with the device-adjusted thresholds, then one step
        of the adjustment."""
        self._check_frame(frame)
        if write_out and out is None:
            out = self.new_output()
        B.st_encode_diff_adaptive(self.handle, frame.data_ptr(),
                                  out.data_ptr() if write_out else None,
                                  self._stream())
        return out

    def thresholds(self):
        """The thresholds the next adaptive frame uses (synchronising)."""
        return B.st_get_thresholds(self.handle, self.n_layers + 1)

    def encode_chunk(self, frames, thr, out=None, write_out=True):
        """frames: contiguous device tensor [n_frames, *in_shape]; returns
        the outputs of every frame, [n_frames, *out_shape] (f32).  thr None:
        the device-adjusted thresholds, then one step of the adjustment
        from the whole chunk."""
        nf = frames.shape[0] if frames.dim() == 5 else -1
        if (frames.device != self.device or frames.dtype != self.tdtype
                or frames.dim() != 5 or tuple(frames.shape[1:]) !=
                self.in_shape or not frames.is_contiguous()):
            raise ValueError("frames must be a contiguous device tensor "
                             f"[n, {self.in_shape}] of {self.tdtype}")
        if thr is not None and len(thr) != self.n_layers + 1:
            raise ValueError("thr needs n_layers + 1 entries")
        if write_out and out is None:
            out = torch.empty((nf,) + tuple(self.out_shape),
                              dtype=torch.float32, device=self.device)
        if write_out and (tuple(out.shape) != (nf,) + tuple(self.out_shape)
                          or out.dtype != torch.float32
                          or not out.is_contiguous()):
            raise ValueError("out must be a contiguous f32 tensor "
                             f"[{nf}, {self.out_shape}]")
        if thr is None:
            B.st_encode_chunk_adaptive(self.handle, frames.data_ptr(), nf,
                                       out.data_ptr() if write_out else None,
                                       self._stream())
        else:
            B.st_encode_chunk(self.handle, frames.data_ptr(), nf, thr,
                              out.data_ptr() if write_out else None,
                              self._stream())
        return out

    def capture_diff(self, thr, out):
        """Capture one diff-frame encode with output `out` into a HIP graph:
        with fixed thresholds `thr` (encode_diff), or with thr None the
        device-adjusted ones and the adjustment's step
        (encode_diff_adaptive).  Returns a callable that encodes a frame by
        copying it into the graph's input slot and replaying the graph
        (the same kernels and arguments as the direct call; the
        squeeze-excitation gate slots are chosen on the device, so replays
        and direct calls interleave freely).  Requires a reference frame to
        have been encoded."""
        return DiffGraph(self, thr, out)

    def density(self, layer: int, image: int = -1) -> float:
        return B.st_layer_density(self.handle, layer, image)

    def tensor_shape(self, layer: int):
        return B.st_tensor_shape(self.handle, layer)

    def close(self):
        if self.handle:
            torch.cuda.current_stream(self.device).synchronize()
            B.st_destroy_net(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class DiffGraph:
    """A diff-frame encode replayed as a HIP graph (see
    SparseTemNet.capture_diff).  Every replay launches the same per-frame
    kernel sequence as st_encode_diff on the current stream."""

    def __init__(self, net: SparseTemNet, thr, out):
        if thr is not None and len(thr) != net.n_layers + 1:
            raise ValueError("thr needs n_layers + 1 entries")
        self.slot = torch.zeros(net.in_shape, dtype=net.tdtype,
                                device=net.device)
        self.out = out
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            if thr is None:
                B.st_encode_diff_adaptive(net.handle, self.slot.data_ptr(),
                                          out.data_ptr(), net._stream())
            else:
                B.st_encode_diff(net.handle, self.slot.data_ptr(), list(thr),
                                 out.data_ptr(), net._stream())

    def __call__(self, frame):
        self.slot.copy_(frame)
        self.graph.replay()
        return self.out
