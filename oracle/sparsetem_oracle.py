"""CPU oracle of SparseTem's Diff Computation (numpy, fp64 accumulation).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

What is computed (paper, section "Skipping Non-zero Delta Pixels" and
"Design of SparseBatch"):

* The chunk's first frame (reference frame) is encoded densely; this
  initialises the Subtraction buffer (the last committed input) and, for
  every layer followed by a non-linear operation or producing the network
  output, the cached pre-activation ``P`` that the non-linear op needs.
* Each later frame (diff frame) is encoded by Diff Computation:
  Subtraction, a per-pixel truncation threshold, convolution on the
  remaining diff pixels only (linearity, Eq. 2), Accumulation onto the
  cached pre-activation, and non-linear handling by reconstructing the dense
  value before the non-linearity and re-sparsifying after it (Eq. 3).

Readings of points the paper leaves open (all listed in the design notes):

1. A pixel is kept iff max over channels of |delta| is strictly greater
   than the threshold, so threshold 0 keeps exactly the diff pixels of the
   Subtraction section (a zero pixel has all channels zero).
2. Subtraction is taken against the last committed input: kept pixels
   commit their new value, truncated ones keep accumulating change.
3. Rows truncated inside the network are dropped (no residual carried);
   the non-linear op reconstructs from the cached pre-activation only.
   Optional residual carry (``carry=True``, the output-buffer semantics the
   paper attributes to DeltaCNN): every emitted tensor keeps the sum of
   the deltas its consumers received (Y_hat); a candidate row emits
   e_new - Y_hat, where e is the layer's dense emitted value (f(P), pooled
   or gated; P itself for a layer without non-linearity, which then keeps
   P too), kept rows add their rounded delta to Y_hat and truncated rows
   carry their residual until the site is affected again.
   Optional frozen squeeze-excitation (``frozen_se=True``, an approximation
   of reading 6, flagged as inexact): the gates s computed in the reference
   frame are kept for the diff frames of the chunk, so the layer emits
   f(P_new) * s - f(P_old) * s at its affected sites only.
4. One threshold per produced tensor: ``thr[0]`` masks the frame delta,
   ``thr[j+1]`` masks layer j's emitted delta (shared by all consumers).
5. Bias enters only the reference pass; it cancels in deltas (Eq. 2).
6. Convolution / max-pool follow PyTorch's conv2d / max_pool2d geometry
   (stride, zero padding, groups; -inf pool padding).  The delta of a
   pooled layer is max_window f(P_new) - max_window f(P_old).  A
   squeeze-excitation layer keeps its gates s (per image and channel) as
   state; its delta is f(P_new) * s_new - f(P_old) * s_old at every site,
   with s recomputed from the dense activation of the frame.
7. Sums are accumulated in fp64 and rounded once to f32; the pre-activation
   state is f32; emitted deltas are rounded to the storage dtype with
   round-to-nearest-even; the mask is taken on the rounded values.
   Optional bf16 state (``state_bf16=True``, an approximation that halves
   the state's memory): every stored pre-activation -- the reference
   pass's and each update's f32 result -- is rounded to bf16 (nearest,
   ties to even) before the activation sees it, so the emitted delta is
   f(P_new) - f(P_old) of the stored values.  Not with max-pooled layers
   or residual carry.

Layout: NHWC; pixel id p = (n * H + y) * W + x.
"""

import numpy as np

ACT_NONE, ACT_RELU, ACT_SILU = 0, 1, 2


# ---------------------------------------------------------------- rounding

def round_storage(x, dtype):
    """Round values (already f32-representable, or rounded to f32 first)
    to the storage dtype with round-to-nearest-even; returns float64."""
    x32 = np.asarray(x, dtype=np.float32)
    if dtype == "f32":
        return x32.astype(np.float64)
    if dtype == "f16":
        return x32.astype(np.float16).astype(np.float64)
    if dtype == "bf16":
        # keep the top 16 bits of the f32 pattern, rounding to nearest even
        # (the sum stays below 2^32 for every finite or infinite pattern)
        u = np.array(x32, dtype=np.float32, copy=True).view(np.uint32)
        r = (u >> 16) & 1
        r += 0x7FFF
        u += r
        u &= 0xFFFF0000
        return u.view(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype}")


def f32(x):
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def activation(x32, act):
    """The layer's non-linearity evaluated on f32 values in fp64 and rounded
    to f32: identity, ReLU max(x, 0), or SiLU x / (1 + exp(-x))."""
    x = np.asarray(x32, dtype=np.float32).astype(np.float64)
    if act == ACT_NONE:
        y = x
    elif act == ACT_RELU:
        y = np.maximum(x, 0.0)
    elif act == ACT_SILU:
        y = x / (1.0 + np.exp(-x))
    else:
        raise ValueError(f"unknown activation {act}")
    return y.astype(np.float32)


# ------------------------------------------------------- dense definitions

def out_size(n, k, s, p):
    return (n + 2 * p - k) // s + 1


def conv2d_nhwc(x, w, b, stride, pad, groups=1):
    """Dense convolution (cross-correlation), Eq. 1 extended to stride,
    zero padding and groups:
    O[n,y,x,co] = b[co] + sum_{ci in group(co)} sum_{ky,kx}
                  W[co, ci', ky, kx] * X[n, y*sh - ph + ky, x*sw - pw + kx, ci]
    x: [N,H,W,Cin], w: [Cout, Cin/groups, kh, kw]; returns float64."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    N, H, W, Cin = x.shape
    Cout, cig, kh, kw = w.shape
    sh, sw = stride
    ph, pw = pad
    Ho, Wo = out_size(H, kh, sh, ph), out_size(W, kw, sw, pw)
    cog = Cout // groups
    xp = np.zeros((N, H + 2 * ph, W + 2 * pw, Cin))
    xp[:, ph:ph + H, pw:pw + W, :] = x
    out = np.zeros((N, Ho, Wo, Cout))
    if b is not None:
        out += np.asarray(b, dtype=np.float64)
    for ky in range(kh):
        for kx in range(kw):
            patch = xp[:, ky:ky + sh * (Ho - 1) + 1:sh,
                       kx:kx + sw * (Wo - 1) + 1:sw, :]
            if cig == 1 and cog == 1:
                # depthwise: each channel with its own weight
                out += patch * w[:, 0, ky, kx]
                continue
            for g in range(groups):
                # contiguous operands, so that the product runs as one
                # library matrix product per offset and group
                pg = np.ascontiguousarray(
                    patch[..., g * cig:(g + 1) * cig]).reshape(-1, cig)
                wg = np.ascontiguousarray(w[g * cog:(g + 1) * cog, :, ky, kx])
                out[..., g * cog:(g + 1) * cog] += (pg @ wg.T).reshape(
                    N, Ho, Wo, cog)
    return out


def maxpool_nhwc(x, k, s, p):
    """Dense max-pool with -inf padding (PyTorch max_pool2d geometry)."""
    x = np.asarray(x, dtype=np.float64)
    N, H, W, C = x.shape
    Ho, Wo = out_size(H, k[0], s[0], p[0]), out_size(W, k[1], s[1], p[1])
    xp = np.full((N, H + 2 * p[0], W + 2 * p[1], C), -np.inf)
    xp[:, p[0]:p[0] + H, p[1]:p[1] + W, :] = x
    out = np.full((N, Ho, Wo, C), -np.inf)
    for ky in range(k[0]):
        for kx in range(k[1]):
            out = np.maximum(out, xp[:, ky:ky + s[0] * (Ho - 1) + 1:s[0],
                                     kx:kx + s[1] * (Wo - 1) + 1:s[1], :])
    return out


def se_gates(a32, L):
    """Squeeze-excitation gates of activation map a32 [N,H,W,C] (f32):
    s[n] = sigmoid(W2 @ silu(W1 @ mean_hw(a[n]) + b1) + b2), each stage
    evaluated in fp64 and rounded to f32."""
    a = np.asarray(a32, dtype=np.float32).astype(np.float64)
    m = f32(a.mean(axis=(1, 2)))                           # [N, C]
    w1 = np.asarray(L.se_w1, np.float64)
    w2 = np.asarray(L.se_w2, np.float64)
    z = f32(m.astype(np.float64) @ w1.T + np.asarray(L.se_b1, np.float64))
    z = activation(z, ACT_SILU)
    e = z.astype(np.float64) @ w2.T + np.asarray(L.se_b2, np.float64)
    return f32(1.0 / (1.0 + np.exp(-f32(e).astype(np.float64))))


def se_apply(a32, s):
    """Channel gating a * s (f32 product) of a [N,H,W,C] by s [N,C]."""
    return f32(np.asarray(a32, np.float64) * np.asarray(s, np.float64)
               [:, None, None, :])


# ------------------------------------------------------- sparse geometry

def window_targets(pix, in_hw, out_hw, k, s, p):
    """Input-to-output geometry of a sliding window (conv or pool).

    For each input site i in ``pix`` (ascending pixel ids on the input grid)
    and each window offset (ky, kx) in row-major order, the output site o
    whose window places offset (ky, kx) on i is
    o = ((iy + ph - ky) / sh, (ix + pw - kx) / sw) when both divisions are
    exact and in range.  Returns (offset, in_pix, out_pix) int64 triples,
    grouped by offset and, within an offset, ascending in in_pix (and hence
    in out_pix).  With a 3x3 window, stride 1 and pad 1, one interior site
    reaches 9 outputs: the dense amplification of the Truncation threshold
    section."""
    pix = np.asarray(pix, dtype=np.int64)
    Hi, Wi = in_hw
    Ho, Wo = out_hw
    n, rem = np.divmod(pix, Hi * Wi)
    iy, ix = np.divmod(rem, Wi)
    ks, ins, outs = [], [], []
    for ky in range(k[0]):
        for kx in range(k[1]):
            ty = iy + p[0] - ky
            tx = ix + p[1] - kx
            ok = (ty >= 0) & (tx >= 0) & (ty % s[0] == 0) & (tx % s[1] == 0)
            oy, ox = ty // s[0], tx // s[1]
            ok &= (oy < Ho) & (ox < Wo)
            ks.append(np.full(int(ok.sum()), ky * k[1] + kx, np.int64))
            ins.append(pix[ok])
            outs.append((n[ok] * Ho + oy[ok]) * Wo + ox[ok])
    if not ks:
        return np.zeros((0, 3), np.int64)
    return np.stack([np.concatenate(ks), np.concatenate(ins),
                     np.concatenate(outs)], axis=1)


def rulebook(pix, in_hw, out_hw, k, s, p):
    """Rulebook of a convolution layer: the (offset, in_pix, out_pix) pairs
    on which the delta convolution must compute (Eq. 2 restricted to diff
    pixels).  Canonical order: offset-major, then ascending in_pix."""
    return window_targets(pix, in_hw, out_hw, k, s, p)


# ------------------------------------------------------------- the network

class _Geom:
    def __init__(self, L, in_shape):
        N, H, W, C = in_shape
        if C != L.c_in:
            raise ValueError(f"channel mismatch {C} != {L.c_in}")
        self.N, self.Hi, self.Wi = N, H, W
        self.Ho = out_size(H, L.k[0], L.s[0], L.p[0])
        self.Wo = out_size(W, L.k[1], L.s[1], L.p[1])
        self.pool = L.pool_k[0] > 0
        if self.pool:
            self.Hp = out_size(self.Ho, L.pool_k[0], L.pool_s[0], L.pool_p[0])
            self.Wp = out_size(self.Wo, L.pool_k[1], L.pool_s[1], L.pool_p[1])
        else:
            self.Hp, self.Wp = self.Ho, self.Wo
        self.C = L.c_out


def _is_stateful(layers, i):
    L = layers[i]
    return (L.act != ACT_NONE or L.pool_k[0] > 0 or L.se_mid > 0
            or i == len(layers) - 1)


def _apply_offset(rows, w, ky, kx, groups):
    """rows [n, Cin] (fp64) times the offset-(ky,kx) slice of the weights,
    respecting groups; returns [n, Cout] fp64."""
    Cout, cig = w.shape[0], w.shape[1]
    cog = Cout // groups
    wk = np.ascontiguousarray(w[:, :, ky, kx])  # [Cout, Cin/groups]
    if groups == 1:
        return rows @ wk.T
    if cig == 1 and cog == 1:                 # depthwise
        return rows * wk[:, 0][None, :]
    out = np.zeros((rows.shape[0], Cout))
    for g in range(groups):
        out[:, g * cog:(g + 1) * cog] = (rows[:, g * cig:(g + 1) * cig]
                                         @ wk[g * cog:(g + 1) * cog].T)
    return out


def dense_forward(layers, frame, dtype, with_se=False, all_pre=False,
                  state_dtype="f32"):
    """Plain dense forward of one frame (the definition the diff chain must
    reproduce at threshold 0): returns (out, P, acts) where P[i] is the f32
    pre-activation of every stateful layer (of every layer with all_pre),
    acts[i] the emitted activation rounded to the storage dtype, and out
    the f32 network output; with with_se also the squeeze-excitation gates
    S[i].  state_dtype "bf16": a stateful layer's pre-activation is rounded
    to bf16 before its activation (the bf16-state reading of item 7)."""
    acts = {-1: round_storage(frame, dtype)}
    P = {}
    S = {}
    out = None
    for i, L in enumerate(layers):
        a = conv2d_nhwc(acts[L.src], L.weight, L.bias, L.s, L.p, L.groups)
        if L.residual_src != -2:
            a = a + acts[L.residual_src]
        p32 = f32(a)
        if all_pre:
            P[i] = p32
        if _is_stateful(layers, i):
            if state_dtype == "bf16":
                p32 = f32(round_storage(p32, "bf16"))
            P[i] = p32
            e = activation(p32, L.act).astype(np.float64)
            if L.pool_k[0] > 0:
                e = maxpool_nhwc(e, L.pool_k, L.pool_s, L.pool_p)
            e32 = f32(e)
            if L.se_mid:
                S[i] = se_gates(e32, L)
                e32 = se_apply(e32, S[i])
        else:
            e32 = p32
        acts[i] = round_storage(e32, dtype)
        if i == len(layers) - 1:
            out = e32
    return (out, P, acts, S) if with_se else (out, P, acts)


class OracleNet:
    """Stateful diff encoder over one stream of frames (batch N images)."""

    def __init__(self, layers, batch, H, W, C, dtype="f32", carry=False,
                 frozen_se=False, state_bf16=False):
        if dtype not in ("f32", "f16", "bf16"):
            raise ValueError(dtype)
        if carry and frozen_se:
            raise ValueError("carry and frozen_se are exclusive")
        if state_bf16 and (carry or any(L.pool_k[0] > 0 for L in layers)):
            raise ValueError("a bf16 state excludes carry and max-pools")
        self.layers = list(layers)
        self.dtype = dtype
        self.carry = carry
        self.frozen_se = frozen_se
        self.state_dtype = "bf16" if state_bf16 else "f32"
        self.in_shape = (batch, H, W, C)
        shapes = {-1: self.in_shape}
        self.geo = []
        for i, L in enumerate(self.layers):
            if not (-1 <= L.src < i):
                raise ValueError("src must name an earlier layer")
            g = _Geom(L, shapes[L.src])
            if L.residual_src != -2:
                rs = shapes[L.residual_src]
                if rs != (batch, g.Ho, g.Wo, L.c_out):
                    raise ValueError("residual shape mismatch")
            self.geo.append(g)
            shapes[i] = (batch, g.Hp, g.Wp, L.c_out)
        self.shapes = shapes
        self.stateful = [_is_stateful(self.layers, i)
                         for i in range(len(self.layers))]
        self.xhat = None
        self.P = {}
        self.S = {}
        self.Y = {}        # residual carry: consumers' view of each tensor
        self.last = None

    # -- reference frame ---------------------------------------------------
    def encode_reference(self, frame):
        """Dense computation on the reference frame; initialises the
        Subtraction buffer and the cached pre-activations (SparseBatch)."""
        frame = np.asarray(frame, dtype=np.float64)
        assert frame.shape == self.in_shape
        out, P, acts, S = dense_forward(self.layers, frame, self.dtype,
                                        with_se=True, all_pre=self.carry,
                                        state_dtype=self.state_dtype)
        self.xhat = round_storage(frame, self.dtype)
        self.P = {i: p.copy() for i, p in P.items()}
        self.S = {i: g.copy() for i, g in S.items()}
        if self.carry:
            # the reference frame emits every site: consumers hold acts
            self.Y = {i: f32(acts[i]).reshape(-1, L.c_out).copy()
                      for i, L in enumerate(self.layers)}
        self.last = dict(kind="reference", out=out, acts=acts)
        return out

    # -- diff frame ----------------------------------------------------------
    def encode_diff(self, frame, thr):
        """Diff Computation of one frame against the committed state.
        ``thr`` has len(layers)+1 entries (reading 4)."""
        if self.xhat is None:
            raise RuntimeError("encode_diff before encode_reference")
        thr = [float(t) for t in thr]
        assert len(thr) == len(self.layers) + 1
        frame = np.asarray(frame, dtype=np.float64)
        N, H, W, C = self.in_shape
        tensors, layer_art = [], []

        # Subtraction: X_delta = X - X_hat, in f32 from the stored values.
        D = (f32(frame) - f32(self.xhat)).reshape(N * H * W, C)
        dmax = np.abs(D).max(axis=1) if C else np.zeros(N * H * W)
        keep = dmax > thr[0]                          # reading 1
        A0 = np.flatnonzero(keep)
        rows0 = round_storage(D[A0], self.dtype)
        # Commit the kept pixels to the Subtraction buffer (reading 2).
        xh = self.xhat.reshape(N * H * W, C)
        xh[A0] = frame.reshape(N * H * W, C)[A0]
        tensors.append(dict(cand=np.arange(N * H * W), cand_max=dmax.astype(
            np.float64), pix=A0, rows=rows0, grid=(N, H, W), C=C))

        for i, L in enumerate(self.layers):
            g = self.geo[i]
            src = tensors[L.src + 1]
            skip = (tensors[L.residual_src + 1] if L.residual_src != -2
                    else None)
            if self.carry:
                R, O, dP32 = self._linear(
                    i, src["pix"], src["rows"],
                    None if skip is None else skip["pix"],
                    None if skip is None else skip["rows"])
                d32, cand, Q = self._carry_delta(i, O, dP32)
                d = round_storage(d32, self.dtype)
            else:
                st = self._step(i, src["pix"], src["rows"],
                                None if skip is None else skip["pix"],
                                None if skip is None else skip["rows"],
                                self.P.get(i), self.S.get(i))
                R, O, Q, cand, d = (st["rulebook"], st["O"], st["Q"],
                                    st["cand"], st["cand_rows"])
                if L.se_mid and not self.frozen_se:
                    self.S[i] = st["S"]
            cmax = np.abs(d).max(axis=1) if len(cand) else np.zeros(0)
            kept = cmax > thr[i + 1]                     # readings 1 and 3
            if self.carry:
                # kept rows reach the consumers; truncated rows carry over
                Y = self.Y[i]
                Y[cand[kept]] = f32(Y[cand[kept]].astype(np.float64)
                                    + d[kept])
            tensors.append(dict(cand=cand, cand_max=cmax, cand_rows=d,
                                pix=cand[kept], rows=d[kept],
                                grid=(N, g.Hp, g.Wp), C=L.c_out))
            layer_art.append(dict(rulebook=R, O=O, Q=Q, pairs=len(R)))

        # Accumulation: the dense output of the current frame.
        out = self._dense_output()
        self.last = dict(kind="diff", out=out, tensors=tensors,
                         layers=layer_art, thr=thr)
        return out

    def _linear(self, i, pix, rows, skip_pix=None, skip_rows=None):
        """Linear part of layer i on its input's kept rows (pixel ids `pix`,
        ascending, values `rows`) and its residual input's (or None):
        the rulebook, the affected output sites O (the rulebook's outputs
        and the residual's kept sites, ascending) and
        dP[o] = sum over rulebook pairs of W_k . delta[i] (+ the residual
        delta), Eq. 2 without bias, accumulated in fp64 and rounded once to
        f32.  Returns (rulebook, O, dP32)."""
        L, g = self.layers[i], self.geo[i]
        R = rulebook(pix, (g.Hi, g.Wi), (g.Ho, g.Wo), L.k, L.s, L.p)
        affected = [R[:, 2]]
        if skip_pix is not None:
            affected.append(np.asarray(skip_pix, np.int64))
        O = np.unique(np.concatenate(affected)).astype(np.int64)
        dP = np.zeros((len(O), L.c_out))
        w = np.asarray(L.weight, dtype=np.float64)
        for k in range(L.k[0] * L.k[1]):
            sel = R[:, 0] == k
            if not sel.any():
                continue
            ri = np.searchsorted(pix, R[sel, 1])
            ro = np.searchsorted(O, R[sel, 2])
            dP[ro] += _apply_offset(np.asarray(rows)[ri], w, k // L.k[1],
                                    k % L.k[1], L.groups)
        if skip_pix is not None and len(skip_pix):
            dP[np.searchsorted(O, skip_pix)] += skip_rows
        return R, O, f32(dP)

    def _step(self, i, pix, rows, skip_pix, skip_rows, P, S):
        """Layer i of Diff Computation (no residual carry) on the given
        inputs: the linear part (_linear), then, for a layer that holds a
        cached pre-activation, Accumulation onto P (the dense f32 state
        [N, Ho, Wo, C], updated in place) and the non-linear handling of
        Eq. 3 -- reconstruct the dense value before f, re-sparsify after it
        (pooled: max_window f(P_new) - max_window f(P_old); squeeze-
        excitation: f(P_new) * s_new - f(P_old) * s_old with the gates S of
        the previous frame, or the frozen gates) -- else the linear delta
        passes on.  Returns the rulebook, O, the pooled candidates Q (or
        None), the candidate sites and their deltas rounded to the storage
        dtype (before truncation), and the new gates S."""
        L, g = self.layers[i], self.geo[i]
        N = self.in_shape[0]
        R, O, dP32 = self._linear(i, pix, rows, skip_pix, skip_rows)
        Q = None
        S_new = S
        if self.stateful[i]:
            Pg = P.reshape(N * g.Ho * g.Wo, L.c_out)
            P_old = Pg[O].copy()
            P_new = f32(P_old.astype(np.float64) + dP32)
            if self.state_dtype == "bf16":
                P_new = f32(round_storage(P_new, "bf16"))
            if L.se_mid and self.frozen_se:
                # frozen gates: a per-image, per-channel scale
                Pg[O] = P_new
                s = S.reshape(N, L.c_out)[O // (g.Ho * g.Wo)]
                d32 = f32(f32(activation(P_new, L.act).astype(np.float64)
                              * s)
                          - f32(activation(P_old, L.act).astype(np.float64)
                                * s))
                cand = O
            elif L.se_mid:
                # Squeeze-excitation (reading 6): the gates follow the
                # dense activation, so every site's output moves:
                # delta = f(P_new) * s_new - f(P_old) * s_old.
                a_old = activation(Pg.reshape(N, g.Ho, g.Wo, L.c_out), L.act)
                Pg[O] = P_new
                a_new = activation(Pg.reshape(N, g.Ho, g.Wo, L.c_out), L.act)
                S_new = se_gates(a_new, L)
                e_old = se_apply(a_old, S).reshape(-1, L.c_out)
                e_new = se_apply(a_new, S_new).reshape(-1, L.c_out)
                d32 = f32(e_new.astype(np.float64)
                          - e_old.astype(np.float64))
                cand = np.arange(N * g.Ho * g.Wo, dtype=np.int64)
            elif g.pool:
                T = window_targets(O, (g.Ho, g.Wo), (g.Hp, g.Wp),
                                   L.pool_k, L.pool_s, L.pool_p)
                Q = np.unique(T[:, 2]).astype(np.int64)
                e_old = maxpool_nhwc(activation(
                    Pg.reshape(N, g.Ho, g.Wo, L.c_out), L.act),
                    L.pool_k, L.pool_s, L.pool_p)
                Pg[O] = P_new
                e_new = maxpool_nhwc(activation(
                    Pg.reshape(N, g.Ho, g.Wo, L.c_out), L.act),
                    L.pool_k, L.pool_s, L.pool_p)
                e_old = e_old.reshape(-1, L.c_out)[Q]
                e_new = e_new.reshape(-1, L.c_out)[Q]
                d32 = f32(f32(e_new).astype(np.float64)
                          - f32(e_old).astype(np.float64))
                cand = Q
            else:
                Pg[O] = P_new
                d32 = f32(activation(P_new, L.act).astype(np.float64)
                          - activation(P_old, L.act).astype(np.float64))
                cand = O
        else:
            d32 = dP32
            cand = O
        return dict(rulebook=R, O=O, Q=Q, cand=cand,
                    cand_rows=round_storage(d32, self.dtype), S=S_new)

    def layer_step(self, i, pix, rows, skip_pix=None, skip_rows=None,
                   P_old=None, S_old=None):
        """One layer of Diff Computation on inputs supplied by the caller,
        leaving the net untouched (a teacher-forced step): the kept rows of
        the layer's input and residual input, the cached pre-activation
        before the frame (dense f32 [N, Ho, Wo, C]; None for a layer
        without one) and the previous frame's squeeze-excitation gates.
        Returns _step's artefacts plus the updated dense state "P"."""
        if self.carry:
            raise ValueError("layer_step follows the drop semantics")
        P = None if P_old is None else f32(P_old).copy()
        st = self._step(i, np.asarray(pix, np.int64),
                        np.asarray(rows, np.float64),
                        None if skip_pix is None else
                        np.asarray(skip_pix, np.int64),
                        None if skip_rows is None else
                        np.asarray(skip_rows, np.float64), P, S_old)
        st["P"] = P
        return st

    def _carry_delta(self, i, O, dP32):
        """Residual carry: apply the update to P (every layer keeps P) and
        return (delta = e_new - Y_hat at the candidate sites, candidates,
        pooled candidates or None), e being the layer's dense emitted value
        (f(P), pooled or gated; P for a layer without non-linearity)."""
        L, g = self.layers[i], self.geo[i]
        N = self.in_shape[0]
        Pg = self.P[i].reshape(N * g.Ho * g.Wo, L.c_out)
        Pg[O] = f32(Pg[O].astype(np.float64) + dP32)
        Y = self.Y[i]
        if L.se_mid:
            a_new = activation(Pg.reshape(N, g.Ho, g.Wo, L.c_out), L.act)
            s_new = se_gates(a_new, L)
            self.S[i] = s_new
            e = se_apply(a_new, s_new).reshape(-1, L.c_out)
            cand = np.arange(N * g.Ho * g.Wo, dtype=np.int64)
            Q = None
        elif g.pool:
            T = window_targets(O, (g.Ho, g.Wo), (g.Hp, g.Wp), L.pool_k,
                               L.pool_s, L.pool_p)
            Q = np.unique(T[:, 2]).astype(np.int64)
            e = f32(maxpool_nhwc(activation(
                Pg.reshape(N, g.Ho, g.Wo, L.c_out), L.act),
                L.pool_k, L.pool_s, L.pool_p)).reshape(-1, L.c_out)[Q]
            cand = Q
        else:
            e = activation(Pg[O], L.act) if self.stateful[i] else Pg[O]
            cand = O
            Q = None
        d32 = f32(np.asarray(e, np.float64) - Y[cand].astype(np.float64))
        return d32, cand, Q

    def emitted(self, i):
        """The dense emitted value of layer i from the current state:
        f(P), pooled or gated (P for a layer without non-linearity)."""
        L, g = self.layers[i], self.geo[i]
        N = self.in_shape[0]
        P = self.P[i]
        if not self.stateful[i]:
            return P.reshape(-1, L.c_out)
        e = activation(P, L.act).astype(np.float64)
        if g.pool:
            e = maxpool_nhwc(e, L.pool_k, L.pool_s, L.pool_p)
        e = f32(e)
        if L.se_mid:
            e = se_apply(e, self.S[i])
        return np.asarray(e).reshape(-1, L.c_out)

    def _dense_output(self):
        i = len(self.layers) - 1
        L, g = self.layers[i], self.geo[i]
        e = activation(self.P[i], L.act).astype(np.float64)
        if g.pool:
            e = maxpool_nhwc(e, L.pool_k, L.pool_s, L.pool_p)
        e = f32(e)
        if L.se_mid:
            e = se_apply(e, self.S[i])
        return e

    # -- introspection -----------------------------------------------------
    def density(self, t):
        """Fraction of kept sites of tensor t (0 = frame delta, j+1 = layer
        j's emitted delta) in the last diff frame."""
        T = self.last["tensors"][t]
        N, H, W = T["grid"]
        return len(T["pix"]) / float(N * H * W)

    def flops(self):
        """Algorithmic FLOPs of the last diff frame:
        2 * sum over layers of pairs * Cin * Cout / groups."""
        tot = 0
        for L, art in zip(self.layers, self.last["layers"]):
            tot += 2 * art["pairs"] * L.c_in * L.c_out // L.groups
        return tot
