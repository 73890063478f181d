"""Online truncation-threshold adjustment by iterative binary search (IBST).

Host-side controller for the per-tensor thresholds ``thr`` that
``st_encode_diff`` takes (Section "Online Truncation Threshold
Adjustment").  Every controlled tensor t (the frame delta, t = 0, or the
delta emitted by layer t - 1) owns a threshold theta_t and a bracket
[lo_t, hi_t].  After each diff frame the measured sparsity s_t (fraction of
sites whose delta was truncated or never produced, 1 - density) moves
theta_t one bisection step toward the target band [T - eps, T + eps]:

* s_t < T - eps (too dense):  lo_t = theta_t, theta_t = (theta_t + hi_t) / 2
* s_t > T + eps (too sparse): hi_t = theta_t, theta_t = (lo_t + theta_t) / 2
* otherwise theta_t stays.

One such search (BST) runs per cycle; ``start_cycle`` restarts every bracket
at [0, theta_max] so that a cycle can follow inputs whose sparsity curve has
moved since the last one (the iterative part).  Readings where the paper
gives no value: theta_max = 1.0, T = 0.9, eps = 0.025, the cycle is the
chunk (one reference frame), theta is carried from one cycle to the next,
and the first cycle starts at theta_max / 2.  Tensors that are not
controlled keep a fixed threshold.

Higher thresholds truncate more rows, so sparsity is non-decreasing in
theta; on such a curve the bracket always contains the band's theta
interval, and a band of width w in theta is reached within
ceil(log2(theta_max / w)) + 1 frames of a cycle.
"""

from typing import Iterable, List, Optional, Sequence

import numpy as np


class IBST:
    def __init__(self, n_tensors: int, controlled: Iterable[int],
                 target: float = 0.9, eps: float = 0.025,
                 theta_max: float = 1.0, fixed: float = 0.0,
                 theta0: Optional[float] = None):
        if not 0.0 <= target <= 1.0 or eps < 0.0 or theta_max <= 0.0:
            raise ValueError("need 0 <= target <= 1, eps >= 0, theta_max > 0")
        self.n = int(n_tensors)
        self.ctl = sorted(set(int(t) for t in controlled))
        if any(t < 0 or t >= self.n for t in self.ctl):
            raise ValueError("controlled tensor index out of range")
        self.target, self.eps, self.theta_max = target, eps, theta_max
        self.theta = np.full(self.n, float(fixed))
        self.theta[self.ctl] = theta_max / 2 if theta0 is None else theta0
        self.lo = np.zeros(self.n)
        self.hi = np.full(self.n, theta_max)
        self.frames_in_cycle = 0

    def thresholds(self) -> List[float]:
        """Thresholds for the next diff frame (``thr`` of st_encode_diff)."""
        return [float(v) for v in self.theta]

    def start_cycle(self) -> None:
        """A new chunk starts: restart every bracket at [0, theta_max]."""
        self.lo[:] = 0.0
        self.hi[:] = self.theta_max
        self.frames_in_cycle = 0

    def update(self, sparsity: Sequence[float]) -> List[float]:
        """One bisection step per controlled tensor from the sparsities the
        last diff frame measured (indexed like ``thr``); returns the
        thresholds for the next frame."""
        s = np.asarray(sparsity, dtype=np.float64)
        if s.shape != (self.n,):
            raise ValueError(f"need {self.n} sparsities, got {s.shape}")
        for t in self.ctl:
            th = self.theta[t]
            if s[t] < self.target - self.eps:
                self.lo[t] = th
                self.theta[t] = 0.5 * (th + self.hi[t])
            elif s[t] > self.target + self.eps:
                self.hi[t] = th
                self.theta[t] = 0.5 * (self.lo[t] + th)
        self.frames_in_cycle += 1
        return self.thresholds()


def sparsity_from_counts(active: Sequence[int],
                         grids: Sequence[int]) -> np.ndarray:
    """1 - |A_t| / sites_t for each emitted tensor, from the kept-row
    counters the library reports."""
    a = np.asarray(active, dtype=np.float64)
    g = np.asarray(grids, dtype=np.float64)
    return 1.0 - a / g


def nonlinear_tensors(layers, include_input: bool = True) -> List[int]:
    """Indices (into ``thr``) of the tensors a controller adjusts: the
    deltas emitted after a non-linearity (activation, max-pool or
    squeeze-excitation), and the frame delta when ``include_input``."""
    out = [0] if include_input else []
    for j, L in enumerate(layers):
        if L.act != 0 or (L.pool_k and L.pool_k[0] > 0) or L.se_mid:
            out.append(j + 1)
    return out
