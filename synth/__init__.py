"""Seeded synthetic inputs for the PyraMiD-LSTM workloads.

Shared by the oracle-side tests and the GPU path's tests/benchmark.  This module
draws random numbers and rounds them to the storage type; it holds none of the
method's arithmetic.

The paper's datasets (ISBI 2012 EM stacks, MRBrainS13 volumes; Section 3) are
not available, so synthetic volumes of their shapes stand in for them:
  mr       48 x 240 x 240 x 3   (MR brain: 48 slices of 240 x 240, 3 sequences)
  em       30 x 512 x 512 x 1   (EM: 30 slices of 512 x 512, one channel)
Weights follow the paper's initialisation, U(-0.1, 0.1) (Section 3,
"Experimental Setup"); biases are 0 except the forget-gate bias, 1.0.

Random streams: numpy default_rng(150607452 + 10 * cfg + k) with k = 0 for the
input volume, 1 for weights, 2 for labels; ad-hoc shapes pass their own seed.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

SEED_BASE = 150607452


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returned as fp32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).reshape(a.shape)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of bf16-representable fp32 values."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    a = np.asarray(a, dtype=np.float32)
    return round_bf16(a) if dtype == "bf16" else np.ascontiguousarray(a)


@dataclass
class LayerParams:
    wx: np.ndarray   # [6][4O][C][3][3]
    wh: np.ndarray   # [6][4O][O][3][3]
    b: np.ndarray    # [6][4O]


def layer_params(rng, C: int, O: int, dtype: str = "f32", K: int = 3,
                 forget_bias: float = 1.0) -> LayerParams:
    wx = rng.uniform(-0.1, 0.1, size=(6, 4 * O, C, K, K))
    wh = rng.uniform(-0.1, 0.1, size=(6, 4 * O, O, K, K))
    b = np.zeros((6, 4 * O))
    b[:, O:2 * O] = forget_bias
    return LayerParams(to_storage(wx, dtype), to_storage(wh, dtype), to_storage(b, dtype))


def fc_params(rng, Cin: int, Cout: int, dtype: str = "f32"):
    w = rng.uniform(-0.1, 0.1, size=(Cout, Cin))
    return to_storage(w, dtype), np.zeros(Cout, dtype=np.float32)


def box_mean3d(v: np.ndarray, k: int) -> np.ndarray:
    """Mean over the in-bounds voxels of a k x k x k box, per channel (fp64)."""
    r = k // 2
    out = np.asarray(v, dtype=np.float64)
    for ax in range(3):
        n = out.shape[ax]
        cs = np.cumsum(out, axis=ax)
        pad = [(0, 0)] * out.ndim
        pad[ax] = (1, 0)
        cs = np.pad(cs, pad)
        idx = np.arange(n)
        hi = np.minimum(idx + r + 1, n)
        lo = np.maximum(idx - r, 0)
        s = np.take(cs, hi, axis=ax) - np.take(cs, lo, axis=ax)
        shape = [1] * out.ndim
        shape[ax] = n
        out = s / (hi - lo).reshape(shape)
    return out


def volume(kind: str, N: int, D: int, H: int, W: int, C: int, rng) -> np.ndarray:
    if kind == "normal":
        v = rng.standard_normal((N, D, H, W, C))
    elif kind == "mr":
        v = rng.standard_normal((N, D, H, W, C))
        v = np.stack([box_mean3d(v[n], 5) for n in range(N)])
    elif kind == "em":
        v = rng.uniform(0.0, 1.0, size=(N, D, H, W, C))
    else:
        raise ValueError(kind)
    return v


@dataclass
class Workload:
    name: str
    N: int
    D: int
    H: int
    W: int
    C: int
    hidden: List[int]               # O of each PyraMiD-LSTM layer
    dtype: str = "f32"              # storage type: "f32" or "bf16"
    fc: bool = False                # per-voxel FC tanh (2 x hidden) after each layer
    classes: int = 0                # > 0: final linear + softmax
    labels: bool = False            # cross-entropy training step
    kind: str = "normal"
    cfg: int = 0
    seed: Optional[int] = None
    K: int = 3                      # filter size of every PyraMiD-LSTM layer
    # explicit hidden FC widths (overrides `fc`); one per layer, or one fewer
    # when the last layer feeds the output layer directly
    fc_widths: Optional[List[int]] = None

    def fc_width(self, li: int) -> Optional[int]:
        """Width of the hidden FC tanh after layer li (None: no FC there)."""
        if self.fc_widths is not None:
            return self.fc_widths[li] if li < len(self.fc_widths) else None
        return 2 * self.hidden[li] if self.fc else None

    def seeds(self):
        base = self.seed if self.seed is not None else SEED_BASE + 10 * self.cfg
        return base, base + 1, base + 2

    @property
    def voxels(self) -> int:
        return self.N * self.D * self.H * self.W

    def vdu_per_pass(self) -> int:
        """Voxel-direction updates per forward pass (6 per voxel per layer)."""
        return 6 * self.voxels * len(self.hidden)

    def layer_shapes(self):
        """(input channels, hidden units) of every PyraMiD-LSTM layer."""
        out, C = [], self.C
        for li, O in enumerate(self.hidden):
            out.append((C, O))
            w = self.fc_width(li)
            C = w if w is not None else O
        return out

    def flops_per_pass(self) -> int:
        """Algorithmic contraction flops of the layers (dense K x K stencils):
        2 * K^2 * 4O * (C + O) per voxel-direction update."""
        return sum(6 * self.voxels * 2 * self.K * self.K * 4 * O * (C + O)
                   for C, O in self.layer_shapes())


CONFIGS = {
    1: Workload("tiny 8x8x8x1 O=4 fwd f32", 1, 8, 8, 8, 1, [4], kind="normal", cfg=1),
    2: Workload("MR-like 48x240x240x3 O=16 fwd f32", 1, 48, 240, 240, 3, [16], kind="mr", cfg=2),
    3: Workload("EM-like 30x512x512x1 O=16 fwd f32", 1, 30, 512, 512, 1, [16], kind="em", cfg=3),
    4: Workload("8x64^3x3 3 layers O=16/32/64 + FC + softmax, bf16 storage", 8, 64, 64, 64, 3,
                [16, 32, 64], dtype="bf16", fc=True, classes=4, kind="normal", cfg=4),
    5: Workload("MR-like 48x240x240x3 2 layers O=16/32 + FC + softmax CE, fwd+bwd f32", 1, 48,
                240, 240, 3, [16, 32], fc=True, classes=4, labels=True, kind="mr", cfg=5),
}

# The network of Section 3 ("Experimental Setup"): 7 x 7 filters, PyraMiD-LSTM
# 16 -> FC tanh 25 -> PyraMiD-LSTM 32 -> FC tanh 45 -> PyraMiD-LSTM 64 -> output
# layer, on the last bootstrapping sub-volume of the MR data (25 slices of
# 240 x 240).  Five input channels and five classes are the reading under which
# the paper's weight count is matched (to within 2); labels for training.
PAPER_NET = Workload("paper network 7x7 16/25/32/45/64, MR sub-volume 25x240x240x5, "
                     "softmax, f32", 1, 25, 240, 240, 5, [16, 32, 64], classes=5,
                     labels=True, kind="mr", cfg=6, K=7, fc_widths=[25, 45])


@dataclass
class Instance:
    wl: Workload
    x: np.ndarray                                  # storage-rounded, fp32 array
    layers: List[LayerParams]
    fcs: List[Tuple[np.ndarray, np.ndarray]] = field(default_factory=list)
    head: Optional[Tuple[np.ndarray, np.ndarray]] = None
    labels: Optional[np.ndarray] = None


def make(wl: Workload) -> Instance:
    s_in, s_w, s_lab = wl.seeds()
    rin, rw, rlab = (np.random.default_rng(s) for s in (s_in, s_w, s_lab))
    x = to_storage(volume(wl.kind, wl.N, wl.D, wl.H, wl.W, wl.C, rin), wl.dtype)
    layers, fcs = [], []
    C = wl.C
    for li, O in enumerate(wl.hidden):
        layers.append(layer_params(rw, C, O, wl.dtype, K=wl.K))
        w = wl.fc_width(li)
        if w is not None:
            fcs.append(fc_params(rw, O, w, wl.dtype))
            C = w
        else:
            C = O
    head = fc_params(rw, C, wl.classes, wl.dtype) if wl.classes else None
    labels = None
    if wl.labels:
        labels = rlab.integers(0, wl.classes, size=wl.voxels).astype(np.int32)
    return Instance(wl, x, layers, fcs, head, labels)


def config(cfg: int) -> Instance:
    return make(CONFIGS[cfg])


def image2d(N: int, H: int, W: int, C: int, O: int, K: int, seed: int, dtype: str = "f32",
            scale: float = 0.2):
    """Seeded image batch x [N][H][W][C] ~ N(0, 1) and 2D layer parameters
    wx [4][4O][C][K], wh [4][4O][O][K] ~ U(-scale, scale), b [4][4O] (forget
    gate 1, others 0), rounded to the storage type."""
    rin, rw = np.random.default_rng(seed), np.random.default_rng(seed + 7919)
    x = rin.standard_normal((N, H, W, C))
    wx = rw.uniform(-scale, scale, size=(4, 4 * O, C, K))
    wh = rw.uniform(-scale, scale, size=(4, 4 * O, O, K))
    b = np.zeros((4, 4 * O))
    b[:, O:2 * O] = 1.0
    return tuple(to_storage(a, dtype) for a in (x, wx, wh, b))


def upstream_grad(shape, seed: int, dtype: str = "f32") -> np.ndarray:
    """Seeded dL/dh for single-layer backward tests: N(0, 1)."""
    return to_storage(np.random.default_rng(seed).standard_normal(shape), dtype)
