"""Helpers for the GPU parity tests: device transfer and error metrics."""
from __future__ import annotations

import sys

import numpy as np
import torch

from paper_1506_07452_amd.network import LayerW

DEV = "cuda:0"
TOL = {"f32": 1e-4, "bf16": 2e-2}


def tdt(dtype: str):
    return torch.float32 if dtype == "f32" else torch.bfloat16


def dev(a, dtype="f32"):
    """numpy (storage-rounded fp32 values) -> contiguous device tensor."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(tdt(dtype)).contiguous()


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def layer_dev(L, dtype="f32"):
    return LayerW(dev(L.wx, dtype), dev(L.wh, dtype), dev(L.b, dtype))


def normwise(got, ref):
    """max|got - ref| / max|ref| (the tolerance metric of the parity tests)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = np.abs(ref).max()
    if scale == 0:
        return float(np.abs(got).max())
    return float(np.abs(got - ref).max() / scale)


def say(*a):
    """Name the case before a GPU step (survives a crash of the process)."""
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def saved_view(saved, name, shape):
    """One array of a training forward's `saved` buffer as float64 numpy, in
    the layout the C header documents: gates, c^d, h^d, each starting at the
    next 256-byte boundary, shape [6][N][D][H][W][4O or O]."""
    N, D, H, W, C, O = shape
    counts = {"gates": 6 * N * D * H * W * 4 * O, "cell": 6 * N * D * H * W * O,
              "hd": 6 * N * D * H * W * O}
    off = 0
    for key in ("gates", "cell", "hd"):
        off = (off + 255) // 256 * 256
        if key == name:
            break
        off += counts[key] * 4
    flat = saved[off:off + counts[name] * 4].view(torch.float32)
    last = 4 * O if name == "gates" else O
    return host(flat).reshape(6, N, D, H, W, last)
