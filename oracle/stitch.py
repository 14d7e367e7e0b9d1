"""Test-time stitching of sub-volume outputs on the oracle -- test
infrastructure only.

Section 3, "Sub-volumes and Augmentation": at test time the network runs on
sub-volumes (no rotation or flipping) and their outputs are stitched together
with a Gaussian kernel.  Readings where the paper is silent:
  - tiles of a fixed size (td, th, tw) start at multiples of a stride along
    each axis, plus one tile flush with the far end of the axis when the grid
    does not reach it (every voxel is covered; tiles larger than the volume
    are cut to it);
  - a tile's weight at its voxel (i, j, k) is the separable Gaussian
    exp(-1/2 sum_axes ((i - c) / sigma)^2), centre c = (size - 1) / 2 and
    sigma = sigma_scale * size per axis (sigma_scale = 1/4 by default);
  - the stitched output of a voxel is the weighted mean of the outputs of
    the tiles covering it.
Plain numpy loops over tiles, fp64.
"""
from __future__ import annotations

import numpy as np


def tile_starts(extent: int, size: int, stride: int):
    """Start offsets along one axis: 0, stride, 2 stride, ... while the tile
    fits, then one tile flush with the end if that was not reached."""
    size = min(size, extent)
    starts = list(range(0, extent - size + 1, stride))
    if starts[-1] + size < extent:
        starts.append(extent - size)
    return starts, size


def gaussian_weights(shape, sigma_scale: float = 0.25):
    """Separable Gaussian over a tile of `shape` (td, th, tw)."""
    w = np.ones(shape)
    for ax, n in enumerate(shape):
        c = (n - 1) / 2.0
        sig = sigma_scale * n
        i = np.arange(n, dtype=np.float64)
        g = np.exp(-0.5 * ((i - c) / sig) ** 2)
        sh = [1, 1, 1]
        sh[ax] = n
        w = w * g.reshape(sh)
    return w


def stitch(volume_shape, tile, stride, tile_fn, classes: int, sigma_scale: float = 0.25,
           origins=None):
    """Weighted mean over tiles.  volume_shape (D, H, W); tile and stride are
    (d, h, w) triples; tile_fn(z0, y0, x0, d, h, w) returns the tile's output
    [d][h][w][classes].  `origins` = (z list, y list, x list) gives the tile
    starts per axis instead of the stride grid.  Returns [D][H][W][classes]."""
    D, H, W = volume_shape
    if origins is None:
        zs, td = tile_starts(D, tile[0], stride[0])
        ys, th = tile_starts(H, tile[1], stride[1])
        xs, tw = tile_starts(W, tile[2], stride[2])
    else:
        (zs, ys, xs), (td, th, tw) = origins, tile
    wt = gaussian_weights((td, th, tw), sigma_scale)
    acc = np.zeros((D, H, W, classes))
    wsum = np.zeros((D, H, W))
    for z0 in zs:
        for y0 in ys:
            for x0 in xs:
                p = np.asarray(tile_fn(z0, y0, x0, td, th, tw), dtype=np.float64)
                acc[z0:z0 + td, y0:y0 + th, x0:x0 + tw] += wt[..., None] * p
                wsum[z0:z0 + td, y0:y0 + th, x0:x0 + tw] += wt
    return acc / wsum[..., None]
