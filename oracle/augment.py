"""Training-time sub-volume sampling with rotation and flips on the oracle --
test infrastructure only.

Section 3, "Sub-volumes and Augmentation": training cubes are cut at random
positions of the full data, possibly rotated by a random angle about an axis
(about z for the EM stacks) and flipped along any axis (EM: x, y and z, each
with probability 1/2; MR: x only, no rotation).  The random draws are inputs
here.  Readings where the paper is silent:
  - the cube (d, h, w) has its unrotated corner at (z0, y0, x0) inside the
    volume and turns about its own centre in the (y, x) plane:
        S[k][i][j] = V(z0 + k, yc + c u - s v, xc + s u + c v),
        u = i - (h - 1) / 2, v = j - (w - 1) / 2,
        yc = y0 + (h - 1) / 2, xc = x0 + (w - 1) / 2, (c, s) = (cos, sin);
  - source positions outside the slice are clamped to its edge;
  - image values are bilinear in (y, x); labels take the nearest voxel,
    floor(y + 1/2) after clamping;
  - the flips act on the sampled cube: out[k][i][j] = S[k'][i'][j'] with
    k' = d - 1 - k when z is flipped (likewise i' for y, j' for x).
The source coordinates are computed in fp32 in the order written above (c u,
s v, their difference, then yc + it; s u, c v, their sum, then xc + it), the
precision the sampler uses, because they decide integers: the interpolation
cell and the nearest label.  The interpolation itself is fp64.
"""
from __future__ import annotations

import numpy as np

FLIP_Z, FLIP_Y, FLIP_X = 1, 2, 4


def source_coords(h, w, y0, x0, c, s):
    """fp32 source (y, x) of every (i, j) of the rotated cube, unclamped."""
    f = np.float32
    c, s = f(c), f(s)
    i = np.arange(h, dtype=np.float64)[:, None] - (h - 1) / 2.0
    j = np.arange(w, dtype=np.float64)[None, :] - (w - 1) / 2.0
    u = np.broadcast_to(i, (h, w)).astype(f)          # half-integers: exact in fp32
    v = np.broadcast_to(j, (h, w)).astype(f)
    yc = f(y0 + (h - 1) / 2.0)
    xc = f(x0 + (w - 1) / 2.0)
    y = yc + ((c * u) - (s * v))
    x = xc + ((s * u) + (c * v))
    return y.astype(f), x.astype(f)


def sample(vol, labels, n, corner, size, c, s, flips):
    """One training cube.  vol [N][D][H][W][C], labels [N][D][H][W] or None;
    corner (z0, y0, x0), size (d, h, w); (c, s) the rotation's cosine and
    sine (taken as fp32); flips a bit set of FLIP_Z / FLIP_Y / FLIP_X.
    Returns (cube [d][h][w][C] fp64, cube labels [d][h][w] or None)."""
    z0, y0, x0 = corner
    d, h, w = size
    N, D, H, W, C = vol.shape
    assert 0 <= z0 and z0 + d <= D and 0 <= y0 and y0 + h <= H and 0 <= x0 and x0 + w <= W
    f = np.float32
    y, x = source_coords(h, w, y0, x0, c, s)
    y = np.minimum(np.maximum(y, f(0)), f(H - 1))
    x = np.minimum(np.maximum(x, f(0)), f(W - 1))
    ya = np.floor(y).astype(np.int64)
    xa = np.floor(x).astype(np.int64)
    yb = np.minimum(ya + 1, H - 1)
    xb = np.minimum(xa + 1, W - 1)
    wy = (y.astype(np.float64) - ya)[..., None]
    wx = (x.astype(np.float64) - xa)[..., None]
    src = np.asarray(vol[n], dtype=np.float64)
    cube = np.empty((d, h, w, C))
    for k in range(d):
        sl = src[z0 + k]
        cube[k] = ((1 - wy) * (1 - wx) * sl[ya, xa] + (1 - wy) * wx * sl[ya, xb]
                   + wy * (1 - wx) * sl[yb, xa] + wy * wx * sl[yb, xb])
    lab = None
    if labels is not None:
        yn = np.floor(y + f(0.5)).astype(np.int64)
        xn = np.floor(x + f(0.5)).astype(np.int64)
        lab = np.stack([labels[n, z0 + k][yn, xn] for k in range(d)])
    axes = [ax for bit, ax in ((FLIP_Z, 0), (FLIP_Y, 1), (FLIP_X, 2)) if flips & bit]
    if axes:
        cube = np.flip(cube, axis=axes)
        if lab is not None:
            lab = np.flip(lab, axis=axes)
    return np.ascontiguousarray(cube), None if lab is None else np.ascontiguousarray(lab)
