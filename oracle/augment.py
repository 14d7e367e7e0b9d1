"""Training-time sub-volume sampling with rotation and flips on the oracle --
test infrastructure only.

Section 3, "Sub-volumes and Augmentation": training cubes are cut at random
positions of the full data, possibly rotated by a random angle about an axis
(about z for the EM stacks) and flipped along any axis (EM: x, y and z, each
with probability 1/2; MR: x only, no rotation).  The random draws are inputs
here.  Readings where the paper is silent:
  - the cube (d, h, w) has its unrotated corner at (z0, y0, x0) inside the
    volume and turns about its own centre in the (y, x) plane: cube voxel
    (k, i, j) reads the volume at z0 + k and at the in-plane point
        centre + R(theta) (i - (h - 1) / 2, j - (w - 1) / 2),
    centre = (y0 + (h - 1) / 2, x0 + (w - 1) / 2), R the rotation with
    cosine c and sine s acting on (y, x) offsets: (c a - s b, s a + c b);
  - source positions outside the slice are clamped to its edge;
  - image values are bilinear in (y, x); labels take the nearest voxel,
    floor(p + 1/2) per axis after clamping;
  - the flips act on the sampled cube: out[k][i][j] = S[k'][i'][j'] with
    k' = d - 1 - k when z is flipped (likewise i' for y, j' for x).
Everything is fp64: the rotation is applied as a 2x2 matrix to the offsets,
then interpolated.  `label_margin` tells how far each position lies from a
nearest-label boundary, so a comparison can set aside the few voxels where
any rounding of the position could pick the other label.
"""
from __future__ import annotations

import numpy as np

FLIP_Z, FLIP_Y, FLIP_X = 1, 2, 4


def source_positions(H, W, h, w, y0, x0, c, s):
    """fp64 source (y, x) of every (i, j) of the turned cube, clamped to the
    H x W slice.  Returns two [h][w] arrays."""
    R = np.array([[c, -s], [s, c]], dtype=np.float64)
    off = np.stack(np.meshgrid(np.arange(h) - (h - 1) / 2.0, np.arange(w) - (w - 1) / 2.0,
                               indexing="ij"), axis=-1)                    # [h][w][2]
    centre = np.array([y0 + (h - 1) / 2.0, x0 + (w - 1) / 2.0])
    pos = centre + off @ R.T
    y = np.clip(pos[..., 0], 0.0, H - 1.0)
    x = np.clip(pos[..., 1], 0.0, W - 1.0)
    return y, x


def _flip(a, flips):
    axes = [ax for bit, ax in ((FLIP_Z, 0), (FLIP_Y, 1), (FLIP_X, 2)) if flips & bit]
    return np.ascontiguousarray(np.flip(a, axis=axes) if axes else a)


def sample(vol, labels, n, corner, size, c, s, flips):
    """One training cube.  vol [N][D][H][W][C], labels [N][D][H][W] or None;
    corner (z0, y0, x0), size (d, h, w); (c, s) the rotation's cosine and
    sine; flips a bit set of FLIP_Z / FLIP_Y / FLIP_X.
    Returns (cube [d][h][w][C] fp64, cube labels [d][h][w] or None)."""
    z0, y0, x0 = corner
    d, h, w = size
    N, D, H, W, C = vol.shape
    assert 0 <= z0 and z0 + d <= D and 0 <= y0 and y0 + h <= H and 0 <= x0 and x0 + w <= W
    y, x = source_positions(H, W, h, w, y0, x0, float(c), float(s))
    src = np.asarray(vol[n, z0:z0 + d], dtype=np.float64)              # [d][H][W][C]
    cube = np.empty((d, h, w, C))
    for i in range(h):
        for j in range(w):
            ya, xa = int(np.floor(y[i, j])), int(np.floor(x[i, j]))
            fy, fx = y[i, j] - ya, x[i, j] - xa
            yb, xb = min(ya + 1, H - 1), min(xa + 1, W - 1)
            top = (1 - fx) * src[:, ya, xa] + fx * src[:, ya, xb]
            bot = (1 - fx) * src[:, yb, xa] + fx * src[:, yb, xb]
            cube[:, i, j] = (1 - fy) * top + fy * bot
    lab = None
    if labels is not None:
        yn = np.floor(y + 0.5).astype(np.int64)
        xn = np.floor(x + 0.5).astype(np.int64)
        lab = np.asarray(labels[n, z0:z0 + d])[:, yn, xn]
        lab = _flip(lab, flips)
    return _flip(cube, flips), lab


def label_margin(shape, size, corner, c, s, flips):
    """Per cube voxel (after the flips), the distance of its source position
    from the nearest-label boundary: min over y and x of the distance of
    p + 1/2 to the nearest integer.  Positions clamped to the slice edge
    count as far from a boundary."""
    N, D, H, W = shape[:4]
    z0, y0, x0 = corner
    d, h, w = size
    y, x = source_positions(H, W, h, w, y0, x0, float(c), float(s))

    def dist(p, hi):
        frac = (p + 0.5) - np.floor(p + 0.5)
        m = np.minimum(frac, 1.0 - frac)
        return np.where((p <= 0.0) | (p >= hi), 0.5, m)

    m = np.minimum(dist(y, H - 1.0), dist(x, W - 1.0))
    return _flip(np.broadcast_to(m, (d, h, w)), flips)
