"""2D PyraMiD-LSTM on the oracle -- test infrastructure only.

Section 2.1-2.2 and Fig. 1: over an image, 2 x d = 4 LSTMs, each scanning
whole lines: y+ (rows, top to bottom), y- (bottom to top), x+ (columns, left
to right), x- (right to left).  With the connections rotated by 45 degrees
and the gaps filled (Fig. 1 (b)-(c)), a pixel's gates at line t take the
previous line's h at the K pixels around it -- a 1D convolution along the
line -- and the input line the same way; the cell update is that of
Eq. (10)-(12) and the image output is the sum of the four directions.
Readings as for the volume: zero "same" padding, cross-correlation
(in[q + k - r] * w[k], r = (K - 1) / 2), h and c of the line before the first
are zero, gates (i, f, g, o).

``forward2d`` is written directly from that definition (numpy over a line,
one line at a time, fp64).  ``embed`` maps a 2D layer onto the volume layer
of ``oracle.c`` with D = 1: the y and x directions of the volume with their
K x K filters zero outside the middle row (the taps across the missing
depth axis), and the z directions all zero, whose output is then exactly 0
(i = f = o = 1/2, g = 0).  ``backward2d`` is the volume oracle's gradient
through that embedding; the embedding itself is pinned by ``forward2d``.
"""
from __future__ import annotations

import numpy as np

from . import backward as _backward3d
from . import forward as _forward3d


def _sig(a):
    return 1.0 / (1.0 + np.exp(-a))


def forward2d(x, wx, wh, b):
    """x [N][H][W][C]; wx [4][4O][C][K]; wh [4][4O][O][K]; b [4][4O].
    Returns h [N][H][W][O] (fp64)."""
    x = np.asarray(x, dtype=np.float64)
    wx = np.asarray(wx, dtype=np.float64)
    wh = np.asarray(wh, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    N, H, W, C = x.shape
    O = wh.shape[2]
    K = wh.shape[3]
    r = (K - 1) // 2
    h_out = np.zeros((N, H, W, O))
    for d in range(4):
        rows = d < 2                       # y+/y- scan rows, x+/x- columns
        for n in range(N):
            img = x[n] if rows else x[n].transpose(1, 0, 2)   # [T][L][C]
            T, L = img.shape[0], img.shape[1]
            order = range(T) if d % 2 == 0 else range(T - 1, -1, -1)
            hp = np.zeros((L, O))
            cp = np.zeros((L, O))
            res = np.zeros((T, L, O))
            for t in order:
                A = np.broadcast_to(b[d], (L, 4 * O)).copy()
                xp = np.zeros((L + 2 * r, C))
                xp[r:r + L] = img[t]
                hpp = np.zeros((L + 2 * r, O))
                hpp[r:r + L] = hp
                for k in range(K):
                    A += xp[k:k + L] @ wx[d, :, :, k].T + hpp[k:k + L] @ wh[d, :, :, k].T
                i = _sig(A[:, :O])
                f = _sig(A[:, O:2 * O])
                g = np.tanh(A[:, 2 * O:3 * O])
                o = _sig(A[:, 3 * O:])
                c = g * i + cp * f
                hh = o * np.tanh(c)
                res[t] = hh
                hp, cp = hh, c
            h_out[n] += res if rows else res.transpose(1, 0, 2)
    return h_out


def embed(wx, wh, b):
    """The volume layer (D = 1) that computes the same image layer."""
    wx = np.asarray(wx, dtype=np.float64)
    wh = np.asarray(wh, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    G, C, K = wx.shape[1], wx.shape[2], wx.shape[3]
    O = wh.shape[2]
    r = (K - 1) // 2
    wx3 = np.zeros((6, G, C, K, K))
    wh3 = np.zeros((6, G, O, K, K))
    b3 = np.zeros((6, G))
    wx3[2:, :, :, r, :] = wx
    wh3[2:, :, :, r, :] = wh
    b3[2:] = b
    return wx3, wh3, b3


def forward2d_via_volume(x, wx, wh, b):
    wx3, wh3, b3 = embed(wx, wh, b)
    return _forward3d(np.asarray(x)[:, None], wx3, wh3, b3)["h"][:, 0]


def backward2d(x, wx, wh, b, dh, want_dx=True):
    """Gradient of sum(h * dh) w.r.t. x, wx, wh, b (batch-summed)."""
    K = np.asarray(wh).shape[3]
    r = (K - 1) // 2
    wx3, wh3, b3 = embed(wx, wh, b)
    g = _backward3d(np.asarray(x)[:, None], wx3, wh3, b3, np.asarray(dh)[:, None],
                    want_dx=want_dx)
    out = {"dwx": g["dwx"][2:, :, :, r, :], "dwh": g["dwh"][2:, :, :, r, :], "db": g["db"][2:]}
    if want_dx:
        out["dx"] = g["dx"][:, 0]
    return out
