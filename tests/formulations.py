"""Independent formulations used to pin the oracle (test code only).

* ``torch_layer``: the layer of Eq. (7)-(13) written with the library 2D
  convolution (torch.nn.functional.conv2d, cross-correlation, weight layout
  [out][in][kh][kw], padding K//2) on whole planes, in fp64 and differentiable,
  so torch.autograd supplies an independent gradient.
* ``brute_force``: a pull-style memoised recursion that evaluates h^d at one
  voxel straight from Eq. (7)-(12), visiting only the voxels it needs.
* ``lstm_lines``: torch.nn.LSTM (fp64) along every line of one axis.
"""
from __future__ import annotations

import math
from functools import lru_cache

import numpy as np
import torch
import torch.nn.functional as F

# Permutations taking x [N][D][H][W][C] to [T][N][C][P][Q] for axis 0, 1, 2.
_PERM = {0: (1, 0, 4, 2, 3), 1: (2, 0, 4, 1, 3), 2: (3, 0, 4, 1, 2)}


def _inverse(perm):
    inv = [0] * len(perm)
    for i, p in enumerate(perm):
        inv[p] = i
    return tuple(inv)


def torch_layer(x, wx, wh, b, per_direction=False):
    """x [N][D][H][W][C] (torch fp64 tensors, may require grad)."""
    O = wh.shape[2]
    K = wh.shape[3]
    outs = []
    for d in range(6):
        a, sign = d // 2, (1 if d % 2 == 0 else -1)
        xp = x.permute(*_PERM[a])                       # [T][N][C][P][Q]
        T = xp.shape[0]
        order = range(T) if sign > 0 else range(T - 1, -1, -1)
        h_prev = c_prev = None
        planes = [None] * T
        for s in order:
            A = F.conv2d(xp[s], wx[d], bias=b[d], padding=K // 2)
            if h_prev is not None:
                A = A + F.conv2d(h_prev, wh[d], padding=K // 2)
            i = torch.sigmoid(A[:, 0 * O:1 * O])
            f = torch.sigmoid(A[:, 1 * O:2 * O])
            g = torch.tanh(A[:, 2 * O:3 * O])
            o = torch.sigmoid(A[:, 3 * O:4 * O])
            c = g * i if c_prev is None else g * i + c_prev * f
            h = o * torch.tanh(c)
            planes[s] = h
            h_prev, c_prev = h, c
        hd = torch.stack(planes)                         # [T][N][O][P][Q]
        outs.append(hd.permute(*_inverse(_PERM[a])))     # [N][D][H][W][O]
    if per_direction:
        return outs
    total = outs[0]
    for o in outs[1:]:
        total = total + o
    return total


def _sig(v):
    return 1.0 / (1.0 + math.exp(-v))


def brute_force(x, wx, wh, b):
    """Per-direction outputs [6][N][D][H][W][O] by memoised recursion.

    Pure Python; use only for volumes of a few dozen voxels."""
    N, D, H, W, C = x.shape
    O = wh.shape[2]
    K = wh.shape[3]
    r = K // 2
    ext = (D, H, W)
    out = np.zeros((6, N, D, H, W, O))
    for d in range(6):
        a, sign = d // 2, (1 if d % 2 == 0 else -1)
        inplane = [ax for ax in range(3) if ax != a]

        def coords(s, p, q):
            v = [0, 0, 0]
            v[a], v[inplane[0]], v[inplane[1]] = s, p, q
            return tuple(v)

        for n in range(N):
            @lru_cache(maxsize=None)
            def state(s, p, q):
                """(h, c) vectors of direction d at plane s, pixel (p, q)."""
                z, y, xx = coords(s, p, q)
                prev = s - sign
                has_prev = 0 <= prev < ext[a]
                A = []
                for gn in range(4 * O):
                    acc = float(b[d, gn])
                    for ka in range(K):
                        for kb in range(K):
                            pp, qq = p + ka - r, q + kb - r
                            if not (0 <= pp < ext[inplane[0]] and 0 <= qq < ext[inplane[1]]):
                                continue
                            zz, yy, xw = coords(s, pp, qq)
                            for c in range(C):
                                acc += float(x[n, zz, yy, xw, c]) * float(wx[d, gn, c, ka, kb])
                            if has_prev:
                                hp, _ = state(prev, pp, qq)
                                for j in range(O):
                                    acc += hp[j] * float(wh[d, gn, j, ka, kb])
                    A.append(acc)
                c_prev = state(prev, p, q)[1] if has_prev else [0.0] * O
                hs, cs = [], []
                for o in range(O):
                    i = _sig(A[o])
                    f = _sig(A[O + o])
                    g = math.tanh(A[2 * O + o])
                    og = _sig(A[3 * O + o])
                    c = g * i + c_prev[o] * f
                    cs.append(c)
                    hs.append(og * math.tanh(c))
                return tuple(hs), tuple(cs)

            for z in range(D):
                for y in range(H):
                    for xx in range(W):
                        v = (z, y, xx)
                        s = v[a]
                        p, q = v[inplane[0]], v[inplane[1]]
                        out[d, n, z, y, xx] = state(s, p, q)[0]
    return out


def lstm_lines(x, wx_c, b, wh_c, axis, sign):
    """torch.nn.LSTM along every line of `axis`; x [N][D][H][W][C] numpy.

    wx_c [4O][C], wh_c [4O][O] (centre taps), b [4O].  Returns [N][D][H][W][O]."""
    N, D, H, W, C = x.shape
    O = wh_c.shape[1]
    lstm = torch.nn.LSTM(C, O, batch_first=False).double()
    with torch.no_grad():
        lstm.weight_ih_l0.copy_(torch.from_numpy(np.asarray(wx_c, dtype=np.float64)))
        lstm.weight_hh_l0.copy_(torch.from_numpy(np.asarray(wh_c, dtype=np.float64)))
        lstm.bias_ih_l0.copy_(torch.from_numpy(np.asarray(b, dtype=np.float64)))
        lstm.bias_hh_l0.zero_()
    xt = torch.from_numpy(np.asarray(x, dtype=np.float64))
    # Bring the sweep axis first: [T][batch of lines][C].
    seq = xt.movedim(axis + 1, 0)                       # [T][N][..][..][C]
    shp = seq.shape
    seq = seq.reshape(shp[0], -1, C)
    if sign < 0:
        seq = torch.flip(seq, [0])
    with torch.no_grad():
        y, _ = lstm(seq)
    if sign < 0:
        y = torch.flip(y, [0])
    y = y.reshape(*shp[:-1], O).movedim(0, axis + 1)
    return y.numpy()
