"""PyraMiD-LSTM CPU oracle (fp64) -- test infrastructure only.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding in ``paper_1506_07452_amd``) never imports, links or calls it, and
the two share no code.

The arithmetic lives in ``oracle.c`` (plain nested loops, fp64): the layer of
Section 2.3, Eq. (7)-(13), its back-propagation through the sweeps, the
per-voxel fully connected tanh layer and the final softmax (Section 2.3,
"Fully-Connected Layer"; Fig. 3).  This module only marshals numpy arrays.
``network.py`` composes these pieces into the stacked networks.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
# PLSTM_ORACLE_LIB selects another build of oracle.c (the sanitizer test
# loads the ASan/UBSan one through it)
_LIB = os.environ.get("PLSTM_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
SAN_LIB = os.path.join(_HERE, "liboracle_san.so")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
             "-fno-omit-frame-pointer", "-g"]

_lib = None


def build(force: bool = True, sanitize: bool = False) -> str:
    """Compile oracle.c with gcc (-O2, OpenMP) into liboracle.so, in-tree;
    with `sanitize`, an AddressSanitizer + UndefinedBehaviorSanitizer build
    into liboracle_san.so instead (host code only)."""
    out = SAN_LIB if sanitize else _LIB
    if force or not os.path.exists(out):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Wextra"] +
            (SAN_FLAGS if sanitize else []) + ["-o", tmp, _SRC, "-lm"])
        os.replace(tmp, out)
    return out


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int)
        i = ctypes.c_int
        lib.oracle_forward.argtypes = [i] * 7 + [dp] * 8
        lib.oracle_forward.restype = i
        lib.oracle_backward.argtypes = [i] * 7 + [dp] * 9
        lib.oracle_backward.restype = i
        lib.oracle_fc_tanh_forward.argtypes = [ctypes.c_long, i, i, dp, dp, dp, dp]
        lib.oracle_fc_tanh_forward.restype = None
        lib.oracle_fc_tanh_backward.argtypes = [ctypes.c_long, i, i] + [dp] * 7
        lib.oracle_fc_tanh_backward.restype = None
        lib.oracle_softmax_ce.argtypes = [ctypes.c_long, i, i, dp, dp, dp, ip, dp, dp, dp, dp]
        lib.oracle_softmax_ce.restype = ctypes.c_double
        lib.oracle_threads.argtypes = []
        lib.oracle_threads.restype = i
        lib.oracle_set_threads.argtypes = [i]
        lib.oracle_set_threads.restype = None
        _lib = lib
    return _lib


def threads() -> int:
    """OpenMP threads used by the oracle's parallel loops."""
    return int(_load().oracle_threads())


def set_threads(n: int) -> None:
    """OpenMP threads for later oracle calls from this thread."""
    _load().oracle_set_threads(int(n))


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a):
    if a is None:
        return ctypes.POINTER(ctypes.c_double)()
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _dims(x, wh):
    N, D, H, W, C = x.shape
    O = wh.shape[2]
    K = wh.shape[3]
    return N, D, H, W, C, O, K


def _check_params(x, wx, wh, b):
    N, D, H, W, C, O, K = _dims(x, wh)
    assert wx.shape == (6, 4 * O, C, K, K), wx.shape
    assert wh.shape == (6, 4 * O, O, K, K), wh.shape
    assert b.shape == (6, 4 * O), b.shape


def forward(x, wx, wh, b, want_hd=False, want_saved=False):
    """One PyraMiD-LSTM layer, Eq. (7)-(13).

    x [N][D][H][W][C]; wx [6][4O][C][K][K]; wh [6][4O][O][K][K]; b [6][4O].
    Returns dict with 'h' [N][D][H][W][O] and, on request, 'hd' (per-direction
    outputs, [6][N][D][H][W][O]), 'gates' ([6][N][D][H][W][4O], i,f,g,o after
    the nonlinearity) and 'cell' ([6][N][D][H][W][O])."""
    x, wx, wh, b = map(_f64, (x, wx, wh, b))
    _check_params(x, wx, wh, b)
    N, D, H, W, C, O, K = _dims(x, wh)
    h = np.empty((N, D, H, W, O))
    hd = np.empty((6, N, D, H, W, O)) if want_hd else None
    gates = np.empty((6, N, D, H, W, 4 * O)) if want_saved else None
    cell = np.empty((6, N, D, H, W, O)) if want_saved else None
    rc = _load().oracle_forward(N, D, H, W, C, O, K, _p(x), _p(wx), _p(wh), _p(b),
                                _p(h), _p(hd), _p(gates), _p(cell))
    if rc != 0:
        raise RuntimeError("oracle_forward failed (%d)" % rc)
    out = {"h": h}
    if want_hd:
        out["hd"] = hd
    if want_saved:
        out["gates"] = gates
        out["cell"] = cell
    return out


def backward(x, wx, wh, b, dh, want_dx=True):
    """Gradient of sum(h * dh) for one layer w.r.t. x, wx, wh, b (batch-summed)."""
    x, wx, wh, b, dh = map(_f64, (x, wx, wh, b, dh))
    _check_params(x, wx, wh, b)
    N, D, H, W, C, O, K = _dims(x, wh)
    assert dh.shape == (N, D, H, W, O)
    dx = np.empty_like(x) if want_dx else None
    dwx = np.empty_like(wx)
    dwh = np.empty_like(wh)
    db = np.empty_like(b)
    rc = _load().oracle_backward(N, D, H, W, C, O, K, _p(x), _p(wx), _p(wh), _p(b),
                                 _p(dh), _p(dx), _p(dwx), _p(dwh), _p(db))
    if rc != 0:
        raise RuntimeError("oracle_backward failed (%d)" % rc)
    return {"dx": dx, "dwx": dwx, "dwh": dwh, "db": db}


def fc_tanh_forward(x2, w, b):
    """y = tanh(x2 @ w.T + b) per row (voxel).  x2 [M][Cin], w [Cout][Cin]."""
    x2, w, b = map(_f64, (x2, w, b))
    M, Cin = x2.shape
    Cout = w.shape[0]
    y = np.empty((M, Cout))
    _load().oracle_fc_tanh_forward(M, Cin, Cout, _p(x2), _p(w), _p(b), _p(y))
    return y


def fc_tanh_backward(x2, w, y, dy, want_dx=True):
    x2, w, y, dy = map(_f64, (x2, w, y, dy))
    M, Cin = x2.shape
    Cout = w.shape[0]
    dx = np.empty((M, Cin)) if want_dx else None
    dw = np.empty((Cout, Cin))
    db = np.empty(Cout)
    _load().oracle_fc_tanh_backward(M, Cin, Cout, _p(x2), _p(w), _p(y), _p(dy),
                                    _p(dx), _p(dw), _p(db))
    return {"dx": dx, "dw": dw, "db": db}


def softmax_ce(x2, w, b, labels=None, grad=False):
    """Final linear layer + per-row softmax; mean cross-entropy when labels given."""
    x2, w, b = map(_f64, (x2, w, b))
    M, Cin = x2.shape
    Kc = w.shape[0]
    p = np.empty((M, Kc))
    lab = None
    if labels is not None:
        lab = np.ascontiguousarray(labels, dtype=np.int32).reshape(M)
        assert lab.min() >= 0 and lab.max() < Kc
    lab_p = lab.ctypes.data_as(ctypes.POINTER(ctypes.c_int)) if lab is not None \
        else ctypes.POINTER(ctypes.c_int)()
    dx = dw = db = None
    if grad:
        assert lab is not None
        dx, dw, db = np.empty((M, Cin)), np.empty((Kc, Cin)), np.empty(Kc)
    loss = _load().oracle_softmax_ce(M, Cin, Kc, _p(x2), _p(w), _p(b), lab_p, _p(p),
                                     _p(dx), _p(dw), _p(db))
    out = {"p": p, "loss": float(loss) if lab is not None else None}
    if grad:
        out.update({"dx": dx, "dw": dw, "db": db})
    return out
