"""Python binding of libpyramid_lstm.so (the MI355X PyraMiD-LSTM library).

Argument marshalling only: every function here has the name of a C entry point
declared in include/pyramid_lstm.h, converts torch tensors to device pointers
and the current HIP stream, calls the entry point and raises on a negative
status.  All computation runs in the library's HIP kernels; torch provides
device memory and streams.  There is no fallback: if the library is not built
the binding raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "PyramidLSTMError", "plstm_shape", "shape_for", "PLSTM_F32", "PLSTM_BF16",
    "pyramid_lstm_status_string", "pyramid_lstm_workspace_size", "pyramid_lstm_saved_size",
    "pyramid_lstm_forward", "pyramid_lstm_backward", "pyramid_fc_tanh_forward",
    "pyramid_fc_workspace_size", "pyramid_fc_tanh_backward", "pyramid_softmax_ce",
    "pyramid_head_workspace_size", "pyramid_head_train", "plstm_param_segment",
    "pyramid_head_forward", "pyramid_head_forward_supported",
    "pyramid_rmsprop_step", "pyramid_rmsprop_learning_rate", "RMSprop", "pyramid_softmax_sq",
    "pyramid_crop", "pyramid_stitch_clear", "pyramid_stitch_add", "pyramid_stitch_finish",
    "pyramid_lstm_timing_enable", "pyramid_lstm_timing_read", "pyramid_lstm_set_forward_path",
    "pyramid_lstm_set_backward_path", "pyramid_lstm_set_step_split", "pyramid_lstm_set_bf16_mfma",
    "pyramid_lstm_set_wgrad_staged",
    "library_path", "load", "plstm2d_shape", "shape2d_for", "pyramid_lstm2d_workspace_size",
    "pyramid_lstm2d_saved_size", "pyramid_lstm2d_forward", "pyramid_lstm2d_backward",
    "plstm_cube", "PLSTM_FLIP_Z", "PLSTM_FLIP_Y", "PLSTM_FLIP_X", "PLSTM_MAX_CUBES",
    "pyramid_sample_cubes", "draw_cubes", "pyramid_lstm_device_status",
    "pyramid_lstm_set_wait_test", "PLSTM_DEVICE_WAIT_GAVE_UP", "pyramid_lstm_forward_noalloc",
    "PLSTM_NOALLOC_SCRATCH_BYTES", "PLSTM_ESCRATCH",
]

PLSTM_F32 = 0
PLSTM_BF16 = 1
PLSTM_FLIP_Z, PLSTM_FLIP_Y, PLSTM_FLIP_X = 1, 2, 4
PLSTM_MAX_CUBES = 64
PLSTM_DEVICE_WAIT_GAVE_UP = 1
PLSTM_NOALLOC_SCRATCH_BYTES = 256 << 20
PLSTM_ESCRATCH = -6

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "libpyramid_lstm.so")
_lib = None


class PyramidLSTMError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (fn, pyramid_lstm_status_string(status), status))


class plstm_shape(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int32), ("D", ctypes.c_int32), ("H", ctypes.c_int32),
                ("W", ctypes.c_int32), ("C", ctypes.c_int32), ("O", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("K", ctypes.c_int32)]


class plstm2d_shape(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int32), ("H", ctypes.c_int32), ("W", ctypes.c_int32),
                ("C", ctypes.c_int32), ("O", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("K", ctypes.c_int32)]


class plstm_cube(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("z0", ctypes.c_int32), ("y0", ctypes.c_int32),
                ("x0", ctypes.c_int32), ("cos_t", ctypes.c_float), ("sin_t", ctypes.c_float),
                ("flips", ctypes.c_int32)]


class plstm_param_segment(ctypes.Structure):
    _fields_ = [("theta", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("ms", ctypes.c_void_p),
                ("mom", ctypes.c_void_p), ("n", ctypes.c_int64)]


def library_path() -> str:
    return _LIB_PATH


def load():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError("libpyramid_lstm.so is not built; run "
                           "`python -m paper_1506_07452_amd.build` first")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, sz, i32, i64 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int64
    sp = ctypes.POINTER(plstm_shape)
    lib.pyramid_lstm_status_string.argtypes = [ctypes.c_int]
    lib.pyramid_lstm_status_string.restype = ctypes.c_char_p
    lib.pyramid_lstm_workspace_size.argtypes = [sp, ctypes.c_int]
    lib.pyramid_lstm_workspace_size.restype = sz
    lib.pyramid_lstm_saved_size.argtypes = [sp]
    lib.pyramid_lstm_saved_size.restype = sz
    lib.pyramid_lstm_forward.argtypes = [sp] + [vp] * 7 + [sz, vp]
    lib.pyramid_lstm_forward.restype = ctypes.c_int
    lib.pyramid_lstm_forward_noalloc.argtypes = [sp] + [vp] * 6
    lib.pyramid_lstm_forward_noalloc.restype = ctypes.c_int
    lib.pyramid_lstm_backward.argtypes = [sp] + [vp] * 11 + [sz, vp]
    lib.pyramid_lstm_backward.restype = ctypes.c_int
    sp2 = ctypes.POINTER(plstm2d_shape)
    lib.pyramid_lstm2d_workspace_size.argtypes = [sp2, ctypes.c_int]
    lib.pyramid_lstm2d_workspace_size.restype = sz
    lib.pyramid_lstm2d_saved_size.argtypes = [sp2]
    lib.pyramid_lstm2d_saved_size.restype = sz
    lib.pyramid_lstm2d_forward.argtypes = [sp2] + [vp] * 7 + [sz, vp]
    lib.pyramid_lstm2d_forward.restype = ctypes.c_int
    lib.pyramid_lstm2d_backward.argtypes = [sp2] + [vp] * 11 + [sz, vp]
    lib.pyramid_lstm2d_backward.restype = ctypes.c_int
    lib.pyramid_fc_tanh_forward.argtypes = [i64, i32, i32, i32] + [vp] * 4 + [vp]
    lib.pyramid_fc_tanh_forward.restype = ctypes.c_int
    lib.pyramid_fc_workspace_size.argtypes = [i64, i32, i32]
    lib.pyramid_fc_workspace_size.restype = sz
    lib.pyramid_fc_tanh_backward.argtypes = [i64, i32, i32] + [vp] * 8 + [sz, vp]
    lib.pyramid_fc_tanh_backward.restype = ctypes.c_int
    lib.pyramid_softmax_ce.argtypes = [i64, i32, i32, i32] + [vp] * 10 + [sz, vp]
    lib.pyramid_softmax_ce.restype = ctypes.c_int
    lib.pyramid_softmax_sq.argtypes = [i64, i32, i32, i32] + [vp] * 10 + [sz, vp]
    lib.pyramid_softmax_sq.restype = ctypes.c_int
    lib.pyramid_head_workspace_size.argtypes = [i64, i32, i32, i32]
    lib.pyramid_head_workspace_size.restype = sz
    lib.pyramid_head_train.argtypes = [i64, i32, i32, i32] + [vp] * 14 + [sz, vp]
    lib.pyramid_head_train.restype = ctypes.c_int
    lib.pyramid_head_forward_supported.argtypes = [i32, i32, i32, i32]
    lib.pyramid_head_forward_supported.restype = ctypes.c_int
    lib.pyramid_head_forward.argtypes = [i64, i32, i32, i32, i32] + [vp] * 7
    lib.pyramid_head_forward.restype = ctypes.c_int
    f32 = ctypes.c_float
    lib.pyramid_rmsprop_step.argtypes = [i32, ctypes.POINTER(plstm_param_segment), f32, f32, f32,
                                         f32, vp]
    lib.pyramid_rmsprop_step.restype = ctypes.c_int
    lib.pyramid_rmsprop_learning_rate.argtypes = [i32]
    lib.pyramid_rmsprop_learning_rate.restype = ctypes.c_double
    lib.pyramid_crop.argtypes = [i32] * 13 + [vp, vp, vp]
    lib.pyramid_crop.restype = ctypes.c_int
    lib.pyramid_sample_cubes.argtypes = [i32] * 7 + [ctypes.POINTER(plstm_cube)] + [i32] * 3 + \
        [vp] * 5
    lib.pyramid_sample_cubes.restype = ctypes.c_int
    lib.pyramid_stitch_clear.argtypes = [i32] * 4 + [vp, vp, vp]
    lib.pyramid_stitch_clear.restype = ctypes.c_int
    lib.pyramid_stitch_add.argtypes = [i32] * 10 + [f32, vp, vp, vp, vp]
    lib.pyramid_stitch_add.restype = ctypes.c_int
    lib.pyramid_stitch_finish.argtypes = [i32] * 4 + [vp, vp, vp, vp]
    lib.pyramid_stitch_finish.restype = ctypes.c_int
    lib.pyramid_lstm_timing_enable.argtypes = [ctypes.c_int]
    lib.pyramid_lstm_timing_enable.restype = ctypes.c_int
    lib.pyramid_lstm_timing_read.argtypes = [ctypes.c_int, ctypes.c_char_p,
                                             ctypes.POINTER(ctypes.c_double),
                                             ctypes.POINTER(ctypes.c_int),
                                             ctypes.POINTER(ctypes.c_int)]
    lib.pyramid_lstm_timing_read.restype = ctypes.c_int
    lib.pyramid_lstm_device_status.argtypes = [ctypes.POINTER(ctypes.c_int32), i32, vp]
    lib.pyramid_lstm_device_status.restype = ctypes.c_int
    lib.pyramid_lstm_set_wait_test.argtypes = [ctypes.c_int]
    lib.pyramid_lstm_set_wait_test.restype = ctypes.c_int
    lib.pyramid_lstm_set_bf16_mfma.argtypes = [ctypes.c_int]
    lib.pyramid_lstm_set_bf16_mfma.restype = ctypes.c_int
    lib.pyramid_lstm_set_step_split.argtypes = [ctypes.c_int]
    lib.pyramid_lstm_set_step_split.restype = ctypes.c_int
    lib.pyramid_lstm_set_wgrad_staged.argtypes = [ctypes.c_int]
    lib.pyramid_lstm_set_wgrad_staged.restype = ctypes.c_int
    lib.pyramid_lstm_set_forward_path.argtypes = [ctypes.c_int]
    lib.pyramid_lstm_set_forward_path.restype = ctypes.c_int
    lib.pyramid_lstm_set_backward_path.argtypes = [ctypes.c_int]
    lib.pyramid_lstm_set_backward_path.restype = ctypes.c_int
    _lib = lib
    return lib


# ----------------------------------------------------------------- marshalling
_DT = {torch.float32: PLSTM_F32, torch.bfloat16: PLSTM_BF16}


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch.Tensor, got %r" % type(t))
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check(fn, rc):
    if rc != 0:
        raise PyramidLSTMError(fn, rc)


def shape_for(x: torch.Tensor, O: int, K: int = 3) -> plstm_shape:
    """plstm_shape of a [N][D][H][W][C] volume, hidden size O and K x K filters."""
    if x.dim() != 5:
        raise ValueError("x must be [N][D][H][W][C]")
    if x.dtype not in _DT:
        raise ValueError("x must be float32 or bfloat16")
    N, D, H, W, C = x.shape
    return plstm_shape(N, D, H, W, C, O, _DT[x.dtype], K)


def shape2d_for(x: torch.Tensor, O: int, K: int = 3) -> plstm2d_shape:
    """plstm2d_shape of a [N][H][W][C] image batch, hidden size O, filters of K taps."""
    if x.dim() != 4:
        raise ValueError("x must be [N][H][W][C]")
    if x.dtype not in _DT:
        raise ValueError("x must be float32 or bfloat16")
    N, H, W, C = x.shape
    return plstm2d_shape(N, H, W, C, O, _DT[x.dtype], K)


def _workspace(nbytes, device):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


# --------------------------------------------------------------- entry points
def pyramid_lstm_status_string(status: int) -> str:
    return load().pyramid_lstm_status_string(int(status)).decode()


def pyramid_lstm_workspace_size(shape: plstm_shape, training: int) -> int:
    return int(load().pyramid_lstm_workspace_size(ctypes.byref(shape), int(training)))


def pyramid_lstm_saved_size(shape: plstm_shape) -> int:
    return int(load().pyramid_lstm_saved_size(ctypes.byref(shape)))


def pyramid_lstm_forward(shape, x, wx, wh, b, h, saved=None, ws=None, stream=None):
    """Layer forward.  ws=None allocates the workspace with torch."""
    lib = load()
    if ws is None:
        ws = _workspace(pyramid_lstm_workspace_size(shape, saved is not None), x.device)
    _check("pyramid_lstm_forward", lib.pyramid_lstm_forward(
        ctypes.byref(shape), _ptr(x), _ptr(wx), _ptr(wh), _ptr(b), _ptr(h), _ptr(saved),
        _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def pyramid_lstm_forward_noalloc(shape, x, wx, wh, b, h, stream=None):
    """Inference forward on the library's own per-GPU scratch (no workspace,
    nothing allocated); raises PyramidLSTMError (PLSTM_ESCRATCH) for shapes
    whose workspace exceeds PLSTM_NOALLOC_SCRATCH_BYTES."""
    _check("pyramid_lstm_forward_noalloc", load().pyramid_lstm_forward_noalloc(
        ctypes.byref(shape), _ptr(x), _ptr(wx), _ptr(wh), _ptr(b), _ptr(h), _stream(stream)))


def pyramid_lstm_backward(shape, x, wx, wh, b, saved, dh, dx, dwx, dwh, db, ws=None,
                          stream=None):
    lib = load()
    if ws is None:
        ws = _workspace(pyramid_lstm_workspace_size(shape, 1), x.device)
    _check("pyramid_lstm_backward", lib.pyramid_lstm_backward(
        ctypes.byref(shape), _ptr(x), _ptr(wx), _ptr(wh), _ptr(b), _ptr(saved), _ptr(dh),
        _ptr(dx), _ptr(dwx), _ptr(dwh), _ptr(db), _ptr(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def pyramid_lstm2d_workspace_size(shape: plstm2d_shape, training: int) -> int:
    return int(load().pyramid_lstm2d_workspace_size(ctypes.byref(shape), int(training)))


def pyramid_lstm2d_saved_size(shape: plstm2d_shape) -> int:
    return int(load().pyramid_lstm2d_saved_size(ctypes.byref(shape)))


def pyramid_lstm2d_forward(shape, x, wx, wh, b, h, saved=None, ws=None, stream=None):
    """2D layer forward over x [N][H][W][C].  ws=None allocates the workspace with torch."""
    lib = load()
    if ws is None:
        ws = _workspace(pyramid_lstm2d_workspace_size(shape, saved is not None), x.device)
    _check("pyramid_lstm2d_forward", lib.pyramid_lstm2d_forward(
        ctypes.byref(shape), _ptr(x), _ptr(wx), _ptr(wh), _ptr(b), _ptr(h), _ptr(saved),
        _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def pyramid_lstm2d_backward(shape, x, wx, wh, b, saved, dh, dx, dwx, dwh, db, ws=None,
                            stream=None):
    lib = load()
    if ws is None:
        ws = _workspace(pyramid_lstm2d_workspace_size(shape, 1), x.device)
    _check("pyramid_lstm2d_backward", lib.pyramid_lstm2d_backward(
        ctypes.byref(shape), _ptr(x), _ptr(wx), _ptr(wh), _ptr(b), _ptr(saved), _ptr(dh),
        _ptr(dx), _ptr(dwx), _ptr(dwh), _ptr(db), _ptr(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def pyramid_fc_tanh_forward(x, w, b, y, stream=None):
    """x [M][Cin], w [Cout][Cin], b [Cout], y [M][Cout] (same dtype)."""
    M, Cin = x.shape
    Cout = w.shape[0]
    _check("pyramid_fc_tanh_forward", load().pyramid_fc_tanh_forward(
        M, Cin, Cout, _DT[x.dtype], _ptr(x), _ptr(w), _ptr(b), _ptr(y), _stream(stream)))


def pyramid_fc_workspace_size(M: int, Cin: int, Cout: int) -> int:
    return int(load().pyramid_fc_workspace_size(M, Cin, Cout))


def pyramid_fc_tanh_backward(x, w, y, dy, dx, dw, db, ws=None, stream=None):
    M, Cin = x.shape
    Cout = w.shape[0]
    if ws is None:
        ws = _workspace(pyramid_fc_workspace_size(M, Cin, Cout), x.device)
    _check("pyramid_fc_tanh_backward", load().pyramid_fc_tanh_backward(
        M, Cin, Cout, _ptr(x), _ptr(w), _ptr(y), _ptr(dy), _ptr(dx), _ptr(dw), _ptr(db),
        _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def pyramid_softmax_ce(x, w, b, p, labels=None, loss=None, dx=None, dw=None, db=None, ws=None,
                       stream=None, squared=False):
    """Final linear + softmax (+ mean cross-entropy, or with `squared` the
    squared error of Eq. (14), and its gradient)."""
    M, Cin = x.shape
    K = w.shape[0]
    if labels is not None and ws is None:
        ws = _workspace(pyramid_fc_workspace_size(M, Cin, K), x.device)
    name = "pyramid_softmax_sq" if squared else "pyramid_softmax_ce"
    _check(name, getattr(load(), name)(
        M, Cin, K, _DT[x.dtype], _ptr(x), _ptr(w), _ptr(b), _ptr(labels), _ptr(p), _ptr(loss),
        _ptr(dx), _ptr(dw), _ptr(db), _ptr(ws),
        0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def pyramid_softmax_sq(x, w, b, p, labels=None, loss=None, dx=None, dw=None, db=None, ws=None,
                       stream=None):
    """Final linear + softmax (+ the squared loss of Eq. (14) and its gradient)."""
    pyramid_softmax_ce(x, w, b, p, labels, loss, dx, dw, db, ws, stream, squared=True)


def pyramid_head_workspace_size(M: int, Cin: int, F: int, K: int) -> int:
    return int(load().pyramid_head_workspace_size(M, Cin, F, K))


def pyramid_head_train(x, w1, b1, w2, b2, labels, p, loss, dx, dw1, db1, dw2, db2, ws=None,
                       stream=None):
    """Fused FC tanh + linear + softmax + mean cross-entropy and their backward."""
    M, Cin = x.shape
    F, K = w1.shape[0], w2.shape[0]
    if ws is None:
        ws = _workspace(max(pyramid_head_workspace_size(M, Cin, F, K), 256), x.device)
    _check("pyramid_head_train", load().pyramid_head_train(
        M, Cin, F, K, _ptr(x), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2), _ptr(labels), _ptr(p),
        _ptr(loss), _ptr(dx), _ptr(dw1), _ptr(db1), _ptr(dw2), _ptr(db2), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def pyramid_head_forward_supported(dtype, Cin: int, F: int, K: int) -> bool:
    return bool(load().pyramid_head_forward_supported(_DT[dtype], Cin, F, K))


def pyramid_head_forward(x, w1, b1, w2, b2, p, stream=None):
    """Fused FC tanh + linear + softmax for inference: x [M][Cin], w1 [F][Cin],
    b1 [F], w2 [K][F], b2 [K] (same dtype), p [M][K] fp32."""
    M, Cin = x.shape
    F, K = w1.shape[0], w2.shape[0]
    _check("pyramid_head_forward", load().pyramid_head_forward(
        M, Cin, F, K, _DT[x.dtype], _ptr(x), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2), _ptr(p),
        _stream(stream)))


def pyramid_rmsprop_step(params, grads, ms, mom, lr, rho_ms=0.9, rho_m=0.9, eps=1e-5,
                         stream=None):
    """RMS-prop with momentum (Section 3, Eq. (15)-(18)) over lists of fp32
    device tensors, in place, in one launch."""
    n = len(params)
    if not (len(grads) == len(ms) == len(mom) == n):
        raise ValueError("params, grads, ms and mom must have the same length")
    segs = (plstm_param_segment * max(n, 1))()
    for k, (t, g, a, m) in enumerate(zip(params, grads, ms, mom)):
        for u in (t, g, a, m):
            if u.dtype != torch.float32 or u.numel() != t.numel():
                raise ValueError("fp32 tensors of one size per parameter expected")
        segs[k] = plstm_param_segment(_ptr(t), _ptr(g), _ptr(a), _ptr(m), t.numel())
    _check("pyramid_rmsprop_step", load().pyramid_rmsprop_step(
        n, segs, float(lr), float(rho_ms), float(rho_m), float(eps), _stream(stream)))


def pyramid_rmsprop_learning_rate(epoch: int) -> float:
    """1e-6 + 1e-2 (2^(-1/100))^epoch (Section 3, "Training")."""
    return load().pyramid_rmsprop_learning_rate(int(epoch))


class RMSprop:
    """Optimiser state (zero-initialised) for a fixed list of parameter
    tensors; `step(grads, epoch)` applies one update with the paper's
    hyper-parameters and learning-rate schedule."""

    def __init__(self, params):
        self.params = list(params)
        self.ms = [torch.zeros_like(p) for p in self.params]
        self.mom = [torch.zeros_like(p) for p in self.params]

    def step(self, grads, epoch: int, stream=None):
        pyramid_rmsprop_step(self.params, list(grads), self.ms, self.mom,
                             pyramid_rmsprop_learning_rate(epoch), stream=stream)


def pyramid_crop(x, n, box, tile, stream=None):
    """tile [d][h][w][C] = x[n, z0:z0+d, y0:y0+h, x0:x0+w, :]; box = (z0, y0,
    x0, d, h, w)."""
    N, D, H, W, C = x.shape
    if tile.dtype != x.dtype or tuple(tile.shape[-4:]) != (box[3], box[4], box[5], C):
        raise ValueError("tile must be [d][h][w][C] of x's dtype")
    _check("pyramid_crop", load().pyramid_crop(N, D, H, W, C, _DT[x.dtype], n, *box, _ptr(x),
                                               _ptr(tile), _stream(stream)))


def pyramid_sample_cubes(x, cubes, size, out, labels=None, out_labels=None, stream=None):
    """Training cubes out [count][d][h][w][C] (and out_labels [count][d][h][w])
    from x [N][D][H][W][C] (labels [N][D][H][W] int32); `cubes` is a sequence
    of plstm_cube (at most PLSTM_MAX_CUBES), `size` = (d, h, w)."""
    N, D, H, W, C = x.shape
    d, h, w = size
    count = len(cubes)
    if count < 1 or count > PLSTM_MAX_CUBES:
        raise ValueError("between 1 and %d cubes per call" % PLSTM_MAX_CUBES)
    if out.dtype != x.dtype or tuple(out.shape) != (count, d, h, w, C):
        raise ValueError("out must be [count][d][h][w][C] of x's dtype")
    if labels is not None:
        if labels.dtype != torch.int32 or out_labels is None or out_labels.dtype != torch.int32:
            raise ValueError("labels and out_labels must be int32")
        if tuple(out_labels.shape) != (count, d, h, w) or tuple(labels.shape) != (N, D, H, W):
            raise ValueError("labels [N][D][H][W], out_labels [count][d][h][w]")
    arr = (plstm_cube * count)(*cubes)
    _check("pyramid_sample_cubes", load().pyramid_sample_cubes(
        N, D, H, W, C, _DT[x.dtype], count, arr, d, h, w, _ptr(x), _ptr(labels), _ptr(out),
        _ptr(out_labels), _stream(stream)))


def draw_cubes(rng, N, volume, size, count, rotate=True, flip_axes="zyx"):
    """Random training cubes (host side): a uniform batch element and corner
    among the boxes of `size` = (d, h, w) inside `volume` = (D, H, W); with
    `rotate` an angle uniform in [0, 2 pi) about z; each axis named in
    `flip_axes` flipped with probability 1/2.  The EM recipe is the default;
    the MR recipe is rotate=False, flip_axes="x".  `rng` is a
    numpy.random.Generator."""
    import math
    D, H, W = volume
    d, h, w = size
    bits = {"z": PLSTM_FLIP_Z, "y": PLSTM_FLIP_Y, "x": PLSTM_FLIP_X}
    out = []
    for _ in range(count):
        n = int(rng.integers(0, N))
        z0, y0, x0 = (int(rng.integers(0, E - e + 1)) for E, e in ((D, d), (H, h), (W, w)))
        theta = float(rng.uniform(0.0, 2.0 * math.pi)) if rotate else 0.0
        flips = 0
        for a in flip_axes:
            if rng.random() < 0.5:
                flips |= bits[a]
        out.append(plstm_cube(n, z0, y0, x0, math.cos(theta), math.sin(theta), flips))
    return out


def pyramid_stitch_clear(acc, wsum, stream=None):
    D, H, W, K = acc.shape
    _check("pyramid_stitch_clear", load().pyramid_stitch_clear(D, H, W, K, _ptr(acc),
                                                               _ptr(wsum), _stream(stream)))


def pyramid_stitch_add(p, box, acc, wsum, sigma_scale=0.25, stream=None):
    """acc += g p, wsum += g for the tile p [d][h][w][K] at box (z0, y0, x0, d,
    h, w) with Gaussian weights g."""
    D, H, W, K = acc.shape
    _check("pyramid_stitch_add", load().pyramid_stitch_add(
        D, H, W, K, *box, float(sigma_scale), _ptr(p), _ptr(acc), _ptr(wsum), _stream(stream)))


def pyramid_stitch_finish(acc, wsum, out, stream=None):
    D, H, W, K = acc.shape
    _check("pyramid_stitch_finish", load().pyramid_stitch_finish(
        D, H, W, K, _ptr(acc), _ptr(wsum), _ptr(out), _stream(stream)))


def pyramid_lstm_timing_enable(on: bool) -> None:
    """Start (clearing earlier records) or stop per-phase HIP-event timing."""
    _check("pyramid_lstm_timing_enable", load().pyramid_lstm_timing_enable(int(bool(on))))


def pyramid_lstm_timing_read(max_phases: int = 32):
    """{phase: (total_ms, launches)} accumulated since timing was enabled."""
    names = ctypes.create_string_buffer(32 * max_phases)
    ms = (ctypes.c_double * max_phases)()
    launches = (ctypes.c_int * max_phases)()
    count = ctypes.c_int(0)
    _check("pyramid_lstm_timing_read", load().pyramid_lstm_timing_read(
        max_phases, names, ms, launches, ctypes.byref(count)))
    out = {}
    for k in range(count.value):
        nm = names.raw[32 * k:32 * k + 32].split(b"\0", 1)[0].decode()
        out[nm] = (ms[k], launches[k])
    return out


def pyramid_lstm_set_forward_path(path: int) -> None:
    """0 = automatic, 1 = generic path only, 2 = MFMA sweep where supported,
    3 = MFMA sweep with every strip staged chunk by chunk, 4 = plane-step
    MFMA path where supported."""
    _check("pyramid_lstm_set_forward_path", load().pyramid_lstm_set_forward_path(int(path)))


def pyramid_lstm_set_backward_path(path: int) -> None:
    """0 = automatic, 1 = generic path only, 2 = MFMA sweep where supported,
    3 = plane-step MFMA path where supported."""
    _check("pyramid_lstm_set_backward_path", load().pyramid_lstm_set_backward_path(int(path)))


def pyramid_lstm_set_step_split(mode: int) -> None:
    """Plane-step launch shape: 0 = automatic, 1 = always split each tile's K
    over a workgroup's waves, 2 = never, 3 = never and the fp32 forward
    reading its operands from L1 instead of LDS-staged pixel blocks."""
    _check("pyramid_lstm_set_step_split", load().pyramid_lstm_set_step_split(int(mode)))


def pyramid_lstm_set_bf16_mfma(on: int) -> None:
    """bf16-storage layers with 32 or 64 hidden units: 1 = bf16 MFMA (fp32
    accumulation) on pixel blocks staged in LDS, 2 = bf16 MFMA reading its
    operands from L1, 0 = fp32 MFMA."""
    _check("pyramid_lstm_set_bf16_mfma", load().pyramid_lstm_set_bf16_mfma(int(on)))


def pyramid_lstm_set_wgrad_staged(on: int) -> None:
    """Plane-step weight gradients: 1 = the LDS-staged GEMM where it applies
    (at most 32 hidden units, C a multiple of 4), 0 = the register-streamed
    kernel."""
    _check("pyramid_lstm_set_wgrad_staged", load().pyramid_lstm_set_wgrad_staged(int(on)))


def pyramid_lstm_device_status(clear: bool = False, stream=None) -> int:
    """This device's sticky status bits (synchronises `stream`):
    PLSTM_DEVICE_WAIT_GAVE_UP when a persistent sweep's bounded wait gave up
    since the last clear (that call's outputs were overwritten with NaN)."""
    out = ctypes.c_int32(0)
    _check("pyramid_lstm_device_status",
           load().pyramid_lstm_device_status(ctypes.byref(out), int(bool(clear)), _stream(stream)))
    return int(out.value)


def pyramid_lstm_set_wait_test(on: bool) -> None:
    """Failure-path test mode: every persistent-sweep wait expects a step that
    is never published and gives up after 16 polls (launches still finish)."""
    _check("pyramid_lstm_set_wait_test", load().pyramid_lstm_set_wait_test(int(bool(on))))
