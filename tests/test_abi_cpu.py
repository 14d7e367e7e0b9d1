"""C-ABI checks that need no GPU: symbols, sizes, argument validation.

Every call here is rejected by validation before the library touches HIP, so
the fake (aligned, never dereferenced) pointers are never used.
"""
from __future__ import annotations

import ctypes
import os
import re

import pytest

import paper_1506_07452_amd as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pyramid_lstm.h")
FAKE = ctypes.c_void_p(0x10000)      # aligned, never dereferenced


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pyramid_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    return P.load()


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("pyramid_lstm_forward", "pyramid_lstm_backward", "pyramid_lstm_workspace_size",
              "pyramid_lstm_saved_size", "pyramid_lstm_status_string", "pyramid_fc_tanh_forward",
              "pyramid_fc_tanh_backward", "pyramid_softmax_ce", "pyramid_fc_workspace_size"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert hasattr(P, name), "binding lacks " + name


def shape(**kw):
    d = dict(N=1, D=8, H=8, W=8, C=1, O=4, dtype=P.PLSTM_F32)
    d.update(kw)
    return P.plstm_shape(**d)


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert P.pyramid_lstm_status_string(code) not in ("", "unknown status")
    assert P.pyramid_lstm_status_string(-99) == "unknown status"


def test_sizes(lib):
    s = shape()
    V = 8 * 8 * 8
    assert P.pyramid_lstm_saved_size(s) >= 6 * V * 5 * 4 * 4
    assert P.pyramid_lstm_workspace_size(s, 0) > 0
    assert P.pyramid_lstm_workspace_size(s, 1) >= P.pyramid_lstm_workspace_size(s, 0)
    for bad in (dict(O=5), dict(O=0), dict(C=0), dict(D=0), dict(dtype=7), dict(C=5000),
                dict(N=20000)):
        assert P.pyramid_lstm_workspace_size(shape(**bad), 0) == 0, bad
        assert P.pyramid_lstm_saved_size(shape(**bad)) == 0, bad
    assert lib.pyramid_lstm_workspace_size(None, 0) == 0


def fwd(lib, s, x=FAKE, wx=FAKE, wh=FAKE, b=FAKE, h=FAKE, saved=None, ws=FAKE, nbytes=None):
    if nbytes is None:
        nbytes = 0
    return lib.pyramid_lstm_forward(ctypes.byref(s) if s is not None else None, x, wx, wh, b, h,
                                    saved, ws, nbytes, None)


def test_forward_validation(lib):
    s = shape()
    assert fwd(lib, None) == -1
    assert fwd(lib, s, x=None) == -1
    assert fwd(lib, s, h=None) == -1
    assert fwd(lib, s, ws=None) == -1
    assert fwd(lib, s, wx=ctypes.c_void_p(0x10004)) == -1            # misaligned
    assert fwd(lib, shape(O=5)) == -2
    assert fwd(lib, shape(D=-1)) == -1
    assert fwd(lib, s, nbytes=0) == -3                                # workspace too small
    need = P.pyramid_lstm_workspace_size(s, 1)
    assert fwd(lib, s, saved=FAKE, nbytes=need - 1) == -3
    assert fwd(lib, shape(dtype=P.PLSTM_BF16), saved=FAKE, nbytes=1 << 40) == -2
    assert fwd(lib, shape(K=4)) == -1                                 # even filter
    assert fwd(lib, shape(K=-3)) == -1
    assert fwd(lib, shape(K=9)) == -2                                 # larger than 7


def test_filter_size_in_sizes(lib):
    """K = 0 means 3; the workspace grows with the filter's taps."""
    assert (P.pyramid_lstm_workspace_size(shape(K=0), 1) ==
            P.pyramid_lstm_workspace_size(shape(K=3), 1))
    assert (P.pyramid_lstm_workspace_size(shape(O=32, K=7), 1) >
            P.pyramid_lstm_workspace_size(shape(O=32, K=3), 1))
    for k in (1, 3, 5, 7):
        assert P.pyramid_lstm_workspace_size(shape(K=k), 1) > 0
    for k in (2, 9, -1):
        assert P.pyramid_lstm_workspace_size(shape(K=k), 1) == 0


def test_backward_validation(lib):
    s = shape()
    args = [FAKE] * 11
    def call(sh=s, nbytes=0, **over):
        a = list(args)
        names = ["x", "wx", "wh", "b", "saved", "dh", "dx", "dwx", "dwh", "db", "ws"]
        for k, v in over.items():
            a[names.index(k)] = v
        return lib.pyramid_lstm_backward(ctypes.byref(sh), *a, nbytes, None)
    assert call(saved=None) == -1
    assert call(dh=None) == -1
    assert call(dwh=None) == -1
    assert call(ws=None) == -1
    assert call(dh=ctypes.c_void_p(0x10002)) == -1
    assert call(shape(dtype=P.PLSTM_BF16), nbytes=1 << 40) == -2
    assert call(nbytes=16) == -3


def test_fc_validation(lib):
    assert lib.pyramid_fc_tanh_forward(0, 4, 4, 0, FAKE, FAKE, FAKE, FAKE, None) == -1
    assert lib.pyramid_fc_tanh_forward(10, 4, 4, 3, FAKE, FAKE, FAKE, FAKE, None) == -1
    assert lib.pyramid_fc_tanh_forward(10, 4, 4, 0, FAKE, None, FAKE, FAKE, None) == -1
    assert lib.pyramid_fc_tanh_forward(10, 4, 4000, 0, FAKE, FAKE, FAKE, FAKE, None) == -2
    assert lib.pyramid_fc_tanh_backward(10, 4, 4, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE,
                                        FAKE, 0, None) == -3
    assert lib.pyramid_fc_workspace_size(0, 4, 4) == 0
    assert lib.pyramid_fc_workspace_size(100, 4, 4) > 0
    # softmax: K too large, missing loss with labels, gradient without labels
    assert lib.pyramid_softmax_ce(10, 4, 17, 0, FAKE, FAKE, FAKE, None, FAKE, None, None, None,
                                  None, None, 0, None) == -2
    assert lib.pyramid_softmax_ce(10, 4, 4, 0, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None,
                                  None, FAKE, 1 << 30, None) == -1
    assert lib.pyramid_softmax_ce(10, 4, 4, 0, FAKE, FAKE, FAKE, None, FAKE, None, None, FAKE,
                                  FAKE, None, 0, None) == -1
    assert lib.pyramid_softmax_ce(10, 4, 4, 0, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None,
                                  None, FAKE, 8, None) == -3


def test_head_validation(lib):
    assert lib.pyramid_head_workspace_size(1000, 16, 32, 4) > 0
    assert lib.pyramid_head_workspace_size(1000, 32, 64, 16) > 0
    for bad in ((1000, 16, 33, 4), (1000, 8, 32, 4), (1000, 16, 32, 17), (0, 16, 32, 4)):
        assert lib.pyramid_head_workspace_size(*bad) == 0, bad
    args = [FAKE] * 13
    def call(M=1000, Cin=16, F=32, K=4, nbytes=1 << 30, **over):
        a = list(args)
        names = ["x", "w1", "b1", "w2", "b2", "labels", "p", "loss", "dx", "dw1", "db1", "dw2",
                 "db2"]
        for k, v in over.items():
            a[names.index(k)] = v
        return lib.pyramid_head_train(M, Cin, F, K, *a, FAKE, nbytes, None)
    assert call(Cin=8) == -2
    assert call(K=17) == -2
    assert call(M=0) == -1
    assert call(labels=None) == -1
    assert call(dw2=None) == -1
    assert call(x=ctypes.c_void_p(0x10008)) == -1
    assert call(nbytes=16) == -3


def test_head_forward_validation(lib):
    bf16, f32 = P.PLSTM_BF16, P.PLSTM_F32
    for cin in (32, 64):
        for f in (32, 64, 128):
            for k in (1, 4, 16):
                assert lib.pyramid_head_forward_supported(bf16, cin, f, k) == 1
    for bad in ((f32, 64, 128, 4), (bf16, 16, 32, 4), (bf16, 64, 48, 4), (bf16, 64, 128, 17),
                (bf16, 64, 128, 0), (bf16, 128, 128, 4)):
        assert lib.pyramid_head_forward_supported(*bad) == 0, bad
    def call(M=1000, Cin=64, F=128, K=4, dtype=bf16, **over):
        names = ["x", "w1", "b1", "w2", "b2", "p"]
        a = [FAKE] * 6
        for k, v in over.items():
            a[names.index(k)] = v
        return lib.pyramid_head_forward(M, Cin, F, K, dtype, *a, None)
    assert call(M=0) == -1
    assert call(K=0) == -1
    assert call(dtype=7) == -1
    assert call(p=None) == -1
    assert call(w2=None) == -1
    assert call(x=ctypes.c_void_p(0x10008)) == -1
    assert call(dtype=f32) == -2
    assert call(F=48) == -2
    assert call(K=17) == -2


def test_binding_refuses_host_tensors():
    import torch
    x = torch.zeros(1, 2, 2, 2, 1)
    with pytest.raises((ValueError, RuntimeError)):
        P.pyramid_fc_tanh_forward(x.view(-1, 1), torch.zeros(1, 1), torch.zeros(1),
                                  torch.zeros(8, 1))


def test_path_knobs_and_timing_without_gpu():
    for fn, top in ((P.pyramid_lstm_set_forward_path, 4), (P.pyramid_lstm_set_backward_path, 3),
                    (P.pyramid_lstm_set_step_split, 3), (P.pyramid_lstm_set_bf16_mfma, 5),
                    (P.pyramid_lstm_set_wgrad_staged, 1)):
        for v in list(range(1, top + 1)) + [0]:
            fn(v)
        with pytest.raises(P.PyramidLSTMError):
            fn(top + 1)
        with pytest.raises(P.PyramidLSTMError):
            fn(-1)
    P.pyramid_lstm_set_bf16_mfma(1)       # back to the defaults
    P.pyramid_lstm_set_wgrad_staged(1)
    P.pyramid_lstm_set_forward_path(0)
    P.pyramid_lstm_timing_enable(True)
    assert P.pyramid_lstm_timing_read() == {}
    P.pyramid_lstm_timing_enable(False)


def test_wait_test_knob_and_status_validation(lib):
    """The failure-path knob takes 0 or 1 only; the status query rejects a
    null output before touching HIP."""
    P.pyramid_lstm_set_wait_test(True)
    P.pyramid_lstm_set_wait_test(False)
    assert lib.pyramid_lstm_set_wait_test(2) == -1
    assert lib.pyramid_lstm_set_wait_test(-1) == -1
    assert lib.pyramid_lstm_device_status(None, 0, None) == -1


def test_rmsprop_validation(lib):
    """Argument checks of the optimiser entry point (no GPU work: an update
    of zero elements returns before any launch)."""
    Seg = P.plstm_param_segment
    segs = (Seg * 2)(Seg(FAKE, FAKE, FAKE, FAKE, 0), Seg(FAKE, FAKE, FAKE, FAKE, 0))
    step = lib.pyramid_rmsprop_step
    assert step(2, segs, 0.01, 0.9, 0.9, 1e-5, None) == 0
    assert step(0, segs, 0.01, 0.9, 0.9, 1e-5, None) == -1
    assert step(65, segs, 0.01, 0.9, 0.9, 1e-5, None) == -1
    assert step(2, None, 0.01, 0.9, 0.9, 1e-5, None) == -1
    assert step(2, segs, -1.0, 0.9, 0.9, 1e-5, None) == -1
    assert step(2, segs, 0.01, 1.0, 0.9, 1e-5, None) == -1
    assert step(2, segs, 0.01, 0.9, -0.1, 1e-5, None) == -1
    assert step(2, segs, 0.01, 0.9, 0.9, 0.0, None) == -1
    bad = (Seg * 1)(Seg(None, FAKE, FAKE, FAKE, 5))
    assert step(1, bad, 0.01, 0.9, 0.9, 1e-5, None) == -1
    bad = (Seg * 1)(Seg(FAKE, FAKE, ctypes.c_void_p(0x10002), FAKE, 5))
    assert step(1, bad, 0.01, 0.9, 0.9, 1e-5, None) == -1
    bad = (Seg * 1)(Seg(FAKE, FAKE, FAKE, FAKE, -1))
    assert step(1, bad, 0.01, 0.9, 0.9, 1e-5, None) == -1


def test_learning_rate_schedule_matches_oracle():
    import oracle.optim as optim
    for e in (0, 1, 50, 100, 1234, 6000):
        assert P.pyramid_rmsprop_learning_rate(e) == pytest.approx(optim.learning_rate(e),
                                                                   rel=1e-14)


def test_stitch_and_crop_validation(lib):
    """Boxes outside the volume, null pointers and a non-positive Gaussian
    width are refused before any launch."""
    assert lib.pyramid_crop(1, 4, 5, 6, 2, 0, 0, 0, 0, 0, 5, 5, 6, FAKE, FAKE, None) == -1
    assert lib.pyramid_crop(1, 4, 5, 6, 2, 0, 1, 0, 0, 0, 4, 5, 6, FAKE, FAKE, None) == -1
    assert lib.pyramid_crop(1, 4, 5, 6, 2, 0, 0, 0, 0, -1, 2, 2, 2, FAKE, FAKE, None) == -1
    assert lib.pyramid_crop(1, 4, 5, 6, 2, 0, 0, 0, 0, 0, 2, 2, 2, None, FAKE, None) == -1
    assert lib.pyramid_crop(1, 4, 5, 6, 2, 7, 0, 0, 0, 0, 2, 2, 2, FAKE, FAKE, None) == -1
    add = lib.pyramid_stitch_add
    assert add(4, 5, 6, 3, 0, 0, 4, 2, 2, 3, 0.25, FAKE, FAKE, FAKE, None) == -1
    assert add(4, 5, 6, 3, 0, 0, 0, 2, 2, 3, 0.0, FAKE, FAKE, FAKE, None) == -1
    assert add(4, 5, 6, 3, 0, 0, 0, 2, 2, 3, 0.25, None, FAKE, FAKE, None) == -1
    assert lib.pyramid_stitch_clear(0, 5, 6, 3, FAKE, FAKE, None) == -1
    assert lib.pyramid_stitch_finish(4, 5, 6, 3, FAKE, None, FAKE, None) == -1



def shape2d(**kw):
    d = dict(N=1, H=8, W=8, C=1, O=4, dtype=P.PLSTM_F32, K=3)
    d.update(kw)
    return P.plstm2d_shape(**d)


def test_2d_sizes_and_validation(lib):
    """The 2D entry points: four directions of saved state, the same shape
    rules as the volume layer, every bad argument rejected before HIP."""
    s = shape2d()
    V = 8 * 8
    assert P.pyramid_lstm2d_saved_size(s) >= 4 * V * 6 * 4 * 4
    assert P.pyramid_lstm2d_saved_size(s) < 6 * V * 6 * 4 * 4
    assert P.pyramid_lstm2d_workspace_size(s, 1) >= P.pyramid_lstm2d_workspace_size(s, 0) > 0
    for bad in (dict(O=5), dict(C=0), dict(H=0), dict(W=-1), dict(dtype=3), dict(K=4),
                dict(K=9), dict(N=0)):
        assert P.pyramid_lstm2d_workspace_size(shape2d(**bad), 1) == 0, bad
        assert P.pyramid_lstm2d_saved_size(shape2d(**bad)) == 0, bad
    assert lib.pyramid_lstm2d_saved_size(None) == 0

    def f(sh=s, nbytes=0, **over):
        a = dict(x=FAKE, wx=FAKE, wh=FAKE, b=FAKE, h=FAKE, saved=None, ws=FAKE)
        a.update(over)
        return lib.pyramid_lstm2d_forward(ctypes.byref(sh), a["x"], a["wx"], a["wh"], a["b"],
                                          a["h"], a["saved"], a["ws"], nbytes, None)
    assert lib.pyramid_lstm2d_forward(None, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, 0,
                                      None) == -1
    assert f(x=None) == -1
    assert f(h=None) == -1
    assert f(b=ctypes.c_void_p(0x10002)) == -1
    assert f(shape2d(O=5)) == -2
    assert f(shape2d(K=2)) == -1
    assert f(shape2d(K=9)) == -2
    assert f(nbytes=0) == -3
    assert f(shape2d(dtype=P.PLSTM_BF16), saved=FAKE, nbytes=1 << 40) == -2

    def bw(sh=s, nbytes=0, **over):
        names = ["x", "wx", "wh", "b", "saved", "dh", "dx", "dwx", "dwh", "db", "ws"]
        a = [FAKE] * 11
        for k, v in over.items():
            a[names.index(k)] = v
        return lib.pyramid_lstm2d_backward(ctypes.byref(sh), *a, nbytes, None)
    assert bw(saved=None) == -1
    assert bw(dwx=None) == -1
    assert bw(shape2d(dtype=P.PLSTM_BF16), nbytes=1 << 40) == -2
    assert bw(nbytes=16) == -3


def test_sample_cubes_validation(lib):
    def call(N=1, D=8, H=10, W=12, C=2, dtype=P.PLSTM_F32, cubes=None, size=(4, 5, 6), x=FAKE,
             labels=None, out=FAKE, out_labels=None):
        if cubes is None:
            cubes = [P.plstm_cube(0, 0, 0, 0, 1.0, 0.0, 0)]
        arr = (P.plstm_cube * len(cubes))(*cubes)
        return lib.pyramid_sample_cubes(N, D, H, W, C, dtype, len(cubes), arr, *size, x, labels,
                                        out, out_labels, None)
    cube = P.plstm_cube
    assert call(x=None) == -1
    assert call(out=None) == -1
    assert call(labels=FAKE) == -1                                    # labels without out_labels
    assert call(cubes=[cube(1, 0, 0, 0, 1.0, 0.0, 0)]) == -1         # n out of range
    assert call(cubes=[cube(0, 5, 0, 0, 1.0, 0.0, 0)]) == -1         # z0 + d > D
    assert call(cubes=[cube(0, 0, 6, 0, 1.0, 0.0, 0)]) == -1
    assert call(cubes=[cube(0, 0, 0, 7, 1.0, 0.0, 0)]) == -1
    assert call(cubes=[cube(0, 0, 0, -1, 1.0, 0.0, 0)]) == -1
    assert call(cubes=[cube(0, 0, 0, 0, 1.0, 0.0, 8)]) == -1         # flips > 7
    assert call(cubes=[cube(0, 0, 0, 0, 1.5, 0.0, 0)]) == -1         # |cos| > 1
    assert call(cubes=[cube(0, 0, 0, 0, float("nan"), 0.0, 0)]) == -1
    assert call(cubes=[cube(0, 0, 0, 0, 1.0, 0.0, 0)] * 65) == -1    # more than the maximum
    assert call(size=(9, 5, 6)) == -1
    assert call(dtype=2) == -1
    assert call(x=ctypes.c_void_p(0x10002)) == -1
    assert lib.pyramid_sample_cubes(1, 8, 10, 12, 2, 0, 0, None, 4, 5, 6, FAKE, None, FAKE, None,
                                    None) == -1


def test_draw_cubes_recipes():
    """Host-side draws: boxes inside the volume, EM recipe (any angle, flips
    on z, y, x each about half the time), MR recipe (no rotation, x only)."""
    import numpy as np
    rng = np.random.default_rng(5)
    em = P.draw_cubes(rng, 2, (30, 512, 512), (15, 128, 128), 2000)
    for c in em:
        assert 0 <= c.n < 2 and 0 <= c.z0 <= 15 and 0 <= c.y0 <= 384 and 0 <= c.x0 <= 384
        assert abs(c.cos_t ** 2 + c.sin_t ** 2 - 1) < 1e-6
    for bit in (P.PLSTM_FLIP_Z, P.PLSTM_FLIP_Y, P.PLSTM_FLIP_X):
        frac = np.mean([(c.flips & bit) != 0 for c in em])
        assert 0.45 < frac < 0.55
    ang = np.arctan2([c.sin_t for c in em], [c.cos_t for c in em])
    assert np.histogram(ang, bins=4, range=(-np.pi, np.pi))[0].min() > 400
    mr = P.draw_cubes(rng, 5, (48, 240, 240), (25, 240, 240), 500, rotate=False, flip_axes="x")
    assert all(c.cos_t == 1.0 and c.sin_t == 0.0 and c.flips in (0, P.PLSTM_FLIP_X) for c in mr)
    assert all(c.y0 == 0 and c.x0 == 0 and 0 <= c.z0 <= 23 for c in mr)
    assert 0.4 < np.mean([c.flips != 0 for c in mr]) < 0.6


def test_noalloc_validation_without_gpu(lib):
    """The no-allocation forward rejects null pointers and shapes beyond its
    scratch before any HIP call."""
    big = shape(D=80, H=64, W=64, C=3, O=16)
    assert P.pyramid_lstm_workspace_size(big, 0) > P.PLSTM_NOALLOC_SCRATCH_BYTES
    f = lib.pyramid_lstm_forward_noalloc
    assert f(ctypes.byref(big), FAKE, FAKE, FAKE, FAKE, FAKE, None) == P.PLSTM_ESCRATCH
    small = shape(C=3, O=16)
    assert f(ctypes.byref(small), None, FAKE, FAKE, FAKE, FAKE, None) == -1
    assert f(ctypes.byref(small), FAKE, FAKE, FAKE, FAKE, None, None) == -1
    assert f(None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == -1
