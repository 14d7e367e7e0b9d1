"""GPU parity of the 2D PyraMiD-LSTM layer (four line sweeps over images,
Section 2.1-2.2 and Fig. 1) against the oracle, through the C ABI."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import oracle.layer2d as o2d
import paper_1506_07452_amd as P
import synth
from paper_1506_07452_amd.network import LayerW, layer2d_backward, layer2d_forward
from tests.gpu_util import TOL, dev, host, normwise, say

pytestmark = pytest.mark.gpu

# (N, H, W, C, O, K): lines shorter and longer than one 64-pixel group,
# ragged groups, single pixel / single row / single column images, every unit
# count of the MFMA kernels and one (O = 8) that only the generic kernels take,
# filters of 1, 3, 5 and 7 taps, channel counts below and above a 16-block.
SHAPES = [(1, 5, 6, 2, 16, 3), (2, 17, 33, 3, 16, 3), (1, 9, 70, 5, 32, 7),
          (1, 40, 3, 20, 64, 5), (1, 1, 1, 1, 16, 3), (1, 13, 1, 2, 16, 1),
          (2, 8, 11, 3, 8, 3), (1, 64, 65, 3, 16, 3), (1, 21, 130, 45, 64, 7),
          # 16 units (line blocks): several dense (tap, channel) K-groups, lines
          # longer than a segment and ragged, the widest filter
          (1, 9, 70, 5, 16, 7), (2, 12, 40, 20, 16, 5), (1, 30, 150, 17, 16, 3),
          (1, 40, 129, 1, 16, 1),
          # 16 units and at most 4 channels: dL/dx from the reverse line
          # blocks, at the widest filters and ragged segments
          (1, 11, 100, 4, 16, 7), (2, 20, 70, 4, 16, 5), (1, 7, 200, 3, 16, 3)]


def ident(s):
    return "x".join(map(str, s))


def case(shape, seed, dtype="f32"):
    N, H, W, C, O, K = shape
    x, wx, wh, b = synth.image2d(N, H, W, C, O, K, seed, dtype)
    return x, wx, wh, b


def run(shape, seed, dh_seed):
    x, wx, wh, b = case(shape, seed)
    N, H, W, C, O, K = shape
    dh = synth.upstream_grad((N, H, W, O), dh_seed)
    ref_h = o2d.forward2d(x, wx, wh, b)
    ref = o2d.backward2d(x, wx, wh, b, dh)
    say("2d layer", shape)
    xd, L = dev(x), LayerW(dev(wx), dev(wh), dev(b))
    P.pyramid_lstm_timing_enable(True)
    h_inf, _ = layer2d_forward(xd, L)
    h, saved = layer2d_forward(xd, L, training=True)
    grads = layer2d_backward(xd, L, saved, dev(dh))
    phases = P.pyramid_lstm_timing_read()
    P.pyramid_lstm_timing_enable(False)
    torch.cuda.synchronize()
    assert normwise(host(h_inf), ref_h) <= TOL["f32"]
    assert torch.equal(h_inf, h)
    for name, got in zip(("dx", "dwx", "dwh", "db"), grads):
        err = normwise(host(got), ref[name])
        assert err <= TOL["f32"], (name, err)
    return phases


@pytest.mark.parametrize("shape", SHAPES, ids=ident)
def test_2d_layer_matches_oracle(shape):
    phases = run(shape, 9000 + sum(shape), 31 + sum(shape))
    if shape[4] in (16, 32, 64):
        assert "sweep_fwd_step" in phases and "sweep_bwd_step" in phases, phases
        # one launch (the sum over directions) when the reverse sweep gives
        # dL/dx: with 16 units the line blocks run it (at most 4 channels),
        # with 32 the staged reverse step (at most 32 channels)
        O, C = shape[4], shape[3]
        fused = C <= 4 if O == 16 else (O == 32 and C <= 32)
        assert (phases["dx_step"][1] == 1) == fused, phases
    else:
        assert "sweep_fwd_generic" in phases and "sweep_bwd_generic" in phases, phases


@pytest.fixture(params=[1, 2, 3], ids=["split", "nosplit", "nosplit_l1"])
def step_split(request):
    P.pyramid_lstm_set_step_split(request.param)
    yield
    P.pyramid_lstm_set_step_split(0)


@pytest.mark.parametrize("shape", [(2, 17, 33, 3, 16, 3), (1, 9, 70, 5, 32, 7),
                                   (1, 40, 3, 20, 64, 5)], ids=ident)
def test_2d_both_launch_shapes(shape, step_split):
    run(shape, 9100 + sum(shape), 37 + sum(shape))


@pytest.mark.parametrize("shape", [(2, 17, 33, 3, 16, 3), (1, 9, 70, 5, 32, 7)], ids=ident)
def test_2d_generic_kernels(shape):
    P.pyramid_lstm_set_forward_path(1)
    P.pyramid_lstm_set_backward_path(1)
    try:
        phases = run(shape, 9200 + sum(shape), 41 + sum(shape))
    finally:
        P.pyramid_lstm_set_forward_path(0)
        P.pyramid_lstm_set_backward_path(0)
    assert "sweep_fwd_step" not in phases and "sweep_bwd_step" not in phases, phases


@pytest.mark.parametrize("shape", [(2, 17, 33, 3, 16, 3), (1, 21, 130, 45, 64, 7)], ids=ident)
def test_2d_saved_state_matches_oracle(shape):
    """The saved h^d, c^d and gates of the four directions: those of the
    y+, y-, x+, x- sweeps of the oracle's D = 1 volume embedding."""
    x, wx, wh, b = case(shape, 9300 + sum(shape))
    N, H, W, C, O, K = shape
    wx3, wh3, b3 = o2d.embed(wx, wh, b)
    ref = oracle.forward(x[:, None], wx3, wh3, b3, want_hd=True, want_saved=True)
    say("2d saved", shape)
    h, saved = layer2d_forward(dev(x), LayerW(dev(wx), dev(wh), dev(b)), training=True)
    torch.cuda.synchronize()
    counts = {"gates": 4 * N * H * W * 4 * O, "cell": 4 * N * H * W * O, "hd": 4 * N * H * W * O}
    off = 0
    for name in ("gates", "cell", "hd"):
        off = (off + 255) // 256 * 256
        got = host(saved[off:off + counts[name] * 4].view(torch.float32))
        off += counts[name] * 4
        want = ref[name][2:, :, 0]
        assert normwise(got.reshape(want.shape), want) <= TOL["f32"], name


@pytest.mark.parametrize("bf16_mfma", [1, 3, 2, 0, 5],
                         ids=["bf16_mt", "bf16_lds", "bf16_l1", "fp32_mfma", "bf16_proj"])
@pytest.mark.parametrize("shape", [(1, 9, 70, 5, 32, 7), (1, 40, 3, 20, 64, 5),
                                   (2, 17, 33, 3, 16, 3)], ids=ident)
def test_2d_bf16_forward(shape, bf16_mfma):
    x, wx, wh, b = case(shape, 9400 + sum(shape), "bf16")
    ref = o2d.forward2d(x, wx, wh, b)
    say("2d bf16", shape, bf16_mfma)
    P.pyramid_lstm_set_bf16_mfma(bf16_mfma)
    try:
        h, _ = layer2d_forward(dev(x, "bf16"), LayerW(dev(wx, "bf16"), dev(wh, "bf16"),
                                                      dev(b, "bf16")))
        torch.cuda.synchronize()
    finally:
        P.pyramid_lstm_set_bf16_mfma(1)
    assert h.dtype == torch.bfloat16
    assert normwise(host(h), ref) <= TOL["bf16"]


def test_2d_large_image_sampled():
    """A 2 x 512 x 512 x 3 batch, 32 units, 7 taps.  The y+ sweep's h^d of
    the first rows depends on those rows alone, so the oracle computes it on
    a 6-row crop (the other three directions given zero weights and bias,
    which makes their output exactly zero) and the saved h^d of the y+
    direction is compared there."""
    shape = (2, 512, 512, 3, 32, 7)
    x, wx, wh, b = case(shape, 9500)
    N, H, W, C, O, K = shape
    rows = 6
    wx1, wh1, b1 = wx.copy(), wh.copy(), b.copy()
    wx1[1:] = 0.0
    wh1[1:] = 0.0
    b1[1:] = 0.0
    ref = o2d.forward2d(x[:, :rows], wx1, wh1, b1)
    say("2d large", shape)
    h, saved = layer2d_forward(dev(x), LayerW(dev(wx), dev(wh), dev(b)), training=True)
    torch.cuda.synchronize()
    cnt_g, cnt_s = 4 * N * H * W * 4 * O, 4 * N * H * W * O
    off = (cnt_g * 4 + 255) // 256 * 256          # gates, then cell
    off = (off + cnt_s * 4 + 255) // 256 * 256    # then hd
    hd = saved[off:off + cnt_s * 4].view(torch.float32).view(4, N, H, W, O)
    assert normwise(host(hd[0, :, :rows]), ref) <= TOL["f32"]
    assert torch.isfinite(h).all()


# The 2D workload that bench.py times: 30 EM-like 512 x 512 slices as images,
# 16 units, one channel, 3 taps (line blocks of 16 lines per launch).
BENCH_2D = (30, 512, 512, 1, 16, 3)
LINES = 40                      # > two 16-line launches
IMAGES = (0, 13, 29)            # images the oracle checks


@pytest.mark.timeout(600)
@pytest.mark.parametrize("d", range(4), ids=["y+", "y-", "x+", "x-"])
def test_2d_line_blocks_at_bench_scale(d):
    """Direction d alone over the full bench batch.  The other three get zero
    filters and an input-gate bias of -200, so i = 0 exactly in fp32: their
    h is exactly zero and so is every gate gradient of theirs (with i = 1/2
    instead, dA_g = dc i (1 - g^2) would carry dL/dc down the opposite sweep
    of the same axis, past the crop).  The sweep's first 40 lines depend only
    on those lines, and with dL/dh zero everywhere else (other images and
    later lines) the backward touches nothing else: the oracle on that
    40-line crop of three images gives h there, dL/dx there (exactly zero
    elsewhere) and every parameter gradient.  Full 512-pixel lines cross
    eight 64-pixel segments and three line-block launches."""
    N, H, W, C, O, K = BENCH_2D
    x, wx, wh, b = synth.image2d(N, H, W, C, O, K, seed=2048, scale=0.1)
    for p in (wx, wh, b):
        keep = p[d].copy()
        p[...] = 0.0
        p[d] = keep
    for e in range(4):
        if e != d:
            b[e, :O] = -200.0
    rows = d < 2
    first = d % 2 == 0
    span = slice(0, LINES) if first else slice((H if rows else W) - LINES, None)
    crop = (slice(None), span) if rows else (slice(None), slice(None), span)
    img = list(IMAGES)
    dh = np.zeros((N, H, W, O), dtype=np.float32)
    dh_crop = synth.upstream_grad(x[img][crop].shape[:-1] + (O,), 4000 + d)
    sub = dh[img]
    sub[crop] = dh_crop
    dh[img] = sub
    say("2d bench scale, direction", d)
    xd, L = dev(x), LayerW(dev(wx), dev(wh), dev(b))
    P.pyramid_lstm_timing_enable(True)
    h, saved = layer2d_forward(xd, L, training=True)
    gdx, gdwx, gdwh, gdb = layer2d_backward(xd, L, saved, dev(dh))
    phases = P.pyramid_lstm_timing_read()
    P.pyramid_lstm_timing_enable(False)
    torch.cuda.synchronize()
    # the reverse line blocks gave dL/dx: only the sum over directions remains
    assert "sweep_fwd_step" in phases and phases["dx_step"][1] == 1, phases
    xc = np.ascontiguousarray(x[img][crop])
    say("2d bench scale oracle", d)
    ref_h = o2d.forward2d(xc, wx, wh, b)
    ref = o2d.backward2d(xc, wx, wh, b, dh_crop)
    hh = host(h)[img][crop]
    err_h = normwise(hh, ref_h)
    dx = host(gdx)
    dx_crop = dx[img][crop]
    mask = np.ones(dx.shape, dtype=bool)
    msub = mask[img]
    msub[crop] = False
    mask[img] = msub
    errs = {"h": err_h, "dx": normwise(dx_crop, ref["dx"]),
            "dwx": normwise(host(gdwx), ref["dwx"]), "dwh": normwise(host(gdwh), ref["dwh"]),
            "db": normwise(host(gdb), ref["db"])}
    print("[2d bench scale] direction %d: %s" % (d, {k: "%.2e" % v for k, v in errs.items()}),
          flush=True)
    assert not np.any(dx[mask]), "dL/dx outside the crop must be exactly zero"
    for k, v in errs.items():
        assert v <= TOL["f32"], (k, v)
