"""GPU parity of one PyraMiD-LSTM layer (forward and backward) against the
fp64 oracle, plus invariants that hold at any size, through the C ABI."""
from __future__ import annotations

import os
import time

import numpy as np
import pytest
import torch

import oracle
import paper_1506_07452_amd as P
import synth
from paper_1506_07452_amd.network import LayerW, layer_backward, layer_forward
from tests.gpu_util import DEV, TOL, dev, host, layer_dev, normwise, saved_view, say

pytestmark = pytest.mark.gpu

# (N, D, H, W, C, O): tiny, ragged (planes not multiples of any tile), several
# tiles per plane, degenerate extents, every supported O.
SHAPES = [
    (1, 8, 8, 8, 1, 4),
    (1, 5, 37, 29, 3, 16),
    (2, 7, 9, 11, 2, 8),
    (1, 3, 3, 3, 1, 32),
    (1, 4, 6, 70, 3, 64),
    (1, 1, 1, 1, 1, 4),
    (1, 1, 13, 1, 2, 16),
    (1, 12, 64, 50, 3, 16),
    (2, 9, 17, 40, 32, 32),
]


def instance(shape, seed, dtype="f32"):
    N, D, H, W, C, O = shape
    wl = synth.Workload("t", N, D, H, W, C, [O], dtype=dtype, seed=seed)
    return synth.make(wl)


@pytest.fixture
def generic_path():
    """Run the forward on the generic per-plane path only."""
    P.pyramid_lstm_set_forward_path(1)
    yield
    P.pyramid_lstm_set_forward_path(0)


@pytest.mark.parametrize("shape", SHAPES + [(3, 6, 20, 18, 2, 16), (1, 9, 2, 300, 4, 16)],
                         ids=lambda s: "x".join(map(str, s)))
def test_forward_matches_oracle(shape):
    inst = instance(shape, 1000 + sum(shape))
    L = inst.layers[0]
    ref = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    say("forward", shape)
    h, _ = layer_forward(dev(inst.x), layer_dev(L))
    torch.cuda.synchronize()
    err = normwise(host(h), ref)
    assert err <= TOL["f32"], err


@pytest.fixture
def chunked_sweep():
    """Run the MFMA forward sweep with every strip staged chunk by chunk (no
    strip kept whole in LDS), so both strip kinds are covered on small shapes."""
    P.pyramid_lstm_set_forward_path(3)
    yield
    P.pyramid_lstm_set_forward_path(0)


# O = 16 shapes of both strip kinds: several strips per direction, ragged
# strips and tiles, single-row / single-column planes, C = 1..4.
O16_SHAPES = [(1, 5, 37, 29, 3, 16), (3, 6, 20, 18, 2, 16), (1, 9, 2, 300, 4, 16),
              (1, 12, 64, 50, 1, 16), (2, 17, 3, 1, 3, 16), (1, 30, 70, 9, 4, 16)]


@pytest.mark.parametrize("shape", O16_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_chunked_sweep_matches_oracle(shape, chunked_sweep):
    inst = instance(shape, 1200 + sum(shape))
    L = inst.layers[0]
    ref = oracle.forward(inst.x, L.wx, L.wh, L.b)
    say("forward chunked", shape)
    x, Ld = dev(inst.x), layer_dev(L)
    h, _ = layer_forward(x, Ld)
    assert normwise(host(h), ref["h"]) <= TOL["f32"]
    h2, saved = layer_forward(x, Ld, training=True)
    torch.cuda.synchronize()
    assert torch.equal(h, h2)


@pytest.mark.parametrize("shape", O16_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_sweep_saved_state_matches_oracle(shape):
    """Training forward of the default sweep: the saved per-direction h^d,
    c^d and gates match the oracle's, not only their sum."""
    inst = instance(shape, 1300 + sum(shape))
    L = inst.layers[0]
    ref = oracle.forward(inst.x, L.wx, L.wh, L.b, want_hd=True, want_saved=True)
    say("forward saved", shape)
    h, saved = layer_forward(dev(inst.x), layer_dev(L), training=True)
    torch.cuda.synchronize()
    assert normwise(host(h), ref["h"]) <= TOL["f32"]
    for name in ("hd", "cell", "gates"):
        got = saved_view(saved, name, shape)
        assert normwise(got, ref[name]) <= TOL["f32"], name


@pytest.mark.parametrize("shape", [(1, 5, 37, 29, 3, 16), (2, 4, 9, 7, 1, 16)],
                         ids=lambda s: "x".join(map(str, s)))
def test_generic_path_forward_matches_oracle(shape, generic_path):
    inst = instance(shape, 1100 + sum(shape))
    L = inst.layers[0]
    ref = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    say("forward generic", shape)
    P.pyramid_lstm_timing_enable(True)
    h, _ = layer_forward(dev(inst.x), layer_dev(L))
    phases = P.pyramid_lstm_timing_read()
    P.pyramid_lstm_timing_enable(False)
    assert "sweep_fwd_generic" in phases and "sweep_fwd_mfma" not in phases
    assert normwise(host(h), ref) <= TOL["f32"]


@pytest.fixture
def generic_backward():
    """Run the backward on the generic per-plane path only."""
    P.pyramid_lstm_set_backward_path(1)
    yield
    P.pyramid_lstm_set_backward_path(0)


@pytest.mark.parametrize("shape", [(1, 5, 37, 29, 3, 16), (2, 4, 9, 7, 1, 16)],
                         ids=lambda s: "x".join(map(str, s)))
def test_generic_path_backward_matches_oracle(shape, generic_backward):
    inst = instance(shape, 3100 + sum(shape))
    L = inst.layers[0]
    dh = synth.upstream_grad(inst.x.shape[:-1] + (shape[-1],), 17 + sum(shape))
    ref = oracle.backward(inst.x, L.wx, L.wh, L.b, dh)
    say("backward generic", shape)
    x, Ld = dev(inst.x), layer_dev(L)
    h, saved = layer_forward(x, Ld, training=True)
    P.pyramid_lstm_timing_enable(True)
    grads = layer_backward(x, Ld, saved, dev(dh))
    phases = P.pyramid_lstm_timing_read()
    P.pyramid_lstm_timing_enable(False)
    assert "sweep_bwd_generic" in phases and "sweep_bwd_mfma" not in phases
    for name, got in zip(("dx", "dwx", "dwh", "db"), grads):
        assert normwise(host(got), ref[name]) <= TOL["f32"], name


@pytest.fixture
def step_path():
    """Run forward and backward on the plane-step MFMA path wherever it
    supports the shape (O = 16 included, which otherwise takes the persistent
    sweeps)."""
    P.pyramid_lstm_set_forward_path(4)
    P.pyramid_lstm_set_backward_path(3)
    yield
    P.pyramid_lstm_set_forward_path(0)
    P.pyramid_lstm_set_backward_path(0)


# every unit count of the plane-step kernels; channel counts below, at and
# above one 16-channel block (zero-padded tails); planes smaller than one
# 64-pixel group, ragged groups, batch > 1
STEP_SHAPES = [(1, 5, 37, 29, 3, 16), (2, 4, 9, 7, 1, 16), (1, 6, 5, 4, 20, 16),
               (1, 3, 3, 3, 1, 32), (2, 9, 17, 40, 32, 32), (1, 4, 6, 70, 3, 64),
               (1, 2, 19, 3, 64, 64)]


@pytest.fixture(params=[0, 1, 2, 3], ids=["auto", "split", "nosplit", "nosplit_l1"])
def step_split(request):
    """Every launch shape of the plane-step kernels: the default (staged pixel
    blocks; the reverse step's K split over a workgroup's waves by gate-unit
    block), K split over a workgroup's waves, or one tile group per wave."""
    P.pyramid_lstm_set_step_split(request.param)
    yield request.param
    P.pyramid_lstm_set_step_split(0)


@pytest.mark.parametrize("shape", STEP_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_step_path_matches_oracle(shape, step_path, step_split):
    inst = instance(shape, 4000 + sum(shape))
    L = inst.layers[0]
    dh = synth.upstream_grad(inst.x.shape[:-1] + (shape[-1],), 11 + sum(shape))
    ref_h = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    ref = oracle.backward(inst.x, L.wx, L.wh, L.b, dh)
    say("step path", shape)
    x, Ld = dev(inst.x), layer_dev(L)
    P.pyramid_lstm_timing_enable(True)
    h_inf, _ = layer_forward(x, Ld)
    h, saved = layer_forward(x, Ld, training=True)
    dx, dwx, dwh, db = layer_backward(x, Ld, saved, dev(dh))
    phases = P.pyramid_lstm_timing_read()
    P.pyramid_lstm_timing_enable(False)
    torch.cuda.synchronize()
    assert "sweep_fwd_step" in phases and "sweep_bwd_step" in phases, phases
    assert "sweep_fwd_mfma" not in phases and "sweep_fwd_generic" not in phases, phases
    assert normwise(host(h_inf), ref_h) <= TOL["f32"]
    assert torch.equal(h_inf, h)
    for name, got in (("dx", dx), ("dwx", dwx), ("dwh", dwh), ("db", db)):
        err = normwise(host(got), ref[name])
        assert err <= TOL["f32"], (name, err)


@pytest.mark.parametrize("staged", [1, 0], ids=["lds", "streamed"])
@pytest.mark.parametrize("shape", [(2, 9, 17, 40, 32, 32), (1, 6, 5, 4, 20, 16),
                                   (1, 5, 12, 70, 8, 32), (1, 3, 21, 5, 4, 16)],
                         ids=lambda s: "x".join(map(str, s)))
def test_step_weight_gradients_both_kernels(shape, staged, step_path):
    """The plane-step weight gradients from the LDS-staged GEMM (several
    N-parts and voxel chunks, ragged 16-voxel units, batch > 1) and from the
    register-streamed kernel, against the oracle."""
    inst = instance(shape, 4500 + sum(shape))
    L = inst.layers[0]
    dh = synth.upstream_grad(inst.x.shape[:-1] + (shape[-1],), 17 + sum(shape))
    ref = oracle.backward(inst.x, L.wx, L.wh, L.b, dh)
    say("wgrad kernels", shape, staged)
    P.pyramid_lstm_set_wgrad_staged(staged)
    try:
        x, Ld = dev(inst.x), layer_dev(L)
        h, saved = layer_forward(x, Ld, training=True)
        dx, dwx, dwh, db = layer_backward(x, Ld, saved, dev(dh))
        torch.cuda.synchronize()
    finally:
        P.pyramid_lstm_set_wgrad_staged(1)
    for name, got in (("dx", dx), ("dwx", dwx), ("dwh", dwh), ("db", db)):
        err = normwise(host(got), ref[name])
        assert err <= TOL["f32"], (name, err)


@pytest.mark.parametrize("shape", [(1, 5, 37, 29, 3, 16), (1, 4, 6, 70, 3, 64)],
                         ids=lambda s: "x".join(map(str, s)))
def test_step_path_saved_state_matches_oracle(shape, step_path):
    """Gates, c^d and h^d that the plane-step forward saves for the backward."""
    inst = instance(shape, 5000 + sum(shape))
    L = inst.layers[0]
    ref = oracle.forward(inst.x, L.wx, L.wh, L.b, want_hd=True, want_saved=True)
    say("step path saved", shape)
    h, saved = layer_forward(dev(inst.x), layer_dev(L), training=True)
    torch.cuda.synchronize()
    assert normwise(host(h), ref["h"]) <= TOL["f32"]
    for name in ("hd", "cell", "gates"):
        got = saved_view(saved, name, shape)
        assert normwise(got, ref[name]) <= TOL["f32"], name


def test_large_hidden_layers_take_the_step_path():
    """O = 32 and 64 run on the plane-step MFMA kernels by default."""
    for shape in [(1, 4, 9, 10, 32, 32), (1, 3, 8, 7, 64, 64)]:
        inst = instance(shape, 6000 + sum(shape))
        say("step path default", shape)
        x, Ld = dev(inst.x), layer_dev(inst.layers[0])
        P.pyramid_lstm_timing_enable(True)
        h, saved = layer_forward(x, Ld, training=True)
        layer_backward(x, Ld, saved, torch.ones_like(h))
        phases = P.pyramid_lstm_timing_read()
        P.pyramid_lstm_timing_enable(False)
        for k in ("sweep_fwd_step", "sweep_bwd_step", "wgrad_step", "dx_step"):
            assert k in phases, (shape, phases)
        assert "sweep_fwd_generic" not in phases and "sweep_bwd_generic" not in phases


def instance_k(shape, K, seed, dtype="f32"):
    N, D, H, W, C, O = shape
    wl = synth.Workload("t", N, D, H, W, C, [O], dtype=dtype, seed=seed, K=K)
    return synth.make(wl)


# K x K filters (Section 3 uses 7 x 7): every unit count, channel counts of
# the paper's network (5, 25, 45), K = 1, a plane smaller than the filter
K_CASES = [((1, 5, 17, 13, 3, 16), 5), ((1, 4, 11, 9, 25, 32), 7), ((2, 3, 8, 12, 5, 16), 7),
           ((1, 6, 9, 10, 2, 16), 1), ((1, 3, 9, 8, 45, 64), 7), ((1, 2, 3, 9, 4, 32), 7)]


@pytest.mark.parametrize("case", K_CASES, ids=lambda c: "x".join(map(str, c[0])) + "_k%d" % c[1])
def test_filter_size_matches_oracle(case, step_split):
    shape, K = case
    inst = instance_k(shape, K, 7000 + sum(shape) + K)
    L = inst.layers[0]
    dh = synth.upstream_grad(inst.x.shape[:-1] + (shape[-1],), 13 + sum(shape))
    ref_h = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    ref = oracle.backward(inst.x, L.wx, L.wh, L.b, dh)
    say("filter size", shape, K)
    x, Ld = dev(inst.x), layer_dev(L)
    assert Ld.K == K
    P.pyramid_lstm_timing_enable(True)
    h_inf, _ = layer_forward(x, Ld)
    h, saved = layer_forward(x, Ld, training=True)
    dx, dwx, dwh, db = layer_backward(x, Ld, saved, dev(dh))
    phases = P.pyramid_lstm_timing_read()
    P.pyramid_lstm_timing_enable(False)
    torch.cuda.synchronize()
    if K != 3:
        assert "sweep_fwd_step" in phases and "sweep_bwd_step" in phases, phases
    assert normwise(host(h_inf), ref_h) <= TOL["f32"]
    assert normwise(host(h), ref_h) <= TOL["f32"]
    for name, got in (("dx", dx), ("dwx", dwx), ("dwh", dwh), ("db", db)):
        err = normwise(host(got), ref[name])
        assert err <= TOL["f32"], (name, err)


@pytest.mark.parametrize("case", [((1, 5, 9, 7, 3, 16), 5), ((1, 3, 6, 5, 2, 8), 7)],
                         ids=lambda c: "x".join(map(str, c[0])) + "_k%d" % c[1])
def test_filter_size_generic_path(case):
    """The generic per-plane kernels with K x K filters (forced)."""
    shape, K = case
    inst = instance_k(shape, K, 7100 + sum(shape) + K)
    L = inst.layers[0]
    dh = synth.upstream_grad(inst.x.shape[:-1] + (shape[-1],), 17 + sum(shape))
    ref_h = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    ref = oracle.backward(inst.x, L.wx, L.wh, L.b, dh)
    say("filter size generic", shape, K)
    P.pyramid_lstm_set_forward_path(1)
    P.pyramid_lstm_set_backward_path(1)
    try:
        x, Ld = dev(inst.x), layer_dev(L)
        h, saved = layer_forward(x, Ld, training=True)
        grads = layer_backward(x, Ld, saved, dev(dh))
        torch.cuda.synchronize()
    finally:
        P.pyramid_lstm_set_forward_path(0)
        P.pyramid_lstm_set_backward_path(0)
    assert normwise(host(h), ref_h) <= TOL["f32"]
    for name, got in zip(("dx", "dwx", "dwh", "db"), grads):
        assert normwise(host(got), ref[name]) <= TOL["f32"], name


# bf16 K x K cases: 32 units with 7 x 7; 64 units with 5 x 5 at 20 input
# channels (the 256-pixel kernel) and at 40 (its LDS does not fit: the
# default falls back to 64-pixel blocks); 1 x 1 filters, whose steps have
# two or three K-groups (one on the first plane)
BF16_K_CASES = [((1, 4, 11, 9, 25, 32), 7), ((2, 3, 19, 35, 20, 64), 5),
                ((1, 3, 21, 18, 40, 64), 5), ((1, 5, 17, 20, 7, 32), 1),
                ((2, 3, 9, 33, 30, 64), 1),
                # 16 units, packed taps: 16 x 16 pixel blocks with ragged
                # edges, every filter size, one to eight input channels
                ((2, 5, 19, 35, 3, 16), 3), ((1, 4, 11, 9, 8, 16), 7),
                ((1, 3, 21, 18, 5, 16), 5), ((1, 5, 17, 20, 1, 16), 1),
                ((1, 2, 3, 9, 4, 16), 7)]


@pytest.mark.parametrize("case", BF16_K_CASES,
                         ids=lambda c: "x".join(map(str, c[0])) + "_k%d" % c[1])
@pytest.mark.parametrize("bf16_mfma", [1, 3, 2, 0, 5],
                         ids=["bf16_mt", "bf16_lds", "bf16_l1", "fp32_mfma", "bf16_proj"])
def test_filter_size_bf16(bf16_mfma, case):
    shape, K = case
    inst = instance_k(shape, K, 7200 + sum(shape), "bf16")
    L = inst.layers[0]
    ref = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    say("filter size bf16", shape, K, bf16_mfma)
    P.pyramid_lstm_set_bf16_mfma(bf16_mfma)
    try:
        h, _ = layer_forward(dev(inst.x, "bf16"), layer_dev(L, "bf16"))
        torch.cuda.synchronize()
    finally:
        P.pyramid_lstm_set_bf16_mfma(1)
    assert normwise(host(h), ref) <= TOL["bf16"]


@pytest.mark.parametrize("shape", O16_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("bwd_path", [0, 2], ids=["resident", "chunked"])
def test_reverse_sweep_strip_kinds_match_oracle(shape, bwd_path):
    """The persistent reverse sweep with strips kept whole in LDS where they
    fit (default) and with every strip staged chunk by chunk: same gradients
    as the oracle."""
    inst = instance(shape, 1400 + sum(shape))
    L = inst.layers[0]
    dh = synth.upstream_grad(inst.x.shape[:-1] + (shape[-1],), 19 + sum(shape))
    ref = oracle.backward(inst.x, L.wx, L.wh, L.b, dh)
    say("reverse sweep", shape, bwd_path)
    x, Ld = dev(inst.x), layer_dev(L)
    h, saved = layer_forward(x, Ld, training=True)
    P.pyramid_lstm_set_backward_path(bwd_path)
    P.pyramid_lstm_timing_enable(True)
    try:
        grads = layer_backward(x, Ld, saved, dev(dh))
        phases = P.pyramid_lstm_timing_read()
        torch.cuda.synchronize()
    finally:
        P.pyramid_lstm_timing_enable(False)
        P.pyramid_lstm_set_backward_path(0)
    assert "sweep_bwd_mfma" in phases, phases
    for name, got in zip(("dx", "dwx", "dwh", "db"), grads):
        assert normwise(host(got), ref[name]) <= TOL["f32"], name


@pytest.mark.parametrize("shape", [(1, 5, 37, 29, 3, 16), (2, 9, 20, 18, 1, 16)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("bf16_mfma", [1, 3], ids=["packed_step", "persistent"])
def test_bf16_o16_forward_paths(shape, bf16_mfma):
    """bf16 storage with 16 units and C <= 8: by default the bf16 plane steps
    with packed taps run (h^d rounded to bf16 for the recurrence and the
    sum); with the 256-pixel blocks off the inputs are widened to fp32 and
    the persistent sweep runs, the output being the bf16-rounded sum."""
    inst = instance(shape, 1500 + sum(shape), "bf16")
    L = inst.layers[0]
    ref = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    say("bf16 o16", shape, bf16_mfma)
    P.pyramid_lstm_set_bf16_mfma(bf16_mfma)
    P.pyramid_lstm_timing_enable(True)
    try:
        h, _ = layer_forward(dev(inst.x, "bf16"), layer_dev(L, "bf16"))
        phases = P.pyramid_lstm_timing_read()
    finally:
        P.pyramid_lstm_timing_enable(False)
        P.pyramid_lstm_set_bf16_mfma(1)
    torch.cuda.synchronize()
    assert h.dtype == torch.bfloat16
    if bf16_mfma == 1:
        assert "sweep_fwd_step_bf16" in phases and "sweep_fwd_mfma" not in phases, phases
        assert normwise(host(h), ref) <= TOL["bf16"]
    else:
        assert "sweep_fwd_mfma" in phases and "sweep_fwd_step" not in phases, phases
        # fp32 arithmetic: only the final rounding to bf16 separates it from the oracle
        assert normwise(host(h), ref) <= 4e-3


@pytest.mark.parametrize("shape", [(2, 6, 20, 34, 3, 16), (1, 4, 18, 16, 8, 16),
                                   (1, 2, 33, 18, 1, 16), (3, 8, 8, 8, 3, 16)],
                         ids=lambda s: "x".join(map(str, s)))
def test_bf16_o16_two_planes_per_launch(shape):
    """16-unit bf16 layers with 3 x 3 filters and an even number of planes in
    every direction run two planes per launch (each block also computes the
    one-pixel ring of its first plane): the same h bit for bit as one plane
    per launch, and the oracle's within the bf16 bound; ragged 16 x 16
    blocks, a single launch pair (D = 2), planes smaller than a block."""
    inst = instance(shape, 1600 + sum(shape), "bf16")
    L = inst.layers[0]
    ref = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    say("bf16 o16 two planes", shape)
    x, Ld = dev(inst.x, "bf16"), layer_dev(L, "bf16")
    out = {}
    for knob in (1, 4):
        P.pyramid_lstm_set_bf16_mfma(knob)
        try:
            out[knob], _ = layer_forward(x, Ld)
            torch.cuda.synchronize()
        finally:
            P.pyramid_lstm_set_bf16_mfma(1)
    assert torch.equal(out[1], out[4])
    assert normwise(host(out[1]), ref) <= TOL["bf16"]


def test_mfma_backward_runs_for_o16():
    """The persistent MFMA reverse sweep and MFMA parameter gradients are the
    path taken for 16 hidden units."""
    inst = instance((1, 12, 40, 36, 3, 16), 77)
    L = inst.layers[0]
    x, Ld = dev(inst.x), layer_dev(L)
    say("mfma backward path")
    h, saved = layer_forward(x, Ld, training=True)
    P.pyramid_lstm_timing_enable(True)
    layer_backward(x, Ld, saved, torch.ones_like(h))
    phases = P.pyramid_lstm_timing_read()
    P.pyramid_lstm_timing_enable(False)
    assert phases.get("sweep_bwd_mfma", (0, 0))[1] == 1, phases
    assert "wgrad_mfma" in phases and "sweep_bwd_generic" not in phases


@pytest.mark.parametrize("cfg", [2, 3])
def test_mfma_sweep_runs_for_the_o16_workloads(cfg):
    """The persistent MFMA sweep (one launch) is the path taken for the
    16-hidden-unit fp32 workloads, not the generic fallback."""
    inst = synth.config(cfg)
    say("mfma path", cfg)
    P.pyramid_lstm_timing_enable(True)
    layer_forward(dev(inst.x), layer_dev(inst.layers[0]))
    phases = P.pyramid_lstm_timing_read()
    P.pyramid_lstm_timing_enable(False)
    assert phases.get("sweep_fwd_mfma", (0, 0))[1] == 1, phases
    assert "sweep_fwd_generic" not in phases


@pytest.mark.parametrize("shape", [SHAPES[0], SHAPES[1], SHAPES[2], SHAPES[4], SHAPES[8]],
                         ids=lambda s: "x".join(map(str, s)))
def test_forward_bf16_matches_oracle(shape):
    inst = instance(shape, 2000 + sum(shape), "bf16")
    L = inst.layers[0]
    ref = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    say("forward bf16", shape)
    h, _ = layer_forward(dev(inst.x, "bf16"), layer_dev(L, "bf16"))
    torch.cuda.synchronize()
    assert h.dtype == torch.bfloat16
    err = normwise(host(h), ref)
    assert err <= TOL["bf16"], err


@pytest.mark.parametrize("bf16_mfma", [1, 3, 2, 0],
                         ids=["bf16_mt", "bf16_lds", "bf16_l1", "fp32_mfma"])
@pytest.mark.parametrize("shape", [(1, 4, 6, 70, 3, 64), (2, 9, 17, 40, 32, 32),
                                   (1, 5, 23, 9, 40, 32), (2, 3, 7, 66, 64, 64)],
                         ids=lambda s: "x".join(map(str, s)))
def test_forward_bf16_large_hidden_matches_oracle(shape, bf16_mfma, step_split):
    """bf16 storage with 32 or 64 hidden units: the bf16-MFMA forward step
    (and the fp32-MFMA one), both launch shapes, channel counts below, at
    and between 32-channel blocks."""
    inst = instance(shape, 2500 + sum(shape), "bf16")
    L = inst.layers[0]
    ref = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    say("forward bf16 large hidden", shape, bf16_mfma)
    P.pyramid_lstm_set_bf16_mfma(bf16_mfma)
    try:
        P.pyramid_lstm_timing_enable(True)
        h, _ = layer_forward(dev(inst.x, "bf16"), layer_dev(L, "bf16"))
        torch.cuda.synchronize()
        phases = P.pyramid_lstm_timing_read()
        P.pyramid_lstm_timing_enable(False)
    finally:
        P.pyramid_lstm_set_bf16_mfma(1)
    assert ("sweep_fwd_step_bf16" in phases) == bool(bf16_mfma), phases
    err = normwise(host(h), ref)
    assert err <= TOL["bf16"], err


@pytest.mark.parametrize("shape", SHAPES + [(3, 6, 20, 18, 2, 16), (1, 7, 130, 90, 1, 16)],
                         ids=lambda s: "x".join(map(str, s)))
def test_training_forward_and_backward_match_oracle(shape):
    inst = instance(shape, 3000 + sum(shape))
    L = inst.layers[0]
    dh = synth.upstream_grad(inst.x.shape[:-1] + (shape[-1],), 7 + sum(shape))
    ref_h = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    ref = oracle.backward(inst.x, L.wx, L.wh, L.b, dh)
    say("backward", shape)
    x, Ld = dev(inst.x), layer_dev(L)
    h, saved = layer_forward(x, Ld, training=True)
    dx, dwx, dwh, db = layer_backward(x, Ld, saved, dev(dh))
    torch.cuda.synchronize()
    assert normwise(host(h), ref_h) <= TOL["f32"]
    for name, got in (("dx", dx), ("dwx", dwx), ("dwh", dwh), ("db", db)):
        err = normwise(host(got), ref[name])
        assert err <= TOL["f32"], (name, err)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_config_forward(cfg):
    """Configs 1-3 at full size, every element of h against the oracle run
    in the test on the host's cores (config 3 takes about a minute there).
    Prints the largest elementwise error and where it is."""
    inst = synth.config(cfg)
    L = inst.layers[0]
    say("config", cfg)
    h, _ = layer_forward(dev(inst.x), layer_dev(L))
    torch.cuda.synchronize()
    got = host(h)
    del h
    say("config oracle", cfg, "threads", oracle.threads())
    t0 = time.time()
    ref = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    err = np.abs(got - ref)
    worst = np.unravel_index(int(np.argmax(err)), err.shape)
    scale = float(np.abs(ref).max())
    print("[config %d] oracle %.1f s; max|h| %.4f, max err %.3e at %s (normwise %.3e), "
          "mean err %.3e" % (cfg, time.time() - t0, scale, err[worst], worst, err[worst] / scale,
                             err.mean()), flush=True)
    assert err[worst] / scale <= TOL["f32"]


def test_zero_parameters_exact_zero():
    """All-zero parameters give h = 0 exactly (sigma(0) = 1/2, tanh(0) = 0)."""
    inst = instance((1, 6, 10, 12, 3, 16), 11)
    L = inst.layers[0]
    Lz = LayerW(*(torch.zeros_like(t) for t in layer_dev(L).__dict__.values()))
    say("zero parameters")
    h, _ = layer_forward(dev(inst.x), Lz)
    torch.cuda.synchronize()
    assert torch.count_nonzero(h).item() == 0


@pytest.mark.parametrize("d", range(6))
def test_dependency_cone_on_gpu(d):
    """Only direction d active: perturbing one input voxel leaves every output
    outside its pyramid bitwise unchanged.  Inside, the change decays along the
    sweep (at the cone's edge it passes only through corner taps and can drop
    below fp32 resolution), so every voxel within one plane of the source must
    change."""
    N, D, H, W, C, O = 1, 7, 9, 11, 1, 16
    inst = instance((N, D, H, W, C, O), 40 + d)
    L = inst.layers[0]
    keep = np.zeros(6)
    keep[d] = 1
    Ld = LayerW(dev(L.wx * keep[:, None, None, None, None]),
                dev(L.wh * keep[:, None, None, None, None]), dev(L.b * keep[:, None]))
    src = (3, 4, 5)
    x2 = inst.x.copy()
    x2[0][src] += 1.0
    say("cone", d)
    h1, _ = layer_forward(dev(inst.x), Ld)
    h2, _ = layer_forward(dev(x2), Ld)
    torch.cuda.synchronize()
    changed = np.any(host(h1)[0] != host(h2)[0], axis=-1)
    a, sign = d // 2, (1 if d % 2 == 0 else -1)
    inplane = [ax for ax in range(3) if ax != a]
    idx = np.indices((D, H, W))
    dt = sign * (idx[a] - src[a])
    cheb = np.maximum(abs(idx[inplane[0]] - src[inplane[0]]),
                      abs(idx[inplane[1]] - src[inplane[1]]))
    cone = (dt >= 0) & (cheb <= 1 + dt)
    assert not np.any(changed & ~cone)
    assert np.all(changed[cone & (dt <= 1)])


@pytest.mark.parametrize("axis", [0, 1, 2])
def test_mirror_swaps_plus_minus_on_gpu(axis):
    """Same parameters for both directions of an axis: mirroring the input
    along that axis mirrors the layer output, bitwise."""
    inst = instance((1, 6, 9, 13, 2, 16), 50 + axis)
    L = inst.layers[0]
    wx, wh, b = L.wx.copy(), L.wh.copy(), L.b.copy()
    dp, dm = 2 * axis, 2 * axis + 1
    wx[dm], wh[dm], b[dm] = wx[dp], wh[dp], b[dp]
    for d in range(6):               # other axes off
        if d // 2 != axis:
            wx[d], wh[d], b[d] = 0, 0, 0
    Ld = LayerW(dev(wx), dev(wh), dev(b))
    say("mirror", axis)
    h1, _ = layer_forward(dev(inst.x), Ld)
    h2, _ = layer_forward(dev(np.flip(inst.x, axis=axis + 1).copy()), Ld)
    torch.cuda.synchronize()
    a, m = host(h1), np.flip(host(h2), axis=axis + 1)
    # h = h^{a+} + h^{a-}; mirroring swaps the two terms, and fp32 addition
    # commutes exactly
    assert np.array_equal(a, m)


def test_repeat_runs_bitwise_identical():
    inst = instance((1, 10, 48, 40, 3, 16), 60)
    L = inst.layers[0]
    x, Ld = dev(inst.x), layer_dev(L)
    say("determinism")
    outs = [layer_forward(x, Ld)[0].clone() for _ in range(3)]
    dh = dev(synth.upstream_grad(tuple(outs[0].shape), 61))
    grads = []
    for _ in range(2):
        h, saved = layer_forward(x, Ld, training=True)
        grads.append([t.clone() for t in layer_backward(x, Ld, saved, dh)])
    torch.cuda.synchronize()
    assert all(torch.equal(outs[0], o) for o in outs[1:])
    assert all(torch.equal(a, b) for a, b in zip(grads[0], grads[1]))


def test_wait_that_gives_up_is_reported():
    """A persistent sweep whose bounded wait gives up cannot return an error
    code (the call has returned): its outputs become NaN and the device's
    sticky status reports it.  The test mode makes every wait expect a step
    that is never published, so each launch takes that path and still ends
    normally; afterwards the status clears and results are right again."""
    shape = (1, 12, 64, 50, 1, 16)          # 7-50 strips per direction in both sweeps
    inst = instance(shape, 77)
    L = inst.layers[0]
    x, Ld = dev(inst.x), layer_dev(L)
    dh = dev(synth.upstream_grad(shape[:4] + (16,), 78))
    say("wait failure path: clean run")
    P.pyramid_lstm_device_status(clear=True)
    h_ok, _ = layer_forward(x, Ld)
    assert P.pyramid_lstm_device_status() == 0
    say("wait failure path: test mode")
    P.pyramid_lstm_set_wait_test(True)
    try:
        h_bad, saved = layer_forward(x, Ld, training=True)
        torch.cuda.synchronize()
        st_fwd = P.pyramid_lstm_device_status(clear=True)
        grads = layer_backward(x, Ld, saved, dh)
        torch.cuda.synchronize()
        st_bwd = P.pyramid_lstm_device_status(clear=True)
    finally:
        P.pyramid_lstm_set_wait_test(False)
    assert st_fwd == P.PLSTM_DEVICE_WAIT_GAVE_UP
    assert st_bwd == P.PLSTM_DEVICE_WAIT_GAVE_UP
    assert torch.isnan(h_bad).all()
    for g in grads:
        assert torch.isnan(g).all()
    say("wait failure path: clean again")
    assert P.pyramid_lstm_device_status() == 0
    h2, saved2 = layer_forward(x, Ld, training=True)
    grads2 = layer_backward(x, Ld, saved2, dh)
    torch.cuda.synchronize()
    assert P.pyramid_lstm_device_status() == 0
    assert torch.equal(h2, h_ok)
    ref = oracle.backward(inst.x, L.wx, L.wh, L.b, host(dh))
    for name, got in zip(("dx", "dwx", "dwh", "db"), grads2):
        assert normwise(host(got), ref[name]) <= TOL["f32"], name
