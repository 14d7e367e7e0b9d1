"""GPU parity of the stacked networks (configs 4 and 5, and small versions of
them checked against the oracle directly), through the C ABI."""
from __future__ import annotations

import os

import numpy as np
import pytest
import torch

import oracle
import oracle.network as onet
import synth
from paper_1506_07452_amd.network import network_forward, network_train_step
from tests.gpu_util import DEV, TOL, dev, host, layer_dev, normwise, say

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def to_device(inst, dtype):
    layers = [layer_dev(L, dtype) for L in inst.layers]
    fcs = [(dev(w, dtype), dev(b, dtype)) for w, b in inst.fcs]
    head = (dev(inst.head[0], dtype), dev(inst.head[1], dtype))
    labels = None
    if inst.labels is not None:
        labels = torch.from_numpy(inst.labels).to(DEV)
    return dev(inst.x, dtype), layers, fcs, head, labels


def oracle_args(inst):
    return ([(L.wx, L.wh, L.b) for L in inst.layers], inst.fcs, inst.head)


def small(wl_kw, seed):
    wl = synth.Workload("small", seed=seed, **wl_kw)
    return synth.make(wl)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_small_network_forward(dtype):
    inst = small(dict(N=2, D=6, H=10, W=9, C=3, hidden=[16, 32], dtype=dtype, fc=True,
                      classes=4), 70)
    ref = onet.forward(inst.x, *oracle_args(inst))["p"]
    say("small network forward", dtype)
    x, layers, fcs, head, _ = to_device(inst, dtype)
    out = network_forward(x, layers, fcs, head)
    torch.cuda.synchronize()
    assert normwise(host(out["p"]), ref) <= TOL[dtype]


@pytest.mark.parametrize("fused", [True, False], ids=["fused_head", "separate_head"])
def test_small_network_training_step(fused):
    inst = small(dict(N=1, D=5, H=12, W=7, C=3, hidden=[16, 32], fc=True, classes=4,
                      labels=True), 80)
    ref = onet.backward(inst.x, *oracle_args(inst), inst.labels)
    say("small network training step", fused)
    x, layers, fcs, head, labels = to_device(inst, "f32")
    g = network_train_step(x, layers, fcs, head, labels, fused_head=fused)
    torch.cuda.synchronize()
    assert abs(g["loss"].item() - ref["loss"]) <= TOL["f32"] * abs(ref["loss"])
    pairs = [(g["head"][0], ref["head"][0]), (g["head"][1], ref["head"][1])]
    for li in range(2):
        pairs += list(zip(g["fcs"][li], ref["fcs"][li]))
        pairs += list(zip(g["layers"][li], ref["layers"][li]))
    for got, want in pairs:
        assert normwise(host(got), want) <= TOL["f32"]


def paper_small(seed, dtype="f32"):
    """The network of Section 3 ("Experimental Setup") on a small volume: 7 x 7
    filters, PyraMiD 16 -> FC tanh 25 -> PyraMiD 32 -> FC tanh 45 ->
    PyraMiD 64 -> output layer (5 classes), 5 input channels."""
    wl = synth.Workload("paper small", 1, 3, 9, 8, 5, [16, 32, 64], dtype=dtype, classes=5,
                        labels=dtype == "f32", K=7, fc_widths=[25, 45], seed=seed)
    return synth.make(wl)


def test_paper_network_training_step():
    inst = paper_small(95)
    ref = onet.backward(inst.x, *oracle_args(inst), inst.labels)
    say("paper network training step")
    x, layers, fcs, head, labels = to_device(inst, "f32")
    g = network_train_step(x, layers, fcs, head, labels)
    torch.cuda.synchronize()
    assert abs(g["loss"].item() - ref["loss"]) <= TOL["f32"] * abs(ref["loss"])
    assert normwise(host(g["p"]), ref["p"]) <= TOL["f32"]
    pairs = [(g["head"][0], ref["head"][0]), (g["head"][1], ref["head"][1])]
    for li in range(2):
        pairs += list(zip(g["fcs"][li], ref["fcs"][li]))
    for li in range(3):
        pairs += list(zip(g["layers"][li], ref["layers"][li]))
    for got, want in pairs:
        assert normwise(host(got), want) <= TOL["f32"]


def test_paper_network_forward_bf16():
    inst = paper_small(96, "bf16")
    ref = onet.forward(inst.x, *oracle_args(inst))["p"]
    say("paper network forward bf16")
    x, layers, fcs, head, _ = to_device(inst, "bf16")
    out = network_forward(x, layers, fcs, head)
    torch.cuda.synchronize()
    assert normwise(host(out["p"]), ref) <= TOL["bf16"]


# input widths of the four softmax kernels: multiples of 4 from 64 (16 lanes
# per row), smaller multiples of 4 (a row per thread, read as vectors), other
# widths up to 128 (rows staged in LDS), wider ones
SOFTMAX_CIN = [(16, "vec"), (64, "coop64"), (128, "coop128"), (200, "coop200"), (18, "rows"),
               (203, "wide")]


@pytest.mark.parametrize("cin", [c for c, _ in SOFTMAX_CIN], ids=[n for _, n in SOFTMAX_CIN])
def test_softmax_squared_loss_matches_oracle(cin):
    """The squared loss of Eq. (14) on the softmax output, and its gradient,
    on every softmax kernel."""
    import oracle.loss as oloss
    import paper_1506_07452_amd as P
    rng = np.random.default_rng(93 + cin)
    M, K = 1037, 5
    xa = rng.standard_normal((M, cin)).astype(np.float32)
    w = rng.uniform(-0.3, 0.3, (K, cin)).astype(np.float32)
    b = rng.uniform(-0.3, 0.3, K).astype(np.float32)
    lab = rng.integers(0, K, M).astype(np.int32)
    say("softmax squared loss", cin)
    p = torch.empty(M, K, device=DEV)
    loss = torch.empty(1, device=DEV)
    dx, dw, db = (torch.empty(M, cin, device=DEV), torch.empty(K, cin, device=DEV),
                  torch.empty(K, device=DEV))
    P.pyramid_softmax_sq(dev(xa), dev(w), dev(b), p, torch.from_numpy(lab).to(DEV), loss, dx,
                         dw, db)
    torch.cuda.synchronize()
    ref = oloss.softmax_sq(xa, w, b, lab, grad=True)
    assert normwise(host(p), ref["p"]) <= TOL["f32"]
    assert abs(loss.item() - ref["loss"]) <= TOL["f32"] * ref["loss"]
    for got, want in ((dx, ref["dx"]), (dw, ref["dw"]), (db, ref["db"])):
        assert normwise(host(got), want) <= TOL["f32"]


def test_paper_network_training_step_squared_loss():
    """The paper's network trained as in Section 3: squared loss, every
    gradient against the oracle."""
    inst = paper_small(99)
    ref = onet.backward(inst.x, *oracle_args(inst), inst.labels, loss="sq")
    say("paper network squared loss")
    x, layers, fcs, head, labels = to_device(inst, "f32")
    g = network_train_step(x, layers, fcs, head, labels, loss="sq")
    torch.cuda.synchronize()
    assert abs(g["loss"].item() - ref["loss"]) <= TOL["f32"] * abs(ref["loss"])
    pairs = [(g["head"][0], ref["head"][0]), (g["head"][1], ref["head"][1])]
    for li in range(2):
        pairs += list(zip(g["fcs"][li], ref["fcs"][li]))
    for li in range(3):
        pairs += list(zip(g["layers"][li], ref["layers"][li]))
    for got, want in pairs:
        assert normwise(host(got), want) <= TOL["f32"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_crop_is_the_subvolume(dtype):
    import paper_1506_07452_amd as P
    rng = np.random.default_rng(101)
    xa = rng.standard_normal((2, 5, 9, 7, 3))
    x = dev(xa, dtype)
    box = (1, 2, 3, 3, 6, 4)
    say("crop", dtype)
    tile = torch.empty((1, 3, 6, 4, 3), dtype=x.dtype, device=DEV)
    P.pyramid_crop(x, 1, box, tile)
    torch.cuda.synchronize()
    want = host(x)[1, 1:4, 2:8, 3:7]
    assert np.array_equal(host(tile)[0], want)


def test_stitched_inference_matches_oracle():
    """A volume run as overlapping sub-volumes and stitched with Gaussian
    weights (Section 3) against the oracle doing the same with its own
    network.  Both sides get the same hand-written tile origins (ragged
    overlaps, the last tile flush with each far end); the stride grids of
    the two sides are pinned separately on the CPU."""
    import oracle.stitch as ostitch
    from paper_1506_07452_amd.network import network_infer_volume
    inst = small(dict(N=1, D=6, H=20, W=18, C=3, hidden=[16, 32], fc=True, classes=4), 102)
    tile = (4, 12, 10)
    origins = ([0, 2], [0, 5, 8], [0, 8])
    lw, fw, hw = oracle_args(inst)

    def tile_fn(z0, y0, x0, d, h, w):
        xs = inst.x[:, z0:z0 + d, y0:y0 + h, x0:x0 + w]
        return onet.forward(xs, lw, fw, hw)["p"].reshape(d, h, w, -1)

    ref = ostitch.stitch((6, 20, 18), tile, None, tile_fn, 4, origins=origins)
    say("stitched inference")
    x, layers, fcs, head, _ = to_device(inst, "f32")
    p = network_infer_volume(x, layers, fcs, head, tile, origins=origins)
    p_grid = network_infer_volume(x, layers, fcs, head, tile, (2, 8, 8))
    torch.cuda.synchronize()
    assert normwise(host(p)[0], ref) <= TOL["f32"]
    assert np.allclose(host(p).sum(-1), 1.0, atol=1e-5)
    # the stride grid (2, 8, 8) lays tiles at z (0, 2), y (0, 8), x (0, 8)
    ref_grid = ostitch.stitch((6, 20, 18), tile, None, tile_fn, 4,
                              origins=([0, 2], [0, 8], [0, 8]))
    assert normwise(host(p_grid)[0], ref_grid) <= TOL["f32"]


def test_single_tile_stitch_is_the_network_output():
    from paper_1506_07452_amd.network import network_infer_volume
    inst = small(dict(N=2, D=4, H=9, W=8, C=3, hidden=[16], fc=True, classes=3), 103)
    say("single tile stitch")
    x, layers, fcs, head, _ = to_device(inst, "f32")
    p = network_infer_volume(x, layers, fcs, head, (4, 9, 8), (4, 9, 8))
    q = network_forward(x, layers, fcs, head)["p"].view(p.shape)
    torch.cuda.synchronize()
    assert normwise(host(p), host(q)) <= 1e-6


def test_rmsprop_matches_oracle():
    """Three RMS-prop updates (Section 3, Eq. (15)-(18)) of four tensors of
    ragged sizes in one launch each, against the fp64 oracle fed the same
    fp32 gradients."""
    import oracle.optim as optim
    import paper_1506_07452_amd as P
    rng = np.random.default_rng(97)
    sizes = [1, 1000, 4097, 3 * 64 * 64]
    th = [rng.uniform(-0.1, 0.1, n).astype(np.float32) for n in sizes]
    ref = [(t.astype(np.float64), np.zeros(n), np.zeros(n)) for t, n in zip(th, sizes)]
    params = [dev(t) for t in th]
    ms = [torch.zeros(n, device=DEV) for n in sizes]
    mom = [torch.zeros(n, device=DEV) for n in sizes]
    say("rmsprop")
    for epoch in range(3):
        grads = [(rng.standard_normal(n) * 10.0 ** rng.integers(-4, 2, n)).astype(np.float32)
                 for n in sizes]
        lr = optim.learning_rate(epoch)
        P.pyramid_rmsprop_step(params, [dev(g) for g in grads], ms, mom, lr)
        ref = [optim.rmsprop_step(t, g, a, m, lr) for (t, a, m), g in zip(ref, grads)]
    torch.cuda.synchronize()
    for k in range(len(sizes)):
        assert normwise(host(params[k]), ref[k][0]) <= 1e-6
        assert normwise(host(ms[k]), ref[k][1]) <= 1e-6
        assert normwise(host(mom[k]), ref[k][2]) <= 1e-5


def test_paper_network_training_reduces_loss():
    """A few full training iterations of the paper's network (train step +
    RMS-prop update with the decaying rate) on one fixed small batch: the
    loss goes down."""
    from paper_1506_07452_amd import RMSprop
    from paper_1506_07452_amd.network import network_gradients, network_parameters
    inst = paper_small(98)
    say("paper network training iterations")
    x, layers, fcs, head, labels = to_device(inst, "f32")
    opt = RMSprop(network_parameters(layers, fcs, head))
    losses = []
    for epoch in range(6):
        g = network_train_step(x, layers, fcs, head, labels)
        losses.append(g["loss"].item())
        opt.step(network_gradients(g), epoch)
    torch.cuda.synchronize()
    assert losses[-1] < 0.9 * losses[0], losses


def test_fc_and_softmax_match_oracle():
    rng = np.random.default_rng(90)
    M, Cin, Cout, K = 1000, 16, 32, 4
    xa = rng.standard_normal((M, Cin)).astype(np.float32)
    w1 = rng.uniform(-0.3, 0.3, (Cout, Cin)).astype(np.float32)
    b1 = rng.uniform(-0.3, 0.3, Cout).astype(np.float32)
    w2 = rng.uniform(-0.3, 0.3, (K, Cout)).astype(np.float32)
    b2 = rng.uniform(-0.3, 0.3, K).astype(np.float32)
    lab = rng.integers(0, K, M).astype(np.int32)
    dy = rng.standard_normal((M, Cout)).astype(np.float32)
    import paper_1506_07452_amd as P
    y = torch.empty(M, Cout, device=DEV)
    P.pyramid_fc_tanh_forward(dev(xa), dev(w1), dev(b1), y)
    dx, dw, db = (torch.empty(M, Cin, device=DEV), torch.empty(Cout, Cin, device=DEV),
                  torch.empty(Cout, device=DEV))
    P.pyramid_fc_tanh_backward(dev(xa), dev(w1), y, dev(dy), dx, dw, db)
    p = torch.empty(M, K, device=DEV)
    loss = torch.empty(1, device=DEV)
    ldx, ldw, ldb = (torch.empty(M, Cout, device=DEV), torch.empty(K, Cout, device=DEV),
                     torch.empty(K, device=DEV))
    P.pyramid_softmax_ce(y, dev(w2), dev(b2), p, torch.from_numpy(lab).to(DEV), loss, ldx, ldw, ldb)
    torch.cuda.synchronize()
    ry = oracle.fc_tanh_forward(xa, w1, b1)
    assert normwise(host(y), ry) <= TOL["f32"]
    rb = oracle.fc_tanh_backward(xa, w1, ry, dy)
    for got, want in ((dx, rb["dx"]), (dw, rb["dw"]), (db, rb["db"])):
        assert normwise(host(got), want) <= TOL["f32"]
    rs = oracle.softmax_ce(host(y), w2, b2, lab, grad=True)
    assert normwise(host(p), rs["p"]) <= TOL["f32"]
    assert abs(loss.item() - rs["loss"]) <= TOL["f32"] * rs["loss"]
    for got, want in ((ldx, rs["dx"]), (ldw, rs["dw"]), (ldb, rs["db"])):
        assert normwise(host(got), want) <= TOL["f32"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cin,cout", [(16, 32), (32, 64), (64, 128), (16, 128), (64, 32),
                                      (24, 40)], ids=lambda v: str(v))
def test_fc_tanh_forward_widths(cin, cout, dtype):
    """FC + tanh at every width the MFMA kernel takes (and one it does not),
    a ragged number of rows, both storage types."""
    rng = np.random.default_rng(91 + cin + cout)
    M = 1037
    xd = dev(rng.standard_normal((M, cin)), dtype)
    wd = dev(rng.uniform(-0.3, 0.3, (cout, cin)), dtype)
    bd = dev(rng.uniform(-0.3, 0.3, cout), dtype)
    import paper_1506_07452_amd as P
    say("fc tanh forward", cin, cout, dtype)
    y = torch.empty(M, cout, device=DEV, dtype=xd.dtype)
    P.pyramid_fc_tanh_forward(xd, wd, bd, y)
    torch.cuda.synchronize()
    ref = oracle.fc_tanh_forward(host(xd), host(wd), host(bd))
    assert normwise(host(y), ref) <= TOL[dtype]


@pytest.mark.parametrize("case", [(1, 32, 32, 4), (1037, 64, 128, 4), (515, 32, 64, 5),
                                  (2049, 64, 32, 16), (777, 64, 64, 1), (140001, 64, 128, 4),
                                  (33, 32, 128, 3)],
                         ids=lambda c: "x".join(map(str, c)))
def test_head_forward_bf16(case):
    """The fused inference head (FC tanh + linear + softmax, bf16 storage)
    against the separate entry points (same y, fp32 sums in another order)
    and the oracle: one row, ragged tiles, one to sixteen classes."""
    import paper_1506_07452_amd as P
    M, cin, F, K = case
    rng = np.random.default_rng(131 + M + cin + F + K)
    xd = dev(rng.standard_normal((M, cin)), "bf16")
    w1 = dev(rng.uniform(-0.3, 0.3, (F, cin)), "bf16")
    b1 = dev(rng.uniform(-0.3, 0.3, F), "bf16")
    w2 = dev(rng.uniform(-0.5, 0.5, (K, F)), "bf16")
    b2 = dev(rng.uniform(-0.5, 0.5, K), "bf16")
    say("head forward bf16", case)
    assert P.pyramid_head_forward_supported(torch.bfloat16, cin, F, K)
    p = torch.full((M, K), float("nan"), device=DEV)
    P.pyramid_head_forward(xd, w1, b1, w2, b2, p)
    y = torch.empty(M, F, device=DEV, dtype=torch.bfloat16)
    P.pyramid_fc_tanh_forward(xd, w1, b1, y)
    p_sep = torch.empty(M, K, device=DEV)
    P.pyramid_softmax_ce(y, w2, b2, p_sep)
    torch.cuda.synchronize()
    assert torch.isfinite(p).all()
    err = (p - p_sep).abs().max().item()
    assert err <= 2e-6, err
    ref_y = oracle.fc_tanh_forward(host(xd), host(w1), host(b1))
    ref = oracle.softmax_ce(ref_y, host(w2), host(b2))["p"]
    assert normwise(host(p), ref) <= TOL["bf16"]


@pytest.mark.parametrize("case", [(1, 16, 32), (129, 16, 32), (1037, 32, 64), (140001, 16, 32),
                                  (2049, 32, 64), (1037, 64, 128), (515, 24, 40)],
                         ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("want_dx", [True, False], ids=["dx", "nodx"])
def test_fc_tanh_backward_widths(case, want_dx):
    """FC + tanh backward on the MFMA kernel (16 -> 32, 32 -> 64) and the row
    kernels (other widths): one row, ragged tiles, more row tiles than
    workgroups, with and without dL/dx."""
    import paper_1506_07452_amd as P
    M, cin, cout = case
    rng = np.random.default_rng(93 + M + cin)
    xa = rng.standard_normal((M, cin)).astype(np.float32)
    w1 = rng.uniform(-0.3, 0.3, (cout, cin)).astype(np.float32)
    ya = np.tanh(rng.standard_normal((M, cout))).astype(np.float32)
    dy = rng.standard_normal((M, cout)).astype(np.float32)
    say("fc tanh backward", case, want_dx)
    dx = torch.empty(M, cin, device=DEV) if want_dx else None
    dw, db = torch.empty(cout, cin, device=DEV), torch.empty(cout, device=DEV)
    P.pyramid_fc_tanh_backward(dev(xa), dev(w1), dev(ya), dev(dy), dx, dw, db)
    torch.cuda.synchronize()
    rb = oracle.fc_tanh_backward(xa, w1, ya, dy)
    pairs = [(dw, rb["dw"]), (db, rb["db"])] + ([(dx, rb["dx"])] if want_dx else [])
    for got, want in pairs:
        assert normwise(host(got), want) <= TOL["f32"]


def oracle_head(xa, w1, b1, w2, b2, lab):
    """FC tanh -> softmax CE -> backward, chained from the oracle's pieces."""
    ry = oracle.fc_tanh_forward(xa, w1, b1)
    rs = oracle.softmax_ce(ry, w2, b2, lab, grad=True)
    rb = oracle.fc_tanh_backward(xa, w1, ry, rs["dx"])
    return {"p": rs["p"], "loss": rs["loss"], "dx": rb["dx"], "dw1": rb["dw"], "db1": rb["db"],
            "dw2": rs["dw"], "db2": rs["db"]}


# (M, Cin, F, K): one row, one ragged tile, several tiles, more row tiles
# than workgroups (each workgroup loops), K at both padded widths.
HEAD_CASES = [(1, 16, 32, 4), (129, 16, 32, 3), (1000, 16, 32, 4), (777, 32, 64, 5),
              (300, 16, 32, 16), (140001, 16, 32, 4), (2049, 32, 64, 2)]


@pytest.mark.parametrize("case", HEAD_CASES, ids=lambda c: "x".join(map(str, c)))
def test_fused_head_matches_oracle(case):
    import paper_1506_07452_amd as P
    M, Cin, F, K = case
    rng = np.random.default_rng(91 + sum(case))
    xa = rng.standard_normal((M, Cin)).astype(np.float32)
    w1 = rng.uniform(-0.3, 0.3, (F, Cin)).astype(np.float32)
    b1 = rng.uniform(-0.3, 0.3, F).astype(np.float32)
    w2 = rng.uniform(-0.3, 0.3, (K, F)).astype(np.float32)
    b2 = rng.uniform(-0.3, 0.3, K).astype(np.float32)
    lab = rng.integers(0, K, M).astype(np.int32)
    say("fused head", case)
    out = {k: torch.empty(shp, device=DEV) for k, shp in
           (("p", (M, K)), ("loss", (1,)), ("dx", (M, Cin)), ("dw1", (F, Cin)), ("db1", (F,)),
            ("dw2", (K, F)), ("db2", (K,)))}
    P.pyramid_head_train(dev(xa), dev(w1), dev(b1), dev(w2), dev(b2),
                         torch.from_numpy(lab).to(DEV), out["p"], out["loss"], out["dx"],
                         out["dw1"], out["db1"], out["dw2"], out["db2"])
    torch.cuda.synchronize()
    ref = oracle_head(xa, w1, b1, w2, b2, lab)
    assert abs(out["loss"].item() - ref["loss"]) <= TOL["f32"] * ref["loss"]
    for k in ("p", "dx", "dw1", "db1", "dw2", "db2"):
        assert normwise(host(out[k]), ref[k]) <= TOL["f32"], k


def test_fused_head_without_dx_and_bad_label():
    """dx is optional; an out-of-range label turns the loss into NaN."""
    import paper_1506_07452_amd as P
    M, Cin, F, K = 300, 16, 32, 4
    rng = np.random.default_rng(5)
    args = [dev(rng.uniform(-0.3, 0.3, s).astype(np.float32))
            for s in ((M, Cin), (F, Cin), (F,), (K, F), (K,))]
    lab = torch.from_numpy(rng.integers(0, K, M).astype(np.int32)).to(DEV)
    outs = [torch.empty(s, device=DEV) for s in ((M, K), (1,), (F, Cin), (F,), (K, F), (K,))]
    say("fused head no dx")
    P.pyramid_head_train(*args, lab, outs[0], outs[1], None, *outs[2:])
    torch.cuda.synchronize()
    assert torch.isfinite(outs[1]).all()
    lab[7] = K
    P.pyramid_head_train(*args, lab, outs[0], outs[1], None, *outs[2:])
    torch.cuda.synchronize()
    assert torch.isnan(outs[1]).all()


def test_fused_training_step_matches_unfused():
    """The training step with the fused head equals the one composed from the
    separate entry points (same math, different summation order)."""
    inst = small(dict(N=1, D=6, H=20, W=18, C=3, hidden=[16, 32], fc=True, classes=4,
                      labels=True), 81)
    x, layers, fcs, head, labels = to_device(inst, "f32")
    say("fused vs unfused step")
    a = network_train_step(x, layers, fcs, head, labels, fused_head=True)
    b = network_train_step(x, layers, fcs, head, labels, fused_head=False)
    torch.cuda.synchronize()
    assert abs(a["loss"].item() - b["loss"].item()) <= 1e-5 * abs(b["loss"].item())
    pairs = [(a["p"], b["p"])] + list(zip(a["head"], b["head"]))
    for fa, fb in zip(a["fcs"], b["fcs"]):
        pairs += list(zip(fa, fb))
    for la, lb in zip(a["layers"], b["layers"]):
        pairs += list(zip(la, lb))
    for ta, tb in pairs:
        assert normwise(host(ta), host(tb)) <= TOL["f32"]


def test_config4_network_forward_bf16():
    """8 x 64^3 x 3, three layers (16, 32, 64) + FC tanh + softmax, bf16
    storage, against the oracle's stored results: every softmax output of
    batch element 0, 4096 sampled voxels across the batch, per-class sums."""
    inst = synth.config(4)
    gold = np.load(os.path.join(GOLDEN, "cfg4.npz"))
    full = np.load(os.path.join(GOLDEN, "cfg4_elem0.npz"))["p"]
    say("config 4")
    x, layers, fcs, head, _ = to_device(inst, "bf16")
    out = network_forward(x, layers, fcs, head)
    torch.cuda.synchronize()
    p = out["p"]
    got0 = host(p[:full.shape[0]])
    err = np.abs(got0 - full)
    worst = int(np.argmax(err.max(1)))
    print("[config 4] element 0: max err %.3e at voxel %d, mean err %.3e" %
          (err.max(), worst, err.mean()), flush=True)
    assert normwise(got0, full) <= TOL["bf16"]
    got = host(p[torch.from_numpy(gold["vox"]).to(DEV)])
    assert normwise(got, gold["p"]) <= TOL["bf16"]
    cs = host(p.sum(0))
    assert np.allclose(cs, gold["class_sum"], rtol=TOL["bf16"])


def test_config5_training_step():
    """48 x 240 x 240 x 3, two layers (16, 32) + FC + softmax + CE, fp32:
    loss, sampled probabilities and every parameter gradient vs the oracle."""
    inst = synth.config(5)
    gold = np.load(os.path.join(GOLDEN, "cfg5.npz"))
    say("config 5")
    x, layers, fcs, head, labels = to_device(inst, "f32")
    g = network_train_step(x, layers, fcs, head, labels)
    torch.cuda.synchronize()
    assert abs(g["loss"].item() - float(gold["loss"])) <= TOL["f32"] * float(gold["loss"])
    got_p = host(g["p"][torch.from_numpy(gold["vox"]).to(DEV)])
    assert normwise(got_p, gold["p"]) <= TOL["f32"]
    named = {"head_dw": g["head"][0], "head_db": g["head"][1]}
    for li in range(2):
        named["l%d_dwx" % li], named["l%d_dwh" % li], named["l%d_db" % li] = g["layers"][li]
        named["fc%d_dw" % li], named["fc%d_db" % li] = g["fcs"][li]
    for k, t in named.items():
        err = normwise(host(t), gold[k])
        assert err <= TOL["f32"], (k, err)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cin", [c for c, _ in SOFTMAX_CIN], ids=[n for _, n in SOFTMAX_CIN])
def test_softmax_ce_kernels_match_oracle(cin, dtype):
    """Linear + softmax + mean cross-entropy and its gradients on every
    softmax kernel, fp32 and bf16 inputs; the forward alone (no labels) gives
    the same probabilities."""
    import paper_1506_07452_amd as P
    rng = np.random.default_rng(97 + cin)
    M, K = 1531, 4
    xa = synth.to_storage(rng.standard_normal((M, cin)), dtype)
    w = synth.to_storage(rng.uniform(-0.3, 0.3, (K, cin)), dtype)
    b = synth.to_storage(rng.uniform(-0.3, 0.3, K), dtype)
    lab = rng.integers(0, K, M).astype(np.int32)
    say("softmax ce", cin, dtype)
    xd, wd, bd = dev(xa, dtype), dev(w, dtype), dev(b, dtype)
    p = torch.empty(M, K, device=DEV)
    p_inf = torch.empty(M, K, device=DEV)
    loss = torch.empty(1, device=DEV)
    # gradients take fp32 inputs only; bf16 gives probabilities and the loss
    grads = dtype == "f32"
    dw = torch.empty(K, cin, device=DEV) if grads else None
    db = torch.empty(K, device=DEV) if grads else None
    dx = torch.empty(M, cin, device=DEV) if grads else None
    P.pyramid_softmax_ce(xd, wd, bd, p, torch.from_numpy(lab).to(DEV), loss, dx, dw, db)
    P.pyramid_softmax_ce(xd, wd, bd, p_inf)
    torch.cuda.synchronize()
    ref = oracle.softmax_ce(xa, w, b, lab, grad=True)
    tol = TOL[dtype] if dtype == "bf16" else TOL["f32"]
    assert normwise(host(p), ref["p"]) <= tol
    assert torch.equal(p, p_inf)
    assert abs(loss.item() - ref["loss"]) <= TOL["f32"] * ref["loss"]
    pairs = [(dw, ref["dw"]), (db, ref["db"]), (dx, ref["dx"])] if grads else []
    for got, want in pairs:
        assert normwise(host(got), want) <= TOL["f32"]

