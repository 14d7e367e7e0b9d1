"""The forward that allocates nothing (pyramid_lstm_forward_noalloc, for
callers that cannot allocate) against pyramid_lstm_forward, through the C
ABI: two calls in a row on the library's per-GPU scratch, the second with a
smaller input, each compared with the existing entry point on the same
inputs and with the oracle."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_1506_07452_amd as P
import synth
from tests.gpu_util import TOL, dev, host, layer_dev, normwise, say

pytestmark = pytest.mark.gpu

# (N, D, H, W, C, O, dtype) pairs: a larger call, then a smaller one.  The
# persistent sweep (16 units), the plane-step path (32 units) and bf16
# storage (widened to fp32 inside the scratch).
PAIRS = [
    ((1, 20, 48, 40, 3, 16, "f32"), (1, 6, 20, 18, 2, 16, "f32")),
    ((2, 9, 17, 40, 32, 32, "f32"), (1, 5, 9, 11, 3, 32, "f32")),
    ((1, 12, 32, 32, 3, 16, "bf16"), (1, 4, 10, 12, 1, 16, "bf16")),
]


def run_pair(pair):
    results = []
    for k, (N, D, H, W, C, O, dtype) in enumerate(pair):
        wl = synth.Workload("noalloc", N, D, H, W, C, [O], dtype=dtype, seed=700 + 31 * k + O)
        inst = synth.make(wl)
        L = inst.layers[0]
        x, Ld = dev(inst.x, dtype), layer_dev(L, dtype)
        s = P.shape_for(x, O)
        h_na = torch.empty(x.shape[:-1] + (O,), dtype=x.dtype, device=x.device)
        say("noalloc", (N, D, H, W, C, O, dtype))
        P.pyramid_lstm_forward_noalloc(s, x, Ld.wx, Ld.wh, Ld.b, h_na)
        results.append((inst, L, dtype, x, Ld, s, h_na))
    torch.cuda.synchronize()
    for inst, L, dtype, x, Ld, s, h_na in results:
        h_ref = torch.empty_like(h_na)
        P.pyramid_lstm_forward(s, x, Ld.wx, Ld.wh, Ld.b, h_ref)
        torch.cuda.synchronize()
        tol = TOL[dtype]
        assert normwise(host(h_na), host(h_ref)) <= tol
        ref = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
        assert normwise(host(h_na), ref) <= tol
        if dtype == "f32":
            assert torch.equal(h_na, h_ref)     # same kernels, same order


@pytest.mark.parametrize("pair", PAIRS, ids=["sweep", "plane_step", "bf16"])
def test_noalloc_two_calls_match_forward(pair):
    run_pair(pair)


def test_noalloc_rejects_shapes_beyond_the_scratch():
    s = P.plstm_shape(1, 80, 64, 64, 3, 16, P.PLSTM_F32, 3)
    assert P.pyramid_lstm_workspace_size(s, 0) > P.PLSTM_NOALLOC_SCRATCH_BYTES
    x = torch.zeros((1, 80, 64, 64, 3), device="cuda:0")
    w = torch.zeros(16, device="cuda:0")
    with pytest.raises(P.PyramidLSTMError) as e:
        P.pyramid_lstm_forward_noalloc(s, x, w, w, w, x)
    assert e.value.status == P.PLSTM_ESCRATCH
