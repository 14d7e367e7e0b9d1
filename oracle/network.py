"""Stacked PyraMiD-LSTM network on the fp64 oracle -- test infrastructure only.

Fig. 3 and Section 2.3 ("Fully-Connected Layer"): PyraMiD-LSTM layers are
followed by per-voxel fully connected layers squashed by tanh; a softmax
follows the last fully connected layer.  Two topologies:
  - len(fcs) == len(layers): a hidden FC tanh after every PyraMiD-LSTM layer,
    then a linear output layer (the synthetic networks: each hidden FC layer
    twice as wide as the layer before it);
  - len(fcs) == len(layers) - 1: the last PyraMiD-LSTM layer feeds the output
    layer directly (the network of Section 3, "Experimental Setup": 16 units ->
    FC 25 -> 32 units -> FC 45 -> 64 units -> output layer).
The output layer is linear + softmax (and, for training, the mean
cross-entropy over all voxels of the batch).  Gradients are the chain rule
through these pieces; each piece is an oracle function from ``oracle.c``.
"""
from __future__ import annotations

import numpy as np

from . import backward as layer_backward
from . import fc_tanh_backward, fc_tanh_forward
from . import forward as layer_forward
from . import softmax_ce
from .loss import softmax_sq


def forward(x, layers, fcs, head, labels=None, loss="ce"):
    """x [N][D][H][W][C]; layers = [(wx, wh, b)], fcs = [(w, b)], head = (w, b).
    loss: "ce" (mean cross-entropy) or "sq" (mean squared error against the
    one-hot target, Eq. (14)).

    Returns dict: 'p' [N*D*H*W][classes], 'loss' (if labels), and the
    per-layer activations needed by ``backward`` under 'acts'."""
    N, D, H, W, _ = x.shape
    assert len(fcs) in (len(layers), len(layers) - 1)
    a = np.asarray(x, dtype=np.float64)
    acts = []
    for li, (wx, wh, b) in enumerate(layers):
        h = layer_forward(a, wx, wh, b)["h"]
        act = {"in": a, "h": h}
        a = h
        if li < len(fcs):
            wf, bf = fcs[li]
            y = fc_tanh_forward(h.reshape(-1, h.shape[-1]), wf, bf).reshape(N, D, H, W, -1)
            act["y"] = y
            a = y
        acts.append(act)
    head_fn = {"ce": softmax_ce, "sq": softmax_sq}[loss]
    out = head_fn(a.reshape(-1, a.shape[-1]), head[0], head[1], labels,
                  grad=labels is not None)
    out["acts"] = acts
    return out


def backward(x, layers, fcs, head, labels, loss="ce"):
    """Gradients of the loss ("ce" or "sq", as in ``forward``) w.r.t. every
    parameter.

    Returns dict: 'loss', 'head' (dw, db), 'fcs' [(dw, db)], 'layers'
    [(dwx, dwh, db)], in the order of the arguments."""
    fwd = forward(x, layers, fcs, head, labels, loss)
    acts = fwd["acts"]
    N, D, H, W, _ = x.shape
    last = acts[-1]["y"] if "y" in acts[-1] else acts[-1]["h"]
    g = fwd["dx"].reshape(last.shape)                 # dL/d(input of the output layer)
    layer_grads = [None] * len(layers)
    fc_grads = [None] * len(fcs)
    for li in range(len(layers) - 1, -1, -1):
        wx, wh, b = layers[li]
        h = acts[li]["h"]
        if li < len(fcs):
            wf, _ = fcs[li]
            y = acts[li]["y"]
            fg = fc_tanh_backward(h.reshape(-1, h.shape[-1]), wf, y.reshape(-1, y.shape[-1]),
                                  g.reshape(-1, g.shape[-1]))
            fc_grads[li] = (fg["dw"], fg["db"])
            dh = fg["dx"].reshape(h.shape)
        else:
            dh = g.reshape(h.shape)
        lg = layer_backward(acts[li]["in"], wx, wh, b, dh, want_dx=li > 0)
        layer_grads[li] = (lg["dwx"], lg["dwh"], lg["db"])
        if li > 0:
            g = lg["dx"]
    return {"loss": fwd["loss"], "p": fwd["p"], "head": (fwd["dw"], fwd["db"]),
            "fcs": fc_grads, "layers": layer_grads}
