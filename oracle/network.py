"""Stacked PyraMiD-LSTM network on the fp64 oracle -- test infrastructure only.

Fig. 3 and Section 2.3 ("Fully-Connected Layer"): every PyraMiD-LSTM layer is
followed by a per-voxel fully connected layer squashed by tanh; a softmax
follows the last fully connected layer.  Reading used for the synthetic
networks: each hidden fully connected layer has twice the width of the
PyraMiD-LSTM layer before it, and a final linear layer maps to the classes,
followed by the softmax (and, for training, the mean cross-entropy over all
voxels of the batch).  Gradients are the chain rule through these pieces; each
piece is an oracle function from ``oracle.c``.
"""
from __future__ import annotations

import numpy as np

from . import backward as layer_backward
from . import fc_tanh_backward, fc_tanh_forward
from . import forward as layer_forward
from . import softmax_ce


def forward(x, layers, fcs, head, labels=None):
    """x [N][D][H][W][C]; layers = [(wx, wh, b)], fcs = [(w, b)], head = (w, b).

    Returns dict: 'p' [N*D*H*W][classes], 'loss' (if labels), and the
    per-layer activations needed by ``backward`` under 'acts'."""
    N, D, H, W, _ = x.shape
    a = np.asarray(x, dtype=np.float64)
    acts = []
    for (wx, wh, b), (wf, bf) in zip(layers, fcs):
        h = layer_forward(a, wx, wh, b)["h"]
        O = h.shape[-1]
        y = fc_tanh_forward(h.reshape(-1, O), wf, bf).reshape(N, D, H, W, -1)
        acts.append({"in": a, "h": h, "y": y})
        a = y
    out = softmax_ce(a.reshape(-1, a.shape[-1]), head[0], head[1], labels,
                     grad=labels is not None)
    out["acts"] = acts
    return out


def backward(x, layers, fcs, head, labels):
    """Gradients of the mean cross-entropy w.r.t. every parameter.

    Returns dict: 'loss', 'head' (dw, db), 'fcs' [(dw, db)], 'layers'
    [(dwx, dwh, db)], in the order of the arguments."""
    fwd = forward(x, layers, fcs, head, labels)
    acts = fwd["acts"]
    N, D, H, W, _ = x.shape
    g = fwd["dx"].reshape(acts[-1]["y"].shape)        # dL/d(last FC output)
    layer_grads = [None] * len(layers)
    fc_grads = [None] * len(fcs)
    for li in range(len(layers) - 1, -1, -1):
        wx, wh, b = layers[li]
        wf, _ = fcs[li]
        h, y = acts[li]["h"], acts[li]["y"]
        O = h.shape[-1]
        fg = fc_tanh_backward(h.reshape(-1, O), wf, y.reshape(-1, y.shape[-1]),
                              g.reshape(-1, g.shape[-1]))
        fc_grads[li] = (fg["dw"], fg["db"])
        dh = fg["dx"].reshape(h.shape)
        lg = layer_backward(acts[li]["in"], wx, wh, b, dh, want_dx=li > 0)
        layer_grads[li] = (lg["dwx"], lg["dwh"], lg["db"])
        if li > 0:
            g = lg["dx"]
    return {"loss": fwd["loss"], "p": fwd["p"], "head": (fwd["dw"], fwd["db"]),
            "fcs": fc_grads, "layers": layer_grads}
