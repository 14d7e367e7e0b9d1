"""Stacked PyraMiD-LSTM networks on the GPU, composed from the C entry points.

Fig. 3 / Section 2.3: PyraMiD-LSTM layer -> per-voxel FC + tanh, repeated;
the last FC layer feeds a per-voxel softmax.  This module only allocates
tensors with torch and calls the library (every arithmetic step runs in the
HIP kernels); gradients flow through the same entry points in reverse.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Tuple

import torch

from . import (plstm_shape, pyramid_fc_tanh_backward, pyramid_fc_tanh_forward,
               pyramid_head_forward, pyramid_head_forward_supported,
               pyramid_head_train, pyramid_head_workspace_size, pyramid_lstm_backward,
               pyramid_lstm_forward, pyramid_lstm_saved_size, pyramid_lstm_workspace_size,
               pyramid_lstm2d_backward, pyramid_lstm2d_forward, pyramid_lstm2d_saved_size,
               pyramid_softmax_ce, shape2d_for, shape_for)


@dataclass
class LayerW:
    wx: torch.Tensor      # [6][4O][C][K][K]
    wh: torch.Tensor      # [6][4O][O][K][K]
    b: torch.Tensor       # [6][4O]

    @property
    def O(self):
        return self.wh.shape[2]

    @property
    def K(self):
        return self.wh.shape[-1]


def layer_forward(x: torch.Tensor, L: LayerW, training: bool = False, ws=None, stream=None):
    """One layer; returns (h, saved or None)."""
    s = shape_for(x, L.O, L.K)
    h = torch.empty(x.shape[:-1] + (L.O,), dtype=x.dtype, device=x.device)
    saved = None
    if training:
        saved = torch.empty(pyramid_lstm_saved_size(s), dtype=torch.uint8, device=x.device)
    pyramid_lstm_forward(s, x, L.wx, L.wh, L.b, h, saved, ws, stream)
    return h, saved


def layer_backward(x, L: LayerW, saved, dh, want_dx=True, ws=None, stream=None):
    s = shape_for(x, L.O, L.K)
    dx = torch.empty_like(x) if want_dx else None
    dwx, dwh, db = (torch.empty_like(t, dtype=torch.float32) for t in (L.wx, L.wh, L.b))
    pyramid_lstm_backward(s, x, L.wx, L.wh, L.b, saved, dh, dx, dwx, dwh, db, ws, stream)
    return dx, dwx, dwh, db


def layer2d_forward(x: torch.Tensor, L: LayerW, training: bool = False, ws=None, stream=None):
    """2D layer over x [N][H][W][C] (weights [4][4O][C|O][K], b [4][4O]);
    returns (h, saved or None)."""
    s = shape2d_for(x, L.O, L.K)
    h = torch.empty(x.shape[:-1] + (L.O,), dtype=x.dtype, device=x.device)
    saved = None
    if training:
        saved = torch.empty(pyramid_lstm2d_saved_size(s), dtype=torch.uint8, device=x.device)
    pyramid_lstm2d_forward(s, x, L.wx, L.wh, L.b, h, saved, ws, stream)
    return h, saved


def layer2d_backward(x, L: LayerW, saved, dh, want_dx=True, ws=None, stream=None):
    s = shape2d_for(x, L.O, L.K)
    dx = torch.empty_like(x) if want_dx else None
    dwx, dwh, db = (torch.empty_like(t, dtype=torch.float32) for t in (L.wx, L.wh, L.b))
    pyramid_lstm2d_backward(s, x, L.wx, L.wh, L.b, saved, dh, dx, dwx, dwh, db, ws, stream)
    return dx, dwx, dwh, db


def workspace_for(x_shape, hidden: List[int], fc: bool, dtype, training: bool, device):
    """One workspace big enough for every layer of a network whose FC layers
    are twice as wide as the layer before (3 x 3 filters)."""
    shapes, C = [], x_shape[-1]
    for O in hidden:
        shapes.append((C, O, 3))
        C = 2 * O if fc else O
    return workspace_for_layers(x_shape, shapes, dtype, training, device)


def workspace_for_layers(x_shape, shapes, dtype, training: bool, device):
    """One workspace big enough for layers of (input channels, hidden units,
    filter size) `shapes` over the volume of `x_shape`."""
    need = 256
    for C, O, K in shapes:
        s = plstm_shape(*x_shape[:-1], C, O, 0 if dtype == torch.float32 else 1, K)
        need = max(need, pyramid_lstm_workspace_size(s, int(training)))
    return torch.empty(need, dtype=torch.uint8, device=device)


def network_forward(x, layers: List[LayerW], fcs: List[Tuple[torch.Tensor, torch.Tensor]],
                    head: Tuple[torch.Tensor, torch.Tensor], labels: Optional[torch.Tensor] = None,
                    training: bool = False, ws=None, stream=None, loss: str = "ce"):
    """Returns dict: 'p' [M][K] fp32, 'loss' (device scalar, with labels),
    'acts' (per-layer inputs/outputs and saved activations for training).
    loss: "ce" (mean cross-entropy) or "sq" (squared error, Eq. (14))."""
    N, D, H, W, _ = x.shape
    M = N * D * H * W
    if len(fcs) not in (len(layers), len(layers) - 1):
        raise ValueError("one hidden FC layer per PyraMiD-LSTM layer, or none after the last")
    K = head[0].shape[0]
    # inference with bf16 storage: the last FC and the softmax as one pass
    # (the last layer's act then has no "y")
    fused = (labels is None and not training and len(fcs) == len(layers) and
             x.dtype == torch.bfloat16 and
             pyramid_head_forward_supported(x.dtype, layers[-1].O, fcs[-1][0].shape[0], K))
    a = x
    acts = []
    for li, L in enumerate(layers):
        h, saved = layer_forward(a, L, training, ws, stream)
        act = {"in": a, "h": h, "saved": saved}
        a = h
        if fused and li == len(layers) - 1:
            acts.append(act)
            p = torch.empty((M, K), dtype=torch.float32, device=x.device)
            pyramid_head_forward(h.view(M, -1), fcs[li][0], fcs[li][1], head[0], head[1], p,
                                 stream)
            return {"p": p, "acts": acts}
        if li < len(fcs):
            wf, bf = fcs[li]
            y = torch.empty((N, D, H, W, wf.shape[0]), dtype=a.dtype, device=a.device)
            pyramid_fc_tanh_forward(h.view(M, -1), wf, bf, y.view(M, -1), stream)
            act["y"] = y
            a = y
        acts.append(act)
    p = torch.empty((M, K), dtype=torch.float32, device=x.device)
    out = {"p": p, "acts": acts}
    if labels is None:
        pyramid_softmax_ce(a.view(M, -1), head[0], head[1], p, stream=stream)
        return out
    if loss not in ("ce", "sq"):
        raise ValueError("loss must be 'ce' or 'sq'")
    lval = torch.empty(1, dtype=torch.float32, device=x.device)
    out["loss"] = lval
    if training:
        dlast = torch.empty((M, a.shape[-1]), dtype=torch.float32, device=x.device)
        dw = torch.empty_like(head[0])
        db = torch.empty_like(head[1])
        pyramid_softmax_ce(a.view(M, -1), head[0], head[1], p, labels, lval, dlast, dw, db,
                           stream=stream, squared=loss == "sq")
        out.update({"dlast": dlast, "head_grad": (dw, db)})
    else:
        pyramid_softmax_ce(a.view(M, -1), head[0], head[1], p, labels, lval, stream=stream,
                           squared=loss == "sq")
    return out


def network_train_step(x, layers, fcs, head, labels, ws=None, stream=None, fused_head=True,
                       loss="ce"):
    """Forward + back-propagation through the whole network (fp32).
    Returns dict with 'loss', 'p', 'head' (dw, db), 'fcs' [(dw, db)],
    'layers' [(dwx, dwh, db)].  With `fused_head` (default) the last FC + tanh,
    the softmax head, the loss and their backward run as one pass over the
    voxels (pyramid_head_train) where it covers the widths."""
    N, D, H, W, _ = x.shape
    M = N * D * H * W
    nl = len(layers)
    O_last, F_last, K = layers[-1].O, fcs[-1][0].shape[0], head[0].shape[0]
    if not (fused_head and loss == "ce" and len(fcs) == nl and
            pyramid_head_workspace_size(M, O_last, F_last, K) > 0):
        return _train_step_unfused(x, layers, fcs, head, labels, ws, stream, loss)
    a = x
    acts = []
    for li in range(nl):
        h, saved = layer_forward(a, layers[li], True, ws, stream)
        act = {"in": a, "h": h, "saved": saved}
        if li < nl - 1:
            wf, bf = fcs[li]
            y = torch.empty((N, D, H, W, wf.shape[0]), dtype=a.dtype, device=a.device)
            pyramid_fc_tanh_forward(h.view(M, -1), wf, bf, y.view(M, -1), stream)
            act["y"] = y
            a = y
        acts.append(act)
    p = torch.empty((M, K), dtype=torch.float32, device=x.device)
    lval = torch.empty(1, dtype=torch.float32, device=x.device)
    dh = torch.empty((M, O_last), dtype=torch.float32, device=x.device)
    wf, bf = fcs[-1]
    dwf, dbf = torch.empty_like(wf), torch.empty_like(bf)
    dw, db = torch.empty_like(head[0]), torch.empty_like(head[1])
    pyramid_head_train(acts[-1]["h"].view(M, O_last), wf, bf, head[0], head[1], labels, p, lval,
                       dh, dwf, dbf, dw, db, stream=stream)
    fc_grads = [None] * len(fcs)
    layer_grads = [None] * nl
    fc_grads[-1] = (dwf, dbf)
    g = None
    for li in range(nl - 1, -1, -1):
        act = acts[li]
        O = act["h"].shape[-1]
        if li < nl - 1:
            wf, _ = fcs[li]
            dh = torch.empty((M, O), dtype=torch.float32, device=x.device)
            dwf, dbf = torch.empty_like(wf), torch.empty(wf.shape[0], device=x.device)
            pyramid_fc_tanh_backward(act["h"].view(M, O), wf, act["y"].view(M, -1),
                                     g.view(M, -1), dh, dwf, dbf, stream=stream)
            fc_grads[li] = (dwf, dbf)
        dx, dwx, dwh, db_l = layer_backward(act["in"], layers[li], act["saved"],
                                            dh.view(act["h"].shape), want_dx=li > 0, ws=ws,
                                            stream=stream)
        layer_grads[li] = (dwx, dwh, db_l)
        g = dx
    return {"loss": lval, "p": p, "head": (dw, db), "fcs": fc_grads, "layers": layer_grads}


def _train_step_unfused(x, layers, fcs, head, labels, ws=None, stream=None, loss="ce"):
    """network_train_step composed from the separate FC / softmax entry points."""
    out = network_forward(x, layers, fcs, head, labels, training=True, ws=ws, stream=stream,
                          loss=loss)
    acts = out["acts"]
    g = out["dlast"]
    N, D, H, W, _ = x.shape
    M = N * D * H * W
    fc_grads = [None] * len(fcs)
    layer_grads = [None] * len(layers)
    for li in range(len(layers) - 1, -1, -1):
        act = acts[li]
        O = act["h"].shape[-1]
        if li < len(fcs):
            wf, _ = fcs[li]
            dh = torch.empty((M, O), dtype=torch.float32, device=x.device)
            dwf, dbf = torch.empty_like(wf), torch.empty(wf.shape[0], device=x.device)
            pyramid_fc_tanh_backward(act["h"].view(M, O), wf, act["y"].view(M, -1),
                                     g.view(M, -1), dh, dwf, dbf, stream=stream)
            fc_grads[li] = (dwf, dbf)
        else:
            dh = g      # the output layer reads h directly
        dx, dwx, dwh, db = layer_backward(act["in"], layers[li], act["saved"],
                                          dh.view(act["h"].shape), want_dx=li > 0, ws=ws,
                                          stream=stream)
        layer_grads[li] = (dwx, dwh, db)
        if li > 0:
            g = dx
    return {"loss": out["loss"], "p": out["p"], "head": out["head_grad"], "fcs": fc_grads,
            "layers": layer_grads}


def network_parameters(layers, fcs, head):
    """Every parameter tensor of a network, in the order of
    `network_gradients`: per layer (wx, wh, b), per hidden FC (w, b), head."""
    out = []
    for L in layers:
        out += [L.wx, L.wh, L.b]
    for w, b in fcs:
        out += [w, b]
    return out + [head[0], head[1]]


def network_gradients(g):
    """The gradients of a `network_train_step` result, in the order of
    `network_parameters`."""
    out = []
    for t in g["layers"]:
        out += list(t)
    for t in g["fcs"]:
        out += list(t)
    return out + [g["head"][0], g["head"][1]]


def grid_axis(extent, size, stride):
    """Tile origins along one axis of `extent` voxels for tiles of `size`
    (cut to the extent) advancing by `stride`: n = ceil((extent - size) /
    stride) + 1 tiles, the i-th at min(i * stride, extent - size), so the
    last one ends flush with the axis.  Returns (origins, size)."""
    if extent < 1 or size < 1 or stride < 1:
        raise ValueError("extent, tile size and stride must be positive")
    size = min(size, extent)
    span = extent - size
    n = -(-span // stride) + 1
    return [min(i * stride, span) for i in range(n)], size


def network_infer_volume(x, layers, fcs, head, tile, stride=None, sigma_scale=0.25, ws=None,
                         stream=None, origins=None):
    """Class probabilities [N][D][H][W][K] of a volume processed as sub-volumes
    (Section 3, "Sub-volumes and Augmentation"): tiles of size `tile` (d, h, w),
    each run through the network on its own and stitched with Gaussian weights
    (sigma = sigma_scale x tile extent).  The tile origins per axis are either
    given (`origins` = (z list, y list, x list), every tile inside the volume)
    or laid on a grid of `stride` (d, h, w) by `grid_axis`."""
    from . import pyramid_crop, pyramid_stitch_add, pyramid_stitch_clear, pyramid_stitch_finish
    N, D, H, W, C = x.shape
    K = head[0].shape[0]
    if origins is None:
        if stride is None:
            raise ValueError("give a stride or explicit tile origins")
        (zs, td), (ys, th), (xs, tw) = (grid_axis(e, t, s) for e, t, s in
                                        zip((D, H, W), tile, stride))
    else:
        td, th, tw = tile
        zs, ys, xs = (list(o) for o in origins)
        for ext, size, starts in ((D, td, zs), (H, th, ys), (W, tw, xs)):
            if not starts or min(starts) < 0 or max(starts) + size > ext:
                raise ValueError("tile origins must keep every tile inside the volume")
    out = torch.empty((N, D, H, W, K), dtype=torch.float32, device=x.device)
    acc = torch.empty((D, H, W, K), dtype=torch.float32, device=x.device)
    wsum = torch.empty((D, H, W), dtype=torch.float32, device=x.device)
    sub = torch.empty((1, td, th, tw, C), dtype=x.dtype, device=x.device)
    for n in range(N):
        pyramid_stitch_clear(acc, wsum, stream)
        for z0 in zs:
            for y0 in ys:
                for x0 in xs:
                    box = (z0, y0, x0, td, th, tw)
                    pyramid_crop(x, n, box, sub, stream)
                    p = network_forward(sub, layers, fcs, head, ws=ws, stream=stream)["p"]
                    pyramid_stitch_add(p.view(td, th, tw, K), box, acc, wsum, sigma_scale,
                                       stream)
        pyramid_stitch_finish(acc, wsum, out[n], stream)
    return out

