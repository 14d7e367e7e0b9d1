"""Write the full-size expected values used by the GPU parity tests.

Calls only the fp64 oracle (``oracle``, ``oracle.network``) on the seeded
synthetic workloads of ``synth``; nothing here touches the GPU path.  The
oracle takes minutes on these workloads, too long to rerun inside every
GPU test, so its results are stored once (the single-layer workloads 2 and 3
are compared in full against the oracle run inside their test instead; jobs
2 and 3 still write their samples for inspection):

  cfg2.npz, cfg3.npz  single layer forward: 4096 sampled entries of h, max|h|,
                      per-slice sums of h and h^2 (not committed)
  cfg4.npz            3-layer network forward: 4096 sampled voxels of the
                      softmax output, per-class sums
  cfg4_elem0.npz      the same network's full softmax output for batch
                      element 0 (64^3 x 4, fp32; 95 s of oracle on 8 cores)
  cfg5.npz            2-layer training step: loss, sampled probabilities and
                      every parameter gradient in full (fp32)

Usage:  python tests/golden/make_golden.py [job ...]   (jobs: 2 3 4 4_elem0 5)
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle                      # noqa: E402
import oracle.network as onet      # noqa: E402
import synth                       # noqa: E402

NSAMPLE = 4096
SAMPLE_SEED = 4242


def _layer_tuple(L):
    return (L.wx, L.wh, L.b)


def single_layer(cfg):
    inst = synth.config(cfg)
    L = inst.layers[0]
    h = oracle.forward(inst.x, L.wx, L.wh, L.b)["h"]
    rng = np.random.default_rng(SAMPLE_SEED + cfg)
    idx = rng.choice(h.size, size=NSAMPLE, replace=False)
    N, D = h.shape[:2]
    return {"idx": idx.astype(np.int64), "val": h.reshape(-1)[idx],
            "absmax": np.abs(h).max(),
            "slice_sum": h.reshape(N * D, -1).sum(1),
            "slice_sumsq": (h.reshape(N * D, -1) ** 2).sum(1)}


def network_forward(cfg):
    inst = synth.config(cfg)
    out = onet.forward(inst.x, [_layer_tuple(L) for L in inst.layers], inst.fcs, inst.head)
    p = out["p"]
    rng = np.random.default_rng(SAMPLE_SEED + cfg)
    vox = np.sort(rng.choice(p.shape[0], size=NSAMPLE, replace=False))
    return {"vox": vox.astype(np.int64), "p": p[vox], "class_sum": p.sum(0),
            "absmax": np.abs(p).max()}


def network_forward_element0(cfg):
    inst = synth.config(cfg)
    out = onet.forward(inst.x[:1], [_layer_tuple(L) for L in inst.layers], inst.fcs, inst.head)
    return {"p": out["p"].astype(np.float32)}


def training_step(cfg):
    inst = synth.config(cfg)
    g = onet.backward(inst.x, [_layer_tuple(L) for L in inst.layers], inst.fcs, inst.head,
                      inst.labels)
    rng = np.random.default_rng(SAMPLE_SEED + cfg)
    p = g["p"]
    vox = np.sort(rng.choice(p.shape[0], size=NSAMPLE, replace=False))
    res = {"loss": np.float64(g["loss"]), "vox": vox.astype(np.int64), "p": p[vox],
           "head_dw": g["head"][0], "head_db": g["head"][1]}
    for li, (dwx, dwh, db) in enumerate(g["layers"]):
        res["l%d_dwx" % li], res["l%d_dwh" % li], res["l%d_db" % li] = dwx, dwh, db
    for li, (dw, db) in enumerate(g["fcs"]):
        res["fc%d_dw" % li], res["fc%d_db" % li] = dw, db
    # gradients in fp32 (relative rounding 6e-8, far inside the tolerance)
    return {k: (v.astype(np.float32) if k.startswith(("l", "fc", "head")) and k != "loss"
                else v) for k, v in res.items()}


JOBS = {"2": single_layer, "3": single_layer, "4": network_forward,
        "4_elem0": network_forward_element0, "5": training_step}


def main(jobs):
    for job in jobs:
        cfg = int(job.split("_")[0])
        t0 = time.time()
        res = JOBS[job](cfg)
        path = os.path.join(HERE, "cfg%s.npz" % job)
        np.savez_compressed(path + ".tmp.npz", **res)
        os.replace(path + ".tmp.npz", path)
        print("cfg%s: %.1f s -> %s" % (job, time.time() - t0, path), flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or ["4", "4_elem0", "5"])
