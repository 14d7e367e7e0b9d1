"""GPU parity of the training-cube sampler (rotation about z, flips; Section 3,
"Sub-volumes and Augmentation") against the oracle, through the C ABI.
Image values within fp32 rounding of the interpolation.  Labels are the
nearest voxel of a rotated position: they must agree bit for bit, except at
voxels whose position lies within 1e-4 of a nearest-label boundary (where any
rounding may pick either side), and those must stay rare."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle.augment as oaug
import paper_1506_07452_amd as P
import synth
from tests.gpu_util import DEV, TOL, dev, host, normwise, say

pytestmark = pytest.mark.gpu


def volume(N, D, H, W, C, seed, kind="em", dtype="f32"):
    rng = np.random.default_rng(seed)
    x = synth.to_storage(synth.volume(kind, N, D, H, W, C, rng), dtype)
    lab = rng.integers(0, 5, size=(N, D, H, W)).astype(np.int32)
    return x, lab


def run(x, lab, cubes, size, dtype="f32"):
    count = len(cubes)
    N, D, H, W, C = x.shape
    xd = dev(x, dtype)
    out = torch.empty((count,) + tuple(size) + (C,), dtype=xd.dtype, device=DEV)
    labd = None if lab is None else torch.from_numpy(lab).to(DEV)
    out_lab = None if lab is None else torch.empty((count,) + tuple(size), dtype=torch.int32,
                                                   device=DEV)
    P.pyramid_sample_cubes(xd, cubes, size, out, labd, out_lab)
    torch.cuda.synchronize()
    return host(out), None if lab is None else out_lab.cpu().numpy()


MARGIN = 1e-4          # positions this close to a label boundary may go either way
MAX_NEAR_TIES = 1e-3   # ... and may make up at most this fraction of a cube


def check(x, lab, cubes, size, got, got_lab, tol):
    for q, cb in enumerate(cubes):
        corner = (cb.z0, cb.y0, cb.x0)
        ref, ref_lab = oaug.sample(x, lab, cb.n, corner, size, cb.cos_t, cb.sin_t, cb.flips)
        assert normwise(got[q], ref) <= tol, (q, normwise(got[q], ref))
        if lab is not None:
            near = oaug.label_margin(x.shape, size, corner, cb.cos_t, cb.sin_t,
                                     cb.flips) < MARGIN
            assert near.mean() <= MAX_NEAR_TIES, (q, near.mean())
            assert np.array_equal(got_lab[q][~near], ref_lab[~near]), q


CASES = [  # (N, D, H, W, C), cube size, count, recipe
    ((2, 9, 70, 61, 3), (5, 32, 40), 7, "em"),
    ((1, 6, 33, 33, 1), (6, 33, 33), 5, "em"),              # the cube is the whole volume
    ((3, 12, 48, 40, 5), (7, 24, 24), 9, "mr"),
    ((1, 4, 1, 50, 2), (2, 1, 17), 4, "em"),                # single-row slices
    ((1, 3, 9, 1, 2), (3, 9, 1), 3, "em"),                  # single-column slices
    ((1, 2, 5, 5, 1), (1, 1, 1), 6, "em"),                  # one-voxel cubes
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c[0])) + "_" + c[3])
def test_cubes_match_oracle(case):
    shape, size, count, recipe = case
    N, D, H, W, C = shape
    x, lab = volume(*shape, seed=300 + sum(shape))
    rng = np.random.default_rng(17 + sum(shape))
    if recipe == "em":
        cubes = P.draw_cubes(rng, N, (D, H, W), size, count)
    else:
        cubes = P.draw_cubes(rng, N, (D, H, W), size, count, rotate=False, flip_axes="x")
    say("cubes", shape, size, count, recipe)
    got, got_lab = run(x, lab, cubes, size)
    check(x, lab, cubes, size, got, got_lab, 1e-5)


def test_unrotated_cubes_equal_the_crop():
    x, lab = volume(2, 8, 30, 20, 3, seed=320)
    cubes = [P.plstm_cube(1, 2, 5, 3, 1.0, 0.0, 0), P.plstm_cube(0, 0, 0, 0, 1.0, 0.0, 0)]
    say("cubes identity")
    got, got_lab = run(x, lab, cubes, (4, 12, 15))
    assert np.array_equal(got[0], x[1, 2:6, 5:17, 3:18])
    assert np.array_equal(got_lab[1], lab[0, 0:4, 0:12, 0:15])
    xd = dev(x)
    tile = torch.empty((4, 12, 15, 3), device=DEV)
    P.pyramid_crop(xd, 1, (2, 5, 3, 4, 12, 15), tile)
    torch.cuda.synchronize()
    assert np.array_equal(host(tile), got[0])


def test_quarter_turns_and_flips_exact():
    """Angles whose cosine and sine are exact in fp32 land on voxel centres:
    bit-exact turns and flips of the crop."""
    x, lab = volume(1, 5, 21, 21, 2, seed=321)
    cubes = [P.plstm_cube(0, 1, 2, 3, c, s, f) for (c, s) in ((0.0, 1.0), (-1.0, 0.0), (0.0, -1.0))
             for f in range(8)]
    say("cubes quarter turns")
    got, got_lab = run(x, lab, cubes, (3, 16, 16))
    check(x, lab, cubes, (3, 16, 16), got, got_lab, 0.0)
    for q, cb in enumerate(cubes):       # on voxel centres: no label is near a boundary
        ref, ref_lab = oaug.sample(x, lab, cb.n, (cb.z0, cb.y0, cb.x0), (3, 16, 16), cb.cos_t,
                                   cb.sin_t, cb.flips)
        assert np.array_equal(got_lab[q], ref_lab)


def test_bf16_storage():
    x, lab = volume(1, 6, 40, 36, 3, seed=322, dtype="bf16")
    rng = np.random.default_rng(23)
    cubes = P.draw_cubes(rng, 1, (6, 40, 36), (4, 20, 24), 6)
    say("cubes bf16")
    got, got_lab = run(x, lab, cubes, (4, 20, 24), "bf16")
    check(x, lab, cubes, (4, 20, 24), got, got_lab, TOL["bf16"])


def test_em_stage_three_cubes_from_a_full_stack():
    """The EM recipe at the size of the last bootstrapping stage: 64 cubes
    of 20 x 256 x 256 (the most one call takes) from a 30 x 512 x 512 stack,
    checked in full against the oracle on four of them and by label range on
    all."""
    x, lab = volume(1, 30, 512, 512, 1, seed=323)
    rng = np.random.default_rng(29)
    cubes = P.draw_cubes(rng, 1, (30, 512, 512), (20, 256, 256), P.PLSTM_MAX_CUBES)
    say("cubes em stage 3")
    got, got_lab = run(x, lab, cubes, (20, 256, 256))
    check(x, lab, cubes[:2] + cubes[-2:], (20, 256, 256), np.concatenate([got[:2], got[-2:]]),
          np.concatenate([got_lab[:2], got_lab[-2:]]), 1e-5)
    assert got_lab.min() >= 0 and got_lab.max() <= 4
    assert got.min() >= x.min() - 1e-6 and got.max() <= x.max() + 1e-6   # convex weights
