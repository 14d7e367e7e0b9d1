// Training cubes (Section 3, "Sub-volumes and Augmentation"): cubes cut at
// given positions of the volume, turned about their own centre in the (y, x)
// plane -- a rotation about z -- and flipped along any of z, y, x.  The
// random draws (position, angle, flips) come from the caller.
//
// Cube voxel (k, i, j) before the flips reads the source position
//   z = z0 + k,  y = yc + c u - s v,  x = xc + s u + c v,
//   u = i - (h - 1) / 2, v = j - (w - 1) / 2, (yc, xc) the cube's centre,
// clamped to the slice.  Image values are bilinear in (y, x); labels take the
// nearest voxel, floor(y + 1/2).  Positions, weights and the blend are fp64:
// the kernel is an HBM gather, so the double arithmetic is free, and the
// interpolation cell and the nearest label are then decided as exactly as the
// rotation allows (only positions within ~1e-13 of a cell or label boundary
// could fall either way).  One thread per cube voxel.
#include "common.h"
#include "timing.h"

namespace plstm {
namespace {

constexpr int kAugThreads = 256;

struct CubeArgs {
    int N, D, H, W, C;
    int d, h, w;
    int n[PLSTM_MAX_CUBES], z0[PLSTM_MAX_CUBES], y0[PLSTM_MAX_CUBES], x0[PLSTM_MAX_CUBES];
    int flips[PLSTM_MAX_CUBES];
    float c[PLSTM_MAX_CUBES], s[PLSTM_MAX_CUBES];
};

// Rotated source position of cube voxel (i, j), clamped to the slice.
__device__ inline void source_yx(const CubeArgs &a, int cube, int i, int j, double &y, double &x)
{
    const double u = (double)i - 0.5 * (double)(a.h - 1);
    const double v = (double)j - 0.5 * (double)(a.w - 1);
    const double yc = (double)a.y0[cube] + 0.5 * (double)(a.h - 1);
    const double xc = (double)a.x0[cube] + 0.5 * (double)(a.w - 1);
    const double c = a.c[cube], s = a.s[cube];
    y = yc + (c * u - s * v);
    x = xc + (s * u + c * v);
    y = fmin(fmax(y, 0.0), (double)(a.H - 1));
    x = fmin(fmax(x, 0.0), (double)(a.W - 1));
}

template <typename TS>
__global__ void __launch_bounds__(kAugThreads)
k_sample_cubes(const CubeArgs a, const TS *__restrict__ vol, const int32_t *__restrict__ labels,
               TS *__restrict__ out, int32_t *__restrict__ out_labels)
{
    const int cube = blockIdx.y;
    const long long vox = (long long)blockIdx.x * kAugThreads + threadIdx.x;
    const long long per = (long long)a.d * a.h * a.w;
    if (vox >= per) return;
    const int j = (int)(vox % a.w), i = (int)((vox / a.w) % a.h), k = (int)(vox / ((long long)a.w * a.h));
    const int fl = a.flips[cube];
    const int kk = (fl & PLSTM_FLIP_Z) ? a.d - 1 - k : k;
    const int ii = (fl & PLSTM_FLIP_Y) ? a.h - 1 - i : i;
    const int jj = (fl & PLSTM_FLIP_X) ? a.w - 1 - j : j;
    double y, x;
    source_yx(a, cube, ii, jj, y, x);
    const int ya = (int)floor(y), xa = (int)floor(x);
    const int yb = min(ya + 1, a.H - 1), xb = min(xa + 1, a.W - 1);
    const double wy = y - (double)ya, wx = x - (double)xa;
    const long long slice = ((long long)a.n[cube] * a.D + a.z0[cube] + kk) * a.H;
    const long long paa = ((slice + ya) * a.W + xa) * a.C, pab = ((slice + ya) * a.W + xb) * a.C;
    const long long pba = ((slice + yb) * a.W + xa) * a.C, pbb = ((slice + yb) * a.W + xb) * a.C;
    const double waa = (1.0 - wy) * (1.0 - wx), wab = (1.0 - wy) * wx;
    const double wba = wy * (1.0 - wx), wbb = wy * wx;
    const long long o = ((long long)cube * per + vox) * a.C;
    for (int ch = 0; ch < a.C; ++ch) {
        const double r = waa * (double)Store<TS>::load(vol, paa + ch) +
                         wab * (double)Store<TS>::load(vol, pab + ch) +
                         wba * (double)Store<TS>::load(vol, pba + ch) +
                         wbb * (double)Store<TS>::load(vol, pbb + ch);
        Store<TS>::store(out, o + ch, (float)r);
    }
    if (labels) {
        const int yn = (int)floor(y + 0.5), xn = (int)floor(x + 0.5);
        out_labels[(long long)cube * per + vox] = labels[(slice + yn) * a.W + xn];
    }
}

}  // namespace
}  // namespace plstm

using namespace plstm;

extern "C" {

int pyramid_sample_cubes(int32_t N, int32_t D, int32_t H, int32_t W, int32_t C, int32_t dtype,
                         int32_t count, const plstm_cube *cubes, int32_t d, int32_t h, int32_t w,
                         const void *x, const int32_t *labels, void *out, int32_t *out_labels,
                         void *stream)
{
    if (!x || !out || !cubes || (labels && !out_labels)) return PLSTM_EINVAL;
    if (N < 1 || D < 1 || H < 1 || W < 1 || C < 1 || d < 1 || h < 1 || w < 1) return PLSTM_EINVAL;
    if (count < 1 || count > PLSTM_MAX_CUBES) return PLSTM_EINVAL;
    if (dtype != PLSTM_F32 && dtype != PLSTM_BF16) return PLSTM_EINVAL;
    if (d > D || h > H || w > W) return PLSTM_EINVAL;
    const size_t esz = dtype == PLSTM_F32 ? 4 : 2;
    if ((((uintptr_t)x | (uintptr_t)out) & (esz - 1)) ||
        (((uintptr_t)labels | (uintptr_t)out_labels) & 3u))
        return PLSTM_EINVAL;
    if ((long long)N * D * H * W * C > (1LL << 40) || H >= (1 << 22) || W >= (1 << 22))
        return PLSTM_EUNSUPPORTED;
    CubeArgs a;
    a.N = N; a.D = D; a.H = H; a.W = W; a.C = C;
    a.d = d; a.h = h; a.w = w;
    for (int q = 0; q < count; ++q) {
        const plstm_cube &cb = cubes[q];
        if (cb.n < 0 || cb.n >= N || cb.z0 < 0 || cb.y0 < 0 || cb.x0 < 0 || cb.z0 + d > D ||
            cb.y0 + h > H || cb.x0 + w > W || cb.flips < 0 || cb.flips > 7)
            return PLSTM_EINVAL;
        if (!(cb.cos_t >= -1.0f && cb.cos_t <= 1.0f && cb.sin_t >= -1.0f && cb.sin_t <= 1.0f))
            return PLSTM_EINVAL;
        a.n[q] = cb.n; a.z0[q] = cb.z0; a.y0[q] = cb.y0; a.x0[q] = cb.x0;
        a.flips[q] = cb.flips; a.c[q] = cb.cos_t; a.s[q] = cb.sin_t;
    }
    const long long per = (long long)d * h * w;
    const dim3 grid((unsigned)((per + kAugThreads - 1) / kAugThreads), (unsigned)count);
    hipStream_t st = (hipStream_t)stream;
    timing_begin("sample_cubes", st);
    if (dtype == PLSTM_F32)
        k_sample_cubes<float><<<grid, kAugThreads, 0, st>>>(a, (const float *)x, labels,
                                                            (float *)out, out_labels);
    else
        k_sample_cubes<uint16_t><<<grid, kAugThreads, 0, st>>>(a, (const uint16_t *)x, labels,
                                                               (uint16_t *)out, out_labels);
    PLSTM_LAUNCH_CHECK();
    timing_end(1, st);
    return PLSTM_OK;
}

}  // extern "C"
