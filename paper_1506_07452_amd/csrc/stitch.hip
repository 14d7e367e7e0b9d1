// Inference over volumes larger than one pass (Section 3, "Sub-volumes and
// Augmentation"): crop a sub-volume out of the input, and stitch the
// per-voxel class probabilities of the sub-volumes into the whole volume as
// a Gaussian-weighted mean.  A tile's weight at its voxel (i, j, k) is the
// separable Gaussian exp(-1/2 sum_axes ((i - c) / sigma)^2) with c the
// tile's centre and sigma = sigma_scale x the tile's extent per axis.  Tiles
// are accumulated one launch after another on the caller's stream, one
// thread per voxel, so the sums are deterministic.
#include "common.h"
#include "timing.h"

namespace plstm {
namespace {

constexpr int kStThreads = 256;

// Sub-volume [z0, z0+d) x [y0, y0+h) x [x0, x0+w) of batch element n of
// x [N][D][H][W][C] into tile [d][h][w][C]; elements of `esize` bytes,
// copied as 2-byte words (esize is 2 or 4).
__global__ void __launch_bounds__(kStThreads)
k_crop(int D, int H, int W, int words, long long n, int z0, int y0, int x0, int d, int h, int w,
       const uint16_t *__restrict__ x, uint16_t *__restrict__ tile)
{
    const long long i = (long long)blockIdx.x * kStThreads + threadIdx.x;
    const long long total = (long long)d * h * w * words;
    if (i >= total) return;
    const int c = (int)(i % words);
    const long long v = i / words;
    const int k = (int)(v % w), j = (int)((v / w) % h), z = (int)(v / ((long long)w * h));
    const long long src = (((n * D + z0 + z) * H + y0 + j) * (long long)W + x0 + k) * words + c;
    tile[i] = x[src];
}

__device__ inline float gauss(int i, int n, float scale)
{
    const float c = 0.5f * (float)(n - 1), sig = scale * (float)n;
    const float u = ((float)i - c) / sig;
    return __expf(-0.5f * u * u);
}

__global__ void __launch_bounds__(kStThreads)
k_stitch_add(int H, int W, int K, int z0, int y0, int x0, int d, int h, int w, float scale,
             const float *__restrict__ p, float *__restrict__ acc, float *__restrict__ wsum)
{
    const long long v = (long long)blockIdx.x * kStThreads + threadIdx.x;
    if (v >= (long long)d * h * w) return;
    const int k = (int)(v % w), j = (int)((v / w) % h), z = (int)(v / ((long long)w * h));
    const float g = gauss(z, d, scale) * gauss(j, h, scale) * gauss(k, w, scale);
    const long long o = ((long long)(z0 + z) * H + y0 + j) * W + x0 + k;
    for (int c = 0; c < K; ++c) acc[o * K + c] += g * p[v * K + c];
    wsum[o] += g;
}

__global__ void __launch_bounds__(kStThreads)
k_stitch_clear(long long V, int K, float *__restrict__ acc, float *__restrict__ wsum)
{
    const long long i = (long long)blockIdx.x * kStThreads + threadIdx.x;
    if (i < V * K) acc[i] = 0.0f;
    if (i < V) wsum[i] = 0.0f;
}

__global__ void __launch_bounds__(kStThreads)
k_stitch_finish(long long V, int K, const float *__restrict__ acc, const float *__restrict__ wsum,
                float *__restrict__ out)
{
    const long long i = (long long)blockIdx.x * kStThreads + threadIdx.x;
    if (i < V * K) out[i] = acc[i] / wsum[i / K];
}

inline unsigned nblocks(long long n) { return (unsigned)((n + kStThreads - 1) / kStThreads); }

bool box_ok(int D, int H, int W, int z0, int y0, int x0, int d, int h, int w)
{
    return D >= 1 && H >= 1 && W >= 1 && d >= 1 && h >= 1 && w >= 1 && z0 >= 0 && y0 >= 0 &&
           x0 >= 0 && z0 + d <= D && y0 + h <= H && x0 + w <= W;
}

}  // namespace
}  // namespace plstm

using namespace plstm;

extern "C" {

int pyramid_crop(int32_t N, int32_t D, int32_t H, int32_t W, int32_t C, int32_t dtype,
                 int32_t n, int32_t z0, int32_t y0, int32_t x0, int32_t d, int32_t h, int32_t w,
                 const void *x, void *tile, void *stream)
{
    if (!x || !tile || N < 1 || C < 1 || n < 0 || n >= N) return PLSTM_EINVAL;
    if (dtype != PLSTM_F32 && dtype != PLSTM_BF16) return PLSTM_EINVAL;
    if (!box_ok(D, H, W, z0, y0, x0, d, h, w)) return PLSTM_EINVAL;
    if (((uintptr_t)x | (uintptr_t)tile) & 3u) return PLSTM_EINVAL;
    if ((long long)N * D * H * W * C > (1LL << 40)) return PLSTM_EUNSUPPORTED;
    const int words = C * (dtype == PLSTM_F32 ? 2 : 1);
    hipStream_t st = (hipStream_t)stream;
    k_crop<<<nblocks((long long)d * h * w * words), kStThreads, 0, st>>>(
        D, H, W, words, n, z0, y0, x0, d, h, w, (const uint16_t *)x, (uint16_t *)tile);
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

int pyramid_stitch_clear(int32_t D, int32_t H, int32_t W, int32_t K, void *acc, void *wsum,
                         void *stream)
{
    if (!acc || !wsum || D < 1 || H < 1 || W < 1 || K < 1) return PLSTM_EINVAL;
    const long long V = (long long)D * H * W;
    k_stitch_clear<<<nblocks(V * K), kStThreads, 0, (hipStream_t)stream>>>(V, K, (float *)acc,
                                                                          (float *)wsum);
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

int pyramid_stitch_add(int32_t D, int32_t H, int32_t W, int32_t K, int32_t z0, int32_t y0,
                       int32_t x0, int32_t d, int32_t h, int32_t w, float sigma_scale,
                       const void *p, void *acc, void *wsum, void *stream)
{
    if (!p || !acc || !wsum || K < 1) return PLSTM_EINVAL;
    if (!box_ok(D, H, W, z0, y0, x0, d, h, w)) return PLSTM_EINVAL;
    if (!(sigma_scale > 0.0f)) return PLSTM_EINVAL;
    timing_begin("stitch", (hipStream_t)stream);
    k_stitch_add<<<nblocks((long long)d * h * w), kStThreads, 0, (hipStream_t)stream>>>(
        H, W, K, z0, y0, x0, d, h, w, sigma_scale, (const float *)p, (float *)acc,
        (float *)wsum);
    PLSTM_LAUNCH_CHECK();
    timing_end(1, (hipStream_t)stream);
    return PLSTM_OK;
}

int pyramid_stitch_finish(int32_t D, int32_t H, int32_t W, int32_t K, const void *acc,
                          const void *wsum, void *out, void *stream)
{
    if (!acc || !wsum || !out || D < 1 || H < 1 || W < 1 || K < 1) return PLSTM_EINVAL;
    const long long V = (long long)D * H * W;
    k_stitch_finish<<<nblocks(V * K), kStThreads, 0, (hipStream_t)stream>>>(
        V, K, (const float *)acc, (const float *)wsum, (float *)out);
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

}  // extern "C"
