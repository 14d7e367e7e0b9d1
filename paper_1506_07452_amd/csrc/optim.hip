// Training update of the paper (Section 3, "Training"): RMS-prop with
// momentum over every parameter tensor of a network in one launch.
//   ms  = rho_ms ms + (1 - rho_ms) g^2       Eq. (15)
//   G   = g / (sqrt(ms) + eps)               Eq. (16)
//   mom = rho_m mom + (1 - rho_m) G          Eq. (17)
//   theta -= lr mom                          Eq. (18)
// fp32 throughout, IEEE square root and division.  The segments (tensors)
// travel in the kernel arguments; a thread updates one element, found by a
// search over the segments' first elements.
#include <math.h>

#include "common.h"
#include "timing.h"

namespace plstm {
namespace {

constexpr int kOptMaxSeg = 64;
constexpr int kOptThreads = 256;

struct OptArgs {
    int count;
    float lr, rho_ms, rho_m, eps;
    long long start[kOptMaxSeg + 1];   // first element of each segment; start[count] = total
    float *theta[kOptMaxSeg];
    const float *grad[kOptMaxSeg];
    float *ms[kOptMaxSeg];
    float *mom[kOptMaxSeg];
};

__global__ void __launch_bounds__(kOptThreads)
k_rmsprop(OptArgs a)
{
    const long long i = (long long)blockIdx.x * kOptThreads + threadIdx.x;
    if (i >= a.start[a.count]) return;
    int lo = 0, hi = a.count - 1;     // last segment with start <= i
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.start[mid] <= i) lo = mid; else hi = mid - 1;
    }
    const long long j = i - a.start[lo];
    const float g = a.grad[lo][j];
    const float ms = a.rho_ms * a.ms[lo][j] + (1.0f - a.rho_ms) * (g * g);
    const float G = g / (sqrtf(ms) + a.eps);
    const float m = a.rho_m * a.mom[lo][j] + (1.0f - a.rho_m) * G;
    a.ms[lo][j] = ms;
    a.mom[lo][j] = m;
    a.theta[lo][j] -= a.lr * m;
}

}  // namespace
}  // namespace plstm

using namespace plstm;

extern "C" {

int pyramid_rmsprop_step(int32_t count, const plstm_param_segment *segs, float lr,
                         float rho_ms, float rho_m, float eps, void *stream)
{
    if (count < 1 || count > kOptMaxSeg || !segs) return PLSTM_EINVAL;
    if (!(lr >= 0.0f) || !(rho_ms >= 0.0f && rho_ms < 1.0f) || !(rho_m >= 0.0f && rho_m < 1.0f) ||
        !(eps > 0.0f))
        return PLSTM_EINVAL;
    OptArgs a;
    a.count = count;
    a.lr = lr; a.rho_ms = rho_ms; a.rho_m = rho_m; a.eps = eps;
    long long total = 0;
    for (int k = 0; k < count; ++k) {
        const plstm_param_segment &s = segs[k];
        if (s.n < 0) return PLSTM_EINVAL;
        if (s.n > 0) {
            if (!s.theta || !s.grad || !s.ms || !s.mom) return PLSTM_EINVAL;
            if (((uintptr_t)s.theta | (uintptr_t)s.grad | (uintptr_t)s.ms | (uintptr_t)s.mom) & 3u)
                return PLSTM_EINVAL;
        }
        a.start[k] = total;
        a.theta[k] = s.theta; a.grad[k] = s.grad; a.ms[k] = s.ms; a.mom[k] = s.mom;
        total += s.n;
        if (total > (1LL << 40)) return PLSTM_EUNSUPPORTED;
    }
    a.start[count] = total;
    if (total == 0) return PLSTM_OK;
    hipStream_t st = (hipStream_t)stream;
    timing_begin("rmsprop", st);
    k_rmsprop<<<(unsigned)((total + kOptThreads - 1) / kOptThreads), kOptThreads, 0, st>>>(a);
    PLSTM_LAUNCH_CHECK();
    timing_end(1, st);
    return PLSTM_OK;
}

double pyramid_rmsprop_learning_rate(int32_t epoch)
{
    return 1e-6 + 1e-2 * pow(pow(0.5, 1.0 / 100.0), (double)epoch);
}

}  // extern "C"
