// Forward dispatch between the persistent MFMA sweep and the generic path.
#pragma once

#include "common.h"

namespace plstm {

// Persistent MFMA sweep (sweep_fwd.hip): O = 16, C <= 4, fp32.
bool sweep_fwd_supported(const Geom &g, int dtype);
size_t sweep_fwd_ws(const Geom &g, bool training);
int sweep_fwd(const Geom &g, const float *x, const float *wx, const float *wh, const float *b,
              float *hd, float *cell, float *gates, int *flags, hipStream_t st,
              bool allow_resident);

// Persistent MFMA backward sweep + MFMA parameter gradients (sweep_bwd.hip):
// O = 16, C <= 4, fp32.
bool sweep_bwd_supported(const Geom &g);
size_t sweep_bwd_ws(const Geom &g);
int sweep_bwd(const Geom &g, const float *x, const float *wx, const float *wh, const Saved &sv,
              const float *dh, float *dx, float *dwx, float *dwh, float *db, void *ws,
              hipStream_t st, bool allow_resident);

// Plane-step MFMA path (sweep_step.hip): O = 16, 32, 64, C <= 64, fp32
// arithmetic (bf16 storage converted on entry), one launch per plane step.
bool step_supported(const Geom &g);
// bf16 inference of a 16-unit layer on the macro-tiled bf16 step (packed taps),
// taken before the persistent fp32 sweep
bool step_b16_packed(const Geom &g, int dtype);
size_t step_fwd_ws(const Geom &g);
// Writes c^d, the gates when `gates` is set, h^d (fp32; bf16 storage on the
// bf16 MFMA keeps h^d in bf16 in the workspace instead) and the direction sum h.
int step_fwd(const Geom &g, int dtype, const void *x, const void *wx, const void *wh,
             const void *b, float *hd, float *cell, float *gates, void *h, void *ws,
             hipStream_t st);
size_t step_bwd_ws(const Geom &g);
int step_bwd(const Geom &g, const float *x, const float *wh, const float *wx, const Saved &sv,
             const float *dh, float *dx, float *dwx, float *dwh, float *db, void *ws,
             hipStream_t st);
// dL/dx from the gate gradients dA [6][N][V][4O] on the MFMA (step_supported
// shapes); `fragx` holds step_dx_ws bytes.
size_t step_dx_ws(const Geom &g);
int step_dx(const Geom &g, const float *wx, const float *dA, float *fragx, float *dx,
            hipStream_t st);

// Outputs overwritten with NaN when a persistent launch's bounded wait gave
// up (status.hip): up to kMax fp32 arrays, null entries skipped.
struct PoisonList {
    static constexpr int kMax = 4;
    float *ptr[kMax] = {nullptr, nullptr, nullptr, nullptr};
    long long count[kMax] = {0, 0, 0, 0};
};
// Enqueues the check after a persistent launch whose error word is `err`.
int wait_check(const int *err, const PoisonList &pl, hipStream_t st);
// This device's sticky status word (null on a HIP error).
int *device_status_word();
// Bounded waits of the persistent sweeps: polls before giving up, and the
// bias added to the step a wait expects (non-zero only in the failure-path
// test mode, pyramid_lstm_set_wait_test).
extern int g_wait_spin_limit;
extern int g_wait_bias;

// h = sum of the six per-direction outputs (generic.hip): from fp32 h^d, or
// (sum_dirs_bf16, bf16 h) from bf16 h^d, added in fp32 and rounded once.
int sum_dirs(const Geom &g, int dtype, const float *hd, void *h, hipStream_t st);
int sum_dirs_bf16(const Geom &g, const uint16_t *hb, void *h, hipStream_t st);

// Workspace bytes of the forward for this shape (covers every path it may take).
size_t forward_ws(const Geom &g, int dtype, bool training);

// Runs the layer forward on the fastest path that supports the shape.
int forward_dispatch(const Geom &g, int dtype, const void *x, const void *wx, const void *wh,
                     const void *b, void *h, const Saved *sv, void *ws, hipStream_t st);

// Backward (fp32): workspace bytes and dispatch.
size_t backward_ws(const Geom &g);
int backward_dispatch(const Geom &g, const float *x, const float *wx, const float *wh,
                      const Saved &sv, const float *dh, float *dx, float *dwx, float *dwh,
                      float *db, void *ws, hipStream_t st);

// Forward: 0 = automatic, 1 = generic path only, 2 = persistent MFMA sweep where
// supported, 3 = as 2 without strips kept whole in LDS, 4 = plane-step MFMA
// path where supported.  Backward: 0 = automatic, 1 = generic path only,
// 2 = persistent MFMA sweep where supported, 3 = plane-step MFMA path where
// supported.
extern int g_forward_path;
extern int g_backward_path;
// Plane-step launches: 0 = automatic, 1 = always split each tile's K over a
// workgroup's waves, 2 = never, 3 = never and the fp32 forward without LDS
// staging.
extern int g_step_split;
// bf16 storage with 32 or 64 hidden units: 1 = contraction on the bf16 MFMA
// with pixel blocks staged in LDS (default), 2 = bf16 MFMA with operands read
// from L1, 0 = on the fp32 MFMA.
extern int g_step_bf16_mfma;
// Weight gradients of the plane-step path: 1 = the LDS-staged GEMM where it
// applies (at most 32 hidden units, C % 4 == 0; default), 0 = the
// register-streamed kernel.
extern int g_wgrad_staged;

}  // namespace plstm
