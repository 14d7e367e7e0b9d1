// C ABI of the PyraMiD-LSTM library: argument validation, workspace sizing and
// carving, and dispatch to the HIP kernels.  Every check happens before the
// first HIP call; errors are status codes (no abort, no exception).
#include <limits.h>

#include <atomic>

#include "common.h"
#include "sweep.h"

using namespace plstm;

namespace {

// Workspace of pyramid_lstm_forward_noalloc.  Every GPU the library runs on
// holds its own copy until the process ends.  In host code `scratch` only
// names the symbol: the device address of the current GPU's copy comes from
// the runtime (scratch_ptr), and only that address reaches a kernel.
static __device__ __align__(256) unsigned char scratch[PLSTM_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch_ptr[kMaxDevices];

// The current device's copy of `scratch`, looked up on the first call made
// with that device current; null on a HIP error.
void *scratch_ptr()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
    return p;
}

bool aligned(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int check_shape(const plstm_shape *s)
{
    if (!s) return PLSTM_EINVAL;
    if (s->N < 1 || s->D < 1 || s->H < 1 || s->W < 1 || s->C < 1 || s->O < 1)
        return PLSTM_EINVAL;
    if (s->dtype != PLSTM_F32 && s->dtype != PLSTM_BF16) return PLSTM_EINVAL;
    if (s->K != 0 && (s->K < 1 || s->K % 2 == 0)) return PLSTM_EINVAL;
    if (s->K > 7) return PLSTM_EUNSUPPORTED;
    if (s->C > 1024) return PLSTM_EUNSUPPORTED;
    if (s->O != 4 && s->O != 8 && s->O != 16 && s->O != 32 && s->O != 64)
        return PLSTM_EUNSUPPORTED;
    // grid limits of the generic path: 6N blocks in z, one plane per launch
    if ((long long)s->N * kDirs > 65535) return PLSTM_EUNSUPPORTED;
    const long long V = (long long)s->D * s->H * s->W;
    if (V >= (1LL << 31) / 64 || (long long)s->N * V * 4 * s->O * kDirs > (1LL << 40))
        return PLSTM_EUNSUPPORTED;
    return PLSTM_OK;
}

// A 2D layer is validated as the volume of one slice it is computed as.
int check_shape2d(const plstm2d_shape *s)
{
    if (!s) return PLSTM_EINVAL;
    const plstm_shape t{s->N, 1, s->H, s->W, s->C, s->O, s->dtype, s->K};
    return check_shape(&t);
}

size_t layer_ws(const Geom &g, int dtype, int training)
{
    size_t need = forward_ws(g, dtype, training != 0);
    if (training) {
        const size_t b = backward_ws(g);
        if (b > need) need = b;
    }
    return need < 256 ? 256 : need;
}

int layer_forward(const Geom &g, int dtype, const void *x, const void *wx, const void *wh,
                  const void *b, void *h, void *saved, void *ws, size_t ws_bytes, void *stream)
{
    if (!x || !wx || !wh || !b || !h || !ws) return PLSTM_EINVAL;
    if (!aligned(x) || !aligned(wx) || !aligned(wh) || !aligned(b) || !aligned(h) ||
        !aligned(ws) || (saved && !aligned(saved)))
        return PLSTM_EINVAL;
    if (saved && dtype != PLSTM_F32) return PLSTM_EUNSUPPORTED;
    if (ws_bytes < layer_ws(g, dtype, saved != nullptr)) return PLSTM_EWORKSPACE;
    Saved sv{};
    if (saved) sv = carve_saved(saved, g);
    return forward_dispatch(g, dtype, x, wx, wh, b, h, saved ? &sv : nullptr, ws,
                            (hipStream_t)stream);
}

int layer_backward(const Geom &g, int dtype, const void *x, const void *wx, const void *wh,
                   const void *b, const void *saved, const void *dh, void *dx, void *dwx,
                   void *dwh, void *db, void *ws, size_t ws_bytes, void *stream)
{
    if (!x || !wx || !wh || !b || !saved || !dh || !dwx || !dwh || !db || !ws)
        return PLSTM_EINVAL;
    if (!aligned(x) || !aligned(wx) || !aligned(wh) || !aligned(b) || !aligned(saved) ||
        !aligned(dh) || (dx && !aligned(dx)) || !aligned(dwx) || !aligned(dwh) ||
        !aligned(db) || !aligned(ws))
        return PLSTM_EINVAL;
    if (dtype != PLSTM_F32) return PLSTM_EUNSUPPORTED;
    if (ws_bytes < layer_ws(g, dtype, 1)) return PLSTM_EWORKSPACE;
    const Saved sv = carve_saved(const_cast<void *>(saved), g);
    return backward_dispatch(g, (const float *)x, (const float *)wx, (const float *)wh, sv,
                             (const float *)dh, (float *)dx, (float *)dwx, (float *)dwh,
                             (float *)db, ws, (hipStream_t)stream);
}

}  // namespace

extern "C" {

const char *pyramid_lstm_status_string(int status)
{
    switch (status) {
    case PLSTM_OK: return "ok";
    case PLSTM_EINVAL: return "invalid argument";
    case PLSTM_EUNSUPPORTED: return "unsupported shape or type";
    case PLSTM_EWORKSPACE: return "workspace too small";
    case PLSTM_EHIP: return "HIP runtime error";
    case PLSTM_ENOTCORESIDENT: return "persistent grid does not fit on the device";
    case PLSTM_ESCRATCH: return "shape needs more than the no-allocation entry point's scratch";
    default: return "unknown status";
    }
}

size_t pyramid_lstm_saved_size(const plstm_shape *s)
{
    if (check_shape(s) != PLSTM_OK) return 0;
    return saved_bytes(make_geom(*s));
}

size_t pyramid_lstm_workspace_size(const plstm_shape *s, int training)
{
    if (check_shape(s) != PLSTM_OK) return 0;
    return layer_ws(make_geom(*s), s->dtype, training);
}

int pyramid_lstm_forward(const plstm_shape *s, const void *x, const void *wx, const void *wh,
                         const void *b, void *h, void *saved, void *ws, size_t ws_bytes,
                         void *stream)
{
    const int rc = check_shape(s);
    if (rc != PLSTM_OK) return rc;
    return layer_forward(make_geom(*s), s->dtype, x, wx, wh, b, h, saved, ws, ws_bytes, stream);
}

int pyramid_lstm_forward_noalloc(const plstm_shape *s, const void *x, const void *wx,
                                 const void *wh, const void *b, void *h, void *stream)
{
    const int rc = check_shape(s);
    if (rc != PLSTM_OK) return rc;
    if (!x || !wx || !wh || !b || !h) return PLSTM_EINVAL;
    const Geom g = make_geom(*s);
    if (layer_ws(g, s->dtype, 0) > (size_t)PLSTM_NOALLOC_SCRATCH_BYTES) return PLSTM_ESCRATCH;
    void *ws = scratch_ptr();
    if (!ws) return PLSTM_EHIP;
    return layer_forward(g, s->dtype, x, wx, wh, b, h, nullptr, ws,
                         (size_t)PLSTM_NOALLOC_SCRATCH_BYTES, stream);
}

int pyramid_lstm_backward(const plstm_shape *s, const void *x, const void *wx, const void *wh,
                          const void *b, const void *saved, const void *dh, void *dx, void *dwx,
                          void *dwh, void *db, void *ws, size_t ws_bytes, void *stream)
{
    const int rc = check_shape(s);
    if (rc != PLSTM_OK) return rc;
    return layer_backward(make_geom(*s), s->dtype, x, wx, wh, b, saved, dh, dx, dwx, dwh, db, ws,
                          ws_bytes, stream);
}

size_t pyramid_lstm2d_saved_size(const plstm2d_shape *s)
{
    if (check_shape2d(s) != PLSTM_OK) return 0;
    return saved_bytes(make_geom2d(*s));
}

size_t pyramid_lstm2d_workspace_size(const plstm2d_shape *s, int training)
{
    if (check_shape2d(s) != PLSTM_OK) return 0;
    return layer_ws(make_geom2d(*s), s->dtype, training);
}

int pyramid_lstm2d_forward(const plstm2d_shape *s, const void *x, const void *wx, const void *wh,
                           const void *b, void *h, void *saved, void *ws, size_t ws_bytes,
                           void *stream)
{
    const int rc = check_shape2d(s);
    if (rc != PLSTM_OK) return rc;
    return layer_forward(make_geom2d(*s), s->dtype, x, wx, wh, b, h, saved, ws, ws_bytes,
                         stream);
}

int pyramid_lstm2d_backward(const plstm2d_shape *s, const void *x, const void *wx,
                            const void *wh, const void *b, const void *saved, const void *dh,
                            void *dx, void *dwx, void *dwh, void *db, void *ws, size_t ws_bytes,
                            void *stream)
{
    const int rc = check_shape2d(s);
    if (rc != PLSTM_OK) return rc;
    return layer_backward(make_geom2d(*s), s->dtype, x, wx, wh, b, saved, dh, dx, dwx, dwh, db,
                          ws, ws_bytes, stream);
}

size_t pyramid_fc_workspace_size(int64_t M, int32_t Cin, int32_t Cout)
{
    if (M < 1 || Cin < 1 || Cout < 1 || Cin > 1024 || Cout > 1024) return 0;
    const size_t need = fc_ws(M, Cin, Cout);
    return need < 256 ? 256 : need;
}

int pyramid_fc_tanh_forward(int64_t M, int32_t Cin, int32_t Cout, int32_t dtype, const void *x,
                            const void *w, const void *b, void *y, void *stream)
{
    if (M < 1 || Cin < 1 || Cout < 1) return PLSTM_EINVAL;
    if (Cin > 1024 || Cout > 1024 || M > (1LL << 40) / Cout) return PLSTM_EUNSUPPORTED;
    if (dtype != PLSTM_F32 && dtype != PLSTM_BF16) return PLSTM_EINVAL;
    if (!x || !w || !b || !y) return PLSTM_EINVAL;
    if (!aligned(x) || !aligned(w) || !aligned(b) || !aligned(y)) return PLSTM_EINVAL;
    return fc_tanh_forward(M, Cin, Cout, dtype, x, w, b, y, (hipStream_t)stream);
}

int pyramid_fc_tanh_backward(int64_t M, int32_t Cin, int32_t Cout, const void *x, const void *w,
                             const void *y, const void *dy, void *dx, void *dw, void *db,
                             void *ws, size_t ws_bytes, void *stream)
{
    if (M < 1 || Cin < 1 || Cout < 1) return PLSTM_EINVAL;
    if (Cin > 1024 || Cout > 1024 || M > (1LL << 40) / Cout) return PLSTM_EUNSUPPORTED;
    if (!x || !w || !y || !dy || !dw || !db || !ws) return PLSTM_EINVAL;
    if (!aligned(x) || !aligned(w) || !aligned(y) || !aligned(dy) || (dx && !aligned(dx)) ||
        !aligned(dw) || !aligned(db) || !aligned(ws))
        return PLSTM_EINVAL;
    if (ws_bytes < pyramid_fc_workspace_size(M, Cin, Cout)) return PLSTM_EWORKSPACE;
    return fc_tanh_backward(M, Cin, Cout, (const float *)x, (const float *)w, (const float *)y,
                            (const float *)dy, (float *)dx, (float *)dw, (float *)db, ws,
                            (hipStream_t)stream);
}

static int softmax_entry(int64_t M, int32_t Cin, int32_t K, int32_t dtype, const void *x,
                         const void *w, const void *b, const int32_t *labels, void *p,
                         void *loss, void *dx, void *dw, void *db, void *ws, size_t ws_bytes,
                         void *stream, bool squared)
{
    if (M < 1 || Cin < 1 || K < 1) return PLSTM_EINVAL;
    if (Cin > 1024 || K > 16 || M > (1LL << 40) / 16) return PLSTM_EUNSUPPORTED;
    if (dtype != PLSTM_F32 && dtype != PLSTM_BF16) return PLSTM_EINVAL;
    if (!x || !w || !b || !p) return PLSTM_EINVAL;
    if (!aligned(x) || !aligned(w) || !aligned(b) || !aligned(p)) return PLSTM_EINVAL;
    const bool grad = dw || db || dx;
    if (labels) {
        if (!loss || !ws || !aligned(labels)) return PLSTM_EINVAL;
        if (ws_bytes < pyramid_fc_workspace_size(M, Cin, K)) return PLSTM_EWORKSPACE;
    }
    if (grad) {
        if (!labels || !dw || !db) return PLSTM_EINVAL;
        if (dtype != PLSTM_F32) return PLSTM_EUNSUPPORTED;
        if ((dx && !aligned(dx)) || !aligned(dw) || !aligned(db)) return PLSTM_EINVAL;
    }
    return softmax_ce(M, Cin, K, dtype, x, w, b, labels, (float *)p, (float *)loss,
                      (float *)dx, (float *)dw, (float *)db, ws, (hipStream_t)stream, squared);
}

int pyramid_softmax_ce(int64_t M, int32_t Cin, int32_t K, int32_t dtype, const void *x,
                       const void *w, const void *b, const int32_t *labels, void *p, void *loss,
                       void *dx, void *dw, void *db, void *ws, size_t ws_bytes, void *stream)
{
    return softmax_entry(M, Cin, K, dtype, x, w, b, labels, p, loss, dx, dw, db, ws, ws_bytes,
                         stream, false);
}

int pyramid_softmax_sq(int64_t M, int32_t Cin, int32_t K, int32_t dtype, const void *x,
                       const void *w, const void *b, const int32_t *labels, void *p, void *loss,
                       void *dx, void *dw, void *db, void *ws, size_t ws_bytes, void *stream)
{
    return softmax_entry(M, Cin, K, dtype, x, w, b, labels, p, loss, dx, dw, db, ws, ws_bytes,
                         stream, true);
}

int pyramid_head_forward_supported(int32_t dtype, int32_t Cin, int32_t F, int32_t K)
{
    return head_fwd_supported(dtype, Cin, F, K) ? 1 : 0;
}

int pyramid_head_forward(int64_t M, int32_t Cin, int32_t F, int32_t K, int32_t dtype,
                         const void *x, const void *w1, const void *b1, const void *w2,
                         const void *b2, void *p, void *stream)
{
    if (M < 1 || M > (1LL << 40) / 256 || Cin < 1 || F < 1 || K < 1) return PLSTM_EINVAL;
    if (dtype != PLSTM_F32 && dtype != PLSTM_BF16) return PLSTM_EINVAL;
    if (!x || !w1 || !b1 || !w2 || !b2 || !p) return PLSTM_EINVAL;
    if (!aligned(x) || !aligned(w1) || !aligned(b1) || !aligned(w2) || !aligned(b2) ||
        !aligned(p))
        return PLSTM_EINVAL;
    if (!head_fwd_supported(dtype, Cin, F, K)) return PLSTM_EUNSUPPORTED;
    return head_forward(M, Cin, F, K, (const uint16_t *)x, (const uint16_t *)w1,
                        (const uint16_t *)b1, (const uint16_t *)w2, (const uint16_t *)b2,
                        (float *)p, (hipStream_t)stream);
}

size_t pyramid_head_workspace_size(int64_t M, int32_t Cin, int32_t F, int32_t K)
{
    if (M < 1 || M > (1LL << 40) / 64 || !head_supported(Cin, F, K)) return 0;
    const size_t need = head_ws(M, Cin, F, K);
    return need < 256 ? 256 : need;
}

int pyramid_head_train(int64_t M, int32_t Cin, int32_t F, int32_t K, const void *x,
                       const void *w1, const void *b1, const void *w2, const void *b2,
                       const int32_t *labels, void *p, void *loss, void *dx, void *dw1,
                       void *db1, void *dw2, void *db2, void *ws, size_t ws_bytes,
                       void *stream)
{
    if (M < 1 || Cin < 1 || F < 1 || K < 1) return PLSTM_EINVAL;
    if (!x || !w1 || !b1 || !w2 || !b2 || !labels || !p || !loss || !dw1 || !db1 || !dw2 ||
        !db2 || !ws)
        return PLSTM_EINVAL;
    if (!aligned(x) || !aligned(w1) || !aligned(b1) || !aligned(w2) || !aligned(b2) ||
        !aligned(labels) || !aligned(p) || !aligned(loss) || (dx && !aligned(dx)) ||
        !aligned(dw1) || !aligned(db1) || !aligned(dw2) || !aligned(db2) || !aligned(ws))
        return PLSTM_EINVAL;
    const size_t need = pyramid_head_workspace_size(M, Cin, F, K);
    if (need == 0) return PLSTM_EUNSUPPORTED;
    if (ws_bytes < need) return PLSTM_EWORKSPACE;
    return head_train(M, Cin, F, K, (const float *)x, (const float *)w1, (const float *)b1,
                      (const float *)w2, (const float *)b2, labels, (float *)p, (float *)loss,
                      (float *)dx, (float *)dw1, (float *)db1, (float *)dw2, (float *)db2, ws,
                      (hipStream_t)stream);
}

}  // extern "C"
