// Chooses the forward implementation for a shape.
#include "sweep.h"

namespace plstm {

int g_forward_path = 0;
int g_backward_path = 0;

namespace {
// fp32 copies of a bf16 layer's input and parameters for the persistent
// sweep (3 x 3 filters), carved after its own workspace.
struct Widened {
    float *x, *wx, *wh, *b;
};
Widened widened_params(Carve &cv, const Geom &g)
{
    Widened w;
    w.x = cv.take<float>((size_t)g.N * g.V * g.C);
    w.wx = cv.take<float>((size_t)g.nd * 4 * g.O * g.C * 9);
    w.wh = cv.take<float>((size_t)g.nd * 4 * g.O * g.O * 9);
    w.b = cv.take<float>((size_t)g.nd * 4 * g.O);
    return w;
}
}  // namespace

size_t forward_ws(const Geom &g, int dtype, bool training)
{
    size_t need = generic_forward_ws(g, training);
    if (sweep_fwd_supported(g, dtype)) {
        Carve cv(nullptr);
        cv.take<char>(sweep_fwd_ws(g, training));
        if (dtype == PLSTM_BF16) widened_params(cv, g);
        if (cv.off > need) need = cv.off;
    }
    if (step_supported(g)) {
        Carve cv(nullptr);
        if (!training) {
            cv.take<float>(saved_state_count(g));   // h^d
            cv.take<float>(saved_state_count(g));   // c^d
        }
        const size_t s = align_up(cv.off, 256) + step_fwd_ws(g);
        if (s > need) need = s;
    }
    return need;
}

int forward_dispatch(const Geom &g, int dtype, const void *x, const void *wx, const void *wh,
                     const void *b, void *h, const Saved *sv, void *ws, hipStream_t st)
{
    const int path = g_forward_path;
    const bool b16_step = !sv && step_supported(g) && step_b16_packed(g, dtype);
    if (path != 1 && path != 4 && !b16_step && sweep_fwd_supported(g, dtype)) {
        Carve cv(ws);
        float *hd = sv ? sv->hd : cv.take<float>(saved_state_count(g));
        float *cellbuf = sv ? sv->cell : cv.take<float>(saved_state_count(g));
        int *flags = cv.take<int>(1024 + 1);
        const float *xf = (const float *)x, *wxf = (const float *)wx, *whf = (const float *)wh,
                    *bf = (const float *)b;
        if (dtype == PLSTM_BF16) {
            // the persistent sweep computes in fp32: widen the bf16 inputs
            const Widened wd = widened_params(cv, g);
            int rc = bf16_to_f32(x, wd.x, (long long)g.N * g.V * g.C, st);
            if (rc == PLSTM_OK) rc = bf16_to_f32(wx, wd.wx, (long long)g.nd * 4 * g.O * g.C * 9, st);
            if (rc == PLSTM_OK) rc = bf16_to_f32(wh, wd.wh, (long long)g.nd * 4 * g.O * g.O * 9, st);
            if (rc == PLSTM_OK) rc = bf16_to_f32(b, wd.b, (long long)g.nd * 4 * g.O, st);
            if (rc != PLSTM_OK) return rc;
            xf = wd.x; wxf = wd.wx; whf = wd.wh; bf = wd.b;
        }
        const int rc = sweep_fwd(g, xf, wxf, whf, bf, hd, cellbuf, sv ? sv->gates : nullptr,
                                 flags, st, path != 3);
        if (rc == PLSTM_OK) return sum_dirs(g, dtype, hd, h, st);
        // A grid that cannot be co-resident or a plane too wide for LDS runs
        // on another path instead.
        if (rc != PLSTM_ENOTCORESIDENT && rc != PLSTM_EUNSUPPORTED) return rc;
    }
    if (path != 1 && step_supported(g)) {
        Carve cv(ws);
        float *hd = sv ? sv->hd : cv.take<float>(saved_state_count(g));
        float *cellbuf = sv ? sv->cell : cv.take<float>(saved_state_count(g));
        char *rest = (char *)ws + align_up(cv.off, 256);
        return step_fwd(g, dtype, x, wx, wh, b, hd, cellbuf, sv ? sv->gates : nullptr, h, rest,
                        st);
    }
    return generic_forward(g, dtype, x, wx, wh, b, h, sv, ws, st);
}

size_t backward_ws(const Geom &g)
{
    size_t need = generic_backward_ws(g);
    if (sweep_bwd_supported(g)) {
        const size_t s = sweep_bwd_ws(g);
        if (s > need) need = s;
    }
    if (step_supported(g)) {
        const size_t s = step_bwd_ws(g);
        if (s > need) need = s;
    }
    return need;
}

int backward_dispatch(const Geom &g, const float *x, const float *wx, const float *wh,
                      const Saved &sv, const float *dh, float *dx, float *dwx, float *dwh,
                      float *db, void *ws, hipStream_t st)
{
    const int path = g_backward_path;
    if (path != 1 && path != 3 && sweep_bwd_supported(g)) {
        const int rc = sweep_bwd(g, x, wx, wh, sv, dh, dx, dwx, dwh, db, ws, st, path != 2);
        if (rc != PLSTM_ENOTCORESIDENT && rc != PLSTM_EUNSUPPORTED) return rc;
    }
    if (path != 1 && step_supported(g))
        return step_bwd(g, x, wh, wx, sv, dh, dx, dwx, dwh, db, ws, st);
    return generic_backward(g, x, wx, wh, sv, dh, dx, dwx, dwh, db, ws, st);
}

}  // namespace plstm

extern "C" int pyramid_lstm_set_forward_path(int path)
{
    if (path < 0 || path > 4) return PLSTM_EINVAL;
    plstm::g_forward_path = path;
    return PLSTM_OK;
}

extern "C" int pyramid_lstm_set_backward_path(int path)
{
    if (path < 0 || path > 3) return PLSTM_EINVAL;
    plstm::g_backward_path = path;
    return PLSTM_OK;
}
