// Chooses the forward implementation for a shape.
#include "sweep.h"

namespace plstm {

int g_forward_path = 0;

size_t forward_ws(const Geom &g, int dtype, bool training)
{
    size_t need = generic_forward_ws(g, training);
    if (sweep_fwd_supported(g, dtype)) {
        const size_t s = sweep_fwd_ws(g, training);
        if (s > need) need = s;
    }
    return need;
}

int forward_dispatch(const Geom &g, int dtype, const void *x, const void *wx, const void *wh,
                     const void *b, void *h, float *gates, float *cell, void *ws,
                     hipStream_t st)
{
    if (g_forward_path != 1 && sweep_fwd_supported(g, dtype)) {
        Carve cv(ws);
        float *hd = cv.take<float>((size_t)kDirs * g.N * g.V * g.O);
        float *cellbuf = cell ? cell : cv.take<float>((size_t)kDirs * g.N * g.V * g.O);
        int *flags = cv.take<int>(1024 + 1);
        const int rc = sweep_fwd(g, (const float *)x, (const float *)wx, (const float *)wh,
                                 (const float *)b, hd, cellbuf, gates, flags, st);
        if (rc == PLSTM_OK) return sum_dirs(g, dtype, hd, h, st);
        // A grid that cannot be co-resident or a plane too wide for LDS runs
        // on the generic path instead.
        if (rc != PLSTM_ENOTCORESIDENT && rc != PLSTM_EUNSUPPORTED) return rc;
    }
    return generic_forward(g, dtype, x, wx, wh, b, h, gates, cell, ws, st);
}

}  // namespace plstm

extern "C" int pyramid_lstm_set_forward_path(int path)
{
    if (path < 0 || path > 2) return PLSTM_EINVAL;
    plstm::g_forward_path = path;
    return PLSTM_OK;
}
