// Chooses the forward implementation for a shape.
#include "sweep.h"

namespace plstm {

size_t forward_ws(const Geom &g, int dtype, bool training)
{
    (void)dtype;
    return generic_forward_ws(g, training);
}

int forward_dispatch(const Geom &g, int dtype, const void *x, const void *wx, const void *wh,
                     const void *b, void *h, float *gates, float *cell, void *ws,
                     hipStream_t st)
{
    return generic_forward(g, dtype, x, wx, wh, b, h, gates, cell, ws, st);
}

}  // namespace plstm
