// Forward dispatch between the persistent MFMA sweep and the generic path.
#pragma once

#include "common.h"

namespace plstm {

// Workspace bytes of the forward actually dispatched for this shape.
size_t forward_ws(const Geom &g, int dtype, bool training);

// Runs the layer forward on the fastest path that supports the shape.
int forward_dispatch(const Geom &g, int dtype, const void *x, const void *wx, const void *wh,
                     const void *b, void *h, float *gates, float *cell, void *ws,
                     hipStream_t st);

}  // namespace plstm
