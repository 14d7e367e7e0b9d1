// Optional per-phase timing with HIP events (off unless enabled).
#pragma once

#include <hip/hip_runtime.h>

namespace plstm {

// Record an event on `st` opening phase `name` (a string literal); no-op when
// timing is disabled.
void timing_begin(const char *name, hipStream_t st);
// Close the most recently opened phase; `launches` kernel launches ran in it.
void timing_end(int launches, hipStream_t st);

}  // namespace plstm
