// Per-phase HIP-event timing of the library's kernels, for measurement tools.
// When enabled, each forward/backward phase is bracketed by two events on the
// caller's stream; pyramid_lstm_timing_read() waits for them and reports the
// accumulated time and launch count per phase name.
#include <mutex>
#include <string.h>
#include <vector>

#include "timing.h"
#include "pyramid_lstm.h"

namespace plstm {
namespace {

struct Rec {
    const char *name;
    hipEvent_t start, stop;
    int launches;
};

std::mutex mu;
bool enabled = false;
std::vector<Rec> recs;
int open_rec = -1;

}  // namespace

void timing_begin(const char *name, hipStream_t st)
{
    std::lock_guard<std::mutex> lk(mu);
    if (!enabled) return;
    Rec r{name, nullptr, nullptr, 0};
    if (hipEventCreate(&r.start) != hipSuccess || hipEventCreate(&r.stop) != hipSuccess) return;
    hipEventRecord(r.start, st);
    recs.push_back(r);
    open_rec = (int)recs.size() - 1;
}

void timing_end(int launches, hipStream_t st)
{
    std::lock_guard<std::mutex> lk(mu);
    if (!enabled || open_rec < 0) return;
    recs[open_rec].launches = launches;
    hipEventRecord(recs[open_rec].stop, st);
    open_rec = -1;
}

}  // namespace plstm

using namespace plstm;

extern "C" {

int pyramid_lstm_timing_enable(int on)
{
    std::lock_guard<std::mutex> lk(mu);
    for (auto &r : recs) {
        hipEventDestroy(r.start);
        hipEventDestroy(r.stop);
    }
    recs.clear();
    open_rec = -1;
    enabled = on != 0;
    return PLSTM_OK;
}

int pyramid_lstm_timing_read(int max_phases, char *names, double *ms, int *launches,
                             int *count)
{
    std::lock_guard<std::mutex> lk(mu);
    if (max_phases < 0 || (max_phases > 0 && (!names || !ms || !launches)) || !count)
        return PLSTM_EINVAL;
    int n = 0;
    for (auto &r : recs) {
        if (hipEventSynchronize(r.stop) != hipSuccess) return PLSTM_EHIP;
        float t = 0.0f;
        if (hipEventElapsedTime(&t, r.start, r.stop) != hipSuccess) return PLSTM_EHIP;
        int k = 0;
        while (k < n && strncmp(names + 32 * k, r.name, 31) != 0) ++k;
        if (k == n) {
            if (n >= max_phases) continue;
            strncpy(names + 32 * n, r.name, 31);
            names[32 * n + 31] = 0;
            ms[n] = 0.0;
            launches[n] = 0;
            ++n;
        }
        ms[k] += t;
        launches[k] += r.launches;
    }
    *count = n;
    return PLSTM_OK;
}

}  // extern "C"
