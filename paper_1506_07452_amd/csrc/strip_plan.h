// Strip decomposition shared by the persistent sweep kernels.
//
// Each direction's plane is cut into k strips of whole rows x about Q/k
// columns; one workgroup owns one strip (of one batch element) for the whole
// sweep and stages a chunk of rows (plus a 1-pixel halo) in LDS per step.
// The planner picks k per axis (both directions of an axis share a geometry)
// to minimise the modelled time of the slowest direction within the number
// of co-resident workgroups.
#pragma once

#include "common.h"

namespace plstm {

struct DevInfo {
    int cus = 0;
    int max_lds = 0;
};

inline DevInfo device_info()
{
    static DevInfo cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return DevInfo{};
    DevInfo &di = cache[dev];
    if (di.cus == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess)
            di.cus = v;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess)
            di.max_lds = v;
    }
    return di;
}

// Per-step cost model of a strip (microseconds; fitted on MI355X): a
// neighbour handshake, then per LDS chunk a staging round trip that grows
// with the staged pixels and the 16-pixel tiles, shared by four SIMDs.
struct StripCostModel {
    size_t fixed_bytes;   // LDS independent of the strip size
    size_t px_bytes;      // LDS per staged pixel
    double c_sync, c_tile, c_stage0, c_stage_px;
    // Resident mode (optional): the whole strip stays in LDS for the sweep,
    // res_px_bytes per staged pixel (incl. halo) plus res_own_bytes per strip
    // pixel plus res_fixed_bytes; one step then costs c_res_step + the tiles.
    bool allow_resident = false;
    size_t res_px_bytes = 0, res_own_bytes = 0, res_fixed_bytes = 0;
    int res_max_staged = 0;   // most staged elements the kernel supports
    long long res_max_own = 0;   // most strip pixels the kernel supports (0: no limit)
    double c_res_step = 0.0;
};

struct Plan {
    int nstrip[kDirs];
    int first[kDirs];
    int chunk_rows[kDirs];
    int max_w[kDirs];
    int resident[kDirs];
    int blocks;
    size_t lds;
};

struct StripShape {
    int w, rows, chunks;
    bool resident;
    size_t lds;
};

inline StripShape strip_shape(const DirGeom &r, int k, const StripCostModel &m, size_t lds_limit)
{
    StripShape sh{};
    sh.w = (r.Q + k - 1) / k;
    if (m.allow_resident) {
        const long long staged = (long long)(r.P + 2) * (sh.w + 2);
        const size_t lds = m.fixed_bytes + m.res_fixed_bytes + (size_t)staged * m.res_px_bytes +
                           (size_t)r.P * sh.w * m.res_own_bytes;
        if (lds <= lds_limit && staged <= m.res_max_staged &&
            (m.res_max_own == 0 || (long long)r.P * sh.w <= m.res_max_own)) {
            sh.rows = r.P;
            sh.chunks = 1;
            sh.resident = true;
            sh.lds = lds;
            return sh;
        }
    }
    const size_t per_row = (size_t)(sh.w + 2) * m.px_bytes;
    const long long max_rows =
        lds_limit > m.fixed_bytes ? (long long)((lds_limit - m.fixed_bytes) / per_row) - 2 : 0;
    if (max_rows < 1) return sh;   // rows = 0: does not fit
    // Rows per chunk: the four SIMDs take a chunk's 16-pixel tiles in rounds
    // of four, so among the row counts that fit, take the one with the
    // fewest modelled rounds plus stagings over the plane (the last chunk
    // holds the remaining rows); ties go to the larger chunk.
    const long long lo = max_rows / 2 > 1 ? max_rows / 2 : 1;
    double best = 1e300;
    for (long long rows = max_rows; rows >= lo; --rows) {
        const long long chunks = (r.P + rows - 1) / rows;
        const long long last = r.P - (chunks - 1) * rows;
        const long long rounds = (chunks - 1) * ((rows * sh.w + 63) / 64) + (last * sh.w + 63) / 64;
        const double c = (double)chunks * (m.c_stage0 + m.c_stage_px * (rows + 2) * (sh.w + 2)) +
                         (double)rounds * m.c_tile;
        if (c < best * (1.0 - 1e-9)) {
            best = c;
            sh.rows = (int)rows;
            sh.chunks = (int)chunks;
        }
    }
    sh.lds = m.fixed_bytes + (size_t)(sh.rows + 2) * per_row;
    return sh;
}

inline double strip_cost(const DirGeom &r, int k, const StripCostModel &m, size_t lds_limit)
{
    const StripShape sh = strip_shape(r, k, m, lds_limit);
    if (sh.rows < 1) return 1e30;
    const int tiles = (sh.rows * sh.w + 15) / 16;
    if (sh.resident) return (double)r.T * (m.c_res_step + ((tiles + 3) / 4) * m.c_tile);
    const double stage = m.c_stage0 + m.c_stage_px * (sh.rows + 2) * (sh.w + 2);
    const int last = r.P - (sh.chunks - 1) * sh.rows;
    const int rounds = (sh.chunks - 1) * ((sh.rows * sh.w + 63) / 64) + (last * sh.w + 63) / 64;
    return (double)r.T * (m.c_sync + sh.chunks * stage + rounds * m.c_tile);
}

// For each axis only the counts k = ceil(Q / w) (the fewest strips of
// widest-strip width w) are candidates; all combinations are searched.
inline Plan make_plan(const Geom &g, int budget, const StripCostModel &m, size_t lds_limit)
{
    Plan pl{};
    int cand[3][64];
    double cost[3][64];
    int ncand[3];
    for (int ax = 0; ax < 3; ++ax) {
        const DirGeom &r = g.dir[2 * ax];
        ncand[ax] = 0;
        int prev_w = -1;
        for (int k = 1; k <= r.Q && ncand[ax] < 64; ++k) {
            const int w = (r.Q + k - 1) / k;
            if (w == prev_w) continue;
            prev_w = w;
            if ((long long)2 * g.N * k > budget) break;
            cand[ax][ncand[ax]] = k;
            cost[ax][ncand[ax]] = strip_cost(r, k, m, lds_limit);
            ++ncand[ax];
        }
    }
    double best = 1e300;
    int bk[3] = {1, 1, 1};
    for (int i = 0; i < ncand[0]; ++i)
        for (int j = 0; j < ncand[1]; ++j)
            for (int l = 0; l < ncand[2]; ++l) {
                const long long blocks = 2LL * g.N * (cand[0][i] + cand[1][j] + cand[2][l]);
                if (blocks > budget) continue;
                double c = cost[0][i];
                if (cost[1][j] > c) c = cost[1][j];
                if (cost[2][l] > c) c = cost[2][l];
                if (c < best * (1.0 - 1e-9) ||
                    (c <= best && blocks < 2LL * g.N * (bk[0] + bk[1] + bk[2]))) {
                    best = c;
                    bk[0] = cand[0][i]; bk[1] = cand[1][j]; bk[2] = cand[2][l];
                }
            }
    int first = 0;
    size_t lds = 0;
    for (int d = 0; d < kDirs; ++d) {
        const int k = bk[d / 2];
        const StripShape sh = strip_shape(g.dir[d], k, m, lds_limit);
        pl.nstrip[d] = k;
        pl.first[d] = first;
        pl.chunk_rows[d] = sh.rows;
        pl.max_w[d] = sh.w;
        pl.resident[d] = sh.resident ? 1 : 0;
        first += k * g.N;
        if (sh.lds > lds) lds = sh.lds;
    }
    pl.blocks = first;
    pl.lds = lds;
    return pl;
}

}  // namespace plstm
