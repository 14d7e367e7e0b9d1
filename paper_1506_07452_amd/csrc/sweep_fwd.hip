// Persistent MFMA forward sweep for O = 16 hidden units, C <= 4 input
// channels, fp32 (Section 2.3, Eq. (7)-(12); the sum of Eq. (13) follows in
// a separate pass).
//
// One cooperative launch runs all six directions (and all batch elements) at
// once.  The plane of each direction is cut into strips of whole rows x a few
// columns; one workgroup (4 waves) owns one strip for the whole sweep:
//
//   for t in 0..T-1:
//     wait until the two neighbouring strips have published h_{t-1}
//     for each chunk of rows of the strip (sized to fit LDS):
//       stage h_{t-1} (chunk + 1-pixel halo) and the input plane x_t into LDS
//       each wave, per tile of 16 pixels:
//         A = bias + im2col(x_t) W_x + im2col(h_{t-1}) W_h   (v_mfma_f32_16x16x4f32)
//         gates, c_t = g i + c_{t-1} f, h_t = o tanh(c_t)    (in registers)
//         write h_t, c_t (and the gates when training) to global memory
//     publish: release fence, flag = t + 1
//
// The weights live in VGPRs as MFMA B fragments for the whole kernel; h of
// every plane stays in the per-direction volume in global memory, so a step
// only reads plane t-1 and writes plane t (no write-after-read hazard), and
// LDS is just a staging copy.  MFMA layout (16x16x4 f32, one block): lane l
// supplies A[m = l%16][k = l/16] and B[k = l/16][n = l%16] and receives
// D[4(l/16) + i][l%16], i = 0..3.  The K index of a tap is permuted so that
// lane group q = l/16 takes hidden channels 4q..4q+3 with one 16-byte LDS
// read; B uses the same permutation.  N-tile g holds gate g (i, f, g, o) of
// the 16 units, so every lane ends with all four gates of unit l%16 for four
// pixels and the cell update needs no data exchange.
#include "common.h"
#include "sweep.h"
#include "timing.h"

namespace plstm {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kO = 16;
constexpr int kG = 4 * kO;
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kHS = 20;          // LDS floats per staged h pixel (16 + 4 pad)
constexpr int kMaxSpin = 1 << 21;

struct SweepArgs {
    Geom g;
    const float *x, *wx, *wh, *b;
    float *hd;          // [6][N][V][16] per-direction h^d
    float *cell;        // [6][N][V][16] c^d
    float *gates;       // [6][N][V][64] or null
    int *flags;         // [blocks] completed steps per strip
    int *err;           // set when a wait gives up
    int nstrip[kDirs];  // strips per (direction, batch element)
    int first[kDirs];   // first block of direction d
    int chunk_rows;     // rows staged per LDS chunk
    int max_w;          // widest strip (LDS layout)
};

__device__ inline float fsig(float a) { return 1.0f / (1.0f + __expf(-a)); }
__device__ inline float ftanh(float a) {
    // tanh(a) = 1 - 2 / (exp(2a) + 1); saturates correctly at +-inf.
    return 1.0f - 2.0f / (__expf(2.0f * a) + 1.0f);
}

template <int C>
__global__ void __launch_bounds__(kThreads, 1) k_sweep_fwd(SweepArgs a)
{
    extern __shared__ float smem[];
    // ---- which strip this workgroup owns -------------------------------
    int d = 0;
#pragma unroll
    for (int k = 1; k < kDirs; ++k)
        if ((int)blockIdx.x >= a.first[k]) d = k;
    const int local = blockIdx.x - a.first[d];
    const int ns = a.nstrip[d];
    const int n = local / ns, strip = local % ns;
    const DirGeom dg = a.g.dir[d];
    const int q0 = (int)((long long)strip * dg.Q / ns);
    const int q1 = (int)((long long)(strip + 1) * dg.Q / ns);
    const int TQ = q1 - q0, W2 = TQ + 2;
    const int nb_lo = strip > 0 ? (int)blockIdx.x - 1 : -1;
    const int nb_hi = strip + 1 < ns ? (int)blockIdx.x + 1 : -1;

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int q4 = lane >> 4, col = lane & 15;
    float *hs = smem;
    float *xs = smem + (a.chunk_rows + 2) * (a.max_w + 2) * kHS;

    // ---- weights as MFMA B fragments (resident for the whole sweep) -----
    const long long V = a.g.V;
    float bh[9][4][4];
#pragma unroll
    for (int tap = 0; tap < 9; ++tap)
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                const int j = 4 * q4 + s, gn = nt * kO + col;
                bh[tap][s][nt] = a.wh[(((long long)d * kG + gn) * kO + j) * 9 + tap];
            }
    constexpr int KXS = (9 * C + 3) / 4;
    float bx[KXS][4];
    int xoff[KXS];
#pragma unroll
    for (int ks = 0; ks < KXS; ++ks) {
        const int k = 4 * ks + q4;
        const int tap = k < 9 * C ? k / C : 0, c = k % C;   // padding lanes read tap 0
        xoff[ks] = k < 9 * C ? ((tap / 3 - 1) * W2 + (tap % 3 - 1)) * C + c : 0;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const int gn = nt * kO + col;
            const float w = a.wx[(((long long)d * kG + gn) * C + c) * 9 + tap];
            bx[ks][nt] = k < 9 * C ? w : 0.0f;
        }
    }
    float bias[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) bias[nt] = a.b[d * kG + nt * kO + col];

    const long long dn = ((long long)d * a.g.N + n) * V;   // h^d / c^d base (voxels)
    const long long xn = (long long)n * V;                  // x base (voxels)

    for (int t = 0; t < dg.T; ++t) {
        const int s = dg.sign > 0 ? t : dg.T - 1 - t;
        const int sprev = s - dg.sign;
        // ---- wait for the neighbours' h_{t-1} ---------------------------
        if (t > 0) {
            const int nb = threadIdx.x == 0 ? nb_lo : (threadIdx.x == 1 ? nb_hi : -1);
            if (nb >= 0) {
                int spins = 0;
                while (__hip_atomic_load(&a.flags[nb], __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT) < t) {
                    __builtin_amdgcn_s_sleep(1);
                    if (++spins > kMaxSpin) {
                        __hip_atomic_store(a.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        break;
                    }
                    if ((spins & 1023) == 0 &&
                        __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
                        break;
                }
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            }
            __syncthreads();
        }
        for (int r0 = 0; r0 < dg.P; r0 += a.chunk_rows) {
            const int CH = min(a.chunk_rows, dg.P - r0);
            const int npl = (CH + 2) * W2;            // staged pixels incl. halo
            // ---- stage h_{t-1} and x_t (zero outside the plane) ----------
            for (int e = threadIdx.x; e < npl * 4; e += kThreads) {
                const int pix = e >> 2, qd = e & 3;
                const int pr = pix / W2 + r0 - 1, pc = pix % W2 + q0 - 1;
                f4 v = {0.0f, 0.0f, 0.0f, 0.0f};
                if (t > 0 && pr >= 0 && pr < dg.P && pc >= 0 && pc < dg.Q)
                    v = *(const f4 *)&a.hd[(dn + sprev * dg.ss + pr * dg.sp + pc * dg.sq) * kO +
                                          qd * 4];
                *(f4 *)&hs[pix * kHS + qd * 4] = v;
            }
            for (int e = threadIdx.x; e < npl * C; e += kThreads) {
                const int pix = e / C, c = e % C;
                const int pr = pix / W2 + r0 - 1, pc = pix % W2 + q0 - 1;
                float v = 0.0f;
                if (pr >= 0 && pr < dg.P && pc >= 0 && pc < dg.Q)
                    v = a.x[(xn + s * dg.ss + pr * dg.sp + pc * dg.sq) * C + c];
                xs[pix * C + c] = v;
            }
            __syncthreads();
            // ---- 16-pixel tiles -----------------------------------------
            const int npx = CH * TQ;
            const int nmt = (npx + 15) >> 4;
            for (int mt = wave; mt < nmt; mt += kWaves) {
                const int pa = min(mt * 16 + col, npx - 1);     // this lane's A row
                const int base = (pa / TQ + 1) * W2 + (pa % TQ + 1);
                f4 acc[4];
#pragma unroll
                for (int nt = 0; nt < 4; ++nt) acc[nt] = f4{bias[nt], bias[nt], bias[nt], bias[nt]};
#pragma unroll
                for (int tap = 0; tap < 9; ++tap) {
                    const int o = (tap / 3 - 1) * W2 + (tap % 3 - 1);
                    const f4 hv = *(const f4 *)&hs[(base + o) * kHS + 4 * q4];
#pragma unroll
                    for (int s2 = 0; s2 < 4; ++s2)
#pragma unroll
                        for (int nt = 0; nt < 4; ++nt)
                            acc[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(hv[s2], bh[tap][s2][nt],
                                                                         acc[nt], 0, 0, 0);
                }
#pragma unroll
                for (int ks = 0; ks < KXS; ++ks) {
                    const float av = (4 * ks + q4 < 9 * C) ? xs[base * C + xoff[ks]] : 0.0f;
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt)
                        acc[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bx[ks][nt], acc[nt],
                                                                     0, 0, 0);
                }
                // ---- gates and cell update: rows 4 q4 + i, unit col ------
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int px = mt * 16 + 4 * q4 + i;
                    if (px >= npx) continue;
                    const int pr = px / TQ + r0, pc = px % TQ + q0;
                    const long long v = dn + s * dg.ss + pr * dg.sp + pc * dg.sq;
                    const float gi = fsig(acc[0][i]);
                    const float gf = fsig(acc[1][i]);
                    const float gg = ftanh(acc[2][i]);
                    const float go = fsig(acc[3][i]);
                    float c = gg * gi;
                    if (t > 0) c += a.cell[(v + (long long)(sprev - s) * dg.ss) * kO + col] * gf;
                    a.cell[v * kO + col] = c;
                    a.hd[v * kO + col] = go * ftanh(c);
                    if (a.gates) {
                        float *gp = a.gates + v * kG + col;
                        gp[0] = gi;
                        gp[kO] = gf;
                        gp[2 * kO] = gg;
                        gp[3 * kO] = go;
                    }
                }
            }
            __syncthreads();
        }
        // ---- publish h_t -------------------------------------------------
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        __syncthreads();
        if (threadIdx.x == 0)
            __hip_atomic_store(&a.flags[blockIdx.x], t + 1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
    }
}

__global__ void k_fill_zero(int *p, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

// ---- launch planning ------------------------------------------------------
struct Plan {
    int nstrip[kDirs];
    int first[kDirs];
    int blocks;
    int chunk_rows;
    int max_w;
    size_t lds;
};

struct DevInfo {
    int cus = 0;
    int max_lds = 0;
};

DevInfo device_info()
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

// Strip counts that balance T_d x (pixels per strip x per-pixel cost +
// per-step synchronisation cost) over the directions, within `budget` blocks.
Plan make_plan(const Geom &g, int budget, int C, size_t lds_limit)
{
    Plan pl{};
    const double px_cost = 1.0, sync_cost = 80.0;   // relative: ~one 16-px tile per sync
    int ns[kDirs];
    for (int d = 0; d < kDirs; ++d) ns[d] = 1;
    auto cost = [&](int d, int k) {
        const DirGeom &r = g.dir[d];
        const double px = (double)r.P * ((r.Q + k - 1) / k);
        return (double)r.T * (px * px_cost + sync_cost);
    };
    int used = kDirs * g.N;
    while (true) {
        int worst = -1;
        double wc = -1.0;
        for (int d = 0; d < kDirs; ++d) {
            const double c = cost(d, ns[d]);
            if (c > wc) { wc = c; worst = d; }
        }
        if (worst < 0 || ns[worst] >= g.dir[worst].Q || used + g.N > budget) break;
        ++ns[worst];
        used += g.N;
    }
    int first = 0, max_w = 1;
    for (int d = 0; d < kDirs; ++d) {
        pl.nstrip[d] = ns[d];
        pl.first[d] = first;
        first += ns[d] * g.N;
        const int w = (g.dir[d].Q + ns[d] - 1) / ns[d];
        max_w = w > max_w ? w : max_w;
    }
    pl.blocks = first;
    pl.max_w = max_w;
    // rows per chunk: fill the LDS budget
    int maxP = 1;
    for (int d = 0; d < kDirs; ++d) maxP = g.dir[d].P > maxP ? g.dir[d].P : maxP;
    const size_t per_row = (size_t)(max_w + 2) * (kHS + C) * sizeof(float);
    long long rows = (long long)(lds_limit / per_row) - 2;
    if (rows > maxP) rows = maxP;
    pl.chunk_rows = rows < 1 ? 0 : (int)rows;
    pl.lds = (size_t)(pl.chunk_rows + 2) * per_row;
    return pl;
}

template <int C>
int launch_sweep(const Plan &pl, SweepArgs &args, hipStream_t st)
{
    const void *fn = (const void *)k_sweep_fwd<C>;
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_sweep_fwd<C>, kThreads, pl.lds) !=
        hipSuccess)
        return PLSTM_EHIP;
    if ((long long)per_cu * device_info().cus < pl.blocks) return PLSTM_ENOTCORESIDENT;
    (void)hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl.lds);
    void *kargs[] = {&args};
    if (hipLaunchCooperativeKernel(fn, dim3(pl.blocks), dim3(kThreads), kargs, pl.lds, st) !=
        hipSuccess)
        return PLSTM_EHIP;
    return PLSTM_OK;
}

}  // namespace

bool sweep_fwd_supported(const Geom &g, int dtype)
{
    return dtype == PLSTM_F32 && g.O == kO && g.C >= 1 && g.C <= 4;
}

size_t sweep_fwd_ws(const Geom &g, bool training)
{
    Carve cv(nullptr);
    cv.take<float>((size_t)kDirs * g.N * g.V * kO);                 // h^d
    if (!training) cv.take<float>((size_t)kDirs * g.N * g.V * kO);  // c^d
    cv.take<int>(1024 + 1);                                          // flags + err
    return cv.off;
}

int sweep_fwd(const Geom &g, const float *x, const float *wx, const float *wh, const float *b,
              float *hd, float *cell, float *gates, int *flags, hipStream_t st)
{
    const DevInfo di = device_info();
    if (di.cus <= 0) return PLSTM_EHIP;
    const size_t lds_limit = (size_t)(di.max_lds > 0 ? di.max_lds : 65536) - 1024;
    const int budget = di.cus < 1024 ? di.cus : 1024;
    const Plan pl = make_plan(g, budget, g.C, lds_limit);
    if (pl.blocks > budget || pl.chunk_rows < 1) return PLSTM_EUNSUPPORTED;

    SweepArgs args;
    args.g = g;
    args.x = x; args.wx = wx; args.wh = wh; args.b = b;
    args.hd = hd; args.cell = cell; args.gates = gates;
    args.flags = flags;
    args.err = flags + 1024;
    for (int d = 0; d < kDirs; ++d) {
        args.nstrip[d] = pl.nstrip[d];
        args.first[d] = pl.first[d];
    }
    args.chunk_rows = pl.chunk_rows;
    args.max_w = pl.max_w;

    k_fill_zero<<<(1025 + 255) / 256, 256, 0, st>>>(flags, 1025);
    PLSTM_LAUNCH_CHECK();
    timing_begin("sweep_fwd_mfma", st);
    int rc;
    switch (g.C) {
    case 1: rc = launch_sweep<1>(pl, args, st); break;
    case 2: rc = launch_sweep<2>(pl, args, st); break;
    case 3: rc = launch_sweep<3>(pl, args, st); break;
    default: rc = launch_sweep<4>(pl, args, st); break;
    }
    timing_end(1, st);
    return rc;
}

}  // namespace plstm
