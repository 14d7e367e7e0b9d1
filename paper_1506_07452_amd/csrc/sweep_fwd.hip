// Persistent MFMA forward sweep for O = 16 hidden units, C <= 4 input
// channels, fp32 (Section 2.3, Eq. (7)-(12); the sum of Eq. (13) follows in
// a separate pass).
//
// One cooperative launch runs all six directions (and all batch elements) at
// once.  The plane of each direction is cut into strips of whole rows x a few
// columns; one workgroup (8 waves, two per SIMD) owns one strip for the whole
// sweep:
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
// The recurrent weights live in VGPRs as MFMA B fragments for the whole
// kernel (the input-convolution fragments in LDS); h of
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
#include "strip_plan.h"
#include "timing.h"

namespace plstm {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kO = 16;
constexpr int kG = 4 * kO;
constexpr int kWaves = 8;          // two waves per SIMD: one computes gates while the other runs MFMAs
constexpr int kThreads = 64 * kWaves;
constexpr int kHS = 20;          // LDS floats per staged h pixel (16 + 4 pad)
constexpr int kMaxSpin = 1 << 21;
constexpr int kWaitVmcnt0 = 0x0F70;   // s_waitcnt vmcnt(0), other counters unconstrained
constexpr int kBatch = 4;        // staging loads in flight per thread

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
    int chunk_rows[kDirs];  // rows staged per LDS chunk, per direction
    int max_w[kDirs];       // widest strip of each direction (LDS layout)
};

// Gate nonlinearities from exp and the hardware reciprocal (1 ulp each):
// sigma(a) = 1 / (1 + e^-a);  tanh(a) = 1 - 2 / (e^{2a} + 1), which saturates
// to +-1 at +-inf.
__device__ inline float frcp(float v) { return __builtin_amdgcn_rcpf(v); }
__device__ inline float fsig(float a) { return frcp(1.0f + __expf(-a)); }
__device__ inline float ftanh(float a) { return 1.0f - 2.0f * frcp(__expf(2.0f * a) + 1.0f); }

// floor(i / w) for 0 <= i < 2^20, w >= 1, from a float reciprocal: the
// fraction of (i + 0.5) / w is at least 0.5 / w away from an integer, while the
// product's rounding error is below (i / w) 2^-23 <= 0.125 / w, so the
// truncation is exact.
__device__ inline int fdiv_floor(int i, float inv_w) {
    return (int)(((float)i + 0.5f) * inv_w);
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
    constexpr int KXS = (9 * C + 3) / 4;    // MFMA k-steps of the input convolution
    float *wxs = smem;                       // [KXS][64 lanes][4 N-tiles] B fragments
    const int chunk_rows = a.chunk_rows[d];
    float *hs = smem + KXS * 256;
    float *xs = hs + (chunk_rows + 2) * (a.max_w[d] + 2) * kHS;

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
    // Input-convolution B fragments go to LDS (they feed few MFMAs; keeping
    // them out of VGPRs lets two waves share a SIMD).
    int xoff[KXS];
#pragma unroll
    for (int ks = 0; ks < KXS; ++ks) {
        const int k = 4 * ks + q4;
        const int tap = k < 9 * C ? k / C : 0, c = k % C;   // padding lanes read tap 0
        xoff[ks] = k < 9 * C ? ((tap / 3 - 1) * W2 + (tap % 3 - 1)) * C + c : 0;
        if (wave == 0) {
            f4 w4;
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                const int gn = nt * kO + col;
                const float w = a.wx[(((long long)d * kG + gn) * C + c) * 9 + tap];
                w4[nt] = k < 9 * C ? w : 0.0f;
            }
            *(f4 *)&wxs[(ks * 64 + lane) * 4] = w4;
        }
    }
    __syncthreads();
    float bias[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) bias[nt] = a.b[d * kG + nt * kO + col];

    // Base pointers of this (direction, batch element); element offsets inside
    // a slice fit in 32 bits (V * 64 < 2^31 is checked at the boundary).
    const long long dn = ((long long)d * a.g.N + n) * V;
    float *const hd_dn = a.hd + dn * kO;
    float *const cell_dn = a.cell + dn * kO;
    float *const gates_dn = a.gates ? a.gates + dn * kG : nullptr;
    const float *const x_n = a.x + (long long)n * V * C;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const float inv_tq = 1.0f / (float)TQ, inv_w2 = 1.0f / (float)W2;

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
        const int splane = s * ss, sprev_plane = sprev * ss;
        const int cplane = t > 0 ? sprev_plane : splane;
        for (int r0 = 0; r0 < dg.P; r0 += chunk_rows) {
            const int CH = min(chunk_rows, dg.P - r0);
            const int npl = (CH + 2) * W2;            // staged pixels incl. halo
            // ---- stage h_{t-1} and x_t (zero outside the plane) ----------
            // Branch-free loads from clamped addresses, kBatch per thread in
            // flight before the LDS stores: one memory round trip per batch.
            const int nh = npl * 4, nx = npl * C;
            for (int e0 = threadIdx.x; e0 < max(nh, nx); e0 += kThreads * kBatch) {
                f4 hv[kBatch];
                float xv[kBatch];
#pragma unroll
                for (int u = 0; u < kBatch; ++u) {
                    const int e = e0 + u * kThreads;
                    {
                        const int pix = e >> 2, qd = e & 3;
                        const int rr = fdiv_floor(pix, inv_w2);
                        const int pr = rr + r0 - 1, pc = pix - rr * W2 + q0 - 1;
                        const bool ok = e < nh && t > 0 && pr >= 0 && pr < dg.P && pc >= 0 &&
                                        pc < dg.Q;
                        const int off = ok ? (sprev_plane + pr * sp + pc * sq) * kO + qd * 4 : 0;
                        const f4 v = *(const f4 *)&hd_dn[off];
                        hv[u] = ok ? v : f4{0.0f, 0.0f, 0.0f, 0.0f};
                    }
                    {
                        const int pix = e / C, c = e - (e / C) * C;
                        const int rr = fdiv_floor(pix, inv_w2);
                        const int pr = rr + r0 - 1, pc = pix - rr * W2 + q0 - 1;
                        const bool ok = e < nx && pr >= 0 && pr < dg.P && pc >= 0 && pc < dg.Q;
                        const int off = ok ? (splane + pr * sp + pc * sq) * C + c : 0;
                        const float v = x_n[off];
                        xv[u] = ok ? v : 0.0f;
                    }
                }
#pragma unroll
                for (int u = 0; u < kBatch; ++u) {
                    const int e = e0 + u * kThreads;
                    if (e < nh) *(f4 *)&hs[(e >> 2) * kHS + (e & 3) * 4] = hv[u];
                    if (e < nx) xs[e] = xv[u];
                }
            }
            __syncthreads();
            // ---- 16-pixel tiles -----------------------------------------
            const int npx = CH * TQ;
            const int nmt = (npx + 15) >> 4;
            for (int mt = wave; mt < nmt; mt += kWaves) {
                const int pa = min(mt * 16 + col, npx - 1);     // this lane's A row
                const int ra = fdiv_floor(pa, inv_tq);
                const int base = (ra + 1) * W2 + (pa - ra * TQ) + 1;
                // Output rows 4 q4 + i of this lane; c_{t-1} is loaded now so
                // the load overlaps the contraction below.
                float cprev[4];
                int vout[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int px = min(mt * 16 + 4 * q4 + i, npx - 1);
                    const int rr = fdiv_floor(px, inv_tq);
                    vout[i] = splane + (rr + r0) * sp + (px - rr * TQ + q0) * sq;
                    // at t = 0 there is no previous plane: read (and discard)
                    // this plane's entry so the address stays inside the slice
                    const float cv = cell_dn[(vout[i] - splane + cplane) * kO + col];
                    cprev[i] = t > 0 ? cv : 0.0f;
                }
                // keep the loads above the contraction (the scheduler would
                // otherwise sink them to their use and expose their latency)
                __builtin_amdgcn_sched_barrier(0);
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
                    const f4 bxv = *(const f4 *)&wxs[(ks * 64 + lane) * 4];
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt)
                        acc[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bxv[nt], acc[nt],
                                                                     0, 0, 0);
                }
                // ---- gates and cell update: rows 4 q4 + i, unit col ------
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (mt * 16 + 4 * q4 + i >= npx) continue;
                    const int v = vout[i];
                    const float gi = fsig(acc[0][i]);
                    const float gf = fsig(acc[1][i]);
                    const float gg = ftanh(acc[2][i]);
                    const float go = fsig(acc[3][i]);
                    const float c = gg * gi + cprev[i] * gf;
                    cell_dn[v * kO + col] = c;
                    hd_dn[v * kO + col] = go * ftanh(c);
                    if (gates_dn) {
                        float *gp = gates_dn + v * kG + col;
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
        // Every wave waits until its own stores have reached L2, then one
        // thread writes L2 back (release at agent scope) and raises the flag:
        // one cache writeback per workgroup and step instead of one per wave.
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if (threadIdx.x == 0) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");   // L2 writeback
            __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);             // ... completed
            __hip_atomic_store(&a.flags[blockIdx.x], t + 1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

__global__ void k_fill_zero(int *p, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

// ---- launch planning ------------------------------------------------------
StripCostModel fwd_model(int C)
{
    StripCostModel m;
    m.fixed_bytes = (size_t)((9 * C + 3) / 4) * 256 * sizeof(float);   // wx fragments
    m.px_bytes = (size_t)(kHS + C) * sizeof(float);                     // h + x per pixel
    m.c_sync = 3.0;
    m.c_tile = 3.2;
    m.c_stage0 = 1.0;
    m.c_stage_px = 0.0031;
    return m;
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
    if (!training) {
        cv.take<float>(saved_state_count(g));   // h^d
        cv.take<float>(saved_state_count(g));   // c^d
    }
    cv.take<int>(1024 + 1);                     // flags + err
    return cv.off;
}

int sweep_fwd(const Geom &g, const float *x, const float *wx, const float *wh, const float *b,
              float *hd, float *cell, float *gates, int *flags, hipStream_t st)
{
    const DevInfo di = device_info();
    if (di.cus <= 0) return PLSTM_EHIP;
    const size_t lds_limit = (size_t)(di.max_lds > 0 ? di.max_lds : 65536) - 1024;
    const int budget = di.cus < 1024 ? di.cus : 1024;
    const Plan pl = make_plan(g, budget, fwd_model(g.C), lds_limit);
    if (pl.blocks > budget) return PLSTM_EUNSUPPORTED;
    for (int d = 0; d < kDirs; ++d)
        if (pl.chunk_rows[d] < 1) return PLSTM_EUNSUPPORTED;

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
    for (int d = 0; d < kDirs; ++d) {
        args.chunk_rows[d] = pl.chunk_rows[d];
        args.max_w[d] = pl.max_w[d];
    }

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
