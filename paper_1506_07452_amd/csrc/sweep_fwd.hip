// Persistent MFMA forward sweep for O = 16 hidden units, C <= 4 input
// channels, fp32 (Section 2.3, Eq. (7)-(12); the sum of Eq. (13) follows in
// a separate pass).
//
// One cooperative launch runs all six directions (and all batch elements) at
// once.  The plane of each direction is cut into strips of whole rows x a few
// columns; one workgroup (16 waves, four per SIMD) owns one strip for the
// whole sweep.  A strip that fits LDS stays there for the whole sweep (h
// double-buffered, c in LDS, only the halo columns and x_t read per step);
// otherwise, per step:
//
//   for t in 0..T-1:
//     wait until the two neighbouring strips have published h_{t-1}
//     for each chunk of rows of the strip (sized to fit LDS):
//       stage h_{t-1} (chunk + 1-pixel halo) and the input plane x_t into LDS
//       each wave, per tile of 16 pixels:
//         A = bias + im2col(x_t) W_x + im2col(h_{t-1}) W_h   (v_mfma_f32_16x16x4f32)
//         gates, c_t = g i + c_{t-1} f, h_t = o tanh(c_t)    (in registers)
//         write h_t, c_t (and the gates when training) to global memory
//     publish: flag = t + 1 once the stores have completed
//
// The weight fragments (recurrent and input) and the bias live in LDS for
// the whole kernel; h of every plane stays in the per-direction volume in
// global memory, so a step only reads plane t-1 and writes plane t (no
// write-after-read hazard).  MFMA layout (16x16x4 f32, one block): lane l
// supplies A[m = l%16][k = l/16] and B[k = l/16][n = l%16] and receives
// D[4(l/16) + i][l%16], i = 0..3.  Gate-units are on M (M-tile g = gate g of
// the 16 units, the weights are the A operand) and pixels on N (B = im2col).
// The K index of a tap is permuted so that lane group q = l/16 takes hidden
// channels 4q..4q+3 of its pixel with one 16-byte LDS read; A uses the same
// permutation.  Every lane ends with all four gates of units 4q..4q+3 of
// pixel l%16, so the cell update needs no data exchange and its loads and
// stores are 16-byte vectors.
#include "common.h"
#include "coherent.h"
#include "sweep.h"
#include "strip_plan.h"
#include "timing.h"

namespace plstm {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kO = 16;
constexpr int kG = 4 * kO;
constexpr int kWaves = 16;         // four waves per SIMD: gate math of some overlaps the MFMAs of others
constexpr int kWhFloats = 9 * 4 * 64 * 4;   // recurrent A fragments in LDS
constexpr int kThreads = 64 * kWaves;
constexpr int kHS = 20;          // LDS floats per staged h pixel (16 + 4 pad)
constexpr int kWaitVmcnt0 = 0x0F70;   // s_waitcnt vmcnt(0), other counters unconstrained
constexpr int kBatch = 4;        // staging loads in flight per thread
constexpr int kCS = 20;          // LDS floats per cell state of a resident strip (16 + 4 pad)
constexpr int kResX = 4;         // x_t staging registers per thread (resident strips)

struct SweepArgs {
    Geom g;
    const float *x, *wx, *wh, *b;
    float *hd;          // [6][N][V][16] per-direction h^d
    float *cell;        // [6][N][V][16] c^d
    float *gates;       // [6][N][V][64] or null
    int *flags;         // [blocks] completed steps per strip
    int *err;           // set when a wait gives up
    int max_spin;       // polls before a wait gives up
    int wait_bias;      // added to the awaited step (0; failure-path test mode only)
    int nstrip[kDirs];  // strips per (direction, batch element)
    int first[kDirs];   // first block of direction d
    int chunk_rows[kDirs];  // rows staged per LDS chunk, per direction
    int max_w[kDirs];       // widest strip of each direction (LDS layout)
    int resident[kDirs];    // 1: strips of this direction stay in LDS
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

// Waits until the strip's neighbours have published `step` steps (bounded:
// a wait that never ends raises the error flag and gives up).  Their shared
// columns are then read at device coherence, so no cache invalidate is
// needed.
__device__ inline void wait_neighbours(const SweepArgs &a, int nb_lo, int nb_hi, int step)
{
    const int nb = threadIdx.x == 0 ? nb_lo : (threadIdx.x == 1 ? nb_hi : -1);
    if (nb >= 0) {
        int spins = 0;
        while (__hip_atomic_load(&a.flags[nb], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <
               step + a.wait_bias) {
            __builtin_amdgcn_s_sleep(1);
            if (++spins > a.max_spin) {
                __hip_atomic_store(a.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
            if ((spins & 1023) == 0 &&
                __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
                break;
        }
    }
}

// Publishes `step` completed steps of this strip.  The columns neighbours
// read are written at device coherence; callers make sure those stores have
// completed (every storing wave waited for vmcnt 0) before the flag goes up.
__device__ inline void publish(const SweepArgs &a, int step)
{
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __hip_atomic_store(&a.flags[blockIdx.x], step, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Gate pre-activations of one 16-pixel tile: bias + W_x im2col(x_t) +
// W_h im2col(h_{t-1}); `base` is the LDS pixel index of this lane's pixel in
// the staged (halo-padded) tile whose rows are `rs` and columns `cs` pixels
// apart.
template <int C>
__device__ __forceinline__ void tile_preact(const float *whs, const float *hsrc,
                                            const float *xs, const float *wxs, const float *bs,
                                            int base, int rs, int cs, const int *xoff, int q4,
                                            int lane, f4 (&acc)[4])
{
    constexpr int KXS = (9 * C + 3) / 4;
#pragma unroll
    for (int g = 0; g < 4; ++g) acc[g] = *(const f4 *)&bs[g * kO + 4 * q4];
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
        const int o = (tap / 3 - 1) * rs + (tap % 3 - 1) * cs;
        const f4 hv = *(const f4 *)&hsrc[(base + o) * kHS + 4 * q4];
        f4 w[4];
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) w[s2] = *(const f4 *)&whs[((tap * 4 + s2) * 64 + lane) * 4];
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(w[s2][g], hv[s2], acc[g], 0,
                                                            0, 0);
    }
#pragma unroll
    for (int ks = 0; ks < KXS; ++ks) {
        const float xv = (4 * ks + q4 < 9 * C) ? xs[base * C + xoff[ks]] : 0.0f;
        const f4 wxv = *(const f4 *)&wxs[(ks * 64 + lane) * 4];
#pragma unroll
        for (int g = 0; g < 4; ++g)
            acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(wxv[g], xv, acc[g], 0, 0, 0);
    }
}

// Gates, cell and hidden update of four units of one pixel (Eq. (7)-(12)).
__device__ __forceinline__ void lstm_cell(const f4 (&acc)[4], f4 cprev, bool has_prev, f4 &gi,
                                          f4 &gf, f4 &gg, f4 &go, f4 &cn, f4 &hn)
{
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        gi[i] = fsig(acc[0][i]);
        gf[i] = fsig(acc[1][i]);
        gg[i] = ftanh(acc[2][i]);
        go[i] = fsig(acc[3][i]);
        cn[i] = gg[i] * gi[i] + (has_prev ? cprev[i] : 0.0f) * gf[i];
        hn[i] = go[i] * ftanh(cn[i]);
    }
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
    float *wxs = smem;                       // [KXS][64 lanes][4 M-tiles] A fragments
    float *bs = wxs + KXS * 256;             // [64] bias
    const bool resident = a.resident[d] != 0;
    const int P = dg.P;
    // LDS pixel strides of a staged tile: chunked strips are row-major,
    // resident strips column-major (a tile then covers one or two columns,
    // so the columns next to a neighbour strip form their own tiles).
    const int rs = resident ? 1 : W2, cs = resident ? P + 2 : 1;

    // ---- recurrent weights as MFMA A fragments (resident for the sweep) ---
    const long long V = a.g.V;
    // Recurrent weights as MFMA A fragments in LDS: entry (tap, s, lane)
    // holds the four gates' weights of gate-unit lane%16 for hidden unit
    // 4 (lane/16) + s, one 16-byte read per k-step (LDS keeps the waves at
    // about 110 VGPRs, so four share a SIMD).
    float *whs = bs + kG;
    for (int e = threadIdx.x; e < 9 * 4 * 64; e += kThreads) {
        const int l = e & 63, s = (e >> 6) & 3, tap = e >> 8;
        const int lq = l >> 4, lc = l & 15;
        f4 v;
#pragma unroll
        for (int g = 0; g < 4; ++g)
            v[g] = a.wh[(((long long)d * kG + g * kO + lc) * kO + 4 * lq + s) * 9 + tap];
        *(f4 *)&whs[e * 4] = v;
    }
    // Input-convolution A fragments in LDS as well (they feed few MFMAs).
    int xoff[KXS];
#pragma unroll
    for (int ks = 0; ks < KXS; ++ks) {
        const int k = 4 * ks + q4;
        const int tap = k < 9 * C ? k / C : 0, c = k % C;   // padding lanes read tap 0
        xoff[ks] = k < 9 * C ? ((tap / 3 - 1) * rs + (tap % 3 - 1) * cs) * C + c : 0;
        if (wave == 0) {
            f4 w4;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int gn = g * kO + col;
                const float w = a.wx[(((long long)d * kG + gn) * C + c) * 9 + tap];
                w4[g] = k < 9 * C ? w : 0.0f;
            }
            *(f4 *)&wxs[(ks * 64 + lane) * 4] = w4;
        }
    }
    if (threadIdx.x < kG) bs[threadIdx.x] = a.b[d * kG + threadIdx.x];

    // Base pointers of this (direction, batch element); element offsets inside
    // a slice fit in 32 bits (V * 64 < 2^31 is checked at the boundary).
    const long long dn = ((long long)d * a.g.N + n) * V;
    float *const hd_dn = a.hd + dn * kO;
    // h^d of the slice as a buffer resource for the device-coherent accesses
    // of the columns shared with neighbour strips (this strip's first and
    // last columns and the halo columns beside them)
    const __amdgpu_buffer_rsrc_t hd_rs = coherent_rsrc(hd_dn, V * kO);
    auto is_shared_col = [&](int pc) {
        return (pc == q0 - 1) | (pc == q1) | ((pc == q0) & (nb_lo >= 0)) |
               ((pc == q1 - 1) & (nb_hi >= 0));
    };
    float *const cell_dn = a.cell + dn * kO;
    float *const gates_dn = a.gates ? a.gates + dn * kG : nullptr;
    const float *const x_n = a.x + (long long)n * V * C;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const float inv_w2 = 1.0f / (float)W2;

    if (resident) {
        // ================= resident strip: the whole strip in LDS ===========
        // h is double-buffered (h_{t-1} read, h_t written by the epilogue),
        // c stays in LDS, only the two halo columns come from global memory
        // each step and x_{t+1} is loaded while step t computes.  Pixels are
        // numbered column by column; the tiles touching a column next to a
        // neighbour strip run first and the step is published as soon as
        // they are stored, so neighbours seldom wait.
        const int P2 = P + 2;
        const int npl = P2 * W2;
        const int npx = P * TQ;
        const int nmt = (npx + 15) >> 4;
        float *hb0 = whs + kWhFloats;
        float *hb1 = hb0 + npl * kHS;
        float *xs = hb1 + npl * kHS;
        float *cb = xs + ((npl * C + 3) & ~3);     // [npx][kCS] cell states (16-byte aligned)
        int *order = (int *)(cb + npx * kCS);      // tile order, edge tiles first
        int *cnt = order + nmt;                    // edge tiles stored this step
        const float inv_p = 1.0f / (float)P;
        for (int e = threadIdx.x; e < 2 * npl * kHS; e += kThreads) hb0[e] = 0.0f;
        if (threadIdx.x == 0) {
            int k = 0;
            for (int pass = 0; pass < 2; ++pass)
                for (int mt = 0; mt < nmt; ++mt) {
                    const int c0 = (mt * 16) / P, c1 = min(mt * 16 + 15, npx - 1) / P;
                    const bool edge = (c0 == 0 && nb_lo >= 0) || (c1 == TQ - 1 && nb_hi >= 0);
                    if (edge == (pass == 0)) order[k++] = mt;
                }
            int ne = 0;
            for (int mt = 0; mt < nmt; ++mt) {
                const int c0 = (mt * 16) / P, c1 = min(mt * 16 + 15, npx - 1) / P;
                ne += ((c0 == 0 && nb_lo >= 0) || (c1 == TQ - 1 && nb_hi >= 0)) ? 1 : 0;
            }
            cnt[0] = 0;
            cnt[1] = ne;
        }
        // x_t staging registers (loaded one step ahead).  Threads walk the
        // staged plane row by row (coalesced in global memory) and store
        // into the column-major LDS copy.
        float xr[kResX];
        auto issue_x = [&](int splane) {
#pragma unroll
            for (int u = 0; u < kResX; ++u) {
                const int e = threadIdx.x + u * kThreads;
                const int pix = e / C, c = e - (e / C) * C;
                const int rr = fdiv_floor(pix, inv_w2);
                const int pr = rr - 1, pc = pix - rr * W2 + q0 - 1;
                const bool ok = e < npl * C && pr >= 0 && pr < P && pc >= 0 && pc < dg.Q;
                const int off = ok ? (splane + pr * sp + pc * sq) * C + c : 0;
                const float v = x_n[off];
                xr[u] = ok ? v : 0.0f;
            }
        };
        auto commit_x = [&]() {
#pragma unroll
            for (int u = 0; u < kResX; ++u) {
                const int e = threadIdx.x + u * kThreads;
                const int pix = e / C, c = e - (e / C) * C;
                const int rr = fdiv_floor(pix, inv_w2);
                if (e < npl * C) xs[((pix - rr * W2) * P2 + rr) * C + c] = xr[u];
            }
        };
        issue_x((dg.sign > 0 ? 0 : dg.T - 1) * ss);
        __syncthreads();
        const int n_edge = cnt[1];
        for (int t = 0; t < dg.T; ++t) {
            const int s = dg.sign > 0 ? t : dg.T - 1 - t;
            const int splane = s * ss;
            float *hprev = (t & 1) ? hb0 : hb1;      // h_{t-1}
            float *hcur = (t & 1) ? hb1 : hb0;       // h_t
            if (t > 0) {
                // halo columns of h_{t-1} from the neighbours
                wait_neighbours(a, nb_lo, nb_hi, t);
                __syncthreads();
                const int pplane = (s - dg.sign) * ss;
                for (int e = threadIdx.x; e < 2 * P * 4; e += kThreads) {
                    const int side = e / (P * 4), rem = e - side * P * 4;
                    const int r = rem >> 2, qd = rem & 3;
                    const int pc = side ? q1 : q0 - 1;
                    if (pc >= 0 && pc < dg.Q) {
                        const f4 v =
                            load_coherent(hd_rs, (pplane + r * sp + pc * sq) * kO + qd * 4);
                        *(f4 *)&hprev[((side ? TQ + 1 : 0) * P2 + r + 1) * kHS + qd * 4] = v;
                    }
                }
            }
            commit_x();
            __syncthreads();
            // One tile: contraction, cell update, stores (h_t to LDS for the
            // next step and to the volume for the neighbours and the sum).
            auto tile = [&](int mt) {
                const int pa = min(mt * 16 + col, npx - 1);     // this lane's pixel
                const int ca = fdiv_floor(pa, inv_p), ra = pa - ca * P;
                const int base = (ca + 1) * P2 + ra + 1;
                const int v = splane + ra * sp + (q0 + ca) * sq;
                const f4 cv = *(const f4 *)&cb[pa * kCS + 4 * q4];
                f4 acc[4];
                tile_preact<C>(whs, hprev, xs, wxs, bs, base, 1, P2, xoff, q4, lane, acc);
                f4 gi, gf, gg, go, cn, hn;
                lstm_cell(acc, cv, t > 0, gi, gf, gg, go, cn, hn);
                if (mt * 16 + col < npx) {
                    *(f4 *)&cb[pa * kCS + 4 * q4] = cn;
                    *(f4 *)&hcur[base * kHS + 4 * q4] = hn;
                    if (is_shared_col(q0 + ca))
                        store_coherent(hd_rs, v * kO + 4 * q4, hn);
                    else
                        *(f4 *)&hd_dn[v * kO + 4 * q4] = hn;
                    if (gates_dn) {
                        *(f4 *)&cell_dn[v * kO + 4 * q4] = cn;
                        float *gp = gates_dn + v * kG + 4 * q4;
                        *(f4 *)&gp[0] = gi;
                        *(f4 *)&gp[kO] = gf;
                        *(f4 *)&gp[2 * kO] = gg;
                        *(f4 *)&gp[3 * kO] = go;
                    }
                }
            };
            // Edge tiles first; once a wave's edge tile has reached L2 it
            // counts it, and the wave that stores the last one publishes.
            // The x_{t+1} prefetch goes out only after a wave's edge tiles,
            // so the store waits do not wait for it.
            int k = wave;
            for (; k < n_edge; k += kWaves) {
                tile(order[k]);
                __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
                if (lane == 0 && atomicAdd(cnt, 1) == n_edge - 1) publish(a, t + 1);
            }
            if (t + 1 < dg.T) issue_x((dg.sign > 0 ? t + 1 : dg.T - 2 - t) * ss);
            for (; k < nmt; k += kWaves) tile(order[k]);
            if (n_edge == 0) __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
            __syncthreads();
            if (threadIdx.x == 0) {
                if (n_edge == 0) publish(a, t + 1);
                cnt[0] = 0;
            }
        }
        return;
    }

    // ================= chunked strip: rows staged per step =================
    const int chunk_rows = a.chunk_rows[d];
    float *hs = whs + kWhFloats;
    float *xs = hs + (chunk_rows + 2) * (a.max_w[d] + 2) * kHS;
    const float inv_tq = 1.0f / (float)TQ;
    __syncthreads();
    for (int t = 0; t < dg.T; ++t) {
        const int s = dg.sign > 0 ? t : dg.T - 1 - t;
        const int sprev = s - dg.sign;
        if (t > 0) {
            wait_neighbours(a, nb_lo, nb_hi, t);
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
                        f4 v;
                        if (is_shared_col(pc))
                            v = load_coherent(hd_rs, off);
                        else
                            v = *(const f4 *)&hd_dn[off];
                        hv[u] = ok ? v : f4{0.0f, 0.0f, 0.0f, 0.0f};
                    }
                    {
                        const int pix = e / C, c = e % C;
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
                const int pa = min(mt * 16 + col, npx - 1);     // this lane's pixel
                const int ra = fdiv_floor(pa, inv_tq);
                const int base = (ra + 1) * W2 + (pa - ra * TQ) + 1;
                const int v = splane + (ra + r0) * sp + (pa - ra * TQ + q0) * sq;
                // c_{t-1} of this lane's units, loaded now so the load overlaps
                // the contraction below; at t = 0 there is no previous plane:
                // read (and discard) this plane's entry so the address stays
                // inside the slice.
                const f4 cv = *(const f4 *)&cell_dn[(v - splane + cplane) * kO + 4 * q4];
                // keep the load above the contraction (the scheduler would
                // otherwise sink it to its use and expose its latency)
                __builtin_amdgcn_sched_barrier(0);
                f4 acc[4];
                tile_preact<C>(whs, hs, xs, wxs, bs, base, W2, 1, xoff, q4, lane, acc);
                if (mt * 16 + col >= npx) continue;
                f4 gi, gf, gg, go, cn, hn;
                lstm_cell(acc, cv, t > 0, gi, gf, gg, go, cn, hn);
                *(f4 *)&cell_dn[v * kO + 4 * q4] = cn;
                if (is_shared_col(pa - ra * TQ + q0))
                    store_coherent(hd_rs, v * kO + 4 * q4, hn);
                else
                    *(f4 *)&hd_dn[v * kO + 4 * q4] = hn;
                if (gates_dn) {
                    float *gp = gates_dn + v * kG + 4 * q4;
                    *(f4 *)&gp[0] = gi;
                    *(f4 *)&gp[kO] = gf;
                    *(f4 *)&gp[2 * kO] = gg;
                    *(f4 *)&gp[3 * kO] = go;
                }
            }
            __syncthreads();
        }
        // ---- publish h_t -------------------------------------------------
        // Every wave waits until its own stores have completed, then one
        // thread raises the flag.
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if (threadIdx.x == 0) publish(a, t + 1);
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
    // wx fragments, bias, recurrent fragments
    m.fixed_bytes = (size_t)(((9 * C + 3) / 4) * 256 + kG + kWhFloats) * sizeof(float);
    m.px_bytes = (size_t)(kHS + C) * sizeof(float);                     // h + x per pixel
    m.c_sync = 3.0;
    m.c_tile = 3.2;
    m.c_stage0 = 1.0;
    m.c_stage_px = 0.0031;
    m.allow_resident = true;
    m.res_px_bytes = (size_t)(2 * kHS + C) * sizeof(float);   // two h buffers + x
    m.res_own_bytes = (size_t)kCS * sizeof(float) + 1 * sizeof(int);   // c + tile order
    m.res_fixed_bytes = 16 * sizeof(int);                      // counters + alignment of c
    m.res_max_staged = kResX * kThreads / C;                   // x_t fits the registers
    m.c_res_step = 1.6;
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
    // bf16 storage: the caller widens x and the parameters to fp32 first
    return (dtype == PLSTM_F32 || dtype == PLSTM_BF16) && g.nd == kDirs && g.KP == 3 &&
           g.KQ == 3 && g.O == kO && g.C >= 1 && g.C <= 4;
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
              float *hd, float *cell, float *gates, int *flags, hipStream_t st,
              bool allow_resident)
{
    const DevInfo di = device_info();
    if (di.cus <= 0) return PLSTM_EHIP;
    const size_t lds_limit = (size_t)(di.max_lds > 0 ? di.max_lds : 65536) - 1024;
    const int budget = di.cus < 1024 ? di.cus : 1024;
    StripCostModel model = fwd_model(g.C);
    model.allow_resident = allow_resident;
    const Plan pl = make_plan(g, budget, model, lds_limit);
    if (pl.blocks > budget) return PLSTM_EUNSUPPORTED;
    for (int d = 0; d < kDirs; ++d) {
        if (pl.chunk_rows[d] < 1) return PLSTM_EUNSUPPORTED;
        // a resident strip's x_t plane must fit the staging registers
        if (pl.resident[d] &&
            (long long)(g.dir[d].P + 2) * (pl.max_w[d] + 2) * g.C > (long long)kResX * kThreads)
            return PLSTM_EUNSUPPORTED;
    }

    SweepArgs args;
    args.g = g;
    args.x = x; args.wx = wx; args.wh = wh; args.b = b;
    args.hd = hd; args.cell = cell; args.gates = gates;
    args.flags = flags;
    args.err = flags + 1024;
    args.max_spin = g_wait_spin_limit;
    args.wait_bias = g_wait_bias;
    for (int d = 0; d < kDirs; ++d) {
        args.nstrip[d] = pl.nstrip[d];
        args.first[d] = pl.first[d];
    }
    for (int d = 0; d < kDirs; ++d) {
        args.chunk_rows[d] = pl.chunk_rows[d];
        args.max_w[d] = pl.max_w[d];
        args.resident[d] = pl.resident[d];
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
    if (rc != PLSTM_OK) return rc;
    PoisonList poison;
    poison.ptr[0] = hd;
    poison.count[0] = (long long)saved_state_count(g);
    return wait_check(args.err, poison, st);
}

}  // namespace plstm
