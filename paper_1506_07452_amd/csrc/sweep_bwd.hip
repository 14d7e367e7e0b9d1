// Backward of the layer for O = 16 hidden units, fp32: back-propagation
// through the six sweeps (the chain rule through Section 2.3, Eq. (7)-(13),
// in reverse plane order) and the parameter gradients.
//
// (1) k_sweep_bwd, persistent, one cooperative launch for all directions, on
//     the forward's strip decomposition.  For plane t (last to first):
//       gh   = dL/dh[plane t] + sum_taps dA_{t+1}[p - tap] W_h^T      (MFMA)
//       gc   = gh o (1 - tanh^2 c_t) + gc_{t+1} f_{t+1}
//       dA_o = gh tanh(c_t) o (1 - o)     dA_i = gc g i (1 - i)
//       dA_g = gc i (1 - g^2)             dA_f = gc c_{t-1} f (1 - f)
//     The transposed 3x3 convolution is an MFMA contraction of K = 9 x 64
//     (tap, gate-unit) with units on M and pixels on N: lane l takes pixel
//     l%16 and gate l/16 (16 units = 4 LDS reads of 16 bytes per tap) for the
//     B operand, the transposed recurrent weights are the A operand, resident
//     in LDS, and each lane ends with four consecutive units of one
//     pixel, so every epilogue load and store is a 16-byte vector.  The
//     product gc_t f_t is what plane t - 1 needs, so that is what is kept.
//     dA of every voxel is kept for (2) and for dL/dx.
// (2) k_wgrad_rows: dW = sum over voxels of dA (x) [im2col(h_{t-1}),
//     im2col(x_t), 1], a register-streamed implicit GEMM (see there), and
//     (3) k_wgrad_reduce sums the per-wave partials in a fixed order.
#include "common.h"
#include "coherent.h"
#include "strip_plan.h"
#include "sweep.h"
#include "timing.h"

namespace plstm {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kO = 16;
constexpr int kG = 4 * kO;
constexpr int kWaves = 16;             // four waves per SIMD
constexpr int kWaFloats = 9 * 4 * 64 * 4;  // W_h^T fragments in LDS
constexpr int kThreads = 64 * kWaves;
// A staged dA pixel is 64 floats in LDS; its 16-byte chunk c sits at
// position c ^ (pixel & 15), so the 16 pixels a read instruction touches
// hit 16 different bank groups.
__device__ inline int swz(int c, int pix) { return c ^ (pix & 15); }
constexpr int kOutOfRange = 0x7ffffff0;    // buffer offset past any resource: reads zero
typedef __attribute__((address_space(3))) void lds_void;
constexpr int kWaitVmcnt0 = 0x0F70;   // s_waitcnt vmcnt(0), other counters unconstrained

__device__ inline float frcp(float v) { return __builtin_amdgcn_rcpf(v); }

__device__ inline float ftanh(float a) { return 1.0f - 2.0f * frcp(__expf(2.0f * a) + 1.0f); }
// floor(i / w) for 0 <= i < 2^20 (see the forward sweep for the error bound)
__device__ inline int fdiv_floor(int i, float inv_w) { return (int)(((float)i + 0.5f) * inv_w); }

struct BwdArgs {
    Geom g;
    const float *wh;
    const float *gates, *cell;   // saved forward activations [6][N][V][64], [6][N][V][16]
    const float *dh;             // dL/dh [N][V][16]
    float *dA;                   // [6][N][V][64] gate pre-activation gradients
    float *gcf;                  // [6][N][V][16] dL/dc_t * f_t, carried to plane t - 1
    int *flags, *err;
    int max_spin;                // polls before a wait gives up
    int wait_bias;               // added to the awaited step (0; failure-path test mode only)
    int nstrip[kDirs], first[kDirs], chunk_rows[kDirs], max_w[kDirs];
    int resident[kDirs];         // 1: the strip's dA stays in LDS for the sweep
};

// Epilogue operands of one tile (this lane's pixel, units 4 q4 .. 4 q4 + 3).
struct BwdEpi {
    f4 dh, gi, gf, gg, go, c, gcfn, cp;
};

// sum over taps of dA_{t+1}[p - tap] W_h^T for one 16-pixel tile, on the
// MFMA: `base` is the lane's LDS pixel, whose row and column neighbours are
// `rs` and `cs` LDS pixels apart.  The K loop runs in quarters of a tap
// (quarter j = 4 tap + s: gate-units 16 q4 + 4 s .. + 3 of the lane's pixel
// as B, the matching W_h^T fragment as A, four MFMAs); each quarter's two LDS
// reads are issued three quarters (twelve MFMAs) before their use, in a
// ring of four register slots, so a wave alone keeps the matrix unit busy.
__device__ __forceinline__ void contract_bwd(const float *as, const float *was, int base, int rs,
                                             int cs, int q4, int lane, f4 (&acc)[4])
{
    constexpr int kQuarters = 36;
    constexpr int kAhead = 2;
    f4 bq[kAhead + 1], aq[kAhead + 1];
    auto load = [&](int j) {
        const int tap = j >> 2, sq = j & 3;
        // h_t at pixel p fed A_{t+1} at p - (tap offset)
        const int pp = base - ((tap / 3 - 1) * rs + (tap % 3 - 1) * cs);
        bq[j % (kAhead + 1)] = *(const f4 *)&as[pp * kG + 4 * swz(4 * q4 + sq, pp)];
        aq[j % (kAhead + 1)] = *(const f4 *)&was[((tap * 4 + sq) * 64 + lane) * 4];
    };
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[k] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int j = 0; j < kAhead; ++j) load(j);
#pragma unroll
    for (int j = 0; j < kQuarters; ++j) {
        if (j + kAhead < kQuarters) load(j + kAhead);
        // keep the reads ahead of this quarter's MFMAs
        __builtin_amdgcn_sched_barrier(0);
        const int sl = j % (kAhead + 1);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(aq[sl][i], bq[sl][i], acc[i], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
    }
}

__global__ void __launch_bounds__(kThreads, 1) k_sweep_bwd(BwdArgs a)
{
    extern __shared__ float smem[];
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
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int q4 = lane >> 4, col = lane & 15;
    const int chunk_rows = a.chunk_rows[d];
    // A fragments of W_h^T in LDS (registers stay free for four waves per
    // SIMD): entry (tap, s4, lane) holds, for lane l, the gate-units
    // 16 (l/16) + 4 s4 .. + 3 of output unit l%16; the tap's K index
    // k = (s, q4) -> gate-unit 16 q4 + s.  The first staging barrier orders
    // these stores before their reads.
    float *was = smem;
    float *as = smem + kWaFloats;
    for (int e = threadIdx.x; e < 9 * 4 * 64; e += kThreads) {
        const int l = e & 63, s4 = (e >> 6) & 3, tap = e >> 8;
        const int lq = l >> 4, lc = l & 15;
        f4 v;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            v[j] = a.wh[(((long long)d * kG + 16 * lq + 4 * s4 + j) * kO + lc) * 9 + tap];
        *(f4 *)&was[e * 4] = v;
    }

    const long long V = a.g.V;
    const long long dn = ((long long)d * a.g.N + n) * V;
    const float *const gates_dn = a.gates + dn * kG;
    const float *const cell_dn = a.cell + dn * kO;
    float *const dA_dn = a.dA + dn * kG;
    // the slice as a buffer resource for the device-coherent accesses
    // (its byte size fits 32 bits: checked on the host)
    const __amdgpu_buffer_rsrc_t dA_rs = coherent_rsrc(dA_dn, V * kG);
    float *const gcf_dn = a.gcf + dn * kO;
    const float *const dh_n = a.dh + (long long)n * V * kO;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const float inv_tq = 1.0f / (float)TQ, inv_w2 = 1.0f / (float)W2;
    // Columns that pass between neighbouring strips (this strip's first and
    // last, and the halo columns beside them).  Their dA is stored and loaded
    // at device coherence (write-through / read-through at agent scope, the
    // accesses relaxed agent-scope atomics use), so a strip's step needs no
    // L2 writeback before its flag and no L2 invalidate after waiting: once a
    // strip's coherent stores have completed (vmcnt) its flag goes up.
    auto is_shared_col = [&](int pc) {
        return (pc == q0 - 1) | (pc == q1) | ((pc == q0) & (nb_lo >= 0)) |
               ((pc == q1 - 1) & (nb_hi >= 0));
    };

    if (a.resident[d]) {
        // ============ resident strip: dA of the whole strip stays in LDS ============
        // dA_t overwrites dA_{t+1} in place: each wave keeps its tiles' dA in
        // registers until every wave's contraction has read dA_{t+1} (one
        // barrier), then writes them.  Only the two halo columns come from
        // the neighbours each step.  Pixels are numbered column by column
        // (LDS pixel (column + 1) (P + 2) + row + 1); the tiles touching a
        // column next to a neighbour strip run first and the step is
        // published as soon as they are stored.  At most two tiles per wave
        // (checked on the host).
        const int P = dg.P, P2 = P + 2;
        const int npl = P2 * W2;
        const int npx = P * TQ;
        const int nmt = (npx + 15) >> 4;
        int *order = (int *)(as + (size_t)npl * kG);   // tile order, edge tiles first
        int *cnt = order + nmt;                         // edge tiles stored this step
        const float inv_p = 1.0f / (float)P;
        for (int e = threadIdx.x; e < npl * (kG / 4); e += kThreads)
            *(f4 *)&as[e * 4] = f4{0.0f, 0.0f, 0.0f, 0.0f};   // dA_T = 0, halo rows
        if (threadIdx.x == 0) {
            int k = 0, ne = 0;
            for (int pass = 0; pass < 2; ++pass)
                for (int mt = 0; mt < nmt; ++mt) {
                    const int c0 = (mt * 16) / P, c1 = min(mt * 16 + 15, npx - 1) / P;
                    const bool edge = (c0 == 0 && nb_lo >= 0) || (c1 == TQ - 1 && nb_hi >= 0);
                    if (edge == (pass == 0)) order[k++] = mt;
                    ne += (pass == 0 && edge) ? 1 : 0;
                }
            cnt[0] = 0;
            cnt[1] = ne;
        }
        __syncthreads();
        const int n_edge = cnt[1];
        // A lane handles the same pixel of its tiles at every step, so it
        // keeps (gc f)_t for the next step and the c_{t-1} it loaded, which is
        // the next step's c_t, in registers: neither is loaded again and gc f
        // is never stored.
        f4 carry_gcf[2], carry_c[2];
#pragma unroll
        for (int it = 0; it < 2; ++it) carry_gcf[it] = carry_c[it] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        for (int r = 0; r < dg.T; ++r) {
            const int t = dg.T - 1 - r;
            const int s = dg.sign > 0 ? t : dg.T - 1 - t;
            const bool has_next = t + 1 < dg.T, has_prev = t > 0;
            const int splane = s * ss;
            const int nplane = has_next ? (s + dg.sign) * ss : splane;
            const int pplane = has_prev ? (s - dg.sign) * ss : splane;
            if (r > 0) {
                // ---- the neighbours' edge columns of dA_{t+1} -> halo columns
                const int nb = threadIdx.x == 0 ? nb_lo : (threadIdx.x == 1 ? nb_hi : -1);
                if (nb >= 0) {
                    int spins = 0;
                    while (__hip_atomic_load(&a.flags[nb], __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT) < r + a.wait_bias) {
                        __builtin_amdgcn_s_sleep(1);
                        if (++spins > a.max_spin) {
                            __hip_atomic_store(a.err, 1, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                            break;
                        }
                        if ((spins & 1023) == 0 &&
                            __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
                            break;
                    }
                }
                __syncthreads();
                // One instruction moves four consecutive rows of a halo
                // column (lane l: chunk position l%16 of row 4 j + l/16);
                // lanes past the last row are inactive, so the halo rows
                // above and below the plane keep their zeros.
                const int nslot = (P + 3) >> 2;
                for (int i = wave; i < 2 * nslot; i += kWaves) {
                    const int side = i >= nslot ? 1 : 0;
                    const int j = i - side * nslot;
                    if ((side ? nb_hi : nb_lo) < 0) continue;
                    const int row = 4 * j + (lane >> 4);
                    const int lcol = side ? TQ + 1 : 0;
                    const int pix = lcol * P2 + 1 + row;
                    const int pc = side ? q1 : q0 - 1;
                    const int boff =
                        ((nplane + row * sp + pc * sq) * kG + (col ^ (pix & 15)) * 4) *
                        (int)sizeof(float);
                    lds_void *dst = (lds_void *)&as[(size_t)(lcol * P2 + 1 + 4 * j) * kG];
                    if (row < P)
                        __builtin_amdgcn_raw_ptr_buffer_load_lds(dA_rs, dst, 16, boff, 0, 0,
                                                                 kCachePolicySC1);
                }
                __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
                __syncthreads();
            }
            f4 hold[2][4];
            int hbase[2];
#pragma unroll
            for (int it = 0; it < 2; ++it) {
                const int k = wave + it * kWaves;
                hbase[it] = -1;
                if (k < nmt) {
                    const int mt = order[k];
                    const int pa = min(mt * 16 + col, npx - 1);
                    const int ca = fdiv_floor(pa, inv_p), ra = pa - ca * P;
                    const int base = (ca + 1) * P2 + ra + 1;
                    const int vo = splane + ra * sp + (ca + q0) * sq;
                    const bool shared = is_shared_col(ca + q0);
                    BwdEpi e;
                    const int vop = vo - splane + pplane;
                    e.dh = *(const f4 *)&dh_n[vo * kO + 4 * q4];
                    e.gi = *(const f4 *)&gates_dn[vo * kG + 0 * kO + 4 * q4];
                    e.gf = *(const f4 *)&gates_dn[vo * kG + 1 * kO + 4 * q4];
                    e.gg = *(const f4 *)&gates_dn[vo * kG + 2 * kO + 4 * q4];
                    e.go = *(const f4 *)&gates_dn[vo * kG + 3 * kO + 4 * q4];
                    e.c = r == 0 ? *(const f4 *)&cell_dn[vo * kO + 4 * q4] : carry_c[it];
                    e.gcfn = carry_gcf[it];
                    e.cp = *(const f4 *)&cell_dn[vop * kO + 4 * q4];
                    __builtin_amdgcn_sched_barrier(0);
                    f4 acc[4];
                    contract_bwd(as, was, base, 1, P2, q4, lane, acc);
                    f4 dAi, dAf, dAg, dAo, gcf;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float gh = acc[0][i] + acc[1][i] + acc[2][i] + acc[3][i] + e.dh[i];
                        const float tc = ftanh(e.c[i]);
                        const float gcs = gh * e.go[i] * (1.0f - tc * tc) +
                                          (has_next ? e.gcfn[i] : 0.0f);
                        const float cprev = has_prev ? e.cp[i] : 0.0f;
                        gcf[i] = gcs * e.gf[i];
                        dAi[i] = gcs * e.gg[i] * e.gi[i] * (1.0f - e.gi[i]);
                        dAf[i] = gcs * cprev * e.gf[i] * (1.0f - e.gf[i]);
                        dAg[i] = gcs * e.gi[i] * (1.0f - e.gg[i] * e.gg[i]);
                        dAo[i] = gh * tc * e.go[i] * (1.0f - e.go[i]);
                    }
                    const int o4 = vo * kG + 4 * q4;
                    if (shared) {
                        store_coherent(dA_rs, o4 + 0 * kO, dAi);
                        store_coherent(dA_rs, o4 + 1 * kO, dAf);
                        store_coherent(dA_rs, o4 + 2 * kO, dAg);
                        store_coherent(dA_rs, o4 + 3 * kO, dAo);
                    } else {
                        float *dst = &dA_dn[o4];
                        *(f4 *)&dst[0 * kO] = dAi;
                        *(f4 *)&dst[1 * kO] = dAf;
                        *(f4 *)&dst[2 * kO] = dAg;
                        *(f4 *)&dst[3 * kO] = dAo;
                    }
                    carry_gcf[it] = gcf;
                    carry_c[it] = e.cp;
                    hold[it][0] = dAi;
                    hold[it][1] = dAf;
                    hold[it][2] = dAg;
                    hold[it][3] = dAo;
                    hbase[it] = base;
                    if (k < n_edge) {
                        // this edge tile's coherent stores have completed:
                        // count it; the wave that counts the last publishes
                        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
                        if (lane == 0 && atomicAdd(cnt, 1) == n_edge - 1)
                            __hip_atomic_store(&a.flags[blockIdx.x], r + 1, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                    }
                }
            }
            // every contraction has read dA_{t+1}: overwrite it with dA_t
            __syncthreads();
#pragma unroll
            for (int it = 0; it < 2; ++it) {
                if (hbase[it] >= 0) {
                    const int pb = hbase[it];
#pragma unroll
                    for (int g = 0; g < 4; ++g)
                        *(f4 *)&as[pb * kG + 4 * swz(4 * g + q4, pb)] = hold[it][g];
                }
            }
            if (threadIdx.x == 0) {
                if (n_edge == 0)
                    __hip_atomic_store(&a.flags[blockIdx.x], r + 1, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                cnt[0] = 0;
            }
            // the next step's first barrier orders these LDS writes before
            // its contractions
        }
        return;
    }

    for (int r = 0; r < dg.T; ++r) {
        const int t = dg.T - 1 - r;                   // plane processed at this step
        const int s = dg.sign > 0 ? t : dg.T - 1 - t;
        const bool has_next = t + 1 < dg.T, has_prev = t > 0;
        // ---- wait for the neighbours' dA_{t+1} --------------------------
        if (r > 0) {
            const int nb = threadIdx.x == 0 ? nb_lo : (threadIdx.x == 1 ? nb_hi : -1);
            if (nb >= 0) {
                int spins = 0;
                while (__hip_atomic_load(&a.flags[nb], __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT) < r + a.wait_bias) {
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
            __syncthreads();
        }
        const int splane = s * ss;
        const int nplane = has_next ? (s + dg.sign) * ss : splane;   // in-slice when read
        const int pplane = has_prev ? (s - dg.sign) * ss : splane;
        for (int r0 = 0; r0 < dg.P; r0 += chunk_rows) {
            const int CH = min(chunk_rows, dg.P - r0);
            const int npl = (CH + 2) * W2;
            // ---- stage dA_{t+1} (chunk + halo) straight into LDS ------------
            // Direct-to-LDS buffer loads (no registers, all in flight at
            // once): one instruction moves 4 pixels, lane l the 16-byte chunk
            // at position l%16 of pixel 4 i + l/16, which holds its chunk
            // (l%16) ^ (pixel & 15) (see `swz`).  Off-plane pixels, the halo
            // past the volume and the plane after the last get an
            // out-of-range offset and the hardware writes zeros.
            const int nslots = (npl + 3) >> 2;
            for (int i = wave; i < nslots; i += kWaves) {
                const int pix = 4 * i + (lane >> 4);
                const int chunk = col ^ (pix & 15);
                const int rr = fdiv_floor(pix, inv_w2);
                const int pr = rr + r0 - 1, pc = pix - rr * W2 + q0 - 1;
                const bool ok = has_next & (pr >= 0) & (pr < dg.P) & (pc >= 0) & (pc < dg.Q);
                const int boff =
                    ok ? ((nplane + pr * sp + pc * sq) * kG + chunk * 4) * (int)sizeof(float)
                       : kOutOfRange;
                lds_void *dst = (lds_void *)&as[i * 4 * kG];
                if (pix < npl) {
                    if (is_shared_col(pc))   // read at device coherence (written that way)
                        __builtin_amdgcn_raw_ptr_buffer_load_lds(dA_rs, dst, 16, boff, 0, 0,
                                                                 kCachePolicySC1);
                    else
                        __builtin_amdgcn_raw_ptr_buffer_load_lds(dA_rs, dst, 16, boff, 0, 0, 0);
                }
            }
            __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
            __syncthreads();
            // ---- 16-pixel tiles ------------------------------------------
            // Each tile's epilogue operands are loaded before its contraction.
            // Lanes past the chunk redo its last pixel (the same values to
            // the same addresses).
            const int npx = CH * TQ;
            const int nmt = (npx + 15) >> 4;
            auto pixel = [&](int mt, int &base, int &vo, bool &shared) {
                const int pb = min(mt * 16 + col, npx - 1);
                const int rb = fdiv_floor(pb, inv_tq);
                const int cb = pb - rb * TQ;
                base = (rb + 1) * W2 + cb + 1;
                vo = splane + (rb + r0) * sp + (cb + q0) * sq;
                shared = is_shared_col(cb + q0);
            };
            auto load_epi = [&](int vo, BwdEpi &e) {
                const int von = vo - splane + nplane, vop = vo - splane + pplane;
                e.dh = *(const f4 *)&dh_n[vo * kO + 4 * q4];
                e.gi = *(const f4 *)&gates_dn[vo * kG + 0 * kO + 4 * q4];
                e.gf = *(const f4 *)&gates_dn[vo * kG + 1 * kO + 4 * q4];
                e.gg = *(const f4 *)&gates_dn[vo * kG + 2 * kO + 4 * q4];
                e.go = *(const f4 *)&gates_dn[vo * kG + 3 * kO + 4 * q4];
                e.c = *(const f4 *)&cell_dn[vo * kO + 4 * q4];
                e.gcfn = *(const f4 *)&gcf_dn[von * kO + 4 * q4];
                e.cp = *(const f4 *)&cell_dn[vop * kO + 4 * q4];
            };
            auto epilogue = [&](int vo, bool shared, const f4 (&acc)[4], const BwdEpi &e) {
                f4 dAi, dAf, dAg, dAo, gcf;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float gh = acc[0][i] + acc[1][i] + acc[2][i] + acc[3][i] + e.dh[i];
                    const float tc = ftanh(e.c[i]);
                    const float gcs = gh * e.go[i] * (1.0f - tc * tc) +
                                      (has_next ? e.gcfn[i] : 0.0f);
                    const float cprev = has_prev ? e.cp[i] : 0.0f;
                    gcf[i] = gcs * e.gf[i];
                    dAi[i] = gcs * e.gg[i] * e.gi[i] * (1.0f - e.gi[i]);
                    dAf[i] = gcs * cprev * e.gf[i] * (1.0f - e.gf[i]);
                    dAg[i] = gcs * e.gi[i] * (1.0f - e.gg[i] * e.gg[i]);
                    dAo[i] = gh * tc * e.go[i] * (1.0f - e.go[i]);
                }
                const int o4 = vo * kG + 4 * q4;
                float *dst = &dA_dn[o4];
                if (shared) {
                    store_coherent(dA_rs, o4 + 0 * kO, dAi);
                    store_coherent(dA_rs, o4 + 1 * kO, dAf);
                    store_coherent(dA_rs, o4 + 2 * kO, dAg);
                    store_coherent(dA_rs, o4 + 3 * kO, dAo);
                } else {
                    *(f4 *)&dst[0 * kO] = dAi;
                    *(f4 *)&dst[1 * kO] = dAf;
                    *(f4 *)&dst[2 * kO] = dAg;
                    *(f4 *)&dst[3 * kO] = dAo;
                }
                *(f4 *)&gcf_dn[vo * kO + 4 * q4] = gcf;
            };
            for (int mt = wave; mt < nmt; mt += kWaves) {
                int base, vo;
                bool shared;
                pixel(mt, base, vo, shared);
                BwdEpi e;
                load_epi(vo, e);
                // keep the loads above the contraction (the scheduler would
                // otherwise sink them to their use and expose their latency)
                __builtin_amdgcn_sched_barrier(0);
                f4 acc[4];
                contract_bwd(as, was, base, W2, 1, q4, lane, acc);
                epilogue(vo, shared, acc, e);
            }
            __syncthreads();
        }
        // ---- publish dA_t: every wave's coherent stores have completed ---
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if (threadIdx.x == 0)
            __hip_atomic_store(&a.flags[blockIdx.x], r + 1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
    }
}

// ---- parameter gradients, register-streamed --------------------------------
// dW[d] = sum over voxels v of dA[v] (x) [im2col(h_{t-1})(v), im2col(x_t)(v), 1],
// an implicit GEMM with M = 64 gate-units, N = 144 + 9C + 1 and K = voxels.
// One wave owns a contiguous range of units (16 voxels of a row: four MFMA
// k-steps) of one direction, walking each column group down the rows of a
// plane, and holds all 4 x ceil(N / 16) output tiles (in AGPRs; one wave per
// SIMD).  Operands come straight from global memory into registers
// (lane col takes a gate-unit (A) or an im2col column (B), so every load is
// 64 contiguous bytes per voxel), the
// next group's loads are in flight while the current group's MFMAs run,
// and the accumulators stay in VGPRs for the whole launch: no LDS, no
// barriers.  Zero padding (off-plane taps, h_{-1}) comes from the buffer
// range check.
constexpr int kWgWaves = 4;                    // one team (wave) per SIMD
constexpr int kWgTeamsPerDir = 170;

struct WgRowArgs {
    Geom g;
    const float *x, *hd, *dA;
    float *partial;     // [6][tpd][64][KCp]
    int tpd;            // teams per direction
    int KCp;            // columns padded to 16
};

template <int C> struct WgN {
    static constexpr int NT = (144 + 9 * C + 1 + 15) / 16;   // N-tiles
};

// Cursor of a team: batch element, sweep step, row, group of 16 columns.
struct WgCursor {
    int n, t, p, qg;
};

template <int C, int NT0, int NTC>
__device__ inline void wg_rows_team(const WgRowArgs &a, int d, long long r0, long long r1, int q,
                                    int col, float *out)
{
    const DirGeom dg = a.g.dir[d];
    const long long V = a.g.V;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int ngrp = (dg.Q + 15) >> 4;
    // per-lane constants of the input-tap columns (tiles 9, 10, ...)
    int xtap_dp[NTC], xtap_dq[NTC], xtap_c[NTC], xkind[NTC];   // kind 0: x, 1: one, 2: zero
#pragma unroll
    for (int j = 0; j < NTC; ++j) {
        const int nt = NT0 + j;
        const int kk = (nt - 9) * 16 + col;
        const int tap = kk < 9 * C && kk >= 0 ? kk / C : 4;
        xtap_dp[j] = tap / 3 - 1;
        xtap_dq[j] = tap % 3 - 1;
        xtap_c[j] = kk >= 0 && kk < 9 * C ? kk % C : 0;
        xkind[j] = kk < 9 * C ? 0 : (kk == 9 * C ? 1 : 2);
    }
    f4 acc[4][NTC];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int j = 0; j < NTC; ++j) acc[g][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};

    // Operands of one group of 16 voxels.  K order inside the group: lane
    // group q takes voxels 4q .. 4q+3 (k-step ks: voxel 4q + ks), so the
    // three column taps of an h_{t-1} row read a sliding window of six
    // loads per lane: tap (r, dq) at k-step ks is hv[r][ks + dq].
    constexpr int NX = NT0 + NTC > 9 ? NT0 + NTC - (NT0 > 9 ? NT0 : 9) : 0;   // input tiles
    constexpr int JX = NT0 > 9 ? 0 : 9 - NT0;                                  // first input j
    struct Ops {
        float a[4][4];                 // [k-step][gate]: dA
        float hv[3][6];                // [row p-1, p, p+1][column 4q-1 .. 4q+4]: h_{t-1}
        float bx[4][NX > 0 ? NX : 1];  // [k-step][input tile]: x_t
    };
    constexpr bool kRow[3] = {NT0 < 3, NT0 < 6 && NT0 + NTC > 3, NT0 + NTC > 6};
    // Row-uniform state of the group being loaded: buffer resources of the
    // slice, planes, row validity.  An invalid lane (off the plane, past the
    // row, h_{-1}) gets an out-of-range offset and the hardware returns 0,
    // so no mask touches a loaded value before its MFMA.
    constexpr int kOOB = 0x7ffffff0;
    struct Row {
        __amdgpu_buffer_rsrc_t rs_a, rs_h, rs_x;
        int s, p, colbase;
        bool live, hok[3];
    };
    auto row_of = [&](const WgCursor &cu, bool live) {
        Row w;
        const long long dn = ((long long)d * a.g.N + cu.n) * V;
        // slice resources (byte sizes fit 31 bits: checked on the host)
        w.rs_a = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(a.dA + dn * kG), (short)0,
                                                   (int)(V * kG * 4), kBufferRsrcWord3);
        w.rs_h = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(a.hd + dn * kO), (short)0,
                                                   (int)(V * kO * 4), kBufferRsrcWord3);
        w.rs_x = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(a.x + (long long)cu.n * V * C),
                                                   (short)0, (int)(V * C * 4), kBufferRsrcWord3);
        w.s = dg.sign > 0 ? cu.t : dg.T - 1 - cu.t;
        w.p = cu.p;
        w.colbase = cu.qg * 16 + 4 * q;
        w.live = live;
#pragma unroll
        for (int r = 0; r < 3; ++r)
            w.hok[r] = live & (cu.t > 0) & ((unsigned)(cu.p + r - 1) < (unsigned)dg.P);
        return w;
    };
    // bounds as non-short-circuit unsigned compares: no branches
    auto load_a = [&](const Row &w, int ks, Ops &o) {
        const int qq = w.colbase + ks;
        const bool vq = w.live & ((unsigned)qq < (unsigned)dg.Q);
        const int off = (w.s * ss + w.p * sp + qq * sq) * kG + col;
#pragma unroll
        for (int g = 0; g < 4; ++g)
            o.a[ks][g] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                w.rs_a, vq ? (off + g * 16) * 4 : kOOB, 0, 0));
    };
    auto load_h = [&](const Row &w, int m, Ops &o) {
        const int c = w.colbase - 1 + m;
        const bool okc = (unsigned)c < (unsigned)dg.Q;
        const int sprev = w.s - dg.sign;
#pragma unroll
        for (int r = 0; r < 3; ++r) {
            if (!kRow[r]) continue;
            const int off = (sprev * ss + (w.p + r - 1) * sp + c * sq) * kO + col;
            o.hv[r][m] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                w.rs_h, (w.hok[r] & okc) ? off * 4 : kOOB, 0, 0));
        }
    };
    auto load_x = [&](const Row &w, int ks, Ops &o) {
#pragma unroll
        for (int jx = 0; jx < NX; ++jx) {
            const int j = JX + jx;
            const int pp = w.p + xtap_dp[j], c = w.colbase + ks + xtap_dq[j];
            const bool ok = w.live & (xkind[j] == 0) & ((unsigned)pp < (unsigned)dg.P) &
                            ((unsigned)c < (unsigned)dg.Q);
            const int off = (w.s * ss + pp * sp + c * sq) * C + xtap_c[j];
            o.bx[ks][jx] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                w.rs_x, ok ? off * 4 : kOOB, 0, 0));
        }
    };
    // ones of the bias column (1 for a voxel on the plane, else 0: its dA
    // is 0 then anyway)
    float bias_one[NTC];
#pragma unroll
    for (int j = 0; j < NTC; ++j) bias_one[j] = (NT0 + j >= 9 && xkind[j] == 1) ? 1.0f : 0.0f;
    auto mfma_k = [&](const Ops &o, int ks) {
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int j = 0; j < NTC; ++j) {
                const int nt = NT0 + j;
                const float b = nt < 9 ? o.hv[nt / 3][ks + nt % 3] : o.bx[ks][j - JX] + bias_one[j];
                acc[g][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a[ks][g], b, acc[g][j], 0, 0, 0);
            }
    };
    // Cursor over units u = ((n T + t) ngrp + qg) P + p: a column group
    // walks down the rows, so the h_{t-1} and x rows of one group are
    // re-read (as p + 1, p, p - 1) by the next two groups from cache.  Past
    // the end it stays on a valid unit and the loads are masked to zero.
    WgCursor cu;
    {
        long long rest = r0;
        cu.p = (int)(rest % dg.P);
        rest /= dg.P;
        cu.qg = (int)(rest % ngrp);
        rest /= ngrp;
        cu.t = (int)(rest % dg.T);
        cu.n = (int)(rest / dg.T);
    }
    auto advance = [&]() {
        if (++cu.p == dg.P) {
            cu.p = 0;
            if (++cu.qg == ngrp) {
                cu.qg = 0;
                if (++cu.t == dg.T) {
                    cu.t = 0;
                    if (cu.n + 1 < a.g.N) ++cu.n;
                }
            }
        }
    };
    const long long total = r1 - r0;
    Ops o;
    {
        const Row w = row_of(cu, total > 0);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            load_a(w, ks, o);
            load_x(w, ks, o);
        }
#pragma unroll
        for (int m = 0; m < 6; ++m) load_h(w, m, o);
    }
    // Each operand register is refilled with the next group's value right
    // after its last use by this group's MFMAs: one group of operands is
    // live, and every load has a whole group of MFMAs to arrive.
    for (long long it = 0; it < total; ++it) {
        advance();
        const Row w = row_of(cu, it + 1 < total);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            mfma_k(o, ks);
            load_a(w, ks, o);
            load_x(w, ks, o);
            load_h(w, ks, o);          // hv[.][ks] was last used at k-step ks
            if (ks == 3) {
                load_h(w, 4, o);
                load_h(w, 5, o);
            }
        }
    }
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int j = 0; j < NTC; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                out[(g * 16 + 4 * q + i) * a.KCp + (NT0 + j) * 16 + col] = acc[g][j][i];
}

template <int C>
__global__ void __launch_bounds__(64 * kWgWaves) __attribute__((amdgpu_waves_per_eu(1)))
k_wgrad_rows(WgRowArgs a)
{
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int q = lane >> 4, col = lane & 15;
    const int team = blockIdx.x * kWgWaves + wave;
    if (team >= kDirs * a.tpd) return;
    const int d = team / a.tpd, tin = team % a.tpd;
    const DirGeom dg = a.g.dir[d];
    const long long units = (long long)a.g.N * dg.T * ((dg.Q + 15) / 16) * dg.P;
    const long long r0 = units * tin / a.tpd, r1 = units * (tin + 1) / a.tpd;
    float *out = a.partial + (long long)team * kG * a.KCp;
    wg_rows_team<C, 0, WgN<C>::NT>(a, d, r0, r1, q, col, out);
}

// dW = sum of the per-workgroup partials in workgroup order.
__global__ void __launch_bounds__(256)
k_wgrad_reduce(int C, int bpd, int KCp, const float *__restrict__ partial,
               float *__restrict__ dwx, float *__restrict__ dwh, float *__restrict__ db)
{
    const int i = blockIdx.x * 256 + threadIdx.x;
    const int KC = 144 + 9 * C + 1;
    if (i >= kDirs * kG * KC) return;
    const int k = i % KC;
    const int gn = (i / KC) % kG;
    const int d = i / (KC * kG);
    float acc = 0.0f;
    for (int b = 0; b < bpd; ++b) acc += partial[(((long long)d * bpd + b) * kG + gn) * KCp + k];
    if (k < 144) {
        const int tap = k / 16, j = k % 16;
        dwh[(((long long)d * kG + gn) * kO + j) * 9 + tap] = acc;
    } else if (k < 144 + 9 * C) {
        const int kk = k - 144, tap = kk / C, c = kk % C;
        dwx[(((long long)d * kG + gn) * C + c) * 9 + tap] = acc;
    } else {
        db[d * kG + gn] = acc;
    }
}

__global__ void k_fill_zero(int *p, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

StripCostModel bwd_model(bool allow_resident)
{
    StripCostModel m;
    m.fixed_bytes = kWaFloats * sizeof(float);
    m.px_bytes = kG * sizeof(float);
    m.c_sync = 3.0;
    m.c_tile = 2.9;
    m.c_stage0 = 1.0;
    m.c_stage_px = 0.008;
    m.allow_resident = allow_resident;
    m.res_px_bytes = kG * sizeof(float);          // dA_{t+1} / dA_t, in place
    m.res_own_bytes = 1;                          // tile order (4 bytes per 16 pixels)
    m.res_fixed_bytes = 16 * sizeof(int);         // counters
    m.res_max_staged = 1 << 30;
    m.res_max_own = 2 * kWaves * 16;              // two tiles per wave
    m.c_res_step = 2.0;
    return m;
}

inline int wgrad_kcp(int C) { return (144 + 9 * C + 1 + 15) / 16 * 16; }
constexpr int kWgradBlocksPerDir = 42;

template <int C>
int launch_wgrad(const Geom &g, const float *x, const float *hd, const float *dA, float *partial,
                 hipStream_t st)
{
    WgRowArgs wa;
    wa.g = g;
    wa.x = x; wa.hd = hd; wa.dA = dA;
    wa.partial = partial;
    wa.tpd = kWgTeamsPerDir;
    wa.KCp = wgrad_kcp(C);
    const int teams = kDirs * kWgTeamsPerDir;
    const int per_block = kWgWaves;
    k_wgrad_rows<C><<<(teams + per_block - 1) / per_block, 64 * kWgWaves, 0, st>>>(wa);
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

}  // namespace

bool sweep_bwd_supported(const Geom &g)
{
    // dA slices are addressed as buffer resources: bytes must fit 32 bits
    return g.nd == kDirs && g.KP == 3 && g.KQ == 3 && g.O == kO && g.C >= 1 && g.C <= 4 &&
           g.V * kG * (long long)sizeof(float) < (1LL << 31);
}

size_t sweep_bwd_ws(const Geom &g)
{
    Carve cv(nullptr);
    cv.take<float>((size_t)kDirs * g.N * g.V * kG);                     // dA
    cv.take<float>((size_t)kDirs * g.N * g.V * kO);                     // dL/dc * f
    cv.take<int>(1024 + 1);                                              // flags + err
    cv.take<float>((size_t)kDirs * kWgTeamsPerDir * kG * wgrad_kcp(g.C));   // partials
    if (step_supported(g)) cv.take<char>(step_dx_ws(g));                     // dL/dx fragments
    return cv.off;
}

int sweep_bwd(const Geom &g, const float *x, const float *wx, const float *wh, const Saved &sv,
              const float *dh, float *dx, float *dwx, float *dwh, float *db, void *ws,
              hipStream_t st, bool allow_resident)
{
    const DevInfo di = device_info();
    if (di.cus <= 0) return PLSTM_EHIP;
    const size_t lds_limit = (size_t)(di.max_lds > 0 ? di.max_lds : 65536) - 1024;
    const int budget = di.cus < 1024 ? di.cus : 1024;
    const Plan pl = make_plan(g, budget, bwd_model(allow_resident), lds_limit);
    if (pl.blocks > budget) return PLSTM_EUNSUPPORTED;
    for (int d = 0; d < kDirs; ++d) {
        if (pl.chunk_rows[d] < 1) return PLSTM_EUNSUPPORTED;
        // a resident strip: at most two 16-pixel tiles per wave
        if (pl.resident[d] && (long long)g.dir[d].P * pl.max_w[d] > 2 * kWaves * 16)
            return PLSTM_EUNSUPPORTED;
    }

    Carve cv(ws);
    float *dA = cv.take<float>((size_t)kDirs * g.N * g.V * kG);
    float *gcf = cv.take<float>((size_t)kDirs * g.N * g.V * kO);
    int *flags = cv.take<int>(1024 + 1);
    float *partial = cv.take<float>((size_t)kDirs * kWgTeamsPerDir * kG * wgrad_kcp(g.C));
    float *fragx = step_supported(g) ? (float *)cv.take<char>(step_dx_ws(g)) : nullptr;

    BwdArgs args;
    args.g = g;
    args.wh = wh;
    args.gates = sv.gates; args.cell = sv.cell;
    args.dh = dh;
    args.dA = dA; args.gcf = gcf;
    args.flags = flags; args.err = flags + 1024;
    args.max_spin = g_wait_spin_limit;
    args.wait_bias = g_wait_bias;
    for (int d = 0; d < kDirs; ++d) {
        args.nstrip[d] = pl.nstrip[d];
        args.first[d] = pl.first[d];
        args.chunk_rows[d] = pl.chunk_rows[d];
        args.max_w[d] = pl.max_w[d];
        args.resident[d] = pl.resident[d];
    }
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_sweep_bwd, kThreads, pl.lds) !=
        hipSuccess)
        return PLSTM_EHIP;
    if ((long long)per_cu * di.cus < pl.blocks) return PLSTM_ENOTCORESIDENT;
    (void)hipFuncSetAttribute((const void *)k_sweep_bwd,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl.lds);

    k_fill_zero<<<(1025 + 255) / 256, 256, 0, st>>>(flags, 1025);
    PLSTM_LAUNCH_CHECK();
    timing_begin("sweep_bwd_mfma", st);
    void *kargs[] = {&args};
    if (hipLaunchCooperativeKernel((const void *)k_sweep_bwd, dim3(pl.blocks), dim3(kThreads),
                                   kargs, pl.lds, st) != hipSuccess)
        return PLSTM_EHIP;
    timing_end(1, st);

    timing_begin("wgrad_mfma", st);
    int rc;
    switch (g.C) {
    case 1: rc = launch_wgrad<1>(g, x, sv.hd, dA, partial, st); break;
    case 2: rc = launch_wgrad<2>(g, x, sv.hd, dA, partial, st); break;
    case 3: rc = launch_wgrad<3>(g, x, sv.hd, dA, partial, st); break;
    default: rc = launch_wgrad<4>(g, x, sv.hd, dA, partial, st); break;
    }
    if (rc != PLSTM_OK) return rc;
    const int nout = kDirs * kG * (144 + 9 * g.C + 1);
    k_wgrad_reduce<<<(nout + 255) / 256, 256, 0, st>>>(g.C, kWgTeamsPerDir, wgrad_kcp(g.C),
                                                       partial, dwx, dwh, db);
    PLSTM_LAUNCH_CHECK();
    timing_end(2, st);
    if (dx) {
        rc = fragx ? step_dx(g, wx, dA, fragx, dx, st) : generic_dx(g, wx, dA, dx, st);
        if (rc != PLSTM_OK) return rc;
    }
    PoisonList poison;
    poison.ptr[0] = dwx; poison.count[0] = (long long)kDirs * kG * g.C * 9;
    poison.ptr[1] = dwh; poison.count[1] = (long long)kDirs * kG * kO * 9;
    poison.ptr[2] = db;  poison.count[2] = (long long)kDirs * kG;
    poison.ptr[3] = dx;  poison.count[3] = dx ? (long long)g.N * g.V * g.C : 0;
    return wait_check(args.err, poison, st);
}

}  // namespace plstm
