// Plane-step MFMA path (Section 2.3, Eq. (7)-(13), and the chain rule
// through them) for O = 16, 32 or 64 hidden units and any number of input
// channels: the layers of the stacked networks whose recurrent weights do
// not fit a workgroup's LDS next to its staged planes.
//
// The sweeps run one launch per plane step t.  Within a launch every
// direction with t < T_d updates its whole plane t as independent GEMM
// tiles on v_mfma_f32_16x16x4f32:
//   forward   A_t = b + W_x im2col(x_t) + W_h im2col(h_{t-1})
//             M = the four gates of 16 units, N = pixels, K = 9 (C' + O),
//             gates and the cell update fused into the epilogue;
//   backward  dL/dh_t = dL/dh + sum_taps W_h^T dA_{t+1}[p - tap]
//             M = 16 units, N = pixels, K = 9 * 4O, the gate gradients
//             fused into the epilogue.
// The kernel boundary between steps makes plane t visible to step t + 1 on
// every XCD, so no flags or coherent accesses are needed.  The weights (a
// few hundred KB per direction) are repacked once per call into MFMA A
// fragments and read from L2; the four waves of a workgroup work on
// neighbouring pixel groups of the same unit group, so they share each
// fragment through the L1.  The input and h_{t-1} planes are read straight
// from global memory with raw buffer loads: a tap off the plane gets an
// out-of-range offset and the hardware returns zero.
//
// MFMA layout (16x16x4 f32): lane l supplies A[m = l%16][k = l/16] and
// B[k = l/16][n = l%16] and receives D[4(l/16) + i][l%16], i = 0..3.  In
// each group of four k-steps lane group q takes channels 4q .. 4q+3 of a
// 16-channel block (k-step i: channel 4q + i), so every operand load is one
// 16-byte vector, and every lane ends with four consecutive units of one
// pixel: the epilogues need no data exchange and move 16-byte vectors.
//
// The input volume is converted once per call to fp32 with its channels
// zero-padded to C' = a multiple of 16 (so bf16 storage and any C share one
// kernel); the arithmetic and the saved states are fp32.
//
// The parameter gradients and dL/dx are implicit GEMMs over all voxels
// (no recurrence) on the same MFMA: dW = sum_v dA (x) [im2col(h_{t-1}),
// im2col(x_t), 1] with K = voxels, and dL/dx = sum_d sum_taps W_x^T dA.
#include "common.h"
#include "strip_plan.h"
#include "sweep.h"
#include "timing.h"

namespace plstm {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kSW = 4;                   // waves per workgroup
constexpr int kXcds = 8;                 // XCDs: workgroup b runs on XCD b % 8
constexpr int kNT = 4;                   // 16-pixel tiles per wave
constexpr int kOOB = 0x7ffffff0;         // byte offset past any buffer: loads return 0
constexpr int kRsrcWord3 = 0x00020000;   // raw buffer, 32-bit data

__device__ inline float frcp(float v) { return __builtin_amdgcn_rcpf(v); }
__device__ inline float fsig(float a) { return frcp(1.0f + __expf(-a)); }
__device__ inline float ftanh(float a) { return 1.0f - 2.0f * frcp(__expf(2.0f * a) + 1.0f); }

// Buffer resource over `nfloats` floats (the host checks that the byte size
// fits 31 bits).
__device__ inline __amdgpu_buffer_rsrc_t slice_rsrc(const float *p, long long nfloats)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p), (short)0,
                                             (int)(nfloats * (long long)sizeof(float)),
                                             kRsrcWord3);
}
__device__ inline f4 bload4(__amdgpu_buffer_rsrc_t rs, unsigned off)
{
    return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)off, 0, 0));
}
__device__ inline float bload1(__amdgpu_buffer_rsrc_t rs, unsigned off)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, (int)off, 0, 0));
}
// Byte offset of a masked load: `off` if `ok`, else past the buffer.  The
// empty asm pins the select in a register, so the compiler cannot turn it
// into a branch around the load.
__device__ inline unsigned sel_off(bool ok, unsigned off)
{
    unsigned o = ok ? off : (unsigned)kOOB;
    asm volatile("" : "+v"(o));
    return o;
}
__device__ inline f4 mfma(float a, float b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Direction of a wave item: the base offsets are non-decreasing, a direction
// with no items this step has base[d] == base[d + 1].
__device__ inline int item_dir(const int *base, int item)
{
    int d = 0;
#pragma unroll
    for (int k = 1; k < kDirs; ++k) d += item >= base[k] ? 1 : 0;
    return d;
}

constexpr int kWaitVmcnt0 = 0x0F70;   // s_waitcnt vmcnt(0), other counters unconstrained
typedef __attribute__((address_space(3))) void lds_void;

// In-plane coordinates of a pixel, or kDead past the plane: no tap offset
// (|offset| <= 3) brings kDead back onto a plane.
constexpr int kDead = -(1 << 20);
__device__ inline bool on_plane(int p, int q, int P, int Q)
{
    return ((unsigned)p < (unsigned)P) & ((unsigned)q < (unsigned)Q);
}
// Tap (ka, kb) of a KP x KQ filter from its index: ka = tap / KQ with the
// multiplier k_mul = ceil(2^16 / KQ) (exact for tap < 2^12).
__device__ inline int tap_row(int tap, int k_mul) { return (tap * k_mul) >> 16; }

// ---- conversion and repacking (once per call) -------------------------------

// x [N][V][C] (fp32 or bf16) -> xp [N][V][C'] fp32, channels >= C zero.
template <typename TS>
__global__ void __launch_bounds__(256)
k_pad_x(long long nvox, int C, int Cp, const TS *__restrict__ x, float *__restrict__ xp)
{
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= nvox * Cp) return;
    const long long v = i / Cp;
    const int c = (int)(i - v * Cp);
    xp[i] = c < C ? Store<TS>::load(x, v * C + c) : 0.0f;
}

// Forward A fragments frag[d][ug][kg][gate][lane][4]: K-group kg < KX is
// input tap kg / (C'/16), channel block kg % (C'/16); the rest are h taps
// (kg - KX) / U, channel block (kg - KX) % U.  Entry i of lane (q, col) is
// the weight of gate-unit gate*O + 16 ug + col for channel 16 cb + 4q + i.
template <typename TS>
__global__ void __launch_bounds__(256)
k_pack_fwd(int nd, int O, int C, int Cp, int KX, int KG, int KK, const TS *__restrict__ wx,
           const TS *__restrict__ wh, const TS *__restrict__ b, float *__restrict__ frag,
           float *__restrict__ bias)
{
    const int U = O / 16, G = 4 * O, CX = Cp / 16;
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i < (long long)nd * G) bias[i] = Store<TS>::load(b, i);
    if (i >= (long long)nd * U * KG * 1024) return;
    const int i4 = (int)(i & 3), lane = (int)((i >> 2) & 63), gate = (int)((i >> 8) & 3);
    long long r = i >> 10;
    const int kg = (int)(r % KG);
    r /= KG;
    const int ug = (int)(r % U), d = (int)(r / U);
    const int q = lane >> 4, col = lane & 15;
    const long long gu = (long long)d * G + gate * O + ug * 16 + col;
    float v = 0.0f;
    if (kg < KX) {
        const int tap = kg / CX, c = (kg % CX) * 16 + 4 * q + i4;
        if (c < C) v = Store<TS>::load(wx, (gu * C + c) * KK + tap);
    } else {
        const int kh = kg - KX, tap = kh / U, j = (kh % U) * 16 + 4 * q + i4;
        v = Store<TS>::load(wh, (gu * O + j) * KK + tap);
    }
    frag[i] = v;
}

// Backward A fragments fragB[d][ug][kg][lane][4], kg = tap * 4U + mb: entry
// i of lane (q, col) is W_h[d][gate-unit 16 mb + 4q + i][unit 16 ug + col][tap].
__global__ void __launch_bounds__(256)
k_pack_bwd(int nd, int O, int KK, const float *__restrict__ wh, float *__restrict__ frag)
{
    const int U = O / 16, G = 4 * O, KG = KK * 4 * U;
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= (long long)nd * U * KG * 256) return;
    const int i4 = (int)(i & 3), lane = (int)((i >> 2) & 63);
    long long r = i >> 8;
    const int kg = (int)(r % KG);
    r /= KG;
    const int ug = (int)(r % U), d = (int)(r / U);
    const int tap = kg / (4 * U), mb = kg % (4 * U);
    const int q = lane >> 4, col = lane & 15;
    const long long gu = (long long)d * G + mb * 16 + 4 * q + i4;
    frag[i] = wh[(gu * O + ug * 16 + col) * KK + tap];
}

// dL/dx A fragments fragX[d][tap][mb][ct][lane][4]: entry i of lane (q, col)
// is W_x[d][gate-unit 16 mb + 4q + i][channel 16 ct + col][tap] (0 past C).
__global__ void __launch_bounds__(256)
k_pack_dx(int nd, int O, int C, int CT, int KK, const float *__restrict__ wx,
          float *__restrict__ frag)
{
    const int G = 4 * O, MB = G / 16;
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= (long long)nd * KK * MB * CT * 256) return;
    const int i4 = (int)(i & 3), lane = (int)((i >> 2) & 63);
    long long r = i >> 8;
    const int ct = (int)(r % CT);
    r /= CT;
    const int mb = (int)(r % MB);
    r /= MB;
    const int tap = (int)(r % KK), d = (int)(r / KK);
    const int q = lane >> 4, col = lane & 15;
    const int c = ct * 16 + col;
    const long long gu = (long long)d * G + mb * 16 + 4 * q + i4;
    frag[i] = c < C ? wx[(gu * C + c) * KK + tap] : 0.0f;
}

// ---- forward step -----------------------------------------------------------

struct FwdStepArgs {
    Geom g;
    int t;
    int Cp, KX, KG;           // padded channels, input K-groups (KK C'/16), all K-groups
    int k_mul;                // ceil(2^16 / K): tap row from tap index
    int cx_mul;               // ceil(2^16 / (C'/16)): division by C'/16
    const float *xp;          // [N][V][C']
    const float *frag;        // [6][U][KG][4][64][4]
    const float *bias;        // [6][4O]
    float *hd, *cell;         // [6][N][V][O]
    float *gates;             // [6][N][V][4O] or null
    int npg[kDirs];           // pixel groups (kNT tiles) of a plane
    int base[kDirs + 1];      // first workgroup of each direction in this launch
    // pixel blocks of the LDS-staged kernel (as in FwdB16Args)
    int bp[kDirs], bq[kDirs], nbq[kDirs], nblk[kDirs];
};

// The four gates of unit group ug for kNT 16-pixel tiles of one plane (an
// item).  Two launch shapes:
//   SPLIT   one item per workgroup; its waves split the K-groups (wave w
//           takes w, w + 4, ...), the partial sums meet in LDS in wave order
//           and wave w finishes tile w: four times as many waves per step,
//           for steps with few pixels;
//   !SPLIT  one item per wave; the four waves of a workgroup take
//           neighbouring pixel groups of the same unit group, so they share
//           every A fragment through the L1.
// Items of a (direction, batch element) are ordered unit group major.
template <int U, bool SPLIT>
__global__ void __launch_bounds__(64 * kSW) __attribute__((amdgpu_waves_per_eu(3)))
k_step_fwd(FwdStepArgs a)
{
    constexpr int O = 16 * U, G = 4 * O;
    constexpr int KS = SPLIT ? kSW : 1;          // waves sharing one item's K
    constexpr int NE = SPLIT ? 1 : kNT;          // tiles a wave finishes
    static_assert(kNT == kSW, "wave w finishes tile w");
    __shared__ f4 red[SPLIT ? kSW : 1][4][kNT][64];
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int item = SPLIT ? (int)blockIdx.x : (int)blockIdx.x * kSW + wave;
    if (item >= a.base[kDirs]) return;
    const int d = item_dir(a.base, item);
    const DirGeom dg = a.g.dir[d];
    const int npg = a.npg[d];
    int r = item - a.base[d];
    const int n = r / (U * npg);
    r -= n * U * npg;
    const int ug = r / npg, pg = r - ug * npg;
    const int t = a.t;
    const int s = dg.sign > 0 ? t : dg.T - 1 - t;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int P = dg.P, Q = dg.Q;
    const long long V = a.g.V;
    const int Cp = a.Cp, CX = Cp >> 4, KX = a.KX;
    const int hoff = -dg.sign * ss;   // voxel of plane t - 1 = voxel of plane t + hoff
    const int uo = ug * 16 + 4 * q4;
    const int KQ = a.g.KQ, radp = a.g.KP >> 1, radq = KQ >> 1;

    // this lane's pixel of each tile: voxel and in-plane coordinates
    int vox[kNT], tp[kNT], tq[kNT];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        const int pix = (pg * kNT + nt) * 16 + col;
        const bool live = pix < P * Q;
        const int p = live ? pix / Q : 0, qq = live ? pix - p * Q : 0;
        vox[nt] = s * ss + p * sp + qq * sq;
        tp[nt] = live ? p : kDead;
        tq[nt] = qq;
    }
    const long long sbase = ((long long)d * a.g.N + n) * V;
    const auto rs_x = slice_rsrc(a.xp + (long long)n * V * Cp, V * Cp);
    const auto rs_h = slice_rsrc(a.hd + sbase * O, V * O);
    const auto rs_c = slice_rsrc(a.cell + sbase * O, V * O);
    const float *fr = a.frag + (long long)(d * U + ug) * a.KG * 1024 + lane * 4;

    // the tiles this wave finishes and their c_{t-1}, in flight during the
    // contraction
    int evox[NE];
    bool elive[NE];
    f4 cprev[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        evox[e] = vox[e];
        elive[e] = tp[e] >= 0;
        if (SPLIT) {
#pragma unroll
            for (int nt = 1; nt < kNT; ++nt)
                if (wave == nt) {
                    evox[e] = vox[nt];
                    elive[e] = tp[nt] >= 0;
                }
        }
        cprev[e] = bload4(rs_c, sel_off(t > 0 && elive[e],
                                        (unsigned)((evox[e] + hoff) * O + uo) * 4u));
    }

    f4 acc[4][kNT];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[g][nt] = f4{0.0f, 0.0f, 0.0f, 0.0f};

    struct Ops {
        f4 a[4];
        f4 b[kNT];
    };
    // K-group kg: input tap / channel block for kg < KX, else h_{t-1}'s
    auto load = [&](int kg, Ops &o) {
        const bool is_x = kg < KX;
        const int kk = is_x ? kg : kg - KX;
        // kk / CX from a multiplier (exact for kk < 2^12, CX <= 4); U is a
        // power of two
        const int tap = is_x ? (kk * a.cx_mul) >> 16 : kk / U;
        const int cb = kk - tap * (is_x ? CX : U);
        const int stride = is_x ? Cp : O;
        const int row = tap_row(tap, a.k_mul), ka = row - radp, kb = tap - row * KQ - radq;
        const int dv = (is_x ? 0 : hoff) + ka * sp + kb * sq;
        const auto rs = is_x ? rs_x : rs_h;
#pragma unroll
        for (int g = 0; g < 4; ++g) o.a[g] = *(const f4 *)(fr + kg * 1024 + g * 256);
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt)
            o.b[nt] = bload4(rs, sel_off(on_plane(tp[nt] + ka, tq[nt] + kb, P, Q),
                                         (unsigned)((vox[nt] + dv) * stride + cb * 16 + 4 * q4) *
                                             4u));
    };
    const int KG = t > 0 ? a.KG : KX;
    const int k0 = SPLIT ? wave : 0;
    // the next K-group's operands are loaded while the current one's MFMAs run
    Ops cur, nxt;
    if (k0 < KG) load(k0, cur);
    for (int kg = k0; kg < KG; kg += KS) {
        if (kg + KS < KG) load(kg + KS, nxt);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int nt = 0; nt < kNT; ++nt)
                    acc[g][nt] = mfma(cur.a[g][i], cur.b[nt][i], acc[g][nt]);
        cur = nxt;
    }
    if (SPLIT) {
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt) red[SPLIT ? wave : 0][g][nt][lane] = acc[g][nt];
        __syncthreads();
    }

    // Eq. (7)-(12): gates, cell and hidden state of units uo .. uo+3
    // (split partials added in wave order, then the bias)
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        if (!elive[e]) continue;
        f4 pre[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            f4 v = acc[g][e];
            if (SPLIT) {
                v = red[0][g][wave][lane];
#pragma unroll
                for (int w = 1; w < KS; ++w) v += red[SPLIT ? w : 0][g][wave][lane];
            }
            pre[g] = v + *(const f4 *)(a.bias + d * G + g * O + uo);
        }
        const long long vo = sbase + evox[e];
        f4 gi, gf, gg, go, c, h;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            gi[i] = fsig(pre[0][i]);
            gf[i] = fsig(pre[1][i]);
            gg[i] = ftanh(pre[2][i]);
            go[i] = fsig(pre[3][i]);
            c[i] = gg[i] * gi[i] + cprev[e][i] * gf[i];
            h[i] = go[i] * ftanh(c[i]);
        }
        *(f4 *)(a.cell + vo * O + uo) = c;
        *(f4 *)(a.hd + vo * O + uo) = h;
        if (a.gates) {
            float *gp = a.gates + vo * G + uo;
            *(f4 *)gp = gi;
            *(f4 *)(gp + O) = gf;
            *(f4 *)(gp + 2 * O) = gg;
            *(f4 *)(gp + 3 * O) = go;
        }
    }
}

// LDS-staged variant of k_step_fwd (steps with enough blocks): a workgroup
// takes a BP x BQ block of 64 pixels of one plane and all U unit groups (wave
// w: units 16 w .. 16 w + 15).  The block's x_t with its filter halo is
// staged in LDS (16-byte chunks of 4 channels, XOR-swizzled by the pixel)
// and the input taps read their B operands from there; then h_{t-1} is
// staged over it for the recurrent taps.  The A fragments stream from global
// memory.  Tile nt of the block is its pixels 16 nt .. 16 nt + 15 in
// row-major order.
template <int U>
__global__ void __launch_bounds__(64 * U) __attribute__((amdgpu_waves_per_eu(3)))
k_step_fwd_blk(FwdStepArgs a)
{
    constexpr int O = 16 * U, G = 4 * O;
    extern __shared__ f4 stf[];
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int ug = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int blk = blockIdx.x;
    if (blk >= a.base[kDirs]) return;
    const int d = item_dir(a.base, blk);
    const DirGeom dg = a.g.dir[d];
    int r = blk - a.base[d];
    const int n = r / a.nblk[d];
    r -= n * a.nblk[d];
    const int BP = a.bp[d], BQ = a.bq[d];
    const int bi = r / a.nbq[d], bj = r - bi * a.nbq[d];
    const int p0 = bi * BP, q0 = bj * BQ;
    const int t = a.t;
    const int s = dg.sign > 0 ? t : dg.T - 1 - t;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int P = dg.P, Q = dg.Q;
    const long long V = a.g.V;
    const int Cp = a.Cp, CX = Cp >> 4, KX = a.KX;
    const int hoff = -dg.sign * ss;
    const int uo = ug * 16 + 4 * q4;
    const int KQ = a.g.KQ, radp = a.g.KP >> 1, radq = KQ >> 1;
    const int SW = BQ + 2 * radq, SH = BP + 2 * radp;
    const long long sbase = ((long long)d * a.g.N + n) * V;
    const auto rs_x = slice_rsrc(a.xp + (long long)n * V * Cp, V * Cp);
    const auto rs_h = slice_rsrc(a.hd + sbase * O, V * O);
    const auto rs_c = slice_rsrc(a.cell + sbase * O, V * O);

    // Stage one operand of the block and its halo: nch chunks per pixel of
    // `stride` floats per voxel from `rs` at voxel offset `dvox` (zero off
    // the plane or when !ok).
    auto stage = [&](__amdgpu_buffer_rsrc_t rs, int nch, int stride, int dvox, bool ok) {
        const int swm = (nch & 7) == 0 ? 7 : 3;
        const int nst = SH * SW * nch;
        for (int e = threadIdx.x; e < nst; e += 64 * U) {
            const int spx = e / nch, c = e - spx * nch;
            const int sy = spx / SW, sx = spx - sy * SW;
            const int pp = p0 - radp + sy, qq = q0 - radq + sx;
            const bool on = ok && on_plane(pp, qq, P, Q);
            const int v = s * ss + pp * sp + qq * sq + dvox;
            stf[spx * nch + (c ^ (spx & swm))] =
                bload4(rs, sel_off(on, (unsigned)(v * stride + 4 * c) * 4u));
        }
    };

    const int lbq = 31 - __builtin_clz(BQ);
    int spix[kNT], evox[kNT];
    bool elive[kNT];
    f4 cprev[kNT];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        const int e = nt * 16 + col;
        const int ey = e >> lbq, ex = e & (BQ - 1);
        spix[nt] = (ey + radp) * SW + ex + radq;
        const int pp = p0 + ey, qq = q0 + ex;
        elive[nt] = on_plane(pp, qq, P, Q);
        evox[nt] = s * ss + (elive[nt] ? pp * sp + qq * sq : 0);
        cprev[nt] = bload4(rs_c, sel_off(t > 0 && elive[nt],
                                         (unsigned)((evox[nt] + hoff) * O + uo) * 4u));
    }

    f4 acc[4][kNT];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[g][nt] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    const float *fr = a.frag + (long long)(d * U + ug) * a.KG * 1024 + lane * 4;
    // K-groups kg0 .. kg1 - 1 of one operand (x: kg < KX, else h) from the
    // staged block; A fragments one K-group ahead
    auto contract = [&](int kg0, int kg1, bool is_x) {
        const int nch = is_x ? CX * 4 : U * 4;
        const int swm = (nch & 7) == 0 ? 7 : 3;
        f4 acur[4], anxt[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) acur[g] = *(const f4 *)(fr + kg0 * 1024 + g * 256);
        for (int kg = kg0; kg < kg1; ++kg) {
            if (kg + 1 < kg1) {
#pragma unroll
                for (int g = 0; g < 4; ++g) anxt[g] = *(const f4 *)(fr + (kg + 1) * 1024 + g * 256);
            }
            const int kk = is_x ? kg : kg - KX;
            const int tap = is_x ? (kk * a.cx_mul) >> 16 : kk / U;
            const int cb = kk - tap * (is_x ? CX : U);
            const int row = tap_row(tap, a.k_mul), ka = row - radp, kb = tap - row * KQ - radq;
            const int chunk = cb * 4 + q4;
            const int doff = ka * SW + kb;
            f4 bv[kNT];
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt) {
                const int spx = spix[nt] + doff;
                bv[nt] = stf[spx * nch + (chunk ^ (spx & swm))];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int g = 0; g < 4; ++g)
#pragma unroll
                    for (int nt = 0; nt < kNT; ++nt)
                        acc[g][nt] = mfma(acur[g][i], bv[nt][i], acc[g][nt]);
#pragma unroll
            for (int g = 0; g < 4; ++g) acur[g] = anxt[g];
        }
    };
    stage(rs_x, CX * 4, Cp, 0, true);
    __syncthreads();
    contract(0, KX, true);
    if (t > 0) {
        __syncthreads();                 // every wave is done with the staged x
        stage(rs_h, U * 4, O, hoff, true);
        __syncthreads();
        contract(KX, a.KG, false);
    }

#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        if (!elive[nt]) continue;
        f4 pre[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) pre[g] = acc[g][nt] + *(const f4 *)(a.bias + d * G + g * O + uo);
        const long long vo = sbase + evox[nt];
        f4 gi, gf, gg, go, c, h;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            gi[i] = fsig(pre[0][i]);
            gf[i] = fsig(pre[1][i]);
            gg[i] = ftanh(pre[2][i]);
            go[i] = fsig(pre[3][i]);
            c[i] = gg[i] * gi[i] + cprev[nt][i] * gf[i];
            h[i] = go[i] * ftanh(c[i]);
        }
        *(f4 *)(a.cell + vo * O + uo) = c;
        *(f4 *)(a.hd + vo * O + uo) = h;
        if (a.gates) {
            float *gp = a.gates + vo * G + uo;
            *(f4 *)gp = gi;
            *(f4 *)(gp + O) = gf;
            *(f4 *)(gp + 2 * O) = gg;
            *(f4 *)(gp + 3 * O) = go;
        }
    }
}

// Forward step on LDS-staged pixel blocks with K split over the waves (U =
// 1, 2 or 4 unit groups).  A workgroup takes a BP x BQ block of 64 pixels of
// one plane; x_t and h_{t-1} of the block and its filter halo are staged in
// LDS once ([x | h] per pixel in 16-byte chunks of 4 channels, XOR-swizzled
// by the pixel), so every tap's B operand comes from LDS.  Wave w owns unit
// group w % U and K-part w / U of the KP = 4 / U parts (K-groups kp,
// kp + KP, ...; input and recurrent K-groups as in k_step_fwd) for all four
// pixel tiles.  It then leaves the partial sums of the tiles it does not
// finish in LDS and finishes tiles kp, kp + KP, ... itself: the KP partials
// added in K-part order, the bias, the gates and the cell update.  Four
// waves per block whatever U is, for steps with few blocks.
template <int U>
__global__ void __launch_bounds__(64 * kSW) __attribute__((amdgpu_waves_per_eu(3)))
k_step_fwd_bls(FwdStepArgs a)
{
    constexpr int O = 16 * U, G = 4 * O;
    constexpr int KP = kSW / U;                  // K-parts
    constexpr int NF = kNT / KP;                 // tiles a wave finishes
    constexpr int NU = kNT - NF;                 // tiles it leaves to others
    static_assert(kSW % U == 0 && kNT % KP == 0, "waves cover unit groups x K-parts");
    extern __shared__ f4 stf[];
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int ug = wave % U, kp = wave / U;
    const int blk = blockIdx.x;
    if (blk >= a.base[kDirs]) return;
    const int d = item_dir(a.base, blk);
    const DirGeom dg = a.g.dir[d];
    int r = blk - a.base[d];
    const int n = r / a.nblk[d];
    r -= n * a.nblk[d];
    const int BP = a.bp[d], BQ = a.bq[d];
    const int bi = r / a.nbq[d], bj = r - bi * a.nbq[d];
    const int p0 = bi * BP, q0 = bj * BQ;
    const int t = a.t;
    const int s = dg.sign > 0 ? t : dg.T - 1 - t;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int P = dg.P, Q = dg.Q;
    const long long V = a.g.V;
    const int Cp = a.Cp, CX = Cp >> 4, KX = a.KX;
    const int hoff = -dg.sign * ss;   // voxel of plane t - 1 = voxel of plane t + hoff
    const int uo = ug * 16 + 4 * q4;
    const int KQ = a.g.KQ, radp = a.g.KP >> 1, radq = KQ >> 1;
    const int SW = BQ + 2 * radq, SH = BP + 2 * radp;
    const long long sbase = ((long long)d * a.g.N + n) * V;
    const auto rs_x = slice_rsrc(a.xp + (long long)n * V * Cp, V * Cp);
    const auto rs_h = slice_rsrc(a.hd + sbase * O, V * O);
    const auto rs_c = slice_rsrc(a.cell + sbase * O, V * O);
    const int nxc = CX * 4, nch = nxc + U * 4;   // staged chunks per pixel: x, then h
    const int swm = (nch & 7) == 0 ? 7 : 3;
    const int lbq = 31 - __builtin_clz(BQ);

    // the bias of this lane's units, and the tiles this wave finishes and
    // their c_{t-1}, in flight meanwhile
    f4 biasv[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) biasv[g] = *(const f4 *)(a.bias + d * G + g * O + uo);
    int evox[NF];
    bool elive[NF];
    f4 cprev[NF];
#pragma unroll
    for (int j = 0; j < NF; ++j) {
        const int e = (kp + KP * j) * 16 + col;
        const int ey = e >> lbq, ex = e & (BQ - 1);
        elive[j] = on_plane(p0 + ey, q0 + ex, P, Q);
        evox[j] = s * ss + (elive[j] ? (p0 + ey) * sp + (q0 + ex) * sq : 0);
        cprev[j] = bload4(rs_c, sel_off(t > 0 && elive[j],
                                        (unsigned)((evox[j] + hoff) * O + uo) * 4u));
    }

    // stage x_t and h_{t-1} of the block and its halo (zero off the plane,
    // and h at t = 0) with direct-to-LDS loads, all in flight at once: one
    // instruction fills 64 consecutive 16-byte slots, slot p of pixel spx
    // holding chunk p ^ (spx & swm), each lane loading the chunk its slot
    // holds; x and h chunks go out as two instructions masked by source.
    {
        const int nslot = SH * SW * nch;
        for (int e0 = wave * 64; e0 < nslot; e0 += 64 * kSW) {
            const int e = e0 + lane;
            const int spx = e / nch, pos = e - spx * nch;
            const int c = pos ^ (spx & swm);
            const int sy = spx / SW, sx = spx - sy * SW;
            const int pp = p0 - radp + sy, qq = q0 - radq + sx;
            const bool on = e < nslot && on_plane(pp, qq, P, Q);
            const int v = s * ss + pp * sp + qq * sq;
            lds_void *dst = (lds_void *)&stf[e0];
            if (e < nslot) {
                if (c < nxc)
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(
                        rs_x, dst, 16, (int)sel_off(on, (unsigned)(v * Cp + 4 * c) * 4u), 0, 0, 0);
                else
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(
                        rs_h, dst, 16,
                        (int)sel_off(on && t > 0, (unsigned)((v + hoff) * O + 4 * (c - nxc)) * 4u),
                        0, 0, 0);
            }
        }
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    }
    __syncthreads();

    int spix[kNT];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        const int e = nt * 16 + col;
        spix[nt] = ((e >> lbq) + radp) * SW + (e & (BQ - 1)) + radq;
    }
    f4 acc[4][kNT];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[g][nt] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    const float *fr = a.frag + (long long)(d * U + ug) * a.KG * 1024 + lane * 4;
    const int KGe = t > 0 ? a.KG : KX;
    f4 acur[4], anxt[4];
    if (kp < KGe) {
#pragma unroll
        for (int g = 0; g < 4; ++g) acur[g] = *(const f4 *)(fr + kp * 1024 + g * 256);
    }
    for (int kg = kp; kg < KGe; kg += KP) {
        if (kg + KP < KGe) {
#pragma unroll
            for (int g = 0; g < 4; ++g) anxt[g] = *(const f4 *)(fr + (kg + KP) * 1024 + g * 256);
        }
        const bool is_x = kg < KX;
        const int kk = is_x ? kg : kg - KX;
        const int tap = is_x ? (kk * a.cx_mul) >> 16 : kk / U;
        const int cb = kk - tap * (is_x ? CX : U);
        const int row = tap_row(tap, a.k_mul), ka = row - radp, kb = tap - row * KQ - radq;
        const int doff = ka * SW + kb;
        const int chunk = (is_x ? 0 : nxc) + cb * 4 + q4;
        f4 bv[kNT];
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) {
            const int spx = spix[nt] + doff;
            bv[nt] = stf[spx * nch + (chunk ^ (spx & swm))];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int nt = 0; nt < kNT; ++nt)
                    acc[g][nt] = mfma(acur[g][i], bv[nt][i], acc[g][nt]);
#pragma unroll
        for (int g = 0; g < 4; ++g) acur[g] = anxt[g];
    }

    // slot of tile nt among the tiles K-part k leaves to others
    auto slot = [](int nt, int k) {
        int sl = 0;
#pragma unroll
        for (int m = 0; m < kNT; ++m) sl += (m < nt && m % KP != k) ? 1 : 0;
        return sl;
    };
    if constexpr (KP > 1) {
        __syncthreads();                 // every wave is done with the staged block
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) {
            if (nt % KP == kp) continue;
            const int sl = slot(nt, kp);
#pragma unroll
            for (int g = 0; g < 4; ++g) stf[((wave * 4 + g) * NU + sl) * 64 + lane] = acc[g][nt];
        }
        __syncthreads();
    }

    // Eq. (7)-(12) for the tiles this wave finishes: the K-parts' partials in
    // order, the bias, gates, cell and hidden state of units uo .. uo+3
#pragma unroll
    for (int j = 0; j < NF; ++j) {
        if (!elive[j]) continue;
        const int nt = kp + KP * j;
        f4 pre[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            f4 v = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int k = 0; k < KP; ++k) {
                if (k == kp) {
#pragma unroll
                    for (int m = 0; m < kNT; ++m)
                        if (m == nt) v += acc[g][m];
                } else {
                    v += stf[(((ug + U * k) * 4 + g) * NU + slot(nt, k)) * 64 + lane];
                }
            }
            pre[g] = v + biasv[g];
        }
        const long long vo = sbase + evox[j];
        f4 gi, gf, gg, go, c, h;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            gi[i] = fsig(pre[0][i]);
            gf[i] = fsig(pre[1][i]);
            gg[i] = ftanh(pre[2][i]);
            go[i] = fsig(pre[3][i]);
            c[i] = gg[i] * gi[i] + cprev[j][i] * gf[i];
            h[i] = go[i] * ftanh(c[i]);
        }
        *(f4 *)(a.cell + vo * O + uo) = c;
        *(f4 *)(a.hd + vo * O + uo) = h;
        if (a.gates) {
            float *gp = a.gates + vo * G + uo;
            *(f4 *)gp = gi;
            *(f4 *)(gp + O) = gf;
            *(f4 *)(gp + 2 * O) = gg;
            *(f4 *)(gp + 3 * O) = go;
        }
    }
}

// ---- line blocks of the 2D layer's forward (16 hidden units) ----------------
// A 2D direction scans whole lines; each step is one line of Q pixels, too
// little work for a launch of its own.  Here a workgroup owns a 64-pixel
// segment of a line and advances S lines in one launch with overlapped
// tiles: at line j of the launch it computes the segment widened by
// (S - 1 - j) r pixels on each side (r = KQ / 2), which is exactly what line
// j + 1 reads, so h_{t-1} and c stay in LDS across the S lines; only the
// segment itself is stored.  The widened pixels are the neighbours' own
// pixels, recomputed.  Pixels past the line keep h = 0 (zero padding).
constexpr int kLineSeg = 64;       // stored pixels of a segment
constexpr int kLineSlots = 112;    // LDS pixel slots: segment + 2 S r (S r <= 16) + a tile
struct LineFwdArgs {
    Geom g;
    int t0, S;                  // first line of this launch, lines per launch
    int Cp, KX, KG;             // padded channels; K-groups of the taps of x (dense), all
    int c_mul;                  // ceil(2^16 / C): (tap, channel) of a dense K index
    const float *xp, *frag, *bias;
    float *hd, *cell, *gates;
    int nseg[kDirs];            // segments per line
    int base[kDirs + 1];        // first workgroup of each direction
};

// A fragments of k_line_fwd, frag[d][kg][gate][lane][4] (16 units): the input
// taps packed densely, K index kk = 16 kg + 4 q + i of the first KX groups
// being (tap, channel) = (kk / C, kk % C) (zero past K C); then one group per
// recurrent tap.  Entry i of lane (q, col) weighs gate-unit gate*16 + col.
template <typename TS>
__global__ void __launch_bounds__(256)
k_pack_line(int nd, int C, int KQ, int KX, int KG, const TS *__restrict__ wx,
            const TS *__restrict__ wh, const TS *__restrict__ b, float *__restrict__ frag,
            float *__restrict__ bias)
{
    constexpr int O = 16, G = 64;
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i < (long long)nd * G) bias[i] = Store<TS>::load(b, i);
    if (i >= (long long)nd * KG * 1024) return;
    const int i4 = (int)(i & 3), lane = (int)((i >> 2) & 63), gate = (int)((i >> 8) & 3);
    const long long r = i >> 10;
    const int kg = (int)(r % KG), d = (int)(r / KG);
    const int q = lane >> 4, col = lane & 15;
    const long long gu = (long long)d * G + gate * O + col;
    float v = 0.0f;
    if (kg < KX) {
        const int kk = 16 * kg + 4 * q + i4;
        if (kk < KQ * C) v = Store<TS>::load(wx, (gu * C + kk % C) * KQ + kk / C);
    } else {
        v = Store<TS>::load(wh, (gu * O + 4 * q + i4) * KQ + (kg - KX));
    }
    frag[i] = v;
}

// LDS bytes of k_line_fwd beyond its static arrays: the launch's A fragments
// and two lines of x (C floats per pixel).
inline size_t line_fwd_dyn_lds(int KG, int C)
{
    return (size_t)KG * 4 * 64 * 16 + 2 * (size_t)kLineSlots * C * 4;
}

__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3)))
k_line_fwd(LineFwdArgs a)
{
    constexpr int O = 16, G = 64;
    __shared__ f4 hbuf[2][kLineSlots][4];   // h of the previous and current line
    __shared__ f4 cbuf[kLineSlots][4];      // c (read and rewritten in place)
    extern __shared__ f4 dyn[];
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int blk = blockIdx.x;
    if (blk >= a.base[kDirs]) return;
    const int d = item_dir(a.base, blk);
    const DirGeom dg = a.g.dir[d];
    int r = blk - a.base[d];
    const int n = r / a.nseg[d], seg = r - n * a.nseg[d];
    const int Q = dg.Q, rq = a.g.KQ >> 1, S = a.S;
    const int q0 = seg * kLineSeg;
    const int pbase = q0 - S * rq;            // pixel of LDS slot 0
    const int ss = (int)dg.ss, sq = (int)dg.sq;
    const long long V = a.g.V;
    const long long sbase = ((long long)d * a.g.N + n) * V;
    const int C = a.g.C, Cp = a.Cp, KX = a.KX, KG = a.KG, KC = a.g.KQ * C;
    const auto rs_x = slice_rsrc(a.xp + (long long)n * V * Cp, V * Cp);
    const auto rs_h = slice_rsrc(a.hd + sbase * O, V * O);
    const auto rs_c = slice_rsrc(a.cell + sbase * O, V * O);
    const int t0 = a.t0;
    const int nlines = min(S, dg.T - t0);
    f4 *afr = dyn;                                 // [KG][4 gates][64 lanes]
    float *xbuf = (float *)(dyn + KG * 256);       // [2][kLineSlots][C]

    // x of line t (pixels pbase + slot, C channels) into buffer b: 4-byte
    // direct-to-LDS loads, 64 floats per instruction; pixels past the line
    // read zero
    auto stage_x = [&](int t, int b) {
        const int s = dg.sign > 0 ? t : dg.T - 1 - t;
        const int nel = kLineSlots * C;
        for (int e0 = wave * 64; e0 < nel; e0 += 256) {
            const int e = e0 + lane;
            const int slot = e / C, c = e - slot * C;
            const int qq = pbase + slot;
            const bool ok = e < nel && (unsigned)qq < (unsigned)Q;
            const unsigned off = sel_off(ok, (unsigned)(((s * ss + qq * sq) * Cp + c) * 4));
            lds_void *dst = (lds_void *)&xbuf[(size_t)b * kLineSlots * C + e0];
            if (e < nel) __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_x, dst, 4, (int)off, 0, 0, 0);
        }
    };

    // the launch's A fragments, h and c of line t0 - 1 over the widest range
    // (zero before the first line and past the line's ends), x of line t0
    {
        const f4 *src = (const f4 *)(a.frag + (long long)d * KG * 1024);
        for (int e = threadIdx.x; e < KG * 256; e += 256) afr[e] = src[e];
        const int sprev = dg.sign > 0 ? t0 - 1 : dg.T - t0;
        const int nsl = kLineSeg + 2 * S * rq;
        for (int e = threadIdx.x; e < kLineSlots * 4; e += 256) {
            const int slot = e >> 2, part = e & 3;
            const int qq = pbase + slot;
            const bool ok = t0 > 0 && slot < nsl && (unsigned)qq < (unsigned)Q;
            const unsigned off = (unsigned)(((sprev * ss + qq * sq) * O + 4 * part) * 4);
            hbuf[0][slot][part] = bload4(rs_h, sel_off(ok, off));
            cbuf[slot][part] = bload4(rs_c, sel_off(ok, off));
        }
        stage_x(t0, 0);
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    }
    __syncthreads();

    for (int j = 0; j < nlines; ++j) {
        const int t = t0 + j;
        const int s = dg.sign > 0 ? t : dg.T - 1 - t;
        if (j + 1 < nlines) stage_x(t + 1, (j + 1) & 1);   // lands while this line computes
        const int lo = (j + 1) * rq;                        // slot of the first computed pixel
        const int W = kLineSeg + 2 * (S - 1 - j) * rq;      // computed pixels
        const int ntl = (W + 15) >> 4;
        const f4 (*hp)[4] = hbuf[j & 1];
        f4 (*hc)[4] = hbuf[(j + 1) & 1];
        const float *xb = xbuf + (size_t)(j & 1) * kLineSlots * C;
        const int kgn = t > 0 ? KG : KX;
        for (int i = wave; i < ntl; i += 4) {               // wave-uniform
            const int slot = lo + 16 * i + col;
            const int qq = pbase + slot;
            const bool on = 16 * i + col < W && (unsigned)qq < (unsigned)Q;
            f4 acc[4];
#pragma unroll
            for (int g = 0; g < 4; ++g) acc[g] = f4{0.0f, 0.0f, 0.0f, 0.0f};
            for (int kg = 0; kg < kgn; ++kg) {
                f4 bv;
                if (kg < KX) {
                    // dense (tap, channel) K indices of this lane's four k-steps
#pragma unroll
                    for (int i4 = 0; i4 < 4; ++i4) {
                        const int kk = 16 * kg + 4 * q4 + i4;
                        const bool real = kk < KC;          // padding reads tap 0, channel 0
                        const int tap = real ? (kk * a.c_mul) >> 16 : 0;
                        const int c = real ? kk - tap * C : 0;
                        const float xv = xb[(slot + tap - rq) * C + c];
                        bv[i4] = real ? xv : 0.0f;
                    }
                } else {
                    bv = hp[slot + (kg - KX) - rq][q4];
                }
                const f4 *ak = afr + kg * 256 + lane;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const f4 av = ak[g * 64];
#pragma unroll
                    for (int i4 = 0; i4 < 4; ++i4) acc[g] = mfma(av[i4], bv[i4], acc[g]);
                }
            }
            f4 gi, gf, gg, go, c, h;
            const f4 cp = cbuf[slot][q4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                gi[u] = fsig(acc[0][u] + a.bias[d * G + 0 * O + 4 * q4 + u]);
                gf[u] = fsig(acc[1][u] + a.bias[d * G + 1 * O + 4 * q4 + u]);
                gg[u] = ftanh(acc[2][u] + a.bias[d * G + 2 * O + 4 * q4 + u]);
                go[u] = fsig(acc[3][u] + a.bias[d * G + 3 * O + 4 * q4 + u]);
                c[u] = gg[u] * gi[u] + (t > 0 ? cp[u] : 0.0f) * gf[u];
                h[u] = go[u] * ftanh(c[u]);
            }
            const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
            cbuf[slot][q4] = on ? c : zero;
            hc[slot][q4] = on ? h : zero;
            if (on && qq >= q0 && qq < q0 + kLineSeg) {
                const long long vo = sbase + s * ss + qq * sq;
                *(f4 *)(a.cell + vo * O + 4 * q4) = c;
                *(f4 *)(a.hd + vo * O + 4 * q4) = h;
                if (a.gates) {
                    float *gp = a.gates + vo * G + 4 * q4;
                    *(f4 *)gp = gi;
                    *(f4 *)(gp + O) = gf;
                    *(f4 *)(gp + 2 * O) = gg;
                    *(f4 *)(gp + 3 * O) = go;
                }
            }
        }
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);            // next line's x has landed
        __syncthreads();
    }
}

// ---- forward step on the bf16 MFMA (bf16 storage, O = 32 or 64) --------------
// For bf16 storage the contraction runs on v_mfma_f32_16x16x32_bf16 with fp32
// accumulation: x and the weights are bf16 values already, and h^d is kept
// in bf16 only (h_{t-1} enters the recurrence as bf16, and the direction sum
// adds the bf16 values in fp32); c stays fp32.  Lane l supplies A[m = l%16][k = 8(l/16) + j] and B[k][n = l%16],
// j = 0..7, so lane group q takes channels 8q .. 8q+7 of a 32-channel block:
// one 16-byte load per operand, one MFMA per block, gate, tile.
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef unsigned short us4 __attribute__((ext_vector_type(4)));

__device__ inline f4 mfma_bf16(bf8 a, bf8 b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// Gates and cell update of four units (Eq. (7)-(12)) for the bf16 steps,
// h rounded to bf16.  The fused multiply-adds are written out, so every
// kernel that uses it rounds alike whatever the compiler would contract.
__device__ inline void lstm_cell4_b16(const f4 (&pre)[4], const f4 &cprev, f4 &c, us4 &hbv)
{
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float gi = fsig(pre[0][i]), gf = fsig(pre[1][i]), go = fsig(pre[3][i]);
        const float gg = __builtin_fmaf(-2.0f, frcp(__expf(2.0f * pre[2][i]) + 1.0f), 1.0f);
        c[i] = __builtin_fmaf(gg, gi, cprev[i] * gf);
        const float tc = __builtin_fmaf(-2.0f, frcp(__expf(2.0f * c[i]) + 1.0f), 1.0f);
        hbv[i] = f32_to_bf16(go * tc);
    }
}
__device__ inline bf8 bload8h(__amdgpu_buffer_rsrc_t rs, unsigned off)
{
    return __builtin_bit_cast(bf8, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)off, 0, 0));
}

// x [N][V][C] bf16 -> xb [N][V][C32] bf16, channels >= C zero.
__global__ void __launch_bounds__(256)
k_pad_x_b16(long long nvox, int C, int C32, const uint16_t *__restrict__ x,
            uint16_t *__restrict__ xb)
{
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= nvox * C32) return;
    const long long v = i / C32;
    const int c = (int)(i - v * C32);
    xb[i] = c < C ? x[v * C + c] : (uint16_t)0;
}

// bf16 A fragments fragb[d][ug][kg][gate][lane][8]: K-group kg < KX is input
// tap kg / (C32/32), channel block kg % (C32/32); the rest are h taps
// (kg - KX) / (O/32), block (kg - KX) % (O/32).  Entry j of lane (q, col)
// is the weight of gate-unit gate*O + 16 ug + col for channel 32 cb + 8q + j.
// Packed taps (pk, 16 units, C <= 8): the four lane groups of a K-group take
// four 8-channel slots, input slot 4 kg + q being tap 4 kg + q, h slot
// 4 (kg - KX) + q being channels 8 (slot & 1) .. + 7 of tap slot / 2; slots
// past the last tap hold zeros.
__global__ void __launch_bounds__(256)
k_pack_fwd_b16(int nd, int O, int C, int C32, int KX, int KG, int KK, int pk,
               const uint16_t *__restrict__ wx,
               const uint16_t *__restrict__ wh, const uint16_t *__restrict__ b,
               uint16_t *__restrict__ frag, float *__restrict__ bias)
{
    const int U = O / 16, G = 4 * O, CX = C32 / 32, UH = O / 32;
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i < (long long)nd * G) bias[i] = bf16_to_f32(b[i]);
    if (i >= (long long)nd * U * KG * 2048) return;
    const int j8 = (int)(i & 7), lane = (int)((i >> 3) & 63), gate = (int)((i >> 9) & 3);
    long long r = i >> 11;
    const int kg = (int)(r % KG);
    r /= KG;
    const int ug = (int)(r % U), d = (int)(r / U);
    const int q = lane >> 4, col = lane & 15;
    const long long gu = (long long)d * G + gate * O + ug * 16 + col;
    uint16_t v = 0;
    if (pk) {
        if (kg < KX) {
            const int tap = 4 * kg + q;
            if (tap < KK && j8 < C) v = wx[(gu * C + j8) * KK + tap];
        } else {
            const int slot = 4 * (kg - KX) + q, tap = slot >> 1;
            if (tap < KK) v = wh[(gu * O + 8 * (slot & 1) + j8) * KK + tap];
        }
    } else if (kg < KX) {
        const int tap = kg / CX, c = (kg % CX) * 32 + 8 * q + j8;
        if (c < C) v = wx[(gu * C + c) * KK + tap];
    } else {
        const int kh = kg - KX, tap = kh / UH, jj = (kh % UH) * 32 + 8 * q + j8;
        v = wh[(gu * O + jj) * KK + tap];
    }
    frag[i] = v;
}

struct FwdB16Args {
    Geom g;
    int t;
    int C32, KX, KG;          // padded channels (a multiple of 32; 8 for packed taps),
                              // input K-groups, all K-groups
    int k_mul;                // ceil(2^16 / K)
    int cx_mul32;             // ceil(2^16 / (C32/32)): division by C32/32
    const uint16_t *xb;       // [N][V][C32] bf16
    const uint16_t *frag;     // [6][U][KG][4][64][8] bf16
    const float *bias;        // [6][4O]
    float *cell;              // [6][N][V][O] fp32 c^d
    uint16_t *hb;             // [6][N][V][O] bf16 h^d (the recurrence's operand and the
                              // direction sum's input)
    uint16_t *preact;         // projection variant: x's part of the pre-activations and
                              // the bias, [6][N][V][4O] bf16
    float *cpp;               // macro-tiled kernel: c^d of the last two planes,
                              // [6][N][2][pqmax][O] fp32, plane t at parity t & 1
    int pqmax;                // largest plane (P Q) over the directions
    int npg[kDirs];
    int base[kDirs + 1];
    // pixel blocks of the LDS-staged kernel: BP x BQ pixels (BP BQ = 64), nbq
    // blocks across a plane row, nblk per plane
    int bp[kDirs], bq[kDirs], nbq[kDirs], nblk[kDirs];
};

// Same items and launch shapes as k_step_fwd.
template <int U, bool SPLIT>
__global__ void __launch_bounds__(64 * kSW) __attribute__((amdgpu_waves_per_eu(3)))
k_step_fwd_b16(FwdB16Args a)
{
    constexpr int O = 16 * U, G = 4 * O, UH = O / 32;
    constexpr int KS = SPLIT ? kSW : 1;
    constexpr int NE = SPLIT ? 1 : kNT;
    static_assert(kNT == kSW && O % 32 == 0, "wave w finishes tile w; 32-channel blocks");
    __shared__ f4 red[SPLIT ? kSW : 1][4][kNT][64];
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int item = SPLIT ? (int)blockIdx.x : (int)blockIdx.x * kSW + wave;
    if (item >= a.base[kDirs]) return;
    const int d = item_dir(a.base, item);
    const DirGeom dg = a.g.dir[d];
    const int npg = a.npg[d];
    int r = item - a.base[d];
    const int n = r / (U * npg);
    r -= n * U * npg;
    const int ug = r / npg, pg = r - ug * npg;
    const int t = a.t;
    const int s = dg.sign > 0 ? t : dg.T - 1 - t;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int P = dg.P, Q = dg.Q;
    const long long V = a.g.V;
    const int C32 = a.C32, CX = C32 >> 5, KX = a.KX;
    const int hoff = -dg.sign * ss;
    const int uo = ug * 16 + 4 * q4;
    const int KQ = a.g.KQ, radp = a.g.KP >> 1, radq = KQ >> 1;

    int vox[kNT], tp[kNT], tq[kNT];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        const int pix = (pg * kNT + nt) * 16 + col;
        const bool live = pix < P * Q;
        const int p = live ? pix / Q : 0, qq = live ? pix - p * Q : 0;
        vox[nt] = s * ss + p * sp + qq * sq;
        tp[nt] = live ? p : kDead;
        tq[nt] = qq;
    }
    const long long sbase = ((long long)d * a.g.N + n) * V;
    // byte sizes: V * C32 * 2 and V * O * 2 (< 2^31, checked on the host)
    const auto rs_x = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(a.xb + (long long)n * V * C32), (short)0, (int)(V * C32 * 2),
        kRsrcWord3);
    const auto rs_h = __builtin_amdgcn_make_buffer_rsrc(a.hb + sbase * O, (short)0,
                                                        (int)(V * O * 2), kRsrcWord3);
    const auto rs_c = slice_rsrc(a.cell + sbase * O, V * O);
    const uint16_t *fr = a.frag + (long long)(d * U + ug) * a.KG * 2048 + lane * 8;

    int evox[NE];
    bool elive[NE];
    f4 cprev[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        evox[e] = vox[e];
        elive[e] = tp[e] >= 0;
        if (SPLIT) {
#pragma unroll
            for (int nt = 1; nt < kNT; ++nt)
                if (wave == nt) {
                    evox[e] = vox[nt];
                    elive[e] = tp[nt] >= 0;
                }
        }
        cprev[e] = bload4(rs_c, sel_off(t > 0 && elive[e],
                                        (unsigned)((evox[e] + hoff) * O + uo) * 4u));
    }

    f4 acc[4][kNT];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[g][nt] = f4{0.0f, 0.0f, 0.0f, 0.0f};

    struct Ops {
        bf8 a[4];
        bf8 b[kNT];
    };
    auto load = [&](int kg, Ops &o) {
        const bool is_x = kg < KX;
        const int kk = is_x ? kg : kg - KX;
        const int tap = is_x ? (kk * a.cx_mul32) >> 16 : kk / UH;
        const int cb = kk - tap * (is_x ? CX : UH);
        const int stride = is_x ? C32 : O;
        const int row = tap_row(tap, a.k_mul), ka = row - radp, kb = tap - row * KQ - radq;
        const int dv = (is_x ? 0 : hoff) + ka * sp + kb * sq;
        const auto rs = is_x ? rs_x : rs_h;
#pragma unroll
        for (int g = 0; g < 4; ++g) o.a[g] = *(const bf8 *)(fr + (kg * 4 + g) * 512);
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt)
            o.b[nt] = bload8h(rs, sel_off(on_plane(tp[nt] + ka, tq[nt] + kb, P, Q),
                                          (unsigned)((vox[nt] + dv) * stride + cb * 32 + 8 * q4) *
                                              2u));
    };
    const int KG = t > 0 ? a.KG : KX;
    const int k0 = SPLIT ? wave : 0;
    Ops cur, nxt;
    if (k0 < KG) load(k0, cur);
    for (int kg = k0; kg < KG; kg += KS) {
        if (kg + KS < KG) load(kg + KS, nxt);
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt) acc[g][nt] = mfma_bf16(cur.a[g], cur.b[nt], acc[g][nt]);
        cur = nxt;
    }
    if (SPLIT) {
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt) red[SPLIT ? wave : 0][g][nt][lane] = acc[g][nt];
        __syncthreads();
    }

#pragma unroll
    for (int e = 0; e < NE; ++e) {
        if (!elive[e]) continue;
        f4 pre[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            f4 v = acc[g][e];
            if (SPLIT) {
                v = red[0][g][wave][lane];
#pragma unroll
                for (int w = 1; w < KS; ++w) v += red[SPLIT ? w : 0][g][wave][lane];
            }
            pre[g] = v + *(const f4 *)(a.bias + d * G + g * O + uo);
        }
        const long long vo = sbase + evox[e];
        f4 c, h;
        us4 hbv;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float gi = fsig(pre[0][i]), gf = fsig(pre[1][i]);
            const float gg = ftanh(pre[2][i]), go = fsig(pre[3][i]);
            c[i] = gg * gi + cprev[e][i] * gf;
            h[i] = go * ftanh(c[i]);
            hbv[i] = f32_to_bf16(h[i]);
        }
        *(f4 *)(a.cell + vo * O + uo) = c;
        *(us4 *)(a.hb + vo * O + uo) = hbv;
    }
}

// LDS-staged variant (steps with enough blocks): a workgroup takes a BP x BQ
// block of 64 pixels of one plane and all U unit groups (wave w: units
// 16 w .. 16 w + 15).  x_t and h_{t-1} of the block and its filter halo are
// staged once into LDS (16-byte chunks of 8 channels, [x | h] per pixel, the
// chunk index XOR-swizzled by the pixel), and every tap reads its B operand
// from there instead of from L1: the taps of a pixel share one staged copy.
// The A fragments stream from global memory as in k_step_fwd_b16.  Tile nt
// of the block is its pixels 16 nt .. 16 nt + 15 in row-major order.
template <int U>
__global__ void __launch_bounds__(64 * U) __attribute__((amdgpu_waves_per_eu(3)))
k_step_fwd_b16_blk(FwdB16Args a)
{
    constexpr int O = 16 * U, G = 4 * O, UH = O / 32;
    extern __shared__ bf8 stg[];
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int ug = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int blk = blockIdx.x;
    if (blk >= a.base[kDirs]) return;
    const int d = item_dir(a.base, blk);
    const DirGeom dg = a.g.dir[d];
    int r = blk - a.base[d];
    const int n = r / a.nblk[d];
    r -= n * a.nblk[d];
    const int BP = a.bp[d], BQ = a.bq[d];
    const int bi = r / a.nbq[d], bj = r - bi * a.nbq[d];
    const int p0 = bi * BP, q0 = bj * BQ;
    const int t = a.t;
    const int s = dg.sign > 0 ? t : dg.T - 1 - t;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int P = dg.P, Q = dg.Q;
    const long long V = a.g.V;
    const int C32 = a.C32, CX = C32 >> 5, KX = a.KX;
    const int hoff = -dg.sign * ss;
    const int uo = ug * 16 + 4 * q4;
    const int KQ = a.g.KQ, radp = a.g.KP >> 1, radq = KQ >> 1;
    const int SW = BQ + 2 * radq, SH = BP + 2 * radp;     // staged block with halo
    const int NXC = C32 >> 3, NCH = NXC + (O >> 3);      // 16-byte chunks per staged pixel
    const int swm = (NCH & 7) == 0 ? 7 : 3;              // swizzle within the pixel's chunks
    const long long sbase = ((long long)d * a.g.N + n) * V;
    // byte sizes: V * C32 * 2 and V * O * 2 (< 2^31, checked on the host)
    const auto rs_x = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(a.xb + (long long)n * V * C32), (short)0, (int)(V * C32 * 2),
        kRsrcWord3);
    const auto rs_h = __builtin_amdgcn_make_buffer_rsrc(a.hb + sbase * O, (short)0,
                                                        (int)(V * O * 2), kRsrcWord3);
    const auto rs_c = slice_rsrc(a.cell + sbase * O, V * O);

    // ---- stage [x_t | h_{t-1}] of the block and its halo (zero off the plane)
    // with direct-to-LDS loads, all in flight at once: one instruction fills
    // 64 consecutive 16-byte slots, slot p of pixel spx holding chunk
    // p ^ (spx & swm), each lane loading the chunk its slot holds; x and h
    // chunks go out as two instructions masked by source
    const int nst = SH * SW * NCH;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    for (int e0 = wv * 64; e0 < nst; e0 += 64 * U) {
        const int e = e0 + (threadIdx.x & 63);
        const int spx = e / NCH, pos = e - spx * NCH;
        const int c = pos ^ (spx & swm);
        const int sy = spx / SW, sx = spx - sy * SW;
        const int pp = p0 - radp + sy, qq = q0 - radq + sx;
        const bool on = on_plane(pp, qq, P, Q);
        const int v = s * ss + pp * sp + qq * sq;
        lds_void *dst = (lds_void *)&stg[e0];
        if (e < nst) {
            if (c < NXC)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rs_x, dst, 16, (int)sel_off(on, (unsigned)(v * C32 + 8 * c) * 2u), 0, 0, 0);
            else
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rs_h, dst, 16,
                    (int)sel_off(on && t > 0, (unsigned)((v + hoff) * O + 8 * (c - NXC)) * 2u),
                    0, 0, 0);
        }
    }

    // this lane's pixel of each tile (block row-major; BQ is a power of two)
    const int lbq = 31 - __builtin_clz(BQ);
    int spix[kNT], evox[kNT];
    bool elive[kNT];
    f4 cprev[kNT];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        const int e = nt * 16 + col;
        const int ey = e >> lbq, ex = e & (BQ - 1);
        spix[nt] = (ey + radp) * SW + ex + radq;
        const int pp = p0 + ey, qq = q0 + ex;
        elive[nt] = on_plane(pp, qq, P, Q);
        evox[nt] = s * ss + (elive[nt] ? pp * sp + qq * sq : 0);
        cprev[nt] = bload4(rs_c, sel_off(t > 0 && elive[nt],
                                         (unsigned)((evox[nt] + hoff) * O + uo) * 4u));
    }
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();

    f4 acc[4][kNT];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[g][nt] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    const uint16_t *fr = a.frag + (long long)(d * U + ug) * a.KG * 2048 + lane * 8;
    auto load_a = [&](int kg, bf8 (&av)[4]) {
#pragma unroll
        for (int g = 0; g < 4; ++g) av[g] = *(const bf8 *)(fr + (kg * 4 + g) * 512);
    };
    const int KG = t > 0 ? a.KG : KX;
    bf8 acur[4], anxt[4];
    load_a(0, acur);
    for (int kg = 0; kg < KG; ++kg) {
        if (kg + 1 < KG) load_a(kg + 1, anxt);
        const bool is_x = kg < KX;
        const int kk = is_x ? kg : kg - KX;
        const int tap = is_x ? (kk * a.cx_mul32) >> 16 : kk / UH;
        const int cb = kk - tap * (is_x ? CX : UH);
        const int row = tap_row(tap, a.k_mul), ka = row - radp, kb = tap - row * KQ - radq;
        const int chunk = (is_x ? 0 : NXC) + cb * 4 + q4;
        const int doff = ka * SW + kb;
        bf8 bv[kNT];
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) {
            const int spx = spix[nt] + doff;
            bv[nt] = stg[spx * NCH + (chunk ^ (spx & swm))];
        }
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt) acc[g][nt] = mfma_bf16(acur[g], bv[nt], acc[g][nt]);
#pragma unroll
        for (int g = 0; g < 4; ++g) acur[g] = anxt[g];
    }

#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        if (!elive[nt]) continue;
        f4 pre[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) pre[g] = acc[g][nt] + *(const f4 *)(a.bias + d * G + g * O + uo);
        const long long vo = sbase + evox[nt];
        f4 c, h;
        us4 hbv;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float gi = fsig(pre[0][i]), gf = fsig(pre[1][i]);
            const float gg = ftanh(pre[2][i]), go = fsig(pre[3][i]);
            c[i] = gg * gi + cprev[nt][i] * gf;
            h[i] = go * ftanh(c[i]);
            hbv[i] = f32_to_bf16(h[i]);
        }
        *(f4 *)(a.cell + vo * O + uo) = c;
        *(us4 *)(a.hb + vo * O + uo) = hbv;
    }
}

// Macro-tiled variant (the default where its LDS fits): a workgroup of
// NW = WM WN waves takes a (4 WN) x 16 block of pixels of one plane and all
// 4O gate rows.  Wave (wm, wn) computes the UGW = U / WM unit groups from
// UGW wm (4 UGW 16-row gate tiles) for block rows 4 wn .. 4 wn + 3 (four
// 16-pixel tiles, one block row each), so every A fragment read from LDS
// feeds four MFMAs and every B fragment 4 UGW.
// - [x_t | h_{t-1}] of the block and its filter halo is staged once, with
//   direct-to-LDS loads as in k_step_fwd_b16_blk; the staged pixel is padded
//   to NCH + 2 chunks (a stride of 8 mod 16 floats), so the 16 lanes that
//   read one chunk of 16 consecutive pixels hit distinct banks.
// - The A fragments of a K-group (4O gate rows x 32 channels, 1 KB per
//   16-row tile) stream through a ring of three LDS arrays, also with
//   direct-to-LDS loads issued two K-groups ahead.  Step kg reads K-group
//   kg + 1 into registers and refills the array that held kg with kg + 3;
//   its barrier publishes kg + 2 (each wave has waited for its own share)
//   and frees the array of kg + 1, which step kg + 1 refills (each wave has
//   waited for its reads).  The arrays are distinct objects and each step names its
//   two statically (the loop is unrolled by six), so the compiler knows that
//   the reads do not touch the array a load is still filling.
// - The reads of K-group kg + 1 are interleaved with kg's MFMAs (one A and
//   at most one B fragment per four MFMAs, the ring load mid-step), so
//   neither waits on the other.
// - 16-unit layers with at most 8 input channels pack their taps (PK): each
//   lane group q of a K-group reads its own 8-channel slot, one input tap or
//   half of an h tap, so a K-group holds four input taps or two h taps instead
//   of one padded to 32 channels.  The staged pixel then has one x chunk, two
//   h chunks and three pad chunks.
// - c^d is needed one plane later only, so it lives in a two-plane buffer
//   (100 MB for the stacked network's 64-unit layer) that stays in the
//   memory-side cache instead of a volume written out to HBM.
// Workgroups are remapped so that each XCD runs a contiguous range of blocks
// (at most two directions' weights per L2).
template <int U, int WM, int WN, int MODE>
__global__ void __launch_bounds__(64 * WM * WN)
__attribute__((amdgpu_waves_per_eu(U / WM == 1 ? 3 : 2)))
k_step_fwd_b16_mt(FwdB16Args a)
{
    constexpr int O = 16 * U, G = 4 * O, NW = WM * WN, T = 4 * U;
    constexpr bool PK = U == 1;                 // packed taps
    constexpr int UGW = U / WM, AT = 4 * UGW;   // unit groups and A tiles per wave
    constexpr int BP = 4 * WN, BQ = 16;
    constexpr int NDMA = T / NW;             // ring loads per wave per K-group
    static_assert(U % WM == 0 && (UGW == 1 || UGW == 2), "one or two unit groups per wave");
    static_assert(T % NW == 0 && NDMA < 16, "ring tiles split evenly over the waves");
    constexpr int kWaitRingLds = 0x0070 | NDMA;  // s_waitcnt vmcnt(NDMA) lgkmcnt(0)
    constexpr int kWaitAllLds = 0x0070;          // s_waitcnt vmcnt(0) lgkmcnt(0)
    __shared__ bf8 ring0[T * 64], ring1[T * 64], ring2[T * 64];
    extern __shared__ bf8 stg[];             // [SH][SW][NCH + 2]: staged pixels
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wv % WM, wn = wv / WM;
    const int per_xcd = gridDim.x / kXcds;
    const int blk = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    if (blk >= a.base[kDirs]) return;
    const int d = item_dir(a.base, blk);
    const DirGeom dg = a.g.dir[d];
    int r = blk - a.base[d];
    int n, t_ = a.t;
    if constexpr (MODE == 1) {
        // projection: every plane of the direction in one launch
        const int per_n = dg.T * a.nblk[d];
        n = r / per_n;
        r -= n * per_n;
        t_ = r / a.nblk[d];
        r -= t_ * a.nblk[d];
    } else {
        n = r / a.nblk[d];
        r -= n * a.nblk[d];
    }
    const int t = t_;
    const int bi = r / a.nbq[d], bj = r - bi * a.nbq[d];
    const int p0 = bi * BP, q0 = bj * BQ;
    const int s = dg.sign > 0 ? t : dg.T - 1 - t;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int P = dg.P, Q = dg.Q;
    const long long V = a.g.V;
    const int C32 = a.C32, CX = C32 >> 5, KX = a.KX, KGA = a.KG;
    const int hoff = -dg.sign * ss;
    const int KQ = a.g.KQ, radp = a.g.KP >> 1, radq = KQ >> 1;
    const int SW = BQ + 2 * radq, SH = BP + 2 * radp;
    const int NXC = C32 >> 3, NCH = NXC + (MODE == 1 ? 0 : O >> 3), NCHP = PK ? 6 : NCH + 2;
    const int KK = a.g.KP * KQ;
    const long long sbase = ((long long)d * a.g.N + n) * V;
    // byte sizes: V * C32 * 2, V * O * 2 and U * KG * 4096 (< 2^31, checked on the host)
    const auto rs_x = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(a.xb + (long long)n * V * C32), (short)0, (int)(V * C32 * 2),
        kRsrcWord3);
    const auto rs_h = __builtin_amdgcn_make_buffer_rsrc(a.hb + sbase * O, (short)0,
                                                        (int)(V * O * 2), kRsrcWord3);
    const auto rs_a = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(a.frag + (long long)d * U * KGA * 2048), (short)0,
        U * KGA * 4096, kRsrcWord3);
    // c of this block's pixels: plane parity t & 1 of the two-plane buffer,
    // c_{t-1} from the other parity
    const long long cpq = (long long)a.pqmax * O;
    float *cpl = a.cpp + ((long long)d * a.g.N + n) * 2 * cpq;
    const auto rs_c = slice_rsrc(cpl + ((t + 1) & 1) * cpq, cpq);

    // A fragments of K-group kg into a ring array: tile j = 4 ug + gate
    auto issue_a = [&](int kg, bf8 *slot) {
#pragma unroll
        for (int j0 = 0; j0 < T; j0 += NW) {
            const int j = j0 + wv, ug = j >> 2, gt = j & 3;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rs_a, (lds_void *)&slot[j * 64], 16,
                (int)((unsigned)(((ug * KGA + kg) * 4 + gt) * 512 + lane * 8) * 2u), 0, 0, 0);
        }
    };

    // ---- stage [x_t | h_{t-1}] of the block and its halo (zero off the
    // plane, before the first plane and in the two pad chunks): one
    // instruction fills 64 consecutive 16-byte slots, x and h chunks as two
    // instructions masked by source
    const int nst = SH * SW * NCHP;
    for (int e0 = wv * 64; e0 < nst; e0 += 64 * NW) {
        const int e = e0 + lane;
        const int spx = e / NCHP, c = e - spx * NCHP;
        const int sy = spx / SW, sx = spx - sy * SW;
        const int pp = p0 - radp + sy, qq = q0 - radq + sx;
        const bool on = on_plane(pp, qq, P, Q);
        const int v = s * ss + pp * sp + qq * sq;
        lds_void *dst = (lds_void *)&stg[e0];
        if (e < nst) {
            if (c < NXC)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rs_x, dst, 16, (int)sel_off(on, (unsigned)(v * C32 + 8 * c) * 2u), 0, 0, 0);
            else
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rs_h, dst, 16,
                    (int)sel_off(on && t > 0 && c < NCH,
                                 (unsigned)((v + hoff) * O + 8 * (c - NXC)) * 2u),
                    0, 0, 0);
        }
    }
    const int KG = MODE == 1 ? KX : (t > 0 ? KGA : KX);   // KX = 0 for MODE 2
    // only the recurrent-only mode has no K-group (its first plane)
    const bool any_kg = MODE != 2 || KG > 0;
    if (any_kg) issue_a(0, ring0);
    if (KG > 1) issue_a(1, ring1);
    if (KG > 2) issue_a(2, ring2);

    // staged chunk of this lane in tile nt (block row 4 wn + nt) at tap
    // (0, 0), channel chunk q4 (chunk 0 with packed taps)
    int spb[kNT];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt)
        spb[nt] = ((4 * wn + nt + radp) * SW + col + radq) * NCHP + (PK ? 0 : q4);
    // B offset of K-group kg past spb: tap shift and chunk block (uniform),
    // with packed taps the lane's own slot (a slot past the last tap, whose
    // weights are zero, reads the last tap)
    auto b_off = [&](int kg) {
        if constexpr (PK) {
            const bool is_x = kg < KX;
            const int slot = 4 * (is_x ? kg : kg - KX) + q4;
            const int tap = min(is_x ? slot : slot >> 1, KK - 1);
            const int row = tap_row(tap, a.k_mul), ka = row - radp, kb = tap - row * KQ - radq;
            return (ka * SW + kb) * NCHP + (is_x ? 0 : NXC + (slot & 1));
        }
        const bool is_x = kg < KX;
        const int kk = is_x ? kg : kg - KX;
        const int tap = is_x ? (kk * a.cx_mul32) >> 16 : kk / (O / 32);
        const int cb = kk - tap * (is_x ? CX : O / 32);
        const int row = tap_row(tap, a.k_mul), ka = row - radp, kb = tap - row * KQ - radq;
        return (ka * SW + kb) * NCHP + (is_x ? 0 : NXC) + cb * 4;
    };

    struct Ops {
        bf8 a[AT];
        bf8 b[kNT];
    };
    f4 acc[AT][kNT];
#pragma unroll
    for (int i = 0; i < AT; ++i)
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[i][nt] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    auto mfmas = [&](const Ops &o) {
#pragma unroll
        for (int i = 0; i < AT; ++i)
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt) acc[i][nt] = mfma_bf16(o.a[i], o.b[nt], acc[i][nt]);
    };
    auto step = [&](int kg, const Ops &cur, Ops &nxt, const bf8 *rd, bf8 *dm) {
        const int bb = b_off(kg + 1);
        const bool more = kg + 3 < KG;
#pragma unroll
        for (int i = 0; i < AT; ++i) {
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt) acc[i][nt] = mfma_bf16(cur.a[i], cur.b[nt], acc[i][nt]);
            if (i == AT / 2 && more) issue_a(kg + 3, dm);
            nxt.a[i] = rd[(AT * wm + i) * 64 + lane];
            if (AT == 2 * kNT) {
                if (i & 1) nxt.b[i >> 1] = stg[spb[i >> 1] + bb];
            } else if (i < kNT) {
                nxt.b[i] = stg[spb[i] + bb];
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // the reads done, this wave's share of kg + 2 landed (kg + 3 may stay
        // in flight), then the barrier; no fence: one would also wait for
        // kg + 3.  The empty asm keeps the compiler from moving LDS accesses
        // across the barrier.
        if (more)
            __builtin_amdgcn_s_waitcnt(kWaitRingLds);
        else
            __builtin_amdgcn_s_waitcnt(kWaitAllLds);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };

    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
    Ops X, Y;
    if (any_kg) {
        const int bb = b_off(0);
#pragma unroll
        for (int i = 0; i < AT; ++i) X.a[i] = ring0[(AT * wm + i) * 64 + lane];
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) X.b[nt] = stg[spb[nt] + bb];
    }
    // step 0 refills ring0: every wave has read K-group 0 from it first
    if (any_kg) __syncthreads();
    // after step kg the operands of kg + 1 are in Y for even kg, X for odd
    for (int kg = 0; kg + 1 < KG; kg += 6) {
        step(kg, X, Y, ring1, ring0);
        if (kg + 2 < KG) step(kg + 1, Y, X, ring2, ring1);
        if (kg + 3 < KG) step(kg + 2, X, Y, ring0, ring2);
        if (kg + 4 < KG) step(kg + 3, Y, X, ring1, ring0);
        if (kg + 5 < KG) step(kg + 4, X, Y, ring2, ring1);
        if (kg + 6 < KG) step(kg + 5, Y, X, ring0, ring2);
    }
    if ((KG - 1) & 1) X = Y;

    // epilogue operands, in flight during the last K-group's MFMAs
    const int ug0 = UGW * wm;
    f4 bias[UGW][4], cprev[UGW][kNT];
    int evox[kNT], epix[kNT];
    bool elive[kNT];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        const int pp = p0 + 4 * wn + nt, qq = q0 + col;
        elive[nt] = on_plane(pp, qq, P, Q);
        evox[nt] = s * ss + (elive[nt] ? pp * sp + qq * sq : 0);
        epix[nt] = elive[nt] ? pp * Q + qq : 0;
    }
#pragma unroll
    for (int ui = 0; ui < UGW; ++ui) {
        const int uo = (ug0 + ui) * 16 + 4 * q4;
#pragma unroll
        for (int gt = 0; gt < 4; ++gt)
            bias[ui][gt] = MODE == 2 ? f4{0.0f, 0.0f, 0.0f, 0.0f}
                                     : *(const f4 *)(a.bias + d * G + gt * O + uo);
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt)
            cprev[ui][nt] = bload4(rs_c, sel_off(MODE != 1 && t > 0 && elive[nt],
                                                 (unsigned)(epix[nt] * O + uo) * 4u));
    }
    if (any_kg) mfmas(X);

#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        if (!elive[nt]) continue;
        const long long vo = sbase + evox[nt];
#pragma unroll
        for (int ui = 0; ui < UGW; ++ui) {
            const int uo = (ug0 + ui) * 16 + 4 * q4;
            f4 pre[4];
#pragma unroll
            for (int gt = 0; gt < 4; ++gt) pre[gt] = acc[ui * 4 + gt][nt] + bias[ui][gt];
            if constexpr (MODE == 1) {
                // x's part of the pre-activations (and the bias), rounded to bf16
#pragma unroll
                for (int gt = 0; gt < 4; ++gt) {
                    us4 pv;
#pragma unroll
                    for (int i = 0; i < 4; ++i) pv[i] = f32_to_bf16(pre[gt][i]);
                    *(us4 *)(a.preact + vo * G + gt * O + uo) = pv;
                }
                continue;
            }
            if constexpr (MODE == 2) {
#pragma unroll
                for (int gt = 0; gt < 4; ++gt) {
                    const us4 pv = *(const us4 *)(a.preact + vo * G + gt * O + uo);
#pragma unroll
                    for (int i = 0; i < 4; ++i) pre[gt][i] += bf16_to_f32(pv[i]);
                }
            }
            f4 c;
            us4 hbv;
            lstm_cell4_b16(pre, cprev[ui][nt], c, hbv);
            *(f4 *)(cpl + (t & 1) * cpq + epix[nt] * O + uo) = c;
            *(us4 *)(a.hb + vo * O + uo) = hbv;
        }
    }
}

// Two plane steps per launch for 16-unit layers on packed taps with 3 x 3
// filters: Eq. (7)-(12) for planes t and t + 1 of every direction.  These
// steps are bound by each launch's fixed latency (staging, a contraction of
// eight K-groups, the epilogue), not by their work, so a workgroup takes a
// 16 x 16 block through both planes:
// - it stages x_t, x_{t+1} and h_{t-1} on the block and a two-pixel halo
//   (a 20 x 20 grid of six 16-byte chunks per pixel: x_t, h_{t-1} twice,
//   x_{t+1}, and h_t twice, written by step t);
// - step t covers the block and the one-pixel ring around it, whose h_t the
//   block's step t + 1 reads (the ring is also computed, identically, by the
//   neighbouring blocks: 27% more work for step t in exchange for half the
//   launches); h_t goes to LDS (zero off the plane) and, for the block, to h^d;
// - step t + 1 covers the block.  Wave w takes block rows 2w and 2w + 1 in
//   both steps, so c_t of its pixels stays in its registers; the 68 ring
//   pixels fill five more tiles, one each for waves 0-4.
// All eight K-groups of A fragments stay in LDS.  The contraction, its order
// and the cell update are those of k_step_fwd_b16_mt, so h^d and c^d are the
// same bit for bit.  c^d alternates between the halves of the two-plane
// buffer by launch: launch L = t / 2 reads c_{t-1} from half (L + 1) & 1 and
// writes c_{t+1} to half L & 1 (a neighbour may still read c_{t-1} of this
// block's pixels).  Every direction's plane count must be even.
constexpr int kS2Grid = 20, kS2Chunks = 6, kS2KG = 8;

template <int NT>
__device__ inline void s2_contract(const bf8 *afr, const bf8 *stg, const int (&pb)[NT], int xch,
                                   int hch, int q4, int lane, f4 (&acc)[NT][4])
{
#pragma unroll
    for (int i = 0; i < NT; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) acc[i][g] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kg = 0; kg < kS2KG; ++kg) {
        // packed taps: input slot 4 kg + q4 is tap 4 kg + q4; h slot
        // 4 (kg - 3) + q4 is half slot & 1 of tap slot / 2; slots past the
        // ninth tap carry zero weights and read the last tap
        const bool is_x = kg < 3;
        const int slot = 4 * (is_x ? kg : kg - 3) + q4;
        const int tap = min(is_x ? slot : slot >> 1, 8);
        const int ka = tap / 3 - 1, kb = tap - (tap / 3) * 3 - 1;
        const int off = (ka * kS2Grid + kb) * kS2Chunks + (is_x ? xch : hch + (slot & 1));
        bf8 av[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) av[g] = afr[(kg * 4 + g) * 64 + lane];
#pragma unroll
        for (int i = 0; i < NT; ++i) {
            const bf8 bv = stg[pb[i] + off];
#pragma unroll
            for (int g = 0; g < 4; ++g) acc[i][g] = mfma_bf16(av[g], bv, acc[i][g]);
        }
    }
}

// eight waves of two block rows each: 118 VGPRs, two workgroups (16 waves)
// per CU; four waves of four rows (198 VGPRs, 8 waves per CU) took 9% longer
constexpr int kS2Waves = 8;

template <int NWV>
__global__ void __launch_bounds__(64 * NWV) __attribute__((amdgpu_waves_per_eu(NWV == 8 ? 4 : 2)))
k_step2_fwd_b16_pk(FwdB16Args a)
{
    constexpr int O = 16, G = 4 * O, SG = kS2Grid, NC = kS2Chunks, KG = kS2KG;
    constexpr int RPW = 16 / NWV;             // block rows per wave
    __shared__ bf8 afr[KG * 4 * 64];          // A fragments [kg][gate][lane]
    extern __shared__ bf8 stg[];              // [SG][SG][NC]
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int per_xcd = gridDim.x / kXcds;
    const int blk = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    if (blk >= a.base[kDirs]) return;
    const int d = item_dir(a.base, blk);
    const DirGeom dg = a.g.dir[d];
    int r = blk - a.base[d];
    const int n = r / a.nblk[d];
    r -= n * a.nblk[d];
    const int bi = r / a.nbq[d], bj = r - bi * a.nbq[d];
    const int p0 = bi * 16, q0 = bj * 16;
    const int t = a.t;                         // even: this launch makes planes t and t + 1
    const int s = dg.sign > 0 ? t : dg.T - 1 - t;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int P = dg.P, Q = dg.Q;
    const int nxt = dg.sign * ss;              // voxel offset of the next plane
    const long long V = a.g.V;
    const long long sbase = ((long long)d * a.g.N + n) * V;
    // byte sizes: V * 16, V * O * 2 and KG * 4096 (< 2^31, checked on the host)
    const auto rs_x = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(a.xb + (long long)n * V * 8), (short)0, (int)(V * 16), kRsrcWord3);
    const auto rs_h = __builtin_amdgcn_make_buffer_rsrc(a.hb + sbase * O, (short)0,
                                                        (int)(V * O * 2), kRsrcWord3);
    const auto rs_a = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(a.frag + (long long)d * KG * 2048), (short)0, KG * 4096,
        kRsrcWord3);
    const long long cpq = (long long)a.pqmax * O;
    float *cpl = a.cpp + ((long long)d * a.g.N + n) * 2 * cpq;
    const int half = (t >> 1) & 1;
    const auto rs_c = slice_rsrc(cpl + (half ^ 1) * cpq, cpq);
    float *cw = cpl + half * cpq;

    // A fragments, tile j = 4 kg + gate
#pragma unroll
    for (int j0 = 0; j0 < KG * 4; j0 += NWV) {
        const int j = j0 + wv;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_a, (lds_void *)&afr[j * 64], 16,
                                                 (int)((unsigned)(j * 512 + lane * 8) * 2u), 0, 0,
                                                 0);
    }
    // staged grid: pixel (gy, gx) is plane pixel (p0 - 2 + gy, q0 - 2 + gx);
    // zero off the plane, h_{t-1} zero before the first plane, chunks 4-5
    // zero until step t writes them
    constexpr int nst = SG * SG * NC;
    for (int e0 = wv * 64; e0 < nst; e0 += 64 * NWV) {
        const int e = e0 + lane;
        const int spx = e / NC, c = e - spx * NC;
        const int gy = spx / SG, gx = spx - gy * SG;
        const int pp = p0 - 2 + gy, qq = q0 - 2 + gx;
        const bool on = on_plane(pp, qq, P, Q);
        const int v = s * ss + pp * sp + qq * sq;
        lds_void *dst = (lds_void *)&stg[e0];
        if (e < nst) {
            if (c == 0 || c == 3)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rs_x, dst, 16, (int)sel_off(on, (unsigned)((c == 0 ? v : v + nxt) * 8) * 2u),
                    0, 0, 0);
            else
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rs_h, dst, 16,
                    (int)sel_off(on && t > 0 && c < 3, (unsigned)((v - nxt) * O + 8 * (c - 1)) * 2u),
                    0, 0, 0);
        }
    }
    const int uo = 4 * q4;
    f4 bias[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) bias[g] = *(const f4 *)(a.bias + d * G + g * O + uo);
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();

    // gates and cell update of one tile (as in k_step_fwd_b16_mt)
    auto cell = [&](const f4 (&acc)[4], const f4 &cprev, f4 &c, us4 &hbv) {
        f4 pre[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) pre[g] = acc[g] + bias[g];
        lstm_cell4_b16(pre, cprev, c, hbv);
    };
    // h_t of staged pixel spx into chunks 4-5 (units uo .. uo + 3)
    auto put_h = [&](int spx, us4 v) {
        *(us4 *)((char *)stg + (size_t)(spx * NC + 4) * 16 + q4 * 8) = v;
    };

    // ---- step t, block rows RPW wv .. RPW wv + RPW - 1
    int pb[RPW];
#pragma unroll
    for (int nt = 0; nt < RPW; ++nt) pb[nt] = ((RPW * wv + nt + 2) * SG + col + 2) * NC;
    bool live[RPW];
    int pix[RPW];
    f4 cprev[RPW], ct[RPW];
#pragma unroll
    for (int nt = 0; nt < RPW; ++nt) {
        const int pp = p0 + RPW * wv + nt, qq = q0 + col;
        live[nt] = on_plane(pp, qq, P, Q);
        pix[nt] = live[nt] ? pp * Q + qq : 0;
        cprev[nt] = bload4(rs_c, sel_off(t > 0 && live[nt], (unsigned)(pix[nt] * O + uo) * 4u));
    }
    {
        f4 acc[RPW][4];
        s2_contract<RPW>(afr, stg, pb, 0, 1, q4, lane, acc);
#pragma unroll
        for (int nt = 0; nt < RPW; ++nt) {
            us4 hbv;
            cell(acc[nt], cprev[nt], ct[nt], hbv);
            if (!live[nt]) hbv = us4{0, 0, 0, 0};
            put_h(pb[nt] / NC, hbv);
            if (live[nt]) {
                const int pp = p0 + RPW * wv + nt, qq = q0 + col;
                *(us4 *)(a.hb + (sbase + s * ss + pp * sp + qq * sq) * O + uo) = hbv;
            }
        }
    }
    // ---- step t, the ring: index k < 68 walks the top row, the bottom row,
    // then the left and right columns of the 18 x 18 region around the block
    for (int j = wv; j < 5; j += NWV) {
        const int k = 16 * j + col;
        const bool slot = k < 68;
        int rr, cc;
        if (k < 18) { rr = 0; cc = k; }
        else if (k < 36) { rr = 17; cc = k - 18; }
        else if (k < 52) { rr = k - 36 + 1; cc = 0; }
        else if (k < 68) { rr = k - 52 + 1; cc = 17; }
        else { rr = 0; cc = 0; }
        const int pp = p0 - 1 + rr, qq = q0 - 1 + cc;
        const bool on = slot && on_plane(pp, qq, P, Q);
        const f4 cp = bload4(rs_c, sel_off(t > 0 && on, (unsigned)((on ? pp * Q + qq : 0) * O + uo) * 4u));
        int rb[1] = {((rr + 1) * SG + cc + 1) * NC};
        f4 acc[1][4];
        s2_contract<1>(afr, stg, rb, 0, 1, q4, lane, acc);
        f4 c;
        us4 hbv;
        cell(acc[0], cp, c, hbv);
        if (!on) hbv = us4{0, 0, 0, 0};
        if (slot) put_h(rb[0] / NC, hbv);
    }
    __syncthreads();

    // ---- step t + 1 of the block: x_{t+1} in chunk 3, h_t in chunks 4-5
    {
        f4 acc[RPW][4];
        s2_contract<RPW>(afr, stg, pb, 3, 4, q4, lane, acc);
#pragma unroll
        for (int nt = 0; nt < RPW; ++nt) {
            if (!live[nt]) continue;
            f4 c;
            us4 hbv;
            cell(acc[nt], ct[nt], c, hbv);
            const int pp = p0 + RPW * wv + nt, qq = q0 + col;
            *(f4 *)(cw + pix[nt] * O + uo) = c;
            *(us4 *)(a.hb + (sbase + s * ss + nxt + pp * sp + qq * sq) * O + uo) = hbv;
        }
    }
}

// ---- backward step ----------------------------------------------------------

struct BwdStepArgs {
    Geom g;
    int t;
    const float *frag;        // [6][U][KK * 4U][64][4]
    int k_mul;                // ceil(2^16 / K)
    const float *gates, *cell, *dh;
    float *dA;                // [6][N][V][4O]
    float *gcf;               // [6][N][V][O]: dL/dc_t * f_t
    int npg[kDirs];
    int base[kDirs + 1];
    // pixel blocks of the LDS-staged kernel (as in FwdStepArgs) and one
    // wave's LDS region in 16-byte units (its staged block + filter halo, or
    // its partial sums, whichever is larger)
    int bp[kDirs], bq[kDirs], nbq[kDirs], nblk[kDirs];
    int reg_f4;
    // dL/dx inside the staged reverse step: W_x^T fragments
    // [6][KK * 4U][CT][64][4] and each direction's share [6][N][V][C]
    const float *fragx;
    float *dxd;
};

// ---- line blocks of the 2D layer's reverse sweep (16 hidden units) ----------
// The reverse of k_line_fwd: a workgroup owns a 64-pixel segment and goes
// back S lines per launch with overlapped tiles.  At reverse line j it
// computes the segment widened by (S - j) r pixels on each side: line j + 1
// reads all but the outer r of them (the outer r serve dL/dx).  dA_{t+1} (64
// gate-units per pixel, 16-byte chunks XOR-swizzled by the pixel; overwritten
// after a barrier) and gc_{t+1} f_{t+1} (in place) stay in LDS, and so does
// the c_{t-1} read at line t, which is the next line's c.  The saved gates and
// dL/dh are read per tile; only the segment's own dA_t is stored, and gc_t f_t
// on the launch's last line.  Pixels past the line keep dA = 0.
//   gh = dL/dh + sum_taps W_h^T dA_{t+1}[p - tap]                 (MFMA)
//   gc = gh o (1 - tanh^2 c) + (gc f)_{t+1}
//   dA_i = gc g i (1 - i), dA_f = gc c_{t-1} f (1 - f), dA_g = gc i (1 - g^2),
//   dA_o = gh tanh(c) o (1 - o)
// With dxd (C <= 4) the line also gives this direction's share of dL/dx,
//   dxd[p] = sum_taps W_x^T dA_t[p - tap],
// from dA_t in LDS: the computed range is one radius wider than the next
// line needs, so the segment's taps are all there.  Wave w sums gate w's 16
// units for the segment's 64 pixels; the four partials meet in LDS and are
// added, in order, after the next barrier.
// With dbp the segment's dA_t columns are summed too (db): per lane over its
// central pixels, then over the lanes and waves in a fixed order, and added
// to the (image, segment) partial of the earlier launches.
struct LineBwdArgs {
    Geom g;
    int r0, S;                  // first reverse step of this launch, steps per launch
    const float *frag;          // [6][KK * 4][64][4] W_h^T fragments
    const float *gates, *cell, *dh;
    float *dA, *gcf;
    const float *wx;            // [4][4O][C][K] input filters (dxd only)
    float *dxd;                 // [4][N][V][C] per-direction dL/dx, or null
    float *dbp;                 // [4][N][nsegmax][4O] bias-gradient partials, or null
    int nsegmax;                // segments of the longest line
    int nseg[kDirs];
    int base[kDirs + 1];
};

// LDS bytes of k_line_bwd beyond its static arrays: W_h^T fragments, one line
// of dA and, for dL/dx, the input filters.
inline size_t line_bwd_dyn_lds(int KG, int wx_floats)
{
    return (size_t)KG * 64 * 16 + (size_t)kLineSlots * 256 + (size_t)(wx_floats + 3) / 4 * 16;
}

// One wave's share of a segment pixel's dL/dx in the reverse line blocks:
// gate w's 16 units over the taps, CC channels.  dab: one line of dA (16
// chunks of 4 gate-units per pixel, chunk ^ (slot & 15)); wxl: [K][4O][CC]
// input filters (wave-uniform reads); cs: the pixel's slot.
template <int CC>
__device__ inline f4 line_dx_px(const f4 *dab, const float *wxl, int cs, int rq, int KQ, int wave)
{
    constexpr int G = 64;
    f4 px = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int tap = 0; tap < KQ; ++tap) {
        const int sx = cs - (tap - rq);
        const f4 *wp = (const f4 *)(wxl + (tap * G + wave * 16) * CC);
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            const f4 v = dab[sx * 16 + ((wave * 4 + h) ^ (sx & 15))];
            f4 w[CC];                       // units 4h .. 4h + 3, CC channels each
#pragma unroll
            for (int k = 0; k < CC; ++k) w[k] = wp[h * CC + k];
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4)
#pragma unroll
                for (int c = 0; c < CC; ++c) {
                    const int e = i4 * CC + c;
                    px[c] += v[i4] * w[e >> 2][e & 3];
                }
        }
    }
    return px;
}

__global__ void __launch_bounds__(256)
k_line_bwd(LineBwdArgs a)
{
    constexpr int O = 16, G = 64;
    __shared__ f4 gcb[kLineSlots][4];           // gc f, chunk ^ (slot & 3)
    __shared__ f4 dxr[4][64];                   // dL/dx partials of the four waves
    __shared__ f4 cl[kLineSlots][4];            // c_{t-1} read at line t: line t - 1's c
    __shared__ f4 dbr[4][4][4];                 // bias-gradient sums [wave][gate][q4]
    extern __shared__ f4 dyn[];
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int blk = blockIdx.x;
    if (blk >= a.base[kDirs]) return;
    const int d = item_dir(a.base, blk);
    const DirGeom dg = a.g.dir[d];
    int r = blk - a.base[d];
    const int n = r / a.nseg[d], seg = r - n * a.nseg[d];
    const int Q = dg.Q, rq = a.g.KQ >> 1, S = a.S, KG = a.g.KQ * 4;
    const int q0 = seg * kLineSeg;
    const int pbase = q0 - (S + 1) * rq;       // pixel of LDS slot 0
    const int ss = (int)dg.ss, sq = (int)dg.sq, T = dg.T;
    const long long V = a.g.V;
    const long long sbase = ((long long)d * a.g.N + n) * V;
    const int C = a.g.C, KQ = a.g.KQ;
    const bool want_dx = a.dxd != nullptr;
    f4 dbacc[4] = {{0.0f, 0.0f, 0.0f, 0.0f}, {0.0f, 0.0f, 0.0f, 0.0f},
                   {0.0f, 0.0f, 0.0f, 0.0f}, {0.0f, 0.0f, 0.0f, 0.0f}};
    const auto rs_dA = slice_rsrc(a.dA + sbase * G, V * G);
    const auto rs_gcf = slice_rsrc(a.gcf + sbase * O, V * O);
    const auto rs_g = slice_rsrc(a.gates + sbase * G, V * G);
    const auto rs_c = slice_rsrc(a.cell + sbase * O, V * O);
    const auto rs_dh = slice_rsrc(a.dh + (long long)n * V * O, V * O);
    const int r0 = a.r0;
    const int nlines = min(S, T - r0);
    const int noff = dg.sign * ss;             // plane t + 1 = plane t + noff
    f4 *afr = dyn;                              // [KG][64 lanes]
    f4 *dab = dyn + KG * 64;                    // [kLineSlots][16], chunk ^ (slot & 15)
    float *wxl = (float *)(dab + kLineSlots * 16);  // [K][4O][C] input filters

    // W_h^T fragments, the input filters; dA and gc f of line t + 1 over the
    // widest range (zero after the last line and past the line's ends)
    {
        const f4 *src = (const f4 *)(a.frag + (long long)d * KG * 256);
        for (int e = threadIdx.x; e < KG * 64; e += 256) afr[e] = src[e];
        if (want_dx) {
            const int nw = KQ * G * C;
            for (int e = threadIdx.x; e < nw; e += 256) {
                const int tap = e / (G * C), mc = e - tap * (G * C);
                wxl[e] = a.wx[((long long)d * G * C + mc) * KQ + tap];
            }
        }
        const int tn = T - r0;                  // line t + 1 for t = T - 1 - r0
        const int sn = dg.sign > 0 ? tn : T - 1 - tn;
        const int nsl = kLineSeg + 2 * (S + 1) * rq;
        for (int e = threadIdx.x; e < kLineSlots * 16; e += 256) {
            const int slot = e >> 4, ch = e & 15;
            const int qq = pbase + slot;
            const bool ok = r0 > 0 && slot < nsl && (unsigned)qq < (unsigned)Q;
            const int v = sn * ss + qq * sq;
            dab[slot * 16 + (ch ^ (slot & 15))] =
                bload4(rs_dA, sel_off(ok, (unsigned)((v * G + 4 * ch) * 4)));
            if (ch < 4)
                gcb[slot][ch ^ (slot & 3)] = bload4(rs_gcf, sel_off(ok, (unsigned)((v * O + 4 * ch) * 4)));
        }
    }
    __syncthreads();

    const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
    // the segment's dL/dx of line s: the four waves' partials, added in order
    auto store_dx = [&](int s) {
        if (threadIdx.x < kLineSeg) {
            const int p = threadIdx.x, qq = q0 + p;
            if (qq < Q) {
                const f4 v = ((dxr[0][p] + dxr[1][p]) + dxr[2][p]) + dxr[3][p];
                float *out = a.dxd + (sbase + s * ss + qq * sq) * C;
                for (int c = 0; c < C; ++c) out[c] = v[c];
            }
        }
    };
    int s_dx = -1;                              // line whose partials wait in dxr
    for (int j = 0; j < nlines; ++j) {
        const int t = T - 1 - (r0 + j);
        const int s = dg.sign > 0 ? t : T - 1 - t;
        const bool has_next = t + 1 < T;
        const int lo = (j + 1) * rq;
        const int W = kLineSeg + 2 * (S - j) * rq;
        const int ntl = (W + 15) >> 4;          // at most 6: two tiles per wave
        // dA_t is held in registers until every wave has read dA_{t+1} from
        // the one LDS buffer
        f4 dv[2][4];
        bool onv[2];
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int i = wave + 4 * k;
            onv[k] = false;
            if (i >= ntl) continue;             // wave-uniform
            const int slot = lo + 16 * i + col;
            const int qq = pbase + slot;
            const bool on = 16 * i + col < W && (unsigned)qq < (unsigned)Q;
            onv[k] = on;
            const int vox = s * ss + (on ? qq : 0) * sq;
            // epilogue operands in flight during the contraction
            f4 gv[4];
#pragma unroll
            for (int g = 0; g < 4; ++g)
                gv[g] = bload4(rs_g, sel_off(on, (unsigned)((vox * G + g * O + 4 * q4) * 4)));
            const int gsw = q4 ^ (slot & 3);
            // c_t: the previous line's c_{t-1}, kept in LDS (same lane and slot)
            const f4 c = j == 0 ? bload4(rs_c, sel_off(on, (unsigned)((vox * O + 4 * q4) * 4)))
                                : cl[slot][gsw];
            const f4 cp = bload4(rs_c, sel_off(on && t > 0, (unsigned)(((vox - noff) * O + 4 * q4) * 4)));
            const f4 dhv = bload4(rs_dh, sel_off(on, (unsigned)((vox * O + 4 * q4) * 4)));
            f4 acc = zero;
            if (has_next) {
                for (int kg = 0; kg < KG; ++kg) {
                    const int tap = kg >> 2, mb = kg & 3;
                    const int sx = slot - (tap - rq);
                    const f4 bv = dab[sx * 16 + ((mb * 4 + q4) ^ (sx & 15))];
                    const f4 av = afr[kg * 64 + lane];
#pragma unroll
                    for (int i4 = 0; i4 < 4; ++i4) acc = mfma(av[i4], bv[i4], acc);
                }
            }
            // gc f and c are read and rewritten by their own lane only
            const f4 gn = has_next ? gcb[slot][gsw] : zero;
            cl[slot][gsw] = cp;
            f4 gco;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const float gi = gv[0][u], gf = gv[1][u], gg = gv[2][u], go = gv[3][u];
                const float gh = acc[u] + dhv[u];
                const float tc = ftanh(c[u]);
                const float gc = gh * go * (1.0f - tc * tc) + gn[u];
                dv[k][0][u] = gc * gg * gi * (1.0f - gi);
                dv[k][1][u] = gc * (t > 0 ? cp[u] : 0.0f) * gf * (1.0f - gf);
                dv[k][2][u] = gc * gi * (1.0f - gg * gg);
                dv[k][3][u] = gh * tc * go * (1.0f - go);
                gco[u] = gc * gf;
            }
            gcb[slot][gsw] = on ? gco : zero;
            if (on && qq >= q0 && qq < q0 + kLineSeg) {
#pragma unroll
                for (int g = 0; g < 4; ++g) dbacc[g] += dv[k][g];
                const long long vo = sbase + vox;
#pragma unroll
                for (int g = 0; g < 4; ++g) *(f4 *)(a.dA + vo * G + g * O + 4 * q4) = dv[k][g];
                // gc f leaves LDS only where the next launch starts
                if (j == nlines - 1) *(f4 *)(a.gcf + vo * O + 4 * q4) = gco;
            }
        }
        __syncthreads();
        if (want_dx && s_dx >= 0) store_dx(s_dx);
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int i = wave + 4 * k;
            if (i >= ntl) continue;
            const int slot = lo + 16 * i + col;
#pragma unroll
            for (int g = 0; g < 4; ++g) dab[slot * 16 + ((g * 4 + q4) ^ (slot & 15))] = onv[k] ? dv[k][g] : zero;
        }
        __syncthreads();
        if (want_dx) {
            // lane = pixel of the segment; wave = gate; taps from dA_t in LDS
            const int cs = (S + 1) * rq + lane;
            f4 px;
            switch (C) {
            case 1: px = line_dx_px<1>(dab, wxl, cs, rq, KQ, wave); break;
            case 2: px = line_dx_px<2>(dab, wxl, cs, rq, KQ, wave); break;
            case 3: px = line_dx_px<3>(dab, wxl, cs, rq, KQ, wave); break;
            default: px = line_dx_px<4>(dab, wxl, cs, rq, KQ, wave); break;
            }
            dxr[wave][lane] = px;
            s_dx = s;
        }
    }
    if (want_dx && s_dx >= 0) {
        __syncthreads();
        store_dx(s_dx);
    }
    if (a.dbp) {
        // over the 16 lanes of a unit group (pixels), then the four waves
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                float v = dbacc[g][u];
                v += __shfl_xor(v, 1);
                v += __shfl_xor(v, 2);
                v += __shfl_xor(v, 4);
                v += __shfl_xor(v, 8);
                dbacc[g][u] = v;
            }
        if (col == 0) {
#pragma unroll
            for (int g = 0; g < 4; ++g) dbr[wave][g][q4] = dbacc[g];
        }
        __syncthreads();
        if (threadIdx.x < G) {
            const int m = threadIdx.x, g = m >> 4, q = (m >> 2) & 3, u = m & 3;
            const float v = ((dbr[0][g][q][u] + dbr[1][g][q][u]) + dbr[2][g][q][u]) + dbr[3][g][q][u];
            float *e = a.dbp + (((long long)d * a.g.N + n) * a.nsegmax + seg) * G + m;
            *e = (r0 == 0 ? 0.0f : *e) + v;
        }
    }
}

// db from the reverse line blocks' partials: each direction's (image,
// segment) partials added in order.
struct LineDbReduceArgs {
    int nd, N, nsegmax;
    int nseg[kDirs];
    const float *dbp;
    float *db;
};

__global__ void __launch_bounds__(256)
k_line_db_reduce(LineDbReduceArgs a)
{
    constexpr int G = 64;
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= a.nd * G) return;
    const int d = i / G, m = i - d * G;
    float acc = 0.0f;
    for (int n = 0; n < a.N; ++n)
        for (int seg = 0; seg < a.nseg[d]; ++seg)
            acc += a.dbp[(((long long)d * a.N + n) * a.nsegmax + seg) * G + m];
    a.db[i] = acc;
}

// dx = the four directions' dL/dx added in order.
__global__ void __launch_bounds__(256)
k_sum_dx4(long long n, const float *__restrict__ dxd, float *__restrict__ dx)
{
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    dx[i] = ((dxd[i] + dxd[n + i]) + dxd[2 * n + i]) + dxd[3 * n + i];
}

// Every unit group of kNT 16-pixel tiles of one plane (an item); the two
// launch shapes of the forward step (SPLIT: one item per workgroup, K split
// over its waves, wave w finishes tile w; !SPLIT: one item per wave).
//   gh = dL/dh + sum_taps W_h^T dA_{t+1}[p - tap]            (MFMA)
//   gc = gh o (1 - tanh^2 c) + (gc f)_{t+1}
//   dA_i = gc g i (1 - i), dA_f = gc c_{t-1} f (1 - f), dA_g = gc i (1 - g^2),
//   dA_o = gh tanh(c) o (1 - o)
template <int U, bool SPLIT>
__global__ void __launch_bounds__(64 * kSW) __attribute__((amdgpu_waves_per_eu(3)))
k_step_bwd(BwdStepArgs a)
{
    constexpr int O = 16 * U, G = 4 * O, MB = 4 * U;
    constexpr int KS = SPLIT ? kSW : 1;
    constexpr int NE = SPLIT ? 1 : kNT;
    static_assert(kNT == kSW, "wave w finishes tile w");
    __shared__ f4 red[SPLIT ? kSW : 1][U][kNT][64];
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int item = SPLIT ? (int)blockIdx.x : (int)blockIdx.x * kSW + wave;
    if (item >= a.base[kDirs]) return;
    const int d = item_dir(a.base, item);
    const DirGeom dg = a.g.dir[d];
    const int npg = a.npg[d];
    const int r = item - a.base[d];
    const int n = r / npg, pg = r - n * npg;
    const int t = a.t;
    const int s = dg.sign > 0 ? t : dg.T - 1 - t;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int P = dg.P, Q = dg.Q;
    const long long V = a.g.V;
    const bool has_next = t + 1 < dg.T;
    const int noff = dg.sign * ss;    // voxel of plane t + 1 = voxel of plane t + noff
    const int KQ = a.g.KQ, radp = a.g.KP >> 1, radq = KQ >> 1, KG = a.g.KP * KQ * MB;

    // this lane's pixel of each tile: voxel and in-plane coordinates (the
    // pixels that received its h through tap (ka, kb) are (p - ka + r, q - kb + r))
    int vox[kNT], tp[kNT], tq[kNT];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        const int pix = (pg * kNT + nt) * 16 + col;
        const bool live = pix < P * Q;
        const int p = live ? pix / Q : 0, qq = live ? pix - p * Q : 0;
        vox[nt] = s * ss + p * sp + qq * sq;
        tp[nt] = live ? p : kDead;
        tq[nt] = qq;
    }
    const long long sbase = ((long long)d * a.g.N + n) * V;
    const auto rs_dA = slice_rsrc(a.dA + sbase * G, V * G);
    const float *fr = a.frag + (long long)d * U * KG * 256 + lane * 4;

    f4 acc[U][kNT];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[u][nt] = f4{0.0f, 0.0f, 0.0f, 0.0f};

    if (has_next) {
        struct Ops {
            f4 a[U];
            f4 b[kNT];
        };
        auto load = [&](int kg, Ops &o) {
            const int tap = kg / MB, mb = kg - tap * MB;
#pragma unroll
            for (int u = 0; u < U; ++u) o.a[u] = *(const f4 *)(fr + ((long long)u * KG + kg) * 256);
            const int row = tap_row(tap, a.k_mul), ka = row - radp, kb = tap - row * KQ - radq;
            const int dv = noff - ka * sp - kb * sq;
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt)
                o.b[nt] = bload4(rs_dA, sel_off(on_plane(tp[nt] - ka, tq[nt] - kb, P, Q),
                                                (unsigned)((vox[nt] + dv) * G + mb * 16 + 4 * q4) *
                                                    4u));
        };
        const int k0 = SPLIT ? wave : 0;
        Ops cur, nxt;
        load(k0, cur);
        for (int kg = k0; kg < KG; kg += KS) {
            if (kg + KS < KG) load(kg + KS, nxt);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int nt = 0; nt < kNT; ++nt)
                        acc[u][nt] = mfma(cur.a[u][i], cur.b[nt][i], acc[u][nt]);
            cur = nxt;
        }
    }
    if (SPLIT) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt) red[SPLIT ? wave : 0][u][nt][lane] = acc[u][nt];
        __syncthreads();
    }

#pragma unroll
    for (int e = 0; e < NE; ++e) {
        int evox = vox[e];
        bool elive = tp[e] >= 0;
        if (SPLIT) {
#pragma unroll
            for (int nt = 1; nt < kNT; ++nt)
                if (wave == nt) {
                    evox = vox[nt];
                    elive = tp[nt] >= 0;
                }
        }
        if (!elive) continue;
        const long long vo = sbase + evox;
        const float *dhp = a.dh + ((long long)n * V + evox) * O;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int uo = u * 16 + 4 * q4;
            const float *gp = a.gates + vo * G + uo;
            const f4 gi = *(const f4 *)gp, gf = *(const f4 *)(gp + O);
            const f4 gg = *(const f4 *)(gp + 2 * O), go = *(const f4 *)(gp + 3 * O);
            const f4 c = *(const f4 *)(a.cell + vo * O + uo);
            f4 cp = {0.0f, 0.0f, 0.0f, 0.0f}, gn = {0.0f, 0.0f, 0.0f, 0.0f};
            if (t > 0) cp = *(const f4 *)(a.cell + (vo - noff) * O + uo);
            if (has_next) gn = *(const f4 *)(a.gcf + (vo + noff) * O + uo);
            f4 ghv = acc[u][e];
            if (SPLIT) {
                ghv = red[0][u][wave][lane];
#pragma unroll
                for (int w = 1; w < KS; ++w) ghv += red[SPLIT ? w : 0][u][wave][lane];
            }
            ghv += *(const f4 *)(dhp + uo);
            f4 di, df, dgv, dov, gco;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float gh = ghv[i];
                const float tc = ftanh(c[i]);
                const float gc = gh * go[i] * (1.0f - tc * tc) + gn[i];
                di[i] = gc * gg[i] * gi[i] * (1.0f - gi[i]);
                df[i] = gc * cp[i] * gf[i] * (1.0f - gf[i]);
                dgv[i] = gc * gi[i] * (1.0f - gg[i] * gg[i]);
                dov[i] = gh * tc * go[i] * (1.0f - go[i]);
                gco[i] = gc * gf[i];
            }
            float *dp = a.dA + vo * G + uo;
            *(f4 *)dp = di;
            *(f4 *)(dp + O) = df;
            *(f4 *)(dp + 2 * O) = dgv;
            *(f4 *)(dp + 3 * O) = dov;
            *(f4 *)(a.gcf + vo * O + uo) = gco;
        }
    }
}

// Reverse step on LDS-staged pixel blocks (U = 1 or 2 unit tiles), with
// this direction's share of dL/dx for the plane before it in sweep order when
// CT > 0.  A workgroup takes a BP x BQ block of 64 pixels of one plane (the
// blocks of the staged forward).  The K dimension of the contraction is (tap,
// gate-unit block of 16): wave w takes the blocks mb = w + 4 j (j < U) of
// every tap.  It stages those channels of dA_{t+1} for the block and its
// filter halo in its own LDS region (16-byte chunks XOR-swizzled by the
// pixel), so every tap's B operand comes from LDS, and contracts them with
//   W_h^T (U unit tiles):     gh_t[p]     = sum_taps W_h^T dA_{t+1}[p - tap]
//   W_x^T (CT channel tiles): dx_{t+1}[p] = sum_taps W_x^T dA_{t+1}[p - tap]
// for the block's four pixel tiles: the input x_{t+1} entered plane t + 1's
// gates through the same taps (Eq. (7)-(9), (11)), so its gradient is the
// same transposed convolution of the same staged dA_{t+1}.  The partial sums
// of the three tiles a wave does not finish then go to its region; after a
// barrier wave w adds tile w's four partials in wave order, runs the
// gate-gradient epilogue and stores dx_{t+1}.  t = -1 gives dL/dx of plane 0
// only.
template <int U, int CT>
__global__ void __launch_bounds__(64 * kSW) __attribute__((amdgpu_waves_per_eu(3)))
k_step_bwd_blk(BwdStepArgs a)
{
    constexpr int O = 16 * U, G = 4 * O, MB = 4 * U;
    constexpr int NCH = 4 * U;                       // staged 16-byte chunks per pixel
    constexpr int SWM = NCH >= 8 ? 7 : 3;
    static_assert(kNT == kSW, "wave w finishes tile w");
    extern __shared__ f4 lds[];
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int blk = blockIdx.x;
    if (blk >= a.base[kDirs]) return;
    const int d = item_dir(a.base, blk);
    const DirGeom dg = a.g.dir[d];
    int r = blk - a.base[d];
    const int n = r / a.nblk[d];
    r -= n * a.nblk[d];
    const int BP = a.bp[d], BQ = a.bq[d];
    const int bi = r / a.nbq[d], bj = r - bi * a.nbq[d];
    const int p0 = bi * BP, q0 = bj * BQ;
    const int t = a.t;
    const bool do_h = t >= 0;                        // plane t exists (t = -1: dL/dx only)
    const int s = dg.sign > 0 ? t : dg.T - 1 - t;
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int P = dg.P, Q = dg.Q;
    const long long V = a.g.V;
    const bool has_next = t + 1 < dg.T;
    const int noff = dg.sign * ss;    // voxel of plane t + 1 = voxel of plane t + noff
    const int KQ = a.g.KQ, radp = a.g.KP >> 1, radq = KQ >> 1, KK = a.g.KP * KQ;
    const int KG = KK * MB;
    const int SW = BQ + 2 * radq, SH = BP + 2 * radp;
    const long long sbase = ((long long)d * a.g.N + n) * V;
    f4 *mine = lds + (long long)wave * a.reg_f4;

    // ---- the epilogue's pixel (tile `wave`)
    const int lbq = 31 - __builtin_clz(BQ);
    const int ee = wave * 16 + col;
    const int ey = ee >> lbq, ex = ee & (BQ - 1);
    const bool elive = on_plane(p0 + ey, q0 + ex, P, Q);
    const int pix = elive ? (p0 + ey) * sp + (q0 + ex) * sq : 0;
    const int evox = s * ss + pix;
    const long long vo = sbase + evox;
    const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};

    // ---- contraction over this wave's gate-unit blocks of dA_{t+1}
    f4 acc[U][kNT], accx[CT > 0 ? CT : 1][kNT];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[u][nt] = zero;
#pragma unroll
    for (int c = 0; c < (CT > 0 ? CT : 1); ++c)
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) accx[c][nt] = zero;
    if (has_next) {
        // direct-to-LDS loads, all in flight at once: one instruction fills
        // 64 consecutive 16-byte slots, slot p of pixel spx holding chunk
        // p ^ (spx & SWM), each lane loading the chunk its slot holds
        const auto rs_dA = slice_rsrc(a.dA + sbase * G, V * G);
        const int nst = SH * SW * NCH;
        for (int e0 = 0; e0 < nst; e0 += 64) {
            const int e = e0 + lane;
            const int spx = e / NCH, pos = e - spx * NCH;
            const int c = pos ^ (spx & SWM);
            const int sy = spx / SW, sx = spx - sy * SW;
            const int pp = p0 - radp + sy, qq = q0 - radq + sx;
            const int mb = wave + kSW * (c >> 2);
            const int v = (s + dg.sign) * ss + pp * sp + qq * sq;
            lds_void *dst = (lds_void *)&mine[e0];
            if (e < nst)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rs_dA, dst, 16,
                    (int)sel_off(on_plane(pp, qq, P, Q),
                                 (unsigned)(v * G + mb * 16 + 4 * (c & 3)) * 4u),
                    0, 0, 0);
        }
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    }
    __syncthreads();
    if (has_next) {
        int spix[kNT];
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) {
            const int e = nt * 16 + col;
            spix[nt] = ((e >> lbq) + radp) * SW + (e & (BQ - 1)) + radq;
        }
        const float *fr = a.frag + (long long)d * U * KG * 256 + lane * 4;
        const float *frx = a.fragx + (long long)d * KG * CT * 256 + lane * 4;
        // K-steps in (tap, j) order; A fragments one K-group ahead
        auto afrag = [&](int tap, int j, f4 *o, f4 *ox) {
            const int kg = tap * MB + wave + kSW * j;
#pragma unroll
            for (int u = 0; u < U; ++u) o[u] = *(const f4 *)(fr + ((long long)u * KG + kg) * 256);
#pragma unroll
            for (int c = 0; c < CT; ++c) ox[c] = *(const f4 *)(frx + ((long long)kg * CT + c) * 256);
        };
        f4 acur[U], anxt[U], axc[CT > 0 ? CT : 1], axn[CT > 0 ? CT : 1];
        afrag(0, 0, acur, axc);
        const int nk = KK * U;
        for (int k = 0; k < nk; ++k) {
            const int tap = k / U, j = k - tap * U;
            if (k + 1 < nk) afrag((k + 1) / U, (k + 1) - ((k + 1) / U) * U, anxt, axn);
            const int row = tap_row(tap, a.k_mul), ka = row - radp, kb = tap - row * KQ - radq;
            // the pixels that received this pixel's h (and x) through tap (ka, kb)
            const int doff = -ka * SW - kb;
            const int chunk = j * 4 + q4;
            f4 bv[kNT];
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt) {
                const int spx = spix[nt] + doff;
                bv[nt] = mine[spx * NCH + (chunk ^ (spx & SWM))];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int nt = 0; nt < kNT; ++nt)
                        acc[u][nt] = mfma(acur[u][i], bv[nt][i], acc[u][nt]);
#pragma unroll
                for (int c = 0; c < CT; ++c)
#pragma unroll
                    for (int nt = 0; nt < kNT; ++nt)
                        accx[c][nt] = mfma(axc[c][i], bv[nt][i], accx[c][nt]);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) acur[u] = anxt[u];
#pragma unroll
            for (int c = 0; c < CT; ++c) axc[c] = axn[c];
        }
    }
    // the epilogue's operands of tile `wave`, in flight during the exchange
    // of partial sums below
    f4 e_g[U][4], e_c[U], e_cp[U], e_gn[U], e_dh[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int k = 0; k < 4; ++k) e_g[u][k] = zero;
        e_c[u] = e_cp[u] = e_gn[u] = e_dh[u] = zero;
    }
    if (do_h && elive) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int uo = u * 16 + 4 * q4;
            const float *gp = a.gates + vo * G + uo;
#pragma unroll
            for (int k = 0; k < 4; ++k) e_g[u][k] = *(const f4 *)(gp + k * O);
            e_c[u] = *(const f4 *)(a.cell + vo * O + uo);
            if (t > 0) e_cp[u] = *(const f4 *)(a.cell + (vo - noff) * O + uo);
            if (has_next) e_gn[u] = *(const f4 *)(a.gcf + (vo + noff) * O + uo);
            e_dh[u] = *(const f4 *)(a.dh + ((long long)n * V + evox) * O + uo);
        }
    }
    // partial sums of the tiles other waves finish, into this wave's own
    // region (only this wave read it): slot nt - (nt > wave) of each M-tile
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        if (nt == wave) continue;
        const int sl = nt - (nt > wave ? 1 : 0);
#pragma unroll
        for (int u = 0; u < U; ++u) mine[(u * (kNT - 1) + sl) * 64 + lane] = acc[u][nt];
#pragma unroll
        for (int c = 0; c < CT; ++c)
            mine[((U + c) * (kNT - 1) + sl) * 64 + lane] = accx[c][nt];
    }
    __syncthreads();
    if (!elive) return;
    // tile `wave` of M-tile m: the four waves' partials in wave order
    auto partial = [&](int m, f4 own) {
        f4 v = zero;
#pragma unroll
        for (int w = 0; w < kSW; ++w) {
            if (w == wave) {
                v += own;
            } else {
                const int sl = wave - (wave > w ? 1 : 0);
                v += lds[(long long)w * a.reg_f4 + (m * (kNT - 1) + sl) * 64 + lane];
            }
        }
        return v;
    };
    f4 own_h[U], own_x[CT > 0 ? CT : 1];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt)
        if (nt == wave) {
#pragma unroll
            for (int u = 0; u < U; ++u) own_h[u] = acc[u][nt];
#pragma unroll
            for (int c = 0; c < CT; ++c) own_x[c] = accx[c][nt];
        }

    if (CT > 0 && has_next) {
        const int C = a.g.C;
        float *out = a.dxd + (sbase + evox + noff) * C;
#pragma unroll
        for (int c = 0; c < CT; ++c) {
            const f4 v = partial(U + c, own_x[c]);
            const int c0 = c * 16 + 4 * q4;
            if ((C & 3) == 0 && c0 + 3 < C) {
                *(f4 *)(out + c0) = v;
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (c0 + i < C) out[c0 + i] = v[i];
            }
        }
    }
    if (!do_h) return;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int uo = u * 16 + 4 * q4;
        const f4 gi = e_g[u][0], gf = e_g[u][1], gg = e_g[u][2], go = e_g[u][3];
        const f4 c = e_c[u], cp = e_cp[u], gn = e_gn[u];
        f4 ghv = partial(u, own_h[u]) + e_dh[u];
        f4 di, df, dgv, dov, gco;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float gh = ghv[i];
            const float tc = ftanh(c[i]);
            const float gcv = gh * go[i] * (1.0f - tc * tc) + gn[i];
            di[i] = gcv * gg[i] * gi[i] * (1.0f - gi[i]);
            df[i] = gcv * cp[i] * gf[i] * (1.0f - gf[i]);
            dgv[i] = gcv * gi[i] * (1.0f - gg[i] * gg[i]);
            dov[i] = gh * tc * go[i] * (1.0f - go[i]);
            gco[i] = gcv * gf[i];
        }
        float *dp = a.dA + vo * G + uo;
        *(f4 *)dp = di;
        *(f4 *)(dp + O) = df;
        *(f4 *)(dp + 2 * O) = dgv;
        *(f4 *)(dp + 3 * O) = dov;
        *(f4 *)(a.gcf + vo * O + uo) = gco;
    }
}

// dx = sum of the nd directions' shares in direction order; four elements
// per thread (n4 = n / 4 vectors, n a multiple of 4), every direction's load
// in flight before the first add.
__global__ void __launch_bounds__(256)
k_sum_dxn(long long n, int nd, const float *__restrict__ dxd, float *__restrict__ dx)
{
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    float v = dxd[i];
    for (int d = 1; d < nd; ++d) v += dxd[d * n + i];
    dx[i] = v;
}
__global__ void __launch_bounds__(256)
k_sum_dxn4(long long n4, int nd, const f4 *__restrict__ dxd, f4 *__restrict__ dx)
{
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= n4) return;
    f4 t[kDirs];
#pragma unroll
    for (int d = 0; d < kDirs; ++d)
        if (d < nd) t[d] = dxd[d * n4 + i];
    f4 v = t[0];
#pragma unroll
    for (int d = 1; d < kDirs; ++d)
        if (d < nd) v += t[d];
    dx[i] = v;
}

// ---- parameter gradients ----------------------------------------------------
// dW[d][m][k] = sum over the voxels of direction d of dA[v][m] col[v][k],
// col = [im2col(h_{t-1}) (KK O) | im2col(x_t) (KK C')]; K of the MFMA runs over
// voxels.  A wave owns 4 M-tiles x NTL N-tiles of one direction, all of the
// h part or all of the x part, and a chunk of the direction's voxels,
// visited as units of 16 pixels of a row (lane group q takes pixels
// 4q .. 4q+3, one per k-step), walking each column group down the rows so
// that the rows read for one unit are re-read from cache by the next ones.
// The partial sums of the chunks are added in order.  db = sum_v dA[v] is the
// product with a column of ones appended to the x part.
constexpr int kWgN = 4;          // most N-tiles a wave holds
constexpr int kWgMaxChunks = 512;

// N-tiles per block: each part (KK U tiles of h; ceil((KK C + 1) / 16) tiles
// of x, whose columns are the (tap, channel) pairs packed densely and then a
// column of ones, which gives db) is cut into the fewest blocks of at most
// kWgN tiles, as even as possible.
struct WgBlocks {
    int nh, nx;       // blocks of each part
    int th, tx;       // tiles per block of each part (the last block may have fewer)
};
__host__ __device__ inline int wg_xtiles(int KK, int C) { return (KK * C + 16) / 16; }
__host__ __device__ inline WgBlocks wg_blocks(int U, int XT, int KK)
{
    WgBlocks w;
    const int h = KK * U, x = XT;
    w.nh = (h + kWgN - 1) / kWgN;
    w.nx = (x + kWgN - 1) / kWgN;
    w.th = (h + w.nh - 1) / w.nh;
    w.tx = (x + w.nx - 1) / w.nx;
    return w;
}

struct WgStepArgs {
    Geom g;
    int Cp;                   // floats per voxel of xp
    int NTt;                  // N-tiles: KK U + KK C'/16
    int kch;                  // voxel chunks per (direction, M-block, N-block)
    int k_mul;                // ceil(2^16 / K)
    const float *xp, *hd, *dA;  // xp: the input x [N][V][Cp] (read one channel per lane)
    float *partial;           // [6][kch][4O][16 NTt]
};

// The wave's share: NTL tiles (compile time) of which `ntl` are real; ONES:
// the block holds the column of ones.
template <int U, int NTL, bool ONES>
__device__ inline void wg_wave(const WgStepArgs &a, int d, int kc, int mblk, bool is_h, int t0,
                               int ntl, int first_nt)
{
    constexpr int O = 16 * U, G = 4 * O;
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int KQ = a.g.KQ, KK = a.g.KP * KQ, radp = a.g.KP >> 1, radq = KQ >> 1;
    const DirGeom dg = a.g.dir[d];
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int P = dg.P, Q = dg.Q;
    const long long V = a.g.V;
    const int Cp = a.Cp, C = a.g.C;
    const int ngrp = (Q + 15) >> 4;
    const int stride = is_h ? O : Cp;           // floats per voxel of the source

    // per tile and lane: tap offset in the slice, tap row and column (packed)
    // and channel (-1: a column past the part).  An h tile is one tap and 16
    // channels (uniform tap); an x tile is 16 (tap, channel) pairs, column
    // kk = 16 tt + col being tap kk / C, channel kk % C; column KK C is the
    // column of ones (db): its lanes load nothing (an out-of-range offset) and
    // their operand becomes 1 where the products use it, so the loads stay
    // unconditional and nothing waits for them early.
    int dtap[NTL], chn[NTL];
    unsigned tapok[NTL];
    bool ones[NTL];
#pragma unroll
    for (int j = 0; j < NTL; ++j) {
        const int tt = t0 + j;
        const int kk = tt * 16 + col;
        ones[j] = ONES && !is_h && j < ntl && kk == KK * C;
        const bool real = j < ntl && (is_h || kk < KK * C);
        const int tap = !real ? radp * KQ + radq : (is_h ? tt / U : kk / C);
        const int ka = tap / KQ, kb = tap % KQ;
        dtap[j] = (ka - radp) * sp + (kb - radq) * sq;
        tapok[j] = ka | kb << 3;
        chn[j] = !real ? -1 : (is_h ? (tt % U) * 16 + col : kk % C);
    }

    f4 acc[4][NTL];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int j = 0; j < NTL; ++j) acc[m][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};

    struct Ops {
        float a[4][4];            // [k-step][M-tile]
        float b[4][NTL];          // [k-step][N-tile]
    };
    struct Cursor {
        int n, t, qg, p;
    };
    const long long units = (long long)a.g.N * dg.T * ngrp * P;
    const long long u0 = units * kc / a.kch, u1 = units * (kc + 1) / a.kch;
    Cursor cu;
    {
        long long rest = u0;
        cu.p = (int)(rest % P);
        rest /= P;
        cu.qg = (int)(rest % ngrp);
        rest /= ngrp;
        cu.t = (int)(rest % dg.T);
        cu.n = (int)(rest / dg.T);
        if (cu.n >= a.g.N) cu.n = a.g.N - 1;
    }
    auto advance = [&]() {
        if (++cu.p == P) {
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
    // Branch-free loads: an operand outside the volume, of h_{-1} or of a
    // tile past the part gets an out-of-range offset.
    auto load = [&](const Cursor &c, bool live_unit, Ops &o) {
        const long long sb = ((long long)d * a.g.N + c.n) * V;
        const auto rs_a = slice_rsrc(a.dA + sb * G, V * G);
        const auto rs_b = is_h ? slice_rsrc(a.hd + sb * O, V * O)
                               : slice_rsrc(a.xp + (long long)c.n * V * Cp, V * Cp);
        const int s = dg.sign > 0 ? c.t : dg.T - 1 - c.t;
        const int pl = is_h ? s - dg.sign : s;
        const bool src_ok = live_unit & (!is_h | (c.t > 0));
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int qq = c.qg * 16 + 4 * q4 + ks;
            const bool live = live_unit & (qq < Q);
            const int v = s * ss + c.p * sp + qq * sq;
#pragma unroll
            for (int m = 0; m < 4; ++m)
                o.a[ks][m] =
                    bload1(rs_a, sel_off(live, (unsigned)(v * G + mblk * 64 + m * 16 + col) * 4u));
            const int vb = pl * ss + c.p * sp + qq * sq;
#pragma unroll
            for (int j = 0; j < NTL; ++j) {
                const int pp = c.p + (int)(tapok[j] & 7) - radp;
                const int qn = qq + (int)(tapok[j] >> 3) - radq;
                const bool ok = src_ok & (chn[j] >= 0) & ((unsigned)pp < (unsigned)P) &
                                ((unsigned)qn < (unsigned)Q);
                o.b[ks][j] =
                    bload1(rs_b, sel_off(ok, (unsigned)((vb + dtap[j]) * stride + chn[j]) * 4u));
            }
        }
    };
    const long long total = u1 - u0;
    auto step = [&](const Ops &o) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
            for (int m = 0; m < 4; ++m)
#pragma unroll
                for (int j = 0; j < NTL; ++j)
                    acc[m][j] = mfma(o.a[ks][m], ONES && ones[j] ? 1.0f : o.b[ks][j], acc[m][j]);
    };
    // two operand sets in ping-pong: each is reloaded only after its
    // products, so no loaded register is copied (a copy would wait for the
    // load just issued), and the loads of one set are all issued before the
    // products of the other (a whole unit of MFMAs in flight behind them)
    Ops o0, o1;
    load(cu, total > 0, o0);
    for (long long it = 0; it < total; it += 2) {
        advance();
        load(cu, it + 1 < total, o1);
        __builtin_amdgcn_sched_barrier(0);
        step(o0);
        __builtin_amdgcn_sched_barrier(0);
        if (it + 1 >= total) break;
        advance();
        load(cu, it + 2 < total, o0);
        __builtin_amdgcn_sched_barrier(0);
        step(o1);
        __builtin_amdgcn_sched_barrier(0);
    }
    const int KCp = a.NTt * 16;
    float *out = a.partial + ((long long)d * a.kch + kc) * G * KCp;
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int j = 0; j < NTL; ++j) {
            if (j >= ntl) continue;
            const int nt = first_nt + j;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                out[(long long)(mblk * 64 + m * 16 + 4 * q4 + i) * KCp + nt * 16 + col] =
                    acc[m][j][i];
        }
}

// Work items run N-block fastest, so the waves that read the same voxel chunk
// of dA (one per N-block) are neighbours; the grid (a multiple of eight
// workgroups) is remapped so that each XCD, which takes every eighth
// workgroup, runs a contiguous range of items and those waves share its L2.
template <int U>
__global__ void __launch_bounds__(64 * kSW) __attribute__((amdgpu_waves_per_eu(2)))
k_wgrad_step(WgStepArgs a)
{
    const int per_xcd = gridDim.x / kXcds;
    const int lblk = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    const int item = lblk * kSW + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int KK = a.g.KP * a.g.KQ, XT = wg_xtiles(KK, a.g.C);
    const WgBlocks wb = wg_blocks(U, XT, KK);
    const int nblk = wb.nh + wb.nx;
    const int per_dir = U * nblk * a.kch;
    if (item >= a.g.nd * per_dir) return;
    const int d = item / per_dir;
    int r = item - d * per_dir;
    const int nb = r % nblk;
    r /= nblk;
    const int kc = r % a.kch, mblk = r / a.kch;
    const bool is_h = nb < wb.nh;
    // first N-tile and tile count of this block; x tiles numbered after h's
    const int tb = is_h ? wb.th : wb.tx;
    const int t0 = is_h ? nb * wb.th : (nb - wb.nh) * wb.tx;
    const int tend = is_h ? KK * U : XT;
    const int ntl = t0 + tb < tend ? tb : tend - t0;
    const int first_nt = (is_h ? 0 : KK * U) + t0;
    // the x block holding the column of ones (tile KK C / 16 of the x part)
    const int ones_tile = KK * a.g.C / 16;
    const bool ones = !is_h && t0 <= ones_tile && ones_tile < t0 + ntl;
    static_assert(kWgN <= 4, "at most four N-tiles per wave");
    // as many products per unit as the block has tiles
    if (ones) {
        if (ntl <= 1)
            wg_wave<U, 1, true>(a, d, kc, mblk, is_h, t0, ntl, first_nt);
        else if (ntl <= 2)
            wg_wave<U, 2, true>(a, d, kc, mblk, is_h, t0, ntl, first_nt);
        else if (ntl <= 3)
            wg_wave<U, 3, true>(a, d, kc, mblk, is_h, t0, ntl, first_nt);
        else
            wg_wave<U, 4, true>(a, d, kc, mblk, is_h, t0, ntl, first_nt);
    } else {
        if (ntl <= 1)
            wg_wave<U, 1, false>(a, d, kc, mblk, is_h, t0, ntl, first_nt);
        else if (ntl <= 2)
            wg_wave<U, 2, false>(a, d, kc, mblk, is_h, t0, ntl, first_nt);
        else if (ntl <= 3)
            wg_wave<U, 3, false>(a, d, kc, mblk, is_h, t0, ntl, first_nt);
        else
            wg_wave<U, 4, false>(a, d, kc, mblk, is_h, t0, ntl, first_nt);
    }
}

// ---- parameter gradients through LDS (up to 32 hidden units, C % 4 == 0) ----
// The same products as k_wgrad_step, organised as a staged GEMM: one
// workgroup of eight waves per (direction, N-part, voxel chunk) holds the
// whole [4O x 16 NT] partial sum of its N-part (at most kWlPartNT N-tiles;
// wave w takes N-tiles w, w + 8, w + 16 and all 4U M-tiles).  Pairs of
// 16-voxel units (as in k_wgrad_step: consecutive rows of a column group)
// are staged once for all eight waves:
//   dA transposed to [gate][voxel] and the im2col columns of the part to
//   [column][voxel] (h_{t-1} taps, x_t taps, the column of ones; zero off
//   the plane and before the first plane),
// each row holding the pair's 32 voxels padded to kWlRow floats; one
// ds_read_b128 gives a lane its four k-steps of a unit (voxels 4 q .. 4 q + 3).
// (On gfx950, 64 lanes reading 16 bytes each at row r = lane % 16, offset
// 4 (lane / 16) run without bank conflicts when the row stride is 8 mod 16
// floats (24, 40, 56, ...); strides of 36 or 20 floats take half as long
// again, measured.)
// Two stage buffers: the next pair's global loads are in flight while this
// pair's MFMAs run, then go to the other buffer, one barrier per pair.  dA
// is read from memory once per N-part instead of once per N-block wave.
constexpr int kWlWaves = 8;
constexpr int kWlThreads = 64 * kWlWaves;
template <int N> struct IntC {
    static constexpr int value = N;
};
constexpr int kWlPartNT = 20;             // most N-tiles of a part
constexpr int kWlNT = 3;                  // N-tiles per wave: ceil(20 / 8)
constexpr int kWlRow = 40;                // floats per staged row: 2 x 16 voxels + pad
constexpr int kWlBSlots = 3;              // column quads x voxels per thread: 20 * 64 / 512

struct WlArgs {
    Geom g;
    int NTt, nparts, kch;
    const float *x, *hd, *dA;
    float *partial;           // [6][kch][4O][16 NTt] (chunk partials of every part)
};

template <int U>
__global__ void __launch_bounds__(kWlThreads, 1) __attribute__((amdgpu_waves_per_eu(1, 2)))
k_wgrad_lds(WlArgs a)
{
    constexpr int O = 16 * U, G = 4 * O, MT = 4 * U;
    extern __shared__ float wl_smem[];
    const int per_dir = a.nparts * a.kch;
    const int d = blockIdx.x / per_dir;
    const int part = (blockIdx.x % per_dir) / a.kch, kc = blockIdx.x % a.kch;
    const int tid = threadIdx.x, lane = tid & 63, q4 = lane >> 4, col = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int KQ = a.g.KQ, KK = a.g.KP * KQ, radp = a.g.KP >> 1, radq = KQ >> 1;
    const int C = a.g.C, NTt = a.NTt, KCp = NTt * 16;
    const int KO = KK * O, KX = KK * C;          // h columns, x columns
    // this part's N-tiles [nt0, nt1)
    const int nt0 = (int)((long long)NTt * part / a.nparts);
    const int nt1 = (int)((long long)NTt * (part + 1) / a.nparts);
    const int ncol = (nt1 - nt0) * 16;
    const DirGeom dg = a.g.dir[d];
    const int ss = (int)dg.ss, sp = (int)dg.sp, sq = (int)dg.sq;
    const int P = dg.P, Q = dg.Q;
    const long long V = a.g.V;
    const int ngrp = (Q + 15) >> 4;
    const int rows = G + ncol;
    float *const buf0 = wl_smem, *const buf1 = wl_smem + (size_t)rows * kWlRow;

    // columns that never change: the column of ones and the padding past it
    for (int e = tid; e < 2 * ncol * 32; e += kWlThreads) {
        const int b = e / (ncol * 32), r = e - b * ncol * 32;
        const int c = nt0 * 16 + r / 32;
        if (c >= KO + KX)
            (b ? buf1 : buf0)[(G + r / 32) * kWlRow + (r & 31)] = c == KO + KX ? 1.0f : 0.0f;
    }

    // unit cursor over this chunk: (n, t, column group, row), row fastest
    const long long units = (long long)a.g.N * dg.T * ngrp * P;
    const long long u0 = units * kc / a.kch, u1 = units * (kc + 1) / a.kch;
    int cn, ct, cg, cp;
    {
        long long rest = u0;
        cp = (int)(rest % P); rest /= P;
        cg = (int)(rest % ngrp); rest /= ngrp;
        ct = (int)(rest % dg.T);
        cn = (int)(rest / dg.T);
        if (cn >= a.g.N) cn = a.g.N - 1;
    }
    auto advance = [&]() __attribute__((always_inline)) {
        if (++cp == P) {
            cp = 0;
            if (++cg == ngrp) {
                cg = 0;
                if (++ct == dg.T) {
                    ct = 0;
                    if (cn + 1 < a.g.N) ++cn;
                }
            }
        }
    };

    // staged registers of a pair of units: dA (one quad of gates of one
    // voxel per thread and unit) and the part's im2col quads (column quad,
    // voxel); a unit past the chunk stages zeros
    struct Stage {
        f4 a[2];
        f4 b[2][kWlBSlots];
    };
    const int nbq = ncol / 4 * 16;                 // column quads x voxels of a unit
    // Branch-free loads: a masked operand (past the plane, off the volume,
    // h_{-1}, a column past the layer's or a unit past the chunk) gets an
    // out-of-range offset and reads zero.  A wave's 64 lanes of one slot
    // cover one 16-column N-tile, all of h or all of x, so the source
    // (resource, stride, plane) is uniform per slot; the slot's tap offset
    // and channel do not change from unit to unit.
    int s_dp[kWlBSlots], s_dq[kWlBSlots], s_ch[kWlBSlots];
    bool s_h[kWlBSlots], s_ok[kWlBSlots];
#pragma unroll
    for (int k = 0; k < kWlBSlots; ++k) {
        const int e = k * kWlThreads + tid;
        const int c = nt0 * 16 + 4 * (e >> 4);   // first column of the lane's quad
        s_h[k] = __builtin_amdgcn_readfirstlane(c < KO ? 1 : 0) != 0;
        const int kk = s_h[k] ? c : c - KO;
        const int tap = s_h[k] ? kk / O : kk / C;
        s_ch[k] = s_h[k] ? kk % O : kk % C;
        s_dp[k] = tap / KQ - radp;
        s_dq[k] = tap % KQ - radq;
        s_ok[k] = (e < nbq) & (c < KO + KX);
    }
    auto fetch_unit = [&](f4 &sa, f4 (&sb4)[kWlBSlots], bool live) __attribute__((always_inline)) {
        const long long sb = ((long long)d * a.g.N + cn) * V;
        const int s = dg.sign > 0 ? ct : dg.T - 1 - ct;
        const auto rs_a = slice_rsrc(a.dA + sb * G, V * G);
        const auto rs_h = slice_rsrc(a.hd + sb * O, V * O);
        const auto rs_x = slice_rsrc(a.x + (long long)cn * V * C, V * C);
        const int q = cg * 16 + (tid & 15);
        {
            // dA: thread -> (voxel, gate quad), voxel fastest
            const int gq = tid >> 4;
            const bool ok = live & (tid < 16 * (G / 4)) & (q < Q);
            sa = bload4(rs_a, sel_off(ok, (unsigned)((s * ss + cp * sp + q * sq) * G + 4 * gq) * 4u));
        }
#pragma unroll
        for (int k = 0; k < kWlBSlots; ++k) {
            const int pp = cp + s_dp[k], qn = q + s_dq[k];
            const bool ok = live & s_ok[k] & ((unsigned)pp < (unsigned)P) &
                            ((unsigned)qn < (unsigned)Q) & (!s_h[k] | (ct > 0));
            const int pl = s_h[k] ? s - dg.sign : s;
            const int stride = s_h[k] ? O : C;
            const auto rs = s_h[k] ? rs_h : rs_x;
            sb4[k] = bload4(rs, sel_off(ok, (unsigned)((pl * ss + pp * sp + qn * sq) * stride +
                                                       s_ch[k]) * 4u));
        }
    };
    // stage units u and u + 1 (of `total`); the cursor is at unit u
    auto fetch = [&](Stage &st, long long u, long long total) __attribute__((always_inline)) {
        fetch_unit(st.a[0], st.b[0], u < total);
        if (u + 1 < total) advance();
        fetch_unit(st.a[1], st.b[1], u + 1 < total);
    };
    auto put = [&](const Stage &st, float *bf) __attribute__((always_inline)) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            {
                const int i = tid & 15, gq = tid >> 4;
                if (tid < 16 * (G / 4)) {
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        bf[(4 * gq + j) * kWlRow + 16 * h + i] = st.a[h][j];
                }
            }
#pragma unroll
            for (int k = 0; k < kWlBSlots; ++k) {
                const int e = k * kWlThreads + tid;
                const int i = e & 15, cq = e >> 4;
                if (e < nbq && nt0 * 16 + 4 * cq < KO + KX) {
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        bf[(G + 4 * cq + j) * kWlRow + 16 * h + i] = st.b[h][k][j];
                }
            }
        }
    };

    f4 acc[MT][kWlNT];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < kWlNT; ++j) acc[m][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    const int nmy = max(0, (nt1 - nt0 - wave + kWlWaves - 1) / kWlWaves);   // this wave's N-tiles

    // products of one staged unit (h: which half of the rows) for the wave's
    // NTW N-tiles
    auto compute = [&](const float *bf, int h, auto ntw) __attribute__((always_inline)) {
        constexpr int NTW = decltype(ntw)::value;
        f4 bv[NTW];
#pragma unroll
        for (int j = 0; j < NTW; ++j)
            bv[j] = *(const f4 *)&bf[(G + (wave + kWlWaves * j) * 16 + col) * kWlRow + 16 * h +
                                     4 * q4];
        f4 av[MT];
#pragma unroll
        for (int m = 0; m < MT; ++m)
            av[m] = *(const f4 *)&bf[(m * 16 + col) * kWlRow + 16 * h + 4 * q4];
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int j = 0; j < NTW; ++j) acc[m][j] = mfma(av[m][ks], bv[j][ks], acc[m][j]);
    };
    auto compute_pair = [&](const float *bf, bool second) __attribute__((always_inline)) {
        if (nmy >= 3) {
            compute(bf, 0, IntC<3>{});
            if (second) compute(bf, 1, IntC<3>{});
        } else if (nmy == 2) {
            compute(bf, 0, IntC<2>{});
            if (second) compute(bf, 1, IntC<2>{});
        } else if (nmy == 1) {
            compute(bf, 0, IntC<1>{});
            if (second) compute(bf, 1, IntC<1>{});
        }
    };

    const long long total = u1 - u0;
    if (total > 0) {
        Stage st;
        fetch(st, 0, total);
        put(st, buf0);
        __syncthreads();
        // the first wave of each SIMD (waves 0-3) issues the next pair's
        // loads before its products, the second one (waves 4-7) after them,
        // so that one wave's address arithmetic runs beside the other's MFMAs
        const bool early = wave < kWlWaves / 2;
        for (long long u = 0; u < total; u += 2) {
            const bool more = u + 2 < total;
            if (more && early) {
                advance();
                fetch(st, u + 2, total);
            }
            compute_pair((u >> 1) & 1 ? buf1 : buf0, u + 1 < total);
            if (more && !early) {
                advance();
                fetch(st, u + 2, total);
            }
            if (more) put(st, (u >> 1) & 1 ? buf0 : buf1);
            __syncthreads();
        }
    }
    float *out = a.partial + ((long long)d * a.kch + kc) * G * KCp;
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < kWlNT; ++j) {
            if (j >= nmy) continue;
            const int nt = nt0 + wave + kWlWaves * j;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                out[(long long)(m * 16 + 4 * q4 + i) * KCp + nt * 16 + col] = acc[m][j][i];
        }
}

// dW = sum of the chunk partials in chunk order, scattered to the ABI layouts;
// the column of ones gives db (skipped when db is null).
__global__ void __launch_bounds__(256)
k_wgrad_step_reduce(int nd, int O, int C, int Cp, int KK, int NTt, int kch,
                    const float *__restrict__ partial, float *__restrict__ dwx,
                    float *__restrict__ dwh, float *__restrict__ db)
{
    // columns: KK O of h (tap-major), then KK C of x ((tap, channel) dense),
    // then the column of ones
    const int G = 4 * O, KC = KK * (O + C) + 1, KCp = NTt * 16;
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= (long long)nd * G * KC) return;
    const int k = (int)(i % KC);
    const int gu = (int)((i / KC) % G);
    const int d = (int)(i / ((long long)KC * G));
    float acc = 0.0f;
    for (int c = 0; c < kch; ++c) acc += partial[(((long long)d * kch + c) * G + gu) * KCp + k];
    if (k < KK * O) {
        dwh[(((long long)d * G + gu) * O + k % O) * KK + k / O] = acc;
    } else if (k < KC - 1) {
        const int kx = k - KK * O;
        dwx[(((long long)d * G + gu) * C + kx % C) * KK + kx / C] = acc;
    } else if (db) {
        db[(long long)d * G + gu] = acc;
    }
}

// ---- dL/dx --------------------------------------------------------------------
// dx[v][c] = sum_d sum_taps sum_m dA^d[v - tap][m] W_x[d][m][c][tap]: M = 16
// channels per tile (CT tiles), N = kNT 16-voxel tiles of consecutive voxels,
// K = 6 directions x 9 taps x 4O gate-units.
struct DxStepArgs {
    Geom g;
    int CT;
    const float *frag;        // [6][KK][4U][CT][64][4]
    int k_mul;                // ceil(2^16 / K)
    const float *dA;          // [6][N][V][4O]
    float *dx;                // [N][V][C]
    int nvg;                  // voxel groups (kNT tiles) per batch element
};

template <int U, int CT>
__global__ void __launch_bounds__(64 * kSW)
k_dx_step(DxStepArgs a)
{
    constexpr int O = 16 * U, G = 4 * O, MB = 4 * U;
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const int item = blockIdx.x * kSW + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (item >= a.g.N * a.nvg) return;
    const int KQ = a.g.KQ, radp = a.g.KP >> 1, radq = KQ >> 1, KG = a.g.KP * KQ * MB;
    const int n = item / a.nvg, vg = item - n * a.nvg;
    const long long V = a.g.V;
    const int H = a.g.H, W = a.g.W, C = a.g.C;
    int vv[kNT], zc[kNT], yc[kNT], xc[kNT];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        const long long v = (long long)(vg * kNT + nt) * 16 + col;
        const bool live = v < V;
        vv[nt] = live ? (int)v : -1;
        const int vl = live ? (int)v : 0;
        zc[nt] = vl / (H * W);
        yc[nt] = (vl / W) % H;
        xc[nt] = vl % W;
    }
    f4 acc[CT][kNT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[ct][nt] = f4{0.0f, 0.0f, 0.0f, 0.0f};

    struct Ops {
        f4 a[CT];
        f4 b[kNT];
    };
    for (int d = 0; d < a.g.nd; ++d) {
        const DirGeom dg = a.g.dir[d];
        const int sp = (int)dg.sp, sq = (int)dg.sq, P = dg.P, Q = dg.Q;
        const int ax = a.g.axis[d];
        // in-plane coordinates of each voxel for this direction (the pixel
        // (p - ka + r, q - kb + r) received x through tap (ka, kb))
        int tp[kNT], tq[kNT];
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) {
            tp[nt] = vv[nt] >= 0 ? (ax == 0 ? yc[nt] : zc[nt]) : kDead;
            tq[nt] = ax < 2 ? xc[nt] : yc[nt];
        }
        const auto rs = slice_rsrc(a.dA + ((long long)d * a.g.N + n) * V * G, V * G);
        const float *fr = a.frag + (long long)d * KG * CT * 256 + lane * 4;
        auto load = [&](int tap, int mb, Ops &o) {
            const int kg = tap * MB + mb;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct)
                o.a[ct] = *(const f4 *)(fr + ((long long)kg * CT + ct) * 256);
            const int row = tap_row(tap, a.k_mul), ka = row - radp, kb = tap - row * KQ - radq;
            const int dv = -ka * sp - kb * sq;
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt)
                o.b[nt] = bload4(rs, sel_off(on_plane(tp[nt] - ka, tq[nt] - kb, P, Q),
                                             (unsigned)((vv[nt] + dv) * G + mb * 16 + 4 * q4) * 4u));
        };
        auto step = [&](const Ops &o) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int ct = 0; ct < CT; ++ct)
#pragma unroll
                    for (int nt = 0; nt < kNT; ++nt)
                        acc[ct][nt] = mfma(o.a[ct][i], o.b[nt][i], acc[ct][nt]);
        };
        auto next = [&](int &tap, int &mb) {
            if (++mb == MB) {
                mb = 0;
                ++tap;
            }
        };
        // two operand sets in ping-pong (KG is a multiple of 4): the loads of
        // one are all issued before the products of the other, and no loaded
        // register is copied
        Ops o0, o1;
        load(0, 0, o0);
        int tap = 0, mb = 0;
        for (int kg = 0; kg < KG; kg += 2) {
            next(tap, mb);
            load(tap, mb, o1);
            __builtin_amdgcn_sched_barrier(0);
            step(o0);
            __builtin_amdgcn_sched_barrier(0);
            next(tap, mb);
            // unconditional (the last pass reloads k-group 0, unused) so that
            // the products below wait for their own loads only
            const bool more = kg + 2 < KG;
            load(more ? tap : 0, more ? mb : 0, o0);
            __builtin_amdgcn_sched_barrier(0);
            step(o1);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
        if (vv[nt] < 0) continue;
        float *out = a.dx + ((long long)n * V + vv[nt]) * C;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            const int c0 = ct * 16 + 4 * q4;
            if ((C & 3) == 0 && c0 + 3 < C) {
                *(f4 *)(out + c0) = acc[ct][nt];
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (c0 + i < C) out[c0 + i] = acc[ct][nt][i];
            }
        }
    }
}

// ---- host side --------------------------------------------------------------

inline int pad16(int c) { return (c + 15) / 16 * 16; }
inline unsigned blocks_for(long long n, int per) { return (unsigned)((n + per - 1) / per); }

inline int npg_of(const DirGeom &dg) { return (dg.P * dg.Q + 16 * kNT - 1) / (16 * kNT); }
inline int k_mul_of(const Geom &g) { return (65536 + g.KQ - 1) / g.KQ; }
inline int max_T(const Geom &g)
{
    int m = 0;
    for (int d = 0; d < g.nd; ++d) m = g.dir[d].T > m ? g.dir[d].T : m;
    return m;
}

struct WgShape {
    int NTt, nblk, kch;
    int lds_parts;    // > 0: k_wgrad_lds with this many N-parts (kch chunks each)
};
// Voxel chunks per (direction, block): the launch takes ceil(waves / slots)
// rounds of 1/kch of a block's work; pick the chunk count that minimises that
// (ties: fewer chunks).  Blocks of four N-tiles count one wave per SIMD;
// blocks of fewer tiles do less MFMA work per load and are given three, the
// kernel's occupancy at its register count.
inline WgShape wg_shape(const Geom &g, bool staged = g_wgrad_staged != 0)
{
    const int U = g.O / 16, KK = g.KP * g.KQ, XT = wg_xtiles(KK, g.C);
    const WgBlocks wb = wg_blocks(U, XT, KK);
    WgShape w;
    w.NTt = KK * U + XT;
    w.nblk = wb.nh + wb.nx;
    const DevInfo di = device_info();
    w.lds_parts = 0;
    // (the staged kernel addresses dA, h and x of a (direction, batch
    // element) slice as buffer resources: byte sizes within 31 bits)
    if (staged && U <= 2 && g.C % 4 == 0 &&
        g.V * 4 * g.O * (long long)sizeof(float) < (1LL << 31)) {
        // N-parts of at most kWlPartNT tiles, about one workgroup per CU
        w.lds_parts = (w.NTt + kWlPartNT - 1) / kWlPartNT;
        const int per = g.nd * w.lds_parts;
        const int cus = di.cus > 0 ? di.cus : 256;
        w.kch = cus / per > 1 ? cus / per : 1;
        return w;
    }
    const int per_simd = (wb.th < kWgN && wb.tx < kWgN) ? 3 : 1;
    const long long simds = 4LL * per_simd * (di.cus > 0 ? di.cus : 256);   // wave slots
    const long long per = (long long)g.nd * U * w.nblk;
    double best = 1e30;
    w.kch = 1;
    for (int k = 1; k <= kWgMaxChunks; ++k) {
        const double cost = (double)((per * k + simds - 1) / simds) / k;
        if (cost < best * (1.0 - 1e-9)) {
            best = cost;
            w.kch = k;
        }
    }
    return w;
}

// Weight-gradient partial sums for either kernel (the choice may change
// between a workspace query and the call).
inline size_t wg_partial_floats(const Geom &g)
{
    const WgShape w0 = wg_shape(g, false), w1 = wg_shape(g, true);
    const int kch = w0.kch > w1.kch ? w0.kch : w1.kch;
    return (size_t)g.nd * kch * 4 * g.O * w0.NTt * 16;
}

// Waves below which a step splits each tile's K over a workgroup's waves:
// about two per SIMD (or always / never, when set for testing).
inline int split_threshold()
{
    if (g_step_split == 1) return 1 << 30;
    if (g_step_split == 2 || g_step_split == 3) return 0;
    const DevInfo di = device_info();
    return 8 * (di.cus > 0 ? di.cus : 256);
}

// LDS bytes of k_step_fwd_bls: the staged [x | h] block or the partial sums,
// whichever is larger.
inline size_t fwd_bls_lds(const Geom &g, const FwdStepArgs &a, int U)
{
    const int KP = kSW / U, NU = kNT - kNT / KP;
    size_t m = (size_t)kSW * 4 * NU * 64 * 16;
    const int nch = a.Cp / 4 + 4 * U;
    for (int d = 0; d < g.nd; ++d) {
        const size_t b = (size_t)(a.bp[d] + 2 * (g.KP / 2)) * (a.bq[d] + 2 * (g.KQ / 2)) * nch * 16;
        if (b > m) m = b;
    }
    return m;
}

template <int U>
int launch_fwd_steps(const Geom &g, FwdStepArgs &a, hipStream_t st)
{
    const int T = max_T(g);
    if (g_step_split == 0) {
        const size_t lds = fwd_bls_lds(g, a, U);
        if (lds <= (size_t)device_info().max_lds) {
            if (hipFuncSetAttribute((const void *)k_step_fwd_bls<U>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize,
                                    (int)lds) != hipSuccess)
                return PLSTM_EHIP;
            for (int t = 0; t < T; ++t) {
                a.t = t;
                int nb = 0;
                for (int d = 0; d < kDirs; ++d) {
                    a.base[d] = nb;
                    if (t < g.dir[d].T) nb += g.N * a.nblk[d];
                }
                a.base[kDirs] = nb;
                k_step_fwd_bls<U><<<nb, 64 * kSW, lds, st>>>(a);
                PLSTM_LAUNCH_CHECK();
            }
            return PLSTM_OK;
        }
    }
    const int few = split_threshold();
    // staged x or h of a block (the larger of the two phases)
    size_t lds = 0;
    const int nch = (a.Cp / 4 > 4 * U ? a.Cp / 4 : 4 * U);
    for (int d = 0; d < g.nd; ++d) {
        const size_t b = (size_t)(a.bp[d] + 2 * (g.KP / 2)) * (a.bq[d] + 2 * (g.KQ / 2)) * nch * 16;
        if (b > lds) lds = b;
    }
    const bool staged = g_step_split != 3 && lds <= 64 * 1024;
    for (int t = 0; t < T; ++t) {
        a.t = t;
        int tot = 0;
        for (int d = 0; d < kDirs; ++d) {
            a.base[d] = tot;
            if (t < g.dir[d].T) tot += g.N * U * a.npg[d];
        }
        a.base[kDirs] = tot;
        if (tot < few) {
            k_step_fwd<U, true><<<tot, 64 * kSW, 0, st>>>(a);
        } else if (staged) {
            int nb = 0;
            for (int d = 0; d < kDirs; ++d) {
                a.base[d] = nb;
                if (t < g.dir[d].T) nb += g.N * a.nblk[d];
            }
            a.base[kDirs] = nb;
            k_step_fwd_blk<U><<<nb, 64 * U, lds, st>>>(a);
        } else {
            k_step_fwd<U, false><<<blocks_for(tot, kSW), 64 * kSW, 0, st>>>(a);
        }
        PLSTM_LAUNCH_CHECK();
    }
    return PLSTM_OK;
}

// One wave's LDS region of the staged reverse step, in 16-byte units: its
// staged block (reg_px pixels of 4U chunks) or its partial sums (three
// tiles of U + CT M-tiles, 64 lanes), whichever is larger.
inline int bwd_blk_reg_f4(int U, int CT, int reg_px)
{
    const int st = reg_px * 4 * U, part = (U + CT) * (kNT - 1) * 64;
    return st > part ? st : part;
}

// The staged reverse step for this shape: U <= 2 unit tiles and, with dL/dx
// inside it, at most two channel tiles; `reg_px` the largest staged block.
inline bool bwd_blk_ok(const Geom &g, bool with_dx, int reg_px)
{
    const int U = g.O / 16, CT = with_dx ? pad16(g.C) / 16 : 0;
    if (g_step_split != 0 || U > 2 || CT > 2) return false;
    return (size_t)kSW * bwd_blk_reg_f4(U, CT, reg_px) * 16 <= (size_t)device_info().max_lds;
}

template <int U, int CT>
int launch_bwd_blk(const Geom &g, BwdStepArgs &a, hipStream_t st)
{
    const size_t lds = (size_t)kSW * a.reg_f4 * 16;
    if (hipFuncSetAttribute((const void *)k_step_bwd_blk<U, CT>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        return PLSTM_EHIP;
    // with dL/dx, a last launch (t = -1) gives plane 0's share
    for (int t = max_T(g) - 1; t >= (CT > 0 ? -1 : 0); --t) {
        a.t = t;
        int nb = 0;
        for (int d = 0; d < kDirs; ++d) {
            a.base[d] = nb;
            if (t < g.dir[d].T && g.dir[d].T > 0) nb += g.N * a.nblk[d];
        }
        a.base[kDirs] = nb;
        k_step_bwd_blk<U, CT><<<nb, 64 * kSW, lds, st>>>(a);
        PLSTM_LAUNCH_CHECK();
    }
    return PLSTM_OK;
}

template <int U>
int launch_bwd_steps(const Geom &g, BwdStepArgs &a, hipStream_t st)
{
    if constexpr (U <= 2) {
        if (a.reg_f4 > 0) {
            const int CT = a.dxd ? pad16(g.C) / 16 : 0;
            switch (CT) {
            case 0: return launch_bwd_blk<U, 0>(g, a, st);
            case 1: return launch_bwd_blk<U, 1>(g, a, st);
            case 2: return launch_bwd_blk<U, 2>(g, a, st);
            default: return PLSTM_EUNSUPPORTED;
            }
        }
    }
    // an item of the reverse step holds every unit group: split up to four
    // waves per SIMD
    const int few = g_step_split == 0 ? 2 * split_threshold() : split_threshold();
    for (int t = max_T(g) - 1; t >= 0; --t) {
        a.t = t;
        int tot = 0;
        for (int d = 0; d < kDirs; ++d) {
            a.base[d] = tot;
            if (t < g.dir[d].T) tot += g.N * a.npg[d];
        }
        a.base[kDirs] = tot;
        if (tot < few)
            k_step_bwd<U, true><<<tot, 64 * kSW, 0, st>>>(a);
        else
            k_step_bwd<U, false><<<blocks_for(tot, kSW), 64 * kSW, 0, st>>>(a);
        PLSTM_LAUNCH_CHECK();
    }
    return PLSTM_OK;
}

template <int U, int CT>
int launch_dx(const DxStepArgs &a, hipStream_t st)
{
    k_dx_step<U, CT><<<blocks_for((long long)a.g.N * a.nvg, kSW), 64 * kSW, 0, st>>>(a);
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

template <int U>
int launch_dx_ct(const DxStepArgs &a, hipStream_t st)
{
    switch (a.CT) {
    case 1: return launch_dx<U, 1>(a, st);
    case 2: return launch_dx<U, 2>(a, st);
    case 3: return launch_dx<U, 3>(a, st);
    case 4: return launch_dx<U, 4>(a, st);
    default: return PLSTM_EUNSUPPORTED;
    }
}

}  // namespace

int g_step_split = 0;
int g_step_bf16_mfma = 1;
int g_wgrad_staged = 1;

namespace {
// knob values 1 and 4 select the macro-tiled bf16 kernels; 4 keeps the
// 16-unit layers at one plane per launch
inline bool b16_mt_mode() { return g_step_bf16_mfma == 1 || g_step_bf16_mfma == 4; }
}  // namespace

bool step_supported(const Geom &g)
{
    if (g.O != 16 && g.O != 32 && g.O != 64) return false;
    if (g.KQ < 1 || g.KQ > 7 || g.KQ % 2 == 0 || (g.KP != 1 && g.KP != g.KQ)) return false;
    const long long Cp = pad16(g.C);
    if (Cp > 64) return false;
    // slices addressed through buffer resources: byte sizes fit 31 bits
    const long long lim = 1LL << 31;
    if (g.V * 4 * g.O * 4 >= lim || g.V * Cp * 4 >= lim) return false;
    // wave items of a step fit an int
    long long items = 0;
    for (int d = 0; d < g.nd; ++d) items += (long long)g.N * (g.O / 16) * npg_of(g.dir[d]);
    return items < (1LL << 30);
}

// bf16 storage with 32 or 64 hidden units takes the bf16 MFMA.
// 16-unit layers take the bf16 MFMA only as the macro-tiled kernel with packed
// taps (3D, at most 8 input channels).
inline bool b16_packed(const Geom &g) { return g.O == 16 && g.C <= 8 && g.nd == kDirs; }
inline bool use_b16(const Geom &g, int dtype)
{
    return dtype == PLSTM_BF16 && g_step_bf16_mfma &&
           (g.O == 32 || g.O == 64 || (b16_packed(g) && b16_mt_mode()));
}
inline int pad32(int c) { return (c + 31) / 32 * 32; }
inline int max_pq(const Geom &g)
{
    int m = 0;
    for (int d = 0; d < g.nd; ++d)
        if (g.dir[d].P * g.dir[d].Q > m) m = g.dir[d].P * g.dir[d].Q;
    return m;
}
// bf16 channel padding and K-groups: taps padded to 32 channels each, or
// packed (four input slots or two h taps per K-group)
struct B16K {
    int C32, KX, KG;
};
inline B16K b16_k(const Geom &g)
{
    const int KK = g.KP * g.KQ;
    if (g.O == 16) return {8, (KK + 3) / 4, (KK + 3) / 4 + (KK + 1) / 2};
    const int C32 = pad32(g.C);
    return {C32, KK * C32 / 32, KK * (C32 + g.O) / 32};
}

bool step_b16_packed(const Geom &g, int dtype) { return use_b16(g, dtype) && g.O == 16; }

size_t step_fwd_ws(const Geom &g)
{
    const int U = g.O / 16, Cp = pad16(g.C), KK = g.KP * g.KQ, KG = KK * (Cp + g.O) / 16;
    Carve cv(nullptr);
    cv.take<float>((size_t)g.N * g.V * Cp);          // padded x
    cv.take<float>((size_t)g.nd * U * KG * 1024);    // A fragments
    cv.take<float>((size_t)g.nd * 4 * g.O);          // bias
    size_t need = cv.off;
    if (g.O % 32 == 0 || b16_packed(g)) {           // bf16 variant
        const B16K k = b16_k(g);
        Carve cb(nullptr);
        cb.take<uint16_t>((size_t)g.N * g.V * k.C32);
        cb.take<uint16_t>((size_t)g.nd * U * k.KG * 2048);
        cb.take<float>((size_t)g.nd * 4 * g.O);
        cb.take<uint16_t>((size_t)g.nd * g.N * g.V * g.O);
        cb.take<float>((size_t)g.nd * g.N * 2 * max_pq(g) * g.O);   // c^d, two planes
        if (g.O >= 32) {                             // projection variant
            cb.take<uint16_t>((size_t)g.nd * (g.O / 16) * k.KX * 2048);
            cb.take<uint16_t>((size_t)g.nd * (g.O / 16) * (k.KG - k.KX) * 2048);
            cb.take<uint16_t>((size_t)g.nd * g.N * g.V * 4 * g.O);
        }
        if (cb.off > need) need = cb.off;
    }
    return need;
}

// 64-pixel blocks of the LDS-staged forward kernels, as square as a plane
// allows: BP the largest power of two up to min(P, 8), BQ = 64 / BP.
void set_blocks(const Geom &g, int *bp, int *bq, int *nbq, int *nblk)
{
    for (int d = 0; d < kDirs; ++d) {
        const DirGeom &dg = g.dir[d];
        int b = 1;
        while (b < 8 && 2 * b <= dg.P) b *= 2;
        bp[d] = b;
        bq[d] = 64 / b;
        nbq[d] = dg.Q > 0 ? (dg.Q + bq[d] - 1) / bq[d] : 0;
        nblk[d] = dg.P > 0 ? (dg.P + b - 1) / b * nbq[d] : 0;
    }
}

// LDS bytes of the staged pixel blocks (the largest over the directions).
size_t b16_block_lds(const Geom &g, const FwdB16Args &a)
{
    size_t m = 0;
    const int nch = (a.C32 + g.O) / 8;
    for (int d = 0; d < g.nd; ++d) {
        const size_t b = (size_t)(a.bp[d] + 2 * (g.KP / 2)) * (a.bq[d] + 2 * (g.KQ / 2)) * nch * 16;
        if (b > m) m = b;
    }
    return m;
}

// Wave layout of the macro-tiled bf16 forward: WM x WN waves, pixel blocks
// of (4 WN) x 16.  64 units: 2 x 4 waves, one workgroup of 256 pixels per
// CU; 32 units: 2 x 2 waves of one unit group each, three workgroups of 128
// pixels per CU.
template <int U> struct MtShape;
template <> struct MtShape<4> { static constexpr int WM = 2, WN = 4; };
template <> struct MtShape<2> { static constexpr int WM = 2, WN = 2; };
template <> struct MtShape<1> { static constexpr int WM = 1, WN = 4; };
void set_mt_blocks(const Geom &g, int wn, int *bp, int *bq, int *nbq, int *nblk)
{
    for (int d = 0; d < kDirs; ++d) {
        const DirGeom &dg = g.dir[d];
        bp[d] = 4 * wn;
        bq[d] = 16;
        nbq[d] = dg.Q > 0 ? (dg.Q + 15) / 16 : 0;
        nblk[d] = dg.P > 0 ? (dg.P + bp[d] - 1) / bp[d] * nbq[d] : 0;
    }
}

// Dynamic LDS bytes of the macro-tiled kernel: the staged block with its
// halo, NCH + 2 chunks per pixel (6 with packed taps).  Its A ring (three
// arrays of 4U tiles of 1 KB) is static.
size_t b16_mt_stage_lds(const Geom &g, const FwdB16Args &a, int wn)
{
    const int nchp = g.O == 16 ? 6 : (a.C32 + g.O) / 8 + 2;
    return (size_t)(4 * wn + 2 * (g.KP / 2)) * (16 + 2 * (g.KQ / 2)) * nchp * 16;
}

template <int U>
int launch_fwd_b16_steps(const Geom &g, FwdB16Args &a, hipStream_t st, int *launches)
{
    *launches = max_T(g);
    const int T = max_T(g);
    const int few = split_threshold();
    constexpr int WM = MtShape<U>::WM, WN = MtShape<U>::WN;
    const size_t lds_mt = b16_mt_stage_lds(g, a, WN);
    const bool mt = b16_mt_mode() &&
                    (size_t)3 * 4 * U * 1024 + lds_mt <= (size_t)device_info().max_lds;
    size_t lds = 0;
    bool staged = false;
    if (U == 1 && !mt) return PLSTM_EUNSUPPORTED;   // packed taps: macro-tiled only
    if constexpr (U == 1) {
        // two planes per launch: 3 x 3 filters, an even number of planes in
        // every direction
        bool two = g_step_bf16_mfma == 1 && g.KP == 3 && g.KQ == 3;
        for (int d = 0; d < g.nd; ++d) two = two && g.dir[d].T % 2 == 0;
        if (two) {
            set_mt_blocks(g, 4, a.bp, a.bq, a.nbq, a.nblk);
            const int lds2 = kS2Grid * kS2Grid * kS2Chunks * 16;
            if (hipFuncSetAttribute((const void *)k_step2_fwd_b16_pk<kS2Waves>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize,
                                    lds2) != hipSuccess)
                return PLSTM_EHIP;
            for (int t = 0; t < T; t += 2) {
                a.t = t;
                int nb = 0;
                for (int d = 0; d < kDirs; ++d) {
                    a.base[d] = nb;
                    if (t < g.dir[d].T) nb += g.N * a.nblk[d];
                }
                a.base[kDirs] = nb;
                if (nb == 0) continue;
                const int grid = (nb + kXcds - 1) / kXcds * kXcds;
                k_step2_fwd_b16_pk<kS2Waves><<<grid, 64 * kS2Waves, lds2, st>>>(a);
                PLSTM_LAUNCH_CHECK();
            }
            *launches = (T + 1) / 2;
            return PLSTM_OK;
        }
    }
    if (mt) {
        set_mt_blocks(g, WN, a.bp, a.bq, a.nbq, a.nblk);
        if (hipFuncSetAttribute((const void *)k_step_fwd_b16_mt<U, WM, WN, 0>,
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)lds_mt) != hipSuccess)
            return PLSTM_EHIP;
    } else {
        set_blocks(g, a.bp, a.bq, a.nbq, a.nblk);
        lds = b16_block_lds(g, a);
        staged = (g_step_bf16_mfma == 1 || g_step_bf16_mfma == 3) && lds <= 64 * 1024;
    }
    for (int t = 0; t < T; ++t) {
        a.t = t;
        if (mt) {
            int nb = 0;
            for (int d = 0; d < kDirs; ++d) {
                a.base[d] = nb;
                if (t < g.dir[d].T) nb += g.N * a.nblk[d];
            }
            a.base[kDirs] = nb;
            if (nb == 0) continue;
            const int grid = (nb + kXcds - 1) / kXcds * kXcds;
            k_step_fwd_b16_mt<U, WM, WN, 0><<<grid, 64 * WM * WN, lds_mt, st>>>(a);
            PLSTM_LAUNCH_CHECK();
            continue;
        }
        if constexpr (U == 1) return PLSTM_EUNSUPPORTED;
        else {
        int tot = 0;
        for (int d = 0; d < kDirs; ++d) {
            a.base[d] = tot;
            if (t < g.dir[d].T) tot += g.N * U * a.npg[d];
        }
        a.base[kDirs] = tot;
        if (tot < few) {
            k_step_fwd_b16<U, true><<<tot, 64 * kSW, 0, st>>>(a);
        } else if (staged) {
            int nb = 0;
            for (int d = 0; d < kDirs; ++d) {
                a.base[d] = nb;
                if (t < g.dir[d].T) nb += g.N * a.nblk[d];
            }
            a.base[kDirs] = nb;
            k_step_fwd_b16_blk<U><<<nb, 64 * U, lds, st>>>(a);
        } else {
            k_step_fwd_b16<U, false><<<blocks_for(tot, kSW), 64 * kSW, 0, st>>>(a);
        }
        PLSTM_LAUNCH_CHECK();
        }
    }
    return PLSTM_OK;
}

// Projection variant (knob value 5, 32 or 64 units): x's contraction for every
// plane of every direction in one launch of the macro-tiled kernel (MODE 1),
// which writes bf16 pre-activations, then one launch per plane of the
// recurrent part alone (MODE 2), which adds them in its epilogue.
template <int U>
int launch_fwd_b16_proj(const Geom &g, FwdB16Args &a, const uint16_t *fragx,
                        const uint16_t *fragh, int KX, int KH, hipStream_t st, int *launches)
{
    constexpr int WM = MtShape<U>::WM, WN = MtShape<U>::WN, O = 16 * U;
    const int T = max_T(g);
    const size_t ring = (size_t)3 * 4 * U * 1024;
    const size_t halo = (size_t)(4 * WN + 2 * (g.KP / 2)) * (16 + 2 * (g.KQ / 2)) * 16;
    const size_t lds1 = halo * (a.C32 / 8 + 2), lds2 = halo * (O / 8 + 2);
    if (ring + lds1 > (size_t)device_info().max_lds || ring + lds2 > (size_t)device_info().max_lds)
        return PLSTM_EUNSUPPORTED;
    if (hipFuncSetAttribute((const void *)k_step_fwd_b16_mt<U, WM, WN, 1>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds1) != hipSuccess ||
        hipFuncSetAttribute((const void *)k_step_fwd_b16_mt<U, WM, WN, 2>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds2) != hipSuccess)
        return PLSTM_EHIP;
    set_mt_blocks(g, WN, a.bp, a.bq, a.nbq, a.nblk);
    // MODE 1: all planes
    FwdB16Args p = a;
    p.KX = KX; p.KG = KX; p.frag = fragx; p.t = 0;
    long long nb = 0;
    for (int d = 0; d < kDirs; ++d) {
        p.base[d] = (int)nb;
        nb += (long long)g.N * g.dir[d].T * a.nblk[d];
    }
    if (nb >= (1LL << 30)) return PLSTM_EUNSUPPORTED;
    p.base[kDirs] = (int)nb;
    int n_launch = 0;
    if (nb > 0) {
        const int grid = (int)((nb + kXcds - 1) / kXcds * kXcds);
        k_step_fwd_b16_mt<U, WM, WN, 1><<<grid, 64 * WM * WN, lds1, st>>>(p);
        PLSTM_LAUNCH_CHECK();
        ++n_launch;
    }
    // MODE 2: the recurrence, plane by plane
    FwdB16Args q = a;
    q.C32 = 0; q.KX = 0; q.KG = KH; q.frag = fragh; q.cx_mul32 = 0;
    for (int t = 0; t < T; ++t) {
        q.t = t;
        int nbt = 0;
        for (int d = 0; d < kDirs; ++d) {
            q.base[d] = nbt;
            if (t < g.dir[d].T) nbt += g.N * a.nblk[d];
        }
        q.base[kDirs] = nbt;
        if (nbt == 0) continue;
        const int grid = (nbt + kXcds - 1) / kXcds * kXcds;
        k_step_fwd_b16_mt<U, WM, WN, 2><<<grid, 64 * WM * WN, lds2, st>>>(q);
        PLSTM_LAUNCH_CHECK();
        ++n_launch;
    }
    *launches = n_launch;
    return PLSTM_OK;
}

static int step_fwd_b16(const Geom &g, const uint16_t *x, const uint16_t *wx,
                        const uint16_t *wh, const uint16_t *b, void *h, float *cell, void *ws,
                        hipStream_t st)
{
    const B16K k = b16_k(g);
    const int U = g.O / 16, C32 = k.C32, KK = g.KP * g.KQ, KX = k.KX, KG = k.KG;
    Carve cv(ws);
    uint16_t *xb = cv.take<uint16_t>((size_t)g.N * g.V * C32);
    uint16_t *frag = cv.take<uint16_t>((size_t)g.nd * U * KG * 2048);
    float *bias = cv.take<float>((size_t)g.nd * 4 * g.O);
    uint16_t *hb = cv.take<uint16_t>((size_t)g.nd * g.N * g.V * g.O);
    float *cpp = cv.take<float>((size_t)g.nd * g.N * 2 * max_pq(g) * g.O);
    const long long nvox = (long long)g.N * g.V;
    const long long nfrag = (long long)g.nd * U * KG * 2048;
    timing_begin("sweep_fwd_step_bf16", st);
    // channels already a multiple of 32: the input is its own padded copy
    if (C32 != g.C) {
        k_pad_x_b16<<<blocks_for(nvox * C32, 256), 256, 0, st>>>(nvox, g.C, C32, x, xb);
        PLSTM_LAUNCH_CHECK();
    }
    k_pack_fwd_b16<<<blocks_for(nfrag, 256), 256, 0, st>>>(g.nd, g.O, g.C, C32, KX, KG, KK,
                                                           g.O == 16, wx, wh, b, frag, bias);
    PLSTM_LAUNCH_CHECK();
    FwdB16Args a;
    a.g = g;
    a.C32 = C32; a.KX = KX; a.KG = KG;
    a.cx_mul32 = C32 >= 32 ? (65536 + C32 / 32 - 1) / (C32 / 32) : 0;
    a.k_mul = k_mul_of(g);
    a.xb = C32 != g.C ? xb : x;
    a.frag = frag; a.bias = bias;
    a.cell = cell; a.hb = hb;
    a.cpp = cpp; a.pqmax = max_pq(g);
    a.preact = nullptr;
    for (int d = 0; d < kDirs; ++d) a.npg[d] = npg_of(g.dir[d]);
    int steps = 0;
    int rc;
    if (g_step_bf16_mfma == 5 && U >= 2) {
        // projection variant: x-only and h-only fragments, pre-activations
        const int KH = KG - KX;
        uint16_t *fragx = cv.take<uint16_t>((size_t)g.nd * U * KX * 2048);
        uint16_t *fragh = cv.take<uint16_t>((size_t)g.nd * U * KH * 2048);
        a.preact = cv.take<uint16_t>((size_t)g.nd * g.N * g.V * 4 * g.O);
        const long long nfx = (long long)g.nd * U * KX * 2048, nfh = (long long)g.nd * U * KH * 2048;
        k_pack_fwd_b16<<<blocks_for(nfx, 256), 256, 0, st>>>(g.nd, g.O, g.C, C32, KX, KX, KK, 0,
                                                              wx, wh, b, fragx, bias);
        PLSTM_LAUNCH_CHECK();
        k_pack_fwd_b16<<<blocks_for(nfh, 256), 256, 0, st>>>(g.nd, g.O, g.C, C32, 0, KH, KK, 0,
                                                              wx, wh, b, fragh, bias);
        PLSTM_LAUNCH_CHECK();
        rc = U == 2 ? launch_fwd_b16_proj<2>(g, a, fragx, fragh, KX, KH, st, &steps)
                    : launch_fwd_b16_proj<4>(g, a, fragx, fragh, KX, KH, st, &steps);
        steps += 2;
    } else {
        rc = U == 1   ? launch_fwd_b16_steps<1>(g, a, st, &steps)
             : U == 2 ? launch_fwd_b16_steps<2>(g, a, st, &steps)
                      : launch_fwd_b16_steps<4>(g, a, st, &steps);
    }
    if (rc != PLSTM_OK) return rc;
    timing_end((C32 != g.C ? 2 : 1) + steps, st);
    return sum_dirs_bf16(g, hb, h, st);
}

int step_fwd(const Geom &g, int dtype, const void *x, const void *wx, const void *wh,
             const void *b, float *hd, float *cell, float *gates, void *h, void *ws,
             hipStream_t st)
{
    if (!step_supported(g)) return PLSTM_EUNSUPPORTED;
    if (use_b16(g, dtype) && !gates)
        return step_fwd_b16(g, (const uint16_t *)x, (const uint16_t *)wx, (const uint16_t *)wh,
                            (const uint16_t *)b, h, cell, ws, st);
    const int U = g.O / 16, Cp = pad16(g.C);
    const int KK = g.KP * g.KQ, KX = KK * Cp / 16, KG = KX + KK * U;
    Carve cv(ws);
    float *xp = cv.take<float>((size_t)g.N * g.V * Cp);
    float *frag = cv.take<float>((size_t)g.nd * U * KG * 1024);
    float *bias = cv.take<float>((size_t)g.nd * 4 * g.O);
    const long long nvox = (long long)g.N * g.V;
    const long long nfrag = (long long)g.nd * U * KG * 1024;

    timing_begin("sweep_fwd_step", st);
    auto pad_x = [&]() {
        if (dtype == PLSTM_BF16)
            k_pad_x<uint16_t><<<blocks_for(nvox * Cp, 256), 256, 0, st>>>(nvox, g.C, Cp,
                                                                          (const uint16_t *)x, xp);
        else
            k_pad_x<float><<<blocks_for(nvox * Cp, 256), 256, 0, st>>>(nvox, g.C, Cp,
                                                                       (const float *)x, xp);
    };

    // 2D layers with 16 units: line blocks, S lines per launch (S r <= 16),
    // the input taps packed densely as (tap, channel) pairs; fp32 x is staged
    // from the input itself (C floats per pixel), bf16 from its fp32 copy
    const int KXL = (g.KQ * g.C + 15) / 16, KGL = KXL + g.KQ;
    if (g.nd == 4 && g.KP == 1 && g.O == 16 && (g_step_split == 0 || g_step_split == 2) &&
        line_fwd_dyn_lds(KGL, g.C) <= 64 * 1024) {
        const bool x_direct = dtype != PLSTM_BF16;
        if (!x_direct) {
            pad_x();
            PLSTM_LAUNCH_CHECK();
        }
        const long long nfl = (long long)g.nd * KGL * 1024;
        if (dtype == PLSTM_BF16)
            k_pack_line<uint16_t><<<blocks_for(nfl, 256), 256, 0, st>>>(
                g.nd, g.C, g.KQ, KXL, KGL, (const uint16_t *)wx, (const uint16_t *)wh,
                (const uint16_t *)b, frag, bias);
        else
            k_pack_line<float><<<blocks_for(nfl, 256), 256, 0, st>>>(
                g.nd, g.C, g.KQ, KXL, KGL, (const float *)wx, (const float *)wh,
                (const float *)b, frag, bias);
        PLSTM_LAUNCH_CHECK();
        LineFwdArgs la;
        la.g = g;
        const int rq = g.KQ / 2;
        la.S = rq == 0 ? 16 : (16 / rq < 16 ? 16 / rq : 16);
        la.Cp = x_direct ? g.C : Cp; la.KX = KXL; la.KG = KGL;
        la.c_mul = (65536 + g.C - 1) / g.C;
        la.xp = x_direct ? (const float *)x : xp; la.frag = frag; la.bias = bias;
        la.hd = hd; la.cell = cell; la.gates = gates;
        for (int d = 0; d < kDirs; ++d) la.nseg[d] = (g.dir[d].Q + kLineSeg - 1) / kLineSeg;
        const int T = max_T(g);
        const size_t dyn = line_fwd_dyn_lds(KGL, g.C);
        if (hipFuncSetAttribute((const void *)k_line_fwd, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)dyn) != hipSuccess)
            return PLSTM_EHIP;
        int launches = 0;
        for (int t0 = 0; t0 < T; t0 += la.S) {
            la.t0 = t0;
            int nb = 0;
            for (int d = 0; d < kDirs; ++d) {
                la.base[d] = nb;
                if (t0 < g.dir[d].T) nb += g.N * la.nseg[d];
            }
            la.base[kDirs] = nb;
            k_line_fwd<<<nb, 256, dyn, st>>>(la);
            PLSTM_LAUNCH_CHECK();
            ++launches;
        }
        timing_end((x_direct ? 1 : 2) + launches, st);
        return sum_dirs(g, dtype, hd, h, st);
    }
    // fp32 x whose channel count is already a multiple of 16 is read in place
    const bool x_in_place = dtype == PLSTM_F32 && Cp == g.C;
    if (!x_in_place) {
        pad_x();
        PLSTM_LAUNCH_CHECK();
    }

    if (dtype == PLSTM_BF16)
        k_pack_fwd<uint16_t><<<blocks_for(nfrag, 256), 256, 0, st>>>(
            g.nd, g.O, g.C, Cp, KX, KG, KK, (const uint16_t *)wx, (const uint16_t *)wh,
            (const uint16_t *)b, frag, bias);
    else
        k_pack_fwd<float><<<blocks_for(nfrag, 256), 256, 0, st>>>(
            g.nd, g.O, g.C, Cp, KX, KG, KK, (const float *)wx, (const float *)wh, (const float *)b,
            frag, bias);
    PLSTM_LAUNCH_CHECK();
    FwdStepArgs a;
    a.g = g;
    a.Cp = Cp; a.KX = KX; a.KG = KG;
    a.cx_mul = (65536 + Cp / 16 - 1) / (Cp / 16);
    a.k_mul = k_mul_of(g);
    a.xp = x_in_place ? (const float *)x : xp; a.frag = frag; a.bias = bias;
    a.hd = hd; a.cell = cell; a.gates = gates;
    for (int d = 0; d < kDirs; ++d) a.npg[d] = npg_of(g.dir[d]);
    set_blocks(g, a.bp, a.bq, a.nbq, a.nblk);
    int rc;
    switch (U) {
    case 1: rc = launch_fwd_steps<1>(g, a, st); break;
    case 2: rc = launch_fwd_steps<2>(g, a, st); break;
    default: rc = launch_fwd_steps<4>(g, a, st); break;
    }
    if (rc != PLSTM_OK) return rc;
    timing_end((x_in_place ? 1 : 2) + max_T(g), st);
    return sum_dirs(g, dtype, hd, h, st);
}

// The 2D layer with 16 units and at most 4 input channels takes dL/dx from
// the reverse line blocks.
inline bool line_bwd_dx(const Geom &g) { return g.nd == 4 && g.KP == 1 && g.O == 16 && g.C <= 4; }
// Segments of the longest line of the 2D layer (bias-gradient partials of
// the reverse line blocks).
inline int line_nsegmax(const Geom &g)
{
    int m = 0;
    for (int d = 0; d < g.nd; ++d) {
        const int ns = (g.dir[d].Q + kLineSeg - 1) / kLineSeg;
        m = ns > m ? ns : m;
    }
    return m;
}
inline bool line_bwd_geom(const Geom &g) { return g.nd == 4 && g.KP == 1 && g.O == 16; }
// Shapes whose reverse sweep may give dL/dx per direction (the 2D line blocks,
// or the staged reverse step with at most 32 units and 32 input channels).
inline bool bwd_dxd(const Geom &g) { return line_bwd_dx(g) || (g.O <= 32 && pad16(g.C) <= 32); }

size_t step_bwd_ws(const Geom &g)
{
    const int U = g.O / 16, Cp = pad16(g.C), G = 4 * g.O, KK = g.KP * g.KQ;
    const WgShape w = wg_shape(g);
    Carve cv(nullptr);
    cv.take<float>((size_t)g.nd * g.N * g.V * G);                  // dA
    cv.take<float>((size_t)g.nd * g.N * g.V * g.O);                // dL/dc * f
    cv.take<float>((size_t)g.nd * U * KK * 4 * U * 256);           // W_h^T fragments
    cv.take<float>(wg_partial_floats(g));                           // weight-gradient partials
    cv.take<float>((size_t)g.nd * KK * 4 * U * (Cp / 16) * 256);   // W_x^T fragments
    if (bwd_dxd(g)) cv.take<float>((size_t)g.nd * g.N * g.V * g.C);   // dL/dx per direction
    if (line_bwd_geom(g)) cv.take<float>((size_t)g.nd * g.N * line_nsegmax(g) * 64);  // db partials
    return cv.off;
}

// dL/dx from the gate gradients of all six directions (any O in 16, 32, 64;
// C <= 64).
int step_dx(const Geom &g, const float *wx, const float *dA, float *fragx, float *dx,
            hipStream_t st)
{
    const int U = g.O / 16, CT = pad16(g.C) / 16;
    const int KK = g.KP * g.KQ;
    const long long nf = (long long)g.nd * KK * 4 * U * CT * 256;
    timing_begin("dx_step", st);
    k_pack_dx<<<blocks_for(nf, 256), 256, 0, st>>>(g.nd, g.O, g.C, CT, KK, wx, fragx);
    PLSTM_LAUNCH_CHECK();
    DxStepArgs a;
    a.g = g;
    a.CT = CT;
    a.frag = fragx;
    a.k_mul = k_mul_of(g);
    a.dA = dA;
    a.dx = dx;
    a.nvg = (int)((g.V + 16 * kNT - 1) / (16 * kNT));
    int rc;
    switch (U) {
    case 1: rc = launch_dx_ct<1>(a, st); break;
    case 2: rc = launch_dx_ct<2>(a, st); break;
    default: rc = launch_dx_ct<4>(a, st); break;
    }
    if (rc != PLSTM_OK) return rc;
    timing_end(2, st);
    return PLSTM_OK;
}

size_t step_dx_ws(const Geom &g)
{
    Carve cv(nullptr);
    cv.take<float>((size_t)g.nd * g.KP * g.KQ * 4 * (g.O / 16) * (pad16(g.C) / 16) * 256);
    return cv.off;
}

int step_bwd(const Geom &g, const float *x, const float *wh, const float *wx, const Saved &sv,
             const float *dh, float *dx, float *dwx, float *dwh, float *db, void *ws,
             hipStream_t st)
{
    if (!step_supported(g)) return PLSTM_EUNSUPPORTED;
    const int U = g.O / 16, Cp = pad16(g.C), G = 4 * g.O, KK = g.KP * g.KQ;
    const WgShape w = wg_shape(g);
    Carve cv(ws);
    float *dA = cv.take<float>((size_t)g.nd * g.N * g.V * G);
    float *gcf = cv.take<float>((size_t)g.nd * g.N * g.V * g.O);
    float *frag = cv.take<float>((size_t)g.nd * U * KK * 4 * U * 256);
    float *partial = cv.take<float>(wg_partial_floats(g));
    float *fragx = cv.take<float>((size_t)g.nd * KK * 4 * U * (Cp / 16) * 256);
    float *dxd = bwd_dxd(g) ? cv.take<float>((size_t)g.nd * g.N * g.V * g.C) : nullptr;
    float *dbl = line_bwd_geom(g) ? cv.take<float>((size_t)g.nd * g.N * line_nsegmax(g) * 64)
                                  : nullptr;
    bool db_done = false;
    const long long nvox = (long long)g.N * g.V;
    bool dx_done = false;

    timing_begin("sweep_bwd_step", st);
    k_pack_bwd<<<blocks_for((long long)g.nd * U * KK * 4 * U * 256, 256), 256, 0, st>>>(
        g.nd, g.O, KK, wh, frag);
    PLSTM_LAUNCH_CHECK();
    const bool fuse_dx = dx && dxd && line_bwd_dx(g);
    const size_t line_dyn = line_bwd_dyn_lds(g.KQ * 4, fuse_dx ? g.KQ * G * g.C : 0);
    if (g.nd == 4 && g.KP == 1 && g.O == 16 && (g_step_split == 0 || g_step_split == 2) &&
        line_dyn + 2 * kLineSlots * 64 + 4 * 64 * 16 + 4 * 4 * 4 * 16 <= (size_t)device_info().max_lds) {
        // 2D layers with 16 units: line blocks, S lines per launch (S r <= 16)
        LineBwdArgs la;
        la.g = g;
        const int rq = g.KQ / 2;
        la.S = rq == 0 ? 16 : (16 / rq < 16 ? 16 / rq : 16);
        if (kLineSeg + 2 * la.S * rq > 96) return PLSTM_EUNSUPPORTED;   // two tiles per wave
        la.frag = frag;
        la.gates = sv.gates; la.cell = sv.cell; la.dh = dh;
        la.dA = dA; la.gcf = gcf;
        la.wx = wx;
        la.dxd = fuse_dx ? dxd : nullptr;
        la.dbp = dbl;
        la.nsegmax = line_nsegmax(g);
        for (int d = 0; d < kDirs; ++d) la.nseg[d] = (g.dir[d].Q + kLineSeg - 1) / kLineSeg;
        const size_t dyn = line_dyn;
        if (hipFuncSetAttribute((const void *)k_line_bwd, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)dyn) != hipSuccess)
            return PLSTM_EHIP;
        const int T = max_T(g);
        int launches = 0;
        for (int r0 = 0; r0 < T; r0 += la.S) {
            la.r0 = r0;
            int nb = 0;
            for (int d = 0; d < kDirs; ++d) {
                la.base[d] = nb;
                if (r0 < g.dir[d].T) nb += g.N * la.nseg[d];
            }
            la.base[kDirs] = nb;
            k_line_bwd<<<nb, 256, dyn, st>>>(la);
            PLSTM_LAUNCH_CHECK();
            ++launches;
        }
        timing_end(1 + launches, st);
        if (fuse_dx) {
            timing_begin("dx_step", st);
            const long long ndx = nvox * g.C;
            k_sum_dx4<<<blocks_for(ndx, 256), 256, 0, st>>>(ndx, dxd, dx);
            PLSTM_LAUNCH_CHECK();
            timing_end(1, st);
            dx_done = true;
        }
        LineDbReduceArgs ra;
        ra.nd = g.nd; ra.N = g.N; ra.nsegmax = la.nsegmax;
        for (int d = 0; d < kDirs; ++d) ra.nseg[d] = la.nseg[d];
        ra.dbp = dbl;
        ra.db = db;
        timing_begin("wgrad_step", st);
        k_line_db_reduce<<<blocks_for(g.nd * G, 256), 256, 0, st>>>(ra);
        PLSTM_LAUNCH_CHECK();
        timing_end(1, st);
        db_done = true;
    } else {
        BwdStepArgs a;
        a.g = g;
        a.frag = frag;
        a.k_mul = k_mul_of(g);
        a.gates = sv.gates; a.cell = sv.cell; a.dh = dh;
        a.dA = dA; a.gcf = gcf;
        for (int d = 0; d < kDirs; ++d) a.npg[d] = npg_of(g.dir[d]);
        set_blocks(g, a.bp, a.bq, a.nbq, a.nblk);
        int reg_px = 64;
        for (int d = 0; d < g.nd; ++d) {
            const int px = (a.bp[d] + 2 * (g.KP / 2)) * (a.bq[d] + 2 * (g.KQ / 2));
            if (px > reg_px) reg_px = px;
        }
        // the staged reverse step, with dL/dx inside it where it takes it
        const bool with_dx = dx && dxd && bwd_blk_ok(g, true, reg_px);
        a.reg_f4 = bwd_blk_ok(g, with_dx, reg_px)
                       ? bwd_blk_reg_f4(U, with_dx ? Cp / 16 : 0, reg_px) : 0;
        a.fragx = fragx;
        a.dxd = with_dx ? dxd : nullptr;
        if (with_dx) {
            const long long nf = (long long)g.nd * KK * 4 * U * (Cp / 16) * 256;
            k_pack_dx<<<blocks_for(nf, 256), 256, 0, st>>>(g.nd, g.O, g.C, Cp / 16, KK, wx,
                                                            fragx);
            PLSTM_LAUNCH_CHECK();
        }
        int rc;
        switch (U) {
        case 1: rc = launch_bwd_steps<1>(g, a, st); break;
        case 2: rc = launch_bwd_steps<2>(g, a, st); break;
        default: rc = launch_bwd_steps<4>(g, a, st); break;
        }
        if (rc != PLSTM_OK) return rc;
        timing_end((with_dx ? 3 : 1) + max_T(g), st);
        if (with_dx) {
            timing_begin("dx_step", st);
            const long long ndx = nvox * g.C;
            if ((ndx & 3) == 0 && ((uintptr_t)dx & 15) == 0)
                k_sum_dxn4<<<blocks_for(ndx / 4, 256), 256, 0, st>>>(ndx / 4, g.nd,
                                                                      (const f4 *)dxd, (f4 *)dx);
            else
                k_sum_dxn<<<blocks_for(ndx, 256), 256, 0, st>>>(ndx, g.nd, dxd, dx);
            PLSTM_LAUNCH_CHECK();
            timing_end(1, st);
            dx_done = true;
        }
    }

    timing_begin("wgrad_step", st);
    if (w.lds_parts > 0) {
        WlArgs la;
        la.g = g;
        la.NTt = w.NTt; la.nparts = w.lds_parts; la.kch = w.kch;
        la.x = x; la.hd = sv.hd; la.dA = dA;
        la.partial = partial;
        const int nb = g.nd * w.lds_parts * w.kch;
        const int nmax = (w.NTt + w.lds_parts - 1) / w.lds_parts * 16;   // widest part's columns
        const size_t lds = 2 * (size_t)(G + nmax) * kWlRow * sizeof(float);
        if (U == 1) {
            (void)hipFuncSetAttribute((const void *)k_wgrad_lds<1>,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            k_wgrad_lds<1><<<nb, kWlThreads, lds, st>>>(la);
        } else {
            (void)hipFuncSetAttribute((const void *)k_wgrad_lds<2>,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            k_wgrad_lds<2><<<nb, kWlThreads, lds, st>>>(la);
        }
        PLSTM_LAUNCH_CHECK();
        const long long nout = (long long)g.nd * G * (KK * (g.O + g.C) + 1);
        k_wgrad_step_reduce<<<blocks_for(nout, 256), 256, 0, st>>>(
            g.nd, g.O, g.C, Cp, KK, w.NTt, w.kch, partial, dwx, dwh, db_done ? nullptr : db);
        PLSTM_LAUNCH_CHECK();
        timing_end(2, st);
        if (dx && !dx_done) return step_dx(g, wx, dA, fragx, dx, st);
        return PLSTM_OK;
    }
    // the x tiles read one channel per lane: x itself, C floats per voxel
    WgStepArgs wa;
    wa.g = g;
    wa.Cp = g.C;
    wa.NTt = w.NTt; wa.kch = w.kch;
    wa.xp = x; wa.hd = sv.hd; wa.dA = dA;
    wa.partial = partial;
    wa.k_mul = k_mul_of(g);
    const long long witems = (long long)g.nd * U * w.nblk * w.kch;
    const long long wblocks = (blocks_for(witems, kSW) + kXcds - 1) / kXcds * kXcds;
    switch (U) {
    case 1: k_wgrad_step<1><<<wblocks, 64 * kSW, 0, st>>>(wa); break;
    case 2: k_wgrad_step<2><<<wblocks, 64 * kSW, 0, st>>>(wa); break;
    default: k_wgrad_step<4><<<wblocks, 64 * kSW, 0, st>>>(wa); break;
    }
    PLSTM_LAUNCH_CHECK();
    // db: the column of ones, unless the line blocks summed it already
    const long long nout = (long long)g.nd * G * (KK * (g.O + g.C) + 1);
    k_wgrad_step_reduce<<<blocks_for(nout, 256), 256, 0, st>>>(
        g.nd, g.O, g.C, Cp, KK, w.NTt, w.kch, partial, dwx, dwh, db_done ? nullptr : db);
    PLSTM_LAUNCH_CHECK();
    timing_end(2, st);
    if (dx && !dx_done) return step_dx(g, wx, dA, fragx, dx, st);
    return PLSTM_OK;
}

}  // namespace plstm

extern "C" int pyramid_lstm_set_step_split(int mode)
{
    if (mode < 0 || mode > 3) return PLSTM_EINVAL;
    plstm::g_step_split = mode;
    return PLSTM_OK;
}

extern "C" int pyramid_lstm_set_bf16_mfma(int on)
{
    if (on < 0 || on > 5) return PLSTM_EINVAL;
    plstm::g_step_bf16_mfma = on;
    return PLSTM_OK;
}

extern "C" int pyramid_lstm_set_wgrad_staged(int on)
{
    if (on != 0 && on != 1) return PLSTM_EINVAL;
    plstm::g_wgrad_staged = on;
    return PLSTM_OK;
}
