// Generic PyraMiD-LSTM path: any supported shape, any KP x KQ filter (K x K
// over a volume's planes, 1 x K along an image's lines), one launch per plane
// step.
//
// Forward (Section 2.3, Eq. (7)-(13)): for step t, every direction d with
// t < T_d updates all pixels of its plane t at once.  One thread owns one
// (direction, batch element, pixel, hidden unit) and produces the four gate
// pre-activations of that unit by direct KP x KQ loops over the input plane and
// the previous plane's h^d; the cell state lives in a per-direction volume.
// The six per-direction outputs are summed in the fixed order d = 0..5.
//
// Backward (the chain rule through Eq. (7)-(13), reverse plane order): for
// step t every thread owns one (d, n, pixel, unit j): it collects dL/dh^d from
// the upstream gradient and from the next plane's gate gradients (a transposed
// KP x KQ convolution with wh), forms dL/dc and the four gate gradients of unit j.
// Parameter gradients are then block-tiled reductions over all voxels
// (deterministic two-stage sums), and dL/dx a transposed KP x KQ convolution with
// wx summed over the six directions.
#include "common.h"
#include "sweep.h"
#include "timing.h"

namespace plstm {
namespace {

constexpr int kThreads = 256;

template <typename TS>
__global__ void __launch_bounds__(kThreads)
k_fwd_step(Geom g, int t, const TS *__restrict__ x, const TS *__restrict__ wx,
           const TS *__restrict__ wh, const TS *__restrict__ b, float *__restrict__ hd,
           float *__restrict__ cellbuf, float *__restrict__ gates)
{
    const int d = blockIdx.z / g.N, n = blockIdx.z % g.N, o = blockIdx.y;
    const DirGeom dg = g.dir[d];
    if (t >= dg.T) return;
    const int px = blockIdx.x * kThreads + threadIdx.x;
    if (px >= dg.P * dg.Q) return;
    const int p = px / dg.Q, q = px % dg.Q;
    const int s = dg.sign > 0 ? t : dg.T - 1 - t;
    const int sprev = s - dg.sign;
    const int C = g.C, O = g.O, G = 4 * O, KP = g.KP, KQ = g.KQ, KK = KP * KQ;
    const int radp = KP / 2, radq = KQ / 2;
    const long long nbase = (long long)n * g.V;
    const long long dbase = (long long)d * g.N * g.V;

    float acc[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[k] = Store<TS>::load(b, (long long)d * G + k * O + o);

    for (int ka = 0; ka < KP; ++ka) {
        const int pp = p + ka - radp;
        if (pp < 0 || pp >= dg.P) continue;
        for (int kb = 0; kb < KQ; ++kb) {
            const int qq = q + kb - radq;
            if (qq < 0 || qq >= dg.Q) continue;
            const long long vin = nbase + s * dg.ss + pp * dg.sp + qq * dg.sq;
            for (int c = 0; c < C; ++c) {
                const float xv = Store<TS>::load(x, vin * C + c);
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    acc[k] += xv * Store<TS>::load(
                        wx, (((long long)d * G + k * O + o) * C + c) * KK + ka * KQ + kb);
            }
            if (t > 0) {
                const long long vh = dbase + nbase + sprev * dg.ss + pp * dg.sp + qq * dg.sq;
                for (int j = 0; j < O; ++j) {
                    const float hv = hd[vh * O + j];
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        acc[k] += hv * Store<TS>::load(
                            wh, (((long long)d * G + k * O + o) * O + j) * KK + ka * KQ + kb);
                }
            }
        }
    }
    const float gi = sigmoidf_(acc[0]);
    const float gf = sigmoidf_(acc[1]);
    const float gg = tanhf(acc[2]);
    const float go = sigmoidf_(acc[3]);
    const long long v = dbase + nbase + s * dg.ss + p * dg.sp + q * dg.sq;
    float c = gg * gi;
    if (t > 0) c += cellbuf[(dbase + nbase + sprev * dg.ss + p * dg.sp + q * dg.sq) * O + o] * gf;
    cellbuf[v * O + o] = c;
    hd[v * O + o] = go * tanhf(c);
    if (gates) {
        gates[v * G + 0 * O + o] = gi;
        gates[v * G + 1 * O + o] = gf;
        gates[v * G + 2 * O + o] = gg;
        gates[v * G + 3 * O + o] = go;
    }
}

// h = sum_d h^d in the fixed order d = 0..5 (Eq. (13)).
template <typename TS>
__global__ void __launch_bounds__(kThreads)
k_sum_dirs(long long count, int nd, const float *__restrict__ hd, TS *__restrict__ h)
{
    const long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (i >= count) return;
    float acc = hd[i];
    for (int d = 1; d < nd; ++d) acc += hd[(long long)d * count + i];
    Store<TS>::store(h, i, acc);
}

// The same sum, four consecutive elements per thread (count a multiple of 4):
// every direction's 16-byte load is in flight before the first add, and the
// additions keep the order d = 0..nd-1, so the result is the scalar kernel's.
typedef float sf4 __attribute__((ext_vector_type(4)));
typedef unsigned short su4 __attribute__((ext_vector_type(4)));
template <typename TS>
__global__ void __launch_bounds__(kThreads)
k_sum_dirs4(long long count4, int nd, const float *__restrict__ hd, TS *__restrict__ h)
{
    const long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (i >= count4) return;
    const sf4 *src = (const sf4 *)hd;
    sf4 v[kDirs];
#pragma unroll
    for (int d = 0; d < kDirs; ++d)
        v[d] = d < nd ? __builtin_nontemporal_load(&src[(long long)d * count4 + i]) : sf4{0, 0, 0, 0};
    sf4 acc = v[0];
#pragma unroll
    for (int d = 1; d < kDirs; ++d)
        if (d < nd) acc += v[d];
    if constexpr (sizeof(TS) == 4) {
        ((sf4 *)h)[i] = acc;
    } else {
        ((su4 *)h)[i] = su4{f32_to_bf16(acc[0]), f32_to_bf16(acc[1]), f32_to_bf16(acc[2]),
                            f32_to_bf16(acc[3])};
    }
}

// Direction sum from bf16 h^d: 8 channels per thread, the directions added
// in fp32 in order, rounded to bf16 once.  Both direction sums read h^d once
// with non-temporal loads (it is not read again soon), about 15% faster than
// ordinary loads.
typedef unsigned su8v __attribute__((ext_vector_type(4)));
__global__ void __launch_bounds__(kThreads)
k_sum_dirs8_b16(long long count8, int nd, const uint16_t *__restrict__ hb, uint16_t *__restrict__ h)
{
    const long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (i >= count8) return;
    const su8v *src = (const su8v *)hb;
    su8v v[kDirs];
#pragma unroll
    for (int d = 0; d < kDirs; ++d)
        v[d] = d < nd ? __builtin_nontemporal_load(&src[(long long)d * count8 + i]) : su8v{0, 0, 0, 0};
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        float a = 0.0f;
#pragma unroll
        for (int d = 0; d < kDirs; ++d) {
            if (d >= nd) continue;
            const unsigned w = v[d][j >> 1];
            a += bf16_to_f32((uint16_t)((j & 1) ? (w >> 16) : (w & 0xffffu)));
        }
        acc[j] = a;
    }
    su8v out;
#pragma unroll
    for (int k = 0; k < 4; ++k)
        out[k] = (unsigned)f32_to_bf16(acc[2 * k]) | ((unsigned)f32_to_bf16(acc[2 * k + 1]) << 16);
    ((su8v *)h)[i] = out;
}

__global__ void __launch_bounds__(kThreads)
k_bwd_step(Geom g, int t, const float *__restrict__ wh, const float *__restrict__ gates,
           const float *__restrict__ cell, const float *__restrict__ dh,
           float *__restrict__ dA, float *__restrict__ gc)
{
    const int d = blockIdx.z / g.N, n = blockIdx.z % g.N, j = blockIdx.y;
    const DirGeom dg = g.dir[d];
    if (t >= dg.T) return;
    const int px = blockIdx.x * kThreads + threadIdx.x;
    if (px >= dg.P * dg.Q) return;
    const int p = px / dg.Q, q = px % dg.Q;
    const int s = dg.sign > 0 ? t : dg.T - 1 - t;
    const int snext = s + dg.sign, sprev = s - dg.sign;
    const int O = g.O, G = 4 * O, KP = g.KP, KQ = g.KQ, KK = KP * KQ;
    const int radp = KP / 2, radq = KQ / 2;
    const long long nbase = (long long)n * g.V;
    const long long dbase = (long long)d * g.N * g.V;
    const long long vloc = nbase + s * dg.ss + p * dg.sp + q * dg.sq;
    const long long v = dbase + vloc;
    const bool has_next = t + 1 < dg.T;

    float gh = dh[vloc * O + j];
    if (has_next) {
        // h_t[p][q][j] entered A_{t+1}[p - (ka-r)][q - (kb-r)] through tap (ka, kb).
        for (int ka = 0; ka < KP; ++ka) {
            const int pp = p - (ka - radp);
            if (pp < 0 || pp >= dg.P) continue;
            for (int kb = 0; kb < KQ; ++kb) {
                const int qq = q - (kb - radq);
                if (qq < 0 || qq >= dg.Q) continue;
                const long long vn = dbase + nbase + snext * dg.ss + pp * dg.sp + qq * dg.sq;
                for (int gn = 0; gn < G; ++gn)
                    gh += dA[vn * G + gn] *
                          wh[(((long long)d * G + gn) * O + j) * KK + ka * KQ + kb];
            }
        }
    }
    const float gi = gates[v * G + 0 * O + j];
    const float gf = gates[v * G + 1 * O + j];
    const float gg = gates[v * G + 2 * O + j];
    const float go = gates[v * G + 3 * O + j];
    const float c = cell[v * O + j];
    const float tc = tanhf(c);
    float gcv = gh * go * (1.0f - tc * tc);
    if (has_next) {
        const long long vn = dbase + nbase + snext * dg.ss + p * dg.sp + q * dg.sq;
        gcv += gc[vn * O + j] * gates[vn * G + 1 * O + j];
    }
    gc[v * O + j] = gcv;
    const float cprev =
        t > 0 ? cell[(dbase + nbase + sprev * dg.ss + p * dg.sp + q * dg.sq) * O + j] : 0.0f;
    dA[v * G + 0 * O + j] = gcv * gg * gi * (1.0f - gi);
    dA[v * G + 1 * O + j] = gcv * cprev * gf * (1.0f - gf);
    dA[v * G + 2 * O + j] = gcv * gi * (1.0f - gg * gg);
    dA[v * G + 3 * O + j] = gh * tc * go * (1.0f - go);
}

// Parameter-gradient partial sums.  For direction d the reduction runs over
// every voxel (n, t, p, q); with KK = KP * KQ taps, column k of the "im2col"
// row is
//   k < KK C          : x at tap (ka, kb) = divmod(k / C, KQ), channel k % C
//   KK C <= k < KK(C+O): h^d_{t-1} at tap, unit, recomputed as o * tanh(c) of
//                       the previous plane (0 for t = 0 or outside the plane)
//   k = KK (C+O)      : 1 (bias)
// Each block owns a 16 x 16 (gate-unit x column) tile and one chunk of voxels;
// partial[d][chunk][gn][k].
constexpr int kTile = 16;
constexpr int kVB = 64;   // voxels staged per LDS batch

__global__ void __launch_bounds__(kThreads)
k_wgrad_partial(Geom g, long long chunk_len, int nchunk, const float *__restrict__ x,
                const float *__restrict__ gates, const float *__restrict__ cell,
                const float *__restrict__ dA, float *__restrict__ partial)
{
    const int C = g.C, O = g.O, G = 4 * O, KQ = g.KQ, KK = g.KP * KQ;
    const int radp = g.KP / 2, radq = KQ / 2;
    const int KT = KK * (C + O) + 1;
    const int d = blockIdx.z / nchunk, chunk = blockIdx.z % nchunk;
    const int k0 = blockIdx.x * kTile, g0 = blockIdx.y * kTile;
    const DirGeom dg = g.dir[d];
    const long long PQ = (long long)dg.P * dg.Q;
    const long long total = (long long)g.N * g.V;   // voxels in sweep order (n, t, p, q)
    const long long v0 = (long long)chunk * chunk_len;
    const long long v1 = v0 + chunk_len < total ? v0 + chunk_len : total;
    const long long dbase = (long long)d * g.N * g.V;

    __shared__ float sA[kVB][kTile + 1];
    __shared__ float sIn[kVB][kTile + 1];
    const int tg = threadIdx.x / kTile, tk = threadIdx.x % kTile;
    float acc = 0.0f;
    for (long long vb = v0; vb < v1; vb += kVB) {
        for (int e = threadIdx.x; e < kVB * kTile; e += kThreads) {
            const int vi = e / kTile, col = e % kTile;
            const long long lin = vb + vi;
            float a = 0.0f, in = 0.0f;
            if (lin < v1) {
                const int n = (int)(lin / g.V);
                const long long rem = lin % g.V;
                const int t = (int)(rem / PQ);
                const int pix = (int)(rem % PQ);
                const int p = pix / dg.Q, q = pix % dg.Q;
                const int s = dg.sign > 0 ? t : dg.T - 1 - t;
                const long long nbase = (long long)n * g.V;
                const long long v = nbase + s * dg.ss + p * dg.sp + q * dg.sq;
                if (g0 + col < G) a = dA[(dbase + v) * G + g0 + col];
                const int k = k0 + col;
                if (k < KK * C) {
                    const int tap = k / C, c = k % C;
                    const int pp = p + tap / KQ - radp, qq = q + tap % KQ - radq;
                    if (pp >= 0 && pp < dg.P && qq >= 0 && qq < dg.Q)
                        in = x[(nbase + s * dg.ss + pp * dg.sp + qq * dg.sq) * C + c];
                } else if (k < KK * (C + O)) {
                    const int kk = k - KK * C;
                    const int tap = kk / O, j = kk % O;
                    const int pp = p + tap / KQ - radp, qq = q + tap % KQ - radq;
                    if (t > 0 && pp >= 0 && pp < dg.P && qq >= 0 && qq < dg.Q) {
                        const long long vp =
                            dbase + nbase + (s - dg.sign) * dg.ss + pp * dg.sp + qq * dg.sq;
                        in = gates[vp * G + 3 * O + j] * tanhf(cell[vp * O + j]);
                    }
                } else if (k == KT - 1) {
                    in = 1.0f;
                }
            }
            sA[vi][col] = a;
            sIn[vi][col] = in;
        }
        __syncthreads();
#pragma unroll 8
        for (int vi = 0; vi < kVB; ++vi) acc += sA[vi][tg] * sIn[vi][tk];
        __syncthreads();
    }
    const int gn = g0 + tg, k = k0 + tk;
    if (gn < G && k < KT)
        partial[(((long long)d * nchunk + chunk) * G + gn) * KT + k] = acc;
}

__global__ void __launch_bounds__(kThreads)
k_wgrad_reduce(Geom g, int nchunk, const float *__restrict__ partial, float *__restrict__ dwx,
               float *__restrict__ dwh, float *__restrict__ db)
{
    const int C = g.C, O = g.O, G = 4 * O, KK = g.KP * g.KQ;
    const int KT = KK * (C + O) + 1;
    const long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (i >= (long long)g.nd * G * KT) return;
    const int k = (int)(i % KT);
    const int gn = (int)((i / KT) % G);
    const int d = (int)(i / ((long long)KT * G));
    float acc = 0.0f;
    for (int ch = 0; ch < nchunk; ++ch)
        acc += partial[(((long long)d * nchunk + ch) * G + gn) * KT + k];
    if (k < KK * C) {
        const int tap = k / C, c = k % C;
        dwx[(((long long)d * G + gn) * C + c) * KK + tap] = acc;
    } else if (k < KK * (C + O)) {
        const int kk = k - KK * C;
        const int tap = kk / O, j = kk % O;
        dwh[(((long long)d * G + gn) * O + j) * KK + tap] = acc;
    } else {
        db[(long long)d * G + gn] = acc;
    }
}

// dL/dx[v][c] = sum_d sum_taps sum_gn dA^d[pixel - (tap - 1)][gn] * wx[d][gn][c][tap].
__global__ void __launch_bounds__(kThreads)
k_dx(Geom g, const float *__restrict__ wx, const float *__restrict__ dA, float *__restrict__ dx)
{
    const long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
    const int C = g.C, O = g.O, G = 4 * O, KP = g.KP, KQ = g.KQ, KK = KP * KQ;
    const int radp = KP / 2, radq = KQ / 2;
    if (i >= (long long)g.N * g.V * C) return;
    const int c = (int)(i % C);
    const long long vloc = i / C;
    const int n = (int)(vloc / g.V);
    const long long r = vloc % g.V;
    const int z = (int)(r / ((long long)g.H * g.W));
    const int y = (int)((r / g.W) % g.H);
    const int xw = (int)(r % g.W);
    const long long nbase = (long long)n * g.V;
    float acc = 0.0f;
    for (int d = 0; d < g.nd; ++d) {
        const DirGeom dg = g.dir[d];
        int s, p, q;
        switch (g.axis[d]) {
        case 0: s = z; p = y; q = xw; break;
        case 1: s = y; p = z; q = xw; break;
        default: s = xw; p = z; q = y; break;
        }
        const long long dbase = (long long)d * g.N * g.V;
        for (int ka = 0; ka < KP; ++ka) {
            const int pp = p - (ka - radp);
            if (pp < 0 || pp >= dg.P) continue;
            for (int kb = 0; kb < KQ; ++kb) {
                const int qq = q - (kb - radq);
                if (qq < 0 || qq >= dg.Q) continue;
                const long long v = dbase + nbase + s * dg.ss + pp * dg.sp + qq * dg.sq;
                const float *a = dA + v * G;
                const float *w = wx + ((long long)d * G * C + c) * KK + ka * KQ + kb;
                for (int gn = 0; gn < G; ++gn) acc += a[gn] * w[(long long)gn * C * KK];
            }
        }
    }
    dx[i] = acc;
}

inline int max_plane(const Geom &g) {
    int m = 0;
    for (int d = 0; d < g.nd; ++d) m = g.dir[d].P * g.dir[d].Q > m ? g.dir[d].P * g.dir[d].Q : m;
    return m;
}
inline int max_T(const Geom &g) {
    int m = 0;
    for (int d = 0; d < g.nd; ++d) m = g.dir[d].T > m ? g.dir[d].T : m;
    return m;
}

// Voxels per reduction chunk: at least 8192, and at most 4096 chunks so that
// the grid's z extent (6 x chunks) stays within HIP's limit.
inline long long wgrad_chunk_len(const Geom &g) {
    const long long nv = (long long)g.N * g.V;
    long long len = 8192;
    if ((nv + len - 1) / len > 4096) len = (nv + 4095) / 4096;
    return len;
}
inline int wgrad_chunks(const Geom &g) {
    const long long len = wgrad_chunk_len(g);
    return (int)(((long long)g.N * g.V + len - 1) / len);
}

}  // namespace

size_t generic_forward_ws(const Geom &g, bool training)
{
    Carve cv(nullptr);
    if (!training) {
        cv.take<float>(saved_state_count(g));   // h^d
        cv.take<float>(saved_state_count(g));   // c^d
    }
    return cv.off;
}

int generic_forward(const Geom &g, int dtype, const void *x, const void *wx, const void *wh,
                    const void *b, void *h, const Saved *sv, void *ws, hipStream_t st)
{
    Carve cv(ws);
    float *hd = sv ? sv->hd : cv.take<float>(saved_state_count(g));
    float *cellbuf = sv ? sv->cell : cv.take<float>(saved_state_count(g));
    float *gates = sv ? sv->gates : nullptr;
    const dim3 grid((max_plane(g) + kThreads - 1) / kThreads, g.O, g.nd * g.N);
    const int T = max_T(g);
    timing_begin("sweep_fwd_generic", st);
    for (int t = 0; t < T; ++t) {
        if (dtype == PLSTM_BF16)
            k_fwd_step<uint16_t><<<grid, kThreads, 0, st>>>(
                g, t, (const uint16_t *)x, (const uint16_t *)wx, (const uint16_t *)wh,
                (const uint16_t *)b, hd, cellbuf, gates);
        else
            k_fwd_step<float><<<grid, kThreads, 0, st>>>(
                g, t, (const float *)x, (const float *)wx, (const float *)wh,
                (const float *)b, hd, cellbuf, gates);
        PLSTM_LAUNCH_CHECK();
    }
    timing_end(T, st);
    return sum_dirs(g, dtype, hd, h, st);
}

namespace {
__global__ void __launch_bounds__(kThreads)
k_bf16_to_f32(long long n, const uint16_t *__restrict__ src, float *__restrict__ dst)
{
    const long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (i < n) dst[i] = bf16_to_f32(src[i]);
}
}  // namespace

int bf16_to_f32(const void *src, float *dst, long long n, hipStream_t st)
{
    if (n <= 0) return PLSTM_OK;
    k_bf16_to_f32<<<(unsigned)((n + kThreads - 1) / kThreads), kThreads, 0, st>>>(
        n, (const uint16_t *)src, dst);
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

int sum_dirs_bf16(const Geom &g, const uint16_t *hb, void *h, hipStream_t st)
{
    const long long count = (long long)g.N * g.V * g.O;
    if (count % 8 != 0) return PLSTM_EUNSUPPORTED;     // O is a multiple of 16 here
    const long long c8 = count / 8;
    timing_begin("sum_dirs", st);
    k_sum_dirs8_b16<<<(unsigned)((c8 + kThreads - 1) / kThreads), kThreads, 0, st>>>(
        c8, g.nd, hb, (uint16_t *)h);
    PLSTM_LAUNCH_CHECK();
    timing_end(1, st);
    return PLSTM_OK;
}

int sum_dirs(const Geom &g, int dtype, const float *hd, void *h, hipStream_t st)
{
    const long long count = (long long)g.N * g.V * g.O;
    const unsigned blocks = (unsigned)((count + kThreads - 1) / kThreads);
    timing_begin("sum_dirs", st);
    if (count % 4 == 0) {
        const long long c4 = count / 4;
        const unsigned b4 = (unsigned)((c4 + kThreads - 1) / kThreads);
        if (dtype == PLSTM_BF16)
            k_sum_dirs4<uint16_t><<<b4, kThreads, 0, st>>>(c4, g.nd, hd, (uint16_t *)h);
        else
            k_sum_dirs4<float><<<b4, kThreads, 0, st>>>(c4, g.nd, hd, (float *)h);
    } else if (dtype == PLSTM_BF16) {
        k_sum_dirs<uint16_t><<<blocks, kThreads, 0, st>>>(count, g.nd, hd, (uint16_t *)h);
    } else {
        k_sum_dirs<float><<<blocks, kThreads, 0, st>>>(count, g.nd, hd, (float *)h);
    }
    PLSTM_LAUNCH_CHECK();
    timing_end(1, st);
    return PLSTM_OK;
}

size_t generic_backward_ws(const Geom &g)
{
    Carve cv(nullptr);
    const int G = 4 * g.O, KT = g.KP * g.KQ * (g.C + g.O) + 1;
    cv.take<float>((size_t)g.nd * g.N * g.V * G);                       // dA
    cv.take<float>((size_t)g.nd * g.N * g.V * g.O);                     // dL/dc
    cv.take<float>((size_t)g.nd * wgrad_chunks(g) * G * KT);            // partials
    return cv.off;
}

int generic_backward(const Geom &g, const float *x, const float *wx, const float *wh,
                     const Saved &sv, const float *dh, float *dx, float *dwx, float *dwh,
                     float *db, void *ws, hipStream_t st)
{
    const float *gates = sv.gates, *cell = sv.cell;
    const int G = 4 * g.O, KT = g.KP * g.KQ * (g.C + g.O) + 1;
    Carve cv(ws);
    float *dA = cv.take<float>((size_t)g.nd * g.N * g.V * G);
    float *gc = cv.take<float>((size_t)g.nd * g.N * g.V * g.O);
    const int nchunk = wgrad_chunks(g);
    float *partial = cv.take<float>((size_t)g.nd * nchunk * G * KT);

    const dim3 grid((max_plane(g) + kThreads - 1) / kThreads, g.O, g.nd * g.N);
    timing_begin("sweep_bwd_generic", st);
    for (int t = max_T(g) - 1; t >= 0; --t) {
        k_bwd_step<<<grid, kThreads, 0, st>>>(g, t, wh, gates, cell, dh, dA, gc);
        PLSTM_LAUNCH_CHECK();
    }
    timing_end(max_T(g), st);
    timing_begin("wgrad_generic", st);
    const dim3 wg_grid((KT + kTile - 1) / kTile, (G + kTile - 1) / kTile, g.nd * nchunk);
    k_wgrad_partial<<<wg_grid, kThreads, 0, st>>>(g, wgrad_chunk_len(g), nchunk, x, gates, cell, dA, partial);
    PLSTM_LAUNCH_CHECK();
    const long long nout = (long long)g.nd * G * KT;
    k_wgrad_reduce<<<(unsigned)((nout + kThreads - 1) / kThreads), kThreads, 0, st>>>(
        g, nchunk, partial, dwx, dwh, db);
    PLSTM_LAUNCH_CHECK();
    timing_end(2, st);
    if (dx) return generic_dx(g, wx, dA, dx, st);
    return PLSTM_OK;
}

int generic_dx(const Geom &g, const float *wx, const float *dA, float *dx, hipStream_t st)
{
    const long long cnt = (long long)g.N * g.V * g.C;
    timing_begin("dx_generic", st);
    k_dx<<<(unsigned)((cnt + kThreads - 1) / kThreads), kThreads, 0, st>>>(g, wx, dA, dx);
    PLSTM_LAUNCH_CHECK();
    timing_end(1, st);
    return PLSTM_OK;
}

}  // namespace plstm
