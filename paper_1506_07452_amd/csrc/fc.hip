// Per-voxel fully connected layers (Section 2.3, "Fully-Connected Layer";
// Fig. 3): FC + tanh after every PyraMiD-LSTM layer, and the last FC layer
// followed by a per-voxel softmax, with the mean cross-entropy and its
// gradient for training.  Weight-gradient sums over voxels are deterministic
// two-stage reductions (fixed chunking, fixed order).
#include "common.h"

namespace plstm {
namespace {

constexpr int kThreads = 256;
constexpr int kTile = 16;
constexpr int kMB = 64;          // rows staged per LDS batch

// y[m][o] = tanh(b[o] + sum_i w[o][i] x[m][i]); one thread per (m, o).
template <typename TS>
__global__ void __launch_bounds__(kThreads)
k_fc_tanh(long long M, int Cin, int Cout, const TS *__restrict__ x, const TS *__restrict__ w,
          const TS *__restrict__ b, TS *__restrict__ y)
{
    const long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (i >= M * Cout) return;
    const int o = (int)(i % Cout);
    const long long m = i / Cout;
    float acc = Store<TS>::load(b, o);
    for (int c = 0; c < Cin; ++c)
        acc += Store<TS>::load(w, (long long)o * Cin + c) * Store<TS>::load(x, m * Cin + c);
    Store<TS>::store(y, i, tanhf(acc));
}

// Row-gradient g[m][o] for the two layer kinds: tanh FC (dy * (1 - y^2)) or
// the softmax head (precomputed dlogits).
struct RowGrad {
    const float *y;      // tanh output, or nullptr when g is given directly
    const float *g;      // dy (tanh) or dlogits (softmax)
    __device__ float at(long long idx) const {
        const float v = g[idx];
        if (!y) return v;
        const float yy = y[idx];
        return v * (1.0f - yy * yy);
    }
};

// dx[m][i] = sum_o grad[m][o] * w[o][i].
__global__ void __launch_bounds__(kThreads)
k_fc_dx(long long M, int Cin, int Cout, RowGrad rg, const float *__restrict__ w,
        float *__restrict__ dx)
{
    const long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (i >= M * Cin) return;
    const int c = (int)(i % Cin);
    const long long m = i / Cin;
    float acc = 0.0f;
    for (int o = 0; o < Cout; ++o) acc += rg.at(m * Cout + o) * w[(long long)o * Cin + c];
    dx[i] = acc;
}

// partial[chunk][o][k] = sum over rows m of the chunk of grad[m][o] * in[m][k],
// in[m][k] = x[m][k] for k < Cin and 1 (bias) for k = Cin.
__global__ void __launch_bounds__(kThreads)
k_fc_wgrad_partial(long long M, int Cin, int Cout, long long chunk_len, RowGrad rg,
                   const float *__restrict__ x, float *__restrict__ partial)
{
    const int KT = Cin + 1;
    const int chunk = blockIdx.z;
    const int k0 = blockIdx.x * kTile, o0 = blockIdx.y * kTile;
    const long long m0 = (long long)chunk * chunk_len;
    const long long m1 = m0 + chunk_len < M ? m0 + chunk_len : M;
    __shared__ float sG[kMB][kTile + 1];
    __shared__ float sX[kMB][kTile + 1];
    const int to = threadIdx.x / kTile, tk = threadIdx.x % kTile;
    float acc = 0.0f;
    for (long long mb = m0; mb < m1; mb += kMB) {
        for (int e = threadIdx.x; e < kMB * kTile; e += kThreads) {
            const int r = e / kTile, col = e % kTile;
            const long long m = mb + r;
            float gv = 0.0f, xv = 0.0f;
            if (m < m1) {
                if (o0 + col < Cout) gv = rg.at(m * Cout + o0 + col);
                const int k = k0 + col;
                if (k < Cin) xv = x[m * Cin + k];
                else if (k == Cin) xv = 1.0f;
            }
            sG[r][col] = gv;
            sX[r][col] = xv;
        }
        __syncthreads();
#pragma unroll 8
        for (int r = 0; r < kMB; ++r) acc += sG[r][to] * sX[r][tk];
        __syncthreads();
    }
    const int o = o0 + to, k = k0 + tk;
    if (o < Cout && k < KT) partial[((long long)chunk * Cout + o) * KT + k] = acc;
}

__global__ void __launch_bounds__(kThreads)
k_fc_wgrad_reduce(int Cin, int Cout, int nchunk, const float *__restrict__ partial,
                  float *__restrict__ dw, float *__restrict__ db)
{
    const int KT = Cin + 1;
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= Cout * KT) return;
    float acc = 0.0f;
    for (int ch = 0; ch < nchunk; ++ch) acc += partial[(long long)ch * Cout * KT + i];
    const int o = i / KT, k = i % KT;
    if (k < Cin) dw[(long long)o * Cin + k] = acc;
    else db[o] = acc;
}

// Softmax head: p = softmax(w x + b) per row; with labels also the per-row
// loss -log p[label] (summed per block into lossp[block]) and
// dlogits = (p - onehot) / M.
constexpr int kMaxK = 16;

template <typename TS>
__global__ void __launch_bounds__(kThreads)
k_softmax(long long M, int Cin, int K, const TS *__restrict__ x, const TS *__restrict__ w,
          const TS *__restrict__ b, const int32_t *__restrict__ labels, float *__restrict__ p,
          float *__restrict__ dlogits, float *__restrict__ lossp)
{
    const long long m = (long long)blockIdx.x * kThreads + threadIdx.x;
    float l = 0.0f;
    if (m < M) {
        float z[kMaxK];
        float mx = -INFINITY;
        for (int k = 0; k < K; ++k) {
            float acc = Store<TS>::load(b, k);
            for (int c = 0; c < Cin; ++c)
                acc += Store<TS>::load(w, (long long)k * Cin + c) * Store<TS>::load(x, m * Cin + c);
            z[k] = acc;
            mx = fmaxf(mx, acc);
        }
        float sum = 0.0f;
        for (int k = 0; k < K; ++k) {
            z[k] = __expf(z[k] - mx);
            sum += z[k];
        }
        const float inv = 1.0f / sum;
        for (int k = 0; k < K; ++k) p[m * K + k] = z[k] * inv;
        if (labels) {
            // An out-of-range label poisons the loss with NaN instead of
            // reading outside the row.
            const int lab = labels[m];
            const bool ok = lab >= 0 && lab < K;
            l = ok ? -logf(z[lab] * inv) : NAN;
            for (int k = 0; k < K; ++k)
                dlogits[m * K + k] = ok ? (z[k] * inv - (k == lab ? 1.0f : 0.0f)) / (float)M : NAN;
        }
    }
    if (labels) {
        __shared__ float red[kThreads];
        red[threadIdx.x] = l;
        __syncthreads();
        for (int off = kThreads / 2; off > 0; off >>= 1) {
            if (threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
            __syncthreads();
        }
        if (threadIdx.x == 0) lossp[blockIdx.x] = red[0];
    }
}

__global__ void __launch_bounds__(kThreads)
k_loss_reduce(long long M, int nblk, const float *__restrict__ lossp, float *__restrict__ loss)
{
    __shared__ float red[kThreads];
    float acc = 0.0f;
    for (int i = threadIdx.x; i < nblk; i += kThreads) acc += lossp[i];
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int off = kThreads / 2; off > 0; off >>= 1) {
        if (threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0) *loss = red[0] / (float)M;
}

// ---- one thread per row, rows staged through LDS ------------------------------
// A block handles kRB consecutive rows: their inputs (contiguous in memory) are
// copied into LDS with coalesced loads, each thread computes its row from LDS
// against the weights (a chunk of up to kOC outputs, also in LDS), and the
// block's outputs leave through LDS with coalesced stores.
constexpr int kRB = 128;          // rows (= threads) per block
constexpr int kOC = 32;           // outputs per thread
constexpr int kRowsMaxIn = 128;   // widest row staged this way

inline bool rows_ok(int in_width) { return in_width <= kRowsMaxIn; }
inline size_t rows_lds(int in_w, int out_w, int wcount) {
    return ((size_t)kRB * (in_w + 1) + (size_t)kRB * (out_w + 1) + wcount) * sizeof(float);
}

// Coalesced copy of rows [m0, m0 + nr) x cols [c0, c0 + nc) of a row-major
// [M][ld] matrix into an LDS tile with row pitch nc + 1 (bank-conflict free).
template <typename TS>
__device__ inline void rows_to_lds(const TS *src, long long m0, int nr, int ld, int c0, int nc,
                                   float *tile)
{
    const int n = nr * nc;
    for (int e = threadIdx.x; e < n; e += kRB) {
        const int r = e / nc, c = e - (e / nc) * nc;
        tile[r * (nc + 1) + c] = Store<TS>::load(src, (m0 + r) * ld + c0 + c);
    }
}

template <typename TS>
__device__ inline void lds_to_rows(const float *tile, long long m0, int nr, int ld, int c0, int nc,
                                   TS *dst)
{
    const int n = nr * nc;
    for (int e = threadIdx.x; e < n; e += kRB) {
        const int r = e / nc, c = e - (e / nc) * nc;
        Store<TS>::store(dst, (m0 + r) * ld + c0 + c, tile[r * (nc + 1) + c]);
    }
}

template <typename TS>
__global__ void __launch_bounds__(kRB)
k_fc_tanh_rows(long long M, int Cin, int Cout, const TS *__restrict__ x, const TS *__restrict__ w,
               const TS *__restrict__ b, TS *__restrict__ y)
{
    extern __shared__ float lds[];
    const int o0 = blockIdx.y * kOC;
    const int oc = min(kOC, Cout - o0);
    const long long m0 = (long long)blockIdx.x * kRB;
    const int nr = (int)min((long long)kRB, M - m0);
    float *xs = lds;                               // [kRB][Cin + 1]
    float *ys = xs + kRB * (Cin + 1);              // [kRB][oc + 1]
    float *sw = ys + kRB * (kOC + 1);              // [oc][Cin], then bias [oc]
    float *sb = sw + oc * Cin;
    for (int e = threadIdx.x; e < oc * Cin; e += kRB)
        sw[e] = Store<TS>::load(w, (long long)o0 * Cin + e);
    for (int e = threadIdx.x; e < oc; e += kRB) sb[e] = Store<TS>::load(b, o0 + e);
    rows_to_lds<TS>(x, m0, nr, Cin, 0, Cin, xs);
    __syncthreads();
    const int r = threadIdx.x;
    if (r < nr) {
        float acc[kOC];
#pragma unroll
        for (int j = 0; j < kOC; ++j) acc[j] = j < oc ? sb[j] : 0.0f;
        const float *xr = xs + r * (Cin + 1);
        for (int c = 0; c < Cin; ++c) {
            const float xv = xr[c];
#pragma unroll
            for (int j = 0; j < kOC; ++j)
                if (j < oc) acc[j] += xv * sw[j * Cin + c];
        }
#pragma unroll
        for (int j = 0; j < kOC; ++j)
            if (j < oc) ys[r * (oc + 1) + j] = tanhf(acc[j]);
    }
    __syncthreads();
    lds_to_rows<TS>(ys, m0, nr, Cout, o0, oc, y);
}

// dx[m][i0 + i] = sum_o grad[m][o] w[o][i0 + i] for a chunk of kOC inputs.
__global__ void __launch_bounds__(kRB)
k_fc_dx_rows(long long M, int Cin, int Cout, RowGrad rg, const float *__restrict__ w,
             float *__restrict__ dx)
{
    extern __shared__ float lds[];
    const int i0 = blockIdx.y * kOC;
    const int ic = min(kOC, Cin - i0);
    const long long m0 = (long long)blockIdx.x * kRB;
    const int nr = (int)min((long long)kRB, M - m0);
    float *gs = lds;                               // [kRB][Cout + 1] row gradients
    float *os = gs + kRB * (Cout + 1);             // [kRB][ic + 1]
    float *sw = os + kRB * (kOC + 1);              // [Cout][ic]
    for (int e = threadIdx.x; e < Cout * ic; e += kRB) {
        const int o = e / ic, i = e % ic;
        sw[e] = w[(long long)o * Cin + i0 + i];
    }
    for (int e = threadIdx.x; e < nr * Cout; e += kRB) {
        const int r = e / Cout, o = e - (e / Cout) * Cout;
        gs[r * (Cout + 1) + o] = rg.at((m0 + r) * Cout + o);
    }
    __syncthreads();
    const int r = threadIdx.x;
    if (r < nr) {
        float acc[kOC];
#pragma unroll
        for (int j = 0; j < kOC; ++j) acc[j] = 0.0f;
        const float *gr = gs + r * (Cout + 1);
        for (int o = 0; o < Cout; ++o) {
            const float gv = gr[o];
#pragma unroll
            for (int j = 0; j < kOC; ++j)
                if (j < ic) acc[j] += gv * sw[o * ic + j];
        }
#pragma unroll
        for (int j = 0; j < kOC; ++j)
            if (j < ic) os[r * (ic + 1) + j] = acc[j];
    }
    __syncthreads();
    lds_to_rows<float>(os, m0, nr, Cin, i0, ic, dx);
}

// Softmax head, one thread per row: logits in registers (K <= 16), the
// label's probability picked by comparison (no dynamically indexed arrays).
template <typename TS>
__global__ void __launch_bounds__(kRB)
k_softmax_rows(long long M, int Cin, int K, const TS *__restrict__ x, const TS *__restrict__ w,
               const TS *__restrict__ b, const int32_t *__restrict__ labels,
               float *__restrict__ p, float *__restrict__ dlogits, float *__restrict__ lossp)
{
    extern __shared__ float lds[];
    const long long m0 = (long long)blockIdx.x * kRB;
    const int nr = (int)min((long long)kRB, M - m0);
    float *xs = lds;                               // [kRB][Cin + 1]
    float *ps = xs + kRB * (Cin + 1);              // [kRB][K + 1] probabilities
    float *sw = ps + kRB * (16 + 1);               // [K][Cin], then bias [K]
    float *sb = sw + K * Cin;
    for (int e = threadIdx.x; e < K * Cin; e += kRB) sw[e] = Store<TS>::load(w, e);
    for (int e = threadIdx.x; e < K; e += kRB) sb[e] = Store<TS>::load(b, e);
    rows_to_lds<TS>(x, m0, nr, Cin, 0, Cin, xs);
    __syncthreads();
    const int r = threadIdx.x;
    float l = 0.0f;
    if (r < nr) {
        float z[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) z[k] = k < K ? sb[k] : 0.0f;
        const float *xr = xs + r * (Cin + 1);
        for (int c = 0; c < Cin; ++c) {
            const float xv = xr[c];
#pragma unroll
            for (int k = 0; k < 16; ++k)
                if (k < K) z[k] += xv * sw[k * Cin + c];
        }
        float mx = -INFINITY;
#pragma unroll
        for (int k = 0; k < 16; ++k)
            if (k < K) mx = fmaxf(mx, z[k]);
        float sum = 0.0f;
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            z[k] = k < K ? __expf(z[k] - mx) : 0.0f;
            sum += z[k];
        }
        const float inv = 1.0f / sum;
#pragma unroll
        for (int k = 0; k < 16; ++k)
            if (k < K) ps[r * (K + 1) + k] = z[k] * inv;
        if (labels) {
            // An out-of-range label poisons the loss with NaN.
            const int lab = labels[m0 + r];
            const bool ok = lab >= 0 && lab < K;
            float pl = 0.0f;
#pragma unroll
            for (int k = 0; k < 16; ++k)
                if (k == lab) pl = z[k] * inv;
            l = ok ? -logf(pl) : NAN;
        }
    }
    __syncthreads();
    lds_to_rows<float>(ps, m0, nr, K, 0, K, p);
    if (labels) {
        // dlogits = (p - onehot(label)) / M, written coalesced from the tile
        const int n = nr * K;
        for (int e = threadIdx.x; e < n; e += kRB) {
            const int rr = e / K, k = e - (e / K) * K;
            const int lab = labels[m0 + rr];
            const bool ok = lab >= 0 && lab < K;
            dlogits[(m0 + rr) * K + k] =
                ok ? (ps[rr * (K + 1) + k] - (k == lab ? 1.0f : 0.0f)) / (float)M : NAN;
        }
        __shared__ float red[kRB];
        red[threadIdx.x] = l;
        __syncthreads();
        for (int off = kRB / 2; off > 0; off >>= 1) {
            if (threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
            __syncthreads();
        }
        if (threadIdx.x == 0) lossp[blockIdx.x] = red[0];
    }
}

inline long long fc_chunk_len(long long M) {
    long long len = 8192;
    if ((M + len - 1) / len > 4096) len = (M + 4095) / 4096;
    return len;
}
inline int fc_chunks(long long M) {
    const long long len = fc_chunk_len(M);
    return (int)((M + len - 1) / len);
}

inline unsigned blocks_for(long long n) { return (unsigned)((n + kThreads - 1) / kThreads); }

int fc_dx(long long M, int Cin, int Cout, RowGrad rg, const float *w, float *dx, hipStream_t st)
{
    if (rows_ok(Cout)) {
        const dim3 grid((unsigned)((M + kRB - 1) / kRB), (Cin + kOC - 1) / kOC);
        k_fc_dx_rows<<<grid, kRB, rows_lds(Cout, kOC, Cout * kOC), st>>>(M, Cin, Cout, rg, w,
                                                                           dx);
    } else {
        k_fc_dx<<<blocks_for(M * Cin), kThreads, 0, st>>>(M, Cin, Cout, rg, w, dx);
    }
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

int fc_wgrad(long long M, int Cin, int Cout, RowGrad rg, const float *x, float *dw, float *db,
             float *partial, hipStream_t st)
{
    const int nchunk = fc_chunks(M);
    const dim3 grid((Cin + 1 + kTile - 1) / kTile, (Cout + kTile - 1) / kTile, nchunk);
    k_fc_wgrad_partial<<<grid, kThreads, 0, st>>>(M, Cin, Cout, fc_chunk_len(M), rg, x, partial);
    PLSTM_LAUNCH_CHECK();
    k_fc_wgrad_reduce<<<blocks_for((long long)Cout * (Cin + 1)), kThreads, 0, st>>>(
        Cin, Cout, nchunk, partial, dw, db);
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

}  // namespace

size_t fc_ws(long long M, int Cin, int Cout)
{
    Carve cv(nullptr);
    cv.take<float>((size_t)fc_chunks(M) * Cout * (Cin + 1));   // weight-gradient partials
    cv.take<float>((size_t)M * (Cout < kMaxK ? Cout : kMaxK)); // dlogits (softmax head)
    cv.take<float>((size_t)(M + kRB - 1) / kRB);               // per-block losses
    return cv.off;
}

int fc_tanh_forward(long long M, int Cin, int Cout, int dtype, const void *x, const void *w,
                    const void *b, void *y, hipStream_t st)
{
    if (rows_ok(Cin)) {
        const dim3 grid((unsigned)((M + kRB - 1) / kRB), (Cout + kOC - 1) / kOC);
        const size_t lds = rows_lds(Cin, kOC, kOC * (Cin + 1));
        if (dtype == PLSTM_BF16)
            k_fc_tanh_rows<uint16_t><<<grid, kRB, lds, st>>>(
                M, Cin, Cout, (const uint16_t *)x, (const uint16_t *)w, (const uint16_t *)b,
                (uint16_t *)y);
        else
            k_fc_tanh_rows<float><<<grid, kRB, lds, st>>>(
                M, Cin, Cout, (const float *)x, (const float *)w, (const float *)b, (float *)y);
        PLSTM_LAUNCH_CHECK();
        return PLSTM_OK;
    }
    const unsigned nb = blocks_for(M * Cout);
    if (dtype == PLSTM_BF16)
        k_fc_tanh<uint16_t><<<nb, kThreads, 0, st>>>(M, Cin, Cout, (const uint16_t *)x,
                                                      (const uint16_t *)w, (const uint16_t *)b,
                                                      (uint16_t *)y);
    else
        k_fc_tanh<float><<<nb, kThreads, 0, st>>>(M, Cin, Cout, (const float *)x,
                                                   (const float *)w, (const float *)b,
                                                   (float *)y);
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

int fc_tanh_backward(long long M, int Cin, int Cout, const float *x, const float *w,
                     const float *y, const float *dy, float *dx, float *dw, float *db,
                     void *ws, hipStream_t st)
{
    Carve cv(ws);
    float *partial = cv.take<float>((size_t)fc_chunks(M) * Cout * (Cin + 1));
    const RowGrad rg{y, dy};
    if (dx) {
        const int rc = fc_dx(M, Cin, Cout, rg, w, dx, st);
        if (rc != PLSTM_OK) return rc;
    }
    return fc_wgrad(M, Cin, Cout, rg, x, dw, db, partial, st);
}

int softmax_ce(long long M, int Cin, int K, int dtype, const void *x, const void *w,
               const void *b, const int32_t *labels, float *p, float *loss, float *dx,
               float *dw, float *db, void *ws, hipStream_t st)
{
    Carve cv(ws);
    float *partial = cv.take<float>((size_t)fc_chunks(M) * K * (Cin + 1));
    float *dlogits = cv.take<float>((size_t)M * K);
    float *lossp = cv.take<float>((size_t)(M + kRB - 1) / kRB);
    unsigned nb = blocks_for(M);
    if (rows_ok(Cin)) {
        nb = (unsigned)((M + kRB - 1) / kRB);
        const size_t lds = rows_lds(Cin, 16, K * (Cin + 1));
        if (dtype == PLSTM_BF16)
            k_softmax_rows<uint16_t><<<nb, kRB, lds, st>>>(
                M, Cin, K, (const uint16_t *)x, (const uint16_t *)w, (const uint16_t *)b, labels,
                p, dlogits, lossp);
        else
            k_softmax_rows<float><<<nb, kRB, lds, st>>>(
                M, Cin, K, (const float *)x, (const float *)w, (const float *)b, labels, p,
                dlogits, lossp);
    } else if (dtype == PLSTM_BF16) {
        k_softmax<uint16_t><<<nb, kThreads, 0, st>>>(M, Cin, K, (const uint16_t *)x,
                                                      (const uint16_t *)w, (const uint16_t *)b,
                                                      labels, p, dlogits, lossp);
    } else {
        k_softmax<float><<<nb, kThreads, 0, st>>>(M, Cin, K, (const float *)x, (const float *)w,
                                                   (const float *)b, labels, p, dlogits, lossp);
    }
    PLSTM_LAUNCH_CHECK();
    if (!labels) return PLSTM_OK;
    k_loss_reduce<<<1, kThreads, 0, st>>>(M, (int)nb, lossp, loss);
    PLSTM_LAUNCH_CHECK();
    if (!dw) return PLSTM_OK;
    const RowGrad rg{nullptr, dlogits};
    if (dx) {
        const int rc = fc_dx(M, Cin, K, rg, (const float *)w, dx, st);
        if (rc != PLSTM_OK) return rc;
    }
    return fc_wgrad(M, Cin, K, rg, (const float *)x, dw, db, partial, st);
}

}  // namespace plstm
