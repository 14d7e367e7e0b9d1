// Per-voxel fully connected layers (Section 2.3, "Fully-Connected Layer";
// Fig. 3): FC + tanh after every PyraMiD-LSTM layer, and the last FC layer
// followed by a per-voxel softmax, with the mean cross-entropy and its
// gradient for training.  Weight-gradient sums over voxels are deterministic
// two-stage reductions (fixed chunking, fixed order).
#include <type_traits>
#include "common.h"
#include "timing.h"

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

// SQ: the squared error of Eq. (14) against the one-hot label, summed over
// the classes, instead of the cross-entropy; its logit gradient is
// 2/M p_j ((p_j - y_j) - sum_k p_k (p_k - y_k)).
template <typename TS, bool SQ>
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
            if (SQ) {
                float e = 0.0f, sd = 0.0f;
                for (int k = 0; k < K; ++k) {
                    const float pk = z[k] * inv, dk = pk - (k == lab ? 1.0f : 0.0f);
                    e += dk * dk;
                    sd += pk * dk;
                }
                l = ok ? e : NAN;
                for (int k = 0; k < K; ++k) {
                    const float pk = z[k] * inv, dk = pk - (k == lab ? 1.0f : 0.0f);
                    dlogits[m * K + k] = ok ? 2.0f * pk * (dk - sd) / (float)M : NAN;
                }
            } else {
                l = ok ? -logf(z[lab] * inv) : NAN;
                for (int k = 0; k < K; ++k)
                    dlogits[m * K + k] =
                        ok ? (z[k] * inv - (k == lab ? 1.0f : 0.0f)) / (float)M : NAN;
            }
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
template <typename TS, bool SQ>
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
            if (SQ) {
                // squared error; sum_k p_k (p_k - y_k) kept in the row's pad slot
                float e = 0.0f, sd = 0.0f;
#pragma unroll
                for (int k = 0; k < 16; ++k) {
                    if (k < K) {
                        const float pk = z[k] * inv, dk = pk - (k == lab ? 1.0f : 0.0f);
                        e += dk * dk;
                        sd += pk * dk;
                    }
                }
                l = ok ? e : NAN;
                ps[r * (K + 1) + K] = sd;
            } else {
                float pl = 0.0f;
#pragma unroll
                for (int k = 0; k < 16; ++k)
                    if (k == lab) pl = z[k] * inv;
                l = ok ? -logf(pl) : NAN;
            }
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
            const float pk = ps[rr * (K + 1) + k], dk = pk - (k == lab ? 1.0f : 0.0f);
            const float g = SQ ? 2.0f * pk * (dk - ps[rr * (K + 1) + K]) : dk;
            dlogits[(m0 + rr) * K + k] = ok ? g / (float)M : NAN;
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

// ---- fused head: FC + tanh, linear + softmax, cross-entropy, backward --------
// Every row is read once and only p and dx are written per row.  A wave
// takes 16 rows at a time and runs the whole chain as MFMA contractions
// whose outputs feed the next one in registers (v_mfma_f32_16x16x4f32: lane
// l gives A[l%16][k], B[k][l%16] and holds D[4(l/16) + i][l%16]; with rows on
// N, lane (q = l/16, col = l%16) holds units 4q..4q+3 of row col, which is
// exactly the B operand of the next contraction when its K index for lane
// group q and k-step i is unit 4q + i):
//   Z^T = W1 X^T + b1,  y = tanh z,  L^T = W2 Y^T + b2,  p = softmax over the
//   lane groups,  dl = (p - onehot) / M,  dY^T = W2^T dl^T,  dz = dy (1 - y^2),
//   dX^T = W1^T dz^T.
// The weight gradients sum over rows (K = rows), so dz, dl, x and y of the 16
// rows are transposed through a per-wave LDS tile; dW1 = dz^T x and
// dW2 = dl^T y accumulate in VGPRs over all rows of the wave, the bias
// gradients as per-lane sums.  Workgroup partials are summed in a fixed
// order (deterministic).
constexpr int kHW = 4;              // waves per workgroup of the fused head
constexpr int kHT = 64 * kHW;

// tanh(a) = 1 - 2 / (e^{2a} + 1), branch-free (saturates to +-1).
__device__ inline float tanh_fast(float a)
{
    return 1.0f - 2.0f * __builtin_amdgcn_rcpf(__expf(2.0f * a) + 1.0f);
}

template <int CIN, int F>
struct HeadCfg {
    static constexpr int CT = CIN / 16, FT = F / 16;
    static constexpr int XP = CIN + 4, YP = F + 4, LP = 20;   // LDS row pitches (floats)
    static constexpr int per_wave = 16 * (XP + 2 * YP + LP);
    static constexpr int red = F * (CIN + 1) + 16 * (F + 1) + 1;
    static constexpr size_t bytes = (size_t)(kHW * per_wave + red) * sizeof(float);
};

template <int CIN, int F>
__global__ void __launch_bounds__(kHT)
k_head_train(long long M, int K, const float *__restrict__ x, const float *__restrict__ w1,
             const float *__restrict__ b1, const float *__restrict__ w2,
             const float *__restrict__ b2, const int32_t *__restrict__ labels,
             float *__restrict__ p, float *__restrict__ dx, float *__restrict__ partial)
{
    typedef float f4 __attribute__((ext_vector_type(4)));
    using HC = HeadCfg<CIN, F>;
    static_assert(CIN % 16 == 0 && F % 16 == 0, "tile multiples");
    constexpr int CT = HC::CT, FT = HC::FT;
    extern __shared__ float lds[];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int q = lane >> 4, col = lane & 15;
    float *xs = lds + wave * HC::per_wave;   // [16][XP]  x
    float *ys = xs + 16 * HC::XP;            // [16][YP]  y
    float *zs = ys + 16 * HC::YP;            // [16][YP]  dz
    float *ls = zs + 16 * HC::YP;            // [16][LP]  dl (zero beyond K)
    float *R = lds + kHW * HC::per_wave;     // workgroup reduction

    // ---- weights as MFMA A fragments, for the whole kernel ---------------
    float a1[FT][CT][4];   // W1[f = 16mt + col][c = 16kt + 4q + i]
    float a2[FT][4];       // W2[k = col][f = 16mt + 4q + i]
    float a3[FT][4];       // W2[k = 4q + i][f = 16mt + col]
    float a4[CT][FT][4];   // W1[f = 16mt + 4q + i][c = 16ct + col]
    f4 bias1[FT], bias2;
#pragma unroll
    for (int mt = 0; mt < FT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int kt = 0; kt < CT; ++kt) {
                a1[mt][kt][i] = w1[(16 * mt + col) * CIN + 16 * kt + 4 * q + i];
                a4[kt][mt][i] = w1[(16 * mt + 4 * q + i) * CIN + 16 * kt + col];
            }
            a2[mt][i] = col < K ? w2[col * F + 16 * mt + 4 * q + i] : 0.0f;
            a3[mt][i] = 4 * q + i < K ? w2[(4 * q + i) * F + 16 * mt + col] : 0.0f;
            bias1[mt][i] = b1[16 * mt + 4 * q + i];
        }
#pragma unroll
    for (int i = 0; i < 4; ++i) bias2[i] = 4 * q + i < K ? b2[4 * q + i] : 0.0f;

    f4 g1[FT][CT], g2[FT], gb1[FT], gb2 = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int mt = 0; mt < FT; ++mt) {
        g2[mt] = gb1[mt] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) g1[mt][ct] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    float lacc = 0.0f;
    const float inv_m = 1.0f / (float)M;
    const long long nsub = (M + 15) / 16;
    const long long gw = (long long)blockIdx.x * kHW + wave, nw = (long long)gridDim.x * kHW;
    // the next 16 rows and labels are loaded while these compute
    f4 xn[CT];
    int labn;
    auto load = [&](long long st) {
        const long long row = st * 16 + col;
        const bool v = st < nsub && row < M;
#pragma unroll
        for (int kt = 0; kt < CT; ++kt) xn[kt] = *(const f4 *)&x[(v ? row : 0) * CIN + 16 * kt + 4 * q];
        labn = labels[v ? row : 0];
    };
    load(gw);
    for (long long st = gw; st < nsub; st += nw) {
        const long long row = st * 16 + col;
        const bool valid = row < M;
        f4 xv[CT];
#pragma unroll
        for (int kt = 0; kt < CT; ++kt) xv[kt] = valid ? xn[kt] : f4{0.0f, 0.0f, 0.0f, 0.0f};
        const int lab = labn;
        load(st + nw);
        // ---- forward: y = tanh(W1 x + b1), logits = W2 y + b2 ------------
        f4 yv[FT];
#pragma unroll
        for (int mt = 0; mt < FT; ++mt) {
            f4 acc = bias1[mt];
#pragma unroll
            for (int kt = 0; kt < CT; ++kt)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[mt][kt][i], xv[kt][i], acc, 0,
                                                               0, 0);
#pragma unroll
            for (int i = 0; i < 4; ++i) yv[mt][i] = tanh_fast(acc[i]);
        }
        f4 lg = bias2;
#pragma unroll
        for (int mt = 0; mt < FT; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                lg = __builtin_amdgcn_mfma_f32_16x16x4f32(a2[mt][i], yv[mt][i], lg, 0, 0, 0);
        // ---- softmax over classes 4q + i, spread over the four lane groups
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (4 * q + i < K) mx = fmaxf(mx, lg[i]);
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        f4 pv;
        float sum = 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            pv[i] = 4 * q + i < K ? __expf(lg[i] - mx) : 0.0f;
            sum += pv[i];
        }
        sum += __shfl_xor(sum, 16);
        sum += __shfl_xor(sum, 32);
        const float inv = 1.0f / sum;
        pv *= inv;
        const bool ok = lab >= 0 && lab < K;     // an out-of-range label poisons with NaN
        f4 dl;
        float pl = 1.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int k = 4 * q + i;
            if (k == lab) pl = pv[i];
            const float g = ok ? (pv[i] - (k == lab ? 1.0f : 0.0f)) * inv_m : NAN;
            dl[i] = (valid && k < K) ? g : 0.0f;
        }
        if (valid) {
            if ((K & 3) == 0) {
                if (4 * q < K) *(f4 *)&p[row * K + 4 * q] = pv;
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (4 * q + i < K) p[row * K + 4 * q + i] = pv[i];
            }
            // the lane holding the label's class adds -log p; a bad label adds NaN once
            if (ok ? (lab >> 2) == q : q == 0) lacc += ok ? -logf(pl) : NAN;
        }
        // ---- backward: dz = (W2^T dl) (1 - y^2), dx = W1^T dz -------------
        f4 dz[FT];
#pragma unroll
        for (int mt = 0; mt < FT; ++mt) {
            f4 acc = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int i = 0; i < 4; ++i)
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a3[mt][i], dl[i], acc, 0, 0, 0);
#pragma unroll
            for (int i = 0; i < 4; ++i) dz[mt][i] = acc[i] * (1.0f - yv[mt][i] * yv[mt][i]);
            gb1[mt] += dz[mt];
        }
        gb2 += dl;
        if (dx) {
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                f4 acc = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int mt = 0; mt < FT; ++mt)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[ct][mt][i], dz[mt][i], acc,
                                                                   0, 0, 0);
                if (valid) *(f4 *)&dx[row * CIN + 16 * ct + 4 * q] = acc;
            }
        }
        // ---- weight gradients over these 16 rows (K = rows) ----------------
#pragma unroll
        for (int kt = 0; kt < CT; ++kt) *(f4 *)&xs[col * HC::XP + 16 * kt + 4 * q] = xv[kt];
#pragma unroll
        for (int mt = 0; mt < FT; ++mt) {
            *(f4 *)&ys[col * HC::YP + 16 * mt + 4 * q] = yv[mt];
            *(f4 *)&zs[col * HC::YP + 16 * mt + 4 * q] = dz[mt];
        }
        *(f4 *)&ls[col * HC::LP + 4 * q] = dl;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int r = 4 * ks + q;
            const float al = ls[r * HC::LP + col];
#pragma unroll
            for (int mt = 0; mt < FT; ++mt) {
                const float az = zs[r * HC::YP + 16 * mt + col];
                const float by = ys[r * HC::YP + 16 * mt + col];
#pragma unroll
                for (int ct = 0; ct < CT; ++ct)
                    g1[mt][ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                        az, xs[r * HC::XP + 16 * ct + col], g1[mt][ct], 0, 0, 0);
                g2[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(al, by, g2[mt], 0, 0, 0);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    // ---- bias sums over the 16 row lanes of each lane group, loss over the wave
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
#pragma unroll
        for (int mt = 0; mt < FT; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) gb1[mt][i] += __shfl_xor(gb1[mt][i], off);
#pragma unroll
        for (int i = 0; i < 4; ++i) gb2[i] += __shfl_xor(gb2[i], off);
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) lacc += __shfl_xor(lacc, off);
    // ---- workgroup sum in wave order: [F][CIN + 1], [K][F + 1], loss --------
    constexpr int P1 = F * (CIN + 1);
    const int P2 = K * (F + 1), PT = P1 + P2 + 1;
    for (int w = 0; w < kHW; ++w) {
        if (wave == w) {
            auto put = [&](int idx, float v) { R[idx] = w == 0 ? v : R[idx] + v; };
#pragma unroll
            for (int mt = 0; mt < FT; ++mt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int f = 16 * mt + 4 * q + i;
#pragma unroll
                    for (int ct = 0; ct < CT; ++ct) put(f * (CIN + 1) + 16 * ct + col, g1[mt][ct][i]);
                    if (col == 0) put(f * (CIN + 1) + CIN, gb1[mt][i]);
                    const int k = 4 * q + i;
                    if (k < K) put(P1 + k * (F + 1) + 16 * mt + col, g2[mt][i]);
                }
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (col == 0 && 4 * q + i < K) put(P1 + (4 * q + i) * (F + 1) + F, gb2[i]);
            if (lane == 0) put(P1 + P2, lacc);
        }
        __syncthreads();
    }
    float *part = partial + (long long)blockIdx.x * PT;
    for (int e = threadIdx.x; e < PT; e += kHT) part[e] = R[e];
}

// Sums the per-block partials and scatters them to the outputs.  A block
// takes 16 outputs; its 256 threads split the partials into 16 interleaved
// parts (thread (part, output)), and the 16 part sums of an output are then
// added in part order: a fixed summation order, 16x shorter dependent chains.
constexpr int kRedOut = 16, kRedParts = kThreads / kRedOut;

__global__ void __launch_bounds__(kThreads)
k_head_reduce(long long M, int Cin, int F, int K, int nblk, const float *__restrict__ partial,
              float *__restrict__ dw1, float *__restrict__ db1, float *__restrict__ dw2,
              float *__restrict__ db2, float *__restrict__ loss)
{
    __shared__ float part_sum[kRedParts][kRedOut];
    const int P1 = F * (Cin + 1), P2 = K * (F + 1), PT = P1 + P2 + 1;
    const int o = threadIdx.x % kRedOut, part = threadIdx.x / kRedOut;
    const int i = blockIdx.x * kRedOut + o;
    float acc = 0.0f;
    if (i < PT)
        for (int b = part; b < nblk; b += kRedParts) acc += partial[(long long)b * PT + i];
    part_sum[part][o] = acc;
    __syncthreads();
    if (part != 0 || i >= PT) return;
    acc = 0.0f;
    for (int k = 0; k < kRedParts; ++k) acc += part_sum[k][o];
    if (i < P1) {
        const int f = i / (Cin + 1), c = i % (Cin + 1);
        if (c < Cin) dw1[f * Cin + c] = acc;
        else db1[f] = acc;
    } else if (i < P1 + P2) {
        const int k = (i - P1) / (F + 1), f = (i - P1) % (F + 1);
        if (f < F) dw2[k * F + f] = acc;
        else db2[k] = acc;
    } else if (loss) {
        *loss = acc / (float)M;
    }
}

constexpr int kHeadMaxBlocks = 1024;

inline int head_blocks(long long M)
{
    const long long t = (M + 16 * kHW - 1) / (16 * kHW);
    return (int)(t < kHeadMaxBlocks ? t : kHeadMaxBlocks);
}

template <int CIN, int F>
int head_launch(long long M, int K, const float *x, const float *w1, const float *b1,
                const float *w2, const float *b2, const int32_t *labels, float *p, float *loss,
                float *dx, float *dw1, float *db1, float *dw2, float *db2, float *partial,
                hipStream_t st)
{
    const int nb = head_blocks(M);
    const size_t lds = HeadCfg<CIN, F>::bytes;
    timing_begin("head_fused", st);
    (void)hipFuncSetAttribute((const void *)k_head_train<CIN, F>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    k_head_train<CIN, F><<<nb, kHT, lds, st>>>(M, K, x, w1, b1, w2, b2, labels, p, dx, partial);
    PLSTM_LAUNCH_CHECK();
    const int PT = F * (CIN + 1) + K * (F + 1) + 1;
    k_head_reduce<<<(PT + kRedOut - 1) / kRedOut, kThreads, 0, st>>>(
        M, CIN, F, K, nb, partial, dw1, db1, dw2, db2, loss);
    PLSTM_LAUNCH_CHECK();
    timing_end(2, st);
    return PLSTM_OK;
}

// ---- FC + tanh backward on the MFMA ---------------------------------------------
// For 16 rows at a time (rows on N, as in the fused head): dz = dy (1 - y^2),
// dX^T = W^T dz^T, and dW = dz^T x, db = sum dz accumulated over the wave's
// rows through a per-wave LDS transpose of dz and x; workgroup partials in
// [F][CIN + 1] (then one unused slot) are summed by k_head_reduce in a fixed
// order.  The next rows' dy, y and x are loaded while these compute.
template <int CIN, int F>
struct FcBwdCfg {
    static constexpr int CT = CIN / 16, FT = F / 16;
    static constexpr int XP = CIN + 4, ZP = F + 4;        // LDS row pitches (floats)
    static constexpr int per_wave = 16 * (XP + ZP);
    static constexpr int red = F * (CIN + 1) + 1;
    static constexpr size_t bytes = (size_t)(kHW * per_wave + red) * sizeof(float);
};

template <int CIN, int F>
__global__ void __launch_bounds__(kHT)
k_fc_tanh_bwd_mfma(long long M, const float *__restrict__ x, const float *__restrict__ w,
                   const float *__restrict__ y, const float *__restrict__ dy,
                   float *__restrict__ dx, float *__restrict__ partial)
{
    typedef float f4 __attribute__((ext_vector_type(4)));
    using FC = FcBwdCfg<CIN, F>;
    static_assert(CIN % 16 == 0 && F % 16 == 0, "tile multiples");
    constexpr int CT = FC::CT, FT = FC::FT;
    extern __shared__ float lds[];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int q = lane >> 4, col = lane & 15;
    float *xs = lds + wave * FC::per_wave;   // [16][XP]  x
    float *zs = xs + 16 * FC::XP;            // [16][ZP]  dz
    float *R = lds + kHW * FC::per_wave;     // workgroup reduction

    float a4[CT][FT][4];   // W[f = 16mt + 4q + i][c = 16ct + col]
#pragma unroll
    for (int mt = 0; mt < FT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) a4[ct][mt][i] = w[(16 * mt + 4 * q + i) * CIN + 16 * ct + col];

    f4 g1[FT][CT], gb1[FT];
#pragma unroll
    for (int mt = 0; mt < FT; ++mt) {
        gb1[mt] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) g1[mt][ct] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    const long long nsub = (M + 15) / 16;
    const long long gw = (long long)blockIdx.x * kHW + wave, nw = (long long)gridDim.x * kHW;
    f4 xn[CT], yn[FT], dn[FT];
    auto load = [&](long long st) {
        const long long row = st * 16 + col;
        const long long rr = (st < nsub && row < M) ? row : 0;
#pragma unroll
        for (int kt = 0; kt < CT; ++kt) xn[kt] = *(const f4 *)&x[rr * CIN + 16 * kt + 4 * q];
#pragma unroll
        for (int mt = 0; mt < FT; ++mt) {
            yn[mt] = *(const f4 *)&y[rr * F + 16 * mt + 4 * q];
            dn[mt] = *(const f4 *)&dy[rr * F + 16 * mt + 4 * q];
        }
    };
    load(gw);
    for (long long st = gw; st < nsub; st += nw) {
        const long long row = st * 16 + col;
        const bool valid = row < M;
        f4 xv[CT], dz[FT];
        const f4 zero = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int kt = 0; kt < CT; ++kt) xv[kt] = valid ? xn[kt] : zero;
#pragma unroll
        for (int mt = 0; mt < FT; ++mt) {
            f4 v;
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = dn[mt][i] * (1.0f - yn[mt][i] * yn[mt][i]);
            dz[mt] = valid ? v : zero;
            gb1[mt] += dz[mt];
        }
        load(st + nw);
        if (dx) {
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                f4 acc = zero;
#pragma unroll
                for (int mt = 0; mt < FT; ++mt)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[ct][mt][i], dz[mt][i], acc,
                                                                   0, 0, 0);
                if (valid) *(f4 *)&dx[row * CIN + 16 * ct + 4 * q] = acc;
            }
        }
#pragma unroll
        for (int kt = 0; kt < CT; ++kt) *(f4 *)&xs[col * FC::XP + 16 * kt + 4 * q] = xv[kt];
#pragma unroll
        for (int mt = 0; mt < FT; ++mt) *(f4 *)&zs[col * FC::ZP + 16 * mt + 4 * q] = dz[mt];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int r = 4 * ks + q;
#pragma unroll
            for (int mt = 0; mt < FT; ++mt) {
                const float az = zs[r * FC::ZP + 16 * mt + col];
#pragma unroll
                for (int ct = 0; ct < CT; ++ct)
                    g1[mt][ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                        az, xs[r * FC::XP + 16 * ct + col], g1[mt][ct], 0, 0, 0);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    // bias sums over the 16 row lanes of each lane group
#pragma unroll
    for (int off = 1; off < 16; off <<= 1)
#pragma unroll
        for (int mt = 0; mt < FT; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) gb1[mt][i] += __shfl_xor(gb1[mt][i], off);
    // workgroup sum in wave order: [F][CIN + 1], then an unused slot
    constexpr int P1 = F * (CIN + 1), PT = P1 + 1;
    for (int wv = 0; wv < kHW; ++wv) {
        if (wave == wv) {
            auto put = [&](int idx, float v) { R[idx] = wv == 0 ? v : R[idx] + v; };
#pragma unroll
            for (int mt = 0; mt < FT; ++mt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int f = 16 * mt + 4 * q + i;
#pragma unroll
                    for (int ct = 0; ct < CT; ++ct) put(f * (CIN + 1) + 16 * ct + col, g1[mt][ct][i]);
                    if (col == 0) put(f * (CIN + 1) + CIN, gb1[mt][i]);
                }
            if (lane == 0) put(P1, 0.0f);
        }
        __syncthreads();
    }
    float *part = partial + (long long)blockIdx.x * PT;
    for (int e = threadIdx.x; e < PT; e += kHT) part[e] = R[e];
}

template <int CIN, int F>
int fc_bwd_mfma_launch(long long M, const float *x, const float *w, const float *y,
                       const float *dy, float *dx, float *dw, float *db, float *partial,
                       hipStream_t st)
{
    const int nb = head_blocks(M);
    const size_t lds = FcBwdCfg<CIN, F>::bytes;
    (void)hipFuncSetAttribute((const void *)k_fc_tanh_bwd_mfma<CIN, F>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    k_fc_tanh_bwd_mfma<CIN, F><<<nb, kHT, lds, st>>>(M, x, w, y, dy, dx, partial);
    PLSTM_LAUNCH_CHECK();
    const int PT = F * (CIN + 1) + 1;
    k_head_reduce<<<(PT + kRedOut - 1) / kRedOut, kThreads, 0, st>>>(
        M, CIN, F, 0, nb, partial, dw, db, nullptr, nullptr, nullptr);
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

// Row counts of the MFMA FC backward's partials (one row of F (CIN + 1) + 1
// floats per workgroup).
inline size_t fc_bwd_mfma_floats(long long M, int Cin, int Cout)
{
    return (size_t)head_blocks(M) * (Cout * (Cin + 1) + 1);
}
inline bool fc_bwd_mfma_ok(int Cin, int Cout)
{
    return (Cin == 16 && Cout == 32) || (Cin == 32 && Cout == 64);
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
    // the MFMA FC backward's workgroup partials use the same workspace
    const size_t mfma = fc_bwd_mfma_ok(Cin, Cout) ? fc_bwd_mfma_floats(M, Cin, Cout) * sizeof(float)
                                                  : 0;
    return cv.off > mfma ? cv.off : mfma;
}

// ---- FC + tanh on the MFMA ----------------------------------------------------
// y = tanh(W x + b) for 16-voxel tiles: M = output units (16 per tile, CO
// tiles), N = voxels, K = inputs in CI blocks of 16 (v_mfma_f32_16x16x4f32).
// In each block lane group q takes inputs 4q .. 4q+3 (k-step i: input
// 4q + i), so W rows and x rows are read as 16-byte (fp32) or 8-byte (bf16)
// vectors in place, and every lane ends with four consecutive outputs of one
// voxel.  A wave takes kFcNT voxel tiles.
constexpr int kFcNT = 2;

template <typename TS> struct Vec4;
template <> struct Vec4<float> {
    typedef float f4v __attribute__((ext_vector_type(4)));
    __device__ static f4v load(const float *p) { return *(const f4v *)p; }
    __device__ static void store(float *p, f4v v) { *(f4v *)p = v; }
};
template <> struct Vec4<uint16_t> {
    typedef float f4v __attribute__((ext_vector_type(4)));
    typedef unsigned short u4 __attribute__((ext_vector_type(4)));
    __device__ static f4v load(const uint16_t *p)
    {
        const u4 v = *(const u4 *)p;
        return f4v{bf16_to_f32(v[0]), bf16_to_f32(v[1]), bf16_to_f32(v[2]), bf16_to_f32(v[3])};
    }
    __device__ static void store(uint16_t *p, f4v v)
    {
        *(u4 *)p = u4{f32_to_bf16(v[0]), f32_to_bf16(v[1]), f32_to_bf16(v[2]), f32_to_bf16(v[3])};
    }
};

template <typename TS, int CI, int CO>
__global__ void __launch_bounds__(256)
k_fc_tanh_mfma(long long M, const TS *__restrict__ x, const TS *__restrict__ w,
               const TS *__restrict__ b, TS *__restrict__ y)
{
    typedef float f4 __attribute__((ext_vector_type(4)));
    constexpr int Cin = 16 * CI, Cout = 16 * CO;
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const long long tile0 = ((long long)blockIdx.x * 4 + (threadIdx.x >> 6)) * kFcNT;
    long long row[kFcNT];
    bool live[kFcNT];
#pragma unroll
    for (int nt = 0; nt < kFcNT; ++nt) {
        row[nt] = (tile0 + nt) * 16 + col;
        live[nt] = row[nt] < M;
    }
    f4 acc[CO][kFcNT];
#pragma unroll
    for (int mt = 0; mt < CO; ++mt) {
        const f4 bv = Vec4<TS>::load(b + mt * 16 + 4 * q4);
#pragma unroll
        for (int nt = 0; nt < kFcNT; ++nt) acc[mt][nt] = bv;
    }
#pragma unroll
    for (int kb = 0; kb < CI; ++kb) {
        f4 xv[kFcNT];
#pragma unroll
        for (int nt = 0; nt < kFcNT; ++nt) {
            xv[nt] = f4{0.0f, 0.0f, 0.0f, 0.0f};
            if (live[nt]) xv[nt] = Vec4<TS>::load(x + row[nt] * Cin + kb * 16 + 4 * q4);
        }
#pragma unroll
        for (int mt = 0; mt < CO; ++mt) {
            const f4 wv = Vec4<TS>::load(w + (long long)(mt * 16 + col) * Cin + kb * 16 + 4 * q4);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int nt = 0; nt < kFcNT; ++nt)
                    acc[mt][nt] =
                        __builtin_amdgcn_mfma_f32_16x16x4f32(wv[i], xv[nt][i], acc[mt][nt], 0, 0, 0);
        }
    }
#pragma unroll
    for (int nt = 0; nt < kFcNT; ++nt) {
        if (!live[nt]) continue;
#pragma unroll
        for (int mt = 0; mt < CO; ++mt) {
            f4 v;
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = tanh_fast(acc[mt][nt][i]);
            Vec4<TS>::store(y + row[nt] * Cout + mt * 16 + 4 * q4, v);
        }
    }
}

template <typename TS, int CI>
int fc_mfma_co(long long M, int Cout, const TS *x, const TS *w, const TS *b, TS *y,
               hipStream_t st)
{
    const long long waves = (M + 16 * kFcNT - 1) / (16 * kFcNT);
    const unsigned blocks = (unsigned)((waves + 3) / 4);
    switch (Cout) {
    case 32: k_fc_tanh_mfma<TS, CI, 2><<<blocks, 256, 0, st>>>(M, x, w, b, y); break;
    case 64: k_fc_tanh_mfma<TS, CI, 4><<<blocks, 256, 0, st>>>(M, x, w, b, y); break;
    case 128: k_fc_tanh_mfma<TS, CI, 8><<<blocks, 256, 0, st>>>(M, x, w, b, y); break;
    default: return PLSTM_EUNSUPPORTED;
    }
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

// bf16 storage with 32 or 64 inputs on the bf16 MFMA: the same tiles as
// k_fc_tanh_mfma, each K-group of 32 inputs one v_mfma_f32_16x16x32_bf16 in
// which lane group q supplies inputs 8q .. 8q+7 of its W row and of its x
// row, each a 16-byte load.  Products of bf16 values are exact in fp32, so
// only the order of the fp32 sums differs from the widened kernel.  A wave
// takes NT voxel tiles (four, two for 128 outputs to keep two waves per
// SIMD), so each W fragment feeds NT MFMAs.
template <int CO> struct FcB16NT {
    static constexpr int value = CO >= 8 ? 2 : 4;
};

template <int CI32, int CO>
__global__ void __launch_bounds__(256)
k_fc_tanh_b16(long long M, const uint16_t *__restrict__ x, const uint16_t *__restrict__ w,
              const uint16_t *__restrict__ b, uint16_t *__restrict__ y)
{
    typedef float f4 __attribute__((ext_vector_type(4)));
    typedef __bf16 bf8v __attribute__((ext_vector_type(8)));
    typedef unsigned u4v __attribute__((ext_vector_type(4)));
    constexpr int Cin = 32 * CI32, Cout = 16 * CO, kFcNTb = FcB16NT<CO>::value;
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const long long tile0 = ((long long)blockIdx.x * 4 + (threadIdx.x >> 6)) * kFcNTb;
    long long row[kFcNTb];
    bool live[kFcNTb];
#pragma unroll
    for (int nt = 0; nt < kFcNTb; ++nt) {
        row[nt] = (tile0 + nt) * 16 + col;
        live[nt] = row[nt] < M;
    }
    f4 acc[CO][kFcNTb];
#pragma unroll
    for (int mt = 0; mt < CO; ++mt) {
        const f4 bv = Vec4<uint16_t>::load(b + mt * 16 + 4 * q4);
#pragma unroll
        for (int nt = 0; nt < kFcNTb; ++nt) acc[mt][nt] = bv;
    }
    const bf8v zero = __builtin_bit_cast(bf8v, u4v{0u, 0u, 0u, 0u});
#pragma unroll
    for (int kb = 0; kb < CI32; ++kb) {
        bf8v xv[kFcNTb];
#pragma unroll
        for (int nt = 0; nt < kFcNTb; ++nt)
            xv[nt] = live[nt] ? *(const bf8v *)(x + row[nt] * Cin + kb * 32 + 8 * q4) : zero;
#pragma unroll
        for (int mt = 0; mt < CO; ++mt) {
            const bf8v wv = *(const bf8v *)(w + (long long)(mt * 16 + col) * Cin + kb * 32 + 8 * q4);
#pragma unroll
            for (int nt = 0; nt < kFcNTb; ++nt)
                acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wv, xv[nt], acc[mt][nt], 0, 0, 0);
        }
    }
#pragma unroll
    for (int nt = 0; nt < kFcNTb; ++nt) {
        if (!live[nt]) continue;
#pragma unroll
        for (int mt = 0; mt < CO; ++mt) {
            f4 v;
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = tanh_fast(acc[mt][nt][i]);
            Vec4<uint16_t>::store(y + row[nt] * Cout + mt * 16 + 4 * q4, v);
        }
    }
}

template <int CI32, int CO>
void launch_fc_b16(long long M, const uint16_t *x, const uint16_t *w, const uint16_t *b,
                   uint16_t *y, hipStream_t st)
{
    constexpr int NT = FcB16NT<CO>::value;
    const long long waves = (M + 16 * NT - 1) / (16 * NT);
    k_fc_tanh_b16<CI32, CO><<<(unsigned)((waves + 3) / 4), 256, 0, st>>>(M, x, w, b, y);
}

template <int CI32>
int fc_b16_co(long long M, int Cout, const uint16_t *x, const uint16_t *w, const uint16_t *b,
              uint16_t *y, hipStream_t st)
{
    switch (Cout) {
    case 32: launch_fc_b16<CI32, 2>(M, x, w, b, y, st); break;
    case 64: launch_fc_b16<CI32, 4>(M, x, w, b, y, st); break;
    case 128: launch_fc_b16<CI32, 8>(M, x, w, b, y, st); break;
    default: return PLSTM_EUNSUPPORTED;
    }
    PLSTM_LAUNCH_CHECK();
    return PLSTM_OK;
}

// Inference output end for bf16 storage (Section 2.3, "Fully-Connected
// Layer"; Fig. 3): the FC + tanh tiles of k_fc_tanh_b16, whose outputs stay
// in registers, then the per-voxel linear layer as a second MFMA with the
// classes as its 16 rows and the voxels as its columns.  After the first
// contraction lane group q of a voxel column holds FC outputs 16 mt + 4q + i
// (i < 4) of tile mt; K-group kk of the second takes outputs 32 kk + 4q + i
// from tile 2 kk and 32 kk + 16 + 4q + i from tile 2 kk + 1 as lane group q's
// eight values, and the W2 fragments are permuted the same way, so nothing
// crosses lanes.  The FC tiles are made two at a time and consumed at once,
// so only two tiles per voxel tile are live and a wave takes four voxel
// tiles.  The logits of a voxel land in the four lane groups of its column
// (class 4q + i); their maximum and sum meet over the groups with two
// exchanges each.  y is rounded to bf16 before the second contraction, as the
// separate kernels store it, and its tiles are summed in the same order, so
// y is the separate kernels' y bit for bit.
constexpr int kHeadNT = 4;

template <int CI32, int FO>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4)))
k_head_fwd_b16(long long M, int K, const uint16_t *__restrict__ x,
               const uint16_t *__restrict__ w1, const uint16_t *__restrict__ b1,
               const uint16_t *__restrict__ w2, const uint16_t *__restrict__ b2,
               float *__restrict__ p)
{
    typedef float f4 __attribute__((ext_vector_type(4)));
    typedef __bf16 bf8v __attribute__((ext_vector_type(8)));
    typedef unsigned u4v __attribute__((ext_vector_type(4)));
    typedef unsigned short us4v __attribute__((ext_vector_type(4)));
    typedef unsigned short us8v __attribute__((ext_vector_type(8)));
    constexpr int Cin = 32 * CI32, F = 16 * FO, NT = kHeadNT, KK2 = FO / 2;
    static_assert(FO % 2 == 0, "F a multiple of 32");
    const int lane = threadIdx.x & 63, q4 = lane >> 4, col = lane & 15;
    const long long tile0 = ((long long)blockIdx.x * 4 + (threadIdx.x >> 6)) * NT;
    long long row[NT];
    bool live[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        row[nt] = (tile0 + nt) * 16 + col;
        live[nt] = row[nt] < M;
    }
    const bf8v zero = __builtin_bit_cast(bf8v, u4v{0u, 0u, 0u, 0u});
    bf8v xv[CI32][NT];
#pragma unroll
    for (int kb = 0; kb < CI32; ++kb)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
            xv[kb][nt] = live[nt] ? *(const bf8v *)(x + row[nt] * Cin + kb * 32 + 8 * q4) : zero;
    f4 z[NT];
    {
        f4 bias2;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            bias2[i] = 4 * q4 + i < K ? bf16_to_f32(b2[4 * q4 + i]) : 0.0f;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) z[nt] = bias2;
    }
#pragma unroll
    for (int kk = 0; kk < KK2; ++kk) {
        // W2 fragment kk: lane (class col, group q4), permuted as above; zero
        // rows past the last class
        us4v lo = us4v{0, 0, 0, 0}, hi = lo;
        if (col < K) {
            lo = *(const us4v *)(w2 + col * F + 32 * kk + 4 * q4);
            hi = *(const us4v *)(w2 + col * F + 32 * kk + 16 + 4 * q4);
        }
        const bf8v a2 = __builtin_bit_cast(bf8v, us8v{lo[0], lo[1], lo[2], lo[3],
                                                      hi[0], hi[1], hi[2], hi[3]});
        f4 acc[2][NT];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int mt = 2 * kk + h;
            const f4 bv = Vec4<uint16_t>::load(b1 + mt * 16 + 4 * q4);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) acc[h][nt] = bv;
#pragma unroll
            for (int kb = 0; kb < CI32; ++kb) {
                const bf8v wv =
                    *(const bf8v *)(w1 + (long long)(mt * 16 + col) * Cin + kb * 32 + 8 * q4);
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
                    acc[h][nt] =
                        __builtin_amdgcn_mfma_f32_16x16x32_bf16(wv, xv[kb][nt], acc[h][nt], 0, 0, 0);
            }
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            us8v yv;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                yv[i] = f32_to_bf16(tanh_fast(acc[0][nt][i]));
                yv[4 + i] = f32_to_bf16(tanh_fast(acc[1][nt][i]));
            }
            z[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, __builtin_bit_cast(bf8v, yv),
                                                            z[nt], 0, 0, 0);
        }
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        // every lane takes part in the exchanges, live or not
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (4 * q4 + i < K) mx = fmaxf(mx, z[nt][i]);
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        f4 e;
        float sum = 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            e[i] = 4 * q4 + i < K ? __expf(z[nt][i] - mx) : 0.0f;
            sum += e[i];
        }
        sum += __shfl_xor(sum, 16);
        sum += __shfl_xor(sum, 32);
        const float inv = 1.0f / sum;
        if (!live[nt]) continue;
        if (K == 4) {
            if (q4 == 0) *(f4 *)(p + row[nt] * 4) = e * inv;
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (4 * q4 + i < K) p[row[nt] * K + 4 * q4 + i] = e[i] * inv;
        }
    }
}

template <int CI32, int FO>
void launch_head_fwd_b16(long long M, int K, const uint16_t *x, const uint16_t *w1,
                         const uint16_t *b1, const uint16_t *w2, const uint16_t *b2, float *p,
                         hipStream_t st)
{
    constexpr int NT = kHeadNT;
    const long long waves = (M + 16 * NT - 1) / (16 * NT);
    k_head_fwd_b16<CI32, FO><<<(unsigned)((waves + 3) / 4), 256, 0, st>>>(M, K, x, w1, b1, w2,
                                                                         b2, p);
}

// Shapes of the MFMA FC: 16, 32 or 64 inputs, 32, 64 or 128 outputs.
inline bool fc_mfma_ok(int Cin, int Cout)
{
    return (Cin == 16 || Cin == 32 || Cin == 64) && (Cout == 32 || Cout == 64 || Cout == 128);
}

template <typename TS>
int fc_mfma(long long M, int Cin, int Cout, const TS *x, const TS *w, const TS *b, TS *y,
            hipStream_t st)
{
    switch (Cin) {
    case 16: return fc_mfma_co<TS, 1>(M, Cout, x, w, b, y, st);
    case 32: return fc_mfma_co<TS, 2>(M, Cout, x, w, b, y, st);
    default: return fc_mfma_co<TS, 4>(M, Cout, x, w, b, y, st);
    }
}

static int fc_tanh_forward_impl(long long M, int Cin, int Cout, int dtype, const void *x,
                                const void *w, const void *b, void *y, hipStream_t st)
{
    if (fc_mfma_ok(Cin, Cout)) {
        if (dtype == PLSTM_BF16 && Cin >= 32)
            return Cin == 32 ? fc_b16_co<1>(M, Cout, (const uint16_t *)x, (const uint16_t *)w,
                                            (const uint16_t *)b, (uint16_t *)y, st)
                             : fc_b16_co<2>(M, Cout, (const uint16_t *)x, (const uint16_t *)w,
                                            (const uint16_t *)b, (uint16_t *)y, st);
        if (dtype == PLSTM_BF16)
            return fc_mfma<uint16_t>(M, Cin, Cout, (const uint16_t *)x, (const uint16_t *)w,
                                     (const uint16_t *)b, (uint16_t *)y, st);
        return fc_mfma<float>(M, Cin, Cout, (const float *)x, (const float *)w,
                              (const float *)b, (float *)y, st);
    }
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

static int fc_tanh_backward_impl(long long M, int Cin, int Cout, const float *x,
                                 const float *w, const float *y, const float *dy, float *dx,
                                 float *dw, float *db, void *ws, hipStream_t st)
{
    if (Cin == 16 && Cout == 32)
        return fc_bwd_mfma_launch<16, 32>(M, x, w, y, dy, dx, dw, db, (float *)ws, st);
    if (Cin == 32 && Cout == 64)
        return fc_bwd_mfma_launch<32, 64>(M, x, w, y, dy, dx, dw, db, (float *)ws, st);
    Carve cv(ws);
    float *partial = cv.take<float>((size_t)fc_chunks(M) * Cout * (Cin + 1));
    const RowGrad rg{y, dy};
    if (dx) {
        const int rc = fc_dx(M, Cin, Cout, rg, w, dx, st);
        if (rc != PLSTM_OK) return rc;
    }
    return fc_wgrad(M, Cin, Cout, rg, x, dw, db, partial, st);
}

// Softmax head, one thread per row read straight from global memory in
// four-element vectors (Cin a multiple of 4), the weights in LDS (every lane
// reads the same address: broadcast).  Logits stay in registers (K <= 16) and
// the label's probability is picked by comparison, as in the row-tile kernel.
template <typename TS, bool SQ>
__global__ void __launch_bounds__(kThreads)
k_softmax_vec(long long M, int Cin, int K, const TS *__restrict__ x, const TS *__restrict__ w,
              const TS *__restrict__ b, const int32_t *__restrict__ labels,
              float *__restrict__ p, float *__restrict__ dlogits, float *__restrict__ lossp)
{
    typedef float f4v __attribute__((ext_vector_type(4)));
    extern __shared__ float lds[];
    float *sw = lds;                               // [K][Cin]
    for (int e = threadIdx.x; e < K * Cin; e += kThreads) sw[e] = Store<TS>::load(w, e);
    __syncthreads();
    const long long m = (long long)blockIdx.x * kThreads + threadIdx.x;
    float l = 0.0f;
    if (m < M) {
        float z[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) z[k] = k < K ? Store<TS>::load(b, k) : 0.0f;
        const TS *xr = x + m * Cin;
        for (int c = 0; c < Cin; c += 4) {
            const f4v xv = Vec4<TS>::load(xr + c);
#pragma unroll
            for (int k = 0; k < 16; ++k)
                if (k < K) {
                    const f4v wv = *(const f4v *)&sw[k * Cin + c];
                    z[k] += (xv[0] * wv[0] + xv[1] * wv[1]) + (xv[2] * wv[2] + xv[3] * wv[3]);
                }
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
            if (k < K) p[m * K + k] = z[k] * inv;
        if (labels) {
            // An out-of-range label poisons the loss and the gradient with NaN.
            const int lab = labels[m];
            const bool ok = lab >= 0 && lab < K;
            if (SQ) {
                float e = 0.0f, sd = 0.0f;
#pragma unroll
                for (int k = 0; k < 16; ++k) {
                    if (k < K) {
                        const float pk = z[k] * inv, dk = pk - (k == lab ? 1.0f : 0.0f);
                        e += dk * dk;
                        sd += pk * dk;
                    }
                }
                l = ok ? e : NAN;
#pragma unroll
                for (int k = 0; k < 16; ++k)
                    if (k < K) {
                        const float pk = z[k] * inv, dk = pk - (k == lab ? 1.0f : 0.0f);
                        dlogits[m * K + k] = ok ? 2.0f * pk * (dk - sd) / (float)M : NAN;
                    }
            } else {
                float pl = 0.0f;
#pragma unroll
                for (int k = 0; k < 16; ++k)
                    if (k == lab) pl = z[k] * inv;
                l = ok ? -logf(pl) : NAN;
#pragma unroll
                for (int k = 0; k < 16; ++k)
                    if (k < K)
                        dlogits[m * K + k] =
                            ok ? (z[k] * inv - (k == lab ? 1.0f : 0.0f)) / (float)M : NAN;
            }
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

// Softmax head, 16 lanes per row (Cin a multiple of 4): lane j of a row's
// group reads elements 4 j .. 4 j + 3 of every 64-element stretch, so a
// group's loads are contiguous; the partial logits meet in a 16-lane
// butterfly, after which every lane of the group holds the row's logits and
// lane k writes class k.  A block of 256 threads takes 128 rows (eight per
// group), and its loss partial lands in lossp[block].
template <typename TS, bool SQ>
__global__ void __launch_bounds__(kThreads)
k_softmax_coop(long long M, int Cin, int K, const TS *__restrict__ x, const TS *__restrict__ w,
               const TS *__restrict__ b, const int32_t *__restrict__ labels,
               float *__restrict__ p, float *__restrict__ dlogits, float *__restrict__ lossp)
{
    typedef float f4v __attribute__((ext_vector_type(4)));
    extern __shared__ float lds[];
    float *sw = lds;                               // [K][Cin]
    for (int e = threadIdx.x; e < K * Cin; e += kThreads) sw[e] = Store<TS>::load(w, e);
    __syncthreads();
    const int j = threadIdx.x & 15, grp = threadIdx.x >> 4;
    float l = 0.0f;
    for (int it = 0; it < 8; ++it) {
        const long long m = (long long)blockIdx.x * 128 + it * 16 + grp;
        if (m >= M) break;                          // the group's 16 lanes agree
        float z[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) z[k] = 0.0f;
        const TS *xr = x + m * Cin;
        for (int c = 4 * j; c < Cin; c += 64) {
            const f4v xv = Vec4<TS>::load(xr + c);
#pragma unroll
            for (int k = 0; k < 16; ++k)
                if (k < K) {
                    const f4v wv = *(const f4v *)&sw[k * Cin + c];
                    z[k] += (xv[0] * wv[0] + xv[1] * wv[1]) + (xv[2] * wv[2] + xv[3] * wv[3]);
                }
        }
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            if (k < K) {
#pragma unroll
                for (int off = 8; off > 0; off >>= 1) z[k] += __shfl_xor(z[k], off, 16);
                z[k] += Store<TS>::load(b, k);
            }
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
        float pj = 0.0f;
#pragma unroll
        for (int k = 0; k < 16; ++k)
            if (k == j) pj = z[k] * inv;
        if (j < K) p[m * K + j] = pj;
        if (labels) {
            // An out-of-range label poisons the loss and the gradient with NaN.
            const int lab = labels[m];
            const bool ok = lab >= 0 && lab < K;
            const float dj = pj - (j == lab ? 1.0f : 0.0f);
            if (SQ) {
                float e = 0.0f, sd = 0.0f;
#pragma unroll
                for (int k = 0; k < 16; ++k) {
                    if (k < K) {
                        const float pk = z[k] * inv, dk = pk - (k == lab ? 1.0f : 0.0f);
                        e += dk * dk;
                        sd += pk * dk;
                    }
                }
                if (j == 0) l += ok ? e : NAN;
                if (j < K) dlogits[m * K + j] = ok ? 2.0f * pj * (dj - sd) / (float)M : NAN;
            } else {
                float pl = 0.0f;
#pragma unroll
                for (int k = 0; k < 16; ++k)
                    if (k == lab) pl = z[k] * inv;
                if (j == 0) l += ok ? -logf(pl) : NAN;
                if (j < K) dlogits[m * K + j] = ok ? dj / (float)M : NAN;
            }
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

template <bool SQ>
static int softmax_loss_impl(long long M, int Cin, int K, int dtype, const void *x,
                             const void *w, const void *b, const int32_t *labels, float *p,
                             float *loss, float *dx, float *dw, float *db, void *ws,
                             hipStream_t st)
{
    Carve cv(ws);
    float *partial = cv.take<float>((size_t)fc_chunks(M) * K * (Cin + 1));
    float *dlogits = cv.take<float>((size_t)M * K);
    float *lossp = cv.take<float>((size_t)(M + kRB - 1) / kRB);
    unsigned nb = blocks_for(M);
    if (Cin % 4 == 0 && Cin >= 64 && (size_t)K * Cin * sizeof(float) <= 65536) {
        // wide rows: 16 lanes per row, 128 rows per block
        nb = (unsigned)((M + 127) / 128);
        const size_t lds = (size_t)K * Cin * sizeof(float);
        if (dtype == PLSTM_BF16)
            k_softmax_coop<uint16_t, SQ><<<nb, kThreads, lds, st>>>(
                M, Cin, K, (const uint16_t *)x, (const uint16_t *)w, (const uint16_t *)b, labels,
                p, dlogits, lossp);
        else
            k_softmax_coop<float, SQ><<<nb, kThreads, lds, st>>>(
                M, Cin, K, (const float *)x, (const float *)w, (const float *)b, labels, p,
                dlogits, lossp);
    } else if (Cin % 4 == 0 && (size_t)K * Cin * sizeof(float) <= 65536) {
        const size_t lds = (size_t)K * Cin * sizeof(float);
        if (dtype == PLSTM_BF16)
            k_softmax_vec<uint16_t, SQ><<<nb, kThreads, lds, st>>>(
                M, Cin, K, (const uint16_t *)x, (const uint16_t *)w, (const uint16_t *)b, labels,
                p, dlogits, lossp);
        else
            k_softmax_vec<float, SQ><<<nb, kThreads, lds, st>>>(
                M, Cin, K, (const float *)x, (const float *)w, (const float *)b, labels, p,
                dlogits, lossp);
    } else if (rows_ok(Cin)) {
        nb = (unsigned)((M + kRB - 1) / kRB);
        const size_t lds = rows_lds(Cin, 16, K * (Cin + 1));
        if (dtype == PLSTM_BF16)
            k_softmax_rows<uint16_t, SQ><<<nb, kRB, lds, st>>>(
                M, Cin, K, (const uint16_t *)x, (const uint16_t *)w, (const uint16_t *)b, labels,
                p, dlogits, lossp);
        else
            k_softmax_rows<float, SQ><<<nb, kRB, lds, st>>>(
                M, Cin, K, (const float *)x, (const float *)w, (const float *)b, labels, p,
                dlogits, lossp);
    } else if (dtype == PLSTM_BF16) {
        k_softmax<uint16_t, SQ><<<nb, kThreads, 0, st>>>(M, Cin, K, (const uint16_t *)x,
                                                      (const uint16_t *)w, (const uint16_t *)b,
                                                      labels, p, dlogits, lossp);
    } else {
        k_softmax<float, SQ><<<nb, kThreads, 0, st>>>(M, Cin, K, (const float *)x, (const float *)w,
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

int fc_tanh_forward(long long M, int Cin, int Cout, int dtype, const void *x, const void *w,
                    const void *b, void *y, hipStream_t st)
{
    timing_begin("fc_tanh_fwd", st);
    const int rc = fc_tanh_forward_impl(M, Cin, Cout, dtype, x, w, b, y, st);
    timing_end(1, st);
    return rc;
}

int fc_tanh_backward(long long M, int Cin, int Cout, const float *x, const float *w,
                     const float *y, const float *dy, float *dx, float *dw, float *db,
                     void *ws, hipStream_t st)
{
    timing_begin("fc_tanh_bwd", st);
    const int rc = fc_tanh_backward_impl(M, Cin, Cout, x, w, y, dy, dx, dw, db, ws, st);
    timing_end(fc_bwd_mfma_ok(Cin, Cout) ? 2 : (dx ? 3 : 2), st);
    return rc;
}

int softmax_ce(long long M, int Cin, int K, int dtype, const void *x, const void *w,
               const void *b, const int32_t *labels, float *p, float *loss, float *dx,
               float *dw, float *db, void *ws, hipStream_t st, bool squared)
{
    timing_begin(squared ? "softmax_sq" : "softmax_ce", st);
    const int rc =
        squared ? softmax_loss_impl<true>(M, Cin, K, dtype, x, w, b, labels, p, loss, dx, dw, db,
                                          ws, st)
                : softmax_loss_impl<false>(M, Cin, K, dtype, x, w, b, labels, p, loss, dx, dw, db,
                                           ws, st);
    timing_end(1 + (labels ? 1 : 0) + (dw ? 2 : 0) + (dx ? 1 : 0), st);
    return rc;
}

bool head_supported(int Cin, int F, int K)
{
    return K >= 1 && K <= 16 && ((Cin == 16 && F == 32) || (Cin == 32 && F == 64));
}

size_t head_ws(long long M, int Cin, int F, int K)
{
    return (size_t)head_blocks(M) * (F * (Cin + 1) + K * (F + 1) + 1) * sizeof(float);
}

bool head_fwd_supported(int dtype, int Cin, int F, int K)
{
    return dtype == PLSTM_BF16 && (Cin == 32 || Cin == 64) && (F == 32 || F == 64 || F == 128) &&
           K >= 1 && K <= 16;
}

int head_forward(long long M, int Cin, int F, int K, const uint16_t *x, const uint16_t *w1,
                 const uint16_t *b1, const uint16_t *w2, const uint16_t *b2, float *p,
                 hipStream_t st)
{
    timing_begin("head_fwd", st);
    auto go = [&](auto ci, auto fo) {
        launch_head_fwd_b16<decltype(ci)::value, decltype(fo)::value>(M, K, x, w1, b1, w2, b2, p,
                                                                      st);
    };
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I4 = std::integral_constant<int, 4>;
    using I8 = std::integral_constant<int, 8>;
    if (Cin == 32) {
        if (F == 32) go(I1(), I2());
        else if (F == 64) go(I1(), I4());
        else go(I1(), I8());
    } else {
        if (F == 32) go(I2(), I2());
        else if (F == 64) go(I2(), I4());
        else go(I2(), I8());
    }
    PLSTM_LAUNCH_CHECK();
    timing_end(1, st);
    return PLSTM_OK;
}

int head_train(long long M, int Cin, int F, int K, const float *x, const float *w1,
               const float *b1, const float *w2, const float *b2, const int32_t *labels,
               float *p, float *loss, float *dx, float *dw1, float *db1, float *dw2, float *db2,
               void *ws, hipStream_t st)
{
    float *partial = (float *)ws;
    if (Cin == 16 && F == 32)
        return head_launch<16, 32>(M, K, x, w1, b1, w2, b2, labels, p, loss, dx, dw1, db1, dw2,
                                   db2, partial, st);
    if (Cin == 32 && F == 64)
        return head_launch<32, 64>(M, K, x, w1, b1, w2, b2, labels, p, loss, dx, dw1, db1, dw2,
                                   db2, partial, st);
    return PLSTM_EUNSUPPORTED;
}

}  // namespace plstm
