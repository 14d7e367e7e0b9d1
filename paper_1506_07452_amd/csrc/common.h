// Internal helpers shared by the library's translation units (host + device).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "pyramid_lstm.h"

namespace plstm {

constexpr int kDirs = 6;

// Geometry of one sweep direction (Section 2.3, direction set).  A voxel of
// batch element n at sweep position s and in-plane pixel (p, q) has linear
// index n * V + s * ss + p * sp + q * sq in the [N][D][H][W] volume.
struct DirGeom {
    int T, P, Q;          // sweep length, in-plane extents (first, second axis)
    int sign;             // +1: plane t is s = t; -1: plane t is s = T - 1 - t
    long long ss, sp, sq; // voxel strides of s, p, q
};

// A layer's geometry.  Directions d < nd are active: the six sweeps of a
// volume (nd = 6, axis[d] = d / 2: z, y, x) or the four line sweeps of an
// image (nd = 4: y+, y-, x+, x-, the image being a volume with D = 1).  The
// filters have KP x KQ taps over the plane's (first, second) axis: K x K for
// a volume, 1 x K along the line for an image.  Per-direction arrays
// (weights, saved states, gradients) hold nd directions.
struct Geom {
    int N, D, H, W, C, O;
    int K;                // filter size (odd)
    int KP, KQ;           // taps along the plane's first and second axis
    int nd;               // active directions
    int axis[kDirs];      // sweep axis of direction d: 0 z, 1 y, 2 x
    long long V;          // D * H * W
    DirGeom dir[kDirs];
};

inline void set_dir(Geom &g, int d, int axis, int sign)
{
    const long long HW = (long long)g.H * g.W;
    DirGeom &r = g.dir[d];
    r.sign = sign;
    g.axis[d] = axis;
    switch (axis) {
    case 0: r.T = g.D; r.P = g.H; r.Q = g.W; r.ss = HW; r.sp = g.W; r.sq = 1; break;
    case 1: r.T = g.H; r.P = g.D; r.Q = g.W; r.ss = g.W; r.sp = HW; r.sq = 1; break;
    default: r.T = g.W; r.P = g.D; r.Q = g.H; r.ss = 1; r.sp = HW; r.sq = g.W; break;
    }
}

inline Geom make_geom(const plstm_shape &s) {
    Geom g;
    g.N = s.N; g.D = s.D; g.H = s.H; g.W = s.W; g.C = s.C; g.O = s.O;
    g.K = s.K == 0 ? 3 : s.K;
    g.KP = g.KQ = g.K;
    g.nd = kDirs;
    g.V = (long long)s.D * s.H * s.W;
    for (int d = 0; d < kDirs; ++d) set_dir(g, d, d / 2, (d % 2 == 0) ? 1 : -1);
    return g;
}

// An image [N][H][W][C] as a volume with D = 1: directions y+, y- (rows top to
// bottom and back, each step a row of W pixels) and x+, x- (columns), 1 x K
// filters along the line.  Unused direction slots have no planes.
inline Geom make_geom2d(const plstm2d_shape &s) {
    Geom g;
    g.N = s.N; g.D = 1; g.H = s.H; g.W = s.W; g.C = s.C; g.O = s.O;
    g.K = s.K == 0 ? 3 : s.K;
    g.KP = 1;
    g.KQ = g.K;
    g.nd = 4;
    g.V = (long long)s.H * s.W;
    for (int d = 0; d < 4; ++d) set_dir(g, d, 1 + d / 2, (d % 2 == 0) ? 1 : -1);
    for (int d = 4; d < kDirs; ++d) {
        set_dir(g, d, 0, 1);
        g.dir[d].T = 0;
    }
    return g;
}

// bf16 <-> fp32 (round to nearest even; NaN kept quiet).
__host__ __device__ inline float bf16_to_f32(uint16_t v) {
    union { uint32_t u; float f; } c;
    c.u = (uint32_t)v << 16;
    return c.f;
}
__host__ __device__ inline uint16_t f32_to_bf16(float f) {
    union { uint32_t u; float f; } c;
    c.f = f;
    if ((c.u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((c.u >> 16) | 0x40);
    const uint32_t lsb = (c.u >> 16) & 1u;
    return (uint16_t)((c.u + 0x7fffu + lsb) >> 16);
}

template <typename T> struct Store;
template <> struct Store<float> {
    __device__ static float load(const float *p, long long i) { return p[i]; }
    __device__ static void store(float *p, long long i, float v) { p[i] = v; }
};
template <> struct Store<uint16_t> {
    __device__ static float load(const uint16_t *p, long long i) { return bf16_to_f32(p[i]); }
    __device__ static void store(uint16_t *p, long long i, float v) { p[i] = f32_to_bf16(v); }
};

__device__ inline float sigmoidf_(float a) { return 1.0f / (1.0f + __expf(-a)); }

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Bump allocator over a caller-provided workspace.
struct Carve {
    char *base;
    size_t off = 0;
    explicit Carve(void *p) : base((char *)p) {}
    template <typename T> T *take(size_t count) {
        off = align_up(off, 256);
        T *p = base ? (T *)(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
};

#define PLSTM_LAUNCH_CHECK()                                   \
    do {                                                       \
        if (hipGetLastError() != hipSuccess) return PLSTM_EHIP; \
    } while (0)

// Saved-activation layout shared by every forward/backward pair (fp32,
// per-direction volumes in [N][D][H][W] voxel order, nd directions):
//   gates [nd][N][V][4O]  i, f, g, o after the nonlinearity
//   cell  [nd][N][V][O]   c^d
//   hd    [nd][N][V][O]   h^d
struct Saved {
    float *gates, *cell, *hd;
};
inline size_t saved_gates_count(const Geom &g) { return (size_t)g.nd * g.N * g.V * 4 * g.O; }
inline size_t saved_state_count(const Geom &g) { return (size_t)g.nd * g.N * g.V * g.O; }
inline Saved carve_saved(void *p, const Geom &g) {
    Carve cv(p);
    Saved s;
    s.gates = cv.take<float>(saved_gates_count(g));
    s.cell = cv.take<float>(saved_state_count(g));
    s.hd = cv.take<float>(saved_state_count(g));
    return s;
}
inline size_t saved_bytes(const Geom &g) {
    Carve cv(nullptr);
    cv.take<float>(saved_gates_count(g));
    cv.take<float>(saved_state_count(g));
    cv.take<float>(saved_state_count(g));
    return cv.off;
}

// ---- launchers implemented in the .hip translation units -------------------

// Generic path (any supported shape): one launch per plane step.
// Forward: with `sv` (training) h^d, c^d and the gates go to the saved buffer,
// otherwise h^d and c^d live in the workspace.
int generic_forward(const Geom &g, int dtype, const void *x, const void *wx, const void *wh,
                    const void *b, void *h, const Saved *sv, void *ws, hipStream_t st);
size_t generic_forward_ws(const Geom &g, bool training);
int generic_backward(const Geom &g, const float *x, const float *wx, const float *wh,
                     const Saved &sv, const float *dh, float *dx, float *dwx, float *dwh,
                     float *db, void *ws, hipStream_t st);
size_t generic_backward_ws(const Geom &g);
// dL/dx from the gate gradients dA [6][N][V][4O] of every direction.
int generic_dx(const Geom &g, const float *wx, const float *dA, float *dx, hipStream_t st);

// dst[i] = src[i] for n bf16 values widened to fp32.
int bf16_to_f32(const void *src, float *dst, long long n, hipStream_t st);

// Fully connected glue.
int fc_tanh_forward(long long M, int Cin, int Cout, int dtype, const void *x, const void *w,
                    const void *b, void *y, hipStream_t st);
int fc_tanh_backward(long long M, int Cin, int Cout, const float *x, const float *w,
                     const float *y, const float *dy, float *dx, float *dw, float *db,
                     void *ws, hipStream_t st);
size_t fc_ws(long long M, int Cin, int Cout);
// `squared`: the squared error of Eq. (14) instead of the cross-entropy.
int softmax_ce(long long M, int Cin, int K, int dtype, const void *x, const void *w,
               const void *b, const int32_t *labels, float *p, float *loss, float *dx,
               float *dw, float *db, void *ws, hipStream_t st, bool squared = false);
// Fused FC + tanh, linear + softmax for inference (bf16 storage).
bool head_fwd_supported(int dtype, int Cin, int F, int K);
int head_forward(long long M, int Cin, int F, int K, const uint16_t *x, const uint16_t *w1,
                 const uint16_t *b1, const uint16_t *w2, const uint16_t *b2, float *p,
                 hipStream_t st);
// Fused FC + tanh, linear + softmax, cross-entropy and backward (fp32).
bool head_supported(int Cin, int F, int K);
size_t head_ws(long long M, int Cin, int F, int K);
int head_train(long long M, int Cin, int F, int K, const float *x, const float *w1,
               const float *b1, const float *w2, const float *b2, const int32_t *labels,
               float *p, float *loss, float *dx, float *dw1, float *db1, float *dw2, float *db2,
               void *ws, hipStream_t st);

}  // namespace plstm
