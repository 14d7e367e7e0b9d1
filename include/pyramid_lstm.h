/*
 * pyramid_lstm.h -- C ABI of the MI355X (gfx950) PyraMiD-LSTM library.
 *
 * The layer (Stollenga et al., arXiv 1506.07452, Section 2.3):
 *   six C-LSTMs, one per direction d in {z+, z-, y+, y-, x+, x-} (paper axes
 *   x, y, z = volume W, H, D; direction set of Section 2.3), each sweeping the
 *   volume plane by plane.  At every plane each voxel computes the gate
 *   pre-activations of Eq. (7)-(9), (11) as a 3x3 2D convolution of the input
 *   plane plus a 3x3 2D convolution of the previous plane's hidden state plus a
 *   per-gate bias shared by all positions, then the cell and hidden update of
 *   Eq. (10), (12); the layer output is the sum of the six directions, Eq. (13).
 *
 * Conventions shared by every entry point:
 *   - All tensor pointers are DEVICE pointers (hipMalloc'd or equivalent),
 *     owned by the caller, aligned to 16 bytes.  The library never allocates,
 *     frees, or synchronises: work is enqueued on `stream` (a hipStream_t; NULL
 *     is the legacy default stream) and completes asynchronously.
 *   - Arguments are validated before anything is enqueued; an error is a
 *     negative return code (never an abort or exception) and nothing has been
 *     launched.  PLSTM_EHIP means a HIP launch failed after validation.
 *   - Calls on distinct streams with distinct buffers are independent.
 *   - Storage type (plstm_shape.dtype): PLSTM_F32 = IEEE fp32; PLSTM_BF16 =
 *     bfloat16 (uint16 bit patterns) for x, wx, wh, b and h.  Accumulation is
 *     always fp32; the cell state is always fp32.
 *   - Layouts are row-major, channels last:
 *       x   [N][D][H][W][C]        volume, C input channels
 *       h   [N][D][H][W][O]        layer output (sum of the six directions)
 *       wx  [6][4*O][C][K][K]      input filters, per direction
 *       wh  [6][4*O][O][K][K]      recurrent filters, per direction
 *       b   [6][4*O]               biases, per direction
 *     Direction order 0..5 = z+, z-, y+, y-, x+, x- (Section 2.3).  Row g*O+o
 *     of wx/wh/b is unit o of gate g, gates in the order (i, f, g=c~, o) of
 *     Eq. (7), (8), (9), (11).  The K x K taps (ka, kb) run over the plane's
 *     two in-plane axes in (D, H, W) order: z+- -> (H, W), y+- -> (D, W),
 *     x+- -> (D, H); the same for the + and - direction of an axis.  The
 *     convolution is a cross-correlation with zero "same" padding, r = (K-1)/2:
 *       A[p][q][g*O+o] += in[p+ka-r][q+kb-r][c] * w[g*O+o][c][ka][kb].
 *     K is odd: 3 is the filter of Section 2.3's examples, 7 the one of the
 *     experiments (Section 3, "Experimental Setup").
 *     Plane t of a + sweep is index t along its axis, of a - sweep index T-1-t;
 *     the first plane has no predecessor (h_{-1} = c_{-1} = 0, Section 2.3).
 *   - Supported: N, D, H, W >= 1; 1 <= C <= 1024; O in {4, 8, 16, 32, 64};
 *     K in {1, 3, 5, 7}.
 */
#ifndef PYRAMID_LSTM_H
#define PYRAMID_LSTM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum plstm_status {
    PLSTM_OK = 0,
    PLSTM_EINVAL = -1,          /* null pointer, bad dimension or alignment */
    PLSTM_EUNSUPPORTED = -2,    /* valid but not supported (O, dtype, size) */
    PLSTM_EWORKSPACE = -3,      /* ws_bytes smaller than the required size */
    PLSTM_EHIP = -4,            /* a HIP runtime call or launch failed */
    PLSTM_ENOTCORESIDENT = -5,  /* the GPU cannot hold the persistent grid */
    PLSTM_ESCRATCH = -6         /* more scratch than pyramid_lstm_forward_noalloc holds */
};

enum plstm_dtype { PLSTM_F32 = 0, PLSTM_BF16 = 1 };

typedef struct plstm_shape {
    int32_t N, D, H, W;   /* batch and volume extents */
    int32_t C;            /* input channels */
    int32_t O;            /* hidden units per direction */
    int32_t dtype;        /* enum plstm_dtype */
    int32_t K;            /* filter size (odd, 1..7) of wx and wh; 0 means 3 */
} plstm_shape;

/* Shape of a 2D PyraMiD-LSTM layer over images (see pyramid_lstm2d_forward). */
typedef struct plstm2d_shape {
    int32_t N, H, W;      /* batch and image extents */
    int32_t C;            /* input channels */
    int32_t O;            /* hidden units per direction */
    int32_t dtype;        /* enum plstm_dtype */
    int32_t K;            /* filter length (odd, 1..7) along the line; 0 means 3 */
} plstm2d_shape;

/* Human-readable name of a status code (static string, never NULL). */
const char *pyramid_lstm_status_string(int status);

/* Bytes of device workspace `ws` needed by pyramid_lstm_forward (training = 0
 * or 1) and pyramid_lstm_backward (training = 1 covers both).  Returns 0 for an
 * invalid or unsupported shape. */
size_t pyramid_lstm_workspace_size(const plstm_shape *s, int training);

/* Bytes of the `saved` buffer that a training forward fills and the backward
 * reads: three fp32 arrays, each starting at the next 256-byte boundary,
 *   gates [6][N][D][H][W][4O]  i, f, g, o of Eq. (7)-(10) after the nonlinearity
 *   c^d   [6][N][D][H][W][O]   cell states, Eq. (11)
 *   h^d   [6][N][D][H][W][O]   per-direction outputs, Eq. (12)
 * with directions in the order z+, z-, y+, y-, x+, x-.  Returns 0 for an
 * invalid or unsupported shape. */
size_t pyramid_lstm_saved_size(const plstm_shape *s);

/* Forward pass of one layer, Eq. (7)-(13).
 *   x, wx, wh, b : inputs (layouts above), read only.
 *   h            : output [N][D][H][W][O], overwritten.
 *   saved        : NULL for inference; else pyramid_lstm_saved_size() bytes,
 *                  overwritten with what pyramid_lstm_backward needs.
 *   ws, ws_bytes : scratch of at least pyramid_lstm_workspace_size(s, saved != NULL)
 *                  bytes; contents undefined on return.
 * Returns PLSTM_OK or a negative status. */
int pyramid_lstm_forward(const plstm_shape *s, const void *x, const void *wx,
                         const void *wh, const void *b, void *h, void *saved,
                         void *ws, size_t ws_bytes, void *stream);

/* Inference forward for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): pyramid_lstm_forward with saved = NULL, whose workspace is
 * instead a scratch array that the library holds on every GPU it runs on
 * (PLSTM_NOALLOC_SCRATCH_BYTES per GPU, until the process ends).  The call
 * allocates nothing.  Arguments, layouts and results are those of
 * pyramid_lstm_forward.  Returns PLSTM_ESCRATCH when the shape needs more
 * than the scratch (pyramid_lstm_workspace_size(s, 0) tells); e.g. a layer
 * of 16 units with C <= 4 needs about 840 bytes per voxel, so a 64^3 volume
 * (262 k voxels) fits.  Every call on a GPU uses
 * that GPU's one array, so calls that overlap on one GPU (other streams, or
 * other host threads) race and must be serialised by the caller; a call on
 * one stream after another needs nothing more, since each call writes the
 * scratch before reading it. */
#define PLSTM_NOALLOC_SCRATCH_BYTES (256u << 20)
int pyramid_lstm_forward_noalloc(const plstm_shape *s, const void *x, const void *wx,
                                 const void *wh, const void *b, void *h, void *stream);

/* Backward pass of one layer: back-propagation through the six sweeps (the
 * chain rule through Eq. (7)-(13); the paper trains the layer by gradient
 * descent, Section 3 "Training").  fp32 only.
 *   x, wx, wh, b : the forward's inputs; saved: the forward's saved buffer.
 *   dh           : dL/dh [N][D][H][W][O].
 *   dx           : NULL, or dL/dx [N][D][H][W][C], overwritten.
 *   dwx, dwh, db : dL/dwx, dL/dwh, dL/db in the layouts of wx, wh, b, summed
 *                  over the batch, overwritten.
 *   ws, ws_bytes : at least pyramid_lstm_workspace_size(s, 1) bytes.
 * Returns PLSTM_OK or a negative status. */
int pyramid_lstm_backward(const plstm_shape *s, const void *x, const void *wx,
                          const void *wh, const void *b, const void *saved,
                          const void *dh, void *dx, void *dwx, void *dwh, void *db,
                          void *ws, size_t ws_bytes, void *stream);

/* Per-voxel fully connected layer squashed by tanh (Section 2.3,
 * "Fully-Connected Layer"):  y[m][o] = tanh(sum_i w[o][i] x[m][i] + b[o]).
 *   x [M][Cin], w [Cout][Cin], b [Cout], y [M][Cout]; storage `dtype` for all
 *   four (fp32 accumulation).  1 <= Cin, Cout <= 1024. */
int pyramid_fc_tanh_forward(int64_t M, int32_t Cin, int32_t Cout, int32_t dtype,
                            const void *x, const void *w, const void *b, void *y,
                            void *stream);

/* Bytes of workspace for pyramid_fc_tanh_backward / pyramid_softmax_ce / _sq. */
size_t pyramid_fc_workspace_size(int64_t M, int32_t Cin, int32_t Cout);

/* Gradient of pyramid_fc_tanh_forward (fp32): given x, w, the forward's output
 * y and dL/dy, writes dL/dx (nullable) [M][Cin], dL/dw [Cout][Cin] and dL/db
 * [Cout] (overwritten; deterministic reduction order). */
int pyramid_fc_tanh_backward(int64_t M, int32_t Cin, int32_t Cout, const void *x,
                             const void *w, const void *y, const void *dy, void *dx,
                             void *dw, void *db, void *ws, size_t ws_bytes, void *stream);

/* Last fully connected layer + per-voxel softmax (Fig. 3; Section 2.3):
 *   p[m][k] = softmax_k(sum_i w[k][i] x[m][i] + b[k]),  1 <= K <= 16.
 *   x [M][Cin], w [K][Cin], b [K] in storage `dtype`; p [M][K] fp32 output.
 * If labels (int32 [M], values in [0, K)) is non-NULL, also writes the mean
 * cross-entropy over the M voxels to *loss (one fp32 on the device) and, when
 * dx/dw/db are non-NULL (fp32 only), its gradient: dL/dx [M][Cin],
 * dL/dw [K][Cin], dL/db [K] (overwritten).  ws: pyramid_fc_workspace_size(M,
 * Cin, K) bytes when labels is non-NULL, else may be NULL. */
int pyramid_softmax_ce(int64_t M, int32_t Cin, int32_t K, int32_t dtype, const void *x,
                       const void *w, const void *b, const int32_t *labels, void *p,
                       void *loss, void *dx, void *dw, void *db, void *ws,
                       size_t ws_bytes, void *stream);

/* As pyramid_softmax_ce, with the squared loss of Section 3 ("Training",
 * Eq. (14)) instead of the cross-entropy: with y the one-hot label,
 *   loss = (1/M) sum_m sum_k (p[m][k] - y[m][k])^2,
 * and its gradient through the softmax.  Same arguments, layouts and
 * workspace. */
int pyramid_softmax_sq(int64_t M, int32_t Cin, int32_t K, int32_t dtype, const void *x,
                       const void *w, const void *b, const int32_t *labels, void *p,
                       void *loss, void *dx, void *dw, void *db, void *ws,
                       size_t ws_bytes, void *stream);

/* The output end of inference in one pass over the rows (Section 2.3,
 * "Fully-Connected Layer"; Fig. 3): the last per-voxel fully connected layer
 * with tanh, then the per-voxel linear layer and softmax,
 *   y = tanh(w1 x + b1) (rounded to the storage type),  p = softmax(w2 y + b2),
 * without writing y.  x [M][Cin], w1 [F][Cin], b1 [F], w2 [K][F], b2 [K] in
 * `dtype`; p [M][K] fp32, overwritten.  All pointers device memory, 16-byte
 * aligned, owned by the caller; runs on `stream`.  y equals
 * pyramid_fc_tanh_forward's output bit for bit and p equals
 * pyramid_softmax_ce's (no labels) up to the order of fp32 sums.  Covers bf16
 * storage with Cin 32 or 64, F 32, 64 or 128 and K <= 16
 * (pyramid_head_forward_supported returns 1 for those, 0 otherwise); other
 * shapes return PLSTM_EUNSUPPORTED, bad sizes or pointers PLSTM_EINVAL. */
int pyramid_head_forward_supported(int32_t dtype, int32_t Cin, int32_t F, int32_t K);
int pyramid_head_forward(int64_t M, int32_t Cin, int32_t F, int32_t K, int32_t dtype,
                         const void *x, const void *w1, const void *b1, const void *w2,
                         const void *b2, void *p, void *stream);

/* Bytes of workspace for pyramid_head_train, or 0 when the fused kernel does
 * not cover (Cin, F, K). */
size_t pyramid_head_workspace_size(int64_t M, int32_t Cin, int32_t F, int32_t K);

/* The output end of a training step in one pass over the rows (fp32): the
 * last per-voxel fully connected layer with tanh, the per-voxel linear layer
 * + softmax and the mean cross-entropy (Section 2.3, "Fully-Connected Layer";
 * Fig. 3), with the gradients of the loss:
 *   y = tanh(w1 x + b1),  p = softmax(w2 y + b2),
 *   loss = (1/M) sum_m -log p[m][labels[m]].
 *   x [M][Cin] (16-byte aligned rows), w1 [F][Cin], b1 [F], w2 [K][F], b2 [K],
 *   labels int32 [M] in [0, K) (an out-of-range label makes loss and the
 *   gradients NaN).  Outputs, all overwritten: p [M][K], *loss (one float),
 *   dx = dL/dx [M][Cin] (nullable), dw1 [F][Cin], db1 [F], dw2 [K][F], db2 [K].
 * Gives the same values as pyramid_fc_tanh_forward + pyramid_softmax_ce +
 * pyramid_fc_tanh_backward (deterministic sums, fixed order).  Covers
 * (Cin, F) = (16, 32) and (32, 64) with K <= 16; other shapes return
 * PLSTM_EUNSUPPORTED (the separate entry points cover every shape).
 * ws: pyramid_head_workspace_size(M, Cin, F, K) bytes. */
int pyramid_head_train(int64_t M, int32_t Cin, int32_t F, int32_t K, const void *x,
                       const void *w1, const void *b1, const void *w2, const void *b2,
                       const int32_t *labels, void *p, void *loss, void *dx, void *dw1,
                       void *db1, void *dw2, void *db2, void *ws, size_t ws_bytes,
                       void *stream);


/* Failures found on the device after a call returned PLSTM_OK.
 * The persistent sweeps (forward and reverse, 16 hidden units) hand the
 * 1-pixel halo between strips of a plane through step flags (Section 2.3:
 * each plane's convolution reads its neighbours' previous plane).  Every wait
 * on a flag is bounded, so a neighbour that never arrives cannot hang the
 * GPU: the wait gives up, the grid drains, and the call's outputs are
 * overwritten with NaN (h and the saved h^d of the forward; dx, dwx, dwh, db
 * of the backward).  The failure also raises a bit in this device's sticky
 * status word:
 *   PLSTM_DEVICE_WAIT_GAVE_UP   a persistent sweep's wait gave up.
 * pyramid_lstm_device_status synchronises `stream`, writes the current
 * device's status bits to *status (host memory; 0 = no failure since the last
 * clear) and, when `clear` is non-zero, resets them.  Returns PLSTM_EINVAL
 * for a null `status`, PLSTM_EHIP when the copy or the synchronisation fails.
 * The word is shared by every caller on the device. */
enum { PLSTM_DEVICE_WAIT_GAVE_UP = 1 };
int pyramid_lstm_device_status(int32_t *status, int32_t clear, void *stream);

/* Failure-path test mode (process-wide, for tests): with on = 1 every wait of
 * the persistent sweeps expects a step no strip ever publishes and gives up
 * after 16 polls, so each such launch takes the path above and still
 * finishes normally; on = 0 (default) restores the normal waits.  Returns
 * PLSTM_EINVAL for other values. */
int pyramid_lstm_set_wait_test(int on);


/* Optional kernel timing for measurement tools (off by default).
 * pyramid_lstm_timing_enable(1) clears earlier records and makes every later
 * call of this library in the process record a pair of HIP events on its
 * stream around each kernel phase ("sweep_fwd", "sum_dirs", "sweep_bwd",
 * "wgrad", "dx", ...); pyramid_lstm_timing_enable(0) clears and stops.
 * pyramid_lstm_timing_read waits for the recorded events and writes, per
 * distinct phase (at most max_phases): its name into names[32*k .. 32*k+31]
 * (NUL-terminated), the summed milliseconds into ms[k] and the number of
 * kernel launches into launches[k]; *count receives the number of phases. */
int pyramid_lstm_timing_enable(int on);
int pyramid_lstm_timing_read(int max_phases, char *names, double *ms, int *launches,
                             int *count);


/* ---- 2D PyraMiD-LSTM (Section 2.1-2.2, Fig. 1) -------------------------- */

/* The layer over images: 2 x 2 = 4 directions instead of 6.  Direction
 * 0 = y+ sweeps the rows top to bottom (each step a row of W pixels),
 * 1 = y- bottom to top, 2 = x+ sweeps the columns left to right (each step a
 * column of H pixels), 3 = x- right to left.  At each step a pixel's gates
 * take a 1D convolution of length K along the line of the input line and of
 * the previous line's h (the rotated connections of Fig. 1 (b)-(c)), then the
 * cell update of Eq. (10)-(12); h = sum of the four directions.
 *   x   [N][H][W][C]     h [N][H][W][O]
 *   wx  [4][4*O][C][K]   wh [4][4*O][O][K]   b [4][4*O]
 *   A[q][g*O+o] += in[q+k-r][c] * w[g*O+o][c][k], r = (K-1)/2, q along the
 *   line, zero padding.
 * Entry points mirror the 3D ones (same conventions, workspace and saved
 * buffers sized by the 2D functions; the saved layout has 4 directions).
 * Supported: as the 3D layer with D = 1. */
size_t pyramid_lstm2d_workspace_size(const plstm2d_shape *s, int training);
size_t pyramid_lstm2d_saved_size(const plstm2d_shape *s);
int pyramid_lstm2d_forward(const plstm2d_shape *s, const void *x, const void *wx,
                           const void *wh, const void *b, void *h, void *saved, void *ws,
                           size_t ws_bytes, void *stream);
int pyramid_lstm2d_backward(const plstm2d_shape *s, const void *x, const void *wx,
                            const void *wh, const void *b, const void *saved, const void *dh,
                            void *dx, void *dwx, void *dwh, void *db, void *ws,
                            size_t ws_bytes, void *stream);

/* ---- training update (Section 3, "Training") ---------------------------- */

/* One parameter tensor for pyramid_rmsprop_step: n fp32 elements of the
 * parameters theta (updated in place), their gradient grad (read), and the
 * optimiser state ms (running mean of grad^2) and mom (smoothed normalised
 * gradient), both updated in place and zero before the first step.  All
 * device pointers, 4-byte aligned, owned by the caller. */
typedef struct plstm_param_segment {
    float *theta;
    const float *grad;
    float *ms;
    float *mom;
    int64_t n;
} plstm_param_segment;

/* RMS-prop with momentum, Eq. (15)-(18), over `count` (1..64) tensors in one
 * launch: ms = rho_ms ms + (1 - rho_ms) g^2; G = g / (sqrt(ms) + eps);
 * mom = rho_m mom + (1 - rho_m) G; theta -= lr mom.  The paper's values are
 * rho_ms = rho_m = 0.9 and eps = 1e-5, with lr from
 * pyramid_rmsprop_learning_rate.  `segs` is a host array read before the call
 * returns; segments must not overlap.  Returns PLSTM_EINVAL for a bad count,
 * null or misaligned pointers, negative n, lr < 0, rho outside [0, 1) or
 * eps <= 0. */
int pyramid_rmsprop_step(int32_t count, const plstm_param_segment *segs, float lr,
                         float rho_ms, float rho_m, float eps, void *stream);

/* The decaying learning rate of Section 3: 1e-6 + 1e-2 (2^(-1/100))^epoch
 * (host function). */
double pyramid_rmsprop_learning_rate(int32_t epoch);

/* ---- inference over volumes larger than one pass (Section 3, "Sub-volumes
 * and Augmentation") -------------------------------------------------------- */

/* Copies the sub-volume [z0, z0+d) x [y0, y0+h) x [x0, x0+w) of batch element n
 * of x [N][D][H][W][C] (storage `dtype`) into tile [d][h][w][C], same type.
 * The box must lie inside the volume (else PLSTM_EINVAL); 4-byte aligned
 * device pointers. */
int pyramid_crop(int32_t N, int32_t D, int32_t H, int32_t W, int32_t C, int32_t dtype,
                 int32_t n, int32_t z0, int32_t y0, int32_t x0, int32_t d, int32_t h, int32_t w,
                 const void *x, void *tile, void *stream);

/* Training cubes (Section 3, "Sub-volumes and Augmentation"): cubes cut at
 * random positions, possibly turned about z by a random angle and flipped
 * along any axis.  The caller draws the randomness and passes one plstm_cube
 * per cube (a host array, copied into the launch; at most PLSTM_MAX_CUBES):
 *   n                 batch element of x;
 *   (z0, y0, x0)      corner of the unrotated d x h x w box, which must lie
 *                     inside the volume;
 *   cos_t, sin_t      cosine and sine of the rotation about z (in [-1, 1]);
 *   flips             bit set of PLSTM_FLIP_Z / _Y / _X.
 * Cube voxel (k, i, j), before the flips, reads the source position
 *   z = z0 + k, y = yc + c u - s v, x = xc + s u + c v,
 *   u = i - (h - 1) / 2, v = j - (w - 1) / 2, (yc, xc) the box's centre,
 * computed in fp64 and clamped to the slice; image values are bilinear in
 * (y, x) (fp64 weights and blend, rounded to the storage type), labels take
 * the nearest voxel floor(y + 1/2).  The
 * flips then act on the cube: out[k][i][j] = cube[k'][i'][j'] with
 * k' = d - 1 - k when z is flipped (likewise y, x).
 * x [N][D][H][W][C] (dtype), labels [N][D][H][W] int32 or NULL;
 * out [count][d][h][w][C] (dtype), out_labels [count][d][h][w] (required when
 * labels is given).  Device buffers, caller-owned; work on `stream`.
 * Returns PLSTM_EINVAL for null or misaligned pointers, a cube outside the
 * volume, count outside 1..PLSTM_MAX_CUBES, flips > 7 or |cos|, |sin| > 1. */
enum { PLSTM_FLIP_Z = 1, PLSTM_FLIP_Y = 2, PLSTM_FLIP_X = 4 };
#define PLSTM_MAX_CUBES 64
typedef struct plstm_cube {
    int32_t n, z0, y0, x0;
    float cos_t, sin_t;
    int32_t flips;
} plstm_cube;
int pyramid_sample_cubes(int32_t N, int32_t D, int32_t H, int32_t W, int32_t C, int32_t dtype,
                         int32_t count, const plstm_cube *cubes, int32_t d, int32_t h, int32_t w,
                         const void *x, const int32_t *labels, void *out, int32_t *out_labels,
                         void *stream);

/* Gaussian-weighted stitching of per-voxel class probabilities (fp32) into a
 * D x H x W volume with K classes.  acc [D][H][W][K] and wsum [D][H][W] are
 * caller-owned fp32 device buffers:
 *   pyramid_stitch_clear   zeroes them;
 *   pyramid_stitch_add     adds tile p [d][h][w][K] placed at (z0, y0, x0):
 *                          acc += g p, wsum += g, with g the separable Gaussian
 *                          exp(-1/2 sum_axes ((i - c) / (sigma_scale * n))^2)
 *                          over the tile (c its centre, n its extent per axis);
 *   pyramid_stitch_finish  out [D][H][W][K] = acc / wsum (every voxel must have
 *                          been covered by a tile).
 * Calls on one stream accumulate in call order (deterministic).  Returns
 * PLSTM_EINVAL for null pointers, a box outside the volume or
 * sigma_scale <= 0. */
int pyramid_stitch_clear(int32_t D, int32_t H, int32_t W, int32_t K, void *acc, void *wsum,
                         void *stream);
int pyramid_stitch_add(int32_t D, int32_t H, int32_t W, int32_t K, int32_t z0, int32_t y0,
                       int32_t x0, int32_t d, int32_t h, int32_t w, float sigma_scale,
                       const void *p, void *acc, void *wsum, void *stream);
int pyramid_stitch_finish(int32_t D, int32_t H, int32_t W, int32_t K, const void *acc,
                          const void *wsum, void *out, void *stream);

/* Forward implementation selection, for testing and tuning (process-wide):
 * 0 = automatic (default): the persistent MFMA sweep where it supports the
 * shape (fp32, O = 16, C <= 4, grid co-resident), else the plane-step MFMA
 * path where it does (O = 16, 32 or 64, C <= 64), else the generic path;
 * 1 = generic path only; 2 = same as 0; 3 = as 0, but the persistent sweep
 * stages every strip chunk by chunk (no strip kept whole in LDS); 4 = the
 * plane-step MFMA path where it supports the shape, else the generic path.
 * Returns PLSTM_EINVAL for other values. */
int pyramid_lstm_set_forward_path(int path);

/* Backward implementation selection, for testing and tuning (process-wide):
 * 0 = automatic (default): persistent MFMA reverse sweep, else plane-step
 * MFMA path, else generic (same shape rules as the forward); 1 = generic
 * per-plane path only; 2 = as 0, but the persistent reverse sweep stages
 * every strip chunk by chunk (no strip kept whole in LDS); 3 = the
 * plane-step MFMA path where it supports the shape, else the generic path.  Returns PLSTM_EINVAL for
 * other values. */
int pyramid_lstm_set_backward_path(int path);

/* Launch shape of the plane-step MFMA path, for testing and tuning
 * (process-wide): 0 = automatic (default): the reverse step (16 or 32 units)
 * runs on 64-pixel blocks with dA_{t+1} staged in LDS, its K split over a
 * workgroup's four waves; a forward step whose tiles would give fewer than
 * about two waves per SIMD splits each tile's K dimension over the four
 * waves of a workgroup, other steps give each wave its own tiles;
 * 1 = always split (the reverse step's operands read from L1); 2 = never
 * split; 3 = never split, and the forward's operands read from L1 per
 * filter tap instead of from 64-pixel blocks staged in LDS (the default for
 * fp32 steps that are not split).  Results are identical up to summation
 * order.  Returns PLSTM_EINVAL for other values. */
int pyramid_lstm_set_step_split(int mode);

/* Contraction type of bf16-storage layers with 32 or 64 hidden units, for
 * testing and tuning (process-wide): 1 = bf16 MFMA with fp32 accumulation
 * (default; h_{t-1} enters the recurrent contraction rounded to bf16) on
 * 256-pixel blocks, the block staged in LDS once for all filter taps and the
 * weights streamed through LDS for all of a workgroup's waves (3 where its
 * LDS does not fit, e.g. 64 units with 5 x 5 filters); 3 = the same
 * contraction on 64-pixel blocks, the weights read by each wave from L1;
 * 2 = operands read from L1 per tap; 0 = fp32 MFMA on the widened values;
 * 4 = as 1, but 16-unit layers (3D, at most 8 input channels, which take
 * the bf16 MFMA on packed taps under 1 and 4 only) run one plane per launch
 * instead of two; 5 = for 32 and 64 units, x's contraction for every plane
 * first (one launch writing bf16 pre-activations, 2 bytes per gate-unit and
 * voxel-direction of workspace), then the recurrent contraction plane by
 * plane (an all-plane input projection; slower than 1, kept for measurement).
 * Results of 1, 2 and 3 differ only in summation order, 1 and 4 not at all;
 * 5 also rounds x's part of the pre-activations to bf16.  Returns
 * PLSTM_EINVAL for other values. */
int pyramid_lstm_set_bf16_mfma(int on);

/* Weight gradients of the plane-step backward, for testing and tuning
 * (process-wide): 1 = a staged GEMM (default where it applies: at most 32
 * hidden units and C a multiple of 4): each workgroup stages a 16-voxel unit
 * of dA and of the im2col columns in LDS once for eight waves; 0 = the
 * register-streamed kernel, each wave reading its own operands from memory.
 * Results differ only in summation order.  Returns PLSTM_EINVAL for other
 * values. */
int pyramid_lstm_set_wgrad_staged(int on);

#ifdef __cplusplus
}
#endif

#endif /* PYRAMID_LSTM_H */
