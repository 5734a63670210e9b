/*
 * tfk.h -- C ABI of the MI355X (gfx950) convnet training-step library.
 *
 * The library implements the dataflow operations of one synchronous SGD step
 * of a convolutional network replica (the paper's single-replica hot path,
 * Sections 4.1, 4.4 and 6.1): Conv2D forward, Conv2DBackpropInput,
 * Conv2DBackpropFilter, fused bias+ReLU forward/backward, MaxPool
 * forward/backward with argmax, and in-place ApplyGradientDescent.  The paper
 * separates client languages from the core by a thin C API (Section 5); this
 * header is that boundary for these operations.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensors are dense device arrays (hipMalloc'd or equivalent).  Activations
 *    are NHWC row-major: element (n,h,w,c) lives at
 *      base[((n*H + h)*W + w) * pixel_stride + c].
 *    pixel_stride == 0 means "dense" (= c).  pixel_stride > c describes a
 *    channel slice of a wider buffer (concat without copies).
 *  - Filters are HWIO row-major: w[kh][kw][ci][co], always dense.
 *  - Element types: TFK_F32 (float) or TFK_BF16 (bfloat16 stored as uint16,
 *    round-to-nearest-even on store).  Accumulation is always fp32.  Filter
 *    gradients, bias, bias gradients and variables are always fp32.
 *  - Convolution is cross-correlation (no filter flip) with explicit stride and
 *    padding (top, bottom, left, right).  Output extent along an axis:
 *      OH = floor((H + pad_top + pad_bottom - KH) / stride_h) + 1.
 *    The library never infers SAME/VALID padding; callers pass the pads.
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream) and returns its status synchronously.  Arguments are validated
 *    before anything is launched: on a non-OK status nothing was enqueued and
 *    no buffer was touched.  tfk_last_error() then holds a message.
 *  - Ownership: the caller owns every buffer.  No call allocates device
 *    memory (the library's only memory of its own is the fixed scratch of
 *    tfk_conv2d_bwd_filter_noalloc) and none keeps a pointer after it returns;
 *    buffers must stay valid until the stream has passed the operation.
 *    Operations that need scratch memory take a caller-provided workspace
 *    sized by the matching *_workspace_bytes query.
 *  - Aliasing: outputs must not overlap inputs except where an argument is
 *    documented as in-place.  A detected overlap returns TFK_ERR_ALIAS.  Two
 *    NHWC views with one pixel stride overlap only if they share an element:
 *    channel slices of one buffer that lie side by side within every pixel
 *    (say a concat's branches, one read while another is written) do not.
 *  - An empty batch (n == 0) is valid: nothing is read; reductions over the
 *    batch (filter and bias gradients) are written as zeros.  Pointers of
 *    empty tensors may be NULL.
 *  - Results are deterministic: no floating-point atomics; every reduction has
 *    a fixed order for a given shape.
 */
#ifndef TFK_H_
#define TFK_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TFK_ABI_VERSION 16

#if defined(__GNUC__)
#define TFK_API __attribute__((visibility("default")))
#else
#define TFK_API
#endif

typedef enum {
    TFK_OK = 0,
    TFK_ERR_NULL = 1,       /* a required pointer is NULL                          */
    TFK_ERR_SHAPE = 2,      /* non-positive extent, mismatched shapes, bad window  */
    TFK_ERR_DTYPE = 3,      /* unknown element type                                */
    TFK_ERR_ALIGN = 4,      /* pointer not aligned to its element size             */
    TFK_ERR_OVERFLOW = 5,   /* an index would not fit its integer type             */
    TFK_ERR_ALIAS = 6,      /* an output overlaps an input it may not overlap      */
    TFK_ERR_WORKSPACE = 7,  /* workspace missing or smaller than the query says    */
    TFK_ERR_HIP = 8,        /* the HIP runtime reported an error at launch         */
    TFK_ERR_ARG = 9         /* any other invalid argument (beta, lr, count, ...)   */
} tfk_status;

typedef enum { TFK_F32 = 0, TFK_BF16 = 1 } tfk_dtype;

/* An NHWC tensor view: extents and the distance between consecutive pixels,
 * in elements (0 = c, i.e. dense). */
typedef struct {
    int32_t n, h, w, c;
    int64_t pixel_stride;
} tfk_nhwc;

/* A sliding window: extent, stride and explicit padding. */
typedef struct {
    int32_t kh, kw;
    int32_t stride_h, stride_w;
    int32_t pad_top, pad_bottom, pad_left, pad_right;
} tfk_window;

/* ---------------------------------------------------------------- convolution
 * Conv2D forward (the mini-batch 2-D convolution of Section 3.1):
 *   y[n,oh,ow,co] = sum_{kh,kw,ci} X[n, oh*sh+kh-pt, ow*sw+kw-pl, ci] * w[kh,kw,ci,co]
 * with X = 0 outside the image.
 *   x   : xd-shaped input, element type dt.
 *   w   : dense HWIO filter [kh][kw][xd.c][cout], element type dt.
 *   y   : yd-shaped output, element type dt, overwritten.  yd.n == xd.n,
 *         yd.h/yd.w must equal the output extents, yd.c == cout.
 *   ws  : workspace of at least tfk_conv2d_workspace_bytes(0, ...) bytes
 *         (may be NULL when that is 0).
 * Requirements: pad < kernel extent on every side.
 * A window that covers the whole unpadded image once (a fully connected layer over a
 * densely stored x, output 1 x 1) runs as the 1 x 1 convolution of the flattened image;
 * with few output tiles (small batch) its reduction is split across blocks into fp32
 * partial sums in the workspace, added in a fixed order.  Image inputs (bf16, 1-4 channels) run as an equivalent 8-channel convolution over the
 * input padded to 4 (or 8) channels.  When x is already stored that way -- e.g. a
 * 3-channel view with pixel_stride 4 of an RGBx buffer, 16-byte aligned -- it is read in
 * place and not copied; the channels past xd.c then meet zero filter weights and must
 * hold finite values.  The same holds for tfk_conv2d_bwd_filter.
 */
TFK_API tfk_status tfk_conv2d_fwd(const void *x, tfk_nhwc xd, const void *w, int32_t cout,
                          tfk_window p, tfk_dtype dt, void *y, tfk_nhwc yd,
                          void *ws, size_t ws_bytes, void *stream);

/*
 * Conv2D forward with BiasAdd and ReLU fused into the same kernel (the hand-fused
 * activation kernels of Section 5):
 *   y[n,oh,ow,co] = max(conv(x, w)[n,oh,ow,co] + bias[co], +0)
 * The sum is formed in fp32 and rounded to dt once, when y is stored (the unfused
 * sequence tfk_conv2d_fwd + tfk_bias_relu_fwd rounds the convolution output first).
 *   bias : cout fp32 values, 4-byte aligned, not overlapping y.
 * Everything else, including the workspace query (op 0 of tfk_conv2d_workspace_bytes),
 * is as for tfk_conv2d_fwd.  A NULL bias is TFK_ERR_NULL.
 */
TFK_API tfk_status tfk_conv2d_fwd_bias_relu(const void *x, tfk_nhwc xd, const void *w, int32_t cout,
                                    const float *bias, tfk_window p, tfk_dtype dt, void *y,
                                    tfk_nhwc yd, void *ws, size_t ws_bytes, void *stream);

/*
 * Conv2DBackpropInput: the gradient of the forward map with respect to x
 * (Section 4.1 backpropagation through the convolution):
 *   dx[n,h,w,ci] = sum over (kh,kw,co) and the (oh,ow) with
 *                  oh*sh+kh-pt == h, ow*sw+kw-pl == w of dy[n,oh,ow,co]*w[kh,kw,ci,co].
 * Input positions reached by no window receive 0.
 *   dy  : dyd-shaped upstream gradient (the forward output's shape), type dt.
 *   w   : dense HWIO filter [kh][kw][dxd.c][dyd.c], type dt.
 *   dx  : dxd-shaped gradient (the forward input's shape: with stride > 1 it
 *         cannot be recovered from dy, so the caller states it), type dt.
 *   beta: 0 overwrites dx; 1 adds to it (summing the partial gradients of
 *         several paths, Section 4.1).  With beta == 1, dx is read and written.
 *   ws  : at least tfk_conv2d_workspace_bytes(1, ...) bytes (split-K partial sums
 *         of fully connected layers at small batch, see tfk_conv2d_fwd; may be NULL
 *         when that is 0).
 */
TFK_API tfk_status tfk_conv2d_bwd_input(const void *dy, tfk_nhwc dyd, const void *w, tfk_window p,
                                tfk_dtype dt, void *dx, tfk_nhwc dxd, float beta,
                                void *ws, size_t ws_bytes, void *stream);

/*
 * Conv2DBackpropFilter: the gradient with respect to the filter (Section 4.1: the
 * backpropagation that the differentiation library derives, whose filter gradients are
 * what the SGD update consumes; Section 6.1 places convolution on the training critical path):
 *   dw[kh,kw,ci,co] = sum_{n,oh,ow} X[n, oh*sh+kh-pt, ow*sw+kw-pl, ci] * dy[n,oh,ow,co]
 *   x   : xd-shaped forward input, type dt.
 *   dy  : dyd-shaped upstream gradient, type dt.
 *   dw  : dense fp32 HWIO [p.kh][p.kw][xd.c][dyd.c], overwritten.
 *   ws  : at least tfk_conv2d_workspace_bytes(2, ...) bytes (split-K partial sums,
 *         reduced in a fixed order).
 * An image input stored with its pixels 4 (or 8) channels apart is read in place as
 * described at tfk_conv2d_fwd (the channels past xd.c must be finite).
 */
TFK_API tfk_status tfk_conv2d_bwd_filter(const void *x, tfk_nhwc xd, const void *dy, tfk_nhwc dyd,
                                 tfk_window p, tfk_dtype dt, float *dw,
                                 void *ws, size_t ws_bytes, void *stream);

/*
 * tfk_conv2d_bwd_filter for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same operation and
 * arguments without the workspace, which is replaced by a scratch array the library keeps in
 * device memory, 128 MiB per GPU, held from the library's load on that GPU until the process
 * ends.  The call allocates nothing.
 *   stream : must belong to the calling thread's current device (else TFK_ERR_HIP).
 * Errors: as tfk_conv2d_bwd_filter; TFK_ERR_WORKSPACE when the shape needs more scratch than
 * 128 MiB (tfk_conv2d_workspace_bytes(2, ...) tells how much it needs).
 * Every call on one GPU uses that GPU's one scratch array: calls that overlap in time on one
 * GPU (on different streams, or from different threads) race and give wrong results; calls
 * ordered on one stream do not.  No scratch content needs to start at zero.
 */
TFK_API tfk_status tfk_conv2d_bwd_filter_noalloc(const void *x, tfk_nhwc xd, const void *dy, tfk_nhwc dyd,
                                         tfk_window p, tfk_dtype dt, float *dw, void *stream);

/*
 * Conv2DBackpropInput fused with the ReLU backward and bias gradient of the layers that
 * produced x (the hand-fused activation-gradient kernels of Section 5), for an x whose
 * channels are all outputs y of BiasAdd + ReLU, when this convolution is the last of x's
 * readers to add its gradient (beta = 1 adds it to what the others stored in dpre; Section
 * 4.1's sum of the gradients of several paths):
 *   g        = the input gradient of tfk_conv2d_bwd_input
 *   dpre[i]  = y[i] > 0 ? beta * dpre[i] + g[i] : +0   (xd-shaped, rounded to dt once when stored)
 *   dbias[c] = sum over the pixels of dpre[., c]   (fp32, of the stored values)
 * It equals tfk_conv2d_bwd_input(..., dx = dpre, beta) followed by tfk_bias_relu_bwd(y,
 * dpre, ...) up to the order of the fp32 bias-gradient sums, without forming g in memory.
 *   dy, dyd, w, p, dt : as tfk_conv2d_bwd_input.
 *   y     : xd-shaped (the same view as dpre), the forward ReLU output; read only.
 *   dpre  : xd-shaped, overwritten; must not overlap dy, w, y or dbias.
 *   dbias : xd.c fp32 values, overwritten; or NULL: deferred (see tfk_bias_grad_finish).
 *   ws    : at least tfk_conv2d_workspace_bytes(3, xd, dyd.c, p, dt) bytes.
 * Requirements: beta is 0 or 1 (else ARG); xd.c <= 16384.  xd.n == 0 sets dbias to 0.
 */
TFK_API tfk_status tfk_conv2d_bwd_input_relu_bwd(const void *dy, tfk_nhwc dyd, const void *w, tfk_window p,
                                         tfk_dtype dt, const void *y, void *dpre, tfk_nhwc xd, float beta,
                                         float *dbias, void *ws, size_t ws_bytes, void *stream);

/* Workspace needed by a convolution (of the Section 4.1 forward and gradient operations
 * above): op 0 = forward, 1 = backprop-input,
 * 2 = backprop-filter, 3 = backprop-input fused with the ReLU backward;
 * xd is the forward input, cout the filter's output channels.  Returns 0
 * for invalid arguments (the operation itself then reports the error). */
TFK_API size_t tfk_conv2d_workspace_bytes(int32_t op, tfk_nhwc xd, int32_t cout, tfk_window p,
                                  tfk_dtype dt);

/* ---------------------------------------------------------------- bias + ReLU
 * Fused BiasAdd + ReLU forward, in place (the hand-fused ReLU kernels of
 * Section 5):  y[p,c] <- max(y[p,c] + bias[c], +0).
 *   y    : yd-shaped, type dt, read and written.
 *   bias : fp32 [yd.c].
 */
TFK_API tfk_status tfk_bias_relu_fwd(void *y, tfk_nhwc yd, const float *bias, tfk_dtype dt,
                             void *stream);

/*
 * ReLU backward fused with the bias gradient (Section 5: the hand-fused kernels of the
 * ReLU activation and its gradient; the bias gradient is the BiasAdd gradient of
 * Section 4.1's backpropagation, summed in the same pass):
 *   dpre[p,c] = (y[p,c] > 0) ? dy[p,c] : 0        (mask from the stored y)
 *   dbias[c]  = sum over all pixels p of dpre[p,c]  (fp32, fixed order)
 *   y, dy, dpre : share the view yd (same extents and pixel stride), type dt.
 *                 dpre may equal dy (in place); any other overlap is an error.
 *   dbias       : fp32 [yd.c], overwritten; or NULL: deferred (see tfk_bias_grad_finish).
 *   ws          : at least tfk_bias_relu_bwd_workspace_bytes(yd, dt) bytes.
 * y may be NULL: a layer with a bias and no ReLU (a classifier's logits), so
 * dpre = dy and dbias holds the column sums of dy.
 */
TFK_API tfk_status tfk_bias_relu_bwd(const void *y, const void *dy, tfk_nhwc yd, void *dpre,
                             float *dbias, tfk_dtype dt, void *ws, size_t ws_bytes,
                             void *stream);

TFK_API size_t tfk_bias_relu_bwd_workspace_bytes(tfk_nhwc yd, tfk_dtype dt);

/*
 * Deferred bias gradients.  Every call that forms a bias gradient from per-block partial sums
 * (tfk_bias_relu_bwd, tfk_conv2d_bwd_input_relu_bwd, tfk_maxpool_bwd_relu_bwd[_taps]) sums
 * them per channel in a second short launch.  Given dbias = NULL it launches only the first:
 * the partials stay in its workspace (channel c's `rows` values at part[c * rows ...]), and
 * tfk_bias_grad_finish later sums the partials that several such calls left, all in one
 * launch, each channel in the same fixed order as the call itself would have summed it (the
 * same bits).  A step issues its bias gradients this way and finishes them together before
 * its update (Section 4.1: every gradient of the step is formed before the update; Section 5:
 * fewer, larger launches).  The caller keeps each deferred call's workspace untouched until
 * the finish has run on the same stream (or after it on another).
 *
 * tfk_last_bias_partials: where the last call on this thread that was given dbias = NULL left
 * its partials (*part inside that call's workspace, *rows per channel; 0 rows: an empty
 * tensor, whose bias gradient is 0).  Errors: NULL (part or rows), ARG (no such call yet).
 */
TFK_API tfk_status tfk_last_bias_partials(const float **part, int32_t *rows);
/*
 * tfk_bias_grad_finish: for i < count, dbias[i][c] = the fixed-order sum of the rows[i]
 * partials of channel c at parts[i] (c < channels[i]).  The arrays are the caller's (read
 * during the call only).  count 0 is a no-op.  Errors: ARG (count < 0), NULL (an array,
 * dbias[i], or parts[i] with rows[i] > 0), SHAPE (rows[i] < 0, channels[i] outside 1..16384),
 * ALIGN (4 bytes), ALIAS (a dbias[i] overlapping partials or another dbias).
 */
TFK_API tfk_status tfk_bias_grad_finish(int32_t count, const float *const *parts, const int32_t *rows,
                                const int32_t *channels, float *const *dbias, void *stream);

/* ---------------------------------------------------------------- max-pool
 * MaxPool forward with argmax (Section 6.1: pooling, with convolution, is on the
 * critical path of the training step).  Each window scans kh (outer) and kw (inner),
 * skipping padded taps; the first maximum in that order wins (a later tap
 * replaces the running maximum only if strictly greater).
 *   x      : xd-shaped input, type dt.
 *   y      : yd-shaped output, type dt, overwritten.
 *   argmax : dense int32 [yd.n][yd.h][yd.w][yd.c]: the flat dense NHWC index
 *            ((n*H + h)*W + w)*C + c into x of the selected tap.
 * Requirements: every window holds at least one in-bounds tap (pad < kernel
 * extent); xd.n*xd.h*xd.w*xd.c <= INT32_MAX (else TFK_ERR_OVERFLOW).
 */
TFK_API tfk_status tfk_maxpool_fwd(const void *x, tfk_nhwc xd, tfk_window p, tfk_dtype dt,
                           void *y, tfk_nhwc yd, int32_t *argmax, void *stream);

/*
 * MaxPool forward (Section 6.1, as tfk_maxpool_fwd) with the selection stored
 * compactly: taps is dense uint8
 * [yd.n][yd.h][yd.w][yd.c] holding the selected window tap kh * p.kw + kw (the
 * element ((n*H + oh*sh - pt + kh)*W + ow*sw - pl + kw)*C + c of x), a quarter
 * of the int32 argmax's bytes.  Requires p.kh * p.kw <= 256.  The _taps backward
 * entry points below take it in place of the argmax.
 */
TFK_API tfk_status tfk_maxpool_fwd_taps(const void *x, tfk_nhwc xd, tfk_window p, tfk_dtype dt,
                                void *y, tfk_nhwc yd, uint8_t *taps, void *stream);

/*
 * Conv2D + BiasAdd + ReLU followed by MaxPool of its output, in one call (Section 5: kernels
 * hand-fused for performance-critical operations, kernel fusion being the direction the paper
 * names; Section 6.1: convolution and pooling on the critical path):
 *   y        = tfk_conv2d_fwd_bias_relu(x, w, bias)          (yd-shaped, written)
 *   py, taps = tfk_maxpool_fwd_taps(y, pp)                   (pyd-shaped pool of y, uint8 taps)
 * with the same values, bit for bit, as those two calls.  Where the convolution's output tiles
 * can be laid out as bands of whole image rows that hold whole pool windows (bf16, a VALID pool,
 * at most 192 output pixels per band), one kernel computes y, keeps each band in LDS and pools
 * it there; other shapes run the two kernels.
 *   x, xd, w, cout, bias, p, dt, y, yd, ws : as tfk_conv2d_fwd_bias_relu (bias required).
 *   pp   : the pool window over y (kh * kw <= 256).
 *   py   : pyd-shaped, type dt, overwritten.   taps : dense uint8 [pyd.n][pyd.h][pyd.w][pyd.c].
 * Errors: as the two calls; py and taps must not overlap x, w, y, bias or each other.
 */
TFK_API tfk_status tfk_conv2d_fwd_bias_relu_maxpool(const void *x, tfk_nhwc xd, const void *w, int32_t cout,
                                            const float *bias, tfk_window p, tfk_dtype dt, void *y, tfk_nhwc yd,
                                            tfk_window pp, void *py, tfk_nhwc pyd, uint8_t *taps, void *ws,
                                            size_t ws_bytes, void *stream);

/*
 * MaxPool backward (Section 6.1 pooling on the critical path; Section 4.1
 * backpropagation, beta = 1 summing the partial gradients of several paths):
 * dx[i] = beta*dx[i] + sum over outputs o with argmax[o] == i of dy[o]
 * (overlapping windows may route several outputs to one input; all are summed).
 *   dy, argmax : yd-shaped (argmax dense), from tfk_maxpool_fwd.
 *   dx         : xd-shaped, type dt; beta 0 overwrites, 1 accumulates.
 */
TFK_API tfk_status tfk_maxpool_bwd(const void *dy, const int32_t *argmax, tfk_nhwc yd, tfk_window p,
                           tfk_dtype dt, void *dx, tfk_nhwc xd, float beta, void *stream);
/* tfk_maxpool_bwd (Section 6.1, Section 4.1) with the selection from tfk_maxpool_fwd_taps. */
TFK_API tfk_status tfk_maxpool_bwd_taps(const void *dy, const uint8_t *taps, tfk_nhwc yd, tfk_window p,
                                tfk_dtype dt, void *dx, tfk_nhwc xd, float beta, void *stream);

/*
 * MaxPool backward, ReLU backward and the bias gradient fused into one pass (the
 * hand-fused activation-gradient kernels of Section 5), for a max-pool whose input y is the
 * output of BiasAdd + ReLU:
 *   g[i]     = beta * dpre[i] + sum over pool outputs o with argmax[o] == i of dy[o]
 *   dpre[i]  = y[i] > 0 ? g[i] : +0              (element i of the pool input, dense index)
 *   dbias[c] = sum over the pixels of dpre[., c]  (of the stored values; fp32)
 * It equals tfk_maxpool_bwd(dy, argmax, ..., dx = dpre, beta) followed by
 * tfk_bias_relu_bwd(y, dpre, ...), with the pool gradient rounded once instead of twice.
 * When beta = 0 the mask can come from the pool's output instead of y: an element receives
 * gradient only from windows whose argmax it is, and each such window's output is exactly the
 * element's value, so routing +0 from windows whose output is not positive gives the same
 * dpre, bit for bit, without reading y (a quarter of the bytes for a 2x2- or 3x3-stride-2 pool).
 *   dy, argmax, yd, p : the max-pool's output gradient, its tfk_maxpool_fwd argmax and window.
 *   y     : xd-shaped pool input (the ReLU output), element type dt; read only.  Not read, and
 *           may be NULL, when py is used.
 *   py, py_stride : NULL, or the pool's output that argmax was selected with (yd-shaped, pixel
 *           stride py_stride >= yd.c elements, element type dt; read only).  Used when beta = 0;
 *           ignored when beta = 1 (the stored gradient then needs y's mask at every element).
 *   dpre  : xd-shaped, written (read first when beta = 1, which adds the gradient the other
 *           consumers of y already stored there); must not overlap y, py, dy or argmax.
 *   dbias : xd.c fp32 values, overwritten; or NULL: deferred (see tfk_bias_grad_finish).
 *   ws    : at least tfk_bias_relu_bwd_workspace_bytes(xd, dt) bytes.
 * Requirements: beta is 0 or 1; xd.c <= 16384.  xd.n == 0 sets dbias to 0.
 * Errors: NULL (dy, argmax, dpre, or y where it is read), SHAPE (pool geometry,
 * xd.c > 16384, py_stride < yd.c), ARG (beta), ALIGN (element alignment), ALIAS (the overlaps
 * above), WORKSPACE (ws too small).
 */
TFK_API tfk_status tfk_maxpool_bwd_relu_bwd(const void *dy, const int32_t *argmax, tfk_nhwc yd, tfk_window p,
                                    tfk_dtype dt, const void *y, const void *py, int64_t py_stride,
                                    void *dpre, tfk_nhwc xd, float beta, float *dbias, void *ws,
                                    size_t ws_bytes, void *stream);
/* tfk_maxpool_bwd_relu_bwd (Section 5 fused activation gradient, Section 6.1 pooling) with the
 * selection from tfk_maxpool_fwd_taps (py: the output of that call, or of
 * tfk_conv2d_fwd_bias_relu_maxpool). */
TFK_API tfk_status tfk_maxpool_bwd_relu_bwd_taps(const void *dy, const uint8_t *taps, tfk_nhwc yd, tfk_window p,
                                         tfk_dtype dt, const void *y, const void *py, int64_t py_stride,
                                         void *dpre, tfk_nhwc xd, float beta, float *dbias, void *ws,
                                         size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------- update
 * ApplyGradientDescent, in place (Section 4.1: W' = W - alpha * dL/dW written
 * with "-=" into the variable's buffer; Section 3.1 variables are mutable
 * buffers updated in place):
 *   var[i] <- fma(-lr, grad[i], var[i])      for 0 <= i < n   (fp32)
 *   var_bf16, if not NULL, receives the bf16 (RNE) copy of the updated var,
 *   used as the next step's low-precision weights.
 * var must not overlap grad or var_bf16.
 */
TFK_API tfk_status tfk_apply_sgd(float *var, const float *grad, int64_t n, float lr,
                         uint16_t *var_bf16, void *stream);

/* ApplyGradientDescent (Section 4.1, W' = W - alpha * dL/dW, as tfk_apply_sgd) over
 * `count` independent (var, grad, n, shadow) tuples in one launch per batch of tensors:
 * every variable of a synchronous step is updated from gradients of the same parameter
 * version (Section 4.4).  shadows may be NULL (no shadows) or hold NULL
 * entries.  The pointer arrays are host memory and are read during the call. */
TFK_API tfk_status tfk_apply_sgd_multi(int32_t count, float *const *vars, const float *const *grads,
                               const int64_t *ns, float lr, uint16_t *const *shadows,
                               void *stream);

/* ---------------------------------------------------------------- classifier loss
 * Softmax cross-entropy of a classifier's logits against integer labels (the
 * loss whose gradient Section 4.1's backpropagation starts from in the image
 * models the paper trains).  For each row i < n of z = logits + bias:
 *   loss[i]       = log(sum_j exp(z[i][j])) - z[i][labels[i]]
 *   dlogits[i][j] = scale * (softmax(z[i])[j] - (j == labels[i]))
 * (scale = 1/n gives the gradient of the batch-mean loss).  The max of each row
 * is taken out before exp, so no finite logit overflows; arithmetic is fp32.
 *   logits, dlogits : n x c row-major, type dt; dlogits may equal logits (in
 *                     place, the logits are then overwritten), any other
 *                     overlap is an error.
 *   bias            : fp32 [c], or NULL for none.
 *   labels          : int32 [n], device memory.  A label outside [0, c) is not
 *                     checked on the host: its row gets a NaN loss and NaN
 *                     gradients.
 *   loss            : fp32 [n], overwritten.
 * Errors: n < 0 or c < 1 (SHAPE); scale not finite (ARG); n * c > 2^40
 * (OVERFLOW); NULL buffers with n > 0 (NULL); misalignment (ALIGN);
 * overlapping operands (ALIAS).  n == 0 is a no-op. */
TFK_API tfk_status tfk_softmax_xent(const void *logits, tfk_dtype dt, int64_t n, int32_t c, const float *bias,
                            const int32_t *labels, float scale, float *loss, void *dlogits,
                            void *stream);

/* ---------------------------------------------------------------- sampled softmax
 * The sampled softmax of Section 4.2 (evaluated in Section 6.4; Jean et al. 2015): a
 * classifier over many classes multiplies its input h (n x d) only by the weight rows of
 * each example's true class and of one shared sample of m classes drawn by the caller from
 * a proposal Q.  The caller lists the distinct candidate classes (the m sampled ones first,
 * then the true classes not among them: u in all) and, per example, the candidate column of
 * its true class; the step then runs as
 *   tfk_gather_rows_t   W[cand] as a d x u_pad filter, b[cand] as u_pad values
 *   tfk_conv2d_fwd      z = h . W[cand]^T (a 1 x 1 convolution of n 1 x 1 images)
 *   tfk_sampled_softmax_xent   loss and dz over the candidates
 *   tfk_bias_relu_bwd (y NULL), tfk_conv2d_bwd_filter, tfk_conv2d_bwd_input
 *                       db, dW of the candidates (d x u_pad), dh
 *   tfk_scatter_apply_sgd   W[cand] -= lr dW, b[cand] -= lr db (rows are distinct)
 *
 * out_t[k][j] = table[idx[j]][k] for j < u, k < d; 0 for u <= j < u_pad or for an index
 * outside [0, rows).  table: rows x d row-major, type dt; out_t: d x u_pad, type dt.
 * Errors: rows < 0, d < 1, u < 0 or u_pad < u (SHAPE); NULL, misaligned or overlapping
 * buffers (NULL, ALIGN, ALIAS). */
TFK_API tfk_status tfk_gather_rows_t(const void *table, tfk_dtype dt, int64_t rows, int32_t d, const int32_t *idx,
                             int32_t u, int32_t u_pad, void *out_t, void *stream);

/* Cross-entropy over candidate logits z (the sampled softmax loss of Section 4.2, as
 * described above) (n x u_pad, type dt): column j < m is sampled class
 * j with log expected count lq_sampled[j]; true_pos[i] is the column of row i's true class,
 * whose log expected count is lq_true[i].  With bc = bias_c (u_pad values, or NULL):
 *   true logit     zt = z[i][t] + bc[t] - lq_true[i]              (t = true_pos[i])
 *   sampled logit  z[i][j] + bc[j] - lq_sampled[j]  for j < m, j != t (j == t: an accidental
 *                  hit, left out)
 *   loss[i] = log(sum of exp over the row's logits) - zt
 *   dz[i][j] = scale * softmax over the row's logits at j, minus scale at the true column;
 *              0 in every other column (excluded, unsampled, padding).
 * true_pos outside [0, u) is not checked on the host: the row gets NaN loss and gradients.
 * Errors: n < 0, not 0 <= m <= u <= u_pad, u < 1 (SHAPE); scale not finite (ARG); NULL,
 * misaligned, or dz / loss overlapping any operand (NULL, ALIGN, ALIAS). */
TFK_API tfk_status tfk_sampled_softmax_xent(const void *z, tfk_dtype dt, int64_t n, int32_t u, int32_t u_pad,
                                    int32_t m, const float *bias_c, const int32_t *true_pos,
                                    const float *lq_true, const float *lq_sampled, float scale, float *loss,
                                    void *dz, void *stream);

/* Sparse ApplyGradientDescent of candidate rows (Section 4.2's sparse variable updates):
 *   var[idx[j]][k] <- fma(-lr, grad_t[k * ld + j], var[idx[j]][k])    j < u, k < d
 * var: rows x d fp32; var_bf16 (optional) its bf16 shadow, rewritten for the touched rows;
 * grad_t: d x ld fp32 (the filter-gradient layout of the candidate convolution).  The rows
 * idx[j] must be distinct (each element then has one writer); an index outside [0, rows)
 * is skipped.
 * Errors: rows < 0, d < 1, u < 0 or ld < u (SHAPE); lr not finite (ARG); NULL, misaligned or
 * overlapping buffers (NULL, ALIGN, ALIAS).  u == 0 is a no-op. */
TFK_API tfk_status tfk_scatter_apply_sgd(float *var, uint16_t *var_bf16, int64_t rows, int32_t d, const int32_t *idx,
                                 int32_t u, const float *grad_t, int64_t ld, float lr, void *stream);

/* Momentum, in place (Section 4.1 lists it among the optimizers built from
 * Variable updates: a per-parameter velocity accumulated over the gradients
 * drives the update).  Velocity form of Sutskever et al. (2013), fp32:
 *   accum[i] <- fma(momentum, accum[i], grad[i])
 *   var[i]   <- fma(-lr, accum[i], var[i])                           nesterov = 0
 *   var[i]   <- fma(-lr, fma(momentum, accum[i], grad[i]), var[i])   nesterov = 1
 * (the second line uses the updated accum).  var_bf16 as in tfk_apply_sgd.
 * Errors: n < 0 (SHAPE); lr or momentum not finite, nesterov not 0/1 (ARG);
 * a NULL buffer with n > 0 (NULL); a buffer not aligned to its element
 * (ALIGN); any two of var, accum, grad, var_bf16 overlapping (ALIAS).  n == 0 is a no-op. */
TFK_API tfk_status tfk_apply_momentum(float *var, float *accum, const float *grad, int64_t n, float lr,
                              float momentum, int32_t nesterov, uint16_t *var_bf16, void *stream);

/* Adam, in place (Section 4.1 lists it; Kingma & Ba (2015), Algorithm 1), step
 * t >= 1 of the moment estimates m and v, fp32:
 *   m[i] <- beta1 m[i] + (1 - beta1) grad[i]
 *   v[i] <- beta2 v[i] + (1 - beta2) grad[i]^2
 *   var[i] <- var[i] - lr / (1 - beta1^t) * m[i] / (sqrt(v[i] / (1 - beta2^t)) + epsilon)
 * The bias corrections 1 - beta^t are computed on the host in fp64 and folded
 * into two fp32 scalars; the per-element arithmetic is fp32 with fma.
 * var_bf16 as in tfk_apply_sgd.  Start from m = v = 0 at t = 1.
 * Errors: n < 0 (SHAPE); lr not finite, beta1 or beta2 outside [0, 1),
 * epsilon negative or not finite, t < 1 (ARG); a bias-corrected scalar that
 * overflows fp32 (OVERFLOW); a NULL buffer with n > 0 (NULL); a buffer not
 * aligned to its element (ALIGN); any two of var, m, v, grad, var_bf16
 * overlapping (ALIAS).  n == 0 is a no-op. */
TFK_API tfk_status tfk_apply_adam(float *var, float *m, float *v, const float *grad, int64_t n, float lr,
                          float beta1, float beta2, float epsilon, int64_t t, uint16_t *var_bf16,
                          void *stream);

/* ---------------------------------------------------------------- streams and programs
 * The dataflow executor runs independent kernels of a step on several GPU streams (Section 5);
 * a step's subgraph is pruned and placed once, cached, and run again for every later step from
 * one small request (Sections 3.2 and 3.3).  Here a step is a sequence of calls to this library;
 * a program records that sequence once and issues it again from C++.
 *
 * tfk_stream_wait: work enqueued on `waiter` after this call starts only after everything
 * enqueued on `producer` before it has completed (an event recorded on producer, waited on by
 * waiter; no host synchronisation).  waiter == producer is a no-op.  NULL is the default stream.
 * Errors: HIP (event creation, record or wait failed). */
TFK_API tfk_status tfk_stream_wait(void *waiter, void *producer);

/* A caller-owned point on a stream: tfk_mark_record places it after everything enqueued on
 * `stream` so far, and work enqueued on `waiter` after tfk_stream_wait_mark starts only once
 * that point (the mark's latest record before the wait call) has been reached.  Unlike
 * tfk_stream_wait, the producer may enqueue more work between the two calls without the waiter
 * waiting for it: the independent branches of a step run on several streams that each wait only
 * for the kernels producing their inputs (the executor's per-edge dependencies, Section 3.1;
 * several GPU streams, Section 5).  Both calls are recorded into a program like the ops (the
 * mark by pointer: it must outlive the program's use).  tfk_mark_create errors: NULL; ARG (out
 * of host memory); HIP (event creation).  tfk_mark_record / tfk_stream_wait_mark errors: NULL
 * (mark is NULL); HIP.  tfk_mark_destroy(NULL) is a no-op; a mark that work still waits for may
 * be destroyed (the runtime keeps the event until it completes).  Waiting on a mark that was
 * never recorded does not wait.  The step keeps marks out of HIP stream captures (a capture of
 * a step whose branches waited on marks ended in a host fault of the process; not investigated
 * further). */
typedef struct tfk_mark tfk_mark;
TFK_API tfk_status tfk_mark_create(tfk_mark **mark);
TFK_API void tfk_mark_destroy(tfk_mark *mark);
TFK_API tfk_status tfk_mark_record(tfk_mark *mark, void *stream);
TFK_API tfk_status tfk_stream_wait_mark(void *waiter, tfk_mark *mark);

/* Opaque recorded call sequence. */
typedef struct tfk_program tfk_program;

/* Creates an empty program in *prog (owned by the caller; release with tfk_program_destroy).
 * Errors: NULL (prog is NULL); ARG (out of host memory). */
TFK_API tfk_status tfk_program_create(tfk_program **prog);
/* Releases a program and the events its recorded stream joins own (work already enqueued is
 * not affected).  Stops its recording if it is recording on the calling thread.  NULL: no-op. */
TFK_API void tfk_program_destroy(tfk_program *prog);
/* Starts recording on the calling thread (previous contents are dropped).  Until
 * tfk_program_end, every tfk_* call on this thread that enqueues work (convolutions, bias/ReLU,
 * pooling, updates, losses, sampled-softmax ops, tfk_stream_wait, marks) runs as usual and, when it
 * returns TFK_OK, is appended to the program with its arguments by value: the same pointers,
 * shapes, scalars and streams.  Calls that fail are not appended.  Queries
 * (*_workspace_bytes) are never recorded.  Errors: NULL; ARG (this thread already records). */
TFK_API tfk_status tfk_program_begin(tfk_program *prog);
/* Stops recording.  Errors: NULL; ARG (prog is not recording on this thread). */
TFK_API tfk_status tfk_program_end(tfk_program *prog);
/* Number of recorded calls (0 for NULL). */
TFK_API int64_t tfk_program_length(const tfk_program *prog);
/* Issues the recorded calls again, in order, each validated as when it was recorded.  Every
 * buffer a recorded call names must still be allocated, and each call's results depend only
 * on what its buffers hold when it runs: scalars are replayed as recorded (a recorded
 * tfk_apply_adam replays its step count t unchanged).  Stops at the first call that fails
 * and returns its status.  Errors: NULL; ARG (a program is recording on this thread); any
 * status a recorded call returns. */
TFK_API tfk_status tfk_program_run(tfk_program *prog);

/* ---------------------------------------------------------------- misc
 * Error reporting of the thin C API that the paper's client libraries sit on (Section 5: a C
 * API separates the user-level code from the core runtime); no tensor arithmetic. */
/* Name of a status code. */
TFK_API const char *tfk_status_string(tfk_status s);
/* Detail of the last non-OK status returned on the calling thread ("" if none). */
TFK_API const char *tfk_last_error(void);
/* Version of this interface (incremented when any declaration here changes). */
TFK_API int32_t tfk_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* TFK_H_ */
