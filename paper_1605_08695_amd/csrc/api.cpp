// C ABI of the gfx950 convnet training-step library (declared in include/tfk.h).
//
// Every entry point validates its arguments completely before anything is
// enqueued; on failure it returns a status, records a message for
// tfk_last_error() and leaves every buffer untouched.  Validation is plain
// host code: it makes no HIP call.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <functional>
#include <memory>
#include <new>
#include <string>
#include <vector>

#include "../../include/tfk.h"
#include "kernels.h"

using namespace tfk;

namespace {

thread_local std::string g_err;

tfk_status fail(tfk_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

tfk_status ok() {
    g_err.clear();
    return TFK_OK;
}

tfk_status hip_status(hipError_t e, const char *what) {
    if (e == hipSuccess) return ok();
    return fail(TFK_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool valid_dt(tfk_dtype dt) { return dt == TFK_F32 || dt == TFK_BF16; }
int64_t esize(tfk_dtype dt) { return dt == TFK_F32 ? 4 : 2; }

// Checks extents, resolves pixel_stride == 0 to c.
tfk_status check_view(const char *name, tfk_nhwc &d) {
    if (d.n < 0 || d.h <= 0 || d.w <= 0 || d.c <= 0)
        return fail(TFK_ERR_SHAPE, "%s: extents must be n >= 0 and h, w, c >= 1 (got %d,%d,%d,%d)", name, d.n,
                    d.h, d.w, d.c);
    if (d.pixel_stride == 0) d.pixel_stride = d.c;
    if (d.pixel_stride < d.c)
        return fail(TFK_ERR_SHAPE, "%s: pixel_stride %lld < c %d", name, (long long)d.pixel_stride, d.c);
    const int64_t pix = (int64_t)d.n * d.h * d.w;
    if (pix > INT32_MAX) return fail(TFK_ERR_OVERFLOW, "%s: n*h*w = %lld exceeds 2^31-1", name, (long long)pix);
    if (d.pixel_stride > ((int64_t)1 << 40))
        return fail(TFK_ERR_OVERFLOW, "%s: pixel_stride too large", name);
    return TFK_OK;
}

int64_t view_bytes(const tfk_nhwc &d, int64_t es) {
    const int64_t pix = (int64_t)d.n * d.h * d.w;
    if (pix == 0) return 0;
    return ((pix - 1) * d.pixel_stride + d.c) * es;
}

tfk_status check_window(const tfk_window &p) {
    if (p.kh < 1 || p.kw < 1) return fail(TFK_ERR_SHAPE, "window: kh, kw must be >= 1");
    if (p.stride_h < 1 || p.stride_w < 1 || p.stride_h > 255 || p.stride_w > 255)
        return fail(TFK_ERR_SHAPE, "window: strides must be in [1, 255]");
    if (p.pad_top < 0 || p.pad_bottom < 0 || p.pad_left < 0 || p.pad_right < 0)
        return fail(TFK_ERR_SHAPE, "window: pads must be >= 0");
    if (p.pad_top >= p.kh || p.pad_bottom >= p.kh || p.pad_left >= p.kw || p.pad_right >= p.kw)
        return fail(TFK_ERR_SHAPE, "window: every pad must be smaller than the kernel extent");
    return TFK_OK;
}

// Output extent along one axis, or 0 when no window fits.
int out_len(int n, int k, int s, int p0, int p1) {
    const int64_t span = (int64_t)n + p0 + p1 - k;
    if (span < 0) return 0;
    return (int)(span / s + 1);
}

bool overlap(const void *a, int64_t abytes, const void *b, int64_t bbytes) {
    if (!a || !b || abytes <= 0 || bbytes <= 0) return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + (uintptr_t)bbytes && b0 < a0 + (uintptr_t)abytes;
}

bool aligned(const void *p, int64_t a) { return ((uintptr_t)p % (uintptr_t)a) == 0; }

// Whether two NHWC views may share an element.  Besides disjoint byte ranges, two views with one
// pixel stride whose channels lie side by side within every pixel (channel slices of one buffer,
// e.g. a concat's branches) share none: b's channels start d bytes into a's pixel period, with
// a's channels before d and b's ending within the period.
bool nhwc_overlap(const void *a, const tfk_nhwc &ad, const void *b, const tfk_nhwc &bd, int64_t es) {
    if (!overlap(a, view_bytes(ad, es), b, view_bytes(bd, es))) return false;
    if (ad.pixel_stride != bd.pixel_stride || ad.pixel_stride <= 0) return true;
    const int64_t S = ad.pixel_stride * es;
    int64_t d = ((int64_t)(intptr_t)b - (int64_t)(intptr_t)a) % S;
    if (d < 0) d += S;
    return !(d >= (int64_t)ad.c * es && d + (int64_t)bd.c * es <= S);
}

tfk_status need_ptr(const void *p, const char *name) {
    if (!p) return fail(TFK_ERR_NULL, "%s is NULL", name);
    return TFK_OK;
}

tfk_status need_align(const void *p, int64_t a, const char *name) {
    if (p && !aligned(p, a)) return fail(TFK_ERR_ALIGN, "%s is not %lld-byte aligned", name, (long long)a);
    return TFK_OK;
}

#define TRY(expr)                         \
    do {                                  \
        tfk_status _s = (expr);           \
        if (_s != TFK_OK) return _s;      \
    } while (0)

// Shared validation of a convolution: input view xd, filter (KH,KW,C,cout), output view yd.
tfk_status check_conv(tfk_nhwc &xd, int32_t cout, const tfk_window &p, tfk_dtype dt, tfk_nhwc &yd,
                      const char *xname, const char *yname, ConvShape &s) {
    if (!valid_dt(dt)) return fail(TFK_ERR_DTYPE, "unknown dtype %d", (int)dt);
    TRY(check_view(xname, xd));
    TRY(check_view(yname, yd));
    TRY(check_window(p));
    if (cout < 1) return fail(TFK_ERR_SHAPE, "cout must be >= 1");
    const int oh = out_len(xd.h, p.kh, p.stride_h, p.pad_top, p.pad_bottom);
    const int ow = out_len(xd.w, p.kw, p.stride_w, p.pad_left, p.pad_right);
    if (oh < 1 || ow < 1) return fail(TFK_ERR_SHAPE, "window does not fit the padded input");
    if (yd.n != xd.n || yd.h != oh || yd.w != ow || yd.c != cout)
        return fail(TFK_ERR_SHAPE, "%s must be [%d,%d,%d,%d], got [%d,%d,%d,%d]", yname, xd.n, oh, ow, cout, yd.n,
                    yd.h, yd.w, yd.c);
    const int64_t kred = (int64_t)p.kh * p.kw * xd.c;
    if (kred > INT32_MAX / 2 || (int64_t)kred * cout > INT32_MAX)
        return fail(TFK_ERR_OVERFLOW, "filter too large");
    s.N = xd.n; s.H = xd.h; s.W = xd.w; s.C = xd.c;
    s.OH = oh; s.OW = ow; s.K = cout;
    s.KH = p.kh; s.KW = p.kw; s.sh = p.stride_h; s.sw = p.stride_w; s.pt = p.pad_top; s.pl = p.pad_left;
    return TFK_OK;
}

int64_t filter_bytes(const ConvShape &s, int64_t es) { return (int64_t)s.KH * s.KW * s.C * s.K * es; }

// A window that covers the whole (unpadded, densely stored) image once is a fully connected layer:
// x[n][h][w][c] and w[h][w][c][k] flatten to the same (h W + w) C + c order, so the convolution is
// the 1 x 1 convolution of the flattened image, whose kernels do no per-tap work.  xs is the pixel
// stride of x (or dx); it becomes the flattened row length.
static void fold_full_window(ConvShape &s, int64_t &xs) {
    if (s.OH == 1 && s.OW == 1 && s.KH == s.H && s.KW == s.W && s.pt == 0 && s.pl == 0 && (s.H > 1 || s.W > 1) &&
        xs == s.C) {
        s.C = s.H * s.W * s.C;
        s.H = s.W = s.KH = s.KW = 1;
        s.sh = s.sw = 1;
        xs = s.C;
    }
}

tfk_status check_ws(void *ws, size_t ws_bytes, size_t need) {
    if (need == 0) return TFK_OK;
    if (!ws) return fail(TFK_ERR_WORKSPACE, "workspace of %zu bytes required, got NULL", need);
    if (ws_bytes < need) return fail(TFK_ERR_WORKSPACE, "workspace of %zu bytes required, got %zu", need, ws_bytes);
    if (!aligned(ws, 16)) return fail(TFK_ERR_ALIGN, "workspace must be 16-byte aligned");
    return TFK_OK;
}

}  // namespace

// A recorded sequence of library calls (arguments by value) that tfk_program_run issues again in
// the same order: one step's kernels, workspaces and stream joins, enqueued from C++ with no
// per-call marshalling by the caller.
struct tfk_program {
    std::vector<std::function<tfk_status()>> calls;
};

namespace {

// The program recording on this thread, if any.
thread_local tfk_program *g_rec = nullptr;

// While a program records on this thread, a call runs with recording paused (so that it is not
// appended twice) and, when it succeeds, is appended with its arguments by value.
#define RECORDED(fn, ...)                                                                        \
    do {                                                                                         \
        if (g_rec != nullptr) {                                                                  \
            tfk_program *const rec_ = g_rec;                                                     \
            g_rec = nullptr;                                                                     \
            const tfk_status s_ = fn(__VA_ARGS__);                                               \
            g_rec = rec_;                                                                        \
            if (s_ != TFK_OK) return s_;                                                         \
            try {                                                                                \
                rec_->calls.emplace_back([=]() { return fn(__VA_ARGS__); });                     \
            } catch (...) {                                                                      \
                return fail(TFK_ERR_ARG, "%s: out of host memory while recording", #fn);         \
            }                                                                                    \
            return s_;                                                                           \
        }                                                                                        \
    } while (0)

// Where the last call on this thread that was given dbias = NULL left its bias-gradient partials.
struct LastPartials {
    const float *part = nullptr;
    int32_t rows = 0;
    bool valid = false;
};
thread_local LastPartials g_partials;

static void note_partials(const float *part, int rows) {
    g_partials.part = part;
    g_partials.rows = rows;
    g_partials.valid = true;
}

// An event owned by a recorded stream join (released with its program).
struct OwnedEvent {
    hipEvent_t e = nullptr;
    ~OwnedEvent() {
        if (e != nullptr) (void)hipEventDestroy(e);
    }
};

// Events of stream joins: no timing, and no system-scope fence (the waiting work runs on the same
// GPU, which every kernel's completion already releases its writes to; the system fence, a cache
// write-back for the host's sake, cost the recording stream about 6 us per join).
constexpr unsigned kJoinEventFlags = hipEventDisableTiming | hipEventDisableSystemFence;

tfk_status join(hipEvent_t e, hipStream_t waiter, hipStream_t producer) {
    hipError_t r = hipEventRecord(e, producer);
    if (r == hipSuccess) r = hipStreamWaitEvent(waiter, e, 0);
    return hip_status(r, "stream_wait");
}

}  // namespace

extern "C" {

int32_t tfk_abi_version(void) { return TFK_ABI_VERSION; }

const char *tfk_last_error(void) { return g_err.c_str(); }

const char *tfk_status_string(tfk_status s) {
    switch (s) {
        case TFK_OK: return "ok";
        case TFK_ERR_NULL: return "null pointer";
        case TFK_ERR_SHAPE: return "invalid shape";
        case TFK_ERR_DTYPE: return "invalid dtype";
        case TFK_ERR_ALIGN: return "misaligned pointer";
        case TFK_ERR_OVERFLOW: return "index overflow";
        case TFK_ERR_ALIAS: return "illegal aliasing";
        case TFK_ERR_WORKSPACE: return "workspace too small";
        case TFK_ERR_HIP: return "HIP runtime error";
        case TFK_ERR_ARG: return "invalid argument";
    }
    return "unknown status";
}

// ------------------------------------------------------------------ convolution
size_t tfk_conv2d_workspace_bytes(int32_t op, tfk_nhwc xd, int32_t cout, tfk_window p, tfk_dtype dt) {
    if (op < 0 || op > 3) return 0;
    if (!valid_dt(dt) || check_view("x", xd) != TFK_OK || check_window(p) != TFK_OK || cout < 1) return 0;
    const int oh = out_len(xd.h, p.kh, p.stride_h, p.pad_top, p.pad_bottom);
    const int ow = out_len(xd.w, p.kw, p.stride_w, p.pad_left, p.pad_right);
    if (oh < 1 || ow < 1 || xd.n == 0) return 0;
    ConvShape s{xd.n, xd.h, xd.w, xd.c, oh, ow, cout, p.kh, p.kw, p.stride_h, p.stride_w, p.pad_top, p.pad_left};
    const int dti = dt == TFK_F32 ? 0 : 1;
    // (the fused ReLU backward sums its bias gradient per channel: no flattening there)
    if (op == 3) return conv_bwd_data_relu_ws_bytes(dti, s, xd.pixel_stride);
    int64_t xs = xd.pixel_stride;
    fold_full_window(s, xs);
    if (op == 0) return std::max(conv_fold_applies(dti, s) ? conv_fold_ws_bytes(0, s) : 0,
                                 conv_fwd_split_ws_bytes(dti, s));
    if (op == 1) return conv_bwd_data_ws_bytes(dti, s);
    return conv_bwd_filter_ws_bytes(dti, s);
}

// Validation of the forward convolution (shared by tfk_conv2d_fwd, tfk_conv2d_fwd_bias_relu and the
// fused max-pool form): fills the shape, x's pixel stride after flattening and the workspace need.
static tfk_status conv_fwd_check(const void *x, tfk_nhwc &xd, const void *w, int32_t cout, const float *bias,
                                 tfk_window p, tfk_dtype dt, void *y, tfk_nhwc &yd, void *ws, size_t ws_bytes,
                                 ConvShape &s, int64_t &xs, size_t &need) {
    TRY(check_conv(xd, cout, p, dt, yd, "x", "y", s));
    xs = xd.pixel_stride;
    need = 0;
    if (xd.n == 0) return TFK_OK;
    const int64_t es = esize(dt);
    TRY(need_ptr(x, "x"));
    TRY(need_ptr(w, "w"));
    TRY(need_ptr(y, "y"));
    TRY(need_align(x, es, "x"));
    TRY(need_align(w, es, "w"));
    TRY(need_align(y, es, "y"));
    const int64_t yb = view_bytes(yd, es);
    if (nhwc_overlap(y, yd, x, xd, es) || overlap(y, yb, w, filter_bytes(s, es)))
        return fail(TFK_ERR_ALIAS, "y overlaps x or w");
    if (bias != nullptr && overlap(y, yb, bias, (int64_t)cout * 4)) return fail(TFK_ERR_ALIAS, "y overlaps bias");
    const int64_t xbytes = view_bytes(xd, es), wbytes = filter_bytes(s, es);
    fold_full_window(s, xs);
    const int dti = dt == TFK_F32 ? 0 : 1;
    need = std::max(conv_fold_applies(dti, s) ? conv_fold_ws_bytes(0, s) : 0, conv_fwd_split_ws_bytes(dti, s));
    TRY(check_ws(ws, ws_bytes, need));
    if (need && (overlap(ws, (int64_t)need, x, xbytes) || overlap(ws, (int64_t)need, w, wbytes) ||
                 overlap(ws, (int64_t)need, y, yb)))
        return fail(TFK_ERR_ALIAS, "workspace overlaps an operand");
    return TFK_OK;
}

// Shared by tfk_conv2d_fwd (bias == nullptr) and tfk_conv2d_fwd_bias_relu.
static tfk_status conv_fwd_impl(const void *x, tfk_nhwc xd, const void *w, int32_t cout, const float *bias,
                                tfk_window p, tfk_dtype dt, void *y, tfk_nhwc yd, void *ws, size_t ws_bytes,
                                void *stream, const char *what) {
    ConvShape s;
    int64_t xs;
    size_t need;
    TRY(conv_fwd_check(x, xd, w, cout, bias, p, dt, y, yd, ws, ws_bytes, s, xs, need));
    if (xd.n == 0) return ok();
    return hip_status(launch_conv_fwd(dt == TFK_F32 ? 0 : 1, x, xs, w, y, yd.pixel_stride, s, bias,
                                      need ? ws : nullptr, (hipStream_t)stream),
                      what);
}

tfk_status tfk_conv2d_fwd(const void *x, tfk_nhwc xd, const void *w, int32_t cout, tfk_window p, tfk_dtype dt,
                          void *y, tfk_nhwc yd, void *ws, size_t ws_bytes, void *stream) {
    RECORDED(tfk_conv2d_fwd, x, xd, w, cout, p, dt, y, yd, ws, ws_bytes, stream);
    return conv_fwd_impl(x, xd, w, cout, nullptr, p, dt, y, yd, ws, ws_bytes, stream, "conv2d_fwd");
}

tfk_status tfk_conv2d_fwd_bias_relu(const void *x, tfk_nhwc xd, const void *w, int32_t cout, const float *bias,
                                    tfk_window p, tfk_dtype dt, void *y, tfk_nhwc yd, void *ws, size_t ws_bytes,
                                    void *stream) {
    RECORDED(tfk_conv2d_fwd_bias_relu, x, xd, w, cout, bias, p, dt, y, yd, ws, ws_bytes, stream);
    if (xd.n > 0 && cout > 0) {
        TRY(need_ptr(bias, "bias"));
        TRY(need_align(bias, 4, "bias"));
    }
    return conv_fwd_impl(x, xd, w, cout, bias, p, dt, y, yd, ws, ws_bytes, stream, "conv2d_fwd_bias_relu");
}

tfk_status tfk_conv2d_bwd_input(const void *dy, tfk_nhwc dyd, const void *w, tfk_window p, tfk_dtype dt, void *dx,
                                tfk_nhwc dxd, float beta, void *ws, size_t ws_bytes, void *stream) {
    RECORDED(tfk_conv2d_bwd_input, dy, dyd, w, p, dt, dx, dxd, beta, ws, ws_bytes, stream);
    ConvShape s;
    TRY(check_conv(dxd, dyd.c, p, dt, dyd, "dx", "dy", s));
    if (!(beta == 0.f || beta == 1.f)) return fail(TFK_ERR_ARG, "beta must be 0 or 1");
    if (dxd.n == 0) return ok();
    const int64_t es = esize(dt);
    TRY(need_ptr(dy, "dy"));
    TRY(need_ptr(w, "w"));
    TRY(need_ptr(dx, "dx"));
    TRY(need_align(dy, es, "dy"));
    TRY(need_align(w, es, "w"));
    TRY(need_align(dx, es, "dx"));
    const int64_t xb = view_bytes(dxd, es);
    if (nhwc_overlap(dx, dxd, dy, dyd, es) || overlap(dx, xb, w, filter_bytes(s, es)))
        return fail(TFK_ERR_ALIAS, "dx overlaps dy or w");
    const int64_t wbytes = filter_bytes(s, es);
    int64_t xs = dxd.pixel_stride;
    fold_full_window(s, xs);
    const int dti = dt == TFK_F32 ? 0 : 1;
    const size_t need = conv_bwd_data_ws_bytes(dti, s);
    TRY(check_ws(ws, ws_bytes, need));
    if (need && (overlap(ws, (int64_t)need, dy, view_bytes(dyd, es)) || overlap(ws, (int64_t)need, w, wbytes) ||
                 overlap(ws, (int64_t)need, dx, xb)))
        return fail(TFK_ERR_ALIAS, "workspace overlaps an operand");
    return hip_status(launch_conv_bwd_data(dti, dy, dyd.pixel_stride, w, dx, xs, beta, s,
                                           need ? (float *)ws : nullptr, (hipStream_t)stream),
                      "conv2d_bwd_input");
}

tfk_status tfk_conv2d_bwd_input_relu_bwd(const void *dy, tfk_nhwc dyd, const void *w, tfk_window p, tfk_dtype dt,
                                         const void *y, void *dpre, tfk_nhwc xd, float beta, float *dbias,
                                         void *ws, size_t ws_bytes, void *stream) {
    RECORDED(tfk_conv2d_bwd_input_relu_bwd, dy, dyd, w, p, dt, y, dpre, xd, beta, dbias, ws, ws_bytes, stream);
    ConvShape s;
    TRY(check_conv(xd, dyd.c, p, dt, dyd, "dpre", "dy", s));
    if (!(beta == 0.f || beta == 1.f)) return fail(TFK_ERR_ARG, "beta must be 0 or 1");
    if (xd.c > 16384) return fail(TFK_ERR_SHAPE, "conv2d_bwd_input_relu_bwd supports at most 16384 channels");
    TRY(need_align(dbias, 4, "dbias"));
    hipStream_t st = (hipStream_t)stream;
    if (xd.n == 0) {
        if (dbias == nullptr) {
            note_partials((const float *)ws, 0);
            return ok();
        }
        return hip_status(launch_fill_zero(dbias, xd.c, st), "conv2d_bwd_input_relu_bwd");
    }
    const int64_t es = esize(dt);
    TRY(need_ptr(dy, "dy"));
    TRY(need_ptr(w, "w"));
    TRY(need_ptr(y, "y"));
    TRY(need_ptr(dpre, "dpre"));
    TRY(need_align(dy, es, "dy"));
    TRY(need_align(w, es, "w"));
    TRY(need_align(y, es, "y"));
    TRY(need_align(dpre, es, "dpre"));
    const int64_t xb = view_bytes(xd, es), yb = view_bytes(dyd, es), wb = filter_bytes(s, es), bb = (int64_t)xd.c * 4;
    if (nhwc_overlap(dpre, xd, dy, dyd, es) || overlap(dpre, xb, w, wb) || nhwc_overlap(dpre, xd, y, xd, es))
        return fail(TFK_ERR_ALIAS, "dpre overlaps dy, w or y");
    if (overlap(dbias, bb, dy, yb) || overlap(dbias, bb, w, wb) || overlap(dbias, bb, y, xb) ||
        overlap(dbias, bb, dpre, xb))
        return fail(TFK_ERR_ALIAS, "dbias overlaps a tensor");
    const int dti = dt == TFK_F32 ? 0 : 1;
    const int64_t xs = xd.pixel_stride;      // (not flattened: the bias gradient is per channel)
    const size_t need = conv_bwd_data_relu_ws_bytes(dti, s, xs);
    TRY(check_ws(ws, ws_bytes, need));
    if (overlap(ws, (int64_t)need, dy, yb) || overlap(ws, (int64_t)need, w, wb) || overlap(ws, (int64_t)need, y, xb) ||
        overlap(ws, (int64_t)need, dpre, xb) || overlap(ws, (int64_t)need, dbias, bb))
        return fail(TFK_ERR_ALIAS, "workspace overlaps an operand");
    BiasPartials bp{nullptr, 0};
    TRY(hip_status(launch_conv_bwd_data_relu(dti, dy, dyd.pixel_stride ? dyd.pixel_stride : dyd.c, w, dpre, xs, y,
                                             beta, dbias, (float *)ws, s, st, dbias ? nullptr : &bp),
                   "conv2d_bwd_input_relu_bwd"));
    if (dbias == nullptr) note_partials(bp.part, bp.rows);
    return ok();
}

tfk_status tfk_conv2d_bwd_filter(const void *x, tfk_nhwc xd, const void *dy, tfk_nhwc dyd, tfk_window p,
                                 tfk_dtype dt, float *dw, void *ws, size_t ws_bytes, void *stream) {
    RECORDED(tfk_conv2d_bwd_filter, x, xd, dy, dyd, p, dt, dw, ws, ws_bytes, stream);
    ConvShape s;
    TRY(check_conv(xd, dyd.c, p, dt, dyd, "x", "dy", s));
    TRY(need_ptr(dw, "dw"));
    TRY(need_align(dw, 4, "dw"));
    const int64_t wb = filter_bytes(s, 4);
    hipStream_t st = (hipStream_t)stream;
    if (xd.n == 0) return hip_status(launch_fill_zero(dw, wb / 4, st), "conv2d_bwd_filter");
    const int64_t es = esize(dt);
    TRY(need_ptr(x, "x"));
    TRY(need_ptr(dy, "dy"));
    TRY(need_align(x, es, "x"));
    TRY(need_align(dy, es, "dy"));
    const int dti = dt == TFK_F32 ? 0 : 1;
    const int64_t xb = view_bytes(xd, es), yb = view_bytes(dyd, es);
    int64_t xs = xd.pixel_stride;
    fold_full_window(s, xs);
    const size_t need = conv_bwd_filter_ws_bytes(dti, s);
    TRY(check_ws(ws, ws_bytes, need));
    if (overlap(dw, wb, x, xb) || overlap(dw, wb, dy, yb))
        return fail(TFK_ERR_ALIAS, "dw overlaps x or dy");
    if (need && (overlap(ws, (int64_t)need, x, xb) || overlap(ws, (int64_t)need, dy, yb) ||
                 overlap(ws, (int64_t)need, dw, wb)))
        return fail(TFK_ERR_ALIAS, "workspace overlaps an operand");
    return hip_status(launch_conv_bwd_filter(dti, x, xs, dy, dyd.pixel_stride, dw, s, ws, st),
                      "conv2d_bwd_filter");
}

tfk_status tfk_conv2d_bwd_filter_noalloc(const void *x, tfk_nhwc xd, const void *dy, tfk_nhwc dyd, tfk_window p,
                                         tfk_dtype dt, float *dw, void *stream) {
    RECORDED(tfk_conv2d_bwd_filter_noalloc, x, xd, dy, dyd, p, dt, dw, stream);
    ConvShape s;
    TRY(check_conv(xd, dyd.c, p, dt, dyd, "x", "dy", s));
    int64_t xs = xd.pixel_stride;
    fold_full_window(s, xs);
    const size_t need = conv_bwd_filter_ws_bytes(dt == TFK_F32 ? 0 : 1, s);
    const size_t have = noalloc_scratch_bytes();
    if (need > have)
        return fail(TFK_ERR_WORKSPACE,
                    "conv2d_bwd_filter_noalloc: this shape needs %zu bytes of scratch, more than the library's "
                    "fixed %zu bytes; use tfk_conv2d_bwd_filter with a workspace",
                    need, have);
    void *scratch = nullptr;
    if (need) {
        const hipError_t e = noalloc_scratch(&scratch, (hipStream_t)stream);
        if (e != hipSuccess) return hip_status(e, "conv2d_bwd_filter_noalloc: device scratch of the stream's GPU");
    }
    return tfk_conv2d_bwd_filter(x, xd, dy, dyd, p, dt, dw, scratch, need, stream);
}

// ------------------------------------------------------------------ bias + ReLU
tfk_status tfk_bias_relu_fwd(void *y, tfk_nhwc yd, const float *bias, tfk_dtype dt, void *stream) {
    RECORDED(tfk_bias_relu_fwd, y, yd, bias, dt, stream);
    if (!valid_dt(dt)) return fail(TFK_ERR_DTYPE, "unknown dtype %d", (int)dt);
    TRY(check_view("y", yd));
    if (yd.n == 0) return ok();
    const int64_t es = esize(dt);
    TRY(need_ptr(y, "y"));
    TRY(need_ptr(bias, "bias"));
    TRY(need_align(y, es, "y"));
    TRY(need_align(bias, 4, "bias"));
    if (overlap(y, view_bytes(yd, es), bias, (int64_t)yd.c * 4)) return fail(TFK_ERR_ALIAS, "bias overlaps y");
    const int64_t P = (int64_t)yd.n * yd.h * yd.w;
    return hip_status(launch_bias_relu_fwd(dt == TFK_F32 ? 0 : 1, y, P, yd.c, yd.pixel_stride, bias,
                                           (hipStream_t)stream),
                      "bias_relu_fwd");
}

size_t tfk_bias_relu_bwd_workspace_bytes(tfk_nhwc yd, tfk_dtype dt) {
    if (!valid_dt(dt) || check_view("y", yd) != TFK_OK || yd.n == 0) return 0;
    int G;
    int64_t ppb;
    relu_bwd_plan(dt == TFK_F32 ? 0 : 1, (int64_t)yd.n * yd.h * yd.w, yd.c, yd.pixel_stride, &G, &ppb);
    return (size_t)G * yd.c * sizeof(float);
}

tfk_status tfk_bias_relu_bwd(const void *y, const void *dy, tfk_nhwc yd, void *dpre, float *dbias, tfk_dtype dt,
                             void *ws, size_t ws_bytes, void *stream) {
    RECORDED(tfk_bias_relu_bwd, y, dy, yd, dpre, dbias, dt, ws, ws_bytes, stream);
    if (!valid_dt(dt)) return fail(TFK_ERR_DTYPE, "unknown dtype %d", (int)dt);
    TRY(check_view("y", yd));
    TRY(need_align(dbias, 4, "dbias"));
    hipStream_t st = (hipStream_t)stream;
    const int64_t es = esize(dt);
    const int64_t vb = view_bytes(yd, es);
    const int64_t bb = (int64_t)yd.c * 4;
    if (yd.n == 0) {
        if (dbias == nullptr) {
            note_partials((const float *)ws, 0);
            return ok();
        }
        return hip_status(launch_fill_zero(dbias, yd.c, st), "bias_relu_bwd");
    }
    TRY(need_ptr(dy, "dy"));
    TRY(need_ptr(dpre, "dpre"));
    TRY(need_align(y, es, "y"));
    TRY(need_align(dy, es, "dy"));
    TRY(need_align(dpre, es, "dpre"));
    if (dpre != dy && overlap(dpre, vb, dy, vb)) return fail(TFK_ERR_ALIAS, "dpre partially overlaps dy");
    if (overlap(dpre, vb, y, vb)) return fail(TFK_ERR_ALIAS, "dpre overlaps y");
    if (overlap(dbias, bb, y, vb) || overlap(dbias, bb, dy, vb) || overlap(dbias, bb, dpre, vb))
        return fail(TFK_ERR_ALIAS, "dbias overlaps a tensor");
    const size_t need = tfk_bias_relu_bwd_workspace_bytes(yd, dt);
    TRY(check_ws(ws, ws_bytes, need));
    if (overlap(ws, (int64_t)need, y, vb) || overlap(ws, (int64_t)need, dy, vb) ||
        overlap(ws, (int64_t)need, dpre, vb) || overlap(ws, (int64_t)need, dbias, bb))
        return fail(TFK_ERR_ALIAS, "workspace overlaps an operand");
    const int64_t P = (int64_t)yd.n * yd.h * yd.w;
    BiasPartials bp{nullptr, 0};
    TRY(hip_status(launch_bias_relu_bwd(dt == TFK_F32 ? 0 : 1, y, dy, dpre, P, yd.c, yd.pixel_stride, dbias,
                                        (float *)ws, st, dbias ? nullptr : &bp),
                   "bias_relu_bwd"));
    if (dbias == nullptr) note_partials(bp.part, bp.rows);
    return ok();
}

// ------------------------------------------------------------------ max-pool
static tfk_status check_pool(tfk_nhwc &xd, const tfk_window &p, tfk_dtype dt, tfk_nhwc &yd, const char *xname,
                             const char *yname, PoolGeom &g) {
    if (!valid_dt(dt)) return fail(TFK_ERR_DTYPE, "unknown dtype %d", (int)dt);
    TRY(check_view(xname, xd));
    TRY(check_view(yname, yd));
    TRY(check_window(p));
    const int oh = out_len(xd.h, p.kh, p.stride_h, p.pad_top, p.pad_bottom);
    const int ow = out_len(xd.w, p.kw, p.stride_w, p.pad_left, p.pad_right);
    if (oh < 1 || ow < 1) return fail(TFK_ERR_SHAPE, "window does not fit the padded input");
    if (yd.n != xd.n || yd.h != oh || yd.w != ow || yd.c != xd.c)
        return fail(TFK_ERR_SHAPE, "%s must be [%d,%d,%d,%d], got [%d,%d,%d,%d]", yname, xd.n, oh, ow, xd.c, yd.n,
                    yd.h, yd.w, yd.c);
    if ((int64_t)xd.n * xd.h * xd.w * xd.c > INT32_MAX)
        return fail(TFK_ERR_OVERFLOW, "%s has more than 2^31-1 elements: argmax would overflow int32", xname);
    g.N = xd.n; g.H = xd.h; g.W = xd.w; g.C = xd.c;
    g.OH = oh; g.OW = ow;
    g.KH = p.kh; g.KW = p.kw; g.sh = p.stride_h; g.sw = p.stride_w; g.pt = p.pad_top; g.pl = p.pad_left;
    g.xs = xd.pixel_stride;
    g.ys = yd.pixel_stride;
    return TFK_OK;
}

// The three max-pool entry points take the argmax as int32 dense indices or (taps) as uint8
// window taps; ab is its byte size.
static tfk_status maxpool_fwd_impl(const void *x, tfk_nhwc xd, tfk_window p, tfk_dtype dt, void *y, tfk_nhwc yd,
                                   void *argmax, bool taps, void *stream) {
    PoolGeom g;
    TRY(check_pool(xd, p, dt, yd, "x", "y", g));
    if (taps && (int64_t)p.kh * p.kw > 256) return fail(TFK_ERR_SHAPE, "tap argmax needs kh * kw <= 256");
    if (xd.n == 0) return ok();
    const int64_t es = esize(dt);
    TRY(need_ptr(x, "x"));
    TRY(need_ptr(y, "y"));
    TRY(need_ptr(argmax, "argmax"));
    TRY(need_align(x, es, "x"));
    TRY(need_align(y, es, "y"));
    TRY(need_align(argmax, taps ? 1 : 4, "argmax"));
    const int64_t xb = view_bytes(xd, es), yb = view_bytes(yd, es);
    const int64_t ab = (int64_t)yd.n * yd.h * yd.w * yd.c * (taps ? 1 : 4);
    if (overlap(y, yb, x, xb) || overlap(argmax, ab, x, xb) || overlap(argmax, ab, y, yb))
        return fail(TFK_ERR_ALIAS, "y / argmax overlap");
    return hip_status(launch_maxpool_fwd(dt == TFK_F32 ? 0 : 1, x, g, y, argmax, taps, (hipStream_t)stream),
                      "maxpool_fwd");
}

tfk_status tfk_maxpool_fwd(const void *x, tfk_nhwc xd, tfk_window p, tfk_dtype dt, void *y, tfk_nhwc yd,
                           int32_t *argmax, void *stream) {
    RECORDED(tfk_maxpool_fwd, x, xd, p, dt, y, yd, argmax, stream);
    return maxpool_fwd_impl(x, xd, p, dt, y, yd, argmax, false, stream);
}

tfk_status tfk_maxpool_fwd_taps(const void *x, tfk_nhwc xd, tfk_window p, tfk_dtype dt, void *y, tfk_nhwc yd,
                                uint8_t *taps, void *stream) {
    RECORDED(tfk_maxpool_fwd_taps, x, xd, p, dt, y, yd, taps, stream);
    return maxpool_fwd_impl(x, xd, p, dt, y, yd, taps, true, stream);
}

tfk_status tfk_conv2d_fwd_bias_relu_maxpool(const void *x, tfk_nhwc xd, const void *w, int32_t cout,
                                            const float *bias, tfk_window p, tfk_dtype dt, void *y, tfk_nhwc yd,
                                            tfk_window pp, void *py, tfk_nhwc pyd, uint8_t *taps, void *ws,
                                            size_t ws_bytes, void *stream) {
    RECORDED(tfk_conv2d_fwd_bias_relu_maxpool, x, xd, w, cout, bias, p, dt, y, yd, pp, py, pyd, taps, ws, ws_bytes, stream);
    ConvShape s;
    int64_t xs;
    size_t need;
    TRY(need_ptr(bias, "bias"));
    TRY(need_align(bias, 4, "bias"));
    TRY(conv_fwd_check(x, xd, w, cout, bias, p, dt, y, yd, ws, ws_bytes, s, xs, need));
    tfk_nhwc yin = yd;
    PoolGeom g;
    TRY(check_pool(yin, pp, dt, pyd, "y", "py", g));
    if ((int64_t)pp.kh * pp.kw > 256) return fail(TFK_ERR_SHAPE, "tap argmax needs kh * kw <= 256");
    if (xd.n == 0) return ok();
    const int64_t es = esize(dt);
    TRY(need_ptr(py, "py"));
    TRY(need_ptr(taps, "taps"));
    TRY(need_align(py, es, "py"));
    const int64_t xb = view_bytes(xd, es), wb = filter_bytes(s, es), yb = view_bytes(yd, es);
    const int64_t pb = view_bytes(pyd, es), tb = (int64_t)pyd.n * pyd.h * pyd.w * pyd.c, bb = (int64_t)cout * 4;
    if (overlap(y, yb, bias, bb)) return fail(TFK_ERR_ALIAS, "y overlaps bias");
    if (overlap(py, pb, x, xb) || overlap(py, pb, w, wb) || overlap(py, pb, y, yb) || overlap(py, pb, bias, bb))
        return fail(TFK_ERR_ALIAS, "py overlaps x, w, y or bias");
    if (overlap(taps, tb, x, xb) || overlap(taps, tb, w, wb) || overlap(taps, tb, y, yb) || overlap(taps, tb, py, pb) ||
        overlap(taps, tb, bias, bb))
        return fail(TFK_ERR_ALIAS, "taps overlap a tensor");
    if (need && (overlap(ws, (int64_t)need, py, pb) || overlap(ws, (int64_t)need, taps, tb)))
        return fail(TFK_ERR_ALIAS, "workspace overlaps an operand");
    hipStream_t st = (hipStream_t)stream;
    const char *what = "conv2d_fwd_bias_relu_maxpool";
    if (dt == TFK_BF16) {
        hipError_t e;
        if (conv_fwd_pool_fused(x, xs, w, y, yd.pixel_stride, s, bias, g, py, pyd.pixel_stride, taps, st, &e))
            return hip_status(e, what);
    }
    // not one kernel for this shape: the convolution, then the max-pool of y
    const hipError_t e = launch_conv_fwd(dt == TFK_F32 ? 0 : 1, x, xs, w, y, yd.pixel_stride, s, bias,
                                         need ? ws : nullptr, st);
    if (e != hipSuccess) return hip_status(e, what);
    return hip_status(launch_maxpool_fwd(dt == TFK_F32 ? 0 : 1, y, g, py, taps, true, st), what);
}

static tfk_status maxpool_bwd_impl(const void *dy, const void *argmax, bool taps, tfk_nhwc yd, tfk_window p,
                                   tfk_dtype dt, void *dx, tfk_nhwc xd, float beta, void *stream) {
    PoolGeom g;
    TRY(check_pool(xd, p, dt, yd, "dx", "dy", g));
    if (!(beta == 0.f || beta == 1.f)) return fail(TFK_ERR_ARG, "beta must be 0 or 1");
    if (taps && (int64_t)p.kh * p.kw > 256) return fail(TFK_ERR_SHAPE, "tap argmax needs kh * kw <= 256");
    if (xd.n == 0) return ok();
    const int64_t es = esize(dt);
    TRY(need_ptr(dy, "dy"));
    TRY(need_ptr(argmax, "argmax"));
    TRY(need_ptr(dx, "dx"));
    TRY(need_align(dy, es, "dy"));
    TRY(need_align(dx, es, "dx"));
    TRY(need_align(argmax, taps ? 1 : 4, "argmax"));
    const int64_t xb = view_bytes(xd, es), yb = view_bytes(yd, es);
    const int64_t ab = (int64_t)yd.n * yd.h * yd.w * yd.c * (taps ? 1 : 4);
    if (overlap(dx, xb, dy, yb) || overlap(dx, xb, argmax, ab)) return fail(TFK_ERR_ALIAS, "dx overlaps dy or argmax");
    return hip_status(launch_maxpool_bwd(dt == TFK_F32 ? 0 : 1, dy, argmax, taps, g, beta, dx, (hipStream_t)stream),
                      "maxpool_bwd");
}

tfk_status tfk_maxpool_bwd(const void *dy, const int32_t *argmax, tfk_nhwc yd, tfk_window p, tfk_dtype dt,
                           void *dx, tfk_nhwc xd, float beta, void *stream) {
    RECORDED(tfk_maxpool_bwd, dy, argmax, yd, p, dt, dx, xd, beta, stream);
    return maxpool_bwd_impl(dy, argmax, false, yd, p, dt, dx, xd, beta, stream);
}

tfk_status tfk_maxpool_bwd_taps(const void *dy, const uint8_t *taps, tfk_nhwc yd, tfk_window p, tfk_dtype dt,
                                void *dx, tfk_nhwc xd, float beta, void *stream) {
    RECORDED(tfk_maxpool_bwd_taps, dy, taps, yd, p, dt, dx, xd, beta, stream);
    return maxpool_bwd_impl(dy, taps, true, yd, p, dt, dx, xd, beta, stream);
}

static tfk_status maxpool_relu_bwd_impl(const void *dy, const void *argmax, bool taps, tfk_nhwc yd, tfk_window p,
                                        tfk_dtype dt, const void *y, const void *py, int64_t py_stride, void *dpre,
                                        tfk_nhwc xd, float beta, float *dbias, void *ws, size_t ws_bytes,
                                        void *stream) {
    PoolGeom g;
    TRY(check_pool(xd, p, dt, yd, "y", "dy", g));
    if (!(beta == 0.f || beta == 1.f)) return fail(TFK_ERR_ARG, "beta must be 0 or 1");
    if (xd.c > 16384) return fail(TFK_ERR_SHAPE, "maxpool_bwd_relu_bwd supports at most 16384 channels");
    if (taps && (int64_t)p.kh * p.kw > 256) return fail(TFK_ERR_SHAPE, "tap argmax needs kh * kw <= 256");
    TRY(need_align(dbias, 4, "dbias"));
    hipStream_t st = (hipStream_t)stream;
    if (xd.n == 0) {
        if (dbias == nullptr) {
            note_partials((const float *)ws, 0);
            return ok();
        }
        return hip_status(launch_fill_zero(dbias, xd.c, st), "maxpool_bwd_relu_bwd");
    }
    const int64_t es = esize(dt);
    TRY(need_ptr(dy, "dy"));
    TRY(need_ptr(argmax, "argmax"));
    // the pool's output replaces y as the mask when the gradient is not accumulated
    if (beta != 0.f) py = nullptr;
    if (py == nullptr) TRY(need_ptr(y, "y"));
    else y = nullptr;
    TRY(need_ptr(dpre, "dpre"));
    TRY(need_align(dy, es, "dy"));
    TRY(need_align(y, es, "y"));
    TRY(need_align(py, es, "py"));
    TRY(need_align(dpre, es, "dpre"));
    TRY(need_align(argmax, taps ? 1 : 4, "argmax"));
    tfk_nhwc pyd = yd;
    pyd.pixel_stride = py_stride;
    if (py != nullptr && py_stride < yd.c) return fail(TFK_ERR_SHAPE, "py_stride is below the channel count");
    const int64_t xb = view_bytes(xd, es), yb = view_bytes(yd, es), pb = py ? view_bytes(pyd, es) : 0;
    const int64_t ab = (int64_t)yd.n * yd.h * yd.w * yd.c * (taps ? 1 : 4), bb = (int64_t)xd.c * 4;
    if (overlap(dpre, xb, y, xb) || overlap(dpre, xb, dy, yb) || overlap(dpre, xb, argmax, ab) ||
        overlap(dpre, xb, py, pb))
        return fail(TFK_ERR_ALIAS, "dpre overlaps y, py, dy or argmax");
    if (overlap(dbias, bb, y, xb) || overlap(dbias, bb, dy, yb) || overlap(dbias, bb, dpre, xb) ||
        overlap(dbias, bb, argmax, ab) || overlap(dbias, bb, py, pb))
        return fail(TFK_ERR_ALIAS, "dbias overlaps a tensor");
    const size_t need = tfk_bias_relu_bwd_workspace_bytes(xd, dt);
    TRY(check_ws(ws, ws_bytes, need));
    if (overlap(ws, (int64_t)need, y, xb) || overlap(ws, (int64_t)need, dy, yb) ||
        overlap(ws, (int64_t)need, dpre, xb) || overlap(ws, (int64_t)need, dbias, bb) ||
        overlap(ws, (int64_t)need, argmax, ab) || overlap(ws, (int64_t)need, py, pb))
        return fail(TFK_ERR_ALIAS, "workspace overlaps an operand");
    BiasPartials bp{nullptr, 0};
    TRY(hip_status(launch_maxpool_relu_bwd(dt == TFK_F32 ? 0 : 1, dy, argmax, taps, g, y, py, py_stride, dpre, beta,
                                           dbias, (float *)ws, st, dbias ? nullptr : &bp),
                   "maxpool_bwd_relu_bwd"));
    if (dbias == nullptr) note_partials(bp.part, bp.rows);
    return ok();
}

tfk_status tfk_maxpool_bwd_relu_bwd(const void *dy, const int32_t *argmax, tfk_nhwc yd, tfk_window p, tfk_dtype dt,
                                    const void *y, const void *py, int64_t py_stride, void *dpre, tfk_nhwc xd,
                                    float beta, float *dbias, void *ws, size_t ws_bytes, void *stream) {
    RECORDED(tfk_maxpool_bwd_relu_bwd, dy, argmax, yd, p, dt, y, py, py_stride, dpre, xd, beta, dbias, ws, ws_bytes,
             stream);
    return maxpool_relu_bwd_impl(dy, argmax, false, yd, p, dt, y, py, py_stride, dpre, xd, beta, dbias, ws, ws_bytes,
                                 stream);
}

tfk_status tfk_maxpool_bwd_relu_bwd_taps(const void *dy, const uint8_t *taps, tfk_nhwc yd, tfk_window p, tfk_dtype dt,
                                         const void *y, const void *py, int64_t py_stride, void *dpre, tfk_nhwc xd,
                                         float beta, float *dbias, void *ws, size_t ws_bytes, void *stream) {
    RECORDED(tfk_maxpool_bwd_relu_bwd_taps, dy, taps, yd, p, dt, y, py, py_stride, dpre, xd, beta, dbias, ws,
             ws_bytes, stream);
    return maxpool_relu_bwd_impl(dy, taps, true, yd, p, dt, y, py, py_stride, dpre, xd, beta, dbias, ws, ws_bytes,
                                 stream);
}

// ------------------------------------------------------------------ deferred bias gradients
tfk_status tfk_last_bias_partials(const float **part, int32_t *rows) {
    TRY(need_ptr(part, "part"));
    TRY(need_ptr(rows, "rows"));
    if (!g_partials.valid) return fail(TFK_ERR_ARG, "no call on this thread has left bias-gradient partials");
    *part = g_partials.part;
    *rows = g_partials.rows;
    return ok();
}

tfk_status tfk_bias_grad_finish(int32_t count, const float *const *parts, const int32_t *rows,
                                const int32_t *channels, float *const *dbias, void *stream) {
    if (g_rec != nullptr && count > 0 && parts != nullptr && rows != nullptr && channels != nullptr &&
        dbias != nullptr) {
        // the arrays belong to the caller: the recorded call keeps copies of them
        tfk_program *const rec_ = g_rec;
        g_rec = nullptr;
        const tfk_status s_ = tfk_bias_grad_finish(count, parts, rows, channels, dbias, stream);
        g_rec = rec_;
        if (s_ != TFK_OK) return s_;
        try {
            std::vector<const float *> p(parts, parts + count);
            std::vector<int32_t> r(rows, rows + count), c(channels, channels + count);
            std::vector<float *> d(dbias, dbias + count);
            rec_->calls.emplace_back(
                [=]() { return tfk_bias_grad_finish(count, p.data(), r.data(), c.data(), d.data(), stream); });
        } catch (...) {
            return fail(TFK_ERR_ARG, "tfk_bias_grad_finish: out of host memory while recording");
        }
        return s_;
    }
    if (count < 0) return fail(TFK_ERR_ARG, "count must be >= 0");
    if (count == 0) return ok();
    TRY(need_ptr(parts, "parts"));
    TRY(need_ptr(rows, "rows"));
    TRY(need_ptr(channels, "channels"));
    TRY(need_ptr(dbias, "dbias"));
    std::vector<int> r(count), c(count);
    for (int i = 0; i < count; ++i) {
        if (rows[i] < 0 || channels[i] < 1 || channels[i] > 16384)
            return fail(TFK_ERR_SHAPE, "tensor %d: rows must be >= 0 and channels in 1..16384", i);
        if (rows[i] > 0) {
            TRY(need_ptr(parts[i], "parts[i]"));
            TRY(need_align(parts[i], 4, "parts[i]"));
        }
        TRY(need_ptr(dbias[i], "dbias[i]"));
        TRY(need_align(dbias[i], 4, "dbias[i]"));
        const int64_t bb = (int64_t)channels[i] * 4;
        for (int j = 0; j < count; ++j) {
            if (overlap(dbias[i], bb, parts[j], (int64_t)rows[j] * channels[j] * 4))
                return fail(TFK_ERR_ALIAS, "dbias[%d] overlaps the partials of tensor %d", i, j);
            if (j != i && overlap(dbias[i], bb, dbias[j], (int64_t)channels[j] * 4))
                return fail(TFK_ERR_ALIAS, "dbias[%d] overlaps dbias[%d]", i, j);
        }
        r[i] = rows[i];
        c[i] = channels[i];
    }
    return hip_status(launch_sum_partials_multi(count, parts, r.data(), c.data(), dbias, (hipStream_t)stream),
                      "bias_grad_finish");
}

// ------------------------------------------------------------------ SGD
static tfk_status check_sgd(float *var, const float *grad, int64_t n, float lr, uint16_t *sh) {
    if (n < 0) return fail(TFK_ERR_SHAPE, "n must be >= 0");
    if (!isfinite(lr)) return fail(TFK_ERR_ARG, "lr must be finite");
    if (n == 0) return TFK_OK;
    TRY(need_ptr(var, "var"));
    TRY(need_ptr(grad, "grad"));
    TRY(need_align(var, 4, "var"));
    TRY(need_align(grad, 4, "grad"));
    TRY(need_align(sh, 2, "var_bf16"));
    if (n > ((int64_t)1 << 40)) return fail(TFK_ERR_OVERFLOW, "n too large");
    if (overlap(var, n * 4, grad, n * 4) || overlap(var, n * 4, sh, n * 2) || overlap(grad, n * 4, sh, n * 2))
        return fail(TFK_ERR_ALIAS, "var, grad and var_bf16 must not overlap");
    return TFK_OK;
}

tfk_status tfk_apply_sgd(float *var, const float *grad, int64_t n, float lr, uint16_t *var_bf16, void *stream) {
    RECORDED(tfk_apply_sgd, var, grad, n, lr, var_bf16, stream);
    TRY(check_sgd(var, grad, n, lr, var_bf16));
    if (n == 0) return ok();
    return hip_status(launch_sgd(var, grad, n, lr, var_bf16, (hipStream_t)stream), "apply_sgd");
}

tfk_status tfk_apply_sgd_multi(int32_t count, float *const *vars, const float *const *grads, const int64_t *ns,
                               float lr, uint16_t *const *shadows, void *stream) {
    if (g_rec != nullptr && count > 0 && vars != nullptr && grads != nullptr && ns != nullptr) {
        // the pointer arrays belong to the caller: the recorded call keeps copies of them
        tfk_program *const rec_ = g_rec;
        g_rec = nullptr;
        const tfk_status s_ = tfk_apply_sgd_multi(count, vars, grads, ns, lr, shadows, stream);
        g_rec = rec_;
        if (s_ != TFK_OK) return s_;
        try {
            std::vector<float *> v(vars, vars + count);
            std::vector<const float *> g(grads, grads + count);
            std::vector<int64_t> n(ns, ns + count);
            std::vector<uint16_t *> sh;
            if (shadows != nullptr) sh.assign(shadows, shadows + count);
            rec_->calls.emplace_back([=]() {
                return tfk_apply_sgd_multi(count, v.data(), g.data(), n.data(), lr,
                                           sh.empty() ? nullptr : sh.data(), stream);
            });
        } catch (...) {
            return fail(TFK_ERR_ARG, "tfk_apply_sgd_multi: out of host memory while recording");
        }
        return s_;
    }
    if (count < 0) return fail(TFK_ERR_ARG, "count must be >= 0");
    if (count == 0) return ok();
    TRY(need_ptr(vars, "vars"));
    TRY(need_ptr(grads, "grads"));
    TRY(need_ptr(ns, "ns"));
    for (int i = 0; i < count; ++i) {
        tfk_status s = check_sgd(vars[i], grads[i], ns[i], lr, shadows ? shadows[i] : nullptr);
        if (s != TFK_OK) return fail(s, "tensor %d: %s", i, g_err.c_str());
    }
    hipStream_t st = (hipStream_t)stream;
    int i = 0;
    while (i < count) {
        SgdBatch b;
        b.count = 0;
        b.blk_start[0] = 0;
        for (; i < count && b.count < kSgdBatch; ++i) {
            if (ns[i] == 0) continue;
            const int k = b.count++;
            b.var[k] = vars[i];
            b.grad[k] = grads[i];
            b.shadow[k] = shadows ? shadows[i] : nullptr;
            b.n[k] = ns[i];
            b.blk_start[k + 1] = b.blk_start[k] + (ns[i] + 1023) / 1024;
        }
        if (b.count == 0) continue;
        if (b.blk_start[b.count] > INT32_MAX) return fail(TFK_ERR_OVERFLOW, "too many elements in one batch");
        hipError_t e = launch_sgd_multi(b, lr, st);
        if (e != hipSuccess) return hip_status(e, "apply_sgd_multi");
    }
    return ok();
}

// ------------------------------------------------------------------ softmax cross-entropy
tfk_status tfk_softmax_xent(const void *logits, tfk_dtype dt, int64_t n, int32_t c, const float *bias,
                            const int32_t *labels, float scale, float *loss, void *dlogits, void *stream) {
    RECORDED(tfk_softmax_xent, logits, dt, n, c, bias, labels, scale, loss, dlogits, stream);
    if (!valid_dt(dt)) return fail(TFK_ERR_DTYPE, "unknown dtype %d", (int)dt);
    if (n < 0 || c < 1) return fail(TFK_ERR_SHAPE, "need n >= 0 and c >= 1 (n=%lld, c=%d)", (long long)n, c);
    if (!isfinite(scale)) return fail(TFK_ERR_ARG, "scale must be finite");
    if (n == 0) return ok();
    if (n > ((int64_t)1 << 40) / c) return fail(TFK_ERR_OVERFLOW, "n * c too large");
    const int64_t es = esize(dt), zb = n * c * es;
    TRY(need_ptr(logits, "logits"));
    TRY(need_ptr(labels, "labels"));
    TRY(need_ptr(loss, "loss"));
    TRY(need_ptr(dlogits, "dlogits"));
    TRY(need_align(logits, es, "logits"));
    TRY(need_align(dlogits, es, "dlogits"));
    TRY(need_align(bias, 4, "bias"));
    TRY(need_align(labels, 4, "labels"));
    TRY(need_align(loss, 4, "loss"));
    if (dlogits != logits && overlap(dlogits, zb, logits, zb))
        return fail(TFK_ERR_ALIAS, "dlogits partially overlaps logits");
    const void *p[5] = {dlogits, bias, labels, loss, logits};
    const int64_t b[5] = {zb, (int64_t)c * 4, n * 4, n * 4, zb};
    for (int i = 0; i < 4; ++i)
        for (int j = i + 1; j < 5; ++j)
            if (!(i == 0 && j == 4) && overlap(p[i], b[i], p[j], b[j]))
                return fail(TFK_ERR_ALIAS, "softmax_xent operands overlap");
    if (n > INT32_MAX) return fail(TFK_ERR_OVERFLOW, "too many rows");
    return hip_status(launch_softmax_xent(dt == TFK_F32 ? 0 : 1, logits, bias, labels, n, c, scale, loss, dlogits,
                                          (hipStream_t)stream),
                      "softmax_xent");
}

// ------------------------------------------------------------------ sampled softmax
tfk_status tfk_gather_rows_t(const void *table, tfk_dtype dt, int64_t rows, int32_t d, const int32_t *idx, int32_t u,
                             int32_t u_pad, void *out_t, void *stream) {
    RECORDED(tfk_gather_rows_t, table, dt, rows, d, idx, u, u_pad, out_t, stream);
    if (!valid_dt(dt)) return fail(TFK_ERR_DTYPE, "unknown dtype %d", (int)dt);
    if (rows < 0 || d < 1 || u < 0 || u_pad < u) return fail(TFK_ERR_SHAPE, "need rows >= 0, d >= 1, 0 <= u <= u_pad");
    if ((int64_t)d * u_pad == 0) return ok();
    if ((int64_t)d * u_pad > ((int64_t)1 << 40) || rows > ((int64_t)1 << 40) / d)
        return fail(TFK_ERR_OVERFLOW, "sizes too large");
    const int64_t es = esize(dt);
    TRY(need_ptr(out_t, "out_t"));
    if (u > 0) {
        TRY(need_ptr(table, "table"));
        TRY(need_ptr(idx, "idx"));
    }
    TRY(need_align(table, es, "table"));
    TRY(need_align(out_t, es, "out_t"));
    TRY(need_align(idx, 4, "idx"));
    const int64_t ob = (int64_t)d * u_pad * es;
    if (overlap(out_t, ob, table, rows * d * es) || overlap(out_t, ob, idx, (int64_t)u * 4))
        return fail(TFK_ERR_ALIAS, "out_t overlaps table or idx");
    return hip_status(launch_gather_rows_t(dt == TFK_F32 ? 0 : 1, table, rows, d, idx, u, u_pad, out_t,
                                           (hipStream_t)stream),
                      "gather_rows_t");
}

tfk_status tfk_sampled_softmax_xent(const void *z, tfk_dtype dt, int64_t n, int32_t u, int32_t u_pad, int32_t m,
                                    const float *bias_c, const int32_t *true_pos, const float *lq_true,
                                    const float *lq_sampled, float scale, float *loss, void *dz, void *stream) {
    RECORDED(tfk_sampled_softmax_xent, z, dt, n, u, u_pad, m, bias_c, true_pos, lq_true, lq_sampled, scale, loss, dz, stream);
    if (!valid_dt(dt)) return fail(TFK_ERR_DTYPE, "unknown dtype %d", (int)dt);
    if (n < 0 || m < 0 || u < m || u < 1 || u_pad < u)
        return fail(TFK_ERR_SHAPE, "need n >= 0 and 0 <= m <= u <= u_pad, u >= 1");
    if (!isfinite(scale)) return fail(TFK_ERR_ARG, "scale must be finite");
    if (n == 0) return ok();
    if (n > INT32_MAX || n > ((int64_t)1 << 40) / u_pad) return fail(TFK_ERR_OVERFLOW, "n * u_pad too large");
    const int64_t es = esize(dt), zb = n * u_pad * es;
    TRY(need_ptr(z, "z"));
    TRY(need_ptr(true_pos, "true_pos"));
    TRY(need_ptr(lq_true, "lq_true"));
    if (m > 0) TRY(need_ptr(lq_sampled, "lq_sampled"));
    TRY(need_ptr(loss, "loss"));
    TRY(need_ptr(dz, "dz"));
    TRY(need_align(z, es, "z"));
    TRY(need_align(dz, es, "dz"));
    TRY(need_align(bias_c, 4, "bias_c"));
    TRY(need_align(true_pos, 4, "true_pos"));
    TRY(need_align(lq_true, 4, "lq_true"));
    TRY(need_align(lq_sampled, 4, "lq_sampled"));
    TRY(need_align(loss, 4, "loss"));
    const void *p[7] = {dz, loss, z, bias_c, true_pos, lq_true, lq_sampled};
    const int64_t b[7] = {zb, n * 4, zb, (int64_t)u_pad * 4, n * 4, n * 4, (int64_t)m * 4};
    for (int i = 0; i < 2; ++i)
        for (int j = i + 1; j < 7; ++j)
            if (overlap(p[i], b[i], p[j], b[j])) return fail(TFK_ERR_ALIAS, "dz or loss overlaps an operand");
    return hip_status(launch_sampled_xent(dt == TFK_F32 ? 0 : 1, z, n, u, u_pad, m, bias_c, true_pos, lq_true,
                                          lq_sampled, scale, loss, dz, (hipStream_t)stream),
                      "sampled_softmax_xent");
}

tfk_status tfk_scatter_apply_sgd(float *var, uint16_t *var_bf16, int64_t rows, int32_t d, const int32_t *idx,
                                 int32_t u, const float *grad_t, int64_t ld, float lr, void *stream) {
    RECORDED(tfk_scatter_apply_sgd, var, var_bf16, rows, d, idx, u, grad_t, ld, lr, stream);
    if (rows < 0 || d < 1 || u < 0 || ld < u) return fail(TFK_ERR_SHAPE, "need rows >= 0, d >= 1, 0 <= u <= ld");
    if (!isfinite(lr)) return fail(TFK_ERR_ARG, "lr must be finite");
    if (u == 0) return ok();
    if ((int64_t)d * ld > ((int64_t)1 << 40) || rows > ((int64_t)1 << 40) / d)
        return fail(TFK_ERR_OVERFLOW, "sizes too large");
    TRY(need_ptr(var, "var"));
    TRY(need_ptr(idx, "idx"));
    TRY(need_ptr(grad_t, "grad_t"));
    TRY(need_align(var, 4, "var"));
    TRY(need_align(var_bf16, 2, "var_bf16"));
    TRY(need_align(idx, 4, "idx"));
    TRY(need_align(grad_t, 4, "grad_t"));
    const int64_t vb = rows * d * 4, gb = (int64_t)d * ld * 4;
    if (overlap(var, vb, grad_t, gb) || overlap(var, vb, idx, (int64_t)u * 4) || overlap(var, vb, var_bf16, rows * d * 2) ||
        overlap(var_bf16, rows * d * 2, grad_t, gb) || overlap(var_bf16, rows * d * 2, idx, (int64_t)u * 4))
        return fail(TFK_ERR_ALIAS, "var or var_bf16 overlaps an operand");
    return hip_status(launch_scatter_sgd(var, var_bf16, rows, d, idx, u, grad_t, ld, lr, (hipStream_t)stream),
                      "scatter_apply_sgd");
}

// ------------------------------------------------------------------ Momentum, Adam
static tfk_status check_slots(float *var, const float *grad, const float *s1, const float *s2, int64_t n,
                              uint16_t *sh, const char *n1, const char *n2) {
    if (n < 0) return fail(TFK_ERR_SHAPE, "n must be >= 0");
    if (n == 0) return TFK_OK;
    TRY(need_ptr(var, "var"));
    TRY(need_ptr(grad, "grad"));
    TRY(need_ptr(s1, n1));
    if (n2) TRY(need_ptr(s2, n2));
    TRY(need_align(var, 4, "var"));
    TRY(need_align(grad, 4, "grad"));
    TRY(need_align(s1, 4, n1));
    if (n2) TRY(need_align(s2, 4, n2));
    TRY(need_align(sh, 2, "var_bf16"));
    if (n > ((int64_t)1 << 40)) return fail(TFK_ERR_OVERFLOW, "n too large");
    const void *p[5] = {var, grad, s1, n2 ? s2 : nullptr, sh};
    const int64_t b[5] = {n * 4, n * 4, n * 4, n * 4, n * 2};
    for (int i = 0; i < 5; ++i)
        for (int j = i + 1; j < 5; ++j)
            if (overlap(p[i], b[i], p[j], b[j]))
                return fail(TFK_ERR_ALIAS, "var, grad, %s%s%s and var_bf16 must not overlap", n1, n2 ? ", " : "",
                            n2 ? n2 : "");
    return TFK_OK;
}

tfk_status tfk_apply_momentum(float *var, float *accum, const float *grad, int64_t n, float lr, float momentum,
                              int32_t nesterov, uint16_t *var_bf16, void *stream) {
    RECORDED(tfk_apply_momentum, var, accum, grad, n, lr, momentum, nesterov, var_bf16, stream);
    if (!isfinite(lr)) return fail(TFK_ERR_ARG, "lr must be finite");
    if (!isfinite(momentum)) return fail(TFK_ERR_ARG, "momentum must be finite");
    if (nesterov != 0 && nesterov != 1) return fail(TFK_ERR_ARG, "nesterov must be 0 or 1");
    TRY(check_slots(var, grad, accum, nullptr, n, var_bf16, "accum", nullptr));
    if (n == 0) return ok();
    OptParams p{};
    p.lr = lr;
    p.mom = momentum;
    return hip_status(launch_opt(nesterov ? 1 : 0, var, accum, nullptr, grad, n, p, var_bf16, (hipStream_t)stream),
                      "apply_momentum");
}

tfk_status tfk_apply_adam(float *var, float *m, float *v, const float *grad, int64_t n, float lr, float beta1,
                          float beta2, float epsilon, int64_t t, uint16_t *var_bf16, void *stream) {
    RECORDED(tfk_apply_adam, var, m, v, grad, n, lr, beta1, beta2, epsilon, t, var_bf16, stream);
    if (!isfinite(lr)) return fail(TFK_ERR_ARG, "lr must be finite");
    if (!(beta1 >= 0.f && beta1 < 1.f)) return fail(TFK_ERR_ARG, "beta1 must be in [0, 1)");
    if (!(beta2 >= 0.f && beta2 < 1.f)) return fail(TFK_ERR_ARG, "beta2 must be in [0, 1)");
    if (!(epsilon >= 0.f) || !isfinite(epsilon)) return fail(TFK_ERR_ARG, "epsilon must be finite and >= 0");
    if (t < 1) return fail(TFK_ERR_ARG, "t must be >= 1");
    TRY(check_slots(var, grad, m, v, n, var_bf16, "m", "v"));
    if (n == 0) return ok();
    const double c1 = 1.0 - pow((double)beta1, (double)t), c2 = 1.0 - pow((double)beta2, (double)t);
    OptParams p{};
    p.lr = (float)((double)lr / c1);
    p.b1 = beta1;
    p.omb1 = (float)(1.0 - (double)beta1);
    p.b2 = beta2;
    p.omb2 = (float)(1.0 - (double)beta2);
    p.rc2 = (float)(1.0 / c2);
    p.eps = epsilon;
    if (!isfinite(p.lr) || !isfinite(p.rc2)) return fail(TFK_ERR_OVERFLOW, "bias-corrected step overflows fp32");
    return hip_status(launch_opt(2, var, m, v, grad, n, p, var_bf16, (hipStream_t)stream), "apply_adam");
}

// ------------------------------------------------------------------ streams and programs
tfk_status tfk_stream_wait(void *waiter, void *producer) {
    if (waiter == producer) return ok();
    if (g_rec != nullptr) {
        auto ev = std::make_shared<OwnedEvent>();
        hipError_t r = hipEventCreateWithFlags(&ev->e, kJoinEventFlags);
        if (r != hipSuccess) {
            ev->e = nullptr;
            return hip_status(r, "stream_wait");
        }
        TRY(join(ev->e, (hipStream_t)waiter, (hipStream_t)producer));
        try {
            g_rec->calls.emplace_back([=]() { return join(ev->e, (hipStream_t)waiter, (hipStream_t)producer); });
        } catch (...) {
            return fail(TFK_ERR_ARG, "tfk_stream_wait: out of host memory while recording");
        }
        return ok();
    }
    hipEvent_t e;
    hipError_t r = hipEventCreateWithFlags(&e, kJoinEventFlags);
    if (r != hipSuccess) return hip_status(r, "stream_wait");
    const tfk_status s = join(e, (hipStream_t)waiter, (hipStream_t)producer);
    (void)hipEventDestroy(e);      // released once the recorded work completes
    return s;
}

// A point on one stream that work on other streams can wait for: the event of its latest record.
struct tfk_mark {
    hipEvent_t e = nullptr;
};

tfk_status tfk_mark_create(tfk_mark **mark) {
    TRY(need_ptr(mark, "mark"));
    *mark = nullptr;
    tfk_mark *m = new (std::nothrow) tfk_mark();
    if (m == nullptr) return fail(TFK_ERR_ARG, "tfk_mark_create: out of host memory");
    const hipError_t r = hipEventCreateWithFlags(&m->e, kJoinEventFlags);
    if (r != hipSuccess) {
        delete m;
        return hip_status(r, "mark_create");
    }
    *mark = m;
    return ok();
}

void tfk_mark_destroy(tfk_mark *mark) {
    if (mark == nullptr) return;
    (void)hipEventDestroy(mark->e);
    delete mark;
}

tfk_status tfk_mark_record(tfk_mark *mark, void *stream) {
    TRY(need_ptr(mark, "mark"));
    RECORDED(tfk_mark_record, mark, stream);
    return hip_status(hipEventRecord(mark->e, (hipStream_t)stream), "mark_record");
}

tfk_status tfk_stream_wait_mark(void *waiter, tfk_mark *mark) {
    TRY(need_ptr(mark, "mark"));
    RECORDED(tfk_stream_wait_mark, waiter, mark);
    return hip_status(hipStreamWaitEvent((hipStream_t)waiter, mark->e, 0), "stream_wait_mark");
}

tfk_status tfk_program_create(tfk_program **prog) {
    TRY(need_ptr(prog, "prog"));
    try {
        *prog = new tfk_program();
    } catch (...) {
        *prog = nullptr;
        return fail(TFK_ERR_ARG, "out of host memory");
    }
    return ok();
}

void tfk_program_destroy(tfk_program *prog) {
    if (prog == nullptr) return;
    if (g_rec == prog) g_rec = nullptr;
    delete prog;
}

tfk_status tfk_program_begin(tfk_program *prog) {
    TRY(need_ptr(prog, "prog"));
    if (g_rec != nullptr) return fail(TFK_ERR_ARG, "a program is already recording on this thread");
    prog->calls.clear();
    g_rec = prog;
    return ok();
}

tfk_status tfk_program_end(tfk_program *prog) {
    TRY(need_ptr(prog, "prog"));
    if (g_rec != prog) return fail(TFK_ERR_ARG, "this program is not recording on this thread");
    g_rec = nullptr;
    return ok();
}

int64_t tfk_program_length(const tfk_program *prog) { return prog == nullptr ? 0 : (int64_t)prog->calls.size(); }

tfk_status tfk_program_run(tfk_program *prog) {
    TRY(need_ptr(prog, "prog"));
    if (g_rec != nullptr) return fail(TFK_ERR_ARG, "cannot run a program while one is recording on this thread");
    for (const auto &call : prog->calls) TRY(call());
    return ok();
}

}  // extern "C"
