// kf355_api.cpp -- the C ABI declared in include/kf355.h.  Each entry point
// validates its arguments on the host (no HIP call happens before the
// arguments are known good), derives the dense 3-D view the kernels work on,
// and hands over to the launch code of its operator.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "kf355.h"
#include "kf_internal.h"

namespace kf {
namespace {
thread_local char g_error[512] = "";
thread_local const char* g_variant = "";
}  // namespace

void set_error(const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_error, sizeof g_error, fmt, ap);
    va_end(ap);
}

namespace {

kf_status fail(kf_status s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_error, sizeof g_error, fmt, ap);
    va_end(ap);
    return s;
}

bool dtype_ok(int t) { return t == KF_FLOAT32 || t == KF_BFLOAT16 || t == KF_FLOAT16; }

int64_t elem_bytes(kf_dtype t) { return t == KF_FLOAT32 ? 4 : 2; }

// Number of elements, or -1 on a negative size or int64 overflow.
int64_t count(int32_t ndim, const int64_t* shape) {
    int64_t n = 1;
    for (int32_t i = 0; i < ndim; ++i) {
        if (shape[i] < 0) return -1;
        if (shape[i] != 0 && n > INT64_MAX / shape[i]) return -1;
        n *= shape[i];
    }
    return n;
}

// Dense row-major check; dimensions of size 1 may carry any stride.
bool dense(int32_t ndim, const int64_t* shape, const int64_t* strides) {
    if (!strides) return true;
    int64_t expect = 1;
    for (int32_t i = ndim - 1; i >= 0; --i) {
        if (shape[i] != 1 && strides[i] != expect) return false;
        expect *= shape[i];
    }
    return true;
}

// Dense channels-last [N, C, H, W] (memory order N, H, W, C); dimensions of
// size 1 may carry any stride.
bool dense_nhwc(const int64_t* shape, const int64_t* strides) {
    if (!strides) return false;
    static const int order[4] = {1, 3, 2, 0};  // innermost first: C, W, H, N
    int64_t expect = 1;
    for (int k = 0; k < 4; ++k) {
        const int i = order[k];
        if (shape[i] != 1 && strides[i] != expect) return false;
        expect *= shape[i];
    }
    return true;
}

// PyTorch's pooling output length (see kf_max_pool2d_output_size).
// Division rounding toward -infinity (b > 0): the span below is negative
// when the dilated kernel is longer than the padded input, and ceil mode
// can still produce one window then.
int64_t floor_div(int64_t a, int64_t b) { return a >= 0 ? a / b : -((-a + b - 1) / b); }

int64_t pool_out(int64_t n, int64_t k, int64_t s, int64_t p, int64_t d, bool ceil_mode) {
    const int64_t span = n + 2 * p - d * (k - 1) - 1;
    int64_t out = floor_div(span + (ceil_mode ? s - 1 : 0), s) + 1;
    if (ceil_mode && (out - 1) * s >= n + p) --out;
    return out;
}

// Window {kh, kw, sh, sw, ph, pw, dh, dw}: positive sizes, strides and
// dilations, padding at most half the kernel (PyTorch's rule).
kf_status check_window(const int64_t* win) {
    if (!win) return fail(KF_ERR_NULL_POINTER, "window is NULL");
    for (int i = 0; i < 8; ++i)
        if (win[i] > INT32_MAX) return fail(KF_ERR_BAD_ARG, "window entry %d too large", i);
    if (win[0] < 1 || win[1] < 1) return fail(KF_ERR_BAD_ARG, "kernel size must be >= 1");
    if (win[2] < 1 || win[3] < 1) return fail(KF_ERR_BAD_ARG, "stride must be >= 1");
    if (win[6] < 1 || win[7] < 1) return fail(KF_ERR_BAD_ARG, "dilation must be >= 1");
    if (win[4] < 0 || win[5] < 0 || win[4] > win[0] / 2 || win[5] > win[1] / 2)
        return fail(KF_ERR_BAD_ARG, "padding must be in [0, kernel / 2]");
    return KF_OK;
}

// Byte ranges [a, a+na) and [b, b+nb) share a byte.
bool overlaps(const void* a, int64_t na, const void* b, int64_t nb) {
    const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
    return pa < pb + (uintptr_t)nb && pb < pa + (uintptr_t)na;
}

kf_status check_shape(int32_t ndim, const int64_t* shape, int32_t lo, int32_t hi, int64_t* n) {
    if (ndim < lo || ndim > hi) return fail(KF_ERR_BAD_SHAPE, "ndim %d outside [%d, %d]", ndim, lo, hi);
    if (ndim > 0 && !shape) return fail(KF_ERR_NULL_POINTER, "shape is NULL");
    *n = count(ndim, shape);
    if (*n < 0) return fail(KF_ERR_BAD_SHAPE, "negative size or element count overflows int64");
    return KF_OK;
}

// The dense [outer, len, inner] view of a softmax over `dim` (wrapped), and
// the element count; validates the shape and dim only.
kf_status softmax_view(int32_t ndim, const int64_t* shape, int64_t dim, SoftmaxArgs* a, int64_t* n) {
    kf_status s = check_shape(ndim, shape, 0, KF_MAX_DIMS, n);
    if (s != KF_OK) return s;
    const int64_t rank = ndim > 0 ? ndim : 1;  // a 0-d tensor accepts dim 0 or -1
    if (dim < -rank || dim >= rank)
        return fail(KF_ERR_BAD_ARG, "dim %lld outside [%lld, %lld)", (long long)dim, (long long)-rank,
                    (long long)rank);
    if (dim < 0) dim += rank;
    *a = SoftmaxArgs{nullptr, nullptr, KF_FLOAT32, KF_FLOAT32, 1, 1, 1};
    if (ndim > 0) {
        a->outer = count((int32_t)dim, shape);
        a->len = shape[dim];
        a->inner = count(ndim - (int32_t)dim - 1, shape + dim + 1);
    }
    return KF_OK;
}

// Every check kf_softmax makes before launching; on KF_OK with *n == 0 the
// call is a no-op.
kf_status check_softmax(const void* x, kf_dtype x_dtype, void* y, kf_dtype y_dtype, int32_t ndim,
                        const int64_t* shape, const int64_t* x_strides, const int64_t* y_strides, int64_t dim,
                        SoftmaxArgs* a, int64_t* n) {
    kf_status s = check_shape(ndim, shape, 0, KF_MAX_DIMS, n);
    if (s != KF_OK) return s;
    if (!dtype_ok(x_dtype) || !dtype_ok(y_dtype))
        return fail(KF_ERR_BAD_DTYPE, "dtype %d -> %d not supported", (int)x_dtype, (int)y_dtype);
    const bool pair_ok = (x_dtype == y_dtype) || (y_dtype == KF_FLOAT32 && x_dtype != KF_FLOAT32);
    if (!pair_ok) return fail(KF_ERR_BAD_DTYPE, "softmax cannot narrow %d to %d", (int)x_dtype, (int)y_dtype);
    s = softmax_view(ndim, shape, dim, a, n);
    if (s != KF_OK) return s;
    a->x = x;
    a->y = y;
    a->xt = x_dtype;
    a->yt = y_dtype;
    if (*n == 0) return KF_OK;
    if (!x || !y) return fail(KF_ERR_NULL_POINTER, "x or y is NULL");
    if ((uintptr_t)x % elem_bytes(x_dtype) || (uintptr_t)y % elem_bytes(y_dtype))
        return fail(KF_ERR_BAD_ARG, "x or y is not aligned to its element size");
    if (!dense(ndim, shape, x_strides) || !dense(ndim, shape, y_strides))
        return fail(KF_ERR_UNSUPPORTED_LAYOUT, "only dense row-major tensors are supported");
    const int64_t xb = *n * elem_bytes(x_dtype), yb = *n * elem_bytes(y_dtype);
    if (x != y && overlaps(x, xb, y, yb)) return fail(KF_ERR_BAD_ARG, "x and y partially overlap");
    if (x == y && x_dtype != y_dtype) return fail(KF_ERR_BAD_ARG, "in-place softmax needs equal dtypes");
    return KF_OK;
}

kf_status begin() {
    g_error[0] = 0;
    return KF_OK;
}

kf_status done(kf_status s, const char* variant) {
    if (s == KF_OK) g_variant = variant ? variant : "";
    return s;
}

// Group-norm shape checks shared by the call and the workspace query.
kf_status check_group_norm_shape(kf_dtype xt, int32_t ndim, const int64_t* shape, int64_t groups, int64_t* n) {
    kf_status s = check_shape(ndim, shape, 2, KF_MAX_DIMS, n);
    if (s != KF_OK) return s;
    if (!dtype_ok(xt)) return fail(KF_ERR_BAD_DTYPE, "x dtype %d not supported", (int)xt);
    if (groups < 1) return fail(KF_ERR_BAD_ARG, "num_groups %lld < 1", (long long)groups);
    if (shape[1] % groups != 0)
        return fail(KF_ERR_BAD_ARG, "C = %lld not divisible by num_groups = %lld", (long long)shape[1],
                    (long long)groups);
    const int64_t spatial = ndim > 2 ? count(ndim - 2, shape + 2) : 1;
    if (shape[1] / groups > INT32_MAX || groups > INT32_MAX || (shape[1] / groups) * spatial > INT32_MAX)
        return fail(KF_ERR_UNSUPPORTED_LAYOUT, "group of %lld elements is too large",
                    (long long)((shape[1] / groups) * spatial));
    return KF_OK;
}

// kf_group_norm and kf_group_norm_static: every check, then the launch.
// With use_static the workspace arguments are ignored and the exchange runs
// in the library's static scratch array.
kf_status group_norm_call(const void* x, kf_dtype x_dtype, void* y, int32_t ndim, const int64_t* shape,
                        const int64_t* x_strides, const int64_t* y_strides, int64_t num_groups, const void* weight,
                        const void* bias, kf_dtype affine_dtype, double eps, void* workspace,
                        size_t workspace_bytes, bool use_static, void* stream) {
    int64_t n = 0;
    kf_status s = check_group_norm_shape(x_dtype, ndim, shape, num_groups, &n);
    if (s != KF_OK) return s;
    if ((weight || bias) && !(affine_dtype == x_dtype || affine_dtype == KF_FLOAT32))
        return fail(KF_ERR_BAD_DTYPE, "affine dtype %d must be x's dtype or FLOAT32", (int)affine_dtype);
    if (!(eps >= 0.0) || !std::isfinite(eps)) return fail(KF_ERR_BAD_ARG, "eps must be finite and >= 0");
    if (n == 0) return done(KF_OK, "noop");
    if (!x || !y) return fail(KF_ERR_NULL_POINTER, "x or y is NULL");
    const int64_t eb = elem_bytes(x_dtype);
    if ((uintptr_t)x % eb || (uintptr_t)y % eb) return fail(KF_ERR_BAD_ARG, "x or y is not element aligned");
    bool nhwc = false;
    if (dense(ndim, shape, x_strides)) {
        if (!dense(ndim, shape, y_strides))
            return fail(KF_ERR_UNSUPPORTED_LAYOUT, "y must be dense in x's layout (NC*)");
    } else if (ndim == 4 && dense_nhwc(shape, x_strides)) {
        if (!dense_nhwc(shape, y_strides))
            return fail(KF_ERR_UNSUPPORTED_LAYOUT, "y must be dense in x's layout (channels last)");
        nhwc = true;
    } else {
        return fail(KF_ERR_UNSUPPORTED_LAYOUT, "x must be dense NC* or dense channels last [N, C, H, W]");
    }
    const int64_t xb = n * eb;
    if (x != y && overlaps(x, xb, y, xb)) return fail(KF_ERR_BAD_ARG, "x and y partially overlap");
    const int64_t ab = shape[1] * ((weight || bias) ? elem_bytes(affine_dtype) : 0);
    if ((weight && overlaps(weight, ab, y, xb)) || (bias && overlaps(bias, ab, y, xb)))
        return fail(KF_ERR_BAD_ARG, "weight or bias overlaps y");
    const int64_t spatial = ndim > 2 ? count(ndim - 2, shape + 2) : 1;
    // What this call's layout needs (the size query, blind to layout, may report more).
    const size_t need = group_norm_workspace_bytes_for(shape[0], shape[1], spatial, num_groups, x_dtype, nhwc);
    if (use_static) {
        // The library's own array: checked against its size, then located.
        if (need > KF_GROUP_NORM_STATIC_SCRATCH_BYTES)
            return fail(KF_ERR_WORKSPACE,
                        "group_norm_static: this shape needs %zu bytes of exchange workspace, the static scratch "
                        "array holds %u; use kf_group_norm with a workspace",
                        need, (unsigned)KF_GROUP_NORM_STATIC_SCRATCH_BYTES);
        s = group_norm_static_scratch(&workspace);
        if (s != KF_OK) return s;
        workspace_bytes = KF_GROUP_NORM_STATIC_SCRATCH_BYTES;
    } else {
        if (!workspace || workspace_bytes < need)
            return fail(KF_ERR_WORKSPACE, "workspace of %zu bytes given, %zu needed",
                        workspace ? workspace_bytes : 0, need);
        if ((uintptr_t)workspace % 256) return fail(KF_ERR_WORKSPACE, "workspace is not 256-byte aligned");
        if (overlaps(workspace, (int64_t)need, x, xb) || overlaps(workspace, (int64_t)need, y, xb))
            return fail(KF_ERR_BAD_ARG, "workspace overlaps x or y");
    }

    GroupNormArgs a{x,     y,    x_dtype,      shape[0],         shape[1], spatial, num_groups, weight, bias,
                    affine_dtype, (float)eps, workspace, workspace_bytes, nhwc};
    const char* variant = nullptr;
    s = group_norm_launch(a, static_cast<hipStream_t>(stream), &variant);
    return done(s, variant);
}

}  // namespace
}  // namespace kf

using namespace kf;

extern "C" {

int kf_abi_version(void) { return KF355_ABI_VERSION; }

const char* kf_status_name(int status) {
    switch (status) {
        case KF_OK: return "KF_OK";
        case KF_ERR_NULL_POINTER: return "KF_ERR_NULL_POINTER";
        case KF_ERR_BAD_SHAPE: return "KF_ERR_BAD_SHAPE";
        case KF_ERR_BAD_DTYPE: return "KF_ERR_BAD_DTYPE";
        case KF_ERR_BAD_ARG: return "KF_ERR_BAD_ARG";
        case KF_ERR_UNSUPPORTED_LAYOUT: return "KF_ERR_UNSUPPORTED_LAYOUT";
        case KF_ERR_WORKSPACE: return "KF_ERR_WORKSPACE";
        case KF_ERR_HIP: return "KF_ERR_HIP";
    }
    return "KF_UNKNOWN";
}

const char* kf_last_error(void) { return g_error; }

const char* kf_last_variant(void) { return g_variant; }

kf_status kf_softmax(const void* x, kf_dtype x_dtype, void* y, kf_dtype y_dtype, int32_t ndim, const int64_t* shape,
                     const int64_t* x_strides, const int64_t* y_strides, int64_t dim, void* stream) {
    begin();
    kf::SoftmaxArgs a;
    int64_t n = 0;
    kf_status s = kf::check_softmax(x, x_dtype, y, y_dtype, ndim, shape, x_strides, y_strides, dim, &a, &n);
    if (s != KF_OK) return s;
    if (n == 0) return done(KF_OK, "noop");
    const char* variant = nullptr;
    s = softmax_launch(a, static_cast<hipStream_t>(stream), &variant);
    return done(s, variant);
}

kf_status kf_softmax_split_workspace_bytes(kf_dtype x_dtype, kf_dtype y_dtype, int32_t ndim, const int64_t* shape,
                                           int64_t dim, size_t* bytes) {
    begin();
    if (!bytes) return fail(KF_ERR_NULL_POINTER, "bytes is NULL");
    if (!dtype_ok(x_dtype) || !dtype_ok(y_dtype))
        return fail(KF_ERR_BAD_DTYPE, "dtype %d -> %d not supported", (int)x_dtype, (int)y_dtype);
    kf::SoftmaxArgs a;
    int64_t n = 0;
    kf_status s = kf::softmax_view(ndim, shape, dim, &a, &n);
    if (s != KF_OK) return s;
    a.xt = x_dtype;
    a.yt = y_dtype;
    *bytes = n == 0 ? 0 : softmax_split_workspace_bytes(a);
    return KF_OK;
}

kf_status kf_softmax_split(const void* x, kf_dtype x_dtype, void* y, kf_dtype y_dtype, int32_t ndim,
                           const int64_t* shape, const int64_t* x_strides, const int64_t* y_strides, int64_t dim,
                           void* workspace, size_t workspace_bytes, void* stream) {
    begin();
    kf::SoftmaxArgs a;
    int64_t n = 0;
    kf_status s = kf::check_softmax(x, x_dtype, y, y_dtype, ndim, shape, x_strides, y_strides, dim, &a, &n);
    if (s != KF_OK) return s;
    if (n == 0) return done(KF_OK, "noop");
    const size_t need = softmax_split_workspace_bytes(a);
    if (need > 0) {
        if (!workspace || workspace_bytes < need)
            return fail(KF_ERR_WORKSPACE, "workspace of %zu bytes given, %zu needed",
                        workspace ? workspace_bytes : 0, need);
        if ((uintptr_t)workspace % 256) return fail(KF_ERR_WORKSPACE, "workspace is not 256-byte aligned");
        if (overlaps(workspace, (int64_t)need, x, n * elem_bytes(x_dtype)) ||
            overlaps(workspace, (int64_t)need, y, n * elem_bytes(y_dtype)))
            return fail(KF_ERR_BAD_ARG, "workspace overlaps x or y");
    }
    const char* variant = nullptr;
    s = softmax_split_launch(a, need > 0 ? workspace : nullptr, static_cast<hipStream_t>(stream), &variant);
    return done(s, variant);
}

kf_status kf_softmax_causal(const void* x, kf_dtype x_dtype, void* y, kf_dtype y_dtype, int32_t ndim,
                            const int64_t* shape, const int64_t* x_strides, const int64_t* y_strides, double scale,
                            void* stream) {
    begin();
    int64_t n = 0;
    kf_status s = check_shape(ndim, shape, 2, KF_MAX_DIMS, &n);
    if (s != KF_OK) return s;
    if (!dtype_ok(x_dtype) || !dtype_ok(y_dtype))
        return fail(KF_ERR_BAD_DTYPE, "dtype %d -> %d not supported", (int)x_dtype, (int)y_dtype);
    const bool pair_ok = (x_dtype == y_dtype) || (y_dtype == KF_FLOAT32 && x_dtype != KF_FLOAT32);
    if (!pair_ok) return fail(KF_ERR_BAD_DTYPE, "softmax cannot narrow %d to %d", (int)x_dtype, (int)y_dtype);
    if (!std::isfinite(scale)) return fail(KF_ERR_BAD_ARG, "scale must be finite");
    if (n == 0) return done(KF_OK, "noop");
    if (!x || !y) return fail(KF_ERR_NULL_POINTER, "x or y is NULL");
    if ((uintptr_t)x % elem_bytes(x_dtype) || (uintptr_t)y % elem_bytes(y_dtype))
        return fail(KF_ERR_BAD_ARG, "x or y is not aligned to its element size");
    if (!dense(ndim, shape, x_strides) || !dense(ndim, shape, y_strides))
        return fail(KF_ERR_UNSUPPORTED_LAYOUT, "only dense row-major tensors are supported");
    const int64_t xb = n * elem_bytes(x_dtype), yb = n * elem_bytes(y_dtype);
    if (x != y && overlaps(x, xb, y, yb)) return fail(KF_ERR_BAD_ARG, "x and y partially overlap");
    if (x == y && x_dtype != y_dtype) return fail(KF_ERR_BAD_ARG, "in-place softmax needs equal dtypes");

    const int64_t q = shape[ndim - 2], k = shape[ndim - 1];
    CausalSoftmaxArgs a{x, y, x_dtype, y_dtype, n / (q * k), q, k, (float)scale};
    const char* variant = nullptr;
    s = softmax_causal_launch(a, static_cast<hipStream_t>(stream), &variant);
    return done(s, variant);
}

kf_status kf_group_norm_workspace_bytes(kf_dtype x_dtype, int32_t ndim, const int64_t* shape, int64_t num_groups,
                                        size_t* bytes) {
    begin();
    if (!bytes) return fail(KF_ERR_NULL_POINTER, "bytes is NULL");
    int64_t n = 0;
    kf_status s = check_group_norm_shape(x_dtype, ndim, shape, num_groups, &n);
    if (s != KF_OK) return s;
    const int64_t spatial = ndim > 2 ? count(ndim - 2, shape + 2) : 1;
    *bytes = n == 0 ? 0 : group_norm_workspace_bytes(shape[0], shape[1], spatial, num_groups, x_dtype);
    return KF_OK;
}

kf_status kf_group_norm(const void* x, kf_dtype x_dtype, void* y, int32_t ndim, const int64_t* shape,
                        const int64_t* x_strides, const int64_t* y_strides, int64_t num_groups, const void* weight,
                        const void* bias, kf_dtype affine_dtype, double eps, void* workspace,
                        size_t workspace_bytes, void* stream) {
    begin();
    return group_norm_call(x, x_dtype, y, ndim, shape, x_strides, y_strides, num_groups, weight, bias, affine_dtype,
                           eps, workspace, workspace_bytes, false, stream);
}

kf_status kf_group_norm_static(const void* x, kf_dtype x_dtype, void* y, int32_t ndim, const int64_t* shape,
                               const int64_t* x_strides, const int64_t* y_strides, int64_t num_groups,
                               const void* weight, const void* bias, kf_dtype affine_dtype, double eps,
                               void* stream) {
    begin();
    return group_norm_call(x, x_dtype, y, ndim, shape, x_strides, y_strides, num_groups, weight, bias, affine_dtype,
                           eps, nullptr, 0, true, stream);
}

kf_status kf_layer_norm(const void* x, kf_dtype x_dtype, void* y, int32_t ndim, const int64_t* shape,
                        const int64_t* x_strides, const int64_t* y_strides, int32_t normalized_ndim,
                        const void* weight, const void* bias, kf_dtype affine_dtype, double eps, void* stream) {
    begin();
    int64_t n = 0;
    kf_status s = check_shape(ndim, shape, 1, KF_MAX_DIMS, &n);
    if (s != KF_OK) return s;
    if (!dtype_ok(x_dtype)) return fail(KF_ERR_BAD_DTYPE, "x dtype %d not supported", (int)x_dtype);
    if (normalized_ndim < 1 || normalized_ndim > ndim)
        return fail(KF_ERR_BAD_ARG, "normalized_ndim %d outside [1, %d]", normalized_ndim, ndim);
    if ((weight || bias) && !(affine_dtype == x_dtype || affine_dtype == KF_FLOAT32))
        return fail(KF_ERR_BAD_DTYPE, "affine dtype %d must be x's dtype or FLOAT32", (int)affine_dtype);
    if (!(eps >= 0.0) || !std::isfinite(eps)) return fail(KF_ERR_BAD_ARG, "eps must be finite and >= 0");
    const int64_t d = count(normalized_ndim, shape + (ndim - normalized_ndim));
    if (n == 0 || d == 0) return done(KF_OK, "noop");
    if (!x || !y) return fail(KF_ERR_NULL_POINTER, "x or y is NULL");
    const int64_t eb = elem_bytes(x_dtype);
    if ((uintptr_t)x % eb || (uintptr_t)y % eb) return fail(KF_ERR_BAD_ARG, "x or y is not element aligned");
    const int64_t ab = (weight || bias) ? elem_bytes(affine_dtype) : 1;
    if ((uintptr_t)weight % ab || (uintptr_t)bias % ab)
        return fail(KF_ERR_BAD_ARG, "weight or bias is not element aligned");
    if (!dense(ndim, shape, x_strides) || !dense(ndim, shape, y_strides))
        return fail(KF_ERR_UNSUPPORTED_LAYOUT, "only dense row-major tensors are supported");
    const int64_t xb = n * eb;
    if (x != y && overlaps(x, xb, y, xb)) return fail(KF_ERR_BAD_ARG, "x and y partially overlap");
    if ((weight && overlaps(weight, d * ab, y, xb)) || (bias && overlaps(bias, d * ab, y, xb)))
        return fail(KF_ERR_BAD_ARG, "weight or bias overlaps y");

    LayerNormArgs a{x, y, x_dtype, n / d, d, weight, bias, affine_dtype, (float)eps};
    const char* variant = nullptr;
    s = layer_norm_launch(a, static_cast<hipStream_t>(stream), &variant);
    return done(s, variant);
}

kf_status kf_adaptive_avgpool2d(const void* x, kf_dtype dtype, void* y, int32_t ndim, const int64_t* shape,
                                const int64_t* x_strides, const int64_t* y_strides, int64_t out_h, int64_t out_w,
                                void* stream) {
    begin();
    int64_t n = 0;
    kf_status s = check_shape(ndim, shape, 3, 4, &n);
    if (s != KF_OK) return s;
    if (!dtype_ok(dtype)) return fail(KF_ERR_BAD_DTYPE, "dtype %d not supported", (int)dtype);
    const int64_t H = shape[ndim - 2], W = shape[ndim - 1];
    if (H < 1 || W < 1) return fail(KF_ERR_BAD_SHAPE, "H and W must be >= 1");
    if (out_h < 1 || out_w < 1) return fail(KF_ERR_BAD_ARG, "output size must be >= 1");
    int64_t yshape[4];
    for (int32_t i = 0; i < ndim - 2; ++i) yshape[i] = shape[i];
    yshape[ndim - 2] = out_h;
    yshape[ndim - 1] = out_w;
    const int64_t ny = count(ndim, yshape);
    if (ny < 0) return fail(KF_ERR_BAD_SHAPE, "output element count overflows int64");
    if (n == 0) return done(KF_OK, "noop");
    if (!x || !y) return fail(KF_ERR_NULL_POINTER, "x or y is NULL");
    const int64_t eb = elem_bytes(dtype);
    if ((uintptr_t)x % eb || (uintptr_t)y % eb) return fail(KF_ERR_BAD_ARG, "x or y is not element aligned");
    bool nhwc = false;
    if (dense(ndim, shape, x_strides)) {
        if (!dense(ndim, yshape, y_strides))
            return fail(KF_ERR_UNSUPPORTED_LAYOUT, "y must be dense in x's layout (NCHW)");
    } else if (ndim == 4 && dense_nhwc(shape, x_strides)) {
        if (!dense_nhwc(yshape, y_strides))
            return fail(KF_ERR_UNSUPPORTED_LAYOUT, "y must be dense in x's layout (channels last)");
        nhwc = true;
    } else {
        return fail(KF_ERR_UNSUPPORTED_LAYOUT, "x must be dense NCHW or dense channels last");
    }
    if (overlaps(x, n * eb, y, ny * eb)) return fail(KF_ERR_BAD_ARG, "x and y overlap");

    AvgPoolArgs a{x, y, dtype, n / (H * W), H, W, out_h, out_w, nhwc, ndim == 4 ? shape[0] : 1, shape[ndim - 3]};
    const char* variant = nullptr;
    s = avgpool_launch(a, static_cast<hipStream_t>(stream), &variant);
    return done(s, variant);
}

kf_status kf_max_pool2d_output_size(int64_t h, int64_t w, const int64_t* window, int32_t ceil_mode,
                                     int64_t* out_hw) {
    begin();
    if (!out_hw) return fail(KF_ERR_NULL_POINTER, "out_hw is NULL");
    kf_status s = check_window(window);
    if (s != KF_OK) return s;
    if (h < 1 || w < 1) return fail(KF_ERR_BAD_SHAPE, "H and W must be >= 1");
    out_hw[0] = pool_out(h, window[0], window[2], window[4], window[6], ceil_mode != 0);
    out_hw[1] = pool_out(w, window[1], window[3], window[5], window[7], ceil_mode != 0);
    if (out_hw[0] < 1 || out_hw[1] < 1) return fail(KF_ERR_BAD_SHAPE, "output would be empty");
    return KF_OK;
}

kf_status kf_stream_copy(const void* src, void* dst, int64_t bytes, void* stream) {
    begin();
    if (bytes < 0 || bytes % 16) return fail(KF_ERR_BAD_SHAPE, "bytes must be a non-negative multiple of 16");
    if (bytes == 0) return done(KF_OK, "noop");
    if (!src || !dst) return fail(KF_ERR_NULL_POINTER, "src or dst is NULL");
    if ((uintptr_t)src % 16 || (uintptr_t)dst % 16) return fail(KF_ERR_BAD_ARG, "src and dst must be 16-byte aligned");
    if (overlaps(src, bytes, dst, bytes)) return fail(KF_ERR_BAD_ARG, "src and dst overlap");
    return done(stream_copy_launch(src, dst, bytes, static_cast<hipStream_t>(stream)), "stream_copy");
}

kf_status kf_stream_read(const void* src, int64_t bytes, void* dst, void* stream) {
    begin();
    if (bytes < 0 || bytes % 16) return fail(KF_ERR_BAD_SHAPE, "bytes must be a non-negative multiple of 16");
    if (bytes == 0) return done(KF_OK, "noop");
    if (!src || !dst) return fail(KF_ERR_NULL_POINTER, "src or dst is NULL");
    if ((uintptr_t)src % 16 || (uintptr_t)dst % 8) return fail(KF_ERR_BAD_ARG, "src must be 16-byte and dst 8-byte aligned");
    const int64_t out_bytes = (bytes + 2047) / 2048 * 8;
    if (overlaps(src, bytes, dst, out_bytes)) return fail(KF_ERR_BAD_ARG, "src and dst overlap");
    return done(stream_read_launch(src, bytes, dst, static_cast<hipStream_t>(stream)), "stream_read");
}

kf_status kf_max_pool2d(const void* x, kf_dtype dtype, void* y, int64_t* indices, int32_t ndim, const int64_t* shape,
                        const int64_t* x_strides, const int64_t* y_strides, const int64_t* window, int32_t ceil_mode,
                        void* stream) {
    begin();
    int64_t n = 0;
    kf_status s = check_shape(ndim, shape, 3, 4, &n);
    if (s != KF_OK) return s;
    if (!dtype_ok(dtype)) return fail(KF_ERR_BAD_DTYPE, "dtype %d not supported", (int)dtype);
    s = check_window(window);
    if (s != KF_OK) return s;
    const int64_t H = shape[ndim - 2], W = shape[ndim - 1];
    if (H < 1 || W < 1) return fail(KF_ERR_BAD_SHAPE, "H and W must be >= 1");
    if (H * W > INT32_MAX) return fail(KF_ERR_BAD_SHAPE, "a plane of %lld elements is too large", (long long)(H * W));
    const int64_t oh = pool_out(H, window[0], window[2], window[4], window[6], ceil_mode != 0);
    const int64_t ow = pool_out(W, window[1], window[3], window[5], window[7], ceil_mode != 0);
    if (oh < 1 || ow < 1) return fail(KF_ERR_BAD_SHAPE, "output would be empty");
    int64_t yshape[4];
    for (int32_t i = 0; i < ndim - 2; ++i) yshape[i] = shape[i];
    yshape[ndim - 2] = oh;
    yshape[ndim - 1] = ow;
    const int64_t ny = count(ndim, yshape);
    const int64_t N = ndim == 4 ? shape[0] : 1, C = shape[ndim - 3];
    if (N > INT32_MAX || C > INT32_MAX) return fail(KF_ERR_BAD_SHAPE, "N or C too large");
    if (n == 0) return done(KF_OK, "noop");
    if (!x || !y) return fail(KF_ERR_NULL_POINTER, "x or y is NULL");
    const int64_t eb = elem_bytes(dtype);
    if ((uintptr_t)x % eb || (uintptr_t)y % eb || (uintptr_t)indices % 8)
        return fail(KF_ERR_BAD_ARG, "x, y or indices is not element aligned");
    bool nhwc = false;
    if (dense(ndim, shape, x_strides)) {
        if (!dense(ndim, yshape, y_strides))
            return fail(KF_ERR_UNSUPPORTED_LAYOUT, "y must be dense in x's layout (NCHW)");
    } else if (ndim == 4 && dense_nhwc(shape, x_strides)) {
        if (!dense_nhwc(yshape, y_strides))
            return fail(KF_ERR_UNSUPPORTED_LAYOUT, "y must be dense in x's layout (channels last)");
        nhwc = true;
    } else {
        return fail(KF_ERR_UNSUPPORTED_LAYOUT, "x must be dense NCHW or dense channels last");
    }
    if (overlaps(x, n * eb, y, ny * eb)) return fail(KF_ERR_BAD_ARG, "x and y overlap");
    if (indices && (overlaps(indices, ny * 8, x, n * eb) || overlaps(indices, ny * 8, y, ny * eb)))
        return fail(KF_ERR_BAD_ARG, "indices overlap x or y");

    MaxPoolArgs a{x, y, indices, dtype, N, C, H, W, oh, ow,
                  (int32_t)window[0], (int32_t)window[1], (int32_t)window[2], (int32_t)window[3],
                  (int32_t)window[4], (int32_t)window[5], (int32_t)window[6], (int32_t)window[7], nhwc};
    const char* variant = nullptr;
    s = max_pool2d_launch(a, static_cast<hipStream_t>(stream), &variant);
    return done(s, variant);
}

}  // extern "C"
