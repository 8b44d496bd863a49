/*
 * kf355.h -- C ABI of libkf355: MI355X (gfx950) kernels for the three
 * memory-bound segmented reductions that Kernel Forge (arXiv 2607.24762)
 * optimises inside real PyTorch models: row softmax (Gemma 4 E2B and
 * Qwen 3.5 35B-A3B attention / router scores), GroupNorm (Stable Diffusion
 * 3.5 Medium) and adaptive_avgpool2d (ResNet-50 head); Section IV-C reports
 * the per-operator results, Table I the workloads.
 *
 * Semantics.  Every call computes exactly what the PyTorch operator of the
 * same name computes: the paper admits a kernel only when it reproduces
 * PyTorch eager's outputs for the captured call, characterised by shapes,
 * dtypes, strides, layouts and scalar arguments (Section III-A,
 * "Model Ingestion Pipeline"; Section III-C, "Kernel Validator"), and a call
 * the kernel does not cover is left to the original PyTorch path
 * (Section III-E, "Packaging, Guarded Dispatch").  Here an uncovered layout
 * is reported as KF_ERR_UNSUPPORTED_LAYOUT, never computed some other way.
 *
 * Conventions shared by all calls.
 *  - Tensor data pointers are DEVICE pointers on the current HIP device.
 *    `shape` and `*_strides` are HOST arrays of `ndim` int64 values;
 *    strides count elements.  A NULL stride array means dense row-major.
 *    Only dense row-major tensors are supported; other strides return
 *    KF_ERR_UNSUPPORTED_LAYOUT (size-1 dimensions may carry any stride).
 *  - `stream` is a hipStream_t (NULL = the default stream).  Calls only
 *    enqueue work: they never synchronise, and device faults surface at the
 *    caller's next synchronisation, as with PyTorch.
 *  - The caller owns every buffer; the library allocates nothing and keeps
 *    no pointer after returning.
 *  - Every argument is checked on the host before anything is enqueued.  On
 *    any status other than KF_OK nothing was enqueued, except KF_ERR_HIP,
 *    which reports a failed launch.  kf_last_error() then describes it.
 *  - A tensor with zero elements is a no-op returning KF_OK.
 *  - Calls are thread-safe; the only global state is a thread-local error
 *    string / variant name and per-device properties cached on first use.
 */
#ifndef KF355_H
#define KF355_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KF355_ABI_VERSION 1
#define KF_MAX_DIMS 8

typedef enum kf_status {
    KF_OK = 0,
    KF_ERR_NULL_POINTER = 1,      /* a required pointer is NULL */
    KF_ERR_BAD_SHAPE = 2,         /* ndim out of range, negative or mismatched sizes */
    KF_ERR_BAD_DTYPE = 3,         /* dtype or dtype combination not supported */
    KF_ERR_BAD_ARG = 4,           /* dim, num_groups, eps, output size, aliasing */
    KF_ERR_UNSUPPORTED_LAYOUT = 5,/* valid for PyTorch but not covered here */
    KF_ERR_WORKSPACE = 6,         /* workspace missing or too small */
    KF_ERR_HIP = 7                /* the HIP runtime rejected a launch */
} kf_status;

typedef enum kf_dtype {
    KF_FLOAT32 = 0,
    KF_BFLOAT16 = 1,
    KF_FLOAT16 = 2
} kf_dtype;

/* KF355_ABI_VERSION of the loaded library. */
int kf_abi_version(void);

/* Static name of a status code ("KF_OK", ...); "KF_UNKNOWN" otherwise. */
const char* kf_status_name(int status);

/* Thread-local detail text of this thread's last non-OK status ("" if none).
 * Valid until the next kf_* call on the same thread. */
const char* kf_last_error(void);

/* Thread-local name of the kernel variant enqueued by this thread's last
 * successful operator call ("" if none). */
const char* kf_last_variant(void);

/*
 * kf_softmax -- y = softmax(x, dim): along `dim`, y_j = exp(x_j - m) / S with
 * m the maximum and S the sum of exp(x_k - m) (PyTorch `torch.softmax`; the
 * operator of the Gemma 4 E2B and Qwen 3.5 35B-A3B results, Section IV-C).
 *
 *  x, y        device pointers, same shape `shape[ndim]` (0 <= ndim <= 8;
 *              ndim 0 is one element, giving 1).
 *  x_dtype,    (FLOAT32 -> FLOAT32), (BFLOAT16 -> BFLOAT16),
 *  y_dtype     (BFLOAT16 -> FLOAT32), (FLOAT16 -> FLOAT16), (FLOAT16 -> FLOAT32);
 *              accumulation is fp32, results are rounded to nearest-even.
 *  dim         in [-ndim, ndim) (wrapped like PyTorch); any dim is
 *              supported, the last one is the fast path.
 *  Special rows follow IEEE evaluation as PyTorch does: a row of only -inf
 *  gives NaN, a NaN or +inf entry gives a NaN row, -inf entries give +0.
 *  y may equal x (in place); any other overlap is KF_ERR_BAD_ARG.
 */
kf_status kf_softmax(const void* x, kf_dtype x_dtype, void* y, kf_dtype y_dtype, int32_t ndim,
                     const int64_t* shape, const int64_t* x_strides, const int64_t* y_strides, int64_t dim,
                     void* stream);

/*
 * kf_softmax_split -- kf_softmax (same arguments, semantics, dtype pairs and
 * results to within rounding) for inputs of few long rows, such as the
 * attention scores of one decode step [batch, heads, 1, kv] in eager
 * attention (the paper's LLM workloads decode greedily with a KV cache,
 * Section IV-B): when the rows alone would leave most of the GPU idle, each
 * row is split over several workgroups that exchange their partial
 * (max, sum of exponentials) states through `workspace` and merge them in a
 * fixed order, so results are deterministic.  Views it does not split (rows
 * many or short, dim not last, x == y, x or y off a 16-byte boundary) run as
 * kf_softmax does.
 *
 *  workspace, workspace_bytes
 *              device memory of at least kf_softmax_split_workspace_bytes()
 *              bytes, 256-byte aligned, owned by the caller, ZERO-FILLED before
 *              its first use.  Layout as for kf_group_norm: a 256-byte status
 *              block at offset 0 whose first 32-bit word counts workgroups
 *              that gave up waiting for the rest of their row and recomputed
 *              the row's state themselves (results are the same either way;
 *              informational, cumulative, reset only by the caller), then the
 *              exchange, which every completed call returns to zero.  One
 *              workspace may serve kf_softmax_split and kf_group_norm calls of
 *              any shapes in stream order; calls that may run concurrently
 *              need separate workspaces.  May be NULL when the required size is
 *              0.  Too small: KF_ERR_WORKSPACE.
 */
kf_status kf_softmax_split(const void* x, kf_dtype x_dtype, void* y, kf_dtype y_dtype, int32_t ndim,
                           const int64_t* shape, const int64_t* x_strides, const int64_t* y_strides, int64_t dim,
                           void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes kf_softmax_split needs for these dtypes, shape and dim
 * (written to *bytes; 0 when such a view is never split). */
kf_status kf_softmax_split_workspace_bytes(kf_dtype x_dtype, kf_dtype y_dtype, int32_t ndim, const int64_t* shape,
                                           int64_t dim, size_t* bytes);

/*
 * kf_softmax_causal -- the attention-score softmax of eager attention fused
 * into one pass: y = softmax(scale * x + M, -1) over the last axis of x
 * viewed as [..., q, k], where M is the causal mask aligned to the end of
 * the key axis (query i sees keys j <= i + k - q, as with a key/value cache;
 * M is 0 there and -inf elsewhere).  The paper's LLM workloads run eager
 * attention (Table I), whose softmax calls (Section IV-C) follow exactly this
 * scale-mask-softmax sequence.
 *
 *  Masked inputs are never used (their values may be anything, NaN
 *  included) and the masked triangle is not read from memory; masked
 *  outputs are +0.  A row with no visible key (q > k) is NaN, as the masked
 *  softmax gives.  Arguments are as for kf_softmax, with ndim >= 2 and
 *  `scale` any finite value.  Rows of any length up to INT32_MAX keys and
 *  up to INT32_MAX rows: rows beyond the register-resident kernels (65536
 *  16-bit / 32768 fp32 elements; 40960 / 36864 when rows are not whole
 *  16-byte vectors; 8192 on bases that are not 16-byte aligned) are read
 *  twice, once for the statistics and once for the output.  y may equal x
 *  (in place).
 */
kf_status kf_softmax_causal(const void* x, kf_dtype x_dtype, void* y, kf_dtype y_dtype, int32_t ndim,
                            const int64_t* shape, const int64_t* x_strides, const int64_t* y_strides, double scale,
                            void* stream);

/*
 * kf_group_norm -- y = group_norm(x, num_groups, weight, bias, eps)
 * (PyTorch `torch.nn.functional.group_norm`; the SD3.5 Medium result,
 * Section IV-C): for each sample and each of `num_groups` groups of
 * C/num_groups consecutive channels, mu and var are the mean and biased
 * variance over the group's channels and spatial positions, and
 * y = (x - mu) / sqrt(var + eps) * weight[c] + bias[c].
 *
 *  x, y          device pointers, shape [N, C, *] (2 <= ndim <= 8), same dtype
 *                (FLOAT32, BFLOAT16 or FLOAT16); statistics are fp32.  Dense
 *                row-major, or for 4-D [N, C, H, W] dense channels last
 *                (memory order N, H, W, C); y in x's layout.  Other layouts:
 *                KF_ERR_UNSUPPORTED_LAYOUT.
 *  num_groups    >= 1 and divides C, else KF_ERR_BAD_ARG.
 *  weight, bias  device pointers to C elements each, or NULL (weight 1 /
 *                bias 0); both use `affine_dtype`, which is x_dtype or
 *                FLOAT32.
 *  eps           >= 0 (used as fp32).
 *  workspace     device buffer of at least kf_group_norm_workspace_bytes()
 *                bytes, 256-byte aligned, ZERO-FILLED before its first use
 *                and otherwise left alone by the caller between calls.  Bytes
 *                0-255 are a status block: its first 32-bit word counts the
 *                workgroups that stopped waiting for the rest of their group
 *                (e.g. because other kernels held the compute units) and
 *                recomputed the group's statistics themselves; the results
 *                are identical either way, so the count is informational.  It
 *                is cumulative and sits at offset 0 for every shape and path;
 *                the caller may read it or reset it to 0 between calls.  The
 *                bytes after it carry the cross-workgroup exchange, which
 *                every completed call returns to zero, so one workspace serves
 *                later calls of any shape (kf_softmax_split's too) in stream
 *                order.  Calls that may run concurrently must not share a
 *                workspace.
 *  y may equal x (in place); any other overlap is KF_ERR_BAD_ARG.
 */
kf_status kf_group_norm(const void* x, kf_dtype x_dtype, void* y, int32_t ndim, const int64_t* shape,
                        const int64_t* x_strides, const int64_t* y_strides, int64_t num_groups,
                        const void* weight, const void* bias, kf_dtype affine_dtype, double eps,
                        void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes kf_group_norm needs for this shape (written to *bytes);
 * a pure function of its arguments, no device access. */
kf_status kf_group_norm_workspace_bytes(kf_dtype x_dtype, int32_t ndim, const int64_t* shape, int64_t num_groups,
                                        size_t* bytes);

/* Bytes of the scratch array kf_group_norm_static uses on each GPU. */
#define KF_GROUP_NORM_STATIC_SCRATCH_BYTES (1u << 20)

/*
 * kf_group_norm_static -- kf_group_norm without a workspace argument, for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  Same arguments
 * (minus workspace / workspace_bytes), semantics, kernels and results as
 * kf_group_norm; the call itself allocates nothing (no hipMalloc, hipFree or
 * allocating library routine).
 *
 *  The cross-workgroup exchange runs in a scratch array of
 *  KF_GROUP_NORM_STATIC_SCRATCH_BYTES (1 MiB) that the library holds in each
 *  GPU's memory from the moment its code is loaded there until the process
 *  ends; it starts zeroed and every completed call returns its exchange
 *  region to zero (its first 32-bit word accumulates the give-up count
 *  described for kf_group_norm and is never reset by the library).  The
 *  array's device address is looked up on the first call on each device.
 *  Shapes whose exchange workspace for their layout exceeds the array
 *  return KF_ERR_WORKSPACE before anything is enqueued ([1, 512, 128, 128]
 *  with 32 groups needs 12544 bytes in NCHW and 270592 in channels last, as
 *  kf_group_norm_workspace_bytes reports for either layout; about 2700
 *  groups of 16 NCHW chunks fit, about 120 groups of 64 channels-last
 *  parts).
 *  All calls on one GPU share that GPU's array: calls that may overlap in
 *  time on one GPU (streams not ordered by events, or other threads) race
 *  and give wrong results; calls in stream order are safe.  A failed lookup
 *  of the array's address returns KF_ERR_HIP.
 */
kf_status kf_group_norm_static(const void* x, kf_dtype x_dtype, void* y, int32_t ndim, const int64_t* shape,
                               const int64_t* x_strides, const int64_t* y_strides, int64_t num_groups,
                               const void* weight, const void* bias, kf_dtype affine_dtype, double eps,
                               void* stream);

/*
 * kf_layer_norm -- y = layer_norm(x, x.shape[-normalized_ndim:], weight,
 * bias, eps) (PyTorch `torch.nn.functional.layer_norm`; the SD3.5 Medium
 * layer_norm result, Section IV-C): for each row of the d = product of the
 * last `normalized_ndim` sizes, mu and var are the mean and biased variance
 * of the row and y = (x - mu) / sqrt(var + eps) * weight[j] + bias[j].
 *
 *  x, y             device pointers, same shape (1 <= ndim <= 8), same dtype
 *                   (FLOAT32, BFLOAT16 or FLOAT16); statistics are fp32.
 *  normalized_ndim  in [1, ndim].
 *  weight, bias     device pointers to d elements each (the normalised
 *                   shape, dense), or NULL (weight 1 / bias 0); both use
 *                   `affine_dtype`, which is x_dtype or FLOAT32.
 *  eps              >= 0 (used as fp32).
 *  y may equal x (in place); any other overlap is KF_ERR_BAD_ARG.
 */
kf_status kf_layer_norm(const void* x, kf_dtype x_dtype, void* y, int32_t ndim, const int64_t* shape,
                        const int64_t* x_strides, const int64_t* y_strides, int32_t normalized_ndim,
                        const void* weight, const void* bias, kf_dtype affine_dtype, double eps, void* stream);

/*
 * kf_adaptive_avgpool2d -- y = adaptive_avg_pool2d(x, (out_h, out_w))
 * (PyTorch `torch.nn.functional.adaptive_avg_pool2d`; the ResNet-50 result,
 * Section IV-C): output cell (i, j) is the mean of input rows
 * [floor(i*H/out_h), ceil((i+1)*H/out_h)) and columns
 * [floor(j*W/out_w), ceil((j+1)*W/out_w)).
 *
 *  x        device pointer, shape [N, C, H, W] or [C, H, W] with H, W >= 1,
 *           dtype FLOAT32, BFLOAT16 or FLOAT16 (fp32 accumulation); dense
 *           NCHW, or (4-D) dense channels last (memory order N, H, W, C).
 *  out_h,   >= 1 each (may exceed H, W, as in PyTorch).
 *  out_w
 *  y        device pointer, shape [N, C, out_h, out_w] (or [C, out_h,
 *           out_w]), x's dtype, dense in x's layout; y_strides describe
 *           it.  y must not overlap x.  Other layouts:
 *           KF_ERR_UNSUPPORTED_LAYOUT.
 */
kf_status kf_adaptive_avgpool2d(const void* x, kf_dtype dtype, void* y, int32_t ndim, const int64_t* shape,
                                const int64_t* x_strides, const int64_t* y_strides, int64_t out_h,
                                int64_t out_w, void* stream);

/*
 * kf_max_pool2d -- y = max_pool2d(x, kernel, stride, padding, dilation,
 * ceil_mode), optionally with return_indices (PyTorch
 * `torch.nn.functional.max_pool2d`; the paper's ResNet-50 max_pool2d,
 * Section IV-C).  Output (i, j) of a plane is the maximum over rows
 * i*sh - ph + a*dh (a < kh) and columns j*sw - pw + b*dw (b < kw) that lie
 * inside the plane (padding is never chosen); NaN wins over any number.
 * With indices, the result is the selected input element, bit for bit.
 * Without them (indices NULL) a running maximum is kept instead, so two
 * results differ from the selected element's bits: a window whose maximum
 * is a zero may give +0 where the first maximum is -0 (the two compare
 * equal), and a window holding NaN gives a quiet NaN that need not carry
 * the NaN element's bits.
 *
 *  x        device pointer, shape [N, C, H, W] or [C, H, W], H, W >= 1,
 *           H * W < 2^31; dtype FLOAT32, BFLOAT16 or FLOAT16; dense NCHW, or
 *           (4-D) dense channels last (memory order N, H, W, C).
 *  window   host array {kh, kw, sh, sw, ph, pw, dh, dw}: kernel, stride and
 *           dilation >= 1, 0 <= padding <= kernel / 2 (PyTorch's rule).
 *  ceil_mode  non-zero: output sizes rounded up (a last window starting in
 *           the right padding is dropped), as in PyTorch.
 *  y        device pointer, shape [N, C, out_h, out_w] (or [C, out_h, out_w])
 *           from kf_max_pool2d_output_size, x's dtype, dense in x's layout;
 *           y_strides describe it.  No overlap with x.
 *  indices  NULL, or device int64 array shaped and laid out like y: the
 *           selected position as row * W + col within its plane.  In a tie
 *           the first position in row-major window order; a window holding
 *           NaN reports its last NaN; a window of only -inf its first
 *           in-plane position.
 *  KF_ERR_UNSUPPORTED_LAYOUT for other layouts; KF_ERR_BAD_SHAPE when the
 *  output would be empty.
 */
kf_status kf_max_pool2d(const void* x, kf_dtype dtype, void* y, int64_t* indices, int32_t ndim, const int64_t* shape,
                        const int64_t* x_strides, const int64_t* y_strides, const int64_t* window, int32_t ceil_mode,
                        void* stream);

/* Output sizes {out_h, out_w} of kf_max_pool2d for an H x W plane (PyTorch's
 * formula: out = floor((H + 2*ph - dh*(kh-1) - 1) / sh) + 1, with ceil in
 * ceil mode, minus one when ceil mode would start the last window at or past
 * H + ph), written to out_hw[2].  Same checks as kf_max_pool2d. */
kf_status kf_max_pool2d_output_size(int64_t h, int64_t w, const int64_t* window, int32_t ceil_mode,
                                    int64_t* out_hw);

/*
 * kf_stream_copy -- measurement aid, not an operator: copies `bytes` from src
 * to dst with the library's own streaming kernel (each wave moves 1 KiB of
 * consecutive 16-byte vectors for copies of at most 8 MiB, 4 KiB above;
 * non-temporal loads and stores), so a benchmark can state what the HBM of
 * this GPU sustains for a plain copy beside the operators' achieved
 * bandwidth.
 *
 *  src, dst  device pointers, 16-byte aligned, not overlapping; the caller
 *            owns both.
 *  bytes     a multiple of 16 (0 is a no-op), else KF_ERR_BAD_SHAPE.
 *  Misaligned pointers or overlap: KF_ERR_BAD_ARG.  Asynchronous on stream.
 */
kf_status kf_stream_copy(const void* src, void* dst, int64_t bytes, void* stream);

/*
 * kf_stream_read -- measurement aid, not an operator: reads `bytes` from src
 * (each wave 2 KiB of consecutive 16-byte vectors, non-temporal loads) and
 * writes, for every 2 KiB block of src (the last one possibly shorter), one
 * 64-bit word of parities: the HBM read alone, the floor of an operator that
 * reads much and writes little (such as adaptive_avgpool2d to 1x1).
 *
 *  src     device pointer, 16-byte aligned; the caller owns it.
 *  bytes   a multiple of 16 (0 is a no-op), else KF_ERR_BAD_SHAPE.
 *  dst     device pointer, 8-byte aligned, ceil(bytes / 2048) * 8 bytes,
 *          not overlapping src (else KF_ERR_BAD_ARG); bit L (0..63) of
 *          64-bit word b is the parity of the number of set bits in src's
 *          16-byte vectors 128 * b + L and 128 * b + 64 + L (a vector past
 *          the end counts as zero).
 *  Asynchronous on stream.
 */
kf_status kf_stream_read(const void* src, int64_t bytes, void* dst, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KF355_H */
