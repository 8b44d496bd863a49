// kf_internal.h -- interfaces between the C-ABI layer (kf355_api.cpp) and
// the per-operator launch code (*.hip).  Arguments arrive here already
// validated: shapes non-empty, dtypes legal, layouts dense.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>

#include "kf355.h"

namespace kf {

// Softmax over the middle axis of a dense [outer, len, inner] view.
struct SoftmaxArgs {
    const void* x;
    void* y;
    kf_dtype xt, yt;
    int64_t outer, len, inner;
};
kf_status softmax_launch(const SoftmaxArgs& a, hipStream_t s, const char** variant);
// Rows split over several workgroups when few long rows would leave most of
// the chip idle: workspace bytes the split needs (0 when this view is not
// split, whatever the pointers), and the launch, which falls back to
// softmax_launch when it does not split (workspace may then be NULL).
size_t softmax_split_workspace_bytes(const SoftmaxArgs& a);
kf_status softmax_split_launch(const SoftmaxArgs& a, void* workspace, hipStream_t s, const char** variant);

// Scaled causal softmax over the last axis of a dense [batch, q, k] view.
struct CausalSoftmaxArgs {
    const void* x;
    void* y;
    kf_dtype xt, yt;
    int64_t batch, q, k;
    float scale;
};
kf_status softmax_causal_launch(const CausalSoftmaxArgs& a, hipStream_t s, const char** variant);

// GroupNorm over a dense [n, c, spatial] view.
struct GroupNormArgs {
    const void* x;
    void* y;
    kf_dtype xt;
    int64_t n, c, spatial, groups;
    const void* weight;
    const void* bias;
    kf_dtype at;
    float eps;
    void* workspace;
    size_t workspace_bytes;
    bool nhwc;  // x, y dense [n, spatial, c] (channels last) instead of [n, c, spatial]
};
size_t group_norm_workspace_bytes(int64_t n, int64_t c, int64_t spatial, int64_t groups, kf_dtype xt);
// The exchange workspace the paths of one layout need (nhwc: channels last),
// never more than group_norm_workspace_bytes, which covers both layouts.
size_t group_norm_workspace_bytes_for(int64_t n, int64_t c, int64_t spatial, int64_t groups, kf_dtype xt,
                                      bool nhwc);
kf_status group_norm_launch(const GroupNormArgs& a, hipStream_t s, const char** variant);
// Device address, on the current device, of the library's static GroupNorm
// scratch array (KF_GROUP_NORM_STATIC_SCRATCH_BYTES); looked up once per
// device.  KF_ERR_HIP when the lookup fails.
kf_status group_norm_static_scratch(void** ptr);

// LayerNorm over the last d elements of a dense [rows, d] view.
struct LayerNormArgs {
    const void* x;
    void* y;
    kf_dtype xt;
    int64_t rows, d;
    const void* weight;
    const void* bias;
    kf_dtype at;
    float eps;
};
kf_status layer_norm_launch(const LayerNormArgs& a, hipStream_t s, const char** variant);

// adaptive_avg_pool2d over a dense [planes, h, w] view -> [planes, oh, ow]
// (NCHW), or with nhwc over x [n, h, w, c] -> y [n, oh, ow, c] (channels
// last; planes = n * c).
struct AvgPoolArgs {
    const void* x;
    void* y;
    kf_dtype t;
    int64_t planes, h, w, oh, ow;
    bool nhwc;
    int64_t n, c;
};
kf_status avgpool_launch(const AvgPoolArgs& a, hipStream_t s, const char** variant);

// max_pool2d over x [n, c, h, w] (NCHW) or [n, h, w, c] (NHWC, channels
// last); y and idx (optional) are [n, c, oh, ow] in the same layout.
struct MaxPoolArgs {
    const void* x;
    void* y;
    int64_t* idx;
    kf_dtype t;
    int64_t n, c, h, w, oh, ow;
    int32_t kh, kw, sh, sw, ph, pw, dh, dw;
    bool nhwc;
};
kf_status max_pool2d_launch(const MaxPoolArgs& a, hipStream_t s, const char** variant);

// Calibration copy of `bytes` (a multiple of 16) between 16-byte aligned,
// non-overlapping device buffers.
kf_status stream_copy_launch(const void* src, void* dst, int64_t bytes, hipStream_t s);
kf_status stream_read_launch(const void* src, int64_t bytes, void* dst, hipStream_t s);

// Records the detail text of the current failure (thread-local).
void set_error(const char* fmt, ...);

// Device properties, cached per device (runtime.cpp).
int device_multiprocessors(int dev);
bool device_cooperative(int dev);
// How many workgroups of `threads` threads of `kernel` can be resident on
// device `dev` at once (0 if unknown); one cache object per kernel.
struct ResidencyCache {
    static constexpr int kDevices = 64;
    std::atomic<int> v[kDevices];
};
int resident_capacity(ResidencyCache& cache, int dev, const void* kernel, int threads);
// Unsigned value of environment variable `name`, or `dflt` when unset.
uint32_t env_u32(const char* name, uint32_t dflt);

}  // namespace kf
