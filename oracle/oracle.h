/*
 * oracle.h -- plain, slow, double-precision CPU reference for the three
 * memory-bound operators of the hot path (row softmax, GroupNorm,
 * adaptive average pooling).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library includes this
 * header or links this code; only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may call it.  It shares no code, header,
 * table or helper with the HIP kernels.
 *
 * What is computed is the PyTorch operator each kernel replaces: the paper
 * admits a generated kernel only if it reproduces PyTorch eager's output on
 * the captured calls (Section III-C, "Kernel Validator"; Section IV-B,
 * "Baselines, Reporting Policy").  Every function below is therefore the
 * plain mathematical definition of that operator, evaluated in IEEE double
 * in the order the definition states, with no blocking, fusion or
 * reordering.
 *
 * All arrays are dense, row-major, caller-owned host memory.  Sizes are
 * element counts.  No function allocates, and none reports errors: the
 * Python wrapper checks shapes before calling.
 */
#ifndef KF_ORACLE_H
#define KF_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Softmax over the last axis of a [rows, len] array:
 *   m = max_j x_j ; e_j = exp(x_j - m) ; S = sum_j e_j ; y_j = e_j / S.
 * IEEE evaluation of exactly these steps yields PyTorch's special cases:
 * a row of all -inf gives NaN (-inf - -inf), a NaN or +inf entry gives a
 * NaN row. */
void oracle_softmax_rows(const double* x, int64_t rows, int64_t len, double* y);

/* Scaled causal softmax over the last axis of x viewed as [batch, q, k]:
 * query row i sees keys j <= i + (k - q) (the causal mask aligned to the
 * end of the key axis, as with a key/value cache); every other key is
 * masked.  z_j = scale * x_j for visible keys and -inf for masked ones, then
 * the softmax definition above: masked outputs are +0, a row with no visible
 * key is NaN, and masked inputs are never read. */
void oracle_softmax_causal(const double* x, int64_t batch, int64_t q, int64_t k, double scale, double* y);

/* GroupNorm over x viewed as [n, c, s] (s = product of spatial dims),
 * with c divisible by groups.  For every (sample, group) the set holds the
 * (c/groups)*s elements of that group's channels:
 *   mu = sum x / |set| ; var = sum (x - mu)^2 / |set|   (biased, two-pass)
 *   y  = (x - mu) / sqrt(var + eps) * w[ch] + b[ch]
 * w == NULL means w = 1, b == NULL means b = 0. */
void oracle_group_norm(const double* x, int64_t n, int64_t c, int64_t s,
                       int64_t groups, const double* w, const double* b,
                       double eps, double* y);

/* LayerNorm over the last axis of x viewed as [rows, d] (d = product of the
 * normalised trailing dims):
 *   mu = sum x / d ; var = sum (x - mu)^2 / d   (biased, two-pass)
 *   y  = (x - mu) / sqrt(var + eps) * w[j] + b[j]
 * w == NULL means w = 1, b == NULL means b = 0. */
void oracle_layer_norm(const double* x, int64_t rows, int64_t d, const double* w, const double* b, double eps,
                       double* y);

/* adaptive_avg_pool2d over x viewed as [planes, h, w] -> [planes, oh, ow].
 * Output cell (i, j) averages rows [floor(i*h/oh), ceil((i+1)*h/oh)) and
 * columns [floor(j*w/ow), ceil((j+1)*w/ow)). */
void oracle_adaptive_avgpool2d(const double* x, int64_t planes, int64_t h,
                               int64_t w, int64_t oh, int64_t ow, double* y);

/* max_pool2d over x viewed as [planes, h, w] (PyTorch `max_pool2d`):
 * output (i, j) is the maximum of its window -- rows i*sh - ph + a*dh
 * (a < kh), columns j*sw - pw + b*dw (b < kw), positions outside the plane
 * being padding that is never chosen -- with NaN winning over any number.
 * The window is scanned row-major from -inf at its first in-plane position,
 * moving to any greater or NaN element: ties keep the first position, a
 * window holding NaN reports its last NaN.  y is [planes, oh, ow]; idx (may
 * be NULL) receives the chosen position as row * w + col within the plane.
 * Max is exact, so y needs no rounding to the input's format. */
void oracle_max_pool2d(const double* x, int64_t planes, int64_t h, int64_t w, int64_t kh, int64_t kw, int64_t sh,
                       int64_t sw, int64_t ph, int64_t pw, int64_t dh, int64_t dw, int64_t oh, int64_t ow, double* y,
                       int64_t* idx);

/* Round each double to the nearest value of a binary floating-point format
 * with `mant_bits` stored significand bits and `exp_bits` exponent bits,
 * ties to even, directly from double (one rounding).  Returns the format's
 * bit pattern in the low bits of out[i].  bfloat16 is (7, 8), IEEE binary16
 * is (10, 5).  NaN maps to a quiet NaN, overflow to infinity. */
void oracle_round_to_format(const double* v, int64_t n, int mant_bits,
                            int exp_bits, uint32_t* out);

#ifdef __cplusplus
}
#endif

#endif /* KF_ORACLE_H */
