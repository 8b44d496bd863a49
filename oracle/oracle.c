/*
 * oracle.c -- plain double-precision CPU reference (TEST INFRASTRUCTURE ONLY;
 * see oracle.h).  Built with gcc, no HIP, no shared headers with the kernels.
 *
 * Each operator is the PyTorch definition that the paper's validator checks
 * generated kernels against (Section III-C; Section IV-B): evaluated
 * literally, in double, in the order the definition states.
 */
#include "oracle.h"

#include <math.h>
#include <stdint.h>

/* Softmax along the last axis (PyTorch `softmax(x, dim)` definition).
 * Step order: row maximum, shifted exponentials, their sequential sum,
 * division.  The maximum uses `>` so NaN never becomes m; a NaN entry then
 * makes its own exponential NaN, the sum NaN, and the whole row NaN, which
 * is PyTorch's result. */
void oracle_softmax_rows(const double* x, int64_t rows, int64_t len, double* y) {
    for (int64_t r = 0; r < rows; ++r) {
        const double* xr = x + r * len;
        double* yr = y + r * len;
        double m = -INFINITY;
        for (int64_t j = 0; j < len; ++j)
            if (xr[j] > m) m = xr[j];
        double total = 0.0;
        for (int64_t j = 0; j < len; ++j) {
            double e = exp(xr[j] - m);
            yr[j] = e;
            total += e;
        }
        for (int64_t j = 0; j < len; ++j) yr[j] = yr[j] / total;
    }
}

/* Scaled causal softmax: the masked score row z (scale * x where visible,
 * -inf where masked) put through the softmax steps above, in the same
 * order.  Only visible entries of x are read. */
void oracle_softmax_causal(const double* x, int64_t batch, int64_t q, int64_t k, double scale, double* y) {
    for (int64_t b = 0; b < batch; ++b) {
        for (int64_t i = 0; i < q; ++i) {
            const double* xr = x + (b * q + i) * k;
            double* yr = y + (b * q + i) * k;
            const int64_t last = i + (k - q);  /* highest visible key index */
            double m = -INFINITY;
            for (int64_t j = 0; j < k; ++j) {
                const double z = (j <= last) ? scale * xr[j] : -INFINITY;
                if (z > m) m = z;
            }
            double total = 0.0;
            for (int64_t j = 0; j < k; ++j) {
                const double z = (j <= last) ? scale * xr[j] : -INFINITY;
                const double e = exp(z - m);
                yr[j] = e;
                total += e;
            }
            for (int64_t j = 0; j < k; ++j) yr[j] = yr[j] / total;
        }
    }
}

/* GroupNorm (PyTorch `group_norm(x, groups, w, b, eps)` definition): biased
 * variance from a second pass over the group, eps inside the square root,
 * per-channel affine after normalisation. */
void oracle_group_norm(const double* x, int64_t n, int64_t c, int64_t s,
                       int64_t groups, const double* w, const double* b,
                       double eps, double* y) {
    const int64_t ch_per_group = c / groups;
    const int64_t count = ch_per_group * s;
    for (int64_t in = 0; in < n; ++in) {
        for (int64_t g = 0; g < groups; ++g) {
            const int64_t base = (in * c + g * ch_per_group) * s;
            const double* xg = x + base;
            double* yg = y + base;
            if (count == 0) continue;
            double sum = 0.0;
            for (int64_t i = 0; i < count; ++i) sum += xg[i];
            const double mu = sum / (double)count;
            double sq = 0.0;
            for (int64_t i = 0; i < count; ++i) {
                const double d = xg[i] - mu;
                sq += d * d;
            }
            const double var = sq / (double)count;
            const double inv_std = 1.0 / sqrt(var + eps);
            for (int64_t k = 0; k < ch_per_group; ++k) {
                const int64_t ch = g * ch_per_group + k;
                const double wc = w ? w[ch] : 1.0;
                const double bc = b ? b[ch] : 0.0;
                for (int64_t i = 0; i < s; ++i) {
                    const int64_t at = k * s + i;
                    yg[at] = (xg[at] - mu) * inv_std * wc + bc;
                }
            }
        }
    }
}

/* LayerNorm (PyTorch `layer_norm(x, normalized_shape, w, b, eps)`
 * definition): per row, biased variance from a second pass, eps inside the
 * square root, elementwise affine after normalisation. */
void oracle_layer_norm(const double* x, int64_t rows, int64_t d, const double* w, const double* b, double eps,
                       double* y) {
    for (int64_t r = 0; r < rows; ++r) {
        const double* xr = x + r * d;
        double* yr = y + r * d;
        if (d == 0) continue;
        double sum = 0.0;
        for (int64_t j = 0; j < d; ++j) sum += xr[j];
        const double mu = sum / (double)d;
        double sq = 0.0;
        for (int64_t j = 0; j < d; ++j) {
            const double dv = xr[j] - mu;
            sq += dv * dv;
        }
        const double inv_std = 1.0 / sqrt(sq / (double)d + eps);
        for (int64_t j = 0; j < d; ++j)
            yr[j] = (xr[j] - mu) * inv_std * (w ? w[j] : 1.0) + (b ? b[j] : 0.0);
    }
}

/* adaptive_avg_pool2d (PyTorch definition): output cell (i, j) is the mean
 * of the input window [floor(i*h/oh), ceil((i+1)*h/oh)) x
 * [floor(j*w/ow), ceil((j+1)*w/ow)), computed with integer arithmetic. */
void oracle_adaptive_avgpool2d(const double* x, int64_t planes, int64_t h,
                               int64_t w, int64_t oh, int64_t ow, double* y) {
    for (int64_t p = 0; p < planes; ++p) {
        const double* xp = x + p * h * w;
        double* yp = y + p * oh * ow;
        for (int64_t i = 0; i < oh; ++i) {
            const int64_t h0 = (i * h) / oh;
            const int64_t h1 = ((i + 1) * h + oh - 1) / oh;
            for (int64_t j = 0; j < ow; ++j) {
                const int64_t w0 = (j * w) / ow;
                const int64_t w1 = ((j + 1) * w + ow - 1) / ow;
                double sum = 0.0;
                for (int64_t r = h0; r < h1; ++r)
                    for (int64_t q = w0; q < w1; ++q) sum += xp[r * w + q];
                yp[i * ow + j] = sum / (double)((h1 - h0) * (w1 - w0));
            }
        }
    }
}

/* Max pooling over x viewed as [planes, h, w].  Output (i, j) scans its
 * window in row-major order -- rows i*sh - ph + a*dh for a = 0..kh-1,
 * columns j*sw - pw + b*dw for b = 0..kw-1 -- skipping positions outside
 * the plane (padding is never chosen).  The running choice starts at -inf
 * on the first in-plane position and moves to an element that is greater,
 * or that is NaN: so the result is the maximum, the first position wins a
 * tie, and a window holding NaN gives NaN at its last NaN.  idx, if not
 * NULL, receives the chosen position as row * w + col. */
void oracle_max_pool2d(const double* x, int64_t planes, int64_t h, int64_t w, int64_t kh, int64_t kw, int64_t sh,
                       int64_t sw, int64_t ph, int64_t pw, int64_t dh, int64_t dw, int64_t oh, int64_t ow, double* y,
                       int64_t* idx) {
    for (int64_t p = 0; p < planes; ++p) {
        const double* xp = x + p * h * w;
        for (int64_t i = 0; i < oh; ++i) {
            for (int64_t j = 0; j < ow; ++j) {
                double best = -INFINITY;
                int64_t at = -1;
                for (int64_t a = 0; a < kh; ++a) {
                    const int64_t r = i * sh - ph + a * dh;
                    if (r < 0 || r >= h) continue;
                    for (int64_t b = 0; b < kw; ++b) {
                        const int64_t c = j * sw - pw + b * dw;
                        if (c < 0 || c >= w) continue;
                        const double v = xp[r * w + c];
                        if (at < 0) at = r * w + c;
                        if (v > best || isnan(v)) {
                            best = v;
                            at = r * w + c;
                        }
                    }
                }
                y[(p * oh + i) * ow + j] = best;
                if (idx) idx[(p * oh + i) * ow + j] = at;
            }
        }
    }
}

/* Round one double to the format (mant_bits, exp_bits), ties to even.
 *
 * The exact value |v| is divided by the format's quantum at its binade
 * (a power of two, so the division is exact), rounded to an integer with
 * rint() under the default round-to-nearest-even mode, and re-encoded.
 * Below the smallest normal the quantum is fixed (gradual underflow). */
static uint32_t round_one(double v, int mant_bits, int exp_bits) {
    const int bias = (1 << (exp_bits - 1)) - 1;
    const int emin = 1 - bias;                  /* exponent of smallest normal */
    const int emax = bias;                      /* exponent of largest finite */
    const uint32_t sign = signbit(v) ? 1u : 0u;
    const uint32_t sign_bit = sign << (mant_bits + exp_bits);
    const uint32_t exp_all_ones = ((1u << exp_bits) - 1u) << mant_bits;

    if (isnan(v)) return exp_all_ones | (1u << (mant_bits - 1)); /* quiet NaN */
    if (isinf(v)) return sign_bit | exp_all_ones;
    double a = fabs(v);
    if (a == 0.0) return sign_bit;

    int k;
    (void)frexp(a, &k);                          /* a = f * 2^k, f in [0.5, 1) */
    int e = k - 1;                               /* a in [2^e, 2^(e+1)) */
    if (e < emin) e = emin;                      /* subnormal range: fixed quantum */
    const double quantum = ldexp(1.0, e - mant_bits);
    const double units = rint(a / quantum);      /* exact division, RNE */
    const double r = units * quantum;            /* rounded magnitude, exact */

    if (r >= ldexp(1.0, emax + 1)) return sign_bit | exp_all_ones; /* overflow */
    if (r < ldexp(1.0, emin)) {                  /* subnormal (or rounded to 0) */
        const uint32_t mant = (uint32_t)(r / ldexp(1.0, emin - mant_bits));
        return sign_bit | mant;
    }
    int kr;
    (void)frexp(r, &kr);
    const int er = kr - 1;                       /* may exceed e after a carry */
    const uint32_t mant =
        (uint32_t)(r / ldexp(1.0, er - mant_bits)) - (1u << mant_bits);
    const uint32_t biased = (uint32_t)(er + bias);
    return sign_bit | (biased << mant_bits) | mant;
}

void oracle_round_to_format(const double* v, int64_t n, int mant_bits,
                            int exp_bits, uint32_t* out) {
    for (int64_t i = 0; i < n; ++i) out[i] = round_one(v[i], mant_bits, exp_bits);
}
