/*
 * Oracle for the convolution backward pass with ReLU-derived sparsity.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the benchmark's CPU
 * baseline leg do.  It shares no code with the HIP library.
 *
 * Plain fp64 direct loops over the definitions, written in the paper's
 * notation (Sec. II-A and Sec. IV-B): a layer maps an input [C,H,W] through
 * filters [M,C,R,S] to an output [M,U,V]; the backward pass is the same
 * operation with M and C interchanged.  Here M is called K and [U,V] is
 * [P,Q].  Every array is in the logical order of that notation:
 *     X, dX   : [N][C][H][W]
 *     W, dW   : [K][C][R][S]
 *     Y, dY   : [N][K][P][Q]
 * with P = (H + 2*pad_h - R)/stride_h + 1 (floor) and likewise Q.
 * Convolution is cross-correlation with zero padding.
 *
 * The only parallelism is OpenMP over independent output elements; every
 * output's sum is accumulated in the order the definition writes it.
 */
#include <stdint.h>
#include <stddef.h>
#include <math.h>
#include <omp.h>

typedef struct {
    int32_t N, C, H, W, K, R, S, P, Q;
    int32_t stride_h, stride_w, pad_h, pad_w;
} oracle_shape;

#define IX4(a, b, c, d, B, C, D) ((((int64_t)(a) * (B) + (b)) * (C) + (c)) * (D) + (d))

/* Forward convolution, Sec. II-A: Y[n,k,p,q] = sum_{c,r,s} X[n,c,h,w] W[k,c,r,s]
 * with h = p*stride_h - pad_h + r, w = q*stride_w - pad_w + s, and X = 0
 * outside [0,H) x [0,W). */
void oracle_conv_fwd(const oracle_shape* sh, const double* X, const double* Wt, double* Y)
{
    const oracle_shape s = *sh;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < s.N; ++n)
        for (int k = 0; k < s.K; ++k)
            for (int p = 0; p < s.P; ++p)
                for (int q = 0; q < s.Q; ++q) {
                    double acc = 0.0;
                    for (int c = 0; c < s.C; ++c)
                        for (int r = 0; r < s.R; ++r)
                            for (int t = 0; t < s.S; ++t) {
                                int h = p * s.stride_h - s.pad_h + r;
                                int w = q * s.stride_w - s.pad_w + t;
                                if (h < 0 || h >= s.H || w < 0 || w >= s.W) continue;
                                acc += X[IX4(n, c, h, w, s.C, s.H, s.W)] *
                                       Wt[IX4(k, c, r, t, s.C, s.R, s.S)];
                            }
                    Y[IX4(n, k, p, q, s.K, s.P, s.Q)] = acc;
                }
}

/* Backward data (Sec. IV-B: the backward pass is the forward operation with
 * M and C interchanged and the filters transposed):
 *     dX[n,c,h,w] = sum_{k,r,s} dY[n,k,p,q] W[k,c,r,s]
 * over the taps where (h + pad_h - r) is a non-negative multiple of stride_h
 * with p = (h + pad_h - r)/stride_h < P, and likewise for w, s, q.
 *
 * Output sparsity (Sec. III-B, boxed ReLU derivative and the Hadamard product
 * that follows it): when mask is given (bytes in [N][C][H][W] order), an
 * output whose mask byte is 0 is never computed and is written as +0.0.
 *
 * abs_out (nullable): sum_{terms} |dY * W| per output, the conditioning of
 * each sum.  nterms (nullable): number of in-range taps per output.
 * Both are 0 at masked outputs. */
void oracle_conv_bwd_data(const oracle_shape* sh, const double* dY, const double* Wt,
                          const uint8_t* mask, double* dX, double* abs_out, int64_t* nterms)
{
    const oracle_shape s = *sh;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < s.N; ++n)
        for (int c = 0; c < s.C; ++c)
            for (int h = 0; h < s.H; ++h)
                for (int w = 0; w < s.W; ++w) {
                    const int64_t o = IX4(n, c, h, w, s.C, s.H, s.W);
                    double acc = 0.0, aacc = 0.0;
                    int64_t cnt = 0;
                    if (mask == NULL || mask[o] != 0) {
                        for (int k = 0; k < s.K; ++k)
                            for (int r = 0; r < s.R; ++r)
                                for (int t = 0; t < s.S; ++t) {
                                    int ph = h + s.pad_h - r, pw = w + s.pad_w - t;
                                    if (ph < 0 || pw < 0) continue;
                                    if (ph % s.stride_h != 0 || pw % s.stride_w != 0) continue;
                                    int p = ph / s.stride_h, q = pw / s.stride_w;
                                    if (p >= s.P || q >= s.Q) continue;
                                    double prod = dY[IX4(n, k, p, q, s.K, s.P, s.Q)] *
                                                  Wt[IX4(k, c, r, t, s.C, s.R, s.S)];
                                    acc += prod;
                                    aacc += fabs(prod);
                                    ++cnt;
                                }
                    }
                    /* a killed output is the +0.0 bit pattern, never -0.0 */
                    dX[o] = (mask != NULL && mask[o] == 0) ? 0.0 : acc;
                    if (abs_out) abs_out[o] = aacc;
                    if (nterms) nterms[o] = cnt;
                }
}

/* Backward weight (weight-gradient phase, Sec. IV-B):
 *     dW[k,c,r,s] = sum_{n,p,q} dY[n,k,p,q] X[n,c,h,w],
 * h = p*stride_h - pad_h + r, w = q*stride_w - pad_w + s, X = 0 outside.
 * abs_out / nterms as for the data gradient. */
void oracle_conv_bwd_weight(const oracle_shape* sh, const double* X, const double* dY,
                            double* dW, double* abs_out, int64_t* nterms)
{
    const oracle_shape s = *sh;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int k = 0; k < s.K; ++k)
        for (int c = 0; c < s.C; ++c)
            for (int r = 0; r < s.R; ++r)
                for (int t = 0; t < s.S; ++t) {
                    double acc = 0.0, aacc = 0.0;
                    int64_t cnt = 0;
                    for (int n = 0; n < s.N; ++n)
                        for (int p = 0; p < s.P; ++p)
                            for (int q = 0; q < s.Q; ++q) {
                                int h = p * s.stride_h - s.pad_h + r;
                                int w = q * s.stride_w - s.pad_w + t;
                                if (h < 0 || h >= s.H || w < 0 || w >= s.W) continue;
                                double prod = dY[IX4(n, k, p, q, s.K, s.P, s.Q)] *
                                              X[IX4(n, c, h, w, s.C, s.H, s.W)];
                                acc += prod;
                                aacc += fabs(prod);
                                ++cnt;
                            }
                    const int64_t o = IX4(k, c, r, t, s.C, s.R, s.S);
                    dW[o] = acc;
                    if (abs_out) abs_out[o] = aacc;
                    if (nterms) nterms[o] = cnt;
                }
}

/* Multiply-accumulate count of the data gradient under the paper's compute
 * model (Sec. II-A; worked example of Fig. "Compaction" in Sec. III-B):
 * an output that the mask kills costs 0 MACs (output sparsity); a live output
 * costs one MAC per in-range tap whose dY operand is non-zero (input
 * sparsity).  per_out (nullable, int64 [N][C][H][W]) receives the per-output
 * count; the return value is the total. */
int64_t oracle_bwd_data_macs(const oracle_shape* sh, const double* dY, const uint8_t* mask,
                             int64_t* per_out)
{
    const oracle_shape s = *sh;
    int64_t total = 0;
    #pragma omp parallel for collapse(2) schedule(static) reduction(+:total)
    for (int n = 0; n < s.N; ++n)
        for (int c = 0; c < s.C; ++c)
            for (int h = 0; h < s.H; ++h)
                for (int w = 0; w < s.W; ++w) {
                    const int64_t o = IX4(n, c, h, w, s.C, s.H, s.W);
                    int64_t cnt = 0;
                    if (mask == NULL || mask[o] != 0) {
                        for (int k = 0; k < s.K; ++k)
                            for (int r = 0; r < s.R; ++r)
                                for (int t = 0; t < s.S; ++t) {
                                    int ph = h + s.pad_h - r, pw = w + s.pad_w - t;
                                    if (ph < 0 || pw < 0) continue;
                                    if (ph % s.stride_h != 0 || pw % s.stride_w != 0) continue;
                                    int p = ph / s.stride_h, q = pw / s.stride_w;
                                    if (p >= s.P || q >= s.Q) continue;
                                    if (dY[IX4(n, k, p, q, s.K, s.P, s.Q)] != 0.0) ++cnt;
                                }
                    }
                    if (per_out) per_out[o] = cnt;
                    total += cnt;
                }
    return total;
}

/* Sampled data gradient: the dense definition evaluated at `count` output
 * coordinates given as (n,c,h,w) quadruples, for checks at sizes where the
 * full tensor is too slow.  out[i], abs_out[i] (nullable), nterms[i]
 * (nullable) as above, without any mask. */
void oracle_conv_bwd_data_at(const oracle_shape* sh, const double* dY, const double* Wt,
                             const int32_t* coords, int64_t count,
                             double* out, double* abs_out, int64_t* nterms)
{
    const oracle_shape s = *sh;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        const int n = coords[4 * i], c = coords[4 * i + 1], h = coords[4 * i + 2], w = coords[4 * i + 3];
        double acc = 0.0, aacc = 0.0;
        int64_t cnt = 0;
        for (int k = 0; k < s.K; ++k)
            for (int r = 0; r < s.R; ++r)
                for (int t = 0; t < s.S; ++t) {
                    int ph = h + s.pad_h - r, pw = w + s.pad_w - t;
                    if (ph < 0 || pw < 0) continue;
                    if (ph % s.stride_h != 0 || pw % s.stride_w != 0) continue;
                    int p = ph / s.stride_h, q = pw / s.stride_w;
                    if (p >= s.P || q >= s.Q) continue;
                    double prod = dY[IX4(n, k, p, q, s.K, s.P, s.Q)] *
                                  Wt[IX4(k, c, r, t, s.C, s.R, s.S)];
                    acc += prod;
                    aacc += fabs(prod);
                    ++cnt;
                }
        out[i] = acc;
        if (abs_out) abs_out[i] = aacc;
        if (nterms) nterms[i] = cnt;
    }
}

/* Sampled weight gradient at `count` (k,c,r,s) coordinates. */
void oracle_conv_bwd_weight_at(const oracle_shape* sh, const double* X, const double* dY,
                               const int32_t* coords, int64_t count,
                               double* out, double* abs_out, int64_t* nterms)
{
    const oracle_shape s = *sh;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        const int k = coords[4 * i], c = coords[4 * i + 1], r = coords[4 * i + 2], t = coords[4 * i + 3];
        double acc = 0.0, aacc = 0.0;
        int64_t cnt = 0;
        for (int n = 0; n < s.N; ++n)
            for (int p = 0; p < s.P; ++p)
                for (int q = 0; q < s.Q; ++q) {
                    int h = p * s.stride_h - s.pad_h + r;
                    int w = q * s.stride_w - s.pad_w + t;
                    if (h < 0 || h >= s.H || w < 0 || w >= s.W) continue;
                    double prod = dY[IX4(n, k, p, q, s.K, s.P, s.Q)] *
                                  X[IX4(n, c, h, w, s.C, s.H, s.W)];
                    acc += prod;
                    aacc += fabs(prod);
                    ++cnt;
                }
        out[i] = acc;
        if (abs_out) abs_out[i] = aacc;
        if (nterms) nterms[i] = cnt;
    }
}

/* Sampled forward convolution at `count` (n,k,p,q) coordinates (Sec. II-A),
 * with sum |X*W| and the number of in-range terms per output. */
void oracle_conv_fwd_at(const oracle_shape* sh, const double* X, const double* Wt,
                        const int32_t* coords, int64_t count,
                        double* out, double* abs_out, int64_t* nterms)
{
    const oracle_shape s = *sh;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        const int n = coords[4 * i], k = coords[4 * i + 1], p = coords[4 * i + 2], q = coords[4 * i + 3];
        double acc = 0.0, aacc = 0.0;
        int64_t cnt = 0;
        for (int c = 0; c < s.C; ++c)
            for (int r = 0; r < s.R; ++r)
                for (int t = 0; t < s.S; ++t) {
                    int h = p * s.stride_h - s.pad_h + r;
                    int w = q * s.stride_w - s.pad_w + t;
                    if (h < 0 || h >= s.H || w < 0 || w >= s.W) continue;
                    double prod = X[IX4(n, c, h, w, s.C, s.H, s.W)] * Wt[IX4(k, c, r, t, s.C, s.R, s.S)];
                    acc += prod;
                    aacc += fabs(prod);
                    ++cnt;
                }
        out[i] = acc;
        if (abs_out) abs_out[i] = aacc;
        if (nterms) nterms[i] = cnt;
    }
}

/* Number of OpenMP threads the oracle's parallel loops use. */
int oracle_num_threads(void)
{
    return omp_get_max_threads();
}
