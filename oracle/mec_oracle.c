/*
 * CPU oracle for MEC, the memory-efficient convolution of Cho & Brand,
 * "MEC: Memory-efficient Convolution for Deep Neural Network" (ICML 2017).
 *
 * TEST INFRASTRUCTURE ONLY. This file is the plain, slow reference against
 * which the GPU library is checked. Only the test suite, the smoke check and
 * the CPU-baseline leg of the benchmark may load it. It shares no code,
 * header, table or helper with the GPU library, and the GPU library must
 * never call it.
 *
 * Notation follows Table 1 of the paper: input I is i_n x i_h x i_w x i_c
 * (n-h-w-c, row-major), kernel K is k_h x k_w x i_c x k_c, output O is
 * i_n x o_h x o_w x k_c, lowered tensor L is i_n x o_w x i_h x k_w x i_c,
 * and s_h, s_w are the kernel strides. Padding is assumed to have been
 * applied to I already (Section 2.1).
 *
 * Element types of I, K and L: dtype 0 is IEEE fp32, dtype 1 is bfloat16
 * stored as its 16-bit pattern, dtype 2 is fp64 (accepted where noted). Every product and sum here is done in fp64;
 * bf16 and fp32 values widen to fp64 exactly, so each output is the exact
 * dot product up to one fp64 rounding per addition.
 *
 * Readings of the paper taken here:
 *  - Eq. (1) gives no rounding rule when s does not divide i - k; the
 *    output size is floor((i - k) / s) + 1.
 *  - Eqs. (2)-(4) write k_c where the lowered row length is i_c; the sizes
 *    use i_c, as Algorithm 2 (its allocation of L) and the shape of K do.
 *  - The operation is cross-correlation: kernel element (a, b) multiplies
 *    input pixel (y*s_h + a, x*s_w + b), with no kernel flip (Section 3.1:
 *    each output is the dot product of K with a sliding sub-matrix of I).
 *  - L spans all i_h input rows (Algorithm 2 allocates and fills
 *    i_n*o_w*i_h*k_w*i_c elements).
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC (see build.py beside this file).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define DT_F32 0
#define DT_BF16 1
#define DT_F64 2

/* Widen one element of a dtype-tagged array to fp64. Both conversions are
 * exact: a bf16 pattern is the top half of an fp32 pattern. */
static double elem(const void* base, int64_t idx, int dtype)
{
    if (dtype == DT_F32) {
        return (double)((const float*)base)[idx];
    } else if (dtype == DT_F64) {
        return ((const double*)base)[idx];
    } else {
        uint32_t bits = (uint32_t)((const uint16_t*)base)[idx] << 16;
        float f;
        memcpy(&f, &bits, sizeof f);
        return (double)f;
    }
}

static int64_t elem_bytes(int dtype) { return dtype == DT_F32 ? 4 : (dtype == DT_F64 ? 8 : 2); }

/* Eq. (1): o = (i - k) / s + 1, read with floor division. Callers keep
 * i >= k >= 1 and s >= 1, so C's truncating division is the floor. */
int64_t oracle_out_dim(int64_t i, int64_t k, int64_t s)
{
    return (i - k) / s + 1;
}

/* Size of MEC's lowered tensor L, in elements: Algorithm 2 allocates
 * i_n*o_w*i_h*k_w*i_c elements (Eq. (3) with the i_c reading). */
int64_t oracle_lowered_elems(int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                             int64_t k_h, int64_t k_w, int64_t k_c,
                             int64_t s_h, int64_t s_w)
{
    (void)k_h; (void)k_c; (void)s_h;
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
    return i_n * o_w * i_h * k_w * i_c;
}

/* Size of the im2col lowered matrix of Section 3.1, in elements:
 * (i_n*o_h*o_w) rows by (k_h*k_w*i_c) columns (Eq. (2), i_c reading). */
int64_t oracle_im2col_elems(int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                            int64_t k_h, int64_t k_w, int64_t k_c,
                            int64_t s_h, int64_t s_w)
{
    (void)k_c;
    int64_t o_h = oracle_out_dim(i_h, k_h, s_h);
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
    return i_n * o_h * o_w * k_h * k_w * i_c;
}

/* Eq. (4), second form: R = i_n*i_c*o_w*k_w*(o_h*k_h - i_h), the number of
 * elements MEC's L saves over im2col. Negative when s_h > k_h. */
int64_t oracle_saving_R(int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                        int64_t k_h, int64_t k_w, int64_t k_c,
                        int64_t s_h, int64_t s_w)
{
    (void)k_c;
    int64_t o_h = oracle_out_dim(i_h, k_h, s_h);
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
    return i_n * i_c * o_w * k_w * (o_h * k_h - i_h);
}

/* Direct convolution, Section 3.1 and Fig. 1(a): each output element is the
 * dot product of K with the sub-matrix of I whose top-left corner is
 * (y*s_h, x*s_w):
 *   O[n,y,x,m] = sum_{a<k_h} sum_{b<k_w} sum_{c<i_c}
 *                I[n, y*s_h + a, x*s_w + b, c] * K[a, b, c, m].
 * O is written in fp64, n-h-w-c. */
void oracle_conv2d_direct(const void* I, const void* K, double* O,
                          int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                          int64_t k_h, int64_t k_w, int64_t k_c,
                          int64_t s_h, int64_t s_w, int dtype)
{
    int64_t o_h = oracle_out_dim(i_h, k_h, s_h);
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t n = 0; n < i_n; ++n)
        for (int64_t y = 0; y < o_h; ++y)
            for (int64_t x = 0; x < o_w; ++x)
                for (int64_t m = 0; m < k_c; ++m) {
                    double acc = 0.0;
                    for (int64_t a = 0; a < k_h; ++a)
                        for (int64_t b = 0; b < k_w; ++b)
                            for (int64_t c = 0; c < i_c; ++c) {
                                int64_t ii = ((n * i_h + (y * s_h + a)) * i_w + (x * s_w + b)) * i_c + c;
                                int64_t kk = ((a * k_w + b) * i_c + c) * k_c + m;
                                acc += elem(I, ii, dtype) * elem(K, kk, dtype);
                            }
                    O[((n * o_h + y) * o_w + x) * k_c + m] = acc;
                }
}

/* The same definition evaluated at chosen output positions only, for
 * sampled checks of outputs too large to compute whole. idx holds npts
 * rows of (n, y, x, m); out[p] receives O[n,y,x,m] in fp64. */
void oracle_conv2d_points(const void* I, const void* K, const int64_t* idx, int64_t npts,
                          double* out,
                          int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                          int64_t k_h, int64_t k_w, int64_t k_c,
                          int64_t s_h, int64_t s_w, int dtype)
{
    (void)i_n;
#pragma omp parallel for schedule(static)
    for (int64_t p = 0; p < npts; ++p) {
        int64_t n = idx[4 * p + 0], y = idx[4 * p + 1], x = idx[4 * p + 2], m = idx[4 * p + 3];
        double acc = 0.0;
        for (int64_t a = 0; a < k_h; ++a)
            for (int64_t b = 0; b < k_w; ++b)
                for (int64_t c = 0; c < i_c; ++c) {
                    int64_t ii = ((n * i_h + (y * s_h + a)) * i_w + (x * s_w + b)) * i_c + c;
                    int64_t kk = ((a * k_w + b) * i_c + c) * k_c + m;
                    acc += elem(I, ii, dtype) * elem(K, kk, dtype);
                }
        out[p] = acc;
    }
}

/* MEC compact lowering, Algorithm 2 (its first parallel loop): for every
 * image n, output column w and input row h, copy the k_w*i_c contiguous
 * elements I[n, h, s_w*w : s_w*w + k_w, 0 : i_c] into L[n, w, h, 0:k_w, 0:i_c].
 * A pure bit copy; works for any element size. */
void oracle_mec_lower(const void* I, void* L,
                      int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                      int64_t k_h, int64_t k_w, int64_t k_c,
                      int64_t s_h, int64_t s_w, int dtype)
{
    (void)k_h; (void)k_c; (void)s_h;
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
    int64_t es = elem_bytes(dtype);
    int64_t run = k_w * i_c; /* elements copied per (n, w, h) */
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t n = 0; n < i_n; ++n)
        for (int64_t w = 0; w < o_w; ++w)
            for (int64_t h = 0; h < i_h; ++h) {
                int64_t dst = (((n * o_w + w) * i_h + h) * k_w) * i_c;  /* L[n, w, h, 0, 0] */
                int64_t src = ((n * i_h + h) * i_w + s_w * w) * i_c;    /* I[n, h, s_w*w, 0] */
                memcpy((char*)L + dst * es, (const char*)I + src * es, (size_t)(run * es));
            }
}

/* MEC for one image and one channel, i_n = i_c = k_c = 1 (Section 3.2,
 * the case Algorithm 1 states): L is o_w x i_h x k_w, and output pixel (h, w)
 * is the dot product of the k_h*k_w-element window of row w of L that starts
 * at s_h*k_w*h with K read row by row.
 * I is i_h x i_w fp32, K is k_h x k_w fp32, O is o_h x o_w fp64;
 * Lout (o_w*i_h*k_w fp32) receives the lowered matrix. */
void oracle_vanilla_mec(const float* I, const float* K, double* O, float* Lout,
                        int64_t i_h, int64_t i_w, int64_t k_h, int64_t k_w,
                        int64_t s_h, int64_t s_w)
{
    int64_t o_h = oracle_out_dim(i_h, k_h, s_h);
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
    /* lowering: L[w, h, 0:k_w] = I[h, s_w*w : s_w*w + k_w] */
    for (int64_t w = 0; w < o_w; ++w)
        for (int64_t h = 0; h < i_h; ++h)
            for (int64_t b = 0; b < k_w; ++b)
                Lout[(w * i_h + h) * k_w + b] = I[h * i_w + s_w * w + b];
    /* o_h small matrix products over shifted column windows of L */
    int64_t ld = i_h * k_w;
    for (int64_t h = 0; h < o_h; ++h)
        for (int64_t w = 0; w < o_w; ++w) {
            double acc = 0.0;
            for (int64_t j = 0; j < k_h * k_w; ++j)
                acc += (double)Lout[w * ld + s_h * k_w * h + j] * (double)K[j];
            O[h * o_w + w] = acc;
        }
}

/* MEC's product phase on an already lowered L, from its definition in
 * Section 3.3 (and Section 3.2 for one channel). With R = k_w*i_c and
 * LD = i_h*R, row (n, w) of L is an LD-element vector; output row h of that
 * pair multiplies the contiguous window of k_h*R elements starting at
 * s_h*R*h (the "slab") by K viewed as a (k_h*k_w*i_c) x k_c matrix:
 *   O[n, h, w, m] = sum_{j < k_h*R} L[n, w][s_h*R*h + j] * K[j, m].
 * The result is written straight in n-h-w-c order. How the products are
 * grouped into matrix calls (Solutions A and B, the threshold T) and the
 * transposition Solution A needs do not change any value, so none of that
 * appears here. O receives fp64. */
void oracle_mec_gemm(const void* L, const void* K, double* O,
                     int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                     int64_t k_h, int64_t k_w, int64_t k_c,
                     int64_t s_h, int64_t s_w, int dtype)
{
    int64_t o_h = oracle_out_dim(i_h, k_h, s_h);
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
    int64_t R = k_w * i_c, LD = i_h * R;
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t n = 0; n < i_n; ++n)
        for (int64_t h = 0; h < o_h; ++h)
            for (int64_t w = 0; w < o_w; ++w) {
                int64_t row = (n * o_w + w) * LD;   /* row (n, w) of L */
                int64_t start = s_h * R * h;        /* first element of output row h's slab */
                for (int64_t m = 0; m < k_c; ++m) {
                    double acc = 0.0;
                    for (int64_t j = 0; j < k_h * R; ++j)
                        acc += elem(L, row + start + j, dtype) * elem(K, j * k_c + m, dtype);
                    O[((n * o_h + h) * o_w + w) * k_c + m] = acc;
                }
            }
}

/* MEC end to end (Section 3.3): the compact lowering of I into L, then the
 * product phase above. O receives fp64 n-h-w-c. Returns 0, or -1 if L cannot
 * be allocated. */
int oracle_mec_conv2d(const void* I, const void* K, double* O,
                      int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                      int64_t k_h, int64_t k_w, int64_t k_c,
                      int64_t s_h, int64_t s_w, int dtype)
{
    int64_t nL = oracle_lowered_elems(i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w);
    void* L = malloc((size_t)(nL * elem_bytes(dtype)));
    if (!L) return -1;
    oracle_mec_lower(I, L, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype);
    oracle_mec_gemm(L, K, O, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype);
    free(L);
    return 0;
}

/* im2col lowering of Section 3.1 / Fig. 1(b), the comparison point for
 * MEC's memory saving: row (n, y, x) of the (i_n*o_h*o_w) x (k_h*k_w*i_c)
 * matrix holds the sub-matrix I[n, y*s_h : y*s_h + k_h, x*s_w : x*s_w + k_w,
 * 0:i_c] linearised in (a, b, c) order. A bit copy. */
void oracle_im2col(const void* I, void* M,
                   int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                   int64_t k_h, int64_t k_w, int64_t k_c,
                   int64_t s_h, int64_t s_w, int dtype)
{
    (void)k_c;
    int64_t o_h = oracle_out_dim(i_h, k_h, s_h);
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
    int64_t es = elem_bytes(dtype);
    int64_t cols = k_h * k_w * i_c;
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t n = 0; n < i_n; ++n)
        for (int64_t y = 0; y < o_h; ++y)
            for (int64_t x = 0; x < o_w; ++x)
                for (int64_t a = 0; a < k_h; ++a)
                    for (int64_t b = 0; b < k_w; ++b)
                        for (int64_t c = 0; c < i_c; ++c) {
                            int64_t dst = ((n * o_h + y) * o_w + x) * cols + (a * k_w + b) * i_c + c;
                            int64_t src = ((n * i_h + (y * s_h + a)) * i_w + (x * s_w + b)) * i_c + c;
                            memcpy((char*)M + dst * es, (const char*)I + src * es, (size_t)es);
                        }
}

/* ------------------------------------------------------------------------
 * Training passes. The paper names training as a use of MEC (Section 1, and
 * the training set-ups of Section 4) but gives no backward algorithm; these
 * are the derivatives of the direct convolution above, written out. For a
 * loss with gradient G = dloss/dO (i_n x o_h x o_w x k_c, n-h-w-c), the
 * definition O[n,y,x,m] = sum_{a,b,c} I[n, y*s_h+a, x*s_w+b, c] K[a,b,c,m]
 * is linear in I and in K, so
 *   dI[n, y*s_h+a, x*s_w+b, c] += G[n,y,x,m] K[a,b,c,m]   over all (n,y,x,m,a,b,c)
 *   dK[a,b,c,m] = sum_{n,y,x} I[n, y*s_h+a, x*s_w+b, c] G[n,y,x,m].
 * Input pixels no window covers receive 0. G, K and I share one dtype tag
 * (0 or 1); results are fp64.
 * ------------------------------------------------------------------------ */

/* dI by the scatter form above. Images are independent, so the loop over n
 * runs in parallel. */
void oracle_conv2d_dgrad(const void* G, const void* K, double* dI,
                         int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                         int64_t k_h, int64_t k_w, int64_t k_c,
                         int64_t s_h, int64_t s_w, int dtype)
{
    int64_t o_h = oracle_out_dim(i_h, k_h, s_h);
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < i_n; ++n) {
        double* d = dI + n * i_h * i_w * i_c;
        for (int64_t e = 0; e < i_h * i_w * i_c; ++e) d[e] = 0.0;
        for (int64_t y = 0; y < o_h; ++y)
            for (int64_t x = 0; x < o_w; ++x)
                for (int64_t m = 0; m < k_c; ++m) {
                    double g = elem(G, ((n * o_h + y) * o_w + x) * k_c + m, dtype);
                    for (int64_t a = 0; a < k_h; ++a)
                        for (int64_t b = 0; b < k_w; ++b)
                            for (int64_t c = 0; c < i_c; ++c)
                                d[((y * s_h + a) * i_w + (x * s_w + b)) * i_c + c] +=
                                    g * elem(K, ((a * k_w + b) * i_c + c) * k_c + m, dtype);
                }
    }
}

/* dK by the sum above; each kernel element is one independent sum. */
void oracle_conv2d_wgrad(const void* I, const void* G, double* dK,
                         int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                         int64_t k_h, int64_t k_w, int64_t k_c,
                         int64_t s_h, int64_t s_w, int dtype)
{
    int64_t o_h = oracle_out_dim(i_h, k_h, s_h);
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t a = 0; a < k_h; ++a)
        for (int64_t b = 0; b < k_w; ++b)
            for (int64_t c = 0; c < i_c; ++c)
                for (int64_t m = 0; m < k_c; ++m) {
                    double acc = 0.0;
                    for (int64_t n = 0; n < i_n; ++n)
                        for (int64_t y = 0; y < o_h; ++y)
                            for (int64_t x = 0; x < o_w; ++x)
                                acc += elem(I, ((n * i_h + (y * s_h + a)) * i_w + (x * s_w + b)) * i_c + c, dtype) *
                                       elem(G, ((n * o_h + y) * o_w + x) * k_c + m, dtype);
                    dK[((a * k_w + b) * i_c + c) * k_c + m] = acc;
                }
}

/* The same two gradients through MEC's lowered tensor. Forward, output row
 * h is the slab A_h = L[:, :][s_h*R*h : s_h*R*h + k_h*R] (one row per pair
 * (n, w), R = k_w*i_c) times K viewed as (k_h*R) x k_c. Differentiating
 * O_h = A_h K gives, with G_h = G[n, h, w, :] as a (i_n*o_w) x k_c matrix:
 *   dL:  every slab receives G_h K^T, added where slabs overlap;
 *   dK:  sum over h of A_h^T G_h.
 * dL has L's shape (i_n x o_w x i_h x k_w x i_c); rows no slab covers are 0. */
void oracle_mec_dgrad_lowered(const void* G, const void* K, double* dL,
                              int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                              int64_t k_h, int64_t k_w, int64_t k_c,
                              int64_t s_h, int64_t s_w, int dtype)
{
    int64_t o_h = oracle_out_dim(i_h, k_h, s_h);
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
    int64_t R = k_w * i_c, KD = k_h * R, LD = i_h * R;
#pragma omp parallel for schedule(static)
    for (int64_t p = 0; p < i_n * o_w; ++p) {
        int64_t n = p / o_w, w = p % o_w;
        double* row = dL + p * LD;
        for (int64_t e = 0; e < LD; ++e) row[e] = 0.0;
        for (int64_t h = 0; h < o_h; ++h)
            for (int64_t j = 0; j < KD; ++j) {
                double acc = 0.0;
                for (int64_t m = 0; m < k_c; ++m)
                    acc += elem(G, ((n * o_h + h) * o_w + w) * k_c + m, dtype) *
                           elem(K, j * k_c + m, dtype);
                row[s_h * R * h + j] += acc;
            }
    }
}

void oracle_mec_wgrad_lowered(const void* L, const void* G, double* dK,
                              int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                              int64_t k_h, int64_t k_w, int64_t k_c,
                              int64_t s_h, int64_t s_w, int dtype)
{
    int64_t o_h = oracle_out_dim(i_h, k_h, s_h);
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
    int64_t R = k_w * i_c, KD = k_h * R, LD = i_h * R;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < KD; ++j)
        for (int64_t m = 0; m < k_c; ++m) {
            double acc = 0.0;
            for (int64_t h = 0; h < o_h; ++h)
                for (int64_t p = 0; p < i_n * o_w; ++p) {
                    int64_t n = p / o_w, w = p % o_w;
                    acc += elem(L, p * LD + s_h * R * h + j, dtype) *
                           elem(G, ((n * o_h + h) * o_w + w) * k_c + m, dtype);
                }
            dK[j * k_c + m] = acc;
        }
}

/* The adjoint of the lowering (the transpose of the copy I -> L): every
 * element of dL is added back to the input pixel it was copied from,
 *   dI[n, h, s_w*w + b, c] += dL[n, w, h, b, c].
 * dL may be fp32, bf16 or fp64 (dtype 0, 1, 2); dI is fp64, 0 where no
 * column strip reaches. */
void oracle_mec_fold(const void* dL, double* dI,
                     int64_t i_n, int64_t i_h, int64_t i_w, int64_t i_c,
                     int64_t k_h, int64_t k_w, int64_t k_c,
                     int64_t s_h, int64_t s_w, int dtype)
{
    (void)k_h; (void)k_c; (void)s_h;
    int64_t o_w = oracle_out_dim(i_w, k_w, s_w);
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < i_n; ++n) {
        double* d = dI + n * i_h * i_w * i_c;
        for (int64_t e = 0; e < i_h * i_w * i_c; ++e) d[e] = 0.0;
        for (int64_t w = 0; w < o_w; ++w)
            for (int64_t h = 0; h < i_h; ++h)
                for (int64_t b = 0; b < k_w; ++b)
                    for (int64_t c = 0; c < i_c; ++c)
                        d[(h * i_w + s_w * w + b) * i_c + c] +=
                            elem(dL, (((n * o_w + w) * i_h + h) * k_w + b) * i_c + c, dtype);
    }
}

/* Number of OpenMP threads a parallel region here would use (0 when built
 * without OpenMP), for reporting the core count of timed runs. */
#ifdef _OPENMP
#include <omp.h>
int oracle_num_threads(void) { return omp_get_max_threads(); }
/* Thread count of later parallel regions (n >= 1), for timing on one core. */
void oracle_set_num_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
#else
int oracle_num_threads(void) { return 0; }
void oracle_set_num_threads(int n) { (void)n; }
#endif
