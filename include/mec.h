/*
 * mec.h -- C ABI of the MI355X (gfx950) library for MEC, the memory-efficient
 * convolution of Cho & Brand, "MEC: Memory-efficient Convolution for Deep
 * Neural Network" (ICML 2017).
 *
 * The operation is the 2-D convolution O = I * K with strides s_h, s_w of
 * Section 2.1, on an input that the caller has already padded:
 *
 *   O[n, y, x, m] = sum_{a < k_h} sum_{b < k_w} sum_{c < i_c}
 *                   I[n, y*s_h + a, x*s_w + b, c] * K[a, b, c, m]
 *
 * (cross-correlation: the kernel is not flipped). MEC computes it in two
 * steps (Section 3.3, Algorithm 2): a compact lowering of I into L, then o_h
 * small matrix products over overlapping column windows ("slabs") of L.
 *
 * Dimensions use the paper's notation (Table 1):
 *   I  input    i_n x i_h x i_w x i_c     (n-h-w-c, row-major)
 *   K  kernel   k_h x k_w x i_c x k_c     (h-w-i-o, row-major)
 *   O  output   i_n x o_h x o_w x k_c     (n-h-w-c, row-major)
 *   L  lowered  i_n x o_w x i_h x k_w x i_c
 * with o_h = floor((i_h - k_h) / s_h) + 1 and o_w likewise (Eq. (1); the
 * floor is this library's reading when s does not divide i - k).
 *
 * Conventions shared by every entry point:
 *  - All tensor pointers are DEVICE pointers to dense row-major memory owned
 *    by the caller. The library never allocates, frees or synchronises.
 *  - Each pointer must be aligned to its element size (4 bytes for fp32,
 *    2 bytes for bf16); otherwise MEC_ERR_ALIGNMENT.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL means
 *    the default stream). Results are visible after the stream is
 *    synchronised.
 *  - Every argument is checked on the host before anything is enqueued; on
 *    any error nothing is launched and no memory is written.
 *  - No global state (except the no-alloc entry point's per-device scratch
 *    address, below): calls are thread-safe. Calls on different streams that
 *    write the same memory race, as with any asynchronous device work.
 *  - Status codes are returned; negative values are errors. No C++ exception
 *    crosses this interface.
 */
#ifndef MEC_H
#define MEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of I, K and L. O is always fp32 (products are accumulated in
 * fp32). MEC_BF16 means bfloat16 bit patterns; it is an extension: the paper
 * works in fp32 only (Section 4). */
enum mec_dtype { MEC_F32 = 0, MEC_BF16 = 1 };

/* MEC_ALGO_LOWERED: Algorithm 2 as two kernels -- the lowering writes L into
 *   the caller's workspace, then the slab products read it.
 * MEC_ALGO_FUSED: one kernel forms each slab of L in on-chip memory straight
 *   from I; L is never written to device memory and no workspace is used.
 * MEC_ALGO_IM2COL: the baseline MEC replaces (Section 3.1): im2col lowering
 *   into the workspace (see mec_im2col), then one matrix product by the same
 *   product kernels with no slab overlap. */
enum mec_algo { MEC_ALGO_LOWERED = 0, MEC_ALGO_FUSED = 1, MEC_ALGO_IM2COL = 2 };

enum mec_status {
    MEC_OK = 0,
    MEC_ERR_INVALID_ARG = -1, /* a dimension or stride < 1, k > i, unknown enum,
                                 NULL tensor pointer, or a size too large    */
    MEC_ERR_WORKSPACE = -2,   /* workspace NULL or smaller than required      */
    MEC_ERR_ALIGNMENT = -3,   /* a pointer not aligned to its element size    */
    MEC_ERR_HIP = -4,         /* the HIP runtime reported a launch error      */
    MEC_ERR_UNSUPPORTED = -5, /* valid but beyond this build's kernel limits
                                 (k_h larger than the on-chip tile allows)    */
    MEC_ERR_SCRATCH = -6      /* a no-alloc call needs more scratch than the
                                 library's static array holds                 */
};

/* Output size, Eq. (1) with the floor reading: o_h = (i_h - k_h) / s_h + 1,
 * o_w = (i_w - k_w) / s_w + 1. Writes *o_h and *o_w (either may be NULL).
 * Returns MEC_OK, or MEC_ERR_INVALID_ARG for a size or stride < 1 or k > i. */
int mec_output_dims(int i_h, int i_w, int k_h, int k_w, int s_h, int s_w,
                    int* o_h, int* o_w);

/* Workspace needed by mec_conv2d, in bytes.
 * MEC_ALGO_LOWERED: exactly |L| * sizeof(element), with
 *   |L| = i_n * o_w * i_h * k_w * i_c -- the size of the lowered tensor that
 *   Algorithm 2 allocates (Section 3.4, Eq. (3), read with i_c where the
 *   printed equation has k_c). No rounding up.
 * MEC_ALGO_FUSED: 0.
 * MEC_ALGO_IM2COL: exactly mec_im2col_bytes.
 * Returns the byte count (>= 0) or a negative status. */
int64_t mec_workspace_bytes(int i_n, int i_h, int i_w, int i_c,
                            int k_h, int k_w, int k_c, int s_h, int s_w,
                            int dtype, int algo);

/* Size of the im2col lowered matrix that MEC's L replaces, in bytes:
 * (i_n*o_h*o_w) x (k_h*k_w*i_c) elements (Section 3.1, Eq. (2), i_c reading).
 * Returns the byte count (>= 0) or a negative status. */
int64_t mec_im2col_bytes(int i_n, int i_h, int i_w, int i_c,
                         int k_h, int k_w, int k_c, int s_h, int s_w, int dtype);

/* MEC compact lowering (Section 3.3, Algorithm 2, first loop):
 *   L[n, w, h, 0:k_w, 0:i_c] = I[n, h, s_w*w : s_w*w + k_w, 0:i_c]
 * for all n < i_n, w < o_w, h < i_h. A bit copy in the element type `dtype`;
 * L must hold |L| = i_n*o_w*i_h*k_w*i_c elements and must not overlap I.
 * k_h, k_c and s_h do not change L but are validated (o_h >= 1) so every
 * entry point takes the same shape contract.
 * Returns MEC_OK or a negative status. */
int mec_lower(const void* I, void* L,
              int i_n, int i_h, int i_w, int i_c,
              int k_h, int k_w, int k_c, int s_h, int s_w,
              int dtype, void* stream);

/* MEC's product phase on an already lowered L (Section 3.3, Algorithm 2,
 * from viewing K as a (k_h*k_w*i_c) x k_c matrix on). For every output row
 * h < o_h, with R = k_w*i_c:
 *   O[n, h, w, 0:k_c] = L[n, w][s_h*R*h : s_h*R*h + k_h*R] x K
 * where L[n, w] is row (n, w) of L viewed as an (i_n*o_w) x (i_h*R) matrix.
 * The result is written straight in n-h-w-c order, so neither Solution A's
 * final transposition nor the |O| <= |L| condition applies. L must hold the
 * output of mec_lower for the same arguments. O must not overlap L or K.
 * Results are reproducible run to run: each output's summation order is fixed
 * by the shape and by whether L, K and O are 16-byte aligned (alignment selects
 * the staging path, and fp32 tiles staged straight into LDS sum their products
 * in another order, within rounding of the others). (For 3x3 layers whose
 * tiles leave compute units idle, each tile's reduction is split in two halves
 * that are added into O after O is zeroed; two partial sums added to zero
 * commute exactly.) Every kernel height runs: where no tile of its own fits,
 * the windows L[n, w][s_h*R*h : s_h*R*h + k_h*R] are read as the rows of one
 * plain product (Section 3.2's flat view).
 * Returns MEC_OK or a negative status. */
int mec_gemm(const void* L, const void* K, float* O,
             int i_n, int i_h, int i_w, int i_c,
             int k_h, int k_w, int k_c, int s_h, int s_w,
             int dtype, void* stream);

/* im2col lowering (Section 3.1, Fig. 1(b)), the method MEC is compared with:
 * every output pixel's k_h x k_w x i_c input patch becomes one row of M. Rows
 * are stored column-major over the output image, (n, x, y):
 *   M[n, x, y, a, b, c] = I[n, y*s_h + a, x*s_w + b, c]
 * for n < i_n, x < o_w, y < o_h, a < k_h, b < k_w, c < i_c. In this order M is
 * the MEC lowered tensor of a 1x1, stride-1 convolution whose input pixel
 * (n, y, x) holds that patch as its k_h*k_w*i_c channels, so
 *   mec_gemm(M, K, O, i_n, o_h, o_w, k_h*k_w*i_c, 1, 1, k_c, 1, 1, dtype, stream)
 * computes O = M x K, the convolution, with the same product kernels.
 * M must hold mec_im2col_bytes and must not overlap I. A bit copy in `dtype`.
 * Returns MEC_OK or a negative status. */
int mec_im2col(const void* I, void* M,
               int i_n, int i_h, int i_w, int i_c,
               int k_h, int k_w, int k_c, int s_h, int s_w,
               int dtype, void* stream);

/* The convolution O = I * K by MEC (Algorithm 2), or by the im2col baseline.
 * MEC_ALGO_LOWERED: mec_lower into `workspace`, then mec_gemm from it;
 *   workspace_bytes must be >= mec_workspace_bytes(..., MEC_ALGO_LOWERED) and
 *   the workspace must be aligned to the element size. On return (after the
 *   stream completes) the workspace holds L exactly as mec_lower writes it.
 * MEC_ALGO_FUSED: one kernel; workspace may be NULL and is not touched. Its
 *   tiles stage the slab rows from I on chip, so kernels taller than they hold
 *   are refused with MEC_ERR_UNSUPPORTED (MEC_ALGO_LOWERED takes them).
 * MEC_ALGO_IM2COL: mec_im2col into `workspace` (at least mec_im2col_bytes),
 *   then the product of M and K; the workspace then holds M.
 * O must not overlap I, K or the workspace.
 * Returns MEC_OK or a negative status. */
int mec_conv2d(const void* I, const void* K, float* O,
               void* workspace, size_t workspace_bytes,
               int i_n, int i_h, int i_w, int i_c,
               int k_h, int k_w, int k_c, int s_h, int s_w,
               int dtype, int algo, void* stream);

/* ------------------------------------------------------------------------
 * Training passes (fp32). The paper names training as a use of MEC (Section
 * 1; Section 4 measures training set-ups) but gives no backward algorithm.
 * These are the derivatives of the convolution above. For a loss whose
 * gradient with respect to O is G (fp32, O's shape i_n x o_h x o_w x k_c):
 *   dI[n, y*s_h + a, x*s_w + b, c] = sum of G[n, y, x, m] * K[a, b, c, m]
 *                                    over all (y, x, m, a, b) that reach it
 *   dK[a, b, c, m] = sum over n, y, x of I[n, y*s_h + a, x*s_w + b, c] * G[n, y, x, m]
 * (input pixels no window covers get dI = 0). Both go through MEC's lowered
 * layout: output row h is O_h = A_h K with A_h the slab of L for row h, so
 *   dL = each slab receives G_h K^T (summed where slabs overlap),  dI = fold(dL),
 *   dK = sum over h of A_h^T G_h,
 * where G_h = G[:, h, :, :] as an (i_n*o_w) x k_c matrix and fold is the
 * adjoint of the lowering (mec_fold). dtype must be MEC_F32 (MEC_BF16 gives
 * MEC_ERR_UNSUPPORTED); all tensors are fp32, 4-byte aligned.
 * ------------------------------------------------------------------------ */

/* MEC_GRAD_INPUT: mec_conv2d_dgrad -- on the sub-pixel phase path (see
 *   mec_conv2d_dgrad): 12 bytes of alignment slack, the largest phase's
 *   zero-padded G' (i_n x (Ny + J - 1) x (Nx + I - 1) x k_c floats, rounded
 *   up to 256 bytes) and the largest phase kernel K' (J*I*k_c*i_c floats),
 *   where phase (py, px) has J = ceil((k_h - py)/s_h), I = ceil((k_w - px)/s_w),
 *   Ny = ceil((i_h - py)/s_h), Nx = ceil((i_w - px)/s_w) (stride 1: one phase,
 *   G' of (o_h + 2(k_h-1)) x (o_w + 2(k_w-1)) pixels); otherwise dL in fp32,
 *   |L| * 4 bytes exactly.
 * MEC_GRAD_KERNEL: mec_conv2d_wgrad -- the partial sums of dK only (its
 *   products read the rows of L straight from I): as MEC_GRAD_KERNEL_FROM_L.
 * MEC_GRAD_KERNEL_FROM_L: mec_wgrad_gemm -- the partial sums of dK only:
 *   s * k_h*k_w*i_c*k_c * 4 bytes, s (1 <= s <= 1024) fixed by the shape. */
enum mec_grad_pass { MEC_GRAD_INPUT = 0, MEC_GRAD_KERNEL = 1, MEC_GRAD_KERNEL_FROM_L = 2 };

/* Workspace of a training pass, in bytes (>= 0), or a negative status. */
int64_t mec_grad_workspace_bytes(int i_n, int i_h, int i_w, int i_c,
                                 int k_h, int k_w, int k_c, int s_h, int s_w,
                                 int dtype, int pass);

/* The adjoint of mec_lower: every element of dL (fp32, L's layout
 * i_n x o_w x i_h x k_w x i_c) is added to the input pixel it was copied from,
 *   dI[n, h, s_w*w + b, c] += dL[n, w, h, b, c],
 * summed in increasing w; dI (fp32, I's shape) is overwritten, 0 where no
 * column strip reaches. dL and dI must not overlap.
 * Returns MEC_OK or a negative status. */
int mec_fold(const float* dL, float* dI,
             int i_n, int i_h, int i_w, int i_c,
             int k_h, int k_w, int k_c, int s_h, int s_w, void* stream);

/* dL = dloss/dL (fp32, L's layout): for every output row h, G_h K^T added
 * into the slab L[n, w][s_h*R*h : s_h*R*h + k_h*R] of every pair (n, w), with
 * R = k_w*i_c; rows of L that no slab covers get 0. dL is overwritten and
 * must not overlap G or K. Returns MEC_OK or a negative status. */
int mec_dgrad_gemm(const float* G, const float* K, float* dL,
                   int i_n, int i_h, int i_w, int i_c,
                   int k_h, int k_w, int k_c, int s_h, int s_w,
                   int dtype, void* stream);

/* dI = dloss/dI. The pixels of one sub-pixel phase (py, px),
 * dI[n, s_h*Y + py, s_w*X + px, :], receive G only through the kernel taps
 * a = py + s_h*j, b = px + s_w*i, so each phase is itself a stride-1
 * convolution: G zero-padded by J - 1 rows above and I - 1 columns to the left
 * (G'), correlated with K'[j, i, m, c] = K[py + s_h(J-1-j), px + s_w(I-1-i), c, m]
 * (the taps turned by 180 degrees, input and output channels swapped); at
 * stride 1 there is one phase, G padded by k - 1 on every side. The library
 * forms G' and K' in the workspace, one phase after another, and runs MEC's
 * fused slab products on them, writing straight into the phase's pixels. This
 * path is taken for i_c >= 32 and, at stride 1, kernels up to 3x3 (where it is
 * the faster one); at larger strides for s_h <= k_h, s_w <= k_w, k_c and i_c
 * multiples of 4, phase kernel heights up to 5, at most 4 phases and
 * k_h*k_w >= 10*s_h*s_w (the phases run one after another; smaller ones lose
 * to the dL path). Otherwise: mec_dgrad_gemm
 * into `workspace` (which then holds dL), then mec_fold into dI.
 * workspace_bytes must be at least mec_grad_workspace_bytes(...,
 * MEC_GRAD_INPUT). dI must not overlap G, K or the workspace.
 * Returns MEC_OK or a negative status. */
int mec_conv2d_dgrad(const float* G, const void* K, float* dI,
                     void* workspace, size_t workspace_bytes,
                     int i_n, int i_h, int i_w, int i_c,
                     int k_h, int k_w, int k_c, int s_h, int s_w,
                     int dtype, void* stream);

/* dK = dloss/dK from an already lowered L (mec_lower's output for the same
 * shape, e.g. the workspace of a MEC_ALGO_LOWERED mec_conv2d, reused):
 * partial sums of A_h^T G_h over shares of the (pair, h) reduction go to
 * `workspace` (mec_grad_workspace_bytes(..., MEC_GRAD_KERNEL_FROM_L)), then
 * dK (k_h x k_w x i_c x k_c, fp32) is their sum, taken in a fixed order.
 * dK must not overlap L, G or the workspace. Returns MEC_OK or a negative
 * status. */
int mec_wgrad_gemm(const void* L, const float* G, float* dK,
                   void* workspace, size_t workspace_bytes,
                   int i_n, int i_h, int i_w, int i_c,
                   int k_h, int k_w, int k_c, int s_h, int s_w,
                   int dtype, void* stream);

/* dK = dloss/dK from I: the products of mec_wgrad_gemm with the rows of L
 * read straight from I, L[n*o_w + w, x, r] = I[n, x, s_w*w*i_c + r], so no
 * lowered copy is made; `workspace` holds the partial sums
 * (mec_grad_workspace_bytes(..., MEC_GRAD_KERNEL)). dK is bit-identical to
 * mec_wgrad_gemm on mec_lower's L. Returns MEC_OK or a negative status. */
int mec_conv2d_wgrad(const void* I, const float* G, float* dK,
                     void* workspace, size_t workspace_bytes,
                     int i_n, int i_h, int i_w, int i_c,
                     int k_h, int k_w, int k_c, int s_h, int s_w,
                     int dtype, void* stream);

/* ------------------------------------------------------------------------
 * No-alloc entry point, for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving or training loops, harnesses
 * that forbid hipMalloc. It computes what mec_conv2d_wgrad computes, with the
 * same kernels, but keeps the partial sums in a static device array of the
 * library (mec_noalloc_scratch_bytes() bytes, 64 MiB) instead of a caller's
 * workspace. It calls no hipMalloc, hipFree or other allocating routine.
 *  - Each GPU the library runs on holds its own copy of the array from the
 *    library's first use on it until the process ends. Its address on a
 *    device is looked up once, at the first call on that device (the only
 *    global state of the library: a per-device pointer set under a lock).
 *  - Every call on one GPU shares that GPU's array and leaves the last
 *    call's partial sums in it. Nothing in it must start at zero: every share
 *    writes its partial sums whole before they are summed. Calls that overlap
 *    on one GPU (other streams or threads) race on the array: serialise them.
 *  - Shapes whose partial sums (mec_grad_workspace_bytes(..., MEC_GRAD_KERNEL))
 *    exceed the array return MEC_ERR_SCRATCH before anything is enqueued.
 *  - dK (fp32) is bit-identical to mec_conv2d_wgrad's for the same arguments.
 * The caller passes I, G and dK as for mec_conv2d_wgrad. Returns MEC_OK or a
 * negative status.
 * ------------------------------------------------------------------------ */
int64_t mec_noalloc_scratch_bytes(void);
int mec_conv2d_wgrad_noalloc(const void* I, const float* G, float* dK,
                             int i_n, int i_h, int i_w, int i_c,
                             int k_h, int k_w, int k_c, int s_h, int s_w,
                             int dtype, void* stream);

/* Static, NUL-terminated description of a status code (never NULL). */
const char* mec_strerror(int status);

/* Detail of the most recent MEC_ERR_HIP returned on the calling thread: the
 * kernel that failed to launch and the HIP error name and text. Empty string
 * when none. The pointer is valid until the next call on the same thread. */
const char* mec_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MEC_H */
