// Host side of the C ABI declared in include/mec.h: argument validation,
// output-size arithmetic (Eq. (1), floor reading), workspace sizes, and the
// choice of kernels. Every check happens before anything is enqueued.
#include "mec.h"

#include <stdint.h>
#include <stdio.h>

#include <initializer_list>

#include "mec_internal.h"

namespace {

// Largest tensor this build accepts, in elements. Far above the 288 GB of one
// MI355X; it keeps every int64 product in this file from overflowing.
constexpr int64_t kMaxElems = int64_t(1) << 40;

bool valid_dtype(int dtype) { return dtype == MEC_F32 || dtype == MEC_BF16; }
int64_t elem_bytes(int dtype) { return dtype == MEC_F32 ? 4 : 2; }

// Product of non-negative factors, or -1 once it exceeds kMaxElems.
int64_t checked_product(std::initializer_list<int64_t> factors) {
    int64_t r = 1;
    for (int64_t f : factors) {
        if (f < 0) return -1;
        if (f != 0 && r > kMaxElems / f) return -1;
        r *= f;
    }
    return r;
}

// Fills s from the arguments; returns MEC_OK or MEC_ERR_INVALID_ARG.
int make_shape(mec::Shape& s, int i_n, int i_h, int i_w, int i_c, int k_h, int k_w, int k_c,
               int s_h, int s_w) {
    if (i_n < 1 || i_h < 1 || i_w < 1 || i_c < 1 || k_h < 1 || k_w < 1 || k_c < 1 || s_h < 1 ||
        s_w < 1)
        return MEC_ERR_INVALID_ARG;
    if (k_h > i_h || k_w > i_w) return MEC_ERR_INVALID_ARG;
    s.i_n = i_n; s.i_h = i_h; s.i_w = i_w; s.i_c = i_c;
    s.k_h = k_h; s.k_w = k_w; s.k_c = k_c; s.s_h = s_h; s.s_w = s_w;
    s.o_h = (s.i_h - s.k_h) / s.s_h + 1;  // Eq. (1), floor
    s.o_w = (s.i_w - s.k_w) / s.s_w + 1;
    s.R = s.k_w * s.i_c;
    s.pairs = s.i_n * s.o_w;
    if (checked_product({s.i_n, s.i_h, s.i_w, s.i_c}) < 0 ||
        checked_product({s.k_h, s.k_w, s.i_c, s.k_c}) < 0 ||
        checked_product({s.i_n, s.o_h, s.o_w, s.k_c}) < 0 ||
        checked_product({s.i_n, s.o_w, s.i_h, s.k_w, s.i_c}) < 0 ||
        checked_product({s.i_n, s.o_h, s.o_w, s.k_h, s.k_w, s.i_c}) < 0)
        return MEC_ERR_INVALID_ARG;
    // the kernels index one L row (R elements) and one block's rows in 32 bits
    if (s.R > (int64_t(1) << 26)) return MEC_ERR_INVALID_ARG;
    return MEC_OK;
}

int64_t lowered_elems(const mec::Shape& s) { return s.i_n * s.o_w * s.i_h * s.k_w * s.i_c; }
int64_t im2col_elems(const mec::Shape& s) { return s.i_n * s.o_h * s.o_w * s.k_h * s.k_w * s.i_c; }

// The product phase of im2col + GEMM as MEC's product phase of a 1x1,
// stride-1 convolution: the image has pixels (n, y, x), each with the
// k_h*k_w*i_c values of its patch as channels; its MEC lowered tensor is the
// (n, x, y)-ordered im2col matrix.
mec::Shape im2col_product_shape(const mec::Shape& s) {
    mec::Shape v = s;
    v.i_h = s.o_h;
    v.i_w = s.o_w;
    v.i_c = s.k_h * s.k_w * s.i_c;
    v.k_h = v.k_w = v.s_h = v.s_w = 1;
    v.o_h = s.o_h;
    v.o_w = s.o_w;
    v.R = v.i_c;
    v.pairs = s.i_n * s.o_w;
    return v;
}

bool aligned(const void* p, int64_t bytes) { return ((uintptr_t)p % (uintptr_t)bytes) == 0; }

thread_local char g_last_error[256];

// Launch status -> MEC status; a failure records which launch and why.
int hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return MEC_OK;
    snprintf(g_last_error, sizeof g_last_error, "%s: %s (%s)", what, hipGetErrorName(e),
             hipGetErrorString(e));
    return MEC_ERR_HIP;
}

// A HIP error left pending by earlier, unrelated work would be reported by the
// hipGetLastError that follows our launch; take it off first.
void clear_stale_error() {
    g_last_error[0] = 0;
    (void)hipGetLastError();
}

}  // namespace

extern "C" {

int mec_output_dims(int i_h, int i_w, int k_h, int k_w, int s_h, int s_w, int* o_h, int* o_w) {
    if (i_h < 1 || i_w < 1 || k_h < 1 || k_w < 1 || s_h < 1 || s_w < 1 || k_h > i_h || k_w > i_w)
        return MEC_ERR_INVALID_ARG;
    if (o_h) *o_h = (i_h - k_h) / s_h + 1;
    if (o_w) *o_w = (i_w - k_w) / s_w + 1;
    return MEC_OK;
}

int64_t mec_workspace_bytes(int i_n, int i_h, int i_w, int i_c, int k_h, int k_w, int k_c,
                            int s_h, int s_w, int dtype, int algo) {
    mec::Shape s;
    int rc = make_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w);
    if (rc != MEC_OK) return rc;
    if (!valid_dtype(dtype)) return MEC_ERR_INVALID_ARG;
    if (algo == MEC_ALGO_FUSED) return 0;
    if (algo == MEC_ALGO_IM2COL) return im2col_elems(s) * elem_bytes(dtype);
    if (algo != MEC_ALGO_LOWERED) return MEC_ERR_INVALID_ARG;
    return lowered_elems(s) * elem_bytes(dtype);
}

int64_t mec_im2col_bytes(int i_n, int i_h, int i_w, int i_c, int k_h, int k_w, int k_c, int s_h,
                         int s_w, int dtype) {
    mec::Shape s;
    int rc = make_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w);
    if (rc != MEC_OK) return rc;
    if (!valid_dtype(dtype)) return MEC_ERR_INVALID_ARG;
    return im2col_elems(s) * elem_bytes(dtype);
}

int mec_lower(const void* I, void* L, int i_n, int i_h, int i_w, int i_c, int k_h, int k_w,
              int k_c, int s_h, int s_w, int dtype, void* stream) {
    mec::Shape s;
    int rc = make_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w);
    if (rc != MEC_OK) return rc;
    if (!valid_dtype(dtype) || !I || !L) return MEC_ERR_INVALID_ARG;
    const int64_t es = elem_bytes(dtype);
    if (!aligned(I, es) || !aligned(L, es)) return MEC_ERR_ALIGNMENT;
    clear_stale_error();
    return hip_status(mec::launch_lower(s, I, L, (int)es, (hipStream_t)stream), "lowering");
}

int mec_im2col(const void* I, void* M, int i_n, int i_h, int i_w, int i_c, int k_h, int k_w,
               int k_c, int s_h, int s_w, int dtype, void* stream) {
    mec::Shape s;
    int rc = make_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w);
    if (rc != MEC_OK) return rc;
    if (!valid_dtype(dtype) || !I || !M) return MEC_ERR_INVALID_ARG;
    const int64_t es = elem_bytes(dtype);
    if (!aligned(I, es) || !aligned(M, es)) return MEC_ERR_ALIGNMENT;
    clear_stale_error();
    return hip_status(mec::launch_im2col(s, I, M, (int)es, (hipStream_t)stream), "im2col");
}

int mec_gemm(const void* L, const void* K, float* O, int i_n, int i_h, int i_w, int i_c, int k_h,
             int k_w, int k_c, int s_h, int s_w, int dtype, void* stream) {
    mec::Shape s;
    int rc = make_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w);
    if (rc != MEC_OK) return rc;
    if (!valid_dtype(dtype) || !L || !K || !O) return MEC_ERR_INVALID_ARG;
    const int64_t es = elem_bytes(dtype);
    if (!aligned(L, es) || !aligned(K, es) || !aligned(O, 4)) return MEC_ERR_ALIGNMENT;
    if (!mec::gemm_supported(s, dtype, false)) return MEC_ERR_UNSUPPORTED;
    clear_stale_error();
    return hip_status(mec::launch_gemm(s, L, K, O, dtype, false, (hipStream_t)stream),
                      "slab products");
}

int mec_conv2d(const void* I, const void* K, float* O, void* workspace, size_t workspace_bytes,
               int i_n, int i_h, int i_w, int i_c, int k_h, int k_w, int k_c, int s_h, int s_w,
               int dtype, int algo, void* stream) {
    mec::Shape s;
    int rc = make_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w);
    if (rc != MEC_OK) return rc;
    if (!valid_dtype(dtype) ||
        (algo != MEC_ALGO_LOWERED && algo != MEC_ALGO_FUSED && algo != MEC_ALGO_IM2COL) || !I ||
        !K || !O)
        return MEC_ERR_INVALID_ARG;
    const int64_t es = elem_bytes(dtype);
    if (!aligned(I, es) || !aligned(K, es) || !aligned(O, 4)) return MEC_ERR_ALIGNMENT;
    if (algo != MEC_ALGO_FUSED) {
        const int64_t need = (algo == MEC_ALGO_IM2COL ? im2col_elems(s) : lowered_elems(s)) * es;
        if (!workspace || (uint64_t)workspace_bytes < (uint64_t)need) return MEC_ERR_WORKSPACE;
        if (!aligned(workspace, es)) return MEC_ERR_ALIGNMENT;
    }
    const mec::Shape g = algo == MEC_ALGO_IM2COL ? im2col_product_shape(s) : s;
    if (g.R > (int64_t(1) << 26) || !mec::gemm_supported(g, dtype, algo == MEC_ALGO_FUSED))
        return MEC_ERR_UNSUPPORTED;
    const hipStream_t st = (hipStream_t)stream;
    clear_stale_error();
    if (algo == MEC_ALGO_FUSED)
        return hip_status(mec::launch_gemm(s, I, K, O, dtype, true, st), "fused slab products");
    if (algo == MEC_ALGO_IM2COL) {
        rc = hip_status(mec::launch_im2col(s, I, workspace, (int)es, st), "im2col");
        if (rc != MEC_OK) return rc;
        return hip_status(mec::launch_gemm(g, workspace, K, O, dtype, false, st), "im2col product");
    }
    rc = hip_status(mec::launch_lower(s, I, workspace, (int)es, st), "lowering");
    if (rc != MEC_OK) return rc;
    return hip_status(mec::launch_gemm(s, workspace, K, O, dtype, false, st), "slab products");
}

// ---------------------------------------------------------------- training passes

namespace {

// Common checks of the training entry points: shape, dtype (fp32 only),
// and the 32-bit index ranges of the kernels.
int grad_shape(mec::Shape& s, int i_n, int i_h, int i_w, int i_c, int k_h, int k_w, int k_c,
               int s_h, int s_w, int dtype) {
    int rc = make_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w);
    if (rc != MEC_OK) return rc;
    if (!valid_dtype(dtype)) return MEC_ERR_INVALID_ARG;
    if (dtype != MEC_F32) return MEC_ERR_UNSUPPORTED;
    if (s.i_n * s.i_h * s.i_w * s.i_c >= (int64_t(1) << 31)) return MEC_ERR_UNSUPPORTED;
    return MEC_OK;
}

}  // namespace

int64_t mec_grad_workspace_bytes(int i_n, int i_h, int i_w, int i_c, int k_h, int k_w, int k_c,
                                 int s_h, int s_w, int dtype, int pass) {
    mec::Shape s;
    int rc = grad_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype);
    if (rc != MEC_OK) return rc;
    switch (pass) {
        case MEC_GRAD_INPUT: return mec::dgrad_workspace_bytes(s);
        case MEC_GRAD_KERNEL:  // the products read L's rows from I: partial sums only
        case MEC_GRAD_KERNEL_FROM_L: return mec::wgrad_partial_bytes(s);
        default: return MEC_ERR_INVALID_ARG;
    }
}

int mec_fold(const float* dL, float* dI, int i_n, int i_h, int i_w, int i_c, int k_h, int k_w,
             int k_c, int s_h, int s_w, void* stream) {
    mec::Shape s;
    int rc = grad_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, MEC_F32);
    if (rc != MEC_OK) return rc;
    if (!dL || !dI) return MEC_ERR_INVALID_ARG;
    if (!aligned(dL, 4) || !aligned(dI, 4)) return MEC_ERR_ALIGNMENT;
    clear_stale_error();
    return hip_status(mec::launch_fold(s, dL, dI, (hipStream_t)stream), "fold");
}

int mec_dgrad_gemm(const float* G, const float* K, float* dL, int i_n, int i_h, int i_w, int i_c,
                   int k_h, int k_w, int k_c, int s_h, int s_w, int dtype, void* stream) {
    mec::Shape s;
    int rc = grad_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype);
    if (rc != MEC_OK) return rc;
    if (!G || !K || !dL) return MEC_ERR_INVALID_ARG;
    if (!aligned(G, 4) || !aligned(K, 4) || !aligned(dL, 4)) return MEC_ERR_ALIGNMENT;
    if (!mec::dgrad_supported(s)) return MEC_ERR_UNSUPPORTED;
    clear_stale_error();
    return hip_status(mec::launch_dgrad_dl(s, G, K, dL, (hipStream_t)stream), "dgrad products");
}

int mec_conv2d_dgrad(const float* G, const void* K, float* dI, void* workspace,
                     size_t workspace_bytes, int i_n, int i_h, int i_w, int i_c, int k_h, int k_w,
                     int k_c, int s_h, int s_w, int dtype, void* stream) {
    mec::Shape s;
    int rc = grad_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype);
    if (rc != MEC_OK) return rc;
    if (!G || !K || !dI) return MEC_ERR_INVALID_ARG;
    if (!aligned(G, 4) || !aligned(K, 4) || !aligned(dI, 4)) return MEC_ERR_ALIGNMENT;
    if (!workspace || (uint64_t)workspace_bytes < (uint64_t)mec::dgrad_workspace_bytes(s))
        return MEC_ERR_WORKSPACE;
    if (!aligned(workspace, 4)) return MEC_ERR_ALIGNMENT;
    const hipStream_t st = (hipStream_t)stream;
    clear_stale_error();
    if (mec::dgrad_phases_ok(s))
        return hip_status(mec::launch_dgrad_phases(s, G, static_cast<const float*>(K), dI,
                                                   workspace, st),
                          "dgrad as sub-pixel phases of the padded gradient");
    if (!mec::dgrad_supported(s)) return MEC_ERR_UNSUPPORTED;
    float* dL = static_cast<float*>(workspace);
    rc = hip_status(mec::launch_dgrad_dl(s, G, static_cast<const float*>(K), dL, st),
                    "dgrad products");
    if (rc != MEC_OK) return rc;
    return hip_status(mec::launch_fold(s, dL, dI, st), "fold");
}

int mec_wgrad_gemm(const void* L, const float* G, float* dK, void* workspace,
                   size_t workspace_bytes, int i_n, int i_h, int i_w, int i_c, int k_h, int k_w,
                   int k_c, int s_h, int s_w, int dtype, void* stream) {
    mec::Shape s;
    int rc = grad_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype);
    if (rc != MEC_OK) return rc;
    if (!L || !G || !dK) return MEC_ERR_INVALID_ARG;
    if (!aligned(L, 4) || !aligned(G, 4) || !aligned(dK, 4)) return MEC_ERR_ALIGNMENT;
    if (!mec::wgrad_supported(s)) return MEC_ERR_UNSUPPORTED;
    if (!workspace || (uint64_t)workspace_bytes < (uint64_t)mec::wgrad_partial_bytes(s))
        return MEC_ERR_WORKSPACE;
    if (!aligned(workspace, 4)) return MEC_ERR_ALIGNMENT;
    clear_stale_error();
    return hip_status(mec::launch_wgrad(s, static_cast<const float*>(L), G,
                                        static_cast<float*>(workspace), dK, (hipStream_t)stream),
                      "wgrad products");
}

int mec_conv2d_wgrad(const void* I, const float* G, float* dK, void* workspace,
                     size_t workspace_bytes, int i_n, int i_h, int i_w, int i_c, int k_h, int k_w,
                     int k_c, int s_h, int s_w, int dtype, void* stream) {
    mec::Shape s;
    int rc = grad_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype);
    if (rc != MEC_OK) return rc;
    if (!I || !G || !dK) return MEC_ERR_INVALID_ARG;
    if (!aligned(I, 4) || !aligned(G, 4) || !aligned(dK, 4)) return MEC_ERR_ALIGNMENT;
    if (!mec::wgrad_supported(s)) return MEC_ERR_UNSUPPORTED;
    if (!workspace || (uint64_t)workspace_bytes < (uint64_t)mec::wgrad_partial_bytes(s))
        return MEC_ERR_WORKSPACE;
    if (!aligned(workspace, 4)) return MEC_ERR_ALIGNMENT;
    const hipStream_t st = (hipStream_t)stream;
    float* part = static_cast<float*>(workspace);
    clear_stale_error();
    // the products read L's rows straight from I: no lowering pass
    return hip_status(mec::launch_wgrad(s, static_cast<const float*>(I), G, part, dK, st, true),
                      "wgrad products from I");
}

int64_t mec_noalloc_scratch_bytes(void) { return mec::kNoAllocScratchBytes; }

int mec_conv2d_wgrad_noalloc(const void* I, const float* G, float* dK, int i_n, int i_h, int i_w,
                             int i_c, int k_h, int k_w, int k_c, int s_h, int s_w, int dtype,
                             void* stream) {
    mec::Shape s;
    int rc = grad_shape(s, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype);
    if (rc != MEC_OK) return rc;
    if (!I || !G || !dK) return MEC_ERR_INVALID_ARG;
    if (!aligned(I, 4) || !aligned(G, 4) || !aligned(dK, 4)) return MEC_ERR_ALIGNMENT;
    if (!mec::wgrad_supported(s)) return MEC_ERR_UNSUPPORTED;
    // the same partial sums as mec_conv2d_wgrad, in the static array
    if (mec::wgrad_partial_bytes(s) > mec::kNoAllocScratchBytes) return MEC_ERR_SCRATCH;
    const hipStream_t st = (hipStream_t)stream;
    clear_stale_error();
    void* part = nullptr;
    rc = hip_status(mec::noalloc_scratch(st, &part), "address of the static scratch");
    if (rc != MEC_OK) return rc;
    return hip_status(mec::launch_wgrad(s, static_cast<const float*>(I), G, static_cast<float*>(part), dK,
                                        st, true),
                      "wgrad products from I, partial sums in the static scratch");
}

const char* mec_strerror(int status) {
    switch (status) {
        case MEC_OK: return "success";
        case MEC_ERR_INVALID_ARG: return "invalid argument (dimension, stride, enum or pointer)";
        case MEC_ERR_WORKSPACE: return "workspace missing or smaller than mec_workspace_bytes";
        case MEC_ERR_ALIGNMENT: return "pointer not aligned to its element size";
        case MEC_ERR_HIP: return "HIP runtime error at kernel launch";
        case MEC_ERR_UNSUPPORTED: return "shape beyond this build's kernel limits";
        case MEC_ERR_SCRATCH: return "the call needs more than the library's static scratch holds";
        default: return "unknown status";
    }
}

const char* mec_last_error(void) { return g_last_error; }

}  // extern "C"
