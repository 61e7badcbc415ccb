// Internal declarations shared by the host API (mec_api.cpp) and the HIP
// kernels (mec_lower.hip, mec_gemm.hip). Not part of the public ABI.
#pragma once

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifndef MEC_HD
#if defined(__HIPCC__)
#define MEC_HD __host__ __device__
#else
#define MEC_HD
#endif
#endif

namespace mec {

// Unsigned division by a runtime constant d >= 1 for dividends below 2^31,
// by one 64-bit multiply and a shift. With l = ceil(log2 d) and
// m = floor(2^(31+l) / d) + 1 (which is below 2^32), floor(x*m / 2^(31+l))
// equals floor(x / d) for every x < 2^31 (Granlund and Montgomery, "Division
// by invariant integers using multiplication", PLDI 1994, round-up method).
struct FastDiv {
    uint32_t d;
    uint32_t shift;  // 31 + l
    uint64_t m;

    FastDiv() = default;
    explicit FastDiv(uint32_t divisor) : d(divisor) {
        uint32_t l = 0;
        while ((uint64_t(1) << l) < divisor) ++l;
        shift = 31 + l;
        m = ((uint64_t(1) << shift) / divisor) + 1;
    }
    MEC_HD inline uint32_t div(uint32_t x) const {
        return (uint32_t)(((uint64_t)x * m) >> shift);
    }
};

// Shape of one convolution in the paper's notation, plus derived sizes.
struct Shape {
    int64_t i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w;
    int64_t o_h, o_w;
    int64_t R;      // k_w * i_c: elements copied per (n, w, h) by the lowering
    int64_t pairs;  // i_n * o_w: rows of L viewed as a matrix
};

// ---------------------------------------------------------------- lowering
struct LowerParams {
    const void* I;
    void* L;
    int64_t rows;          // i_n * o_w * i_h rows of R elements in L
    int64_t R;             // k_w * i_c
    int64_t i_h, o_w, i_w, i_c, s_w;
    int32_t rows_per_block;
    uint32_t nblocks;
    FastDiv divR;          // division by R (elements) or by R / VEC (vectors)
};

// Enqueue the lowering. elem_bytes is 4 (fp32) or 2 (bf16). Returns a
// hipError_t from the launch.
hipError_t launch_lower(const Shape& s, const void* I, void* L, int elem_bytes,
                        hipStream_t stream);

// Enqueue the im2col lowering, rows in (n, x, y) order. Returns the launch
// status.
hipError_t launch_im2col(const Shape& s, const void* I, void* M, int elem_bytes,
                         hipStream_t stream);

// ---------------------------------------------------------------- slab products
struct GemmParams {
    const void* A;     // L (lowered) or I (fused)
    const void* K;     // k_h x k_w x i_c x k_c
    float* O;          // i_n x o_h x o_w x k_c
    int64_t i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, o_h, o_w;
    int64_t R;         // k_w * i_c
    int64_t pairs;     // i_n * o_w
    int64_t a_xstride; // elements between rows x and x+1 of one pair's source
    int32_t hrows;     // input rows staged per tile: (HT - 1) * s_h + k_h
    int32_t nchunks;   // r-chunks of KT covering R
    int32_t pair_tiles, h_tiles, n_tiles;
    uint32_t ntiles;
};

struct OutLayout;

// Enqueue the slab products. fused selects the I-sourced variant.
// Returns hipErrorInvalidValue when the shape exceeds the kernels' on-chip
// limits (see gemm_supported), else the launch status. A strided output
// layout (fp32 only) is taken by the fixed kernels alone: hipErrorNotSupported
// when none of them matches.
hipError_t launch_gemm(const Shape& s, const void* A, const void* K, float* O, int dtype,
                       bool fused, hipStream_t stream, const OutLayout* layout = nullptr);

// Whether the slab-product kernels can run this shape (LDS limits), from L
// (fused = false) or staged from I (fused = true): from L, every kernel height
// runs (the flat windows of L through the one-row tiles); from I, the generic
// kernel's tiles bound k_h.
bool gemm_supported(const Shape& s, int dtype, bool fused);

// Where the fp32 kernels of mec_gemm_fixed.hip write output element
// (n, h, w, c): O + n*img + h*row + w*col + off + c. The default (nullptr)
// is dense n-h-w-c; a strided layout lets one sub-pixel phase of the input
// gradient write straight into its positions of dI.
struct OutLayout {
    int64_t img, row, col, off;
};

// The kernels specialised for a compile-time kernel height and stride.
// Returns hipErrorNotSupported when none matches the shape (or the pointers'
// alignment, or a non-default layout with dtype bf16); with dry_run, only
// reports whether one matches.
hipError_t launch_gemm_fixed(const Shape& s, const void* A, const void* K, float* O, int dtype,
                             bool fused, hipStream_t stream, bool dry_run,
                             const OutLayout* layout = nullptr);

// The flat-window kernel for tall strided fp32 kernels over few channels
// (mec_gemm_ring.hip): whether its ring of LDS holds the shape's windows, and
// the launch (dense n-h-w-c O).
bool gemm_ring_usable(const Shape& s, int dtype);
// the window takes at most two blocks of k-steps: K stays in registers for an
// item and fills run several blocks ahead
bool gemm_ring_short(const Shape& s);
hipError_t launch_gemm_ring(const Shape& s, const void* A, const void* K, float* O, bool fused,
                            hipStream_t stream);

// ---------------------------------------------------------------- training passes
// dL (fp32, L's layout) from G = dloss/dO and K, fp32.
bool dgrad_supported(const Shape& s);
hipError_t launch_dgrad_dl(const Shape& s, const float* G, const float* K, float* dL,
                           hipStream_t stream);
// dI as s_h*s_w sub-pixel phases, each a stride-1 forward convolution of the
// zero-padded G with the taps of K that reach it, turned by 180 degrees and
// transposed (fused slab products, written straight into the phase's pixels
// of dI); the padded G and K' go to the workspace (dgrad_workspace_bytes),
// one phase after the other.
bool dgrad_phases_ok(const Shape& s);
int64_t dgrad_workspace_bytes(const Shape& s);
hipError_t launch_dgrad_phases(const Shape& s, const float* G, const float* K, float* dI,
                               void* workspace, hipStream_t stream);
// dI from dL: the adjoint of the lowering.
hipError_t launch_fold(const Shape& s, const float* dL, float* dI, hipStream_t stream);
// dK from L and G: partial sums over shares of the reduction into `part`
// (wgrad_partial_bytes), then their sum into dK.
bool wgrad_supported(const Shape& s);
int64_t wgrad_splits(const Shape& s);
int64_t wgrad_partial_bytes(const Shape& s);
// fused: the kernels read the rows of L from I (the L argument is I then).
hipError_t launch_wgrad(const Shape& s, const float* L, const float* G, float* part, float* dK,
                        hipStream_t stream, bool fused = false);
// The static device array that mec_conv2d_wgrad_noalloc uses for the partial
// sums: its size, and its address on the stream's device (looked up once per
// device; no allocation).
constexpr int64_t kNoAllocScratchBytes = int64_t(64) << 20;
hipError_t noalloc_scratch(hipStream_t stream, void** ptr);

}  // namespace mec

#if defined(__HIP__)
namespace mec {
// Block index remapped so that each of the 8 XCDs of the MI355X, which
// receive workgroups round-robin (block b runs on XCD b % 8), processes one
// contiguous range of logical blocks. Neighbouring tiles then share an XCD's
// L2 cache. A bijection on [0, G).
__device__ inline uint32_t xcd_remap(uint32_t b, uint32_t G) {
    const uint32_t xcd = b & 7u, slot = b >> 3;
    const uint32_t base = G >> 3, rem = G & 7u;
    return xcd * base + (xcd < rem ? xcd : rem) + slot;
}

// Block index remapped so that the 8 XCDs take turns over runs of g
// consecutive logical blocks: XCD x processes runs x, x + 8, x + 16, ...
// The blocks of one run share an XCD's L2 cache, while the blocks in flight
// across the chip cover one compact range of the work (and of the memory it
// writes) instead of eight ranges far apart. Blocks past the last whole round
// of 8 runs keep their own index. A bijection on [0, G).
__device__ inline uint32_t xcd_interleave(uint32_t b, uint32_t G, uint32_t g) {
    const uint32_t full = G / (8 * g) * (8 * g);
    if (b >= full) return b;
    const uint32_t xcd = b & 7u, slot = b >> 3;
    return (slot / g) * 8 * g + xcd * g + slot % g;
}

// 16-byte store of four output values that bypasses the caches' retention
// policy: O is written once and not read back by the kernel, so streaming it
// out keeps dirty O lines from being evicted later, on the time of whichever
// kernel runs next.
__device__ inline void store_o4_nt(float* dst, const float4& v) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const f32x4 t = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(t, reinterpret_cast<f32x4*>(dst));
}
}  // namespace mec
#endif
