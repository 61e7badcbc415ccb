// im2col lowering (Section 3.1, Fig. 1(b)), the method MEC is measured
// against, stored in (n, x)-major order:
//   M[n, x, y, a, b, c] = I[n, y*s_h + a, x*s_w + b, c]
// i.e. the k_h*k_w*i_c patch of every output pixel (n, y, x), with the o_h
// pixels of one output column (n, x) stored together. In this order M is
// exactly MEC's lowered tensor L for a 1x1, stride-1 convolution of the image
// whose pixel (n, y, x) has the patch as its channels, so the slab-product
// kernels with k_h = k_w = 1 multiply it by K: im2col + GEMM on the same
// engine, with no slab overlap to exploit.
//
// band   One workgroup per column (n, x) and block of Y output rows
//        y0 <= y < y0 + Y: it reads the band I[n, y0*s_h : (y0+Y-1)*s_h + k_h,
//        x*s_w : x*s_w + k_w, :] -- runs of R = k_w*i_c elements, the runs MEC
//        copies into L[n, x] -- into LDS once, then writes the Y*k_h*R
//        contiguous elements of M[n, x, y0:y0+Y] (run y*s_h + a for a < k_h)
//        with 16-byte non-temporal stores. Y is the largest block whose band
//        fits the LDS budget (all o_h rows when possible). Runs that are not
//        multiples of 16 bytes are packed element by element into aligned
//        16-byte stores, with element stores at the block's unaligned head and
//        tail.
// gather Fallback when not even one output row's k_h runs fit in LDS: each
//        thread gathers one element of M straight from I.
#include <hip/hip_runtime.h>

#include "mec_internal.h"

namespace mec {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBandThreads = 256;
constexpr int kGatherThreads = 256;
constexpr int64_t kBandLdsLimit = 64 * 1024;

inline bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }

struct BandParams {
    const void* I;
    void* M;
    uint32_t blocks;     // i_n * o_w * nyb
    uint32_t i_h, o_w, o_h, k_h, s_h;
    uint32_t R;          // k_w * i_c
    uint32_t in_row;     // elements between consecutive rows of I: i_w * i_c
    uint32_t in_col;     // elements between consecutive columns x: s_w * i_c
    uint32_t yblk;       // output rows per workgroup (Y)
    uint32_t nyb;        // row blocks per column: ceil(o_h / Y)
    FastDiv div_nyb;
    FastDiv div_ow, div_R, div_kh;
    FastDiv div_RV;      // by R / (16-byte vector), vector path only
};

// E: fp32 or bf16 payload. VEC: every run and every column of I and M starts
// on a 16-byte boundary, so both phases move 16-byte vectors.
template <typename E, bool VEC>
__global__ __launch_bounds__(kBandThreads) void im2col_band_kernel(BandParams p) {
    constexpr uint32_t N = 16 / sizeof(E);
    extern __shared__ u32x4 band_v[];
    E* band = reinterpret_cast<E*>(band_v);
    const uint32_t blk = xcd_remap(blockIdx.x, p.blocks);
    const uint32_t pair = p.div_nyb.div(blk);
    const uint32_t y0 = (blk - pair * p.nyb) * p.yblk;
    const uint32_t ny = p.o_h - y0 < p.yblk ? p.o_h - y0 : p.yblk;  // output rows here
    const uint32_t nrows = (ny - 1) * p.s_h + p.k_h;                  // staged input rows
    const uint32_t len = ny * p.k_h * p.R;                            // elements written
    const uint32_t n = p.div_ow.div(pair), x = pair - n * p.o_w;
    const E* __restrict__ src = reinterpret_cast<const E*>(p.I) +
                                ((size_t)n * p.i_h * p.in_row + (size_t)y0 * p.s_h * p.in_row +
                                 (size_t)x * p.in_col);
    E* __restrict__ dst =
        reinterpret_cast<E*>(p.M) + ((size_t)pair * p.o_h + y0) * p.k_h * p.R;

    if constexpr (VEC) {
        const uint32_t RV = p.R / N, nv = nrows * RV;
        const FastDiv& div_RV = p.div_RV;
        for (uint32_t v = threadIdx.x; v < nv; v += kBandThreads) {
            const uint32_t row = div_RV.div(v), c = v - row * RV;
            band_v[v] = *reinterpret_cast<const u32x4*>(src + (size_t)row * p.in_row + c * N);
        }
        __syncthreads();
        const uint32_t lenv = len / N;
        u32x4* out = reinterpret_cast<u32x4*>(dst);
        for (uint32_t v = threadIdx.x; v < lenv; v += kBandThreads) {
            const uint32_t seg = div_RV.div(v), c = v - seg * RV;  // seg = y*k_h + a
            const uint32_t y = p.div_kh.div(seg), a = seg - y * p.k_h;
            __builtin_nontemporal_store(band_v[(y * p.s_h + a) * RV + c], out + v);
        }
    } else {
        const uint32_t nb = nrows * p.R;
        for (uint32_t e = threadIdx.x; e < nb; e += kBandThreads) {
            const uint32_t row = p.div_R.div(e), r = e - row * p.R;
            band[e] = src[(size_t)row * p.in_row + r];
        }
        __syncthreads();
        auto value = [&](uint32_t e) {
            const uint32_t seg = p.div_R.div(e), r = e - seg * p.R;
            const uint32_t y = p.div_kh.div(seg), a = seg - y * p.k_h;
            return band[(y * p.s_h + a) * p.R + r];
        };
        // elements before the first 16-byte boundary of this column, and after the last
        const uint32_t mis = (uint32_t)(((uintptr_t)dst / sizeof(E)) % N);
        const uint32_t head = mis ? (N - mis < len ? N - mis : len) : 0;
        const uint32_t nvec = (len - head) / N;
        const uint32_t tail0 = head + nvec * N;
        if (threadIdx.x < head) dst[threadIdx.x] = value(threadIdx.x);
        if (threadIdx.x < len - tail0) dst[tail0 + threadIdx.x] = value(tail0 + threadIdx.x);
        u32x4* out = reinterpret_cast<u32x4*>(dst + head);
        for (uint32_t v = threadIdx.x; v < nvec; v += kBandThreads) {
            union {
                u32x4 q;
                E e[N];
            } u;
#pragma unroll
            for (uint32_t k = 0; k < N; ++k) u.e[k] = value(head + v * N + k);
            __builtin_nontemporal_store(u.q, out + v);
        }
    }
}

struct GatherParams {
    const void* I;
    void* M;
    int64_t total;  // |M|
    int64_t i_h, i_w, i_c, k_h, k_w, s_h, s_w, o_h, o_w;
};

template <typename E>
__global__ __launch_bounds__(kGatherThreads) void im2col_gather_kernel(GatherParams p) {
    const E* __restrict__ I = reinterpret_cast<const E*>(p.I);
    E* __restrict__ M = reinterpret_cast<E*>(p.M);
    const int64_t stride = (int64_t)gridDim.x * kGatherThreads;
    for (int64_t e = (int64_t)blockIdx.x * kGatherThreads + threadIdx.x; e < p.total; e += stride) {
        int64_t t = e;
        const int64_t c = t % p.i_c; t /= p.i_c;
        const int64_t b = t % p.k_w; t /= p.k_w;
        const int64_t a = t % p.k_h; t /= p.k_h;
        const int64_t y = t % p.o_h; t /= p.o_h;
        const int64_t x = t % p.o_w;
        const int64_t n = t / p.o_w;
        M[e] = I[((n * p.i_h + y * p.s_h + a) * p.i_w + x * p.s_w + b) * p.i_c + c];
    }
}

template <typename E>
hipError_t launch_typed(const Shape& s, const void* I, void* M, hipStream_t stream) {
    constexpr int64_t N = 16 / sizeof(E);
    const int64_t row_bytes = s.R * (int64_t)sizeof(E);
    // output rows per workgroup: the most whose staged input rows fit in LDS
    int64_t yblk = s.o_h;
    const int64_t fit_rows = kBandLdsLimit / row_bytes;
    if ((yblk - 1) * s.s_h + s.k_h > fit_rows)
        yblk = fit_rows >= s.k_h ? (fit_rows - s.k_h) / s.s_h + 1 : 0;
    const int64_t nyb = yblk > 0 ? (s.o_h + yblk - 1) / yblk : 0;
    const bool small = yblk > 0 && s.pairs * nyb < (int64_t(1) << 31) &&
                       s.i_h * s.R < (int64_t(1) << 31) && s.i_w * s.i_c < (int64_t(1) << 31) &&
                       yblk * s.k_h * s.R < (int64_t(1) << 31);
    if (small) {
        BandParams p{};
        p.I = I;
        p.M = M;
        p.blocks = (uint32_t)(s.pairs * nyb);
        p.i_h = (uint32_t)s.i_h;
        p.o_w = (uint32_t)s.o_w;
        p.o_h = (uint32_t)s.o_h;
        p.k_h = (uint32_t)s.k_h;
        p.s_h = (uint32_t)s.s_h;
        p.R = (uint32_t)s.R;
        p.in_row = (uint32_t)(s.i_w * s.i_c);
        p.in_col = (uint32_t)(s.s_w * s.i_c);
        p.yblk = (uint32_t)yblk;
        p.nyb = (uint32_t)nyb;
        p.div_nyb = FastDiv((uint32_t)nyb);
        p.div_ow = FastDiv(p.o_w);
        p.div_R = FastDiv(p.R);
        p.div_kh = FastDiv(p.k_h);
        const bool vec = s.R % N == 0 && (s.i_w * s.i_c) % N == 0 && (s.s_w * s.i_c) % N == 0 &&
                         aligned16(I) && aligned16(M);
        if (vec) p.div_RV = FastDiv((uint32_t)(s.R / N));
        const int64_t band_bytes = ((yblk - 1) * s.s_h + s.k_h) * row_bytes;
        const size_t lds = (size_t)((band_bytes + 15) / 16 * 16);
        auto kern = vec ? im2col_band_kernel<E, true> : im2col_band_kernel<E, false>;
        hipLaunchKernelGGL(kern, dim3(p.blocks), dim3(kBandThreads), lds, stream, p);
        return hipGetLastError();
    }
    GatherParams g{};
    g.I = I;
    g.M = M;
    g.total = s.pairs * s.o_h * s.k_h * s.R;
    g.i_h = s.i_h; g.i_w = s.i_w; g.i_c = s.i_c; g.k_h = s.k_h; g.k_w = s.k_w;
    g.s_h = s.s_h; g.s_w = s.s_w; g.o_h = s.o_h; g.o_w = s.o_w;
    int64_t blocks = (g.total + kGatherThreads - 1) / kGatherThreads;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(im2col_gather_kernel<E>, dim3((uint32_t)blocks), dim3(kGatherThreads), 0,
                       stream, g);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_im2col(const Shape& s, const void* I, void* M, int elem_bytes,
                         hipStream_t stream) {
    if (s.pairs == 0 || s.o_h == 0) return hipSuccess;
    return elem_bytes == 4 ? launch_typed<uint32_t>(s, I, M, stream)
                           : launch_typed<uint16_t>(s, I, M, stream);
}

}  // namespace mec
