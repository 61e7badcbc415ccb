// MEC compact lowering on gfx950 (Section 3.3, Algorithm 2, first loop):
//   L[n, w, h, 0:k_w, 0:i_c] = I[n, h, s_w*w : s_w*w + k_w, 0:i_c]
// L viewed as (i_n*o_w*i_h) rows of R = k_w*i_c elements: row q = (n*o_w + w)*i_h + h
// is the contiguous run of R elements of I that starts at ((n*i_h + h)*i_w + s_w*w)*i_c.
//
// A pure copy, bound by HBM bandwidth. Each workgroup owns a contiguous range of
// L rows, so its stores form one contiguous, 16-byte-vectorised stream. The
// source offset of each of its rows is computed once into LDS. Reads of I are
// contiguous inside each run; the k_w/s_w-fold re-reads of I by neighbouring
// w hit in L2 because workgroups are remapped so that each XCD walks one
// contiguous range of L.
#include <hip/hip_runtime.h>

#include "mec_internal.h"

namespace mec {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxRowsPerBlock = 1024;
constexpr int64_t kTargetElemsPerBlock = 8192;

// E is a 32-bit (fp32) or 16-bit (bf16) payload; VEC elements make 16 bytes.
template <typename E>
struct Vec16 {
    static constexpr int N = 16 / sizeof(E);
    union {
        uint4 v;
        E e[N];
    };
};

// Source offset (elements of I) of the first element of each L row of the block.
__device__ inline void fill_row_sources(int64_t* src, const LowerParams& p, int64_t row0,
                                        int nrows) {
    for (int i = threadIdx.x; i < nrows; i += kThreads) {
        const int64_t q = row0 + i;
        const int64_t h = q % p.i_h;
        const int64_t nw = q / p.i_h;
        const int64_t w = nw % p.o_w;
        const int64_t n = nw / p.o_w;
        src[i] = ((n * p.i_h + h) * p.i_w + p.s_w * w) * p.i_c;
    }
}

// Every run start is a multiple of VEC elements and both tensors are 16-byte
// aligned: one 16-byte load and one 16-byte store per vector.
template <typename E>
__global__ __launch_bounds__(kThreads) void lower_vec_kernel(LowerParams p) {
    constexpr int VEC = Vec16<E>::N;
    __shared__ int64_t src[kMaxRowsPerBlock];
    const uint32_t blk = xcd_remap(blockIdx.x, p.nblocks);
    const int64_t row0 = (int64_t)blk * p.rows_per_block;
    const int nrows = (int)min((int64_t)p.rows_per_block, p.rows - row0);
    fill_row_sources(src, p, row0, nrows);
    __syncthreads();

    const uint32_t RV = (uint32_t)(p.R / VEC);  // vectors per row
    const uint32_t total = (uint32_t)nrows * RV;
    const uint4* __restrict__ I = reinterpret_cast<const uint4*>(p.I);
    uint4* __restrict__ L = reinterpret_cast<uint4*>(p.L) + row0 * (int64_t)RV;
    for (uint32_t f = threadIdx.x; f < total; f += kThreads) {
        const uint32_t r = p.divR.div(f);
        const uint32_t c = f - r * RV;
        L[f] = I[src[r] / VEC + c];
    }
}

// General runs (any R, any alignment of the run starts). Each thread gathers
// VEC consecutive L elements and writes them with one 16-byte store when the
// block's slice of L is 16-byte aligned (VECDST), element by element otherwise.
template <typename E, bool VECDST>
__global__ __launch_bounds__(kThreads) void lower_gather_kernel(LowerParams p) {
    constexpr int VEC = Vec16<E>::N;
    __shared__ int64_t src[kMaxRowsPerBlock];
    const uint32_t blk = xcd_remap(blockIdx.x, p.nblocks);
    const int64_t row0 = (int64_t)blk * p.rows_per_block;
    const int nrows = (int)min((int64_t)p.rows_per_block, p.rows - row0);
    fill_row_sources(src, p, row0, nrows);
    __syncthreads();

    const uint32_t R = (uint32_t)p.R;
    const uint32_t count = (uint32_t)nrows * R;  // elements of L this block writes
    const E* __restrict__ I = reinterpret_cast<const E*>(p.I);
    E* __restrict__ L = reinterpret_cast<E*>(p.L) + row0 * p.R;
    for (uint32_t e0 = threadIdx.x * VEC; e0 < count; e0 += kThreads * VEC) {
        uint32_t r = p.divR.div(e0);
        uint32_t c = e0 - r * R;
        Vec16<E> v;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            v.e[k] = (e0 + k < count) ? I[src[r] + c] : E(0);
            if (++c == R) {
                c = 0;
                ++r;
            }
        }
        if (VECDST && e0 + VEC <= count) {
            *reinterpret_cast<uint4*>(L + e0) = v.v;
        } else {
#pragma unroll
            for (int k = 0; k < VEC; ++k)
                if (e0 + k < count) L[e0 + k] = v.e[k];
        }
    }
}

inline bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }

template <typename E>
hipError_t launch_typed(const Shape& s, const void* I, void* L, hipStream_t stream) {
    constexpr int VEC = Vec16<E>::N;
    LowerParams p{};
    p.I = I;
    p.L = L;
    p.rows = s.i_n * s.o_w * s.i_h;
    p.R = s.R;
    p.i_h = s.i_h;
    p.o_w = s.o_w;
    p.i_w = s.i_w;
    p.i_c = s.i_c;
    p.s_w = s.s_w;
    // Rows per block: about kTargetElemsPerBlock elements, a multiple of VEC so
    // every block's slice of L starts 16-byte aligned when L does.
    int64_t rpb = (kTargetElemsPerBlock + s.R - 1) / s.R;
    rpb = (rpb + VEC - 1) / VEC * VEC;
    if (rpb > kMaxRowsPerBlock) rpb = kMaxRowsPerBlock;
    p.rows_per_block = (int32_t)rpb;
    const int64_t nblocks = (p.rows + rpb - 1) / rpb;
    p.nblocks = (uint32_t)nblocks;

    const bool vec_runs = (s.R % VEC == 0) && ((s.s_w * s.i_c) % VEC == 0) &&
                          ((s.i_w * s.i_c) % VEC == 0) && aligned16(I) && aligned16(L);
    if (vec_runs) {
        p.divR = FastDiv((uint32_t)(s.R / VEC));
        hipLaunchKernelGGL(lower_vec_kernel<E>, dim3(p.nblocks), dim3(kThreads), 0, stream, p);
    } else {
        p.divR = FastDiv((uint32_t)s.R);
        if (aligned16(L))
            hipLaunchKernelGGL((lower_gather_kernel<E, true>), dim3(p.nblocks), dim3(kThreads), 0,
                               stream, p);
        else
            hipLaunchKernelGGL((lower_gather_kernel<E, false>), dim3(p.nblocks), dim3(kThreads), 0,
                               stream, p);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_lower(const Shape& s, const void* I, void* L, int elem_bytes,
                        hipStream_t stream) {
    if (elem_bytes == 4) return launch_typed<uint32_t>(s, I, L, stream);
    return launch_typed<uint16_t>(s, I, L, stream);
}

}  // namespace mec
