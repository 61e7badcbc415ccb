// MFMA operand traits and small vector helpers shared by the slab-product
// kernels (mec_gemm.hip: any k_h; mec_gemm_fixed.hip: compile-time k_h, s_h).
#pragma once

#include <hip/hip_runtime.h>

#include "mec_internal.h"

namespace mec {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;  // four 64-wide waves per workgroup
constexpr int kPairs = 32;     // (n, w) pairs per tile = rows of one 32x32 MFMA block

// fp32: v_mfma_f32_32x32x2_f32. Lane l supplies A[l % 32][k0 + l / 32] and
// B[k0 + l / 32][l % 32]; one instruction reduces over 2 values of k.
struct TraitsF32 {
    using E = uint32_t;           // fp32 bits in LDS and registers
    static constexpr int KS = 2;  // reduction length of one MFMA
    static constexpr int KL = 1;  // k values each lane supplies
    using Frag = float;
    static __device__ inline Frag frag(const E* p) { return __builtin_bit_cast(float, *p); }
    static __device__ inline floatx16 mfma(Frag a, Frag b, floatx16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
};

// bf16: v_mfma_f32_32x32x16_bf16 with fp32 accumulation. Lane l supplies the
// 8 consecutive k values k0 + 8*(l / 32) + 0..7 of row (or column) l % 32.
struct TraitsBF16 {
    using E = uint16_t;  // bf16 bits
    static constexpr int KS = 16;
    static constexpr int KL = 8;
    using Frag = bf16x8;
    static __device__ inline Frag frag(const E* p) {
        return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
    }
    static __device__ inline floatx16 mfma(Frag a, Frag b, floatx16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
};

// N consecutive elements moved as one load: one 16-byte access when
// N*sizeof(E) == 16, element by element otherwise.
template <int N, typename E, bool WIDE = (N * sizeof(E) == 16)>
struct VecN {
    E e[N];
    __device__ inline void load(const E* src) {
#pragma unroll
        for (int k = 0; k < N; ++k) e[k] = src[k];
    }
    __device__ inline void zero() {
#pragma unroll
        for (int k = 0; k < N; ++k) e[k] = 0;
    }
};
template <int N, typename E>
struct VecN<N, E, true> {
    union {
        uint4 v;
        E e[N];
    };
    __device__ inline void load(const E* src) { v = *reinterpret_cast<const uint4*>(src); }
    __device__ inline void zero() { v = make_uint4(0, 0, 0, 0); }
};

// Row of the 32x32 accumulator block held in register v of lane `lane`
// (the column is lane % 32).
__device__ inline int acc_row(int v, int lane) { return (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3); }

}  // namespace mec
