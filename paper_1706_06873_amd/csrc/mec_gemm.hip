// MEC's slab products on gfx950 MFMA (Section 3.3, Algorithm 2, product phase),
// and the fused variant that forms the slabs on chip straight from I.
//
// With R = k_w*i_c, row (n, w) of L is the i_h x R block L[n, w, 0:i_h, :, :].
// Output row h of image n, column w is
//   O[n, h, w, :] = sum_{a < k_h} L[n, w, h*s_h + a, :] x K[a]      (K[a] is R x k_c)
// i.e. the slab L[n, w][s_h*R*h : s_h*R*h + k_h*R] times K viewed as
// (k_h*R) x k_c. Adjacent output rows h, h+1 share k_h - s_h of their k_h
// rows of L: the "overlap" that MEC's compact lowering exposes.
//
// Tiling. A workgroup computes a tile of 32 consecutive (n, w) pairs x HT
// consecutive output rows h0..h0+HT-1 x NT = 32*NB output channels. It stages
// the union of the L rows those HT slabs need -- hrows = (HT-1)*s_h + k_h rows,
// not HT*k_h -- once per r-chunk of KT columns into LDS, and every one of the
// k_h kernel rows reads its shifted window of that stage. This is where the
// slab overlap saves traffic: each staged L row feeds up to ceil(k_h/s_h)
// output rows. The fused variant stages exactly the same rows, read from I
// (L[n, w, x, r] = I[n, x, s_w*w*i_c + r]) instead of L.
//
// MFMA mapping (32x32 blocks): block rows are the 32 pairs, block columns 32
// output channels, and the reduction runs over (a, r). fp32 uses
// v_mfma_f32_32x32x2_f32 (each lane supplies A[pair][k] and B[k][col] for one
// k); bf16 uses v_mfma_f32_32x32x16_bf16 (8 consecutive k per lane) with fp32
// accumulation. The epilogue stores each accumulator straight into n-h-w-c O,
// which replaces Solution A's h-n-w-c result and its transposition, with
// non-temporal stores (O is not read again by the kernel).
#include "mec_mfma.h"

namespace mec {
namespace {

// Launch-time layout of the LDS stages (elements of E).
struct Lds {
    int ps;      // stride between pairs in the A stage (>= hrows*KT)
    int ktb;     // stride between (a, col) rows of the B stage (>= KT)
    int a_elems; // kPairs * ps
    int stage;   // a_elems + k_h*NT*ktb, rounded up to 8 elements
    int nbuf;    // 2: double-buffered stages; 1: one stage (when two do not fit)
};

struct Args {
    GemmParams g;
    Lds lds;
    FastDiv div_hrows;
    int32_t o_vec;  // k_c % 4 == 0 and O 16-byte aligned: O rows stored 16 bytes per lane
};

// PF: stage through registers so the next chunk's global loads overlap this
// chunk's MFMAs (the register arrays are sized by HROWS_MAX and KH_MAX);
// without PF each chunk is copied global -> LDS directly, for the generic
// configurations whose stages would not fit in registers.
template <class Tr, int HT, int NB, int WAVES_H, int KT, int HROWS_MAX, int KH_MAX, int VA,
          bool PF, bool FUSED>
struct Cfg {
    using T = Tr;
    static constexpr int kHT = HT, kNB = NB, kWavesH = WAVES_H, kKT = KT;
    static constexpr int kHrowsMax = HROWS_MAX, kKhMax = KH_MAX, kVA = VA;
    static constexpr bool kPF = PF;
    static constexpr bool kFused = FUSED;
    static constexpr int NT = 32 * NB;
    static constexpr int WAVES_N = 4 / WAVES_H;
    static constexpr int HW = HT / WAVES_H;
    static constexpr int NBW = NB / WAVES_N;
    static_assert(4 % WAVES_H == 0 && HT % WAVES_H == 0 && NB % WAVES_N == 0, "wave split");
    static_assert(KT % Tr::KS == 0 && KT % VA == 0, "chunk");
    // elements of one stage each thread moves (A in vectors of VA, B singly)
    static constexpr int AVEC = PF ? (kPairs * HROWS_MAX * KT / VA + kThreads - 1) / kThreads : 1;
    static constexpr int BREG = PF ? (KH_MAX * NT * KT + kThreads - 1) / kThreads : 1;
};

template <class C>
__global__ __launch_bounds__(kThreads) void slab_gemm_kernel(Args args) {
    using Tr = typename C::T;
    using E = typename Tr::E;
    constexpr int KT = C::kKT, NT = C::NT, HW = C::HW, NBW = C::NBW, VA = C::kVA;
    const GemmParams& p = args.g;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wh = wave % C::kWavesH, wn = wave / C::kWavesH;

    extern __shared__ __align__(16) char smem[];
    int64_t* abase = reinterpret_cast<int64_t*>(smem);  // [kPairs] source of pair row 0, or -1
    int64_t* obase = abase + kPairs;                     // [kPairs] O offset of (n, 0, w, 0)
    E* stages = reinterpret_cast<E*>(obase + kPairs);

    // tile -> (pair tile, h tile, channel tile); channel tiles fastest so that
    // tiles sharing A land next to each other (and on one XCD)
    const uint32_t t = xcd_remap(blockIdx.x, p.ntiles);
    const int n_tile = (int)(t % (uint32_t)p.n_tiles);
    const uint32_t rest = t / (uint32_t)p.n_tiles;
    const int h_tile = (int)(rest % (uint32_t)p.h_tiles);
    const int pair_tile = (int)(rest / (uint32_t)p.h_tiles);
    const int64_t pair0 = (int64_t)pair_tile * kPairs;
    const int64_t h0 = (int64_t)h_tile * C::kHT;
    const int64_t x0 = h0 * p.s_h;  // first staged input row
    const int n0 = n_tile * NT;
    const int hrows = p.hrows;
    const int k_h = (int)p.k_h;
    const int64_t R = p.R;

    if (tid < kPairs) {
        const int64_t pair = pair0 + tid;
        if (pair < p.pairs) {
            const int64_t n = pair / p.o_w, w = pair % p.o_w;
            abase[tid] = C::kFused ? ((n * p.i_h) * p.i_w + p.s_w * w) * p.i_c : pair * p.i_h * R;
            obase[tid] = (n * p.o_h * p.o_w + w) * p.k_c;
        } else {
            abase[tid] = -1;
            obase[tid] = -1;
        }
    }
    __syncthreads();

    const E* __restrict__ Ag = reinterpret_cast<const E*>(p.A);
    const E* __restrict__ Kg = reinterpret_cast<const E*>(p.K);
    const int a_count = kPairs * hrows * KT;  // elements of one A stage
    const int b_count = k_h * NT * KT;        // elements of one B stage

    // A-stage element e (a multiple of VA) of r-chunk starting at r0: its LDS
    // offset, and its global source or nullptr where the stage holds zeros
    // (pairs past the end, rows past i_h, columns past R).
    auto a_map = [&](int e, int64_t r0, int& lds_off) -> const E* {
        const int r = e % KT;
        const int pr = e / KT;
        const int pp = (int)args.div_hrows.div((uint32_t)pr);
        const int x = pr - pp * hrows;
        lds_off = pp * args.lds.ps + x * KT + r;
        const int64_t ab = abase[pp];
        if (ab >= 0 && x0 + x < p.i_h && r0 + r < R) return Ag + ab + (x0 + x) * p.a_xstride + r0 + r;
        return nullptr;
    };
    // B-stage element e: K[a][r0 + r][n0 + n] stored at LDS (a*NT + n)*ktb + r
    auto b_map = [&](int e, int64_t r0, int& lds_off) -> const E* {
        const int n = e % NT;
        const int ar = e / NT;
        const int r = ar % KT;
        const int a = ar / KT;
        lds_off = args.lds.a_elems + (a * NT + n) * args.lds.ktb + r;
        if (r0 + r < R && n0 + n < p.k_c) return Kg + ((int64_t)a * R + r0 + r) * p.k_c + n0 + n;
        return nullptr;
    };

    VecN<VA, E> areg[C::AVEC];
    E breg[C::BREG];

    // PF: global -> registers for r-chunk rc
    auto load_stage = [&](int rc) {
        const int64_t r0 = (int64_t)rc * KT;
        int off;
#pragma unroll
        for (int j = 0; j < C::AVEC; ++j) {
            const int e = (tid + j * kThreads) * VA;
            VecN<VA, E> v;
            v.zero();
            if (e < a_count) {
                const E* src = a_map(e, r0, off);
                if (src) v.load(src);
            }
            areg[j] = v;
        }
#pragma unroll
        for (int j = 0; j < C::BREG; ++j) {
            const int e = tid + j * kThreads;
            E v = 0;
            if (e < b_count) {
                const E* src = b_map(e, r0, off);
                if (src) v = *src;
            }
            breg[j] = v;
        }
    };

    // PF: registers -> LDS stage st (the offsets repeat the maps of load_stage)
    auto store_stage = [&](E* st) {
        int off;
#pragma unroll
        for (int j = 0; j < C::AVEC; ++j) {
            const int e = (tid + j * kThreads) * VA;
            if (e < a_count) {
                (void)a_map(e, 0, off);
#pragma unroll
                for (int k = 0; k < VA; ++k) st[off + k] = areg[j].e[k];
            }
        }
#pragma unroll
        for (int j = 0; j < C::BREG; ++j) {
            const int e = tid + j * kThreads;
            if (e < b_count) {
                (void)b_map(e, 0, off);
                st[off] = breg[j];
            }
        }
    };

    // no PF: global -> LDS stage st directly
    auto copy_stage = [&](int rc, E* st) {
        const int64_t r0 = (int64_t)rc * KT;
        int off;
#pragma unroll 2
        for (int e = tid * VA; e < a_count; e += kThreads * VA) {
            VecN<VA, E> v;
            v.zero();
            const E* src = a_map(e, r0, off);
            if (src) v.load(src);
#pragma unroll
            for (int k = 0; k < VA; ++k) st[off + k] = v.e[k];
        }
#pragma unroll 4
        for (int e = tid; e < b_count; e += kThreads) {
            const E* src = b_map(e, r0, off);
            st[off] = src ? *src : E(0);
        }
    };

    floatx16 acc[HW][NBW];
#pragma unroll
    for (int i = 0; i < HW; ++i)
#pragma unroll
        for (int j = 0; j < NBW; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int row = lane & 31;
    const int kofs = (lane >> 5) * Tr::KL;
    const int ps = args.lds.ps, ktb = args.lds.ktb;

    auto compute = [&](const E* As) {
        const E* Bs = As + args.lds.a_elems;
#pragma unroll
        for (int kk = 0; kk < KT; kk += Tr::KS) {
            for (int a = 0; a < k_h; ++a) {
                typename Tr::Frag bf[NBW];
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
                    bf[nb] = Tr::frag(Bs + (a * NT + (wn * NBW + nb) * 32 + row) * ktb + kk + kofs);
#pragma unroll
                for (int hw = 0; hw < HW; ++hw) {
                    const int x = (wh * HW + hw) * (int)p.s_h + a;
                    const typename Tr::Frag af = Tr::frag(As + row * ps + x * KT + kk + kofs);
#pragma unroll
                    for (int nb = 0; nb < NBW; ++nb) acc[hw][nb] = Tr::mfma(af, bf[nb], acc[hw][nb]);
                }
            }
        }
    };

    const bool dbuf = args.lds.nbuf == 2;
    auto buf = [&](int rc) { return stages + (dbuf ? (rc & 1) * args.lds.stage : 0); };
    if (C::kPF) {
        load_stage(0);
        store_stage(buf(0));
    } else {
        copy_stage(0, buf(0));
    }
    __syncthreads();
    for (int rc = 0; rc < p.nchunks; ++rc) {
        const bool more = rc + 1 < p.nchunks;
        if (C::kPF) {
            if (more) load_stage(rc + 1);  // in flight during the MFMAs below
            compute(buf(rc));
            if (more) {
                if (!dbuf) __syncthreads();  // every wave is done reading the single stage
                store_stage(buf(rc + 1));
            }
        } else {
            if (more && dbuf) copy_stage(rc + 1, buf(rc + 1));
            compute(buf(rc));
            if (more && !dbuf) {
                __syncthreads();
                copy_stage(rc + 1, buf(rc + 1));
            }
        }
        __syncthreads();
    }

    // epilogue: lane holds C[i][j], j = lane % 32, i = (v/4)*8 + (lane/32)*4 + v%4
    const int64_t ostride_h = p.o_w * p.k_c;
    if (args.o_vec) {
        // Through LDS (the stages are free after the loop's last barrier): each
        // 32x32 block is written row-major (rows 40 floats apart) and read back
        // as 16-byte pieces, so each lane stores 16 contiguous bytes of an O row.
        float* blk = reinterpret_cast<float*>(stages) + wave * (32 * 40);
        const int rr = lane >> 3, cc = (lane & 7) * 4;
#pragma unroll
        for (int hw = 0; hw < HW; ++hw) {
            const int64_t h = h0 + wh * HW + hw;
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
#pragma unroll
                for (int v = 0; v < 16; ++v) blk[acc_row(v, lane) * 40 + row] = acc[hw][nb][v];
                __syncthreads();
                const int c = n0 + (wn * NBW + nb) * 32 + cc;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int r = rr + 8 * i;
                    const float4 val = *reinterpret_cast<const float4*>(blk + r * 40 + cc);
                    const int64_t ob = obase[r];
                    if (h < p.o_h && c < p.k_c && ob >= 0)
                        store_o4_nt(p.O + ob + h * ostride_h + c, val);
                }
                __syncthreads();
            }
        }
        return;
    }
#pragma unroll
    for (int hw = 0; hw < HW; ++hw) {
        const int64_t h = h0 + wh * HW + hw;
        if (h >= p.o_h) continue;
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) {
            const int c = n0 + (wn * NBW + nb) * 32 + row;
            if (c >= p.k_c) continue;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t ob = obase[acc_row(v, lane)];
                if (ob >= 0) __builtin_nontemporal_store(acc[hw][nb][v], p.O + ob + h * ostride_h + c);
            }
        }
    }
}

// ---------------------------------------------------------------- host side

constexpr size_t kLdsBudget = 64 * 1024;

template <class C>
size_t lds_bytes(const Lds& l) {
    return 2 * kPairs * sizeof(int64_t) + (size_t)l.nbuf * l.stage * sizeof(typename C::T::E);
}

template <class C>
Lds lds_layout(int hrows, int k_h) {
    Lds l{};
    if (sizeof(typename C::T::E) == 4) {
        l.ps = hrows * C::kKT + 1;   // odd: the 32 pair rows of a fragment hit 32 banks
        l.ktb = C::kKT + 1;
    } else {
        l.ps = hrows * C::kKT + 8;   // 16-byte aligned fragments, rows offset by 16 bytes
        l.ktb = C::kKT + 8;
    }
    l.a_elems = kPairs * l.ps;
    l.stage = (l.a_elems + k_h * C::NT * l.ktb + 7) / 8 * 8;
    l.nbuf = 2;
    if (lds_bytes<C>(l) > kLdsBudget) l.nbuf = 1;
    return l;
}

template <class C>
bool fits(const Shape& s) {
    const int64_t hrows = (C::kHT - 1) * s.s_h + s.k_h;
    if (hrows > C::kHrowsMax || s.k_h > C::kKhMax) return false;
    return lds_bytes<C>(lds_layout<C>((int)hrows, (int)s.k_h)) <= kLdsBudget;
}

inline bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }

template <class C>
hipError_t run(const Shape& s, const void* A, const void* K, float* O, hipStream_t stream) {
    Args args{};
    GemmParams& g = args.g;
    g.A = A;
    g.K = K;
    g.O = O;
    g.i_h = s.i_h; g.i_w = s.i_w; g.i_c = s.i_c;
    g.k_h = s.k_h; g.k_w = s.k_w; g.k_c = s.k_c;
    g.s_h = s.s_h; g.s_w = s.s_w; g.o_h = s.o_h; g.o_w = s.o_w;
    g.R = s.R;
    g.pairs = s.pairs;
    g.a_xstride = C::kFused ? s.i_w * s.i_c : s.R;
    g.hrows = (int32_t)((C::kHT - 1) * s.s_h + s.k_h);
    g.nchunks = (int32_t)((s.R + C::kKT - 1) / C::kKT);
    g.pair_tiles = (int32_t)((s.pairs + kPairs - 1) / kPairs);
    g.h_tiles = (int32_t)((s.o_h + C::kHT - 1) / C::kHT);
    g.n_tiles = (int32_t)((s.k_c + C::NT - 1) / C::NT);
    const int64_t ntiles = (int64_t)g.pair_tiles * g.h_tiles * g.n_tiles;
    if (ntiles > 0x7fffffff) return hipErrorInvalidValue;
    g.ntiles = (uint32_t)ntiles;
    args.lds = lds_layout<C>(g.hrows, (int)s.k_h);
    args.div_hrows = FastDiv((uint32_t)g.hrows);
    args.o_vec = s.k_c % 4 == 0 && aligned16(O);
    // the epilogue reuses the stage memory for one 32x40 fp32 block per wave
    const size_t epi = 2 * kPairs * sizeof(int64_t) + (size_t)(kThreads / 64) * 32 * 40 * sizeof(float);
    const size_t lds = lds_bytes<C>(args.lds) > epi ? lds_bytes<C>(args.lds) : epi;
    hipLaunchKernelGGL(slab_gemm_kernel<C>, dim3(g.ntiles), dim3(kThreads), lds, stream, args);
    return hipGetLastError();
}

// Whether the A stage may be loaded in 16-byte vectors of VA elements: every
// pair's staged rows then start on a multiple of VA elements.
template <int VA>
bool vec_ok(const Shape& s, bool fused, const void* A) {
    if (!aligned16(A)) return false;
    if (s.R % VA) return false;
    if (fused) return (s.i_c % VA == 0);  // row stride i_w*i_c, column offset s_w*w*i_c
    return true;                           // row stride R, pair stride i_h*R
}

// Instantiated configurations: tile HT output rows x 32*NB channels, r-chunk
// KT, A loaded in vectors of VA elements.
//   f32 "wide":   HT 8, 64 channels, KT 8, 4-wide A loads -- long L rows
//                 (R % 4 == 0), short kernels (ResNet-style 3x3).
//   f32 "narrow": HT 8, 64 channels, KT 2 -- short or odd rows (R = 9, 3x3x1).
//   f32 "tall":   HT 8, 96 channels, KT 2 -- tall strided kernels (11x11 s4).
//   f32 generic:  HT 4 (32 channels) or HT 1 (128 channels), KT 2.
//   bf16:         HT 4, 64 channels, KT 16 (8-wide A loads when R % 8 == 0);
//                 generic HT 4 with 64 or 32 channels, or HT 1 with 128.
template <bool F> using F32Wide = Cfg<TraitsF32, 8, 2, 4, 8, 16, 8, 4, true, F>;
template <bool F> using F32Narrow = Cfg<TraitsF32, 8, 2, 4, 2, 16, 8, 1, true, F>;
template <bool F> using F32Tall = Cfg<TraitsF32, 8, 3, 4, 2, 40, 12, 1, true, F>;
template <bool F> using F32Gen4 = Cfg<TraitsF32, 4, 1, 4, 2, 64, 64, 1, false, F>;
// 2 output rows per tile, tried first: the strided kernels that reach this
// kernel (from I; from L they take the flat windows) lose little overlap at
// 2 rows and gain four times the tiles. Measured from I at batch 32: 5x5
// stride 2 197 -> 67 us, 2x2 stride 2 100 -> 59 us, 1x1 stride 2 349 -> 218 us,
// 7x7 stride 1 150 us either way. (bf16 at 2 rows lost on every shape tried.)
template <bool F> using F32Wide2 = Cfg<TraitsF32, 2, 2, 2, 8, 16, 8, 4, true, F>;
template <bool F> using F32Narrow2 = Cfg<TraitsF32, 2, 2, 2, 2, 16, 8, 1, true, F>;
template <bool F> using F32Gen1 = Cfg<TraitsF32, 1, 4, 1, 2, 64, 64, 1, false, F>;
template <bool F> using BF16Vec4 = Cfg<TraitsBF16, 4, 2, 2, 16, 16, 8, 8, true, F>;
template <bool F> using BF16Gen4 = Cfg<TraitsBF16, 4, 2, 2, 16, 16, 8, 1, false, F>;
template <bool F> using BF16Gen4n = Cfg<TraitsBF16, 4, 1, 4, 16, 64, 64, 1, false, F>;
template <bool F> using BF16Gen1 = Cfg<TraitsBF16, 1, 4, 1, 16, 32, 32, 1, false, F>;

template <bool F>
hipError_t dispatch(const Shape& s, const void* A, const void* K, float* O, int dtype,
                    hipStream_t stream, bool dry_run) {
#define MEC_TRY(CFG)                                              \
    if (fits<CFG>(s)) {                                           \
        return dry_run ? hipSuccess : run<CFG>(s, A, K, O, stream); \
    }
    if (dtype == 0) {
        if (s.R % 4 == 0 && s.R >= 16 && (dry_run || vec_ok<4>(s, F, A))) MEC_TRY(F32Wide2<F>);
        MEC_TRY(F32Narrow2<F>);
        if (s.k_c > 64 && s.s_h > 1) MEC_TRY(F32Tall<F>);
        if (s.R % 4 == 0 && s.R >= 16 && (dry_run || vec_ok<4>(s, F, A))) MEC_TRY(F32Wide<F>);
        MEC_TRY(F32Narrow<F>);
        MEC_TRY(F32Tall<F>);
        MEC_TRY(F32Gen4<F>);
        MEC_TRY(F32Gen1<F>);
    } else {
        if (s.R % 8 == 0 && (dry_run || vec_ok<8>(s, F, A))) MEC_TRY(BF16Vec4<F>);
        MEC_TRY(BF16Gen4<F>);
        MEC_TRY(BF16Gen4n<F>);
        MEC_TRY(BF16Gen1<F>);
    }
#undef MEC_TRY
    return hipErrorInvalidValue;
}

}  // namespace

bool gemm_supported(const Shape& s, int dtype, bool fused) {
    if (launch_gemm_fixed(s, nullptr, nullptr, nullptr, dtype, fused, nullptr, true) == hipSuccess)
        return true;
    if (fused) return dispatch<true>(s, nullptr, nullptr, nullptr, dtype, nullptr, true) == hipSuccess;
    return dispatch<false>(s, nullptr, nullptr, nullptr, dtype, nullptr, true) == hipSuccess;
}

hipError_t launch_gemm(const Shape& s, const void* A, const void* K, float* O, int dtype,
                       bool fused, hipStream_t stream, const OutLayout* layout) {
    // kernels specialised for this kernel height and stride first; only they
    // take a strided output layout
    const hipError_t e = launch_gemm_fixed(s, A, K, O, dtype, fused, stream, false, layout);
    if (e != hipErrorNotSupported || layout) return e;
    if (fused) return dispatch<true>(s, A, K, O, dtype, stream, false);
    return dispatch<false>(s, A, K, O, dtype, stream, false);
}

}  // namespace mec
