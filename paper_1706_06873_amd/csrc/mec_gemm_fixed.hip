// MEC's slab products (Section 3.3, Algorithm 2, product phase) for kernel
// heights and strides fixed at compile time: 3x3 stride 1 and 11x11 stride 4
// in fp32, 3x3 stride 1 in bf16. Same tiling as mec_gemm.hip -- a tile of 32
// (n, w) pairs x HT output rows x NT channels stages the union of the slab rows
// it needs, hrows = (HT-1)*s_h + k_h, once per r-chunk -- but with k_h and s_h
// known the reduction over the kernel rows is fully unrolled: each wave loads
// every staged row fragment it needs once per MFMA k-step and feeds it to all
// (h, a) pairs with h*s_h + a equal to that row, so the slab overlap is reused
// in registers as well as in LDS. Staging offsets are computed once per tile.
#include "mec_mfma.h"

namespace mec {
namespace {

template <class Tr, int HT, int NB, int WAVES_H, int KT, int KH, int SH, int VA, int VB,
          bool FUSED>
struct FCfg {
    using T = Tr;
    using E = typename Tr::E;
    static constexpr int kHT = HT, kKT = KT, kKH = KH, kSH = SH, kVA = VA, kVB = VB;
    static constexpr bool kFused = FUSED;
    static constexpr int NT = 32 * NB;
    static constexpr int WAVES_N = 4 / WAVES_H;
    static constexpr int HW = HT / WAVES_H;    // output rows per wave
    static constexpr int NBW = NB / WAVES_N;   // 32-channel blocks per wave
    static constexpr int HROWS = (HT - 1) * SH + KH;  // staged input rows per tile
    static constexpr int XW = (HW - 1) * SH + KH;     // staged rows one wave reads
    static constexpr bool kF32 = sizeof(E) == 4;
    // LDS strides: fp32 fragments are single dwords, so odd strides put the 32
    // rows of a fragment in 32 different banks; bf16 fragments are 16-byte
    // reads, so strides stay multiples of 8 elements and are offset by 16 bytes.
    static constexpr int PS = kF32 ? ((HROWS * KT) | 1) : HROWS * KT + 8;
    static constexpr int KTB = kF32 ? (KT | 1) : KT + 8;
    static constexpr int A_ELEMS = kPairs * PS;
    static constexpr int STAGE = (A_ELEMS + KH * NT * KTB + 7) / 8 * 8;
    static constexpr int A_VECS = kPairs * HROWS * KT / VA;
    static constexpr int AJ = (A_VECS + kThreads - 1) / kThreads;
    static constexpr int B_VECS = KH * NT * KT / VB;
    static constexpr int BJ = (B_VECS + kThreads - 1) / kThreads;
    static constexpr size_t LDS_BYTES = 2 * STAGE * sizeof(E);
    static_assert(4 % WAVES_H == 0 && HT % WAVES_H == 0 && NB % WAVES_N == 0, "wave split");
    static_assert(KT % Tr::KS == 0 && KT % VA == 0 && NT % VB == 0, "chunk");
    static_assert(LDS_BYTES + 512 <= 160 * 1024, "LDS");
};

struct FixedParams {
    const void* A;     // L (lowered) or I (fused)
    const void* K;
    float* O;
    int64_t i_h, i_w, i_c, k_c, s_w, o_h, o_w, R, pairs;
    int64_t a_xstride;  // elements between consecutive rows x of one pair's source
    int32_t nchunks, h_tiles, n_tiles;
    uint32_t ntiles;
};

template <class C>
__global__ __launch_bounds__(kThreads) void slab_gemm_fixed_kernel(FixedParams p) {
    using Tr = typename C::T;
    using E = typename C::E;
    using Frag = typename Tr::Frag;
    constexpr int KT = C::kKT, NT = C::NT, HW = C::HW, NBW = C::NBW, VA = C::kVA, VB = C::kVB;
    constexpr int KH = C::kKH, SH = C::kSH, HROWS = C::HROWS, XW = C::XW;
    constexpr int PS = C::PS, KTB = C::KTB, STAGE = C::STAGE, A_ELEMS = C::A_ELEMS;
    constexpr int AJ = C::AJ, BJ = C::BJ;

    __shared__ __align__(16) E lds[2 * STAGE];
    __shared__ int64_t abase_s[kPairs];  // source element of (pair, row 0), or -1
    __shared__ int64_t obase_s[kPairs];  // O element of (n, 0, w, 0), or -1

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wh = wave % (4 / C::WAVES_N), wn = wave / (4 / C::WAVES_N);

    const uint32_t t = xcd_remap(blockIdx.x, p.ntiles);
    const int n_tile = (int)(t % (uint32_t)p.n_tiles);
    const uint32_t rest = t / (uint32_t)p.n_tiles;
    const int h_tile = (int)(rest % (uint32_t)p.h_tiles);
    const int64_t pair0 = (int64_t)(rest / (uint32_t)p.h_tiles) * kPairs;
    const int64_t h0 = (int64_t)h_tile * C::kHT;
    const int64_t x0 = h0 * SH;
    const int n0 = n_tile * NT;

    if (tid < kPairs) {
        const int64_t pair = pair0 + tid;
        if (pair < p.pairs) {
            const int64_t n = pair / p.o_w, w = pair % p.o_w;
            abase_s[tid] = C::kFused ? ((n * p.i_h) * p.i_w + p.s_w * w) * p.i_c : pair * p.i_h * p.R;
            obase_s[tid] = (n * p.o_h * p.o_w + w) * p.k_c;
        } else {
            abase_s[tid] = -1;
            obase_s[tid] = -1;
        }
    }
    __syncthreads();

    // Per-thread staging entries, fixed for the whole tile. A entry j covers VA
    // consecutive r of (pair pp, staged row x); B entry j covers VB consecutive
    // channels of (kernel row a, r). g: element offset from the tile's source
    // base (or from K) at r-chunk 0, -1 when the entry stages zeros; l: LDS
    // offset | r << 24, -1 when the entry does not exist.
    const int64_t abase0 = abase_s[0];
    const E* __restrict__ Atile = reinterpret_cast<const E*>(p.A) + abase0;
    const E* __restrict__ Kg = reinterpret_cast<const E*>(p.K);
    int ag[AJ], al[AJ], bg[BJ], bl[BJ];
#pragma unroll
    for (int j = 0; j < AJ; ++j) {
        const int e = (tid + j * kThreads) * VA;
        ag[j] = -1;
        al[j] = -1;
        if (e < kPairs * HROWS * KT) {
            const int r = e % KT, pr = e / KT;
            const int pp = pr / HROWS, x = pr - pp * HROWS;
            al[j] = (pp * PS + x * KT + r) | (r << 24);
            const int64_t ab = abase_s[pp];
            if (ab >= 0 && x0 + x < p.i_h) ag[j] = (int)(ab - abase0 + (x0 + x) * p.a_xstride + r);
        }
    }
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
        const int e = (tid + j * kThreads) * VB;
        bg[j] = -1;
        bl[j] = -1;
        if (e < KH * NT * KT) {
            const int n = e % NT, ar = e / NT;
            const int r = ar % KT, a = ar / KT;
            bl[j] = ((a * NT + n) * KTB + r) | (r << 24);
            if (n0 + n < p.k_c) bg[j] = (int)(((int64_t)a * p.R + r) * p.k_c + n0 + n);
        }
    }

    VecN<VA, E> areg[AJ];
    VecN<VB, E> breg[BJ];
    auto load_stage = [&](int rc) {
        const int r0 = rc * KT;
#pragma unroll
        for (int j = 0; j < AJ; ++j) {
            areg[j].zero();
            if (ag[j] >= 0 && r0 + (al[j] >> 24) < p.R) areg[j].load(Atile + ag[j] + r0);
        }
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            breg[j].zero();
            if (bg[j] >= 0 && r0 + (bl[j] >> 24) < p.R) breg[j].load(Kg + bg[j] + (int64_t)r0 * p.k_c);
        }
    };
    auto store_stage = [&](int buf) {
        E* st = lds + buf * STAGE;
#pragma unroll
        for (int j = 0; j < AJ; ++j) {
            if (al[j] >= 0) {
                E* d = st + (al[j] & 0xffffff);
#pragma unroll
                for (int k = 0; k < VA; ++k) d[k] = areg[j].e[k];
            }
        }
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            if (bl[j] >= 0) {
                E* d = st + A_ELEMS + (bl[j] & 0xffffff);
#pragma unroll
                for (int k = 0; k < VB; ++k) d[k * KTB] = breg[j].e[k];
            }
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
    // this wave's first staged row is wh*HW*SH; its fragments cover XW rows
    const int a_lane = row * PS + (wh * HW * SH) * KT + kofs;
    const int b_lane = A_ELEMS + ((wn * NBW) * 32 + row) * KTB + kofs;

    auto compute = [&](int buf) {
        const E* As = lds + buf * STAGE + a_lane;
        const E* Bs = lds + buf * STAGE + b_lane;
#pragma unroll
        for (int kk = 0; kk < KT; kk += Tr::KS) {
            Frag af[XW];
            Frag bf[KH][NBW];
#pragma unroll
            for (int i = 0; i < XW; ++i) af[i] = Tr::frag(As + i * KT + kk);
#pragma unroll
            for (int a = 0; a < KH; ++a)
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb) bf[a][nb] = Tr::frag(Bs + (a * NT + nb * 32) * KTB + kk);
            // kernel row outermost: consecutive MFMAs update different accumulators
#pragma unroll
            for (int a = 0; a < KH; ++a)
#pragma unroll
                for (int hw = 0; hw < HW; ++hw)
#pragma unroll
                    for (int nb = 0; nb < NBW; ++nb)
                        acc[hw][nb] = Tr::mfma(af[hw * SH + a], bf[a][nb], acc[hw][nb]);
        }
    };

    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int rc = 0; rc < p.nchunks; ++rc) {
        const bool more = rc + 1 < p.nchunks;
        if (more) load_stage(rc + 1);  // global loads in flight during the MFMAs
        compute(rc & 1);
        if (more) store_stage((rc + 1) & 1);
        __syncthreads();
    }

    const int64_t ostride_h = p.o_w * p.k_c;
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
                const int64_t ob = obase_s[acc_row(v, lane)];
                if (ob >= 0) p.O[ob + h * ostride_h + c] = acc[hw][nb][v];
            }
        }
    }
}

inline bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }

// Offsets staged through 32-bit registers must fit: the source span of one
// tile's 32 pairs, and K.
bool offsets_fit(const Shape& s, bool fused) {
    const int64_t lim = int64_t(1) << 31;
    if (s.k_h * s.R * s.k_c >= lim) return false;
    if (!fused) return kPairs * s.i_h * s.R < lim;
    const int64_t images = (kPairs - 1) / s.o_w + 2;  // images 32 consecutive pairs can touch
    return images * s.i_h * s.i_w * s.i_c < lim;
}

template <class C>
bool usable(const Shape& s, const void* A, const void* K) {
    if (s.k_h != C::kKH || s.s_h != C::kSH) return false;
    if (!offsets_fit(s, C::kFused)) return false;
    if (C::kVA > 1) {
        if (A && !aligned16(A)) return false;
        if (s.R % C::kVA) return false;
        if (C::kFused && s.i_c % C::kVA) return false;
    }
    if (C::kVB > 1) {
        if (K && !aligned16(K)) return false;
        if (s.k_c % C::kVB) return false;
    }
    return true;
}

template <class C>
hipError_t run_fixed(const Shape& s, const void* A, const void* K, float* O, hipStream_t stream) {
    FixedParams p{};
    p.A = A;
    p.K = K;
    p.O = O;
    p.i_h = s.i_h; p.i_w = s.i_w; p.i_c = s.i_c; p.k_c = s.k_c; p.s_w = s.s_w;
    p.o_h = s.o_h; p.o_w = s.o_w; p.R = s.R; p.pairs = s.pairs;
    p.a_xstride = C::kFused ? s.i_w * s.i_c : s.R;
    p.nchunks = (int32_t)((s.R + C::kKT - 1) / C::kKT);
    const int64_t pair_tiles = (s.pairs + kPairs - 1) / kPairs;
    p.h_tiles = (int32_t)((s.o_h + C::kHT - 1) / C::kHT);
    p.n_tiles = (int32_t)((s.k_c + C::NT - 1) / C::NT);
    const int64_t ntiles = pair_tiles * p.h_tiles * p.n_tiles;
    if (ntiles > 0x7fffffff) return hipErrorInvalidValue;
    p.ntiles = (uint32_t)ntiles;
    hipLaunchKernelGGL(slab_gemm_fixed_kernel<C>, dim3(p.ntiles), dim3(kThreads), 0, stream, p);
    return hipGetLastError();
}

// fp32, 3x3 stride 1, long rows (R % 4 == 0): 32 pairs x 8 rows x 64 channels,
// r-chunks of 16, 16-byte loads of L (or I) and K.
template <bool F> using F32K3S1Wide = FCfg<TraitsF32, 8, 2, 4, 16, 3, 1, 4, 4, F>;
// fp32, 3x3 stride 1, short rows (R = 3 i_c with i_c not a multiple of 4).
template <bool F> using F32K3S1Narrow = FCfg<TraitsF32, 8, 2, 4, 2, 3, 1, 1, 1, F>;
// fp32, 11x11 stride 4: 32 pairs x 8 rows x 96 channels, 39 staged rows.
template <bool F> using F32K11S4 = FCfg<TraitsF32, 8, 3, 4, 2, 11, 4, 1, 1, F>;
// bf16, 3x3 stride 1: 32 pairs x 14 rows x 128 channels, r-chunks of 32.
template <bool F> using BF16K3S1 = FCfg<TraitsBF16, 14, 4, 2, 32, 3, 1, 8, 8, F>;

template <bool F>
hipError_t dispatch_fixed(const Shape& s, const void* A, const void* K, float* O, int dtype,
                          hipStream_t stream, bool dry_run) {
#define MEC_TRY_FIXED(CFG)                                                  \
    if (usable<CFG>(s, A, K)) {                                             \
        return dry_run ? hipSuccess : run_fixed<CFG>(s, A, K, O, stream);   \
    }
    if (dtype == 0) {
        if (s.R >= 32) MEC_TRY_FIXED(F32K3S1Wide<F>);
        MEC_TRY_FIXED(F32K3S1Narrow<F>);
        MEC_TRY_FIXED(F32K11S4<F>);
    } else {
        MEC_TRY_FIXED(BF16K3S1<F>);
    }
#undef MEC_TRY_FIXED
    return hipErrorNotSupported;
}

}  // namespace

hipError_t launch_gemm_fixed(const Shape& s, const void* A, const void* K, float* O, int dtype,
                             bool fused, hipStream_t stream, bool dry_run) {
    if (fused) return dispatch_fixed<true>(s, A, K, O, dtype, stream, dry_run);
    return dispatch_fixed<false>(s, A, K, O, dtype, stream, dry_run);
}

}  // namespace mec
