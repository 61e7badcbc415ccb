// MEC's slab products (Section 3.3, Algorithm 2, product phase) for kernel
// heights and strides fixed at compile time: in fp32 3x3 stride 1 and 2, 5x5
// stride 1, 7x7 stride 2, 11x11 stride 4 and k_h = 1; in bf16 3x3 and 5x5 stride 1,
// 7x7 stride 2 and k_h = 1 (the shapes of the paper's benchmark layers, Table 2). Same tiling as mec_gemm.hip -- a tile of 32
// (n, w) pairs x HT output rows x NT channels stages the union of the slab rows
// it needs, hrows = (HT-1)*s_h + k_h, once per r-chunk -- but with k_h and s_h
// known the reduction over the kernel rows is fully unrolled: each wave loads
// every staged row fragment it needs once per MFMA k-step and feeds it to all
// (h, a) pairs with h*s_h + a equal to that row, so the slab overlap is reused
// in registers as well as in LDS. Staging offsets are computed once per tile,
// relative to the tile's first pair so they fit 32-bit registers; the next
// r-chunk's global loads are issued during the current one (fp32: spread over
// its first k-steps; bf16, two k-steps per chunk: before the first), and their
// LDS stores go to the other of two stage buffers. O is written
// n-h-w-c with non-temporal stores. Layers whose whole reduction fits one stage
// and whose time goes to writing O (3x3 over 1-3 channels) use a persistent
// streaming variant that overlaps each tile's O stores with the next tile's
// products. From L, every other kernel height runs through the k_h = 1 tiles
// over the flat windows of L (Section 3.2's view: the slab of output row h is
// one contiguous window of its pair's row of L), read s_h*R elements apart.
#include <initializer_list>
#include <type_traits>

#include "mec_mfma.h"

namespace mec {
namespace {

struct FixedParams {
    const void* A;     // L (lowered) or I (fused)
    const void* K;
    float* O;
    int64_t i_h, i_w, i_c, k_c, s_w, o_h, o_w, R, pairs;
    int64_t a_xstride;  // elements between consecutive rows x of one pair's source
    int64_t a_pstride;  // from L: elements between consecutive pairs' rows of L
    int32_t nchunks, h_tiles, n_tiles;
    int32_t band, pair_tiles;  // streaming kernel: tile order (below)
    uint32_t ntiles;    // workgroups: tiles x ksplit
    int32_t ksplit;     // fp32 kernel: 1, or 2 = each tile's r-chunks split between two
                        // workgroups that add their partial sums into a zeroed O
    int32_t o_vec;      // k_c % 4 == 0 and O 16-byte aligned: O rows stored 16 bytes per lane
    FastDiv div_ow;     // pair -> image (streaming kernel; pairs < 2^31)
    // fp32 kernels: O element (n, h, w, c) at n*o_img + h*o_row + w*o_col + o_off + c
    int64_t o_img, o_row, o_col, o_off;
};

// One 16-byte load per lane from base + voff straight into LDS at byte address
// lds + 16 * lane (M0 holds the wave's LDS address; its previous value is put
// back, since M0 cannot be declared clobbered). The compiler does not see the
// load: the caller waits on vmcnt before the data is read.
__device__ inline void lds_dma16(const void* base, uint32_t voff, uint32_t lds) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %2, %3\n\ts_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds), "v"(voff), "s"(base)
        : "memory");
}

// ---------------------------------------------------------------- fp32 kernel
// The fp32 variant lays both stages out so that MFMA fragment reads are
// consecutive across lanes (conflict-free) and stage writes are 16-byte:
//   A stage [x][r][pair]   (the 32 pairs innermost: lane l of a fragment
//                           reads pair l % 32)
//   B stage [a][r][channel]
// Each thread loads 4 pairs x VA consecutive r (global reads keep their runs
// along r) and transposes them in registers into VA 16-byte LDS writes of 4
// consecutive pairs.
// DMA = true (KT = 16, 16-byte rows): both stages are filled by direct-to-LDS
// loads, A two r-chunks ahead through three stages and B one chunk ahead
// through two:
//   A [x][pair][16 r]       granule g of row q at g ^ ((q >> 2) & 3)
//   B [a][r][channel]       K's own layout
// A lane reads 4 consecutive r of its pair with one 16-byte read, and the
// four MFMAs of each 8-r block take r = j (lanes 0-31) and r = 4 + j (lanes
// 32-63), j = 0..3, from A and B alike. Needs R % 16 == 0.
template <int HT, int NB, int WAVES_H, int KT, int KH, int SH, int VA, int VB, bool FUSED,
          int WAVES = 4, bool DMA = false>
struct F32Cfg {
    using T = TraitsF32;
    using E = uint32_t;
    static constexpr int kHT = HT, kKT = KT, kKH = KH, kSH = SH, kVA = VA, kVB = VB;
    static constexpr bool kFused = FUSED;
    static constexpr bool kDMA = DMA;
    static constexpr int NT = 32 * NB;
    static constexpr int kWaves = WAVES;
    static constexpr int THREADS = 64 * WAVES;
    static constexpr int WAVES_N = WAVES / WAVES_H;
    static constexpr int HW = HT / WAVES_H;
    static constexpr int NBW = NB / WAVES_N;
    static constexpr int HROWS = (HT - 1) * SH + KH;
    static constexpr int XW = (HW - 1) * SH + KH;
    static constexpr int A_SIZE = HROWS * KT * kPairs;
    static constexpr int B_SIZE = KH * KT * NT;
    static constexpr int STAGE = A_SIZE + B_SIZE;
    static constexpr int ADMA = DMA ? A_SIZE / 4 / THREADS : 0;  // DMA: granules per thread
    static constexpr int BDMA = DMA ? B_SIZE / 4 / THREADS : 0;
    static constexpr int RG = KT / VA;                  // r-groups per staged row
    static constexpr int A_ITEMS = HROWS * RG * 8;      // (x, r-group, 4-pair group)
    static constexpr int AJ = (A_ITEMS + THREADS - 1) / THREADS;
    static constexpr int NG = NT / 4;                   // 4-channel groups
    static constexpr int B_ITEMS = KH * KT * NG;        // (a, r, 4-channel group)
    static constexpr int BJ = (B_ITEMS + THREADS - 1) / THREADS;
    // Epilogue through LDS: a wave's NBW blocks of one output row side by side
    // (rows EPI_LD floats apart) when that fits in the stage memory or in
    // 40 KB; otherwise one 32x32 block at a time (rows 40 floats apart).
    static constexpr int EPI_WIDE_WORDS = WAVES * 32 * (32 * NBW + 8);
    static constexpr bool WIDE_EPI = EPI_WIDE_WORDS <= 2 * STAGE || EPI_WIDE_WORDS <= 10240;
    static constexpr int EPI_LD = WIDE_EPI ? 32 * NBW + 8 : 40;
    static constexpr int EPI_WORDS = WAVES * 32 * EPI_LD;
    static constexpr int MAIN_WORDS = DMA ? 3 * A_SIZE + 2 * B_SIZE : 2 * STAGE;
    static constexpr int LDS_WORDS = MAIN_WORDS > EPI_WORDS ? MAIN_WORDS : EPI_WORDS;
    static constexpr size_t LDS_BYTES = LDS_WORDS * sizeof(E);
    static_assert(WAVES % WAVES_H == 0 && HT % WAVES_H == 0 && NB % WAVES_N == 0, "wave split");
    static_assert(KT % 2 == 0 && KT % VA == 0 && (VB == 1 || VB == 4), "chunk");
    static_assert(!DMA || (KT == 16 && VA == 4 && VB == 4 && ADMA * 4 * THREADS == A_SIZE &&
                           BDMA * 4 * THREADS == B_SIZE && ADMA + BDMA < 16), "DMA stage");
    static_assert(LDS_BYTES + 1024 <= 160 * 1024, "LDS");
};

template <class C>
__global__ __launch_bounds__(C::THREADS) void slab_gemm_f32_kernel(FixedParams p) {
    constexpr int KT = C::kKT, NT = C::NT, HW = C::HW, NBW = C::NBW, VA = C::kVA, VB = C::kVB;
    constexpr int KH = C::kKH, SH = C::kSH, HROWS = C::HROWS, XW = C::XW, RG = C::RG, NG = C::NG;
    constexpr int A_SIZE = C::A_SIZE, STAGE = C::STAGE, AJ = C::AJ, BJ = C::BJ;

    __shared__ __align__(16) uint32_t lds[C::LDS_WORDS];
    __shared__ int64_t abase_s[kPairs];
    __shared__ int64_t obase_s[kPairs];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wh = wave % (C::kWaves / C::WAVES_N), wn = wave / (C::kWaves / C::WAVES_N);

    // the two halves of a split tile are neighbours, so they land on one XCD
    const uint32_t tw = xcd_remap(blockIdx.x, p.ntiles);
    const uint32_t t = tw / (uint32_t)p.ksplit, part = tw - t * (uint32_t)p.ksplit;
    const int c_begin = (int)(part * (uint32_t)p.nchunks / (uint32_t)p.ksplit);
    const int c_end = (int)((part + 1) * (uint32_t)p.nchunks / (uint32_t)p.ksplit);
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
            abase_s[tid] = C::kFused ? ((n * p.i_h) * p.i_w + p.s_w * w) * p.i_c : pair * p.a_pstride;
            obase_s[tid] = n * p.o_img + w * p.o_col + p.o_off;
        } else {
            abase_s[tid] = -1;
            obase_s[tid] = -1;
        }
    }
    __syncthreads();

    // The tile's source base, computed from uniform values so it stays in
    // scalar registers and every staging load is base + 32-bit offset.
    int64_t abase0;
    {
        const int64_t n_first = pair0 / p.o_w, w_first = pair0 % p.o_w;
        abase0 = C::kFused ? ((n_first * p.i_h) * p.i_w + p.s_w * w_first) * p.i_c : pair0 * p.a_pstride;
    }
    const uint32_t* __restrict__ Atile = reinterpret_cast<const uint32_t*>(p.A) + abase0;
    const uint32_t* __restrict__ Kg = reinterpret_cast<const uint32_t*>(p.K);
    // An interior tile (all pairs, staged rows, r-chunks and channels in range)
    // stages without any predication.
    const bool full = pair0 + kPairs <= p.pairs && x0 + HROWS <= p.i_h && p.R % KT == 0 &&
                      n0 + NT <= p.k_c && (VB == 4 || p.k_c % 4 == 0);

    // staging entries, fixed for the tile: element offsets at r-chunk 0 (-1 =
    // stage zeros), LDS offsets (-1 = no such entry) and the entry's first r
    uint32_t ag[AJ][4];
    int al[AJ], ar[AJ];
#pragma unroll
    for (int j = 0; j < AJ; ++j) {
        const int it = tid + j * C::THREADS;
        al[j] = -1;
        ar[j] = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) ag[j][q] = 0xffffffffu;
        if (it < C::A_ITEMS) {
            const int pg = it % 8, t2 = it / 8;
            const int rg = t2 % RG, x = t2 / RG;
            al[j] = (x * KT + rg * VA) * kPairs + 4 * pg;
            ar[j] = rg * VA;
            if (x0 + x < p.i_h) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int64_t ab = abase_s[4 * pg + q];
                    if (ab >= 0) ag[j][q] = (uint32_t)(ab - abase0 + (x0 + x) * p.a_xstride + rg * VA);
                }
            }
        }
    }
    uint32_t bg[BJ];
    int bl[BJ], br[BJ], bn[BJ];
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
        const int it = tid + j * C::THREADS;
        bg[j] = 0xffffffffu;
        bl[j] = -1;
        br[j] = 0;
        bn[j] = 0;
        if (it < C::B_ITEMS) {
            const int ng = it % NG, t2 = it / NG;
            const int r = t2 % KT, a = t2 / KT;
            bl[j] = A_SIZE + (a * KT + r) * NT + 4 * ng;
            br[j] = r;
            const int64_t c0 = n0 + 4 * ng;
            bn[j] = (int)(p.k_c - c0 < 4 ? (p.k_c - c0 > 0 ? p.k_c - c0 : 0) : 4);  // valid channels
            if (bn[j] > 0) bg[j] = (uint32_t)(((int64_t)a * p.R + r) * p.k_c + c0);
        }
    }
    const uint32_t kstep = (uint32_t)(KT * p.k_c);  // K elements per r-chunk

    // DMA: this thread's granules, as byte offsets from the tile's A and from
    // K; instruction j of a wave fills LDS slots (j * waves + wave) * 64 + lane
    // of a stage. A pair past the end reads the tile's first pair, a row past
    // the input its last row and a channel group past k_c the tile's first:
    // all three only reach outputs that are never stored.
    uint32_t adma[C::ADMA > 0 ? C::ADMA : 1], bdma[C::BDMA > 0 ? C::BDMA : 1];
    if constexpr (C::kDMA) {
#pragma unroll
        for (int j = 0; j < C::ADMA; ++j) {
            const int G = (j * C::kWaves + wave) * 64 + lane;
            const int q = G >> 2, g = (G & 3) ^ ((q >> 2) & 3);
            const int pp = q % kPairs, x = q / kPairs;
            const int64_t ab = abase_s[pp] >= 0 ? abase_s[pp] : abase0;
            const int64_t xr = x0 + x < p.i_h ? x0 + x : p.i_h - 1;
            adma[j] = (uint32_t)(4 * (ab - abase0 + xr * p.a_xstride + g * 4));
        }
#pragma unroll
        for (int j = 0; j < C::BDMA; ++j) {
            const int G = (j * C::kWaves + wave) * 64 + lane;
            const int q = G / (NT / 4), gc = G % (NT / 4);
            const int r = q % KT, a = q / KT;
            const int nc = n0 + 4 * gc < p.k_c ? n0 + 4 * gc : n0;
            bdma[j] = (uint32_t)(4 * (((int64_t)a * p.R + r) * p.k_c + nc));
        }
    }
    const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) uint32_t*)lds;
    const uint32_t wave_u = (uint32_t)__builtin_amdgcn_readfirstlane(wave);
    auto dma_a = [&](int rc, int sa) {
        const uint32_t dst = lds0 + 4u * (uint32_t)(sa * A_SIZE) + wave_u * 1024u;
        const uint32_t r0 = (uint32_t)rc * (4u * KT);
#pragma unroll
        for (int j = 0; j < C::ADMA; ++j) lds_dma16(Atile, adma[j] + r0, dst + (uint32_t)(j * C::kWaves) * 1024u);
    };
    auto dma_b = [&](int rc, int sb) {
        const uint32_t dst = lds0 + 4u * (uint32_t)(3 * A_SIZE + sb * C::B_SIZE) + wave_u * 1024u;
        const uint32_t r0 = (uint32_t)rc * (4u * KT) * (uint32_t)p.k_c;
#pragma unroll
        for (int j = 0; j < C::BDMA; ++j) lds_dma16(Kg, bdma[j] + r0, dst + (uint32_t)(j * C::kWaves) * 1024u);
    };

    VecN<VA, uint32_t> areg[AJ][4];
    VecN<4, uint32_t> breg[BJ];
    // global -> registers for r-chunk rc, one load ("piece") at a time: pieces
    // 0 .. 4*AJ-1 are the A loads (item j, pair q), the rest the K loads.
    // FULL: no entry needs predication.
    constexpr int NPA = AJ * 4, NP = NPA + BJ;
    auto load_piece = [&](int rc, auto full_tag, int pc) {
        constexpr bool FULL = decltype(full_tag)::value;
        const uint32_t r0 = (uint32_t)(rc * KT);
        if (pc < NPA) {
            const int j = pc / 4, q = pc % 4;
            if (FULL && (j + 1) * C::THREADS <= C::A_ITEMS) {
                areg[j][q].load(Atile + (ag[j][q] + r0));
            } else {
                areg[j][q].zero();
                if ((int64_t)r0 + ar[j] < p.R && ag[j][q] != 0xffffffffu)
                    areg[j][q].load(Atile + (ag[j][q] + r0));
            }
        } else {
            const int j = pc - NPA;
            const uint32_t off = bg[j] + (uint32_t)rc * kstep;
            if (FULL && VB == 4 && (j + 1) * C::THREADS <= C::B_ITEMS) {
                breg[j].load(Kg + off);
            } else {
                breg[j].zero();
                if (bg[j] != 0xffffffffu && (int64_t)r0 + br[j] < p.R) {
                    if (VB == 4) {
                        breg[j].load(Kg + off);
                    } else {
#pragma unroll
                        for (int k = 0; k < 4; ++k)
                            if (k < bn[j]) breg[j].e[k] = Kg[off + k];
                    }
                }
            }
        }
    };
    auto load_stage = [&](int rc, auto full_tag) {
#pragma unroll
        for (int pc = 0; pc < NP; ++pc) load_piece(rc, full_tag, pc);
    };
    auto store_stage = [&](int buf) {
        uint32_t* st = lds + buf * STAGE;
#pragma unroll
        for (int j = 0; j < AJ; ++j) {
            if ((j + 1) * C::THREADS <= C::A_ITEMS || al[j] >= 0) {
#pragma unroll
                for (int k = 0; k < VA; ++k) {
                    uint4 v;
                    v.x = areg[j][0].e[k];
                    v.y = areg[j][1].e[k];
                    v.z = areg[j][2].e[k];
                    v.w = areg[j][3].e[k];
                    *reinterpret_cast<uint4*>(st + al[j] + k * kPairs) = v;
                }
            }
        }
#pragma unroll
        for (int j = 0; j < BJ; ++j)
            if ((j + 1) * C::THREADS <= C::B_ITEMS || bl[j] >= 0)
                *reinterpret_cast<uint4*>(st + bl[j]) =
                    make_uint4(breg[j].e[0], breg[j].e[1], breg[j].e[2], breg[j].e[3]);
    };

    floatx16 acc[HW][NBW];
#pragma unroll
    for (int i = 0; i < HW; ++i)
#pragma unroll
        for (int j = 0; j < NBW; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int row = lane & 31;
    const int kofs = lane >> 5;
    const int a_lane = (wh * HW * SH) * KT * kPairs + kofs * kPairs + row;
    const int b_lane = A_SIZE + kofs * NT + (wn * NBW) * 32 + row;

    // The MFMAs of one r-chunk. After k-step ks, issue(ks) issues its share of
    // the next chunk's global loads. When a k-step carries enough MFMAs to cover
    // them, the loads are spread over the first half of the chunk so that the
    // wave never stalls on a burst of loads with the matrix pipe idle, and still
    // have half a chunk to land; with few MFMAs per k-step they all go out after
    // the first one, to have as long as possible to land.
    constexpr int KS = KT / 2;                    // MFMA k-steps per chunk
    constexpr int KSL = (KH * HW * NBW >= 8 && KS > 1) ? KS / 2 : 1;  // k-steps that issue loads
    // DMA: a lane's 16-byte A read of 8-r block kb is granule 2 * kb + kofs of
    // its row, at its swizzled position; B row r = 8 * kb + 4 * kofs + j
    const int a_drow = ((wh * HW * SH) * kPairs + row) * KT;
    const int swz = (row >> 2) & 3;
    const int b_dlane = 4 * kofs * NT + (wn * NBW) * 32 + row;
    auto compute_dma = [&](int abuf, int bbuf) {
        const uint32_t* As = lds + abuf * A_SIZE + a_drow;
        const uint32_t* Bs = lds + 3 * A_SIZE + bbuf * C::B_SIZE + b_dlane;
#pragma unroll
        for (int kb = 0; kb < KT / 8; ++kb) {
            uint4 af[XW];
            const int ga = 4 * ((2 * kb + kofs) ^ swz);
#pragma unroll
            for (int i = 0; i < XW; ++i) af[i] = *reinterpret_cast<const uint4*>(As + i * kPairs * KT + ga);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                float bf[KH][NBW];
#pragma unroll
                for (int a = 0; a < KH; ++a)
#pragma unroll
                    for (int nb = 0; nb < NBW; ++nb)
                        bf[a][nb] = __builtin_bit_cast(float, Bs[(a * KT + 8 * kb + j) * NT + nb * 32]);
#pragma unroll
                for (int a = 0; a < KH; ++a)
#pragma unroll
                    for (int hw = 0; hw < HW; ++hw) {
                        const uint4& v = af[hw * SH + a];
                        const float av = __builtin_bit_cast(float, j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w);
#pragma unroll
                        for (int nb = 0; nb < NBW; ++nb)
                            acc[hw][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bf[a][nb], acc[hw][nb], 0, 0, 0);
                    }
            }
        }
    };
    auto compute = [&](int buf, auto issue) {
        const uint32_t* As = lds + buf * STAGE + a_lane;
        const uint32_t* Bs = lds + buf * STAGE + b_lane;
#pragma unroll
        for (int kk = 0; kk < KT; kk += 2) {
            float af[XW];
            float bf[KH][NBW];
#pragma unroll
            for (int i = 0; i < XW; ++i) af[i] = __builtin_bit_cast(float, As[(i * KT + kk) * kPairs]);
#pragma unroll
            for (int a = 0; a < KH; ++a)
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
                    bf[a][nb] = __builtin_bit_cast(float, Bs[(a * KT + kk) * NT + nb * 32]);
#pragma unroll
            for (int a = 0; a < KH; ++a)
#pragma unroll
                for (int hw = 0; hw < HW; ++hw)
#pragma unroll
                    for (int nb = 0; nb < NBW; ++nb)
                        acc[hw][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[hw * SH + a], bf[a][nb],
                                                                         acc[hw][nb], 0, 0, 0);
            const int ks = kk / 2;
            if (ks < KSL) issue(ks * NP / KSL, (ks + 1) * NP / KSL);
        }
    };

    // r-chunks [c_begin, c_end): all of them, or this workgroup's half
    auto main_loop = [&](auto full_tag) {
        load_stage(c_begin, full_tag);
        store_stage(0);
        __syncthreads();
        for (int rc = c_begin; rc < c_end; ++rc) {
            const bool more = rc + 1 < c_end;
            compute((rc - c_begin) & 1, [&](int pc0, int pc1) {
                if (more)
#pragma unroll
                    for (int pc = pc0; pc < pc1; ++pc) load_piece(rc + 1, full_tag, pc);
            });
            if (more) store_stage((rc + 1 - c_begin) & 1);
            __syncthreads();
        }
    };
    // DMA: as in the bf16 kernel, B chunk i + 1 goes out before A chunk i + 2,
    // so waiting until only this wave's ADMA newest operations are outstanding
    // completes chunk i + 1 and leaves A chunk i + 2 in flight; wait and
    // barrier are one statement that no LDS access may cross.
    auto sync_keep_a = [] {
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(C::ADMA) : "memory");
    };
    auto sync_all = [] { asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory"); };
    auto main_loop_dma = [&]() {
        const int n = c_end - c_begin;
        dma_b(c_begin, 0);
        dma_a(c_begin, 0);
        if (n > 1) {
            dma_a(c_begin + 1, 1);
            sync_keep_a();
        } else {
            sync_all();
        }
        for (int i = 0; i < n; ++i) {
            const int rc = c_begin + i;
            if (i + 1 < n) dma_b(rc + 1, (i + 1) & 1);
            if (i + 2 < n) dma_a(rc + 2, (i + 2) % 3);
            compute_dma(i % 3, i & 1);
            if (i + 2 < n)
                sync_keep_a();
            else
                sync_all();
        }
    };
    if constexpr (C::kDMA) {
        main_loop_dma();
    } else {
        if (full)
            main_loop(std::true_type{});
        else
            main_loop(std::false_type{});
    }

    const int64_t ostride_h = p.o_row;
    // split tiles: exactly two partial sums added to +0 in either order give
    // the same value, so O stays deterministic
    const bool add = p.ksplit > 1;
    if (p.o_vec) {
        // Through LDS (free since the loop's last barrier): accumulator blocks
        // are written row-major, rows EPI_LD floats apart, then read back as
        // 16-byte pieces, so each lane stores 16 contiguous bytes of O. With
        // WIDE_EPI a wave's NBW blocks of one output row sit side by side and a
        // store instruction covers whole 32*NBW-channel row segments of several
        // consecutive pairs; otherwise 128-byte segments of one block.
        constexpr int LD = C::EPI_LD;
        constexpr int NBS = C::WIDE_EPI ? NBW : 1;  // blocks per LDS pass
        constexpr int Q = 8 * NBS;                  // 16-byte pieces per row segment
        constexpr int RPI = 64 / Q;                 // rows per store instruction
        float* blk = reinterpret_cast<float*>(lds) + wave * (32 * LD);
        const int rr = lane / Q, cc = (lane % Q) * 4;
#pragma unroll
        for (int hw = 0; hw < HW; ++hw) {
            const int64_t h = h0 + wh * HW + hw;
#pragma unroll
            for (int nb0 = 0; nb0 < NBW; nb0 += NBS) {
#pragma unroll
                for (int nb = 0; nb < NBS; ++nb)
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        blk[acc_row(v, lane) * LD + nb * 32 + row] = acc[hw][nb0 + nb][v];
                __syncthreads();
                const int c = n0 + (wn * NBW + nb0) * 32 + cc;
#pragma unroll
                for (int i = 0; i < (32 + RPI - 1) / RPI; ++i) {
                    const int r = rr + RPI * i;
                    if (rr < RPI && r < 32) {
                        const float4 val = *reinterpret_cast<const float4*>(blk + r * LD + cc);
                        const int64_t ob = obase_s[r];
                        if (h < p.o_h && c < p.k_c && ob >= 0) {
                            float* dst = p.O + ob + h * ostride_h + c;
                            if (add) {
                                unsafeAtomicAdd(dst, val.x);
                                unsafeAtomicAdd(dst + 1, val.y);
                                unsafeAtomicAdd(dst + 2, val.z);
                                unsafeAtomicAdd(dst + 3, val.w);
                            } else {
                                store_o4_nt(dst, val);
                            }
                        }
                    }
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
                const int64_t ob = obase_s[acc_row(v, lane)];
                if (ob < 0) continue;
                if (add)
                    unsafeAtomicAdd(p.O + ob + h * ostride_h + c, acc[hw][nb][v]);
                else
                    __builtin_nontemporal_store(acc[hw][nb][v], p.O + ob + h * ostride_h + c);
            }
        }
    }
}

// O = 0 before the two halves of split tiles add into it (a kernel rather than
// a memset so that the call stays safe to capture in a graph)
__global__ __launch_bounds__(256) void zero_o_kernel(float* __restrict__ O, int64_t n) {
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
#pragma unroll
    for (int k = 0; k < 4; ++k)
        if (i + k < n) __builtin_nontemporal_store(0.f, O + i + k);
}

// ---------------------------------------------------------------- fp32 streaming kernel
// For layers whose whole reduction fits one stage (R <= KT: the 3x3x3 first
// layers, 27 multiply-adds and 256 bytes of O per output pixel), whose time
// goes to writing O. Run tile by tile, as above, such a layer proceeds in
// lock-step rounds: every workgroup of a round stages and multiplies while HBM
// idles, then all of them write their O tiles at once while the matrix cores
// idle. Here a persistent workgroup walks the tiles b, b + G, b + 2G, ... and
// issues the next tile's operand loads before the current tile's O stores.
// Vector memory operations complete in issue order, so the loads it waits for
// next are never queued behind its own stores, and those stores drain while
// the next tile is multiplied. The O epilogue goes through a per-wave LDS
// region of its own (no barrier), one 32x32 block at a time.
template <class C>
__global__ __launch_bounds__(C::THREADS) void slab_gemm_f32_stream_kernel(FixedParams p) {
    constexpr int KT = C::kKT, NT = C::NT, HW = C::HW, NBW = C::NBW, VA = C::kVA, VB = C::kVB;
    constexpr int KH = C::kKH, SH = C::kSH, XW = C::XW, RG = C::RG, NG = C::NG;
    constexpr int A_SIZE = C::A_SIZE, STAGE = C::STAGE, AJ = C::AJ, BJ = C::BJ;
    // epilogue: a wave's NBW blocks of one output row side by side, rows LD
    // floats apart, so a store instruction covers whole 32*NBW-channel row
    // segments of consecutive pairs
    constexpr int LD = 32 * NBW + 8;
    constexpr int Q = 8 * NBW;     // 16-byte pieces per row segment
    constexpr int RPI = 64 / Q;    // rows per store instruction
    static_assert(64 % Q == 0, "row segments per store instruction");
    __shared__ __align__(16) uint32_t lds[STAGE + C::kWaves * 32 * LD];
    // per tile, for the three in flight (stores, stage, loads): each pair's
    // source offset from the tile's first pair (-1: no such pair) and O offset
    __shared__ int32_t src_s[3][kPairs];
    __shared__ int64_t dst_s[3][kPairs];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wh = wave % (C::kWaves / C::WAVES_N), wn = wave / (C::kWaves / C::WAVES_N);
    const int row = lane & 31;
    const int kofs = lane >> 5;
    const int a_lane = (wh * HW * SH) * KT * kPairs + kofs * kPairs + row;
    const int b_lane = A_SIZE + kofs * NT + (wn * NBW) * 32 + row;
    float* blk = reinterpret_cast<float*>(lds + STAGE) + wave * (32 * LD);
    const int64_t ostride_h = p.o_row;

    struct Tile {
        int64_t pair0, h0, abase0;  // abase0: source element of the first pair
        int n0;
    };
    // source element of a pair's slab (L row base, or I pixel for the fused form)
    auto pair_base = [&](int64_t pair) -> int64_t {
        if (!C::kFused) return pair * p.a_pstride;
        const int64_t n = p.div_ow.div((uint32_t)pair), w = pair - n * p.o_w;
        return ((n * p.i_h) * p.i_w + p.s_w * w) * p.i_c;
    };
    // Tile i of the grid-stride walk, in the hardware's block order, so that
    // the tiles in flight across the chip write one compact range of O. Pair
    // tiles go in bands of p.band (one image's width of output columns): a
    // band's tiles of one row block, then its next row block, so the tiles
    // in flight at once cover a few row blocks of a few images (vgg_first
    // 59.6 -> 58.0 us from L, 55.7 -> 54.0 us fused, against tiles of one pair
    // tile's row blocks in a row, with each XCD walking a range of its own).
    auto coords = [&](uint32_t t) {
        Tile c;
        const uint32_t rest = t / (uint32_t)p.n_tiles;
        c.n0 = (int)(t - rest * (uint32_t)p.n_tiles) * NT;
        const uint32_t per_band = (uint32_t)(p.band * p.h_tiles);
        const uint32_t band = rest / per_band, within = rest - band * per_band;
        const uint32_t pt0 = band * (uint32_t)p.band;
        const uint32_t wide = (uint32_t)p.pair_tiles - pt0 < (uint32_t)p.band ? (uint32_t)p.pair_tiles - pt0
                                                                              : (uint32_t)p.band;
        const uint32_t ht = within / wide;
        c.h0 = (int64_t)ht * C::kHT;
        c.pair0 = (int64_t)(pt0 + (within - ht * wide)) * kPairs;
        c.abase0 = pair_base(c.pair0);
        return c;
    };
    auto write_offsets = [&](const Tile& c, int b) {
        if (tid < kPairs) {
            const int64_t pair = c.pair0 + tid;
            if (pair < p.pairs) {
                const int64_t n = p.div_ow.div((uint32_t)pair), w = pair - n * p.o_w;
                src_s[b][tid] = (int32_t)(pair_base(pair) - c.abase0);
                dst_s[b][tid] = n * p.o_img + w * p.o_col + p.o_off;
            } else {
                src_s[b][tid] = -1;
                dst_s[b][tid] = -1;
            }
        }
    };

    VecN<VA, uint32_t> areg[AJ][4];
    VecN<4, uint32_t> breg[BJ];
    // global -> registers for a whole tile (one r-chunk), every entry predicated
    auto load = [&](const Tile& c, int b) {
        const uint32_t* __restrict__ Atile = reinterpret_cast<const uint32_t*>(p.A) + c.abase0;
        const int32_t x0 = (int32_t)(c.h0 * SH);
#pragma unroll
        for (int j = 0; j < AJ; ++j) {
            const int it = tid + j * C::THREADS;
            const int pg = it % 8, t2 = it / 8;
            const int rg = t2 % RG, x = t2 / RG;
            const bool ok = it < C::A_ITEMS && rg * VA < p.R && x0 + x < p.i_h;
            const uint32_t rofs = (uint32_t)((x0 + x) * (int32_t)p.a_xstride + rg * VA);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                areg[j][q].zero();
                const int32_t sb = ok ? src_s[b][4 * pg + q] : -1;
                if (sb >= 0) areg[j][q].load(Atile + ((uint32_t)sb + rofs));
            }
        }
        const uint32_t* __restrict__ Kg = reinterpret_cast<const uint32_t*>(p.K);
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            const int it = tid + j * C::THREADS;
            const int ng = it % NG, t2 = it / NG;
            const int r = t2 % KT, a = t2 / KT;
            const int c0 = c.n0 + 4 * ng;
            breg[j].zero();
            if (it < C::B_ITEMS && r < p.R && c0 < p.k_c) {
                const uint32_t off = (uint32_t)((a * (int32_t)p.R + r) * (int32_t)p.k_c + c0);
                if (VB == 4) {
                    breg[j].load(Kg + off);
                } else {
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        if (c0 + k < p.k_c) breg[j].e[k] = Kg[off + k];
                }
            }
        }
    };
    auto store_stage = [&]() {
#pragma unroll
        for (int j = 0; j < AJ; ++j) {
            const int it = tid + j * C::THREADS;
            if (it < C::A_ITEMS) {
                const int pg = it % 8, t2 = it / 8;
                const int rg = t2 % RG, x = t2 / RG;
                const int al = (x * KT + rg * VA) * kPairs + 4 * pg;
#pragma unroll
                for (int k = 0; k < VA; ++k)
                    *reinterpret_cast<uint4*>(lds + al + k * kPairs) =
                        make_uint4(areg[j][0].e[k], areg[j][1].e[k], areg[j][2].e[k], areg[j][3].e[k]);
            }
        }
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            const int it = tid + j * C::THREADS;
            if (it < C::B_ITEMS) {
                const int ng = it % NG, t2 = it / NG;
                const int r = t2 % KT, a = t2 / KT;
                *reinterpret_cast<uint4*>(lds + A_SIZE + (a * KT + r) * NT + 4 * ng) =
                    make_uint4(breg[j].e[0], breg[j].e[1], breg[j].e[2], breg[j].e[3]);
            }
        }
    };

    // Tile t is multiplied from the stage while tile t+1's operands are in
    // registers (loaded one tile earlier) and tile t-1's O stores drain; then
    // tile t+1 is staged, tile t+2's loads are issued, and only then tile t's
    // stores. Waiting for a tile's operands thus waits for the stores issued
    // before them one tile earlier, which had a whole tile of products to drain.
    const uint64_t G = gridDim.x;
    uint64_t i = blockIdx.x;
    int b = 0;  // offsets buffer of tile t; t+1 uses b+1, t+2 b+2 (mod 3)
    Tile cur = coords((uint32_t)i);
    bool more1 = i + G < p.ntiles;
    Tile nxt = more1 ? coords((uint32_t)(i + G)) : cur;
    write_offsets(cur, 0);
    if (more1) write_offsets(nxt, 1);
    __syncthreads();
    load(cur, 0);
    store_stage();
    if (more1) load(nxt, 1);
    __syncthreads();
    for (;;) {
        floatx16 acc[HW][NBW];
        // one k-step of the products; the first starts every accumulator from
        // an MFMA with a zero addend (no zeroed registers kept around)
        auto kstep = [&](int kk, auto first_tag) {
            constexpr bool FIRST = decltype(first_tag)::value;
            float af[XW];
            float bf[KH][NBW];
#pragma unroll
            for (int x = 0; x < XW; ++x) af[x] = __builtin_bit_cast(float, lds[a_lane + (x * KT + kk) * kPairs]);
#pragma unroll
            for (int a = 0; a < KH; ++a)
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
                    bf[a][nb] = __builtin_bit_cast(float, lds[b_lane + (a * KT + kk) * NT + nb * 32]);
#pragma unroll
            for (int a = 0; a < KH; ++a)
#pragma unroll
                for (int h = 0; h < HW; ++h)
#pragma unroll
                    for (int nb = 0; nb < NBW; ++nb)
                        acc[h][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                            af[h * SH + a], bf[a][nb], (FIRST && a == 0) ? floatx16{} : acc[h][nb], 0, 0, 0);
        };
        kstep(0, std::true_type{});
#pragma unroll 1
        for (int kk = 2; kk < KT; kk += 2) kstep(kk, std::false_type{});

        const bool more2 = more1 && i + 2 * G < p.ntiles;
        Tile nn = nxt;
        const int b1 = b == 2 ? 0 : b + 1, b2 = b1 == 2 ? 0 : b1 + 1;
        if (more2) {
            nn = coords((uint32_t)(i + 2 * G));
            write_offsets(nn, b2);
        }
        __syncthreads();  // the stage is free; tile t+2's offsets visible
        if (more1) store_stage();  // tile t+1
        if (more2) load(nn, b2);

        if (p.o_vec) {
            // each lane stores 16 contiguous bytes: rows rr, rr + RPI, ... of
            // the wave's blocks, channels cc .. cc + 3 of the row segment
            const int rr = lane / Q, cc = (lane % Q) * 4;
            const int c = cur.n0 + wn * NBW * 32 + cc;
#pragma unroll
            for (int h = 0; h < HW; ++h) {
                const int64_t oh = cur.h0 + wh * HW + h;
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
                    for (int v = 0; v < 16; ++v) blk[acc_row(v, lane) * LD + nb * 32 + row] = acc[h][nb][v];
#pragma unroll
                for (int k = 0; k < 32 / RPI; ++k) {
                    const float4 val = *reinterpret_cast<const float4*>(blk + (rr + RPI * k) * LD + cc);
                    const int64_t ob = dst_s[b][rr + RPI * k];
                    if (oh < p.o_h && c < p.k_c && ob >= 0) store_o4_nt(p.O + ob + oh * ostride_h + c, val);
                }
            }
        } else {
#pragma unroll
            for (int h = 0; h < HW; ++h) {
                const int64_t oh = cur.h0 + wh * HW + h;
                if (oh >= p.o_h) continue;
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb) {
                    const int c = cur.n0 + (wn * NBW + nb) * 32 + row;
                    if (c >= p.k_c) continue;
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int64_t ob = dst_s[b][acc_row(v, lane)];
                        if (ob >= 0) __builtin_nontemporal_store(acc[h][nb][v], p.O + ob + oh * ostride_h + c);
                    }
                }
            }
        }
        if (!more1) break;
        __syncthreads();  // tile t+1's stage visible
        i += G;
        b = b1;
        cur = nxt;
        nxt = nn;
        more1 = more2;
    }
}

// ---------------------------------------------------------------- bf16 kernel
// bf16 fragments hold 8 consecutive k per lane (v_mfma_f32_32x32x16_bf16), so
// both stages keep r innermost, rows padded by 8 elements (16 bytes):
//   A stage [x][pair][KT + 8]   filled by 16-byte loads and 16-byte LDS stores
//   B stage [a][channel][KT + 8] K is channel-contiguous in memory, so each
//        thread loads an 8 (r) x 8 (channel) block with eight 16-byte loads and
//        transposes it in registers into eight 16-byte LDS stores.
// The padding puts the 8 rows of each 128-byte LDS access phase in distinct banks.
// VECA = false: rows whose length R is not a multiple of 8 (e.g. 11x11x3):
// the A pieces are gathered element by element and each row of a K block is
// bounded by R on its own.
// DMA = true: A and B go from global memory straight into LDS (16 bytes per
// lane, no registers): A two r-chunks ahead through three stages, B one
// chunk ahead through two. Stages are unpadded and their 16-byte granules
// permuted so that fragment reads spread over the banks:
//   A [x][pair][32 r]      granule g of row q at g ^ ((q >> 2) & 3)
//   B [a][32 r][channel]   K's own layout; granule g of row r at g ^ (2 (r % 4) | (r & 8))
// A B fragment (8 consecutive r of one channel) is two transposing LDS reads
// (ds_read_b64_tr_b16, 4 rows each).
// Needs R % 32 == 0, so that no chunk holds a partial row.
template <int HT, int NB, int WAVES_H, int KT, int KH, int SH, bool FUSED, int WAVES = 4,
          bool VECA = true, bool DMA = false>
struct BF16Cfg {
    using T = TraitsBF16;
    using E = uint16_t;
    static constexpr int kHT = HT, kKT = KT, kKH = KH, kSH = SH, kVA = VECA ? 8 : 1, kVB = 8;
    static constexpr bool kVecA = VECA;
    static constexpr bool kDMA = DMA;
    static constexpr bool kFused = FUSED;
    static constexpr int kWaves = WAVES;
    static constexpr int NT = 32 * NB;
    static constexpr int THREADS = 64 * WAVES;
    static constexpr int WAVES_N = WAVES / WAVES_H;
    static constexpr int HW = HT / WAVES_H;
    static constexpr int NBW = NB / WAVES_N;
    static constexpr int HROWS = (HT - 1) * SH + KH;
    static constexpr int XW = (HW - 1) * SH + KH;
    static constexpr int KTP = KT + 8;                      // padded row (elements)
    static constexpr int A_SIZE = HROWS * kPairs * (DMA ? KT : KTP);
    static constexpr int B_SIZE = KH * NT * (DMA ? KT : KTP);
    static constexpr int STAGE = A_SIZE + B_SIZE;
    // DMA: 16-byte granules per thread and chunk (one instruction each)
    static constexpr int ADMA = DMA ? A_SIZE / 8 / THREADS : 0;
    static constexpr int BDMA = DMA ? B_SIZE / 8 / THREADS : 0;
    static constexpr int RG = KT / 8;
    static constexpr int A_ITEMS = HROWS * kPairs * RG;     // (x, pair, 8-r group)
    static constexpr int AJ = (A_ITEMS + THREADS - 1) / THREADS;
    static constexpr int B_ITEMS = KH * RG * (NT / 8);      // (a, 8-r group, 8-channel group)
    static constexpr int BJ = (B_ITEMS + THREADS - 1) / THREADS;
    static constexpr int EPI_HALVES = WAVES * 32 * 40 * 2;  // epilogue: one 32x40 fp32 block per wave
    static constexpr int MAIN_HALVES = DMA ? 3 * A_SIZE + 2 * B_SIZE : 2 * STAGE;
    static constexpr int LDS_HALVES = MAIN_HALVES > EPI_HALVES ? MAIN_HALVES : EPI_HALVES;
    static constexpr size_t LDS_BYTES = LDS_HALVES * sizeof(E);
    static_assert(WAVES % WAVES_H == 0 && HT % WAVES_H == 0 && NB % WAVES_N == 0, "wave split");
    static_assert(KT % 16 == 0, "chunk");
    static_assert(!DMA || (KT == 32 && VECA && NB == 4 && ADMA * 8 * THREADS == A_SIZE &&
                           BDMA * 8 * THREADS == B_SIZE && ADMA + BDMA < 16), "DMA stage");
    static_assert(LDS_BYTES + 1024 <= 160 * 1024, "LDS");
};

// Transpose an 8x8 block of 16-bit values: in[i] holds row i (8 values),
// out[j] receives column j.
__device__ inline void transpose8x8_b16(const uint4 (&in)[8], uint4 (&out)[8]) {
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        uint32_t d[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&in[2 * j]);
            const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&in[2 * j + 1]);
            const uint32_t a = r0[c >> 1], b = r1[c >> 1];
            d[j] = (c & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
        }
        out[c] = make_uint4(d[0], d[1], d[2], d[3]);
    }
}

template <class C>
__global__ __launch_bounds__(C::THREADS) void slab_gemm_bf16_kernel(FixedParams p) {
    constexpr int KT = C::kKT, NT = C::NT, HW = C::HW, NBW = C::NBW, KTP = C::KTP;
    constexpr int KH = C::kKH, SH = C::kSH, HROWS = C::HROWS, XW = C::XW, RG = C::RG;
    constexpr int A_SIZE = C::A_SIZE, STAGE = C::STAGE, AJ = C::AJ, BJ = C::BJ;

    __shared__ __align__(16) uint16_t lds[C::LDS_HALVES];
    __shared__ int64_t abase_s[kPairs];
    __shared__ int64_t obase_s[kPairs];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wh = wave % (C::kWaves / C::WAVES_N), wn = wave / (C::kWaves / C::WAVES_N);

    // the two halves of a split tile are neighbours, so they land on one XCD
    const uint32_t tw = xcd_remap(blockIdx.x, p.ntiles);
    const uint32_t t = tw / (uint32_t)p.ksplit, part = tw - t * (uint32_t)p.ksplit;
    const int c_begin = (int)(part * (uint32_t)p.nchunks / (uint32_t)p.ksplit);
    const int c_end = (int)((part + 1) * (uint32_t)p.nchunks / (uint32_t)p.ksplit);
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
            abase_s[tid] = C::kFused ? ((n * p.i_h) * p.i_w + p.s_w * w) * p.i_c : pair * p.a_pstride;
            obase_s[tid] = (n * p.o_h * p.o_w + w) * p.k_c;
        } else {
            abase_s[tid] = -1;
            obase_s[tid] = -1;
        }
    }
    __syncthreads();

    int64_t abase0;
    {
        const int64_t n_first = pair0 / p.o_w, w_first = pair0 % p.o_w;
        abase0 = C::kFused ? ((n_first * p.i_h) * p.i_w + p.s_w * w_first) * p.i_c : pair0 * p.a_pstride;
    }
    const uint16_t* __restrict__ Atile = reinterpret_cast<const uint16_t*>(p.A) + abase0;
    const uint16_t* __restrict__ Kg = reinterpret_cast<const uint16_t*>(p.K);
    const bool full = pair0 + kPairs <= p.pairs && x0 + HROWS <= p.i_h && p.R % KT == 0 &&
                      n0 + NT <= p.k_c;

    // A entries: one 16-byte piece (8 consecutive r) of (x, pair)
    uint32_t ag[AJ];
    int al[AJ], ar[AJ];
#pragma unroll
    for (int j = 0; j < AJ; ++j) {
        const int it = tid + j * C::THREADS;
        ag[j] = 0xffffffffu;
        al[j] = -1;
        ar[j] = 0;
        if (it < C::A_ITEMS) {
            const int rg = it % RG, t2 = it / RG;
            const int pp = t2 % kPairs, x = t2 / kPairs;
            al[j] = (x * kPairs + pp) * KTP + rg * 8;
            ar[j] = rg * 8;
            const int64_t ab = abase_s[pp];
            if (ab >= 0 && x0 + x < p.i_h) ag[j] = (uint32_t)(ab - abase0 + (x0 + x) * p.a_xstride + rg * 8);
        }
    }
    // B entries: an 8 (r) x 8 (channel) block of K for kernel row a
    uint32_t bg[BJ];
    int bl[BJ], br[BJ];
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
        const int it = tid + j * C::THREADS;
        bg[j] = 0xffffffffu;
        bl[j] = -1;
        br[j] = 0;
        if (it < C::B_ITEMS) {
            const int rg = it % RG, t2 = it / RG;
            const int cg = t2 % (NT / 8), a = t2 / (NT / 8);
            bl[j] = (a * NT + cg * 8) * KTP + rg * 8;
            br[j] = rg * 8;
            if (n0 + cg * 8 < p.k_c) bg[j] = (uint32_t)(((int64_t)a * p.R + rg * 8) * p.k_c + n0 + cg * 8);
        }
    }
    // DMA: this thread's granules, as byte offsets from the tile's A and from
    // K; instruction j of a wave fills LDS slots (j * waves + wave) * 64 + lane
    // of a stage. A pair past the end reads the tile's first pair, a row past
    // the input its last row and a channel group past k_c the tile's first:
    // all three only reach outputs that are never stored.
    uint32_t adma[C::ADMA > 0 ? C::ADMA : 1], bdma[C::BDMA > 0 ? C::BDMA : 1];
    if constexpr (C::kDMA) {
#pragma unroll
        for (int j = 0; j < C::ADMA; ++j) {
            const int G = (j * C::kWaves + wave) * 64 + lane;
            const int q = G >> 2, g = (G & 3) ^ ((q >> 2) & 3);
            const int pp = q % kPairs, x = q / kPairs;
            const int64_t ab = abase_s[pp] >= 0 ? abase_s[pp] : abase0;
            const int64_t xr = x0 + x < p.i_h ? x0 + x : p.i_h - 1;
            adma[j] = (uint32_t)(2 * (ab - abase0 + xr * p.a_xstride + g * 8));
        }
#pragma unroll
        for (int j = 0; j < C::BDMA; ++j) {
            const int G = (j * C::kWaves + wave) * 64 + lane;
            const int q = G >> 4, r = q % KT, a = q / KT;
            const int g = (G & 15) ^ (((r & 3) << 1) | (r & 8));
            const int nc = n0 + 8 * g < p.k_c ? n0 + 8 * g : n0;
            bdma[j] = (uint32_t)(2 * (((int64_t)a * p.R + r) * p.k_c + nc));
        }
    }
    const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) uint16_t*)lds;
    const uint32_t wave_u = (uint32_t)__builtin_amdgcn_readfirstlane(wave);
    auto a_stage = [&](int sa) { return lds + (C::kDMA ? sa * A_SIZE : sa * STAGE); };
    auto b_stage = [&](int sb) { return lds + (C::kDMA ? 3 * A_SIZE + sb * C::B_SIZE : sb * STAGE + A_SIZE); };
    auto dma_a = [&](int rc, int sa) {
        const uint32_t dst = lds0 + 2u * (uint32_t)(sa * A_SIZE) + wave_u * 1024u;
        const uint32_t r0 = (uint32_t)rc * (2u * KT);
#pragma unroll
        for (int j = 0; j < C::ADMA; ++j) lds_dma16(Atile, adma[j] + r0, dst + (uint32_t)(j * C::kWaves) * 1024u);
    };
    auto dma_b = [&](int rc, int sb) {
        const uint32_t dst = lds0 + 2u * (uint32_t)(3 * A_SIZE + sb * C::B_SIZE) + wave_u * 1024u;
        const uint32_t r0 = (uint32_t)rc * (2u * KT) * (uint32_t)p.k_c;
#pragma unroll
        for (int j = 0; j < C::BDMA; ++j) lds_dma16(Kg, bdma[j] + r0, dst + (uint32_t)(j * C::kWaves) * 1024u);
    };
    const uint32_t kstep = (uint32_t)(KT * p.k_c);
    const uint32_t krow = (uint32_t)p.k_c;

    uint4 areg[AJ];
    uint4 breg[BJ][8];
    auto load_stage = [&](int rc, auto full_tag) {
        constexpr bool FULL = decltype(full_tag)::value;
        const uint32_t r0 = (uint32_t)(rc * KT);
#pragma unroll
        for (int j = 0; j < (C::kDMA ? 0 : AJ); ++j) {
            if (C::kVecA && FULL && (j + 1) * C::THREADS <= C::A_ITEMS) {
                areg[j] = *reinterpret_cast<const uint4*>(Atile + (ag[j] + r0));
            } else {
                areg[j] = make_uint4(0, 0, 0, 0);
                if (ag[j] != 0xffffffffu && (int64_t)r0 + ar[j] < p.R) {
                    if (C::kVecA) {
                        areg[j] = *reinterpret_cast<const uint4*>(Atile + (ag[j] + r0));
                    } else {
                        // element by element, each bounded by R
                        uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
                        for (int k = 0; k < 8; ++k)
                            if ((int64_t)r0 + ar[j] + k < p.R)
                                w[k >> 1] |= (uint32_t)Atile[ag[j] + r0 + k] << (16 * (k & 1));
                        areg[j] = make_uint4(w[0], w[1], w[2], w[3]);
                    }
                }
            }
        }
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            const uint32_t off = bg[j] + (uint32_t)rc * kstep;
            const bool ok = (C::kVecA && FULL && (j + 1) * C::THREADS <= C::B_ITEMS) ||
                            (bg[j] != 0xffffffffu && (int64_t)r0 + br[j] < p.R);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                // rows past R belong to the next kernel row: zero (R % 8 != 0 only)
                const bool row_ok = ok && (C::kVecA || (int64_t)r0 + br[j] + i < p.R);
                breg[j][i] = row_ok ? *reinterpret_cast<const uint4*>(Kg + (off + i * krow))
                                    : make_uint4(0, 0, 0, 0);
            }
        }
    };
    auto store_stage = [&](int buf) {
        uint16_t* st = a_stage(buf);
        uint16_t* sb = b_stage(buf);
#pragma unroll
        for (int j = 0; j < (C::kDMA ? 0 : AJ); ++j)
            if ((j + 1) * C::THREADS <= C::A_ITEMS || al[j] >= 0)
                *reinterpret_cast<uint4*>(st + al[j]) = areg[j];
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            if ((j + 1) * C::THREADS <= C::B_ITEMS || bl[j] >= 0) {
                uint4 col[8];
                transpose8x8_b16(breg[j], col);
#pragma unroll
                for (int c = 0; c < 8; ++c) *reinterpret_cast<uint4*>(sb + bl[j] + c * KTP) = col[c];
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
    const int kofs = (lane >> 5) * 8;
    const int a_lane = ((wh * HW * SH) * kPairs + row) * KTP + kofs;
    const int b_lane = ((wn * NBW) * 32 + row) * KTP + kofs;
    // DMA: a lane's two k-steps read granules (lane >> 5) and 2 + (lane >> 5)
    // of its row, at their swizzled positions
    const int a_row = ((wh * HW * SH) * kPairs + row) * KT;
    const int swz = (lane >> 2) & 3;
    const int a_dma0 = a_row + 8 * ((lane >> 5) ^ swz);
    const int a_dma1 = a_row + 8 * ((2 + (lane >> 5)) ^ swz);
    // DMA: B fragments by transposing reads. ds_read_b64_tr_b16 gives lane j of
    // each 16-lane group the elements 4k + (j / 4), j % 4 (k = 0..3) of the
    // 8-byte pieces its 16 lanes address; lane i of a group addresses row
    // r0 + i / 4 at channel c0 + 4 (i % 4), so lane j receives rows r0..r0+3 of
    // channel c0 + j: half of its fragment (k = 8 (lane / 32) + 0..3; the
    // second read takes rows r0 + 4..7). Row r's 16-byte granule g sits at
    // g ^ (2 (r % 4) | (r & 8)): the four rows of one read and the two lane
    // halves land on distinct banks.
    int b_tr[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        const int i = lane & 15;
        const int ch = (wn * NBW + nb) * 32 + 16 * ((lane >> 4) & 1) + 4 * (i & 3);
        const int swzb = ((i >> 2) << 1) | (8 * (lane >> 5));
        b_tr[nb] = (kofs + (i >> 2)) * NT + (((ch >> 3) ^ swzb) << 3) + (ch & 7);
    }

    auto compute = [&](int abuf, int bbuf, auto mid) {
        const uint16_t* As = a_stage(abuf);
        const uint16_t* Bs = b_stage(bbuf) + b_lane;
        mid();  // the next chunks' global loads, in flight during both k-steps
#pragma unroll
        for (int kk = 0; kk < KT; kk += 16) {
            bf16x8 af[XW];
            bf16x8 bf[KH][NBW];
#pragma unroll
            for (int i = 0; i < XW; ++i) {
                const uint16_t* src = C::kDMA ? As + (kk == 0 ? a_dma0 : a_dma1) + i * kPairs * KT
                                              : As + a_lane + i * kPairs * KTP + kk;
                af[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(src));
            }
#pragma unroll
            for (int a = 0; a < KH; ++a)
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb) {
                    if constexpr (C::kDMA) {
                        typedef short short4v __attribute__((ext_vector_type(4)));
                        typedef __attribute__((address_space(3))) short4v lds_short4v;
                        const uint16_t* src = b_stage(bbuf) + b_tr[nb] + (a * KT + kk) * NT;
                        const short4v lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)src);
                        const short4v hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)(src + 4 * NT));
                        typedef short short8v __attribute__((ext_vector_type(8)));
                        const short8v v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                        bf[a][nb] = __builtin_bit_cast(bf16x8, v);
                    } else {
                        bf[a][nb] = __builtin_bit_cast(
                            bf16x8, *reinterpret_cast<const uint4*>(Bs + (a * NT + nb * 32) * KTP + kk));
                    }
                }
#pragma unroll
            for (int a = 0; a < KH; ++a)
#pragma unroll
                for (int hw = 0; hw < HW; ++hw)
#pragma unroll
                    for (int nb = 0; nb < NBW; ++nb)
                        acc[hw][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[hw * SH + a], bf[a][nb],
                                                                           acc[hw][nb], 0, 0, 0);
        }
    };

    // r-chunks [c_begin, c_end): all of them, or this workgroup's half
    auto main_loop = [&](auto full_tag) {
        load_stage(c_begin, full_tag);
        store_stage(0);
        __syncthreads();
        for (int rc = c_begin; rc < c_end; ++rc) {
            const bool more = rc + 1 < c_end;
            compute((rc - c_begin) & 1, (rc - c_begin) & 1, [&] {
                if (more) load_stage(rc + 1, full_tag);
            });
            if (more) store_stage((rc + 1 - c_begin) & 1);
            __syncthreads();
        }
    };
    // DMA: in step i, B chunk i + 1 is issued before A chunk i + 2, so waiting
    // until only this wave's ADMA newest operations are outstanding completes
    // A and B chunk i + 1 and leaves A chunk i + 2 in flight; the barrier then
    // publishes every wave's part. The loads are invisible to the compiler,
    // so the wait and the barrier are one statement that no LDS access may
    // cross.
    auto sync_keep_a = [] {
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(C::ADMA) : "memory");
    };
    auto sync_all = [] { asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory"); };
    auto main_loop_dma = [&]() {
        const int n = c_end - c_begin;
        dma_b(c_begin, 0);
        dma_a(c_begin, 0);
        if (n > 1) {
            dma_a(c_begin + 1, 1);
            sync_keep_a();
        } else {
            sync_all();
        }
        for (int i = 0; i < n; ++i) {
            const int rc = c_begin + i;
            compute(i % 3, i & 1, [&] {
                if (i + 1 < n) dma_b(rc + 1, (i + 1) & 1);
                if (i + 2 < n) dma_a(rc + 2, (i + 2) % 3);
            });
            if (i + 2 < n)
                sync_keep_a();
            else
                sync_all();
        }
    };
    if constexpr (C::kDMA) {
        main_loop_dma();
    } else {
        if (full)
            main_loop(std::true_type{});
        else
            main_loop(std::false_type{});
    }

    const int64_t ostride_h = p.o_w * p.k_c;
    const bool add = p.ksplit > 1;  // split tile: add into the zeroed O, as in the fp32 kernel
    if (p.o_vec) {
        // 16-byte O stores through LDS, as in the fp32 kernel
        float* blk = reinterpret_cast<float*>(lds) + wave * (32 * 40);
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
                    const int64_t ob = obase_s[r];
                    if (h < p.o_h && c < p.k_c && ob >= 0) {
                        float* dst = p.O + ob + h * ostride_h + c;
                        if (add) {
                            unsafeAtomicAdd(dst, val.x);
                            unsafeAtomicAdd(dst + 1, val.y);
                            unsafeAtomicAdd(dst + 2, val.z);
                            unsafeAtomicAdd(dst + 3, val.w);
                        } else {
                            store_o4_nt(dst, val);
                        }
                    }
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
                const int64_t ob = obase_s[acc_row(v, lane)];
                if (ob < 0) continue;
                if (add)
                    unsafeAtomicAdd(p.O + ob + h * ostride_h + c, acc[hw][nb][v]);
                else
                    __builtin_nontemporal_store(acc[hw][nb][v], p.O + ob + h * ostride_h + c);
            }
        }
    }
}

inline bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }

// Offsets staged through 32-bit registers must fit: the source span of one
// tile's 32 pairs, and K.
bool offsets_fit(const Shape& s, bool fused) {
    const int64_t lim = int64_t(1) << 30;  // element offsets, as 32-bit byte offsets
    if (s.k_h * s.R * s.k_c >= lim) return false;
    if (!fused) return kPairs * s.i_h * s.R < lim;
    const int64_t images = (kPairs - 1) / s.o_w + 2;  // images 32 consecutive pairs can touch
    return images * s.i_h * s.i_w * s.i_c < lim;
}

template <class C>
bool usable(const Shape& s, const void* A, const void* K) {
    if (s.k_h != C::kKH || s.s_h != C::kSH) return false;
    if (!offsets_fit(s, C::kFused)) return false;
    if (C::kDMA && s.R % C::kKT) return false;
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
struct KernelOf;
template <int HT, int NB, int WH, int KT, int KH, int SH, bool F, int W, bool V, bool D>
struct KernelOf<BF16Cfg<HT, NB, WH, KT, KH, SH, F, W, V, D>> {
    static constexpr auto fn = slab_gemm_bf16_kernel<BF16Cfg<HT, NB, WH, KT, KH, SH, F, W, V, D>>;
    static constexpr int threads = 64 * W;
};
template <int HT, int NB, int WH, int KT, int KH, int SH, int VA, int VB, bool F, int W, bool D>
struct KernelOf<F32Cfg<HT, NB, WH, KT, KH, SH, VA, VB, F, W, D>> {
    static constexpr auto fn = slab_gemm_f32_kernel<F32Cfg<HT, NB, WH, KT, KH, SH, VA, VB, F, W, D>>;
    static constexpr int threads = 64 * W;
};

// Output layout fields and the 16-byte store test: dense n-h-w-c unless a
// layout is given (fp32 kernels only).
inline void set_layout(FixedParams& p, const Shape& s, float* O, const OutLayout* layout) {
    if (layout) {
        p.o_img = layout->img;
        p.o_row = layout->row;
        p.o_col = layout->col;
        p.o_off = layout->off;
    } else {
        p.o_img = s.o_h * s.o_w * s.k_c;
        p.o_row = s.o_w * s.k_c;
        p.o_col = s.k_c;
        p.o_off = 0;
    }
    p.o_vec = s.k_c % 4 == 0 && ((uintptr_t)O & 15u) == 0 &&
              ((p.o_img | p.o_row | p.o_col | p.o_off) & 3) == 0;
}

// The rows of L a product reads, when they are not L's own rows: row x of
// pair q starts at q * pstride + x * xstride (the flat windows below).
struct RowView {
    int64_t xstride, pstride;
};

template <class C>
hipError_t run_fixed(const Shape& s, const void* A, const void* K, float* O, hipStream_t stream,
                     int ksplit = 1, const OutLayout* layout = nullptr, const RowView* view = nullptr) {
    if (layout) ksplit = 1;  // the zeroing would clear other parts of a strided O
    FixedParams p{};
    p.A = A;
    p.K = K;
    p.O = O;
    p.i_h = s.i_h; p.i_w = s.i_w; p.i_c = s.i_c; p.k_c = s.k_c; p.s_w = s.s_w;
    p.o_h = s.o_h; p.o_w = s.o_w; p.R = s.R; p.pairs = s.pairs;
    p.a_xstride = view ? view->xstride : C::kFused ? s.i_w * s.i_c : s.R;
    p.a_pstride = view ? view->pstride : s.i_h * s.R;
    p.nchunks = (int32_t)((s.R + C::kKT - 1) / C::kKT);
    const int64_t pair_tiles = (s.pairs + kPairs - 1) / kPairs;
    p.h_tiles = (int32_t)((s.o_h + C::kHT - 1) / C::kHT);
    p.n_tiles = (int32_t)((s.k_c + C::NT - 1) / C::NT);
    const int64_t ntiles = pair_tiles * p.h_tiles * p.n_tiles * ksplit;
    if (ntiles > 0x7fffffff) return hipErrorInvalidValue;
    p.ntiles = (uint32_t)ntiles;
    p.ksplit = ksplit;
    set_layout(p, s, O, layout);
    if (ksplit > 1) {
        const int64_t n = s.i_n * s.o_h * s.o_w * s.k_c;
        hipLaunchKernelGGL(zero_o_kernel, dim3((uint32_t)((n + 1023) / 1024)), dim3(256), 0, stream, O, n);
    }
    hipLaunchKernelGGL(KernelOf<C>::fn, dim3(p.ntiles), dim3(KernelOf<C>::threads), 0, stream, p);
    return hipGetLastError();
}

template <class C>
bool stream_usable(const Shape& s, const void* A, const void* K) {
    return usable<C>(s, A, K) && s.R <= C::kKT && s.pairs < (int64_t(1) << 31);
}

template <class C>
hipError_t run_stream(const Shape& s, const void* A, const void* K, float* O, hipStream_t stream,
                      const OutLayout* layout = nullptr) {
    FixedParams p{};
    p.A = A;
    p.K = K;
    p.O = O;
    p.i_h = s.i_h; p.i_w = s.i_w; p.i_c = s.i_c; p.k_c = s.k_c; p.s_w = s.s_w;
    p.o_h = s.o_h; p.o_w = s.o_w; p.R = s.R; p.pairs = s.pairs;
    p.a_xstride = C::kFused ? s.i_w * s.i_c : s.R;
    p.a_pstride = s.i_h * s.R;
    p.nchunks = 1;
    const int64_t pair_tiles = (s.pairs + kPairs - 1) / kPairs;
    p.h_tiles = (int32_t)((s.o_h + C::kHT - 1) / C::kHT);
    p.n_tiles = (int32_t)((s.k_c + C::NT - 1) / C::NT);
    const int64_t ntiles = pair_tiles * p.h_tiles * p.n_tiles;
    if (ntiles > 0x7fffffff) return hipErrorInvalidValue;
    p.ntiles = (uint32_t)ntiles;
    p.pair_tiles = (int32_t)pair_tiles;
    p.band = (int32_t)std::min<int64_t>(pair_tiles, (s.o_w + kPairs - 1) / kPairs);
    set_layout(p, s, O, layout);
    p.div_ow = FastDiv((uint32_t)s.o_w);
    // persistent grid: the workgroups every compute unit of the stream's device
    // holds at once (LDS and registers), a multiple of 8
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, slab_gemm_f32_stream_kernel<C>,
                                                     C::THREADS, 0) != hipSuccess || per_cu < 1)
        per_cu = 1;
    int dev = 0, cus = 0;
    if (hipStreamGetDevice(stream, &dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 1;
    int64_t grid = (int64_t)per_cu * cus / 8 * 8;
    if (grid < 8) grid = 8;
    if (grid > ntiles) grid = ntiles;
    hipLaunchKernelGGL(slab_gemm_f32_stream_kernel<C>, dim3((uint32_t)grid), dim3(C::THREADS), 0, stream,
                       p);
    return hipGetLastError();
}

// fp32, 3x3 stride 1, rows of at most 10 elements (3x3 kernels over 3 channels):
// the streaming kernel, 32 pairs x 8 rows x 64 channels, the whole reduction
// in one stage.
template <bool F> using F32K3S1Stream = F32Cfg<8, 2, 4, 10, 3, 1, 1, 4, F>;
template <bool F> using F32K3S1StreamScalar = F32Cfg<8, 2, 4, 10, 3, 1, 1, 1, F>;

// fp32, 3x3 stride 1, long rows (R % 4 == 0): 32 pairs x 14 rows x 64 channels,
// r-chunks of 16, 16-byte loads of L (or I) and K.
template <bool F> using F32K3S1Wide = F32Cfg<14, 2, 2, 16, 3, 1, 4, 4, F>;
// The same tile staged by direct-to-LDS loads (rows of a multiple of 16).
template <bool F> using F32K3S1WideD = F32Cfg<14, 2, 2, 16, 3, 1, 4, 4, F, 4, true>;
// the same with 4 and 2 output rows per tile, for layers whose few pair tiles
// and small o_h would leave most compute units idle with 14-row tiles
template <bool F> using F32K3S1Wide4 = F32Cfg<4, 2, 2, 16, 3, 1, 4, 4, F>;
template <bool F> using F32K3S1Wide2 = F32Cfg<2, 2, 2, 16, 3, 1, 4, 4, F>;
template <bool F> using F32K3S1Wide4D = F32Cfg<4, 2, 2, 16, 3, 1, 4, 4, F, 4, true>;
template <bool F> using F32K3S1Wide2D = F32Cfg<2, 2, 2, 16, 3, 1, 4, 4, F, 4, true>;
// 2-row tiles with r-chunks of 32 where there is at most one workgroup per
// compute unit: twice the MFMAs per global-load round trip (one wave per SIMD
// by registers, so only where no second tile would share the compute unit;
// cv12 3%, the batch-1 Table 3 layers 6% faster, layers with more tiles slower).
template <bool F> using F32K3S1Wide2L = F32Cfg<2, 2, 2, 32, 3, 1, 4, 4, F>;
// fp32, 3x3 stride 1, short rows (R = 3 i_c with i_c not a multiple of 4).
template <bool F> using F32K3S1Narrow = F32Cfg<8, 2, 4, 2, 3, 1, 1, 4, F>;
template <bool F> using F32K3S1NarrowScalar = F32Cfg<8, 2, 4, 2, 3, 1, 1, 1, F>;
// fp32, 11x11 stride 4, 96-channel tiles. From L: 32 pairs x 4 rows (23 staged
// rows), r-chunks of 4. From I: 8 waves, 32 pairs x 8 rows (39 staged rows),
// r-chunks of 2. VB = 4 loads K four channels at a time (k_c % 4 == 0).
template <bool F, int VB>
using F32K11S4 = typename std::conditional<F, F32Cfg<8, 3, 8, 2, 11, 4, 1, VB, true, 8>,
                                           F32Cfg<4, 3, 4, 4, 11, 4, 1, VB, false>>::type;
// fp32, 7x7 stride 2: 32 pairs x 8 rows (21 staged rows) x 64 channels.
// fp32, 3x3 stride 2 (the downsampling layers of residual networks): 32 pairs x
// 2 rows (5 staged rows) x 64 channels. Measured at batch 32 against 4, 6 and 8
// rows: 2 rows the fastest on every shape (e.g. 15x15x512 -> 512: 122 us, 4 rows
// 290 us), and faster than the generic kernel from I by 3.5-11x and than the
// flat windows from L by 1.0-3.2x.
template <bool F> using F32K3S2Wide = F32Cfg<2, 2, 2, 16, 3, 2, 4, 4, F>;
template <bool F> using F32K3S2Narrow = F32Cfg<2, 2, 2, 4, 3, 2, 1, 4, F>;
template <bool F> using F32K3S2Scalar = F32Cfg<2, 2, 2, 4, 3, 2, 1, 1, F>;
template <bool F> using F32K7S2Wide = F32Cfg<8, 2, 2, 8, 7, 2, 4, 4, F>;
// the same with 4 and 2 output rows, where 8-row tiles leave the chip idle
// or rows 4 at a time run faster (chosen in dispatch_fixed)
template <bool F> using F32K7S2Wide4 = F32Cfg<4, 2, 2, 8, 7, 2, 4, 4, F>;
template <bool F> using F32K7S2Wide2 = F32Cfg<2, 2, 2, 8, 7, 2, 4, 4, F>;
template <bool F> using F32K7S2Narrow = F32Cfg<8, 2, 4, 4, 7, 2, 1, 4, F>;
template <bool F> using F32K7S2Scalar = F32Cfg<8, 2, 4, 4, 7, 2, 1, 1, F>;
// fp32, 2x2 and 4x4 (any k_w) stride 1, 16-byte rows: 32 pairs x 8 rows x 64
// channels (the sub-pixel phases of stride-2 input gradients: 3x3 -> 2x2,
// 7x7 -> 4x4 and 3x3 kernels).
template <bool F> using F32K2S1Wide = F32Cfg<8, 2, 2, 16, 2, 1, 4, 4, F>;
template <bool F> using F32K4S1Wide = F32Cfg<8, 2, 2, 16, 4, 1, 4, 4, F>;
// fp32, 5x5 stride 1: 32 pairs x 4 rows (8 staged rows) x 64 channels.
template <bool F> using F32K5S1Wide = F32Cfg<4, 2, 2, 16, 5, 1, 4, 4, F>;
// direct-to-LDS staging: 2.4% faster from I on cv5, 1% slower from L
template <bool F> using F32K5S1WideD = F32Cfg<4, 2, 2, 16, 5, 1, 4, 4, F, 4, true>;
// 2 output rows, where 4-row tiles leave the chip idle (chosen in dispatch_fixed)
template <bool F> using F32K5S1Wide2 = F32Cfg<2, 2, 2, 16, 5, 1, 4, 4, F>;
template <bool F> using F32K5S1Wide2D = F32Cfg<2, 2, 2, 16, 5, 1, 4, 4, F, 4, true>;
template <bool F> using F32K5S1Narrow = F32Cfg<4, 2, 2, 4, 5, 1, 1, 4, F>;
template <bool F> using F32K5S1Scalar = F32Cfg<4, 2, 2, 4, 5, 1, 1, 1, F>;
// k_h = 1, stride 1: plain products with no slab overlap (1x1 convolutions,
// and the im2col baseline's product). 32 pairs x 8 rows x 64 channels, or
// 96 channels for the short-row form when k_c > 64; bf16: 7 rows x 256
// channels.
template <bool F> using F32K1S1Wide = F32Cfg<8, 2, 2, 16, 1, 1, 4, 4, F>;
template <bool F> using F32K1S1Narrow = F32Cfg<8, 2, 2, 4, 1, 1, 1, 4, F>;
template <bool F> using F32K1S1Narrow96 = F32Cfg<8, 3, 4, 8, 1, 1, 1, 4, F>;
template <bool F> using F32K1S1Scalar = F32Cfg<8, 2, 2, 4, 1, 1, 1, 1, F>;
template <bool F> using BF16K1S1 = BF16Cfg<7, 8, 1, 32, 1, 1, F, 8>;
// bf16, 3x3 stride 1: 8 waves, 32 pairs x 14 rows x 128 channels, r-chunks of 32.
template <bool F> using BF16K3S1 = BF16Cfg<14, 4, 2, 32, 3, 1, F, 8>;
// The same tile staged by direct-to-LDS loads (rows of a multiple of 32).
template <bool F> using BF16K3S1D = BF16Cfg<14, 4, 2, 32, 3, 1, F, 8, true, true>;
template <bool F> using BF16K3S1R4 = BF16Cfg<4, 4, 2, 32, 3, 1, F, 8>;
template <bool F> using BF16K3S1R2 = BF16Cfg<2, 4, 2, 32, 3, 1, F, 8>;
template <bool F> using BF16K3S1R2D = BF16Cfg<2, 4, 2, 32, 3, 1, F, 8, true, true>;
// bf16, 5x5 stride 1 (8 staged rows, r-chunks of 32) and 7x7 stride 2 (13
// staged rows, r-chunks of 16): 32 pairs x 4 rows x 128 channels.
template <bool F> using BF16K5S1 = BF16Cfg<4, 4, 2, 32, 5, 1, F, 8>;
template <bool F> using BF16K5S1D = BF16Cfg<4, 4, 2, 32, 5, 1, F, 8, true, true>;
template <bool F> using BF16K7S2 = BF16Cfg<4, 4, 2, 16, 7, 2, F, 8>;
// at most 64 output channels: 2 rows x 64 channels, 4 waves (224x224x64 -> 64,
// from L / fused, against the 128-channel tile: batch 1 45 / 44 -> 34 / 33 us,
// batch 4 95 / 84 -> 75 / 68 us, batch 32 557 / 513 -> 453 / 421 us)
template <bool F> using BF16K7S2N64 = BF16Cfg<2, 2, 2, 16, 7, 2, F, 4>;
// bf16, 11x11 stride 4 over few channels (rows of 33 elements, gathered element
// by element): 32 pairs x 2 rows (15 staged rows) x 96 channels, r-chunks of 16.
template <bool F> using BF16K11S4 = BF16Cfg<2, 3, 2, 16, 11, 4, F, 6, false>;
// bf16 flat windows (from L, one row per window; see dispatch_fixed): 32 pairs x
// 8 windows x 96 or 128 channels, r-chunks of 32, windows gathered element by
// element or, when their length and both strides are multiples of 8, in
// 16-byte pieces.
using BF16FlatG96 = BF16Cfg<8, 3, 2, 32, 1, 1, false, 6, false>;
using BF16FlatG128 = BF16Cfg<8, 4, 2, 32, 1, 1, false, 8, false>;
using BF16FlatV128 = BF16Cfg<8, 4, 2, 32, 1, 1, false, 8, true>;

// Of tiles that differ only in their number of output rows, the one that
// minimises (rounds of tiles over the 256 compute units) x (input rows each
// tile stages): fewer, taller tiles stage the overlap rows less often; more,
// shorter tiles keep every compute unit busy on small layers.
int pick_rows(const Shape& s, int nt, std::initializer_list<int> rows) {
    int best = 0;
    int64_t best_cost = 0;
    for (int ht : rows) {
        const int64_t tiles = ((s.pairs + kPairs - 1) / kPairs) * ((s.o_h + ht - 1) / ht) *
                              ((s.k_c + nt - 1) / nt);
        const int64_t cost = ((tiles + 255) / 256) * ((ht - 1) * s.s_h + s.k_h);
        if (best == 0 || cost < best_cost) {
            best = ht;
            best_cost = cost;
        }
    }
    return best;
}

// bf16 3x3 tiles: split a tile's r-chunks between two workgroups only where
// that shortens the busiest compute unit's chunk count (counted at one
// workgroup per compute unit), the tiles are 2-row tiles at most two per
// compute unit unsplit, and each half keeps at least 4 chunks (the small deep
// layers, e.g. cv12: 60 tiles of 48 chunks on 256 compute units). Measured
// on the register-staged tiles; the direct-to-LDS ones add a bound on the
// output size at the call.
bool split_shortens(const Shape& s, int ht, int nt, int kt) {
    const int64_t nchunks = (s.R + kt - 1) / kt;
    if (nchunks < 8) return false;
    const int64_t tiles = ((s.pairs + kPairs - 1) / kPairs) * ((s.o_h + ht - 1) / ht) * ((s.k_c + nt - 1) / nt);
    if (ht != 2 || tiles > 512) return false;  // measured on 2-row tiles only
    return ((2 * tiles + 255) / 256) * ((nchunks + 1) / 2) < ((tiles + 255) / 256) * nchunks;
}

// fp32 3x3 stride 1: rows per tile (14, 4 or 2, the Wide, Wide4 and Wide2
// configurations) and whether to split each tile's r-chunks between two
// workgroups, by a cost model measured on this GPU: a tile's time is
// nchunks x (t1 + (c - 1) * 1.31 * mfma) when c tiles share a compute unit,
// with t1 = per-chunk overhead + MFMA cycles of one wave per chunk (overheads
// 4600, 2300 and 1500 cycles; MFMA 1536 cycles per output row of a wave), and
// at most w = 1, 3, 4 tiles resident per compute unit (LDS). Tiles beyond w
// per compute unit run in further rounds. A split tile is two workgroups of
// half the r-chunks each, plus zeroing O and adding both halves into it
// (costed as a 4 us launch and three passes over O at 5 TB/s). On ResNet/VGG layers of Table 2
// the unsplit choice is the fastest of the three row counts in every case
// measured (e.g. cv10 2 rows, 21% faster than 4; cv9 4 rows, 13% faster than
// 14; resnet_mid 14). A split is only considered where it shortens the
// busiest compute unit's chunk count, for 2-row tiles at most two per compute
// unit unsplit: layers whose tiles leave compute units idle (cv11 12%, cv12
// 38% faster; the batch-1 layers). The model was measured on the
// register-staged tiles; their direct-to-LDS forms (R % 16 == 0) are faster
// at each of its choices measured and take them over unchanged.
struct TileChoice {
    int ht, ksplit;
};
TileChoice pick_tiles_f32_3x3(const Shape& s, bool allow_split) {
    struct Opt { int ht, w; double ovh; };
    const Opt opts[3] = {{14, 1, 4600.0}, {4, 3, 2300.0}, {2, 4, 1500.0}};
    const int64_t nchunks = (s.R + 15) / 16;
    const double o_bytes = 4.0 * (double)(s.i_n * s.o_h * s.o_w * s.k_c);
    TileChoice best{14, 1};
    double best_t = 0.0;
    for (int split = 1; split <= 2; ++split) {
        if (split == 2 && (nchunks < 4 || !allow_split)) break;
        const int64_t nch = (nchunks + split - 1) / split;
        for (const Opt& o : opts) {
            const int64_t tiles1 = ((s.pairs + kPairs - 1) / kPairs) * ((s.o_h + o.ht - 1) / o.ht) *
                                   ((s.k_c + 63) / 64);
            const int64_t tiles = tiles1 * split;
            const double mfma = 1536.0 * (o.ht / 2);
            const int64_t per_cu = (tiles + 255) / 256;
            // split only where it shortens the busiest compute unit's r-chunks
            // and the unsplit tiles are at most two per compute unit; otherwise
            // it mostly multiplies the tiles sharing each one (measured slower
            // than the model says: cv6 122 -> 144 us; the input-gradient
            // convolution of cv10, 784 tiles, 113 -> 176 us)
            // (and on 2-row tiles only: split 14-row tiles measured far off the
            // model, cv10's input gradient 156 us against ~104 unsplit)
            const int64_t per_cu1 = (tiles1 + 255) / 256;
            if (split == 2 && (o.ht != 2 || per_cu1 > 2 || per_cu * nch >= per_cu1 * nchunks))
                continue;
            // split: the zeroing launch (~4 us) and three passes over O
            double t = split == 1 ? 0.0 : 9600.0 + 3.0 * o_bytes / 5.0e12 * 2.4e9;
            for (int64_t done = 0; done < per_cu; done += o.w) {
                const int64_t c = per_cu - done < o.w ? per_cu - done : o.w;
                t += (double)nch * (o.ovh + mfma + (double)(c - 1) * 1.31 * mfma);
            }
            if (best_t == 0.0 || t < best_t) {
                best = {o.ht, split};
                best_t = t;
            }
        }
    }
    return best;
}

// Section 3.2's flat view of L: the slab of output row h of pair (n, w) is the
// window L[n, w][s_h*R*h : s_h*R*h + k_h*R]. flat_windows gives the one-row
// product over those windows (row x of a pair = output row x, reduction over
// k_h*R), flat_view where its rows lie in L.
Shape flat_windows(const Shape& s) {
    Shape f = s;
    f.k_h = f.k_w = 1;
    f.s_h = f.s_w = 1;
    f.i_c = f.R = s.k_h * s.R;
    f.i_h = s.o_h;  // one row x per output row
    return f;
}
RowView flat_view(const Shape& s) { return RowView{s.s_h * s.R, s.i_h * s.R}; }

template <bool F>
hipError_t dispatch_fixed(const Shape& s, const void* A, const void* K, float* O, int dtype,
                          hipStream_t stream, bool dry_run, const OutLayout* layout) {
#define MEC_TRY_FIXED(CFG)                                                          \
    if (usable<CFG>(s, A, K)) {                                                     \
        return dry_run ? hipSuccess : run_fixed<CFG>(s, A, K, O, stream, 1, layout); \
    }
#define MEC_TRY_FIXED_SPLIT(CFG, KSPLIT)                                                  \
    if (usable<CFG>(s, A, K)) {                                                           \
        return dry_run ? hipSuccess : run_fixed<CFG>(s, A, K, O, stream, KSPLIT, layout); \
    }
#define MEC_TRY_STREAM(CFG)                                                         \
    if (stream_usable<CFG>(s, A, K)) {                                              \
        return dry_run ? hipSuccess : run_stream<CFG>(s, A, K, O, stream, layout);  \
    }
    if (dtype == 0) {
        // tall kernels over short rows of L (11x11 over 3 channels: 33 elements):
        // the flat windows through a ring of LDS (mec_gemm_ring.hip), where the
        // ring holds four output rows' windows (strides up to 4 for 11x11).
        // Measured at batch 32 against the tiles, from L / fused: cv1 stride 3
        // 207 -> 141 us; 7x7 stride 2 over 3 channels (cv3) 101 / 93 -> 86 us;
        // 5x5 stride 2 over 3 channels 24 / 30 -> 18 us, over 6 channels 28 /
        // 28 -> 21 us; fused, rows of at most 10 elements, 3x3 over 3 channels
        // (vgg_first, cv7) 51 -> 46 us and 93 -> 83 us. From L the ring takes
        // only windows of at most two blocks (K held in registers, fills five
        // blocks ahead): with L read from HBM, vgg_first 59 -> 54 us and cv7
        // 116 -> 99 us against the streaming kernel, which keeps the longer
        // windows (the ring read those more slowly). At stride 1 with longer
        // rows it is even or slower (3x3 over 16 channels 92 / 81 -> 92 / 89
        // us, 5x5 over 8 channels even): those keep the tiles.
        if (!layout &&
            (s.k_h >= 9 || (s.k_h >= 5 && s.s_h >= 2) || (s.k_h >= 3 && s.R <= 10 && (F || gemm_ring_short(s)))) &&
            s.R <= 48 && gemm_ring_usable(s, dtype))
            return dry_run ? hipSuccess : launch_gemm_ring(s, A, K, O, F, stream);
        if (s.R >= 32) {
            // no split into a strided layout: zeroing O would clear other pixels
            const TileChoice tc =
                s.k_h == 3 && s.s_h == 1 ? pick_tiles_f32_3x3(s, layout == nullptr) : TileChoice{14, 1};
            // the direct-to-LDS form of the chosen tile where R % 16 == 0 (faster
            // at every row count measured: cv9-cv12 and their input gradients)
            if (tc.ht == 2) {
                MEC_TRY_FIXED_SPLIT(F32K3S1Wide2D<F>, tc.ksplit);
                const int64_t wgs = ((s.pairs + kPairs - 1) / kPairs) * ((s.o_h + 1) / 2) *
                                    ((s.k_c + 63) / 64) * tc.ksplit;
                if (wgs <= 256) MEC_TRY_FIXED_SPLIT(F32K3S1Wide2L<F>, tc.ksplit);
                MEC_TRY_FIXED_SPLIT(F32K3S1Wide2<F>, tc.ksplit);
            }
            if (tc.ht == 4) {
                MEC_TRY_FIXED_SPLIT(F32K3S1Wide4D<F>, tc.ksplit);
                MEC_TRY_FIXED_SPLIT(F32K3S1Wide4<F>, tc.ksplit);
            }
            MEC_TRY_FIXED_SPLIT(F32K3S1WideD<F>, tc.ksplit);
            MEC_TRY_FIXED_SPLIT(F32K3S1Wide<F>, tc.ksplit);
        }
        MEC_TRY_STREAM(F32K3S1Stream<F>);
        MEC_TRY_STREAM(F32K3S1StreamScalar<F>);
        MEC_TRY_FIXED(F32K3S1Narrow<F>);
        MEC_TRY_FIXED(F32K3S1NarrowScalar<F>);
        MEC_TRY_FIXED(F32K3S2Wide<F>);
        MEC_TRY_FIXED(F32K3S2Narrow<F>);
        MEC_TRY_FIXED(F32K3S2Scalar<F>);
        if (s.k_h == 7 && s.s_h == 2) {
            // Rows per tile: 4 where that gives a tile per compute unit, else 2,
            // split between two workgroups where 2-row tiles still leave compute
            // units idle. Measured on 224x224x64 -> 64 (cv4's shape), 8 / 4 / 2
            // rows / 2 rows split, from L: batch 1 267 / 129 / 84 / 78 us,
            // batch 4 283 / 227 / 250 / 255 us, batch 32 1416 / 1338 / 1452 us.
            const int64_t ptiles = (s.pairs + kPairs - 1) / kPairs, ctiles = (s.k_c + 63) / 64;
            const int64_t t4 = ptiles * ((s.o_h + 3) / 4) * ctiles, t2 = ptiles * ((s.o_h + 1) / 2) * ctiles;
            if (t4 >= 256) {
                MEC_TRY_FIXED(F32K7S2Wide4<F>);
            } else {
                const bool split = t2 < 256 && !layout && s.pairs * s.o_h * s.k_c <= (int64_t(1) << 20);
                MEC_TRY_FIXED_SPLIT(F32K7S2Wide2<F>, split ? 2 : 1);
            }
        }
        MEC_TRY_FIXED(F32K7S2Wide<F>);
        MEC_TRY_FIXED(F32K7S2Narrow<F>);
        MEC_TRY_FIXED(F32K7S2Scalar<F>);
        if (s.k_h == 5 && s.s_h == 1) {
            // 2 rows per tile where 4-row tiles number fewer than the compute
            // units, split between two workgroups where even 2-row tiles fill
            // at most half of them. Measured on 24x24x96 -> 256 (cv5's shape),
            // from L / fused, 4 rows -> 2 rows -> 2 rows split: batch 1 94 / 79
            // -> 57 / 47 -> 35 / 29 us; batch 8 86 / 80 -> 56 / 47 (split 62 /
            // 56); batch 32 (400 4-row tiles) unchanged at 157 / 158 us.
            const int64_t ptiles = (s.pairs + kPairs - 1) / kPairs, ctiles = (s.k_c + 63) / 64;
            const int64_t t4 = ptiles * ((s.o_h + 3) / 4) * ctiles, t2 = ptiles * ((s.o_h + 1) / 2) * ctiles;
            if (t4 < 256) {
                const int ks =
                    2 * t2 <= 256 && !layout && s.pairs * s.o_h * s.k_c <= (int64_t(1) << 20) ? 2 : 1;
                if (F) MEC_TRY_FIXED_SPLIT(F32K5S1Wide2D<F>, ks);
                MEC_TRY_FIXED_SPLIT(F32K5S1Wide2<F>, ks);
            }
        }
        if (F) MEC_TRY_FIXED(F32K5S1WideD<F>);
        MEC_TRY_FIXED(F32K5S1Wide<F>);
        MEC_TRY_FIXED(F32K2S1Wide<F>);
        MEC_TRY_FIXED(F32K4S1Wide<F>);
        MEC_TRY_FIXED(F32K5S1Narrow<F>);
        MEC_TRY_FIXED(F32K5S1Scalar<F>);
        using K11V4 = F32K11S4<F, 4>;
        using K11V1 = F32K11S4<F, 1>;
        MEC_TRY_FIXED(K11V4);
        MEC_TRY_FIXED(K11V1);
        MEC_TRY_FIXED(F32K1S1Wide<F>);
        if (s.k_c > 64) MEC_TRY_FIXED(F32K1S1Narrow96<F>);
        MEC_TRY_FIXED(F32K1S1Narrow<F>);
        MEC_TRY_FIXED(F32K1S1Scalar<F>);
        // From L, every other kernel taller than one row (or one row at a stride
        // above 1): Section 3.2's flat view again. The slab of output row h of pair (n, w) is the contiguous window
        // L[n, w][s_h*R*h : s_h*R*h + k_h*R], so O is one plain product whose
        // rows (pair, h) are these windows, s_h*R elements apart, and whose
        // reduction runs over k_h*R elements with no per-kernel-row padding: the
        // k_h = 1 tiles with their rows read through that view. Consecutive
        // windows overlap by (k_h - s_h)*R elements, served by the L2 cache.
        // Against the generic slab kernel (mec_gemm.hip), batch 32: cv1 at
        // strides 1, 2, 5, 10 1284 -> 1063, 353 -> 281, 178 -> 96, 73 -> 57 us;
        // 3x3 stride 2 over 64 channels 183 -> 52 us; 5x5 stride 2 197 -> 70 us;
        // 7x7 stride 1 over 16 channels 153 -> 122 us.
        if (!F && !layout && (s.k_h > 1 || s.s_h > 1) && offsets_fit(s, false)) {
            const Shape f = flat_windows(s);
            const RowView view = flat_view(s);
#define MEC_TRY_FLAT(CFG)                                                                  \
    if (usable<CFG>(f, A, K) && (CFG::kVA == 1 || view.xstride % CFG::kVA == 0) &&         \
        (CFG::kVA == 1 || view.pstride % CFG::kVA == 0)) {                                 \
        return dry_run ? hipSuccess : run_fixed<CFG>(f, A, K, O, stream, 1, nullptr, &view); \
    }
            MEC_TRY_FLAT(F32K1S1Wide<false>);
            if (s.k_c > 64) MEC_TRY_FLAT(F32K1S1Narrow96<false>);
            MEC_TRY_FLAT(F32K1S1Narrow<false>);
            MEC_TRY_FLAT(F32K1S1Scalar<false>);
#undef MEC_TRY_FLAT
        }
    } else {
        if (layout) return hipErrorNotSupported;  // dense O only
        {
            // Whole r-chunks (R % 32 == 0): the direct-to-LDS tiles, 14 rows (one
            // workgroup per compute unit) where they occupy at least three
            // quarters of the 256 compute units, else 2 rows (two per compute
            // unit); the faster of the two on every 3x3 layer of Table 2 and on a
            // 14x14x512 layer at batch 256 (the rows-x-rounds model below picks 2
            // rows there, 1.7x slower than 14 with these kernels).
            const int64_t tiles14 = ((s.pairs + kPairs - 1) / kPairs) * ((s.o_h + 13) / 14) * ((s.k_c + 127) / 128);
            const bool dma = s.R % 32 == 0;
            const int ht = dma ? (tiles14 >= 192 ? 14 : 2)
                               : s.k_h == 3 && s.s_h == 1 ? pick_rows(s, 128, {14, 4, 2}) : 14;
            // With these tiles a split pays only on small outputs: adding the
            // halves into O costs ~24 us per million outputs (cv10 at batch 32,
            // 2.8M outputs: 20 -> 87 us split; cv12, 0.4M: 37 -> 33 us).
            const int64_t n_out = s.i_n * s.o_h * s.o_w * s.k_c;
            const int ks = split_shortens(s, ht, 128, 32) && (!dma || n_out <= (int64_t(1) << 20)) ? 2 : 1;
            if (ht == 2) MEC_TRY_FIXED_SPLIT(BF16K3S1R2D<F>, ks);
            if (ht == 2) MEC_TRY_FIXED_SPLIT(BF16K3S1R2<F>, ks);
            if (ht == 4) MEC_TRY_FIXED_SPLIT(BF16K3S1R4<F>, ks);
            MEC_TRY_FIXED_SPLIT(BF16K3S1D<F>, ks);
            MEC_TRY_FIXED_SPLIT(BF16K3S1<F>, ks);
        }
        MEC_TRY_FIXED(BF16K5S1D<F>);
        MEC_TRY_FIXED(BF16K5S1<F>);
        if (s.k_c <= 64) MEC_TRY_FIXED(BF16K7S2N64<F>);
        MEC_TRY_FIXED(BF16K7S2<F>);
        MEC_TRY_FIXED(BF16K11S4<F>);
        MEC_TRY_FIXED(BF16K1S1<F>);
        // From L, the flat windows (as for fp32 above) where consecutive windows
        // overlap most (k_h >= 5 s_h) and no tile of its own fits: cv1 in bf16
        // at stride 1 2473 -> 1213 us, stride 2 476 -> 325 us against the
        // generic kernel; at stride 5 (118 against 113 us) and on 7x7 stride 2
        // over 3 channels (170 against 110 us) the element-by-element gathering
        // of bf16 windows loses.
        if (!F && s.k_h > 1 && s.k_h >= 5 * s.s_h && offsets_fit(s, false)) {
            const Shape f = flat_windows(s);
            const RowView view = flat_view(s);
            const bool vec = f.R % 8 == 0 && view.xstride % 8 == 0 && view.pstride % 8 == 0;
            if (s.k_c <= 96 && usable<BF16FlatG96>(f, A, K))
                return dry_run ? hipSuccess : run_fixed<BF16FlatG96>(f, A, K, O, stream, 1, nullptr, &view);
            if (vec && usable<BF16FlatV128>(f, A, K))
                return dry_run ? hipSuccess : run_fixed<BF16FlatV128>(f, A, K, O, stream, 1, nullptr, &view);
            if (usable<BF16FlatG128>(f, A, K))
                return dry_run ? hipSuccess : run_fixed<BF16FlatG128>(f, A, K, O, stream, 1, nullptr, &view);
        }
    }
#undef MEC_TRY_FIXED
#undef MEC_TRY_STREAM
#undef MEC_TRY_FIXED_SPLIT
    return hipErrorNotSupported;
}

}  // namespace

hipError_t launch_gemm_fixed(const Shape& s, const void* A, const void* K, float* O, int dtype,
                             bool fused, hipStream_t stream, bool dry_run, const OutLayout* layout) {
    if (fused) return dispatch_fixed<true>(s, A, K, O, dtype, stream, dry_run, layout);
    return dispatch_fixed<false>(s, A, K, O, dtype, stream, dry_run, layout);
}

}  // namespace mec
