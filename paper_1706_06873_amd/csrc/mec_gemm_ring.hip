// MEC's slab products (Section 3.3, Algorithm 2, product phase) for kernels
// over few channels (fp32): the tall, strided 11x11 first layers of Table 2
// (cv1 and cv2, at strides 3 and 4), 5x5 or 7x7 kernels at stride 2 such as
// cv3, and, from I, 3x3 kernels over 3 channels (vgg_first, cv7). A row of L
// is short there (R = k_w*i_c = 33 for 11x11 over 3 channels) and the slab of
// one output row, k_h*R = 363 elements for that layer, spans many of them.
//
// Section 3.2 views output row h of pair (n, w) as one dot product over a
// contiguous window of that pair's row of L:
//   O[n, h, w, :] = sum_{j < k_h*R} L[n, w][s_h*R*h + j] * K[j, :]
// with K viewed as a (k_h*k_w*i_c) x k_c matrix. Consecutive output rows'
// windows start s_h*R elements apart and overlap by (k_h - s_h)*R.
//
// This kernel takes that flat view literally. One wave is one workgroup. Its
// 32x32 MFMA block has as rows 8 pairs x 4 consecutive output rows, so all 32
// rows reduce over the same index j at every step and share one fragment of
// K (read from global memory, where every wave finds it in the L2 cache). The
// reduction runs over the window's k_h*R elements in steps of 2 (one
// v_mfma_f32_32x32x2_f32), padded with zeros to whole blocks of 7 or 8 steps
// (363 -> 364): no per-row padding of R to a staging width. The wave streams
// its 8 pairs' rows of L (or, fused, the same elements of I) through a ring in
// LDS, 512 elements per pair, filled 64 elements at a time by direct-to-LDS
// loads one block of k-steps ahead of use, or, where the window takes at most
// two blocks (3x3 over 1 to 3 channels: K then stays in registers for the
// whole item), five blocks ahead with waits counted per block. Every element
// of the rows it covers is loaded once per item, the overlap between output
// rows is read from the ring. Waves share nothing, so there is no barrier:
// several waves per SIMD hide each other's load latency.
#include "mec_mfma.h"

namespace mec {
namespace {

constexpr int kRPairs = 8;                 // pairs per wave tile
constexpr int kRRows = 4;                  // output rows per wave tile: 8 x 4 = 32 MFMA rows
constexpr int kChunk = 64;                 // elements per fill: one dword per lane
constexpr int kRingChunks = 8;             // ring capacity in chunks
constexpr int kRingLen = kChunk * kRingChunks;
// floats between pairs' rings: 8 x 636 x 4 B = 19.9 KB per wave, so eight
// waves fit a compute unit, two per SIMD (16.5 KB would fit nine, three on one
// SIMD and two on the others: measured 1.5% slower); 636 = -4 mod 64 banks, so
// a fragment read of 8 pairs x 4 rows spreads over the banks
constexpr int kRingLD = kRingLen + 124;
// k-steps between fill points (BS): 8, or 7 where that pads the reduction less
// (the window's ceil(k_h*R / 2) steps are rounded up to whole blocks)
constexpr int kWavesPerCU = 8;             // resident waves per compute unit (LDS: 8 rings)
constexpr uint32_t kStoreDrop = 0x80000000u;  // O byte offsets from here on are out of range
constexpr int kStoreNT = 2;                // cache policy of the O stores: non-temporal

struct RingParams {
    const float* A;   // L (lowered) or I (fused)
    const float* K;   // (k_h*k_w*i_c) x k_c
    float* O;
    int64_t pairs, o_w, o_h, k_c;
    int64_t rowlen;          // i_h * R: elements of one pair's row of L
    int64_t img_stride;      // fused: i_h * i_w * i_c
    int64_t x_stride;        // fused: i_w * i_c (next input row); lowered: R
    int64_t w_stride;        // fused: s_w * i_c; lowered: i_h * R (next pair)
    int32_t R, KR, nks, srow;  // KR = k_h*R; nks = ceil(KR / 2) rounded up to a whole block of
                               // k-steps (the steps past KR multiply zeros); srow = s_h*R
    int32_t ngroups;         // ceil(o_h / 4)
    int32_t gpi;             // row groups per item
    int32_t items_pg;        // items per pair group: ceil(ngroups / gpi)
    int32_t n_tiles;         // channel tiles of 32*NB
    uint32_t nfull;          // whole items: (pair group, items_pg) x n_tiles, or fewer (below)
    FastDiv divR;
    FastDiv div_ow;          // pair -> (image, column); pairs < 2^31
};

// One chunk of the ring for all 8 pairs: for each pair q, one dword per lane
// from base + voff[q] (bytes) straight into LDS at lds[q] + 4*lane. M0 holds
// the LDS address of each load; its previous value is saved once and put back
// once (M0 cannot be declared clobbered; saving it around every load cost 14
// scalar instructions per chunk, 1-1.7% of alexnet_conv1's and cv3's products).
// The caller waits (s_waitcnt lgkmcnt(0)) first: every LDS read issued earlier
// has returned before a slot can be overwritten.
__device__ inline void ring_dma8(const float* base, const uint32_t (&voff)[kRPairs], const uint32_t (&lds)[kRPairs]) {
    static_assert(kRPairs == 8, "one load per pair");
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %9\n\ts_nop 0\n\tglobal_load_lds_dword %1, %17\n\t"
        "s_mov_b32 m0, %10\n\ts_nop 0\n\tglobal_load_lds_dword %2, %17\n\t"
        "s_mov_b32 m0, %11\n\ts_nop 0\n\tglobal_load_lds_dword %3, %17\n\t"
        "s_mov_b32 m0, %12\n\ts_nop 0\n\tglobal_load_lds_dword %4, %17\n\t"
        "s_mov_b32 m0, %13\n\ts_nop 0\n\tglobal_load_lds_dword %5, %17\n\t"
        "s_mov_b32 m0, %14\n\ts_nop 0\n\tglobal_load_lds_dword %6, %17\n\t"
        "s_mov_b32 m0, %15\n\ts_nop 0\n\tglobal_load_lds_dword %7, %17\n\t"
        "s_mov_b32 m0, %16\n\ts_nop 0\n\tglobal_load_lds_dword %8, %17\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(voff[0]), "v"(voff[1]), "v"(voff[2]), "v"(voff[3]), "v"(voff[4]), "v"(voff[5]), "v"(voff[6]),
          "v"(voff[7]), "s"(lds[0]), "s"(lds[1]), "s"(lds[2]), "s"(lds[3]), "s"(lds[4]), "s"(lds[5]), "s"(lds[6]),
          "s"(lds[7]), "s"(base)
        : "memory");
}

// Waits until at most n vector memory operations of this wave are in flight
// (n >= 0, wave-uniform), rounded down to a multiple of 8 and at most 56: a
// stricter wait than asked, never a looser one. The counter retires loads,
// direct-to-LDS loads and stores in the order they were issued.
__device__ __forceinline__ void wait_vm_at_most(int n) {
    switch (n >> 3) {
    case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    case 1: asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
    case 2: asm volatile("s_waitcnt vmcnt(16)" ::: "memory"); break;
    case 3: asm volatile("s_waitcnt vmcnt(24)" ::: "memory"); break;
    case 4: asm volatile("s_waitcnt vmcnt(32)" ::: "memory"); break;
    case 5: asm volatile("s_waitcnt vmcnt(40)" ::: "memory"); break;
    case 6: asm volatile("s_waitcnt vmcnt(48)" ::: "memory"); break;
    default: asm volatile("s_waitcnt vmcnt(56)" ::: "memory"); break;
    }
}

// s_waitcnt vmcnt(0) as the instruction the compiler knows (expcnt and
// lgkmcnt fields at their maxima): its own wait analysis then sees the loads
// it issued before as complete.
constexpr int kWaitVm0 = 0x0F70;

// Short windows (at most two blocks of k-steps): blocks whose fills are
// issued this many blocks ahead of their reads.
constexpr int kShortLead = 5;

// One piece of work: row groups g_begin .. g_end-1 of the 8 pairs from pair0,
// channels n0 .. n0 + 32*NB.
template <int NB, bool FUSED, int BS, bool SHORT>
__device__ __forceinline__ void ring_item(const RingParams& p, float* ring, int64_t pair0, int g_begin,
                                          int g_end, int n0) {
    const int lane = threadIdx.x;
    const int m = lane & 31, kofs = lane >> 5;
    const int pp = m & 7, ii = m >> 3;  // this lane's A row: pair pp, output row ii

    // Source of each pair's row of L: element o of pair q's row is at
    // srcq[q] + (o / R) * x_stride + o % R (lowered: x_stride = R, so srcq[q] + o).
    // Offsets are relative to the first pair's source, in elements.
    int64_t src0;
    {
        const int64_t n = p.div_ow.div((uint32_t)pair0), w = pair0 - n * p.o_w;
        src0 = FUSED ? n * p.img_stride + w * p.w_stride : pair0 * p.rowlen;
    }
    const float* __restrict__ Abase = p.A + src0;
    uint32_t srcq[kRPairs];
#pragma unroll
    for (int q = 0; q < kRPairs; ++q) {
        int64_t pr = pair0 + q;
        if (pr >= p.pairs) pr = pair0;  // past the end: the first pair (never stored)
        const int64_t n = p.div_ow.div((uint32_t)pr), w = pr - n * p.o_w;
        const int64_t s = FUSED ? n * p.img_stride + w * p.w_stride : pr * p.rowlen;
        srcq[q] = (uint32_t)(s - src0);
    }
    const uint32_t ring_lds =
        (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(size_t)(__attribute__((address_space(3))) float*)ring);

    // O through a buffer resource based at the first pair's image. A lane's
    // byte offset for each (pair, channel block) it stores is fixed for the
    // item and the output row adds a scalar offset, so a group's stores are
    // one instruction each. Channels past k_c and pairs past the end get an
    // offset past the resource's range, whose check drops those stores.
    const int64_t img0 = p.div_ow.div((uint32_t)pair0);
    const int64_t obase = img0 * p.o_h * p.o_w * p.k_c;
    const int64_t orange = (p.pairs * p.o_h * p.k_c - obase) * 4;
    const __amdgpu_buffer_rsrc_t orsrc = __builtin_amdgcn_make_buffer_rsrc(
        p.O + obase, (short)0, (int)(orange < kStoreDrop - 1 ? orange : kStoreDrop - 1), 0x00020000);
    uint32_t ooff[4][NB];
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
        const int64_t pr = pair0 + kofs * 4 + q4;
        const int64_t n = p.div_ow.div((uint32_t)pr), w = pr - n * p.o_w;
        const int64_t rel = ((n - img0) * p.o_h * p.o_w + w) * p.k_c + n0 + m;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
            ooff[q4][nb] = pr < p.pairs && n0 + 32 * nb + m < p.k_c ? (uint32_t)((rel + 32 * nb) * 4) : kStoreDrop;
    }

    // Fill chunk c (elements [64c, 64c + 64) of every pair's row) into its ring
    // slot. Elements past the row's end repeat its last one: they only reach
    // output rows past o_h, which are never stored.
    auto fill = [&](int c) {
        int64_t o = (int64_t)c * kChunk + lane;
        if (o > p.rowlen - 1) o = p.rowlen - 1;
        uint32_t rel;
        if (FUSED) {
            const uint32_t x = p.divR.div((uint32_t)o);
            rel = x * (uint32_t)p.x_stride + ((uint32_t)o - x * (uint32_t)p.R);
        } else {
            rel = (uint32_t)o;
        }
        const uint32_t slot = ((uint32_t)c % kRingChunks) * kChunk;
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        uint32_t voff[kRPairs], lds[kRPairs];
#pragma unroll
        for (int q = 0; q < kRPairs; ++q) {
            voff[q] = 4u * (srcq[q] + rel);
            lds[q] = ring_lds + 4u * (uint32_t)(q * kRingLD) + 4u * slot;
        }
        ring_dma8(Abase, voff, lds);
    };
    int filled = -1;  // highest chunk issued (set at the item's start below)
    auto fill_upto = [&](int target) {
        for (int c = filled + 1; c <= target; ++c) fill(c);
        if (target > filled) filled = target;
    };
    // chunks read by block b of group g: [lo, hi] (the element offsets are
    // never negative: divided as unsigned, one shift each instead of the
    // signed division's four scalar instructions; with the ring slot's
    // unsigned remainder and K's 32-bit resource offset below, 1.5-2.5%
    // faster on alexnet_conv1, cv1 and cv3)
    const int rspan = (kRRows - 1) * p.srow;
    auto blk_lo = [&](int g, int b) { return (int)((uint32_t)(g * kRRows * p.srow + 2 * BS * b) / kChunk); };
    auto blk_hi = [&](int g, int b) {
        return (int)((uint32_t)(g * kRRows * p.srow + rspan + 2 * BS * b + 2 * BS - 1) / kChunk);
    };
    const int nblk = (p.nks + BS - 1) / BS;

    // K fragment of k-step t, channel block nb: K[2t + kofs][n0 + 32 nb + m],
    // by buffer loads whose range check returns 0 past K's last element: the
    // padding steps' rows j >= KR, and channels past k_c in the last row (the
    // columns past k_c are never stored). Each block's loads go through a
    // resource based at its first k-step, whose range ends at K's end, with a
    // fixed vector offset per lane and step (the channel block's is the
    // instruction's immediate): every offset stays in the vector operand that
    // the range check covers, and the loads need no vector temporaries.
    const uint32_t klane = (uint32_t)((kofs * (int)p.k_c + n0 + m) * 4);
    const uint32_t kstep = (uint32_t)(2 * p.k_c * 4);  // bytes per k-step
    const uint32_t kbytes = (uint32_t)(p.KR * p.k_c * 4);
    uint32_t kvoff[BS];
#pragma unroll
    for (int u = 0; u < BS; ++u) kvoff[u] = klane + (uint32_t)u * kstep;
    // K fragments of a whole block are loaded one block ahead, into the other
    // of two register sets; the stream of k-steps wraps at nks (every group
    // reduces over the same rows of K).
    float kb0[BS][NB], kb1[BS][NB];
    int kt = 0;  // first k-step (mod nks) of the next block of K fragments
    auto kload_block = [&](float (*dst)[NB]) {
        // kt <= nks - BS, whose first row 2 kt lies inside K (the
        // padding is less than one block), so the range is not empty
        const uint32_t kfirst = (uint32_t)kt * kstep;
        const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(
            reinterpret_cast<char*>(const_cast<float*>(p.K)) + kfirst, (short)0, (int)(kbytes - kfirst), 0x00020000);
#pragma unroll
        for (int u = 0; u < BS; ++u)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                dst[u][nb] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(kr, kvoff[u] + 128 * nb, 0, 0));
        kt = kt + BS == p.nks ? 0 : kt + BS;
        asm volatile("" ::: "memory");  // issued here, not sunk towards their use
    };
    kload_block(kb0);

    if constexpr (SHORT) {
        // A window of at most two blocks (nks <= 2 BS): kb0 holds block 0 and
        // kb1 block 1 (block 0 again when there is one) for the whole item, so
        // the loop issues no loads into registers, only fills and stores, and
        // its waits are counted: the fills of block beta's chunks go out
        // kShortLead blocks ahead, and block beta waits only for what was
        // issued up to the end of the oldest of the last kShortLead blocks
        // (or the item's start) by which its chunks had been issued; what was
        // issued after that may still be in flight. Where the ring could not
        // hold the chunks that far ahead, the lead is shorter (not on 3x3 or
        // 5x5 kernels over 1 to 3 channels at strides up to 2).
        kload_block(kb1);
        const int nbeta = (g_end - g_begin) * nblk;
        auto g_of = [&](int beta) { return g_begin + (nblk == 2 ? beta >> 1 : beta); };
        auto lo_b = [&](int beta) { return blk_lo(g_of(beta), nblk == 2 ? beta & 1 : 0); };
        auto hi_b = [&](int beta) { return blk_hi(g_of(beta), nblk == 2 ? beta & 1 : 0); };
        filled = lo_b(0) - 1;
        {
            const int want = hi_b(kShortLead - 1 < nbeta - 1 ? kShortLead - 1 : nbeta - 1);
            const int cap = lo_b(0) + kRingChunks - 1;
            fill_upto(want < cap ? want : cap);
        }
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        // mark[i]: the highest chunk issued by the end of block beta - kShortLead + i;
        // nops[i]: the operations that block issued (the item's start: before block 0)
        int mark[kShortLead], nops[kShortLead];
#pragma unroll
        for (int i = 0; i < kShortLead; ++i) {
            mark[i] = filled;
            nops[i] = 0;
        }
        floatx16 acc[NB];
        uint32_t ridx = 0;
        const uint32_t abase = (uint32_t)(pp * kRingLD);
        auto short_block = [&](int beta, float (*kuse)[NB]) {
            const int g = g_of(beta), b = nblk == 2 ? beta & 1 : 0;
            if (b == 0) {
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int v = 0; v < 16; ++v) acc[nb][v] = 0.f;
                ridx = (uint32_t)(g * kRRows * p.srow + ii * p.srow + kofs) & (kRingLen - 1);
            }
            const int before = filled;
            int ops = 0;
            // the oldest block of the history whose fills reach this block's
            // chunks: everything issued after it may stay in flight
            int n = -1, later = 0;
#pragma unroll
            for (int i = kShortLead - 1; i >= 0; --i) {
                if (hi_b(beta) <= mark[i]) n = later;
                later += nops[i];
            }
            if (n >= 0) {
                wait_vm_at_most(n);
            } else {  // not issued yet: the ring could not take it that far ahead
                fill_upto(hi_b(beta));
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            }
            {
                const int want = hi_b(beta + kShortLead < nbeta - 1 ? beta + kShortLead : nbeta - 1);
                const int cap = lo_b(beta) + kRingChunks - 1;
                fill_upto(want < cap ? want : cap);
            }
            ops += kRPairs * (filled - before);
            float a[BS];
#pragma unroll
            for (int u = 0; u < BS; ++u) a[u] = ring[abase + ((ridx + 2 * u) & (kRingLen - 1))];
            const int t = b * BS;
            if (2 * (t + BS) > p.KR) {
#pragma unroll
                for (int u = 0; u < BS; ++u)
                    if (2 * (t + u) + kofs >= p.KR) a[u] = 0.f;
            }
            ridx = (ridx + 2 * BS) & (kRingLen - 1);
#pragma unroll
            for (int u = 0; u < BS; ++u)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
                    acc[nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[u], kuse[u][nb], acc[nb], 0, 0, 0);
            if (b + 1 == nblk) {
#pragma unroll
                for (int r = 0; r < kRRows; ++r) {
                    const int64_t h = (int64_t)g * kRRows + r;
                    if (h >= p.o_h) break;
                    const int32_t soff = __builtin_amdgcn_readfirstlane((int32_t)(h * p.o_w * p.k_c * 4));
#pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4)
#pragma unroll
                        for (int nb = 0; nb < NB; ++nb) {
                            const float v = acc[nb][r * 4 + q4];
                            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), orsrc,
                                                                  (int32_t)ooff[q4][nb], soff, kStoreNT);
                        }
                    ops += 4 * NB;
                }
            }
#pragma unroll
            for (int i = 0; i + 1 < kShortLead; ++i) {
                mark[i] = mark[i + 1];
                nops[i] = nops[i + 1];
            }
            mark[kShortLead - 1] = filled;
            nops[kShortLead - 1] = ops;
        };
        for (int beta = 0; beta < nbeta; beta += 2) {
            short_block(beta, kb0);
            if (beta + 1 < nbeta) short_block(beta + 1, kb1);
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        return;
    }

    // first group: everything its first two blocks read
    filled = blk_lo(g_begin, 0) - 1;
    fill_upto(blk_hi(g_begin, nblk > 1 ? 1 : 0) < blk_lo(g_begin, 0) + kRingChunks - 1
                  ? blk_hi(g_begin, nblk > 1 ? 1 : 0)
                  : blk_lo(g_begin, 0) + kRingChunks - 1);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

    floatx16 acc[NB];
    uint32_t ridx = 0;
    const uint32_t abase = (uint32_t)(pp * kRingLD);
    // The item's blocks in one sequence: block beta is block b = beta % nblk of
    // group g = g_begin + beta / nblk. Even blocks multiply kb0 and load kb1,
    // odd ones the reverse (the loop is unrolled by two so that both register
    // sets keep fixed roles).
    auto do_block = [&](int g, int b, float (*kuse)[NB], float (*knext)[NB]) {
        if (b == 0) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[nb][v] = 0.f;
            // this lane's ring position: element g*4*srow + ii*srow + kofs of its row
            ridx = (uint32_t)(g * kRRows * p.srow + ii * p.srow + kofs) & (kRingLen - 1);
        }
        // Everything the previous block issued has landed: this block's K
        // fragments and chunks (and, at the start of a later group, the
        // previous group's O stores, issued last).
        if (b > 0 || g > g_begin) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        if (filled < blk_hi(g, b)) {  // not reached while the ring holds a block ahead
            fill_upto(blk_hi(g, b));
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        }
        // The next block's K fragments, issued before this block's fills: the
        // registers they land in are then in flight when the fills' addresses
        // are formed, so the compiler takes other registers for those (reusing
        // a K register there would make it wait for every load in flight).
        kload_block(knext);
        // prefetch the next block's chunks as far as the ring allows
        if (b + 1 < nblk) {
            const int cap = blk_lo(g, b) + kRingChunks - 1;
            const int want = blk_hi(g, b + 1);
            fill_upto(want < cap ? want : cap);
        }
        // the block's A fragments, all read up front (one LDS round trip per block)
        float a[BS];
#pragma unroll
        for (int u = 0; u < BS; ++u) a[u] = ring[abase + ((ridx + 2 * u) & (kRingLen - 1))];
        const int t = b * BS;
        if (2 * (t + BS) > p.KR) {  // the block reaches past KR: zeros there
#pragma unroll
            for (int u = 0; u < BS; ++u)
                if (2 * (t + u) + kofs >= p.KR) a[u] = 0.f;
        }
        ridx = (ridx + 2 * BS) & (kRingLen - 1);
#pragma unroll
        for (int u = 0; u < BS; ++u)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                acc[nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[u], kuse[u][nb], acc[nb], 0, 0, 0);
        if (b + 1 < nblk) return;
        // end of group g. The next group's first two blocks: its chunks as far
        // as the ring allows once this group's reads are done (the fill waits
        // for them).
        if (g + 1 < g_end) {
            const int cap = blk_lo(g + 1, 0) + kRingChunks - 1;
            const int want = blk_hi(g + 1, nblk > 1 ? 1 : 0);
            fill_upto(want < cap ? want : cap);
        }
        // O rows (pair, h) of this group, 32 channels per block: for register v
        // of lane l the row is acc_row(v, l) = 8*(v/4) + 4*(l/32) + v%4, i.e.
        // output row h = 4g + v/4 of pair 4*(l/32) + v%4. One buffer store per
        // register, at the lane's fixed offset plus the row's scalar offset.
#pragma unroll
        for (int r = 0; r < kRRows; ++r) {
            const int64_t h = (int64_t)g * kRRows + r;
            if (h >= p.o_h) break;
            const int32_t soff = __builtin_amdgcn_readfirstlane((int32_t)(h * p.o_w * p.k_c * 4));
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    // the element as a value first: a vector element has no
                    // object representation of its own to reinterpret
                    const float v = acc[nb][r * 4 + q4];
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), orsrc,
                                                          (int32_t)ooff[q4][nb], soff, kStoreNT);
                }
        }
    };
    const int nbeta = (g_end - g_begin) * nblk;
    int g = g_begin, b = 0;
    for (int beta = 0; beta < nbeta; beta += 2) {
        do_block(g, b, kb0, kb1);
        if (++b == nblk) { b = 0; ++g; }
        if (beta + 1 < nbeta) {
            do_block(g, b, kb1, kb0);
            if (++b == nblk) { b = 0; ++g; }
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// Items 0 .. nfull-1 whole (gpi row groups, all NB channel blocks of their
// channel tile), in an XCD-contiguous order; then, dispatched last, the
// remaining items split into one workgroup per row group and 32-channel
// block: when the whole items leave a last, partial round on the wave slots,
// its items would otherwise run alone at the end while the other slots idle
// (alexnet_conv1: 12320 one-group items on 2048 slots leave 32).
template <int NB, bool FUSED, int BS, bool SHORT>
__global__ __launch_bounds__(64) void slab_gemm_f32_ring_kernel(RingParams p) {
    __shared__ __align__(16) float ring[kRPairs * kRingLD];
    if (blockIdx.x < p.nfull) {
        const uint32_t t = xcd_remap(blockIdx.x, p.nfull);
        const uint32_t unit = t / (uint32_t)p.n_tiles;
        const int g_begin = (int)(unit % (uint32_t)p.items_pg) * p.gpi;
        const int g_end = g_begin + p.gpi < p.ngroups ? g_begin + p.gpi : p.ngroups;
        ring_item<NB, FUSED, BS, SHORT>(p, ring, (int64_t)(unit / (uint32_t)p.items_pg) * kRPairs, g_begin, g_end,
                             (int)(t % (uint32_t)p.n_tiles) * 32 * NB);
    } else {
        // one channel tile (n_tiles == 1): piece = (item, group of the item, channel block)
        const uint32_t piece = blockIdx.x - p.nfull;
        const uint32_t per = (uint32_t)(p.gpi * NB);
        const uint32_t unit = p.nfull + piece / per, sub = piece % per;
        const int g = (int)(unit % (uint32_t)p.items_pg) * p.gpi + (int)(sub / NB);
        if (g < p.ngroups)
            ring_item<1, FUSED, BS, SHORT>(p, ring, (int64_t)(unit / (uint32_t)p.items_pg) * kRPairs, g, g + 1,
                                (int)(sub % NB) * 32);
    }
}

struct RingPlan {
    int gpi;                 // row groups per item
    int64_t nfull, npieces;  // whole items, then single-group single-block pieces
};

// k-steps per block for a window of KR elements: 7 where whole blocks of 7 pad
// its ceil(KR / 2) steps less than blocks of 8 (alexnet_conv1: 182 steps, no
// padding against 184; 3x3 over 3 channels: 14 against 16), else 8.
int ring_block_steps(int64_t KR) {
    const int64_t st = (KR + 1) / 2;
    return (st + 6) / 7 * 7 < (st + 7) / 8 * 8 ? 7 : 8;
}
int64_t ring_nks(int64_t KR, int bs) { return ((KR + 1) / 2 + bs - 1) / bs * bs; }

constexpr int kMaxGroupsPerItem = 16;
// An item's start in k-steps of one channel block (one MFMA each): its first
// chunks are loaded before any product, about 2 us with two waves per SIMD.
constexpr int64_t kItemStart = 37;

// Estimated time, in sixteenths of a k-step of one channel block, of n
// workgroups of `work` k-steps plus a start each over `slots` wave slots (two
// per SIMD). Whole rounds run two waves to a SIMD. A last round over at most
// half the slots leaves most of its waves alone on a SIMD, where the products
// take about 0.7 of the time (measured 0.62-0.71 with one item per SIMD on
// vgg_first and cv3) and the start, mostly load latency, no less; a last
// round over more than half of them takes about 1/16 longer than a whole
// round (measured +4% to +8%).
int64_t ring_rounds_cost(int64_t n, int64_t work, int64_t slots) {
    const int64_t q = n / slots, r = n % slots, unit = work + kItemStart;
    int64_t t = q * unit * 16;
    if (r > 0) t += 2 * r <= slots ? work * 56 / 5 + kItemStart * 16 : unit * 17;
    return t;
}

// The launch's layout: gpi row groups per item, and the items of a last,
// partial round on the wave slots split into one workgroup per row group and
// 32-channel block when they are few (at most a quarter of the slots) and
// there is something to split (one channel tile of several blocks, or items
// of several groups). gpi (1 to 16) minimises the estimated time of the
// busiest slot (ring_rounds_cost), where a whole item's products take
// gpi * steps * nb k-steps of one channel block and a split piece's steps.
// More groups per item amortise the start over short reductions (3x3 over 3
// channels, 14 steps per group: vgg_first fused takes 14 groups per item, one
// round of 1792 items on 2048 slots, 44.0 us against 46.3 with 7 groups in
// 3584 items); long ones keep few (alexnet_conv1, 182 steps: 6160 two-group
// items, 16 of them split). The model still keeps cv3 at batch 32 on 2 groups
// per item and a split tail (84.9 us, against 89.5 with 7 groups in one
// round) and cv7 at batch 1 on one group per item (7.5 us, against 7.8 with 2).
RingPlan ring_plan(int64_t pgroups, int ngroups, int n_tiles, int nb, int64_t slots, int64_t steps) {
    RingPlan best{1, pgroups * ngroups * n_tiles, 0};
    if (slots <= 0) return best;
    int64_t best_cost = -1;
    for (int gpi = 1; gpi <= kMaxGroupsPerItem && gpi <= ngroups; ++gpi) {
        const int64_t items = pgroups * ((ngroups + gpi - 1) / gpi) * n_tiles;
        const int64_t rounds = items / slots, r = items % slots;
        const bool split = n_tiles == 1 && nb * gpi > 1 && rounds > 0 && r > 0 && 4 * r <= slots;
        const int64_t work = gpi * steps * nb;
        const int64_t cost = split ? rounds * (work + kItemStart) * 16 + ring_rounds_cost(r * nb * gpi, steps, slots)
                                   : ring_rounds_cost(items, work, slots);
        if (best_cost < 0 || cost < best_cost) {
            best = {gpi, split ? items - r : items, split ? r * nb * gpi : 0};
            best_cost = cost;
        }
    }
    return best;
}

}  // namespace

bool gemm_ring_usable(const Shape& s, int dtype) {
    if (dtype != 0) return false;
    const int64_t srow = s.s_h * s.R;
    const int bs = ring_block_steps(s.k_h * s.R);
    // the ring holds the chunks one block of the four rows reads plus the next
    // block's: (3 srow + 4 bs + 62) / 64 < 8 chunks
    if ((kRRows - 1) * srow + 4 * bs + 62 > (int64_t)kRingLen - 1) return false;
    // the next group's first chunk is not older than this group's last block's:
    // reads never move back past what the ring has already dropped
    if (2 * (ring_nks(s.k_h * s.R, bs) - bs) > kRRows * srow) return false;
    if (s.R * s.k_h > (int64_t(1) << 20) || s.pairs >= (int64_t(1) << 31)) return false;
    // byte offsets of one dword load within a pair group's source fit 32 bits:
    // lowered, 8 rows of L; fused, three images
    if (8 * s.i_h * s.R >= (int64_t(1) << 30)) return false;
    if (3 * s.i_h * s.i_w * s.i_c >= (int64_t(1) << 30)) return false;
    // O byte offsets from the first image of an item's 8 pairs (at most 8
    // images) plus an output row's stay below the dropped range
    if (9 * s.o_h * s.o_w * s.k_c * 4 >= (int64_t)kStoreDrop) return false;
    return true;
}

bool gemm_ring_short(const Shape& s) {
    const int64_t KR = s.k_h * s.R;
    const int bs = ring_block_steps(KR);
    return ring_nks(KR, bs) <= 2 * bs;
}

hipError_t launch_gemm_ring(const Shape& s, const void* A, const void* K, float* O, bool fused,
                            hipStream_t stream) {
    RingParams p{};
    p.A = static_cast<const float*>(A);
    p.K = static_cast<const float*>(K);
    p.O = O;
    p.pairs = s.pairs;
    p.o_w = s.o_w;
    p.o_h = s.o_h;
    p.k_c = s.k_c;
    p.rowlen = s.i_h * s.R;
    p.img_stride = s.i_h * s.i_w * s.i_c;
    p.x_stride = fused ? s.i_w * s.i_c : s.R;
    p.w_stride = fused ? s.s_w * s.i_c : s.i_h * s.R;
    p.R = (int32_t)s.R;
    p.KR = (int32_t)(s.k_h * s.R);
    const int bs = ring_block_steps(p.KR);
    p.nks = (int32_t)ring_nks(p.KR, bs);
    p.srow = (int32_t)(s.s_h * s.R);
    p.ngroups = (int32_t)((s.o_h + kRRows - 1) / kRRows);
    p.divR = FastDiv((uint32_t)s.R);
    p.div_ow = FastDiv((uint32_t)s.o_w);
    const int nb = s.k_c > 64 ? 3 : s.k_c > 32 ? 2 : 1;
    p.n_tiles = (int32_t)((s.k_c + 32 * nb - 1) / (32 * nb));
    const int64_t pgroups = (s.pairs + kRPairs - 1) / kRPairs;
    int64_t slots = 0;  // wave slots of the stream's device: eight per compute unit
    {
        int dev = 0, cus = 0;
        if (hipStreamGetDevice(stream, &dev) == hipSuccess &&
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
            slots = (int64_t)kWavesPerCU * cus;
    }
    const RingPlan plan = ring_plan(pgroups, p.ngroups, p.n_tiles, nb, slots, p.nks);
    if (plan.nfull + plan.npieces > 0x7fffffff) return hipErrorInvalidValue;
    p.gpi = plan.gpi;
    p.items_pg = (p.ngroups + p.gpi - 1) / p.gpi;
    p.nfull = (uint32_t)plan.nfull;
    const int64_t nfull = plan.nfull, npieces = plan.npieces;
    const dim3 grid((uint32_t)(nfull + npieces)), block(64);
    const bool short_win = gemm_ring_short(s);  // K fits two blocks: held for the whole item
#define MEC_RING(NB_, BS_, SHORT_)                                                                \
    if (nb == NB_ && bs == BS_ && short_win == SHORT_) {                                          \
        if (fused)                                                                                \
            hipLaunchKernelGGL((slab_gemm_f32_ring_kernel<NB_, true, BS_, SHORT_>), grid, block, 0, stream, p); \
        else                                                                                      \
            hipLaunchKernelGGL((slab_gemm_f32_ring_kernel<NB_, false, BS_, SHORT_>), grid, block, 0, stream, p); \
    }
    MEC_RING(1, 7, false)
    MEC_RING(2, 7, false)
    MEC_RING(3, 7, false)
    MEC_RING(1, 8, false)
    MEC_RING(2, 8, false)
    MEC_RING(3, 8, false)
    MEC_RING(1, 7, true)
    MEC_RING(2, 7, true)
    MEC_RING(3, 7, true)
    MEC_RING(1, 8, true)
    MEC_RING(2, 8, true)
    MEC_RING(3, 8, true)
#undef MEC_RING
    return hipGetLastError();
}

}  // namespace mec
