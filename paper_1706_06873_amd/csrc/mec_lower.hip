// MEC compact lowering on gfx950 (Section 3.3, Algorithm 2, first loop):
//   L[n, w, h, 0:k_w, 0:i_c] = I[n, h, s_w*w : s_w*w + k_w, 0:i_c]
// L viewed as (i_n*o_w*i_h) rows of R = k_w*i_c elements: row q = (n*o_w + w)*i_h + h
// is the contiguous run of R elements of I that starts at ((n*i_h + h)*i_w + s_w*w)*i_c.
//
// A pure copy, bound by HBM bandwidth, and write-heavy: |L| is about
// k_w/s_w times |I|. Three kernels, chosen per shape on the host:
//
//  rows   Every run starts on a 16-byte boundary (R, s_w*i_c and i_w*i_c are
//         multiples of the 16-byte vector). A workgroup reads one input row
//         (n, h) into LDS once -- a contiguous, fully coalesced read, so I is
//         read from HBM exactly once -- and writes its o_w runs
//         L[n, w, h, :] as 16-byte non-temporal stores. The runs are
//         scattered through L (stride i_h*R); streaming them past the caches
//         is what lets the write stream run near copy speed.
//  strip  Short or unaligned runs (e.g. R = 33 fp32 for 11x11x3 kernels). A
//         workgroup reads Hb (+ a few) consecutive input rows of one image
//         (again one contiguous span of I) and, for every w, writes the chunk
//         L[n, w, h0:h0+Hb, :] -- contiguous in L, Hb*R elements. It owns the
//         128-byte lines of L that start in its chunk (16-byte vectors when
//         chunks are short), so no line inside a column is written in two
//         parts by two workgroups, and every store there is one whole
//         non-temporal 16-byte vector; only the units that straddle two
//         columns are written element by element. (Granule ownership left a
//         quarter of the lines of 11x11x3 layers split, ~16% slower.)
//  gather Fallback when an input row does not fit in LDS: each thread
//         gathers 16 bytes of L straight from I.
//
// Block order: the write stream runs faster when the workgroups in flight
// across all 8 XCDs write one compact range of L than when each XCD walks a
// range of its own far from the others' (measured: rows kernel on deep_bf16
// 46.7 -> 43.9 us, on Table 2's cv8 75.8 -> 71.8 us). The rows kernel, which
// shares nothing between workgroups, keeps the hardware's order; the strip
// kernel, whose neighbouring chunks of one image stage the same overlap rows,
// gives each XCD the chunks of whole images in turn (alexnet_conv1 57.8 ->
// 55.9 us).
#include <hip/hip_runtime.h>

#include "mec_internal.h"

namespace mec {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kStripThreads = 512;
constexpr int kLineBytes = 128;           // cache line
constexpr int64_t kStripLineMinChunk = 512;  // bytes of L per chunk for line ownership
constexpr int kGatherThreads = 256;
constexpr int kMaxRowsPerBlock = 1024;
constexpr int64_t kTargetElemsPerBlock = 8192;
constexpr int64_t kRowsLdsLimit = 64 * 1024;   // one input row, rows kernel
constexpr int64_t kStripLdsLimit = 48 * 1024;  // Hb input rows, strip kernel

// E is a 32-bit (fp32) or 16-bit (bf16) payload; VEC elements make 16 bytes.
template <typename E>
struct Vec16 {
    static constexpr int N = 16 / sizeof(E);
    union {
        u32x4 v;
        E e[N];
    };
};

inline bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }

// ---------------------------------------------------------------- rows
struct RowsParams {
    const void* I;
    void* L;
    uint32_t nrows_in;  // i_n * i_h
    uint32_t i_h, o_w;
    uint32_t rowv;      // vectors per input row: i_w*i_c / VEC
    uint32_t RV;        // vectors per run: R / VEC
    uint32_t swv;       // vectors between consecutive runs in a row: s_w*i_c / VEC
    FastDiv div_ih, div_RV;
};

template <typename E, int THREADS>
__global__ __launch_bounds__(THREADS) void lower_rows_kernel(RowsParams p) {
    extern __shared__ u32x4 row[];
    const uint32_t blk = blockIdx.x;  // input row n*i_h + h
    const uint32_t n = p.div_ih.div(blk), h = blk - n * p.i_h;
    const u32x4* __restrict__ I = reinterpret_cast<const u32x4*>(p.I) + (size_t)blk * p.rowv;
    // I is read once: streamed past the caches like the stores of L
    for (uint32_t i = threadIdx.x; i < p.rowv; i += THREADS) row[i] = __builtin_nontemporal_load(I + i);
    __syncthreads();
    u32x4* __restrict__ L = reinterpret_cast<u32x4*>(p.L);
    const uint32_t total = p.o_w * p.RV;
    for (uint32_t f = threadIdx.x; f < total; f += THREADS) {
        const uint32_t w = p.div_RV.div(f);
        const uint32_t c = f - w * p.RV;
        __builtin_nontemporal_store(row[w * p.swv + c],
                                    L + (((size_t)n * p.o_w + w) * p.i_h + h) * p.RV + c);
    }
}

// ---------------------------------------------------------------- strip
struct StripParams {
    const void* I;
    void* L;
    uint32_t i_h, o_w, rowlen, R, swic, Hb, hblocks, vpw, nblocks;
    uint32_t extra;      // rows staged beyond the chunk: an owned unit may reach into them
    int32_t in_total;    // elements of I (bound of the staging loads)
    int32_t ioff;        // elements from the 16-byte boundary below I
    int32_t loff;        // elements from the unit-of-ownership boundary below L
    FastDiv div_hblocks, div_R, div_vpw;
};

// Chunk j of column (n, w) is written by workgroup (n, j). Ownership goes by
// aligned units of OWN bytes of L (a cache line or a 16-byte vector): the
// workgroup writes every unit whose first address lies in its chunk,
// L[n, w, h0 : h0+Hb, :], so no unit inside a column is split between
// workgroups and every store there is one 16-byte vector; only the units that
// straddle two columns (or the ends of L) are written element by element,
// each column's part by its own workgroup. A unit starting near the chunk's
// end reaches into the next rows, so the workgroup stages `extra` rows past
// its chunk. The staged rows are one contiguous span of I, loaded as 16-byte
// granules of I, with element loads for the granules that cross either end
// of I.
template <typename E, int OWN>
__global__ __launch_bounds__(kStripThreads) void lower_strip_kernel(StripParams p) {
    constexpr int VEC = Vec16<E>::N;
    constexpr int LINE = OWN / sizeof(E);  // elements per unit of ownership
    extern __shared__ u32x4 strip4[];
    E* rows = reinterpret_cast<E*>(strip4);
    const uint32_t blk = xcd_interleave(blockIdx.x, p.nblocks, p.hblocks);  // one image per run
    const uint32_t n = p.div_hblocks.div(blk), j = blk - n * p.hblocks;
    const uint32_t h0 = j * p.Hb;
    const uint32_t hend = min(h0 + p.Hb, p.i_h);          // chunk rows [h0, hend)
    const uint32_t sh = min(hend + p.extra, p.i_h) - h0;  // staged rows
    {
        // span [first, first + nin) of I; granules of I start at k*VEC - ioff
        const int32_t first = (int32_t)((n * p.i_h + h0) * p.rowlen);
        const int32_t nin = (int32_t)(sh * p.rowlen);
        const int32_t a0 = ((first + p.ioff) & ~(VEC - 1)) - p.ioff;
        const int32_t nv = (first - a0 + nin + VEC - 1) / VEC;
        const E* __restrict__ I = reinterpret_cast<const E*>(p.I);
        for (int32_t i = threadIdx.x; i < nv; i += kStripThreads) {
            const int32_t a = a0 + i * VEC;
            if (a >= 0 && a + VEC <= p.in_total) {
                strip4[i] = *reinterpret_cast<const u32x4*>(I + a);
            } else {
                for (int32_t k = 0; k < VEC; ++k)
                    if (a + k >= 0 && a + k < p.in_total) rows[i * VEC + k] = I[a + k];
            }
        }
    }
    __syncthreads();
    const uint32_t shift = (uint32_t)((((n * p.i_h + h0) * p.rowlen) + p.ioff) & (VEC - 1));

    E* __restrict__ L = reinterpret_cast<E*>(p.L);
    const int64_t col_len = (int64_t)p.i_h * p.R;
    const uint32_t total = p.o_w * p.vpw;
    for (uint32_t f = threadIdx.x; f < total; f += kStripThreads) {
        const uint32_t w = p.div_vpw.div(f);
        const uint32_t v = f - w * p.vpw;
        const int64_t base = ((int64_t)n * p.o_w + w) * col_len;  // column start in L
        // units of L start at k*LINE - loff; the chunk's granules run from its
        // first unit's start (chunk 0: the unit that starts before the column)
        // to the end of the last unit that starts below hi
        const int64_t from = base + (int64_t)h0 * p.R + (j == 0 ? 0 : LINE - 1);
        const int64_t lo = ((from + p.loff) & ~(int64_t)(LINE - 1)) - p.loff;
        const int64_t hi = base + (int64_t)hend * p.R;
        const int64_t gv = lo + (int64_t)v * VEC;
        if (((gv + p.loff) & ~(int64_t)(LINE - 1)) - p.loff >= hi) continue;
        const int e0 = (int)(gv - base);  // column index of the granule's first element
        const uint32_t ee = e0 < 0 ? 0u : (uint32_t)e0;
        const uint32_t r = p.div_R.div(ee);
        uint32_t c = ee - r * p.R;
        const E* src = rows + shift + w * p.swic + (r - h0) * p.rowlen;
        Vec16<E> val;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            const int e = e0 + k;
            val.e[k] = E(0);
            if (e >= 0 && e < (int)col_len) {
                val.e[k] = src[c];
                if (++c == p.R) {
                    c = 0;
                    src += p.rowlen;
                }
            }
        }
        if (e0 >= 0 && e0 + VEC <= (int)col_len) {
            __builtin_nontemporal_store(val.v, reinterpret_cast<u32x4*>(L + gv));
        } else {
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const int e = e0 + k;
                if (e >= 0 && e < (int)col_len) L[gv + k] = val.e[k];
            }
        }
    }
}

// ---------------------------------------------------------------- gather
// Each workgroup owns a contiguous range of L rows; the source offset of each
// of its rows is computed once into LDS.
template <typename E, bool VECDST>
__global__ __launch_bounds__(kGatherThreads) void lower_gather_kernel(LowerParams p) {
    constexpr int VEC = Vec16<E>::N;
    __shared__ int64_t src[kMaxRowsPerBlock];
    const uint32_t blk = xcd_remap(blockIdx.x, p.nblocks);
    const int64_t row0 = (int64_t)blk * p.rows_per_block;
    const int nrows = (int)min((int64_t)p.rows_per_block, p.rows - row0);
    for (int i = threadIdx.x; i < nrows; i += kGatherThreads) {
        const int64_t q = row0 + i;
        const int64_t h = q % p.i_h;
        const int64_t nw = q / p.i_h;
        const int64_t w = nw % p.o_w;
        const int64_t n = nw / p.o_w;
        src[i] = ((n * p.i_h + h) * p.i_w + p.s_w * w) * p.i_c;
    }
    __syncthreads();

    const uint32_t R = (uint32_t)p.R;
    const uint32_t count = (uint32_t)nrows * R;  // elements of L this block writes
    const E* __restrict__ I = reinterpret_cast<const E*>(p.I);
    E* __restrict__ L = reinterpret_cast<E*>(p.L) + row0 * p.R;
    for (uint32_t e0 = threadIdx.x * VEC; e0 < count; e0 += kGatherThreads * VEC) {
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
            *reinterpret_cast<u32x4*>(L + e0) = v.v;
        } else {
#pragma unroll
            for (int k = 0; k < VEC; ++k)
                if (e0 + k < count) L[e0 + k] = v.e[k];
        }
    }
}

// ---------------------------------------------------------------- host side

template <typename E>
hipError_t launch_rows(const Shape& s, const void* I, void* L, hipStream_t stream) {
    constexpr int VEC = Vec16<E>::N;
    RowsParams p{};
    p.I = I;
    p.L = L;
    p.nrows_in = (uint32_t)(s.i_n * s.i_h);
    p.i_h = (uint32_t)s.i_h;
    p.o_w = (uint32_t)s.o_w;
    p.rowv = (uint32_t)(s.i_w * s.i_c / VEC);
    p.RV = (uint32_t)(s.R / VEC);
    p.swv = (uint32_t)(s.s_w * s.i_c / VEC);
    p.div_ih = FastDiv(p.i_h);
    p.div_RV = FastDiv(p.RV);
    // Threads per workgroup (one input row each): 256 where the rows fill
    // every compute unit with 4 to 12 workgroups, 512 where there are fewer
    // (more bytes in flight per row) or more (measured: deep_bf16, 16 rows per
    // compute unit, 43.8 -> 41.7 us; Table 2's cv4 350 -> 341 us, cv10-cv12 6-20%
    // faster; resnet_mid and cv9, about 7 per compute unit, 2-3% slower at 512).
    int dev = 0, cus = 0;
    if (hipStreamGetDevice(stream, &dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 256;
    const int64_t per_cu = (int64_t)p.nrows_in / cus;
    if (per_cu >= 4 && per_cu < 12)
        hipLaunchKernelGGL((lower_rows_kernel<E, 256>), dim3(p.nrows_in), dim3(256), (size_t)p.rowv * 16,
                           stream, p);
    else
        hipLaunchKernelGGL((lower_rows_kernel<E, 512>), dim3(p.nrows_in), dim3(512), (size_t)p.rowv * 16,
                           stream, p);
    return hipGetLastError();
}

// Rows staged past a chunk so that every unit of `own` bytes starting in it
// is covered.
inline int64_t strip_extra(int64_t R, int64_t elem_bytes, int64_t own) {
    return (own / elem_bytes - 2) / R + 1;
}

// Rows per chunk for an ownership unit of `own` bytes: chunks of about 1 KB of
// L, enough workgroups to fill the chip (about 512, two per compute unit), and
// the chunk plus its extra rows within the LDS limit; 0 if not even one row
// fits.
inline int64_t strip_rows(const Shape& s, int64_t es, int64_t own) {
    const int64_t row_bytes = s.i_w * s.i_c * es;
    const int64_t extra = strip_extra(s.R, es, own);
    const int64_t fit = (kStripLdsLimit - 2 * 16) / row_bytes - extra;
    if (fit < 1) return 0;
    int64_t hb = (1024 + s.R * es - 1) / (s.R * es);
    const int64_t by_count = (s.i_n * s.i_h) / 512;
    if (hb > by_count) hb = by_count;
    if (hb > fit) hb = fit;
    if (hb > s.i_h) hb = s.i_h;
    if (hb < 1) hb = 1;
    return hb;
}

// OWN: bytes of L a workgroup owns as a unit (a 16-byte vector or a 128-byte
// line).
template <typename E, int OWN>
hipError_t launch_strip(const Shape& s, int64_t hb, const void* I, void* L, hipStream_t stream) {
    constexpr int VEC = Vec16<E>::N;
    const int64_t es = sizeof(E);
    const int64_t row_bytes = s.i_w * s.i_c * es;
    const int64_t extra = strip_extra(s.R, es, OWN);
    StripParams p{};
    p.I = I;
    p.L = L;
    p.i_h = (uint32_t)s.i_h;
    p.o_w = (uint32_t)s.o_w;
    p.rowlen = (uint32_t)(s.i_w * s.i_c);
    p.R = (uint32_t)s.R;
    p.swic = (uint32_t)(s.s_w * s.i_c);
    p.Hb = (uint32_t)hb;
    p.extra = (uint32_t)extra;
    p.in_total = (int32_t)(s.i_n * s.i_h * s.i_w * s.i_c);
    p.ioff = (int32_t)(((uintptr_t)I / es) % VEC);
    p.loff = (int32_t)(((uintptr_t)L / es) % (OWN / es));
    p.hblocks = (uint32_t)((s.i_h + hb - 1) / hb);
    // granules from the first owned unit's start to the last one's end
    p.vpw = (uint32_t)((hb * s.R + 2 * (OWN / es) + VEC - 1) / VEC);
    p.nblocks = (uint32_t)(s.i_n * p.hblocks);
    p.div_hblocks = FastDiv(p.hblocks);
    p.div_R = FastDiv(p.R);
    p.div_vpw = FastDiv(p.vpw);
    // staged rows plus up to one granule on each side of the span
    const int64_t staged = std::min<int64_t>(hb + extra, s.i_h);
    const size_t lds = (size_t)(staged * row_bytes + 2 * 16);
    hipLaunchKernelGGL((lower_strip_kernel<E, OWN>), dim3(p.nblocks), dim3(kStripThreads), lds, stream,
                       p);
    return hipGetLastError();
}

template <typename E>
hipError_t launch_gather(const Shape& s, const void* I, void* L, hipStream_t stream) {
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
    // rows per block: about kTargetElemsPerBlock elements, a multiple of VEC so
    // every block's slice of L starts 16-byte aligned when L does
    int64_t rpb = (kTargetElemsPerBlock + s.R - 1) / s.R;
    rpb = (rpb + VEC - 1) / VEC * VEC;
    if (rpb > kMaxRowsPerBlock) rpb = kMaxRowsPerBlock;
    p.rows_per_block = (int32_t)rpb;
    p.nblocks = (uint32_t)((p.rows + rpb - 1) / rpb);
    p.divR = FastDiv((uint32_t)s.R);
    if (aligned16(L))
        hipLaunchKernelGGL((lower_gather_kernel<E, true>), dim3(p.nblocks), dim3(kGatherThreads),
                           0, stream, p);
    else
        hipLaunchKernelGGL((lower_gather_kernel<E, false>), dim3(p.nblocks), dim3(kGatherThreads),
                           0, stream, p);
    return hipGetLastError();
}

template <typename E>
hipError_t launch_typed(const Shape& s, const void* I, void* L, hipStream_t stream) {
    constexpr int VEC = Vec16<E>::N;
    const int64_t row_bytes = s.i_w * s.i_c * (int64_t)sizeof(E);
    const bool vec_runs = s.R % VEC == 0 && (s.s_w * s.i_c) % VEC == 0 &&
                          (s.i_w * s.i_c) % VEC == 0 && aligned16(I) && aligned16(L);
    // 32-bit indices inside the row-based kernels
    const bool small = s.i_n * s.i_h < (int64_t(1) << 31) && s.i_h * s.R < (int64_t(1) << 31) &&
                       s.o_w * (s.R / VEC + 2) < (int64_t(1) << 31);
    if (small && vec_runs && row_bytes <= kRowsLdsLimit) return launch_rows<E>(s, I, L, stream);
    // strip: 32-bit offsets into I and within a workgroup's o_w chunks, and at
    // least one chunk row plus its extra rows in LDS
    const bool strip_ok = small && s.i_n * s.i_h * s.i_w * s.i_c < (int64_t(1) << 31) &&
                          s.o_w * (s.i_h * s.R / VEC + 18) < (int64_t(1) << 31);
    if (strip_ok) {
        // whole cache lines per workgroup when the chunks are long enough that
        // the lines' extra rows and idle lanes cost less than lines written in
        // two parts by two workgroups; 16-byte vectors otherwise
        const int64_t es = sizeof(E);
        const int64_t hb_line = strip_rows(s, es, kLineBytes);
        if (hb_line > 0 && hb_line * s.R * es >= kStripLineMinChunk)
            return launch_strip<E, kLineBytes>(s, hb_line, I, L, stream);
        const int64_t hb_vec = strip_rows(s, es, 16);
        if (hb_vec > 0) return launch_strip<E, 16>(s, hb_vec, I, L, stream);
    }
    return launch_gather<E>(s, I, L, stream);
}

}  // namespace

hipError_t launch_lower(const Shape& s, const void* I, void* L, int elem_bytes,
                        hipStream_t stream) {
    if (elem_bytes == 4) return launch_typed<uint32_t>(s, I, L, stream);
    return launch_typed<uint16_t>(s, I, L, stream);
}

}  // namespace mec
