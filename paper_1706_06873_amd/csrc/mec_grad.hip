// Training passes of the convolution through MEC's lowered layout, fp32.
//
// The paper names training as a use of MEC (Section 1; the set-ups of
// Section 4 include training) but gives no backward algorithm. With R =
// k_w*i_c, the product phase computes for every output row h
//   O_h = A_h K,   A_h = L[:, :][s_h*R*h : s_h*R*h + k_h*R]   ((i_n*o_w) x (k_h*R))
// with K viewed as (k_h*R) x k_c. For a loss with gradient G = dloss/dO and
// G_h = G[n, h, w, :] as an (i_n*o_w) x k_c matrix, differentiating gives
//   dL = every slab receives G_h K^T, summed where slabs overlap,
//   dK = sum over h of A_h^T G_h,
// and since the lowering copies I into L, dI is the fold of dL: each element
// of dL added back to the input pixel it was copied from.
//
//  dgrad_dl  dL from G and K on fp32 MFMA (v_mfma_f32_32x32x2_f32). A
//            workgroup computes 32 (n, w) pairs x RT consecutive rows r of dL
//            x 64 columns (b, c). Row r receives G[n, h, w, :] K[a]^T for every
//            (h, a) with h*s_h + a = r, so the tile stages the hspan rows of G
//            its rows draw on and the k_h kernel rows, once per chunk of KT
//            output channels; each staged G row feeds up to ceil(k_h/s_h) rows
//            of dL, the slab overlap of the forward pass seen from the other
//            side. Rows of dL that no slab covers are written as zeros.
//  fold      dI[n, h, x, c] = sum over w with 0 <= x - s_w*w < k_w of
//            dL[n, w, h, x - s_w*w, c], in increasing w: a gather, one thread
//            per element (or per 4 channels), bound by HBM bandwidth.
//  dI as sub-pixel phases  the pixels dI[n, s_h*Y + py, s_w*X + px, :] of
//            one phase receive G only through the taps a = py + s_h*j,
//            b = px + s_w*i, so each phase is a stride-1 convolution: G zero-
//            padded by J-1 rows and I-1 columns, correlated with those taps
//            turned by 180 degrees and transposed (stride 1: one phase, padding
//            k-1). pad_grad and phase_kernel form the operands; the forward's
//            fused slab products write each phase straight into its pixels.
//  wgrad     a share of the reduction over (pair, output row) on fp32 MFMA: a
//            workgroup computes a 128 x 64 tile of dK (rows j = a*R + b*i_c + c,
//            columns m) over the stages in its share, a stage being 16 pairs x
//            4 output rows, and writes the tile to its own partial buffer;
//            wgrad_slab, for short rows, takes all k_h kernel rows of 64
//            columns at once and feeds each staged L row to every (h, a) that
//            reads it.
//  reduce    dK = the partial buffers summed in a fixed order (groups of
//            consecutive shares, then the groups), so the result does not
//            depend on scheduling.
// Global loads of the next stage go to registers before the current stage's
// MFMAs and to LDS after them.
#include <mutex>

#include "mec_mfma.h"

namespace mec {
namespace {

constexpr int kGradThreads = 256;

// ---------------------------------------------------------------- dgrad: dL
constexpr int kDgRT = 8;   // rows of dL per tile
constexpr int kDgJT = 64;  // columns of dL per tile: two 32-wide MFMA blocks
constexpr int kDgRW = 4;   // rows per wave; waves = 2 row groups x 2 column blocks
constexpr size_t kDgLdsBudget = 80 * 1024;  // two workgroups per compute unit

struct DgradParams {
    const float* G;
    const float* K;
    float* dL;
    int32_t i_h, o_h, o_w, k_h, s_h, k_c, R;
    int32_t pairs;
    int32_t r_tiles, j_tiles;
    uint32_t ntiles;
    int32_t hspan;    // G rows a tile stages: (RT + k_h - 2) / s_h + 1
    int32_t nchunks;  // chunks of KT output channels
    int32_t gps;      // LDS stride between pairs in the G stage: hspan*KT + 1 (odd)
    int32_t gunits;   // load units of the G stage: 32 * hspan * KT / VW
    int32_t kbase;    // LDS offset of the K stage
    int32_t kunits;   // load units of the K stage: k_h * JT * KT / VW
    int32_t stage;    // LDS floats of one stage
    int32_t nbuf;     // stages in LDS: 2 (double-buffered) or 1
    FastDiv div_gu;   // by hspan * KT / VW (units per staged pair)
};

// KT: output channels per chunk. VW: channels per global load (4: one
// 16-byte load, k_c % 4 == 0 and G, K aligned; 1: one element). MAXU: load
// units one thread moves per stage (the prefetch registers); the host checks
// that a stage fits. LDS rows have odd strides, so the MFMA operand reads of
// the 32 rows of a block hit 32 different banks; the staging therefore
// writes LDS one element at a time.
template <int KT, int VW, int MAXU>
__global__ __launch_bounds__(kGradThreads) void dgrad_dl_kernel(DgradParams p) {
    typedef float vec_t __attribute__((ext_vector_type(VW)));
    constexpr int QU = KT / VW;  // load units per staged row
    extern __shared__ __align__(16) float dg_smem[];
    __shared__ int64_t gbase[kPairs];  // G offset of (n, 0, w, 0), or -1 past the last pair
    __shared__ int64_t lbase[kPairs];  // dL offset of pair row (n, w)
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave & 1, wn = wave >> 1;

    const uint32_t t = xcd_remap(blockIdx.x, p.ntiles);
    const int jt = (int)(t % (uint32_t)p.j_tiles);
    const uint32_t rest = t / (uint32_t)p.j_tiles;
    const int rt = (int)(rest % (uint32_t)p.r_tiles);
    const int pt = (int)(rest / (uint32_t)p.r_tiles);
    const int r0 = rt * kDgRT, j0 = jt * kDgJT;
    const int64_t pair0 = (int64_t)pt * kPairs;
    // first G row any of rows r0.. needs: the smallest h with h*s_h >= r0 - k_h + 1
    const int lo = r0 - p.k_h + 1;
    const int h_min = lo > 0 ? (lo + p.s_h - 1) / p.s_h : 0;

    if (tid < kPairs) {
        const int64_t pair = pair0 + tid;
        if (pair < p.pairs) {
            const int64_t n = pair / p.o_w, w = pair - n * p.o_w;
            gbase[tid] = (n * p.o_h * p.o_w + w) * p.k_c;
            lbase[tid] = pair * p.i_h * p.R;
        } else {
            gbase[tid] = -1;
            lbase[tid] = -1;
        }
    }
    __syncthreads();

    const int total = p.gunits + p.kunits;
    // load unit u of the chunk starting at channel m0: its LDS offset and
    // global source (nullptr where the stage holds zeros). With VW = 4 and
    // k_c % 4 == 0 a unit is wholly inside or wholly past the k_c channels.
    auto map = [&](int u, int m0, int& off) -> const float* {
        if (u < p.gunits) {
            const int pp = (int)p.div_gu.div((uint32_t)u);
            const int rem = u - pp * p.hspan * QU;
            const int hh = rem / QU, q = rem - (rem / QU) * QU;
            off = pp * p.gps + hh * KT + q * VW;
            const int h = h_min + hh, m = m0 + q * VW;
            const int64_t gb = gbase[pp];
            if (gb >= 0 && h < p.o_h && m < p.k_c) return p.G + gb + (int64_t)h * p.o_w * p.k_c + m;
            return nullptr;
        }
        const int u2 = u - p.gunits;
        const int a = u2 / (kDgJT * QU);
        const int rem = u2 - a * (kDgJT * QU);
        const int jj = rem / QU, q = rem - (rem / QU) * QU;
        off = p.kbase + (a * kDgJT + jj) * (KT + 1) + q * VW;
        const int j = j0 + jj, m = m0 + q * VW;
        if (j < p.R && m < p.k_c) return p.K + ((int64_t)a * p.R + j) * p.k_c + m;
        return nullptr;
    };

    vec_t regs[MAXU];
    auto load = [&](int rc) {
        int off;
#pragma unroll
        for (int i = 0; i < MAXU; ++i) {
            const int u = tid + i * kGradThreads;
            vec_t v = {};
            if (u < total) {
                const float* src = map(u, rc * KT, off);
                if (src) v = *reinterpret_cast<const vec_t*>(src);
            }
            regs[i] = v;
        }
    };
    auto store = [&](float* st) {
        int off;
#pragma unroll
        for (int i = 0; i < MAXU; ++i) {
            const int u = tid + i * kGradThreads;
            if (u < total) {
                (void)map(u, 0, off);
#pragma unroll
                for (int k = 0; k < VW; ++k) st[off + k] = regs[i][k];
            }
        }
    };

    floatx16 acc[kDgRW];
#pragma unroll
    for (int i = 0; i < kDgRW; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][v] = 0.f;

    const int row = lane & 31, khalf = lane >> 5;
    auto compute = [&](const float* st) {
        const float* Gs = st;
        const float* Ks = st + p.kbase;
#pragma unroll
        for (int rr = 0; rr < kDgRW; ++rr) {
            const int r = r0 + wr * kDgRW + rr;
            for (int a = 0; a < p.k_h && a <= r; ++a) {
                const int d = r - a;
                const int h = d / p.s_h;
                if (d - h * p.s_h != 0 || h >= p.o_h) continue;
                const float* gp = Gs + row * p.gps + (h - h_min) * KT + khalf;
                const float* kp = Ks + (a * kDgJT + wn * 32 + row) * (KT + 1) + khalf;
#pragma unroll
                for (int kk = 0; kk < KT; kk += 2)
                    acc[rr] = __builtin_amdgcn_mfma_f32_32x32x2f32(gp[kk], kp[kk], acc[rr], 0, 0, 0);
            }
        }
    };

    const bool dbuf = p.nbuf == 2;
    auto buf = [&](int rc) { return dg_smem + (dbuf ? (rc & 1) * p.stage : 0); };
    load(0);
    store(buf(0));
    __syncthreads();
    for (int rc = 0; rc < p.nchunks; ++rc) {
        const bool more = rc + 1 < p.nchunks;
        if (more) load(rc + 1);  // in flight during the MFMAs below
        compute(buf(rc));
        if (more) {
            if (!dbuf) __syncthreads();  // every wave is done reading the single stage
            store(buf(rc + 1));
        }
        __syncthreads();
    }

    // lane holds C[pair][col]: pair = acc_row(v, lane), col = lane % 32
    const int col = j0 + wn * 32 + row;
    if (col >= p.R) return;
#pragma unroll
    for (int rr = 0; rr < kDgRW; ++rr) {
        const int r = r0 + wr * kDgRW + rr;
        if (r >= p.i_h) continue;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int64_t lb = lbase[acc_row(v, lane)];
            if (lb >= 0) p.dL[lb + (int64_t)r * p.R + col] = acc[rr][v];
        }
    }
}

// ---------------------------------------------------------------- fold
struct FoldParams {
    const float* dL;
    float* dI;
    uint32_t units;  // elements of dI, or groups of 4 channels
    uint32_t i_h, i_w, i_c, k_w, s_w, o_w, R;
    FastDiv div_ic, div_iw, div_ih;
};

// V = 4: four consecutive channels per thread (i_c % 4 == 0, 16-byte aligned
// dL and dI); V = 1: one element.
template <int V>
__global__ __launch_bounds__(kGradThreads) void fold_kernel(FoldParams p) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const uint32_t stride = gridDim.x * kGradThreads;
    for (uint32_t u = blockIdx.x * kGradThreads + threadIdx.x; u < p.units; u += stride) {
        const uint32_t q = u * V;  // element index in dI
        const uint32_t t = p.div_ic.div(q), c = q - t * p.i_c;
        const uint32_t t2 = p.div_iw.div(t), x = t - t2 * p.i_w;
        const uint32_t n = p.div_ih.div(t2), h = t2 - n * p.i_h;
        // columns w whose strip [s_w*w, s_w*w + k_w) holds x
        const uint32_t w_lo = x >= p.k_w ? (x - p.k_w) / p.s_w + 1 : 0;
        uint32_t w_hi = x / p.s_w;
        if (w_hi > p.o_w - 1) w_hi = p.o_w - 1;
        const size_t col = (size_t)p.i_h * p.R;  // elements of one column strip L[n, w]
        const float* src = p.dL + ((size_t)n * p.o_w * p.i_h + h) * p.R + c;
        if (V == 4) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            for (uint32_t w = w_lo; w <= w_hi; ++w)
                acc += *reinterpret_cast<const f32x4*>(src + w * col + (size_t)(x - p.s_w * w) * p.i_c);
            __builtin_nontemporal_store(acc, reinterpret_cast<f32x4*>(p.dI + q));
        } else {
            float acc = 0.f;
            for (uint32_t w = w_lo; w <= w_hi; ++w) acc += src[w * col + (size_t)(x - p.s_w * w) * p.i_c];
            __builtin_nontemporal_store(acc, p.dI + q);
        }
    }
}

// ---------------------------------------------------------------- wgrad
constexpr int kWgPT = 16, kWgHT = 4;  // a stage: 16 pairs x 4 output rows
constexpr int kWgC = kWgPT * kWgHT;   // (pair, row) combinations per stage
constexpr int kWgJT = 128;            // dK rows per tile: one 32-row block per wave
constexpr int kWgMT = 64;             // dK columns per tile: two 32-wide blocks
constexpr int kWgA4 = kWgC * kWgJT / 4 / kGradThreads;  // float4 of the A stage per thread
constexpr int kWgB4 = kWgC * kWgMT / 4 / kGradThreads;  // float4 of the B stage per thread

struct WgradParams {
    const float* L;   // L, or I when fused
    const float* G;
    float* part;      // splits x KD x k_c partial sums
    int32_t i_h, o_h, o_w, k_c, s_h, R, KD, pairs;
    int32_t h_chunks;  // ceil(o_h / HT)
    int32_t nstages;   // ceil(pairs / PT) * h_chunks
    int32_t splits;
    int32_t j_tiles, m_tiles;
    uint32_t ntiles;
    int32_t lvec;      // L loads as 16-byte vectors (R % 4 == 0, L aligned)
    int32_t gvec;      // G loads as 16-byte vectors (k_c % 4 == 0, G aligned)
    int32_t fused;     // the rows of L read from I: L[n*o_w + w, x, r] = I[n, x, s_w*w*i_c + r]
    int32_t i_w, i_c, s_w;
    FastDiv div_ow;
    FastDiv div_R;     // fused wgrad_kernel: j -> (kernel row, r)
};

__global__ __launch_bounds__(kGradThreads) void wgrad_kernel(WgradParams p) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    __shared__ __align__(16) float As[kWgC * kWgJT];  // [combination][j]
    __shared__ __align__(16) float Bs[kWgC * kWgMT];  // [combination][m]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

    const uint32_t t = xcd_remap(blockIdx.x, p.ntiles);
    const int jt = (int)(t % (uint32_t)p.j_tiles);
    const uint32_t rest = t / (uint32_t)p.j_tiles;
    const int mt = (int)(rest % (uint32_t)p.m_tiles);
    const int s = (int)(rest / (uint32_t)p.m_tiles);
    const int j0 = jt * kWgJT, m0 = mt * kWgMT;
    const int st_begin = (int)((int64_t)s * p.nstages / p.splits);
    const int st_end = (int)((int64_t)(s + 1) * p.nstages / p.splits);

    f32x4 ra[kWgA4], rb[kWgB4];
    auto load = [&](int st) {
        const int pc = st / p.h_chunks, hc = st - (st / p.h_chunks) * p.h_chunks;
#pragma unroll
        for (int i = 0; i < kWgA4; ++i) {
            const int u = tid + i * kGradThreads;
            const int cidx = u >> 5, jq = (u & 31) * 4;
            const int pair = pc * kWgPT + (cidx >> 2), h = hc * kWgHT + (cidx & 3);
            const int j = j0 + jq;
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (pair < p.pairs && h < p.o_h && p.fused) {
                // j = a*R + r of this (pair, h): I[n, h*s_h + a, s_w*w*i_c + r]; with
                // R % 4 == 0 the four j of a vector stay in one kernel row
                const int n = (int)p.div_ow.div((uint32_t)pair), w = pair - n * p.o_w;
                const int64_t pix = ((int64_t)n * p.i_h + (int64_t)h * p.s_h) * p.i_w + (int64_t)p.s_w * w;
                auto at = [&](int jj) {
                    const int a = (int)p.div_R.div((uint32_t)jj);
                    return p.L + (pix + (int64_t)a * p.i_w) * p.i_c + (jj - a * p.R);
                };
                if (p.lvec && j + 3 < p.KD) {
                    v = *reinterpret_cast<const f32x4*>(at(j));
                } else {
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        if (j + k < p.KD) v[k] = *at(j + k);
                }
            } else if (pair < p.pairs && h < p.o_h) {
                const float* src = p.L + ((int64_t)pair * p.i_h + (int64_t)h * p.s_h) * p.R + j;
                if (p.lvec && j + 3 < p.KD) {
                    v = *reinterpret_cast<const f32x4*>(src);
                } else {
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        if (j + k < p.KD) v[k] = src[k];
                }
            }
            ra[i] = v;
        }
#pragma unroll
        for (int i = 0; i < kWgB4; ++i) {
            const int u = tid + i * kGradThreads;
            const int cidx = u >> 4, mq = (u & 15) * 4;
            const int pair = pc * kWgPT + (cidx >> 2), h = hc * kWgHT + (cidx & 3);
            const int m = m0 + mq;
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (pair < p.pairs && h < p.o_h) {
                const int n = (int)p.div_ow.div((uint32_t)pair), w = pair - n * p.o_w;
                const float* src = p.G + (((int64_t)n * p.o_h + h) * p.o_w + w) * p.k_c + m;
                if (p.gvec && m + 3 < p.k_c) {
                    v = *reinterpret_cast<const f32x4*>(src);
                } else {
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        if (m + k < p.k_c) v[k] = src[k];
                }
            }
            rb[i] = v;
        }
    };
    auto store = [&]() {
#pragma unroll
        for (int i = 0; i < kWgA4; ++i) {
            const int u = tid + i * kGradThreads;
            *reinterpret_cast<f32x4*>(As + (u >> 5) * kWgJT + (u & 31) * 4) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < kWgB4; ++i) {
            const int u = tid + i * kGradThreads;
            *reinterpret_cast<f32x4*>(Bs + (u >> 4) * kWgMT + (u & 15) * 4) = rb[i];
        }
    };

    floatx16 acc[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[nb][v] = 0.f;
    const int row = lane & 31, khalf = lane >> 5;

    if (st_begin < st_end) {
        load(st_begin);
        store();
        __syncthreads();
        for (int st = st_begin; st < st_end; ++st) {
            const bool more = st + 1 < st_end;
            if (more) load(st + 1);  // in flight during the MFMAs below
#pragma unroll 8
            for (int kk = 0; kk < kWgC; kk += 2) {
                const float af = As[(kk + khalf) * kWgJT + wave * 32 + row];
#pragma unroll
                for (int nb = 0; nb < 2; ++nb) {
                    const float bf = Bs[(kk + khalf) * kWgMT + nb * 32 + row];
                    acc[nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(af, bf, acc[nb], 0, 0, 0);
                }
            }
            __syncthreads();  // every wave is done with this stage
            if (more) {
                store();
                __syncthreads();
            }
        }
    }

    // lane holds C[j][m]: j = wave*32 + acc_row(v, lane), m = nb*32 + lane % 32
    float* out = p.part + (int64_t)s * p.KD * p.k_c;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        const int m = m0 + nb * 32 + row;
        if (m >= p.k_c) continue;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int j = j0 + wave * 32 + acc_row(v, lane);
            if (j < p.KD) out[(int64_t)j * p.k_c + m] = acc[nb][v];
        }
    }
}

// wgrad for the common kernel heights, reusing the slab overlap: a
// workgroup computes every kernel row a < KH for 64 columns (b, c) and 64
// output channels, i.e. the dK rows j = a*R + r for r in [r0, r0 + 64). A
// stage is 16 pairs x 4 output rows as above, but it holds the union of the L
// rows those output rows read -- hrows = 3*s_h + KH rows per pair, 64 columns
// each -- and every staged row feeds each (h, a) with h*s_h + a equal to it:
// KH MFMAs per G fragment instead of one. Wave w computes the 32-column block
// w & 1 and the 32-channel block w >> 1 for all KH kernel rows. VEC: 16-byte
// staging loads (R and k_c multiples of 4, L and G 16-byte aligned).
constexpr int kWs = 64;     // columns r and channels m per tile
constexpr int kWsRows = 8;  // LDS rows per staged pair: 3*s_h + KH <= 8 (host check)
template <int KH, bool VEC>
__global__ __launch_bounds__(kGradThreads) void wgrad_slab_kernel(WgradParams p) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    constexpr int HR_MAX = kWsRows;
    constexpr int A4 = kWgPT * HR_MAX * (kWs / 4) / kGradThreads;  // float4 per thread, max
    constexpr int B4 = kWgC * kWs / 4 / kGradThreads;
    __shared__ __align__(16) float As[kWgPT * HR_MAX * kWs];  // [pair][staged row][r]
    __shared__ __align__(16) float Bs[kWgC * kWs];            // [combination][m]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int hrows = (kWgHT - 1) * p.s_h + KH;
    const int a_units = kWgPT * hrows * (kWs / 4);

    const uint32_t t = xcd_remap(blockIdx.x, p.ntiles);
    const int rt = (int)(t % (uint32_t)p.j_tiles);
    const uint32_t rest = t / (uint32_t)p.j_tiles;
    const int mt = (int)(rest % (uint32_t)p.m_tiles);
    const int s = (int)(rest / (uint32_t)p.m_tiles);
    const int r0 = rt * kWs, m0 = mt * kWs;
    const int st_begin = (int)((int64_t)s * p.nstages / p.splits);
    const int st_end = (int)((int64_t)(s + 1) * p.nstages / p.splits);

    f32x4 ra[A4], rb[B4];
    auto load = [&](int st) {
        const int pc = st / p.h_chunks, hc = st - (st / p.h_chunks) * p.h_chunks;
        const int x0 = hc * kWgHT * p.s_h;  // first staged input row
#pragma unroll
        for (int i = 0; i < A4; ++i) {
            const int u = tid + i * kGradThreads;
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (u < a_units) {
                const int pp = u / (hrows * (kWs / 4)), rem = u - pp * hrows * (kWs / 4);
                const int x = rem / (kWs / 4), r = r0 + (rem - x * (kWs / 4)) * 4;
                const int pair = pc * kWgPT + pp;
                if (pair < p.pairs && x0 + x < p.i_h) {
                    // L[n*o_w + w][x][r] = I[n][x][s_w*w*i_c + r] (the lowering's definition)
                    int64_t base;
                    if (p.fused) {
                        const int n = (int)p.div_ow.div((uint32_t)pair), w = pair - n * p.o_w;
                        base = (((int64_t)n * p.i_h + x0 + x) * p.i_w + (int64_t)p.s_w * w) * p.i_c;
                    } else {
                        base = ((int64_t)pair * p.i_h + x0 + x) * p.R;
                    }
                    const float* src = p.L + base + r;
                    if (VEC) {
                        if (r < p.R) v = *reinterpret_cast<const f32x4*>(src);
                    } else {
#pragma unroll
                        for (int k = 0; k < 4; ++k)
                            if (r + k < p.R) v[k] = src[k];
                    }
                }
            }
            ra[i] = v;
        }
#pragma unroll
        for (int i = 0; i < B4; ++i) {
            const int u = tid + i * kGradThreads;
            const int cidx = u >> 4, m = m0 + (u & 15) * 4;
            const int pair = pc * kWgPT + (cidx >> 2), h = hc * kWgHT + (cidx & 3);
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (pair < p.pairs && h < p.o_h) {
                const int n = (int)p.div_ow.div((uint32_t)pair), w = pair - n * p.o_w;
                const float* src = p.G + (((int64_t)n * p.o_h + h) * p.o_w + w) * p.k_c + m;
                if (VEC) {
                    if (m < p.k_c) v = *reinterpret_cast<const f32x4*>(src);
                } else {
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        if (m + k < p.k_c) v[k] = src[k];
                }
            }
            rb[i] = v;
        }
    };
    auto store = [&]() {
#pragma unroll
        for (int i = 0; i < A4; ++i) {
            const int u = tid + i * kGradThreads;
            if (u < a_units) {
                const int pp = u / (hrows * (kWs / 4)), rem = u - pp * hrows * (kWs / 4);
                const int x = rem / (kWs / 4), q = rem - x * (kWs / 4);
                *reinterpret_cast<f32x4*>(As + (pp * HR_MAX + x) * kWs + q * 4) = ra[i];
            }
        }
#pragma unroll
        for (int i = 0; i < B4; ++i) {
            const int u = tid + i * kGradThreads;
            *reinterpret_cast<f32x4*>(Bs + (u >> 4) * kWs + (u & 15) * 4) = rb[i];
        }
    };

    floatx16 acc[KH];
#pragma unroll
    for (int a = 0; a < KH; ++a)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[a][v] = 0.f;
    const int row = lane & 31, khalf = lane >> 5;
    const int rblk = (wave & 1) * 32, mblk = (wave >> 1) * 32;

    if (st_begin < st_end) {
        load(st_begin);
        store();
        __syncthreads();
        for (int st = st_begin; st < st_end; ++st) {
            const bool more = st + 1 < st_end;
            if (more) load(st + 1);  // in flight during the MFMAs below
#pragma unroll 4
            for (int kk = 0; kk < kWgC; kk += 2) {
                const int c = kk + khalf;  // this lane's (pair, output row) combination
                const int pp = c >> 2, hh = c & 3;
                const float bf = Bs[c * kWs + mblk + row];
                const float* ap = As + (pp * HR_MAX + hh * p.s_h) * kWs + rblk + row;
#pragma unroll
                for (int a = 0; a < KH; ++a)
                    acc[a] = __builtin_amdgcn_mfma_f32_32x32x2f32(ap[a * kWs], bf, acc[a], 0, 0, 0);
            }
            __syncthreads();  // every wave is done with this stage
            if (more) {
                store();
                __syncthreads();
            }
        }
    }

    // lane holds C[r][m] of kernel row a: r = r0 + rblk + acc_row(v, lane), m = m0 + mblk + lane % 32
    float* out = p.part + (int64_t)s * p.KD * p.k_c;
    const int m = m0 + mblk + row;
    if (m >= p.k_c) return;
#pragma unroll
    for (int a = 0; a < KH; ++a)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int r = r0 + rblk + acc_row(v, lane);
            if (r < p.R) out[((int64_t)a * p.R + r) * p.k_c + m] = acc[a][v];
        }
}

// dK[e] = the sum over shares s of part[s][e], in two passes so that many
// workgroups share the reading: pass 1 sums each group of consecutive shares
// (group g = shares [g*S/NG, (g+1)*S/NG)) in increasing order and writes the
// result over the group's first share; pass 2 sums the NG group results in
// increasing order into dK. The order is fixed, so dK does not depend on
// scheduling. V = 4 when E % 4 == 0 and both buffers are 16-byte aligned.
template <int V>
__global__ __launch_bounds__(kGradThreads) void wgrad_reduce_groups_kernel(float* part, uint32_t units,
                                                                           uint32_t E, int32_t splits,
                                                                           int32_t groups) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const uint32_t u = blockIdx.x * kGradThreads + threadIdx.x;
    if (u >= units) return;
    const int g = blockIdx.y;
    const int s0 = (int)((int64_t)g * splits / groups), s1 = (int)((int64_t)(g + 1) * splits / groups);
    if (V == 4) {
        f32x4 acc = *reinterpret_cast<const f32x4*>(part + (size_t)s0 * E + (size_t)u * 4);
        for (int s = s0 + 1; s < s1; ++s)
            acc += *reinterpret_cast<const f32x4*>(part + (size_t)s * E + (size_t)u * 4);
        *reinterpret_cast<f32x4*>(part + (size_t)s0 * E + (size_t)u * 4) = acc;
    } else {
        float acc = part[(size_t)s0 * E + u];
        for (int s = s0 + 1; s < s1; ++s) acc += part[(size_t)s * E + u];
        part[(size_t)s0 * E + u] = acc;
    }
}

template <int V>
__global__ __launch_bounds__(kGradThreads) void wgrad_reduce_kernel(const float* part, float* dK,
                                                                    uint32_t units, uint32_t E,
                                                                    int32_t splits, int32_t groups) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const uint32_t stride = gridDim.x * kGradThreads;
    for (uint32_t u = blockIdx.x * kGradThreads + threadIdx.x; u < units; u += stride) {
        if (V == 4) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            for (int g = 0; g < groups; ++g) {
                const size_t s0 = (size_t)((int64_t)g * splits / groups);
                acc += *reinterpret_cast<const f32x4*>(part + s0 * E + (size_t)u * 4);
            }
            *reinterpret_cast<f32x4*>(dK + (size_t)u * 4) = acc;
        } else {
            float acc = 0.f;
            for (int g = 0; g < groups; ++g) {
                const size_t s0 = (size_t)((int64_t)g * splits / groups);
                acc += part[s0 * E + u];
            }
            dK[u] = acc;
        }
    }
}

// ---------------------------------------------------------------- dI for stride 1
// With s_h = s_w = 1 the input gradient is itself a convolution: zero-pad G by
// k_h - 1 rows and k_w - 1 columns on every side and correlate it with the
// kernel turned by 180 degrees and transposed, K'[a, b, m, c] =
// K[k_h-1-a, k_w-1-b, c, m]; its output is i_h x i_w. These two kernels form
// G' and K'; the slab products then run as for any forward convolution.
struct PadParams {
    const float* G;
    float* Gp;
    uint32_t units;          // 4-channel groups (or elements) of G'
    uint32_t o_h, o_w, k_c;  // G's shape
    uint32_t ph, pw;         // zero rows above and columns left of G in G'
    uint32_t hp, wp;         // G' rows and columns (G's rows and columns past them unused)
    FastDiv div_kc, div_wp, div_hp;
};

template <int V>
__global__ __launch_bounds__(kGradThreads) void pad_grad_kernel(PadParams p) {
    typedef float vec_t __attribute__((ext_vector_type(V)));
    const uint32_t stride = gridDim.x * kGradThreads;
    for (uint32_t u = blockIdx.x * kGradThreads + threadIdx.x; u < p.units; u += stride) {
        const uint32_t q = u * V;  // element of G'
        const uint32_t t = p.div_kc.div(q), m = q - t * p.k_c;
        const uint32_t t2 = p.div_wp.div(t), x = t - t2 * p.wp;
        const uint32_t n = p.div_hp.div(t2), y = t2 - n * p.hp;
        vec_t v = {};
        if (y >= p.ph && y < p.ph + p.o_h && x >= p.pw && x < p.pw + p.o_w)
            v = *reinterpret_cast<const vec_t*>(
                p.G + (((size_t)n * p.o_h + (y - p.ph)) * p.o_w + (x - p.pw)) * p.k_c + m);
        *reinterpret_cast<vec_t*>(p.Gp + q) = v;
    }
}

// The sub-kernel of sub-pixel phase (py, px) of the input gradient:
// K'[j, i, m, c] = K[py + s_h*(J-1-j), px + s_w*(I-1-i), c, m] for j < J, i < I
// (the kernel taps that reach the phase, turned by 180 degrees, with input and
// output channels swapped). Stride 1: K turned by 180 degrees and transposed.
// One thread per element of K'.
struct PhaseKernelParams {
    const float* K;
    float* Kp;
    uint32_t total, J, I, i_c, k_c, k_w, py, px, s_h, s_w;
};

__global__ __launch_bounds__(kGradThreads) void phase_kernel_kernel(PhaseKernelParams p) {
    const uint32_t stride = gridDim.x * kGradThreads;
    for (uint32_t e = blockIdx.x * kGradThreads + threadIdx.x; e < p.total; e += stride) {
        const uint32_t c = e % p.i_c, t = e / p.i_c;
        const uint32_t m = t % p.k_c, t2 = t / p.k_c;
        const uint32_t i = t2 % p.I, j = t2 / p.I;
        const uint32_t a = p.py + p.s_h * (p.J - 1 - j), bb = p.px + p.s_w * (p.I - 1 - i);
        p.Kp[e] = p.K[((a * p.k_w + bb) * p.i_c + c) * p.k_c + m];
    }
}

// ---------------------------------------------------------------- host side

inline bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }

template <int KT, int VW, int MAXU>
bool dgrad_config(const Shape& s, DgradParams& p) {
    p.hspan = (int32_t)((kDgRT + s.k_h - 2) / s.s_h + 1);
    p.gps = p.hspan * KT + 1;
    p.gunits = kPairs * p.hspan * (KT / VW);
    p.kbase = kPairs * p.gps;
    p.kunits = (int32_t)(s.k_h * kDgJT * (KT / VW));
    p.stage = p.kbase + (int32_t)(s.k_h * kDgJT * (KT + 1));
    if ((int64_t)p.gunits + p.kunits > (int64_t)MAXU * kGradThreads) return false;
    if ((size_t)p.stage * sizeof(float) > kDgLdsBudget) return false;
    p.nbuf = (size_t)2 * p.stage * sizeof(float) <= kDgLdsBudget ? 2 : 1;
    p.nchunks = (int32_t)((s.k_c + KT - 1) / KT);
    p.div_gu = FastDiv((uint32_t)(p.hspan * (KT / VW)));
    return true;
}

int64_t wgrad_tiles(const Shape& s) {
    return ((s.k_h * s.R + kWgJT - 1) / kWgJT) * ((s.k_c + kWgMT - 1) / kWgMT);
}

int64_t wgrad_stages(const Shape& s) {
    return ((s.pairs + kWgPT - 1) / kWgPT) * ((s.o_h + kWgHT - 1) / kWgHT);
}

}  // namespace

bool dgrad_supported(const Shape& s) {
    DgradParams p{};
    if (s.R > (int64_t(1) << 26) || s.k_h > 4096) return false;
    return dgrad_config<16, 1, 32>(s, p) || dgrad_config<8, 1, 32>(s, p) ||
           dgrad_config<2, 1, 32>(s, p);
}

hipError_t launch_dgrad_dl(const Shape& s, const float* G, const float* K, float* dL,
                           hipStream_t stream) {
    DgradParams p{};
    p.G = G;
    p.K = K;
    p.dL = dL;
    p.i_h = (int32_t)s.i_h;
    p.o_h = (int32_t)s.o_h;
    p.o_w = (int32_t)s.o_w;
    p.k_h = (int32_t)s.k_h;
    p.s_h = (int32_t)s.s_h;
    p.k_c = (int32_t)s.k_c;
    p.R = (int32_t)s.R;
    p.pairs = (int32_t)s.pairs;
    p.r_tiles = (int32_t)((s.i_h + kDgRT - 1) / kDgRT);
    p.j_tiles = (int32_t)((s.R + kDgJT - 1) / kDgJT);
    const int64_t ntiles = ((s.pairs + kPairs - 1) / kPairs) * p.r_tiles * p.j_tiles;
    if (ntiles > 0x7fffffff) return hipErrorInvalidValue;
    p.ntiles = (uint32_t)ntiles;
    // 16-byte loads when every chunk row starts on a 16-byte boundary; the
    // smallest prefetch that holds one stage (fewer registers, no spills);
    // double-buffered stages first, then single.
    const bool vec = s.k_c % 4 == 0 && ((uintptr_t)G & 15u) == 0 && ((uintptr_t)K & 15u) == 0;
#define MEC_DGRAD(KT, VW, MAXU)                                                                \
    if (dgrad_config<KT, VW, MAXU>(s, p) && p.nbuf >= min_buf) {                               \
        auto kern = dgrad_dl_kernel<KT, VW, MAXU>;                                             \
        hipLaunchKernelGGL(kern, dim3(p.ntiles), dim3(kGradThreads),                           \
                           (size_t)p.nbuf * p.stage * sizeof(float), stream, p);               \
        return hipGetLastError();                                                              \
    }
    for (int min_buf = 2; min_buf >= 1; --min_buf) {
        if (vec) {
            MEC_DGRAD(16, 4, 8)
            MEC_DGRAD(16, 4, 16)
            MEC_DGRAD(8, 4, 16)
            MEC_DGRAD(4, 4, 16)
        }
        MEC_DGRAD(16, 1, 32)
        MEC_DGRAD(8, 1, 32)
        MEC_DGRAD(2, 1, 32)
    }
#undef MEC_DGRAD
    return hipErrorInvalidValue;
}

hipError_t launch_fold(const Shape& s, const float* dL, float* dI, hipStream_t stream) {
    FoldParams p{};
    p.dL = dL;
    p.dI = dI;
    p.i_h = (uint32_t)s.i_h;
    p.i_w = (uint32_t)s.i_w;
    p.i_c = (uint32_t)s.i_c;
    p.k_w = (uint32_t)s.k_w;
    p.s_w = (uint32_t)s.s_w;
    p.o_w = (uint32_t)s.o_w;
    p.R = (uint32_t)s.R;
    p.div_ic = FastDiv(p.i_c);
    p.div_iw = FastDiv(p.i_w);
    p.div_ih = FastDiv(p.i_h);
    const int64_t elems = s.i_n * s.i_h * s.i_w * s.i_c;
    const bool vec = s.i_c % 4 == 0 && aligned16(dL) && aligned16(dI);
    p.units = (uint32_t)(vec ? elems / 4 : elems);
    int64_t blocks = ((int64_t)p.units + kGradThreads - 1) / kGradThreads;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    if (vec)
        hipLaunchKernelGGL(fold_kernel<4>, dim3((uint32_t)blocks), dim3(kGradThreads), 0, stream, p);
    else
        hipLaunchKernelGGL(fold_kernel<1>, dim3((uint32_t)blocks), dim3(kGradThreads), 0, stream, p);
    return hipGetLastError();
}

// The slab-reuse kernel serves k_h = 1, 3 and 5 when R is a multiple of 4,
// at least 48, and the staged rows fit its 8 LDS rows per pair; measured on
// the benchmark layers it beats the plain tiles where rows are short (R <= 256)
// or the kernel is 5 tall, and loses on long rows with few output tiles. The
// choice depends on the shape only, so the workspace query and the launch agree.
bool wgrad_slab_ok(const Shape& s) {
    return (s.k_h == 1 || s.k_h == 3 || s.k_h == 5) && s.R % 4 == 0 && s.R >= 48 &&
           (kWgHT - 1) * s.s_h + s.k_h <= kWsRows && (s.R <= 256 || s.k_h >= 5);
}

// Shares of the (pair, output row) reduction per dK tile. The time of the
// products is set by the busiest compute unit: it holds ceil(tiles * splits /
// 256) workgroups (the workspace size must not depend on the device, so the
// 256 compute units of the MI355X are assumed), each running ceil(stages /
// splits) stages one after another on shared SIMDs. Every share adds its
// partial tile to write and to read back in the reduction. The count that
// minimises the sum of the two, measured on this GPU: a stage costs the
// products of one wave (32 k-steps x KH 64-cycle MFMAs in the slab kernel, 32
// x 2 in the general one), a partial sum 8 bytes per element at 5 TB/s, with
// the occupancy factors below. Choosing the
// share count by workgroup count alone (about 512 or 1024) left 1 to 3
// workgroups beyond whole rounds on some compute units: resnet_mid's 3 tiles
// in 171 shares, 513 workgroups, ran 124.6 us against 91.0 us in 170 (cv8
// 813 -> 547 us, cv4 2049 -> 1741 us, alexnet_conv1 645 -> 523 us).
int64_t wgrad_splits(const Shape& s) {
    const int64_t stages = wgrad_stages(s);
    const int64_t E = s.k_h * s.R * s.k_c;
    const bool slab = wgrad_slab_ok(s);
    const int64_t tiles = slab ? ((s.R + kWs - 1) / kWs) * ((s.k_c + kWs - 1) / kWs) : wgrad_tiles(s);
    // partial sums within 32 MiB (slab) or 256 MiB
    int64_t cap = slab ? (int64_t(8) << 20) / E : (int64_t(64) << 20) / E;
    if (cap > stages) cap = stages;  // at most one share per stage
    if (cap > 1024) cap = 1024;
    if (cap < 1) return 1;
    const double stage_us = (slab ? 32.0 * s.k_h : 64.0) * 64.0 / 2400.0;
    const double share_us = 8.0 * (double)E / 5.0e6;
    int64_t best = 1;
    double best_t = 0.0;
    for (int64_t sp = 1; sp <= cap; ++sp) {
        const int64_t per_cu = (tiles * sp + 255) / 256;
        double t = (double)per_cu * (double)((stages + sp - 1) / sp) * stage_us + (double)sp * share_us;
        // one workgroup per compute unit leaves one wave per SIMD; the general
        // kernel fits three per compute unit and runs best with three
        if (per_cu == 1) t *= 1.25;
        if (per_cu == 2 && !slab) t *= 1.07;
        if (sp == 1 || t < best_t) {
            best = sp;
            best_t = t;
        }
    }
    return best;
}

int64_t wgrad_partial_bytes(const Shape& s) {
    return wgrad_splits(s) * s.k_h * s.R * s.k_c * (int64_t)sizeof(float);
}

bool wgrad_supported(const Shape& s) {
    const int64_t E = s.k_h * s.R * s.k_c;
    return E < (int64_t(1) << 30) && s.k_h * s.R < (int64_t(1) << 30) &&
           wgrad_stages(s) < (int64_t(1) << 30) && s.pairs < (int64_t(1) << 30) &&
           wgrad_tiles(s) * wgrad_splits(s) < (int64_t(1) << 31);
}

hipError_t launch_wgrad(const Shape& s, const float* L, const float* G, float* part, float* dK,
                        hipStream_t stream, bool fused) {
    WgradParams p{};
    p.L = L;
    p.fused = fused;
    p.i_w = (int32_t)s.i_w;
    p.i_c = (int32_t)s.i_c;
    p.s_w = (int32_t)s.s_w;
    p.G = G;
    p.part = part;
    p.i_h = (int32_t)s.i_h;
    p.o_h = (int32_t)s.o_h;
    p.o_w = (int32_t)s.o_w;
    p.k_c = (int32_t)s.k_c;
    p.s_h = (int32_t)s.s_h;
    p.R = (int32_t)s.R;
    p.KD = (int32_t)(s.k_h * s.R);
    p.pairs = (int32_t)s.pairs;
    p.h_chunks = (int32_t)((s.o_h + kWgHT - 1) / kWgHT);
    p.nstages = (int32_t)wgrad_stages(s);
    p.splits = (int32_t)wgrad_splits(s);
    p.lvec = s.R % 4 == 0 && aligned16(L) && (!fused || s.i_c % 4 == 0);
    p.gvec = s.k_c % 4 == 0 && aligned16(G);
    p.div_ow = FastDiv((uint32_t)s.o_w);
    p.div_R = FastDiv((uint32_t)s.R);
    if (wgrad_slab_ok(s)) {
        p.j_tiles = (int32_t)((s.R + kWs - 1) / kWs);
        p.m_tiles = (int32_t)((s.k_c + kWs - 1) / kWs);
        p.ntiles = (uint32_t)((int64_t)p.j_tiles * p.m_tiles * p.splits);
        const bool vec = p.lvec && p.gvec;
#define MEC_WGS(KH)                                                                            \
    if (s.k_h == KH) {                                                                         \
        auto kern = vec ? wgrad_slab_kernel<KH, true> : wgrad_slab_kernel<KH, false>;          \
        hipLaunchKernelGGL(kern, dim3(p.ntiles), dim3(kGradThreads), 0, stream, p);            \
    }
        MEC_WGS(1) MEC_WGS(3) MEC_WGS(5)
#undef MEC_WGS
    } else {
        p.j_tiles = (int32_t)((p.KD + kWgJT - 1) / kWgJT);
        p.m_tiles = (int32_t)((s.k_c + kWgMT - 1) / kWgMT);
        p.ntiles = (uint32_t)((int64_t)p.j_tiles * p.m_tiles * p.splits);
        hipLaunchKernelGGL(wgrad_kernel, dim3(p.ntiles), dim3(kGradThreads), 0, stream, p);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t E = (int64_t)p.KD * s.k_c;
    const bool vec = E % 4 == 0 && aligned16(part) && aligned16(dK);
    const uint32_t units = (uint32_t)(vec ? E / 4 : E);
    const uint32_t ublocks = (units + kGradThreads - 1) / kGradThreads;
    // groups of about 8 consecutive shares, at most 64 groups; with 8 shares
    // or fewer every share is its own group and pass 1 is skipped
    int32_t groups = p.splits <= 8 ? p.splits : (p.splits + 7) / 8;
    if (groups > 64) groups = 64;
    if (groups < p.splits) {
        if (vec)
            hipLaunchKernelGGL(wgrad_reduce_groups_kernel<4>, dim3(ublocks, groups), dim3(kGradThreads),
                               0, stream, part, units, (uint32_t)E, p.splits, groups);
        else
            hipLaunchKernelGGL(wgrad_reduce_groups_kernel<1>, dim3(ublocks, groups), dim3(kGradThreads),
                               0, stream, part, units, (uint32_t)E, p.splits, groups);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    int64_t blocks = ublocks;
    if (blocks > 65536) blocks = 65536;
    if (vec)
        hipLaunchKernelGGL(wgrad_reduce_kernel<4>, dim3((uint32_t)blocks), dim3(kGradThreads), 0,
                           stream, part, dK, units, (uint32_t)E, p.splits, groups);
    else
        hipLaunchKernelGGL(wgrad_reduce_kernel<1>, dim3((uint32_t)blocks), dim3(kGradThreads), 0,
                           stream, part, dK, units, (uint32_t)E, p.splits, groups);
    return hipGetLastError();
}

// Sub-pixel phase (py, px) of the input gradient: the pixels
// dI[n, s_h*Y + py, s_w*X + px, :] receive G through the kernel taps
// a = py + s_h*j (j < J) and b = px + s_w*i (i < I) only:
//   dI[n, s_h*Y+py, s_w*X+px, c] = sum_{j,i,m} G[n, Y-j, X-i, m] K[py+s_h*j, px+s_w*i, c, m]
// (G zero outside its o_h x o_w), which is a stride-1 correlation of G
// zero-padded by J-1 rows above and I-1 columns to the left with the
// sub-kernel K' of phase_kernel_kernel. Stride 1 has one phase: G padded by
// k-1 on every side, K turned by 180 degrees and transposed.
struct Phase {
    Shape t;          // the phase's stride-1 convolution
    int64_t py, px;   // which phase
    int64_t gp_elems; // padded G
};

Phase dgrad_phase(const Shape& s, int64_t py, int64_t px) {
    Phase ph{};
    ph.py = py;
    ph.px = px;
    const int64_t J = (s.k_h - py + s.s_h - 1) / s.s_h, I = (s.k_w - px + s.s_w - 1) / s.s_w;
    const int64_t Ny = (s.i_h - py + s.s_h - 1) / s.s_h, Nx = (s.i_w - px + s.s_w - 1) / s.s_w;
    Shape& t = ph.t;
    t.i_n = s.i_n;
    t.i_h = Ny + J - 1;
    t.i_w = Nx + I - 1;
    t.i_c = s.k_c;
    t.k_h = J;
    t.k_w = I;
    t.k_c = s.i_c;
    t.s_h = t.s_w = 1;
    t.o_h = Ny;
    t.o_w = Nx;
    t.R = t.k_w * t.i_c;
    t.pairs = t.i_n * t.o_w;
    ph.gp_elems = t.i_n * t.i_h * t.i_w * t.i_c;
    return ph;
}

// Where phase (py, px) writes in dI (nullptr: dense, stride 1).
OutLayout phase_layout(const Shape& s, const Phase& ph) {
    OutLayout o{};
    o.img = s.i_h * s.i_w * s.i_c;
    o.row = s.s_h * s.i_w * s.i_c;
    o.col = s.s_w * s.i_c;
    o.off = (ph.py * s.i_w + ph.px) * s.i_c;
    return o;
}

// Taken for i_c >= 32 (the phases' output channels) and, at stride 1, kernels
// up to 3x3: measured on the benchmark layers it beats the dL path there (cv9
// 1.4x, cv8 1.26x, resnet_mid 1.2x) and loses on 5x5 kernels (cv5) and on
// few-channel outputs. Strided (s <= k, every phase reaches some tap): k_c and
// i_c multiples of 4 and phase kernel heights up to 5, so that every phase has
// a fixed kernel with 16-byte rows that takes a strided output layout, and at
// most 4 phases of at least 10 taps each on average: the phases run one after
// another as small convolutions, and measured faster than the dL path for
// 7x7 stride 2 (cv4: 4.85 -> 1.77 ms, workspace 1.3 GB -> 104 MB) but slower
// for 3x3 (1.0-1.7x) and 5x5 (2.9x) stride 2.
bool dgrad_phases_ok(const Shape& s) {
    if (s.i_c < 32) return false;
    if (s.k_h * s.k_w * s.i_c * s.k_c >= (int64_t(1) << 31)) return false;
    const bool unit = s.s_h == 1 && s.s_w == 1;
    if (unit && (s.k_h > 3 || s.k_w > 3)) return false;
    if (!unit && (s.s_h > s.k_h || s.s_w > s.k_w || s.k_c % 4 || s.i_c % 4 ||
                  (s.k_h + s.s_h - 1) / s.s_h > 5))
        return false;  // phase kernels with 16-byte rows, heights 1-5
    if (!unit && (s.k_h * s.k_w < 10 * s.s_h * s.s_w || s.s_h * s.s_w > 4))
        return false;  // phases too small: one small launch each
    if (s.i_n * s.i_h * s.i_w * s.i_c >= (int64_t(1) << 31)) return false;
    for (int64_t py = 0; py < s.s_h; ++py)
        for (int64_t px = 0; px < s.s_w; ++px) {
            const Phase ph = dgrad_phase(s, py, px);
            if (ph.gp_elems >= (int64_t(1) << 31) || ph.t.R > (int64_t(1) << 26)) return false;
            if (unit) {
                if (!gemm_supported(ph.t, 0, true)) return false;
            } else {
                const OutLayout o = phase_layout(s, ph);
                if (launch_gemm_fixed(ph.t, nullptr, nullptr, nullptr, 0, true, nullptr, true, &o) !=
                    hipSuccess)
                    return false;
            }
        }
    return true;
}

namespace {
// workspace: from its first 16-byte boundary (the caller guarantees 4-byte
// alignment), the largest phase's padded G (rounded to 256 bytes), then the
// largest K'
int64_t phases_gp_bytes(const Shape& s) {
    int64_t gp = 0;
    for (int64_t py = 0; py < s.s_h; ++py)
        for (int64_t px = 0; px < s.s_w; ++px) {
            const int64_t e = dgrad_phase(s, py, px).gp_elems;
            if (e > gp) gp = e;
        }
    return (gp * 4 + 255) / 256 * 256;
}
}  // namespace

int64_t dgrad_workspace_bytes(const Shape& s) {
    if (!dgrad_phases_ok(s)) return s.i_n * s.o_w * s.i_h * s.k_w * s.i_c * 4;  // dL
    int64_t kp = 0;
    for (int64_t py = 0; py < s.s_h; ++py)
        for (int64_t px = 0; px < s.s_w; ++px) {
            const Shape& t = dgrad_phase(s, py, px).t;
            if (t.k_h * t.k_w * t.i_c * t.k_c > kp) kp = t.k_h * t.k_w * t.i_c * t.k_c;
        }
    return 12 + phases_gp_bytes(s) + kp * 4;
}

hipError_t launch_dgrad_phases(const Shape& s, const float* G, const float* K, float* dI,
                               void* workspace, hipStream_t stream) {
    char* base = static_cast<char*>(workspace) + ((16 - ((uintptr_t)workspace & 15u)) & 15u);
    float* Gp = reinterpret_cast<float*>(base);
    float* Kp = reinterpret_cast<float*>(base + phases_gp_bytes(s));
    const bool unit = s.s_h == 1 && s.s_w == 1;
    for (int64_t py = 0; py < s.s_h; ++py)
        for (int64_t px = 0; px < s.s_w; ++px) {
            const Phase ph = dgrad_phase(s, py, px);
            const Shape& t = ph.t;
            PadParams p{};
            p.G = G;
            p.Gp = Gp;
            p.o_h = (uint32_t)s.o_h;
            p.o_w = (uint32_t)s.o_w;
            p.k_c = (uint32_t)s.k_c;
            p.ph = (uint32_t)(t.k_h - 1);
            p.pw = (uint32_t)(t.k_w - 1);
            p.hp = (uint32_t)t.i_h;
            p.wp = (uint32_t)t.i_w;
            p.div_kc = FastDiv(p.k_c);
            p.div_wp = FastDiv(p.wp);
            p.div_hp = FastDiv(p.hp);
            const bool vec = s.k_c % 4 == 0 && aligned16(G) && aligned16(Gp);
            p.units = (uint32_t)(vec ? ph.gp_elems / 4 : ph.gp_elems);
            int64_t blocks = ((int64_t)p.units + kGradThreads - 1) / kGradThreads;
            if (blocks > 65536) blocks = 65536;
            if (vec)
                hipLaunchKernelGGL(pad_grad_kernel<4>, dim3((uint32_t)blocks), dim3(kGradThreads), 0,
                                   stream, p);
            else
                hipLaunchKernelGGL(pad_grad_kernel<1>, dim3((uint32_t)blocks), dim3(kGradThreads), 0,
                                   stream, p);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            PhaseKernelParams q{};
            q.K = K;
            q.Kp = Kp;
            q.total = (uint32_t)(t.k_h * t.k_w * t.i_c * t.k_c);
            q.J = (uint32_t)t.k_h;
            q.I = (uint32_t)t.k_w;
            q.i_c = (uint32_t)s.i_c;
            q.k_c = (uint32_t)s.k_c;
            q.k_w = (uint32_t)s.k_w;
            q.py = (uint32_t)py;
            q.px = (uint32_t)px;
            q.s_h = (uint32_t)s.s_h;
            q.s_w = (uint32_t)s.s_w;
            int64_t kblocks = ((int64_t)q.total + kGradThreads - 1) / kGradThreads;
            if (kblocks > 65536) kblocks = 65536;
            hipLaunchKernelGGL(phase_kernel_kernel, dim3((uint32_t)kblocks), dim3(kGradThreads), 0,
                               stream, q);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
            const OutLayout o = phase_layout(s, ph);
            e = launch_gemm(t, Gp, Kp, dI, 0, true, stream, unit ? nullptr : &o);
            if (e != hipSuccess) return e;
        }
    return hipSuccess;
}

// ---------------------------------------------------------------- no-alloc weight gradient
// The partial sums of the weight gradient in a static device array instead of
// a caller's workspace, for callers that cannot allocate device memory. Each
// GPU the library runs on holds its own copy until the process ends. Host code
// never passes `scratch` itself to a kernel (in host code the name is a
// host-side stand-in, not a device address): it uses the address that
// hipGetSymbolAddress returns for the stream's device, taken once per device
// with that device current.
static __device__ __align__(256) float scratch[kNoAllocScratchBytes / sizeof(float)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // per device, set once under g_scratch_mu
}  // namespace

hipError_t noalloc_scratch(hipStream_t stream, void** ptr) {
    int dev = 0;
    hipError_t e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        int cur = 0;
        e = hipGetDevice(&cur);
        if (e != hipSuccess) return e;
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev) {
            const hipError_t e2 = hipSetDevice(cur);
            if (e == hipSuccess) e = e2;
        }
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace mec
