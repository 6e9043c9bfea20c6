// bf16 conv2d through an internal channel-last layout.
//
// The bf16 MFMA (v_mfma_f32_32x32x16_bf16) wants 8 consecutive reduction
// elements per lane.  With the reduction ordered (r, s, c), c innermost, and
// the activations channel-last, those 8 elements are 8 adjacent channels of
// one input pixel: one aligned 16-byte load, one padding check.  So a call
//  1. transposes x from NCHW to an internal NHWC copy (x_cl, one HBM pass,
//     through LDS so both the reads and the writes are contiguous),
//  2. reads filters packed KRSC (w_p[k][(r*S+s)*Cg + c], packed once by the
//     stack executor or per call),
//  3. runs the implicit GEMM D[k][m] = sum_kr W[k][kr] X[kr][m] with both
//     operand tiles staged reduction-contiguous in LDS (rows padded by 16
//     bytes: conflict-free 16-byte reads), double-buffered, MFMA 32x32x16,
//     and stores y in NCHW fp32 with bias + activation.
// Requirements: C/groups % KRC == 0 (every reduction chunk of KRC elements
// is KRC channels at one filter position), so the chunk's (r, s) is uniform.
#include "internal.h"

#include <cstdio>

namespace miconv {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// x [N][C][H][W] -> x_cl [N][P][Q][C], where P x Q are the pixels the conv
// reads in channel-last form: all of them (P = H, Q = W, S = 1), or, for a
// 1x1 stride-S layer without padding, only the ones it samples (row p*S,
// column q*S), so the layer then runs as a stride-1 conv on a P x Q image
// and reads 1/S^2 of x.  The pixel axis is flattened over images (a tile of
// 64 pixels may span images), so small planes waste no lanes.  A
// work-group moves 64 channels x 64 pixels through LDS: a lane reads RV
// consecutive pixels of one channel per load (RV = 8 or 4 when S = 1 and
// H*W and the base address allow it; 1 otherwise) and writes 8 channels of
// one pixel per 16-byte store (C % 8 == 0 on every path that uses it).
struct NhwcCopyArgs {
    const uint16_t *x;
    uint16_t *xt;
    int C, H, W, Q, S, HW, PQ;
    int npq;             // N * P * Q
    int tiles_c;
    int cb;              // channels per work-group (whole-plane kernel)
    FastDiv dv_hw, dv_pq, dv_q;
};

// Writes a staged tile ([64 channels][64 pixels], channel row c at row
// c ^ ((c >> 3) & 7)) to the channel-last copy: a lane gathers 8 channels of
// one pixel and stores them as 16 bytes.
__device__ __forceinline__ void copy_tile_out(const NhwcCopyArgs &a, const uint16_t (*tile)[64 + 8], int c0,
                                              int p0, int t)
{
    auto row = [](int c) { return c ^ ((c >> 3) & 7); };
#pragma unroll
    for (int i = 0; i < 64 / 32; ++i) {   // 64 pixels x 8 channel octets
        const int id = t + 256 * i;
        const int px = id >> 3, o = id & 7;
        if (c0 + 8 * o < a.C && p0 + px < a.npq) {
            uint32_t d[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                d[e] = (uint32_t)tile[row(8 * o + 2 * e)][px] | ((uint32_t)tile[row(8 * o + 2 * e + 1)][px] << 16);
            *reinterpret_cast<uint4 *>(a.xt + (long)(p0 + px) * a.C + c0 + 8 * o) =
                make_uint4(d[0], d[1], d[2], d[3]);
        }
    }
}

template <int RV>
__global__ __launch_bounds__(256) void nchw_to_nhwc_bf16_kernel(NhwcCopyArgs a)
{
    constexpr int PX = 64;
    // [channel][pixel]; channel row c is stored at row c ^ ((c >> 3) & 7), so
    // the transposed reads (8 lanes on channel rows 8*o + e, o = 0..7) fall in
    // 8 distinct bank groups
    __shared__ __attribute__((aligned(16))) uint16_t tile[64][PX + 8];
    auto row = [](int c) { return c ^ ((c >> 3) & 7); };
    const int t = threadIdx.x;
    const int c0 = (blockIdx.x % a.tiles_c) * 64;
    const int p0 = (blockIdx.x / a.tiles_c) * PX;
    if constexpr (RV > 1) {
        constexpr int GR = PX / RV;                 // pixel groups per channel row
#pragma unroll
        for (int i = 0; i < 64 * GR / 256; ++i) {
            const int id = t + 256 * i;
            const int c = id / GR, o = id % GR;
            const int px = p0 + RV * o;             // a group never spans images: H*W % RV == 0
            const bool ok = c0 + c < a.C && px < a.npq;
            const unsigned n = fdiv(ok ? px : 0, a.dv_hw);
            const uint16_t *src = a.x + ((long)n * a.C + c0 + c) * a.HW + (px - (int)n * a.HW);
            if constexpr (RV == 8) {
                const uint4 v = ok ? *reinterpret_cast<const uint4 *>(src) : make_uint4(0, 0, 0, 0);
                *reinterpret_cast<uint4 *>(&tile[row(c)][8 * o]) = v;
            } else {
                const uint2 v = ok ? *reinterpret_cast<const uint2 *>(src) : make_uint2(0, 0);
                *reinterpret_cast<uint2 *>(&tile[row(c)][4 * o]) = v;
            }
        }
    } else {
#pragma unroll
        for (int sub = 0; sub < PX / 64; ++sub) {
            const int px = p0 + 64 * sub + (t & 63);
            const bool pok = px < a.npq;
            const unsigned n = fdiv(pok ? px : 0, a.dv_pq);
            const unsigned pq = (pok ? px : 0) - n * a.PQ;
            const unsigned pp = fdiv(pq, a.dv_q);
            const unsigned q = pq - pp * a.Q;
            const long off = (long)(pp * a.S) * a.W + q * a.S;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int c = (t >> 6) + 4 * i;
                const bool ok = pok && c0 + c < a.C;
                tile[row(c)][64 * sub + (t & 63)] = ok ? a.x[((long)n * a.C + c0 + c) * a.HW + off] : 0;
            }
        }
    }
    __syncthreads();
    copy_tile_out(a, tile, c0, p0, t);
}

// Stride-2 subsampling copy (1x1 stride-2 layers) reading G sampled pixels
// per load: output pixels q .. q+G-1 of a row sample input columns 2q ..
// 2q+2G-2, so one 4G-byte load of 2G consecutive input pixels holds them at
// its even positions.  Requires Q % G == 0 (a group stays in one output row),
// W % G == 0 and H*W % 2G == 0 (every load aligned) and W = 2Q (a load never
// passes the end of its input row).
template <int G>
__global__ __launch_bounds__(256) void nchw_to_nhwc_sampled_bf16_kernel(NhwcCopyArgs a)
{
    static_assert(G == 2 || G == 4, "8- or 16-byte loads");
    constexpr int PX = 64;
    __shared__ __attribute__((aligned(16))) uint16_t tile[64][PX + 8];
    auto row = [](int c) { return c ^ ((c >> 3) & 7); };
    const int t = threadIdx.x;
    const int c0 = (blockIdx.x % a.tiles_c) * 64;
    const int p0 = (blockIdx.x / a.tiles_c) * PX;
    constexpr int GR = PX / G;                  // sampled groups per channel row
#pragma unroll
    for (int i = 0; i < 64 * GR / 256; ++i) {
        const int id = t + 256 * i;
        const int c = id / GR, o = id % GR;
        const int px = p0 + G * o;
        const bool ok = c0 + c < a.C && px < a.npq;
        const unsigned m = ok ? px : 0;
        const unsigned n = fdiv(m, a.dv_pq);
        const unsigned pq = m - n * a.PQ;
        const unsigned pp = fdiv(pq, a.dv_q);
        const unsigned q = pq - pp * a.Q;
        const uint16_t *src = a.x + ((long)n * a.C + c0 + c) * a.HW + (long)(2 * pp) * a.W + 2 * q;
        if constexpr (G == 4) {
            const uint4 v = ok ? *reinterpret_cast<const uint4 *>(src) : make_uint4(0, 0, 0, 0);
            *reinterpret_cast<uint2 *>(&tile[row(c)][4 * o]) =
                make_uint2((v.x & 0xFFFFu) | (v.y << 16), (v.z & 0xFFFFu) | (v.w << 16));
        } else {
            const uint2 v = ok ? *reinterpret_cast<const uint2 *>(src) : make_uint2(0, 0);
            *reinterpret_cast<uint32_t *>(&tile[row(c)][2 * o]) = (v.x & 0xFFFFu) | (v.y << 16);
        }
    }
    __syncthreads();
    copy_tile_out(a, tile, c0, p0, t);
}

// Small planes (32*H*W <= kPlaneElems): a work-group moves one image's block
// of cb channels (64, or fewer so that the block fits in LDS and the grid
// still fills the chip; a multiple of 8).  In NCHW that block, [cb][H][W], is one contiguous run of cb*H*W
// values, so it is read with 16-byte loads whatever H*W is (no pixel group of
// a load can straddle two images), staged in LDS as is, and each lane then
// gathers 8 channels of one sampled pixel from LDS and writes them as one
// 16-byte store.  Requires C % 8 == 0 and a 16-byte aligned x.
constexpr int kPlaneElems = 16384;    // 32 KB of LDS

__global__ __launch_bounds__(256) void nchw_to_nhwc_plane_bf16_kernel(NhwcCopyArgs a)
{
    __shared__ __attribute__((aligned(16))) uint16_t plane[kPlaneElems];
    const int t = threadIdx.x;
    const int n = blockIdx.x / a.tiles_c;
    const int c0 = (blockIdx.x % a.tiles_c) * a.cb;
    const int cn = min(a.cb, a.C - c0);                // a multiple of 8
    const uint4 *src = reinterpret_cast<const uint4 *>(a.x + ((long)n * a.C + c0) * a.HW);
    const int units = cn * a.HW / 8;
    uint4 *dst = reinterpret_cast<uint4 *>(plane);
    for (int u = t; u < units; u += 256) dst[u] = src[u];
    __syncthreads();
    const int oct = cn / 8;
    uint16_t *out = a.xt + (long)n * a.PQ * a.C + c0;
    for (int id = t; id < a.PQ * oct; id += 256) {
        const int pq = id / oct, o = id - pq * oct;
        const int pp = (int)fdiv((unsigned)pq, a.dv_q);
        const int hw = pp * a.S * a.W + (pq - pp * a.Q) * a.S;
        const uint16_t *col = plane + 8 * o * a.HW + hw;
        uint32_t d[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
            d[e] = (uint32_t)col[2 * e * a.HW] | ((uint32_t)col[(2 * e + 1) * a.HW] << 16);
        *reinterpret_cast<uint4 *>(out + (long)pq * a.C + 8 * o) = make_uint4(d[0], d[1], d[2], d[3]);
    }
}

// MFMA roles: the pixel tile is the MFMA's A operand (rows i) and the filter
// tile its B operand (columns j), so accumulator register v of lane l holds
// pixel 8*(v/4) + 4*(l/32) + v%4 of column (channel) l%32: four consecutive
// output pixels of one channel per group of 4 registers, stored as one
// 16-byte write when the plane size allows.
//
// Pipeline: two LDS stages plus two chunks of global loads held in
// registers, so while the wavefronts multiply chunk t, chunks t+1 and t+2
// are in flight.
template <int R_, int S_, int BKC, int BPX, int KRC>
__global__ __launch_bounds__(256) void igemm_bf16_nhwc_kernel(ConvArgs a)
{
    constexpr int NT = 256;
    constexpr int WTK = BKC / 2, WTP = BPX / 2;      // 2 x 2 wavefronts
    constexpr int BI = WTK / 32, BJ = WTP / 32;      // channel blocks, pixel blocks
    constexpr int LDR = KRC + 8;                     // row stride in bf16 (16-byte pad)
    constexpr int G8 = KRC / 8;                      // 8-element groups per row chunk
    constexpr int A_PER = BKC * G8 / NT;             // groups per lane
    constexpr int B_PER = BPX * G8 / NT;
    static_assert(BI >= 1 && BJ >= 1 && A_PER >= 1 && B_PER >= 1, "tile shape");
    static_assert((BKC * G8) % NT == 0 && (BPX * G8) % NT == 0 && NT % G8 == 0, "loader shape");

    __shared__ __attribute__((aligned(16))) uint16_t As[2][BKC][LDR];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BPX][LDR];

    const uint16_t *__restrict__ xcl = static_cast<const uint16_t *>(a.x);   // [N][H][W][C]
    const uint16_t *__restrict__ wp = static_cast<const uint16_t *>(a.w);    // [K][R][S][Cg]
    const int S = S_ ? S_ : a.S;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wk = wid >> 1, wq = wid & 1;
    const int h = lane >> 5, ll = lane & 31;
    const int g = blockIdx.z % a.groups;
    const int split = blockIdx.z / a.groups;
    const int m0 = blockIdx.x * BPX;
    const int k0 = blockIdx.y * BKC;
    const int kr_begin = split * a.kr_per_split;
    const int kr_end = min(a.Kred, kr_begin + a.kr_per_split);

    // Loader lanes: group column j8 = tid % G8 (8 channels), row = tid / G8 + i * RSTEP.
    const int j8 = tid % G8;
    const int row0 = tid / G8;
    constexpr int RSTEP = NT / G8;

    const uint16_t *arow[A_PER];
    bool aok[A_PER];
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
        const int k = k0 + row0 + i * RSTEP;
        aok[i] = k < a.Kg;
        arow[i] = wp + ((long)g * a.Kg + (aok[i] ? k : 0)) * a.Kred + j8 * 8;
    }
    int bih[B_PER], biw[B_PER];
    long bbase[B_PER];
    bool bok[B_PER];
#pragma unroll
    for (int i = 0; i < B_PER; ++i) {
        const int m = m0 + row0 + i * RSTEP;
        bok[i] = m < a.M;
        const int mm = bok[i] ? m : 0;
        const int n = mm / a.PQ;
        const int pq = mm - n * a.PQ;
        const int p = pq / a.Q;
        const int q = pq - p * a.Q;
        bih[i] = p * a.stride - a.pad;
        biw[i] = q * a.stride - a.pad;
        bbase[i] = (long)n * a.H * a.W * a.C + (long)g * a.Cg + j8 * 8;
    }

    struct Regs {
        uint4 a[A_PER], b[B_PER];
    };
    auto gload = [&](Regs &rg, int t) {
        const int kr0 = kr_begin + t * KRC;
        // the chunk [kr0, kr0 + KRC) is KRC channels at filter position rs
        const int rs = kr0 / a.Cg;
        const int c0 = kr0 - rs * a.Cg;
        const int r = rs / S;
        const int s = rs - r * S;
        const bool live = kr0 < kr_end;
#pragma unroll
        for (int i = 0; i < A_PER; ++i)
            rg.a[i] = (live && aok[i]) ? *reinterpret_cast<const uint4 *>(arow[i] + kr0)
                                       : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int i = 0; i < B_PER; ++i) {
            const int ih = bih[i] + r, iw = biw[i] + s;
            const bool ok = live && bok[i] && (unsigned)ih < (unsigned)a.H &&
                            (unsigned)iw < (unsigned)a.W;
            rg.b[i] = ok ? *reinterpret_cast<const uint4 *>(xcl + bbase[i] +
                                                            ((long)ih * a.W + iw) * a.C + c0)
                         : make_uint4(0, 0, 0, 0);
        }
    };
    auto sstore = [&](const Regs &rg, int buf) {
#pragma unroll
        for (int i = 0; i < A_PER; ++i)
            *reinterpret_cast<uint4 *>(&As[buf][row0 + i * RSTEP][j8 * 8]) = rg.a[i];
#pragma unroll
        for (int i = 0; i < B_PER; ++i)
            *reinterpret_cast<uint4 *>(&Bs[buf][row0 + i * RSTEP][j8 * 8]) = rg.b[i];
    };

    // acc[bj][bi]: rows = pixel block bj, columns = channel block bi
    floatx16 acc[BJ][BI];
#pragma unroll
    for (int bj = 0; bj < BJ; ++bj)
#pragma unroll
        for (int bi = 0; bi < BI; ++bi)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[bj][bi][v] = 0.f;

    auto compute = [&](int buf) {
#pragma unroll
        for (int ks = 0; ks < KRC; ks += 16) {
            bf16x8 wv[BI], xv[BJ];
#pragma unroll
            for (int bi = 0; bi < BI; ++bi)
                wv[bi] = *reinterpret_cast<const bf16x8 *>(&As[buf][wk * WTK + bi * 32 + ll][ks + 8 * h]);
#pragma unroll
            for (int bj = 0; bj < BJ; ++bj)
                xv[bj] = *reinterpret_cast<const bf16x8 *>(&Bs[buf][wq * WTP + bj * 32 + ll][ks + 8 * h]);
#pragma unroll
            for (int bj = 0; bj < BJ; ++bj)
#pragma unroll
                for (int bi = 0; bi < BI; ++bi)
                    acc[bj][bi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xv[bj], wv[bi], acc[bj][bi],
                                                                         0, 0, 0);
        }
    };

    const int nchunks = kr_end > kr_begin ? (kr_end - kr_begin) / KRC : 0;
    Regs r0, r1;
    if (nchunks > 0) {
        gload(r0, 0);
        gload(r1, 1);          // beyond the last chunk the loads are masked to zero
        sstore(r0, 0);
        gload(r0, 2);
    }
    __syncthreads();
    // Step t: the register set holding chunk t+1 goes to LDS stage (t+1)&1 and
    // is refilled with chunk t+3, then stage t&1 is multiplied.  The loop is
    // unrolled by two so that each register set has a fixed role (a runtime
    // choice between them would push both into scratch memory).
    auto step = [&](int t, Regs &nx) {
        if (t + 1 < nchunks) sstore(nx, (t + 1) & 1);
        if (t + 3 < nchunks) gload(nx, t + 3);
        compute(t & 1);
        __syncthreads();
    };
    for (int t = 0; t < nchunks; t += 2) {
        step(t, r1);
        if (t + 1 < nchunks) step(t + 1, r0);
    }

    // Epilogue: lane l holds channel column l%32 and, per group of 4
    // registers, 4 consecutive pixels.
    const bool vec = a.splits == 1 && (a.PQ & 3) == 0 && ((uintptr_t)a.y & 15) == 0 && (a.ysn & 3) == 0;
    const long cstride = a.splits > 1 ? (long)a.M : (long)a.PQ;
    float *out = a.splits > 1 ? a.ws + (long)split * a.K * a.M : a.y;
#pragma unroll
    for (int bi = 0; bi < BI; ++bi) {
        const int k = k0 + wk * WTK + bi * 32 + ll;
        if (k >= a.Kg) continue;
        const int kg = g * a.Kg + k;
        const float bv = (a.splits == 1 && a.bias) ? a.bias[kg] : 0.f;
        const long coff = (long)kg * cstride;
#pragma unroll
        for (int bj = 0; bj < BJ; ++bj) {
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int mb = m0 + wq * WTP + bj * 32 + 8 * q4 + 4 * h;   // first of 4 pixels
                float v4[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float val = acc[bj][bi][4 * q4 + e];
                    if (a.splits == 1) {
                        val += bv;
                        if (a.relu && !a.res) val = fmaxf(val, 0.f);
                    }
                    v4[e] = val;
                }
                if (vec && mb + 3 < a.M) {
                    const int n = mb / a.PQ;
                    const long off = (long)n * a.ysn + (mb - n * a.PQ) + coff;
                    if (a.res) {
                        const float4 r = *reinterpret_cast<const float4 *>(a.res + off);
                        const float re[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            v4[e] += re[e];
                            if (a.relu) v4[e] = fmaxf(v4[e], 0.f);
                        }
                    }
                    *reinterpret_cast<float4 *>(out + off) = make_float4(v4[0], v4[1], v4[2], v4[3]);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int m = mb + e;
                        if (m >= a.M) continue;
                        const int n = m / a.PQ;
                        const long off = a.splits > 1 ? (long)m + coff
                                                      : (long)n * a.ysn + (m - n * a.PQ) + coff;
                        float val = v4[e];
                        if (a.splits == 1 && a.res) {
                            val += a.res[off];
                            if (a.relu) val = fmaxf(val, 0.f);
                        }
                        out[off] = val;
                    }
                }
            }
        }
    }
}

// Direct-to-LDS variant (64-channel reduction chunks).  Every lane's
// global_load_lds_dwordx4 writes its 16 bytes straight into LDS, at the
// wavefront's base plus 16 bytes per lane, so operand tiles never pass through
// registers: the pipeline can run NST chunks deep with few VGPRs.  A chunk
// row (one pixel or one filter, 64 channels = 128 bytes = 8 units of 16 bytes)
// is stored with its units permuted, unit kg at slot kg ^ f(row), with
// f(row) = (row & 7) ^ ((row >> 3) & 1): the MFMA operand reads (16
// consecutive rows, one unit each) then hit 16 distinct 16-byte bank groups,
// and each load instruction still fills 1 KB of LDS contiguously.
// The LDS epilogue of the channel-last kernels writes the tile [BKC filters]
// [BPX pixels] (row pitch OP floats, bias added, activation applied unless a
// residual follows) in rows of 4 pixels: element (filter kl, pixels 4*c4 ..
// 4*c4+3) is row idx = kl * BPX/4 + c4, and thread tid takes rows tid,
// tid + NT, ...  Rows go to y -- or, with a reduction split, to this split's
// partials [K][M] -- as 16-byte stores where y's alignment and the plane
// allow.
template <int BPX, int BKC, int NT, int OP>
__device__ inline void store_tile(const ConvArgs &a, const float *ot, int tid, int k0, int m0, int g,
                                  int split)
{
    const bool split_out = a.splits > 1;
    float *out = split_out ? a.ws + (long)split * a.K * a.M : a.y;
    const bool vec = split_out ? (a.M & 3) == 0 : ((a.PQ & 3) == 0 && ((uintptr_t)a.y & 15) == 0 && (a.ysn & 3) == 0);
    constexpr int C4 = BPX / 4;
    constexpr int KS = NT / C4;                     // filter rows per pass of the work-group
    constexpr int IT = BKC / KS;                    // passes
    static_assert(NT % C4 == 0 && BKC % KS == 0, "epilogue rows per thread");
    // A thread's rows share one quad of pixels, m .. m+3 (c4 = tid % C4), and
    // step through the filters KS at a time.
    const int c4 = tid % C4, kl0 = tid / C4;
    const int m = m0 + 4 * c4;
    if (m >= a.M) return;
    if (vec && m + 3 < a.M) {
        // the quad lies in one image plane (P*Q % 4 == 0): one image index and
        // one base offset; every row is a constant stride further
        const int n = split_out ? 0 : (int)fdiv(m, a.dv_pq);
        const long kstride = split_out ? (long)a.M : (long)a.PQ;
        const long base = split_out ? (long)m : (long)n * a.ysn + (m - n * a.PQ);
        float *dst = out + base + ((long)g * a.Kg + k0 + kl0) * kstride;
        const long step = KS * kstride;
        typedef float f32x4 __attribute__((ext_vector_type(4)));
        constexpr int B = IT < 8 ? IT : 8;          // LDS reads in flight per batch
        static_assert(IT % B == 0, "batches");
#pragma unroll
        for (int i0 = 0; i0 < IT; i0 += B) {
            f32x4 v[B];
#pragma unroll
            for (int i = 0; i < B; ++i)
                v[i] = *reinterpret_cast<const f32x4 *>(ot + (kl0 + (i0 + i) * KS) * OP + 4 * c4);
#pragma unroll
            for (int i = 0; i < B; ++i) {
                if (k0 + kl0 + (i0 + i) * KS < a.Kg)
                    __builtin_nontemporal_store(v[i], reinterpret_cast<f32x4 *>(dst + (i0 + i) * step));
            }
        }
        return;
    }
    for (int it = 0; it < IT; ++it) {
        const int kl = kl0 + it * KS;
        const int k = k0 + kl;
        if (k >= a.Kg) break;
        const int kg = g * a.Kg + k;
        const float4 v = *reinterpret_cast<const float4 *>(ot + kl * OP + 4 * c4);
        const float ve[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int mm = m + e;
            if (mm >= a.M) break;
            const int n = split_out ? 0 : (int)fdiv(mm, a.dv_pq);
            const long off = split_out ? (long)kg * a.M + mm : ((long)n * a.ysn + (long)kg * a.PQ) + (mm - n * a.PQ);
            out[off] = ve[e];
        }
    }
}

// The same rows with the residual joined (no split).  load_res_tile requests
// every residual value this thread needs in one burst, before the epilogue's
// barriers, so the loads overlap each other and the accumulator pass; they all
// precede the thread's first store, so res may be y itself.  store_tile_res
// then joins, activates and stores.
template <int BPX, int BKC, int NT>
__device__ inline void load_res_tile(const ConvArgs &a, int tid, int k0, int m0, int g,
                                     float (&rv)[BKC * (BPX / 4) / NT][4])
{
    constexpr int C4 = BPX / 4;
    constexpr int IT = BKC * C4 / NT;
    static_assert(BKC * C4 % NT == 0, "epilogue rows per thread");
    const int ysn = (int)a.ysn;   // every y offset is below 2^31 (checked on the host)
    const bool vec = (a.PQ & 3) == 0 && ((uintptr_t)a.y & 15) == 0 && (ysn & 3) == 0;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int idx = tid + it * NT;
        const int kl = idx / C4, c4 = idx - kl * C4;
        const int k = k0 + kl;
        const int m = m0 + 4 * c4;
#pragma unroll
        for (int e = 0; e < 4; ++e) rv[it][e] = 0.f;
        if (k >= a.Kg || m >= a.M) continue;
        const int kg = g * a.Kg + k;
        if (vec && m + 3 < a.M) {
            const int n = (int)fdiv(m, a.dv_pq);
            const float4 r = *reinterpret_cast<const float4 *>(
                a.res + (n * ysn + kg * a.PQ) + (m - n * a.PQ));
            rv[it][0] = r.x;
            rv[it][1] = r.y;
            rv[it][2] = r.z;
            rv[it][3] = r.w;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int mm = m + e;
                if (mm >= a.M) break;
                const int n = (int)fdiv(mm, a.dv_pq);
                rv[it][e] = a.res[(n * ysn + kg * a.PQ) + (mm - n * a.PQ)];
            }
        }
    }
}

template <int BPX, int BKC, int NT, int OP>
__device__ inline void store_tile_res(const ConvArgs &a, const float *ot, int tid, int k0, int m0, int g,
                                      const float (&rv)[BKC * (BPX / 4) / NT][4])
{
    constexpr int C4 = BPX / 4;
    constexpr int IT = BKC * C4 / NT;
    const int ysn = (int)a.ysn;
    const bool vec = (a.PQ & 3) == 0 && ((uintptr_t)a.y & 15) == 0 && (ysn & 3) == 0;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int idx = tid + it * NT;
        const int kl = idx / C4, c4 = idx - kl * C4;
        const int k = k0 + kl;
        const int m = m0 + 4 * c4;
        if (k >= a.Kg || m >= a.M) continue;
        const int kg = g * a.Kg + k;
        const float4 v = *reinterpret_cast<const float4 *>(ot + kl * OP + 4 * c4);
        float ve[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            ve[e] += rv[it][e];
            if (a.relu) ve[e] = fmaxf(ve[e], 0.f);
        }
        if (vec && m + 3 < a.M) {
            const int n = (int)fdiv(m, a.dv_pq);
            typedef float f32x4 __attribute__((ext_vector_type(4)));
            const f32x4 nv = {ve[0], ve[1], ve[2], ve[3]};
            __builtin_nontemporal_store(
                nv, reinterpret_cast<f32x4 *>(a.y + (n * ysn + kg * a.PQ) + (m - n * a.PQ)));
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int mm = m + e;
                if (mm >= a.M) break;
                const int n = (int)fdiv(mm, a.dv_pq);
                a.y[(n * ysn + kg * a.PQ) + (mm - n * a.PQ)] = ve[e];
            }
        }
    }
}

__device__ inline int unit_swz(int row) { return (row & 7) ^ ((row >> 3) & 1); }

// 32-channel chunks (rows of 4 units, 64 bytes): unit u of row r sits at
// slot u ^ ((r >> 2) & 3), so 16 consecutive rows read at one logical unit
// cover all 16 bank groups of 256 bytes.
template <int UPR>
__device__ inline int row_swz(int row)
{
    if constexpr (UPR == 8) return unit_swz(row);
    else return (row >> 2) & 3;
}

template <int N>
__device__ inline void wait_vmcnt()
{
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most `ahead` (uniform, 0 <= ahead <= MAXA) groups of LOADS
// loads of this lane are outstanding.
template <int LOADS, int MAXA>
__device__ inline void wait_ahead(int ahead)
{
    if constexpr (MAXA > 0) {
        if (ahead >= MAXA) {
            wait_vmcnt<MAXA * LOADS>();
            return;
        }
        wait_ahead<LOADS, MAXA - 1>(ahead);
    } else {
        wait_vmcnt<0>();
    }
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16_t;

// Channel-last bf16 epilogue (layers inside a channel-last network: y and
// the residual are bf16 [N*P*Q][K]).  In these instantiations the MFMA runs
// with the filters as its A operand, so accumulator register v of lane l
// holds channel 8*(v/4) + 4*(l/32) + v%4 of the channel block and pixel l%32
// of the pixel block: four consecutive channels of one pixel, written to LDS
// as one 16-byte store into a pixel-major tile [BPX][BKC + 4] fp32 (16 lanes
// of a store phase cover the 64 banks once).  Each thread then takes 8
// consecutive channels of one pixel: bias, the bf16 residual, activation,
// round to bf16 (nearest even), one 16-byte store.  With a reduction split
// the raw fp32 sums go to this split's partials [M][K] instead (two 16-byte
// stores) for splitk_reduce_cl_kernel.  Requires K/groups % 8 == 0 and y,
// res 16-byte aligned (checked on the host).
template <int BPX, int BKC, int NT>
struct ClRes {
    static constexpr int C8 = BKC / 8;
    static constexpr int IT = BPX / (NT / C8);       // pixels per thread
    uint4 rv[IT];
};

// The thread's residual octets (the ones its epilogue_cl stores), requested
// ahead so that their round trips overlap other work (all precede the
// thread's first store, so res may be y itself).
template <int BPX, int BKC, int NT>
__device__ inline void cl_res_load(const ConvArgs &a, ClRes<BPX, BKC, NT> &r, int tid, int k0, int m0, int g)
{
    constexpr int C8 = BKC / 8;
    constexpr int IT = BPX / (NT / C8);
    static_assert(NT % C8 == 0 && BPX % (NT / C8) == 0, "a thread keeps one channel octet");
    const int o = tid % C8;
    const int k = k0 + 8 * o;
    const int kg = g * a.Kg + k;
    const uint16_t *res = reinterpret_cast<const uint16_t *>(a.res);
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int m = m0 + tid / C8 + it * (NT / C8);
        r.rv[it] = make_uint4(0, 0, 0, 0);
        if (res && a.splits == 1 && k < a.Kg && m < a.M)
            r.rv[it] = *reinterpret_cast<const uint4 *>(res + (long)m * a.K + kg);
    }
}

// NH = 2: the tile is staged in two passes of half its pixels (each the
// pixels of one column of wavefronts, WPX = 2), which halves the staging LDS.
template <int BPX, int BKC, int NT, int TPX, int TCH, int BJ, int BI, int NH = 1>
__device__ inline void epilogue_cl(const ConvArgs &a, const floatx16 (&acc)[BJ][BI], float *ot, int tid,
                                   int wpx, int wch, int h, int ll, int k0, int m0, int g, int split,
                                   const ClRes<BPX, BKC, NT> &cr)
{
    constexpr int CP = BKC + 4;
    constexpr int C8 = BKC / 8;
    constexpr int IT = BPX / (NT / C8);              // pixels per thread
    constexpr int PH = BPX / NH;                     // pixels per pass
    static_assert(NH == 1 || (NH == 2 && TPX == PH && IT % 2 == 0), "a pass is one column of wavefronts");
    const int o = tid % C8;
    const int k = k0 + 8 * o;
    const int kg = g * a.Kg + k;
    const bool kok = k < a.Kg;                       // K/groups % 8 == 0: the octet is whole
    const uint4 *rv = cr.rv;
    float bv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) bv[e] = (kok && a.splits == 1 && a.bias) ? a.bias[kg + e] : 0.f;
    uint16_t *y = reinterpret_cast<uint16_t *>(a.y);
#pragma unroll
    for (int hp = 0; hp < NH; ++hp) {
        if (hp) __syncthreads();                     // every thread is done reading the last pass
        if (NH == 1 || wpx == hp) {
#pragma unroll
            for (int bi = 0; bi < BI; ++bi)
#pragma unroll
                for (int bj = 0; bj < BJ; ++bj)
#pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4) {
                        const int kl = wch * TCH + bi * 32 + 8 * q4 + 4 * h;
                        const int pl = wpx * TPX + bj * 32 + ll - hp * PH;
                        *reinterpret_cast<float4 *>(ot + pl * CP + kl) =
                            make_float4(acc[bj][bi][4 * q4], acc[bj][bi][4 * q4 + 1], acc[bj][bi][4 * q4 + 2],
                                        acc[bj][bi][4 * q4 + 3]);
                    }
        }
        __syncthreads();
#pragma unroll
        for (int it = hp * (IT / NH); it < (hp + 1) * (IT / NH); ++it) {
            const int pl = tid / C8 + it * (NT / C8);
            const int m = m0 + pl;
            if (!kok || m >= a.M) continue;
            const float4 lo = *reinterpret_cast<const float4 *>(ot + (pl - hp * PH) * CP + 8 * o);
            const float4 hi = *reinterpret_cast<const float4 *>(ot + (pl - hp * PH) * CP + 8 * o + 4);
            float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
            const long off = (long)m * a.K + kg;
            if (a.splits > 1) {
                float *dst = a.ws + (long)split * a.M * a.K + off;
                *reinterpret_cast<float4 *>(dst) = lo;
                *reinterpret_cast<float4 *>(dst + 4) = hi;
                continue;
            }
            const uint32_t rr[4] = {rv[it].x, rv[it].y, rv[it].z, rv[it].w};
            uint32_t d[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float v0 = v[2 * e] + bv[2 * e], v1 = v[2 * e + 1] + bv[2 * e + 1];
                if (a.res) {
                    v0 += bf16_to_f32((uint16_t)(rr[e] & 0xFFFFu));
                    v1 += bf16_to_f32((uint16_t)(rr[e] >> 16));
                }
                if (a.relu) {
                    v0 = fmaxf(v0, 0.f);
                    v1 = fmaxf(v1, 0.f);
                }
                d[e] = pack_bf16x2(v0, v1);
            }
            // plain stores: the next layer reads y, and the lines it finds in
            // the last-level cache it does not fetch from HBM
            *reinterpret_cast<uint4 *>(y + off) = make_uint4(d[0], d[1], d[2], d[3]);
        }
    }
}

// NCHWB (1x1, stride 1, H*W % 8 == 0, 128-pixel tiles): the pixel operand is
// read from the NCHW input itself, no channel-last copy.  A chunk's pixel tile
// is staged as 64 channel rows of 128 pixels (16 units of 8 pixels, unit s of
// row c stored at s ^ 4*(c & 3)), and each MFMA fragment (8 channels of one
// pixel per lane) is assembled by two ds_read_b64_tr_b16: in every group of 16
// lanes, lane 4e+t points at 4 pixels of channel row e and lane i receives
// pixel i of the 4 rows.  The permuted units put the 4 rows of one read in 4
// different 64-byte bank groups.
//
// NCHWB == 2 (even H*W that is not a multiple of 8, e.g. 14x14): 8 pixels of
// a channel may straddle two images, so the rows are loaded 4 bytes per lane
// (2 pixels, never straddling): one load instruction fills one 256-byte
// channel row, each lane fetching the pixel pair its LDS dword holds under
// the unit permutation.  Same bandwidth per byte through the load path,
// 4x the instructions.
template <int R_, int S_, int BPX, int BKC, int WPX, int WCH, int NST, int NCHWB, int KRC, bool RES, bool YCL>
__device__ __forceinline__ void dma_body(const ConvArgs &a)
{
    constexpr int NT = 64 * WPX * WCH;
    constexpr int UPR = KRC / 8;                        // 16-byte units per operand row
    constexpr int TPX = BPX / WPX, TCH = BKC / WCH;     // one wavefront's tile
    constexpr int BJ = TPX / 32, BI = TCH / 32;         // pixel blocks, channel blocks
    constexpr int UA = BKC * UPR, UB = BPX * UPR;       // 16-byte units per stage
    constexpr int LA = UA / NT, LB = UB / NT;           // load instructions per lane per chunk
    constexpr int LOADS = LA + (NCHWB == 2 ? KRC / (WPX * WCH) : LB);
    static_assert(BJ >= 1 && BI >= 1 && UA % NT == 0 && UB % NT == 0, "tile shape");
    static_assert(NST >= 1 && NST <= 8 && (NST - 2) * LOADS <= 63, "pipeline depth");
    static_assert(!NCHWB || (BPX == 128 && R_ == 1 && S_ == 1 && KRC == 64), "NCHW pixel operand: 1x1, 128-pixel tiles");
    static_assert(NCHWB != 2 || (KRC / WPX / WCH) * WPX * WCH == KRC, "one channel row per load");
    static_assert(KRC == 64 || KRC == 32, "reduction chunk");

    constexpr int OP = BPX + 4;                          // output tile row pitch (floats)
    // one-stage 128-pixel channel-last tiles stage their epilogue in two
    // passes, so the operand stage sets the LDS size
    constexpr int NHE = YCL && NST == 1 && BPX == 128 && WPX == 2 ? 2 : 1;
    constexpr int EPI = YCL ? BPX / NHE * (BKC + 4) / 4 : BKC * OP / 4;   // epilogue tile, 16-byte units
    constexpr int SMEM = NST * (UA + UB) > EPI ? NST * (UA + UB) : EPI;
    __shared__ __attribute__((aligned(16))) uint4 smem[SMEM];

    const uint16_t *__restrict__ xcl = static_cast<const uint16_t *>(a.x);   // [N][H][W][C]
    const uint16_t *__restrict__ wp = static_cast<const uint16_t *>(a.w);    // [K][R][S][Cg]
    const int S = S_ ? S_ : a.S;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wpx = wid % WPX, wch = wid / WPX;
    const int h = lane >> 5, ll = lane & 31;
    // XCD-aware tile order: the hardware deals work-groups to the 8 XCDs
    // round-robin, so work-group w runs on XCD w % 8.  Logical tiles are
    // renumbered so that each XCD gets one contiguous range of them, with the
    // channel tiles of one pixel tile adjacent: tiles that read the same
    // input pixels share that XCD's L2.
    const int T = gridDim.x;
    const int xcd = blockIdx.x % 8, j = blockIdx.x / 8;
    const int L = xcd * (T / 8) + min(xcd, T % 8) + j;
    const int ktiles = (a.Kg + BKC - 1) / BKC;
    const int mtiles = (a.M + BPX - 1) / BPX;
    const int ky = L % ktiles;
    const int mx = (L / ktiles) % mtiles;
    const int z = L / (ktiles * mtiles);
    const int g = z % a.groups;
    const int split = z / a.groups;
    const int m0 = mx * BPX;
    const int k0 = ky * BKC;
    const int kr_begin = split * a.kr_per_split;
    const int kr_end = min(a.Kred, kr_begin + a.kr_per_split);

    // Operands are read through buffer resources: an offset past the end
    // (kOutside) makes the hardware range check return zeros, which is how
    // padding taps, pixels past M and filters past K are loaded.
    constexpr unsigned kOutside = 0xffffffffu;
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(wp), (short)0, (int)((long)a.K * a.Kred * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(xcl), (short)0, (int)((long)a.N * a.H * a.W * a.C * 2), 0x00020000);

    // Loader: load i of lane tid fills unit u = i*NT + tid of its operand.
    // Byte offsets of the lane's row at reduction index 0 / tap (0, 0).
    unsigned aoffs[LA];
    bool aok[LA];
#pragma unroll
    for (int i = 0; i < LA; ++i) {
        const int u = i * NT + tid;
        const int row = u / UPR;
        const int kg = (u % UPR) ^ row_swz<UPR>(row);
        const int k = k0 + row;
        aok[i] = k < a.Kg;
        aoffs[i] = (unsigned)((((long)g * a.Kg + (aok[i] ? k : 0)) * a.Kred + kg * 8) * 2);
    }
    int bih[LB], biw[LB], boffs[LB];
    // NCHWB == 2: byte offset of the lane's pixel pair at channel 0 of the
    // group, for each value of (row & 3) (the permutation of the row's units)
    unsigned doff[4];
    if constexpr (NCHWB == 2) {
#pragma unroll
        for (int c3 = 0; c3 < 4; ++c3) {
            const int sl = (lane >> 2) ^ (4 * c3);              // logical 8-pixel unit of LDS unit lane/4
            const int m = m0 + 8 * sl + 2 * (lane & 3);
            const int n = m / a.HW;
            doff[c3] = m < a.M ? (unsigned)((((long)n * a.C + (long)g * a.Cg) * a.HW + (m - n * a.HW)) * 2)
                               : 0x80000000u;
        }
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
        const int u = i * NT + tid;
        if constexpr (NCHWB == 2) {
            break;
        } else if constexpr (NCHWB) {
            // unit u: channel row c = u / 16 of the chunk, 8 pixels at unit s
            const int c = u >> 4;
            const int sl = (u & 15) ^ (4 * (c & 3));
            const int m = m0 + 8 * sl;
            const bool ok = m < a.M;
            const int mm = ok ? m : 0;
            const int n = mm / a.HW;
            bih[i] = ok ? 0 : -(1 << 28);               // 1x1: only the pixel range test
            biw[i] = 0;
            boffs[i] = (int)(((long)n * a.C + (long)g * a.Cg + c) * a.HW + (mm - n * a.HW));
            continue;
        }
        const int row = u / UPR;
        const int kg = (u % UPR) ^ row_swz<UPR>(row);
        const int m = m0 + row;
        const bool ok = m < a.M;
        const int mm = ok ? m : 0;
        const int n = mm / a.PQ;
        const int pq = mm - n * a.PQ;
        const int p = pq / a.Q;
        const int q = pq - p * a.Q;
        bih[i] = ok ? p * a.stride - a.pad : -(1 << 28);      // never inside the image
        biw[i] = q * a.stride - a.pad;
        // element offset of (n, bih, biw, g*Cg + kg*8); negative for a top/left
        // padding origin, but every tap that passes the bounds test is >= 0
        boffs[i] = (int)((long)n * a.H * a.W * a.C + ((long)bih[i] * a.W + biw[i]) * a.C +
                         (long)g * a.Cg + kg * 8);
    }

    auto issue = [&](int t) {
        // chunk parameters are uniform: keep them in scalar registers
        const int kr0 = __builtin_amdgcn_readfirstlane(kr_begin + t * KRC);
        const int rs = kr0 / a.Cg;                  // the chunk is 64 channels at tap rs
        const int c0 = kr0 - rs * a.Cg;
        const int r = rs / S;
        const int s = rs - r * S;
        const int delta = (r * a.W + s) * a.C + c0;    // element offset of the tap
        const int stage = t % NST;
        uint4 *st = smem + stage * (UA + UB);
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            const unsigned off = aok[i] ? aoffs[i] + 2u * kr0 : kOutside;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(wres, (lds_void_t *)(st + i * NT + wid * 64), 16,
                                                     off, 0, 0, 0);
        }
        if constexpr (NCHWB == 2) {
            // channel rows wid, wid + NW, ...: one 256-byte row per load
            constexpr int NW = WPX * WCH;
#pragma unroll
            for (int i = 0; i < KRC / NW; ++i) {
                const int c = wid + i * NW;
                const unsigned off = doff[c & 3] + 2u * (unsigned)((c0 + c) * a.HW);   // >= 2^31: zeros
                __builtin_amdgcn_raw_ptr_buffer_load_lds(xres, (lds_void_t *)(st + UA + c * 16), 4, off, 0, 0, 0);
            }
            return;
        }
#pragma unroll
        for (int i = 0; i < LB; ++i) {
            bool ok;
            unsigned off;
            if constexpr (NCHWB) {
                ok = bih[i] == 0;
                off = ok ? 2u * (unsigned)(boffs[i] + c0 * a.HW) : kOutside;
            } else {
                ok = (unsigned)(bih[i] + r) < (unsigned)a.H && (unsigned)(biw[i] + s) < (unsigned)a.W;
                off = ok ? 2u * (unsigned)(boffs[i] + delta) : kOutside;
            }
            __builtin_amdgcn_raw_ptr_buffer_load_lds(xres, (lds_void_t *)(st + UA + i * NT + wid * 64),
                                                     16, off, 0, 0, 0);
        }
    };

    // Operand reads: row offsets (in units) and the permuted slot of unit
    // 2*ks + h, per 16-wide reduction step ks.
    const int fl = row_swz<UPR>(ll);
    int aoff[BI], boff[BJ];
#pragma unroll
    for (int bi = 0; bi < BI; ++bi) aoff[bi] = (wch * TCH + bi * 32 + ll) * UPR;
#pragma unroll
    for (int bj = 0; bj < BJ; ++bj) boff[bj] = UA + (wpx * TPX + bj * 32 + ll) * UPR;

    floatx16 acc[BJ][BI];
#pragma unroll
    for (int bj = 0; bj < BJ; ++bj)
#pragma unroll
        for (int bi = 0; bi < BI; ++bi)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[bj][bi][v] = 0.f;

    // All operand reads of a chunk are issued before its first MFMA, so LDS
    // latency overlaps the MFMAs of the earlier reduction steps.
    auto compute = [&](int t) {
        const uint4 *st = smem + (t % NST) * (UA + UB);
        constexpr int KS = KRC / 16;
        bf16x8 wv[KS][BI], xv[KS][BJ];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int slot = (2 * ks + h) ^ fl;
#pragma unroll
            for (int bi = 0; bi < BI; ++bi)
                wv[ks][bi] = *reinterpret_cast<const bf16x8 *>(st + aoff[bi] + slot);
#pragma unroll
            for (int bj = 0; bj < BJ; ++bj) {
                if constexpr (NCHWB) {
                    // rows kb+e and kb+4+e of the chunk, pixels n0 + 4t .. n0 + 4t + 3
                    const int kb = 16 * ks + 8 * (lane >> 5) + ((lane >> 2) & 3);
                    const int px = wpx * TPX + bj * 32 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
                    const char *base = reinterpret_cast<const char *>(st + UA);
                    const int o1 = (kb * 16 + ((px >> 3) ^ (4 * (kb & 3)))) * 16 + (px & 7) * 2;
                    const int o2 = ((kb + 4) * 16 + ((px >> 3) ^ (4 * (kb & 3)))) * 16 + (px & 7) * 2;
                    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(base + o1));
                    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(base + o2));
                    const v8i16 both = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                    xv[ks][bj] = __builtin_bit_cast(bf16x8, both);
                } else {
                    xv[ks][bj] = *reinterpret_cast<const bf16x8 *>(st + boff[bj] + slot);
                }
            }
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int bj = 0; bj < BJ; ++bj)
#pragma unroll
                for (int bi = 0; bi < BI; ++bi) {
                    if constexpr (YCL)   // filters as the A operand: a lane holds channels of one pixel
                        acc[bj][bi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wv[ks][bi], xv[ks][bj],
                                                                             acc[bj][bi], 0, 0, 0);
                    else
                        acc[bj][bi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xv[ks][bj], wv[ks][bi],
                                                                             acc[bj][bi], 0, 0, 0);
                }
    };

    // the residual of the channel-last epilogue: the work-group's first
    // requests, landed by the time the first reduction chunk has
    ClRes<BPX, BKC, NT> cr;
    if constexpr (YCL) cl_res_load<BPX, BKC, NT>(a, cr, tid, k0, m0, g);

    const int nchunks = kr_end > kr_begin ? (kr_end - kr_begin) / KRC : 0;
    if constexpr (NST == 1) {
        // one stage (layers of one or two chunks): no overlap inside the
        // work-group, a third of the LDS, more work-groups per CU
        for (int t = 0; t < nchunks; ++t) {
            if (t) asm volatile("s_barrier" ::: "memory");   // every wavefront is done with chunk t-1
            issue(t);
            wait_vmcnt<0>();
            asm volatile("s_barrier" ::: "memory");
            compute(t);
        }
    } else {
#pragma unroll
        for (int t = 0; t < NST - 1; ++t)
            if (t < nchunks) issue(t);
        for (int t = 0; t < nchunks; ++t) {
            // this lane's loads of chunk t are done once at most `ahead` later
            // chunks' loads are outstanding
            const int ahead = min(NST - 2, nchunks - 1 - t);
            wait_ahead<LOADS, NST - 2>(ahead);
            // every lane's chunk t is in LDS, and every wavefront is done with chunk t-1
            asm volatile("s_barrier" ::: "memory");
            if (t + NST - 1 < nchunks) issue(t + NST - 1);
            compute(t);
        }
    }

    if constexpr (YCL) {
        __syncthreads();   // every wavefront is done with the operand stages
        epilogue_cl<BPX, BKC, NT, TPX, TCH, BJ, BI, NHE>(a, acc, reinterpret_cast<float *>(smem), tid, wpx, wch,
                                                         h, ll, k0, m0, g, split, cr);
        return;
    }
    // Epilogue through LDS: the tile (BKC channels x BPX pixels, fp32, bias and
    // activation applied) is laid out channel-major in the shared buffer, free
    // once every wavefront has passed the barrier, then each channel row is
    // written out with contiguous 16-byte stores (a lane's own accumulators
    // would give 32 scattered 32-byte pieces per store instruction).
    float rv[RES ? BKC * (BPX / 4) / NT : 1][4];
    if constexpr (RES) load_res_tile<BPX, BKC, NT>(a, tid, k0, m0, g, rv);
    __syncthreads();
    float *ot = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int bi = 0; bi < BI; ++bi) {
        const int kl = wch * TCH + bi * 32 + ll;
        const int k = k0 + kl;
        const float bv = (a.splits == 1 && a.bias && k < a.Kg) ? a.bias[g * a.Kg + k] : 0.f;
#pragma unroll
        for (int bj = 0; bj < BJ; ++bj) {
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                float v4[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float val = acc[bj][bi][4 * q4 + e];
                    if (a.splits == 1) {
                        val += bv;
                        if (a.relu && !RES) val = fmaxf(val, 0.f);
                    }
                    v4[e] = val;
                }
                const int pl = wpx * TPX + bj * 32 + 8 * q4 + 4 * h;
                *reinterpret_cast<float4 *>(ot + kl * OP + pl) = make_float4(v4[0], v4[1], v4[2], v4[3]);
            }
        }
    }
    __syncthreads();
    if constexpr (RES)
        store_tile_res<BPX, BKC, NT, OP>(a, ot, tid, k0, m0, g, rv);
    else
        store_tile<BPX, BKC, NT, OP>(a, ot, tid, k0, m0, g, split);
}

template <int R_, int S_, int BPX, int BKC, int WPX, int WCH, int NST, int NCHWB, int KRC = 64>
__global__ __launch_bounds__(64 * WPX * WCH) void igemm_bf16_dma_kernel(ConvArgs a)
{
    dma_body<R_, S_, BPX, BKC, WPX, WCH, NST, NCHWB, KRC, false, false>(a);
}

// Channel-last bf16 output (and residual): the epilogue_cl instantiation.
template <int R_, int S_, int BPX, int BKC, int WPX, int WCH, int NST, int NCHWB, int KRC = 64>
__global__ __launch_bounds__(64 * WPX * WCH, NST == 1 && BPX == 128 ? 5 : 1) void igemm_bf16_dma_cl_kernel(ConvArgs a)
{
    dma_body<R_, S_, BPX, BKC, WPX, WCH, NST, NCHWB, KRC, false, true>(a);
}

// The same kernel with the residual join in its epilogue (layers without a
// reduction split): the residual loads are issued before the epilogue's
// barriers, which costs registers the plain kernel does not spend.
template <int R_, int S_, int BPX, int BKC, int WPX, int WCH, int NST, int NCHWB, int KRC = 64>
__global__ __launch_bounds__(64 * WPX * WCH, 2) void igemm_bf16_dma_res_kernel(ConvArgs a)
{
    dma_body<R_, S_, BPX, BKC, WPX, WCH, NST, NCHWB, KRC, true, false>(a);
}

// 3x3, stride 1, padding 1 (the middle layers of bottleneck blocks): the
// pixel operand of all nine taps of one 64-channel block comes from one
// staged patch.  In the channel-last copy, flattened over (n, p, q), output
// pixel m reads input pixel m + (r-1)*W + (s-1) at tap (r, s), so the pixels
// that output pixels m0 .. m0+BPX-1 read at any tap lie in the contiguous run
// m0-W-1 .. m0+BPX+W: the work-group stages that run once per channel block
// (rows of 64 channels, units permuted as in igemm_bf16_dma_kernel) and reads
// tap (r, s) at row offset r*W + s.  Taps that fall into the padding (input
// row or column outside the image, which in the flattened run is a
// neighbouring row or image) are zeroed after the read.  The pixel operand
// moves once per channel block instead of once per tap: 3.5x less staging
// traffic for a 128-pixel tile at 28x28.  Filters are packed in 64-channel
// blocks ((block, r, s, c) order), so chunk t = (block t/9, tap t%9) is again
// 64 contiguous values per filter, double-buffered in LDS; the patches are
// double-buffered by block parity, the next block's patch loaded with the
// last tap of the current one.  PR = patch rows allocated (BPX + 2W + 2 used).
// NPB = 1 (one channel block, C/groups == 64): a single patch buffer, loaded
// once, and a single filter stage, which keeps a 128 x 64 tile at 40 KB of
// LDS: four work-groups per CU, each waiting for a tap's filters while the
// others compute.
template <int BPX, int BKC, int WPX, int WCH, int PR, int NPB, bool RES, bool YCL>
__device__ __forceinline__ void halo_body(const ConvArgs &a)
{
    constexpr int NT = 64 * WPX * WCH;
    constexpr int TPX = BPX / WPX, TCH = BKC / WCH;     // one wavefront's tile
    constexpr int BJ = TPX / 32, BI = TCH / 32;         // pixel blocks, channel blocks
    constexpr int UA = BKC * 8;                         // 16-byte units per filter stage
    constexpr int UP = PR * 8;                          // 16-byte units per patch buffer
    constexpr int LA = UA / NT;
    static_assert(BJ >= 1 && BI >= 1 && UA % NT == 0 && UP % NT == 0, "tile shape");
    constexpr int OP = BPX + 4;                          // output tile row pitch (floats)
    static_assert(NPB == 1 || NPB == 2, "patch buffers");
    constexpr int EPI = YCL ? BPX * (BKC + 4) / 4 : BKC * OP / 4;   // epilogue tile, 16-byte units
    constexpr int FA = NPB == 1 ? UA : 2 * UA;           // filter stages (one with one patch buffer)
    constexpr int SMEM = FA + NPB * UP > EPI ? FA + NPB * UP : EPI;
    __shared__ __attribute__((aligned(16))) uint4 smem[SMEM];   // [A 0][A 1 (NPB 2)][patch 0][patch 1 (NPB 2)]
    if (NPB == 1 && a.Cg != 64) return;                 // the launcher never sends such a layer

    const uint16_t *__restrict__ xcl = static_cast<const uint16_t *>(a.x);   // [N][H][W][C]
    const uint16_t *__restrict__ wp = static_cast<const uint16_t *>(a.w);    // [K][Cg/64][3][3][64]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wpx = wid % WPX, wch = wid / WPX;
    const int h = lane >> 5, ll = lane & 31;
    // XCD-aware tile order, as in igemm_bf16_dma_kernel
    const int T = gridDim.x;
    const int xcd = blockIdx.x % 8, jx = blockIdx.x / 8;
    const int L = xcd * (T / 8) + min(xcd, T % 8) + jx;
    const int ktiles = (a.Kg + BKC - 1) / BKC;
    const int mtiles = (a.M + BPX - 1) / BPX;
    const int ky = L % ktiles;
    const int mx = (L / ktiles) % mtiles;
    const int z = L / (ktiles * mtiles);
    const int g = z % a.groups;
    const int split = z / a.groups;
    const int m0 = mx * BPX;
    const int k0 = ky * BKC;
    const int t_begin = split * a.kr_per_split / 64;
    const int t_end = min(a.Kred, (split + 1) * a.kr_per_split) / 64;

    constexpr unsigned kOutside = 0xffffffffu;
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(wp), (short)0, (int)((long)a.K * a.Kred * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(xcl), (short)0, (int)((long)a.N * a.H * a.W * a.C * 2), 0x00020000);

    // Filter loader: load i of lane tid fills unit u = i*NT + tid (row u/8).
    unsigned aoffs[LA];
    bool aok[LA];
#pragma unroll
    for (int i = 0; i < LA; ++i) {
        const int u = i * NT + tid;
        const int row = u >> 3;
        const int kg = (u & 7) ^ unit_swz(row);
        const int k = k0 + row;
        aok[i] = k < a.Kg;
        aoffs[i] = (unsigned)((((long)g * a.Kg + (aok[i] ? k : 0)) * a.Kred + kg * 8) * 2);
    }
    auto issue_a = [&](int t) {
        const int kr0 = __builtin_amdgcn_readfirstlane(t * 64);
        uint4 *st = smem + (NPB == 1 ? 0 : (t & 1) * UA);
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            const unsigned off = aok[i] ? aoffs[i] + 2u * kr0 : kOutside;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(wres, (lds_void_t *)(st + i * NT + wid * 64), 16,
                                                     off, 0, 0, 0);
        }
    };
    // Patch loader: rows 0 .. BPX+2W+1 are pixels m0-W-1+row, 64 channels of
    // block cb; pixels outside 0 .. M-1 load as zeros.
    const int prow = BPX + 2 * a.W + 2;
    if (prow > PR) return;                              // the launcher never sends such a layer
    const int pinstr = (prow * 8 + NT - 1) / NT;        // uniform
    auto issue_patch = [&](int cb) {
        uint4 *pb = smem + FA + (NPB == 2 ? (cb & 1) * UP : 0);
        const int cbase = g * a.Cg + cb * 64;
        for (int i = 0; i < pinstr; ++i) {
            const int u = i * NT + tid;
            const int row = u >> 3;
            const int kg = (u & 7) ^ unit_swz(row);
            const int gm = m0 - a.W - 1 + row;
            const bool ok = row < prow && gm >= 0 && gm < a.M;
            const unsigned off = ok ? (unsigned)(((long)gm * a.C + cbase + kg * 8) * 2) : kOutside;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(xres, (lds_void_t *)(pb + i * NT + wid * 64), 16,
                                                     off, 0, 0, 0);
        }
    };

    // This lane's output pixels (one per 32-pixel block): row and column.
    int pp[BJ], qq[BJ];
#pragma unroll
    for (int bj = 0; bj < BJ; ++bj) {
        const int m = m0 + wpx * TPX + bj * 32 + ll;
        const int mm = m < a.M ? m : 0;
        const int pq = mm - (int)fdiv(mm, a.dv_pq) * a.PQ;
        const int p = fdiv(pq, a.dv_q);
        pp[bj] = m < a.M ? p : -4;                     // never inside the image
        qq[bj] = pq - p * a.Q;
    }
    const int fl = unit_swz(ll);
    int aoff[BI];
#pragma unroll
    for (int bi = 0; bi < BI; ++bi) aoff[bi] = (wch * TCH + bi * 32 + ll) * 8;

    floatx16 acc[BJ][BI];
#pragma unroll
    for (int bj = 0; bj < BJ; ++bj)
#pragma unroll
        for (int bi = 0; bi < BI; ++bi)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[bj][bi][v] = 0.f;

    auto compute = [&](int t) {
        const int cb = t / 9, tap = t - cb * 9;
        const int r = tap / 3, s = tap - r * 3;
        const uint4 *sa = smem + (NPB == 1 ? 0 : (t & 1) * UA);
        const uint4 *pb = smem + FA + (NPB == 2 ? (cb & 1) * UP : 0);
        bf16x8 wv[4][BI], xv[4][BJ];
        int prow_l[BJ];
        bool ok[BJ];
#pragma unroll
        for (int bj = 0; bj < BJ; ++bj) {
            prow_l[bj] = wpx * TPX + bj * 32 + ll + r * a.W + s;
            ok[bj] = (unsigned)(pp[bj] + r - 1) < (unsigned)a.H && (unsigned)(qq[bj] + s - 1) < (unsigned)a.W;
        }
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int slot = (2 * ks + h) ^ fl;
#pragma unroll
            for (int bi = 0; bi < BI; ++bi)
                wv[ks][bi] = *reinterpret_cast<const bf16x8 *>(sa + aoff[bi] + slot);
#pragma unroll
            for (int bj = 0; bj < BJ; ++bj) {
                const int row = prow_l[bj];
                xv[ks][bj] = *reinterpret_cast<const bf16x8 *>(pb + row * 8 + ((2 * ks + h) ^ unit_swz(row)));
            }
        }
#pragma unroll
        for (int bj = 0; bj < BJ; ++bj)
            if (!ok[bj])
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) xv[ks][bj] = bf16x8{};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
            for (int bj = 0; bj < BJ; ++bj)
#pragma unroll
                for (int bi = 0; bi < BI; ++bi) {
                    if constexpr (YCL)   // filters as the A operand, as in epilogue_cl
                        acc[bj][bi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wv[ks][bi], xv[ks][bj],
                                                                             acc[bj][bi], 0, 0, 0);
                    else
                        acc[bj][bi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xv[ks][bj], wv[ks][bi],
                                                                             acc[bj][bi], 0, 0, 0);
                }
    };

    // the residual of the channel-last epilogue: the work-group's first
    // requests, landed by the time the first reduction chunk has
    ClRes<BPX, BKC, NT> cr;
    if constexpr (YCL) cl_res_load<BPX, BKC, NT>(a, cr, tid, k0, m0, g);

    if constexpr (NPB == 1) {
        // one filter stage: a tap's filters are requested once every
        // wavefront is done with the last tap's; the other work-groups on
        // the CU (four fit) cover the round trip
        issue_patch(0);
        for (int t = t_begin; t < t_end; ++t) {
            if (t > t_begin) asm volatile("s_barrier" ::: "memory");
            issue_a(t);
            wait_vmcnt<0>();
            asm volatile("s_barrier" ::: "memory");
            compute(t);
        }
    } else {
    if (t_begin < t_end) {
        issue_a(t_begin);
        issue_patch(t_begin / 9);
    }
    for (int t = t_begin; t < t_end; ++t) {
        // every lane's loads of chunk t (and of its patch) are done ...
        wait_vmcnt<0>();
        // ... and every wavefront is done with chunk t-1
        asm volatile("s_barrier" ::: "memory");
        if (t + 1 < t_end) {
            issue_a(t + 1);
            if ((t + 1) % 9 == 0) issue_patch((t + 1) / 9);
        }
        compute(t);
    }
    }

    if constexpr (YCL) {
        __syncthreads();   // every wavefront is done with the filter stages and patches
        epilogue_cl<BPX, BKC, NT, TPX, TCH, BJ, BI>(a, acc, reinterpret_cast<float *>(smem), tid, wpx, wch, h,
                                                    ll, k0, m0, g, split, cr);
        return;
    }
    // Epilogue through LDS, as in igemm_bf16_dma_kernel.
    float rv[RES ? BKC * (BPX / 4) / NT : 1][4];
    if constexpr (RES) load_res_tile<BPX, BKC, NT>(a, tid, k0, m0, g, rv);
    __syncthreads();
    float *ot = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int bi = 0; bi < BI; ++bi) {
        const int kl = wch * TCH + bi * 32 + ll;
        const int k = k0 + kl;
        const float bv = (a.splits == 1 && a.bias && k < a.Kg) ? a.bias[g * a.Kg + k] : 0.f;
#pragma unroll
        for (int bj = 0; bj < BJ; ++bj) {
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                float v4[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float val = acc[bj][bi][4 * q4 + e];
                    if (a.splits == 1) {
                        val += bv;
                        if (a.relu && !RES) val = fmaxf(val, 0.f);
                    }
                    v4[e] = val;
                }
                const int pl = wpx * TPX + bj * 32 + 8 * q4 + 4 * h;
                *reinterpret_cast<float4 *>(ot + kl * OP + pl) = make_float4(v4[0], v4[1], v4[2], v4[3]);
            }
        }
    }
    __syncthreads();
    if constexpr (RES)
        store_tile_res<BPX, BKC, NT, OP>(a, ot, tid, k0, m0, g, rv);
    else
        store_tile<BPX, BKC, NT, OP>(a, ot, tid, k0, m0, g, split);
}

template <int BPX, int BKC, int WPX, int WCH, int PR, int NPB = 2>
__global__ __launch_bounds__(64 * WPX * WCH) void igemm_bf16_halo_kernel(ConvArgs a)
{
    halo_body<BPX, BKC, WPX, WCH, PR, NPB, false, false>(a);
}

// With the residual join in the epilogue (no reduction split).
template <int BPX, int BKC, int WPX, int WCH, int PR, int NPB = 2>
__global__ __launch_bounds__(64 * WPX * WCH, 2) void igemm_bf16_halo_res_kernel(ConvArgs a)
{
    halo_body<BPX, BKC, WPX, WCH, PR, NPB, true, false>(a);
}

// Channel-last bf16 output (and residual).
template <int BPX, int BKC, int WPX, int WCH, int PR, int NPB = 2>
__global__ __launch_bounds__(64 * WPX * WCH) void igemm_bf16_halo_cl_kernel(ConvArgs a)
{
    halo_body<BPX, BKC, WPX, WCH, PR, NPB, false, true>(a);
}

template <int R_, int S_, int BPX, int BKC, int WPX, int WCH, int NST, int NCHWB, int KRC = 64>
void launch_dma(const ConvArgs &a, dim3 grid, hipStream_t st)
{
    if constexpr (NCHWB == 0) {
        if (a.ycl) {
            launch_kernel((igemm_bf16_dma_cl_kernel<R_, S_, BPX, BKC, WPX, WCH, NST, NCHWB, KRC>), grid,
                          dim3(64 * WPX * WCH), 0, st, a);
            return;
        }
    }
    if (a.res && a.splits == 1)
        launch_kernel((igemm_bf16_dma_res_kernel<R_, S_, BPX, BKC, WPX, WCH, NST, NCHWB, KRC>), grid,
                      dim3(64 * WPX * WCH), 0, st, a);
    else
        launch_kernel((igemm_bf16_dma_kernel<R_, S_, BPX, BKC, WPX, WCH, NST, NCHWB, KRC>), grid,
                      dim3(64 * WPX * WCH), 0, st, a);
}

template <int BPX, int BKC, int WPX, int WCH, int PR, int NPB = 2>
void launch_halo_k(const ConvArgs &a, dim3 grid, hipStream_t st)
{
    if (a.ycl)
        launch_kernel((igemm_bf16_halo_cl_kernel<BPX, BKC, WPX, WCH, PR, NPB>), grid, dim3(64 * WPX * WCH), 0,
                      st, a);
    else if (a.res && a.splits == 1)
        launch_kernel((igemm_bf16_halo_res_kernel<BPX, BKC, WPX, WCH, PR, NPB>), grid,
                      dim3(64 * WPX * WCH), 0, st, a);
    else
        launch_kernel((igemm_bf16_halo_kernel<BPX, BKC, WPX, WCH, PR, NPB>), grid, dim3(64 * WPX * WCH),
                      0, st, a);
}

struct TileN {
    int bkc, bpx;
};
const TileN kTilesN[] = {{128, 128}, {64, 64}};

template <int R_, int S_, int KRC>
void launch_tile(const ConvArgs &a, int tile, dim3 grid, hipStream_t st)
{
    if (tile == 0)
        launch_kernel((igemm_bf16_nhwc_kernel<R_, S_, 128, 128, KRC>), grid, dim3(256), 0, st, a);
    else
        launch_kernel((igemm_bf16_nhwc_kernel<R_, S_, 64, 64, KRC>), grid, dim3(256), 0, st, a);
}

template <int KRC>
void launch_krc(const ConvArgs &a, int tile, dim3 grid, hipStream_t st)
{
    if (a.R == 1 && a.S == 1)
        launch_tile<1, 1, KRC>(a, tile, grid, st);
    else if (a.R == 3 && a.S == 3)
        launch_tile<3, 3, KRC>(a, tile, grid, st);
    else
        launch_tile<0, 0, KRC>(a, tile, grid, st);
}

int rs_template(int v) { return (v == 1 || v == 3) ? v : 0; }

// 1x1 layers with stride > 1 and no padding copy only the pixels they
// sample into the channel-last buffer.
bool copy_subsamples(const ConvProblem &p)
{
    return p.R == 1 && p.S == 1 && p.pad == 0 && p.stride > 1;
}

// Pixels per global read of the channel-last copy (x may be null: describe);
// 0 selects the whole-plane kernel, used for planes of up to 512 pixels that
// the tiled kernel could only read pixel by pixel (measured at batch 64:
// 49-pixel planes 10 -> 4.5 us, 14x14 planes sampled at stride 2 12 -> 7.8
// us; 28x28 planes sampled at stride 2, in 16-channel blocks, 15.3 -> 16.6
// us, so larger planes stay with the tiled kernel; for 196-pixel planes, which
// it reads 4 pixels at a time, the two are even).
int copy_read_width(const ConvProblem &p, const void *x)
{
    const uintptr_t xa = (uintptr_t)x;
    const int HW = p.H * p.W;
    const bool scalar = copy_subsamples(p) || HW % 4 != 0;
    if (scalar && 32 * HW <= kPlaneElems && p.C % 8 == 0 && xa % 16 == 0) return 0;
    if (copy_subsamples(p)) {
        // stride 2: negative = sampled pixels per load (8- or 16-byte loads)
        const bool s2 = p.stride == 2 && p.W == 2 * p.Q;
        if (s2 && p.Q % 4 == 0 && p.W % 4 == 0 && HW % 8 == 0 && xa % 16 == 0) return -4;
        if (s2 && p.Q % 2 == 0 && p.W % 2 == 0 && HW % 4 == 0 && xa % 8 == 0) return -2;
        return 1;
    }
    if (HW % 8 == 0 && xa % 16 == 0) return 8;
    if (HW % 4 == 0 && xa % 8 == 0) return 4;
    return 1;
}

// The problem the GEMM kernels see after the copy: a subsampling copy turns
// a 1x1 stride-S layer into a stride-1 layer on its P x Q sampled pixels.
ConvProblem copied_problem(const ConvProblem &p)
{
    ConvProblem q = p;
    if (copy_subsamples(p)) {
        q.H = p.P;
        q.W = p.Q;
        q.stride = 1;
    }
    return q;
}

// Channel block of the whole-plane copy: 64, halved (down to 8) while the
// block exceeds the LDS buffer or the grid of N * C / cb work-groups would
// hold fewer than two per CU.
int plane_copy_block(const ConvProblem &p, int num_cus)
{
    const long hw = (long)p.H * p.W;
    int cb = 64;
    while (cb > 8 && (cb * hw > kPlaneElems || (long)p.N * ceil_div(p.C, cb) < 2L * num_cus)) cb /= 2;
    return cb;
}

// Direct-to-LDS tiles: pixels x channels, wavefronts along pixels x channels,
// pipeline depth.  LDS per work-group = depth * (bpx + bkc) * 128 bytes.
struct TileD {
    int bpx, bkc, wpx, wch, nst;
};
const TileD kTilesD[] = {
    {128, 128, 2, 2, 2},   // 64 KB: two work-groups per CU, wavefront tile 64 x 64
    {128, 64, 2, 2, 2},    // 48 KB: three per CU, wavefront tile 64 x 32
    {64, 64, 2, 2, 3},     // 48 KB: three per CU, wavefront tile 32 x 32, three stages
    {128, 64, 2, 2, 3},    // tile 1 with a third stage: 72 KB, two per CU
    {128, 64, 2, 2, 1},    // one stage (1x1 only): 34 KB with the channel-last epilogue, four per CU
    {64, 64, 2, 2, 1},     // one stage (1x1 only): 17 KB, eight per CU
};

template <int R_, int S_>
void launch_dma_rs(const ConvArgs &a, int tile, dim3 grid, hipStream_t st)
{
    switch (tile) {
    case 0: launch_dma<R_, S_, 128, 128, 2, 2, 2, 0>(a, grid, st); break;
    case 1: launch_dma<R_, S_, 128, 64, 2, 2, 2, 0>(a, grid, st); break;
    case 2: launch_dma<R_, S_, 64, 64, 2, 2, 3, 0>(a, grid, st); break;
    case 3: launch_dma<R_, S_, 128, 64, 2, 2, 3, 0>(a, grid, st); break;
    default:
        // tiles 4 and 5 are instantiated with one stage for 1x1 layers only
        // (the planner's choice); any other layer gets the same tile shape
        // pipelined
        if constexpr (R_ == 1 && S_ == 1) {
            if (tile == 4) launch_dma<1, 1, 128, 64, 2, 2, 1, 0>(a, grid, st);
            else launch_dma<1, 1, 64, 64, 2, 2, 1, 0>(a, grid, st);
        } else {
            if (tile == 4) launch_dma<R_, S_, 128, 64, 2, 2, 2, 0>(a, grid, st);
            else launch_dma<R_, S_, 64, 64, 2, 2, 3, 0>(a, grid, st);
        }
        break;
    }
}

void launch_dma_nchw(const ConvArgs &a, int tile, int mode, dim3 grid, hipStream_t st)
{
    if (mode == 2) {
        if (tile == 0)
            launch_dma<1, 1, 128, 128, 2, 2, 2, 2>(a, grid, st);
        else if (tile == 3)
            launch_dma<1, 1, 128, 64, 2, 2, 3, 2>(a, grid, st);
        else
            launch_dma<1, 1, 128, 64, 2, 2, 2, 2>(a, grid, st);
    } else if (tile == 0) {
        launch_dma<1, 1, 128, 128, 2, 2, 2, 1>(a, grid, st);
    } else if (tile == 4) {
        launch_dma<1, 1, 128, 64, 2, 2, 1, 1>(a, grid, st);
    } else {
        launch_dma<1, 1, 128, 64, 2, 2, 2, 1>(a, grid, st);
    }
}

// Halo kernel instances: 128 x 128 tiles with patches of up to 192 rows
// (BPX + 2W + 2 rows: W <= 31; 80 KB of LDS, two work-groups per CU), and
// 128 x 64 tiles over one 64-channel block with one patch of up to 256 rows
// and one filter stage (W <= 63; 40 KB, four per CU).
hipError_t launch_halo(const ConvArgs &a, int bkc, int pr, dim3 grid, hipStream_t st)
{
    if (128 + 2 * a.W + 2 > pr || a.R != 3 || a.S != 3 || a.stride != 1 || a.pad != 1 || a.Cg % 64 != 0)
        return hipErrorInvalidValue;
    if (bkc == 128 && pr == 192)
        launch_halo_k<128, 128, 2, 2, 192>(a, grid, st);
    else if (bkc == 64 && pr == 256 && a.Cg == 64 && a.splits == 1)
        launch_halo_k<128, 64, 2, 2, 256, 1>(a, grid, st);
    else
        return hipErrorInvalidValue;
    return hipSuccess;
}

void launch_dma(const ConvArgs &a, int tile, dim3 grid, hipStream_t st)
{
    if (a.R == 1 && a.S == 1)
        launch_dma_rs<1, 1>(a, tile, grid, st);
    else if (a.R == 3 && a.S == 3)
        launch_dma_rs<3, 3>(a, tile, grid, st);
    else
        launch_dma_rs<0, 0>(a, tile, grid, st);
}


}  // namespace

bool nhwc_bf16_eligible(const ConvProblem &p) { return p.Cg % 32 == 0; }

// Direct-to-LDS plan.  Measured on ResNet-50's bf16 layers at batch 64:
// the 128 x 128 tile is fastest while it yields at least 1.5 work-groups per
// CU; below that, 128 x 64 while it still covers every CU, then 64 x 64.
// Filters of at most 64 channels take the 64-wide channel tiles.  A launch
// with fewer than half as many 64 x 64 tiles as CUs splits the reduction.
static NhwcPlan plan_dma(const ConvProblem &p, int num_cus, const void *x, int max_splits, bool x_nhwc)
{
    NhwcPlan plan{};
    plan.dma = 1;
    plan.krc = 64;
    plan.x_nhwc = x_nhwc ? 1 : 0;
    auto wgs = [&](int t) {
        return (long)ceil_div(p.M, kTilesD[t].bpx) * ceil_div(p.Kg, kTilesD[t].bkc) * p.groups;
    };
    const int chunks = p.Kred / 64;
    // Long reductions over few pixels (512-channel 3x3 and 2048-channel 1x1
    // layers at 7x7): 128 x 128 tiles with the reduction split to about 1.5
    // work-groups per CU beat 64 x 64 tiles over the whole reduction
    // (measured at batch 64: 3x3 25 + 8 us reduce vs 44 us; 1x1 15 + 9 vs 28).
    const bool long_red = chunks >= 32 && p.Kg > 64 && wgs(0) * 2 < num_cus;
    if (long_red || (p.Kg > 64 && wgs(0) * 2 >= 3L * num_cus))
        plan.tile = 0;
    else if (wgs(1) >= num_cus)
        plan.tile = 1;
    else
        plan.tile = 2;
    int splits = 1;
    const long tiles = wgs(plan.tile);
    if (long_red) {
        splits = (int)((3L * num_cus / 2 + tiles - 1) / tiles);
        if (splits > chunks / 8) splits = chunks / 8;
        const int per = ceil_div(chunks, splits);
        splits = ceil_div(chunks, per);
    } else if (tiles * 2 < num_cus && chunks >= 8) {
        splits = (int)((num_cus + tiles - 1) / tiles);
        if (splits > chunks / 4) splits = chunks / 4;
        const int per = ceil_div(chunks, splits);
        splits = ceil_div(chunks, per);
    }
    if (splits > max_splits) splits = max_splits;
    plan.splits = splits;
    plan.kr_per_split = ceil_div(chunks, splits) * 64;
    plan.partial_bytes = splits > 1 ? (size_t)splits * p.K * p.M * sizeof(float) : 0;
    // 1x1 stride-1 layers read x in NCHW directly: 16-byte loads when every
    // 8-pixel group lies in one image; for other even planes 4-byte loads, 4x
    // the load instructions, which pays off only for short reductions
    // (measured at batch 64, 14x14: 256 -> 1024 channels 26.4 + 6.7 us copy ->
    // 32.2 us; 1024 -> 256 channels 15.7 + 11.3 us copy -> 28.7 us)
    const bool nchw_ok = !x_nhwc && p.R == 1 && p.S == 1 && p.stride == 1 && p.pad == 0 && plan.tile <= 1;
    plan.nchwb = nchw_ok && (p.H * p.W) % 8 == 0 && (uintptr_t)x % 16 == 0 ? 1
                 : nchw_ok && (p.H * p.W) % 2 == 0 && (uintptr_t)x % 4 == 0 && chunks <= 8 ? 2 : 0;
    // A 128 x 64 grid that fits in two work-groups per CU loses no occupancy
    // to a third LDS stage, which then hides more of the global -> LDS
    // latency (measured at batch 64: 14x14 3x3 layers 33.2 -> 29.2 us,
    // 1024-channel 1x1 at 14x14 19.0 -> 16.0 us; grids of several rounds, as
    // at 56x56, lose 10%).  64 x 64 grids are never larger than that (the
    // planner takes them only when 128 x 64 leaves CUs idle), so tile 2 always
    // has three stages (1024-channel 1x1, stride 2, 14x14 -> 7x7: 17.7 -> 14.1 us).
    if (plan.nchwb != 1 && plan.tile == 1 && wgs(1) * splits <= 2L * num_cus) plan.tile = 3;
    // Channel-last 1x1 layers with at most 4 reduction chunks (ResNet's
    // expansions and projections, the 256-channel reductions at 56x56) are
    // bound by HBM and by each tile's load -> epilogue latency.  One LDS stage
    // (no overlap inside a work-group) leaves room for four 128 x 64 or eight
    // 64 x 64 work-groups per CU, whose loads overlap each other's epilogues
    // (measured at batch 64, bf16 channel-last, against the best two-stage
    // tile: 64 -> 256 at 56x56 with the residual 56.0 -> 51.2 us, 64 -> 256
    // projection 48.6 -> 40.5 us, 128 -> 512 at 28x28 34.7 -> 31.7 us,
    // 256 -> 1024 at 14x14 24.4 -> 21.6 us, 256 -> 64 at 56x56 on 64 x 64
    // tiles 35.3 -> 30.2 us); with more chunks the pipelined tiles stay ahead.
    if (x_nhwc && p.R == 1 && p.S == 1 && chunks <= 4 && splits == 1 && wgs(4) >= num_cus)
        plan.tile = p.Kg >= 128 ? 4 : 5;
    // The same for 1x1 layers reading NCHW x with 16-byte loads (fp32 NCHW
    // output): 128 x 64 one-stage tiles, four per CU (measured at batch 64:
    // 64 -> 256 at 56x56 58.2 -> 54.5 us, 128 -> 512 at 28x28 38.1 -> 34.8 us;
    // the 4-byte-load layers at 14x14 even, so they keep their tiles).
    // Not with a residual: its kernel's registers allow two work-groups per CU.
    if (plan.nchwb == 1 && !p.res && chunks <= 4 && splits == 1 && wgs(4) >= num_cus) plan.tile = 4;
    // 3x3 stride-1 layers on 128 x 128 tiles stage one input patch per
    // 64-channel block for all nine taps (igemm_bf16_halo_kernel; measured at
    // batch 64: 28x28 24.5 -> 22.4 us, 7x7 23.2 -> 21.8 us per launch).  With
    // 128 x 64 tiles its 64-80 KB of LDS cost a work-group per CU: 56x56 32.3
    // -> 35.5 us, 14x14 even.
    if (p.R == 3 && p.S == 3 && p.stride == 1 && p.pad == 1 && plan.tile == 0 && 128 + 2 * p.W + 2 <= 192)
        plan.halo = 192;
    else if (p.R == 3 && p.S == 3 && p.stride == 1 && p.pad == 1 && plan.tile == 1 && p.Cg == 64 &&
             splits == 1 && 128 + 2 * p.W + 2 <= 256)
        plan.halo = 256;
    const ConvProblem cp = copied_problem(p);
    plan.xcl_bytes = plan.nchwb || x_nhwc ? 0 : (size_t)cp.N * cp.C * cp.H * cp.W * sizeof(uint16_t);
    plan.copy_cb = plane_copy_block(p, num_cus);
    return plan;
}

NhwcPlan plan_nhwc_bf16(const ConvProblem &p, int num_cus, const void *x, int max_splits, bool x_nhwc)
{
    // the direct-to-LDS kernel addresses x and w through 32-bit buffer offsets
    const bool fits = (long)p.N * p.C * p.H * p.W * 2 < (1L << 31) &&
                      (long)p.K * p.Cg * p.R * p.S * 2 < (1L << 31);
    if (p.Cg % 64 == 0 && fits) return plan_dma(p, num_cus, x, max_splits, x_nhwc);
    NhwcPlan plan{};
    plan.krc = p.Cg % 64 == 0 ? 64 : 32;
    plan.tile = 1;
    const long target = num_cus;
    for (int t = 0; t < 2; ++t) {
        const long tiles = (long)ceil_div(p.M, kTilesN[t].bpx) * ceil_div(p.Kg, kTilesN[t].bkc) * p.groups;
        if (tiles < target && t == 0) continue;
        plan.tile = t;
        const int chunks = p.Kred / plan.krc;
        int splits = tiles < target ? (int)((target + tiles - 1) / tiles) : 1;
        if (splits > chunks / 2) splits = chunks / 2;
        if (splits > max_splits) splits = max_splits;
        if (splits < 1) splits = 1;
        const int per = ceil_div(chunks, splits);
        splits = ceil_div(chunks, per);
        plan.splits = splits;
        plan.kr_per_split = per * plan.krc;
        plan.partial_bytes = splits > 1 ? (size_t)splits * p.K * p.M * sizeof(float) : 0;
        break;
    }
    const ConvProblem cp = copied_problem(p);
    plan.xcl_bytes = (size_t)cp.N * cp.C * cp.H * cp.W * sizeof(uint16_t);
    plan.copy_cb = plane_copy_block(p, num_cus);
    return plan;
}

void describe_nhwc_bf16(const ConvProblem &p, const NhwcPlan &plan, char *buf, int len,
                        int *launches)
{
    int R = rs_template(p.R), S = rs_template(p.S);
    if (R != S) R = S = 0;
    char tname[64];
    const int rv = copy_read_width(p, nullptr);
    if (rv == 0)
        snprintf(tname, sizeof tname, "nchw_to_nhwc_plane_bf16_kernel + ");
    else if (rv < 0)
        snprintf(tname, sizeof tname, "nchw_to_nhwc_sampled_bf16_kernel<%d> + ", -rv);
    else
        snprintf(tname, sizeof tname, "nchw_to_nhwc_bf16_kernel<%d> + ", rv);
    const bool copy = !plan.nchwb && !plan.x_nhwc;
    const char *variant = p.ycl ? "_cl" : p.res && plan.splits == 1 ? "_res" : "";
    const char *reduce = plan.splits == 1 ? "" : p.ycl ? " + splitk_reduce_cl_kernel" : " + splitk_reduce_kernel";
    if (plan.dma && plan.halo) {
        const TileD &d = kTilesD[plan.tile];
        snprintf(buf, len, "%sigemm_bf16_halo%s_kernel<%d, %d, 2, 2, %d, %d>%s", copy ? tname : "", variant,
                 d.bpx, d.bkc, plan.halo, d.bkc == 64 ? 1 : 2, reduce);
        *launches = (copy ? 2 : 1) + (plan.splits > 1 ? 1 : 0);
        return;
    }
    if (plan.dma) {
        const TileD &d = kTilesD[plan.tile];
        // the instantiation's full name, reduction chunk included (every launch uses 64)
        snprintf(buf, len, "%sigemm_bf16_dma%s_kernel<%d, %d, %d, %d, %d, %d, %d, %d, 64>%s", copy ? tname : "",
                 variant, R, S, d.bpx, d.bkc, d.wpx, d.wch, d.nst, plan.nchwb, reduce);
        *launches = (copy ? 2 : 1) + (plan.splits > 1 ? 1 : 0);
        return;
    } else {
        const TileN &t = kTilesN[plan.tile];
        snprintf(buf, len, "%sigemm_bf16_nhwc_kernel<%d, %d, %d, %d, %d>%s", tname, R, S, t.bkc,
                 t.bpx, plan.krc,
                 plan.splits > 1 ? " + splitk_reduce_kernel" : "");
    }
    *launches = plan.splits > 1 ? 3 : 2;
}

hipError_t launch_nhwc_bf16(const ConvProblem &p, const NhwcPlan &plan, const uint16_t *x,
                            const uint16_t *w_krsc, const float *bias, float *y, uint16_t *xcl,
                            float *partials, hipStream_t st, const LaunchHook *hook)
{
    hipError_t e = hipSuccess;
    if (plan.dma && plan.nchwb) {
        ConvArgs a = make_args(p);
        a.x = x;
        a.w = w_krsc;
        a.bias = bias;
        a.y = y;
        a.ws = plan.splits > 1 ? partials : nullptr;
        a.splits = plan.splits;
        a.kr_per_split = plan.kr_per_split;
        const TileD &d = kTilesD[plan.tile];
        const long wgs = (long)ceil_div(p.M, d.bpx) * ceil_div(p.Kg, d.bkc) * p.groups * plan.splits;
        if (hook && (e = hook->before_launch(hook->ctx, st)) != hipSuccess) return e;
        launch_dma_nchw(a, plan.tile, plan.nchwb, dim3((unsigned)wgs), st);
        if ((e = hipGetLastError()) != hipSuccess || plan.splits == 1) return e;
        if (hook && (e = hook->before_launch(hook->ctx, st)) != hipSuccess) return e;
        return launch_splitk_reduce(a, st);
    }
    if (plan.x_nhwc) {
        // x is already channel-last: the GEMM reads it as given, strides included
        if (!plan.dma) return hipErrorInvalidValue;
        ConvArgs a = make_args(p);
        a.x = x;
        a.w = w_krsc;
        a.bias = bias;
        a.y = y;
        a.ws = plan.splits > 1 ? partials : nullptr;
        a.splits = plan.splits;
        a.kr_per_split = plan.kr_per_split;
        const TileD &d = kTilesD[plan.tile];
        const long wgs = (long)ceil_div(p.M, d.bpx) * ceil_div(p.Kg, d.bkc) * p.groups * plan.splits;
        if (hook && (e = hook->before_launch(hook->ctx, st)) != hipSuccess) return e;
        if (plan.halo) {
            if ((e = launch_halo(a, d.bkc, plan.halo, dim3((unsigned)wgs), st)) != hipSuccess) return e;
        } else
            launch_dma(a, plan.tile, dim3((unsigned)wgs), st);
        if ((e = hipGetLastError()) != hipSuccess || plan.splits == 1) return e;
        if (hook && (e = hook->before_launch(hook->ctx, st)) != hipSuccess) return e;
        return launch_splitk_reduce(a, st);
    }
    e = hook ? hook->before_launch(hook->ctx, st) : hipSuccess;
    if (e != hipSuccess) return e;
    if (p.C % 8 != 0) return hipErrorInvalidValue;   // every channel-last path has C % 32 == 0
    const ConvProblem cp = copied_problem(p);
    NhwcCopyArgs ca{};
    ca.x = x;
    ca.xt = xcl;
    ca.C = p.C;
    ca.H = p.H;
    ca.W = p.W;
    ca.Q = cp.W;
    ca.S = copy_subsamples(p) ? p.stride : 1;
    ca.HW = p.H * p.W;
    ca.PQ = cp.H * cp.W;
    ca.npq = p.N * ca.PQ;
    ca.tiles_c = ceil_div(p.C, 64);
    ca.dv_hw = make_fastdiv(ca.HW);
    ca.dv_pq = make_fastdiv(ca.PQ);
    ca.dv_q = make_fastdiv(ca.Q);
    const int rv = copy_read_width(p, x);
    const dim3 tg((unsigned)((long)ceil_div(ca.npq, 64) * ca.tiles_c)), tb(256);
    if (rv == 0) {
        // the block must fit the kernel's LDS buffer (32 * H*W always does here)
        ca.cb = plan.copy_cb >= 8 ? plan.copy_cb : 64;
        while (ca.cb > 8 && ca.cb * ca.HW > kPlaneElems) ca.cb /= 2;
        ca.tiles_c = ceil_div(p.C, ca.cb);
        launch_kernel(nchw_to_nhwc_plane_bf16_kernel, dim3((unsigned)((long)p.N * ca.tiles_c)), tb, 0, st, ca);
    }
    else if (rv == 8)
        launch_kernel(nchw_to_nhwc_bf16_kernel<8>, tg, tb, 0, st, ca);
    else if (rv == 4)
        launch_kernel(nchw_to_nhwc_bf16_kernel<4>, tg, tb, 0, st, ca);
    else if (rv == -4)
        launch_kernel(nchw_to_nhwc_sampled_bf16_kernel<4>, tg, tb, 0, st, ca);
    else if (rv == -2)
        launch_kernel(nchw_to_nhwc_sampled_bf16_kernel<2>, tg, tb, 0, st, ca);
    else
        launch_kernel(nchw_to_nhwc_bf16_kernel<1>, tg, tb, 0, st, ca);
    if ((e = hipGetLastError()) != hipSuccess) return e;

    ConvArgs a = make_args(cp);
    a.x = xcl;
    a.w = w_krsc;
    a.bias = bias;
    a.y = y;
    a.ws = plan.splits > 1 ? partials : nullptr;
    a.splits = plan.splits;
    a.kr_per_split = plan.kr_per_split;
    if (hook && (e = hook->before_launch(hook->ctx, st)) != hipSuccess) return e;
    if (plan.dma) {
        const TileD &d = kTilesD[plan.tile];
        const long wgs = (long)ceil_div(p.M, d.bpx) * ceil_div(p.Kg, d.bkc) * p.groups * plan.splits;
        if (plan.halo) {
            if ((e = launch_halo(a, d.bkc, plan.halo, dim3((unsigned)wgs), st)) != hipSuccess) return e;
        } else
            launch_dma(a, plan.tile, dim3((unsigned)wgs), st);
        if ((e = hipGetLastError()) != hipSuccess || plan.splits == 1) return e;
        if (hook && (e = hook->before_launch(hook->ctx, st)) != hipSuccess) return e;
        return launch_splitk_reduce(a, st);
    }
    const TileN &t = kTilesN[plan.tile];
    dim3 grid(ceil_div(p.M, t.bpx), ceil_div(p.Kg, t.bkc), p.groups * plan.splits);
    if (plan.krc == 64)
        launch_krc<64>(a, plan.tile, grid, st);
    else
        launch_krc<32>(a, plan.tile, grid, st);
    if ((e = hipGetLastError()) != hipSuccess || plan.splits == 1) return e;
    if (hook && (e = hook->before_launch(hook->ctx, st)) != hipSuccess) return e;
    return launch_splitk_reduce(a, st);
}

}  // namespace miconv
