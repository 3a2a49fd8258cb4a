// CONVGEMM on gfx950: the convolution O = conv(F, I) as one fp32 matrix product
// O^ = F^ . im2col(I) whose second operand is gathered from the input tensor
// while it is staged into LDS (the paper's section 4, Figure 6: im2col folded
// into the packing of the GEMM's B operand, so the augmented matrix of
// section 3 is never formed in memory).
//
// Mapping to CDNA4.  One workgroup (4 waves, 2 x 2) owns an MT x NT tile of O^
// (MT filters x NT output positions).  The contraction runs in chunks of
// KC = 16 or 32 rows of im2col(I) (= columns of F^):
//   * F^ chunk (MT x KC): coalesced loads along the filter index, kept in LDS
//     as rows of KC contraction values per filter;
//   * im2col chunk (KC x NT): each thread owns one output position (column)
//     of the tile, decoded once into (oh, ow, n), and walks its contraction
//     rows r -> (y, x, c) incrementally; the value is I at
//     (s*oh + y - p, s*ow + x - p, c, n) or zero outside the input, exactly
//     Figure 6's index maps.  Neighbouring threads hold neighbouring output
//     positions, so each load instruction reads a contiguous (stride s) run of
//     one input row.  Stored in LDS as KC contraction values per column;
//   * v_mfma_f32_16x16x4_f32 on 16 x 16 blocks.  Because the contraction may
//     be taken in any order, lane group q of a wave (lanes 16q .. 16q+15)
//     takes contraction rows 4q .. 4q+3 of each group of 16 for that group's
//     four MFMAs, so one ds_read_b128 feeds four MFMAs;
//   * two LDS buffers: the next chunk's global loads are issued before the
//     current chunk's MFMAs and written to the other buffer after them, one
//     barrier per chunk.
// Tiles are handed out XCD-aware: consecutive workgroup ids go to different
// XCDs (round-robin), so ids are remapped to give each XCD a contiguous range of
// tiles, filter tiles fastest; tiles that share output positions (and the input
// rows they read) then run on the same XCD and share its L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "convgemm.h"

namespace convgemm {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kDirectMaxK = 16384;   // register-direct kernel: its row table (4 bytes a row) fits 64 KiB of LDS

struct Geometry {
    int M, K, N;        // kn, kh*kw*ci, ho*wo*b
    int kh, khw;        // kh, kh*kw
    int kw;
    int hi, wi, hiwi;   // input height, width, hi*wi
    int ho, hw;         // ho, ho*wo
    int s, p;
    int64_t sample;     // hi*wi*ci: input floats per batch entry
    uint32_t ibytes;    // bytes of I (< 2^32)
    uint32_t fbytes;    // bytes of F (< 2^32)
};

// Raw buffer resource over a whole tensor: base address, no stride, the
// tensor's size in bytes as the range, 32-bit data format.  A buffer load
// then takes a per-lane byte offset (vector) plus a wave-uniform byte offset
// (scalar), so the gather needs no per-element address arithmetic.
__device__ inline __amdgpu_buffer_rsrc_t tensor_rsrc(const float* p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ inline float buffer_load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, 0));
}

// One lane's share of a 16 x 16 output block: filters m .. m+3 of output
// position n (the v_mfma_f32_16x16x4_f32 result layout), contiguous in O;
// one 16-byte store when kn is a multiple of 4 and O is 16-byte aligned (vec).
__device__ inline void store_block(float* __restrict__ O, const Geometry& g, int m, int n, f4 v, int accumulate,
                                   int vec)
{
    if (n >= g.N || m >= g.M) return;
    float* o = O + (int64_t)n * g.M + m;
    if (vec) {
        if (accumulate) v += *reinterpret_cast<const f4*>(o);
        *reinterpret_cast<f4*>(o) = v;
    } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (m + q < g.M) o[q] = accumulate ? o[q] + v[q] : v[q];
    }
}

template <int MT, int NT, bool PAD, int KC>
__global__ __launch_bounds__(kThreads) void convgemm_kernel(Geometry g, const float* __restrict__ F,
                                                            const float* __restrict__ I,
                                                            float* __restrict__ O, int accumulate,
                                                            int vec, int mtiles, int ntiles)
{
    constexpr int kKC = KC;                        // contraction rows per staged chunk
    constexpr int kKP = KC + 4;                    // LDS floats per tile row (padded against bank conflicts)
    constexpr int WM = MT / 2, WN = NT / 2;        // wave tile
    constexpr int BM = WM / 16, BN = WN / 16;      // 16 x 16 blocks per wave
    constexpr int AK = MT == 192 ? kKC : MT * kKC / kThreads; // contraction rows per F^-loading thread
    constexpr int ATHREADS = MT * kKC / AK;        // threads that load F^ (whole waves)
    constexpr int RPT = kKC * NT / kThreads;       // im2col rows per thread per chunk
    static_assert(ATHREADS <= kThreads && ATHREADS % 64 == 0 && ATHREADS * AK == MT * kKC && AK % 4 == 0,
                  "F^ loader split");
    static_assert(RPT * kThreads == kKC * NT && RPT % 4 == 0 && BM >= 1 && BN >= 1 && kKC % 16 == 0,
                  "tile shape");

    __shared__ __attribute__((aligned(16))) float As[2][MT * kKP];
    __shared__ __attribute__((aligned(16))) float Bs[2][NT * kKP];

    // XCD-aware tile order: within the largest multiple of 8 of the tile
    // count, workgroup id -> XCD (id mod 8) gets the contiguous tile range
    // [xcd * T8/8, (xcd + 1) * T8/8); the remainder keeps the identity.
    const int T = mtiles * ntiles;
    const int T8 = T & ~7;
    const int bid = blockIdx.x;
    const int t = bid < T8 ? (bid & 7) * (T8 >> 3) + (bid >> 3) : bid;
    const int m0 = (t % mtiles) * MT;
    const int n0 = (t / mtiles) * NT;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;

    // F^ loader: filter am (clamped: rows past kn only feed outputs that are
    // never stored), contraction rows akg .. akg+AK-1 of each chunk.
    const bool a_loader = tid < ATHREADS;            // whole waves
    const int am = tid % MT;
    const int akg = (tid / MT) * AK;
    const int am_c = min(m0 + am, g.M - 1);
    const uint32_t aoff = (uint32_t)(akg * g.M + am_c) * 4u;   // bytes from row k0 of F^

    // im2col gatherer: output position bcol of the tile (clamped to the last
    // one: columns past N only feed outputs that are never stored), decoded
    // once into (oh, ow, n); contraction rows brow .. brow+RPT-1 of each chunk.
    // brow is the same for a whole wave, so the row -> (y, x, c) walk and the
    // row's offset y + hi*x + hi*wi*c live in scalar registers.
    const int bcol = tid % NT;
    const int brow = __builtin_amdgcn_readfirstlane((tid / NT) * RPT);
    const int ncol = min(n0 + bcol, g.N - 1);
    const int nb = ncol / g.hw;
    const int prem = ncol - nb * g.hw;
    const int ow = prem / g.ho;
    const int oh = prem - ow * g.ho;
    const int hbase = oh * g.s - g.p;
    const int wbase = ow * g.s - g.p;
    // without padding every tap of a valid column is inside the input: the
    // element is I[colpos + row offset], colpos < 2^30 (checked on the host)
    const uint32_t colbyte = PAD ? 0u : (uint32_t)(nb * g.sample + hbase + g.hi * wbase) * 4u;
    const float* __restrict__ Ib = I + (int64_t)nb * g.sample;
    const __amdgpu_buffer_rsrc_t irs = tensor_rsrc(I, g.ibytes);
    const __amdgpu_buffer_rsrc_t frs = tensor_rsrc(F, g.fbytes);

    float ra[AK];
    float rb[RPT];
    uint32_t amask = ~0u, bmask = ~0u;   // bit j: value j is a real entry (else stored as 0)

    auto load_chunk = [&](int chunk) {
        const int k0 = chunk * kKC;
        const bool tail = k0 + kKC > g.K;            // uniform: only the last chunk can be partial
        if (a_loader) {
            if (!tail) {
#pragma unroll
                for (int i = 0; i < AK; ++i) ra[i] = buffer_load(frs, aoff, (uint32_t)(k0 + i) * g.M * 4u);
                amask = ~0u;
            } else {
                amask = 0;
#pragma unroll
                for (int i = 0; i < AK; ++i) {
                    const int k = k0 + akg + i;
                    const bool ok = k < g.K;
                    ra[i] = F[(int64_t)(ok ? k : g.K - 1) * g.M + am_c];
                    amask |= (uint32_t)ok << i;
                }
            }
        }
        const int r0 = k0 + brow;
        int c = r0 / g.khw;
        const int rem = r0 - c * g.khw;
        int x = rem / g.kh;
        int y = rem - x * g.kh;
        bmask = 0;
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            const bool rok = r0 + j < g.K;           // uniform
            if (!PAD) {
                const int roff = rok ? y + g.hi * x + g.hiwi * c : 0;
                rb[j] = buffer_load(irs, colbyte, (uint32_t)roff * 4u);
                bmask |= (uint32_t)rok << j;
            } else {
                const int hh = hbase + y, ww = wbase + x;
                const bool ok = rok && (unsigned)hh < (unsigned)g.hi && (unsigned)ww < (unsigned)g.wi;
                const float v = Ib[ok ? hh + g.hi * ww + g.hiwi * c : 0];
                rb[j] = v;
                bmask |= (uint32_t)ok << j;
            }
            // next contraction row: y fastest, then x, then c
            ++y;
            const bool wy = y == g.kh;
            y = wy ? 0 : y;
            x += wy;
            const bool wx = x == g.kw;
            x = wx ? 0 : x;
            c += wx;
        }
    };

    // The zeroing is applied here, after the MFMAs, so that nothing waits for
    // the loads before the MFMAs are issued; full chunks without padding store
    // the loaded values as they are.
    auto store_chunk = [&](int buf, bool tail) {
        if (a_loader) {
            float* ap = &As[buf][am * kKP + akg];
#pragma unroll
            for (int i = 0; i < AK; i += 4) {
                f4 v = f4{ra[i], ra[i + 1], ra[i + 2], ra[i + 3]};
                if (tail) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) v[q] = (amask >> (i + q)) & 1 ? v[q] : 0.0f;
                }
                *reinterpret_cast<f4*>(ap + i) = v;
            }
        }
        float* bp = &Bs[buf][bcol * kKP + brow];
#pragma unroll
        for (int j = 0; j < RPT; j += 4) {
            f4 v = f4{rb[j], rb[j + 1], rb[j + 2], rb[j + 3]};
            if (PAD || tail) {
#pragma unroll
                for (int q = 0; q < 4; ++q) v[q] = (bmask >> (j + q)) & 1 ? v[q] : 0.0f;
            }
            *reinterpret_cast<f4*>(bp + j) = v;
        }
    };

    f4 acc[BM][BN];
#pragma unroll
    for (int i = 0; i < BM; ++i)
#pragma unroll
        for (int j = 0; j < BN; ++j) acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};

    // Each group of 16 contraction rows: lane group q = lane/16 takes rows
    // 4q .. 4q+3 of the group, one per MFMA of the group's four.
    auto compute = [&](int buf) {
        const float* ap = &As[buf][(wm * WM + (lane & 15)) * kKP + 4 * (lane >> 4)];
        const float* bp = &Bs[buf][(wn * WN + (lane & 15)) * kKP + 4 * (lane >> 4)];
#pragma unroll
        for (int g16 = 0; g16 < kKC; g16 += 16) {
            f4 a[BM], b[BN];
#pragma unroll
            for (int i = 0; i < BM; ++i) a[i] = *reinterpret_cast<const f4*>(ap + i * 16 * kKP + g16);
#pragma unroll
            for (int j = 0; j < BN; ++j) b[j] = *reinterpret_cast<const f4*>(bp + j * 16 * kKP + g16);
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
#pragma unroll
                for (int i = 0; i < BM; ++i)
#pragma unroll
                    for (int j = 0; j < BN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][kk], b[j][kk], acc[i][j], 0, 0, 0);
        }
    };

    const int nchunks = (g.K + kKC - 1) / kKC;
    load_chunk(0);
    store_chunk(0, kKC > g.K);
    __syncthreads();
    // The scheduling barriers keep the next chunk's loads ahead of the MFMAs
    // and their LDS stores behind them, so the loads' latency is covered.
    for (int chunk = 0; chunk + 1 < nchunks; ++chunk) {
        const int buf = chunk & 1;
        load_chunk(chunk + 1);
        __builtin_amdgcn_sched_barrier(0);
        compute(buf);
        __builtin_amdgcn_sched_barrier(0);
        store_chunk(buf ^ 1, (chunk + 2) * kKC > g.K);
        __syncthreads();
    }
    compute((nchunks - 1) & 1);

    // Epilogue: lane holds rows 4*(lane/16) .. +3 of column lane%16 of each
    // 16 x 16 block.
#pragma unroll
    for (int i = 0; i < BM; ++i)
#pragma unroll
        for (int j = 0; j < BN; ++j)
            store_block(O, g, m0 + wm * WM + i * 16 + 4 * (lane >> 4), n0 + wn * WN + j * 16 + (lane & 15),
                        acc[i][j], accumulate, vec);
}

// Register-direct CONVGEMM (no padding): every wave loads the operand values
// its own MFMAs consume straight into registers, so there is no LDS staging
// and no barrier in the contraction loop; waves run independently and the
// operands they share (F^ rows between the two waves of a tile row, input
// positions between the two of a tile column, and the im2col duplication of
// the input) are served by the L1 and L2 caches.
//
// Tile: 4 waves (2 x 2), wave tile 16BM x 16BN, workgroup tile 32BM x 32BN.
// Contraction in groups of 16 rows; lane group q = lane/16 takes rows
// 4q .. 4q+3 of a group, one per MFMA, so that:
//   * F^ value (filter m, row k0 + 4q + kk): byte (k0 + kk)*4kn [wave-uniform,
//     the scalar offset] + (4q kn + m)*4 [per lane, fixed];
//   * im2col value (row k0 + 4q + kk, position n): byte colpos(n) [per lane,
//     fixed] + rowoff(k0 + 4q + kk) [per lane group], where rowoff(r) =
//     4 (y + hi x + hi wi c) comes from a table of all rows built in LDS when
//     the workgroup starts (one ds_read_b128 gives a lane its four rows of a
//     group).  Without padding every tap of a valid position is inside the
//     input, so no element needs a check.
// Two register sets pipeline the groups: the next group's loads are issued
// before the current group's MFMAs.
// O += v with one atomic add per element: the contraction of a tile split
// over several workgroups (O cleared first unless accumulating).
__device__ inline void add_block(float* __restrict__ O, const Geometry& g, int m, int n, f4 v)
{
    if (n >= g.N || m >= g.M) return;
    float* o = O + (int64_t)n * g.M + m;
#pragma unroll
    for (int q = 0; q < 4; ++q)
        if (m + q < g.M) unsafeAtomicAdd(o + q, v[q]);
}

__global__ void zero_kernel(float* __restrict__ O, int64_t count)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x)
        O[i] = 0.0f;
}

template <int BM, int BN, bool SPLIT>
__global__ __launch_bounds__(kThreads) void convgemm_direct_kernel(Geometry g, const float* __restrict__ F,
                                                                   const float* __restrict__ I,
                                                                   float* __restrict__ O, int accumulate,
                                                                   int vec, int mtiles, int ntiles, int kpad,
                                                                   int kparts)
{
    constexpr int WM = 16 * BM, WN = 16 * BN;
    constexpr int MT = 2 * WM, NT = 2 * WN;
    extern __shared__ int rowoff[];                // kpad entries; rows past K read offset 0
    // workgroup T * part + b takes groups [part * G / kparts, (part + 1) * G /
    // kparts) of the contraction of tile b; only its rows' offsets are formed
    const int T = mtiles * ntiles;
    const int ngroups = (g.K + 15) / 16;
    int part = 0, glo = 0, ghi = ngroups;
    if (SPLIT) {
        part = blockIdx.x / T;
        glo = part * ngroups / kparts;
        ghi = (part + 1) * ngroups / kparts;
    }
    for (int r = glo * 16 + threadIdx.x; r < ghi * 16; r += kThreads) {
        int v = 0;
        if (r < g.K) {
            const int c = r / g.khw, rem = r - c * g.khw, x = rem / g.kh, y = rem - x * g.kh;
            v = (y + g.hi * x + g.hiwi * c) * 4;
        }
        rowoff[r] = v;
    }
    __syncthreads();

    // XCD-aware tile order, as in the LDS-staged kernel
    const int T8 = T & ~7;
    const int bid = blockIdx.x - part * T;
    const int t = bid < T8 ? (bid & 7) * (T8 >> 3) + (bid >> 3) : bid;
    const int m0 = (t % mtiles) * MT;
    const int n0 = (t / mtiles) * NT;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int q = lane >> 4, l16 = lane & 15;
    const __amdgpu_buffer_rsrc_t irs = tensor_rsrc(I, g.ibytes);
    const __amdgpu_buffer_rsrc_t frs = tensor_rsrc(F, g.fbytes);

    // per-lane fixed offsets; filters and positions past the edge are clamped
    // (they only feed outputs that are never stored)
    int am[BM];
    uint32_t aoff[BM], coff[BN];
#pragma unroll
    for (int i = 0; i < BM; ++i) {
        am[i] = min(m0 + wm * WM + 16 * i + l16, g.M - 1);
        aoff[i] = (uint32_t)(4 * q * g.M + am[i]) * 4u;
    }
#pragma unroll
    for (int j = 0; j < BN; ++j) {
        const int n = min(n0 + wn * WN + 16 * j + l16, g.N - 1);
        const int nb = n / g.hw, rem = n - nb * g.hw, ow = rem / g.ho, oh = rem - ow * g.ho;
        coff[j] = (uint32_t)(nb * g.sample + oh * g.s + g.hi * (ow * g.s)) * 4u;
    }

    f4 acc[BM][BN];
#pragma unroll
    for (int i = 0; i < BM; ++i)
#pragma unroll
        for (int j = 0; j < BN; ++j) acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};

    float a[2][BM][4], b[2][BN][4];
    auto load = [&](int grp, int set) {
        const int k0 = grp * 16;
        const int4 r4 = *reinterpret_cast<const int4*>(&rowoff[k0 + 4 * q]);
        const uint32_t rr[4] = {(uint32_t)r4.x, (uint32_t)r4.y, (uint32_t)r4.z, (uint32_t)r4.w};
        if (k0 + 16 <= g.K) {
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
                for (int i = 0; i < BM; ++i) a[set][i][kk] = buffer_load(frs, aoff[i], (uint32_t)(k0 + kk) * g.M * 4u);
#pragma unroll
                for (int j = 0; j < BN; ++j) b[set][j][kk] = buffer_load(irs, coff[j] + rr[kk], 0u);
            }
        } else {
            // last, partial group: F^ rows past K are loaded clamped and zeroed
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const int row = k0 + 4 * q + kk;
                const bool ok = row < g.K;
                const int rc = ok ? row : g.K - 1;
#pragma unroll
                for (int i = 0; i < BM; ++i) {
                    const float v = buffer_load(frs, (uint32_t)(rc * g.M + am[i]) * 4u, 0u);
                    a[set][i][kk] = ok ? v : 0.0f;
                }
#pragma unroll
                for (int j = 0; j < BN; ++j) b[set][j][kk] = buffer_load(irs, coff[j] + rr[kk], 0u);
            }
        }
    };
    auto compute = [&](int set) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
#pragma unroll
            for (int i = 0; i < BM; ++i)
#pragma unroll
                for (int j = 0; j < BN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[set][i][kk], b[set][j][kk], acc[i][j], 0, 0, 0);
    };

    int grp = glo;
    if (grp < ghi) load(grp, 0);
    for (; grp + 2 <= ghi; grp += 2) {
        load(grp + 1, 1);
        __builtin_amdgcn_sched_barrier(0);
        compute(0);
        __builtin_amdgcn_sched_barrier(0);
        if (grp + 2 < ghi) load(grp + 2, 0);
        __builtin_amdgcn_sched_barrier(0);
        compute(1);
        __builtin_amdgcn_sched_barrier(0);
    }
    if (grp < ghi) compute(0);

    if (SPLIT) {
#pragma unroll
        for (int i = 0; i < BM; ++i)
#pragma unroll
            for (int j = 0; j < BN; ++j)
                add_block(O, g, m0 + wm * WM + 16 * i + 4 * q, n0 + wn * WN + 16 * j + l16, acc[i][j]);
        return;
    }

#pragma unroll
    for (int i = 0; i < BM; ++i)
#pragma unroll
        for (int j = 0; j < BN; ++j)
            store_block(O, g, m0 + wm * WM + 16 * i + 4 * q, n0 + wn * WN + 16 * j + l16, acc[i][j], accumulate,
                        vec);
}

int out_size(int h, int k, int s, int p)
{
    if (k < 1 || s < 1 || p < 0 || h < 1) return -1;
    const int64_t span = (int64_t)h - k + 2 * (int64_t)p;
    if (span < 0) return -1;
    return (int)(span / s + 1);
}

struct Tile {
    int mt, nt;
};

// Tile choice (measured on the AlexNet layers): 128 x 128 tiles when the
// filter count is a multiple of 128 and they still give at least four
// workgroups per compute unit; otherwise 64 x 64 tiles, whose small register
// and LDS footprint keeps four or more workgroups resident per compute unit.
Tile choose_tile(int M, int N, int cus)
{
    const int64_t t128 = (int64_t)((M + 127) / 128) * ((N + 127) / 128);
    if (M % 128 == 0 && t128 >= 4 * (int64_t)cus) return Tile{128, 128};
    return Tile{64, 64};
}

// KC: 32-row chunks when the grid is short (fewer than four tiles per compute
// unit: long contractions over few output positions, where fewer and larger
// chunks pay), else 16-row chunks (smaller LDS footprint, more resident
// workgroups).
template <int MT, int NT>
hipError_t launch(const Geometry& g, const float* F, const float* I, float* O, int accumulate, int vec,
                  int cus, hipStream_t stream)
{
    const int mtiles = (g.M + MT - 1) / MT;
    const int ntiles = (g.N + NT - 1) / NT;
    const int64_t tiles = (int64_t)mtiles * ntiles;
    if (tiles > 0x7fffffff) return hipErrorInvalidConfiguration;
    const bool long_k = tiles < 4 * (int64_t)cus;
    const dim3 grid((unsigned)tiles), block(kThreads);
    if (g.p == 0 && !long_k)
        hipLaunchKernelGGL((convgemm_kernel<MT, NT, false, 16>), grid, block, 0, stream, g, F, I, O, accumulate, vec,
                           mtiles, ntiles);
    else if (g.p == 0)
        hipLaunchKernelGGL((convgemm_kernel<MT, NT, false, 32>), grid, block, 0, stream, g, F, I, O, accumulate, vec,
                           mtiles, ntiles);
    else if (!long_k)
        hipLaunchKernelGGL((convgemm_kernel<MT, NT, true, 16>), grid, block, 0, stream, g, F, I, O, accumulate, vec,
                           mtiles, ntiles);
    else
        hipLaunchKernelGGL((convgemm_kernel<MT, NT, true, 32>), grid, block, 0, stream, g, F, I, O, accumulate, vec,
                           mtiles, ntiles);
    return hipGetLastError();
}

// kparts: workgroups sharing one tile's contraction (atomic adds into O)
template <int BM, int BN>
hipError_t launch_direct(const Geometry& g, const float* F, const float* I, float* O, int accumulate, int vec,
                         int kparts, hipStream_t stream)
{
    const int mtiles = (g.M + 32 * BM - 1) / (32 * BM);
    const int ntiles = (g.N + 32 * BN - 1) / (32 * BN);
    const int64_t tiles = (int64_t)mtiles * ntiles;
    if (tiles * kparts > 0x7fffffff) return hipErrorInvalidConfiguration;
    const int kpad = (g.K + 15) / 16 * 16;
    if (kparts > 1 && !accumulate) {
        const int64_t count = (int64_t)g.M * g.N;
        const int64_t blocks = std::min<int64_t>((count + 255) / 256, 4096);
        hipLaunchKernelGGL(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, O, count);
    }
    if (kparts > 1)
        hipLaunchKernelGGL((convgemm_direct_kernel<BM, BN, true>), dim3((unsigned)(tiles * kparts)), dim3(kThreads),
                           (size_t)kpad * sizeof(int), stream, g, F, I, O, accumulate, vec, mtiles, ntiles, kpad, kparts);
    else
        hipLaunchKernelGGL((convgemm_direct_kernel<BM, BN, false>), dim3((unsigned)tiles), dim3(kThreads),
                           (size_t)kpad * sizeof(int), stream, g, F, I, O, accumulate, vec, mtiles, ntiles, kpad, 1);
    return hipGetLastError();
}

int device_cus()
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        return 256;
    return cus;
}

}  // namespace
}  // namespace convgemm

extern "C" int convgemm_out_size(int h, int k, int stride, int pad)
{
    return convgemm::out_size(h, k, stride, pad);
}

extern "C" int convgemm_f32(int kn, int kh, int kw, int ci, int hi, int wi, int b, int stride, int pad,
                            const float* F, const float* I, float* O, int accumulate, int path, int mt, int nt,
                            hipStream_t stream)
{
    using namespace convgemm;
    if (kn < 1) return -1;
    if (kh < 1) return -2;
    if (kw < 1) return -3;
    if (ci < 1) return -4;
    if (hi < 1) return -5;
    if (wi < 1) return -6;
    if (b < 0) return -7;
    if (stride < 1) return -8;
    if (pad < 0) return -9;
    const int ho = out_size(hi, kh, stride, pad);
    const int wo = out_size(wi, kw, stride, pad);
    if (ho < 1) return -5;
    if (wo < 1) return -6;
    if ((int64_t)hi * wi * ci >= ((int64_t)1 << 31)) return -5;
    if ((int64_t)kh * kw * ci >= ((int64_t)1 << 31)) return -2;
    if ((int64_t)ho * wo * b >= ((int64_t)1 << 31)) return -7;
    if ((int64_t)hi * wi * ci * b >= ((int64_t)1 << 30)) return -7;
    if (kn >= (1 << 24) || (int64_t)kn * kh * kw * ci >= ((int64_t)1 << 30)) return -1;
    if (accumulate != 0 && accumulate != 1) return -13;
    // path: 0 automatic, 1 LDS-staged gather, 2 register-direct (no padding,
    // contraction up to kDirectMaxK rows: its row table lives in LDS)
    const int64_t kk = (int64_t)kh * kw * ci;
    if (path < 0 || path > 2 || (path == 2 && (pad != 0 || kk > kDirectMaxK)) || (path == 0 && (mt || nt)))
        return -14;
    const bool lds_tile = (mt == 64 && (nt == 64 || nt == 128 || nt == 256)) || (mt == 128 && nt == 128) ||
                          (mt == 192 && nt == 128);
    const bool direct_tile = (mt == 64 || mt == 128) && (nt == 64 || nt == 128);
    if (path == 1 && !(lds_tile || (mt == 0 && nt == 0))) return -15;
    if (path == 2 && !(direct_tile || (mt == 0 && nt == 0))) return -15;
    if (b == 0) return CONVGEMM_OK;
    if (!F) return -10;
    if (!I) return -11;
    if (!O) return -12;

    Geometry g;
    g.M = kn;
    g.K = kh * kw * ci;
    g.N = ho * wo * b;
    g.kh = kh;
    g.kw = kw;
    g.khw = kh * kw;
    g.hi = hi;
    g.wi = wi;
    g.hiwi = hi * wi;
    g.ho = ho;
    g.hw = ho * wo;
    g.s = stride;
    g.p = pad;
    g.sample = (int64_t)hi * wi * ci;
    g.ibytes = (uint32_t)(g.sample * b * 4);
    g.fbytes = (uint32_t)((int64_t)kn * g.K * 4);

    const int vec = (kn % 4 == 0) && ((uintptr_t)O % 16 == 0);
    const int cus = device_cus();
    hipError_t e;
    // automatic: the register-direct kernel for unit-stride
    // convolutions without padding (the im2col columns of neighbouring
    // positions are then contiguous input runs that the caches serve well);
    // the LDS-staged gather otherwise (measured: the direct kernel is slower
    // at stride 4, where each load instruction spans four times the lines)
    if (path == 0) path = (pad == 0 && stride == 1 && kk <= kDirectMaxK) ? 2 : 1;
    if (path == 2) {
        int dm = mt, dn = nt;
        if (dm == 0) {
            // measured on the AlexNet layers: 64 x 128 while that still gives
            // four tiles per CU; 128 x 64 for filter counts divisible by 128
            // with at least 1.5 tiles per CU; 64 x 64 otherwise
            const int64_t t64x128 = (int64_t)((g.M + 63) / 64) * ((g.N + 127) / 128);
            const int64_t t128x64 = (int64_t)((g.M + 127) / 128) * ((g.N + 63) / 64);
            if (t64x128 >= 4 * (int64_t)cus)
                dm = 64, dn = 128;
            else if (g.M % 128 == 0 && 2 * t128x64 >= 3 * (int64_t)cus)
                dm = 128, dn = 64;
            else
                dm = 64, dn = 64;
        }
        // grids short even with the smallest tile, and long contractions: the
        // contraction of each tile is split over several workgroups (atomic
        // adds into O) so that every CU holds about three, each part keeping
        // at least 64 groups of 16 (measured on AlexNet layer 8, 608 tiles:
        // 0.227 -> 0.209 ms; layer 7's 456 larger tiles were slower split)
        int kparts = 1;
        if (mt == 0 && dm == 64 && dn == 64) {
            const int64_t tl = (int64_t)((g.M + 63) / 64) * ((g.N + 63) / 64);
            const int ngroups = (g.K + 15) / 16;
            while (kparts < 4 && tl * kparts < 3 * (int64_t)cus && ngroups / (2 * kparts) >= 64) kparts *= 2;
        }
        if (dm == 64 && dn == 64)
            e = launch_direct<2, 2>(g, F, I, O, accumulate, vec, kparts, stream);
        else if (dm == 64)
            e = launch_direct<2, 4>(g, F, I, O, accumulate, vec, 1, stream);
        else if (dn == 64)
            e = launch_direct<4, 2>(g, F, I, O, accumulate, vec, 1, stream);
        else
            e = launch_direct<4, 4>(g, F, I, O, accumulate, vec, 1, stream);
        return e == hipSuccess ? CONVGEMM_OK : CONVGEMM_ERR_HIP_BASE - (int)e;
    }
    Tile t = (mt == 0 && nt == 0) ? choose_tile(g.M, g.N, cus) : Tile{mt, nt};
    if (t.mt == 64 && t.nt == 64)
        e = launch<64, 64>(g, F, I, O, accumulate, vec, cus, stream);
    else if (t.mt == 64 && t.nt == 128)
        e = launch<64, 128>(g, F, I, O, accumulate, vec, cus, stream);
    else if (t.mt == 64)
        e = launch<64, 256>(g, F, I, O, accumulate, vec, cus, stream);
    else if (t.mt == 128)
        e = launch<128, 128>(g, F, I, O, accumulate, vec, cus, stream);
    else
        e = launch<192, 128>(g, F, I, O, accumulate, vec, cus, stream);
    return e == hipSuccess ? CONVGEMM_OK : CONVGEMM_ERR_HIP_BASE - (int)e;
}
