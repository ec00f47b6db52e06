// Codebook gradient of an AQ layer: the continuous step of PV-Tuning
// (Sec. 3.2), which tunes the codebooks while the codes stay fixed.
//
// With the loss gradient dY at the layer output, the chain rule through
// Y = X W^T and eq. (4) gives
//     dC[m][k][t] = sum over (i, j) with b[i][j][m] == k of s[i] * (dY^T X)[i][j*g + t].
// Two kernels compute it:
//   1. wgrad_kernel: the weight gradient dY^T X on the matrix cores.  The
//      reduction runs over tokens, so both operands are staged into LDS with
//      tokens contiguous: token-major linear operands are transposed in
//      registers in 8x8 blocks; NCHW convolution operands already run along
//      tokens (im2col rows are shifted input rows, Sec. 3.1.1).  Each tile
//      may cover a slice of the tokens (a split); it writes s[i] * partial.
//   2. cbgrad_gather_kernel: for every codebook entry, the (row, group) pairs
//      that select it are listed (a counting sort of the codes, built once);
//      the kernel sums their s-scaled gradient groups over all splits in a
//      fixed order.  No atomics: repeated calls give identical bits.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "aq_device.h"

namespace aq {

namespace {

constexpr int kGradChunk = 64;   // tokens per chunk: four 16-deep MFMA steps
constexpr int kGradPitch = 72;   // halves per LDS row: 64 tokens plus 8 padding halves

struct GradArgs {
    const uint16_t* X;
    const uint16_t* dY;
    const float* scales;
    float* P;                    // [S][C_out][K] fp32, s[i]-scaled partial weight gradients
    int nchunk;                  // token chunks in the whole input
    int cps;                     // chunks per split
    int S;                       // splits (every split owns at least one chunk)
    int tiles_m, tiles_n;        // tiles along C_out and K
};

template <int DT>
__device__ __forceinline__ floatx16 mfma_grad(const u32x4& a, const u32x4& b, const floatx16& c) {
    if constexpr (DT == AQ_BF16)
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                       0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a), __builtin_bit_cast(half8, b), c, 0,
                                                      0, 0);
}

// Column e of an 8x8 block of 16-bit values whose row a is r[a]: o[e] holds
// r[0][e], r[1][e], ..., r[7][e].
__device__ __forceinline__ u32x4 block_column(const u32x4 (&r)[8], int e) {
    u32x4 o;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const uint32_t lo = r[2 * p][e >> 1], hi = r[2 * p + 1][e >> 1];
        o[p] = (e & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
    return o;
}

// Eight input values shifted by d in {-1, 0, +1} positions along the row:
// out[e] = in[e + d], with `nb` the value that enters at the open end.
// Branch-free: d differs between the lanes of a wave.
__device__ __forceinline__ u32x4 shift_row(const u32x4& v, uint32_t nb, int d) {
    const u32x4 lo{__builtin_amdgcn_alignbyte(v[0], nb << 16, 2), __builtin_amdgcn_alignbyte(v[1], v[0], 2),
                   __builtin_amdgcn_alignbyte(v[2], v[1], 2), __builtin_amdgcn_alignbyte(v[3], v[2], 2)};
    const u32x4 hi{__builtin_amdgcn_alignbyte(v[1], v[0], 2), __builtin_amdgcn_alignbyte(v[2], v[1], 2),
                   __builtin_amdgcn_alignbyte(v[3], v[2], 2), __builtin_amdgcn_alignbyte(nb, v[3], 2)};
    u32x4 o;
#pragma unroll
    for (int w = 0; w < 4; ++w) o[w] = d < 0 ? lo[w] : (d > 0 ? hi[w] : v[w]);
    return o;
}

// KIND: 0 linear (token-major X [N][K], dY [N][C_out]); 1 3x3 and 2 1x1
// convolutions with stride 1 and same padding (NCHW X and dY, OW % 8 == 0).
// Two workgroups per CU, except the 128 x 128 convolution tile, whose two
// register sets of eight staged rows each need the whole register file.
template <int KIND, int DT, int BM, int BN>
__global__ void __launch_bounds__(256, (KIND != 0 && BM == 128 && BN == 128) ? 1 : 2)
    wgrad_kernel(Geom geo, GradArgs ga) {
    constexpr bool CONV = KIND != 0;
    constexpr int KHW = KIND == 1 ? 9 : 1, KW = KIND == 1 ? 3 : 1, PAD = KIND == 1 ? 1 : 0;
    constexpr int WM = BM / 2, WN = BN / 2, AM = WM / 32, AN = WN / 32;
    constexpr int ROWS = BM + BN;
    constexpr int STAGE = ROWS * kGradPitch;                 // halves per stage
    constexpr int VPT = CONV ? ROWS * 8 / 256 : 1;           // staged units per thread
    __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];

    // XCD-aware order: consecutive workgroups land on different XCDs, so each
    // XCD takes a contiguous run of (split, row tile, column tile).
    const int total = ga.S * ga.tiles_m * ga.tiles_n;
    const int per_xcd = (total + 7) / 8;
    const int w = (int)(blockIdx.x % 8) * per_xcd + (int)(blockIdx.x / 8);
    if (w >= total) return;
    const int tn = w % ga.tiles_n;
    const int tm = (w / ga.tiles_n) % ga.tiles_m;
    const int z = w / (ga.tiles_n * ga.tiles_m);
    const int i0 = tm * BM, k0 = tn * BN;
    const int c_beg = z * ga.cps, c_end = min(ga.nchunk, c_beg + ga.cps);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31, hi = lane >> 5;
    const int64_t N = geo.tokens;

    // ---- staging: global -> registers -> LDS ----
    // Register sets hold whole chunks; loads run two chunks ahead of the
    // matrix cores.  Offsets are 32-bit (the host checks the sizes).
    constexpr int NV = CONV ? VPT : 8;
    constexpr int NB = CONV ? VPT : 1;
    const int N32 = (int)N;
    // convolution: every unit of this thread shares the token block tb = tid % 8;
    // per-row parts of the addresses are fixed for the whole loop
    int roff[NB], rmeta[NB];     // A: i*P; B: c*H*W | meta: bit0 live, bits 1..4 kernel row, bits 5..6 shift+1
    if constexpr (CONV) {
        const int P = geo.OH * geo.OW;
#pragma unroll
        for (int u = 0; u < VPT; ++u) {
            const int row = (tid >> 3) + 32 * u;
            if (u < BM / 32) {
                const int i = i0 + row;
                roff[u] = i * P;
                rmeta[u] = (i < geo.C_out) ? 1 : 0;
            } else {
                const int k = k0 + row - BM;
                const int c = k / KHW, rs = k - c * KHW;
                const int r = rs / KW, q = rs - r * KW;
                roff[u] = c * geo.H * geo.W;
                rmeta[u] = (k < geo.K ? 1 : 0) | (r << 1) | ((q - PAD + 1) << 5);
            }
        }
    }
    // Loads are branch-free buffer loads: an invalid element's offset lies past
    // the buffer, which returns zero.
    const int64_t xbytes = CONV ? (N / (geo.OH * geo.OW)) * geo.cin * geo.H * geo.W * 2 : N * geo.K * 2;
    const __amdgpu_buffer_rsrc_t rx = buffer_rsrc(ga.X, (uint64_t)xbytes);
    const __amdgpu_buffer_rsrc_t ry = buffer_rsrc(ga.dY, (uint64_t)(N * geo.C_out * 2));
    auto load_chunk = [&](int chunk, u32x4 (&rv)[NV], uint32_t (&nbv)[NB]) {
        const int n0 = chunk * kGradChunk;
        if constexpr (!CONV) {
            // one 8x8 block per thread: 8 tokens x 8 channels (dY) or 8 inputs (X);
            // BM is a multiple of 64, so whole waves load dY
            const bool isA = __builtin_amdgcn_readfirstlane(tid >> 6) * 64 < BM;
            const int bid = isA ? tid : tid - BM;
            const int nb8 = isA ? BM / 8 : BN / 8;
            const int cb = bid % nb8, tb = bid / nb8;
            const int len = isA ? geo.C_out : geo.K;
            const int col = (isA ? i0 : k0) + 8 * cb;
            const bool live = tid < ROWS && col < len && chunk < c_end;
            uint32_t off[8];
#pragma unroll
            for (int a = 0; a < 8; ++a) {
                const int n = n0 + 8 * tb + a;
                off[a] = (live && n < N32) ? (uint32_t)(n * len + col) * 2u : kOutOfRange;
            }
            if (isA) {
#pragma unroll
                for (int a = 0; a < 8; ++a) rv[a] = __builtin_amdgcn_raw_buffer_load_b128(ry, off[a], 0, 0);
            } else {
#pragma unroll
                for (int a = 0; a < 8; ++a) rv[a] = __builtin_amdgcn_raw_buffer_load_b128(rx, off[a], 0, 0);
            }
        } else {
            const int P = geo.OH * geo.OW;
            const int n = n0 + 8 * (tid & 7);
            const bool live_n = n < N32 && chunk < c_end;
            // unconditional (a select around the division becomes a branch)
            const int b = (int)((unsigned)n / (unsigned)P);
            const int p = n - b * P;
            const int oh = (int)((unsigned)p / (unsigned)geo.OW);
            const int ow0 = p - oh * geo.OW;
            const int ybase = b * geo.C_out * P + p;
            const int xbase = b * geo.cin * geo.H * geo.W + ow0;
#pragma unroll
            for (int u = 0; u < VPT; ++u) {
                const bool live = live_n && (rmeta[u] & 1);
                if (u < BM / 32) {           // rows of dY (the row index is 32u + tid / 8)
                    const uint32_t off = live ? (uint32_t)(ybase + roff[u]) * 2u : kOutOfRange;
                    rv[u] = __builtin_amdgcn_raw_buffer_load_b128(ry, off, 0, 0);
                    nbv[u] = 0;
                } else {                     // im2col rows of X: a shifted input row
                    const int ih = oh + ((rmeta[u] >> 1) & 15) - PAD;
                    const bool ok = live && ih >= 0 && ih < geo.H;
                    const uint32_t off = ok ? (uint32_t)(xbase + roff[u] + ih * geo.W) * 2u : kOutOfRange;
                    const int d = (rmeta[u] >> 5) - 1;
                    const bool nb_ok = ok && ((d < 0 && ow0 > 0) || (d > 0 && ow0 + 8 < geo.W));
                    const uint32_t noff = nb_ok ? (d < 0 ? off - 2u : off + 16u) : kOutOfRange;
                    rv[u] = __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, 0);
                    nbv[u] = __builtin_amdgcn_raw_buffer_load_b16(rx, noff, 0, 0);
                }
            }
        }
    };
    auto store_chunk = [&](uint16_t* st, const u32x4 (&rv)[NV], const uint32_t (&nbv)[NB]) {
        if constexpr (!CONV) {
            if (tid < ROWS) {
                const bool isA = tid < BM;
                const int bid = isA ? tid : tid - BM;
                const int nb8 = isA ? BM / 8 : BN / 8;
                const int cb = bid % nb8, tb = bid / nb8;
                const int rbase = (isA ? 0 : BM) + 8 * cb;
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    *reinterpret_cast<u32x4*>(st + (rbase + e) * kGradPitch + 8 * tb) = block_column(rv, e);
            }
        } else {
#pragma unroll
            for (int u = 0; u < VPT; ++u) {
                const int row = (tid >> 3) + 32 * u;
                const int d = u < BM / 32 ? 0 : (rmeta[u] >> 5) - 1;
                *reinterpret_cast<u32x4*>(st + row * kGradPitch + 8 * (tid & 7)) = shift_row(rv[u], nbv[u], d);
            }
        }
    };

    floatx16 acc[AM][AN];
#pragma unroll
    for (int a = 0; a < AM; ++a)
#pragma unroll
        for (int b = 0; b < AN; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

    auto compute = [&](const uint16_t* st) {
#pragma unroll
        for (int s = 0; s < kGradChunk / 16; ++s) {
            u32x4 af[AM], bf[AN];
#pragma unroll
            for (int a = 0; a < AM; ++a)
                af[a] = *reinterpret_cast<const u32x4*>(st + (WM * wm + 32 * a + l32) * kGradPitch + 16 * s + 8 * hi);
#pragma unroll
            for (int b = 0; b < AN; ++b)
                bf[b] = *reinterpret_cast<const u32x4*>(st + (BM + WN * wn + 32 * b + l32) * kGradPitch + 16 * s +
                                                        8 * hi);
#pragma unroll
            for (int a = 0; a < AM; ++a)
#pragma unroll
                for (int b = 0; b < AN; ++b) acc[a][b] = mfma_grad<DT>(af[a], bf[b], acc[a][b]);
        }
    };

    // Chunk c computes from LDS stage c % 2.  At the top of its iteration one
    // register set holds chunk c + 1 and the other receives chunk c + 2; chunk
    // c + 1 goes to the free stage after the MFMAs.  The loop body is written
    // twice so that the two register sets swap roles without copies.  Loads
    // past the split's last chunk are issued anyway with out-of-range offsets:
    // unconditional loads keep the compiler's wait counts exact (a load that
    // is issued on one path only makes it wait for every load at the join).
    if (c_beg < c_end) {
        u32x4 ra[NV], rb[NV];
        uint32_t na[NB], nbr[NB];
        load_chunk(c_beg, ra, na);
        store_chunk(lds, ra, na);
        load_chunk(c_beg + 1, ra, na);
        __syncthreads();
        int c = c_beg;
        while (true) {
            load_chunk(c + 2, rb, nbr);
            compute(lds + ((c - c_beg) & 1) * STAGE);
            store_chunk(lds + ((c + 1 - c_beg) & 1) * STAGE, ra, na);   // past the end: zeros, never read
            __syncthreads();
            if (++c >= c_end) break;
            load_chunk(c + 2, ra, na);
            compute(lds + ((c - c_beg) & 1) * STAGE);
            store_chunk(lds + ((c + 1 - c_beg) & 1) * STAGE, rb, nbr);
            __syncthreads();
            if (++c >= c_end) break;
        }
    }

    // ---- epilogue: s[i] * partial, fp32, rows i (output channels), columns k ----
    float* Pz = ga.P + (int64_t)z * geo.C_out * geo.K;
#pragma unroll
    for (int a = 0; a < AM; ++a)
#pragma unroll
        for (int b = 0; b < AN; ++b) {
            const int k = k0 + WN * wn + 32 * b + l32;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int i = i0 + WM * wm + 32 * a + 8 * (r >> 2) + 4 * hi + (r & 3);
                if (i < geo.C_out && k < geo.K) Pz[(int64_t)i * geo.K + k] = ga.scales[i] * acc[a][b][r];
            }
        }
}

// Eight values moved one position along the row: out[e] = in[e + 1] with nb
// entering at the top (up), or out[e] = in[e - 1] with nb entering at the
// bottom (down).
__device__ __forceinline__ u32x4 shift_up(const u32x4& v, uint32_t nb) {
    return u32x4{__builtin_amdgcn_alignbyte(v[1], v[0], 2), __builtin_amdgcn_alignbyte(v[2], v[1], 2),
                 __builtin_amdgcn_alignbyte(v[3], v[2], 2), __builtin_amdgcn_alignbyte(nb, v[3], 2)};
}
__device__ __forceinline__ u32x4 shift_down(const u32x4& v, uint32_t nb) {
    return u32x4{__builtin_amdgcn_alignbyte(v[0], nb << 16, 2), __builtin_amdgcn_alignbyte(v[1], v[0], 2),
                 __builtin_amdgcn_alignbyte(v[2], v[1], 2), __builtin_amdgcn_alignbyte(v[3], v[2], 2)};
}

// Convolution weight gradient with both operands streamed into LDS by
// direct-to-LDS loads.  Needs stride 1, same padding, OW dividing 64 and
// OH * OW a multiple of 64, so that a 64-token chunk is whole output rows of
// one image.  Column (c, r, q) of the im2col matrix is input row r of channel
// c shifted by q - pad along each output row; the shift moves onto dY:
//     sum_n dY[i][n] * x[c][oh + r - pad][ow + q - pad]
//   = sum_m dYq[i][(oh, m)] * x[c][oh + r - pad][m],
// with dYq[i][(oh, m)] = dY[i][(oh, m - q + pad)] and zero past the row ends.
// LDS then holds unshifted spans -- 64 tokens of dY row i, and of input rows
// (c, r) -- and the q variants of every dY fragment are built in registers
// from the fragment and its two neighbouring values.  Rows are 128 bytes with
// the 16-byte pieces XOR-swizzled by the row index (conflict-free fragment
// reads); three stages keep two chunks of loads in flight.
template <int KIND, int DT, int BM, int BNP>
__global__ void __launch_bounds__(256, 2) wgrad_conv_dma_kernel(Geom geo, GradArgs ga, const uint8_t* zero) {
    constexpr int KQ = KIND == 1 ? 3 : 1;        // kernel columns: variants of dY
    constexpr int KR = KIND == 1 ? 3 : 1;        // kernel rows
    constexpr int PAD = KIND == 1 ? 1 : 0;
    constexpr int WM = BM / 2, WN = BNP / 2, AM = WM / 32, AN = WN / 32;
    constexpr int ROWS = BM + BNP;
    constexpr int STAGE = ROWS * 128;
    constexpr int NST = 3;
    constexpr int LOADS = ROWS / 32;             // 16-byte loads per thread per chunk
    static_assert(ROWS % 32 == 0, "rows per stage");
    __shared__ __attribute__((aligned(16))) uint8_t lds[NST * STAGE];

    const int total = ga.S * ga.tiles_m * ga.tiles_n;
    const int per_xcd = (total + 7) / 8;
    const int w = (int)(blockIdx.x % 8) * per_xcd + (int)(blockIdx.x / 8);
    if (w >= total) return;
    const int tn = w % ga.tiles_n;
    const int tm = (w / ga.tiles_n) % ga.tiles_m;
    const int z = w / (ga.tiles_n * ga.tiles_m);
    const int i0 = tm * BM, p0 = tn * BNP;
    const int c_beg = z * ga.cps, c_end = min(ga.nchunk, c_beg + ga.cps);
    const int nch = max(0, c_end - c_beg);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31, hi = lane >> 5;
    const int P = geo.OH * geo.OW;
    const int npairs = geo.cin * KR;
    const uint8_t* dyb = reinterpret_cast<const uint8_t*>(ga.dY);
    const uint8_t* xb = reinterpret_cast<const uint8_t*>(ga.X);

    // this lane's slot in every load: row (8 g + lane / 8), logical piece pc
    const int lrow = lane >> 3;
    const int lpc = (lane & 7) ^ lrow;
    auto issue = [&](int chunk, uint8_t* st) {
        const int n0 = chunk * 64;
        const int b = n0 / P;
        const int pb = n0 - b * P;
        const int t = 8 * lpc;                   // token of the piece within the chunk
        const int oh = pb / geo.OW + t / geo.OW, ow = t % geo.OW;
#pragma unroll
        for (int j = 0; j < LOADS; ++j) {
            const int grp = wave + 4 * j;
            const int row = 8 * grp + lrow;
            const uint8_t* src = zero;
            if (8 * grp < BM) {
                const int i = i0 + row;
                if (i < geo.C_out) src = dyb + ((int64_t)(b * geo.C_out + i) * P + pb + t) * 2;
            } else {
                const int pr = p0 + row - BM;
                const int c = pr / KR, r = pr - c * KR;
                const int ih = oh + r - PAD;
                if (pr < npairs && ih >= 0 && ih < geo.H)
                    src = xb + ((int64_t)(b * geo.cin + c) * geo.H * geo.W + ih * geo.W + ow) * 2;
            }
            lds_dma16(src, st + grp * 1024);
        }
    };

    // neighbour masks: the piece starts (ends) an output row
    bool lft_ok[4], rgt_ok[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const int pc = 2 * s + hi;
        lft_ok[s] = (8 * pc) % geo.OW != 0;
        rgt_ok[s] = (8 * pc + 8) % geo.OW != 0;
    }

    floatx16 acc[KQ][AM][AN];
#pragma unroll
    for (int q = 0; q < KQ; ++q)
#pragma unroll
        for (int a = 0; a < AM; ++a)
#pragma unroll
            for (int b = 0; b < AN; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[q][a][b][r] = 0.0f;

    auto compute = [&](const uint8_t* st) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int pc = 2 * s + hi;
            u32x4 av[KQ][AM], bf[AN];
#pragma unroll
            for (int a = 0; a < AM; ++a) {
                const int row = WM * wm + 32 * a + l32;
                const uint8_t* rp = st + row * 128;
                const u32x4 v = *reinterpret_cast<const u32x4*>(rp + ((pc ^ (row & 7)) << 4));
                if constexpr (KQ == 3) {
                    const uint32_t left = lft_ok[s] ? *reinterpret_cast<const uint16_t*>(
                                                          rp + ((((pc - 1) & 7) ^ (row & 7)) << 4) + 14)
                                                    : 0u;
                    const uint32_t right =
                        rgt_ok[s] ? *reinterpret_cast<const uint16_t*>(rp + ((((pc + 1) & 7) ^ (row & 7)) << 4)) : 0u;
                    av[0][a] = shift_up(v, right);     // q = 0: dY[m + 1]
                    av[1][a] = v;                      // q = 1
                    av[2][a] = shift_down(v, left);    // q = 2: dY[m - 1]
                } else {
                    av[0][a] = v;
                }
            }
#pragma unroll
            for (int b = 0; b < AN; ++b) {
                const int row = BM + WN * wn + 32 * b + l32;
                bf[b] = *reinterpret_cast<const u32x4*>(st + row * 128 + ((pc ^ (row & 7)) << 4));
            }
#pragma unroll
            for (int q = 0; q < KQ; ++q)
#pragma unroll
                for (int a = 0; a < AM; ++a)
#pragma unroll
                    for (int b = 0; b < AN; ++b) acc[q][a][b] = mfma_grad<DT>(av[q][a], bf[b], acc[q][a][b]);
        }
    };

    auto stg = [&](int c) { return lds + (c % NST) * STAGE; };
    if (nch > 0) issue(c_beg, stg(0));
    if (nch > 1) issue(c_beg + 1, stg(1));
    if (nch > 1) wait_vmcnt<LOADS>();
    else wait_vmcnt<0>();
    lds_barrier();
    for (int t = 0; t < nch; ++t) {
        if (t + 2 < nch) issue(c_beg + t + 2, stg(t + 2));
        compute(stg(t));
        if (t + 2 < nch) wait_vmcnt<LOADS>();    // chunk t + 1 landed
        else wait_vmcnt<0>();
        lds_barrier();
    }

    float* Pz = ga.P + (int64_t)z * geo.C_out * geo.K;
#pragma unroll
    for (int a = 0; a < AM; ++a)
#pragma unroll
        for (int b = 0; b < AN; ++b) {
            const int pr = p0 + WN * wn + 32 * b + l32;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int i = i0 + WM * wm + 32 * a + 8 * (r >> 2) + 4 * hi + (r & 3);
                if (i < geo.C_out && pr < npairs) {
                    const float sc = ga.scales[i];
#pragma unroll
                    for (int q = 0; q < KQ; ++q) Pz[(int64_t)i * geo.K + pr * KQ + q] = sc * acc[q][a][b][r];
                }
            }
        }
}

// Linear weight gradient with both operands streamed into LDS by
// direct-to-LDS loads, untransposed: a chunk is 64 tokens x 64 channels of dY
// and 64 tokens x 64 inputs of X, each row 128 bytes (one token), so the
// reduction dimension (tokens) is the slow one in LDS.  The MFMA fragments
// come out with the gfx950 transpose read ds_read_b64_tr_b16: within each
// group of 16 lanes, lane l receives element l % 4 of the 8-byte rows
// addressed by lanes 4f + l / 4 (f = 0..3).  So lane 16 g + 4 f + q addresses
// the four channels 16 (g % 2) + 4 q .. + 3 at token 8 (g / 2) + f, and
// lane l obtains channel l % 32 at tokens 8 (l / 32) + 0..3 -- half of its
// fragment; a second read 4 tokens on gives the other half.  The 16-byte
// pieces of a row are XOR-swizzled with 4 * ((token / 2) % 2), which spreads
// the 32 lanes of a half-wave over all banks.
__device__ __forceinline__ int lin_swz(int n) { return ((n >> 1) & 1) << 2; }

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Four transpose reads at LDS byte addresses, completed before returning.
// Written as one asm block: through the builtin the compiler orders every
// such read after all outstanding direct-to-LDS loads (it cannot tell the
// addresses apart), which would drain the prefetched chunks.  The loads of
// the chunk read here were awaited explicitly before the barrier.
__device__ __forceinline__ void tr_read4(u32x2& a0, u32x2& a1, u32x2& b0, u32x2& b1, uint32_t pa0, uint32_t pa1,
                                         uint32_t pb0, uint32_t pb1) {
    asm volatile(
        "ds_read_b64_tr_b16 %0, %4\n\t"
        "ds_read_b64_tr_b16 %1, %5\n\t"
        "ds_read_b64_tr_b16 %2, %6\n\t"
        "ds_read_b64_tr_b16 %3, %7\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(a0), "=&v"(a1), "=&v"(b0), "=&v"(b1)
        : "v"(pa0), "v"(pa1), "v"(pb0), "v"(pb1)
        : "memory");
}

template <int DT>
__global__ void __launch_bounds__(256, 2) wgrad_linear_dma_kernel(Geom geo, GradArgs ga, const uint8_t* zero) {
    constexpr int BM = 64, BN = 64;
    constexpr int STAGE = 64 * 128 * 2;          // A then B: 64 tokens x 128 bytes each
    constexpr int NST = 3;
    constexpr int LOADS = 4;                     // 16-byte loads per thread per chunk
    __shared__ __attribute__((aligned(16))) uint8_t lds[NST * STAGE];

    const int total = ga.S * ga.tiles_m * ga.tiles_n;
    const int per_xcd = (total + 7) / 8;
    const int w = (int)(blockIdx.x % 8) * per_xcd + (int)(blockIdx.x / 8);
    if (w >= total) return;
    const int tn = w % ga.tiles_n;
    const int tm = (w / ga.tiles_n) % ga.tiles_m;
    const int z = w / (ga.tiles_n * ga.tiles_m);
    const int i0 = tm * BM, k0 = tn * BN;
    const int c_beg = z * ga.cps, c_end = min(ga.nchunk, c_beg + ga.cps);
    const int nch = max(0, c_end - c_beg);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31, hi = lane >> 5;
    const int64_t N = geo.tokens;
    const uint8_t* dyb = reinterpret_cast<const uint8_t*>(ga.dY);
    const uint8_t* xb = reinterpret_cast<const uint8_t*>(ga.X);

    // load slot of this lane: row 8 * grp + lane / 8 of a region, slot piece lane % 8
    const int lrow = lane >> 3;
    auto issue = [&](int chunk, uint8_t* st) {
        const int64_t n0 = (int64_t)chunk * 64;
#pragma unroll
        for (int j = 0; j < LOADS; ++j) {
            const int grp = wave + 4 * j;        // 0..7: dY rows, 8..15: X rows
            const int row = 8 * (grp & 7) + lrow;
            const int pc = (lane & 7) ^ lin_swz(row);
            const int64_t n = n0 + row;
            const uint8_t* src = zero;
            if (grp < 8) {
                const int i = i0 + 8 * pc;
                if (n < N && i < geo.C_out) src = dyb + (n * geo.C_out + i) * 2;
            } else {
                const int k = k0 + 8 * pc;
                if (n < N && k < geo.K) src = xb + (n * geo.K + k) * 2;
            }
            lds_dma16(src, st + grp * 1024);
        }
    };

    // transpose-read addresses (bytes within a stage) for every step and half:
    // lane 16 g + 4 f + q reads channels (inputs) c .. c + 3, c = 16 (g % 2) + 4 q
    // of the wave's 32-wide block, at token 16 s + 8 (g / 2) + 4 h + f
    const int g16 = lane >> 4, j16 = lane & 15;
    const int fo = j16 >> 2, qo = j16 & 3;
    int offa[4][2], offb[4][2];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int n = 16 * s + 8 * (g16 >> 1) + 4 * h + fo;
            const int ca = 32 * wm + 16 * (g16 & 1) + 4 * qo;
            const int cb = 32 * wn + 16 * (g16 & 1) + 4 * qo;
            offa[s][h] = n * 128 + (((ca >> 3) ^ lin_swz(n)) << 4) + (ca & 7) * 2;
            offb[s][h] = 64 * 128 + n * 128 + (((cb >> 3) ^ lin_swz(n)) << 4) + (cb & 7) * 2;
        }

    floatx16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.0f;

    const uint32_t lds0 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)lds;
    auto compute = [&](int stage) {
        const uint32_t st = lds0 + stage * STAGE;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            u32x2 a0, a1, b0, b1;
            tr_read4(a0, a1, b0, b1, st + offa[s][0], st + offa[s][1], st + offb[s][0], st + offb[s][1]);
            acc = mfma_grad<DT>(u32x4{a0[0], a0[1], a1[0], a1[1]}, u32x4{b0[0], b0[1], b1[0], b1[1]}, acc);
        }
    };

    auto stg = [&](int c) { return lds + (c % NST) * STAGE; };
    if (nch > 0) issue(c_beg, stg(0));
    if (nch > 1) issue(c_beg + 1, stg(1));
    if (nch > 1) wait_vmcnt<LOADS>();
    else wait_vmcnt<0>();
    lds_barrier();
    for (int t = 0; t < nch; ++t) {
        if (t + 2 < nch) issue(c_beg + t + 2, stg(t + 2));
        compute(t % NST);
        if (t + 2 < nch) wait_vmcnt<LOADS>();
        else wait_vmcnt<0>();
        lds_barrier();
    }

    float* Pz = ga.P + (int64_t)z * geo.C_out * geo.K;
    const int k = k0 + 32 * wn + l32;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int i = i0 + 32 * wm + 8 * (r >> 2) + 4 * hi + (r & 3);
        if (i < geo.C_out && k < geo.K) Pz[(int64_t)i * geo.K + k] = ga.scales[i] * acc[r];
    }
}

// One group of LPB lanes per codebook entry (m, k); lanes split into
// LPB / g entry slots times g positions t.  Each slot sums its entries in
// list order, then lane t adds the slots in order.
template <int LPB>
__global__ void __launch_bounds__(256) cbgrad_gather_kernel(const float* __restrict__ P, int64_t slice, int S,
                                                            const int32_t* __restrict__ offs,
                                                            const int32_t* __restrict__ ent, int64_t nent, int nk,
                                                            int M, int g, float* __restrict__ dC) {
    constexpr int BPW = 256 / LPB;
    __shared__ float red[256];
    const int tid = threadIdx.x;
    const int sub = tid / LPB, lt = tid % LPB;
    const int64_t bucket = (int64_t)blockIdx.x * BPW + sub;
    const bool live_bucket = bucket < (int64_t)M * nk;
    const int EP = LPB / g;
    const int e = lt / g, t = lt - (lt / g) * g;
    float acc = 0.0f;
    if (live_bucket && e < EP) {
        const int m = (int)(bucket / nk), k = (int)(bucket - (int64_t)m * nk);
        const int32_t beg = offs[(int64_t)m * (nk + 1) + k], end = offs[(int64_t)m * (nk + 1) + k + 1];
        const int32_t* list = ent + (int64_t)m * nent;
        // four entries per step, all loads issued before any add (branch-free
        // buffer loads; an entry past the list reads zero): short lists, as a
        // large codebook has, finish in one step
        const __amdgpu_buffer_rsrc_t lr = buffer_rsrc(list, (uint64_t)nent * 4);
        const __amdgpu_buffer_rsrc_t pr = buffer_rsrc(P, (uint64_t)S * slice * 4);
        const uint32_t sstride = (uint32_t)(slice * 4);
        int32_t idx = beg + e;
        for (; idx + 3 * EP < end; idx += 4 * EP) {     // whole steps: no bounds checks
            int64_t base[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) base[u] = (int64_t)list[idx + u * EP] * g + t;
            float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            for (int s = 0; s < S; ++s)
#pragma unroll
                for (int u = 0; u < 4; ++u) v[u] += P[s * slice + base[u]];
#pragma unroll
            for (int u = 0; u < 4; ++u) acc += v[u];
        }
        if (idx < end) {                                  // the last, partial step
            uint32_t boff[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int32_t iu = idx + u * EP;
                const int32_t p = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(
                    lr, iu < end ? (uint32_t)iu * 4u : kOutOfRange, 0, 0);
                boff[u] = iu < end ? (uint32_t)(p * g + t) * 4u : kOutOfRange;
            }
            float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            for (int s = 0; s < S; ++s)
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    v[u] += __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(pr, boff[u] + s * sstride, 0, 0));
#pragma unroll
            for (int u = 0; u < 4; ++u) acc += v[u];
        }
    }
    red[tid] = acc;
    __syncthreads();
    if (live_bucket && lt < g) {
        float sum = 0.0f;
        for (int e2 = 0; e2 < EP; ++e2) sum += red[sub * LPB + e2 * g + lt];
        dC[bucket * g + lt] = sum;
    }
}

// Sum of the S partial weight gradients into the first, in split order
// (streaming; float4 per thread when every slice starts 16-byte aligned).
__global__ void __launch_bounds__(256) split_sum_kernel(float* __restrict__ P, int64_t slice, int S) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (slice % 4 == 0) {
        for (int64_t i = t0; i < slice / 4; i += stride) {
            floatx4 a = reinterpret_cast<const floatx4*>(P)[i];
            for (int s = 1; s < S; ++s) a += reinterpret_cast<const floatx4*>(P + s * slice)[i];
            reinterpret_cast<floatx4*>(P)[i] = a;
        }
    } else {
        for (int64_t i = t0; i < slice; i += stride) {
            float a = P[i];
            for (int s = 1; s < S; ++s) a += P[s * slice + i];
            P[i] = a;
        }
    }
}

template <int KIND, int DT, int BM, int BN>
hipError_t wgrad_launch(const Geom& geo, const GradArgs& ga, hipStream_t st) {
    const int total = ga.S * ga.tiles_m * ga.tiles_n;
    const unsigned grid = (unsigned)(8 * ((total + 7) / 8));
    wgrad_kernel<KIND, DT, BM, BN><<<grid, 256, 0, st>>>(geo, ga);
    note_launch(st, "wgrad_kernel", {KIND, DT, BM, BN});
    return hipGetLastError();
}

template <int KIND, int DT, int BM, int BNP>
hipError_t wgrad_dma_launch(const Geom& geo, const GradArgs& ga, const uint8_t* zero, hipStream_t st) {
    const int total = ga.S * ga.tiles_m * ga.tiles_n;
    const unsigned grid = (unsigned)(8 * ((total + 7) / 8));
    wgrad_conv_dma_kernel<KIND, DT, BM, BNP><<<grid, 256, 0, st>>>(geo, ga, zero);
    note_launch(st, "wgrad_conv_dma_kernel", {KIND, DT, BM, BNP});
    return hipGetLastError();
}

template <int KIND, int DT>
hipError_t wgrad_dma_dispatch(const Geom& geo, const GradPlan& gp, const GradArgs& ga, const uint8_t* zero,
                              hipStream_t st) {
    if (gp.bm == 128 && gp.bn == 64) return wgrad_dma_launch<KIND, DT, 128, 64>(geo, ga, zero, st);
    if (gp.bm == 64 && gp.bn == 64) return wgrad_dma_launch<KIND, DT, 64, 64>(geo, ga, zero, st);
    return hipErrorInvalidConfiguration;
}

template <int KIND, int DT>
hipError_t wgrad_dispatch(const Geom& geo, const GradPlan& gp, const GradArgs& ga, hipStream_t st) {
    if (gp.bm == 128 && gp.bn == 128) return wgrad_launch<KIND, DT, 128, 128>(geo, ga, st);
    if (gp.bm == 64 && gp.bn == 128) return wgrad_launch<KIND, DT, 64, 128>(geo, ga, st);
    if (gp.bm == 64 && gp.bn == 64) return wgrad_launch<KIND, DT, 64, 64>(geo, ga, st);
    return hipErrorInvalidConfiguration;
}

}  // namespace

// Linear layers, and convolutions whose 64-token chunks are whole output rows
// of one image, take the direct-to-LDS kernels.
static bool grad_dma_ok(const Geom& geo, const Options& opt) {
    if (opt.grad_regs) return false;
    if (!geo.conv) return true;                  // linear: C_out and K are multiples of 8
    if (geo.stride != 1 || geo.OW != geo.W || geo.OH != geo.H || geo.W % 8 != 0) return false;
    return 64 % geo.OW == 0 && ((int64_t)geo.OH * geo.OW) % 64 == 0;
}

// Tile and split choice: the largest tile that still gives about one
// workgroup per CU, then token splits up to about four workgroups per CU
// while the partial gradients stay within 32 MiB (each split adds a full
// C_out x K fp32 partial to write and to sum).
GradPlan grad_plan_create(const Geom& geo, int64_t max_tokens, const Options& opt) {
    GradPlan gp{};
    gp.dma = grad_dma_ok(geo, opt);
    const int want_bm = opt.grad_bm, want_bn = opt.grad_bn;
    if (gp.dma && !geo.conv) {
        gp.bm = gp.bn = 64;
        gp.tiles_m = (geo.C_out + 63) / 64;
        gp.tiles_n = (geo.K + 63) / 64;
    } else if (gp.dma) {
        // rows of C_out x (input channel, kernel row) pairs; 64 x 64 measured
        // faster than 128 x 64 on every layer shape here (more workgroups per
        // CU hide the load latency better)
        const int npairs = geo.cin * (geo.kh == 3 ? 3 : 1);
        gp.bm = want_bm == 128 ? 128 : 64;
        gp.bn = 64;
        gp.tiles_m = (geo.C_out + gp.bm - 1) / gp.bm;
        gp.tiles_n = (npairs + gp.bn - 1) / gp.bn;
    } else {
        const int shapes[3][2] = {{128, 128}, {64, 128}, {64, 64}};
        int pick = 2;
        for (int s = 0; s < 3; ++s) {
            if (want_bm) {
                if (shapes[s][0] == want_bm && shapes[s][1] == want_bn) {
                    pick = s;
                    break;
                }
                continue;
            }
            const int64_t tiles = (int64_t)((geo.C_out + shapes[s][0] - 1) / shapes[s][0]) *
                                  ((geo.K + shapes[s][1] - 1) / shapes[s][1]);
            if (tiles >= 240) {
                pick = s;
                break;
            }
        }
        gp.bm = shapes[pick][0];
        gp.bn = shapes[pick][1];
        gp.tiles_m = (geo.C_out + gp.bm - 1) / gp.bm;
        gp.tiles_n = (geo.K + gp.bn - 1) / gp.bn;
    }
    const int64_t tiles = (int64_t)gp.tiles_m * gp.tiles_n;
    const int64_t nchunk = std::max<int64_t>(1, (max_tokens + kGradChunk - 1) / kGradChunk);
    const int64_t slice = (int64_t)geo.C_out * geo.K * 4;
    gp.s_max = (int)std::min<int64_t>({16, nchunk, std::max<int64_t>(1, (960 + tiles - 1) / tiles),
                                       std::max<int64_t>(1, (int64_t(32) << 20) / slice)});
    if (opt.grad_splits > 0) gp.s_max = (int)std::min<int64_t>({16, nchunk, (int64_t)opt.grad_splits});
    return gp;
}

int grad_kind(const Geom& geo) {
    if (!geo.conv) return 0;
    return geo.kh == 3 ? 1 : 2;
}

hipError_t launch_codebook_grad(const Geom& geo, const GradPlan& gp, int dtype, const void* X, const void* dY,
                                const float* scales, float* P, const int32_t* offs, const int32_t* ent, float* dC,
                                const void* zero, int splits_override, hipStream_t st) {
    GradArgs ga;
    ga.X = static_cast<const uint16_t*>(X);
    ga.dY = static_cast<const uint16_t*>(dY);
    ga.scales = scales;
    ga.P = P;
    ga.nchunk = (int)((geo.tokens + kGradChunk - 1) / kGradChunk);
    int S = std::min(gp.s_max, ga.nchunk);
    if (splits_override > 0) S = std::min(S, splits_override);
    ga.cps = (ga.nchunk + S - 1) / S;
    ga.S = (ga.nchunk + ga.cps - 1) / ga.cps;     // every split owns at least one chunk
    ga.tiles_m = gp.tiles_m;
    ga.tiles_n = gp.tiles_n;
    const int kind = grad_kind(geo);
    hipError_t e;
    const uint8_t* z16 = static_cast<const uint8_t*>(zero);
    if (gp.dma && kind == 0) {
        const unsigned grid = (unsigned)(8 * ((ga.S * ga.tiles_m * ga.tiles_n + 7) / 8));
        if (dtype == AQ_BF16)
            wgrad_linear_dma_kernel<AQ_BF16><<<grid, 256, 0, st>>>(geo, ga, z16);
        else
            wgrad_linear_dma_kernel<AQ_F16><<<grid, 256, 0, st>>>(geo, ga, z16);
        note_launch(st, "wgrad_linear_dma_kernel", {dtype});
        e = hipGetLastError();
    } else if (gp.dma) {
        e = kind == 1 ? (dtype == AQ_BF16 ? wgrad_dma_dispatch<1, AQ_BF16>(geo, gp, ga, z16, st)
                                          : wgrad_dma_dispatch<1, AQ_F16>(geo, gp, ga, z16, st))
                      : (dtype == AQ_BF16 ? wgrad_dma_dispatch<2, AQ_BF16>(geo, gp, ga, z16, st)
                                          : wgrad_dma_dispatch<2, AQ_F16>(geo, gp, ga, z16, st));
    } else if (dtype == AQ_BF16) {
        e = kind == 0 ? wgrad_dispatch<0, AQ_BF16>(geo, gp, ga, st)
            : kind == 1 ? wgrad_dispatch<1, AQ_BF16>(geo, gp, ga, st)
                        : wgrad_dispatch<2, AQ_BF16>(geo, gp, ga, st);
    } else {
        e = kind == 0 ? wgrad_dispatch<0, AQ_F16>(geo, gp, ga, st)
            : kind == 1 ? wgrad_dispatch<1, AQ_F16>(geo, gp, ga, st)
                        : wgrad_dispatch<2, AQ_F16>(geo, gp, ga, st);
    }
    if (e != hipSuccess) return e;
    const int64_t slice = (int64_t)geo.C_out * geo.K;
    int S_gather = ga.S;
    if (ga.S > 1) {
        // the gather visits every (row, group) once per codebook: sum the splits first
        const int64_t n4 = std::max<int64_t>(1, slice / 4);
        const unsigned grid = (unsigned)std::min<int64_t>((n4 + 255) / 256, 4096);
        split_sum_kernel<<<grid, 256, 0, st>>>(P, slice, ga.S);
        note_launch(st, "split_sum_kernel", {});
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        S_gather = 1;
    }
    const int nk = 1 << geo.B;
    const int64_t buckets = (int64_t)geo.M * nk;
    const int64_t nent = (int64_t)geo.C_out * geo.G;
    // a wave per entry when lists are short (large codebooks), a workgroup otherwise
    if (nent / nk < 64) {
        cbgrad_gather_kernel<64><<<(unsigned)((buckets + 3) / 4), 256, 0, st>>>(P, slice, S_gather, offs, ent, nent,
                                                                               nk, geo.M, geo.g, dC);
    } else {
        cbgrad_gather_kernel<256><<<(unsigned)buckets, 256, 0, st>>>(P, slice, S_gather, offs, ent, nent, nk, geo.M,
                                                                     geo.g, dC);
    }
    note_launch(st, "cbgrad_gather_kernel", {nent / nk < 64 ? 64 : 256});
    return hipGetLastError();
}

// Counting sort of the codes: for codebook m, entries offs[m][k] ..
// offs[m][k+1] of ent[m] list the (row, group) pairs i*G + j with
// b[i][j][m] == k, in increasing order.
void build_code_index(const void* codes, int B, int C_out, int G, int M, std::vector<int32_t>& offs,
                      std::vector<int32_t>& ent) {
    const int nk = 1 << B;
    const int64_t nent = (int64_t)C_out * G;
    offs.assign((size_t)M * (nk + 1), 0);
    ent.assign((size_t)M * nent, 0);
    auto code = [&](int64_t p, int m) -> int {
        return B <= 8 ? static_cast<const uint8_t*>(codes)[p * M + m] : static_cast<const uint16_t*>(codes)[p * M + m];
    };
    for (int m = 0; m < M; ++m) {
        int32_t* o = offs.data() + (size_t)m * (nk + 1);
        for (int64_t p = 0; p < nent; ++p) ++o[code(p, m) + 1];
        for (int k = 0; k < nk; ++k) o[k + 1] += o[k];
        std::vector<int32_t> pos(o, o + nk);
        int32_t* list = ent.data() + (size_t)m * nent;
        for (int64_t p = 0; p < nent; ++p) list[pos[code(p, m)]++] = (int32_t)p;
    }
}

}  // namespace aq
