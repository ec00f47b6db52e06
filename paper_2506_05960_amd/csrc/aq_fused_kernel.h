// Fused decode + matrix-core forward (fp16 tiles, group size 8), gfx950.
//
// Work split.  A workgroup owns a BM (tokens) x BN (output channels) tile of Y
// and its four waves split the reduction dimension: wave w takes K chunks
// w, w+4, w+8, ... and accumulates the whole tile for them, so the main loop
// needs no workgroup barrier.  At the end the four partial tiles meet in LDS
// and each wave sums (in a fixed order) and stores a quarter of the tile.
// With a K split over S workgroups (layers with too few tiles to fill the
// chip), workgroup s of a tile takes chunks 4 s + w, 4 s + w + 4 S, ...;
// each writes its fp32 partial tile to a workspace and bumps the tile's
// arrival counter, and the last to arrive adds the S partials in split order
// (so the result does not depend on arrival order), stores Y and resets the
// counter for the next launch.
//
// Operands.  v_mfma_f32_32x32x16_f16 takes 8 fp16 values per lane for each
// operand; lane l holds row (l % 32) and a k-slice of 8 chosen by (l / 32).
// Any assignment of the 16 logical k values of a step to (lane half, slot)
// works as long as both operands use the same one.
//  * Weights: each lane decodes its own groups straight into registers.  The
//    codes a lane needs (one output channel, one half of a chunk's k-slices)
//    are stored contiguously at create time as 8-bit codes (16-bit when the
//    codebook is larger than 256 rows); a group is the sum of its M codewords,
//    accumulated with packed fp16 adds in ascending m (for M = 2 this equals
//    the fp32 sum rounded once to fp16).  The per-channel scale multiplies the
//    fp32 accumulator in the epilogue.
//  * Activations sit in a per-wave, double-buffered LDS staging area split
//    into planes of 8 channels (or 8 consecutive k), 16 bytes per pixel (or
//    token), so that one lane's 8 operand values are one 16-byte read and 16
//    lanes read 256 contiguous bytes.
//  * Linear layer: a chunk is 64 consecutive k (4 MFMA steps).
//  * Convolution (implicit im2col): the staging area holds the input rows the
//    token tile touches, with zero padding columns.  A 3x3 chunk is 16 input
//    channels and one MFMA step is one kernel position (kh, kw) over them.
//    The weight groups of a chunk run over (channel, kh, kw) with the channel
//    outermost, so a lane decodes the 9 groups of its 8 channels and regroups
//    the 72 values per position with byte permutes.  A 1x1 chunk is 64
//    channels (4 steps).
#pragma once

#include <type_traits>

#include "aq_device.h"

namespace aq {

constexpr int kWaves = 4;

// Orders this wave's LDS accesses at the compiler level.  LDS instructions of
// one wave execute in issue order, so no hardware wait is needed (a memory
// fence here would also wait for the global prefetches in flight).
__device__ __forceinline__ void wave_sync() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_wave_barrier();
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ floatx16 mfma_f16(const u32x4& a, const u32x4& b, const floatx16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a), __builtin_bit_cast(half8, b), c, 0, 0,
                                                  0);
}

// Dword made of fp16 half `hlo` of xlo (low half) and half `hhi` of xhi (high half).
__device__ __forceinline__ uint32_t pick2(uint32_t xlo, int hlo, uint32_t xhi, int hhi) {
    const uint32_t sel = (uint32_t)(2 * hlo) | ((uint32_t)(2 * hlo + 1) << 8) | ((uint32_t)(4 + 2 * hhi) << 16) |
                         ((uint32_t)(5 + 2 * hhi) << 24);
    return __builtin_amdgcn_perm(xhi, xlo, sel);
}


// Quotient of non-negative a < 2^24 by 1 <= d < 2^24 through an fp32
// reciprocal, corrected to the exact integer quotient (24-bit multiplies).
__device__ __forceinline__ int fdiv(int a, int d, float inv_d) {
    int qt = (int)((float)a * inv_d);
    qt += (int)__umul24(qt + 1, d) <= a;
    qt -= (int)__umul24(qt, d) > a;
    return qt;
}

// Raw codewords of one group as read from the codebook: M x 16 bytes (fp16)
// or M x 32 bytes (fp32).
template <int DEC, int MC>
struct GroupRaw {
    u32x4 w[DEC == FUSED_DEC_F32L ? 2 * MC : MC];
};

// Code i of a lane's packed record words (8- or 16-bit codes, little-endian).
// Extracted with shifts: reading the 32-bit words through a 16-bit pointer
// would break type-based aliasing, and the compiler then reuses stale codes.
template <typename EntT>
__device__ __forceinline__ uint32_t code_at(const uint32_t* dw, int i) {
    if constexpr (sizeof(EntT) == 1) return (dw[i >> 2] >> (8 * (i & 3))) & 0xFFu;
    else return (dw[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
}

// Issue the codebook reads of one group, whose M codes are codes i0 .. i0+M-1
// of the record words `dw`.  The LDS codebook keeps 256 rows per codebook
// (rows past 2^B unused), so codebook m starts at a fixed byte offset and a
// codeword address is a shift.
template <int DEC, int MC, typename EntT>
__device__ __forceinline__ void gather_group(GroupRaw<DEC, MC>& g, const uint32_t* dw, int i0, const uint8_t* cb_lds,
                                             const void* cb_glob) {
    if constexpr (DEC == FUSED_DEC_T16G) {
        g.w[0] = static_cast<const u32x4*>(cb_glob)[code_at<EntT>(dw, i0)];
    } else if constexpr (DEC == FUSED_DEC_F32L) {
#pragma unroll
        for (int m = 0; m < MC; ++m) {
            const u32x4* p = reinterpret_cast<const u32x4*>(cb_lds + m * 256 * 32 + code_at<EntT>(dw, i0 + m) * 32u);
            g.w[2 * m] = p[0];
            g.w[2 * m + 1] = p[1];
        }
    } else {
#pragma unroll
        for (int m = 0; m < MC; ++m)
            g.w[m] = *reinterpret_cast<const u32x4*>(cb_lds + m * 256 * 16 + code_at<EntT>(dw, i0 + m) * 16u);
    }
}

// Sum the gathered codewords of one group and round once to fp16 (4 dwords).
template <int DEC, int MC>
__device__ __forceinline__ u32x4 combine_group(const GroupRaw<DEC, MC>& g) {
    if constexpr (DEC == FUSED_DEC_PK16) {
        // fp16 accumulation in ascending m (for M = 2 identical to the fp32 sum rounded once)
        u32x4 r = g.w[0];
#pragma unroll
        for (int m = 1; m < MC; ++m) {
            r[0] = add_f16x2(r[0], g.w[m][0]);
            r[1] = add_f16x2(r[1], g.w[m][1]);
            r[2] = add_f16x2(r[2], g.w[m][2]);
            r[3] = add_f16x2(r[3], g.w[m][3]);
        }
        return r;
    } else if constexpr (DEC == FUSED_DEC_F32L) {
        float s[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            s[e] = __uint_as_float(g.w[0][e]);
            s[4 + e] = __uint_as_float(g.w[1][e]);
        }
#pragma unroll
        for (int m = 1; m < MC; ++m)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                s[e] = __fadd_rn(s[e], __uint_as_float(g.w[2 * m][e]));
                s[4 + e] = __fadd_rn(s[4 + e], __uint_as_float(g.w[2 * m + 1][e]));
            }
        u32x4 r;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            const float a = opaque_f32(s[2 * d]), b = opaque_f32(s[2 * d + 1]);
            r[d] = (uint32_t)f32_to_f16(a) | ((uint32_t)f32_to_f16(b) << 16);
        }
        return r;
    } else {   // M == 1: the codeword is already the fp16 weight
        return g.w[0];
    }
}

// 8 fp16 values from 8 int8 values, exactly: the fp16 bit pattern
// 0x6400 | (x ^ 0x80) encodes 1024 + (x + 128), and subtracting 1152 (exact for
// integers below 2048) leaves x.
__device__ __forceinline__ u32x4 i8x8_to_f16(uint64_t q) {
    const uint32_t lo = (uint32_t)q ^ 0x80808080u, hi = (uint32_t)(q >> 32) ^ 0x80808080u;
    const uint32_t k64 = 0x64646464u;
    const uint32_t bias = 0xE480E480u;   // fp16 -1152 in both halves
    u32x4 r;
    r[0] = add_f16x2(__builtin_amdgcn_perm(k64, lo, 0x04010400u), bias);
    r[1] = add_f16x2(__builtin_amdgcn_perm(k64, lo, 0x04030402u), bias);
    r[2] = add_f16x2(__builtin_amdgcn_perm(k64, hi, 0x04010400u), bias);
    r[3] = add_f16x2(__builtin_amdgcn_perm(k64, hi, 0x04030402u), bias);
    return r;
}

// KIND: 0 linear, 1 conv 3x3, 2 conv 1x1.  OCC: waves per SIMD the register
// budget is sized for (2 lets two workgroups share a compute unit, so one's
// prologue and epilogue overlap the other's main loop).
template <int KIND, int CM, int XT, int DEC, int MC, int BM, int BN, int UPL, int OCC = 1>
__global__ void __launch_bounds__(256, OCC)
fused_fwd_kernel(Geom geo, FusedPlan plan, const void* __restrict__ cb, const uint8_t* __restrict__ crec,
                 const float* __restrict__ scales, const void* __restrict__ X, const float* __restrict__ x_scales,
                 void* __restrict__ Y, int y_dtype, float* __restrict__ part, uint32_t* __restrict__ arrivals) {
    constexpr bool CONV = KIND != 0;
    constexpr int KH = KIND == 1 ? 3 : 1;
    constexpr int NS = KIND == 1 ? 9 : CM;         // MFMA steps per chunk (= groups per lane)
    constexpr int AM = BM / 32, AN = BN / 32;
    using EntT = typename std::conditional<DEC == FUSED_DEC_T16G, uint16_t, uint8_t>::type;   // one code
    constexpr bool CB_LDS = DEC != FUSED_DEC_T16G && DEC != FUSED_DEC_REC;   // codebook copied to LDS
    static_assert(KIND != 1 || CM == 1, "3x3 chunks are 16 channels");

    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    // Every kernel argument the prologue reads is pinned to scalar registers
    // here, so they arrive in one scalar-memory round trip.  Left to itself the
    // compiler loads each group next to its first use and waits for it there:
    // four round trips before the first activation load, each a scalar-cache
    // miss while every wave of the launch starts at once.
    asm volatile("" ::"s"(geo.tokens), "s"(geo.C_out), "s"(geo.K), "s"(geo.B), "s"(geo.H), "s"(geo.W),
                 "s"(geo.cin), "s"(geo.OW), "s"(geo.OH), "s"(geo.stride), "s"(geo.pad));
    asm volatile("" ::"s"(plan.nchunk), "s"(plan.ps), "s"(plan.pw), "s"(plan.pr), "s"(plan.pbuf_bytes),
                 "s"(plan.nmajor), "s"(plan.units), "s"(plan.tile_div), "s"(plan.rec_bytes), "s"(plan.inv_pr),
                 "s"(plan.inv_ow), "s"(plan.cb_bytes), "s"(plan.x_bytes), "s"(plan.total_rows), "s"(plan.inv_wp),
                 "s"(plan.inv_tile_div), "s"(plan.inv_oh), "s"(cb), "s"(crec), "s"(X), "s"(gridDim.x),
                 "s"(plan.sr), "s"(plan.rpb), "s"(plan.inv_sr), "s"(plan.inv_rpb), "s"(plan.splitk),
                 "s"(plan.ntiles), "s"(plan.inv_ntiles));
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // uniform per wave: held in a scalar register, so chunk offsets are scalar arithmetic
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31;
    const int q = lane >> 5;
    // XCD-aware tile order: consecutive workgroup ids go to the 8 XCDs in turn,
    // so id h runs on XCD h % 8.  Giving each XCD a contiguous range of logical
    // tiles (output-channel tile fastest) keeps the input rows a token tile
    // shares with its neighbours, and with its other channel tiles, in one L2.
    int tile_m, tile_n, tile_lin, ksplit;
    {
        const int nwg = (int)gridDim.x, h = (int)blockIdx.x;
        const int xcd = h & 7, j = h >> 3;
        const int per = nwg >> 3, rem = nwg & 7;
        const int Lg = xcd * per + min(xcd, rem) + j;
        // K split slowest: an XCD's range of workgroups covers one split (the
        // same K range) of neighbouring tiles
        ksplit = __builtin_amdgcn_readfirstlane(fdiv(Lg, plan.ntiles, plan.inv_ntiles));
        const int L = Lg - ksplit * plan.ntiles;
        tile_lin = L;
        // plan.nmajor: channel tile slowest (an XCD's range then covers few
        // channel tiles, so the weight operands it streams stay in its L2);
        // else token tile slowest.  The host supplies the count of the fastest
        // tile index and its reciprocal, so this is branch-free.
        const int hi = __builtin_amdgcn_readfirstlane(fdiv(L, plan.tile_div, plan.inv_tile_div));
        const int lo = L - hi * plan.tile_div;
        tile_n = plan.nmajor ? hi : lo;
        tile_m = plan.nmajor ? lo : hi;
    }
    const int cstep = kWaves * plan.splitk;          // chunk stride of one wave
    const int T0 = tile_m * BM;                     // token and element counts fit in 31 bits (host check)
    const int N0 = tile_n * BN;
    const int tokens = (int)geo.tokens;

    // ---- codebook: global -> registers (stored to LDS once the first chunk's loads are in flight) ----
    // LDS layout [m][256 rows][row bytes]; the source is [m][2^B rows][row bytes].
    uint8_t* cb_lds = lds;
    constexpr int ROWB = DEC == FUSED_DEC_F32L ? 32 : 16;
    constexpr int CB_PER_T = CB_LDS ? (MC * 256 * ROWB) / (16 * 256) : 0;
    u32x4 cbr[CB_PER_T > 0 ? CB_PER_T : 1];
    const int rows_b = 1 << geo.B;
    if constexpr (CB_LDS) {
        const __amdgpu_buffer_rsrc_t cbs = buffer_rsrc(cb, (uint64_t)MC * rows_b * ROWB);
#pragma unroll
        for (int i = 0; i < CB_PER_T; ++i) {
            const int idx = tid + 256 * i;                 // 16-byte unit of the LDS layout
            const int m = idx / (256 * ROWB / 16);
            const int rem = idx - m * (256 * ROWB / 16);
            const int row = rem / (ROWB / 16), part = rem - row * (ROWB / 16);
            const uint32_t off = row < rows_b ? (uint32_t)(((m * rows_b + row) * (ROWB / 16) + part) * 16) : kOutOfRange;
            cbr[i] = __builtin_amdgcn_raw_buffer_load_b128(cbs, off, 0, 0);   // rows past 2^B read zeros
        }
    }
    uint8_t* pbuf0 = lds + plan.cb_bytes + wave * 2 * plan.pbuf_bytes;
    uint8_t* pbuf1 = pbuf0 + plan.pbuf_bytes;

    // ---- per-lane addressing, computed once (a chunk only adds a uniform offset) ----
    // Only what the first loads need is computed before they are issued; the
    // staging destinations and fragment offsets follow them.  Predicates are
    // bitwise (no branches) and products of small non-negative values use
    // 24-bit multiplies.
    const int HW = CONV ? geo.H * geo.W : 0;
    uint32_t a_base[AM];            // byte offset of this lane's A slice in a staging buffer
    uint32_t g_off[UPL];            // element offset of the unit's first value for chunk 0
    uint32_t l_off[UPL];            // byte offset of the unit's destination in a staging buffer
    bool g_ok[UPL];                 // the unit loads data (false: zeros)
    bool l_ok[UPL];                 // the unit exists
    int k_first[UPL];               // linear: first k of the unit for chunk 0
    const int gr0 = CONV ? fdiv(T0, geo.OW, plan.inv_ow) : 0;
    if constexpr (CONV) {
        const int wp = geo.W >> 1;  // pixel pairs per row
#pragma unroll
        for (int j = 0; j < UPL; ++j) {
            const int u = lane + 64 * j;
            const int t = fdiv(u, wp, plan.inv_wp);
            const int pp = u - __umul24(t, wp);
            const int o = fdiv(t, plan.pr, plan.inv_pr);
            const int pr = t - __umul24(o, plan.pr);
            // staged row pr: row jr of block blk, the input rows of plan.rpb
            // consecutive output rows starting at output row gr (one image)
            const int blk = fdiv(pr, plan.sr, plan.inv_sr), jr = pr - __umul24(blk, plan.sr);
            const int gr = gr0 + __umul24(blk, plan.rpb);
            const int b = fdiv(gr, geo.OH, plan.inv_oh), oh = gr - __umul24(b, geo.OH);
            const int ih = __umul24(oh, geo.stride) - geo.pad + jr;
            l_ok[j] = u < plan.units;
            g_ok[j] = l_ok[j] & (gr < plan.total_rows) & (ih >= 0) & (ih < geo.H);
            const uint32_t ga = (uint32_t)(__umul24(__umul24(b, geo.cin) + 8 * o, geo.H) + ih) * (uint32_t)geo.W + 2u * pp;
            g_off[j] = g_ok[j] ? ga : 0u;
            k_first[j] = 0;
            l_off[j] = l_ok[j] ? (uint32_t)(__umul24(o, plan.ps) + (__umul24(pr, plan.pw) + 2 * pp + geo.pad) * 16)
                               : (uint32_t)(plan.pbuf_bytes - 32);
        }
    } else {
#pragma unroll
        for (int j = 0; j < UPL; ++j) {
            const int u = lane + 64 * j;
            const int o = u % (2 * CM);
            const int tt = u / (2 * CM);
            const int T = T0 + tt;
            l_ok[j] = u < plan.units;
            g_ok[j] = l_ok[j] & (T < tokens);
            k_first[j] = 8 * o;
            const uint32_t ga = (uint32_t)(T * geo.K + 8 * o);
            g_off[j] = g_ok[j] ? ga : 0u;
            l_off[j] = l_ok[j] ? (uint32_t)(o * plan.ps + tt * 16) : (uint32_t)(plan.pbuf_bytes - 32);
        }
    }
    uint32_t c_off[AN];
    bool c_ok[AN];
#pragma unroll
    for (int b = 0; b < AN; ++b) {
        const int n = N0 + 32 * b + l32;
        c_ok[b] = n < geo.C_out;
        c_off[b] = c_ok[b] ? (uint32_t)__umul24(n * 2 + q, plan.rec_bytes) : 0u;
    }
    const uint32_t chunk_rec_stride = (uint32_t)geo.C_out * 2u * (uint32_t)plan.rec_bytes;

    // ---- staging of one chunk: global -> registers (out-of-range offsets read zeros) ----
    constexpr int SREG = CONV ? 8 : 4;    // dwords per unit
    constexpr int XB = XT == AQ_I8 ? 1 : 2;   // bytes per activation
    const __amdgpu_buffer_rsrc_t xr = buffer_rsrc(X, (uint64_t)plan.x_bytes);   // computed on the host
    uint32_t stage[UPL][SREG];
    // Chunks past the last one read zeros (no branch, so the compiler's wait
    // counts stay exact across the prefetch).
    auto stage_load = [&](int chunk) {
        const bool cv = chunk < plan.nchunk;
#pragma unroll
        for (int j = 0; j < UPL; ++j) {
            if constexpr (CONV) {
                // 8 channels x 2 pixels
                const uint32_t base = g_ok[j] & cv ? (g_off[j] + (uint32_t)(chunk * 16 * CM) * HW) * 2u : kOutOfRange;
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    stage[j][e] = __builtin_amdgcn_raw_buffer_load_b32(xr, base + (uint32_t)(e * HW * 2), 0, 0);
            } else {
                const int k = chunk * 16 * CM + k_first[j];
                const bool ok = g_ok[j] & cv & (k < geo.K);
                const uint32_t off = ok ? (g_off[j] + (uint32_t)(chunk * 16 * CM)) * XB : kOutOfRange;
                if constexpr (XT == AQ_I8) {
                    const auto v = __builtin_amdgcn_raw_buffer_load_b64(xr, off, 0, 0);
                    stage[j][0] = v[0];
                    stage[j][1] = v[1];
                } else {
                    const auto v = __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0);
                    stage[j][0] = v[0]; stage[j][1] = v[1]; stage[j][2] = v[2]; stage[j][3] = v[3];
                }
            }
        }
    };
    // registers -> LDS buffer (channel transpose for a convolution)
    auto stage_store = [&](uint8_t* buf) {
#pragma unroll
        for (int j = 0; j < UPL; ++j) {
            uint8_t* dst = buf + l_off[j];   // units past the end write a spare slot
            if constexpr (CONV) {
                u32x4 p0, p1;   // pixel 0 / pixel 1, channels 0..7
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    p0[d] = pick2(stage[j][2 * d], 0, stage[j][2 * d + 1], 0);
                    p1[d] = pick2(stage[j][2 * d], 1, stage[j][2 * d + 1], 1);
                }
                reinterpret_cast<u32x4*>(dst)[0] = p0;
                reinterpret_cast<u32x4*>(dst)[1] = p1;
            } else {
                u32x4 v;
                if constexpr (XT == AQ_I8) v = i8x8_to_f16((uint64_t)stage[j][0] | ((uint64_t)stage[j][1] << 32));
                else v = u32x4{stage[j][0], stage[j][1], stage[j][2], stage[j][3]};
                *reinterpret_cast<u32x4*>(dst) = v;
            }
        }
    };

    // ---- code records of one chunk: global -> registers ----
    constexpr int REC_DW = DEC == FUSED_DEC_REC ? 1 : (NS * MC * (int)sizeof(EntT) + 3) / 4;   // record dwords
    const __amdgpu_buffer_rsrc_t cr = buffer_rsrc(crec, (uint64_t)plan.nchunk * chunk_rec_stride);
    // pre-decoded mode: operand record (chunk, step, channel, lane half), 16 bytes each
    const __amdgpu_buffer_rsrc_t wr = buffer_rsrc(crec, (uint64_t)plan.nchunk * NS * geo.C_out * 32u);
    uint32_t crg[AN][REC_DW];
    auto codes_load = [&](int chunk) {
        if constexpr (DEC == FUSED_DEC_REC) return;
        const bool cv = chunk < plan.nchunk;
#pragma unroll
        for (int b = 0; b < AN; ++b) {
            const uint32_t off = c_ok[b] & cv ? c_off[b] + (uint32_t)chunk * chunk_rec_stride : kOutOfRange;
#pragma unroll
            for (int d = 0; d < REC_DW; d += 4) {
                if constexpr (true) {
                    if (d + 4 <= REC_DW) {
                        const auto v = __builtin_amdgcn_raw_buffer_load_b128(cr, off + 4 * d, 0, 0);
                        crg[b][d] = v[0]; crg[b][d + 1] = v[1]; crg[b][d + 2] = v[2]; crg[b][d + 3] = v[3];
                    } else if (d + 3 == REC_DW) {
                        const auto v = __builtin_amdgcn_raw_buffer_load_b96(cr, off + 4 * d, 0, 0);
                        crg[b][d] = v[0]; crg[b][d + 1] = v[1]; crg[b][d + 2] = v[2];
                    } else if (d + 2 == REC_DW) {
                        const auto v = __builtin_amdgcn_raw_buffer_load_b64(cr, off + 4 * d, 0, 0);
                        crg[b][d] = v[0]; crg[b][d + 1] = v[1];
                    } else {
                        crg[b][d] = __builtin_amdgcn_raw_buffer_load_b32(cr, off + 4 * d, 0, 0);
                    }
                }
            }
        }
    };

    // Prologue, first part: the chunk's codes and activations go out right
    // after the codebook, before the remaining index arithmetic.
    int chunk = wave + kWaves * ksplit;
    codes_load(chunk);
    stage_load(chunk);
    __builtin_amdgcn_sched_barrier(0);   // issue them here, not next to their uses
    if constexpr (CONV) {
#pragma unroll
        for (int a = 0; a < AM; ++a) {
            const int T = T0 + 32 * a + l32;
            const int gT = fdiv(T, geo.OW, plan.inv_ow);
            const int r = gT - gr0;
            const int ow = T - __umul24(gT, geo.OW);
            // output row r: block r / rpb, whose row (r % rpb) * stride is kernel row 0
            const int blk = fdiv(r, plan.rpb, plan.inv_rpb), rr = r - __umul24(blk, plan.rpb);
            const int R0 = __umul24(blk, plan.sr) + __umul24(rr, geo.stride);
            a_base[a] = (uint32_t)(q * plan.ps + (__umul24(R0, plan.pw) + __umul24(ow, geo.stride)) * 16);
        }
        // zero the padding columns of both buffers once: (buffer, plane, row, pad column)
        const int padc = plan.pw - geo.W;
        const int nrow = 2 * 2 * CM * plan.pr;
        for (int i = lane; i < nrow * padc; i += 64) {
            const int row = i / padc, pcx = i - row * padc;       // padc is 2 * pad, a small constant
            const int bsel = row & 1, rest = row >> 1;
            const int o = fdiv(rest, plan.pr, plan.inv_pr), pr = rest - o * plan.pr;
            const int pcol = pcx < geo.pad ? pcx : geo.W + pcx;
            uint8_t* dst = (bsel ? pbuf1 : pbuf0) + o * plan.ps + (pr * plan.pw + pcol) * 16;
            *reinterpret_cast<u32x4*>(dst) = u32x4{0u, 0u, 0u, 0u};
        }
    } else {
#pragma unroll
        for (int a = 0; a < AM; ++a) a_base[a] = (uint32_t)(q * plan.ps + (32 * a + l32) * 16);
    }

    // Accumulators start in matrix-core (AGPR) registers: the empty asm pins the
    // register class of the zero start value, so the loop-carried values stay
    // there instead of being copied from VGPRs before every block of products.
    floatx16 acc[AM][AN];
#pragma unroll
    for (int a = 0; a < AM; ++a)
#pragma unroll
        for (int b = 0; b < AN; ++b) {
            floatx16 z;
#pragma unroll
            for (int r = 0; r < 16; ++r) z[r] = 0.0f;
            asm volatile("" : "=a"(acc[a][b]) : "0"(z));
        }

    // activation fragments of one step (every token block), and of a whole chunk
    auto load_af_step = [&](const uint8_t* buf, u32x4 (&af)[NS][AM], int s) {
        uint32_t soff;
        if constexpr (KIND == 1) soff = (uint32_t)(((s / 3) * plan.pw + (s % 3)) * 16);
        else soff = (uint32_t)(2 * s * plan.ps);
#pragma unroll
        for (int a = 0; a < AM; ++a) af[s][a] = *reinterpret_cast<const u32x4*>(buf + a_base[a] + soff);
    };
    auto load_af = [&](const uint8_t* buf, u32x4 (&af)[NS][AM]) {
#pragma unroll
        for (int s = 0; s < NS; ++s) load_af_step(buf, af, s);
    };
    constexpr bool LOOKAHEAD = DEC != FUSED_DEC_F32L && NS * MC <= 18;
    // weights of one 32-channel block of a chunk, decoded into MFMA operands
    auto decode_block = [&](const uint32_t* codes_dw, int dchunk, int db, u32x4 (&d)[NS]) {
        if constexpr (LOOKAHEAD) {
            GroupRaw<DEC, MC> raw[NS];
#pragma unroll
            for (int g = 0; g < NS; ++g) gather_group<DEC, MC, EntT>(raw[g], codes_dw, g * MC, cb_lds, cb);
#pragma unroll
            for (int g = 0; g < NS; ++g) d[g] = combine_group<DEC, MC>(raw[g]);
        } else {
            GroupRaw<DEC, MC> raw1;
#pragma unroll
            for (int g = 0; g < NS; ++g) {
                gather_group<DEC, MC, EntT>(raw1, codes_dw, g * MC, cb_lds, cb);
                d[g] = combine_group<DEC, MC>(raw1);
            }
        }
    };
    // Software pipeline: the next block's codewords (for the last block, block 0
    // of this wave's next chunk) are read and summed while the current block's
    // MFMAs run, and the next chunk's activation fragments are read right after
    // its staging store, so a chunk starts with its operands in flight.  The
    // look-ahead is used when a block of raw codewords (groups x M x 16 bytes
    // per lane) fits in 72 registers.
    //
    // Prologue, second part.  The codebook store and the first block's decode
    // wait only for the codebook and the codes, so the decode runs while the
    // activations are still in flight.
    u32x4 af[NS][AM];
    u32x4 dec[NS];
    if constexpr (CB_LDS) {
#pragma unroll
        for (int i = 0; i < CB_PER_T; ++i) reinterpret_cast<u32x4*>(cb_lds)[tid + 256 * i] = cbr[i];
    }
    lds_barrier();   // codebook and padding visible (global loads stay in flight)
    if constexpr (DEC == FUSED_DEC_REC) {
        // Pre-decoded operands, steps outermost.  Each step's activation
        // fragments are read from LDS one step ahead of its products (two steps
        // of registers instead of a whole chunk's), the records of every channel
        // block of a step are loaded a chunk ahead into two register sets (chunk
        // parity P, static), and the next chunk is staged mid-chunk: the products
        // never drain at a chunk end.  Loads past the last chunk read zeros.
        u32x4 rec[2][NS][AN];
        u32x4 afb[2][AM];
        auto rec_step = [&](u32x4 (&dst)[AN], int c, int s) {
            const bool cv = c < plan.nchunk;
#pragma unroll
            for (int b = 0; b < AN; ++b) {
                const uint32_t base = (uint32_t)(((c * NS + s) * geo.C_out + N0 + 32 * b + l32) * 2 + q) * 16u;
                dst[b] = __builtin_amdgcn_raw_buffer_load_b128(wr, c_ok[b] & cv ? base : kOutOfRange, 0, 0);
            }
        };
        auto frag_step = [&](const uint8_t* buf, u32x4 (&dst)[AM], int s) {
            uint32_t soff;
            if constexpr (KIND == 1) soff = (uint32_t)(((s / 3) * plan.pw + (s % 3)) * 16);
            else soff = (uint32_t)(2 * s * plan.ps);
#pragma unroll
            for (int a = 0; a < AM; ++a) dst[a] = *reinterpret_cast<const u32x4*>(buf + a_base[a] + soff);
        };
#pragma unroll
        for (int s = 0; s < NS; ++s) rec_step(rec[0][s], chunk, s);
        stage_store(pbuf0);
        wave_sync();
        frag_step(pbuf0, afb[0], 0);
        // step s of a chunk of parity P uses fragment buffer (s + P NS) & 1, so
        // the buffers alternate across chunk boundaries for odd NS too
        auto body = [&](auto pc, int c) {
            constexpr int P = decltype(pc)::value;
            const uint8_t* cur = P ? pbuf1 : pbuf0;
            uint8_t* nxt = P ? pbuf0 : pbuf1;
            stage_load(c + cstep);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                rec_step(rec[1 - P][s], c + cstep, s);
                if (s == NS / 2) {
                    wave_sync();
                    stage_store(nxt);
                    wave_sync();
                }
                if (s + 1 < NS) frag_step(cur, afb[(s + 1 + P * NS) & 1], s + 1);
                else frag_step(nxt, afb[(s + 1 + P * NS) & 1], 0);
#pragma unroll
                for (int b = 0; b < AN; ++b)
#pragma unroll
                    for (int a = 0; a < AM; ++a) {
                        if constexpr (CONV) acc[a][b] = mfma_f16(rec[P][s][b], afb[(s + P * NS) & 1][a], acc[a][b]);
                        else acc[a][b] = mfma_f16(afb[(s + P * NS) & 1][a], rec[P][s][b], acc[a][b]);
                    }
                // each product followed by a share of the loads and fragment reads
#pragma unroll
                for (int i = 0; i < AN * AM; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                 // MFMA
                    if (i < AN) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);                    // VMEM read
                    if (i >= AN * AM - AM) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);         // DS read
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        for (; chunk + cstep < plan.nchunk; chunk += 2 * cstep) {
            body(std::integral_constant<int, 0>{}, chunk);
            body(std::integral_constant<int, 1>{}, chunk + cstep);
        }
        if (chunk < plan.nchunk) body(std::integral_constant<int, 0>{}, chunk);
    } else {
    // A wave without a chunk runs this on zeros, in its own staging buffer;
    // no branch here keeps the loads above from being sunk below the barrier.
    if constexpr (LOOKAHEAD) decode_block(crg[0], chunk, 0, dec);
    stage_store(pbuf0);
    wave_sync();
    load_af(pbuf0, af);
    int it = 0;
    for (; chunk < plan.nchunk; chunk += cstep, ++it) {
        uint8_t* nxt = (it & 1) ? pbuf0 : pbuf1;
        const bool more = chunk + cstep < plan.nchunk;
        uint32_t crn[AN][REC_DW];
#pragma unroll
        for (int b = 0; b < AN; ++b)
#pragma unroll
            for (int d = 0; d < REC_DW; ++d) crn[b][d] = crg[b][d];
        if (more) {
            stage_load(chunk + cstep);   // next chunk's activations and codes
            codes_load(chunk + cstep);
        }
#pragma unroll
        for (int b = 0; b < AN; ++b) {
            __builtin_amdgcn_sched_barrier(0);
            u32x4 dnext[NS];
            bool have_next = false;
            if constexpr (LOOKAHEAD) {
                if (b + 1 < AN) {
                    decode_block(crn[b + 1], chunk, b + 1, dnext);
                    have_next = true;
                } else if (more) {
                    decode_block(crg[0], chunk + cstep, 0, dnext);   // block 0 of the next chunk
                    have_next = true;
                }
            } else {
                decode_block(crn[b], chunk, b, dec);
            }
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                u32x4 bf;
                if constexpr (KIND == 1 && DEC != FUSED_DEC_REC) {
                    // position s: channel e of the lane's 8 is decoded value 9e + s
#pragma unroll
                    for (int d = 0; d < 4; ++d) {
                        const int v0 = 9 * (2 * d) + s, v1 = 9 * (2 * d + 1) + s;
                        bf[d] = pick2(dec[v0 >> 3][(v0 & 7) >> 1], v0 & 1, dec[v1 >> 3][(v1 & 7) >> 1], v1 & 1);
                    }
                } else {
                    bf = dec[s];
                }
#pragma unroll
                for (int a = 0; a < AM; ++a) {
                    if constexpr (CONV) acc[a][b] = mfma_f16(bf, af[s][a], acc[a][b]);   // rows: channels
                    else acc[a][b] = mfma_f16(af[s][a], bf, acc[a][b]);                  // rows: tokens
                }
            }
            if (have_next) {
#pragma unroll
                for (int g = 0; g < NS; ++g) dec[g] = dnext[g];
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        if (more) {
            wave_sync();
            stage_store(nxt);
            wave_sync();
            load_af(nxt, af);
        }
    }

    }   // in-loop decode

    // ---- epilogue: the four partial tiles meet in LDS, interleaved by 4 along
    // the MFMA row so that each lane writes float4s; then every thread sums 8
    // columns x 4 rows over the partials, scales, converts and writes four
    // 16-byte row segments.  Rows are output channels (convolution) or tokens
    // (linear); columns are tokens (convolution) or output channels (linear).
    constexpr int ROWS = CONV ? BN : BM;     // MFMA A rows of the tile
    constexpr int COLS = CONV ? BM : BN;     // MFMA B columns of the tile
    __syncthreads();   // every wave is done with its staging buffers
    // [wave][ROWS / 4][COLS + 1] float4; the padding float4 puts consecutive row
    // quads 4 banks apart, so the epilogue's reads (row quad fastest across
    // lanes) are conflict free
    constexpr int COLSP = COLS + 1;
    floatx4* red = reinterpret_cast<floatx4*>(lds + plan.cb_bytes);
#pragma unroll
    for (int a = 0; a < AM; ++a)
#pragma unroll
        for (int b = 0; b < AN; ++b)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                // register quad i holds rows 8 i + 4 q + (0..3) of the 32 x 32 block
                const int row0 = (CONV ? 32 * b : 32 * a) + 8 * i + 4 * q;
                const int col = (CONV ? 32 * a : 32 * b) + l32;
                red[(wave * (ROWS / 4) + row0 / 4) * COLSP + col] =
                    floatx4{acc[a][b][4 * i], acc[a][b][4 * i + 1], acc[a][b][4 * i + 2], acc[a][b][4 * i + 3]};
            }
    // Scales of this thread's epilogue task (one task per thread for every tile
    // used), loaded only once the accumulators are in LDS: live any earlier,
    // they push the accumulators out of the matrix-core registers (measured
    // on the linear kernels).  The partial-tile reads below hide their latency.
    constexpr int EROWS = CONV ? BN : BM, ECOLS = CONV ? BM : BN;
    float esc[8];
    float exs[4];
    const bool has_xs = !CONV && x_scales != nullptr;
    {
        const __amdgpu_buffer_rsrc_t sr = buffer_rsrc(scales, (uint64_t)geo.C_out * 4u);
        const __amdgpu_buffer_rsrc_t xsr = buffer_rsrc(x_scales, has_xs ? (uint64_t)geo.tokens * 4u : 0u);
        const int task = tid;
        const bool tok_task = task < (EROWS / 4) * (ECOLS / 8);
        const int c8 = (task / (EROWS / 4)) * 8;
        const int rq = task - (task / (EROWS / 4)) * (EROWS / 4);
        if constexpr (CONV) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                esc[e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                    sr, tok_task ? (uint32_t)(N0 + 4 * rq + e) * 4u : kOutOfRange, 0, 0));
#pragma unroll
            for (int e = 4; e < 8; ++e) esc[e] = 0.0f;
#pragma unroll
            for (int e = 0; e < 4; ++e) exs[e] = 0.0f;
        } else {
#pragma unroll
            for (int c = 0; c < 8; ++c)
                esc[c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                    sr, tok_task ? (uint32_t)(N0 + c8 + c) * 4u : kOutOfRange, 0, 0));
#pragma unroll
            for (int e = 0; e < 4; ++e)
                exs[e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                    xsr, tok_task && has_xs ? (uint32_t)(T0 + 4 * rq + e) * 4u : kOutOfRange, 0, 0));
        }
    }
    __syncthreads();
    const int ybytes = y_dtype == AQ_F32 ? 4 : 2;
    const __amdgpu_buffer_rsrc_t yr = buffer_rsrc(Y, (uint64_t)geo.tokens * geo.C_out * ybytes);
    const int plane = CONV ? geo.OH * geo.OW : 0;
    constexpr int TASKS = (ROWS / 4) * (COLS / 8);   // (4 rows, 8 columns) per task
    static_assert(TASKS <= 256, "one epilogue task per thread");
    const int task = tid;
    floatx4 v[8];
    if (task < TASKS) {
        const int c8 = (task / (ROWS / 4)) * 8;
        const int rq = task - (task / (ROWS / 4)) * (ROWS / 4);
        floatx4 pv[kWaves][8];
#pragma unroll
        for (int w = 0; w < kWaves; ++w)
#pragma unroll
            for (int c = 0; c < 8; ++c) pv[w][c] = red[(w * (ROWS / 4) + rq) * COLSP + c8 + c];
#pragma unroll
        for (int c = 0; c < 8; ++c) v[c] = ((pv[0][c] + pv[1][c]) + pv[2][c]) + pv[3][c];
    }
    if (plan.splitk > 1) {
        // K split over workgroups: publish this split's partial tile, count the
        // arrival; the last workgroup of the tile sums every split in order.
        // The partial tiles are written and read with device-coherent buffer
        // accesses (past the per-XCD L2, which may hold stale copies), so no
        // cache-wide write-back or invalidation is needed: each thread's stores
        // have completed (vmcnt 0) before the barrier that precedes the
        // arrival count, and the loads are issued after it.  Layout
        // [tile][split][8][TASKS] of 16-byte pieces, task fastest: one store or
        // load instruction of a wave covers 1 KB.
        const int S = plan.splitk;
        const __amdgpu_buffer_rsrc_t pr = buffer_rsrc(part, (uint64_t)plan.ntiles * S * TASKS * 8 * 16);
        const uint32_t mine = (uint32_t)(((tile_lin * S + ksplit) * 8 * TASKS + task) * 16);
        if (task < TASKS) {
#pragma unroll
            for (int c = 0; c < 8; ++c)
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v[c]), pr, mine + (uint32_t)(c * TASKS * 16),
                                                       0, kCoherent);
        }
        wait_vmcnt<0>();
        __syncthreads();                         // (every thread is also done reading the partial tiles in LDS)
        uint32_t* arrived = reinterpret_cast<uint32_t*>(lds);
        if (tid == 0) *arrived = __hip_atomic_fetch_add(arrivals + tile_lin, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        if (*arrived != (uint32_t)(S - 1)) return;   // not the last split of this tile (uniform)
        if (task < TASKS) {
            const uint32_t base = (uint32_t)((tile_lin * S * 8 * TASKS + task) * 16);
            for (int k = 0; k < S; ++k) {
                u32x4 q[8];
#pragma unroll
                for (int c = 0; c < 8; ++c)
                    q[c] = __builtin_amdgcn_raw_buffer_load_b128(pr, base + (uint32_t)((k * 8 + c) * TASKS * 16), 0,
                                                                 kCoherent);
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    const floatx4 f = __builtin_bit_cast(floatx4, q[c]);
                    v[c] = k == 0 ? f : v[c] + f;      // splits added in order 0, 1, ..., S - 1
                }
            }
        }
        if (tid == 0) __hip_atomic_store(arrivals + tile_lin, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (task < TASKS) {
        const int c8 = (task / (ROWS / 4)) * 8;
        const int rq = task - (task / (ROWS / 4)) * (ROWS / 4);
        // Columns are tokens (convolution: 8 consecutive tokens stay in one image
        // plane when the plane size is a multiple of 8) or output channels
        // (linear: 16-byte aligned when C_out is a multiple of 8).
        int col0, ncols, rows_left;
        bool aligned;
        if constexpr (CONV) {
            col0 = T0 + c8;
            ncols = min(8, tokens - col0);
            rows_left = geo.C_out - (N0 + 4 * rq);
            aligned = plane % 8 == 0;
        } else {
            col0 = N0 + c8;
            ncols = min(8, geo.C_out - col0);
            rows_left = tokens - (T0 + 4 * rq);
            aligned = geo.C_out % 8 == 0;
        }
        if (ncols == 8 && aligned) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (e >= rows_left) break;
                int yi0;
                float o[8];
                if constexpr (CONV) {
                    const int co = N0 + 4 * rq + e;
                    const int bimg = col0 / plane;
                    yi0 = (bimg * geo.C_out + co) * plane + (col0 - bimg * plane);
#pragma unroll
                    for (int c = 0; c < 8; ++c) o[c] = v[c][e] * esc[e];
                } else {
                    yi0 = (T0 + 4 * rq + e) * geo.C_out + col0;
#pragma unroll
                    for (int c = 0; c < 8; ++c) o[c] = v[c][e] * esc[c] * (has_xs ? exs[e] : 1.0f);
                }
                if (y_dtype == AQ_F32) {
                    __builtin_amdgcn_raw_buffer_store_b128(
                        u32x4{__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]), __float_as_uint(o[3])},
                        yr, yi0 * 4, 0, 0);
                    __builtin_amdgcn_raw_buffer_store_b128(
                        u32x4{__float_as_uint(o[4]), __float_as_uint(o[5]), __float_as_uint(o[6]), __float_as_uint(o[7])},
                        yr, yi0 * 4 + 16, 0, 0);
                } else {
                    u32x4 h;
#pragma unroll
                    for (int d = 0; d < 4; ++d)
                        h[d] = (uint32_t)f32_to_f16(o[2 * d]) | ((uint32_t)f32_to_f16(o[2 * d + 1]) << 16);
                    __builtin_amdgcn_raw_buffer_store_b128(h, yr, yi0 * 2, 0, 0);
                }
            }
        } else {
            for (int e = 0; e < 4 && e < rows_left; ++e)
                for (int c = 0; c < ncols; ++c) {
                    int yi;
                    float o;
                    if constexpr (CONV) {
                        const int tk = col0 + c, bb = tk / plane;
                        yi = (bb * geo.C_out + N0 + 4 * rq + e) * plane + (tk - bb * plane);
                        o = v[c][e] * esc[e];
                    } else {
                        yi = (T0 + 4 * rq + e) * geo.C_out + col0 + c;
                        o = v[c][e] * esc[c] * (has_xs ? exs[e] : 1.0f);
                    }
                    if (y_dtype == AQ_F32) __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(o), yr, yi * 4, 0, 0);
                    else __builtin_amdgcn_raw_buffer_store_b16(f32_to_f16(o), yr, yi * 2, 0, 0);
                }
        }
    }
}

template <int KIND, int CM, int XT, int DEC, int MC, int BM, int BN, int UPL, int OCC = 1>
static hipError_t fused_launch_cfg(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl) {
    auto kern = fused_fwd_kernel<KIND, CM, XT, DEC, MC, BM, BN, UPL, OCC>;
    hipError_t e = ensure_dynamic_lds((const void*)kern, plan.lds_bytes);
    if (e != hipSuccess) return e;
    if (fl.occupancy) return hipOccupancyMaxActiveBlocksPerMultiprocessor(fl.occupancy, kern, 256, plan.lds_bytes);
    const dim3 grid((unsigned)(((geo.tokens + BM - 1) / BM) * ((geo.C_out + BN - 1) / BN) * plan.splitk));
    kern<<<grid, 256, plan.lds_bytes, fl.stream>>>(geo, plan, fl.cb, fl.crec, fl.scales, fl.X, fl.x_scales, fl.Y,
                                                   fl.y_dtype, fl.part, fl.arrivals);
    note_launch(fl.stream, "fused_fwd_kernel", {KIND, CM, XT, DEC, MC, BM, BN, UPL, OCC});
    return hipGetLastError();
}

}  // namespace aq
