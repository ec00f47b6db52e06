// Matrix-core product of a 3x3 or 1x1 convolution over its pre-decoded
// operand records, gfx950 (Y = conv(X, W) with W decoded once per forward,
// Sec. 2.4 eq. (4); the convolution as an implicit im2col product, K ordered
// (input channel, kernel row, kernel column)).
//
// Work split.  A workgroup owns a BM (tokens) x BN (output channels) tile and
// its four waves split it 2 x 2: wave w covers token half (w & 1) and channel
// half (w >> 1) over the whole reduction dimension (WK = 1), or, for layers
// with too few such tiles to fill the chip, channel half (w & 1) of a tile
// half as tall over every other chunk (WK = 2; the two partial tiles are
// summed in LDS at the end, in a fixed order).  The fused decode kernel
// splits K between its waves instead (so that each wave decodes its own
// weights), which leaves each wave a quarter of the reduction and makes the
// workgroup reduce four partial tiles at the end; with the weights already
// decoded, every wave here runs the whole reduction, the prologue and
// epilogue are paid once per tile, and the input rows are staged once per
// workgroup for both token halves' four waves.
//
// Operands, per chunk (3x3: 16 input channels, 9 matrix-core steps, one per
// kernel position (kh, kw); 1x1: 64 input channels, 4 steps of 16):
//  * Activations (A operand, rows = tokens): the input rows the token tile
//    touches, the chunk's channels as planes of 8, are loaded two pixels of
//    one channel per 32-bit load, transposed with byte permutes to 16 bytes
//    per pixel (8 channels) and stored to one of two LDS buffers, whose zero
//    padding columns are written once.  A lane's 8 operand values for a step
//    are one 16-byte LDS read at its output pixel's input position.
//  * Weights (B operand, columns = output channels): record (chunk, step,
//    channel, lane half) holds the lane's 8 fp16 weights (3x3: channels
//    8 half + 0..7 of the chunk at kernel position step; 1x1: channels
//    16 step + 8 half + 0..7).  They are read straight into
//    registers, D - 1 steps ahead of their products, through a ring of D
//    register sets; the two waves of a channel half read the same records,
//    the second read hitting the L1 cache.
// One workgroup barrier per chunk: the next chunk's activations, loaded at the
// start of the chunk, are stored to the other LDS buffer after the chunk's
// last products are issued.  Loads past the data (channels, chunks, image
// borders) use an out-of-range buffer offset and return zeros.
//
// Output: lane (l32, q) ends with, for each 32-token block a, channel block b
// and register quad i, tokens 32 a + 8 i + 4 q + (0..3) of channel 32 b + l32;
// four consecutive tokens of one image are consecutive in NCHW, so each quad
// is scaled by the channel scale, rounded and stored as one 8-byte (fp16) or
// 16-byte (fp32) piece.
#include <algorithm>

#include "aq_device.h"

namespace aq {

namespace {

__device__ __forceinline__ floatx16 mfma_16(const u32x4& a, const u32x4& b, const floatx16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a), __builtin_bit_cast(half8, b), c, 0, 0,
                                                  0);
}

// Quotient of non-negative a < 2^24 by 1 <= d < 2^24 through an fp32
// reciprocal, corrected to the exact integer quotient.
__device__ __forceinline__ int qdiv_rc(int a, int d, float inv_d) {
    int qt = (int)((float)a * inv_d);
    qt += (int)__umul24(qt + 1, d) <= a;
    qt -= (int)__umul24(qt, d) > a;
    return qt;
}

// Dword made of fp16 half `hlo` of xlo (low half) and half `hhi` of xhi (high half).
__device__ __forceinline__ uint32_t halves(uint32_t xlo, int hlo, uint32_t xhi, int hhi) {
    const uint32_t sel = (uint32_t)(2 * hlo) | ((uint32_t)(2 * hlo + 1) << 8) | ((uint32_t)(4 + 2 * hhi) << 16) |
                         ((uint32_t)(5 + 2 * hhi) << 24);
    return __builtin_amdgcn_perm(xhi, xlo, sel);
}

// KIND: 1 for 3x3, 2 for 1x1; WK: waves sharing the reduction (1 or 2);
// TM / TN: 32-wide token / channel blocks per wave (tile 32 TM (3 - WK) x
// 64 TN); UPL: staging units (chunk of the iteration, plane, staged row, pixel
// pair) per thread; D: record register sets (records are loaded D - 1 steps
// ahead; D divides the steps of the two iterations the loop body covers).
template <int KIND, int WK, int TM, int TN, int UPL, int D>
__global__ void __launch_bounds__(256, 2)
rec_conv_kernel(Geom geo, FusedPlan plan, const uint8_t* __restrict__ rec, const float* __restrict__ scales,
                const void* __restrict__ X, void* __restrict__ Y, int y_dtype) {
    constexpr int NS = KIND == 1 ? 9 : 4;           // steps per chunk
    constexpr int CM = KIND == 1 ? 1 : 4;           // 16-channel slices per chunk (2 CM planes of 8)
    static_assert((2 * NS) % D == 0, "the record ring must divide two chunks");
    static_assert(WK == 1 || WK == 2, "one or two waves per reduction");
    constexpr int BM = 32 * TM * (3 - WK), BN = 64 * TN;
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    asm volatile("" ::"s"(geo.tokens), "s"(geo.C_out), "s"(geo.H), "s"(geo.W), "s"(geo.cin), "s"(geo.OW),
                 "s"(geo.OH), "s"(geo.stride), "s"(geo.pad));
    asm volatile("" ::"s"(plan.nchunk), "s"(plan.ps), "s"(plan.pw), "s"(plan.pr), "s"(plan.pbuf_bytes),
                 "s"(plan.nmajor), "s"(plan.units), "s"(plan.tile_div), "s"(plan.inv_pr), "s"(plan.inv_ow),
                 "s"(plan.x_bytes), "s"(plan.total_rows), "s"(plan.inv_wp), "s"(plan.inv_tile_div), "s"(plan.inv_oh),
                 "s"(plan.sr), "s"(plan.rpb), "s"(plan.inv_sr), "s"(plan.inv_rpb), "s"(rec), "s"(X));
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31, q = lane >> 5;

    // XCD-aware tile order: workgroup id h runs on XCD h % 8; each XCD gets a
    // contiguous range of logical tiles, the faster index varying first.
    int tile_m, tile_n;
    {
        const int nwg = (int)gridDim.x, h = (int)blockIdx.x;
        const int xcd = h & 7, j = h >> 3;
        const int per = nwg >> 3, rem = nwg & 7;
        const int L = xcd * per + min(xcd, rem) + j;
        const int hi = __builtin_amdgcn_readfirstlane(qdiv_rc(L, plan.tile_div, plan.inv_tile_div));
        const int lo = L - hi * plan.tile_div;
        tile_n = plan.nmajor ? hi : lo;
        tile_m = plan.nmajor ? lo : hi;
    }
    const int T0 = tile_m * BM, N0 = tile_n * BN;
    const int WT = WK == 1 ? (wave & 1) * 32 * TM : 0;          // the wave's token offset in the tile
    const int WN = (WK == 1 ? wave >> 1 : wave & 1) * 32 * TN;  // the wave's channel offset in the tile
    const int wk = WK == 1 ? 0 : wave >> 1;                      // the wave's chunks: wk, wk + WK, ...
    const int tokens = (int)geo.tokens;
    const int HW = geo.H * geo.W;
    // staging buffer (chunk g of an iteration, parity p) at lds + (2 g + p) pbuf_bytes

    // ---- staging units of this thread: unit tid + 256 j is (chunk g of the
    // iteration, plane o, staged row, pixel pair) ----
    const int gr0 = qdiv_rc(T0, geo.OW, plan.inv_ow);   // first output row of the tile
    uint32_t g_off[UPL];   // element offset of the unit's first value for iteration 0
    uint32_t l_off[UPL];   // byte offset of the unit's destination from its parity's buffer of chunk 0
    int u_chunk[UPL];      // the unit's chunk within an iteration
    bool g_ok[UPL];
    {
        const int wp = geo.W >> 1;
#pragma unroll
        for (int j = 0; j < UPL; ++j) {
            const int uu = tid + 256 * j;
            const int g = WK == 2 && uu >= plan.units ? 1 : 0;
            const int u = uu - g * plan.units;
            u_chunk[j] = g;
            const int t = qdiv_rc(u, wp, plan.inv_wp);
            const int pp = u - __umul24(t, wp);
            const int o = qdiv_rc(t, plan.pr, plan.inv_pr);
            const int pr = t - __umul24(o, plan.pr);
            // staged row pr: row jr of block blk, the input rows of plan.rpb
            // consecutive output rows starting at output row gr (one image)
            const int blk = qdiv_rc(pr, plan.sr, plan.inv_sr), jr = pr - __umul24(blk, plan.sr);
            const int gr = gr0 + __umul24(blk, plan.rpb);
            const int b = qdiv_rc(gr, geo.OH, plan.inv_oh), oh = gr - __umul24(b, geo.OH);
            const int ih = __umul24(oh, geo.stride) - geo.pad + jr;
            const bool l_ok = u < plan.units;
            g_ok[j] = l_ok & (gr < plan.total_rows) & (ih >= 0) & (ih < geo.H);
            g_off[j] = g_ok[j] ? (uint32_t)(__umul24(__umul24(b, geo.cin) + 8 * o + 16 * CM * g, geo.H) + ih) *
                                         (uint32_t)geo.W +
                                     2u * pp
                               : 0u;
            l_off[j] = l_ok ? (uint32_t)(2 * g * plan.pbuf_bytes + __umul24(o, plan.ps) +
                                         (__umul24(pr, plan.pw) + 2 * pp + geo.pad) * 16)
                            : (uint32_t)(plan.pbuf_bytes - 32);   // a spare slot
        }
    }
    const __amdgpu_buffer_rsrc_t xr = buffer_rsrc(X, (uint64_t)plan.x_bytes);
    uint32_t stg[UPL][8];
    // 8 channels x 2 pixels per unit of iteration it; chunks past the last read zeros
    auto stage_load = [&](int it) {
#pragma unroll
        for (int j = 0; j < UPL; ++j) {
            const bool cv = WK * it + u_chunk[j] < plan.nchunk;
            const uint32_t base =
                g_ok[j] & cv ? (g_off[j] + (uint32_t)(WK * it * 16 * CM) * (uint32_t)HW) * 2u : kOutOfRange;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                stg[j][e] = __builtin_amdgcn_raw_buffer_load_b32(xr, base + (uint32_t)(e * HW * 2), 0, 0);
        }
    };
    auto stage_store = [&](uint8_t* buf) {   // buf: the parity's buffer of chunk 0
#pragma unroll
        for (int j = 0; j < UPL; ++j) {
            u32x4 p0, p1;   // pixel 0 / pixel 1, channels 0..7
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                p0[d] = halves(stg[j][2 * d], 0, stg[j][2 * d + 1], 0);
                p1[d] = halves(stg[j][2 * d], 1, stg[j][2 * d + 1], 1);
            }
            uint8_t* dst = buf + l_off[j];
            reinterpret_cast<u32x4*>(dst)[0] = p0;
            reinterpret_cast<u32x4*>(dst)[1] = p1;
        }
    };

    // ---- A fragments: lane (l32, q) reads token WT + 32 a + l32, plane q ----
    uint32_t a_base[TM];
#pragma unroll
    for (int a = 0; a < TM; ++a) {
        const int T = T0 + WT + 32 * a + l32;
        const int gT = qdiv_rc(T, geo.OW, plan.inv_ow);
        const int r = gT - gr0;
        const int ow = T - __umul24(gT, geo.OW);
        // output row r: block r / rpb, whose row (r % rpb) * stride is kernel row 0
        const int blk = qdiv_rc(r, plan.rpb, plan.inv_rpb), rr = r - __umul24(blk, plan.rpb);
        const int R0 = __umul24(blk, plan.sr) + __umul24(rr, geo.stride);
        a_base[a] = (uint32_t)(2 * wk * plan.pbuf_bytes + q * plan.ps +
                               (__umul24(R0, plan.pw) + __umul24(ow, geo.stride)) * 16);
    }
    auto frag = [&](u32x4 (&dst)[TM], const uint8_t* buf, int s) {
        uint32_t soff;
        if constexpr (KIND == 1) soff = (uint32_t)(((s / 3) * plan.pw + (s % 3)) * 16);   // kernel position
        else soff = (uint32_t)(2 * s * plan.ps);                                           // planes 2 s, 2 s + 1
#pragma unroll
        for (int a = 0; a < TM; ++a) dst[a] = *reinterpret_cast<const u32x4*>(buf + a_base[a] + soff);
    };

    // ---- B operands: records of channel block b ----
    const uint32_t step_bytes = (uint32_t)geo.C_out * 32u;
    const __amdgpu_buffer_rsrc_t wr = buffer_rsrc(rec, (uint64_t)plan.nchunk * NS * step_bytes);
    uint32_t roff[TN];
    bool n_ok[TN];
#pragma unroll
    for (int b = 0; b < TN; ++b) {
        const int n = N0 + WN + 32 * b + l32;
        n_ok[b] = n < geo.C_out;
        roff[b] = (uint32_t)((n * 2 + q) * 16);
    }
    u32x4 rc[D][TN];
    // records of step s of this wave's chunk of iteration it
    auto rec_load = [&](u32x4 (&dst)[TN], int it, int s) {
        const int c = WK * it + wk;
        const bool cv = c < plan.nchunk;
#pragma unroll
        for (int b = 0; b < TN; ++b)
            dst[b] = __builtin_amdgcn_raw_buffer_load_b128(
                wr, n_ok[b] & cv ? roff[b] + (uint32_t)(c * NS + s) * step_bytes : kOutOfRange, 0, 0);
    };

    floatx16 acc[TM][TN];
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) {
            floatx16 z;
#pragma unroll
            for (int r = 0; r < 16; ++r) z[r] = 0.0f;
            asm volatile("" : "=a"(acc[a][b]) : "0"(z));   // accumulators live in AGPRs
        }

    // ---- prologue: iteration 0 staged, the first D - 1 steps' records in flight ----
    stage_load(0);
#pragma unroll
    for (int i = 0; i < D - 1; ++i) rec_load(rc[i], 0, i);
    __builtin_amdgcn_sched_barrier(0);
    {
        // zero padding columns of every buffer: (buffer, plane, staged row, pad column)
        const int padc = plan.pw - geo.W;
        const int nrow = 2 * WK * 2 * CM * plan.pr;
        for (int i = tid; i < nrow * padc; i += 256) {
            const int row = i / padc, pcx = i - row * padc;
            const int bsel = row % (2 * WK), rest = row / (2 * WK);
            const int o = rest / plan.pr, pr = rest - o * plan.pr;
            const int pcol = pcx < geo.pad ? pcx : geo.W + pcx;
            uint8_t* dst = lds + bsel * plan.pbuf_bytes + o * plan.ps + (pr * plan.pw + pcol) * 16;
            *reinterpret_cast<u32x4*>(dst) = u32x4{0u, 0u, 0u, 0u};
        }
    }
    uint8_t* buf0 = lds;
    uint8_t* buf1 = lds + plan.pbuf_bytes;
    stage_store(buf0);
    lds_barrier();
    u32x4 af[2][TM];
    frag(af[0], buf0, 0);

    // One iteration c of parity P (this wave's chunk WK c + wk): step s uses
    // fragment set (s + P NS) & 1 (the sets alternate across iterations for
    // odd NS too) and record set (s + P NS) % D.
    auto body = [&](auto pc, int c) {
        constexpr int P = decltype(pc)::value;
        const uint8_t* cur = P ? buf1 : buf0;
        uint8_t* nxt = P ? buf0 : buf1;
        stage_load(c + 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            // the next step's fragments first (the step's products cover their
            // latency), then the records D - 1 steps ahead into the set the
            // previous step used
            if (s + 1 < NS) frag(af[(s + 1 + P * NS) & 1], cur, s + 1);
            rec_load(rc[(s + P * NS + D - 1) % D], c + (s + D - 1) / NS, (s + D - 1) % NS);
#pragma unroll
            for (int b = 0; b < TN; ++b)
#pragma unroll
                for (int a = 0; a < TM; ++a)
                    acc[a][b] = mfma_16(af[(s + P * NS) & 1][a], rc[(s + P * NS) % D][b], acc[a][b]);
#pragma unroll
            for (int i = 0; i < TN * TM; ++i) {
                if (i < TM && s + 1 < NS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                             // MFMA
                if (i < TN) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);                // VMEM read
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // the next chunk's activations into the other buffer (its last reads
        // were issued before the previous barrier), then its first fragments
        stage_store(nxt);
        lds_barrier();
        frag(af[(NS + P * NS) & 1], nxt, 0);
    };
    const int niter = (plan.nchunk + WK - 1) / WK;
    int c = 0;
    for (; c + 1 < niter; c += 2) {
        body(std::integral_constant<int, 0>{}, c);
        body(std::integral_constant<int, 1>{}, c + 1);
    }
    if (c < niter) body(std::integral_constant<int, 0>{}, c);

    if constexpr (WK == 2) {
        // the second reduction half's partial tiles meet the first's in LDS
        // (the staging buffers are free once every wave is past this barrier)
        lds_barrier();
        floatx4* red = reinterpret_cast<floatx4*>(lds) + (WN / (32 * TN)) * (TM * TN * 4 * 64);
        if (wk == 1) {
#pragma unroll
            for (int a = 0; a < TM; ++a)
#pragma unroll
                for (int b = 0; b < TN; ++b)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        red[((a * TN + b) * 4 + i) * 64 + lane] =
                            floatx4{acc[a][b][4 * i], acc[a][b][4 * i + 1], acc[a][b][4 * i + 2], acc[a][b][4 * i + 3]};
        }
        lds_barrier();
        if (wk == 1) return;
#pragma unroll
        for (int a = 0; a < TM; ++a)
#pragma unroll
            for (int b = 0; b < TN; ++b)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const floatx4 o = red[((a * TN + b) * 4 + i) * 64 + lane];
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[a][b][4 * i + e] += o[e];
                }
    }

    // ---- epilogue: scale, round, store 4 consecutive tokens of one channel per quad ----
    const __amdgpu_buffer_rsrc_t sr = buffer_rsrc(scales, (uint64_t)geo.C_out * 4u);
    float esc[TN];
#pragma unroll
    for (int b = 0; b < TN; ++b)
        esc[b] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
            sr, n_ok[b] ? (uint32_t)(N0 + WN + 32 * b + l32) * 4u : kOutOfRange, 0, 0));
    const int ybytes = y_dtype == AQ_F32 ? 4 : 2;
    const __amdgpu_buffer_rsrc_t yr = buffer_rsrc(Y, (uint64_t)geo.tokens * geo.C_out * ybytes);
    const int plane = geo.OH * geo.OW;
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int t0 = T0 + WT + 32 * a + 8 * i + 4 * q;   // a multiple of 4; plane % 4 == 0 (host check)
            const int img = qdiv_rc(qdiv_rc(t0, geo.OW, plan.inv_ow), geo.OH, plan.inv_oh);
            const uint32_t pos = (uint32_t)(t0 - img * plane);
#pragma unroll
            for (int b = 0; b < TN; ++b) {
                const int n = N0 + WN + 32 * b + l32;
                if (!(n_ok[b] & (t0 < tokens))) continue;
                const uint32_t yi = (uint32_t)(img * geo.C_out + n) * (uint32_t)plane + pos;
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = acc[a][b][4 * i + e] * esc[b];
                if (y_dtype == AQ_F32) {
                    __builtin_amdgcn_raw_buffer_store_b128(
                        u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])},
                        yr, yi * 4u, 0, 0);
                } else {
                    const u32x2 h{(uint32_t)f32_to_f16(v[0]) | ((uint32_t)f32_to_f16(v[1]) << 16),
                                  (uint32_t)f32_to_f16(v[2]) | ((uint32_t)f32_to_f16(v[3]) << 16)};
                    __builtin_amdgcn_raw_buffer_store_b64(h, yr, yi * 2u, 0, 0);
                }
            }
        }
}

template <int KIND, int WK, int TM, int TN, int UPL, int D>
hipError_t rec_conv_cfg(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl) {
    auto kern = rec_conv_kernel<KIND, WK, TM, TN, UPL, D>;
    hipError_t e = ensure_dynamic_lds((const void*)kern, plan.lds_bytes);
    if (e != hipSuccess) return e;
    if (fl.occupancy) return hipOccupancyMaxActiveBlocksPerMultiprocessor(fl.occupancy, kern, 256, plan.lds_bytes);
    const dim3 grid((unsigned)plan.ntiles);
    kern<<<grid, 256, plan.lds_bytes, fl.stream>>>(geo, plan, fl.crec, fl.scales, fl.X, fl.Y, fl.y_dtype);
    note_launch(fl.stream, "rec_conv_kernel", {KIND, WK, TM, TN, UPL, D});
    return hipGetLastError();
}

// Instantiated (UPL, D) per tile: what fits 256 registers per lane without
// spills (192 channels: six record sets with one staging unit per thread; the
// two-wave reduction: three record sets, and at most two units for 192 channels).
template <int WK, int TN, int D>
hipError_t rec_conv3_upl(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl) {
    if (plan.upl == 1) return rec_conv_cfg<1, WK, 2, TN, 1, D>(geo, plan, fl);
    if constexpr (TN == 3 && D == 6) {
        return hipErrorInvalidConfiguration;
    } else {
        if (plan.upl == 2) return rec_conv_cfg<1, WK, 2, TN, 2, D>(geo, plan, fl);
        if constexpr (WK == 2 && TN == 3) {
            return hipErrorInvalidConfiguration;
        } else {
            if (plan.upl == 3) return rec_conv_cfg<1, WK, 2, TN, 3, D>(geo, plan, fl);
            return hipErrorInvalidConfiguration;
        }
    }
}

template <int WK>
hipError_t rec_conv_wk(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl) {
    if (plan.kind == 2) {
        // 1x1: 64 (3 - WK) tokens stage 8 planes x 64 pixels per chunk, two
        // units per thread; records three steps ahead (four sets)
        if (plan.upl != 2 || plan.rdepth != 4) return hipErrorInvalidConfiguration;
        return plan.bn == 192 ? rec_conv_cfg<2, WK, 2, 3, 2, 4>(geo, plan, fl)
                              : rec_conv_cfg<2, WK, 2, 2, 2, 4>(geo, plan, fl);
    }
    if (plan.kind != 1) return hipErrorInvalidConfiguration;
    if constexpr (WK == 2) {
        if (plan.rdepth != 3) return hipErrorInvalidConfiguration;
        return plan.bn == 192 ? rec_conv3_upl<2, 3, 3>(geo, plan, fl) : rec_conv3_upl<2, 2, 3>(geo, plan, fl);
    } else {
        if (plan.rdepth != 3 && plan.rdepth != 6) return hipErrorInvalidConfiguration;
        if (plan.bn == 192)
            return plan.rdepth == 6 ? rec_conv3_upl<1, 3, 6>(geo, plan, fl) : rec_conv3_upl<1, 3, 3>(geo, plan, fl);
        return plan.rdepth == 6 ? rec_conv3_upl<1, 2, 6>(geo, plan, fl) : rec_conv3_upl<1, 2, 3>(geo, plan, fl);
    }
}

}  // namespace

hipError_t launch_rec_conv(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl) {
    if (plan.dec != FUSED_DEC_REC || (plan.bn != 128 && plan.bn != 192)) return hipErrorInvalidConfiguration;
    if (plan.bm == 128) return rec_conv_wk<1>(geo, plan, fl);
    if (plan.bm == 64) return rec_conv_wk<2>(geo, plan, fl);
    return hipErrorInvalidConfiguration;
}

}  // namespace aq
