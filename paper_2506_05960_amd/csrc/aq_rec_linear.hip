// Matrix-core product of a linear layer over its pre-decoded operand records,
// gfx950 (Y = X W^T with W decoded once per forward, Sec. 2.4 eq. (4)).
//
// Work split.  A workgroup owns a BM (tokens) x BN (output channels) tile and
// its four waves split it 2 x 2: wave w covers token half (w & 1) and channel
// half (w >> 1) over the whole reduction dimension, so no partial tiles meet
// at the end.  Splitting K between the waves instead (as the fused decode
// kernel does, to share its decode work) makes every wave stream the operands
// of the whole tile; here each byte brought into the compute unit feeds 2-4x
// more products, which is what a layer without an in-loop decode needs.
//
// Operands, per 64-wide K chunk (4 matrix-core steps of 16):
//  * Weights: record (chunk, step, channel, lane half) holds the 8 fp16
//    weights of that lane's v_mfma_f32_32x32x16_f16 A operand (k = 64 chunk +
//    16 step + 8 half + 0..7).  A wave reads its channel blocks' records
//    straight into registers; the two waves of a channel half read the same
//    records, the second read hitting the L1 cache.
//  * Activations: the tile's 64-wide slice of X (fp16, or int8 widened exactly
//    to fp16 on the way) goes through registers into an LDS buffer of 8 planes
//    (8 consecutive k each) with 16 bytes per token, so a lane's 8 B-operand
//    values are one ds_read_b128 and 16 lanes read 256 contiguous bytes.
// Pipeline: record and activation loads are issued two chunks ahead of the
// products (three register sets, rotated by chunk mod 3), spread over the
// chunk's four steps between the products; the two LDS buffers alternate with
// one workgroup barrier per chunk.  Loads past the data (tokens, K or chunks) use an
// out-of-range buffer offset and return zeros, so the pipeline has no branch.
//
// Output: the products are arranged as (channel rows, token columns), so a
// lane ends with 4 consecutive channels of one token in 4 consecutive
// accumulator registers; they are scaled (channel scale, then the int8 token
// scale).  fp16 outputs (C_out a multiple of 8) pass through LDS so that each
// store instruction writes whole 128-byte row segments; otherwise each
// 4-channel piece is stored directly (8 bytes fp16, 16 bytes fp32).
#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include "aq_device.h"

namespace aq {

namespace {

struct RecLinArgs {
    int tokens, K, C_out, nchunk;
    int tile_div;             // tiles along the faster tile index
    float inv_tile_div;
    int nmajor;               // channel tile slowest (else token tile slowest)
    int y_dtype;
    uint32_t x_bytes;         // bytes of X
    uint32_t rec_bytes;       // bytes of the records
    uint32_t y_bytes;         // bytes of Y
    uint32_t step_bytes;      // record bytes of one (chunk, step): C_out * 32
};

__device__ __forceinline__ floatx16 mfma16(const u32x4& a, const u32x4& b, const floatx16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a), __builtin_bit_cast(half8, b), c, 0, 0,
                                                  0);
}

// 8 fp16 values from 8 int8 values, exactly: the fp16 bit pattern
// 0x6400 | (x ^ 0x80) encodes 1024 + (x + 128), and subtracting 1152 (exact for
// integers below 2048) leaves x.
__device__ __forceinline__ u32x4 widen_i8x8(uint32_t lo, uint32_t hi) {
    lo ^= 0x80808080u;
    hi ^= 0x80808080u;
    const uint32_t k64 = 0x64646464u;
    const uint32_t bias = 0xE480E480u;   // fp16 -1152 in both halves
    u32x4 r;
    r[0] = add_f16x2(__builtin_amdgcn_perm(k64, lo, 0x04010400u), bias);
    r[1] = add_f16x2(__builtin_amdgcn_perm(k64, lo, 0x04030402u), bias);
    r[2] = add_f16x2(__builtin_amdgcn_perm(k64, hi, 0x04010400u), bias);
    r[3] = add_f16x2(__builtin_amdgcn_perm(k64, hi, 0x04030402u), bias);
    return r;
}

// Byte offset `off` (< 2^31), or past the end of every buffer when !ok.  Set
// as a bit, not chosen: a select between an offset and a constant is turned
// into branches around the load, whose joins make the compiler wait for every
// load in flight.
__device__ __forceinline__ uint32_t off_if(bool ok, uint32_t off) { return off | ((uint32_t)!ok << 31); }

// Quotient of non-negative a < 2^24 by 1 <= d < 2^24 through an fp32
// reciprocal, corrected to the exact integer quotient.
__device__ __forceinline__ int qdiv(int a, int d, float inv_d) {
    int qt = (int)((float)a * inv_d);
    qt += (int)__umul24(qt + 1, d) <= a;
    qt -= (int)__umul24(qt, d) > a;
    return qt;
}

// TM / TN: 32-wide token / channel blocks per wave; WGT: waves along the
// tokens (2: a 2 x 2 split, 1: the four waves side by side along the channels).
// Tile 32 TM WGT tokens x 32 TN (4 / WGT) channels.
template <int XT, int TM, int TN, int WGT>
__global__ void __launch_bounds__(256, 1)
rec_linear_kernel(RecLinArgs ar, const uint8_t* __restrict__ rec, const float* __restrict__ scales,
                  const void* __restrict__ X, const float* __restrict__ x_scales, void* __restrict__ Y) {
    constexpr int WGN = 4 / WGT;                 // waves along the channels
    constexpr int BM = 32 * TM * WGT, BN = 32 * TN * WGN;
    constexpr int UPL = BM / 32;                 // staging units (token, plane) per thread
    constexpr int PS = BM * 16 + 32;             // plane stride: consecutive planes 2 banks apart
    constexpr int BUF = 8 * PS;                  // one staging buffer
    constexpr int XB = XT == AQ_I8 ? 1 : 2;      // bytes per activation
    constexpr int SW = XT == AQ_I8 ? 2 : 4;      // dwords per staging unit (8 values)
    constexpr int RS = 64 * TN + 16;             // epilogue: bytes per fp16 output row of a wave, padded

    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
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
        const int hi = __builtin_amdgcn_readfirstlane(qdiv(L, ar.tile_div, ar.inv_tile_div));
        const int lo = L - hi * ar.tile_div;
        tile_n = ar.nmajor ? hi : lo;
        tile_m = ar.nmajor ? lo : hi;
    }
    const int T0 = tile_m * BM, N0 = tile_n * BN;
    const int WT = (wave % WGT) * 32 * TM;       // the wave's token offset in the tile
    const int WN = (wave / WGT) * 32 * TN;       // the wave's channel offset in the tile

    // ---- activation staging: unit j of this thread is (token tt + 32 j, plane o) ----
    const __amdgpu_buffer_rsrc_t xr = buffer_rsrc(X, ar.x_bytes);
    const int o = tid & 7, tt = tid >> 3;
    uint32_t xoff[UPL];                          // byte offset of the unit for chunk 0 (kOutOfRange: none)
#pragma unroll
    for (int j = 0; j < UPL; ++j) {
        const int t = T0 + tt + 32 * j;
        xoff[j] = off_if(t < ar.tokens, (uint32_t)(t * ar.K + 8 * o) * XB);
    }
    uint32_t xs[3][UPL][SW];
    // activations of chunk c, units [j0, j0 + n)
    auto x_load = [&](uint32_t (&dst)[UPL][SW], int c, int j0, int n) {
        const bool kin = 64 * c + 8 * o < ar.K;    // also false past the last chunk
#pragma unroll
        for (int j = j0; j < j0 + n; ++j) {
            const uint32_t off = off_if(kin, xoff[j] + (uint32_t)(64 * c * XB));
            if constexpr (XT == AQ_I8) {
                const auto v = __builtin_amdgcn_raw_buffer_load_b64(xr, off, 0, 0);
                dst[j][0] = v[0];
                dst[j][1] = v[1];
            } else {
                const auto v = __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0);
                dst[j][0] = v[0]; dst[j][1] = v[1]; dst[j][2] = v[2]; dst[j][3] = v[3];
            }
        }
    };
    const uint32_t st_base = (uint32_t)(o * PS + tt * 16);
    auto x_store = [&](const uint32_t (&src)[UPL][SW], uint8_t* buf, int j0, int n) {
#pragma unroll
        for (int j = j0; j < j0 + n; ++j) {
            u32x4 v;
            if constexpr (XT == AQ_I8) v = widen_i8x8(src[j][0], src[j][1]);
            else v = u32x4{src[j][0], src[j][1], src[j][2], src[j][3]};
            *reinterpret_cast<u32x4*>(buf + st_base + 512 * j) = v;
        }
    };

    // ---- weight records: block b, step s of chunk c ----
    const __amdgpu_buffer_rsrc_t rr = buffer_rsrc(rec, ar.rec_bytes);
    uint32_t roff[TN];
#pragma unroll
    for (int b = 0; b < TN; ++b) {
        const int n = N0 + WN + 32 * b + l32;
        roff[b] = off_if(n < ar.C_out, (uint32_t)((n * 2 + q) * 16));
    }
    u32x4 rc[3][TN][4];
    // records of step s of chunk c (every channel block)
    auto rec_load = [&](u32x4 (&dst)[TN][4], int c, int s) {
        const bool cin = c < ar.nchunk;
#pragma unroll
        for (int b = 0; b < TN; ++b) {
            const uint32_t off = off_if(cin, roff[b] + (uint32_t)(4 * c + s) * ar.step_bytes);
            dst[b][s] = __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0);
        }
    };

    // B-operand (activation) fragment of step s, token block a: plane 2 s + q, token WT + 32 a + l32
    const uint32_t fr_base = (uint32_t)(q * PS + (WT + l32) * 16);

    floatx16 acc[TN][TM];
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int a = 0; a < TM; ++a) {
            floatx16 z;
#pragma unroll
            for (int r = 0; r < 16; ++r) z[r] = 0.0f;
            asm volatile("" : "=a"(acc[b][a]) : "0"(z));   // accumulators live in AGPRs
        }

    // One chunk c; P = c mod 3 picks the register sets (static), the LDS
    // buffer is c mod 2.  Chunk c + 2's records and activations are issued
    // and chunk c + 1's activations (issued one chunk ago) are staged a quarter
    // per step, interleaved with the step's products so that neither the
    // vector-memory queue nor the widening stalls the matrix cores.
    constexpr int XU = UPL / 4;                  // staging units per step
    auto body = [&](auto pc, int c) {
        constexpr int P = decltype(pc)::value;
        const uint8_t* cur = lds + (c & 1) * BUF;
        uint8_t* nxt = lds + ((c + 1) & 1) * BUF;
        // activation fragments double-buffered across steps
        u32x4 xf[2][TM];
        auto frag = [&](u32x4 (&dst)[TM], int s) {
#pragma unroll
            for (int a = 0; a < TM; ++a)
                dst[a] = *reinterpret_cast<const u32x4*>(cur + fr_base + (uint32_t)(2 * s * PS + 512 * a));
        };
        frag(xf[0], 0);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            rec_load(rc[(P + 2) % 3], c + 2, s);
            x_load(xs[(P + 2) % 3], c + 2, XU * s, XU);
            if (s + 1 < 4) frag(xf[(s + 1) & 1], s + 1);
            x_store(xs[(P + 1) % 3], nxt, XU * s, XU);
#pragma unroll
            for (int b = 0; b < TN; ++b)
#pragma unroll
                for (int a = 0; a < TM; ++a) acc[b][a] = mfma16(rc[P][b][s], xf[s & 1][a], acc[b][a]);
            // order within the step: each product followed by a share of the
            // loads, fragment reads, widening and staging writes
#pragma unroll
            for (int i = 0; i < TN * TM; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                               // MFMA
                if (i < TN + XU) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);             // VMEM read
                if (i >= TN * TM - TM && s + 1 < 4) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
                __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);                               // VALU
                if (i % (TN * TM / XU) == TN * TM / XU - 1) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);   // DS write
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        lds_barrier();
    };

    rec_load(rc[0], 0, 0); rec_load(rc[0], 0, 1); rec_load(rc[0], 0, 2); rec_load(rc[0], 0, 3);
    x_load(xs[0], 0, 0, UPL);
    rec_load(rc[1], 1, 0); rec_load(rc[1], 1, 1); rec_load(rc[1], 1, 2); rec_load(rc[1], 1, 3);
    x_load(xs[1], 1, 0, UPL);
    x_store(xs[0], lds, 0, UPL);
    lds_barrier();
    int c = 0;
    for (; c + 3 <= ar.nchunk; c += 3) {
        body(std::integral_constant<int, 0>{}, c);
        body(std::integral_constant<int, 1>{}, c + 1);
        body(std::integral_constant<int, 2>{}, c + 2);
    }
    if (c < ar.nchunk) body(std::integral_constant<int, 0>{}, c);
    if (c + 1 < ar.nchunk) body(std::integral_constant<int, 1>{}, c + 1);

    // ---- epilogue: lane (l32, q) holds, for channel block b and register quad
    // r, channels WN + 32 b + 8 r + 4 q + (0..3) of token WT + 32 a + l32 ----
    const __amdgpu_buffer_rsrc_t sr = buffer_rsrc(scales, (uint64_t)ar.C_out * 4u);
    const bool has_xs = x_scales != nullptr;
    const __amdgpu_buffer_rsrc_t xsr = buffer_rsrc(x_scales, has_xs ? (uint64_t)ar.tokens * 4u : 0u);
    floatx4 esc[TN][4];
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int ch = N0 + WN + 32 * b + 8 * r + 4 * q;
            const auto v = __builtin_amdgcn_raw_buffer_load_b128(sr, off_if(ch < ar.C_out, (uint32_t)ch * 4u), 0, 0);
            esc[b][r] = floatx4{__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]),
                                __uint_as_float(v[3])};
        }
    float exs[TM];
#pragma unroll
    for (int a = 0; a < TM; ++a) {
        const int t = T0 + WT + 32 * a + l32;
        exs[a] = __uint_as_float(
            __builtin_amdgcn_raw_buffer_load_b32(xsr, off_if(has_xs & (t < ar.tokens), (uint32_t)t * 4u), 0, 0));
    }
    const __amdgpu_buffer_rsrc_t yr = buffer_rsrc(Y, ar.y_bytes);
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    if (ar.y_dtype != AQ_F32 && (ar.C_out & 7) == 0) {
        // fp16 rows through LDS (the staging buffers are free after the last
        // barrier): each wave writes its 32 TM x 32 TN sub-tile as rows of RS
        // bytes, then 4 TN lanes store one row's 64 TN contiguous bytes
        uint8_t* ew = lds + wave * (32 * TM * RS);
#pragma unroll
        for (int a = 0; a < TM; ++a) {
            const float xa = has_xs ? exs[a] : 1.0f;   // times 1 is exact
#pragma unroll
            for (int b = 0; b < TN; ++b)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    float v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = (acc[b][a][4 * r + e] * esc[b][r][e]) * xa;
                    const u32x2 h{(uint32_t)f32_to_f16(v[0]) | ((uint32_t)f32_to_f16(v[1]) << 16),
                                  (uint32_t)f32_to_f16(v[2]) | ((uint32_t)f32_to_f16(v[3]) << 16)};
                    *reinterpret_cast<u32x2*>(ew + (32 * a + l32) * RS + 64 * b + 16 * r + 8 * q) = h;
                }
        }
        asm volatile("" ::: "memory");
        __builtin_amdgcn_wave_barrier();   // one wave's LDS accesses execute in order
        asm volatile("" ::: "memory");
#pragma unroll
        for (int i = 0; i < 2 * TM * TN; ++i) {
            const int R = (16 / TN) * i + lane / (4 * TN), C = lane % (4 * TN);
            const u32x4 v = *reinterpret_cast<const u32x4*>(ew + R * RS + 16 * C);
            const int t = T0 + WT + R, ch = N0 + WN + 8 * C;
            const bool ok = (t < ar.tokens) & (ch < ar.C_out);   // C_out % 8 == 0: the segment is whole
            __builtin_amdgcn_raw_buffer_store_b128(v, yr, off_if(ok, ((uint32_t)t * (uint32_t)ar.C_out + (uint32_t)ch) * 2u),
                                                   0, 0);
        }
        return;
    }
#pragma unroll
    for (int a = 0; a < TM; ++a) {
        const int t = T0 + WT + 32 * a + l32;
#pragma unroll
        for (int b = 0; b < TN; ++b)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int ch = N0 + WN + 32 * b + 8 * r + 4 * q;
                const bool ok = (t < ar.tokens) & (ch < ar.C_out);   // C_out % 4 == 0: the quad is whole
                const uint32_t idx = (uint32_t)t * (uint32_t)ar.C_out + (uint32_t)ch;
                const float xa = has_xs ? exs[a] : 1.0f;   // times 1 is exact
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = (acc[b][a][4 * r + e] * esc[b][r][e]) * xa;
                if (ar.y_dtype == AQ_F32) {
                    __builtin_amdgcn_raw_buffer_store_b128(
                        u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])},
                        yr, off_if(ok, idx * 4u), 0, 0);
                } else {
                    const u32x2 h{(uint32_t)f32_to_f16(v[0]) | ((uint32_t)f32_to_f16(v[1]) << 16),
                                  (uint32_t)f32_to_f16(v[2]) | ((uint32_t)f32_to_f16(v[3]) << 16)};
                    __builtin_amdgcn_raw_buffer_store_b64(h, yr, off_if(ok, idx * 2u), 0, 0);
                }
            }
    }
}

// staging (two buffers of 8 planes) or the epilogue's fp16 rows (4 waves x 32 TM rows of 64 TN + 16 bytes)
constexpr size_t rec_linear_lds_bytes(int BM, int TM, int TN) {
    return (size_t)2 * 8 * (BM * 16 + 32) > (size_t)4 * 32 * TM * (64 * TN + 16)
               ? (size_t)2 * 8 * (BM * 16 + 32)
               : (size_t)4 * 32 * TM * (64 * TN + 16);
}

template <int XT, int TM, int TN, int WGT>
hipError_t rec_linear_cfg(const RecLinArgs& ar, const FusedLaunch& fl) {
    auto kern = rec_linear_kernel<XT, TM, TN, WGT>;
    constexpr int BM = 32 * TM * WGT, BN = 32 * TN * (4 / WGT);
    constexpr size_t lds = rec_linear_lds_bytes(BM, TM, TN);
    const hipError_t e = ensure_dynamic_lds((const void*)kern, lds);
    if (e != hipSuccess) return e;
    const int64_t tm = (ar.tokens + BM - 1) / BM, tn = (ar.C_out + BN - 1) / BN;
    const dim3 grid((unsigned)(tm * tn));
    kern<<<grid, 256, lds, fl.stream>>>(ar, fl.crec, fl.scales, fl.X, fl.x_scales, fl.Y);
    note_launch(fl.stream, "rec_linear_kernel", {XT, TM, TN, WGT});
    return hipGetLastError();
}

}  // namespace

bool rec_linear_supported(const Geom& geo, const FusedPlan& plan, int x_dtype) {
    if (geo.conv || plan.kind != 0 || plan.cm != 4 || geo.g != 8) return false;
    if (x_dtype != AQ_F16 && x_dtype != AQ_I8) return false;
    if (geo.C_out % 4 != 0) return false;
    const int64_t lim = int64_t(1) << 31;
    const int64_t rec_bytes = (int64_t)plan.nchunk * 4 * geo.C_out * 32;
    return geo.tokens * (int64_t)std::max(geo.K, geo.C_out) * 4 < lim && rec_bytes < lim && geo.tokens < (1 << 24);
}

// Tile variant: 0 = 128 x 128 in a 2 x 2 wave split, 1 = 256 x 128 in a 2 x 2
// split, 2 = 128 x 128 with the four waves side by side along the channels.
// `forced` is the option value (0 planner, 1 = variant 1, 2 = variant 2,
// 3 = variant 0).  The planner takes variant 2: each wave then reads one
// channel block of records and all four token blocks of the activations per
// step, and measured 3-6 % faster than the 2 x 2 split on every linear shape
// here (U-Net 8192 tokens x 384 -> 1152: 19.2 vs 20.2 us per forward; 8192 x
// 576 -> 1728 int8: 29.4-31.5 vs 31.3-33.3 us); the 256-token tile is slower
// (one workgroup per compute unit).
int rec_linear_tile(const Geom& geo, int forced) {
    (void)geo;
    if (forced == 1 || forced == 2) return forced;
    if (forced == 3) return 0;
    return 2;
}

hipError_t launch_rec_linear(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl) {
    RecLinArgs ar{};
    ar.tokens = (int)geo.tokens;
    ar.K = geo.K;
    ar.C_out = geo.C_out;
    ar.nchunk = plan.nchunk;
    const int var = plan.rlin_var;
    const int bm = var == 1 ? 256 : 128, bn = 128;
    const int tm = (int)((geo.tokens + bm - 1) / bm), tn = (geo.C_out + bn - 1) / bn;
    ar.nmajor = plan.nmajor;
    ar.tile_div = ar.nmajor ? tm : tn;
    ar.inv_tile_div = 1.0f / (float)ar.tile_div;
    ar.y_dtype = fl.y_dtype;
    const int xb = fl.x_dtype == AQ_I8 ? 1 : 2;
    ar.x_bytes = (uint32_t)(geo.tokens * geo.K * xb);
    ar.rec_bytes = (uint32_t)((int64_t)plan.nchunk * 4 * geo.C_out * 32);
    ar.y_bytes = (uint32_t)(geo.tokens * geo.C_out * (fl.y_dtype == AQ_F32 ? 4 : 2));
    ar.step_bytes = (uint32_t)geo.C_out * 32u;
    if (fl.x_dtype == AQ_I8) {
        if (var == 1) return rec_linear_cfg<AQ_I8, 4, 2, 2>(ar, fl);
        if (var == 2) return rec_linear_cfg<AQ_I8, 4, 1, 1>(ar, fl);
        return rec_linear_cfg<AQ_I8, 2, 2, 2>(ar, fl);
    }
    if (var == 1) return rec_linear_cfg<AQ_F16, 4, 2, 2>(ar, fl);
    if (var == 2) return rec_linear_cfg<AQ_F16, 4, 1, 1>(ar, fl);
    return rec_linear_cfg<AQ_F16, 2, 2, 2>(ar, fl);
}

}  // namespace aq
