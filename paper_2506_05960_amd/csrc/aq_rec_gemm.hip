// Matrix-core forward over pre-decoded operand records (the decompress-then-
// compute route; Sec. 4.4 describes decompressing the weights before the
// dense product).  The records are the B operands of v_mfma_f32_32x32x16_f16
// exactly as the fused kernel would decode them (`operand_records_kernel`),
// so this kernel is a dense fp16 implicit-im2col product:
//
//  * A workgroup of 4 waves owns a BM (tokens) x BN (output channels) tile;
//    the waves sit 2 x 2 on it, each accumulating a (BM/2) x (BN/2) quarter.
//  * K is walked in the fused kernel's chunks (16 input channels x 9 kernel
//    positions for a 3x3 convolution, 64 consecutive k otherwise).  Each chunk's
//    activations (the input rows the tile touches, 8-channel planes of 16 B
//    per pixel, zero padding columns) and weight records (BN channels x steps
//    x 32 B, stored step- and lane-half-major so that 16 consecutive lanes read
//    16 consecutive records) are staged in LDS by the whole workgroup, double
//    buffered with one barrier per chunk, and every wave reads its A and B
//    fragments from there.
//  * No partial tiles to combine; the tile passes through LDS once so that
//    the stores are 16-byte row segments.
#include "aq_fused_kernel.h"

namespace aq {

template <int KIND, int XT, int BM, int BN>
__global__ void __launch_bounds__(256, 1)
rec_gemm_kernel(Geom geo, FusedPlan plan, const uint8_t* __restrict__ recs, const float* __restrict__ scales,
                const void* __restrict__ X, const float* __restrict__ x_scales, void* __restrict__ Y, int y_dtype) {
    constexpr bool CONV = KIND != 0;
    constexpr int KH = KIND == 1 ? 3 : 1;
    constexpr int CM = KIND == 1 ? 1 : 4;
    constexpr int NS = KIND == 1 ? 9 : CM;          // MFMA steps per chunk
    constexpr int WM = BM / 2, WN = BN / 2;         // a wave's quarter
    constexpr int AM = WM / 32, AN = WN / 32;
    constexpr int UPL = CONV ? 3 : 4;               // staging units per thread (the planner keeps units <= 256 UPL)
    constexpr int BREC = NS * BN * 2;               // 16-byte weight records per chunk
    constexpr int BPT = (BREC + 255) / 256;         // weight records per thread

    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int l32 = lane & 31;
    const int q = lane >> 5;
    int tile_m, tile_n;
    {
        const int nwg = (int)gridDim.x, h = (int)blockIdx.x;
        const int xcd = h & 7, j = h >> 3;
        const int per = nwg >> 3, rem = nwg & 7;
        const int L = xcd * per + min(xcd, rem) + j;
        if (plan.nmajor) {
            // channel tile slowest: an XCD's range covers few channel tiles, so the
            // weight operands it streams stay in its L2
            const int ntm = (int)((geo.tokens + BM - 1) / BM);
            tile_n = L / ntm;
            tile_m = L - tile_n * ntm;
        } else {
            const int ntn = (geo.C_out + BN - 1) / BN;
            tile_m = L / ntn;
            tile_n = L - tile_m * ntn;
        }
    }
    const int T0 = tile_m * BM;
    const int N0 = tile_n * BN;
    const int tokens = (int)geo.tokens;

    // LDS: two stages, each [activation planes | weight records]
    const int abytes = plan.pbuf_bytes;              // activation planes (+ spare slot)
    const int stage_bytes = abytes + BREC * 16;
    uint8_t* st0 = lds;
    uint8_t* st1 = lds + stage_bytes;

    // ---- activation staging addresses (whole workgroup) ----
    const int HW = CONV ? geo.H * geo.W : 0;
    uint32_t a_base[AM];
    uint32_t g_off[UPL], l_off[UPL];
    bool g_ok[UPL];
    int k_first[UPL];
    if constexpr (CONV) {
        const float inv_ow = 1.0f / (float)geo.OW, inv_oh = 1.0f / (float)geo.OH;
        const float inv_pr = 1.0f / (float)plan.pr;
        const int gr0 = fdiv(T0, geo.OW, inv_ow);
#pragma unroll
        for (int a = 0; a < AM; ++a) {
            const int T = T0 + WM * wm + 32 * a + l32;
            const int gT = fdiv(T, geo.OW, inv_ow);
            const int r = gT - gr0;
            const int ow = T - gT * geo.OW;
            a_base[a] = (uint32_t)(q * plan.ps + ((r * KH) * plan.pw + ow * geo.stride) * 16);
        }
        const int wp = geo.W >> 1;
        const float inv_wp = 1.0f / (float)wp;
#pragma unroll
        for (int j = 0; j < UPL; ++j) {
            const int u = tid + 256 * j;
            const int t = fdiv(u, wp, inv_wp);
            const int pp = u - t * wp;
            const int o = fdiv(t, plan.pr, inv_pr);
            const int pr = t - o * plan.pr;
            const int r = pr / KH, kh = pr - r * KH;
            const int gr = gr0 + r;
            const int b = fdiv(gr, geo.OH, inv_oh), oh = gr - b * geo.OH;
            const int ih = oh * geo.stride - geo.pad + kh;
            const bool l_ok = u < plan.units;
            g_ok[j] = l_ok && gr < plan.total_rows && ih >= 0 && ih < geo.H;
            g_off[j] = g_ok[j] ? (uint32_t)(__umul24(__umul24(b, geo.cin) + 8 * o, geo.H) + ih) * (uint32_t)geo.W + 2u * pp : 0u;
            l_off[j] = l_ok ? (uint32_t)(o * plan.ps + (pr * plan.pw + 2 * pp + geo.pad) * 16) : (uint32_t)(abytes - 32);
            k_first[j] = 0;
        }
        // zero the padding columns of both stages once
        const int padc = plan.pw - geo.W;
        const int nrow = 2 * 2 * CM * plan.pr;
        for (int i = tid; i < nrow * padc; i += 256) {
            const int row = i / padc, pcx = i - row * padc;
            const int bsel = row & 1, rest = row >> 1;
            const int o = fdiv(rest, plan.pr, inv_pr), pr = rest - o * plan.pr;
            const int pcol = pcx < geo.pad ? pcx : geo.W + pcx;
            uint8_t* dst = (bsel ? st1 : st0) + o * plan.ps + (pr * plan.pw + pcol) * 16;
            *reinterpret_cast<u32x4*>(dst) = u32x4{0u, 0u, 0u, 0u};
        }
    } else {
#pragma unroll
        for (int a = 0; a < AM; ++a) a_base[a] = (uint32_t)(q * plan.ps + (WM * wm + 32 * a + l32) * 16);
#pragma unroll
        for (int j = 0; j < UPL; ++j) {
            const int u = tid + 256 * j;
            const int o = u % (2 * CM);
            const int tt = u / (2 * CM);
            const int T = T0 + tt;
            const bool l_ok = u < plan.units;
            g_ok[j] = l_ok && T < tokens;
            k_first[j] = 8 * o;
            g_off[j] = g_ok[j] ? (uint32_t)(T * geo.K + 8 * o) : 0u;
            l_off[j] = l_ok ? (uint32_t)(o * plan.ps + tt * 16) : (uint32_t)(abytes - 32);
        }
    }

    constexpr int SREG = CONV ? 8 : 4;
    constexpr int XB = XT == AQ_I8 ? 1 : 2;
    const uint64_t xbytes = CONV ? (uint64_t)plan.total_rows / geo.OH * geo.cin * HW * 2
                                 : (uint64_t)geo.tokens * geo.K * XB;
    const __amdgpu_buffer_rsrc_t xr = buffer_rsrc(X, xbytes);
    const __amdgpu_buffer_rsrc_t wr = buffer_rsrc(recs, (uint64_t)plan.nchunk * NS * geo.C_out * 32u);
    struct Regs {
        uint32_t stage[UPL][SREG];
    };
    Regs ra;                                         // the next chunk's activations, in flight
    // weight records go straight from global memory into the stage's LDS area
    // (direct-to-LDS loads: lane l of a wave fills slot base + l); every wave
    // issues whole 64-record runs, so the stage's run count is wave-uniform
    auto issue_weights = [&](int chunk, uint8_t* stg) {
        uint8_t* wdst = stg + abytes;
#pragma unroll
        for (int i = 0; i < BPT; ++i) {
            const int run0 = 256 * i + 64 * wave;    // first slot of this wave's run
            if (run0 < BREC) {
                // LDS slot e = (s * 2 + h) * BN + n holds record (chunk, s, N0 + n, h); channels
                // past C_out read a valid record whose products are never stored
                const int e = run0 + lane;
                const int sh = e / BN;
                const int n = e - sh * BN;
                const int st = sh >> 1, h = sh & 1;
                const int nc = min(N0 + n, geo.C_out - 1);
                const uint8_t* src = recs + ((size_t)((chunk * NS + st) * geo.C_out + nc) * 2 + h) * 16;
                __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                                 (__attribute__((address_space(3))) void*)(wdst + (size_t)run0 * 16),
                                                 16, 0, 0);
            }
        }
    };
    auto load_chunk = [&](int chunk, Regs& rg) {
        auto& stage = rg.stage;
#pragma unroll
        for (int j = 0; j < UPL; ++j) {
            if constexpr (CONV) {
                const uint32_t base = g_ok[j] ? (g_off[j] + (uint32_t)(chunk * 16 * CM) * HW) * 2u : kOutOfRange;
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    stage[j][e] = __builtin_amdgcn_raw_buffer_load_b32(xr, base + (uint32_t)(e * HW * 2), 0, 0);
            } else {
                const int k = chunk * 16 * CM + k_first[j];
                const bool ok = g_ok[j] && k < geo.K;
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
    auto store_chunk = [&](uint8_t* stg, const Regs& rg) {
        const auto& stage = rg.stage;
#pragma unroll
        for (int j = 0; j < UPL; ++j) {
            uint8_t* dst = stg + l_off[j];
            if constexpr (CONV) {
                u32x4 p0, p1;
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

    floatx16 acc[AM][AN];
#pragma unroll
    for (int a = 0; a < AM; ++a)
#pragma unroll
        for (int b = 0; b < AN; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

    // fragments of step s: the A slices of the wave's token blocks and the B
    // records of its channel blocks; step s + 1's are read before step s's
    // MFMAs are issued, so LDS latency hides behind the matrix cores
    auto frag_load = [&](const uint8_t* cur, int s, u32x4 (&af)[AM], u32x4 (&bf)[AN]) {
        const u32x4* wl = reinterpret_cast<const u32x4*>(cur + abytes);
        uint32_t soff;
        if constexpr (KIND == 1) soff = (uint32_t)(((s / 3) * plan.pw + (s % 3)) * 16);
        else soff = (uint32_t)(2 * s * plan.ps);
#pragma unroll
        for (int a = 0; a < AM; ++a) af[a] = *reinterpret_cast<const u32x4*>(cur + a_base[a] + soff);
#pragma unroll
        for (int b = 0; b < AN; ++b) bf[b] = wl[(s * 2 + q) * BN + WN * wn + 32 * b + l32];
    };
    auto compute = [&](const uint8_t* cur) {
        u32x4 af[2][AM], bf[2][AN];
        frag_load(cur, 0, af[0], bf[0]);
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            if (s + 1 < NS) frag_load(cur, s + 1, af[(s + 1) & 1], bf[(s + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);   // keep the reads ahead of this step's MFMAs
#pragma unroll
            for (int a = 0; a < AM; ++a)
#pragma unroll
                for (int b = 0; b < AN; ++b) {
                    if constexpr (CONV) acc[a][b] = mfma_f16(bf[s & 1][b], af[s & 1][a], acc[a][b]);   // rows: channels
                    else acc[a][b] = mfma_f16(af[s & 1][a], bf[s & 1][b], acc[a][b]);                  // rows: tokens
                }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // chunk c is computed from stage c % 2 while chunk c + 1 is fetched into registers
    const int nch = plan.nchunk;
    if (nch > 0) {
        issue_weights(0, st0);
        load_chunk(0, ra);
        store_chunk(st0, ra);
    }
    __builtin_amdgcn_s_waitcnt(0);                   // the direct-to-LDS loads have landed
    __syncthreads();
    for (int chunk = 0; chunk < nch; ++chunk) {
        uint8_t* cur = (chunk & 1) ? st1 : st0;
        uint8_t* nxt = (chunk & 1) ? st0 : st1;
        const bool more = chunk + 1 < nch;
        if (more) {
            load_chunk(chunk + 1, ra);
            issue_weights(chunk + 1, nxt);
        }
        compute(cur);
        if (more) store_chunk(nxt, ra);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    }

    // ---- epilogue: the tile meets in LDS (rows interleaved by 4 so that each
    // lane writes float4s, plus one padding float4 per row quad), then every
    // thread scales, converts and writes 4 rows x 8 columns as 16-byte segments.
    // Rows are output channels (convolution) or tokens (linear).
    constexpr int ROWS = CONV ? BN : BM, COLS = CONV ? BM : BN;
    constexpr int COLSP = COLS + 1;
    floatx4* red = reinterpret_cast<floatx4*>(lds);   // the stages are free after the last barrier
#pragma unroll
    for (int a = 0; a < AM; ++a)
#pragma unroll
        for (int b = 0; b < AN; ++b)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row0 = (CONV ? WN * wn + 32 * b : WM * wm + 32 * a) + 8 * i + 4 * q;
                const int col = (CONV ? WM * wm + 32 * a : WN * wn + 32 * b) + l32;
                red[(row0 / 4) * COLSP + col] =
                    floatx4{acc[a][b][4 * i], acc[a][b][4 * i + 1], acc[a][b][4 * i + 2], acc[a][b][4 * i + 3]};
            }
    __syncthreads();
    const int ybytes = y_dtype == AQ_F32 ? 4 : 2;
    const __amdgpu_buffer_rsrc_t yr = buffer_rsrc(Y, (uint64_t)geo.tokens * geo.C_out * ybytes);
    const int plane = CONV ? geo.OH * geo.OW : 0;
    constexpr int TASKS = (ROWS / 4) * (COLS / 8);
    for (int task = tid; task < TASKS; task += 256) {
        const int c8 = (task / (ROWS / 4)) * 8;
        const int rq = task - (task / (ROWS / 4)) * (ROWS / 4);
        floatx4 v[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) v[c] = red[rq * COLSP + c8 + c];
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
        if (ncols <= 0 || rows_left <= 0) continue;
        // row scales (channel for a convolution, token for a linear layer) and column scales
        float rs[4], cs[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if constexpr (CONV) {
                const int co = min(N0 + 4 * rq + e, geo.C_out - 1);
                rs[e] = scales[co];
            } else {
                const int tok = min(T0 + 4 * rq + e, tokens - 1);
                rs[e] = x_scales ? x_scales[tok] : 1.0f;
            }
        }
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            if constexpr (CONV) cs[c] = 1.0f;
            else cs[c] = scales[min(col0 + c, geo.C_out - 1)];
        }
        if (ncols == 8 && aligned) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (e >= rows_left) break;
                int yi0;
                if constexpr (CONV) {
                    const int co = N0 + 4 * rq + e;
                    const int bimg = col0 / plane;
                    yi0 = (bimg * geo.C_out + co) * plane + (col0 - bimg * plane);
                } else {
                    yi0 = (T0 + 4 * rq + e) * geo.C_out + col0;
                }
                float o[8];
#pragma unroll
                for (int c = 0; c < 8; ++c) o[c] = v[c][e] * cs[c] * rs[e];
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
                    if constexpr (CONV) {
                        const int tk = col0 + c, bb = tk / plane;
                        yi = (bb * geo.C_out + N0 + 4 * rq + e) * plane + (tk - bb * plane);
                    } else {
                        yi = (T0 + 4 * rq + e) * geo.C_out + col0 + c;
                    }
                    const float o = v[c][e] * cs[c] * rs[e];
                    if (y_dtype == AQ_F32) __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(o), yr, yi * 4, 0, 0);
                    else __builtin_amdgcn_raw_buffer_store_b16(f32_to_f16(o), yr, yi * 2, 0, 0);
                }
        }
    }
}

template <int KIND, int XT, int BM, int BN>
static hipError_t rec_gemm_cfg(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl) {
    auto kern = rec_gemm_kernel<KIND, XT, BM, BN>;
    static size_t attr_bytes = 0;
    if (plan.lds_bytes > attr_bytes) {
        hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)plan.lds_bytes);
        if (e != hipSuccess) return e;
        attr_bytes = plan.lds_bytes;
    }
    const dim3 grid((unsigned)(((geo.tokens + BM - 1) / BM) * ((geo.C_out + BN - 1) / BN)));
    kern<<<grid, 256, plan.lds_bytes, fl.stream>>>(geo, plan, fl.crec, fl.scales, fl.X, fl.x_scales, fl.Y, fl.y_dtype);
    return hipGetLastError();
}

hipError_t launch_rec_gemm(const Geom& geo, const FusedPlan& p, const FusedLaunch& fl) {
#define AQ_G(K, XT, TBM, TBN) \
    if (p.bm == TBM && p.bn == TBN) return rec_gemm_cfg<K, XT, TBM, TBN>(geo, p, fl);
    if (p.kind == 1) {
        AQ_G(1, AQ_F16, 128, 128)
        AQ_G(1, AQ_F16, 128, 64)
        AQ_G(1, AQ_F16, 64, 128)
    } else if (p.kind == 2) {
        AQ_G(2, AQ_F16, 128, 128)
        AQ_G(2, AQ_F16, 128, 64)
        AQ_G(2, AQ_F16, 64, 128)
    } else if (fl.x_dtype == AQ_I8) {
        AQ_G(0, AQ_I8, 128, 128)
        AQ_G(0, AQ_I8, 128, 64)
        AQ_G(0, AQ_I8, 64, 128)
    } else {
        AQ_G(0, AQ_F16, 128, 128)
        AQ_G(0, AQ_F16, 128, 64)
        AQ_G(0, AQ_F16, 64, 128)
    }
#undef AQ_G
    return hipErrorInvalidConfiguration;
}

}  // namespace aq
