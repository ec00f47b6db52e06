// Matrix-core forward over pre-decoded operand records (the decompress-then-
// compute route; Sec. 4.4 describes decompressing the weights before the
// dense product).  The records are the B operands of v_mfma_f32_32x32x16_f16
// exactly as the fused kernel would decode them (`operand_records_kernel`),
// so this kernel is a dense fp16 implicit-im2col product:
//
//  * A workgroup of 4 waves owns a BM (tokens) x BN (output channels) tile;
//    the waves sit 2 x 2 on it, each accumulating a (BM/2) x (BN/2) quarter.
//  * K is walked in the fused kernel's chunks (16 input channels x 9 kernel
//    positions for a 3x3 convolution, 64 consecutive k otherwise).  Each
//    chunk's activations and weight records reach LDS through direct-to-LDS
//    loads (lane l of a wave fills slot base + l): no registers, no staging
//    arithmetic.  Three LDS stages keep two chunks in flight; every thread
//    issues the same number of loads per chunk (slots with nothing to load
//    read a zero block), so one vmcnt wait retires exactly one chunk.
//  * Activations come in channel-interleaved fp16: a convolution's input is
//    repacked per forward to [n][C/8][H][W][8] (`act_pack_conv_kernel`), an
//    int8 token matrix is widened to fp16, an fp16 one is read in place.  A
//    convolution stages every input row its tile touches once per image
//    (kernel rows become LDS offsets), zero outside the image.
//  * No partial tiles to combine; the tile passes through LDS once so that
//    the stores are 16-byte row segments.
#include "aq_fused_kernel.h"

namespace aq {

struct GemmArgs {
    const uint8_t* recs;       // operand records [chunk][step][C_out][2] x 16 B
    const uint8_t* xa;         // activations: packed conv input / fp16 tokens [T][K]
    const uint8_t* zero;       // 16 zero bytes
    const float* scales;
    const float* x_scales;
    void* Y;
    int y_dtype;
    int ni, rpi, pw;           // convolution staging: image slots, rows per slot, padded row width
    uint32_t cstride;          // bytes between consecutive chunks of activations
};

constexpr int kGemmStages = 3;


template <int KIND, int XT, int BM, int BN>
__global__ void __launch_bounds__(256, 1)
rec_gemm_kernel(Geom geo, FusedPlan plan, GemmArgs ga) {
    constexpr bool CONV = KIND != 0;
    constexpr int KH = KIND == 1 ? 3 : 1;
    constexpr int NS = KIND == 1 ? 9 : 4;            // MFMA steps per chunk
    constexpr int WM = BM / 2, WN = BN / 2;          // a wave's quarter
    constexpr int AM = WM / 32, AN = WN / 32;
    constexpr int ACT_T = CONV ? 4 : 5;              // activation slots per thread per chunk
    constexpr int BREC = NS * BN * 2;                // 16-byte weight records per chunk
    constexpr int WREC_T = (BREC + 255) / 256;       // weight slots per thread per chunk
    constexpr int ASLOTS = ACT_T * 256;
    constexpr int STAGE = (ASLOTS + WREC_T * 256) * 16;
    constexpr int LOADS = ACT_T + WREC_T;            // direct-to-LDS loads per thread per chunk
    constexpr int LPS = BM + 1;                      // linear: slots per plane (one spare)

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

    // ---- activation slots: this thread's slots z = tid + 256 j of a stage ----
    // convolution: z = ((o * ni + i) * rpi + rr) * pw + pc  (plane o of 8 channels, image
    // slot i, staged row rr, padded column pc); linear: z = o * (BM + 1) + tt (plane o of
    // 8 consecutive k, token tt; tt == BM is a spare slot)
    uint32_t aoff[ACT_T];        // byte offset of chunk 0's source
    bool aok[ACT_T];
    int ako[ACT_T];              // linear: first k of the slot within its chunk (bounds the last chunk)
    int gr0 = 0, b0 = 0;
    if constexpr (CONV) {
        gr0 = T0 / geo.OW;
        b0 = gr0 / geo.OH;
    }
#pragma unroll
    for (int j = 0; j < ACT_T; ++j) {
        const int z = tid + 256 * j;
        aok[j] = false;
        aoff[j] = 0;
        ako[j] = 0;
        if constexpr (CONV) {
            const int pc = z % ga.pw;
            const int t1 = z / ga.pw;
            const int rr = t1 % ga.rpi;
            const int t2 = t1 / ga.rpi;
            const int i = t2 % ga.ni;
            const int o = t2 / ga.ni;
            const int b = b0 + i;
            const int oh_first = i == 0 ? gr0 - b0 * geo.OH : 0;
            const int ih = oh_first * geo.stride - geo.pad + rr;
            const int iw = pc - geo.pad;
            const int nimg = (int)(geo.tokens / ((int64_t)geo.OH * geo.OW));
            aok[j] = o < (KIND == 1 ? 2 : 8) && b < nimg && ih >= 0 && ih < geo.H && iw >= 0 && iw < geo.W;
            if (aok[j])
                aoff[j] = ((((uint32_t)b * (uint32_t)(geo.cin / 8) + (uint32_t)o) * (uint32_t)geo.H + (uint32_t)ih) *
                               (uint32_t)geo.W + (uint32_t)iw) * 16u;
        } else {
            const int o = z / LPS;
            const int tt = z - o * LPS;
            const int T = T0 + tt;
            aok[j] = o < 8 && tt < BM && T < tokens;
            ako[j] = 8 * o;
            if (aok[j]) aoff[j] = ((uint32_t)T * (uint32_t)geo.K + 8u * (uint32_t)o) * 2u;
        }
    }
    // A-fragment base of each of the wave's token blocks (plane q of the step)
    uint32_t a_base[AM];
#pragma unroll
    for (int a = 0; a < AM; ++a) {
        const int T = T0 + WM * wm + 32 * a + l32;
        if constexpr (CONV) {
            const int gr = T / geo.OW;
            const int ow = T - gr * geo.OW;
            const int b = gr / geo.OH;
            const int oh = gr - b * geo.OH;
            const int i = min(b - b0, ga.ni - 1);        // tokens past the end: any slot, never stored
            const int oh_first = i == 0 ? gr0 - b0 * geo.OH : 0;
            const int rr = min(max(oh - oh_first, 0) * geo.stride, ga.rpi - KH);
            a_base[a] = (uint32_t)((((q * ga.ni + i) * ga.rpi + rr) * ga.pw + ow * geo.stride) * 16);
        } else {
            a_base[a] = (uint32_t)((q * LPS + WM * wm + 32 * a + l32) * 16);
        }
    }

    // ---- one chunk's direct-to-LDS loads ----
    auto issue = [&](int chunk, uint8_t* stg) {
        const uint32_t cshift = (uint32_t)chunk * ga.cstride;
#pragma unroll
        for (int j = 0; j < ACT_T; ++j) {
            bool ok = aok[j];
            if constexpr (!CONV) ok = ok && 64 * chunk + ako[j] < geo.K;   // K need not be a multiple of 64
            const uint8_t* src = ok ? ga.xa + aoff[j] + cshift : ga.zero;
            lds_dma16(src, stg + (size_t)(256 * j + 64 * wave) * 16);
        }
        uint8_t* wdst = stg + ASLOTS * 16;
#pragma unroll
        for (int i = 0; i < WREC_T; ++i) {
            // LDS slot e = (s * 2 + h) * BN + n holds record (chunk, s, N0 + n, h); channels
            // past C_out read a valid record whose products are never stored
            const int e = 256 * i + tid;
            const int sh = e / BN;
            const int n = e - sh * BN;
            const int st = sh >> 1, h = sh & 1;
            const int nc = min(N0 + n, geo.C_out - 1);
            const uint8_t* src = e < BREC ? ga.recs + ((size_t)((chunk * NS + st) * geo.C_out + nc) * 2 + h) * 16
                                          : ga.zero;
            lds_dma16(src, wdst + (size_t)(256 * i + 64 * wave) * 16);
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
        const u32x4* wl = reinterpret_cast<const u32x4*>(cur + ASLOTS * 16);
        uint32_t soff;
        if constexpr (KIND == 1) soff = (uint32_t)(((s / 3) * ga.pw + (s % 3)) * 16);
        else if constexpr (CONV) soff = (uint32_t)(2 * s * ga.ni * ga.rpi * ga.pw * 16);
        else soff = (uint32_t)(2 * s * LPS * 16);
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

    // ---- main loop: chunk c computes from stage c % 3 while chunks c + 1 and c + 2 land ----
    const int nch = plan.nchunk;
    auto stg = [&](int c) { return lds + (size_t)(c % kGemmStages) * STAGE; };
    if (nch > 0) issue(0, stg(0));
    if (nch > 1) issue(1, stg(1));
    if (nch > 1) wait_vmcnt<LOADS>();                // chunk 0 landed (chunk 1 may be in flight)
    else wait_vmcnt<0>();
    lds_barrier();
    for (int chunk = 0; chunk < nch; ++chunk) {
        if (chunk + 2 < nch) issue(chunk + 2, stg(chunk + 2));
        compute(stg(chunk));
        if (chunk + 2 < nch) wait_vmcnt<LOADS>();    // chunk + 1 landed
        else wait_vmcnt<0>();
        lds_barrier();
    }

    const float* scales = ga.scales;
    const float* x_scales = ga.x_scales;
    void* Y = ga.Y;
    const int y_dtype = ga.y_dtype;
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
static hipError_t rec_gemm_cfg(const Geom& geo, const FusedPlan& plan, const GemmArgs& ga, hipStream_t st) {
    auto kern = rec_gemm_kernel<KIND, XT, BM, BN>;
    hipError_t e = ensure_dynamic_lds((const void*)kern, plan.lds_bytes);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)(((geo.tokens + BM - 1) / BM) * ((geo.C_out + BN - 1) / BN)));
    kern<<<grid, 256, plan.lds_bytes, st>>>(geo, plan, ga);
    note_launch(st, "rec_gemm_kernel", {KIND, XT, BM, BN});
    return hipGetLastError();
}

// LDS bytes of a tile: three stages (activation and weight slots) or the epilogue's tile
size_t rec_gemm_lds_bytes(int kind, int bm, int bn) {
    const int act_t = kind != 0 ? 4 : 5;
    const int ns = kind == 1 ? 9 : 4;
    const int wrec_t = (ns * bn * 2 + 255) / 256;
    const size_t stage = (size_t)(act_t * 256 + wrec_t * 256) * 16;
    const size_t rows = kind != 0 ? bn : bm, cols = kind != 0 ? bm : bn;
    const size_t red = (rows / 4) * (cols + 1) * 16;
    return std::max<size_t>(kGemmStages * stage, red);
}

// Repack an NCHW fp16 input to [n][C/8][H][W][8] (one thread per pixel and 8 channels).
__global__ void __launch_bounds__(256)
act_pack_conv_kernel(const uint16_t* __restrict__ x, u32x4* __restrict__ out, int nimg, int C, int H, int W) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t hw = (int64_t)H * W;
    const int64_t total = (int64_t)nimg * (C / 8) * hw;
    if (idx >= total) return;
    const int64_t p = idx % hw;
    const int64_t nc8 = idx / hw;                    // n * C/8 + cblk
    const int64_t src0 = nc8 * 8 * hw + p;           // channel 8 cblk of image n
    u32x4 v;
#pragma unroll
    for (int d = 0; d < 4; ++d)
        v[d] = (uint32_t)x[src0 + (2 * d) * hw] | ((uint32_t)x[src0 + (2 * d + 1) * hw] << 16);
    out[idx] = v;
}

// Widen an int8 token matrix to fp16 (exact), 8 values per thread.
__global__ void __launch_bounds__(256)
act_widen_i8_kernel(const uint64_t* __restrict__ x, u32x4* __restrict__ out, int64_t n8) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= n8) return;
    out[idx] = i8x8_to_f16(x[idx]);
}

hipError_t launch_rec_gemm(const Geom& geo, const FusedPlan& p, const FusedLaunch& fl, void* xpack,
                           const void* zero) {
    GemmArgs ga;
    ga.recs = fl.crec;
    ga.zero = static_cast<const uint8_t*>(zero);
    ga.scales = fl.scales;
    ga.x_scales = fl.x_scales;
    ga.Y = fl.Y;
    ga.y_dtype = fl.y_dtype;
    ga.ni = p.pr;              // the planner keeps the staging geometry in pr / ps / pw
    ga.rpi = p.ps;
    ga.pw = p.pw;
    hipStream_t st = fl.stream;
    if (p.kind != 0) {
        const int nimg = (int)(geo.tokens / ((int64_t)geo.OH * geo.OW));
        const int64_t total = (int64_t)nimg * (geo.cin / 8) * geo.H * geo.W;
        act_pack_conv_kernel<<<(unsigned)((total + 255) / 256), 256, 0, st>>>(
            static_cast<const uint16_t*>(fl.X), static_cast<u32x4*>(xpack), nimg, geo.cin, geo.H, geo.W);
        note_launch(st, "act_pack_conv_kernel", {});
        ga.xa = static_cast<const uint8_t*>(xpack);
        ga.cstride = (uint32_t)((p.kind == 1 ? 2 : 8) * geo.H * geo.W * 16);   // the chunk's 8-channel planes
    } else if (fl.x_dtype == AQ_I8) {
        const int64_t n8 = geo.tokens * geo.K / 8;
        act_widen_i8_kernel<<<(unsigned)((n8 + 255) / 256), 256, 0, st>>>(static_cast<const uint64_t*>(fl.X),
                                                                           static_cast<u32x4*>(xpack), n8);
        note_launch(st, "act_widen_i8_kernel", {});
        ga.xa = static_cast<const uint8_t*>(xpack);
        ga.cstride = 64 * 2;
    } else {
        ga.xa = static_cast<const uint8_t*>(fl.X);
        ga.cstride = 64 * 2;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
#define AQ_G(K, XT, TBM, TBN) \
    if (p.bm == TBM && p.bn == TBN) return rec_gemm_cfg<K, XT, TBM, TBN>(geo, p, ga, st);
    if (p.kind == 1) {
        AQ_G(1, AQ_F16, 128, 128)
        AQ_G(1, AQ_F16, 128, 64)
        AQ_G(1, AQ_F16, 64, 128)
    } else if (p.kind == 2) {
        AQ_G(2, AQ_F16, 128, 128)
        AQ_G(2, AQ_F16, 128, 64)
        AQ_G(2, AQ_F16, 64, 128)
    } else {
        AQ_G(0, AQ_F16, 128, 128)
        AQ_G(0, AQ_F16, 128, 64)
        AQ_G(0, AQ_F16, 64, 128)
    }
#undef AQ_G
    return hipErrorInvalidConfiguration;
}

}  // namespace aq
