// Decode path of the AQ forward on gfx950 matrix cores.
//
// Per workgroup: a BM (tokens) x BN (output channels) tile of Y.  Each K step
// of 32 inputs (4 groups of g = 8) stages the activation tile in LDS (with
// implicit im2col for a convolution and int8 -> fp16 conversion for A8
// inputs) and expands the weight tile from its codes: each thread sums the M
// fp32 codewords of a group in ascending m and rounds once to the tile dtype
// (the per-channel scale is applied to the fp32 accumulator in the epilogue,
// which is algebraically the same product).  With fp16 codebooks and an fp16
// tile the codeword sum is accumulated in fp16 instead.  Four waves then contract the
// tiles with v_mfma_f32_32x32x16_{f16,bf16}; one lane's 8 operand values are
// exactly one decoded group.
#include <type_traits>

#include "aq_device.h"

namespace aq {

enum DecodeMode { DEC_LDS_F32 = 0, DEC_GLOBAL_F32 = 1, DEC_GLOBAL_TILE = 2 };

constexpr int kBK = 32;        // K per step: 4 groups of 8
constexpr int kLDT = kBK + 8;  // padded LDS row (16-bit elements), 80 bytes
constexpr int kThreads = 256;

template <int TILE>
__device__ __forceinline__ floatx16 mfma32(const u32x4& a, const u32x4& b, const floatx16& c) {
    if constexpr (TILE == AQ_F16)
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a), __builtin_bit_cast(half8, b), c, 0,
                                                      0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                       0, 0, 0);
}

__device__ __forceinline__ uint32_t pack2(uint16_t lo, uint16_t hi) { return (uint32_t)lo | ((uint32_t)hi << 16); }

template <int TILE>
__device__ __forceinline__ u32x4 pack8_f32(const float* v) {
    u32x4 r;
    r[0] = pack2(f32_to_tile<TILE>(v[0]), f32_to_tile<TILE>(v[1]));
    r[1] = pack2(f32_to_tile<TILE>(v[2]), f32_to_tile<TILE>(v[3]));
    r[2] = pack2(f32_to_tile<TILE>(v[4]), f32_to_tile<TILE>(v[5]));
    r[3] = pack2(f32_to_tile<TILE>(v[6]), f32_to_tile<TILE>(v[7]));
    return r;
}

// 8 consecutive activations X[tok][k..k+7] of a linear layer, as tile bits.
template <int XT, int TILE>
__device__ __forceinline__ u32x4 load_x8_linear(const void* X, int64_t off) {
    if constexpr (XT == TILE) {
        return *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(X) + off);
    } else {
        float v[8];
        if constexpr (XT == AQ_F32) {
            const floatx4* p = reinterpret_cast<const floatx4*>(static_cast<const float*>(X) + off);
            floatx4 a = p[0], b = p[1];
            v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
            v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
        } else if constexpr (XT == AQ_I8) {
            const uint64_t q = *reinterpret_cast<const uint64_t*>(static_cast<const int8_t*>(X) + off);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = (float)(int8_t)((q >> (8 * e)) & 0xff);
        } else {
            const u32x4 r = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(X) + off);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint16_t lo = (uint16_t)(r[e] & 0xffffu), hi = (uint16_t)(r[e] >> 16);
                v[2 * e] = (XT == AQ_F16) ? f16_to_f32(lo) : bf16_to_f32(lo);
                v[2 * e + 1] = (XT == AQ_F16) ? f16_to_f32(hi) : bf16_to_f32(hi);
            }
        }
        return pack8_f32<TILE>(v);
    }
}

template <int MODE, int XT, int TILE, bool CONV, int BM, int BN>
__global__ void __launch_bounds__(kThreads, 2)
mfma_fwd_kernel(Geom geo, const void* __restrict__ cbdev, const void* __restrict__ codes_v,
                const float* __restrict__ scales, const void* __restrict__ X, const float* __restrict__ x_scales,
                void* __restrict__ Y, int y_dtype, int acc16) {
    static_assert(BM % 64 == 0 && BN % 64 == 0, "tile must split into 2x2 waves of 32x32 blocks");
    constexpr int WM = BM / 2, WN = BN / 2;        // per-wave tile
    constexpr int AM = WM / 32, AN = WN / 32;      // 32x32 blocks per wave
    using CodeT = typename std::conditional<MODE == DEC_LDS_F32, uint8_t, uint16_t>::type;
    const CodeT* codes = static_cast<const CodeT*>(codes_v);

    __shared__ __attribute__((aligned(16))) uint16_t xs[BM * kLDT];
    __shared__ __attribute__((aligned(16))) uint16_t wsh[BN * kLDT];
    extern __shared__ floatx4 cb_lds[];            // DEC_LDS_F32: [M][2^B][8] fp32

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int64_t m0 = (int64_t)blockIdx.x * BM;
    const int n0 = blockIdx.y * BN;
    const int M = geo.M;
    const int nk = 1 << geo.B;

    if constexpr (MODE == DEC_LDS_F32) {
        const int n4 = (M * nk * 8) / 4;
        const floatx4* src = static_cast<const floatx4*>(cbdev);
        for (int i = tid; i < n4; i += kThreads) cb_lds[i] = src[i];
    }

    // Per-thread token bookkeeping for the implicit im2col loader.
    constexpr int KSLICES = kThreads / BM;          // conv: threads per token row
    constexpr int KPER = kBK / KSLICES;             // conv: k values per thread per step
    int conv_row = 0, conv_kslice = 0;
    int64_t conv_xbase = 0;
    int conv_ih0 = 0, conv_iw0 = 0;
    bool conv_valid = false;
    if constexpr (CONV) {
        conv_row = tid % BM;
        conv_kslice = tid / BM;
        const int64_t tok = m0 + conv_row;
        conv_valid = tok < geo.tokens;
        if (conv_valid) {
            const int64_t plane = (int64_t)geo.OH * geo.OW;
            const int64_t b = tok / plane;
            const int p = (int)(tok - b * plane);
            const int oh = p / geo.OW;
            const int ow = p - oh * geo.OW;
            conv_ih0 = oh * geo.stride - geo.pad;
            conv_iw0 = ow * geo.stride - geo.pad;
            conv_xbase = b * geo.cin * (int64_t)geo.H * geo.W;
        }
    }

    floatx16 acc[AM][AN];
#pragma unroll
    for (int a = 0; a < AM; ++a)
#pragma unroll
        for (int b = 0; b < AN; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

    constexpr int XCH = BM * (kBK / 8) / kThreads;  // linear: 8-element chunks per thread
    constexpr int WGR = BN * (kBK / 8) / kThreads;  // groups decoded per thread per step

    for (int k0 = 0; k0 < geo.K; k0 += kBK) {
        // ---- activations -> registers
        u32x4 xv[CONV ? KPER / 8 : XCH];
        if constexpr (!CONV) {
#pragma unroll
            for (int c = 0; c < XCH; ++c) {
                const int ch = tid + c * kThreads;
                const int row = ch >> 2;
                const int k = k0 + (ch & 3) * 8;
                const int64_t tok = m0 + row;
                if (tok < geo.tokens && k < geo.K) xv[c] = load_x8_linear<XT, TILE>(X, tok * geo.K + k);
                else xv[c] = u32x4{0u, 0u, 0u, 0u};
            }
        } else {
            const int khw = geo.kh * geo.kw;
            int k = k0 + conv_kslice * KPER;
            int c = k / khw;
            int rs = k - c * khw;
            int r = rs / geo.kw;
            int s = rs - r * geo.kw;
            float v[KPER];
#pragma unroll
            for (int e = 0; e < KPER; ++e) {
                float val = 0.0f;
                const int ih = conv_ih0 + r, iw = conv_iw0 + s;
                if (conv_valid && k + e < geo.K && ih >= 0 && ih < geo.H && iw >= 0 && iw < geo.W)
                    val = load_as_f32<XT>(X, conv_xbase + ((int64_t)c * geo.H + ih) * geo.W + iw);
                v[e] = val;
                if (++s == geo.kw) {
                    s = 0;
                    if (++r == geo.kh) { r = 0; ++c; }
                }
            }
#pragma unroll
            for (int q = 0; q < KPER / 8; ++q) xv[q] = pack8_f32<TILE>(v + 8 * q);
        }

        // ---- weights: decode WGR groups -> registers
        u32x4 wv[WGR];
#pragma unroll
        for (int q = 0; q < WGR; ++q) {
            const int gi = tid + q * kThreads;
            const int row = gi >> 2;
            const int j = (k0 >> 3) + (gi & 3);
            const int co = n0 + row;
            if (co < geo.C_out && j < geo.G) {
                const CodeT* bp = codes + ((int64_t)co * geo.G + j) * M;
                if constexpr (MODE == DEC_GLOBAL_TILE) {
                    wv[q] = static_cast<const u32x4*>(cbdev)[bp[0]];
                } else {
                    float sum[8];
                    const floatx4* cbv = (MODE == DEC_LDS_F32) ? cb_lds : static_cast<const floatx4*>(cbdev);
                    {
                        const floatx4* p = cbv + (int64_t)bp[0] * 2;
                        const floatx4 lo = p[0], hi = p[1];
                        sum[0] = lo[0]; sum[1] = lo[1]; sum[2] = lo[2]; sum[3] = lo[3];
                        sum[4] = hi[0]; sum[5] = hi[1]; sum[6] = hi[2]; sum[7] = hi[3];
                    }
                    for (int m = 1; m < M; ++m) {
                        const floatx4* p = cbv + ((int64_t)m * nk + bp[m]) * 2;
                        const floatx4 lo = p[0], hi = p[1];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            if (acc16) {   // fp16 codebooks and tile: fp16 accumulation
                                sum[e] = (float)((_Float16)sum[e] + (_Float16)lo[e]);
                                sum[4 + e] = (float)((_Float16)sum[4 + e] + (_Float16)hi[e]);
                            } else {
                                sum[e] = __fadd_rn(sum[e], lo[e]);
                                sum[4 + e] = __fadd_rn(sum[4 + e], hi[e]);
                            }
                        }
                    }
#pragma unroll
                    for (int e = 0; e < 8; ++e) sum[e] = opaque_f32(sum[e]);
                    wv[q] = pack8_f32<TILE>(sum);
                }
            } else {
                wv[q] = u32x4{0u, 0u, 0u, 0u};
            }
        }

        __syncthreads();   // previous step's MFMA reads are done
        if constexpr (!CONV) {
#pragma unroll
            for (int c = 0; c < XCH; ++c) {
                const int ch = tid + c * kThreads;
                *reinterpret_cast<u32x4*>(&xs[(ch >> 2) * kLDT + (ch & 3) * 8]) = xv[c];
            }
        } else {
#pragma unroll
            for (int q = 0; q < KPER / 8; ++q)
                *reinterpret_cast<u32x4*>(&xs[conv_row * kLDT + conv_kslice * KPER + 8 * q]) = xv[q];
        }
#pragma unroll
        for (int q = 0; q < WGR; ++q) {
            const int gi = tid + q * kThreads;
            *reinterpret_cast<u32x4*>(&wsh[(gi >> 2) * kLDT + (gi & 3) * 8]) = wv[q];
        }
        __syncthreads();

        // ---- contraction: two k16 sub-steps
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            const int kofs = kk * 16 + (lane >> 5) * 8;
            u32x4 fx[AM], fw[AN];
#pragma unroll
            for (int a = 0; a < AM; ++a)
                fx[a] = *reinterpret_cast<const u32x4*>(&xs[(wm * WM + a * 32 + (lane & 31)) * kLDT + kofs]);
#pragma unroll
            for (int b = 0; b < AN; ++b)
                fw[b] = *reinterpret_cast<const u32x4*>(&wsh[(wn * WN + b * 32 + (lane & 31)) * kLDT + kofs]);
#pragma unroll
            for (int a = 0; a < AM; ++a)
#pragma unroll
                for (int b = 0; b < AN; ++b) {
                    if constexpr (CONV) acc[a][b] = mfma32<TILE>(fw[b], fx[a], acc[a][b]);
                    else acc[a][b] = mfma32<TILE>(fx[a], fw[b], acc[a][b]);
                }
        }
    }

    // ---- epilogue: D row p / column q of each 32x32 block
    // (linear: p = token, q = channel; conv: p = channel, q = token)
#pragma unroll
    for (int a = 0; a < AM; ++a)
#pragma unroll
        for (int b = 0; b < AN; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int p = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                const int q = lane & 31;
                int64_t tok;
                int co;
                if constexpr (CONV) {
                    co = n0 + wn * WN + b * 32 + p;
                    tok = m0 + wm * WM + a * 32 + q;
                } else {
                    tok = m0 + wm * WM + a * 32 + p;
                    co = n0 + wn * WN + b * 32 + q;
                }
                if (tok < geo.tokens && co < geo.C_out) {
                    float v = acc[a][b][r] * scales[co];
                    if (x_scales) v *= x_scales[tok];
                    const int64_t yi = y_index(geo, tok, co);
                    if (y_dtype == AQ_F32) static_cast<float*>(Y)[yi] = v;
                    else static_cast<uint16_t*>(Y)[yi] = f32_to_f16(v);
                }
            }
}

template <int MODE, int XT, int TILE, bool CONV, int BM, int BN>
static hipError_t launch_cfg(const Geom& geo, const DeviceWeights& w, const void* cbdev, const void* X,
                             const float* x_scales, void* Y, int y_dtype, hipStream_t st) {
    auto kern = mfma_fwd_kernel<MODE, XT, TILE, CONV, BM, BN>;
    size_t dyn = 0;
    if constexpr (MODE == DEC_LDS_F32) {
        dyn = (size_t)geo.M * (1 << geo.B) * 8 * sizeof(float);
        hipError_t e = ensure_dynamic_lds((const void*)kern, dyn);
        if (e != hipSuccess) return e;
    }
    const dim3 grid((unsigned)((geo.tokens + BM - 1) / BM), (unsigned)((geo.C_out + BN - 1) / BN));
    const int acc16 = w.cb_dtype == AQ_F16 && TILE == AQ_F16;
    kern<<<grid, kThreads, dyn, st>>>(geo, cbdev, w.codes, w.scales, X, x_scales, Y, y_dtype, acc16);
    note_launch(st, "mfma_fwd_kernel", {MODE, XT, TILE, (int)CONV, BM, BN});
    return hipGetLastError();
}

template <int MODE, int XT, int TILE, bool CONV>
static hipError_t launch_tiles(const Geom& geo, const DeviceWeights& w, const void* cbdev, const void* X,
                               const float* x_scales, void* Y, int y_dtype, hipStream_t st) {
    auto tiles = [&](int bm, int bn) {
        return ((geo.tokens + bm - 1) / bm) * (int64_t)((geo.C_out + bn - 1) / bn);
    };
    if (tiles(128, 128) >= 256)
        return launch_cfg<MODE, XT, TILE, CONV, 128, 128>(geo, w, cbdev, X, x_scales, Y, y_dtype, st);
    if (tiles(128, 64) >= 256)
        return launch_cfg<MODE, XT, TILE, CONV, 128, 64>(geo, w, cbdev, X, x_scales, Y, y_dtype, st);
    return launch_cfg<MODE, XT, TILE, CONV, 64, 64>(geo, w, cbdev, X, x_scales, Y, y_dtype, st);
}

template <int XT, int TILE, bool CONV>
static hipError_t launch_mode(const Geom& geo, const DeviceWeights& w, const void* cb32, const void* cbtile,
                              const void* X, const float* x_scales, void* Y, int y_dtype, hipStream_t st) {
    if (geo.B <= 8) return launch_tiles<DEC_LDS_F32, XT, TILE, CONV>(geo, w, cb32, X, x_scales, Y, y_dtype, st);
    if (geo.M == 1) return launch_tiles<DEC_GLOBAL_TILE, XT, TILE, CONV>(geo, w, cbtile, X, x_scales, Y, y_dtype, st);
    return launch_tiles<DEC_GLOBAL_F32, XT, TILE, CONV>(geo, w, cb32, X, x_scales, Y, y_dtype, st);
}

template <int TILE>
static hipError_t launch_tile_dtype(const Geom& geo, const DeviceWeights& w, const void* cb32, const void* cbtile,
                                    const void* X, int x_dtype, const float* x_scales, void* Y, int y_dtype,
                                    hipStream_t st) {
    if (geo.conv) {
        switch (x_dtype) {
        case AQ_F32: return launch_mode<AQ_F32, TILE, true>(geo, w, cb32, cbtile, X, x_scales, Y, y_dtype, st);
        case AQ_F16: return launch_mode<AQ_F16, TILE, true>(geo, w, cb32, cbtile, X, x_scales, Y, y_dtype, st);
        default: return launch_mode<AQ_BF16, TILE, true>(geo, w, cb32, cbtile, X, x_scales, Y, y_dtype, st);
        }
    }
    switch (x_dtype) {
    case AQ_F32: return launch_mode<AQ_F32, TILE, false>(geo, w, cb32, cbtile, X, x_scales, Y, y_dtype, st);
    case AQ_F16: return launch_mode<AQ_F16, TILE, false>(geo, w, cb32, cbtile, X, x_scales, Y, y_dtype, st);
    case AQ_BF16: return launch_mode<AQ_BF16, TILE, false>(geo, w, cb32, cbtile, X, x_scales, Y, y_dtype, st);
    default: return launch_mode<AQ_I8, TILE, false>(geo, w, cb32, cbtile, X, x_scales, Y, y_dtype, st);
    }
}

hipError_t launch_mfma_forward(const Geom& geo, const DeviceWeights& w, const void* X, int x_dtype,
                               const float* x_scales, void* Y, int y_dtype, int tile_dtype, hipStream_t stream) {
    if (tile_dtype == AQ_F16)
        return launch_tile_dtype<AQ_F16>(geo, w, w.cb32, w.cbtile, X, x_dtype, x_scales, Y, y_dtype, stream);
    return launch_tile_dtype<AQ_BF16>(geo, w, w.cb32, w.cbtile, X, x_dtype, x_scales, Y, y_dtype, stream);
}

// ---- create-time codebook preparation ----

template <int CBT>
__global__ void codebook_prep_kernel(const void* __restrict__ cb, int64_t n, float* __restrict__ cb32,
                                     uint16_t* __restrict__ cbtile, int tile_dtype) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float v = load_as_f32<CBT>(cb, i);
    cb32[i] = v;
    if (cbtile) cbtile[i] = (tile_dtype == AQ_BF16) ? f32_to_bf16(v) : f32_to_f16(v);
}

hipError_t launch_codebook_prep(const void* cb, int cb_dtype, int64_t n, float* cb32, void* cbtile, int tile_dtype,
                                hipStream_t stream) {
    const dim3 grid((unsigned)((n + 255) / 256));
    uint16_t* ct = static_cast<uint16_t*>(cbtile);
    switch (cb_dtype) {
    case AQ_F32: codebook_prep_kernel<AQ_F32><<<grid, 256, 0, stream>>>(cb, n, cb32, ct, tile_dtype); break;
    case AQ_F16: codebook_prep_kernel<AQ_F16><<<grid, 256, 0, stream>>>(cb, n, cb32, ct, tile_dtype); break;
    default: codebook_prep_kernel<AQ_BF16><<<grid, 256, 0, stream>>>(cb, n, cb32, ct, tile_dtype); break;
    }
    return hipGetLastError();
}

}  // namespace aq
