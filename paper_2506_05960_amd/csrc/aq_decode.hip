// Decode-to-global: writes the dense weight matrix W [C_out][K] in the tile
// dtype.  Test hook for bit-exact checks of the decode arithmetic used by the
// matrix-core paths: the codewords are summed in ascending m (in fp16 when
// both the codebook and the tile are fp16, else in fp32), multiplied by the
// channel scale in fp32 and rounded once to the tile dtype.
#include "aq_device.h"

namespace aq {

template <int CBT, typename CodeT, int TILE>
__global__ void __launch_bounds__(256)
decode_to_global_kernel(const void* __restrict__ cb, const CodeT* __restrict__ codes,
                        const float* __restrict__ scales, void* __restrict__ W, int C_out, int G, int g, int M,
                        int B) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // (row, group)
    if (idx >= (int64_t)C_out * G) return;
    const int i = (int)(idx / G);
    const int j = (int)(idx - (int64_t)i * G);
    const CodeT* b = codes + idx * M;
    const float s = scales[i];
    const int64_t rows = (int64_t)1 << B;
    const int64_t K = (int64_t)G * g;
    for (int t = 0; t < g; ++t) {
        float acc;
        if constexpr (CBT == AQ_F16 && TILE == AQ_F16) {
            // fp16 codebooks, fp16 tile: accumulate in fp16, ascending m
            _Float16 h = (_Float16)load_as_f32<CBT>(cb, (int64_t)b[0] * g + t);
            for (int m = 1; m < M; ++m) h = h + (_Float16)load_as_f32<CBT>(cb, ((int64_t)m * rows + b[m]) * g + t);
            acc = (float)h;
        } else {
            acc = load_as_f32<CBT>(cb, (int64_t)b[0] * g + t);
            for (int m = 1; m < M; ++m)
                acc = __fadd_rn(acc, load_as_f32<CBT>(cb, ((int64_t)m * rows + b[m]) * g + t));
        }
        acc = opaque_f32(__fmul_rn(acc, s));
        const int64_t o = (int64_t)i * K + (int64_t)j * g + t;
        if constexpr (TILE == AQ_F32) static_cast<float*>(W)[o] = acc;
        else static_cast<uint16_t*>(W)[o] = f32_to_tile<TILE>(acc);
    }
}

template <int CBT, typename CodeT>
static hipError_t decode_dispatch_tile(const Geom& geo, const DeviceWeights& w, int tile, void* W,
                                       hipStream_t st) {
    const int64_t n = (int64_t)geo.C_out * geo.G;
    const dim3 grid((unsigned)((n + 255) / 256)), block(256);
    const CodeT* codes = static_cast<const CodeT*>(w.codes);
    switch (tile) {
    case AQ_F32:
        decode_to_global_kernel<CBT, CodeT, AQ_F32><<<grid, block, 0, st>>>(w.codebooks, codes, w.scales, W, geo.C_out,
                                                                             geo.G, geo.g, geo.M, geo.B);
        break;
    case AQ_F16:
        decode_to_global_kernel<CBT, CodeT, AQ_F16><<<grid, block, 0, st>>>(w.codebooks, codes, w.scales, W, geo.C_out,
                                                                             geo.G, geo.g, geo.M, geo.B);
        break;
    default:
        decode_to_global_kernel<CBT, CodeT, AQ_BF16><<<grid, block, 0, st>>>(w.codebooks, codes, w.scales, W,
                                                                              geo.C_out, geo.G, geo.g, geo.M, geo.B);
        break;
    }
    return hipGetLastError();
}

template <typename CodeT>
static hipError_t decode_dispatch_cb(const Geom& geo, const DeviceWeights& w, int tile, void* W, hipStream_t st) {
    switch (w.cb_dtype) {
    case AQ_F32: return decode_dispatch_tile<AQ_F32, CodeT>(geo, w, tile, W, st);
    case AQ_F16: return decode_dispatch_tile<AQ_F16, CodeT>(geo, w, tile, W, st);
    default: return decode_dispatch_tile<AQ_BF16, CodeT>(geo, w, tile, W, st);
    }
}

hipError_t launch_decode_to_global(const Geom& geo, const DeviceWeights& w, int tile_dtype, void* W,
                                   hipStream_t stream) {
    if (geo.B <= 8) return decode_dispatch_cb<uint8_t>(geo, w, tile_dtype, W, stream);
    return decode_dispatch_cb<uint16_t>(geo, w, tile_dtype, W, stream);
}

}  // namespace aq
