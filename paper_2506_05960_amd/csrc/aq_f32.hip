// fp32 decode path: weight tiles are expanded from codes into LDS in fp32
// (any group size g) and contracted with fp32 FMAs.  Serves layers whose
// tile dtype is fp32, where the matrix-core fp16/bf16 rounding of the weight
// tile is not wanted.
#include "aq_device.h"

namespace aq {

constexpr int kF32BM = 64, kF32BN = 64, kF32BK = 16;

template <int XT, typename CodeT>
__global__ void __launch_bounds__(256)
f32_fwd_kernel(Geom geo, const float* __restrict__ cb32, const CodeT* __restrict__ codes,
               const float* __restrict__ scales, const void* __restrict__ X, const float* __restrict__ x_scales,
               void* __restrict__ Y, int y_dtype) {
    __shared__ float xs[kF32BK][kF32BM + 4];
    __shared__ float wsh[kF32BK][kF32BN + 4];
    const int tid = threadIdx.x;
    const int tx = tid & 15, ty = tid >> 4;
    const int64_t m0 = (int64_t)blockIdx.x * kF32BM;
    const int n0 = blockIdx.y * kF32BN;
    const int g = geo.g, M = geo.M;
    const int64_t nk = (int64_t)1 << geo.B;
    float acc[4][4] = {};

    for (int k0 = 0; k0 < geo.K; k0 += kF32BK) {
        // 64 x 16 activations and 64 x 16 decoded weights, 4 of each per thread
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = tid + q * 256;
            const int row = e & 63;
            const int kk = e >> 6;
            const int k = k0 + kk;
            const int64_t tok = m0 + row;
            xs[kk][row] = (tok < geo.tokens && k < geo.K) ? x_elem<XT>(geo, X, tok, k) : 0.0f;
            const int co = n0 + row;
            float w = 0.0f;
            if (co < geo.C_out && k < geo.K) {
                const int j = k / g;
                const int t = k - j * g;
                const CodeT* bp = codes + ((int64_t)co * geo.G + j) * M;
                w = cb32[(int64_t)bp[0] * g + t];
                for (int m = 1; m < M; ++m) w = __fadd_rn(w, cb32[((int64_t)m * nk + bp[m]) * g + t]);
            }
            wsh[kk][row] = w;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < kF32BK; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                a[i] = xs[kk][ty * 4 + i];
                b[i] = wsh[kk][tx * 4 + i];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) acc[i][jj] = fmaf(a[i], b[jj], acc[i][jj]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t tok = m0 + ty * 4 + i;
        if (tok >= geo.tokens) continue;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int co = n0 + tx * 4 + jj;
            if (co >= geo.C_out) continue;
            float v = acc[i][jj] * scales[co];
            if (x_scales) v *= x_scales[tok];
            const int64_t yi = y_index(geo, tok, co);
            if (y_dtype == AQ_F32) static_cast<float*>(Y)[yi] = v;
            else static_cast<uint16_t*>(Y)[yi] = f32_to_f16(v);
        }
    }
}

template <typename CodeT>
static hipError_t f32_launch_codes(const Geom& geo, const DeviceWeights& w, const void* X, int x_dtype,
                                   const float* x_scales, void* Y, int y_dtype, hipStream_t st) {
    const dim3 grid((unsigned)((geo.tokens + kF32BM - 1) / kF32BM), (unsigned)((geo.C_out + kF32BN - 1) / kF32BN));
    const CodeT* codes = static_cast<const CodeT*>(w.codes);
    switch (x_dtype) {
    case AQ_F32: f32_fwd_kernel<AQ_F32, CodeT><<<grid, 256, 0, st>>>(geo, w.cb32, codes, w.scales, X, x_scales, Y, y_dtype); break;
    case AQ_F16: f32_fwd_kernel<AQ_F16, CodeT><<<grid, 256, 0, st>>>(geo, w.cb32, codes, w.scales, X, x_scales, Y, y_dtype); break;
    case AQ_BF16: f32_fwd_kernel<AQ_BF16, CodeT><<<grid, 256, 0, st>>>(geo, w.cb32, codes, w.scales, X, x_scales, Y, y_dtype); break;
    default: f32_fwd_kernel<AQ_I8, CodeT><<<grid, 256, 0, st>>>(geo, w.cb32, codes, w.scales, X, x_scales, Y, y_dtype); break;
    }
    note_launch(st, "f32_fwd_kernel", {x_dtype, 8 * (int)sizeof(CodeT)});
    return hipGetLastError();
}

hipError_t launch_f32_forward(const Geom& geo, const DeviceWeights& w, const void* X, int x_dtype,
                              const float* x_scales, void* Y, int y_dtype, hipStream_t stream) {
    if (geo.B <= 8) return f32_launch_codes<uint8_t>(geo, w, X, x_dtype, x_scales, Y, y_dtype, stream);
    return f32_launch_codes<uint16_t>(geo, w, X, x_dtype, x_scales, Y, y_dtype, stream);
}

}  // namespace aq
