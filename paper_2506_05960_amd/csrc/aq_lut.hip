// LUT path of the AQ forward (paper appendix, eq. (12)): for a tile of tokens
// and a chunk of weight groups, tabulate every codeword's dot product with
// the tokens' input slice in LDS, then accumulate, for each output channel,
// the table entries its codes select.  Partial sums per group chunk go to a
// workspace and a second kernel reduces them in a fixed order, applies the
// per-channel (and per-token) scales and stores Y.
#include "aq_device.h"

namespace aq {

// One workgroup: group chunk blockIdx.x, token tile blockIdx.y (4 tokens).
// LDS: LUT [jc*M][2^B] of floatx4 (one value per token), then x [4][jc*g].
template <int CBT, int XT>
__global__ void __launch_bounds__(256)
lut_gather_kernel(Geom geo, const void* __restrict__ cb, const uint8_t* __restrict__ codes_lut, int jc,
                  const void* __restrict__ X, int64_t tok0, int ntok, int tok_block, float* __restrict__ ws) {
    extern __shared__ floatx4 lds_lut[];
    const int chunk = blockIdx.x;
    const int tile = blockIdx.y;
    const int g = geo.g, M = geo.M;
    const int nk = 1 << geo.B;
    const int nent = jc * M * nk;
    const int kspan = jc * g;
    float* xs = reinterpret_cast<float*>(lds_lut + nent);
    const int k_base = chunk * kspan;

    for (int e = threadIdx.x; e < kLutTokTile * kspan; e += blockDim.x) {
        const int n = e / kspan;
        const int kk = e - n * kspan;
        const int tok = tile * kLutTokTile + n;
        const int k = k_base + kk;
        float v = 0.0f;
        if (tok < ntok && k < geo.K) v = x_elem<XT>(geo, X, tok0 + tok, k);
        xs[e] = v;
    }
    __syncthreads();

    for (int e = threadIdx.x; e < nent; e += blockDim.x) {
        const int k = e % nk;
        const int jm = e / nk;
        const int m = jm % M;
        const int jj = jm / M;
        const int64_t cbase = ((int64_t)m * nk + k) * g;
        const float* x0 = xs + jj * g;
        floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
        for (int t = 0; t < g; ++t) {
            const float c = load_as_f32<CBT>(cb, cbase + t);
            acc[0] = fmaf(x0[t], c, acc[0]);
            acc[1] = fmaf(x0[kspan + t], c, acc[1]);
            acc[2] = fmaf(x0[2 * kspan + t], c, acc[2]);
            acc[3] = fmaf(x0[3 * kspan + t], c, acc[3]);
        }
        lds_lut[e] = acc;
    }
    __syncthreads();

    const int rowbytes = jc * M;
    const uint8_t* cbase = codes_lut + (int64_t)chunk * geo.C_out * rowbytes;
    for (int i = threadIdx.x; i < geo.C_out; i += blockDim.x) {
        const uint8_t* b = cbase + (int64_t)i * rowbytes;
        floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
        for (int jm = 0; jm < rowbytes; ++jm) acc += lds_lut[jm * nk + b[jm]];
        for (int n = 0; n < kLutTokTile; ++n) {
            const int tok = tile * kLutTokTile + n;
            if (tok < ntok) ws[((int64_t)chunk * tok_block + tok) * geo.C_out + i] = acc[n];
        }
    }
}

// Fixed-order reduction over group chunks, scales, dtype cast and store.
template <int YT>
__global__ void __launch_bounds__(256)
lut_reduce_kernel(Geom geo, const float* __restrict__ ws, int nchunk, int tok_block, int64_t tok0, int ntok,
                  const float* __restrict__ scales, const float* __restrict__ x_scales, void* __restrict__ Y) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)ntok * geo.C_out) return;
    const int tok = (int)(idx / geo.C_out);
    const int i = (int)(idx - (int64_t)tok * geo.C_out);
    float acc = 0.0f;
    for (int c = 0; c < nchunk; ++c) acc += ws[((int64_t)c * tok_block + tok) * geo.C_out + i];
    float v = acc * scales[i];
    if (x_scales) v *= x_scales[tok0 + tok];
    store_y<YT>(Y, y_index(geo, tok0 + tok, i), v);
}

template <int CBT, int XT>
static void launch_gather(const Geom& geo, const DeviceWeights& w, const LutPlan& plan, const void* X,
                          int64_t tok0, int ntok, float* ws, hipStream_t st) {
    const int nent = plan.jc * geo.M * (1 << geo.B);
    const size_t lds = (size_t)nent * sizeof(floatx4) + (size_t)kLutTokTile * plan.jc * geo.g * sizeof(float);
    const dim3 grid(plan.nchunk, (ntok + kLutTokTile - 1) / kLutTokTile);
    static size_t attr_bytes = 64 * 1024;
    if (lds > attr_bytes) {
        if (hipFuncSetAttribute((const void*)lut_gather_kernel<CBT, XT>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)lds) != hipSuccess)
            return;
        attr_bytes = lds;
    }
    lut_gather_kernel<CBT, XT><<<grid, 256, lds, st>>>(geo, w.codebooks, w.codes_lut, plan.jc, X, tok0, ntok,
                                                       plan.tok_block, ws);
}

template <int CBT>
static void launch_gather_x(int x_dtype, const Geom& geo, const DeviceWeights& w, const LutPlan& plan,
                            const void* X, int64_t tok0, int ntok, float* ws, hipStream_t st) {
    switch (x_dtype) {
    case AQ_F32: launch_gather<CBT, AQ_F32>(geo, w, plan, X, tok0, ntok, ws, st); break;
    case AQ_F16: launch_gather<CBT, AQ_F16>(geo, w, plan, X, tok0, ntok, ws, st); break;
    case AQ_BF16: launch_gather<CBT, AQ_BF16>(geo, w, plan, X, tok0, ntok, ws, st); break;
    default: launch_gather<CBT, AQ_I8>(geo, w, plan, X, tok0, ntok, ws, st); break;
    }
}

size_t lut_lds_bytes(const Geom& geo, const LutPlan& plan) {
    return (size_t)plan.jc * geo.M * (1 << geo.B) * sizeof(floatx4) +
           (size_t)kLutTokTile * plan.jc * geo.g * sizeof(float);
}

hipError_t launch_lut_forward(const Geom& geo, const DeviceWeights& w, const LutPlan& plan, const void* X,
                              int x_dtype, const float* x_scales, void* Y, int y_dtype, float* ws,
                              hipStream_t stream) {
    for (int64_t tok0 = 0; tok0 < geo.tokens; tok0 += plan.tok_block) {
        const int ntok = (int)((geo.tokens - tok0 < plan.tok_block) ? geo.tokens - tok0 : plan.tok_block);
        switch (w.cb_dtype) {
        case AQ_F32: launch_gather_x<AQ_F32>(x_dtype, geo, w, plan, X, tok0, ntok, ws, stream); break;
        case AQ_F16: launch_gather_x<AQ_F16>(x_dtype, geo, w, plan, X, tok0, ntok, ws, stream); break;
        default: launch_gather_x<AQ_BF16>(x_dtype, geo, w, plan, X, tok0, ntok, ws, stream); break;
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t nout = (int64_t)ntok * geo.C_out;
        const dim3 grid((unsigned)((nout + 255) / 256));
        if (y_dtype == AQ_F32)
            lut_reduce_kernel<AQ_F32><<<grid, 256, 0, stream>>>(geo, ws, plan.nchunk, plan.tok_block, tok0, ntok,
                                                                w.scales, x_scales, Y);
        else
            lut_reduce_kernel<AQ_F16><<<grid, 256, 0, stream>>>(geo, ws, plan.nchunk, plan.tok_block, tok0, ntok,
                                                                w.scales, x_scales, Y);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace aq
