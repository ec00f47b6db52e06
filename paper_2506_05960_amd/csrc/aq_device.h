// Device-side helpers shared by the gfx950 kernels: storage conversions,
// vector types, activation loads with implicit im2col, and output stores.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "aq.h"
#include "aq_internal.h"

namespace aq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---- scalar conversions (storage bits <-> fp32) ----

__device__ __forceinline__ float f16_to_f32(uint16_t b) { return (float)__builtin_bit_cast(_Float16, b); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
// round-to-nearest-even conversions
__device__ __forceinline__ uint16_t f32_to_f16(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }
__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

// Materialise an fp32 value in a register.  Keeps the compiler from folding
// an fp32 multiply or add with a following fp16 conversion into one
// mixed-precision instruction (which would round once instead of twice).
__device__ __forceinline__ float opaque_f32(float v) {
    asm volatile("" : "+v"(v));
    return v;
}

template <int DT>
__device__ __forceinline__ float load_as_f32(const void* p, int64_t i) {
    if constexpr (DT == AQ_F32) return static_cast<const float*>(p)[i];
    else if constexpr (DT == AQ_F16) return f16_to_f32(static_cast<const uint16_t*>(p)[i]);
    else if constexpr (DT == AQ_BF16) return bf16_to_f32(static_cast<const uint16_t*>(p)[i]);
    else return (float)static_cast<const int8_t*>(p)[i];
}

template <int DT>
__device__ __forceinline__ uint16_t f32_to_tile(float f) {
    if constexpr (DT == AQ_BF16) return f32_to_bf16(f);
    else return f32_to_f16(f);
}

template <int YT>
__device__ __forceinline__ void store_y(void* Y, int64_t i, float v) {
    if constexpr (YT == AQ_F32) static_cast<float*>(Y)[i] = v;
    else static_cast<uint16_t*>(Y)[i] = f32_to_f16(v);
}

// Flat index of output (token, channel) in Y: linear [tokens][C_out]; conv NCHW.
__device__ __forceinline__ int64_t y_index(const Geom& geo, int64_t tok, int ch) {
    if (!geo.conv) return tok * geo.C_out + ch;
    const int64_t plane = (int64_t)geo.OH * geo.OW;
    const int64_t b = tok / plane;
    const int64_t p = tok - b * plane;
    return (b * geo.C_out + ch) * plane + p;
}

// Element (tok, k) of the implicit X matrix as fp32 (im2col with zero padding
// for a convolution).  int8 values are returned unscaled.
template <int XT>
__device__ __forceinline__ float x_elem(const Geom& geo, const void* X, int64_t tok, int k) {
    if (!geo.conv) return load_as_f32<XT>(X, tok * geo.K + k);
    const int khw = geo.kh * geo.kw;
    const int c = k / khw;
    const int rs = k - c * khw;
    const int r = rs / geo.kw;
    const int s = rs - r * geo.kw;
    const int64_t plane = (int64_t)geo.OH * geo.OW;
    const int64_t b = tok / plane;
    const int p = (int)(tok - b * plane);
    const int oh = p / geo.OW;
    const int ow = p - oh * geo.OW;
    const int ih = oh * geo.stride - geo.pad + r;
    const int iw = ow * geo.stride - geo.pad + s;
    if (ih < 0 || ih >= geo.H || iw < 0 || iw >= geo.W) return 0.0f;
    return load_as_f32<XT>(X, ((b * geo.cin + c) * geo.H + ih) * (int64_t)geo.W + iw);
}

}  // namespace aq
