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

// Raw buffer resource over `bytes` bytes; loads at offsets >= bytes return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* p, uint64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0,
                                             (int)(uint32_t)(bytes < 0xFFFFFFFFull ? bytes : 0xFFFFFFFFull), 0x00020000);
}
constexpr uint32_t kOutOfRange = 0x80000000u;   // byte offset past every buffer the kernels read

// Cache policy of a buffer access that is coherent across the whole device
// (the SC1 bit): it reads and writes memory past this XCD's L2, which may
// hold stale copies of lines another XCD wrote.  Used for the partial sums
// that one workgroup publishes and another, possibly on another XCD, reads.
constexpr int kCoherent = 16;

typedef _Float16 half2v __attribute__((ext_vector_type(2)));

// Two IEEE fp16 additions (round to nearest even) on packed halves.
__device__ __forceinline__ uint32_t add_f16x2(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, a) + __builtin_bit_cast(half2v, b));
}

// ---- direct-to-LDS loads ----

// 16 bytes from global memory into LDS: lane l of the wave writes slot
// dst_wave_base + 16 * l (the base must be wave-uniform).
__device__ __forceinline__ void lds_dma16(const uint8_t* src, uint8_t* dst_wave_base) {
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                     (__attribute__((address_space(3))) void*)dst_wave_base, 16, 0, 0);
}

// s_waitcnt with vmcnt <= n (n < 64), expcnt and lgkmcnt unrestricted (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt field");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier without the release fence of __syncthreads(): that fence
// waits for every outstanding vector-memory operation, which would also drain
// the direct-to-LDS prefetches of later chunks.  LDS reads issued before the
// barrier are drained here; the DMA writes are awaited by wait_vmcnt.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

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
