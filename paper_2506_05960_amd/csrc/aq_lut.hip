// LUT path of the AQ forward (appendix, eq. (12)-(13)): because every group
// of a row is reconstructed from the same M codebooks, the product of one
// token's input slice x_j (g values) with a reconstructed group is the sum of
// M table entries T[j][m][b] = x_j . C_m[b], one per code.  A workgroup owns a
// chunk of jc groups at a time, NT tokens and a slice of output rows:
//
//  1. Table.  T for the chunk's jc*M (group, codebook) slots and all 2^B
//     codewords, NT tokens per entry, fp32, in LDS.  With an fp16 codebook
//     and fp16 / int8 input and g = 8 this is a small matrix product with
//     reduction length 8 -- rows (group, token), columns codewords -- run on
//     v_mfma_f32_32x32x8_f16 (fp16 products are exact in fp32).  Otherwise
//     threads form the dot products with fp32 FMAs.
//  2. Gather.  The chunk's codes of a row are one contiguous run of jc*M
//     bytes (repacked at create time), read by a few lanes with 16-byte loads
//     so that a wavefront streams one contiguous block of codes.  Each lane
//     adds the table entries its codes select, then the lanes of a row
//     combine their sums with cross-lane reductions.
//
// A workgroup walks a few consecutive chunks, keeping its rows' sums in
// registers, and writes one partial sum per row and token to a workspace.
// The partial sums are then added in a fixed order, the per-channel (and
// per-token) scales applied and Y stored, in one of two ways:
//  * a second kernel (the default): 64 threads per output each add every
//    64th chunk group's partial, then one adds the 64 results in order;
//  * in this kernel: the workgroups of one row slice and token pass (one per
//    chunk group) count their arrivals, and the last to arrive adds every
//    chunk group's partial in chunk-group order and resets the counter (one
//    launch, no memset).  Measured slower: the last workgroup of each slice
//    reduces its whole slice alone, a latency chain longer than the launch
//    it saves.
//
// Table layout: slot s = (group jj, codebook m) = jj*M + m, entry s*256 + code,
// NT consecutive floats per entry (one 4/8/16-byte LDS read).  Every slot has
// 256 entries; entries past 2^B, and the slots of groups past the end of K
// (whose staged inputs are zero), hold zeros, so the gather needs no bounds
// test on codes or slots.
#include "aq_device.h"

namespace aq {

typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef _Float16 half2 __attribute__((ext_vector_type(2)));

template <int NT>
struct TblVec;
template <>
struct TblVec<1> {
    typedef float type;
};
template <>
struct TblVec<2> {
    typedef float type __attribute__((ext_vector_type(2)));
};
template <>
struct TblVec<4> {
    typedef float type __attribute__((ext_vector_type(4)));
};

struct LutArgs {
    const void* cb;          // [M][2^B][g] codebooks (codebook dtype)
    const uint8_t* codes;    // [nchunk][C_out][jc*M]
    uint32_t code_bytes;     // size of `codes`
    const void* X;           // first image (convolution) or token (linear) of this launch
    uint32_t x_bytes;        // bytes of X from there on that this launch may read
    int tok0;                // first token of this launch, counted from X
    int ntok;                // tokens in this launch
    int jc;                  // groups per chunk
    int nchunk;              // chunks along K
    int cpw;                 // consecutive chunks per workgroup, 1 .. kLutMaxSteps
    int rpl;                 // row steps per workgroup, 1 .. kLutMaxSteps
    int tok_block;           // workspace rows per chunk group
    float* ws;               // [chunk groups][tok_block][C_out]
    uint32_t* arrivals;      // [row slices][token passes] arrival counters, zero between launches
    int ncg;                 // chunk groups (gridDim.y)
    const float* scales;     // [C_out]
    const float* x_scales;   // [tokens] per-token scales (int8 input), else null
    void* Y;                 // the whole output
    int64_t tok_out0;        // first token of this launch in Y (and x_scales)
    int y_dtype;
    int one_launch;          // reduce in this kernel (last-arriving workgroup) instead of a second kernel
};

constexpr int kLutMaxSteps = 4;      // chunks per workgroup, and row steps per workgroup
constexpr int kLutMaxM = 8;
constexpr int kLutPreFrags = 8;      // codebook fragments kept in registers per wave (2M of them, M <= 4)

constexpr uint32_t kLutOob = 0x80000000u;   // byte offset past every buffer read here

// Element (tok, k) of the implicit X matrix, read without branches: its byte
// offset (out of range for padding, k >= K or tok >= ntok, so the load returns
// zero), the raw storage bits, and their value.  Offsets are relative to the
// launch's first image (convolution) or token (linear layer).
template <int XT>
__device__ __forceinline__ uint32_t x_offset(const Geom& geo, int tok, int k, bool ok) {
    uint32_t idx;
    if (!geo.conv) {
        idx = (uint32_t)tok * (uint32_t)geo.K + (uint32_t)k;
    } else {
        const int khw = geo.kh * geo.kw;
        const int c = k / khw;
        const int rs = k - c * khw;
        const int r = rs / geo.kw;
        const int s = rs - r * geo.kw;
        const int plane = geo.OH * geo.OW;
        const int b = tok / plane;
        const int pp = tok - b * plane;
        const int oh = pp / geo.OW;
        const int ow = pp - oh * geo.OW;
        const int ih = oh * geo.stride - geo.pad + r;
        const int iw = ow * geo.stride - geo.pad + s;
        ok = ok && ih >= 0 && ih < geo.H && iw >= 0 && iw < geo.W;
        idx = ((uint32_t)(b * geo.cin + c) * (uint32_t)geo.H + (uint32_t)ih) * (uint32_t)geo.W + (uint32_t)iw;
    }
    constexpr uint32_t xb = XT == AQ_F32 ? 4u : XT == AQ_I8 ? 1u : 2u;
    return ok ? idx * xb : kLutOob;
}

template <int XT>
__device__ __forceinline__ uint32_t x_load_raw(__amdgpu_buffer_rsrc_t xr, uint32_t off) {
    if constexpr (XT == AQ_F32) return __builtin_amdgcn_raw_buffer_load_b32(xr, off, 0, 0);
    else if constexpr (XT == AQ_I8) return __builtin_amdgcn_raw_buffer_load_b8(xr, off, 0, 0);
    else return __builtin_amdgcn_raw_buffer_load_b16(xr, off, 0, 0);
}

template <int XT>
__device__ __forceinline__ uint32_t x_raw(const Geom& geo, __amdgpu_buffer_rsrc_t xr, int tok, int k, bool ok) {
    return x_load_raw<XT>(xr, x_offset<XT>(geo, tok, k, ok));
}

template <int XT>
__device__ __forceinline__ float x_value(uint32_t raw) {
    if constexpr (XT == AQ_F32) return __uint_as_float(raw);
    else if constexpr (XT == AQ_I8) return (float)(int8_t)(uint8_t)raw;
    else if constexpr (XT == AQ_F16) return f16_to_f32((uint16_t)raw);
    else return bf16_to_f32((uint16_t)raw);
}

// Two fp16 values packed in a dword.  (Copied through memory: a bit cast of a
// vector element inside an unrolled loop has been seen to read element 0.)
__device__ __forceinline__ half2 u32_as_half2(uint32_t u) {
    half2 h;
    __builtin_memcpy(&h, &u, 4);
    return h;
}

// fp16 bits of an element whose value fp16 holds exactly (fp16 or int8 input)
template <int XT>
__device__ __forceinline__ _Float16 x_half(uint32_t raw) {
    if constexpr (XT == AQ_F16) return __builtin_bit_cast(_Float16, (uint16_t)raw);
    else return (_Float16)(int)(int8_t)(uint8_t)raw;
}

template <int NT, bool MF, int CBT, int XT>
__global__ void __launch_bounds__(256)
lut_fwd_kernel(Geom geo, LutArgs a) {
    typedef typename TblVec<NT>::type vecT;
    extern __shared__ __attribute__((aligned(16))) float lds[];
    const int slice = blockIdx.x;
    const int cgrp = blockIdx.y;
    const int tok_first = blockIdx.z * NT;
    const int M = geo.M, g = geo.g;
    const int nk = 1 << geo.B;
    const int jc = a.jc;
    const int slots = jc * M;
    const int kspan = jc * g;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    vecT* tbl = reinterpret_cast<vecT*>(lds);

    // gather mapping: LPR = jc*M/16 adjacent lanes per row, one 16-code run each;
    // the workgroup covers a.rpl steps of 4 * (64 / LPR) rows
    const int LPR = slots >> 4;
    const int rpw = 64 / LPR;                          // rows per wave (lanes past rpw*LPR idle)
    const int part = lane % LPR;
    const int rows_step = 4 * rpw;
    const int row0 = lane < rpw * LPR ? slice * rows_step * a.rpl + wave * rpw + lane / LPR : geo.C_out;
    const __amdgpu_buffer_rsrc_t cr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(a.codes), 0,
                                                                        (int)a.code_bytes, 0x00020000);
    const uint8_t* tb = reinterpret_cast<const uint8_t*>(lds);

    // ---- every global read this workgroup needs, issued before any is used ----
    // (all offsets are computed first so that the loads go out back to back)
    const int p = lane & 31;
    const int th = lane >> 5;                          // which 4 of the 8 reduction values
    const int c_lo = cgrp * a.cpw;
    const int ncw = min(a.nchunk - c_lo, a.cpw);       // chunks of this workgroup
    // inputs: element e = n*kspan + kk of each chunk, one per thread when they fit
    const bool xone = NT * kspan <= 256;
    uint32_t xoff[kLutMaxSteps];
    {
        const int e = threadIdx.x;
        const int n = e / kspan;
        const int kk = e - n * kspan;
        const int tok = tok_first + n;
#pragma unroll
        for (int ci = 0; ci < kLutMaxSteps; ++ci) {
            const int k = (c_lo + ci) * kspan + kk;
            const bool ok = xone && ci < ncw && e < NT * kspan && tok < a.ntok && k < geo.K;
            xoff[ci] = x_offset<XT>(geo, a.tok0 + tok, ok ? k : 0, ok);
        }
    }
    // codes of chunk c_lo + ci for row step r; the first chunk's are requested now,
    // each later chunk's one chunk ahead of its use
    auto code_off = [&](int ci, int r) -> uint32_t {
        const int row = row0 + r * rows_step;
        return ci < ncw && r < a.rpl && row < geo.C_out
            ? ((uint32_t)(c_lo + ci) * geo.C_out + row) * (uint32_t)slots + (uint32_t)part * 16u
            : kLutOob;
    };
    uint32_t coff[kLutMaxSteps];
#pragma unroll
    for (int r = 0; r < kLutMaxSteps; ++r) coff[r] = code_off(0, r);
    const __amdgpu_buffer_rsrc_t cbr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.cb), 0, (int)((uint32_t)M * nk * g * 2u), 0x00020000);
    // one-token table by dot products: thread k keeps codeword k of every codebook;
    // several-token table on the matrix cores: this wave's (codebook, 32-codeword block)
    // fragments, pairs wave, wave+4, ... (2M of them)
    constexpr bool DOT = MF && NT == 1;
    constexpr int NPRE = DOT ? kLutMaxM : kLutPreFrags;
    uint32_t boff[NPRE];
#pragma unroll
    for (int i = 0; i < NPRE; ++i) {
        if constexpr (DOT) {
            const int k = threadIdx.x;
            boff[i] = i < M && k < nk ? (uint32_t)(i * nk + k) * 16u : kLutOob;
        } else {
            const int pi = wave + 4 * i;
            const int k = (pi & 7) * 32 + p;
            const bool ok = MF && i < 2 * M && 2 * M <= kLutPreFrags && k < nk;
            boff[i] = ok ? ((uint32_t)((pi >> 3) * nk + k) * 8u + 4u * th) * 2u : kLutOob;
        }
    }
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.X), 0, (int)a.x_bytes,
                                                                        0x00020000);
    u32x4 creg[kLutMaxSteps][kLutMaxSteps];
#pragma unroll
    for (int r = 0; r < kLutMaxSteps; ++r) creg[0][r] = __builtin_amdgcn_raw_buffer_load_b128(cr, coff[r], 0, 0);
    uint32_t xpre[kLutMaxSteps];
#pragma unroll
    for (int ci = 0; ci < kLutMaxSteps; ++ci) xpre[ci] = x_load_raw<XT>(xr, xoff[ci]);
    half4 bfr[kLutPreFrags];
    u32x4 hcb[kLutMaxM];
    if constexpr (DOT) {
#pragma unroll
        for (int i = 0; i < kLutMaxM; ++i) hcb[i] = __builtin_amdgcn_raw_buffer_load_b128(cbr, boff[i], 0, 0);
    } else if constexpr (MF) {
#pragma unroll
        for (int i = 0; i < kLutPreFrags; ++i)
            bfr[i] = __builtin_bit_cast(half4, __builtin_amdgcn_raw_buffer_load_b64(cbr, boff[i], 0, 0));
    }

    vecT acc[kLutMaxSteps];
#pragma unroll
    for (int r = 0; r < kLutMaxSteps; ++r) acc[r] = vecT{};

#pragma unroll
    for (int ci = 0; ci < kLutMaxSteps; ++ci) {
        if (ci >= ncw) break;
        const int k0 = (c_lo + ci) * kspan;
        if (ci + 1 < kLutMaxSteps) {
#pragma unroll
            for (int r = 0; r < kLutMaxSteps; ++r)
                creg[ci + 1 < kLutMaxSteps ? ci + 1 : 0][r] =
                    __builtin_amdgcn_raw_buffer_load_b128(cr, code_off(ci + 1, r), 0, 0);
        }
        if (ci) __syncthreads();                       // previous chunk's gathers are done with the table
        // ---- stage the NT tokens' inputs for this chunk (zero past K / past the tokens) ----
        if constexpr (MF) {
            _Float16* xs = reinterpret_cast<_Float16*>(lds + (size_t)slots * 256 * NT);
            if (xone) {
                if (threadIdx.x < NT * kspan) xs[threadIdx.x] = x_half<XT>(xpre[ci]);   // exact: fp16 or int8 value
            } else {
                for (int e = threadIdx.x; e < NT * kspan; e += 256) {
                    const int n = e / kspan;
                    const int kk = e - n * kspan;
                    const int tok = tok_first + n;
                    const int k = k0 + kk;
                    const bool ok = tok < a.ntok && k < geo.K;
                    xs[e] = x_half<XT>(x_raw<XT>(geo, xr, a.tok0 + tok, ok ? k : 0, ok));
                }
            }
            __syncthreads();
            if constexpr (DOT) {
                // ---- one-token table: entry (group jj, codebook m, codeword k) = x_jj . C_m[k] ----
                float* tf = lds;
                const int k = threadIdx.x;               // 256 threads, 256 entries per slot
                for (int jj = 0; jj < jc; ++jj) {
                    const u32x4 xv = *reinterpret_cast<const u32x4*>(xs + jj * 8);   // same address in every lane
#pragma unroll
                    for (int m = 0; m < kLutMaxM; ++m) {
                        if (m >= M) break;
                        float v = 0.0f;
#pragma unroll
                        for (int w = 0; w < 4; ++w)
                            v = __builtin_amdgcn_fdot2(u32_as_half2(xv[w]), u32_as_half2(hcb[m][w]), v, false);
                        tf[(jj * M + m) * 256 + k] = v;
                    }
                }
            } else {
                // ---- several-token table on the matrix cores: D[(group, token)][codeword] ----
                const int gpb = 32 / NT;                   // groups per 32-row block
                const int nrb = (jc + gpb - 1) / gpb;
                for (int i = 0; i < 2 * M; ++i) {
                    const int pi = wave + 4 * i;
                    const int m = pi >> 3;
                    const int k = (pi & 7) * 32 + p;
                    half4 bv = {0, 0, 0, 0};
                    if (2 * M <= kLutPreFrags) {
#pragma unroll
                        for (int f = 0; f < kLutPreFrags; ++f)
                            if (f == i) bv = bfr[f];
                    } else {
                        const uint32_t off = k < nk ? ((uint32_t)(m * nk + k) * 8u + 4u * th) * 2u : kLutOob;
                        bv = __builtin_bit_cast(half4, __builtin_amdgcn_raw_buffer_load_b64(cbr, off, 0, 0));
                    }
                    for (int rb = 0; rb < nrb; ++rb) {
                        half4 av = {0, 0, 0, 0};
                        {
                            const int jj = rb * gpb + p / NT;
                            const int n = p % NT;
                            if (jj < jc) av = *reinterpret_cast<const half4*>(xs + n * kspan + jj * 8 + 4 * th);
                        }
                        floatx16 d = {};
                        d = __builtin_amdgcn_mfma_f32_32x32x8f16(av, bv, d, 0, 0, 0);
                        // lane holds column k, rows 8*(r/4) + 4*th + r%4
#pragma unroll
                        for (int rq = 0; rq < 4; ++rq) {
                            const int rw = 8 * rq + 4 * th;  // rows rw .. rw+3
                            if constexpr (NT == 4) {
                                const int jj = rb * gpb + rw / 4;
                                if (jj < jc) {
                                    vecT v = {d[4 * rq], d[4 * rq + 1], d[4 * rq + 2], d[4 * rq + 3]};
                                    tbl[(jj * M + m) * 256 + k] = v;
                                }
                            } else {
#pragma unroll
                                for (int h = 0; h < 2; ++h) {
                                    const int jj = rb * gpb + (rw + 2 * h) / 2;
                                    if (jj < jc) {
                                        vecT v;
                                        v[0] = d[4 * rq + 2 * h];
                                        v[1] = d[4 * rq + 2 * h + 1];
                                        tbl[(jj * M + m) * 256 + k] = v;
                                    }
                                }
                            }
                        }
                    }
                }
            }
        } else {
            float* xs = lds + (size_t)slots * 256 * NT;
            if (xone) {
                if (threadIdx.x < NT * kspan) xs[threadIdx.x] = x_value<XT>(xpre[ci]);
            } else {
                for (int e = threadIdx.x; e < NT * kspan; e += 256) {
                    const int n = e / kspan;
                    const int kk = e - n * kspan;
                    const int tok = tok_first + n;
                    const int k = k0 + kk;
                    const bool ok = tok < a.ntok && k < geo.K;
                    xs[e] = x_value<XT>(x_raw<XT>(geo, xr, a.tok0 + tok, ok ? k : 0, ok));
                }
            }
            __syncthreads();
            // ---- table with fp32 FMAs: one thread per (slot, codeword) entry ----
            float* tf = lds;
            for (int e = threadIdx.x; e < slots * 256; e += 256) {
                const int s = e >> 8;
                const int k = e & 255;
                const int jj = s / M;
                const int m = s - jj * M;
                float t_acc[NT];
#pragma unroll
                for (int n = 0; n < NT; ++n) t_acc[n] = 0.0f;
                if (k < nk) {
                    const int64_t cbase = ((int64_t)m * nk + k) * g;
                    const float* x0 = xs + jj * g;
                    for (int t = 0; t < g; ++t) {
                        const float c = load_as_f32<CBT>(a.cb, cbase + t);
#pragma unroll
                        for (int n = 0; n < NT; ++n) t_acc[n] = fmaf(x0[n * kspan + t], c, t_acc[n]);
                    }
                }
#pragma unroll
                for (int n = 0; n < NT; ++n) tf[(size_t)e * NT + n] = t_acc[n];
            }
        }
        __syncthreads();

        // ---- gather: slot of byte b is part*16 + b; its entry starts at (slot*256 + code) * NT floats ----
        const uint8_t* tq = tb + (size_t)part * 16 * 256 * sizeof(vecT);
#pragma unroll
        for (int r = 0; r < kLutMaxSteps; ++r) {
            if (r >= a.rpl) break;
            const u32x4 cw = creg[ci][r];
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const uint32_t v = cw[w];
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const uint32_t code = (v >> (8 * b)) & 0xFFu;
                    acc[r] += *reinterpret_cast<const vecT*>(tq + ((4 * w + b) * 256 + code) * sizeof(vecT));
                }
            }
        }
    }

    // ---- combine the LPR lanes of a row (adjacent lanes) and store this chunk group's partial sums ----
    const __amdgpu_buffer_rsrc_t wsr = buffer_rsrc(a.ws, (uint64_t)a.ncg * a.tok_block * geo.C_out * 4);
#pragma unroll
    for (int r = 0; r < kLutMaxSteps; ++r) {
        if (r >= a.rpl) break;
        vecT v = acc[r];
        for (int j = 1; j < LPR; ++j) {
            const int src = min(lane + j, 63);
            if constexpr (NT == 1) {
                v += __shfl(acc[r], src, 64);
            } else {
#pragma unroll
                for (int n = 0; n < NT; ++n) v[n] += __shfl(acc[r][n], src, 64);
            }
        }
        const int row = row0 + r * rows_step;
        if (row < geo.C_out && part == 0) {
#pragma unroll
            for (int n = 0; n < NT; ++n) {
                const int tok = tok_first + n;
                if (tok < a.ntok) {
                    float e;
                    if constexpr (NT == 1) e = v;
                    else e = v[n];
                    const uint32_t off = (uint32_t)(((cgrp * a.tok_block + tok) * geo.C_out + row) * 4);
                    // device-coherent when this kernel reduces (the last workgroup may run on another XCD)
                    if (a.one_launch) __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(e), wsr, off, 0, kCoherent);
                    else __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(e), wsr, off, 0, 0);
                }
            }
        }
    }

    if (!a.one_launch) return;       // the reduction kernel follows
    // ---- arrival of this chunk group; the last one of the (row slice, token
    // pass) adds every chunk group's partial sums in order and stores Y ----
    wait_vmcnt<0>();                 // this thread's partial sums have reached memory
    __syncthreads();                 // (and every thread is done with the table in LDS)
    uint32_t* arrived = reinterpret_cast<uint32_t*>(lds);
    uint32_t* cnt = a.arrivals + (size_t)slice * gridDim.z + blockIdx.z;
    if (threadIdx.x == 0) *arrived = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (*arrived != (uint32_t)(a.ncg - 1)) return;    // uniform over the workgroup
    const int nrows = rows_step * a.rpl;
    const int rbase = slice * nrows;
    for (int e = threadIdx.x; e < nrows * NT; e += 256) {
        const int n = e / nrows;
        const int row = rbase + (e - n * nrows);
        const int tok = tok_first + n;
        if (row >= geo.C_out || tok >= a.ntok) continue;
        // every chunk group's partial sum, 16 device-coherent loads in flight at
        // a time (past the end: zeros), added in chunk-group order
        const uint32_t src = (uint32_t)((tok * geo.C_out + row) * 4);
        const uint32_t cstride = (uint32_t)(a.tok_block * geo.C_out * 4);
        float t = 0.0f;
        for (int c0 = 0; c0 < a.ncg; c0 += 16) {
            uint32_t q[16];
#pragma unroll
            for (int c = 0; c < 16; ++c)
                q[c] = __builtin_amdgcn_raw_buffer_load_b32(wsr, c0 + c < a.ncg ? src + (uint32_t)(c0 + c) * cstride
                                                                              : kOutOfRange, 0, kCoherent);
#pragma unroll
            for (int c = 0; c < 16; ++c)
                if (c0 + c < a.ncg) t = (c0 + c == 0) ? __uint_as_float(q[c]) : t + __uint_as_float(q[c]);
        }
        float y = t * a.scales[row];
        if (a.x_scales) y *= a.x_scales[a.tok_out0 + tok];
        const int64_t yi = y_index(geo, a.tok_out0 + tok, row);
        if (a.y_dtype == AQ_F32) static_cast<float*>(a.Y)[yi] = y;
        else static_cast<uint16_t*>(a.Y)[yi] = f32_to_f16(y);
    }
    if (threadIdx.x == 0) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Fixed-order reduction over chunk groups, scales, dtype cast and store.
// A workgroup covers 16 outputs; 64 threads per output each add every 64th
// partial sum, then one thread adds the 64 results in order.
constexpr int kRedParts = 64;

template <int YT>
__global__ void __launch_bounds__(1024)
lut_reduce_kernel(Geom geo, const float* __restrict__ ws, int ncg, int tok_block, int64_t tok0, int ntok,
                  const float* __restrict__ scales, const float* __restrict__ x_scales, void* __restrict__ Y) {
    __shared__ float red[kRedParts][17];
    const int ol = threadIdx.x & 15;
    const int part = threadIdx.x >> 4;
    const int64_t idx = (int64_t)blockIdx.x * 16 + ol;
    const bool valid = idx < (int64_t)ntok * geo.C_out;
    const int tok = valid ? (int)(idx / geo.C_out) : 0;
    const int i = valid ? (int)(idx - (int64_t)tok * geo.C_out) : 0;
    float acc = 0.0f;
    if (valid)
        for (int c = part; c < ncg; c += kRedParts) acc += ws[((int64_t)c * tok_block + tok) * geo.C_out + i];
    red[part][ol] = acc;
    __syncthreads();
    if (part == 0 && valid) {
        float t = 0.0f;
        for (int p = 0; p < kRedParts; ++p) t += red[p][ol];
        float v = t * scales[i];
        if (x_scales) v *= x_scales[tok0 + tok];
        store_y<YT>(Y, y_index(geo, tok0 + tok, i), v);
    }
}

size_t lut_lds_bytes(const Geom& geo, const LutPlan& plan, int nt) {
    const bool mf = plan.mfma_table;
    return (size_t)plan.jc * geo.M * 256 * nt * sizeof(float) +
           (size_t)nt * plan.jc * geo.g * (mf ? 2 : 4);
}

template <int NT, bool MF, int CBT, int XT>
static hipError_t launch_table(const Geom& geo, const LutPlan& plan, const LutArgs& a, hipStream_t st) {
    const size_t lds = lut_lds_bytes(geo, plan, NT);
    hipError_t e = ensure_dynamic_lds((const void*)lut_fwd_kernel<NT, MF, CBT, XT>, lds);
    if (e != hipSuccess) return e;
    const int rows_wg = 4 * (64 / (plan.jc * geo.M / 16)) * a.rpl;
    const dim3 grid((unsigned)((geo.C_out + rows_wg - 1) / rows_wg), (unsigned)((a.nchunk + a.cpw - 1) / a.cpw),
                    (unsigned)((a.ntok + NT - 1) / NT));
    lut_fwd_kernel<NT, MF, CBT, XT><<<grid, 256, lds, st>>>(geo, a);
    note_launch(st, "lut_fwd_kernel", {NT, (int)MF, CBT, XT});
    return hipGetLastError();
}

template <int NT>
static hipError_t launch_table_nt(const Geom& geo, const LutPlan& plan, int cb_dtype, int x_dtype, const LutArgs& a,
                                  hipStream_t st) {
    if (plan.mfma_table) {
        if (x_dtype == AQ_I8) return launch_table<NT, true, AQ_F16, AQ_I8>(geo, plan, a, st);
        return launch_table<NT, true, AQ_F16, AQ_F16>(geo, plan, a, st);
    }
#define AQ_LUT_X(CBT)                                                                            \
    switch (x_dtype) {                                                                           \
    case AQ_F32: return launch_table<NT, false, CBT, AQ_F32>(geo, plan, a, st);                 \
    case AQ_F16: return launch_table<NT, false, CBT, AQ_F16>(geo, plan, a, st);                 \
    case AQ_BF16: return launch_table<NT, false, CBT, AQ_BF16>(geo, plan, a, st);               \
    default: return launch_table<NT, false, CBT, AQ_I8>(geo, plan, a, st);                      \
    }
    switch (cb_dtype) {
    case AQ_F32: AQ_LUT_X(AQ_F32)
    case AQ_F16: AQ_LUT_X(AQ_F16)
    default: AQ_LUT_X(AQ_BF16)
    }
#undef AQ_LUT_X
}

// Arrival counters of one launch: one per (row slice, token pass).  A table
// has at most 144 slots (144 KB of LDS), so a row takes at most 9 lanes and a
// row step (four waves) at least 28 rows; a launch covers at most 32 tokens.
size_t lut_arrival_count(int C_out) { return (size_t)((C_out + 15) / 16) * 32; }

int lut_tokens_per_entry(const LutPlan& plan, int ntok) {
    int nt = ntok >= 3 ? 4 : ntok;
    while (nt > plan.nt_max) nt >>= 1;
    return nt;
}

hipError_t launch_lut_forward(const Geom& geo, const DeviceWeights& w, const LutPlan& plan, const void* X,
                              int x_dtype, const float* x_scales, void* Y, int y_dtype, float* ws,
                              uint32_t* arrivals, bool one_launch, hipStream_t stream) {
    for (int64_t tok0 = 0; tok0 < geo.tokens; tok0 += plan.tok_block) {
        const int ntok = (int)((geo.tokens - tok0 < plan.tok_block) ? geo.tokens - tok0 : plan.tok_block);
        const int nt = lut_tokens_per_entry(plan, ntok);
        LutArgs a;
        a.cb = w.codebooks;
        a.codes = w.codes_lut;
        a.code_bytes = (uint32_t)((size_t)plan.nchunk * geo.C_out * plan.jc * geo.M);
        const int xb = x_dtype == AQ_F32 ? 4 : x_dtype == AQ_I8 ? 1 : 2;
        int64_t first = tok0, count = ntok, row_elems = geo.K;   // linear: whole token rows
        if (geo.conv) {                                           // convolution: whole images
            const int64_t plane = (int64_t)geo.OH * geo.OW;
            first = tok0 / plane;
            count = (tok0 + ntok - 1) / plane - first + 1;
            row_elems = (int64_t)geo.cin * geo.H * geo.W;
            a.tok0 = (int)(tok0 - first * plane);
        } else {
            a.tok0 = 0;
        }
        const int64_t xbytes = count * row_elems * xb;
        if (xbytes >= (int64_t(1) << 31)) return hipErrorInvalidValue;   // 32-bit buffer offsets
        a.X = static_cast<const char*>(X) + first * row_elems * xb;
        a.x_bytes = (uint32_t)xbytes;
        a.ntok = ntok;
        a.jc = plan.jc;
        a.nchunk = plan.nchunk;
        // rows: a row step is 4 * (64 / LPR) rows, LPR = jc*M/16 lanes per row; one
        // workgroup takes up to kLutMaxSteps steps, so that each chunk's table serves
        // as many output rows as possible.  chunks: up to kLutMaxSteps consecutive
        // chunks per workgroup (fewer partial sums) while the grid stays near 512.
        const int rows_step = 4 * (64 / (plan.jc * geo.M / 16));
        const int64_t passes = (ntok + nt - 1) / nt;
        const int rpl = (int)std::min<int64_t>(kLutMaxSteps, (geo.C_out + rows_step - 1) / rows_step);
        const int64_t slices = (geo.C_out + (int64_t)rows_step * rpl - 1) / ((int64_t)rows_step * rpl);
        const int cpw =
            (int)std::min<int64_t>(kLutMaxSteps, std::max<int64_t>(1, (plan.nchunk * slices * passes + 511) / 512));
        a.cpw = cpw;
        a.rpl = rpl;
        const int64_t cgs = (plan.nchunk + cpw - 1) / cpw;
        if ((size_t)(slices * passes) > lut_arrival_count(geo.C_out)) return hipErrorInvalidValue;
        a.tok_block = plan.tok_block;
        a.ws = ws;
        a.arrivals = arrivals;
        a.ncg = (int)cgs;
        a.scales = w.scales;
        a.x_scales = x_scales;
        a.Y = Y;
        a.tok_out0 = tok0;
        a.y_dtype = y_dtype;
        a.one_launch = one_launch ? 1 : 0;
        hipError_t e;
        switch (nt) {
        case 4: e = launch_table_nt<4>(geo, plan, w.cb_dtype, x_dtype, a, stream); break;
        case 2: e = launch_table_nt<2>(geo, plan, w.cb_dtype, x_dtype, a, stream); break;
        default: e = launch_table_nt<1>(geo, plan, w.cb_dtype, x_dtype, a, stream); break;
        }
        if (e != hipSuccess) return e;
        if (one_launch) continue;
        const int64_t nout = (int64_t)ntok * geo.C_out;
        const dim3 grid((unsigned)((nout + 15) / 16));
        if (y_dtype == AQ_F32)
            lut_reduce_kernel<AQ_F32><<<grid, 16 * kRedParts, 0, stream>>>(geo, ws, (int)cgs, plan.tok_block, tok0, ntok,
                                                                w.scales, x_scales, Y);
        else
            lut_reduce_kernel<AQ_F16><<<grid, 16 * kRedParts, 0, stream>>>(geo, ws, (int)cgs, plan.tok_block, tok0, ntok,
                                                                w.scales, x_scales, Y);
        note_launch(stream, "lut_reduce_kernel", {y_dtype == AQ_F32 ? AQ_F32 : AQ_F16});
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace aq
