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
    note_launch(st, "decode_to_global_kernel", {CBT, 8 * (int)sizeof(CodeT), tile});
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

// ---- operand records for the fused kernel's pre-decoded mode ----
//
// One thread per (chunk c, channel n, lane half q).  It decodes the groups
// that lane of the fused kernel covers -- a 3x3 chunk's 72 weights of 8 input
// channels (K indices [(16c + 8q) * 9, + 72), channel outermost), or a
// 64-wide chunk's groups 8c + 2s + q, s < 4 -- with the decode arithmetic
// (codewords summed in ascending m: in fp16 for an fp16 codebook, else in fp32
// rounded once), and writes the B operand of each step s.  For a 3x3 chunk the
// operand of kernel position s is weight 9e + s of the 72 (e = channel 0..7);
// otherwise it is group s itself.  Groups past the end of K are zero.
template <int CBT, typename CodeT, int G>
__device__ __forceinline__ void decode_group_f16(const void* cb, const CodeT* code, int M, int64_t rows,
                                                 uint16_t (&v)[G]) {
    if constexpr (CBT == AQ_F16) {
        const uint16_t* c16 = static_cast<const uint16_t*>(cb);
        _Float16 h[G];
#pragma unroll
        for (int t = 0; t < G; ++t) h[t] = __builtin_bit_cast(_Float16, c16[(int64_t)code[0] * G + t]);
        for (int m = 1; m < M; ++m)
#pragma unroll
            for (int t = 0; t < G; ++t)
                h[t] = h[t] + __builtin_bit_cast(_Float16, c16[((int64_t)m * rows + code[m]) * G + t]);
#pragma unroll
        for (int t = 0; t < G; ++t) v[t] = __builtin_bit_cast(uint16_t, h[t]);
    } else {
        float a[G];
#pragma unroll
        for (int t = 0; t < G; ++t) a[t] = load_as_f32<CBT>(cb, (int64_t)code[0] * G + t);
        for (int m = 1; m < M; ++m)
#pragma unroll
            for (int t = 0; t < G; ++t) a[t] = __fadd_rn(a[t], load_as_f32<CBT>(cb, ((int64_t)m * rows + code[m]) * G + t));
#pragma unroll
        for (int t = 0; t < G; ++t) v[t] = f32_to_f16(opaque_f32(a[t]));
    }
}

// K3: a 3x3 chunk (16 input channels); G: group size 8, or 9 (one group per
// input channel's filter, the kernel-aware format of Sec. 3.1.2).  The lane's
// 72 weights are K indices [(16c + 8q) * 9, + 72): nine groups of 8 or eight
// groups of 9.
template <int CBT, typename CodeT, bool K3, int G>
__global__ void __launch_bounds__(256)
operand_records_kernel(const void* __restrict__ cb, const CodeT* __restrict__ codes, u32x4* __restrict__ rec,
                       int nchunk, int C_out, int Gn, int M, int B) {
    constexpr int ns = K3 ? 9 : 4;
    constexpr int NG = K3 ? 72 / G : 4;            // groups a thread decodes
    static_assert(K3 || G == 8, "64-wide chunks use groups of 8");
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // (chunk, channel, half)
    if (idx >= (int64_t)nchunk * C_out * 2) return;
    const int c = (int)(idx / (2 * C_out));
    const int rem = (int)(idx - (int64_t)c * 2 * C_out);
    const int n = rem >> 1, q = rem & 1;
    const int64_t rows = (int64_t)1 << B;
    const int j0 = K3 ? (16 * c + 8 * q) * 9 / G : 0;
    uint16_t v[NG][G];
#pragma unroll
    for (int s = 0; s < NG; ++s) {
        const int j = K3 ? j0 + s : c * 2 * ns + 2 * s + q;
        if (j < Gn) {
            decode_group_f16<CBT, CodeT, G>(cb, codes + ((int64_t)n * Gn + j) * M, M, rows, v[s]);
        } else {
#pragma unroll
            for (int t = 0; t < G; ++t) v[s][t] = 0;
        }
    }
#pragma unroll
    for (int s = 0; s < ns; ++s) {
        u32x4 o;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            uint32_t lo, hi;
            if constexpr (K3) {
                // position s of channel e (of the lane's 8) is weight 9e + s of the run
                const int v0 = 9 * (2 * d) + s, v1 = 9 * (2 * d + 1) + s;
                lo = v[v0 / G][v0 % G];
                hi = v[v1 / G][v1 % G];
            } else {
                lo = v[s][2 * d];
                hi = v[s][2 * d + 1];
            }
            o[d] = lo | (hi << 16);
        }
        rec[(((int64_t)c * ns + s) * C_out + n) * 2 + q] = o;
    }
}

// Same records for fp16 codebooks with g = 8 and M in {1, 2, 4}: a codeword is
// one 16-byte load, the M codewords of a group are summed with packed fp16
// adds in ascending m (the same IEEE fp16 sums as above), and every load of a
// thread is issued before any sum.
template <typename CodeT, bool K3, int MC>
__device__ __forceinline__ void records_f16_body(const u32x4* __restrict__ cb, const CodeT* __restrict__ codes,
                                                 u32x4* __restrict__ rec, int nchunk, int C_out, int Gn, int B,
                                                 int64_t idx) {   // idx: (chunk, channel, half)
    constexpr int ns = K3 ? 9 : 4;
    constexpr int NG = K3 ? 9 : 4;                 // groups a thread decodes
    if (idx >= (int64_t)nchunk * C_out * 2) return;
    const int c = (int)(idx / (2 * C_out));
    const int rem = (int)(idx - (int64_t)c * 2 * C_out);
    const int n = rem >> 1, q = rem & 1;
    const uint32_t rows = 1u << B;
    const int j0 = K3 ? (16 * c + 8 * q) * 9 / 8 : 0;
    uint32_t code[NG][MC];
#pragma unroll
    for (int s = 0; s < NG; ++s) {
        const int j = K3 ? j0 + s : c * 2 * ns + 2 * s + q;
        const int jc = j < Gn ? j : Gn - 1;       // groups past the end of K are zeroed below
#pragma unroll
        for (int m = 0; m < MC; ++m) code[s][m] = codes[((int64_t)n * Gn + jc) * MC + m];
    }
    u32x4 w[NG][MC];
#pragma unroll
    for (int s = 0; s < NG; ++s)
#pragma unroll
        for (int m = 0; m < MC; ++m) w[s][m] = cb[m * rows + code[s][m]];
    u32x4 g[NG];
#pragma unroll
    for (int s = 0; s < NG; ++s) {
        const int j = K3 ? j0 + s : c * 2 * ns + 2 * s + q;
        g[s] = w[s][0];
#pragma unroll
        for (int m = 1; m < MC; ++m)
#pragma unroll
            for (int d = 0; d < 4; ++d) g[s][d] = add_f16x2(g[s][d], w[s][m][d]);
        if (j >= Gn) g[s] = u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int s = 0; s < ns; ++s) {
        u32x4 o;
        if constexpr (K3) {
            // position s of channel e (of the lane's 8) is weight 9e + s of the run
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                const int v0 = 9 * (2 * d) + s, v1 = 9 * (2 * d + 1) + s;
                const uint32_t lo = (g[v0 >> 3][(v0 & 7) >> 1] >> (16 * (v0 & 1))) & 0xFFFFu;
                const uint32_t hi = (g[v1 >> 3][(v1 & 7) >> 1] >> (16 * (v1 & 1))) & 0xFFFFu;
                o[d] = lo | (hi << 16);
            }
        } else {
            o = g[s];
        }
        rec[(((int64_t)c * ns + s) * C_out + n) * 2 + q] = o;
    }
}

template <typename CodeT, bool K3, int MC>
__global__ void __launch_bounds__(256)
operand_records_f16_kernel(const u32x4* __restrict__ cb, const CodeT* __restrict__ codes, u32x4* __restrict__ rec,
                           int nchunk, int C_out, int Gn, int B) {
    records_f16_body<CodeT, K3, MC>(cb, codes, rec, nchunk, C_out, Gn, B,
                                    (int64_t)blockIdx.x * blockDim.x + threadIdx.x);
}

// Records of a 3x3 chunk in the kernel-aware format (g = 9: one group per
// input channel's 3x3 filter) from fp16 codebooks padded to 16 values per row:
// a codeword is one 16-byte and one 4-byte load, every load of a thread is
// issued before any sum, and the M codewords of a group are summed in fp16 in
// ascending m (the same IEEE fp16 sums as operand_records_kernel).  A record
// (chunk c, position s, channel n, lane half q) holds tap s of the 8 input
// channels 16c + 8q + e; two threads share it, each decoding 4 channels and
// writing its 8-byte half.
template <typename CodeT, int MC>
__device__ __forceinline__ void records_g9_f16_body(const uint8_t* __restrict__ cbp, const CodeT* __restrict__ codes,
                                                    uint8_t* __restrict__ rec, int nchunk, int C_out, int Gn, int B,
                                                    int64_t idx) {   // idx: (chunk, channel, half, quarter)
    if (idx >= (int64_t)nchunk * C_out * 4) return;
    const int hq = (int)(idx & 1);
    const int64_t rid = idx >> 1;
    const int c = (int)(rid / (2 * C_out));
    const int rem = (int)(rid - (int64_t)c * 2 * C_out);
    const int n = rem >> 1, q = rem & 1;
    const uint32_t rows = 1u << B;
    const int j0 = 16 * c + 8 * q + 4 * hq;
    uint32_t code[4][MC];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int jc = j0 + e < Gn ? j0 + e : Gn - 1;   // groups past the end of K are zeroed below
#pragma unroll
        for (int m = 0; m < MC; ++m) code[e][m] = codes[((int64_t)n * Gn + jc) * MC + m];
    }
    u32x4 lo[4][MC];
    uint32_t hi[4][MC];
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int m = 0; m < MC; ++m) {
            const uint8_t* row = cbp + ((size_t)m * rows + code[e][m]) * 32u;
            lo[e][m] = *reinterpret_cast<const u32x4*>(row);
            hi[e][m] = *reinterpret_cast<const uint32_t*>(row + 16);
        }
    uint16_t v[4][9];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        _Float16 h[9];
#pragma unroll
        for (int t = 0; t < 9; ++t) {
            const uint32_t w = t < 8 ? lo[e][0][t >> 1] : hi[e][0];
            h[t] = __builtin_bit_cast(_Float16, (uint16_t)(w >> (16 * (t & 1))));
        }
#pragma unroll
        for (int m = 1; m < MC; ++m)
#pragma unroll
            for (int t = 0; t < 9; ++t) {
                const uint32_t w = t < 8 ? lo[e][m][t >> 1] : hi[e][m];
                h[t] = h[t] + __builtin_bit_cast(_Float16, (uint16_t)(w >> (16 * (t & 1))));
            }
        const bool in = j0 + e < Gn;
#pragma unroll
        for (int t = 0; t < 9; ++t) v[e][t] = in ? __builtin_bit_cast(uint16_t, h[t]) : (uint16_t)0;
    }
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int s = 0; s < 9; ++s) {
        const u32x2 o{(uint32_t)v[0][s] | ((uint32_t)v[1][s] << 16), (uint32_t)v[2][s] | ((uint32_t)v[3][s] << 16)};
        *reinterpret_cast<u32x2*>(rec + ((((int64_t)c * 9 + s) * C_out + n) * 2 + q) * 16 + 8 * hq) = o;
    }
}

template <typename CodeT, int MC>
__global__ void __launch_bounds__(256)
operand_records_g9_f16_kernel(const uint8_t* __restrict__ cbp, const CodeT* __restrict__ codes,
                              uint8_t* __restrict__ rec, int nchunk, int C_out, int Gn, int B) {
    records_g9_f16_body<CodeT, MC>(cbp, codes, rec, nchunk, C_out, Gn, B,
                                   (int64_t)blockIdx.x * blockDim.x + threadIdx.x);
}

// Batched forms: one launch decodes the records of several layers that share
// the kernel; workgroup b belongs to the job whose range [start, next start)
// holds it (binary search over the kernel argument, uniform per workgroup),
// and decodes exactly what the single-layer launch's workgroup b - start does.
__device__ __forceinline__ int record_job_of(const RecordBatch& b, uint32_t blk) {
    int lo = 0, hi = b.count - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (b.start[mid] <= blk) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

template <typename CodeT, bool K3, int MC>
__global__ void __launch_bounds__(256) operand_records_f16_batch_kernel(const RecordBatch b) {
    const int l = record_job_of(b, blockIdx.x);
    const RecordJob& j = b.job[l];
    records_f16_body<CodeT, K3, MC>(static_cast<const u32x4*>(j.cb), static_cast<const CodeT*>(j.codes),
                                    static_cast<u32x4*>(j.rec), j.nchunk, j.C_out, j.G, j.B,
                                    (int64_t)(blockIdx.x - b.start[l]) * blockDim.x + threadIdx.x);
}

template <typename CodeT, int MC>
__global__ void __launch_bounds__(256) operand_records_g9_f16_batch_kernel(const RecordBatch b) {
    const int l = record_job_of(b, blockIdx.x);
    const RecordJob& j = b.job[l];
    records_g9_f16_body<CodeT, MC>(static_cast<const uint8_t*>(j.cb), static_cast<const CodeT*>(j.codes),
                                   static_cast<uint8_t*>(j.rec), j.nchunk, j.C_out, j.G, j.B,
                                   (int64_t)(blockIdx.x - b.start[l]) * blockDim.x + threadIdx.x);
}

size_t operand_record_bytes(const Geom& geo, const FusedPlan& plan) {
    const int ns = plan.kind == 1 ? 9 : plan.cm;
    return (size_t)plan.nchunk * ns * geo.C_out * 2 * 16;
}

template <typename CodeT>
static hipError_t records_dispatch(const Geom& geo, const FusedPlan& plan, const DeviceWeights& w, void* rec,
                                   hipStream_t st) {
    const int64_t n = (int64_t)plan.nchunk * geo.C_out * 2;
    const dim3 grid((unsigned)((n + 255) / 256)), block(256);
    const CodeT* codes = static_cast<const CodeT*>(w.codes);
    u32x4* r = static_cast<u32x4*>(rec);
    if (plan.kind != 1 && plan.cm != 4) return hipErrorInvalidConfiguration;
    if (geo.g != 8 && !(geo.g == 9 && plan.kind == 1)) return hipErrorInvalidConfiguration;
    if (w.cb_dtype == AQ_F16 && geo.g == 8 && (geo.M == 1 || geo.M == 2 || geo.M == 4)) {
        const u32x4* cb = static_cast<const u32x4*>(w.codebooks);
#define AQ_REC16(K3, MC) \
    operand_records_f16_kernel<CodeT, K3, MC><<<grid, block, 0, st>>>(cb, codes, r, plan.nchunk, geo.C_out, geo.G, geo.B)
        if (plan.kind == 1) {
            if (geo.M == 1) AQ_REC16(true, 1);
            else if (geo.M == 2) AQ_REC16(true, 2);
            else AQ_REC16(true, 4);
        } else {
            if (geo.M == 1) AQ_REC16(false, 1);
            else if (geo.M == 2) AQ_REC16(false, 2);
            else AQ_REC16(false, 4);
        }
#undef AQ_REC16
        note_launch(st, "operand_records_f16_kernel", {8 * (int)sizeof(CodeT), plan.kind == 1, geo.M});
        return hipGetLastError();
    }
    if (w.cb_dtype == AQ_F16 && geo.g == 9 && plan.kind == 1 && w.cb9 && (geo.M == 1 || geo.M == 2 || geo.M == 4)) {
        const uint8_t* cbp = static_cast<const uint8_t*>(w.cb9);
        const dim3 grid9((unsigned)((2 * n + 255) / 256));   // two threads per record
        uint8_t* r8 = static_cast<uint8_t*>(rec);
#define AQ_REC9(MC)                                                                                       \
    operand_records_g9_f16_kernel<CodeT, MC><<<grid9, block, 0, st>>>(cbp, codes, r8, plan.nchunk, geo.C_out, \
                                                                      geo.G, geo.B)
        if (geo.M == 1) AQ_REC9(1);
        else if (geo.M == 2) AQ_REC9(2);
        else AQ_REC9(4);
#undef AQ_REC9
        note_launch(st, "operand_records_g9_f16_kernel", {8 * (int)sizeof(CodeT), geo.M});
        return hipGetLastError();
    }
#define AQ_REC(CBT)                                                                                             \
    if (plan.kind == 1 && geo.g == 9)                                                                          \
        operand_records_kernel<CBT, CodeT, true, 9><<<grid, block, 0, st>>>(w.codebooks, codes, r, plan.nchunk, \
                                                                             geo.C_out, geo.G, geo.M, geo.B);   \
    else if (plan.kind == 1)                                                                                   \
        operand_records_kernel<CBT, CodeT, true, 8><<<grid, block, 0, st>>>(w.codebooks, codes, r, plan.nchunk, \
                                                                             geo.C_out, geo.G, geo.M, geo.B);   \
    else                                                                                                       \
        operand_records_kernel<CBT, CodeT, false, 8><<<grid, block, 0, st>>>(w.codebooks, codes, r,            \
                                                                              plan.nchunk, geo.C_out, geo.G,   \
                                                                              geo.M, geo.B);
    switch (w.cb_dtype) {
    case AQ_F32: AQ_REC(AQ_F32) break;
    case AQ_F16: AQ_REC(AQ_F16) break;
    default: AQ_REC(AQ_BF16) break;
    }
    note_launch(st, "operand_records_kernel", {w.cb_dtype, 8 * (int)sizeof(CodeT), plan.kind == 1, geo.g});
#undef AQ_REC
    return hipGetLastError();
}

hipError_t launch_operand_records(const Geom& geo, const FusedPlan& plan, const DeviceWeights& w, void* rec,
                                  hipStream_t stream) {
    if (geo.B <= 8) return records_dispatch<uint8_t>(geo, plan, w, rec, stream);
    return records_dispatch<uint16_t>(geo, plan, w, rec, stream);
}

int records_batch_key(const Geom& geo, const FusedPlan& plan, const DeviceWeights& w) {
    if (w.cb_dtype != AQ_F16) return -1;
    const int mi = geo.M == 1 ? 0 : geo.M == 2 ? 1 : geo.M == 4 ? 2 : -1;
    if (mi < 0) return -1;
    const int c16 = geo.B > 8;
    if (geo.g == 8 && (plan.kind == 1 || plan.cm == 4)) return ((0 * 2 + c16) * 2 + (plan.kind == 1)) * 3 + mi;
    if (geo.g == 9 && plan.kind == 1 && w.cb9) return ((1 * 2 + c16) * 2 + 1) * 3 + mi;
    return -1;
}

RecordJob records_batch_job(const Geom& geo, const FusedPlan& plan, const DeviceWeights& w, void* rec,
                            uint32_t* blocks) {
    const int64_t n = (int64_t)plan.nchunk * geo.C_out * (geo.g == 9 ? 4 : 2);   // threads
    *blocks = (uint32_t)((n + 255) / 256);
    return RecordJob{geo.g == 9 ? w.cb9 : w.codebooks, w.codes, rec, plan.nchunk, geo.C_out, geo.G, geo.B};
}

hipError_t launch_operand_records_batch(int key, const RecordBatch& b, hipStream_t st) {
    if (key < 0 || key >= 24 || b.count < 1 || b.count > kRecordBatchMax) return hipErrorInvalidValue;
    const dim3 grid(b.start[b.count]), block(256);
    const int mi = key % 3, k3 = (key / 3) % 2, c16 = (key / 6) % 2, fam = key / 12;
    const int MC = mi == 0 ? 1 : mi == 1 ? 2 : 4;
#define AQ_B16(CT, K3, MC) operand_records_f16_batch_kernel<CT, K3, MC><<<grid, block, 0, st>>>(b)
#define AQ_B9(CT, MC) operand_records_g9_f16_batch_kernel<CT, MC><<<grid, block, 0, st>>>(b)
#define AQ_BM(CT)                                                                   \
    if (fam == 1) {                                                                 \
        if (MC == 1) AQ_B9(CT, 1);                                                  \
        else if (MC == 2) AQ_B9(CT, 2);                                             \
        else AQ_B9(CT, 4);                                                          \
    } else if (k3) {                                                                \
        if (MC == 1) AQ_B16(CT, true, 1);                                           \
        else if (MC == 2) AQ_B16(CT, true, 2);                                      \
        else AQ_B16(CT, true, 4);                                                   \
    } else {                                                                        \
        if (MC == 1) AQ_B16(CT, false, 1);                                          \
        else if (MC == 2) AQ_B16(CT, false, 2);                                     \
        else AQ_B16(CT, false, 4);                                                  \
    }
    if (c16) { AQ_BM(uint16_t) } else { AQ_BM(uint8_t) }
#undef AQ_BM
#undef AQ_B9
#undef AQ_B16
    if (fam == 1) note_launch(st, "operand_records_g9_f16_batch_kernel", {c16 ? 16 : 8, MC, b.count});
    else note_launch(st, "operand_records_f16_batch_kernel", {c16 ? 16 : 8, k3, MC, b.count});
    return hipGetLastError();
}

hipError_t launch_decode_to_global(const Geom& geo, const DeviceWeights& w, int tile_dtype, void* W,
                                   hipStream_t stream) {
    if (geo.B <= 8) return decode_dispatch_cb<uint8_t>(geo, w, tile_dtype, W, stream);
    return decode_dispatch_cb<uint16_t>(geo, w, tile_dtype, W, stream);
}

}  // namespace aq
