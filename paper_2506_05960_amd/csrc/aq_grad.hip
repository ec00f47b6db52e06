// Codebook gradient of an AQ layer: the continuous step of PV-Tuning
// (Sec. 3.2), which tunes the codebooks while the codes stay fixed.
//
// With the loss gradient dY at the layer output, the chain rule through
// Y = X W^T and eq. (4) gives
//     dC[m][k][t] = sum over (i, j) with b[i][j][m] == k of s[i] * (dY^T X)[i][j*g + t].
// Two kernels compute it:
//   1. wgrad_kernel: the weight gradient dY^T X on the matrix cores.  The
//      reduction runs over tokens, so both operands are staged into LDS with
//      tokens contiguous: token-major linear operands are transposed in
//      registers in 8x8 blocks; NCHW convolution operands already run along
//      tokens (im2col rows are shifted input rows, Sec. 3.1.1).  Each tile
//      may cover a slice of the tokens (a split); it writes s[i] * partial.
//   2. cbgrad_gather_kernel: for every codebook entry, the (row, group) pairs
//      that select it are listed (a counting sort of the codes, built once);
//      the kernel sums their s-scaled gradient groups over all splits in a
//      fixed order.  No atomics: repeated calls give identical bits.
#include <algorithm>
#include <vector>

#include "aq_device.h"

namespace aq {

namespace {

constexpr int kGradChunk = 64;   // tokens per chunk: four 16-deep MFMA steps
constexpr int kGradPitch = 72;   // halves per LDS row: 64 tokens plus 8 padding halves

struct GradArgs {
    const uint16_t* X;
    const uint16_t* dY;
    const float* scales;
    float* P;                    // [S][C_out][K] fp32, s[i]-scaled partial weight gradients
    int nchunk;                  // token chunks in the whole input
    int cps;                     // chunks per split
    int S;                       // splits (every split owns at least one chunk)
    int tiles_m, tiles_n;        // tiles along C_out and K
};

template <int DT>
__device__ __forceinline__ floatx16 mfma_grad(const u32x4& a, const u32x4& b, const floatx16& c) {
    if constexpr (DT == AQ_BF16)
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                       0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a), __builtin_bit_cast(half8, b), c, 0,
                                                      0, 0);
}

// Column e of an 8x8 block of 16-bit values whose row a is r[a]: o[e] holds
// r[0][e], r[1][e], ..., r[7][e].
__device__ __forceinline__ u32x4 block_column(const u32x4 (&r)[8], int e) {
    u32x4 o;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const uint32_t lo = r[2 * p][e >> 1], hi = r[2 * p + 1][e >> 1];
        o[p] = (e & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
    return o;
}

// Eight input values shifted by d in {-1, 0, +1} positions along the row:
// out[e] = in[e + d], with `nb` the value that enters at the open end.
__device__ __forceinline__ u32x4 shift_row(const u32x4& v, uint32_t nb, int d) {
    if (d == 0) return v;
    u32x4 o;
    if (d < 0) {
        o[0] = __builtin_amdgcn_alignbyte(v[0], nb << 16, 2);
        o[1] = __builtin_amdgcn_alignbyte(v[1], v[0], 2);
        o[2] = __builtin_amdgcn_alignbyte(v[2], v[1], 2);
        o[3] = __builtin_amdgcn_alignbyte(v[3], v[2], 2);
    } else {
        o[0] = __builtin_amdgcn_alignbyte(v[1], v[0], 2);
        o[1] = __builtin_amdgcn_alignbyte(v[2], v[1], 2);
        o[2] = __builtin_amdgcn_alignbyte(v[3], v[2], 2);
        o[3] = __builtin_amdgcn_alignbyte(nb, v[3], 2);
    }
    return o;
}

// KIND: 0 linear (token-major X [N][K], dY [N][C_out]); 1 3x3 and 2 1x1
// convolutions with stride 1 and same padding (NCHW X and dY, OW % 8 == 0).
template <int KIND, int DT, int BM, int BN>
__global__ void __launch_bounds__(256, 2) wgrad_kernel(Geom geo, GradArgs ga) {
    constexpr bool CONV = KIND != 0;
    constexpr int KHW = KIND == 1 ? 9 : 1, KW = KIND == 1 ? 3 : 1, PAD = KIND == 1 ? 1 : 0;
    constexpr int WM = BM / 2, WN = BN / 2, AM = WM / 32, AN = WN / 32;
    constexpr int ROWS = BM + BN;
    constexpr int STAGE = ROWS * kGradPitch;                 // halves per stage
    constexpr int VPT = CONV ? ROWS * 8 / 256 : 1;           // staged units per thread
    __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];

    // XCD-aware order: consecutive workgroups land on different XCDs, so each
    // XCD takes a contiguous run of (split, row tile, column tile).
    const int total = ga.S * ga.tiles_m * ga.tiles_n;
    const int per_xcd = (total + 7) / 8;
    const int w = (int)(blockIdx.x % 8) * per_xcd + (int)(blockIdx.x / 8);
    if (w >= total) return;
    const int tn = w % ga.tiles_n;
    const int tm = (w / ga.tiles_n) % ga.tiles_m;
    const int z = w / (ga.tiles_n * ga.tiles_m);
    const int i0 = tm * BM, k0 = tn * BN;
    const int c_beg = z * ga.cps, c_end = min(ga.nchunk, c_beg + ga.cps);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31, hi = lane >> 5;
    const int64_t N = geo.tokens;

    // ---- staging: global -> registers (next chunk) -> LDS ----
    u32x4 rv[CONV ? VPT : 8];
    uint32_t nbv[CONV ? VPT : 1];
    int dsh[CONV ? VPT : 1];
    auto load_chunk = [&](int chunk) {
        const int64_t n0 = (int64_t)chunk * kGradChunk;
        if constexpr (!CONV) {
            // one 8x8 block per thread: 8 tokens x 8 channels (dY) or 8 inputs (X)
            const bool isA = tid < BM;
            const int bid = isA ? tid : tid - BM;
            const int nb8 = isA ? BM / 8 : BN / 8;
            const int cb = bid % nb8, tb = bid / nb8;
            const int len = isA ? geo.C_out : geo.K;
            const int col = (isA ? i0 : k0) + 8 * cb;
            const uint16_t* src = isA ? ga.dY : ga.X;
            const bool live = tid < ROWS && col < len;
#pragma unroll
            for (int a = 0; a < 8; ++a) {
                const int64_t n = n0 + 8 * tb + a;
                rv[a] = (live && n < N) ? *reinterpret_cast<const u32x4*>(src + n * len + col) : u32x4{0, 0, 0, 0};
            }
        } else {
            const int64_t P = (int64_t)geo.OH * geo.OW;
#pragma unroll
            for (int u = 0; u < VPT; ++u) {
                const int v = tid + 256 * u;
                const int row = v >> 3, tb = v & 7;
                const int64_t n = n0 + 8 * tb;
                rv[u] = u32x4{0, 0, 0, 0};
                nbv[u] = 0;
                dsh[u] = 0;
                if (n >= N) continue;
                const int64_t b = n / P;
                const int64_t p = n - b * P;
                if (row < BM) {
                    const int i = i0 + row;
                    if (i < geo.C_out)
                        rv[u] = *reinterpret_cast<const u32x4*>(ga.dY + (b * geo.C_out + i) * P + p);
                } else {
                    const int k = k0 + row - BM;
                    if (k >= geo.K) continue;
                    const int c = k / KHW, rs = k - c * KHW;
                    const int r = rs / KW, q = rs - r * KW;
                    const int oh = (int)(p / geo.OW), ow0 = (int)(p - (int64_t)oh * geo.OW);
                    const int ih = oh + r - PAD;
                    if (ih < 0 || ih >= geo.H) continue;
                    const uint16_t* rowp = ga.X + ((b * geo.cin + c) * geo.H + ih) * (int64_t)geo.W;
                    rv[u] = *reinterpret_cast<const u32x4*>(rowp + ow0);
                    const int d = q - PAD;
                    dsh[u] = d;
                    if (d < 0 && ow0 > 0) nbv[u] = rowp[ow0 - 1];
                    if (d > 0 && ow0 + 8 < geo.W) nbv[u] = rowp[ow0 + 8];
                }
            }
        }
    };
    auto store_chunk = [&](uint16_t* st) {
        if constexpr (!CONV) {
            if (tid < ROWS) {
                const bool isA = tid < BM;
                const int bid = isA ? tid : tid - BM;
                const int nb8 = isA ? BM / 8 : BN / 8;
                const int cb = bid % nb8, tb = bid / nb8;
                const int rbase = (isA ? 0 : BM) + 8 * cb;
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    *reinterpret_cast<u32x4*>(st + (rbase + e) * kGradPitch + 8 * tb) = block_column(rv, e);
            }
        } else {
#pragma unroll
            for (int u = 0; u < VPT; ++u) {
                const int v = tid + 256 * u;
                const int row = v >> 3, tb = v & 7;
                *reinterpret_cast<u32x4*>(st + row * kGradPitch + 8 * tb) = shift_row(rv[u], nbv[u], dsh[u]);
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

    auto compute = [&](const uint16_t* st) {
#pragma unroll
        for (int s = 0; s < kGradChunk / 16; ++s) {
            u32x4 af[AM], bf[AN];
#pragma unroll
            for (int a = 0; a < AM; ++a)
                af[a] = *reinterpret_cast<const u32x4*>(st + (WM * wm + 32 * a + l32) * kGradPitch + 16 * s + 8 * hi);
#pragma unroll
            for (int b = 0; b < AN; ++b)
                bf[b] = *reinterpret_cast<const u32x4*>(st + (BM + WN * wn + 32 * b + l32) * kGradPitch + 16 * s +
                                                        8 * hi);
#pragma unroll
            for (int a = 0; a < AM; ++a)
#pragma unroll
                for (int b = 0; b < AN; ++b) acc[a][b] = mfma_grad<DT>(af[a], bf[b], acc[a][b]);
        }
    };

    if (c_beg < c_end) {
        load_chunk(c_beg);
        store_chunk(lds);
        __syncthreads();
        for (int c = c_beg; c < c_end; ++c) {
            const int cur = (c - c_beg) & 1;
            if (c + 1 < c_end) load_chunk(c + 1);
            compute(lds + cur * STAGE);
            if (c + 1 < c_end) store_chunk(lds + (cur ^ 1) * STAGE);
            __syncthreads();
        }
    }

    // ---- epilogue: s[i] * partial, fp32, rows i (output channels), columns k ----
    float* Pz = ga.P + (int64_t)z * geo.C_out * geo.K;
#pragma unroll
    for (int a = 0; a < AM; ++a)
#pragma unroll
        for (int b = 0; b < AN; ++b) {
            const int k = k0 + WN * wn + 32 * b + l32;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int i = i0 + WM * wm + 32 * a + 8 * (r >> 2) + 4 * hi + (r & 3);
                if (i < geo.C_out && k < geo.K) Pz[(int64_t)i * geo.K + k] = ga.scales[i] * acc[a][b][r];
            }
        }
}

// One group of LPB lanes per codebook entry (m, k); lanes split into
// LPB / g entry slots times g positions t.  Each slot sums its entries in
// list order, then lane t adds the slots in order.
template <int LPB>
__global__ void __launch_bounds__(256) cbgrad_gather_kernel(const float* __restrict__ P, int64_t slice, int S,
                                                            const int32_t* __restrict__ offs,
                                                            const int32_t* __restrict__ ent, int64_t nent, int nk,
                                                            int M, int g, float* __restrict__ dC) {
    constexpr int BPW = 256 / LPB;
    __shared__ float red[256];
    const int tid = threadIdx.x;
    const int sub = tid / LPB, lt = tid % LPB;
    const int64_t bucket = (int64_t)blockIdx.x * BPW + sub;
    const bool live_bucket = bucket < (int64_t)M * nk;
    const int EP = LPB / g;
    const int e = lt / g, t = lt - (lt / g) * g;
    float acc = 0.0f;
    if (live_bucket && e < EP) {
        const int m = (int)(bucket / nk), k = (int)(bucket - (int64_t)m * nk);
        const int32_t beg = offs[(int64_t)m * (nk + 1) + k], end = offs[(int64_t)m * (nk + 1) + k + 1];
        const int32_t* list = ent + (int64_t)m * nent;
        int32_t idx = beg + e;
        // four entries per step keep several independent loads in flight
        for (; idx + 3 * EP < end; idx += 4 * EP) {
            int64_t base[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) base[u] = (int64_t)list[idx + u * EP] * g + t;
            float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            for (int s = 0; s < S; ++s)
#pragma unroll
                for (int u = 0; u < 4; ++u) v[u] += P[s * slice + base[u]];
#pragma unroll
            for (int u = 0; u < 4; ++u) acc += v[u];
        }
        for (; idx < end; idx += EP) {
            const int64_t base = (int64_t)list[idx] * g + t;
            float v = 0.0f;
            for (int s = 0; s < S; ++s) v += P[s * slice + base];
            acc += v;
        }
    }
    red[tid] = acc;
    __syncthreads();
    if (live_bucket && lt < g) {
        float sum = 0.0f;
        for (int e2 = 0; e2 < EP; ++e2) sum += red[sub * LPB + e2 * g + lt];
        dC[bucket * g + lt] = sum;
    }
}

template <int KIND, int DT, int BM, int BN>
hipError_t wgrad_launch(const Geom& geo, const GradArgs& ga, hipStream_t st) {
    const int total = ga.S * ga.tiles_m * ga.tiles_n;
    const unsigned grid = (unsigned)(8 * ((total + 7) / 8));
    wgrad_kernel<KIND, DT, BM, BN><<<grid, 256, 0, st>>>(geo, ga);
    return hipGetLastError();
}

template <int KIND, int DT>
hipError_t wgrad_dispatch(const Geom& geo, const GradPlan& gp, const GradArgs& ga, hipStream_t st) {
    if (gp.bm == 128 && gp.bn == 128) return wgrad_launch<KIND, DT, 128, 128>(geo, ga, st);
    if (gp.bm == 64 && gp.bn == 128) return wgrad_launch<KIND, DT, 64, 128>(geo, ga, st);
    if (gp.bm == 64 && gp.bn == 64) return wgrad_launch<KIND, DT, 64, 64>(geo, ga, st);
    return hipErrorInvalidConfiguration;
}

}  // namespace

// Tile and split choice: the largest tile that still gives about one
// workgroup per CU, then token splits up to about two workgroups per CU.
GradPlan grad_plan_create(const Geom& geo, int64_t max_tokens) {
    GradPlan gp{};
    const int shapes[3][2] = {{128, 128}, {64, 128}, {64, 64}};
    int pick = 2;
    for (int s = 0; s < 3; ++s) {
        const int64_t tiles = (int64_t)((geo.C_out + shapes[s][0] - 1) / shapes[s][0]) *
                              ((geo.K + shapes[s][1] - 1) / shapes[s][1]);
        if (tiles >= 240) {
            pick = s;
            break;
        }
    }
    gp.bm = shapes[pick][0];
    gp.bn = shapes[pick][1];
    gp.tiles_m = (geo.C_out + gp.bm - 1) / gp.bm;
    gp.tiles_n = (geo.K + gp.bn - 1) / gp.bn;
    const int64_t tiles = (int64_t)gp.tiles_m * gp.tiles_n;
    const int64_t nchunk = std::max<int64_t>(1, (max_tokens + kGradChunk - 1) / kGradChunk);
    gp.s_max = (int)std::min<int64_t>({16, nchunk, std::max<int64_t>(1, (480 + tiles - 1) / tiles)});
    return gp;
}

int grad_kind(const Geom& geo) {
    if (!geo.conv) return 0;
    return geo.kh == 3 ? 1 : 2;
}

hipError_t launch_codebook_grad(const Geom& geo, const GradPlan& gp, int dtype, const void* X, const void* dY,
                                const float* scales, float* P, const int32_t* offs, const int32_t* ent, float* dC,
                                int splits_override, hipStream_t st) {
    GradArgs ga;
    ga.X = static_cast<const uint16_t*>(X);
    ga.dY = static_cast<const uint16_t*>(dY);
    ga.scales = scales;
    ga.P = P;
    ga.nchunk = (int)((geo.tokens + kGradChunk - 1) / kGradChunk);
    int S = std::min(gp.s_max, ga.nchunk);
    if (splits_override > 0) S = std::min(S, splits_override);
    ga.cps = (ga.nchunk + S - 1) / S;
    ga.S = (ga.nchunk + ga.cps - 1) / ga.cps;     // every split owns at least one chunk
    ga.tiles_m = gp.tiles_m;
    ga.tiles_n = gp.tiles_n;
    const int kind = grad_kind(geo);
    hipError_t e;
    if (dtype == AQ_BF16) {
        e = kind == 0 ? wgrad_dispatch<0, AQ_BF16>(geo, gp, ga, st)
            : kind == 1 ? wgrad_dispatch<1, AQ_BF16>(geo, gp, ga, st)
                        : wgrad_dispatch<2, AQ_BF16>(geo, gp, ga, st);
    } else {
        e = kind == 0 ? wgrad_dispatch<0, AQ_F16>(geo, gp, ga, st)
            : kind == 1 ? wgrad_dispatch<1, AQ_F16>(geo, gp, ga, st)
                        : wgrad_dispatch<2, AQ_F16>(geo, gp, ga, st);
    }
    if (e != hipSuccess) return e;
    const int nk = 1 << geo.B;
    const int64_t buckets = (int64_t)geo.M * nk;
    const int64_t nent = (int64_t)geo.C_out * geo.G;
    const int64_t slice = (int64_t)geo.C_out * geo.K;
    // a wave per entry when lists are short (large codebooks), a workgroup otherwise
    if (nent / nk < 64) {
        cbgrad_gather_kernel<64><<<(unsigned)((buckets + 3) / 4), 256, 0, st>>>(P, slice, ga.S, offs, ent, nent, nk,
                                                                               geo.M, geo.g, dC);
    } else {
        cbgrad_gather_kernel<256><<<(unsigned)buckets, 256, 0, st>>>(P, slice, ga.S, offs, ent, nent, nk, geo.M, geo.g,
                                                                     dC);
    }
    return hipGetLastError();
}

// Counting sort of the codes: for codebook m, entries offs[m][k] ..
// offs[m][k+1] of ent[m] list the (row, group) pairs i*G + j with
// b[i][j][m] == k, in increasing order.
void build_code_index(const void* codes, int B, int C_out, int G, int M, std::vector<int32_t>& offs,
                      std::vector<int32_t>& ent) {
    const int nk = 1 << B;
    const int64_t nent = (int64_t)C_out * G;
    offs.assign((size_t)M * (nk + 1), 0);
    ent.assign((size_t)M * nent, 0);
    auto code = [&](int64_t p, int m) -> int {
        return B <= 8 ? static_cast<const uint8_t*>(codes)[p * M + m] : static_cast<const uint16_t*>(codes)[p * M + m];
    };
    for (int m = 0; m < M; ++m) {
        int32_t* o = offs.data() + (size_t)m * (nk + 1);
        for (int64_t p = 0; p < nent; ++p) ++o[code(p, m) + 1];
        for (int k = 0; k < nk; ++k) o[k + 1] += o[k];
        std::vector<int32_t> pos(o, o + nk);
        int32_t* list = ent.data() + (size_t)m * nent;
        for (int64_t p = 0; p < nent; ++p) list[pos[code(p, m)]++] = (int32_t)p;
    }
}

}  // namespace aq
