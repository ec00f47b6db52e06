// Internal declarations shared by the host entry points and the kernel
// launchers.  Nothing here crosses the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <initializer_list>
#include <vector>

#include "aq.h"

namespace aq {

// Geometry of one forward call, resolved on the host.
struct Geom {
    int C_out, K, G, g, M, B;
    int64_t tokens;               // rows of the (implicit) X matrix
    bool conv;
    int cin, kh, kw, stride, pad, H, W, OH, OW;
};

// Per-layer route options (aq_layer_set_option); 0 everywhere is the default.
struct Options {
    int64_t lut_max_tokens;   // 0: the measured rule, -1: never, else the token limit
    int weights;              // 0 auto, 1 in-loop decode, 2 pre-decoded records
    int generic;              // 1: generic decode kernel instead of the fused kernel
    int rec_product;          // 0 auto, 1 fused kernel's pre-decoded loop, 2 dense product
    int fused_bm, fused_bn;   // forced fused tile (0: planner)
    int dense_bm, dense_bn;   // forced dense-product tile (0: planner)
    int rlin_tile;            // wave-split linear kernel tile variant (0, 1, 2)
    int tile_order;           // 0 auto, 1 token tiles slowest, 2 channel tiles slowest
    int stage_rows;           // 1: kh staged rows per output row
    int split_k;              // fused kernel K split over workgroups (0: planner)
    int grad_splits;          // codebook gradient token splits (0: planner)
    int grad_regs;            // 1: register-staged weight-gradient kernels
    int grad_bm, grad_bn;     // forced weight-gradient tile (0: planner)
    int table_one_launch;     // 1: table path reduces in its own kernel (last-arriving workgroup)
};

constexpr int kMaxSplitK = 8;   // most workgroups sharing one output tile along K

// Launch trace of the entry point running on this thread (aq_layer_set_launch_events):
// every launcher reports each kernel it puts on `st` right after the launch, by
// name and template arguments, so that the caller's timing events bracket it.
void note_launch(hipStream_t st, const char* kernel, std::initializer_list<int> template_args);

// Raise a kernel's dynamic-LDS limit to at least `bytes` on the current
// device (once per kernel and device; thread-safe).
hipError_t ensure_dynamic_lds(const void* kernel, size_t bytes);

// Device-resident copy of a layer's quantized weights.
struct DeviceWeights {
    const void* codebooks;        // [M][2^B][g] in codebook dtype
    const float* cb32;            // [M][2^B][g] fp32 (exact widening of codebooks)
    const void* cbtile;           // [2^B][g] codebook rounded to the tile dtype (M == 1, B > 8), else null
    const void* codes;            // [C_out][G][M] uint8 | uint16
    const uint8_t* codes_lut;     // [nchunk][C_out][jc*M] uint8 (B <= 8), zero padded past G
    const float* scales;          // [C_out]
    int cb_dtype;                 // aq_dtype
    const void* cb9;              // g = 9 fp16 codebooks padded to 16 values per row [M][2^B][16], else null
};

// LUT-path blocking chosen at create time.
struct LutPlan {
    int jc;                       // groups per chunk (jc * M is a multiple of 16)
    int nchunk;                   // ceil(G / jc)
    int tok_block;                // tokens per launch (workspace rows)
    int nt_max;                   // most tokens per table entry (1, 2 or 4) that fit LDS
    bool mfma_table;              // table built on the matrix cores (fp16 codebook, fp16/int8 input, g == 8)
};

// ---- fused decode + matrix-core path (fp16 tiles, g == 8) ----

enum FusedDec {
    FUSED_DEC_PK16 = 0,   // fp16 codebooks in LDS, codewords accumulated with packed fp16 adds
    FUSED_DEC_F32L = 1,   // fp32 codebooks in LDS, fp32 sum in ascending m
    FUSED_DEC_T16L = 2,   // M == 1, codebook pre-rounded to fp16, in LDS
    FUSED_DEC_T16G = 3,   // M == 1, codebook pre-rounded to fp16, read from global memory (B > 8)
    FUSED_DEC_REC = 4     // operands decoded beforehand into per-step records (one 16-byte load each)
};

struct FusedPlan {
    int kind;             // 0 linear, 1 conv 3x3, 2 conv 1x1
    int cm;               // 16-wide k steps per chunk (per kernel position for a convolution)
    int nchunk;           // chunks along K
    int rec_bytes;        // code record bytes per (chunk, output channel, lane half)
    int dec;              // FusedDec
    int mc;               // M
    int cb_bytes;         // LDS codebook bytes (0 when read from global memory)
    int rec_only;         // no in-loop decode for this format: always the pre-decoded mode
    int nmajor;           // workgroup order: channel tile slowest (else token tile slowest)
    int rlin_var;         // wave-split linear kernel tile variant (rec_linear_tile)
    // chosen per forward
    int bm, bn, upl;      // tile and staging units per lane
    int units;            // staging units per chunk
    int pr, pw, ps;       // patch rows, patch width (pixels), pixel / token-row stride (bytes)
    // convolution: the staged rows are blocks of sr rows, each holding every input
    // row of rpb consecutive output rows of one image (output row i of a block
    // reads block rows i * stride + kernel row)
    int sr, rpb;
    float inv_sr, inv_rpb;
    int pbuf_bytes;       // one staging buffer
    int total_rows;       // convolution: images * OH
    size_t lds_bytes;     // dynamic LDS per workgroup
    // convolution: fp32 reciprocals of OW, OH, pr and W / 2 (correctly rounded)
    // for the kernel's quotient-with-correction index arithmetic
    float inv_ow, inv_oh, inv_pr, inv_wp;
    int64_t x_bytes;      // bytes of this forward's input X (the bound of the kernel's activation loads)
    int tile_div;         // tiles along the faster tile index (token tiles if nmajor, else channel tiles)
    float inv_tile_div;   // its fp32 reciprocal
    int wsplit;           // 1: convolution on the 2 x 2 wave-split records kernel (tile bm x bn)
    int rdepth;           // wave-split kernel: record register sets (loads run rdepth - 1 steps ahead)
    int splitk;           // workgroups sharing one tile along K (1: no split)
    int ntiles;           // output tiles (the grid is ntiles * splitk workgroups)
    float inv_ntiles;     // its fp32 reciprocal
};

struct FusedLaunch {
    const void* cb;       // codebook source (LDS copy source or global table)
    const uint8_t* crec;  // code records
    const float* scales;
    const void* X;
    const float* x_scales;
    void* Y;
    int y_dtype;
    int x_dtype;
    hipStream_t stream;
    float* part;          // K split: fp32 partial tiles [ntiles][splitk][BM * BN] (null without a split)
    uint32_t* arrivals;   // K split: arrival counter per tile, zero between launches
    int* occupancy;       // non-null: store the instantiation's workgroups per compute unit
                          // at plan.lds_bytes and launch nothing
};

hipError_t launch_fused_forward(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl);
// 3x3 or 1x1 convolution over pre-decoded operand records (fl.crec) with the
// four waves splitting a 128 x bn tile 2 x 2 (plan.wsplit; bn 128 or 192,
// plan.upl staging units per thread; plan.rdepth 3 or 6 for 3x3, 4 for 1x1).
hipError_t launch_rec_conv(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl);
// Dense matrix-core product over pre-decoded operand records (fl.crec), tile plan.bm x plan.bn;
// for a convolution plan.pr / plan.ps / plan.pw are the staging's image slots, rows per
// slot and padded row width.  `xpack` receives the repacked activations (convolution, int8
// input), `zero` points at 16 zero bytes.
hipError_t launch_rec_gemm(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl, void* xpack,
                           const void* zero);
size_t rec_gemm_lds_bytes(int kind, int bm, int bn);

// Operand records of the pre-decoded mode: record (chunk, step, channel, lane
// half) = the 8 fp16 weights of that matrix-core B operand, unscaled.
size_t operand_record_bytes(const Geom& geo, const FusedPlan& plan);
hipError_t launch_operand_records(const Geom& geo, const FusedPlan& plan, const DeviceWeights& w, void* rec,
                                  hipStream_t stream);
// Several layers' record decodes in one launch (aq_layers_prepare): jobs whose
// records kernel is the same, passed by value as the kernel argument.
struct RecordJob {
    const void* cb;       // fp16 codebooks [M][2^B][8], or the padded g = 9 rows [M][2^B][16]
    const void* codes;    // [C_out][G][M] uint8 | uint16
    void* rec;            // the layer's record buffer
    int nchunk, C_out, G, B;
};
constexpr int kRecordBatchMax = 32;
struct RecordBatch {
    int count;                              // jobs, 1 .. kRecordBatchMax
    uint32_t start[kRecordBatchMax + 1];    // first workgroup of each job; start[count] = grid size
    RecordJob job[kRecordBatchMax];
};
// Key of the records kernel of this decode (equal keys batch together), or -1
// where that kernel has no batched form.
int records_batch_key(const Geom& geo, const FusedPlan& plan, const DeviceWeights& w);
// The decode as a batch job, and its workgroup count.
RecordJob records_batch_job(const Geom& geo, const FusedPlan& plan, const DeviceWeights& w, void* rec,
                            uint32_t* blocks);
hipError_t launch_operand_records_batch(int key, const RecordBatch& b, hipStream_t stream);
// Linear layer over pre-decoded operand records (plan.cm == 4): 2 x 2 wave
// split of a 256- or 128-token by 128-channel tile, no K split.
bool rec_linear_supported(const Geom& geo, const FusedPlan& plan, int x_dtype);
int rec_linear_tile(const Geom& geo, int forced);
hipError_t launch_rec_linear(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl);
hipError_t launch_fused_conv3(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl);
hipError_t launch_fused_conv1(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl);
hipError_t launch_fused_linear(const Geom& geo, const FusedPlan& plan, const FusedLaunch& fl);

// ---- launchers (each returns the launch's hipError_t) ----

hipError_t launch_decode_to_global(const Geom& geo, const DeviceWeights& w, int tile_dtype, void* W,
                                   hipStream_t stream);

// ws: [chunk groups][tok_block][C_out] fp32 partial sums; arrivals: lut_arrival_count(geo) counters, zero
// between launches (the last workgroup of each row slice and token pass resets its own)
hipError_t launch_lut_forward(const Geom& geo, const DeviceWeights& w, const LutPlan& plan, const void* X,
                              int x_dtype, const float* x_scales, void* Y, int y_dtype, float* ws,
                              uint32_t* arrivals, bool one_launch, hipStream_t stream);
size_t lut_arrival_count(int C_out);

hipError_t launch_mfma_forward(const Geom& geo, const DeviceWeights& w, const void* X, int x_dtype,
                               const float* x_scales, void* Y, int y_dtype, int tile_dtype,
                               hipStream_t stream);

// Codebook preparation at create time: fp32 widening and tile-dtype rounding.
hipError_t launch_codebook_prep(const void* cb, int cb_dtype, int64_t n, float* cb32, void* cbtile, int tile_dtype,
                                hipStream_t stream);

size_t lut_lds_bytes(const Geom& geo, const LutPlan& plan, int nt);
int lut_tokens_per_entry(const LutPlan& plan, int ntok);

hipError_t launch_f32_forward(const Geom& geo, const DeviceWeights& w, const void* X, int x_dtype,
                              const float* x_scales, void* Y, int y_dtype, hipStream_t stream);

// ---- codebook gradient ----

struct GradPlan {
    bool dma;                     // convolution kernel with direct-to-LDS staging
    int bm, bn;                   // weight-gradient tile: output channels x inputs (x (channel, kernel row) pairs)
    int tiles_m, tiles_n;
    int s_max;                    // most token splits (partial buffers in the workspace)
};

GradPlan grad_plan_create(const Geom& geo, int64_t max_tokens, const Options& opt);
// X, dY: fp16 or bf16 (dtype); P: [s_max][C_out][K] fp32 workspace; offs / ent: the code index
hipError_t launch_codebook_grad(const Geom& geo, const GradPlan& gp, int dtype, const void* X, const void* dY,
                                const float* scales, float* P, const int32_t* offs, const int32_t* ent, float* dC,
                                const void* zero, int splits_override, hipStream_t st);
void build_code_index(const void* codes, int B, int C_out, int G, int M, std::vector<int32_t>& offs,
                      std::vector<int32_t>& ent);

}  // namespace aq
