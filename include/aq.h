/*
 * aq.h -- C ABI of the additively-quantized (AQ) layer forward for AMD
 * Instinct MI355X (gfx950).
 *
 * Operation (AQUATIC-Diff, arXiv 2506.05960, Sec. 2.4 eq. (4) and Sec. 3.1.1):
 * the weight matrix W [C_out][K] of a linear or im2col-lowered convolution
 * layer is split along K into G = K/g groups of g consecutive weights.  Group
 * j of output row i is stored as M integer codes b[i][j][m] < 2^B, and
 *
 *     W[i][j*g + t] = s[i] * sum_{m<M} C[m][ b[i][j][m] ][t]
 *
 * with M codebooks C[m] of 2^B rows of g values and one scale s[i] per output
 * channel.  The forward computes Y = X * W^T (tokens as rows).  A convolution
 * runs on NCHW input; its token order is (image, output row, output column)
 * and its K order is (input channel, kernel row, kernel column) with the
 * channel outermost (Sec. 3.1.1).
 *
 * Two device paths implement the forward:
 *   - LUT: per token and group, tabulate x_g . C[m][k] for every codeword k,
 *     then sum code-indexed table entries (the appendix's rearrangement,
 *     eq. (12)).  Needs B <= 8.  W is never formed.
 *   - DECODE: expand codes into fp16/bf16 (or fp32) weight operands and
 *     contract them with matrix-core instructions.  Its weights come from one
 *     of two sources:
 *       * in-loop decode: each workgroup decodes its weight tile on chip
 *         (registers / LDS) right before the products; W never reaches
 *         memory;
 *       * pre-decoded records: a first kernel writes the unscaled decoded
 *         weights, C_out * K fp16 values (2 * C_out * K bytes), to a
 *         layer-owned buffer, which the product kernel then reads.  This is
 *         the paper's decompress-then-compute route (Sec. 4.4), with the
 *         decompressed weights a per-forward temporary.
 *     The dispatcher takes the records per layer shape where they measured
 *     faster (formats without an in-loop decode always take them);
 *     AQ_OPT_WEIGHTS forces either source.
 * aq_layer_forward picks a path per call (AQ_PATH_AUTO) unless one is forced.
 *
 * Conventions for every entry point:
 *   - Return value is an aq_status; nothing aborts or throws across the ABI.
 *     On failure aq_last_error() returns a message (thread-local, valid until
 *     the next failing call on the same thread).
 *   - Arguments are validated on the host before any launch, allocation or
 *     copy (a call may first query the current device).
 *   - "host" pointers are read synchronously during the call; "device"
 *     pointers must be HIP device allocations on the layer's device.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 */
#ifndef AQ_H
#define AQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct aq_layer aq_layer; /* opaque, owned by the library */

typedef enum {
    AQ_OK = 0,
    AQ_ERR_INVALID_ARGUMENT = 1, /* bad pointer, size, dtype, alignment or code value */
    AQ_ERR_UNSUPPORTED = 2,      /* valid request the library has no kernel for      */
    AQ_ERR_OUT_OF_MEMORY = 3,    /* device allocation failed                          */
    AQ_ERR_DEVICE = 4            /* any other HIP error (or no GPU present)           */
} aq_status;

typedef enum { AQ_F32 = 0, AQ_F16 = 1, AQ_BF16 = 2, AQ_I8 = 3 } aq_dtype;

typedef enum { AQ_PATH_AUTO = 0, AQ_PATH_LUT = 1, AQ_PATH_DECODE = 2 } aq_path;

typedef struct {
    int32_t  out_features;   /* C_out >= 1                                                  */
    int32_t  in_features;    /* K = G*g; for a convolution K = conv_cin*conv_kh*conv_kw      */
    int32_t  codebook_dtype; /* aq_dtype: F32 | F16 | BF16                                   */
    int32_t  x_dtype;        /* aq_dtype: F32 | F16 | BF16 | I8 (I8: linear only, x_scales)  */
    int32_t  y_dtype;        /* aq_dtype: F32 | F16                                          */
    int32_t  tile_dtype;     /* aq_dtype: F16 | BF16 (matrix-core decode path) | F32         */
    int32_t  conv_kh, conv_kw;  /* 0,0 => linear layer: X [n][K], Y [n][C_out] row-major      */
    int32_t  conv_cin, conv_stride, conv_pad, in_h, in_w; /* conv: X NCHW [n][cin][in_h][in_w],
                                                              Y NCHW [n][C_out][OH][OW]         */
    int64_t  max_tokens;     /* workspace sizing: every forward needs tokens <= max_tokens    */
} aq_layer_desc;

/*
 * Create a layer: validate, copy and repack the quantized weights into
 * library-owned device memory on the current HIP device, and allocate the
 * workspace for up to desc->max_tokens tokens.  Synchronous; the caller may
 * free its buffers on return.
 *   codebooks  host, [M][2^B][g] in desc->codebook_dtype (bf16 as raw bits)
 *   codes      host, [C_out][K/g][M], uint8 when B <= 8, uint16 otherwise;
 *              every code must be < 2^B (scanned; AQ_ERR_INVALID_ARGUMENT)
 *   scales     host, [C_out] fp32, the per-output-channel scale s[i]
 *   g, M, B    group size 1..16, codebooks 1..8, index bits 1..16
 *   out        receives the handle (set to NULL on failure)
 * Supported: the LUT path needs B <= 8; the fp16/bf16 decode path needs
 * g == 8; the fp32 decode path takes any g.  A layer with no usable path
 * returns AQ_ERR_UNSUPPORTED.  Without a GPU: AQ_ERR_DEVICE.
 */
aq_status aq_layer_create(const aq_layer_desc* desc, const void* codebooks, const void* codes,
                          const float* scales, int g, int M, int B, aq_layer** out);

/*
 * Forward Y = X * W^T on `stream`; asynchronous, allocates nothing and never
 * synchronises.  The layer's workspace (table partial sums, pre-decoded
 * records, split-K partial tiles and arrival counters) makes concurrent
 * forwards on one layer a race: serialise them on one stream.
 *   X          device; linear: [n][K] row-major; conv: NCHW [n][cin][in_h][in_w];
 *              dtype desc->x_dtype; 16-byte aligned
 *   x_scales   device [n] fp32 per-token scales, required iff x_dtype == I8
 *              (x[t][k] = x_scales[t] * q[t][k]); otherwise ignored
 *   Y          device; linear [n][C_out]; conv NCHW [n][C_out][OH][OW];
 *              dtype desc->y_dtype; 16-byte aligned
 *   n          tokens (linear) or images (conv); 1 <= tokens <= max_tokens
 */
aq_status aq_layer_forward(aq_layer* layer, const void* X, const float* x_scales, void* Y, int64_t n,
                           void* stream);

/*
 * Decode the per-forward weight records of a forward over n tokens (linear)
 * or images (convolution) ahead of that forward, on `stream` (row a4 on the
 * pre-decoded route: the unscaled fp16 weights of Sec. 2.4 eq. (4), written
 * to the layer's record buffer).  The decode depends on the weights alone,
 * so a caller may run it on another stream, overlapped with other work (the
 * previous layer's product, say).  The next aq_layer_forward of this layer
 * with the same n then launches only its product kernel.  Ordering is the
 * caller's: that forward must be stream-ordered after this call's work (its
 * stream waits for `stream`, with an event), and no earlier forward of this
 * layer may still be reading the record buffer when this call's decode runs.
 * A route without pre-decoded records launches nothing and leaves the
 * forward unchanged; a forward with another n, and the allocation-free
 * forward, decode their own records.  Errors: AQ_ERR_INVALID_ARGUMENT (null
 * layer, n < 1, tokens beyond max_tokens), AQ_ERR_DEVICE (launch failed).
 */
aq_status aq_layer_prepare(aq_layer* layer, int64_t n, void* stream);

/*
 * aq_layer_prepare for `count` layers at once: layers[i] is prepared for a
 * forward over n[i] tokens (linear) or images (convolution).  The result, and
 * the ordering the caller owes each layer, are those of calling
 * aq_layer_prepare on every entry; but the record decodes of all layers whose
 * format shares one records kernel (fp16 codebooks, g = 8 or the kernel-aware
 * g = 9, M in {1, 2, 4}) go out as one launch per 32 layers, so that a whole
 * network's decodes (each one short and latency-bound) fill the chip
 * together.  Each layer's records land in its own buffer, bit-identical to
 * its own decode.  Other formats get one launch per layer.
 *   layers     host array [count] of layer handles, each listed at most once,
 *              all created on the current device
 *   n          host array [count]
 *   count      >= 0 (0: nothing to do)
 *   stream     the stream every decode is launched on
 * Every entry is checked before anything is launched; errors:
 * AQ_ERR_INVALID_ARGUMENT (null array or layer, n < 1, tokens beyond
 * max_tokens, a layer listed twice or created on another device),
 * AQ_ERR_DEVICE (launch failed; the layers launched before the failure stay
 * prepared).
 */
aq_status aq_layers_prepare(aq_layer* const* layers, const int64_t* n, int32_t count, void* stream);

/*
 * Allocation-free forward, for callers that cannot allocate device memory
 * during the call or keep per-layer workspace (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  Arguments,
 * validation, route, kernels and results (bit for bit) are those of
 * aq_layer_forward; the per-call scratch of the kernels -- the table path's
 * partial sums and arrival counters, the fused kernel's K-split partial tiles
 * and arrival counters, the pre-decoded operand records and the dense
 * product's repacked activations -- lives in one static device array of the
 * library (64 MiB per GPU, 256 KiB of it counters) instead of the layer's
 * workspace.  It calls no hipMalloc, hipFree or allocating library routine.
 * A call whose scratch would exceed the array returns AQ_ERR_UNSUPPORTED
 * before launching anything.  The first call on a device resolves the
 * array's address and clears its counters with a small kernel on `stream`.
 * Every call on one GPU shares that GPU's array: calls that overlap on one
 * GPU (other streams, other threads) race; serialise them.
 */
aq_status aq_layer_forward_static(aq_layer* layer, const void* X, const float* x_scales, void* Y, int64_t n,
                                  void* stream);

/*
 * Decoded weights W [C_out][K] in desc->tile_dtype (device, caller-owned),
 * computed as the decode path does (eq. (4) with the per-channel scale): the
 * M codewords summed in ascending m -- in fp16, rounding each partial sum,
 * when both codebooks and tile are fp16, otherwise in fp32 -- then times s[i]
 * in fp32, then one round-to-nearest-even to the tile dtype.  (For M <= 2
 * the fp16 sum equals the fp32 sum rounded once.)  Asynchronous on `stream`.
 * A test hook for bit-exact checks (the pre-decoded records of the forward
 * hold the same values before the scale, in the matrix-core operand order).
 */
aq_status aq_layer_decode(aq_layer* layer, void* W, void* stream);

/*
 * Codebook gradient, the continuous step of PV-Tuning (Sec. 3.2): codebooks
 * are tuned by gradient descent while the codes stay fixed.  With dY the loss
 * gradient at the layer output, the chain rule through Y = X * W^T and
 * eq. (4) with the per-channel scale gives
 *     dC[m][k][t] = sum over (i, j) with b[i][j][m] == k of s[i] * (dY^T X)[i][j*g + t],
 * where X is the im2col matrix for a convolution (Sec. 3.1.1).
 *   X      device; the forward's input layout (linear [n][K], conv NCHW);
 *          dtype `dtype`; 16-byte aligned
 *   dY     device; the forward's output layout (linear [n][C_out], conv NCHW
 *          [n][C_out][OH][OW]); dtype `dtype`; 16-byte aligned
 *   dtype  aq_dtype F16 or BF16, for both X and dY (others: AQ_ERR_UNSUPPORTED)
 *   dC     device [M][2^B][g] fp32, caller-owned, overwritten
 *   n      tokens (linear) or images (conv); tokens <= max_tokens
 * Supported: linear layers with C_out and K multiples of 8; 1x1 and 3x3
 * convolutions with stride 1, same padding and in_w a multiple of 8.  Other
 * layers return AQ_ERR_UNSUPPORTED.  The first call on a layer builds an
 * index of the codes (4 * C_out * (K/g) * M bytes) and a workspace of fp32
 * partial weight gradients, one C_out x K slice per token split, at most
 * max(32 MiB, C_out * K * 4) bytes (synchronous).  Later calls are
 * asynchronous on `stream` and allocate nothing.  Summation orders are
 * fixed: repeated calls give identical bits.
 * Calls on one layer share its workspace: serialise them on one stream.
 */
aq_status aq_layer_codebook_grad(aq_layer* layer, const void* X, const void* dY, int32_t dtype, float* dC,
                                 int64_t n, void* stream);

/* Force a path for later forwards (AUTO restores the dispatcher).  Forcing an
 * unavailable path returns AQ_ERR_UNSUPPORTED and leaves the setting as is. */
aq_status aq_layer_set_path(aq_layer* layer, aq_path path);

/*
 * Per-layer options of the dispatcher and planners, for benchmarks and tests
 * that compare routes.  Every option defaults to 0 (the measured rule) unless
 * stated; setting 0 restores the default.  The library reads no environment
 * variables.  Options are read on the host at each call; setting one while a
 * forward of the same layer is being issued on another thread is a race.
 * Forward results are identical across routes only where the entry says so.
 *   AQ_OPT_LUT_MAX_TOKENS   table path for tokens <= value when both paths
 *                           exist; 0 = the measured rule, -1 = never
 *   AQ_OPT_WEIGHTS          decode path weight source: 0 auto, 1 in-loop
 *                           decode (W never in memory), 2 pre-decoded
 *                           records (W written per forward); formats with
 *                           no in-loop decode (g = 9, M not in {1, 2, 4},
 *                           fp32/bf16 codebooks) always take the records
 *   AQ_OPT_GENERIC          1 = generic decode kernel instead of the fused
 *                           decode kernel (0: fused kernel where it applies)
 *   AQ_OPT_RECORD_PRODUCT   product kernel over records: 0 auto (linear
 *                           layers: the wave-split linear kernel), 1 the
 *                           fused kernel's own pre-decoded loop (outputs
 *                           bit-identical to its in-loop decode), 2 the
 *                           dense product with both operands staged in LDS,
 *                           3 the wave-split convolution kernel (3x3 and
 *                           1x1) where it applies (image planes a multiple
 *                           of 4 pixels): 128-token tiles, or, with a
 *                           64-token AQ_OPT_FUSED_TILE, 64-token tiles with
 *                           two waves per reduction
 *   AQ_OPT_FUSED_TILE       fused kernel tile BM * 1000 + BN (0 = planner);
 *                           a tile that does not fit falls back to the planner
 *   AQ_OPT_DENSE_TILE       dense product tile BM * 1000 + BN (0 = planner)
 *   AQ_OPT_REC_LINEAR_TILE  wave-split linear kernel: 0 = planner (128 x 128
 *                           with the four waves side by side along the
 *                           channels), 1 = 256 x 128 in 2 x 2 waves, 2 = 128 x
 *                           128 side by side, 3 = 128 x 128 in 2 x 2
 *                           (bit-identical outputs)
 *   AQ_OPT_TILE_ORDER       workgroup order: 0 auto, 1 token tiles slowest,
 *                           2 channel tiles slowest (bit-identical outputs)
 *   AQ_OPT_STAGE_ROWS       convolution staging: 0 each input row once per
 *                           block of output rows, 1 kh rows per output row
 *                           (bit-identical outputs)
 *   AQ_OPT_SPLIT_K          fused kernel: workgroups sharing one output tile
 *                           along K (0 = planner, 1 = none, up to 8); partial
 *                           tiles are summed in a fixed order, so repeated
 *                           runs are bitwise identical
 *   AQ_OPT_GRAD_SPLITS      codebook gradient: most token splits (0 = planner)
 *   AQ_OPT_GRAD_REGS        codebook gradient: 1 = register-staged kernels
 *                           (0: direct-to-LDS kernels where they apply)
 *   AQ_OPT_GRAD_TILE        codebook gradient tile BM * 1000 + BN (0 = planner)
 *   AQ_OPT_TABLE_ONE_LAUNCH table path: 1 = the table kernel also adds the
 *                           chunk groups' partial sums (the last workgroup of
 *                           each row slice to arrive does, in chunk-group
 *                           order); 0 = a second, reduction kernel (measured
 *                           faster).  Both orders are fixed: repeated runs
 *                           are bitwise identical
 * The gradient options take effect at the next gradient call; if they need a
 * larger partial-gradient workspace, that call reallocates it (synchronous).
 * Unknown options or out-of-range values return AQ_ERR_INVALID_ARGUMENT.
 */
typedef enum {
    AQ_OPT_LUT_MAX_TOKENS = 1,
    AQ_OPT_WEIGHTS = 2,
    AQ_OPT_GENERIC = 3,
    AQ_OPT_RECORD_PRODUCT = 4,
    AQ_OPT_FUSED_TILE = 5,
    AQ_OPT_DENSE_TILE = 6,
    AQ_OPT_REC_LINEAR_TILE = 7,
    AQ_OPT_TILE_ORDER = 8,
    AQ_OPT_STAGE_ROWS = 9,
    AQ_OPT_SPLIT_K = 10,
    AQ_OPT_GRAD_SPLITS = 11,
    AQ_OPT_GRAD_REGS = 12,
    AQ_OPT_GRAD_TILE = 13,
    AQ_OPT_TABLE_ONE_LAUNCH = 14
} aq_option;

aq_status aq_layer_set_option(aq_layer* layer, int32_t option, int64_t value);
aq_status aq_layer_get_option(const aq_layer* layer, int32_t option, int64_t* value);

/*
 * Launch timing without a profiler.  After aq_layer_set_launch_events with n
 * events (hipEvent_t handles created by the caller with timing enabled), each
 * later aq_layer_forward, aq_layer_prepare or aq_layer_codebook_grad call on
 * the layer (not aq_layers_prepare, whose launches serve several layers) records
 * events[0] on its stream before its first kernel launch and events[k] right
 * after its k-th launch (k < n; further launches are not bracketed).  Calls
 * on a stream under graph capture record no events (the runtime has no
 * external event nodes).  hipEventElapsedTime(events[k-1], events[k]) is then
 * the duration of launch k (plus the gap before it).  n = 0 stops
 * the recording; n is at most 64.  The events stay owned by the caller and
 * must outlive their use.
 * aq_layer_last_launches reports how many kernels the layer's last forward,
 * prepare or gradient call launched and, in `names` (truncated to names_size - 1 bytes
 * and terminated), their kernels one per line, as name<template arguments>
 * with the arguments as integers (a code type as its bit width).
 */
aq_status aq_layer_set_launch_events(aq_layer* layer, void* const* events, int32_t n_events);
aq_status aq_layer_last_launches(const aq_layer* layer, int32_t* n_launches, char* names, int64_t names_size);

/*
 * Text description of the route a forward over n tokens (linear) or images
 * (conv) would take, as "key=value" pairs: the path and kernel route, and for
 * the matrix-core kernels the weight source (in-loop decode or pre-decoded
 * records, with the bytes the records write), tile, K split, workgroup
 * order and workgroups per compute unit.  Host function: it launches nothing
 * and queries only kernel occupancy on the current device; `buf` receives at
 * most size - 1 characters and a terminating zero.
 */
aq_status aq_layer_describe(const aq_layer* layer, int64_t n, char* buf, int64_t size);

/* The path a forward over `tokens` tokens would take (pure host function). */
aq_status aq_layer_choose_path(const aq_layer* layer, int64_t tokens, aq_path* out);

/* Release the layer's device memory (synchronises the device).  NULL is a no-op. */
aq_status aq_layer_destroy(aq_layer* layer);

/* Message for the last failing call on this thread ("" if none). */
const char* aq_last_error(void);

/* Library version string. */
const char* aq_version(void);

#ifdef __cplusplus
}
#endif

#endif /* AQ_H */
