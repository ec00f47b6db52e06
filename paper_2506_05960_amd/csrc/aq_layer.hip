// C ABI entry points: argument validation (host only, before any HIP call),
// device copies and repacking of the quantized weights, path dispatch.
#include <algorithm>
#include <array>
#include <cmath>
#include <cstdio>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "aq_internal.h"

using aq::DeviceWeights;
using aq::Geom;
using aq::LutPlan;

struct aq_layer {
    aq_layer_desc desc;
    int g, M, B, G;
    int device;
    void* d_cb;
    float* d_cb32;
    void* d_cbtile;
    void* d_cb9;              // g = 9 fp16 codebooks padded to 16 values per row (records kernel)
    void* d_codes;
    uint8_t* d_codes_lut;
    float* d_scales;
    float* d_ws;
    uint32_t* d_lut_arrivals; // table path: arrival counters (zero between launches)
    LutPlan plan;
    aq::FusedPlan fplan;
    uint8_t* d_crec;          // fused-path code records (null when the fused path does not apply)
    void* d_wrec;             // fused-path operand records, decoded per forward in the pre-decoded mode
    void* d_xpack;            // dense product: activations repacked per forward
    void* d_zero;             // 256 zero bytes
    float* d_part;            // fused kernel K split: fp32 partial tiles
    size_t part_bytes;        // bytes at d_part
    uint32_t* d_arrivals;     // fused kernel K split: one arrival counter per tile (zero between launches)
    // codebook gradient, prepared by the first gradient call
    bool grad_ready;
    aq::GradPlan gplan;
    int32_t* d_gidx_offs;     // [M][2^B + 1] list offsets per codebook entry
    int32_t* d_gidx_ent;      // [M][C_out * G] (row, group) pairs i * G + j, sorted by code
    float* d_gpart;           // [s_max][C_out][K] fp32 partial weight gradients
    bool grad_stale;          // a gradient option changed since the plan was made
    size_t gpart_bytes;       // bytes allocated at d_gpart
    bool lut_ok, dec_ok, fused_ok;
    aq_path path;
    int64_t lut_max_tokens;   // the measured rule for this layer
    aq::Options opt;
    std::vector<hipEvent_t> events;   // caller's timing events (aq_layer_set_launch_events)
    int32_t last_launches;            // kernel launches of the last traced call
    std::string last_names;           // and their kernels, one per line
    int64_t prepared_n;               // aq_layer_prepare decoded the records of a forward of this
                                      // many tokens / images into d_wrec (0: none pending)
};

namespace aq {

namespace {

struct LaunchTrace {
    bool active = false;
    const hipEvent_t* ev = nullptr;
    int n_ev = 0;
    int count = 0;
    hipError_t err = hipSuccess;
    std::string names;
};
thread_local LaunchTrace g_trace;

}  // namespace

void note_launch(hipStream_t st, const char* kernel, std::initializer_list<int> template_args) {
    LaunchTrace& t = g_trace;
    if (!t.active) return;
    if (!t.names.empty()) t.names += '\n';
    t.names += kernel;
    if (template_args.size()) {
        t.names += '<';
        bool first = true;
        for (int a : template_args) {
            if (!first) t.names += ", ";
            t.names += std::to_string(a);
            first = false;
        }
        t.names += '>';
    }
    ++t.count;
    if (t.ev && t.count < t.n_ev && t.err == hipSuccess) {
        t.err = hipEventRecordWithFlags(t.ev[t.count], st, 0u);
        if (t.err != hipSuccess) (void)hipGetLastError();
    }
}

hipError_t ensure_dynamic_lds(const void* kernel, size_t bytes) {
    static std::mutex mu;
    static std::map<std::pair<const void*, int>, size_t> done;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(mu);
    size_t& have = done[{kernel, dev}];
    if (bytes <= have) return hipSuccess;
    e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e == hipSuccess) have = bytes;
    return e;
}

}  // namespace aq

namespace {

thread_local std::string g_err;

aq_status fail(aq_status s, const std::string& msg) {
    g_err = msg;
    return s;
}

aq_status hip_fail(hipError_t e, const char* what) {
    if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation)
        return fail(AQ_ERR_OUT_OF_MEMORY, std::string(what) + ": " + hipGetErrorString(e));
    return fail(AQ_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

// Starts the launch trace of one entry-point call: event 0 is recorded on the
// call's stream before its first launch.  A stream under graph capture gets
// no event records (this runtime has no external event nodes).  A failed
// record is reported by the entry point and cleared from the runtime's
// last-error state, which the launchers read.
struct TraceScope {
    aq_layer* L;
    explicit TraceScope(aq_layer* layer, hipStream_t st) : L(layer) {
        aq::LaunchTrace& t = aq::g_trace;
        t = aq::LaunchTrace{};
        t.active = true;
        t.ev = L->events.empty() ? nullptr : L->events.data();
        t.n_ev = (int)L->events.size();
        if (t.ev) {
            hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
            t.err = hipStreamIsCapturing(st, &cs);
            if (t.err == hipSuccess && cs != hipStreamCaptureStatusNone) t.ev = nullptr;
            if (t.err == hipSuccess && t.ev) t.err = hipEventRecordWithFlags(t.ev[0], st, 0u);
            if (t.err != hipSuccess) (void)hipGetLastError();
        }
    }
    hipError_t error() const { return aq::g_trace.err; }
    ~TraceScope() {
        aq::LaunchTrace& t = aq::g_trace;
        L->last_launches = t.count;
        L->last_names = t.names;
        t.active = false;
        t.ev = nullptr;
    }
};

size_t dtype_bytes(int dt) {
    switch (dt) {
    case AQ_F32: return 4;
    case AQ_F16:
    case AQ_BF16: return 2;
    default: return 1;
    }
}

bool is_conv(const aq_layer_desc& d) { return d.conv_kh != 0 || d.conv_kw != 0; }

int conv_out(int in, int pad, int k, int stride) { return (in + 2 * pad - k) / stride + 1; }

aq_status validate_desc(const aq_layer_desc* d, int g, int M, int B) {
    if (g < 1 || g > 16) return fail(AQ_ERR_INVALID_ARGUMENT, "g must be in [1, 16]");
    if (M < 1 || M > 8) return fail(AQ_ERR_INVALID_ARGUMENT, "M must be in [1, 8]");
    if (B < 1 || B > 16) return fail(AQ_ERR_INVALID_ARGUMENT, "B must be in [1, 16]");
    if (d->out_features < 1) return fail(AQ_ERR_INVALID_ARGUMENT, "out_features must be >= 1");
    if (d->in_features < 1) return fail(AQ_ERR_INVALID_ARGUMENT, "in_features must be >= 1");
    if (d->in_features % g != 0) return fail(AQ_ERR_INVALID_ARGUMENT, "in_features must be a multiple of g");
    if (d->codebook_dtype != AQ_F32 && d->codebook_dtype != AQ_F16 && d->codebook_dtype != AQ_BF16)
        return fail(AQ_ERR_INVALID_ARGUMENT, "codebook_dtype must be F32, F16 or BF16");
    if (d->x_dtype < AQ_F32 || d->x_dtype > AQ_I8) return fail(AQ_ERR_INVALID_ARGUMENT, "bad x_dtype");
    if (d->y_dtype != AQ_F32 && d->y_dtype != AQ_F16) return fail(AQ_ERR_INVALID_ARGUMENT, "y_dtype must be F32 or F16");
    if (d->tile_dtype != AQ_F32 && d->tile_dtype != AQ_F16 && d->tile_dtype != AQ_BF16)
        return fail(AQ_ERR_INVALID_ARGUMENT, "tile_dtype must be F32, F16 or BF16");
    if (d->max_tokens < 1) return fail(AQ_ERR_INVALID_ARGUMENT, "max_tokens must be >= 1");
    if (is_conv(*d)) {
        if (d->conv_kh < 1 || d->conv_kw < 1 || d->conv_cin < 1 || d->conv_stride < 1 || d->conv_pad < 0 ||
            d->in_h < 1 || d->in_w < 1)
            return fail(AQ_ERR_INVALID_ARGUMENT, "bad convolution geometry");
        if ((int64_t)d->conv_cin * d->conv_kh * d->conv_kw != d->in_features)
            return fail(AQ_ERR_INVALID_ARGUMENT, "in_features must equal conv_cin*conv_kh*conv_kw");
        if (d->in_h + 2 * d->conv_pad < d->conv_kh || d->in_w + 2 * d->conv_pad < d->conv_kw)
            return fail(AQ_ERR_INVALID_ARGUMENT, "convolution output would be empty");
        if (d->x_dtype == AQ_I8)
            return fail(AQ_ERR_UNSUPPORTED, "int8 activations are supported for linear layers only");
    }
    return AQ_OK;
}

Geom make_geom(const aq_layer* L, int64_t n) {
    Geom geo{};
    const aq_layer_desc& d = L->desc;
    geo.C_out = d.out_features;
    geo.K = d.in_features;
    geo.g = L->g;
    geo.M = L->M;
    geo.B = L->B;
    geo.G = L->G;
    geo.conv = is_conv(d);
    if (geo.conv) {
        geo.cin = d.conv_cin;
        geo.kh = d.conv_kh;
        geo.kw = d.conv_kw;
        geo.stride = d.conv_stride;
        geo.pad = d.conv_pad;
        geo.H = d.in_h;
        geo.W = d.in_w;
        geo.OH = conv_out(d.in_h, d.conv_pad, d.conv_kh, d.conv_stride);
        geo.OW = conv_out(d.in_w, d.conv_pad, d.conv_kw, d.conv_stride);
        geo.tokens = n * (int64_t)geo.OH * geo.OW;
    } else {
        geo.tokens = n;
    }
    return geo;
}

aq_path choose(const aq_layer* L, int64_t tokens) {
    if (L->path != AQ_PATH_AUTO) return L->path;
    const int64_t lim = L->opt.lut_max_tokens == 0 ? L->lut_max_tokens : L->opt.lut_max_tokens < 0 ? 0
                                                                                                     : L->opt.lut_max_tokens;
    if (L->lut_ok && (!L->dec_ok || tokens <= lim)) return AQ_PATH_LUT;
    return AQ_PATH_DECODE;
}

void free_layer(aq_layer* L) {
    if (!L) return;
    void* ptrs[] = {L->d_cb,     L->d_cb32, L->d_cbtile, L->d_codes, L->d_codes_lut, L->d_scales,
                    L->d_ws,     L->d_crec, L->d_wrec,   L->d_xpack, L->d_zero, L->d_gidx_offs,
                    L->d_gidx_ent, L->d_gpart, L->d_part, L->d_arrivals, L->d_lut_arrivals, L->d_cb9};
    for (void* p : ptrs)
        if (p) (void)hipFree(p);
    delete L;
}

template <typename T>
aq_status dev_upload(T** dst, const void* src, size_t bytes, const char* what) {
    hipError_t e = hipMalloc(reinterpret_cast<void**>(dst), bytes);
    if (e != hipSuccess) {
        *dst = nullptr;
        return hip_fail(e, what);
    }
    if (src) {
        e = hipMemcpy(*dst, src, bytes, hipMemcpyHostToDevice);
        if (e != hipSuccess) return hip_fail(e, what);
    }
    return AQ_OK;
}

// ---- fused decode + matrix-core path: eligibility, code records, tiles ----

constexpr size_t kLdsBytes = 160 * 1024;

// Decide whether the fused path applies and fill the create-time part of the plan.
// LUT blocking: a chunk of jc groups with jc*M a multiple of 16 (one or more
// 16-byte code runs per row), its table (jc*M slots x 256 entries x NT fp32)
// within 64 KB at the largest token count per entry that fits, and never
// above 144 KB.
bool lut_plan_create(const aq_layer_desc& d, int g, int M, int G, LutPlan* p) {
    int q = 16;
    for (int m = M; m % 2 == 0 && q > 1; m /= 2) q /= 2;        // 16 / gcd(M, 16)
    const size_t slot_bytes = (size_t)256 * sizeof(float);      // per token
    int nt = 4;
    while (nt > 1 && (size_t)q * M * slot_bytes * nt > 144 * 1024) nt /= 2;
    if ((size_t)q * M * slot_bytes * nt > 144 * 1024) return false;
    int jc = q;
    while ((size_t)(jc + q) * M * slot_bytes * nt <= 64 * 1024 && jc + q <= (G + q - 1) / q * q) jc += q;
    p->jc = jc;
    p->nchunk = (G + jc - 1) / jc;
    p->nt_max = nt;
    p->mfma_table = d.codebook_dtype == AQ_F16 && (d.x_dtype == AQ_F16 || d.x_dtype == AQ_I8) && g == 8;
    int64_t tb = std::min<int64_t>(d.max_tokens, 32);   // the table path serves few tokens per launch
    p->tok_block = (int)((tb + 3) / 4 * 4);
    // 32-bit code and partial-sum offsets in the kernel
    return (int64_t)p->nchunk * d.out_features * jc * M < (int64_t(1) << 31) &&
           (int64_t)p->nchunk * p->tok_block * d.out_features * 4 < (int64_t(1) << 31);
}

bool fused_plan_create(const aq_layer_desc& d, int g, int M, int B, aq::FusedPlan* p) {
    std::memset(p, 0, sizeof(*p));
    if (d.tile_dtype != AQ_F16 || (g != 8 && g != 9)) return false;
    const bool conv = is_conv(d);
    if (g == 9 && !(conv && d.conv_kh == 3 && d.conv_kw == 3)) return false;   // g = 9: one 3x3 filter per group
    if (conv) {
        if (d.x_dtype != AQ_F16 || d.in_w % 2 != 0) return false;
        if (d.conv_kh == 3 && d.conv_kw == 3 && d.conv_cin % 16 == 0) {
            p->kind = 1;
            p->cm = 1;
            p->nchunk = d.conv_cin / 16;
        } else if (d.conv_kh == 1 && d.conv_kw == 1 && d.conv_pad == 0 && d.conv_cin % 64 == 0) {
            p->kind = 2;
            p->cm = 4;
            p->nchunk = d.conv_cin / 64;
        } else {
            return false;
        }
    } else {
        if (d.x_dtype != AQ_F16 && d.x_dtype != AQ_I8) return false;
        p->kind = 0;
        p->cm = 4;
        p->nchunk = (d.in_features + 63) / 64;
    }
    if (g == 8 && (M == 2 || M == 4) && B <= 8 && d.codebook_dtype == AQ_F16) {
        p->dec = aq::FUSED_DEC_PK16;
        p->cb_bytes = M * 256 * 16;             // LDS keeps 256 rows per codebook
    } else if (g == 8 && M == 1 && B > 8 && d.codebook_dtype == AQ_F16) {
        p->dec = aq::FUSED_DEC_T16G;
        p->cb_bytes = 0;
    } else {
        // any other codebook count, size or dtype, and g = 9: operands decoded
        // once per forward by the records kernel
        p->dec = aq::FUSED_DEC_REC;
        p->cb_bytes = 0;
        p->rec_only = 1;
    }
    p->mc = M;
    const int ns = p->kind == 1 ? 9 : p->cm;
    const int ent_b = p->dec == aq::FUSED_DEC_T16G ? 2 : 1;
    p->rec_bytes = (ns * M * ent_b + 3) / 4 * 4;
    return true;
}

// Code records: for chunk c, output channel n and lane half q, the M codes of
// every group the lane decodes, in decode order (8-bit codes, or 16-bit codes
// when B > 8), padded to whole dwords.
std::vector<uint8_t> fused_records(const aq::FusedPlan& p, const void* codes, int C_out, int G, int M, int B) {
    const int ns = p.kind == 1 ? 9 : p.cm;
    const int ent_b = p.dec == aq::FUSED_DEC_T16G ? 2 : 1;
    std::vector<uint8_t> rec((size_t)p.nchunk * C_out * 2 * p.rec_bytes, 0);
    for (int c = 0; c < p.nchunk; ++c)
        for (int n = 0; n < C_out; ++n)
            for (int q = 0; q < 2; ++q) {
                uint8_t* r = rec.data() + (((size_t)c * C_out + n) * 2 + q) * p.rec_bytes;
                for (int s = 0; s < ns; ++s) {
                    const int j = p.kind == 1 ? 18 * c + 9 * q + s : c * 2 * p.cm + 2 * s + q;
                    if (j >= G) continue;
                    for (int m = 0; m < M; ++m) {
                        const size_t src = ((size_t)n * G + j) * M + m;
                        if (ent_b == 1) r[s * M + m] = static_cast<const uint8_t*>(codes)[src];
                        else std::memcpy(r + 2 * (s * M + m), static_cast<const uint16_t*>(codes) + src, 2);
                    }
                }
            }
    return rec;
}

struct TileCand {
    int bm, bn, upl;
};

// Per-forward tile choice; fills the remaining plan fields.  Returns false when
// no instantiated tile fits (the caller then uses the generic kernel).
// K split over workgroups (fused kernel): a layer whose tiles do not fill one
// round of the compute units may give each tile to S workgroups that share its
// K chunks.  Cost per workgroup in chunk-time units: the chunks of one wave,
// plus the fixed prologue and epilogue, plus one for publishing and summing the
// partial tiles.  Layers that fill the chip keep the fitted model (fixed cost
// about three chunks); for under-filled layers (fewer than 256 tiles of 64 x 64)
// the fixed cost measured about twelve chunks on the U-Net's 512-token
// convolutions, and the in-loop decode's codeword gathers (per output channel
// and codebook) weigh against the products (per token and channel) by a factor
// 1 + M 32 / BM (measured: M = 2 favours 64 x 64 tiles, M = 4 128 x 64).
constexpr double kFixedChunks = 3.0;
constexpr double kFixedChunksUnderfilled = 12.0;
constexpr double kSplitChunks = 1.0;

// Fewer than 256 tiles of 64 tokens x 64 channels: the layer cannot fill the chip.
bool underfilled(const Geom& geo) {
    return ((geo.tokens + 63) / 64) * (int64_t)((geo.C_out + 63) / 64) < 256;
}

// Workgroups of one fused-kernel instantiation that a compute unit holds at once
// (registers and LDS), as the runtime reports it; cached per device and
// instantiation, 1 where the query fails.
int fused_occupancy(const Geom& geo, const aq::FusedPlan& q, int x_dtype) {
    static std::mutex mu;
    static std::map<std::array<int64_t, 11>, int> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 1;
    const std::array<int64_t, 11> key{dev,  q.kind, q.cm, x_dtype, q.dec, q.mc, q.bm, q.bn, q.upl, (int64_t)q.lds_bytes,
                                      q.wsplit * 16 + q.rdepth};
    {
        std::lock_guard<std::mutex> lock(mu);
        auto it = cache.find(key);
        if (it != cache.end()) return it->second;
    }
    int occ = 0;
    aq::FusedLaunch fl{};
    fl.x_dtype = x_dtype;
    fl.occupancy = &occ;
    const hipError_t e = q.wsplit ? aq::launch_rec_conv(geo, q, fl) : aq::launch_fused_forward(geo, q, fl);
    if (e != hipSuccess || occ < 1) {
        (void)hipGetLastError();
        occ = 1;
    }
    std::lock_guard<std::mutex> lock(mu);
    cache[key] = occ;
    return occ;
}

// Time of `n` workgroups on one compute unit that holds `occ` at once, each
// with `loop` units of main-loop work and `fixed` of prologue and epilogue:
// workgroups sharing a compute unit share its matrix and LDS throughput in the
// main loop (each one more adds 0.9 of its loop time) and hide each other's
// fixed costs (fitted to forced-tile timings of the U-Net's convolutions at
// 512 to 32768 tokens, both weight modes, M = 2 and 4).
constexpr double kShareLoop = 0.9;
constexpr double kShareFixed = 0.0;

double cu_time(int64_t n, int occ, double loop, double fixed) {
    auto together = [&](int64_t k) {
        return k > 0 ? loop * (1.0 + kShareLoop * (double)(k - 1)) + fixed * (1.0 + kShareFixed * (double)(k - 1))
                     : 0.0;
    };
    return (double)(n / occ) * together(occ) + together(n % occ);
}

// Staging geometry of a convolution tile of `bm` output pixels: the input
// rows it reads (each input row once per block of output rows of one image: a
// tile of whole images, or of consecutive rows of one image; kh rows per output
// row when that stages fewer rows or AQ_OPT_STAGE_ROWS = 1), their padded width,
// and the staging units (plane of 8 channels, staged row, pixel pair).  With
// `widen`, a staged row is widened until consecutive output rows start OW
// 16-byte slots apart (mod 64 banks), which makes A-fragment reads of rows
// shorter than 16 tokens conflict free.  False when bm and OW do not tile
// each other.
bool conv_staging(const Geom& geo, const aq::Options& opt, int kind, int cm, int bm, bool widen, aq::FusedPlan* q) {
    if (!(bm % geo.OW == 0 || geo.OW % bm == 0)) return false;
    const int tr = bm >= geo.OW ? bm / geo.OW : 1;
    const int kh = kind == 1 ? 3 : 1;
    const int img = geo.OH * geo.OW;
    int rpb = 1;
    if (opt.stage_rows != 1) {
        if (bm % img == 0) rpb = geo.OH;
        else if (img % bm == 0 && tr > 1) rpb = tr;
    }
    int sr = (rpb - 1) * geo.stride + kh;
    if (rpb > 1 && (tr / rpb) * sr >= tr * kh) {
        rpb = 1;
        sr = kh;
    }
    q->rpb = rpb;
    q->sr = sr;
    q->inv_rpb = 1.0f / (float)rpb;
    q->inv_sr = 1.0f / (float)sr;
    q->pr = (tr / rpb) * sr;
    q->pw = geo.W + 2 * geo.pad;
    // consecutive output rows of a block are `stride` staged rows apart (kh
    // apart with one output row per block)
    const int rstep = rpb > 1 ? geo.stride : kh;
    if (widen)
        while ((rstep * q->pw - geo.OW) % 16 != 0) ++q->pw;
    q->ps = q->pr * q->pw * 16;                    // one plane of 8 channels
    q->units = 2 * cm * q->pr * (geo.W / 2);       // (plane, row, pixel pair)
    q->total_rows = (int)(geo.tokens / geo.OW);
    q->inv_ow = 1.0f / (float)geo.OW;
    q->inv_oh = 1.0f / (float)geo.OH;
    q->inv_pr = 1.0f / (float)q->pr;
    q->inv_wp = 1.0f / (float)(geo.W / 2);
    return true;
}

bool fused_plan_tile(const Geom& geo, const aq::Options& opt, size_t part_cap, int x_dtype, aq::FusedPlan* p) {
    static const TileCand conv3[] = {{64, 96, 3}, {64, 64, 3}, {128, 64, 3}, {128, 64, 6}, {64, 64, 6}};
    static const TileCand conv1[] = {{64, 96, 4}, {64, 64, 4}};
    static const TileCand lin[] = {{64, 96, 8}, {64, 64, 8}, {32, 128, 4}, {32, 64, 4}};
    const TileCand* cands = p->kind == 1 ? conv3 : p->kind == 2 ? conv1 : lin;
    const int ncand = p->kind == 1 ? 5 : p->kind == 2 ? 2 : 4;
    const int want_bm = opt.fused_bm, want_bn = opt.fused_bn;
    double best = 0;
    aq::FusedPlan bestp{};
    bool found = false;
    // Output rows shorter than 16 tokens put two rows in one 16-lane group of an
    // A-fragment read; a staged row widened until consecutive rows start OW
    // 16-byte slots apart (mod 64 banks) makes those reads conflict free.  Each
    // tile is tried widened and, at a cost penalty, as is.
    const bool narrow = p->kind != 0 && geo.OW < 16 && geo.stride == 1;
    for (int ci = 0; ci < 2 * ncand; ++ci) {
        const int i = ci % ncand;
        const bool widen = ci < ncand;
        if (widen && !narrow) continue;
        const TileCand& t = cands[i];
        if (want_bm && (t.bm != want_bm || t.bn != want_bn)) continue;
        aq::FusedPlan q = *p;
        q.bm = t.bm;
        q.bn = t.bn;
        q.upl = t.upl;
        if (p->kind != 0) {
            if (!conv_staging(geo, opt, p->kind, p->cm, t.bm, widen, &q)) continue;
        } else {
            q.pr = q.pw = 0;
            q.sr = q.rpb = 1;
            q.inv_ow = q.inv_oh = q.inv_pr = q.inv_wp = q.inv_sr = q.inv_rpb = 0.0f;
            q.ps = t.bm * 16 + 16;                      // one plane of 8 consecutive k
            q.units = t.bm * 2 * p->cm;                 // (token, plane)
            q.total_rows = 0;
        }
        q.pbuf_bytes = 2 * p->cm * q.ps + 32;       // + a spare slot for padding units
        if ((q.units + 63) / 64 > t.upl) continue;
        const size_t rows = p->kind != 0 ? t.bn : t.bm, cols = p->kind != 0 ? t.bm : t.bn;
        const size_t red = (size_t)4 * (rows / 4) * (cols + 1) * 16;       // four padded partial tiles
        q.lds_bytes = (size_t)p->cb_bytes + std::max<size_t>((size_t)8 * q.pbuf_bytes, red);
        if (q.lds_bytes > kLdsBytes) continue;
        const int64_t nwg = ((geo.tokens + t.bm - 1) / t.bm) * (int64_t)((geo.C_out + t.bn - 1) / t.bn);
        // convolutions: workgroups per compute unit (the grid spread over 256) timed
        // by cu_time; linear layers' tile costs were fitted with one workgroup per
        // compute unit and keep that model
        const int occ = p->kind != 0 ? fused_occupancy(geo, q, x_dtype) : 1;
        // each workgroup weighted by a per-tile overhead term; linear layers also
        // weigh the staging units per lane (fitted to measured tiles)
        double tcost = (double)t.bm * t.bn * (1.0 + 48.0 / t.bm + 48.0 / t.bn);
        if (p->kind == 0) tcost *= t.upl / (t.upl + 2.0);
        // pre-decoded operands of a linear layer: the 64 x 64 tile measured best
        if (p->kind == 0 && p->dec == aq::FUSED_DEC_REC && !(t.bm == 64 && t.bn == 64)) tcost *= 1.25;
        if (narrow && !widen) tcost *= 1.15;             // bank conflicts on the A-fragment reads (measured)
        const bool under = underfilled(geo);
        if (under && p->dec == aq::FUSED_DEC_PK16) tcost *= 1.0 + 32.0 * p->mc / t.bm;
        for (int S = 1; S <= aq::kMaxSplitK; ++S) {
            if (opt.split_k != 0 && S != opt.split_k && !(S == 1 && opt.split_k > 1)) continue;
            if (S > 1) {
                if (opt.split_k == 0 && (!under || nwg * S > 256)) continue;   // planner: one round, under-filled layers
                if (4 * S > p->nchunk) continue;                                 // every wave keeps a chunk
                if ((size_t)S * nwg * t.bm * t.bn * 4 > part_cap) continue;
                if (nwg * S >= (int64_t(1) << 24)) continue;
            }
            const double cpw = std::ceil((double)p->nchunk / (4.0 * S)) + (S > 1 ? kSplitChunks : 0.0);
            double cost = tcost * cu_time((nwg * S + 255) / 256, occ, cpw,
                                          under ? kFixedChunksUnderfilled : kFixedChunks);
            // a forced split wins over the unsplit fallback of the same tile
            if (opt.split_k > 1 && S == 1) cost *= 1e6;
            if (!found || cost < best) {
                best = cost;
                bestp = q;
                bestp.splitk = S;
                bestp.ntiles = (int)nwg;
                bestp.inv_ntiles = 1.0f / (float)nwg;
                found = true;
            }
        }
    }
    if (!found && want_bm) {
        aq::Options o = opt;
        o.fused_bm = o.fused_bn = 0;      // the forced tile does not fit: the planner's choice
        return fused_plan_tile(geo, o, part_cap, x_dtype, p);
    }
    if (found) *p = bestp;
    return found;
}

// Tile of the dense product over pre-decoded records: the workgroup stages
// each chunk's activations (all BM tokens) and weight records (BN channels)
// in two LDS stages.  Returns false when no tile fits.
bool gemm_plan_tile(const Geom& geo, const aq::Options& opt, aq::FusedPlan* p) {
    static const TileCand cands[] = {{128, 128, 0}, {128, 64, 0}, {64, 128, 0}};
    const int want_bm = opt.dense_bm, want_bn = opt.dense_bn;
    double best = 0;
    aq::FusedPlan bestp{};
    bool found = false;
    for (const TileCand& t : cands) {
        if (want_bm && (t.bm != want_bm || t.bn != want_bn)) continue;
        aq::FusedPlan q = *p;
        q.bm = t.bm;
        q.bn = t.bn;
        if (p->kind != 0) {
            if (!(t.bm % geo.OW == 0 || geo.OW % t.bm == 0)) continue;
            const int kh = p->kind == 1 ? 3 : 1;
            const int tr = t.bm >= geo.OW ? t.bm / geo.OW : 1;
            const int64_t rows_total = geo.tokens / geo.OW;
            const int64_t ntm = (geo.tokens + t.bm - 1) / t.bm;
            int ni = 1;                                      // most images one tile's rows span
            for (int64_t m = 0; m < std::min<int64_t>(ntm, 4 * geo.OH + 4); ++m) {
                const int64_t g0 = m * t.bm / geo.OW;
                const int64_t gl = std::min<int64_t>((m * t.bm + t.bm - 1) / geo.OW, rows_total - 1);
                ni = std::max<int>(ni, (int)(gl / geo.OH - g0 / geo.OH + 1));
            }
            const int rpi = (std::min(tr, geo.OH) - 1) * geo.stride + kh;
            const int planes = p->kind == 1 ? 2 : 8;
            // staged rows `stride` apart per output row: widen so that two rows in one
            // 16-lane fragment read fall on different banks when an output row is short
            int pw = geo.W + 2 * geo.pad;
            if (geo.OW < 16) {
                int w = pw;
                while ((geo.stride * w - geo.OW) % 16 != 0 && w < pw + 16) ++w;
                if ((geo.stride * w - geo.OW) % 16 == 0 && (int64_t)planes * ni * rpi * w <= 1024) pw = w;
            }
            if ((int64_t)planes * ni * rpi * pw > 1024) continue;
            q.pr = ni;
            q.ps = rpi;
            q.pw = pw;
        }
        q.lds_bytes = aq::rec_gemm_lds_bytes(p->kind, t.bm, t.bn);
        if (q.lds_bytes > kLdsBytes) continue;
        const int64_t nwg = ((geo.tokens + t.bm - 1) / t.bm) * (int64_t)((geo.C_out + t.bn - 1) / t.bn);
        const int64_t rounds = (nwg + 255) / 256;
        const double cost = (double)rounds * t.bm * t.bn * (1.0 + 64.0 / t.bm + 64.0 / t.bn);
        if (!found || cost < best) {
            best = cost;
            bestp = q;
            found = true;
        }
    }
    if (found) *p = bestp;
    return found;
}

// Pre-decoded mode (operands decoded once per forward into records the main
// loop reads with plain 16-byte loads) instead of decoding inside the main
// loop: chosen for codebooks too large for LDS (their codeword reads from L2
// repeat for every token tile) once there are enough token tiles to repay the
// extra pass.  Option AQ_OPT_WEIGHTS = 2 / 1 forces it on / off.
bool use_predecoded(const aq_layer* L, const Geom& geo) {
    if (L->fplan.rec_only) return true;
    if (L->opt.weights != 0) return L->opt.weights == 2;
    const int64_t token_tiles = (geo.tokens + 63) / 64;
    const aq::FusedPlan& p = L->fplan;
    if (p.dec == aq::FUSED_DEC_T16G) return token_tiles >= 8;
    // measured on the U-Net layer shapes: the in-loop decode is repeated for every
    // token tile, so the single decode pass wins once tokens x M is large enough
    const int64_t tm = geo.tokens * p.mc;
    // under-filled convolutions with K to split: the in-loop decode with a K split
    // over workgroups (no record pass) measured faster on the U-Net's 512-token
    // 3x3 layers for M = 2 and 4 (8 x 8 level, K = 8640: 21.8 / 27.1 us against
    // 29.5 in-loop unsplit and 32.8 with records)
    if (p.kind != 0 && p.dec == aq::FUSED_DEC_PK16 && underfilled(geo) && p.nchunk >= 8) return false;
    if (p.kind == 1) {
        // 3x3 convolutions of the U-Net shapes (both routes timed per shape): with
        // M = 4 the pre-decoded route won on every shape from 512 tokens up; with
        // M = 2 once the reduction is long for the token count (conv64, 8192
        // tokens x K = 1728, stays in-loop: 13.5 vs 15.1 us)
        if (p.mc >= 4 && geo.tokens >= 512) return true;
        return tm >= 32768 || (geo.K >= 3456 && geo.tokens >= 8192) || (geo.K >= 5000 && geo.tokens >= 2048) ||
               geo.K >= 13000;
    }
    if (p.kind == 0) {
        if (aq::rec_linear_supported(geo, p, L->desc.x_dtype)) {
            // the wave-split product over records (measured on the U-Net linear shapes):
            // faster once its 128 x 128 tiles cover three quarters of the compute units,
            // at 2048 tokens and up or M >= 4 (the in-loop decode then gathers 4 codewords
            // per group); with fewer tiles the in-loop decode's K split keeps more units busy
            const int64_t tiles = ((geo.tokens + 127) / 128) * (int64_t)((geo.C_out + 127) / 128);
            return tiles >= 192 && (geo.tokens >= 2048 || p.mc >= 4);
        }
        return p.mc >= 4 && geo.C_out >= 1152 && geo.tokens >= 2048;
    }
    return p.mc >= 4 && geo.tokens >= 32768;
}

// The route of one forward, resolved on the host (shared by the forward and
// aq_layer_describe).
// The 2 x 2 wave-split records kernel for a 3x3 or 1x1 convolution, `wk`
// waves per reduction: a 128-token tile (wk = 1) or a 64-token tile whose
// two channel halves each take every other chunk in two waves (wk = 2); 192
// channels where C_out is a multiple of 192 (else 128); and its staging.
// AQ_OPT_FUSED_TILE picks 128 or 192 channels when its token count matches.
// False where the kernel does not apply (tile rows, image planes not a
// multiple of 4 tokens, more staging units than instantiated).
bool wsplit_plan(const Geom& geo, const aq::Options& opt, int wk, aq::FusedPlan* p) {
    if (p->dec != aq::FUSED_DEC_REC || !(p->kind == 1 || (p->kind == 2 && p->cm == 4))) return false;
    if ((geo.OH * geo.OW) % 4 != 0 || geo.W % 2 != 0) return false;
    const int bm = wk == 1 ? 128 : 64;
    aq::FusedPlan q = *p;
    if (!conv_staging(geo, opt, p->kind, p->cm, bm, false, &q)) return false;
    q.upl = (wk * q.units + 255) / 256;
    if (p->kind == 1 ? q.upl > 3 : q.upl != 2) return false;
    int bn = geo.C_out % 192 == 0 ? 192 : 128;
    if (opt.fused_bm == bm && (opt.fused_bn == 128 || opt.fused_bn == 192)) bn = opt.fused_bn;
    if (p->kind == 1 && wk == 2 && bn == 192 && q.upl > 2) bn = 128;   // registers (see the launcher)
    q.bm = bm;
    q.bn = bn;
    q.wsplit = 1;
    // 3x3: records five steps ahead (six register sets) where the registers
    // allow (not with the two-wave reduction); 1x1: three steps ahead
    q.rdepth = p->kind == 2 ? 4 : wk == 2 || (bn == 192 && q.upl > 1) ? 3 : 6;
    q.splitk = 1;
    q.pbuf_bytes = 2 * p->cm * q.ps + 32;        // the chunk's planes and a spare slot
    // staging: two buffers per chunk of an iteration; wk = 2: then the partial
    // tiles of the second reduction half (4 KB per 32 x 32 block)
    const size_t red = wk == 2 ? (size_t)2 * 2 * (bn / 64) * 4 * 64 * 16 : 0;
    q.lds_bytes = std::max((size_t)2 * wk * q.pbuf_bytes, red);
    if (q.lds_bytes > kLdsBytes) return false;
    const int64_t nt = ((geo.tokens + bm - 1) / bm) * (int64_t)((geo.C_out + bn - 1) / bn);
    if (nt >= (int64_t(1) << 24)) return false;
    q.ntiles = (int)nt;
    q.inv_ntiles = 1.0f / (float)nt;
    *p = q;
    return true;
}

struct Route {
    enum Kind { LUT = 0, F32 = 1, GENERIC = 2, DENSE = 3, FUSED = 4, REC_LINEAR = 5, NONE = 6 } kind;
    aq::FusedPlan fp;
};

Route plan_route(const aq_layer* L, const Geom& geo) {
    Route r{};
    const aq_layer_desc& d = L->desc;
    if (choose(L, geo.tokens) == AQ_PATH_LUT) {
        r.kind = Route::LUT;
        return r;
    }
    if (d.tile_dtype == AQ_F32) {
        r.kind = Route::F32;
        return r;
    }
    const aq::Options& opt = L->opt;
    aq::FusedPlan fp = L->fplan;
    // the fused kernel uses 32-bit element and byte offsets
    const int64_t nimg = geo.conv ? geo.tokens / ((int64_t)geo.OH * geo.OW) : 0;
    const bool fits31 = geo.tokens * (int64_t)std::max(geo.K, geo.C_out) * 4 < (int64_t(1) << 31) &&
                        (!geo.conv || nimg * (int64_t)geo.cin * geo.H * geo.W * 2 < (int64_t(1) << 31));
    if (L->fused_ok && use_predecoded(L, geo)) {
        // pre-decoded mode: operands decoded once per forward, then read with plain loads
        fp.dec = aq::FUSED_DEC_REC;
        fp.mc = 1;
        fp.cb_bytes = 0;
    }
    auto order = [&opt](aq::FusedPlan& q) {
        // channel-major order for pre-decoded convolution operands; linear layers
        // measured faster token-major (qkv 8192 x 576 -> 1728: 59.5 vs 61.8 us)
        q.nmajor = q.dec == aq::FUSED_DEC_REC && q.kind != 0;
        if (opt.tile_order != 0) q.nmajor = opt.tile_order == 2;
    };
    aq::FusedPlan gp = fp;
    // dense product over the records: a comparator route (AQ_OPT_RECORD_PRODUCT = 2);
    // measured slower than the fused kernel's pre-decoded mode on most layer shapes here
    if (L->fused_ok && fits31 && fp.dec == aq::FUSED_DEC_REC && opt.rec_product == 2 && gemm_plan_tile(geo, opt, &gp)) {
        order(gp);
        r.kind = Route::DENSE;
        r.fp = gp;
        return r;
    }
    // Convolutions on the wave-split records kernel where its tiles fill the
    // chip (measured on the U-Net shapes, records included):
    //  * 128-token tiles (one wave per reduction) for 3x3 layers with at least
    //    192 of them (20-25 % faster than the fused kernel's best tile at 32768
    //    tokens) and 1x1 layers with at least 256 (24.0 -> 17.6 us at 32768
    //    tokens x 384 -> 192 channels, M = 2);
    //  * else 64-token tiles with two waves per reduction where there are at
    //    least 256 of them and every wave keeps 4 chunks or more (8192 tokens
    //    x 384 channels: 3-8 % faster than the fused kernel, 3x3 and 1x1);
    //  * else, for 1x1 layers with M >= 4, 128-token tiles from 128 of them
    //    (the in-loop decode gathers 4 codewords per group).
    // Fewer tiles leave compute units idle: the fused kernel stays ahead; so
    // does it for output rows under 16 tokens (the rule needs OW >= 16).
    // Layers switch to records for it even where the in-loop decode was chosen
    // (3x3 at 8192 tokens, M = 2: 23.6 -> 20.8 us at K = 1728 -> 192 with
    // stride 2, 24.1 -> 21.7 us at K = 1728 -> 384).  AQ_OPT_RECORD_PRODUCT =
    // 3 forces the kernel where it applies (a forced 64-token AQ_OPT_FUSED_TILE
    // selects the two-wave reduction), 1 and 2 exclude it; AQ_OPT_WEIGHTS = 1
    // keeps a layer on the in-loop decode.
    bool planned = false;
    const bool ws_switch = fp.kind != 0 && fp.dec != aq::FUSED_DEC_REC && opt.weights == 0;
    if (L->fused_ok && fits31 && opt.generic != 1 && fp.kind != 0 && (fp.dec == aq::FUSED_DEC_REC || ws_switch) &&
        (opt.rec_product == 3 || opt.rec_product == 0)) {
        aq::FusedPlan rp = fp;
        rp.dec = aq::FUSED_DEC_REC;
        rp.mc = 1;
        rp.cb_bytes = 0;
        aq::FusedPlan w1 = rp, w2 = rp;
        const bool ok1 = wsplit_plan(geo, opt, 1, &w1), ok2 = wsplit_plan(geo, opt, 2, &w2);
        const aq::FusedPlan* pick = nullptr;
        if (opt.rec_product == 3 && !ws_switch) {
            if (opt.fused_bm == 64 ? ok2 : ok1) pick = opt.fused_bm == 64 ? &w2 : &w1;
        } else if (opt.rec_product == 0 && geo.OW >= 16) {
            // (output rows under 16 tokens: this kernel does not widen its staged
            // rows, and its fragment reads conflict; 8 x 8 images measured slower)
            if (ok1 && w1.ntiles >= (fp.kind == 1 ? 192 : 256)) pick = &w1;
            else if (ok2 && w2.ntiles >= 256 && fp.nchunk >= 8) pick = &w2;
            else if (ok1 && fp.kind == 2 && geo.M >= 4 && w1.ntiles >= 128) pick = &w1;
        }
        if (pick) {
            fp = *pick;
            planned = true;
        }
    }
    if (!planned && L->fused_ok && fits31 && opt.generic != 1)
        planned = fused_plan_tile(geo, opt, L->part_bytes, d.x_dtype, &fp);
    if (planned) {
        order(fp);
        fp.tile_div = fp.nmajor ? (int)((geo.tokens + fp.bm - 1) / fp.bm) : (geo.C_out + fp.bn - 1) / fp.bn;
        fp.inv_tile_div = 1.0f / (float)fp.tile_div;
        fp.rlin_var = aq::rec_linear_tile(geo, opt.rlin_tile);
        // a linear layer's records feed the 2 x 2 wave-split product (AQ_OPT_RECORD_PRODUCT = 1:
        // the fused kernel's own pre-decoded mode, whose partial-tile order matches its in-loop mode)
        const bool rlin = fp.dec == aq::FUSED_DEC_REC && opt.rec_product != 1 && aq::rec_linear_supported(geo, fp, d.x_dtype);
        r.kind = rlin ? Route::REC_LINEAR : Route::FUSED;
        r.fp = fp;
        return r;
    }
    r.kind = geo.g == 8 ? Route::GENERIC : Route::NONE;
    return r;
}

// Where a forward's per-call scratch lives: the layer's workspace, or the
// static array of the allocation-free entry point.
struct Workspace {
    float* lut_ws;            // table path: [chunk groups][tok_block][C_out] partial sums
    uint32_t* lut_arrivals;   // table path: arrival counters
    void* wrec;               // pre-decoded operand records
    float* part;              // fused kernel K split: partial tiles
    uint32_t* arrivals;       // fused kernel K split: arrival counters
    void* xpack;              // dense product: repacked activations
};

aq_status check_forward(const aq_layer* L, const void* X, const float* x_scales, const void* Y, int64_t n, Geom* geo,
                        Route* r) {
    if (!L || !X || !Y) return fail(AQ_ERR_INVALID_ARGUMENT, "null pointer argument");
    if (n < 1) return fail(AQ_ERR_INVALID_ARGUMENT, "n must be >= 1");
    const aq_layer_desc& d = L->desc;
    *geo = make_geom(L, n);
    if (geo->tokens > d.max_tokens) return fail(AQ_ERR_INVALID_ARGUMENT, "tokens exceed max_tokens");
    if (d.x_dtype == AQ_I8 && !x_scales) return fail(AQ_ERR_INVALID_ARGUMENT, "int8 activations need x_scales");
    if ((reinterpret_cast<uintptr_t>(X) | reinterpret_cast<uintptr_t>(Y)) & 15)
        return fail(AQ_ERR_INVALID_ARGUMENT, "X and Y must be 16-byte aligned");
    *r = plan_route(L, *geo);
    if (r->kind == Route::NONE)
        return fail(AQ_ERR_UNSUPPORTED, "g = 9 layers run on the fused kernel only (it was disabled or its "
                                        "tiles do not fit this shape)");
    return AQ_OK;
}

// Whether aq_layer_prepare already decoded this forward's records into the
// layer's own buffer (and the forward uses that buffer).  Any forward on the
// layer's workspace consumes the pending preparation.
bool records_prepared(aq_layer* L, const Workspace& wk, int64_t n) {
    return wk.wrec == L->d_wrec && L->prepared_n == n;
}

aq_status run_route(aq_layer* L, const Geom& geo, const Route& r, const void* X, const float* x_scales, void* Y,
                    int64_t n, hipStream_t st, const Workspace& wk) {
    const aq_layer_desc& d = L->desc;
    const float* xs = d.x_dtype == AQ_I8 ? x_scales : nullptr;
    const DeviceWeights w{L->d_cb,         L->d_cb32,   L->d_cbtile,      L->d_codes,
                          L->d_codes_lut, L->d_scales, d.codebook_dtype, L->d_cb9};
    TraceScope trace(L, st);
    if (trace.error() != hipSuccess) return hip_fail(trace.error(), "launch event");
    hipError_t e = hipSuccess;
    aq::FusedPlan fp = r.fp;
    switch (r.kind) {
    case Route::LUT:
        e = aq::launch_lut_forward(geo, w, L->plan, X, d.x_dtype, xs, Y, d.y_dtype, wk.lut_ws, wk.lut_arrivals,
                                   L->opt.table_one_launch != 0, st);
        break;
    case Route::F32:
        e = aq::launch_f32_forward(geo, w, X, d.x_dtype, xs, Y, d.y_dtype, st);
        break;
    case Route::GENERIC:
        e = aq::launch_mfma_forward(geo, w, X, d.x_dtype, xs, Y, d.y_dtype, d.tile_dtype, st);
        break;
    case Route::DENSE: {
        if (!records_prepared(L, wk, n)) e = aq::launch_operand_records(geo, fp, w, wk.wrec, st);
        const aq::FusedLaunch fl{nullptr, static_cast<const uint8_t*>(wk.wrec), L->d_scales, X, xs, Y,
                                 d.y_dtype, d.x_dtype, st, nullptr, nullptr};
        if (e == hipSuccess) e = aq::launch_rec_gemm(geo, fp, fl, wk.xpack, L->d_zero);
        break;
    }
    default: {   // FUSED, REC_LINEAR
        const void* cbsrc = fp.dec == aq::FUSED_DEC_PK16   ? L->d_cb
                            : fp.dec == aq::FUSED_DEC_F32L ? static_cast<const void*>(L->d_cb32)
                                                           : L->d_cbtile;
        const uint8_t* recs = L->d_crec;
        if (fp.dec == aq::FUSED_DEC_REC) {
            if (!records_prepared(L, wk, n)) e = aq::launch_operand_records(geo, fp, w, wk.wrec, st);
            recs = static_cast<const uint8_t*>(wk.wrec);
        }
        fp.x_bytes = geo.conv ? n * (int64_t)geo.cin * geo.H * geo.W * 2
                              : geo.tokens * (int64_t)geo.K * (d.x_dtype == AQ_I8 ? 1 : 2);
        const aq::FusedLaunch fl{cbsrc, recs, L->d_scales, X, xs, Y, d.y_dtype, d.x_dtype, st, wk.part, wk.arrivals};
        if (e == hipSuccess)
            e = r.kind == Route::REC_LINEAR ? aq::launch_rec_linear(geo, fp, fl)
                : fp.wsplit                  ? aq::launch_rec_conv(geo, fp, fl)
                                             : aq::launch_fused_forward(geo, fp, fl);
        break;
    }
    }
    if (wk.wrec == L->d_wrec) L->prepared_n = 0;
    if (e != hipSuccess) return hip_fail(e, "forward launch");
    if (trace.error() != hipSuccess) return hip_fail(trace.error(), "launch event");
    return AQ_OK;
}

// ---- allocation-free forward: scratch in a static device array ----

constexpr size_t kScratchBytes = size_t(64) << 20;             // per GPU
constexpr size_t kScratchCounterBytes = size_t(256) << 10;     // arrival counters first (table, then K split)
constexpr size_t kScratchLutCounters = 0;
constexpr size_t kScratchSplitCounters = size_t(128) << 10;
constexpr int kScratchMaxDevices = 64;

}  // namespace

// The scratch of aq_layer_forward_static.  Every GPU the library runs on holds
// its own copy until the process ends.  Host code never uses this name as an
// address: the per-device address comes from hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

__global__ void scratch_clear_kernel(uint32_t* p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0u;
}

struct ScratchDev {
    uint8_t* ptr = nullptr;
};
std::mutex g_scratch_mu;
ScratchDev g_scratch[kScratchMaxDevices];

// The current device's scratch address; the first call on a device resolves it
// and clears the counter area with a fill kernel on `st` (a memset could not
// be captured into a graph safely).  The counters return to zero at the end of
// every launch that uses them.
aq_status scratch_for_current_device(hipStream_t st, uint8_t** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kScratchMaxDevices) return fail(AQ_ERR_UNSUPPORTED, "device index beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    ScratchDev& sd = g_scratch[dev];
    if (!sd.ptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "scratch address");
        const int n = (int)(kScratchCounterBytes / 4);
        scratch_clear_kernel<<<(n + 255) / 256, 256, 0, st>>>(static_cast<uint32_t*>(p), n);
        e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "scratch counter clear");
        sd.ptr = static_cast<uint8_t*>(p);
    }
    *out = sd.ptr;
    return AQ_OK;
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

// Lay the route's scratch out in the static array, or refuse.
aq_status static_workspace(const aq_layer* L, const Geom& geo, const Route& r, uint8_t* base, Workspace* wk) {
    *wk = Workspace{};
    uint8_t* data = base + kScratchCounterBytes;
    const size_t cap = kScratchBytes - kScratchCounterBytes;
    size_t used = 0;
    auto take = [&](size_t bytes) {
        uint8_t* p = data + used;
        used += align256(bytes);
        return p;
    };
    if (r.kind == Route::LUT) {
        const LutPlan& p = L->plan;
        if (aq::lut_arrival_count(geo.C_out) * 4 > kScratchSplitCounters - kScratchLutCounters)
            return fail(AQ_ERR_UNSUPPORTED, "static forward: too many table arrival counters (C_out > 16384)");
        wk->lut_arrivals = reinterpret_cast<uint32_t*>(base + kScratchLutCounters);
        wk->lut_ws = reinterpret_cast<float*>(take((size_t)p.nchunk * p.tok_block * geo.C_out * 4));
    } else if (r.kind == Route::FUSED || r.kind == Route::REC_LINEAR || r.kind == Route::DENSE) {
        const aq::FusedPlan& fp = r.fp;
        if (fp.dec == aq::FUSED_DEC_REC) wk->wrec = take(aq::operand_record_bytes(geo, fp));
        if (r.kind == Route::FUSED && fp.splitk > 1) {
            if ((size_t)fp.ntiles * 4 > kScratchCounterBytes - kScratchSplitCounters)
                return fail(AQ_ERR_UNSUPPORTED, "static forward: too many split arrival counters");
            wk->arrivals = reinterpret_cast<uint32_t*>(base + kScratchSplitCounters);
            wk->part = reinterpret_cast<float*>(take((size_t)fp.splitk * fp.ntiles * fp.bm * fp.bn * 4));
        }
        if (r.kind == Route::DENSE) {
            const size_t xp = geo.conv ? (size_t)(geo.tokens / ((int64_t)geo.OH * geo.OW)) * geo.cin * geo.H * geo.W * 2
                                       : L->desc.x_dtype == AQ_I8 ? (size_t)geo.tokens * geo.K * 2 : 0;
            wk->xpack = take(xp);
        }
    }
    if (used > cap)
        return fail(AQ_ERR_UNSUPPORTED, "static forward: needs " + std::to_string(used) + " bytes of scratch, above the " +
                                             std::to_string(cap) + " the static array holds");
    return AQ_OK;
}

}  // namespace

extern "C" {

const char* aq_last_error(void) { return g_err.c_str(); }

const char* aq_version(void) { return "aq-mi355x 0.1.0 (gfx950)"; }

aq_status aq_layer_create(const aq_layer_desc* desc, const void* codebooks, const void* codes, const float* scales,
                          int g, int M, int B, aq_layer** out) {
    g_err.clear();
    if (out) *out = nullptr;
    if (!desc || !codebooks || !codes || !scales || !out)
        return fail(AQ_ERR_INVALID_ARGUMENT, "null pointer argument");
    aq_status st = validate_desc(desc, g, M, B);
    if (st != AQ_OK) return st;

    const int C_out = desc->out_features;
    const int K = desc->in_features;
    const int G = K / g;
    const int64_t nk = (int64_t)1 << B;
    const int64_t ncodes = (int64_t)C_out * G * M;
    if (B <= 8) {
        const uint8_t* c = static_cast<const uint8_t*>(codes);
        for (int64_t i = 0; i < ncodes; ++i)
            if (c[i] >= nk) return fail(AQ_ERR_INVALID_ARGUMENT, "code value >= 2^B at index " + std::to_string(i));
    } else {
        const uint16_t* c = static_cast<const uint16_t*>(codes);
        for (int64_t i = 0; i < ncodes; ++i)
            if (c[i] >= nk) return fail(AQ_ERR_INVALID_ARGUMENT, "code value >= 2^B at index " + std::to_string(i));
    }
    const bool lut_ok = B <= 8;
    aq::FusedPlan fplan;
    const bool fused_ok = fused_plan_create(*desc, g, M, B, &fplan);
    const bool dec_ok = desc->tile_dtype == AQ_F32 || g == 8 || fused_ok;
    if (!lut_ok && !dec_ok)
        return fail(AQ_ERR_UNSUPPORTED, "no kernel for this format: LUT needs B <= 8; the fp16/bf16 decode needs "
                                        "g == 8, or g == 9 on an fp16 3x3 convolution with C_in % 16 == 0");

    int ndev = 0;
    hipError_t e = hipGetDeviceCount(&ndev);
    if (e != hipSuccess || ndev < 1) return fail(AQ_ERR_DEVICE, "no HIP device available");

    aq_layer* L = new aq_layer();
    L->desc = *desc;
    L->g = g;
    L->M = M;
    L->B = B;
    L->G = G;
    L->lut_ok = lut_ok;
    L->dec_ok = dec_ok;
    L->path = AQ_PATH_AUTO;
    // Measured crossover on MI355X (fp16 layers with 256-entry codebooks, codes
    // read from HBM): the table path beats the matrix-core path (which splits
    // such under-filled layers along K) only for long reductions and the
    // fewest tokens: up to 4 tokens with M <= 2, one token with more codebooks
    // (K = 8640 and 17280 to 960 outputs).
    L->lut_max_tokens = desc->in_features >= 4096 ? (M <= 2 ? 4 : 1) : 0;
    e = hipGetDevice(&L->device);
    if (e != hipSuccess) {
        free_layer(L);
        return hip_fail(e, "hipGetDevice");
    }

    const size_t cb_elems = (size_t)M * nk * g;
    const size_t code_bytes = (size_t)ncodes * (B <= 8 ? 1 : 2);
#define AQ_TRY(x)                \
    do {                         \
        aq_status s_ = (x);      \
        if (s_ != AQ_OK) {       \
            free_layer(L);       \
            return s_;           \
        }                        \
    } while (0)
    AQ_TRY(dev_upload(&L->d_cb, codebooks, cb_elems * dtype_bytes(desc->codebook_dtype), "codebooks"));
    AQ_TRY(dev_upload(&L->d_cb32, nullptr, cb_elems * sizeof(float), "codebooks fp32"));
    const bool want_tile_cb = B > 8 && M == 1 && desc->tile_dtype != AQ_F32;
    if (want_tile_cb) AQ_TRY(dev_upload(&L->d_cbtile, nullptr, cb_elems * 2, "codebook tile"));
    if (g == 9 && desc->codebook_dtype == AQ_F16) {
        // 18-byte codewords padded to 32 bytes: one 16- and one 4-byte load each
        std::vector<uint16_t> pad((size_t)M * nk * 16, 0);
        const uint16_t* src = static_cast<const uint16_t*>(codebooks);
        for (size_t r = 0; r < (size_t)M * nk; ++r) std::memcpy(&pad[r * 16], src + r * 9, 9 * sizeof(uint16_t));
        AQ_TRY(dev_upload(&L->d_cb9, pad.data(), pad.size() * sizeof(uint16_t), "padded codebooks"));
    }
    AQ_TRY(dev_upload(&L->d_codes, codes, code_bytes, "codes"));
    AQ_TRY(dev_upload(&L->d_scales, scales, (size_t)C_out * sizeof(float), "scales"));

    if (lut_ok) {
        LutPlan& p = L->plan;
        if (!lut_plan_create(*desc, g, M, G, &p)) {
            free_layer(L);
            return fail(AQ_ERR_UNSUPPORTED, "LUT plan: layer too large for the table kernel");
        }
        const int jc = p.jc;
        // codes regrouped per chunk: [nchunk][C_out][jc*M], zero padded past G
        std::vector<uint8_t> rep((size_t)p.nchunk * C_out * jc * M, 0);
        const uint8_t* c = static_cast<const uint8_t*>(codes);
        for (int i = 0; i < C_out; ++i)
            for (int j = 0; j < G; ++j) {
                const int ch = j / jc, jj = j - ch * jc;
                for (int m = 0; m < M; ++m)
                    rep[(((size_t)ch * C_out + i) * jc + jj) * M + m] = c[((size_t)i * G + j) * M + m];
            }
        AQ_TRY(dev_upload(&L->d_codes_lut, rep.data(), rep.size(), "LUT codes"));
        AQ_TRY(dev_upload(&L->d_ws, nullptr, (size_t)p.nchunk * p.tok_block * C_out * sizeof(float), "workspace"));
        const size_t ncnt = aq::lut_arrival_count(C_out) * sizeof(uint32_t);
        AQ_TRY(dev_upload(&L->d_lut_arrivals, nullptr, ncnt, "table arrival counters"));
        e = hipMemset(L->d_lut_arrivals, 0, ncnt);
        if (e != hipSuccess) {
            free_layer(L);
            return hip_fail(e, "table arrival counters");
        }
    }

    L->fused_ok = fused_ok;
    L->fplan = fplan;
    if (L->fused_ok) {
        if (!fplan.rec_only) {
            std::vector<uint8_t> rec = fused_records(L->fplan, codes, C_out, G, M, B);
            AQ_TRY(dev_upload(&L->d_crec, rec.data(), rec.size(), "fused code records"));
        }
        const Geom g1 = make_geom(L, 1);
        AQ_TRY(dev_upload(&L->d_wrec, nullptr, aq::operand_record_bytes(g1, L->fplan), "operand records"));
        // the dense product's repacked activations (convolution, int8 input) and a zero block
        size_t xpack = 0;
        if (is_conv(*desc)) {
            const int64_t nimg_max = (desc->max_tokens + (int64_t)g1.OH * g1.OW - 1) / ((int64_t)g1.OH * g1.OW);
            xpack = (size_t)nimg_max * desc->conv_cin * desc->in_h * desc->in_w * 2;
        } else if (desc->x_dtype == AQ_I8) {
            xpack = (size_t)desc->max_tokens * K * 2;
        }
        if (xpack) AQ_TRY(dev_upload(&L->d_xpack, nullptr, xpack, "packed activations"));
        AQ_TRY(dev_upload(&L->d_zero, nullptr, 256, "zero block"));
        e = hipMemset(L->d_zero, 0, 256);
        if (e != hipSuccess) {
            free_layer(L);
            return hip_fail(e, "zero block");
        }
        // K-split workspace: what the planner takes for a forward of max_tokens
        // tokens in either weight mode (fewer tokens may split further only
        // within it), and one arrival counter per smallest tile
        {
            const int64_t per = g1.conv ? (int64_t)g1.OH * g1.OW : 1;
            const Geom gmax = make_geom(L, std::max<int64_t>(1, desc->max_tokens / per));
            size_t need = 0;
            for (int mode = 0; mode < 2; ++mode) {
                aq::FusedPlan q = L->fplan;
                if (mode == 1 || q.rec_only) {
                    q.dec = aq::FUSED_DEC_REC;
                    q.mc = 1;
                    q.cb_bytes = 0;
                }
                // room for every split count the planner allows on its tile, so a
                // forced split (AQ_OPT_SPLIT_K) fits too
                if (fused_plan_tile(gmax, aq::Options{}, SIZE_MAX, desc->x_dtype, &q) && q.ntiles < 256) {
                    const int smax = std::min<int>({aq::kMaxSplitK, 512 / q.ntiles, q.nchunk / 4});
                    if (smax > 1) need = std::max(need, (size_t)smax * q.ntiles * q.bm * q.bn * 4);
                }
            }
            if (need) {
                AQ_TRY(dev_upload(&L->d_part, nullptr, need, "split partial tiles"));
                L->part_bytes = need;
            }
            const size_t ncnt = (size_t)((desc->max_tokens + 31) / 32) * ((C_out + 63) / 64);
            AQ_TRY(dev_upload(&L->d_arrivals, nullptr, ncnt * 4, "split arrival counters"));
            e = hipMemset(L->d_arrivals, 0, ncnt * 4);
            if (e != hipSuccess) {
                free_layer(L);
                return hip_fail(e, "split arrival counters");
            }
        }
    }

    e = aq::launch_codebook_prep(L->d_cb, desc->codebook_dtype, (int64_t)cb_elems, L->d_cb32, L->d_cbtile,
                                 desc->tile_dtype, nullptr);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        free_layer(L);
        return hip_fail(e, "codebook preparation");
    }
#undef AQ_TRY

    *out = L;
    return AQ_OK;
}

aq_status aq_layer_forward(aq_layer* L, const void* X, const float* x_scales, void* Y, int64_t n, void* stream) {
    Route r;
    Geom geo;
    const aq_status s = check_forward(L, X, x_scales, Y, n, &geo, &r);
    if (s != AQ_OK) return s;
    const Workspace wk{L->d_ws, L->d_lut_arrivals, L->d_wrec, L->d_part, L->d_arrivals, L->d_xpack};
    return run_route(L, geo, r, X, x_scales, Y, n, static_cast<hipStream_t>(stream), wk);
}

aq_status aq_layer_prepare(aq_layer* L, int64_t n, void* stream) {
    if (!L) return fail(AQ_ERR_INVALID_ARGUMENT, "null layer");
    if (n < 1) return fail(AQ_ERR_INVALID_ARGUMENT, "n must be >= 1");
    const Geom geo = make_geom(L, n);
    if (geo.tokens > L->desc.max_tokens) return fail(AQ_ERR_INVALID_ARGUMENT, "tokens exceed max_tokens");
    const Route r = plan_route(L, geo);
    L->prepared_n = 0;
    hipStream_t st = static_cast<hipStream_t>(stream);
    TraceScope trace(L, st);
    if (trace.error() != hipSuccess) return hip_fail(trace.error(), "launch event");
    const bool rec = (r.kind == Route::FUSED || r.kind == Route::REC_LINEAR || r.kind == Route::DENSE) &&
                     r.fp.dec == aq::FUSED_DEC_REC;
    if (!rec) return AQ_OK;                      // nothing of this forward depends on the weights alone
    const aq_layer_desc& d = L->desc;
    const DeviceWeights w{L->d_cb,         L->d_cb32,   L->d_cbtile,      L->d_codes,
                          L->d_codes_lut, L->d_scales, d.codebook_dtype, L->d_cb9};
    const hipError_t e = aq::launch_operand_records(geo, r.fp, w, L->d_wrec, st);
    if (e != hipSuccess) return hip_fail(e, "records launch");
    if (trace.error() != hipSuccess) return hip_fail(trace.error(), "launch event");
    L->prepared_n = n;
    return AQ_OK;
}

aq_status aq_layers_prepare(aq_layer* const* layers, const int64_t* n, int32_t count, void* stream) {
    if (count < 0) return fail(AQ_ERR_INVALID_ARGUMENT, "count < 0");
    if (count == 0) return AQ_OK;
    if (!layers || !n) return fail(AQ_ERR_INVALID_ARGUMENT, "null layer or n array");
    for (int32_t i = 0; i < count; ++i) {
        const std::string at = " (entry " + std::to_string(i) + ")";
        if (!layers[i]) return fail(AQ_ERR_INVALID_ARGUMENT, "null layer" + at);
        if (n[i] < 1) return fail(AQ_ERR_INVALID_ARGUMENT, "n must be >= 1" + at);
        for (int32_t j = 0; j < i; ++j)
            if (layers[j] == layers[i]) return fail(AQ_ERR_INVALID_ARGUMENT, "layer listed twice" + at);
    }
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    struct Item {
        aq_layer* L;
        int64_t n;
        Geom geo;
        Route r;
        int key;
    };
    std::vector<Item> items;
    items.reserve((size_t)count);
    // every argument is checked before anything is launched
    for (int32_t i = 0; i < count; ++i) {
        aq_layer* L = layers[i];
        const std::string at = " (entry " + std::to_string(i) + ")";
        if (L->device != dev) return fail(AQ_ERR_INVALID_ARGUMENT, "layer created on another device" + at);
        const Geom geo = make_geom(L, n[i]);
        if (geo.tokens > L->desc.max_tokens) return fail(AQ_ERR_INVALID_ARGUMENT, "tokens exceed max_tokens" + at);
        items.push_back(Item{L, n[i], geo, plan_route(L, geo), -1});
    }
    hipStream_t st = static_cast<hipStream_t>(stream);
    std::vector<int> keys;                     // batched kernels in order of first use
    for (Item& it : items) {
        it.L->prepared_n = 0;
        const bool rec = (it.r.kind == Route::FUSED || it.r.kind == Route::REC_LINEAR || it.r.kind == Route::DENSE) &&
                         it.r.fp.dec == aq::FUSED_DEC_REC;
        if (!rec) continue;
        aq_layer* L = it.L;
        const DeviceWeights w{L->d_cb,         L->d_cb32,   L->d_cbtile,      L->d_codes,
                              L->d_codes_lut, L->d_scales, L->desc.codebook_dtype, L->d_cb9};
        it.key = aq::records_batch_key(it.geo, it.r.fp, w);
        if (it.key < 0) {                       // no batched form: the layer's own launch
            e = aq::launch_operand_records(it.geo, it.r.fp, w, L->d_wrec, st);
            if (e != hipSuccess) return hip_fail(e, "records launch");
            L->prepared_n = it.n;
            it.key = -2;
            continue;
        }
        if (std::find(keys.begin(), keys.end(), it.key) == keys.end()) keys.push_back(it.key);
    }
    for (int key : keys) {
        aq::RecordBatch b{};
        std::vector<Item*> members;
        auto flush = [&]() -> aq_status {
            if (b.count == 0) return AQ_OK;
            const hipError_t fe = aq::launch_operand_records_batch(key, b, st);
            if (fe != hipSuccess) return hip_fail(fe, "batched records launch");
            for (Item* m : members) m->L->prepared_n = m->n;
            b = aq::RecordBatch{};
            members.clear();
            return AQ_OK;
        };
        for (Item& it : items) {
            if (it.key != key) continue;
            aq_layer* L = it.L;
            const DeviceWeights w{L->d_cb,         L->d_cb32,   L->d_cbtile,      L->d_codes,
                                  L->d_codes_lut, L->d_scales, L->desc.codebook_dtype, L->d_cb9};
            uint32_t blocks = 0;
            const aq::RecordJob job = aq::records_batch_job(it.geo, it.r.fp, w, L->d_wrec, &blocks);
            if (b.count == aq::kRecordBatchMax ||
                (uint64_t)b.start[b.count] + blocks > (uint64_t)INT32_MAX) {
                const aq_status fs = flush();
                if (fs != AQ_OK) return fs;
            }
            b.job[b.count] = job;
            b.start[b.count + 1] = b.start[b.count] + blocks;
            ++b.count;
            members.push_back(&it);
        }
        const aq_status fs = flush();
        if (fs != AQ_OK) return fs;
    }
    return AQ_OK;
}

aq_status aq_layer_forward_static(aq_layer* L, const void* X, const float* x_scales, void* Y, int64_t n,
                                  void* stream) {
    Route r;
    Geom geo;
    aq_status s = check_forward(L, X, x_scales, Y, n, &geo, &r);
    if (s != AQ_OK) return s;
    uint8_t* base = nullptr;
    Workspace wk;
    // sizes first, so a refused call launches nothing
    s = static_workspace(L, geo, r, reinterpret_cast<uint8_t*>(uintptr_t(256)), &wk);
    if (s != AQ_OK) return s;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    s = scratch_for_current_device(st, &base);
    if (s != AQ_OK) return s;
    s = static_workspace(L, geo, r, base, &wk);
    if (s != AQ_OK) return s;
    return run_route(L, geo, r, X, x_scales, Y, n, st, wk);
}

aq_status aq_layer_describe(const aq_layer* L, int64_t n, char* buf, int64_t size) {
    if (!L || !buf || size < 1) return fail(AQ_ERR_INVALID_ARGUMENT, "null pointer argument or empty buffer");
    if (n < 1) return fail(AQ_ERR_INVALID_ARGUMENT, "n must be >= 1");
    const Geom geo = make_geom(L, n);
    if (geo.tokens > L->desc.max_tokens) return fail(AQ_ERR_INVALID_ARGUMENT, "tokens exceed max_tokens");
    const Route r = plan_route(L, geo);
    static const char* kinds[] = {"table", "fp32", "generic", "dense-records", "fused", "rec-linear", "none"};
    static const char* decs[] = {"in-loop-lds-fp16", "in-loop-lds-fp32", "in-loop-lds-fp16", "in-loop-l2-fp16",
                                 "records"};
    const char* route = r.kind == Route::FUSED && r.fp.wsplit ? "rec-conv" : kinds[r.kind];
    std::string t = std::string("path=") + (r.kind == Route::LUT ? "lut" : "decode") + " route=" + route;
    if (r.kind == Route::FUSED || r.kind == Route::REC_LINEAR || r.kind == Route::DENSE) {
        const aq::FusedPlan& p = r.fp;
        const bool rl = r.kind == Route::REC_LINEAR;
        const int bm = rl ? (p.rlin_var == 1 ? 256 : 128) : p.bm, bn = rl ? 128 : p.bn;
        t += std::string(" weights=") + decs[p.dec] + " tile=" + std::to_string(bm) + "x" + std::to_string(bn);
        if (r.kind == Route::FUSED && p.wsplit) t += " depth=" + std::to_string(p.rdepth);
        if (r.kind == Route::FUSED)
            t += " upl=" + std::to_string(p.upl) + " split_k=" + std::to_string(p.splitk) +
                 " order=" + (p.nmajor ? "channel" : "token") +
                 " wg_per_cu=" + std::to_string(fused_occupancy(geo, p, L->desc.x_dtype));
        if (r.kind == Route::REC_LINEAR) t += " variant=" + std::to_string(p.rlin_var);
        if (p.dec == aq::FUSED_DEC_REC)
            t += " records_bytes=" + std::to_string(aq::operand_record_bytes(geo, p));
    }
    const size_t m = std::min<size_t>(t.size(), (size_t)size - 1);
    std::memcpy(buf, t.data(), m);
    buf[m] = '\0';
    return AQ_OK;
}

// Codebook gradient: validation, one-time preparation (code index and
// partial-gradient workspace), then the two launches.
aq_status aq_layer_codebook_grad(aq_layer* L, const void* X, const void* dY, int32_t dtype, float* dC, int64_t n,
                                 void* stream) {
    if (!L || !X || !dY || !dC) return fail(AQ_ERR_INVALID_ARGUMENT, "null pointer argument");
    if (n < 1) return fail(AQ_ERR_INVALID_ARGUMENT, "n must be >= 1");
    if (dtype < AQ_F32 || dtype > AQ_I8) return fail(AQ_ERR_INVALID_ARGUMENT, "bad dtype");
    if (dtype != AQ_F16 && dtype != AQ_BF16)
        return fail(AQ_ERR_UNSUPPORTED, "the codebook gradient takes fp16 or bf16 X and dY");
    const aq_layer_desc& d = L->desc;
    const Geom geo = make_geom(L, n);
    if (geo.tokens > d.max_tokens) return fail(AQ_ERR_INVALID_ARGUMENT, "tokens exceed max_tokens");
    if ((reinterpret_cast<uintptr_t>(X) | reinterpret_cast<uintptr_t>(dY)) & 15)
        return fail(AQ_ERR_INVALID_ARGUMENT, "X and dY must be 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(dC) & 3) return fail(AQ_ERR_INVALID_ARGUMENT, "dC must be 4-byte aligned");
    if (geo.conv) {
        const bool k3 = geo.kh == 3 && geo.kw == 3 && geo.pad == 1, k1 = geo.kh == 1 && geo.kw == 1 && geo.pad == 0;
        if (!(k3 || k1) || geo.stride != 1 || geo.W % 8 != 0)
            return fail(AQ_ERR_UNSUPPORTED, "the codebook gradient supports 1x1 and 3x3 convolutions with stride 1, "
                                            "same padding and an input width that is a multiple of 8");
    } else if (geo.C_out % 8 != 0 || geo.K % 8 != 0) {
        return fail(AQ_ERR_UNSUPPORTED, "the codebook gradient of a linear layer needs C_out and K multiples of 8");
    }
    if ((int64_t)geo.C_out * geo.G >= (int64_t(1) << 31))
        return fail(AQ_ERR_UNSUPPORTED, "too many code groups for the 32-bit code index");
    // the weight-gradient kernel addresses X and dY with 32-bit byte offsets
    const int64_t lim = int64_t(1) << 31;
    const int64_t xbytes = geo.conv ? n * geo.cin * (int64_t)geo.H * geo.W * 2 : geo.tokens * geo.K * 2;
    if (xbytes >= lim || geo.tokens * geo.C_out * 2 >= lim)
        return fail(AQ_ERR_UNSUPPORTED, "X or dY of 2 GiB or more: beyond the codebook-gradient kernel's offsets");
    if ((int64_t)geo.C_out * geo.K * 4 * 16 >= lim)
        return fail(AQ_ERR_UNSUPPORTED, "C_out * K too large for the codebook-gradient workspace offsets");
    if (!L->grad_ready) {
        // one-time preparation: synchronous and allocating
        const size_t ncodes = (size_t)geo.C_out * geo.G * geo.M;
        std::vector<uint8_t> host(ncodes * (geo.B <= 8 ? 1 : 2));
        hipError_t e = hipMemcpy(host.data(), L->d_codes, host.size(), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e, "codes readback");
        std::vector<int32_t> offs, ent;
        aq::build_code_index(host.data(), geo.B, geo.C_out, geo.G, geo.M, offs, ent);
        aq_status s = dev_upload(&L->d_gidx_offs, offs.data(), offs.size() * sizeof(int32_t), "code index");
        if (s == AQ_OK) s = dev_upload(&L->d_gidx_ent, ent.data(), ent.size() * sizeof(int32_t), "code index");
        if (s == AQ_OK && !L->d_zero) {
            s = dev_upload(&L->d_zero, nullptr, 256, "zero block");
            if (s == AQ_OK && (e = hipMemset(L->d_zero, 0, 256)) != hipSuccess) s = hip_fail(e, "zero block");
        }
        if (s != AQ_OK) {
            for (void** p : {(void**)&L->d_gidx_offs, (void**)&L->d_gidx_ent})
                if (*p) {
                    (void)hipFree(*p);
                    *p = nullptr;
                }
            return s;
        }
        L->grad_ready = true;
        L->grad_stale = true;
    }
    if (L->grad_stale) {
        // plan (again, after a gradient option changed); the partial-gradient
        // workspace grows when the new plan needs more splits (synchronous)
        const aq::GradPlan gp = aq::grad_plan_create(geo, d.max_tokens, L->opt);
        const size_t need = (size_t)gp.s_max * geo.C_out * geo.K * sizeof(float);
        if (need > L->gpart_bytes) {
            if (L->d_gpart) {
                hipError_t e = hipDeviceSynchronize();
                if (e != hipSuccess) return hip_fail(e, "gradient workspace");
                (void)hipFree(L->d_gpart);
                L->d_gpart = nullptr;
                L->gpart_bytes = 0;
            }
            aq_status s = dev_upload(&L->d_gpart, nullptr, need, "gradient workspace");
            if (s != AQ_OK) return s;
            L->gpart_bytes = need;
        }
        L->gplan = gp;
        L->grad_stale = false;
    }
    TraceScope trace(L, static_cast<hipStream_t>(stream));
    if (trace.error() != hipSuccess) return hip_fail(trace.error(), "launch event");
    const hipError_t e =
        aq::launch_codebook_grad(geo, L->gplan, dtype, X, dY, L->d_scales, L->d_gpart, L->d_gidx_offs, L->d_gidx_ent,
                                 dC, L->d_zero, L->opt.grad_splits, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "codebook gradient launch");
    if (trace.error() != hipSuccess) return hip_fail(trace.error(), "launch event");
    return AQ_OK;
}

aq_status aq_layer_decode(aq_layer* L, void* W, void* stream) {
    if (!L || !W) return fail(AQ_ERR_INVALID_ARGUMENT, "null pointer argument");
    const Geom geo = make_geom(L, 1);
    const DeviceWeights w{L->d_cb, L->d_cb32, L->d_cbtile, L->d_codes, L->d_codes_lut, L->d_scales,
                          L->desc.codebook_dtype};
    hipError_t e = aq::launch_decode_to_global(geo, w, L->desc.tile_dtype, W, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "decode launch");
    return AQ_OK;
}

aq_status aq_layer_set_path(aq_layer* L, aq_path path) {
    if (!L) return fail(AQ_ERR_INVALID_ARGUMENT, "null layer");
    if (path != AQ_PATH_AUTO && path != AQ_PATH_LUT && path != AQ_PATH_DECODE)
        return fail(AQ_ERR_INVALID_ARGUMENT, "bad path");
    if (path == AQ_PATH_LUT && !L->lut_ok) return fail(AQ_ERR_UNSUPPORTED, "LUT path needs B <= 8");
    if (path == AQ_PATH_DECODE && !L->dec_ok)
        return fail(AQ_ERR_UNSUPPORTED, "fp16/bf16 decode path needs g == 8 (or g == 9 on a 3x3 convolution)");
    L->path = path;
    return AQ_OK;
}

aq_status aq_layer_set_option(aq_layer* L, int32_t option, int64_t value) {
    if (!L) return fail(AQ_ERR_INVALID_ARGUMENT, "null layer");
    aq::Options& o = L->opt;
    auto in = [&](int64_t lo, int64_t hi) { return value >= lo && value <= hi; };
    auto bad = [&]() { return fail(AQ_ERR_INVALID_ARGUMENT, "option " + std::to_string(option) +
                                                                ": value " + std::to_string(value) + " out of range"); };
    auto tile = [&](int* bm, int* bn) {
        if (value == 0) {
            *bm = *bn = 0;
            return true;
        }
        const int64_t m = value / 1000, nn = value % 1000;
        if (m < 16 || m > 512 || nn < 16 || nn > 512 || m % 16 || nn % 16) return false;
        *bm = (int)m;
        *bn = (int)nn;
        return true;
    };
    switch (option) {
    case AQ_OPT_LUT_MAX_TOKENS:
        if (!in(-1, int64_t(1) << 40)) return bad();
        o.lut_max_tokens = value;
        return AQ_OK;
    case AQ_OPT_WEIGHTS:
        if (!in(0, 2)) return bad();
        o.weights = (int)value;
        return AQ_OK;
    case AQ_OPT_GENERIC:
        if (!in(0, 1)) return bad();
        o.generic = (int)value;
        return AQ_OK;
    case AQ_OPT_RECORD_PRODUCT:
        if (!in(0, 3)) return bad();
        o.rec_product = (int)value;
        return AQ_OK;
    case AQ_OPT_FUSED_TILE:
        return tile(&o.fused_bm, &o.fused_bn) ? AQ_OK : bad();
    case AQ_OPT_DENSE_TILE:
        return tile(&o.dense_bm, &o.dense_bn) ? AQ_OK : bad();
    case AQ_OPT_REC_LINEAR_TILE:
        if (!in(0, 3)) return bad();
        o.rlin_tile = (int)value;
        return AQ_OK;
    case AQ_OPT_TILE_ORDER:
        if (!in(0, 2)) return bad();
        o.tile_order = (int)value;
        return AQ_OK;
    case AQ_OPT_STAGE_ROWS:
        if (!in(0, 1)) return bad();
        o.stage_rows = (int)value;
        return AQ_OK;
    case AQ_OPT_SPLIT_K:
        if (!in(0, aq::kMaxSplitK)) return bad();
        o.split_k = (int)value;
        return AQ_OK;
    case AQ_OPT_GRAD_SPLITS:
        if (!in(0, 16)) return bad();
        o.grad_splits = (int)value;
        L->grad_stale = true;
        return AQ_OK;
    case AQ_OPT_GRAD_REGS:
        if (!in(0, 1)) return bad();
        o.grad_regs = (int)value;
        L->grad_stale = true;
        return AQ_OK;
    case AQ_OPT_GRAD_TILE:
        if (!tile(&o.grad_bm, &o.grad_bn)) return bad();
        L->grad_stale = true;
        return AQ_OK;
    case AQ_OPT_TABLE_ONE_LAUNCH:
        if (!in(0, 1)) return bad();
        o.table_one_launch = (int)value;
        return AQ_OK;
    default:
        return fail(AQ_ERR_INVALID_ARGUMENT, "unknown option " + std::to_string(option));
    }
}

aq_status aq_layer_get_option(const aq_layer* L, int32_t option, int64_t* value) {
    if (!L || !value) return fail(AQ_ERR_INVALID_ARGUMENT, "null pointer argument");
    const aq::Options& o = L->opt;
    switch (option) {
    case AQ_OPT_LUT_MAX_TOKENS: *value = o.lut_max_tokens; return AQ_OK;
    case AQ_OPT_WEIGHTS: *value = o.weights; return AQ_OK;
    case AQ_OPT_GENERIC: *value = o.generic; return AQ_OK;
    case AQ_OPT_RECORD_PRODUCT: *value = o.rec_product; return AQ_OK;
    case AQ_OPT_FUSED_TILE: *value = o.fused_bm * 1000 + o.fused_bn; return AQ_OK;
    case AQ_OPT_DENSE_TILE: *value = o.dense_bm * 1000 + o.dense_bn; return AQ_OK;
    case AQ_OPT_REC_LINEAR_TILE: *value = o.rlin_tile; return AQ_OK;
    case AQ_OPT_TILE_ORDER: *value = o.tile_order; return AQ_OK;
    case AQ_OPT_STAGE_ROWS: *value = o.stage_rows; return AQ_OK;
    case AQ_OPT_SPLIT_K: *value = o.split_k; return AQ_OK;
    case AQ_OPT_GRAD_SPLITS: *value = o.grad_splits; return AQ_OK;
    case AQ_OPT_GRAD_REGS: *value = o.grad_regs; return AQ_OK;
    case AQ_OPT_GRAD_TILE: *value = o.grad_bm * 1000 + o.grad_bn; return AQ_OK;
    case AQ_OPT_TABLE_ONE_LAUNCH: *value = o.table_one_launch; return AQ_OK;
    default: return fail(AQ_ERR_INVALID_ARGUMENT, "unknown option " + std::to_string(option));
    }
}

aq_status aq_layer_set_launch_events(aq_layer* L, void* const* events, int32_t n_events) {
    if (!L) return fail(AQ_ERR_INVALID_ARGUMENT, "null layer");
    if (n_events < 0 || n_events > 64 || (n_events > 0 && !events))
        return fail(AQ_ERR_INVALID_ARGUMENT, "n_events must be in [0, 64] with a non-null array");
    for (int i = 0; i < n_events; ++i)
        if (!events[i]) return fail(AQ_ERR_INVALID_ARGUMENT, "null event at index " + std::to_string(i));
    L->events.assign(reinterpret_cast<hipEvent_t const*>(events), reinterpret_cast<hipEvent_t const*>(events) + n_events);
    return AQ_OK;
}

aq_status aq_layer_last_launches(const aq_layer* L, int32_t* n_launches, char* names, int64_t names_size) {
    if (!L || !n_launches) return fail(AQ_ERR_INVALID_ARGUMENT, "null pointer argument");
    *n_launches = L->last_launches;
    if (names && names_size > 0) {
        const size_t n = std::min<size_t>(L->last_names.size(), (size_t)names_size - 1);
        std::memcpy(names, L->last_names.data(), n);
        names[n] = '\0';
    }
    return AQ_OK;
}

aq_status aq_layer_choose_path(const aq_layer* L, int64_t tokens, aq_path* out) {
    if (!L || !out) return fail(AQ_ERR_INVALID_ARGUMENT, "null pointer argument");
    if (tokens < 1) return fail(AQ_ERR_INVALID_ARGUMENT, "tokens must be >= 1");
    *out = choose(L, tokens);
    return AQ_OK;
}

aq_status aq_layer_destroy(aq_layer* L) {
    if (!L) return AQ_OK;
    hipError_t e = hipDeviceSynchronize();
    free_layer(L);
    if (e != hipSuccess) return hip_fail(e, "destroy");
    return AQ_OK;
}

}  // extern "C"
