// Partition runtime behind the C ABI in include/ppipe.h.
//
// create: validates the layer range [begin, end) (a partition spans layers i
//   to j exclusive and receives only layer i-1's feature map: the paper's
//   MILP inputs C_ldbij and Y_bj, Appendix A.1), derives every layer shape
//   from the model input, folds batch norm into fp32 per-channel scale and
//   shift, repacks weights to the kernels' layouts in the storage dtype,
//   assigns activation buffers by liveness, chooses a kernel plan for every
//   (layer, batch) pair and allocates everything once for max_batch.
// run: walks the range in index order on the caller's stream, or replays a
//   captured HIP graph; no allocation, no host synchronisation.
// profile: per-layer and per-launch HIP event timing that produces the
//   latency table L[i][b] and the feature-map sizes S_i (Sec. 3 inputs,
//   Sec. 5.1 offline profiling).
#include "ppipe.h"
#include "kernels.h"

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

using namespace ppipe;

namespace {

thread_local std::string g_err;
thread_local int g_status = 0;

int fail(int code, const std::string& msg)
{
    g_err = msg;
    g_status = code;
    return code;
}

}  // namespace

// the host-only parts of the library report errors through the same slot
int ppipe::set_error(int status, const std::string& msg) { return fail(status, msg); }

namespace {

std::string hip_msg(const char* what, hipError_t e)
{
    return std::string(what) + ": " + hipGetErrorString(e);
}

// ---- host-side rounding for weight packing (fp32 -> 16-bit, nearest even) ----
uint16_t f32_to_f16_bits(float f)
{
    uint32_t x;
    std::memcpy(&x, &f, 4);
    const uint32_t sign = (x >> 16) & 0x8000u;
    const uint32_t ax = x & 0x7fffffffu;
    if (ax >= 0x7f800000u)                      // inf / nan
        return (uint16_t)(sign | (ax > 0x7f800000u ? 0x7e00u : 0x7c00u));
    if (ax >= 0x477ff000u)                      // >= 65520 rounds to inf
        return (uint16_t)(sign | 0x7c00u);
    if (ax < 0x38800000u) {                     // below 2^-14: multiples of 2^-24
        float af;
        std::memcpy(&af, &ax, 4);
        return (uint16_t)(sign | (uint32_t)std::nearbyint(af * 16777216.0f));
    }
    uint32_t h = ((((ax >> 23) - 127u + 15u) << 10) | ((ax & 0x7fffffu) >> 13));
    const uint32_t rem = ax & 0x1fffu;
    if (rem > 0x1000u || (rem == 0x1000u && (h & 1u)))
        ++h;
    return (uint16_t)(sign | h);
}

uint16_t f32_to_bf16_bits(float f)
{
    uint32_t x;
    std::memcpy(&x, &f, 4);
    if ((x & 0x7fffffffu) > 0x7f800000u)
        return (uint16_t)((x >> 16) | 0x40u);
    return (uint16_t)((x + 0x7fffu + ((x >> 16) & 1u)) >> 16);
}

void put_elem(std::vector<uint8_t>& blob, size_t off, int dt, size_t i, float v)
{
    if (dt == DT_F32) {
        std::memcpy(&blob[off + i * 4], &v, 4);
    } else {
        uint16_t b = dt == DT_F16 ? f32_to_f16_bits(v) : f32_to_bf16_bits(v);
        std::memcpy(&blob[off + i * 2], &b, 2);
    }
}

enum Kind { K_GEMM = 0, K_DW = 1, K_MAXPOOL = 2, K_GAP = 3 };
enum { BUF_IN = -1, BUF_OUT = -2, BUF_NONE = -3 };

struct Plan {
    int cfg, wk, splits, chunks_per_split, total_chunks, tiles_m, tiles_co, co_fastest;
    int grid = 0;   // pointwise kernel: cap on blocks along the pixels (0: resident set)
    bool forced = false;   // chosen by a tuning override, not by the planner
};

struct Shape {
    int c, h, w;
};

// Scratch memory of a run: split-K partial sums followed by the fp32 logits
// of a final FC + softmax (ws), and the channel-padded input of a stem (pad).
struct Workspace {
    float* ws;
    void* pad;
};

}  // namespace

struct LayerRT {
    int index, op, src, res_src, act, k, stride, pad, groups;
    int H, W, C, Ho, Wo, Co;
    int kind;
    bool tapv = false, softmax = false, skinny_ok = false, pad_in = false;
    bool pw_ok = false;         // the streaming 1x1 kernel applies (GEMM_PW)
    bool stem_ok = false;       // the stem kernel applies (GEMM_STEM)
    int KH = 1, KW = 1, gstride = 1, gpad = 0, K = 0, Kpad = 0;
    int cpad = 0;               // channels as the GEMM reads them (C rounded up to a vector)
    size_t w_off = 0, scale_off = 0, bias_off = 0;
    void* w = nullptr;
    float* scale = nullptr;
    float* bias = nullptr;
    int in_buf = BUF_IN, res_buf = BUF_NONE, out_buf = BUF_OUT;
    // position in the partition of the layer this GEMM shares its input with
    // and may run with in one launch (-1: none); pair_lead on the earlier one
    int pair = -1;
    bool pair_lead = false;
    std::vector<Plan> plans;   // [batch - 1]
    std::string name;          // the description's layer name, or "layer<i>"
    int64_t out_bytes_b1 = 0;
    double flops_b1 = 0, in_bytes_b1 = 0, res_bytes_b1 = 0, param_bytes = 0;
};

struct GraphEntry {
    int batch;
    const void* in;
    void* out;
    hipGraph_t graph;
    hipGraphExec_t exec;
};

struct ppipe_partition {
    int begin = 0, end = 0, dtype = 0, max_batch = 64, device = 0;
    ppipe_tuning tune{-1, 0, 1, 0, 0, 0, 0, 0};   // planner overrides given at create
    int cus = 256;                                // compute units the plans are sized for
    bool tuned = false;                           // any override active
    Shape in{}, out{};
    int out_dtype = 0;
    std::vector<LayerRT> L;
    std::vector<void*> slots;
    std::vector<size_t> slot_bytes;
    float* ws = nullptr;          // split-K partials, then fp32 logits of a final FC + softmax
    size_t ws_bytes = 0;
    void* pad_buf = nullptr;      // channel-padded input of layers with C < 16 bytes
    size_t pad_bytes = 0;
    void* wblob = nullptr;
    size_t wbytes = 0;
    std::vector<uint8_t> host_blob;   // packed parameters between validation and upload
    hipStream_t cap_stream = nullptr;
    std::vector<GraphEntry> graphs;
    // timed runs: an event before and after every launch of one run
    struct {
        int batch = 0;
        const void* in = nullptr;
        void* out = nullptr;
        std::vector<hipEvent_t> ev;
        bool ran = false;
    } timed;
};

LaunchEvents& ppipe::launch_events()
{
    thread_local LaunchEvents ev;
    return ev;
}

namespace {

// Kernel plan of a GEMM-shaped layer at one batch: kernel family, tile
// shape, waves per tile (skinny) and tile order.  Deterministic in (M, Co, K,
// dtype, eligibility) so that the latency table, the benchmark and the
// parity tests exercise the same launches.
Plan choose_plan(int M, int Co, int K, int dt, bool skinny_ok, bool pw_ok, bool stem_ok,
                 bool split_free, const ppipe_tuning& tune, int cus)
{
    // Grid-size thresholds below are stated for the 256 CUs of a whole
    // MI355X and scale with the CUs the handle runs on (a CU share of a
    // virtual GPU has fewer).
    const int64_t C = cus;
    auto at = [&](int64_t n256) { return n256 * C / 256; };
    auto tiles = [&](int cfg) {
        GemmCfgInfo c = gemm_cfg_info(cfg);
        return (int64_t)((M + c.bn - 1) / c.bn) * ((Co + c.bm - 1) / c.bm);
    };
    auto steps = [&](int cfg) { return (K + gemm_bk(cfg, dt) - 1) / gemm_bk(cfg, dt); };
    // Fitted to per-layer sweeps of every plan over the five partition
    // workloads on MI355X, timed in layer order (weights cold as in a real
    // run, the split-K reduction at its in-order cost of ~4 us):
    //  * 16-bit layers with Co >= 128 take 8-wave 128x128 tiles: with 192 to
    //    255 of them (128 with K >= 1024) on the four-stage ring, one block
    //    per CU with two stages in flight (ResNet-152's 14x14 layer3 at batch
    //    64: 3x3 29.6 -> 23.2 us, 1x1 1024->256 17.5 -> 14.9 us against
    //    64x64 tiles, the whole model 8.8% faster, batch 44-56 6-8%); from
    //    256 of them on the two-stage ring, two blocks per CU (from 384
    //    before, ResNet-152 at batch 42-56 2.5% faster); with a long K loop,
    //    a hundred of them split over K;
    //  * everything else takes 64x64 tiles; K is split in two only when each
    //    half keeps >= 12 steps and the split grid has at most 192 blocks
    //    (three quarters of the CUs), or 384 with >= 24 steps per half: a
    //    split halves the K loop but adds a reduction launch (ResNet-152's
    //    196-pixel 3x3 layers at batch 11-15 ran both halves of a CU's two
    //    blocks in turn and paid the reduction on top, 16.5 against 11.2 us,
    //    the whole model 8-10% faster unsplit; at batch 8-10, 100-136 tiles,
    //    1.4-2.9% faster unsplit); further splits while the grid is short
    //    of about 1.5 blocks per CU and each split keeps >= 4 steps, or up to
    //    2 blocks per CU with >= 12 steps per split;
    //  * sparse grids (up to two 64x64 blocks, or under one 8-wave 128x128
    //    block, per CU) take software-pipelined loops; sparse 64x64 grids use
    //    8 waves and four stages (two in flight), because a lone block
    //    streams every operand byte from beyond L2 and is bound by the bytes
    //    it keeps in flight (VGG-16's 25088-input FC at batch 16, 64 tiles
    //    split 8 ways: 45 -> 36 us); dense grids take the two-stage loop (fewest registers and
    //    LDS, highest occupancy), on 8-wave 64x128 tiles for layers of at
    //    most 64 output channels with at least 512 such tiles (fewer operand
    //    bytes per FLOP: VGG-16 conv1_2 at batch 16 124 -> 108 us, ResNet-152's
    //    7x7 stem at batch 64 116 -> 93 us);
    //  * small fp32 layers take the skinny kernel (no reduction pass); so do
    //    16-bit layers with a long K loop (>= 1024) whose 16x16 skinny grid
    //    holds at least 128 pixels and fits one block per CU: ResNet-152's
    //    196-pixel layer3 convolutions at batch 1, where 64x64 tiles leave 16
    //    blocks (1x1, 6.5 -> 5.5 us) or 8 K splits and a reduction (3x3, 9.7
    //    -> 7.2 us); the whole model 4% faster at batch 1.  Smaller grids
    //    (layer4's 49 pixels) ran faster per layer but slower in a replayed
    //    graph, and FC layers gained nothing.
    const bool wide = dt != PPIPE_F32 && Co >= 128;
    const int64_t t128 = tiles(GEMM_DMA_128x128_8W_S2);
    const int k128 = steps(GEMM_DMA_128x128_8W_S2);
    int cfg = GEMM_DMA_64x64_S2, wk = 0, splits = 1;
    const int64_t sk16 = (int64_t)((M + 15) / 16) * ((Co + 15) / 16);
    if (dt == PPIPE_F32 && skinny_ok && M <= 4096 && K >= 256) {
        cfg = GEMM_SK_32x32;
        wk = 4;
    } else if (dt != PPIPE_F32 && skinny_ok && !split_free && K >= 1024 && M >= 128 &&
               sk16 <= C) {
        cfg = GEMM_SK_16x16;
        wk = 4;
    } else if (wide && t128 < C && (t128 >= at(192) || (t128 >= at(128) && K >= 1024))) {
        cfg = GEMM_DMA_128x128_8W_S4;
    } else if (wide && (t128 >= C || (t128 >= at(96) && k128 >= 64))) {
        cfg = GEMM_DMA_128x128_8W_S2;
        if (t128 < C)
            while (splits < 16 && t128 * splits * 2 <= at(512) && k128 / (splits * 2) >= 8)
                splits *= 2;
        if (t128 * splits < C)
            cfg = GEMM_DMA_128x128_8W_S3;
    } else if (split_free) {
        // the softmax kernel of an FC + softmax layer adds the partials as it
        // loads the logits, so splitting K costs no reduction launch: eight
        // ways (each split keeping >= 2 steps) on the 8-wave four-stage tile
        // (MobileNetV2's classifier at batch 32 11.9 -> 8.5 us, VGG-16's at
        // batch 16 10.7 -> 8.6 us)
        const int k = steps(GEMM_DMA_64x64_8W_S4);
        cfg = GEMM_DMA_64x64_8W_S4;
        while (splits < 8 && k / (splits * 2) >= 2)
            splits *= 2;
    } else {
        const int64_t t = tiles(cfg);
        const int k = steps(cfg);
        while (splits < 32) {
            const int64_t nb = t * splits * 2;
            const int cps = k / (splits * 2);
            const bool ok = splits == 1
                                ? (cps >= 12 && (nb <= at(192) || (nb <= at(384) && cps >= 24)))
                                : ((nb <= at(128) && cps >= 2) || (nb <= at(384) && cps >= 4) ||
                                   (nb <= at(512) && cps >= 12));
            if (!ok) break;
            splits *= 2;
        }
        if (t * splits <= at(512))
            cfg = GEMM_DMA_64x64_8W_S4;
        else if (splits == 1 && Co <= 64 && tiles(GEMM_DMA_64x128_8W_S2) >= at(512))
            cfg = GEMM_DMA_64x128_8W_S2;
    }
    //  * 16-bit 1x1 stride-1 layers with at most 32 input channels (or 160
    //    with at most 32 output channels) and at least 16384 output pixels
    //    stream through the pointwise kernel (2-3x faster on MobileNetV2's
    //    large expansion layers; the GEMM stays ahead on small grids).
    //    The no_pointwise tuning override turns it off (A/B timing).
    if (pw_ok && M >= 16384 && !tune.no_pointwise) {
        cfg = GEMM_PW;
        wk = pointwise_channel_frags(Co);
        splits = 1;
    }
    //  * stems of 3-channel images take the stem kernel (no channel-padding
    //    pass): 3x3 stems 1.7-2.4x faster than the padded GEMM; ResNet-152's
    //    7x7 stem as a whole model 0.3-3.6% faster at batch 6-32 and even from
    //    40 to 64.  The no_stem tuning override turns it off.
    if (stem_ok && !tune.no_stem) {
        cfg = GEMM_STEM;
        wk = stem_channel_frags(Co);
        splits = 1;
    }
    // The gemm_cfg tuning override (with gemm_waves, gemm_splits) forces one
    // configuration on every eligible GEMM layer (tuning sweeps and kernel tests).
    bool forced = false;
    {
        const int fc = tune.gemm_cfg, fw = tune.gemm_waves, fs = tune.gemm_splits;
        if (fc >= 0 && fc < GEMM_NCFG) {
            const int cfg0 = cfg;
            const bool sk = gemm_cfg_info(fc).skinny;
            const bool wk_ok = fw == 4 || fw == 8 || (fw == 16 && fc == GEMM_SK_16x16);
            if (fc == GEMM_PW) {
                if (pw_ok) {
                    cfg = fc;
                    wk = pointwise_channel_frags(Co);
                    splits = 1;
                }
            } else if (fc == GEMM_STEM) {
                if (stem_ok) {
                    cfg = fc;
                    wk = stem_channel_frags(Co);
                    splits = 1;
                }
            } else if (!sk) {
                cfg = fc;
                wk = 0;
                splits = std::max(1, std::min(fs, 64));
            } else if (skinny_ok && wk_ok) {
                cfg = fc;
                wk = fw;
                splits = 1;
            }
            forced = cfg != cfg0 || fc == cfg0;
        }
    }
    const GemmCfgInfo c = gemm_cfg_info(cfg);
    Plan p;
    p.cfg = cfg;
    p.wk = wk;
    p.total_chunks = steps(cfg);
    p.chunks_per_split = (p.total_chunks + splits - 1) / splits;
    p.splits = (p.total_chunks + p.chunks_per_split - 1) / p.chunks_per_split;
    p.tiles_m = (M + c.bn - 1) / c.bn;
    p.tiles_co = (Co + c.bm - 1) / c.bm;
    if (cfg == GEMM_PW || cfg == GEMM_STEM) {   // 16-pixel groups x channel slices of wk fragments
        p.tiles_co = (Co + 16 * wk - 1) / (16 * wk);
        if (tune.stream_grid > 0) {                 // tuning sweeps
            p.grid = tune.stream_grid;
            forced = true;
        }
    }
    p.forced = forced;
    p.co_fastest = M > Co ? 1 : 0;   // keep the larger operand's slices on one XCD
    return p;
}

// The per-vector-tap variant applies to the LDS-staged kernel only; a layer
// planned on the skinny kernel has whole K steps per tap (skinny_ok).
bool tapv_of(const LayerRT& l, const Plan& p)
{
    return l.tapv && !gemm_cfg_info(p.cfg).skinny && p.cfg != GEMM_PW && p.cfg != GEMM_STEM;
}

// The stem kernel reads the image itself; other kernels read it channel-padded.
bool pads_input(const LayerRT& l, const Plan& p)
{
    return l.pad_in && p.cfg != GEMM_STEM;
}

const void* buf_ptr(const ppipe_partition* P, int id, const void* in, void* out)
{
    if (id == BUF_IN) return in;
    if (id == BUF_OUT) return out;
    if (id == BUF_NONE) return nullptr;
    return P->slots[id];
}

// Receives a callback around every kernel launch (profiling).
struct LaunchHook {
    virtual ~LaunchHook() = default;
    virtual void before(const LayerRT&, int, hipStream_t) {}
    virtual void after(const LayerRT&, int, hipStream_t) {}
};

// Hands the k-th event pair to the k-th launch of a run (the launch records
// them around the kernel itself).
struct TimedHook : LaunchHook {
    explicit TimedHook(const std::vector<hipEvent_t>& e) : ev(e) {}
    ~TimedHook() override { launch_events() = LaunchEvents{}; }
    const std::vector<hipEvent_t>& ev;
    size_t k = 0;
    void before(const LayerRT&, int, hipStream_t) override
    {
        if (2 * k + 1 < ev.size()) launch_events() = LaunchEvents{ev[2 * k], ev[2 * k + 1]};
    }
    void after(const LayerRT&, int, hipStream_t) override
    {
        launch_events() = LaunchEvents{};
        ++k;
    }
};

// Launch sequence of a GEMM layer: [channel pad], GEMM, [split-K reduce], [softmax].
enum LaunchRole { L_PAD, L_GEMM, L_REDUCE, L_SOFTMAX, L_OTHER };

std::vector<int> launch_roles(const LayerRT& l, int batch)
{
    if (l.kind != K_GEMM) return {L_OTHER};
    std::vector<int> r;
    if (pads_input(l, l.plans[batch - 1])) r.push_back(L_PAD);
    r.push_back(L_GEMM);
    // the softmax launch of an FC + softmax layer also reduces its K splits
    if (l.plans[batch - 1].splits > 1 && !l.softmax) r.push_back(L_REDUCE);
    if (l.softmax) r.push_back(L_SOFTMAX);
    return r;
}

int layer_launches(const LayerRT& l, int batch) { return (int)launch_roles(l, batch).size(); }

std::string launch_name(const ppipe_partition* P, const LayerRT& l, int batch, int launch)
{
    switch (l.kind) {
    case K_GEMM: {
        const Plan& p = l.plans[batch - 1];
        switch (launch_roles(l, batch)[launch]) {
        case L_PAD: return pad_channels_name(P->dtype);
        case L_GEMM: return conv_gemm_name(P->dtype, p.cfg, p.wk, tapv_of(l, p));
        case L_REDUCE: return splitk_reduce_name(P->dtype);
        default: return softmax_rows_name();
        }
    }
    case K_DW: return dwconv_name(P->dtype, l.k);
    case K_MAXPOOL: return maxpool_name(P->dtype);
    default: return gap_name(P->dtype);
    }
}

// Algorithmic work of one launch: FLOPs, and the layer's input, weight,
// output and residual bytes each counted once.  In a multi-launch layer the
// first launch owns the input (the GEMM also the weights and FLOPs) and the
// last launch the output and residual; a split-K reduction in between owns
// nothing.
void launch_work(const ppipe_partition* P, const LayerRT& l, int batch, int launch,
                 double* flops, double* bytes)
{
    const double b = batch;
    const double out_bytes = b * (double)l.out_bytes_b1 *
                             (l.softmax ? 4.0 / dtype_size(P->dtype) : 1.0);
    const std::vector<int> roles = launch_roles(l, batch);
    const int n = (int)roles.size(), role = roles[launch];
    *flops = (role == L_GEMM || role == L_OTHER) ? b * l.flops_b1 : 0.0;
    double by = 0.0;
    if (launch == 0) by += b * l.in_bytes_b1;
    if (role == L_GEMM || role == L_OTHER) by += l.param_bytes;
    if (launch == n - 1) by += out_bytes + b * l.res_bytes_b1;
    *bytes = by;
}

// GEMM arguments of layer l at a batch (x: the layer's input as the GEMM reads it).
ConvGemmArgs gemm_args(const ppipe_partition* P, const LayerRT& l, int batch, const void* x,
                       const void* res, void* y, bool padded, const Workspace& W)
{
    const Plan& p = l.plans[batch - 1];
    ConvGemmArgs a;
    a.x = x;
    a.w = l.w;
    a.scale = l.scale;
    a.bias = l.bias;
    a.res = res;
    a.y = y;
    a.M = batch * l.Ho * l.Wo;
    a.partial = W.ws;
    a.logits = W.ws + (p.splits > 1 ? (size_t)p.splits * a.M * l.Co : 0);
    a.N = batch;
    a.H = l.H; a.W = l.W; a.C = padded ? l.cpad : l.C;
    a.Ho = l.Ho; a.Wo = l.Wo; a.Co = l.Co;
    a.KH = l.KH; a.KW = l.KW; a.stride = l.gstride; a.pad = l.gpad;
    a.K = l.K; a.Kpad = l.Kpad;
    a.act = l.act;
    a.total_chunks = p.total_chunks;
    a.splits = p.splits;
    a.chunks_per_split = p.chunks_per_split;
    a.tiles_m = p.tiles_m;
    a.tiles_co = p.tiles_co;
    a.co_fastest = p.co_fastest;
    a.softmax = l.softmax ? 1 : 0;
    a.grid_blocks = p.grid;
    return a;
}

// Whether paired layers a (lead) and b run as one launch at this batch: both
// planned unsplit on the sparse-grid configuration (8-wave 64x64, four
// stages), where neither grid fills the chip and each launch is bound by its
// latency.  Dense grids gain nothing from sharing a launch (ResNet-152 at
// batch 16 ran 0.7% slower with its two dense pairs joined).  The no_pair
// tuning override turns pairing off (A/B timing).
bool pair_runs(const ppipe_partition* P, const LayerRT& a, const LayerRT& b, int batch)
{
    const bool off = P->tune.no_pair != 0;
    const Plan& p = a.plans[batch - 1];
    const Plan& q = b.plans[batch - 1];
    return !off && p.cfg == GEMM_DMA_64x64_8W_S4 && q.cfg == GEMM_DMA_64x64_8W_S4 &&
           p.splits == 1 && q.splits == 1 && !pads_input(a, p) && !pads_input(b, q) &&
           !tapv_of(a, p) && !tapv_of(b, q);
}

// Enqueue the launches of one layer; only >= 0 restricts to that launch.
Workspace handle_workspace(const ppipe_partition* P) { return Workspace{P->ws, P->pad_buf}; }

hipError_t enqueue_layer(const ppipe_partition* P, const LayerRT& l, int batch, const void* in,
                         void* out, hipStream_t s, LaunchHook* hook, int only = -1,
                         const Workspace* wsp = nullptr)
{
    const Workspace W = wsp ? *wsp : handle_workspace(P);
    const void* x = buf_ptr(P, l.in_buf, in, out);
    void* y = const_cast<void*>(buf_ptr(P, l.out_buf, in, out));
    const void* res = buf_ptr(P, l.res_buf, in, out);
    hipError_t e = hipSuccess;
    switch (l.kind) {
    case K_GEMM: {
        const Plan& p = l.plans[batch - 1];
        const std::vector<int> roles = launch_roles(l, batch);
        auto want = [&](int i) { return only < 0 || only == i; };
        int li = 0;
        const bool pad = pads_input(l, p);
        if (pad) {
            if (want(li)) {
                if (hook) hook->before(l, li, s);
                e = launch_pad_channels(P->dtype, x, W.pad, (size_t)batch * l.H * l.W, l.C,
                                        l.cpad, s);
                if (hook) hook->after(l, li, s);
                if (e != hipSuccess) return e;
            }
            ++li;
        }
        const ConvGemmArgs a =
            gemm_args(P, l, batch, pad ? (const void*)W.pad : x, res, y, pad, W);
        if (want(li)) {
            if (hook) hook->before(l, li, s);
            e = launch_conv_gemm(P->dtype, p.cfg, p.wk, tapv_of(l, p), a, s);
            if (hook) hook->after(l, li, s);
            if (e != hipSuccess) return e;
        }
        ++li;
        if (p.splits > 1 && !l.softmax) {
            if (want(li)) {
                if (hook) hook->before(l, li, s);
                e = launch_splitk_reduce(P->dtype, a, s);
                if (hook) hook->after(l, li, s);
                if (e != hipSuccess) return e;
            }
            ++li;
        }
        if (l.softmax && want(li)) {
            if (hook) hook->before(l, li, s);
            e = p.splits > 1 ? launch_softmax_rows(a.partial, p.splits, l.scale, l.bias, a.M,
                                                   l.Co, (float*)y, s)
                             : launch_softmax_rows(a.logits, 1, nullptr, nullptr, a.M, l.Co,
                                                   (float*)y, s);
            if (hook) hook->after(l, li, s);
        }
        (void)roles;
        return e;
    }
    case K_DW:
        if (hook) hook->before(l, 0, s);
        e = launch_dwconv(P->dtype, x, l.w, l.scale, l.bias, y, batch, l.H, l.W, l.C, l.Ho,
                          l.Wo, l.k, l.stride, l.pad, l.act, P->tune.dw_outputs, s);
        if (hook) hook->after(l, 0, s);
        return e;
    case K_MAXPOOL:
        if (hook) hook->before(l, 0, s);
        e = launch_maxpool(P->dtype, x, y, batch, l.H, l.W, l.C, l.Ho, l.Wo, l.k, l.stride,
                           l.pad, s);
        if (hook) hook->after(l, 0, s);
        return e;
    default:
        if (hook) hook->before(l, 0, s);
        e = launch_gap(P->dtype, x, y, batch, l.H * l.W, l.C, s);
        if (hook) hook->after(l, 0, s);
        return e;
    }
}

// The whole range in layer order.  Without a hook (the run and capture
// paths), paired layers whose plans allow it go out as one launch at the
// lead's position; runs with a hook (per-layer and per-launch timing) keep
// one launch sequence per layer.
hipError_t enqueue_all(const ppipe_partition* P, int batch, const void* in, void* out,
                       hipStream_t s, LaunchHook* hook, const Workspace* wsp = nullptr)
{
    const Workspace W = wsp ? *wsp : handle_workspace(P);
    for (const LayerRT& l : P->L) {
        hipError_t e;
        if (!hook && l.pair >= 0 && pair_runs(P, l.pair_lead ? l : P->L[l.pair],
                                              l.pair_lead ? P->L[l.pair] : l, batch)) {
            if (!l.pair_lead)
                continue;   // ran with its lead
            const LayerRT& m = P->L[l.pair];
            const ConvGemmArgs a0 = gemm_args(P, l, batch, buf_ptr(P, l.in_buf, in, out),
                                              buf_ptr(P, l.res_buf, in, out),
                                              const_cast<void*>(buf_ptr(P, l.out_buf, in, out)),
                                              false, W);
            const ConvGemmArgs a1 = gemm_args(P, m, batch, buf_ptr(P, m.in_buf, in, out),
                                              buf_ptr(P, m.res_buf, in, out),
                                              const_cast<void*>(buf_ptr(P, m.out_buf, in, out)),
                                              false, W);
            e = launch_conv_gemm_pair(P->dtype, l.plans[batch - 1].cfg, a0, a1, s);
        } else {
            e = enqueue_layer(P, l, batch, in, out, s, hook, -1, &W);
        }
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

int check_run_args(const ppipe_partition* P, int batch, const void* in, const void* out)
{
    if (!P) return fail(PPIPE_E_INVALID, "null partition handle");
    if (batch < 1 || batch > P->max_batch)
        return fail(PPIPE_E_INVALID, "batch " + std::to_string(batch) + " outside [1, " +
                                         std::to_string(P->max_batch) + "]");
    if (!in || !out) return fail(PPIPE_E_INVALID, "null input or output pointer");
    if (in == out) return fail(PPIPE_E_INVALID, "input and output must not alias");
    return PPIPE_OK;
}

int ensure_device(const ppipe_partition* P)
{
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipGetDevice", e));
    if (cur != P->device) {
        e = hipSetDevice(P->device);
        if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipSetDevice", e));
    }
    return PPIPE_OK;
}

void release_timed(ppipe_partition* P)
{
    for (hipEvent_t e : P->timed.ev) (void)hipEventDestroy(e);
    P->timed.ev.clear();
    P->timed.batch = 0;
    P->timed.ran = false;
}

void release(ppipe_partition* P)
{
    release_timed(P);
    for (GraphEntry& g : P->graphs) {
        (void)hipGraphExecDestroy(g.exec);
        (void)hipGraphDestroy(g.graph);
    }
    P->graphs.clear();
    for (void* s : P->slots) (void)hipFree(s);
    P->slots.clear();
    if (P->ws) (void)hipFree(P->ws);
    if (P->pad_buf) (void)hipFree(P->pad_buf);
    P->pad_buf = nullptr;

    if (P->wblob) (void)hipFree(P->wblob);
    if (P->cap_stream) (void)hipStreamDestroy(P->cap_stream);
    P->ws = nullptr;
    P->wblob = nullptr;
    P->cap_stream = nullptr;
}

float median_of(std::vector<float> v)
{
    if (v.empty()) return 0.0f;
    std::sort(v.begin(), v.end());
    const size_t n = v.size();
    return n % 2 ? v[n / 2] : 0.5f * (v[n / 2 - 1] + v[n / 2]);
}

int build(ppipe_partition* P, const ppipe_model_desc* d, int begin, int end, int dt)
{
    const int n = d->n_layers;
    const int esz = dtype_size(dt);
    const int epv = 16 / esz;
    // ---- shapes of every layer up to end, from the model input ----
    std::vector<Shape> sh(end);
    auto shape_of = [&](int i) { return i < 0 ? Shape{d->in_c, d->in_h, d->in_w} : sh[i]; };
    for (int i = 0; i < end; ++i) {
        const ppipe_layer_desc& ld = d->layers[i];
        const std::string who = "layer " + std::to_string(i);
        if (ld.src < -1 || ld.src >= i)
            return fail(PPIPE_E_INVALID, who + ": src must name an earlier layer or -1");
        if (ld.res_src < -1 || ld.res_src >= i)
            return fail(PPIPE_E_INVALID, who + ": res_src must name an earlier layer or -1");
        const Shape x = shape_of(ld.src);
        if (ld.op == PPIPE_OP_CONV || ld.op == PPIPE_OP_MAXPOOL) {
            if (ld.k < 1 || ld.stride < 1 || ld.pad < 0 || ld.pad >= ld.k)
                return fail(PPIPE_E_INVALID, who + ": need k >= 1, stride >= 1, 0 <= pad < k");
            const int ho = (x.h + 2 * ld.pad - ld.k) / ld.stride + 1;
            const int wo = (x.w + 2 * ld.pad - ld.k) / ld.stride + 1;
            if (x.h + 2 * ld.pad < ld.k || x.w + 2 * ld.pad < ld.k || ho < 1 || wo < 1)
                return fail(PPIPE_E_INVALID, who + ": window larger than the padded input");
            if (ld.op == PPIPE_OP_CONV) {
                if (ld.c_in != x.c)
                    return fail(PPIPE_E_INVALID, who + ": c_in " + std::to_string(ld.c_in) +
                                                     " != producer channels " + std::to_string(x.c));
                if (ld.c_out < 1 || ld.groups < 1 || ld.c_in % ld.groups || ld.c_out % ld.groups)
                    return fail(PPIPE_E_INVALID, who + ": bad groups / channel counts");
                sh[i] = {ld.c_out, ho, wo};
            } else {
                sh[i] = {x.c, ho, wo};
            }
        } else if (ld.op == PPIPE_OP_AVGPOOL_GLOBAL) {
            sh[i] = {x.c, 1, 1};
        } else if (ld.op == PPIPE_OP_FC || ld.op == PPIPE_OP_FC_SOFTMAX) {
            if ((int64_t)ld.c_in != (int64_t)x.c * x.h * x.w)
                return fail(PPIPE_E_INVALID, who + ": fc c_in != flattened producer size");
            if (ld.c_out < 1)
                return fail(PPIPE_E_INVALID, who + ": fc c_out < 1");
            sh[i] = {ld.c_out, 1, 1};
        } else {
            return fail(PPIPE_E_INVALID, who + ": unknown op " + std::to_string(ld.op));
        }
        if (ld.res_src != -1) {
            const Shape r = shape_of(ld.res_src);
            if (ld.op != PPIPE_OP_CONV)
                return fail(PPIPE_E_UNSUPPORTED, who + ": residual add only on CONV layers");
            if (r.c != sh[i].c || r.h != sh[i].h || r.w != sh[i].w)
                return fail(PPIPE_E_INVALID, who + ": residual shape differs from output");
        }
    }
    // ---- the split: one feature map enters, one leaves ----
    for (int i = begin; i < end; ++i) {
        const ppipe_layer_desc& ld = d->layers[i];
        const int refs[2] = {ld.src, ld.res_src};
        for (int t = 0; t < 2; ++t) {
            const int r = refs[t];
            if (t == 1 && r == -1) continue;   // no residual
            if (r >= begin || r == begin - 1) continue;
            return fail(PPIPE_E_SPLIT, "layer " + std::to_string(i) + " reads layer " +
                                           std::to_string(r) + ", produced before the partition "
                                           "input (layer " + std::to_string(begin - 1) + ")");
        }
        if (ld.op == PPIPE_OP_FC_SOFTMAX && i != end - 1)
            return fail(PPIPE_E_UNSUPPORTED, "layer " + std::to_string(i) +
                                                 ": FC_SOFTMAX must be the range's last layer");
    }
    for (int j = end; j < n; ++j) {
        const ppipe_layer_desc& ld = d->layers[j];
        const int refs[2] = {ld.src, ld.res_src};
        for (int r : refs)
            if (r >= begin && r < end - 1)
                return fail(PPIPE_E_SPLIT, "layer " + std::to_string(j) + " (after the range) "
                                           "reads layer " + std::to_string(r) + " inside it");
    }

    // ---- per-layer runtime records and kernel constraints ----
    P->L.resize(end - begin);
    for (int i = begin; i < end; ++i) {
        const ppipe_layer_desc& ld = d->layers[i];
        LayerRT& l = P->L[i - begin];
        const Shape x = shape_of(ld.src), o = sh[i];
        const std::string who = "layer " + std::to_string(i);
        l.index = i; l.op = ld.op; l.src = ld.src; l.res_src = ld.res_src; l.act = ld.act;
        l.name = ld.name && ld.name[0] ? std::string(ld.name) : "layer" + std::to_string(i);
        l.k = ld.k; l.stride = ld.stride; l.pad = ld.pad; l.groups = ld.groups;
        l.H = x.h; l.W = x.w; l.C = x.c; l.Ho = o.h; l.Wo = o.w; l.Co = o.c;
        if (ld.act < PPIPE_ACT_NONE || ld.act > PPIPE_ACT_RELU6)
            return fail(PPIPE_E_INVALID, who + ": unknown activation");
        l.out_bytes_b1 = (int64_t)o.c * o.h * o.w * esz;
        l.in_bytes_b1 = (double)x.c * x.h * x.w * esz;
        l.res_bytes_b1 = ld.res_src >= 0 ? (double)l.out_bytes_b1 : 0.0;
        if (ld.op == PPIPE_OP_CONV && ld.groups > 1) {
            if (!(ld.groups == ld.c_in && ld.c_in == ld.c_out))
                return fail(PPIPE_E_UNSUPPORTED, who + ": grouped conv other than depthwise");
            if (ld.k != 3 || x.c % epv || ld.res_src >= 0 || (ld.stride != 1 && ld.stride != 2))
                return fail(PPIPE_E_UNSUPPORTED, who + ": depthwise kernel needs k = 3, stride 1 "
                                                     "or 2, C % " + std::to_string(epv) +
                                                     " == 0, no residual");
            // input is addressed with 32-bit byte offsets (buffer loads)
            if ((double)P->max_batch * x.c * x.h * x.w * esz >= 2147483648.0)
                return fail(PPIPE_E_UNSUPPORTED, who + ": input reaches 2 GiB at max_batch");
            if (!ld.weight)
                return fail(PPIPE_E_INVALID, who + ": missing weight");
            l.kind = K_DW;
            l.flops_b1 = 2.0 * o.c * o.h * o.w * ld.k * ld.k;
            l.param_bytes = (double)ld.k * ld.k * o.c * esz + 8.0 * o.c;
        } else if (ld.op == PPIPE_OP_CONV || ld.op == PPIPE_OP_FC ||
                   ld.op == PPIPE_OP_FC_SOFTMAX) {
            l.kind = K_GEMM;
            l.softmax = ld.op == PPIPE_OP_FC_SOFTMAX;
            if (ld.op == PPIPE_OP_CONV) {
                l.KH = l.KW = ld.k;
                l.gstride = ld.stride;
                l.gpad = ld.pad;
            } else {   // fc = valid H x W convolution producing 1 x 1
                l.KH = x.h;
                l.KW = x.w;
                l.gstride = 1;
                l.gpad = 0;
                if (l.softmax && o.c > SOFTMAX_MAX_O)
                    return fail(PPIPE_E_UNSUPPORTED, who + ": softmax over more than " +
                                                         std::to_string(SOFTMAX_MAX_O) + " classes");
            }
            if (o.c % 4)
                return fail(PPIPE_E_UNSUPPORTED, who + ": output channels must be a multiple of 4");
            // channels as the GEMM reads them: whole 16-byte vectors
            l.cpad = (x.c + epv - 1) / epv * epv;
            l.pad_in = l.cpad != x.c;
            l.K = l.KH * l.KW * l.cpad;
            l.Kpad = (l.K + 63) / 64 * 64;
            const int bk = gemm_bk(GEMM_64x64, dt);   // every LDS config uses the same BK
            // stage-uniform tap (1x1, or C a multiple of the stage) or per-vector taps
            l.tapv = !(l.KH * l.KW == 1 || l.cpad % bk == 0);
            // skinny kernel: each 64-byte K step lies in one (kh, kw) tap
            l.skinny_ok = l.KH * l.KW == 1 || l.cpad % (4 * epv) == 0;
            // streaming 1x1 kernel: 16-bit, stride 1, unpadded, one MFMA k-step
            // (up to five with at most 32 output channels)
            l.pw_ok = dt != DT_F32 && ld.op == PPIPE_OP_CONV && l.KH * l.KW == 1 &&
                      l.gstride == 1 && l.gpad == 0 && !l.pad_in &&
                      (x.c <= 32 || (x.c <= 160 && o.c <= 32));
            // stem kernel: an image of at most 4 channels (below one vector), <= 52 taps
            l.stem_ok = ld.op == PPIPE_OP_CONV && l.pad_in && x.c <= 4 && l.KH * l.KW <= 52;
            if (l.tapv && l.Kpad / epv > GEMM_VTAB_MAX)
                return fail(PPIPE_E_UNSUPPORTED, who + ": reduction length " +
                                                     std::to_string(l.K) + " with C = " +
                                                     std::to_string(x.c) + " is not supported");
            if (!ld.weight)
                return fail(PPIPE_E_INVALID, who + ": missing weight");
            // operands are addressed with 32-bit byte offsets (buffer loads)
            if ((double)P->max_batch * l.cpad * x.h * x.w * esz >= 2147483648.0 ||
                (double)o.c * ((l.K + 63) / 64 * 64) * esz >= 2147483648.0)
                return fail(PPIPE_E_UNSUPPORTED, who + ": input or weights reach 2 GiB at "
                                                       "max_batch");
            if (l.KH > 32 || l.KW > 32)
                return fail(PPIPE_E_UNSUPPORTED, who + ": window larger than 32");
            l.flops_b1 = 2.0 * o.c * o.h * o.w * (double)(l.KH * l.KW * x.c);
            l.param_bytes = (double)o.c * l.KH * l.KW * x.c * esz + 8.0 * o.c;
        } else if (ld.op == PPIPE_OP_MAXPOOL) {
            if (x.c % epv)
                return fail(PPIPE_E_UNSUPPORTED, who + ": maxpool needs C % " +
                                                     std::to_string(epv) + " == 0");
            l.kind = K_MAXPOOL;
            l.flops_b1 = 0;
        } else {
            if (x.c % epv)
                return fail(PPIPE_E_UNSUPPORTED, who + ": avgpool needs C % " +
                                                     std::to_string(epv) + " == 0");
            l.kind = K_GAP;
            l.flops_b1 = (double)x.c * x.h * x.w;
        }
        if (ld.op == PPIPE_OP_CONV && ld.bn_gamma &&
            !(ld.bn_beta && ld.bn_mean && ld.bn_var))
            return fail(PPIPE_E_INVALID, who + ": batch norm needs gamma, beta, mean and var");
    }

    // ---- weights, folded scale / shift: one device blob ----
    auto align = [](size_t v) { return (v + 255) / 256 * 256; };
    size_t total = 0;
    for (LayerRT& l : P->L) {
        if (l.kind == K_GEMM) {
            l.w_off = total; total = align(total + (size_t)l.Co * l.Kpad * esz);
        } else if (l.kind == K_DW) {
            l.w_off = total; total = align(total + (size_t)l.k * l.k * l.Co * esz);
        } else {
            continue;
        }
        l.scale_off = total; total = align(total + (size_t)l.Co * 4);
        l.bias_off = total; total = align(total + (size_t)l.Co * 4);
    }
    std::vector<uint8_t> blob(std::max<size_t>(total, 256), 0);
    for (LayerRT& l : P->L) {
        if (l.kind != K_GEMM && l.kind != K_DW) continue;
        const ppipe_layer_desc& ld = d->layers[l.index];
        if (l.kind == K_GEMM) {
            if (l.op == PPIPE_OP_CONV) {
                // OIHW [co][ci][kh][kw] -> [co][(kh * KW + kw) * cpad + ci]
                for (int co = 0; co < l.Co; ++co)
                    for (int ci = 0; ci < l.C; ++ci)
                        for (int kh = 0; kh < l.KH; ++kh)
                            for (int kw = 0; kw < l.KW; ++kw)
                                put_elem(blob, l.w_off, dt,
                                         (size_t)co * l.Kpad + (size_t)(kh * l.KW + kw) * l.cpad + ci,
                                         ld.weight[(((size_t)co * l.C + ci) * l.KH + kh) * l.KW + kw]);
            } else {
                // [o][c * H * W + h * W + w] -> [o][(h * W + w) * cpad + c]
                const size_t in_feat = (size_t)l.C * l.KH * l.KW;
                for (int co = 0; co < l.Co; ++co)
                    for (int c = 0; c < l.C; ++c)
                        for (int h = 0; h < l.KH; ++h)
                            for (int w = 0; w < l.KW; ++w)
                                put_elem(blob, l.w_off, dt,
                                         (size_t)co * l.Kpad + (size_t)(h * l.KW + w) * l.cpad + c,
                                         ld.weight[(size_t)co * in_feat + ((size_t)c * l.KH + h) * l.KW + w]);
            }
        } else {
            // depthwise OIHW [c][1][kh][kw] -> [kh][kw][c]
            for (int c = 0; c < l.Co; ++c)
                for (int kh = 0; kh < l.k; ++kh)
                    for (int kw = 0; kw < l.k; ++kw)
                        put_elem(blob, l.w_off, dt, (size_t)(kh * l.k + kw) * l.Co + c,
                                 ld.weight[((size_t)c * l.k + kh) * l.k + kw]);
        }
        float* sc = (float*)&blob[l.scale_off];
        float* bi = (float*)&blob[l.bias_off];
        const bool bn = l.op == PPIPE_OP_CONV && ld.bn_gamma;
        const double eps = ld.bn_eps > 0.0f ? (double)ld.bn_eps : 1e-5;
        for (int c = 0; c < l.Co; ++c) {
            const double b0 = ld.bias ? (double)ld.bias[c] : 0.0;
            if (bn) {
                // (acc + b0 - mean) / sqrt(var + eps) * gamma + beta = acc * s + t
                const double s = (double)ld.bn_gamma[c] / std::sqrt((double)ld.bn_var[c] + eps);
                sc[c] = (float)s;
                bi[c] = (float)((double)ld.bn_beta[c] + (b0 - (double)ld.bn_mean[c]) * s);
            } else {
                sc[c] = 1.0f;
                bi[c] = (float)b0;
            }
        }
    }
    P->host_blob.swap(blob);

    // ---- paired GEMMs ----
    // A GEMM layer and a later GEMM layer reading the same tensor (a residual
    // stage's first convolution and its downsample projection) may run as one
    // launch; the later one's output is then written at the earlier one's
    // position.  Neither may be the last layer, take the softmax or need the
    // channel-padding pass or the per-vector tap table.
    auto pairable = [&](const LayerRT& l, int i) {
        return l.kind == K_GEMM && !l.softmax && !l.pad_in && !l.tapv && i < end - 1;
    };
    for (int i = begin; i < end; ++i) {
        LayerRT& a = P->L[i - begin];
        if (a.pair >= 0 || !pairable(a, i)) continue;
        for (int j = i + 1; j < end; ++j) {
            LayerRT& b = P->L[j - begin];
            // the pair runs at i's position, so j's residual (if any) must
            // already exist there: produced before layer i
            const int rj = d->layers[j].res_src;
            if (b.pair < 0 && pairable(b, j) && d->layers[j].src == d->layers[i].src &&
                (rj == -1 || rj < i)) {
                a.pair = j - begin;
                a.pair_lead = true;
                b.pair = i - begin;
                break;
            }
        }
    }

    // ---- activation buffers by liveness ----
    // A paired layer's output slot is taken at its lead's position, so that
    // it is reserved whichever order the two run in.
    std::vector<int> last_use(end - begin, -1);
    for (int i = begin; i < end; ++i) {
        const ppipe_layer_desc& ld = d->layers[i];
        for (int r : {ld.src, ld.res_src})
            if (r >= begin) last_use[r - begin] = std::max(last_use[r - begin], i);
    }
    std::vector<int> slot_busy_until;
    auto take_slot = [&](LayerRT& l, int i, int at) {
        const size_t need = (size_t)P->max_batch * (size_t)l.out_bytes_b1;
        int slot = -1;
        for (size_t s = 0; s < slot_busy_until.size(); ++s)
            if (slot_busy_until[s] < at) {
                // prefer a free slot that is already large enough
                if (slot < 0 || (P->slot_bytes[s] >= need && P->slot_bytes[slot] < need))
                    slot = (int)s;
            }
        if (slot < 0) {
            slot = (int)slot_busy_until.size();
            slot_busy_until.push_back(-1);
            P->slot_bytes.push_back(0);
        }
        slot_busy_until[slot] = std::max(last_use[i - begin], i);
        P->slot_bytes[slot] = std::max(P->slot_bytes[slot], need);
        l.out_buf = slot;
    };
    for (int i = begin; i < end; ++i) {
        LayerRT& l = P->L[i - begin];
        const ppipe_layer_desc& ld = d->layers[i];
        l.in_buf = ld.src >= begin ? P->L[ld.src - begin].out_buf : BUF_IN;
        l.res_buf = ld.res_src == -1 ? BUF_NONE
                    : (ld.res_src >= begin ? P->L[ld.res_src - begin].out_buf : BUF_IN);
        if (i == end - 1) {
            l.out_buf = BUF_OUT;
            break;
        }
        if (l.pair >= 0 && !l.pair_lead)
            continue;                        // slot taken with its lead
        take_slot(l, i, i);
        if (l.pair_lead)
            take_slot(P->L[l.pair], begin + l.pair, i);
    }

    // ---- kernel plans for every batch, logits workspace ----
    size_t ws = 0;
    for (LayerRT& l : P->L) {
        if (l.kind != K_GEMM) continue;
        l.plans.resize(P->max_batch);
        for (int b = 1; b <= P->max_batch; ++b) {
            const int M = b * l.Ho * l.Wo;
            const Plan p = choose_plan(M, l.Co, l.K, dt, l.skinny_ok, l.pw_ok, l.stem_ok,
                                       l.softmax, P->tune, P->cus);
            l.plans[b - 1] = p;
            size_t need = 0;
            if (p.splits > 1) need += (size_t)p.splits * M * l.Co;
            if (l.softmax) need += (size_t)M * l.Co;
            ws = std::max(ws, need * sizeof(float));
        }
    }
    P->ws_bytes = ws;
    for (const LayerRT& l : P->L)
        if (l.kind == K_GEMM)
            for (int b = 1; b <= P->max_batch; ++b)
                if (pads_input(l, l.plans[b - 1]))
                    P->pad_bytes = std::max(P->pad_bytes, (size_t)b * l.H * l.W * l.cpad * esz);
    const LayerRT& last = P->L.back();
    P->in = shape_of(d->layers[begin].src);
    P->out = {last.Co, last.Ho, last.Wo};
    P->out_dtype = last.softmax ? DT_F32 : dt;
    return PPIPE_OK;
}

// Device side of create: upload weights, allocate buffers, make the capture stream.
int allocate(ppipe_partition* P)
{
    hipError_t e = hipGetDevice(&P->device);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipGetDevice", e));
    e = hipMalloc(&P->wblob, P->host_blob.size());
    if (e != hipSuccess) return fail(PPIPE_E_NOMEM, hip_msg("hipMalloc(weights)", e));
    P->wbytes = P->host_blob.size();
    e = hipMemcpy(P->wblob, P->host_blob.data(), P->host_blob.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipMemcpy(weights)", e));
    std::vector<uint8_t>().swap(P->host_blob);
    for (LayerRT& l : P->L) {
        if (l.kind != K_GEMM && l.kind != K_DW) continue;
        l.w = (uint8_t*)P->wblob + l.w_off;
        l.scale = (float*)((uint8_t*)P->wblob + l.scale_off);
        l.bias = (float*)((uint8_t*)P->wblob + l.bias_off);
    }
    P->slots.assign(P->slot_bytes.size(), nullptr);
    for (size_t s = 0; s < P->slots.size(); ++s) {
        e = hipMalloc(&P->slots[s], P->slot_bytes[s]);
        if (e != hipSuccess) return fail(PPIPE_E_NOMEM, hip_msg("hipMalloc(activations)", e));
    }
    if (P->ws_bytes) {
        e = hipMalloc((void**)&P->ws, P->ws_bytes);
        if (e != hipSuccess) return fail(PPIPE_E_NOMEM, hip_msg("hipMalloc(split-K)", e));
    }

    if (P->pad_bytes) {
        e = hipMalloc(&P->pad_buf, P->pad_bytes);
        if (e != hipSuccess) return fail(PPIPE_E_NOMEM, hip_msg("hipMalloc(channel pad)", e));
    }
    e = hipStreamCreateWithFlags(&P->cap_stream, hipStreamNonBlocking);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipStreamCreate", e));
    return PPIPE_OK;
}

struct ProfileBuffers {
    void* in = nullptr;
    void* out = nullptr;
    hipStream_t s = nullptr;
    ~ProfileBuffers()
    {
        if (s) (void)hipStreamSynchronize(s);
        if (in) (void)hipFree(in);
        if (out) (void)hipFree(out);
        if (s) (void)hipStreamDestroy(s);
    }
};

int setup_profile(ppipe_partition* P, ProfileBuffers& pb)
{
    const size_t in_b = (size_t)P->max_batch * P->in.c * P->in.h * P->in.w * dtype_size(P->dtype);
    const size_t out_b = (size_t)P->max_batch * P->out.c * P->out.h * P->out.w *
                         dtype_size(P->out_dtype);
    hipError_t e = hipStreamCreateWithFlags(&pb.s, hipStreamNonBlocking);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipStreamCreate", e));
    if ((e = hipMalloc(&pb.in, in_b)) != hipSuccess ||
        (e = hipMalloc(&pb.out, out_b)) != hipSuccess)
        return fail(PPIPE_E_NOMEM, hip_msg("hipMalloc(profile buffers)", e));
    e = launch_fill_uniform(P->dtype, pb.in, in_b / dtype_size(P->dtype), 12345u, pb.s);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("fill", e));
    return PPIPE_OK;
}

}  // namespace

// Timing method shared by both profilers: a layer (or one launch) is
// enqueued `reps` times back to back between two events on the profiling
// stream; the per-launch time is the elapsed time / reps.  Repeating the
// same launch amortises the event and dispatch overhead that a pair of
// events around one short kernel would add.  Three such trials are taken
// and the median (and minimum) reported.
namespace {
constexpr int PROFILE_TRIALS = 3;

struct Events {
    hipEvent_t a = nullptr, b = nullptr;
    ~Events()
    {
        if (a) (void)hipEventDestroy(a);
        if (b) (void)hipEventDestroy(b);
    }
    hipError_t make()
    {
        hipError_t e = hipEventCreate(&a);
        return e == hipSuccess ? hipEventCreate(&b) : e;
    }
};

struct EventPool {
    std::vector<hipEvent_t> ev;
    ~EventPool()
    {
        for (hipEvent_t e : ev) (void)hipEventDestroy(e);
    }
    hipError_t make(int n)
    {
        ev.assign(n, nullptr);
        for (hipEvent_t& e : ev) {
            const hipError_t r = hipEventCreate(&e);
            if (r != hipSuccess) return r;
        }
        return hipSuccess;
    }
};

// Hands layer i's event pair to its first launch (start) and its last launch
// (stop), so that the pair spans the layer's kernels in a run.
struct LayerEventsHook : LaunchHook {
    LayerEventsHook(const std::vector<hipEvent_t>& e, int b) : ev(e), batch(b) {}
    ~LayerEventsHook() override { launch_events() = LaunchEvents{}; }
    const std::vector<hipEvent_t>& ev;
    int batch, layer = 0;
    void before(const LayerRT& l, int li, hipStream_t) override
    {
        const int n = layer_launches(l, batch);
        launch_events() = LaunchEvents{li == 0 ? ev[2 * layer] : nullptr,
                                       li == n - 1 ? ev[2 * layer + 1] : nullptr};
    }
    void after(const LayerRT& l, int li, hipStream_t) override
    {
        launch_events() = LaunchEvents{};
        if (li == layer_launches(l, batch) - 1) ++layer;
    }
};

template <typename F>
hipError_t time_reps(hipStream_t s, Events& ev, int reps, F&& enqueue, std::vector<float>& us)
{
    hipError_t e = hipEventRecord(ev.a, s);
    for (int r = 0; r < reps && e == hipSuccess; ++r)
        e = enqueue();
    if (e == hipSuccess) e = hipEventRecord(ev.b, s);
    if (e == hipSuccess) e = hipEventSynchronize(ev.b);
    if (e != hipSuccess) return e;
    float ms = 0;
    e = hipEventElapsedTime(&ms, ev.a, ev.b);
    us.push_back(ms * 1000.0f / (float)reps);
    return e;
}
// ---- fixed scratch memory of ppipe_partition_run_static_scratch ----
// One copy per device, allocated with the code object and held until the
// process ends.  Host code must not use the array's name as a device address
// (on the host it is only a stand-in): the device address comes from
// hipGetSymbolAddress, resolved once per device with that device current.
static __device__ __align__(256) unsigned char scratch[PPIPE_STATIC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};
hipError_t g_scratch_err[MAX_DEVICES] = {};
bool g_scratch_done[MAX_DEVICES] = {};

// Resolves the scratch array's address on the current device (once).
void resolve_scratch(int dev)
{
    if (dev < 0 || dev >= MAX_DEVICES) return;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (g_scratch_done[dev]) return;
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    g_scratch_err[dev] = e;
    g_scratch_ptr[dev] = e == hipSuccess ? ptr : nullptr;
    g_scratch_done[dev] = true;
}

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// Scratch bytes a run at `batch` needs: split-K partials and logits (the
// largest over the layers, each layer reuses the region), then the padded
// stem input.
void scratch_need(const ppipe_partition* P, int batch, size_t* ws_bytes, size_t* pad_bytes)
{
    size_t ws = 0, pad = 0;
    const int esz = dtype_size(P->dtype);
    for (const LayerRT& l : P->L) {
        if (l.kind != K_GEMM) continue;
        const Plan& p = l.plans[batch - 1];
        const size_t M = (size_t)batch * l.Ho * l.Wo;
        size_t n = 0;
        if (p.splits > 1) n += (size_t)p.splits * M * l.Co;
        if (l.softmax) n += M * l.Co;
        ws = std::max(ws, n * sizeof(float));
        if (pads_input(l, p)) pad = std::max(pad, (size_t)batch * l.H * l.W * l.cpad * esz);
    }
    *ws_bytes = ws;
    *pad_bytes = pad;
}

}  // namespace

extern "C" {

const char* ppipe_last_error(void) { return g_err.c_str(); }

int32_t ppipe_last_status(void) { return g_status; }

ppipe_partition* ppipe_partition_create(const ppipe_model_desc* desc, int32_t layer_begin,
                                        int32_t layer_end, int32_t dtype)
{
    return ppipe_partition_create_tuned(desc, layer_begin, layer_end, dtype, nullptr);
}

}   // extern "C"

namespace {

// Compute units of one of `parts` CU shares of the current device: the
// device's CUs in groups of 8 dealt round-robin to the shares (as
// ppipe_stream_create_cu_share deals them), the smallest share; 256 (one
// MI355X) when the device cannot be queried.
int share_cus(int parts)
{
    int cus = 256, dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        n > 0)
        cus = n;
    return std::max(8, cus / 8 / parts * 8);
}

ppipe_partition* create_partition(const ppipe_model_desc* desc, int32_t layer_begin,
                                  int32_t layer_end, int32_t dtype, const ppipe_tuning* tuning,
                                  int32_t parts)
{
    g_err.clear();
    g_status = 0;
    if (parts < 1 || parts > 8) {
        fail(PPIPE_E_INVALID, "CU shares must be 1..8, got " + std::to_string(parts));
        return nullptr;
    }
    if (tuning) {
        const ppipe_tuning& t = *tuning;
        if (t.gemm_cfg < -1 || t.gemm_cfg >= GEMM_NCFG || t.gemm_splits < 0 ||
            t.gemm_splits > 64 || t.stream_grid < 0 ||
            (t.dw_outputs != 0 && t.dw_outputs != 2 && t.dw_outputs != 4)) {
            fail(PPIPE_E_INVALID, "tuning override out of range");
            return nullptr;
        }
    }
    if (!desc || !desc->layers || desc->n_layers < 1) {
        fail(PPIPE_E_INVALID, "model description is empty");
        return nullptr;
    }
    if (dtype < PPIPE_F32 || dtype > PPIPE_BF16) {
        fail(PPIPE_E_INVALID, "unknown dtype " + std::to_string(dtype));
        return nullptr;
    }
    if (layer_begin < 0 || layer_end > desc->n_layers || layer_begin >= layer_end) {
        fail(PPIPE_E_INVALID, "layer range [" + std::to_string(layer_begin) + ", " +
                                  std::to_string(layer_end) + ") is empty or outside the model");
        return nullptr;
    }
    if (desc->in_c < 1 || desc->in_h < 1 || desc->in_w < 1) {
        fail(PPIPE_E_INVALID, "model input shape must be positive");
        return nullptr;
    }
    ppipe_partition* P = new ppipe_partition();
    if (tuning) {
        P->tune = *tuning;
        P->tuned = tuning->gemm_cfg >= 0 || tuning->no_pointwise || tuning->no_stem ||
                   tuning->stream_grid > 0 || tuning->no_pair || tuning->dw_outputs;
    }
    P->begin = layer_begin;
    P->end = layer_end;
    P->dtype = dtype;
    P->max_batch = desc->max_batch > 0 ? desc->max_batch : 64;
    P->cus = share_cus(parts);
    // host-side validation and packing first: a bad description fails
    // without touching the device
    if (build(P, desc, layer_begin, layer_end, dtype) != PPIPE_OK || allocate(P) != PPIPE_OK) {
        std::string msg = g_err;
        const int st = g_status;
        release(P);
        delete P;
        g_err = msg;
        g_status = st;
        return nullptr;
    }
    // set-up of the fixed scratch memory on this device (its address is
    // looked up once per device; ppipe_partition_run_static_scratch reports
    // a failure)
    resolve_scratch(P->device);
    return P;
}

}  // namespace

extern "C" {

ppipe_partition* ppipe_partition_create_tuned(const ppipe_model_desc* desc,
                                              int32_t layer_begin, int32_t layer_end,
                                              int32_t dtype, const ppipe_tuning* tuning)
{
    return create_partition(desc, layer_begin, layer_end, dtype, tuning, 1);
}

ppipe_partition* ppipe_partition_create_on_share(const ppipe_model_desc* desc,
                                                 int32_t layer_begin, int32_t layer_end,
                                                 int32_t dtype, int32_t parts)
{
    return create_partition(desc, layer_begin, layer_end, dtype, nullptr, parts);
}

void ppipe_partition_destroy(ppipe_partition* h)
{
    if (!h) return;
    ensure_device(h);
    // runs on the caller's streams are the caller's to finish (hipFree itself
    // waits for the device); the handle's own timed events are waited for here
    if (h->timed.ran && !h->timed.ev.empty()) (void)hipEventSynchronize(h->timed.ev.back());
    release(h);
    delete h;
}

int ppipe_partition_run(ppipe_partition* h, int32_t batch, const void* in, void* out,
                        void* stream)
{
    int rc = check_run_args(h, batch, in, out);
    if (rc != PPIPE_OK) return rc;
    if ((rc = ensure_device(h)) != PPIPE_OK) return rc;
    hipStream_t s = (hipStream_t)stream;
    for (const GraphEntry& g : h->graphs) {
        if (g.batch == batch && g.in == in && g.out == out) {
            hipError_t e = hipGraphLaunch(g.exec, s);
            if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipGraphLaunch", e));
            return PPIPE_OK;
        }
    }
    hipError_t e = enqueue_all(h, batch, in, out, s, nullptr);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("kernel launch", e));
    return PPIPE_OK;
}

int ppipe_partition_run_static_scratch(ppipe_partition* h, int32_t batch, const void* in,
                                       void* out, void* stream)
{
    int rc = check_run_args(h, batch, in, out);
    if (rc != PPIPE_OK) return rc;
    if ((rc = ensure_device(h)) != PPIPE_OK) return rc;
    size_t ws = 0, pad = 0;
    scratch_need(h, batch, &ws, &pad);
    if (align256(ws) + pad > (size_t)PPIPE_STATIC_SCRATCH_BYTES)
        return fail(PPIPE_E_INVALID,
                    "batch " + std::to_string(batch) + " needs " +
                        std::to_string(align256(ws) + pad) + " bytes of scratch, more than the " +
                        std::to_string((long long)PPIPE_STATIC_SCRATCH_BYTES) + " held");
    const int dev = h->device;
    if (dev < 0 || dev >= MAX_DEVICES)
        return fail(PPIPE_E_INVALID, "device index beyond the scratch table");
    void* base = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_scratch_mu);
        if (!g_scratch_done[dev] || g_scratch_err[dev] != hipSuccess || !g_scratch_ptr[dev])
            return fail(PPIPE_E_HIP, hip_msg("scratch address (hipGetSymbolAddress)",
                                             g_scratch_done[dev] ? g_scratch_err[dev]
                                                                 : hipErrorNotInitialized));
        base = g_scratch_ptr[dev];
    }
    // every scratch byte a kernel reads was written earlier in the same run
    // (split partials by the GEMM, logits by the GEMM, the padded input by
    // the pad kernel), so nothing needs clearing
    const Workspace W{ws ? (float*)base : nullptr, pad ? (uint8_t*)base + align256(ws) : nullptr};
    hipError_t e = enqueue_all(h, batch, in, out, (hipStream_t)stream, nullptr, &W);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("kernel launch", e));
    return PPIPE_OK;
}

int ppipe_partition_capture(ppipe_partition* h, int32_t batch, const void* in, void* out)
{
    int rc = check_run_args(h, batch, in, out);
    if (rc != PPIPE_OK) return rc;
    if ((rc = ensure_device(h)) != PPIPE_OK) return rc;
    for (const GraphEntry& g : h->graphs)
        if (g.batch == batch && g.in == in && g.out == out) return PPIPE_OK;
    hipError_t e = hipStreamBeginCapture(h->cap_stream, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipStreamBeginCapture", e));
    hipError_t le = enqueue_all(h, batch, in, out, h->cap_stream, nullptr);
    hipGraph_t g = nullptr;
    e = hipStreamEndCapture(h->cap_stream, &g);
    if (le != hipSuccess || e != hipSuccess) {
        if (g) (void)hipGraphDestroy(g);
        return fail(PPIPE_E_HIP, hip_msg("graph capture", le != hipSuccess ? le : e));
    }
    hipGraphExec_t x = nullptr;
    e = hipGraphInstantiate(&x, g, nullptr, nullptr, 0);
    if (e != hipSuccess) {
        (void)hipGraphDestroy(g);
        return fail(PPIPE_E_HIP, hip_msg("hipGraphInstantiate", e));
    }
    h->graphs.push_back({batch, in, out, g, x});
    return PPIPE_OK;
}

int ppipe_profile_layers(ppipe_partition* h, const int32_t* batch_sizes, int32_t n_batches,
                         int32_t warmup, int32_t reps, float* out_us, float* out_partition_us)
{
    if (!h) return fail(PPIPE_E_INVALID, "null partition handle");
    if (!batch_sizes || n_batches < 1 || warmup < 0 || reps < 1)
        return fail(PPIPE_E_INVALID, "need batch sizes, warmup >= 0 and reps >= 1");
    for (int j = 0; j < n_batches; ++j)
        if (batch_sizes[j] < 1 || batch_sizes[j] > h->max_batch)
            return fail(PPIPE_E_INVALID, "batch size outside [1, max_batch]");
    int rc = ensure_device(h);
    if (rc != PPIPE_OK) return rc;
    ProfileBuffers pb;
    if ((rc = setup_profile(h, pb)) != PPIPE_OK) return rc;
    Events ev;
    hipError_t e = ev.make();
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipEventCreate", e));
    const int nl = (int)h->L.size();
    EventPool lev;
    if ((e = lev.make(2 * nl)) != hipSuccess)
        return fail(PPIPE_E_HIP, hip_msg("hipEventCreate", e));
    for (int j = 0; j < n_batches; ++j) {
        const int b = batch_sizes[j];
        for (int w = 0; w < warmup && e == hipSuccess; ++w)
            e = enqueue_all(h, b, pb.in, pb.out, pb.s, nullptr);
        if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("kernel launch", e));
        // in sequence: every repetition runs the range in layer order; layer
        // i's time runs from its first kernel's start to its last kernel's end
        std::vector<std::vector<float>> t(nl);
        for (int r = 0; r < reps && e == hipSuccess; ++r) {
            LayerEventsHook hook(lev.ev, b);
            e = enqueue_all(h, b, pb.in, pb.out, pb.s, &hook);
            if (e == hipSuccess) e = hipStreamSynchronize(pb.s);
            for (int i = 0; i < nl && e == hipSuccess; ++i) {
                float ms = 0;
                e = hipEventElapsedTime(&ms, lev.ev[2 * i], lev.ev[2 * i + 1]);
                t[i].push_back(ms * 1000.0f);
            }
        }
        if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("profile run", e));
        for (int i = 0; i < nl; ++i)
            if (out_us) out_us[(size_t)i * n_batches + j] = median_of(t[i]);
        // whole range as run() executes it: one captured graph replayed
        hipGraph_t g = nullptr;
        hipGraphExec_t x = nullptr;
        e = hipStreamBeginCapture(pb.s, hipStreamCaptureModeThreadLocal);
        if (e == hipSuccess) {
            hipError_t le = enqueue_all(h, b, pb.in, pb.out, pb.s, nullptr);
            e = hipStreamEndCapture(pb.s, &g);
            if (e == hipSuccess) e = le;
        }
        if (e == hipSuccess) e = hipGraphInstantiate(&x, g, nullptr, nullptr, 0);
        std::vector<float> tp;
        for (int k = 0; k < PROFILE_TRIALS && e == hipSuccess; ++k)
            e = time_reps(pb.s, ev, reps, [&] { return hipGraphLaunch(x, pb.s); }, tp);
        if (x) (void)hipGraphExecDestroy(x);
        if (g) (void)hipGraphDestroy(g);
        if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("profile graph run", e));
        if (out_partition_us) out_partition_us[j] = median_of(tp);
    }
    return PPIPE_OK;
}

int ppipe_profile_kernels(ppipe_partition* h, int32_t batch, int32_t warmup, int32_t reps,
                          ppipe_kernel_record* records, int32_t capacity, int32_t* count)
{
    if (!h) return fail(PPIPE_E_INVALID, "null partition handle");
    if (batch < 1 || batch > h->max_batch || warmup < 0 || reps < 1 || !count)
        return fail(PPIPE_E_INVALID, "bad batch, warmup, reps or count pointer");
    int rc = ensure_device(h);
    if (rc != PPIPE_OK) return rc;
    int nlaunch = 0;
    for (const LayerRT& l : h->L) nlaunch += layer_launches(l, batch);
    *count = nlaunch;
    ProfileBuffers pb;
    if ((rc = setup_profile(h, pb)) != PPIPE_OK) return rc;
    Events ev;
    hipError_t e = ev.make();
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipEventCreate", e));
    for (int w = 0; w < warmup && e == hipSuccess; ++w)
        e = enqueue_all(h, batch, pb.in, pb.out, pb.s, nullptr);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("kernel launch", e));
    int k = 0;
    for (const LayerRT& l : h->L) {
        for (int j = 0; j < layer_launches(l, batch); ++j, ++k) {
            std::vector<float> t;
            for (int q = 0; q < PROFILE_TRIALS && e == hipSuccess; ++q)
                e = time_reps(pb.s, ev, reps, [&] {
                    return enqueue_layer(h, l, batch, pb.in, pb.out, pb.s, nullptr, j);
                }, t);
            if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("profile run", e));
            if (!records || k >= capacity) continue;
            ppipe_kernel_record& rec = records[k];
            std::memset(&rec, 0, sizeof(rec));
            rec.layer = l.index;
            rec.launch = j;
            std::snprintf(rec.kernel, sizeof(rec.kernel), "%s",
                          launch_name(h, l, batch, j).c_str());
            launch_work(h, l, batch, j, &rec.flops, &rec.bytes);
            double sum = 0;
            for (float v : t) sum += v;
            rec.mean_us = (float)(sum / t.size());
            rec.median_us = median_of(t);
            rec.min_us = *std::min_element(t.begin(), t.end());
        }
    }
    return PPIPE_OK;
}

int ppipe_profile_kernels_cold(ppipe_partition* h, int32_t batch, int32_t reps,
                               int64_t sweep_bytes, ppipe_kernel_record* records,
                               int32_t capacity, int32_t* count)
{
    if (!h) return fail(PPIPE_E_INVALID, "null partition handle");
    if (batch < 1 || batch > h->max_batch || reps < 1 || !count || sweep_bytes < (32 << 20))
        return fail(PPIPE_E_INVALID, "bad batch, reps, sweep size or count pointer");
    int rc = ensure_device(h);
    if (rc != PPIPE_OK) return rc;
    int nlaunch = 0;
    for (const LayerRT& l : h->L) nlaunch += layer_launches(l, batch);
    *count = nlaunch;
    ProfileBuffers pb;
    if ((rc = setup_profile(h, pb)) != PPIPE_OK) return rc;
    struct Sweep {
        void* p = nullptr;
        ~Sweep() { if (p) (void)hipFree(p); }
    } sw;
    hipError_t e = hipMalloc(&sw.p, (size_t)sweep_bytes);
    if (e != hipSuccess) return fail(PPIPE_E_NOMEM, hip_msg("hipMalloc(sweep buffer)", e));
    if ((e = hipMemsetAsync(sw.p, 0, (size_t)sweep_bytes, pb.s)) != hipSuccess)
        return fail(PPIPE_E_HIP, hip_msg("hipMemsetAsync", e));
    Events ev;
    if ((e = ev.make()) != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipEventCreate", e));
    // one warm run so that every buffer a launch reads holds its producer's data
    if ((e = enqueue_all(h, batch, pb.in, pb.out, pb.s, nullptr)) != hipSuccess)
        return fail(PPIPE_E_HIP, hip_msg("kernel launch", e));
    int k = 0;
    for (const LayerRT& l : h->L) {
        for (int j = 0; j < layer_launches(l, batch); ++j, ++k) {
            std::vector<float> t;
            for (int r = 0; r < reps && e == hipSuccess; ++r) {
                e = launch_cache_sweep(sw.p, (size_t)sweep_bytes, pb.s);
                if (e != hipSuccess) break;
                launch_events() = LaunchEvents{ev.a, ev.b};
                e = enqueue_layer(h, l, batch, pb.in, pb.out, pb.s, nullptr, j);
                launch_events() = LaunchEvents{};
                if (e == hipSuccess) e = hipEventSynchronize(ev.b);
                float ms = 0;
                if (e == hipSuccess) e = hipEventElapsedTime(&ms, ev.a, ev.b);
                t.push_back(ms * 1000.0f);
            }
            if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("cold profile run", e));
            if (!records || k >= capacity) continue;
            ppipe_kernel_record& rec = records[k];
            std::memset(&rec, 0, sizeof(rec));
            rec.layer = l.index;
            rec.launch = j;
            std::snprintf(rec.kernel, sizeof(rec.kernel), "%s",
                          launch_name(h, l, batch, j).c_str());
            launch_work(h, l, batch, j, &rec.flops, &rec.bytes);
            double sum = 0;
            for (float v : t) sum += v;
            rec.mean_us = (float)(sum / t.size());
            rec.median_us = median_of(t);
            rec.min_us = *std::min_element(t.begin(), t.end());
        }
    }
    return PPIPE_OK;
}

int ppipe_cast(const void* in, int32_t in_dtype, void* out, int32_t out_dtype, int64_t n,
               void* stream)
{
    if (n < 0 || in_dtype < PPIPE_F32 || in_dtype > PPIPE_BF16 || out_dtype < PPIPE_F32 ||
        out_dtype > PPIPE_BF16)
        return fail(PPIPE_E_INVALID, "bad dtype or negative element count");
    if (n > 0 && (!in || !out)) return fail(PPIPE_E_INVALID, "null buffer");
    const hipError_t e = launch_cast(in, in_dtype, out, out_dtype, (size_t)n,
                                     (hipStream_t)stream);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("cast launch", e));
    return PPIPE_OK;
}

int ppipe_stream_create_cu_share(int32_t part, int32_t parts, void** stream)
{
    if (parts < 1 || part < 0 || part >= parts || !stream)
        return fail(PPIPE_E_INVALID, "need 0 <= part < parts and a stream pointer");
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipGetDevice", e));
    hipDeviceProp_t prop;
    if ((e = hipGetDeviceProperties(&prop, dev)) != hipSuccess)
        return fail(PPIPE_E_HIP, hip_msg("hipGetDeviceProperties", e));
    const int ncu = prop.multiProcessorCount;
    if (ncu < parts) return fail(PPIPE_E_INVALID, "more shares than compute units");
    // CU i belongs to share (i / 8) mod parts.  The mask's CU numbering
    // goes round-robin over the 8 XCDs, and a mask that leaves an XCD empty
    // is refused (measured: strides of 2 and 4 fail, every mask below that
    // keeps CUs on all XCDs works); each share thus spans all XCDs.
    std::vector<uint32_t> mask((ncu + 31) / 32, 0u);
    int picked = 0;
    for (int cu = 0; cu < ncu; ++cu)
        if ((cu / 8) % parts == part) {
            mask[cu / 32] |= 1u << (cu % 32);
            ++picked;
        }
    if (picked == 0) return fail(PPIPE_E_INVALID, "empty compute-unit share");
    hipStream_t st = nullptr;
    e = hipExtStreamCreateWithCUMask(&st, (uint32_t)mask.size(), mask.data());
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipExtStreamCreateWithCUMask", e));
    *stream = (void*)st;
    return PPIPE_OK;
}

int ppipe_stream_destroy(void* stream)
{
    if (!stream) return PPIPE_OK;
    const hipError_t e = hipStreamDestroy((hipStream_t)stream);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipStreamDestroy", e));
    return PPIPE_OK;
}

int ppipe_split_points(const ppipe_model_desc* desc, int32_t* ok)
{
    if (!desc || !desc->layers || desc->n_layers < 1 || !ok)
        return fail(PPIPE_E_INVALID, "null or empty model description");
    const int n = desc->n_layers;
    // earliest layer index read by any layer at or after p (src -1 = model input)
    int earliest = n;   // sentinel: nothing read
    for (int p = n; p >= 0; --p) {
        if (p < n) {
            const ppipe_layer_desc& ld = desc->layers[p];
            earliest = std::min(earliest, ld.src);
            if (ld.res_src >= 0) earliest = std::min(earliest, ld.res_src);
        }
        ok[p] = (p == 0 || p == n || earliest >= p - 1) ? 1 : 0;
    }
    return PPIPE_OK;
}

int ppipe_prepartition(const double* layer_us, const int32_t* split_ok, int32_t n_layers,
                       int32_t n_blocks, int32_t* block_begin, int32_t* n_out)
{
    if (!layer_us || !split_ok || !block_begin || !n_out || n_layers < 1 || n_blocks < 1)
        return fail(PPIPE_E_INVALID, "null argument, no layers or no blocks");
    double total = 0;
    for (int i = 0; i < n_layers; ++i) {
        if (!(layer_us[i] >= 0.0)) return fail(PPIPE_E_INVALID, "negative or NaN layer latency");
        total += layer_us[i];
    }
    const double target = total / n_blocks;
    int nb = 0, start = 0;
    while (start < n_layers) {
        block_begin[nb++] = start;
        // the valid end whose block latency is closest to the target (the
        // earliest of equally close ones); sums only grow, so the scan stops
        // once the sum exceeds the target by the best gap found
        double sum = 0, best_gap = -1;
        int best_end = n_layers;
        for (int p = start + 1; p <= n_layers; ++p) {
            sum += layer_us[p - 1];
            if (p < n_layers && !split_ok[p]) continue;
            const double gap = std::fabs(sum - target);
            if (best_gap < 0 || gap < best_gap) {
                best_gap = gap;
                best_end = p;
            }
            if (sum - target >= best_gap) break;
        }
        start = best_end;
    }
    block_begin[nb] = n_layers;
    *n_out = nb;
    return PPIPE_OK;
}

int ppipe_timing_setup(ppipe_partition* h, int32_t batch, const void* in, void* out)
{
    int rc = check_run_args(h, batch, in, out);
    if (rc != PPIPE_OK) return rc;
    if ((rc = ensure_device(h)) != PPIPE_OK) return rc;
    // the events of an earlier timed run may still be pending: its last
    // event is recorded after its last launch on the same stream
    if (h->timed.ran && !h->timed.ev.empty()) (void)hipEventSynchronize(h->timed.ev.back());
    release_timed(h);
    int nlaunch = 0;
    for (const LayerRT& l : h->L) nlaunch += layer_launches(l, batch);
    h->timed.ev.assign(2 * (size_t)nlaunch, nullptr);
    for (hipEvent_t& e : h->timed.ev) {
        const hipError_t he = hipEventCreate(&e);
        if (he != hipSuccess) {
            release_timed(h);
            return fail(PPIPE_E_HIP, hip_msg("hipEventCreate", he));
        }
    }
    h->timed.batch = batch;
    h->timed.in = in;
    h->timed.out = out;
    return PPIPE_OK;
}

int ppipe_partition_run_timed(ppipe_partition* h, void* stream)
{
    if (!h) return fail(PPIPE_E_INVALID, "null partition handle");
    if (h->timed.batch < 1) return fail(PPIPE_E_INVALID, "ppipe_timing_setup was not called");
    int rc = ensure_device(h);
    if (rc != PPIPE_OK) return rc;
    TimedHook hook(h->timed.ev);
    const hipError_t e = enqueue_all(h, h->timed.batch, h->timed.in, h->timed.out,
                                     (hipStream_t)stream, &hook);
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("timed run", e));
    h->timed.ran = true;
    return PPIPE_OK;
}

int ppipe_timing_read(ppipe_partition* h, ppipe_kernel_record* records, int32_t capacity,
                      int32_t* count)
{
    if (!h || !count) return fail(PPIPE_E_INVALID, "null argument");
    if (!h->timed.ran) return fail(PPIPE_E_INVALID, "no timed run since ppipe_timing_setup");
    int rc = ensure_device(h);
    if (rc != PPIPE_OK) return rc;
    hipError_t e = hipEventSynchronize(h->timed.ev.back());
    if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipEventSynchronize", e));
    const int batch = h->timed.batch;
    int k = 0;
    for (const LayerRT& l : h->L) {
        for (int j = 0; j < layer_launches(l, batch); ++j, ++k) {
            if (!records || k >= capacity) continue;
            float ms = 0;
            e = hipEventElapsedTime(&ms, h->timed.ev[2 * k], h->timed.ev[2 * k + 1]);
            if (e != hipSuccess) return fail(PPIPE_E_HIP, hip_msg("hipEventElapsedTime", e));
            ppipe_kernel_record& rec = records[k];
            std::memset(&rec, 0, sizeof(rec));
            rec.layer = l.index;
            rec.launch = j;
            std::snprintf(rec.kernel, sizeof(rec.kernel), "%s",
                          launch_name(h, l, batch, j).c_str());
            launch_work(h, l, batch, j, &rec.flops, &rec.bytes);
            rec.mean_us = rec.median_us = rec.min_us = ms * 1000.0f;
        }
    }
    *count = k;
    return PPIPE_OK;
}

int ppipe_partition_info(const ppipe_partition* h, ppipe_partition_info_t* info)
{
    if (!h || !info) return fail(PPIPE_E_INVALID, "null argument");
    std::memset(info, 0, sizeof(*info));
    info->layer_begin = h->begin;
    info->layer_end = h->end;
    info->dtype = h->dtype;
    info->max_batch = h->max_batch;
    info->in_c = h->in.c; info->in_h = h->in.h; info->in_w = h->in.w;
    info->out_c = h->out.c; info->out_h = h->out.h; info->out_w = h->out.w;
    info->out_dtype = h->out_dtype;
    info->in_bytes_per_image = (int64_t)h->in.c * h->in.h * h->in.w * dtype_size(h->dtype);
    info->out_bytes_per_image = (int64_t)h->out.c * h->out.h * h->out.w * dtype_size(h->out_dtype);
    info->weight_bytes = (int64_t)h->wbytes;
    size_t ws = h->ws_bytes + h->pad_bytes;
    for (size_t b : h->slot_bytes) ws += b;
    info->workspace_bytes = (int64_t)ws;
    info->tuned = h->tuned ? 1 : 0;
    info->cus = h->cus;
    return PPIPE_OK;
}

int ppipe_layer_info(const ppipe_partition* h, int32_t index, int32_t batch,
                     ppipe_layer_info_t* info)
{
    if (!h || !info) return fail(PPIPE_E_INVALID, "null argument");
    if (index < h->begin || index >= h->end)
        return fail(PPIPE_E_INVALID, "layer index outside the partition");
    if (batch < 1 || batch > h->max_batch)
        return fail(PPIPE_E_INVALID, "batch outside [1, max_batch]");
    const LayerRT& l = h->L[index - h->begin];
    std::memset(info, 0, sizeof(*info));
    info->index = l.index;
    info->op = l.op;
    std::snprintf(info->name, sizeof(info->name), "%s", l.name.c_str());
    info->out_c = l.Co; info->out_h = l.Ho; info->out_w = l.Wo;
    info->kernel_count = layer_launches(l, batch);
    info->out_bytes_b1 = l.softmax ? (int64_t)l.Co * 4 : l.out_bytes_b1;
    info->flops_b1 = l.flops_b1;
    info->act_bytes_b1 = l.in_bytes_b1 + l.res_bytes_b1 + (double)info->out_bytes_b1;
    info->param_bytes = l.param_bytes;
    // name the GEMM launch of a GEMM layer, not its channel-pad prologue
    const std::vector<int> roles = launch_roles(l, batch);
    int main_launch = 0;
    for (size_t i = 0; i < roles.size(); ++i)
        if (roles[i] == L_GEMM) main_launch = (int)i;
    std::string k = launch_name(h, l, batch, main_launch);
    if (l.kind == K_GEMM) {
        const Plan& p = l.plans[batch - 1];
        k += " tiles=" + std::to_string(p.tiles_m * p.tiles_co) + " splits=" +
             std::to_string(p.splits);
        if (l.pair >= 0 && pair_runs(h, l.pair_lead ? l : h->L[l.pair],
                                     l.pair_lead ? h->L[l.pair] : l, batch))
            k += " paired=" + std::to_string(h->L[l.pair].index);
        info->forced = p.forced ? 1 : 0;
    }
    if (l.kind == K_DW && h->tune.dw_outputs) info->forced = 1;
    std::snprintf(info->kernel, sizeof(info->kernel), "%s", k.c_str());
    return PPIPE_OK;
}

}  // extern "C"
