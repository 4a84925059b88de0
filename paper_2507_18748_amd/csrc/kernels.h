// Internal interface between the partition runtime and the gfx950 kernels.
// Not part of the public ABI (include/ppipe.h is).
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <cstddef>
#include <cstdint>
#include <string>

namespace ppipe {

enum DType : int { DT_F32 = 0, DT_F16 = 1, DT_BF16 = 2 };

// Timing events for the next kernel launch of this host thread (set by the
// runtime's timed runs, null otherwise; either may be null alone).  With an
// event set, launches go through hipExtLaunchKernelGGL, which records the
// start event before and the stop event after the kernel itself.
struct LaunchEvents {
    hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents& launch_events();

#define PPIPE_LAUNCH(KERNEL, GRID, BLOCK, SHMEM, STREAM, ...)                                   \
    do {                                                                                         \
        const ::ppipe::LaunchEvents ev_ = ::ppipe::launch_events();                              \
        if (ev_.start || ev_.stop)                                                               \
            hipExtLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, ev_.start, ev_.stop, 0u,   \
                                  __VA_ARGS__);                                                  \
        else                                                                                     \
            hipLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, __VA_ARGS__);                 \
    } while (0)
enum Act : int { ACT_NONE = 0, ACT_RELU = 1, ACT_RELU6 = 2 };

// Records a failing call's status and message for ppipe_last_error(); returns status.
int set_error(int status, const std::string& msg);

inline int dtype_size(int dt) { return dt == DT_F32 ? 4 : 2; }

// Implicit-GEMM convolution over NHWC activations.
//   GEMM rows    co in [0, Co)            (weights, MFMA A operand)
//   GEMM columns m = (n, ho, wo) in [0, M) (activations gathered on the fly, MFMA B operand)
//   reduction    k = (kh, kw, ci) in [0, K), K = KH * KW * C
// Weights are packed [Co][Kpad] in the storage dtype with k ordered (kh, kw, ci)
// and zero padding up to Kpad (a multiple of 64 elements).
// Softmax mode writes fp32 logits (scale * sum + bias) to `logits` instead of
// the activation epilogue; launch_softmax_rows then normalises them.
struct ConvGemmArgs {
    const void* x;        // [N][H][W][C]
    const void* w;        // [Co][Kpad]
    const float* scale;   // [Co] folded batch-norm scale (1 without BN)
    const float* bias;    // [Co] folded shift
    const void* res;      // [M][Co] residual in dtype, or nullptr
    void* y;              // [M][Co] output in dtype
    float* logits;        // [M][Co] fp32 (softmax mode)
    float* partial;       // [splits][M][Co] fp32 raw sums (LDS kernel with splits > 1)
    int N, H, W, C;
    int Ho, Wo, Co;
    int KH, KW, stride, pad;
    int K, Kpad, M;
    int act;
    int total_chunks;     // LDS kernel: ceil(K / BK); skinny kernel: ceil(K / KS)
    int splits;           // LDS kernel: K ranges per tile (blockIdx spans tiles x splits)
    int chunks_per_split;
    int tiles_m, tiles_co;
    int co_fastest;       // tile order: 0 = m tiles of one weight slice adjacent, 1 = co tiles adjacent
    int softmax;          // 1: write fp32 logits for a following softmax
    int grid_blocks;      // pointwise kernel: cap on blocks along the pixels (0: resident set)
};

// Bring every field of the kernel arguments into scalar registers at once.
// Left to itself the compiler loads the argument struct in several batches,
// each waited for before the next goes out; a kernel-argument read costs
// ~0.25 us, so a GEMM block spent ~0.8 us before its first operand load.
// One asm statement that names every field makes all loads go out together;
// the block index passes through it, so no work that uses the arguments can
// be scheduled before it (which would split the loads again), and so does
// the grid size (a hidden kernel argument after the struct).
__device__ __forceinline__ int3 load_args_now(const ConvGemmArgs& a, int bid, int grid,
                                              int bid_y = 0)
{
    asm volatile("" : "+s"(bid), "+s"(grid), "+s"(bid_y) : "s"(a.x), "s"(a.w), "s"(a.scale), "s"(a.bias), "s"(a.res), "s"(a.y),
                 "s"(a.logits), "s"(a.partial), "s"(a.N), "s"(a.H), "s"(a.W), "s"(a.C),
                 "s"(a.Ho), "s"(a.Wo), "s"(a.Co), "s"(a.KH), "s"(a.KW), "s"(a.stride),
                 "s"(a.pad), "s"(a.K), "s"(a.Kpad), "s"(a.M), "s"(a.act), "s"(a.total_chunks),
                 "s"(a.splits), "s"(a.chunks_per_split), "s"(a.tiles_m), "s"(a.tiles_co),
                 "s"(a.co_fastest), "s"(a.softmax), "s"(a.grid_blocks));
    return make_int3(bid, grid, bid_y);
}

// Tile configurations (rows = co, columns = m).
//   LDS-tiled kernel for large M: blocks of 4 waves share staged tiles.
//   Skinny kernel for small M: a block of WK waves computes one small tile,
//   each wave a slice of K, operands loaded straight into registers.
enum GemmCfg : int {
    GEMM_128x128 = 0,   // LDS, 4 waves, 64x64 per wave
    GEMM_64x64 = 1,     // LDS, 4 waves, 32x32 per wave
    GEMM_64x128 = 2,    // LDS, 4 waves, 32x64 per wave (64 output channels, many pixels)
    GEMM_SK_32x32 = 3,  // skinny 32x32 tile
    GEMM_SK_32x16 = 4,  // skinny 32 co x 16 m
    GEMM_SK_16x32 = 5,  // skinny 16 co x 32 m
    GEMM_SK_16x16 = 6,  // skinny 16x16 tile
    GEMM_128x128_8W = 7,  // LDS, 8 waves, 64x32 per wave
    GEMM_128x64 = 8,    // LDS, 4 waves, 64x32 per wave
    // Operands loaded straight into a ring of LDS stages (no register staging).
    GEMM_DMA_64x64_S2 = 9,        // 4 waves, 32x32 per wave, 2 stages
    GEMM_DMA_64x64_S3 = 10,       // 4 waves, 3 stages, software-pipelined
    GEMM_DMA_128x128_8W_S2 = 11,  // 8 waves, 64x32 per wave, 2 stages
    GEMM_DMA_128x128_8W_S3 = 12,  // 8 waves, 3 stages, software-pipelined
    GEMM_DMA_64x64_8W_S2 = 13,    // 8 waves, 32x16 per wave, 2 stages
    GEMM_DMA_64x64_8W_S3 = 14,    // 8 waves, 3 stages, software-pipelined
    GEMM_DMA_64x64_8W_S4 = 15,    // 8 waves, 4 stages (two in flight)
    GEMM_DMA_64x64_8W_S6 = 16,    // 8 waves, 6 stages (four in flight; few blocks per CU)
    // Streaming 1x1 convolution (stride 1, C <= 32, or <= 160 into <= 32
    // channels): weights in registers,
    // 16-pixel groups loaded straight into MFMA fragments.  wk = 16-channel
    // fragments per block (pointwise_channel_frags).
    GEMM_PW = 17,
    // Stem of a C <= 4 channel image: one tap per 16-byte operand vector,
    // channels gathered per lane, weights staged in LDS.  wk = 16-channel
    // fragments per block (stem_channel_frags).
    GEMM_STEM = 18,
    GEMM_DMA_64x128_8W_S2 = 19,   // 8 waves, 32x32 per wave, 2 stages
    GEMM_DMA_64x256_8W_S2 = 20,   // 8 waves, 32 co x 64 m per wave, 2 stages
    // 32x32x16 matrix instructions (16-bit types only), 64x64 per wave,
    // per-k-step double-buffered fragments, NS-stage LDS-direct ring
    GEMM_MX_128x128_S2 = 21,      // 4 waves (2 x 2)
    GEMM_MX_128x128_S3 = 22,
    GEMM_MX_128x128_S4 = 23,
    GEMM_MX_256x128_S2 = 24,      // 8 waves (4 x 2): 256 channels x 128 pixels
    GEMM_MX_128x256_S2 = 25,      // 8 waves (2 x 4): 128 channels x 256 pixels
    GEMM_MX_256x128_S3 = 26,
    GEMM_MX_128x128_8W_S2 = 27,   // 8 waves (2 x 4): 64x32 per wave
    GEMM_MX_128x128_8W_S3 = 28,
    GEMM_DMA_64x64_2W_S2 = 29,    // 2 waves, 64x32 per wave, 2 stages
    GEMM_DMA_64x64_1W_S2 = 30,    // 1 wave, 64x64, 2 stages
    GEMM_DMA_64x64_2W_S3 = 31,    // 2 waves, 3 stages, software-pipelined
    GEMM_DMA_128x128_8W_S4 = 32,  // 8 waves, 4 stages (two in flight, one block per CU)
    GEMM_NCFG = 33
};
struct GemmCfgInfo {
    int bm, bn, kv;       // tile rows (co), columns (m); kv: 16-byte vectors of K per LDS stage
    bool skinny;
    int dma = 0;          // LDS stages of the DMA-staged kernel (0: register-staged)
    int waves = 4;        // waves per block (LDS kernels)
    int mfma = 16;        // 16: 16x16 matrix instructions; 32: 32x32x16 (16-bit types only)
};
GemmCfgInfo gemm_cfg_info(int cfg);
// K elements per pipeline step: an LDS stage, or one 64-byte MFMA k-step (skinny)
inline int gemm_bk(int cfg, int dt)
{
    const GemmCfgInfo c = gemm_cfg_info(cfg);
    return (c.skinny ? 4 : c.kv) * (16 / dtype_size(dt));
}

// Largest number of 16-byte K vectors the per-vector-tap (TAPV) path supports.
constexpr int GEMM_VTAB_MAX = 1024;
constexpr int SOFTMAX_MAX_O = 8192;
constexpr int SKINNY_MAX_WAVES = 16;

// wk: waves per block of the skinny kernel (K split), ignored by the LDS kernel.
// tapv: the LDS kernel looks up each 16-byte K vector's (kh, kw, ci) in a
// table (channel count a multiple of the vector width but not of the stage).
hipError_t launch_conv_gemm(int dt, int cfg, int wk, bool tapv, const ConvGemmArgs& a,
                            hipStream_t s);
// Two layers of one DMA tile configuration, each unsplit and without a
// softmax, in one launch (blocks of a0 first, then of a1).  The layers must
// not depend on each other; both take plain per-tap K steps (no per-vector
// tap table).
hipError_t launch_conv_gemm_pair(int dt, int cfg, const ConvGemmArgs& a0, const ConvGemmArgs& a1,
                                 hipStream_t s);
const char* conv_gemm_name(int dt, int cfg, int wk, bool tapv);

// Streaming 1x1 convolution (GEMM_PW) of a 16-bit layer with C <= 32, or
// C <= 160 with cf <= 2 (C a multiple of 8), Co % 4 == 0, stride 1, no
// padding, no K split, no softmax;
// cf 16-channel fragments per block, at most grid_blocks blocks along the
// pixels (0: one resident set), each wave walking 16-pixel groups grid-stride.
hipError_t launch_pointwise(int dt, int cf, const ConvGemmArgs& a, int grid_blocks, hipStream_t s);
int pointwise_channel_frags(int Co);

// Stem (GEMM_STEM): x is the unpadded image [N][H][W][C], C <= 4 and below
// one 16-byte vector, weights packed with the channels padded to a vector
// per tap, at most 52 taps; cf 16-channel fragments per block.
hipError_t launch_stem(int dt, int cf, const ConvGemmArgs& a, int grid_blocks, hipStream_t s);
int stem_channel_frags(int Co);

// Copy NHWC [npix][C] into [npix][Cp] (Cp > C) with zero channels appended,
// so that a layer with fewer channels than a 16-byte vector can be gathered
// with vector loads.
hipError_t launch_pad_channels(int dt, const void* x, void* y, size_t npix, int C, int Cp,
                               hipStream_t s);
const char* pad_channels_name(int dt);

// Sum of the split-K partials in split order, then the layer epilogue
// (scale, bias, residual, activation, rounding; or fp32 logits in softmax mode).
hipError_t launch_splitk_reduce(int dt, const ConvGemmArgs& a, hipStream_t s);
const char* splitk_reduce_name(int dt);

// Row-wise softmax into out [M][O] of fp32 logits z [M][O] (splits = 1,
// scale = bias = nullptr), or of raw split-K sums z [splits][M][O] finished
// as scale[o] * sum + bias[o] (the FC epilogue) before the softmax.
hipError_t launch_softmax_rows(const float* z, int splits, const float* scale, const float* bias,
                               int M, int O, float* out, hipStream_t s);
const char* softmax_rows_name();

// Depthwise k x k convolution (NHWC, weights [k][k][C] in dtype) with the
// folded batch norm and activation.  C % (16 / sizeof(dtype)) == 0.
hipError_t launch_dwconv(int dt, const void* x, const void* w, const float* scale,
                         const float* bias, void* y, int N, int H, int W, int C, int Ho,
                         int Wo, int k, int stride, int pad, int act, int pw_force,
                         hipStream_t s);
const char* dwconv_name(int dt, int k);

// k x k max pooling, NHWC; out-of-range taps never win.
hipError_t launch_maxpool(int dt, const void* x, void* y, int N, int H, int W, int C,
                          int Ho, int Wo, int k, int stride, int pad, hipStream_t s);
const char* maxpool_name(int dt);

// Mean over H x W per (n, c), fp32 sum, NHWC in -> [N][C] out.
hipError_t launch_gap(int dt, const void* x, void* y, int N, int HW, int C, hipStream_t s);
const char* gap_name(int dt);

// n elements of x (in_dt) converted to y (out_dt); narrowing rounds to
// nearest even.
hipError_t launch_cast(const void* x, int in_dt, void* y, int out_dt, size_t n, hipStream_t s);

// Read `buf` (all but its last 16 MiB, which receive one result per
// thread): isolated-cold profiling, evicts L2 and the memory-side cache
// before a timed launch.  bytes >= 32 MiB.
hipError_t launch_cache_sweep(void* buf, size_t bytes, hipStream_t s);

// Deterministic pseudo-random fill in [0, 1) for profiling inputs.
hipError_t launch_fill_uniform(int dt, void* p, size_t n, uint32_t seed, hipStream_t s);

}  // namespace ppipe
