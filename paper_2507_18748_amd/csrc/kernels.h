// Internal interface between the partition runtime and the gfx950 kernels.
// Not part of the public ABI (include/ppipe.h is).
#pragma once
#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

namespace ppipe {

enum DType : int { DT_F32 = 0, DT_F16 = 1, DT_BF16 = 2 };
enum Act : int { ACT_NONE = 0, ACT_RELU = 1, ACT_RELU6 = 2 };

inline int dtype_size(int dt) { return dt == DT_F32 ? 4 : 2; }

// Implicit-GEMM convolution over NHWC activations.
//   GEMM rows    co in [0, Co)            (weights, MFMA A operand)
//   GEMM columns m = (n, ho, wo) in [0, M) (activations gathered on the fly, MFMA B operand)
//   reduction    k = (kh, kw, ci) in [0, K), K = KH * KW * C
// Weights are packed [Co][Kpad] in the storage dtype with k ordered (kh, kw, ci)
// and zero padding up to Kpad (a multiple of 64 elements).
struct ConvGemmArgs {
    const void* x;        // [N][H][W][C]
    const void* w;        // [Co][Kpad]
    const float* scale;   // [Co] folded batch-norm scale (1 without BN)
    const float* bias;    // [Co] folded shift
    const void* res;      // [M][Co] residual in dtype, or nullptr
    void* y;              // [M][Co] output in dtype (out_mode 0)
    float* partial;       // [splits][M][Co] fp32 (out_mode 1)
    int N, H, W, C;
    int Ho, Wo, Co;
    int KH, KW, stride, pad;
    int K, Kpad, M;
    int act;
    int total_chunks;     // ceil(K / BK)
    int chunks_per_split; // BK chunks handled by each blockIdx.z
    int out_mode;         // 0: fused epilogue into y; 1: raw fp32 sums into partial[split]
};

// Tile configurations of the MFMA kernel (rows = co, columns = m).
enum GemmCfg : int {
    GEMM_128x128 = 0,   // 4 waves, 64x64 per wave
    GEMM_64x64 = 1,     // 4 waves, 32x32 per wave
    GEMM_64x16 = 2,     // 4 waves, 16x16 per wave (small M: FC at batch <= 16)
    GEMM_NCFG = 3
};
struct GemmCfgInfo {
    int bm, bn, threads, kv;   // kv: 16-byte vectors of K per LDS stage
};
GemmCfgInfo gemm_cfg_info(int cfg);
inline int gemm_bk(int cfg, int dt) { return gemm_cfg_info(cfg).kv * (16 / dtype_size(dt)); }

// Largest K (elements) the generic (scalar-gather) path supports.
constexpr int GEMM_KTAB_MAX = 2048;

hipError_t launch_conv_gemm(int dt, int cfg, bool generic, const ConvGemmArgs& a,
                            int splits, hipStream_t s);
const char* conv_gemm_name(int dt, int cfg, bool generic);

// Sum of split-K partials followed by the conv epilogue (scale, bias,
// residual, activation, rounding to dtype).  Co % 4 == 0.
hipError_t launch_splitk_epilogue(int dt, const float* partial, int splits, int M, int Co,
                                  const float* scale, const float* bias, const void* res,
                                  int act, void* y, hipStream_t s);
const char* splitk_epilogue_name(int dt);

// Sum of split-K partials + bias, then softmax over each row; fp32 output [M][O].
constexpr int SOFTMAX_MAX_O = 8192;
hipError_t launch_splitk_softmax(const float* partial, int splits, int M, int O,
                                 const float* bias, float* out, hipStream_t s);
const char* splitk_softmax_name();

// Depthwise k x k convolution (NHWC, weights [k][k][C] in dtype) with the
// folded batch norm and activation.  C % (16 / sizeof(dtype)) == 0.
hipError_t launch_dwconv(int dt, const void* x, const void* w, const float* scale,
                         const float* bias, void* y, int N, int H, int W, int C, int Ho,
                         int Wo, int k, int stride, int pad, int act, hipStream_t s);
const char* dwconv_name(int dt, int k);

// k x k max pooling, NHWC; out-of-range taps never win.
hipError_t launch_maxpool(int dt, const void* x, void* y, int N, int H, int W, int C,
                          int Ho, int Wo, int k, int stride, int pad, hipStream_t s);
const char* maxpool_name(int dt);

// Mean over H x W per (n, c), fp32 sum, NHWC in -> [N][C] out.
hipError_t launch_gap(int dt, const void* x, void* y, int N, int HW, int C, hipStream_t s);
const char* gap_name(int dt);

// Deterministic pseudo-random fill in [0, 1) for profiling inputs.
hipError_t launch_fill_uniform(int dt, void* p, size_t n, uint32_t seed, hipStream_t s);

}  // namespace ppipe
