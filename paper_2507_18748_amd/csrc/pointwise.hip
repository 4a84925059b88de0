// Streaming 1x1 convolution for layers with few input channels.
//
// A 1x1, stride-1 convolution with C <= 32 input channels reduces over one
// 32-element MFMA k-step per output, so the GEMM's machinery (K loop, LDS
// stage ring, staged epilogue) is overhead: these layers (the expansion and
// projection convolutions of MobileNetV2's early blocks) are bound by
// streaming their input and output through HBM.  Here each wave keeps the
// weights of its block's output-channel slice (at most 96 channels, to keep
// registers, and so resident waves, in check) in registers as MFMA A
// fragments and walks 16-pixel groups of the NHWC input grid-stride, in a
// grid of as many blocks as stay resident:
//   * the B fragment of a group is one 16-byte load per lane straight from
//     HBM (lane l: pixel l % 16, channels 8 (l / 16) .. + 8; past C the
//     buffer range check returns zeros), issued PF groups ahead;
//   * 16 x 16 x 32 MFMAs (one per 16 output channels and k-step) give each
//     lane four consecutive output channels of one pixel;
//   * the epilogue (folded BN scale and shift from LDS, residual, activation,
//     rounding) stores those four channels as one 8-byte vector, so a wave's
//     store covers 32 contiguous bytes of each of its 16 pixel rows.
#include "kernels.h"

#include <algorithm>

namespace ppipe {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int NUM_CUS_PW = 256;            // MI355X compute units
constexpr uint32_t PW_OOB = 0x80000000u;   // beyond any buffer: the load returns zeros
constexpr int PW_WAVES = 4;
constexpr int PW_PF = 3;                   // groups in flight ahead of the one computed

template <typename T> __device__ __forceinline__ floatx4 pw_mfma(uint4 a, uint4 b, floatx4 c);
template <> __device__ __forceinline__ floatx4 pw_mfma<_Float16>(uint4 a, uint4 b, floatx4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(halfx8, a),
                                                  __builtin_bit_cast(halfx8, b), c, 0, 0, 0);
}
template <> __device__ __forceinline__ floatx4 pw_mfma<__bf16>(uint4 a, uint4 b, floatx4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t pw_rsrc(const void* p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                             0x00020000);
}
__device__ __forceinline__ uint4 pw_load16(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

__device__ __forceinline__ float pw_act(float v, int act)
{
    if (act == ACT_RELU) return fmaxf(v, 0.0f);
    if (act == ACT_RELU6) return fminf(fmaxf(v, 0.0f), 6.0f);
    return v;
}

// Block: PW_WAVES waves on output channels [co0, co0 + 16 CF); blockIdx.y is
// the channel slice, waves of all blocks along x share the pixel groups.
// KS: 32-element k-steps (C <= 32 KS).
template <typename T, int CF, int KS>
__global__ void __launch_bounds__(PW_WAVES * 64) pw_conv_kernel(ConvGemmArgs a)
{
    constexpr int ESZ = (int)sizeof(T);
    __shared__ float s_scale[CF * 16], s_bias[CF * 16];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int co0 = blockIdx.y * CF * 16;
    for (int i = tid; i < CF * 16; i += PW_WAVES * 64) {
        const bool in = co0 + i < a.Co;
        s_scale[i] = in ? a.scale[co0 + i] : 0.0f;
        s_bias[i] = in ? a.bias[co0 + i] : 0.0f;
    }

    // weights [Co][Kpad]: fragment f, k-step ks of lane l is row co0 + 16 f + l % 16,
    // elements 32 ks + 8 (l / 16) .. + 8
    const auto wsrc = pw_rsrc(a.w, (uint32_t)a.Co * a.Kpad * ESZ);
    uint4 af[CF][KS];
#pragma unroll
    for (int f = 0; f < CF; ++f)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int row = co0 + 16 * f + (lane & 15);
            const int k = 32 * ks + 8 * (lane >> 4);
            af[f][ks] = pw_load16(wsrc, row < a.Co ? (uint32_t)((row * a.Kpad + k) * ESZ) : PW_OOB);
        }

    // input [M][C]: lane l reads pixel 16 g + l % 16, channels 32 ks + 8 (l / 16) .. + 8
    const auto xsrc = pw_rsrc(a.x, (uint32_t)a.M * a.C * ESZ);
    const int groups = (a.M + 15) / 16;
    const int stride = gridDim.x * PW_WAVES;
    int g = blockIdx.x * PW_WAVES + wave;
    auto bload = [&](int gg, uint4 (&b)[KS]) {
        const int p = gg * 16 + (lane & 15);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int c = 32 * ks + 8 * (lane >> 4);
            b[ks] = pw_load16(xsrc, gg < groups && p < a.M && c < a.C
                                        ? (uint32_t)((p * a.C + c) * ESZ)
                                        : PW_OOB);
        }
    };
    uint4 bq[PW_PF + 1][KS];
#pragma unroll
    for (int d = 0; d < PW_PF; ++d) bload(g + d * stride, bq[d]);
    __syncthreads();   // scale and shift in LDS

    const int cl = 4 * (lane >> 4);   // first of this lane's four channels in a fragment
    for (; g < groups; g += stride) {
        bload(g + PW_PF * stride, bq[PW_PF]);
        floatx4 acc[CF];
#pragma unroll
        for (int f = 0; f < CF; ++f) {
            acc[f] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) acc[f] = pw_mfma<T>(af[f][ks], bq[0][ks], acc[f]);
        }
#pragma unroll
        for (int d = 0; d < PW_PF; ++d)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) bq[d][ks] = bq[d + 1][ks];

        const int p = g * 16 + (lane & 15);
        if (p < a.M) {
#pragma unroll
            for (int f = 0; f < CF; ++f) {
                const int c = 16 * f + cl, co = co0 + c;
                if (co >= a.Co)
                    break;
                const size_t off = (size_t)p * a.Co + co;
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = acc[f][r] * s_scale[c + r] + s_bias[c + r];
                if (a.res) {
                    const uint2 u = *(const uint2*)((const T*)a.res + off);
                    T rr[4];
                    __builtin_memcpy(rr, &u, 8);
#pragma unroll
                    for (int r = 0; r < 4; ++r) v[r] += (float)rr[r];
                }
                T e[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) e[r] = (T)pw_act(v[r], a.act);
                uint2 u;
                __builtin_memcpy(&u, e, 8);
                *(uint2*)((T*)a.y + off) = u;
            }
        }
    }
}

template <typename T, int CF>
hipError_t launch_pw_t(const ConvGemmArgs& a, int grid_blocks, hipStream_t s)
{
    // one resident set of blocks (the kernel's occupancy on every CU, split
    // over the channel slices); each wave then walks its share of the groups
    // with loads in flight ahead
    static int resident = 0;
    if (!resident) {
        int n = 0;
        const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, pw_conv_kernel<T, CF, 1>, PW_WAVES * 64, 0);
        if (e != hipSuccess)
            return e;
        resident = std::max(1, n);
    }
    const int groups = (a.M + 15) / 16;
    const int slices = (a.Co + CF * 16 - 1) / (CF * 16);
    const int cap = grid_blocks > 0 ? grid_blocks
                                    : std::max(NUM_CUS_PW * resident / slices, NUM_CUS_PW);
    const int gx = std::min((groups + PW_WAVES - 1) / PW_WAVES, cap);
    const dim3 grid((unsigned)gx, (unsigned)slices), block(PW_WAVES * 64);
    PPIPE_LAUNCH((pw_conv_kernel<T, CF, 1>), grid, block, 0, s, a);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_pw_dt(int cf, const ConvGemmArgs& a, int grid_blocks, hipStream_t s)
{
    switch (cf) {
    case 1:  return launch_pw_t<T, 1>(a, grid_blocks, s);
    case 2:  return launch_pw_t<T, 2>(a, grid_blocks, s);
    case 4:  return launch_pw_t<T, 4>(a, grid_blocks, s);
    case 6:  return launch_pw_t<T, 6>(a, grid_blocks, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

int pointwise_channel_frags(int Co)
{
    // output channels per block in 16-channel fragments: slices of at most
    // 96 channels, split evenly, rounded up to a compiled fragment count
    const int slices = (Co + 95) / 96;
    const int need = (Co + 16 * slices - 1) / (16 * slices);
    for (int cf : {1, 2, 4, 6})
        if (cf >= need) return cf;
    return 6;
}

hipError_t launch_pointwise(int dt, int cf, const ConvGemmArgs& a, int grid_blocks, hipStream_t s)
{
    if (a.C > 32 || a.C % 8 != 0 || a.Co % 4 != 0 || a.KH != 1 || a.KW != 1 || a.stride != 1 ||
        a.pad != 0 || a.softmax || a.splits != 1)
        return hipErrorInvalidValue;
    switch (dt) {
    case DT_F16:  return launch_pw_dt<_Float16>(cf, a, grid_blocks, s);
    case DT_BF16: return launch_pw_dt<__bf16>(cf, a, grid_blocks, s);
    default:      return hipErrorInvalidValue;
    }
}

}  // namespace ppipe
