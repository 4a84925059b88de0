// Streaming convolutions for thin layers: 1x1 layers with few input
// channels, and stems with a 3-channel input.
//
// Pointwise (GEMM_PW).
// A 1x1, stride-1 convolution with C <= 32 input channels reduces over one
// 32-element MFMA k-step per output (up to five with at most 32 output
// channels), so the GEMM's machinery (K loop, LDS stage ring, staged
// epilogue) is overhead: these layers (the expansion and projection
// convolutions of MobileNetV2's early blocks) are bound by streaming their
// input and output through HBM.  Here each wave keeps the
// weights of its block's output-channel slice (at most 96 channels, to keep
// registers, and so resident waves, in check) in registers as MFMA A
// fragments and walks 16-pixel groups of the NHWC input grid-stride, in a
// grid of as many blocks as stay resident:
//   * the B fragment of a group is one 16-byte load per lane straight from
//     HBM (lane l: pixel l % 16, channels 8 (l / 16) .. + 8; past C the
//     buffer range check returns zeros), issued PF groups ahead;
//   * 16 x 16 x 32 MFMAs (one per 16 output channels and k-step) give each
//     lane four consecutive output channels of one pixel;
//   * the epilogue stages the group's scaled sums (folded BN scale and shift
//     from LDS) as a [16 pixel][channel] fp32 tile in the wave's own LDS
//     rows; each lane then finishes one 8-channel vector of one pixel
//     (residual, activation, rounding) and stores 16 contiguous bytes, so a
//     wave's stores run along the pixels' channel rows (output channels a
//     multiple of 8; otherwise each lane stores its four channels as one
//     8-byte vector, 32-byte pieces of 16 rows per store).
//
// Stem (GEMM_STEM).  A k x k convolution of a C <= 4 channel image (RGB
// stems) is bound by writing its output.  The weights are packed as for the
// GEMM, one 16-byte vector per tap with the channels zero-padded, so a
// 16-byte MFMA operand vector is one tap: in k-step ks, lane group q handles
// tap 4 ks + q, gathering the C channels of the input pixel under that tap
// for its output pixel (zero outside the image) and reading the tap's weight
// vector from LDS, where the block stages its channel slice once.  The same
// row-contiguous epilogue follows; fp32 stems run on the 16x16x4 fp32 MFMA.
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
// fp32: a 16-byte vector is 4 consecutive k; instruction t takes component t
// of both operands from every lane group, which pairs them as a dot product.
template <> __device__ __forceinline__ floatx4 pw_mfma<float>(uint4 a, uint4 b, floatx4 c)
{
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
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

// The activation as one clamp (v_med3_f32): [-inf, inf], [0, inf] or [0, 6].
__device__ __forceinline__ float pw_act(float v, int act)
{
    const float lo = act == ACT_NONE ? -INFINITY : 0.0f;
    const float hi = act == ACT_RELU6 ? 6.0f : INFINITY;
    return __builtin_amdgcn_fmed3f(v, lo, hi);
}

// Epilogue of four consecutive output channels co.. (c.. within the block's
// slice) of pixel p: folded BN, residual, activation, one vector store.
template <typename T>
__device__ __forceinline__ void pw_store4(const ConvGemmArgs& a, int p, int co, int c,
                                          const floatx4& acc, const float* s_scale,
                                          const float* s_bias)
{
    const size_t off = (size_t)p * a.Co + co;
    float v[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = acc[r] * s_scale[c + r] + s_bias[c + r];
    if constexpr (sizeof(T) == 4) {
        if (a.res) {
            const float4 u = *(const float4*)((const float*)a.res + off);
            v[0] += u.x; v[1] += u.y; v[2] += u.z; v[3] += u.w;
        }
        *(float4*)((float*)a.y + off) = make_float4(pw_act(v[0], a.act), pw_act(v[1], a.act),
                                                    pw_act(v[2], a.act), pw_act(v[3], a.act));
    } else {
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

// Row-contiguous epilogue of one 16-pixel group (output channels a multiple
// of the 16-byte vector): the wave stages the scaled sums as a [16 pixel]
// [16 CF channel] fp32 tile in its own LDS rows tw (row pitch TROW floats),
// then every lane finishes one 16-byte vector of one pixel (residual,
// activation, rounding) and stores it, so consecutive lanes write along each
// pixel's channel row instead of 8- or 16-byte pieces of 16 rows.
template <int CF>
constexpr int pw_trow() { return CF * 16 + 4; }
// Pixels p0 .. p0 + nvalid - 1 (nvalid <= 16) are lane rows 0 .. nvalid - 1.
template <typename T, int CF>
__device__ __forceinline__ void pw_rows_store_at(const ConvGemmArgs& a, const floatx4 (&acc)[CF],
                                                 const float* __restrict__ s_scale,
                                                 const float* __restrict__ s_bias,
                                                 float* __restrict__ tw, int p0, int nvalid,
                                                 int co0, int lane)
{
    constexpr int VE = 16 / (int)sizeof(T);     // channels per 16-byte vector
    constexpr int NV = 16 * CF / VE;            // vectors of a pixel's slice
    constexpr int NIT = (16 * NV + 63) / 64;    // vectors per lane and group
    constexpr int TROW = pw_trow<CF>();
    const int cl = 4 * (lane >> 4);
#pragma unroll
    for (int f = 0; f < CF; ++f) {
        const int c = 16 * f + cl;
        const float4 sc = *(const float4*)(s_scale + c);   // 16-byte aligned arrays
        const float4 bi = *(const float4*)(s_bias + c);
        float4 v;
        v.x = acc[f][0] * sc.x + bi.x;
        v.y = acc[f][1] * sc.y + bi.y;
        v.z = acc[f][2] * sc.z + bi.z;
        v.w = acc[f][3] * sc.w + bi.w;
        *(float4*)(tw + (lane & 15) * TROW + c) = v;
    }
    __builtin_amdgcn_wave_barrier();   // one wave's LDS operations run in order
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        const int v = it * 64 + lane;
        const int px = v / NV, cv = v - px * NV;
        const int p = p0 + px, co = co0 + VE * cv;
        if (v < 16 * NV && px < nvalid && co < a.Co) {
            const size_t off = (size_t)p * a.Co + co;
            uint4 r = make_uint4(0u, 0u, 0u, 0u);
            if (a.res)
                r = *(const uint4*)((const T*)a.res + off);
            float o[VE];
#pragma unroll
            for (int q = 0; q < VE; q += 4) {
                const float4 t = *(const float4*)(tw + px * TROW + VE * cv + q);
                o[q] = t.x; o[q + 1] = t.y; o[q + 2] = t.z; o[q + 3] = t.w;
            }
            if (a.res) {
                T rr[VE];
                __builtin_memcpy(rr, &r, 16);
#pragma unroll
                for (int q = 0; q < VE; ++q) o[q] += (float)rr[q];
            }
            T e[VE];
#pragma unroll
            for (int q = 0; q < VE; ++q) e[q] = (T)pw_act(o[q], a.act);
            uint4 u;
            __builtin_memcpy(&u, e, 16);
            *(uint4*)((T*)a.y + off) = u;
        }
    }
    __builtin_amdgcn_wave_barrier();
}
// Group g: pixels 16 g .. 16 g + 15 (those below M).
template <typename T, int CF>
__device__ __forceinline__ void pw_rows_store(const ConvGemmArgs& a, const floatx4 (&acc)[CF],
                                              const float* __restrict__ s_scale,
                                              const float* __restrict__ s_bias,
                                              float* __restrict__ tw, int g, int co0, int lane)
{
    pw_rows_store_at<T, CF>(a, acc, s_scale, s_bias, tw, g * 16, a.M - g * 16, co0, lane);
}

// Block: PW_WAVES waves on output channels [co0, co0 + 16 CF); blockIdx.y is
// the channel slice, waves of all blocks along x share the pixel groups.
// KS: 32-element k-steps (C <= 32 KS); groups in flight ahead of the one
// computed: 3 with one k-step, 1 with more (registers).
template <typename T, int CF, int KS>
__global__ void __launch_bounds__(PW_WAVES * 64) pw_conv_kernel(ConvGemmArgs a)
{
    constexpr int PW_PF = KS == 1 ? 3 : 1;
    constexpr int ESZ = (int)sizeof(T);
    __shared__ __attribute__((aligned(16))) float s_scale[CF * 16], s_bias[CF * 16];
    // each wave's rows of the row-contiguous epilogue (pw_rows_store)
    __shared__ __attribute__((aligned(16))) float s_tile[PW_WAVES][16][pw_trow<CF>()];
    const bool rows_out = a.Co % (16 / ESZ) == 0;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int3 bg = load_args_now(a, (int)blockIdx.x, (int)gridDim.x, (int)blockIdx.y);
    const int co0 = bg.z * CF * 16;
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
    const int stride = bg.y * PW_WAVES;
    int g = bg.x * PW_WAVES + wave;
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

        if (rows_out) {
            pw_rows_store<T, CF>(a, acc, s_scale, s_bias, &s_tile[wave][0][0], g, co0, lane);
        } else {
            const int p = g * 16 + (lane & 15);
            if (p < a.M) {
#pragma unroll
                for (int f = 0; f < CF; ++f) {
                    const int c = 16 * f + cl, co = co0 + c;
                    if (co >= a.Co)
                        break;
                    pw_store4<T>(a, p, co, c, acc[f], s_scale, s_bias);
                }
            }
        }
    }
}

// Stem: block of PW_WAVES waves on output channels [co0, co0 + 16 CF), KST
// k-steps of four taps (taps past KH KW have zero weights and load nothing).
template <typename T, int CF, int KST>
__global__ void __launch_bounds__(PW_WAVES * 64) stem_conv_kernel(ConvGemmArgs a)
{
    constexpr int ESZ = (int)sizeof(T);
    constexpr int EPV = 16 / ESZ;
    constexpr int ROWS = CF * 16;
    __shared__ __attribute__((aligned(16))) float s_scale[ROWS], s_bias[ROWS];
    // weights [ks][row][4 taps x 16 bytes]: a fragment read is 1 KB contiguous
    __shared__ uint4 s_w[KST * ROWS * 4];
    // each wave's rows of the row-contiguous epilogue (pw_rows_store)
    __shared__ __attribute__((aligned(16))) float s_tile[PW_WAVES][16][pw_trow<CF>()];
    const bool rows_out = a.Co % EPV == 0;

    const int tid = threadIdx.x, lane = tid & 63;
    const int3 bg = load_args_now(a, (int)blockIdx.x, (int)gridDim.x, (int)blockIdx.y);
    const int co0 = bg.z * ROWS;
    for (int i = tid; i < ROWS; i += PW_WAVES * 64) {
        const bool in = co0 + i < a.Co;
        s_scale[i] = in ? a.scale[co0 + i] : 0.0f;
        s_bias[i] = in ? a.bias[co0 + i] : 0.0f;
    }
    const auto wsrc = pw_rsrc(a.w, (uint32_t)a.Co * a.Kpad * ESZ);
    for (int i = tid; i < KST * ROWS * 4; i += PW_WAVES * 64) {
        const int q = i & 3, r = (i >> 2) % ROWS, ks = (i >> 2) / ROWS;
        const int row = co0 + r, k = (4 * ks + q) * EPV;
        s_w[i] = pw_load16(wsrc, row < a.Co && k < a.Kpad ? (uint32_t)((row * a.Kpad + k) * ESZ)
                                                          : PW_OOB);
    }
    __syncthreads();

    const auto xsrc = pw_rsrc(a.x, (uint32_t)a.N * a.H * a.W * a.C * ESZ);
    const int taps = a.KH * a.KW, hw = a.Ho * a.Wo;
    const int groups = (a.M + 15) / 16;
    const int stride = bg.y * PW_WAVES;
    const int q = lane >> 4, cl = 4 * q;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    for (int g = bg.x * PW_WAVES + wave; g < groups; g += stride) {
        const int p = g * 16 + (lane & 15);
        const int n = p / hw, rem = p - n * hw;
        const int ho = rem / a.Wo, wo = rem - (rem / a.Wo) * a.Wo;
        const int h0 = ho * a.stride - a.pad, w0 = wo * a.stride - a.pad;
        // gather: this lane group's tap of every k-step, C channels each
        uint32_t e[KST][4];
#pragma unroll
        for (int ks = 0; ks < KST; ++ks) {
            const int t = 4 * ks + q;
            const int kh = t / a.KW, kw = t - (t / a.KW) * a.KW;
            const int hi = h0 + kh, wi = w0 + kw;
            const bool ok = p < a.M && t < taps && hi >= 0 && hi < a.H && wi >= 0 && wi < a.W;
            const uint32_t base = (uint32_t)((((n * a.H + hi) * a.W + wi) * a.C) * ESZ);
#pragma unroll
            for (int ci = 0; ci < 4; ++ci) {
                const uint32_t off = ok && ci < a.C ? base + ci * ESZ : PW_OOB;
                if constexpr (ESZ == 4)
                    e[ks][ci] = __builtin_amdgcn_raw_buffer_load_b32(xsrc, off, 0, 0);
                else
                    e[ks][ci] = __builtin_amdgcn_raw_buffer_load_b16(xsrc, off, 0, 0);
            }
        }
        floatx4 acc[CF];
#pragma unroll
        for (int f = 0; f < CF; ++f) acc[f] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ks = 0; ks < KST; ++ks) {
            uint4 b;
            if constexpr (ESZ == 4)
                b = uint4{e[ks][0], e[ks][1], e[ks][2], e[ks][3]};
            else
                b = uint4{e[ks][0] | (e[ks][1] << 16), e[ks][2] | (e[ks][3] << 16), 0u, 0u};
#pragma unroll
            for (int f = 0; f < CF; ++f)
                acc[f] = pw_mfma<T>(s_w[(ks * ROWS + 16 * f + (lane & 15)) * 4 + q], b, acc[f]);
        }
        if (rows_out) {
            pw_rows_store<T, CF>(a, acc, s_scale, s_bias, &s_tile[wave][0][0], g, co0, lane);
        } else if (p < a.M) {
#pragma unroll
            for (int f = 0; f < CF; ++f) {
                const int c = 16 * f + cl, co = co0 + c;
                if (co >= a.Co)
                    break;
                pw_store4<T>(a, p, co, c, acc[f], s_scale, s_bias);
            }
        }
    }
}

// Stem with the input window in LDS.  A block's tile is PW_WAVES output rows
// (wave w: row w) by 16 output columns of one image; the input rows and
// columns those outputs read are loaded into LDS once per tile (each pixel's
// C <= 4 channels padded to four, zeros outside the image), and every lane
// reads its taps from there instead of gathering them from global memory
// (the gather kernel above issues KH KW C two-byte loads per output pixel).
// The tap order, the weights and the MFMA sequence are the gather kernel's,
// so the sums are bit-identical to it.  Blocks walk the tiles with a
// block-uniform stride; the weights of the block's channel slice stay in LDS.
template <typename T>
constexpr int stem_patch_bytes() { return sizeof(T) == 4 ? 16 : 8; }   // one padded pixel
template <typename T>
constexpr int stem_patch_px() { return 8192 / stem_patch_bytes<T>(); }   // 8 KB window buffer

template <typename T, int CF, int KST>
__global__ void __launch_bounds__(PW_WAVES * 64) stem_patch_kernel(ConvGemmArgs a)
{
    constexpr int ESZ = (int)sizeof(T);
    constexpr int EPV = 16 / ESZ;
    constexpr int ROWS = CF * 16;
    constexpr int PB = stem_patch_bytes<T>();
    __shared__ __attribute__((aligned(16))) float s_scale[ROWS], s_bias[ROWS];
    __shared__ uint4 s_w[KST * ROWS * 4];
    __shared__ __attribute__((aligned(16))) unsigned char s_patch[stem_patch_px<T>() * PB];
    __shared__ __attribute__((aligned(16))) float s_tile[PW_WAVES][16][pw_trow<CF>()];
    const bool rows_out = a.Co % EPV == 0;

    const int tid = threadIdx.x, lane = tid & 63;
    const int3 bg = load_args_now(a, (int)blockIdx.x, (int)gridDim.x, (int)blockIdx.y);
    const int co0 = bg.z * ROWS;
    for (int i = tid; i < ROWS; i += PW_WAVES * 64) {
        const bool in = co0 + i < a.Co;
        s_scale[i] = in ? a.scale[co0 + i] : 0.0f;
        s_bias[i] = in ? a.bias[co0 + i] : 0.0f;
    }
    const auto wsrc = pw_rsrc(a.w, (uint32_t)a.Co * a.Kpad * ESZ);
    for (int i = tid; i < KST * ROWS * 4; i += PW_WAVES * 64) {
        const int q = i & 3, r = (i >> 2) % ROWS, ks = (i >> 2) / ROWS;
        const int row = co0 + r, k = (4 * ks + q) * EPV;
        s_w[i] = pw_load16(wsrc, row < a.Co && k < a.Kpad ? (uint32_t)((row * a.Kpad + k) * ESZ)
                                                          : PW_OOB);
    }

    const auto xsrc = pw_rsrc(a.x, (uint32_t)a.N * a.H * a.W * a.C * ESZ);
    const int taps = a.KH * a.KW;
    const int PR = (PW_WAVES - 1) * a.stride + a.KH;     // window rows and columns
    const int PC = 15 * a.stride + a.KW;
    const int TY = (a.Ho + PW_WAVES - 1) / PW_WAVES, TX = (a.Wo + 15) / 16;
    const int tiles = a.N * TY * TX;
    const int q = lane >> 4, px = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // this lane's window offset (in pixels) of each k-step's tap, or -1 past the taps
    int toff[KST];
#pragma unroll
    for (int ks = 0; ks < KST; ++ks) {
        const int t = 4 * ks + q;
        const int kh = t / a.KW, kw = t - (t / a.KW) * a.KW;
        toff[ks] = t < taps ? (wave * a.stride + kh) * PC + px * a.stride + kw : -1;
    }
    // The window of the block's next tile is loaded into registers while the
    // current tile is computed (NPT window pixels per thread at most).
    constexpr int NPT = stem_patch_px<T>() / (PW_WAVES * 64);
    uint32_t e[NPT][4];
    auto load_window = [&](int tile) {
        const int n = tile / (TY * TX), r = tile - n * (TY * TX);
        const int iy0 = (r / TX) * PW_WAVES * a.stride - a.pad;
        const int ix0 = (r - (r / TX) * TX) * 16 * a.stride - a.pad;
#pragma unroll
        for (int j = 0; j < NPT; ++j) {
            const int i = tid + j * PW_WAVES * 64;
            const int py = i / PC, pc = i - (i / PC) * PC;
            const int hi = iy0 + py, wi = ix0 + pc;
            const bool ok = tile < tiles && i < PR * PC && hi >= 0 && hi < a.H && wi >= 0 &&
                            wi < a.W;
            const uint32_t base = (uint32_t)((((n * a.H + hi) * a.W + wi) * a.C) * ESZ);
#pragma unroll
            for (int ci = 0; ci < 4; ++ci) {
                const uint32_t off = ok && ci < a.C ? base + ci * ESZ : PW_OOB;
                if constexpr (ESZ == 4)
                    e[j][ci] = __builtin_amdgcn_raw_buffer_load_b32(xsrc, off, 0, 0);
                else
                    e[j][ci] = __builtin_amdgcn_raw_buffer_load_b16(xsrc, off, 0, 0);
            }
        }
    };
    load_window(bg.x);
    for (int tile = bg.x; tile < tiles; tile += bg.y) {   // the same trip count in every wave
        const int n = tile / (TY * TX), r = tile - n * (TY * TX);
        const int oy0 = (r / TX) * PW_WAVES, ox0 = (r - (r / TX) * TX) * 16;
        __syncthreads();   // the previous tile's window reads are done (and the weights stored)
#pragma unroll
        for (int j = 0; j < NPT; ++j) {
            const int i = tid + j * PW_WAVES * 64;
            if (i < PR * PC) {
                if constexpr (ESZ == 4)
                    *(uint4*)(s_patch + i * PB) = uint4{e[j][0], e[j][1], e[j][2], e[j][3]};
                else
                    *(uint2*)(s_patch + i * PB) =
                        uint2{e[j][0] | (e[j][1] << 16), e[j][2] | (e[j][3] << 16)};
            }
        }
        load_window(tile + bg.y);
        __syncthreads();
        const int oy = oy0 + wave;
        if (oy < a.Ho) {
            uint4 b[KST];
#pragma unroll
            for (int ks = 0; ks < KST; ++ks) {
                if constexpr (ESZ == 4) {
                    b[ks] = toff[ks] >= 0 ? *(const uint4*)(s_patch + toff[ks] * PB)
                                          : uint4{0u, 0u, 0u, 0u};
                } else {
                    const uint2 v = toff[ks] >= 0 ? *(const uint2*)(s_patch + toff[ks] * PB)
                                                  : uint2{0u, 0u};
                    b[ks] = uint4{v.x, v.y, 0u, 0u};
                }
            }
            floatx4 acc[CF];
#pragma unroll
            for (int f = 0; f < CF; ++f) acc[f] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int ks = 0; ks < KST; ++ks)
#pragma unroll
                for (int f = 0; f < CF; ++f)
                    acc[f] = pw_mfma<T>(s_w[(ks * ROWS + 16 * f + px) * 4 + q], b[ks], acc[f]);
            const int p0 = (n * a.Ho + oy) * a.Wo + ox0;
            const int nvalid = min(16, a.Wo - ox0);
            if (rows_out) {
                pw_rows_store_at<T, CF>(a, acc, s_scale, s_bias, &s_tile[wave][0][0], p0, nvalid,
                                        co0, lane);
            } else if (px < nvalid) {
#pragma unroll
                for (int f = 0; f < CF; ++f) {
                    const int c = 16 * f + 4 * q, co = co0 + c;
                    if (co >= a.Co)
                        break;
                    pw_store4<T>(a, p0 + px, co, c, acc[f], s_scale, s_bias);
                }
            }
        }
    }
}

template <typename T, int CF, int KS>
hipError_t launch_pw_t(const ConvGemmArgs& a, int grid_blocks, hipStream_t s)
{
    // one resident set of blocks (the kernel's occupancy on every CU, split
    // over the channel slices); each wave then walks its share of the groups
    // with loads in flight ahead
    static int resident = 0;
    if (!resident) {
        int n = 0;
        const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, pw_conv_kernel<T, CF, KS>, PW_WAVES * 64, 0);
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
    PPIPE_LAUNCH((pw_conv_kernel<T, CF, KS>), grid, block, 0, s, a);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_pw_dt(int cf, const ConvGemmArgs& a, int grid_blocks, hipStream_t s)
{
    const int ks = (a.C + 31) / 32;
    if (ks == 1) {
        switch (cf) {
        case 1:  return launch_pw_t<T, 1, 1>(a, grid_blocks, s);
        case 2:  return launch_pw_t<T, 2, 1>(a, grid_blocks, s);
        case 4:  return launch_pw_t<T, 4, 1>(a, grid_blocks, s);
        case 6:  return launch_pw_t<T, 6, 1>(a, grid_blocks, s);
        default: return hipErrorInvalidValue;
        }
    }
    // more k-steps: at most 32 output channels per block
#define PPIPE_PW_KS(CF_)                                                                         \
    switch (ks) {                                                                                \
    case 2:  return launch_pw_t<T, CF_, 2>(a, grid_blocks, s);                                   \
    case 3:  return launch_pw_t<T, CF_, 3>(a, grid_blocks, s);                                   \
    case 4:  return launch_pw_t<T, CF_, 4>(a, grid_blocks, s);                                   \
    case 5:  return launch_pw_t<T, CF_, 5>(a, grid_blocks, s);                                   \
    default: return hipErrorInvalidValue;                                                        \
    }
    if (cf == 1) { PPIPE_PW_KS(1) }
    if (cf == 2) { PPIPE_PW_KS(2) }
#undef PPIPE_PW_KS
    return hipErrorInvalidValue;
}

template <typename T, int CF, int KST>
hipError_t launch_stem_t(const ConvGemmArgs& a, int grid_blocks, hipStream_t s)
{
    static int resident = 0;
    if (!resident) {
        int n = 0;
        const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, stem_conv_kernel<T, CF, KST>, PW_WAVES * 64, 0);
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
    PPIPE_LAUNCH((stem_conv_kernel<T, CF, KST>), grid, block, 0, s, a);
    return hipGetLastError();
}

template <typename T, int CF, int KST>
hipError_t launch_stem_patch_t(const ConvGemmArgs& a, int grid_blocks, hipStream_t s)
{
    static int resident = 0;
    if (!resident) {
        int n = 0;
        const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, stem_patch_kernel<T, CF, KST>, PW_WAVES * 64, 0);
        if (e != hipSuccess)
            return e;
        resident = std::max(1, n);
    }
    const int tiles = a.N * ((a.Ho + PW_WAVES - 1) / PW_WAVES) * ((a.Wo + 15) / 16);
    const int slices = (a.Co + CF * 16 - 1) / (CF * 16);
    const int cap = grid_blocks > 0 ? grid_blocks
                                    : std::max(NUM_CUS_PW * resident / slices, NUM_CUS_PW);
    const dim3 grid((unsigned)std::min(tiles, cap), (unsigned)slices), block(PW_WAVES * 64);
    PPIPE_LAUNCH((stem_patch_kernel<T, CF, KST>), grid, block, 0, s, a);
    return hipGetLastError();
}

// Filters of more than 12 taps take the window kernel when one tile's input
// window fits its LDS buffer (ResNet-152's 7x7 stem at batch 64: the whole
// model 0.7% faster); 3x3 stems keep the gather kernel, which was ahead on
// them (VGG-16 0.6%, MobileNetV2 1.3%).
template <typename T, int CF>
hipError_t launch_stem_cf(const ConvGemmArgs& a, int grid_blocks, hipStream_t s)
{
    const int kst = (a.KH * a.KW + 3) / 4;
    const int window = ((PW_WAVES - 1) * a.stride + a.KH) * (15 * a.stride + a.KW);
    if (kst > 3 && window <= stem_patch_px<T>()) {
        if (kst <= 7) return launch_stem_patch_t<T, CF, 7>(a, grid_blocks, s);
        if (kst <= 13) return launch_stem_patch_t<T, CF, 13>(a, grid_blocks, s);
        return hipErrorInvalidValue;
    }
    if (kst <= 3) return launch_stem_t<T, CF, 3>(a, grid_blocks, s);
    if (kst <= 7) return launch_stem_t<T, CF, 7>(a, grid_blocks, s);
    if (kst <= 13) return launch_stem_t<T, CF, 13>(a, grid_blocks, s);
    return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_stem_dt(int cf, const ConvGemmArgs& a, int grid_blocks, hipStream_t s)
{
    switch (cf) {
    case 1:  return launch_stem_cf<T, 1>(a, grid_blocks, s);
    case 2:  return launch_stem_cf<T, 2>(a, grid_blocks, s);
    case 4:  return launch_stem_cf<T, 4>(a, grid_blocks, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

int stem_channel_frags(int Co)
{
    // slices of at most 64 output channels, split evenly
    const int slices = (Co + 63) / 64;
    const int need = (Co + 16 * slices - 1) / (16 * slices);
    return need <= 1 ? 1 : need <= 2 ? 2 : 4;
}

hipError_t launch_stem(int dt, int cf, const ConvGemmArgs& a, int grid_blocks, hipStream_t s)
{
    if (a.C > 4 || a.C >= 16 / dtype_size(dt) || a.Co % 4 != 0 || a.KH * a.KW > 52 ||
        a.softmax || a.splits != 1)
        return hipErrorInvalidValue;
    switch (dt) {
    case DT_F32:  return launch_stem_dt<float>(cf, a, grid_blocks, s);
    case DT_F16:  return launch_stem_dt<_Float16>(cf, a, grid_blocks, s);
    case DT_BF16: return launch_stem_dt<__bf16>(cf, a, grid_blocks, s);
    default:      return hipErrorInvalidValue;
    }
}

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
    if (a.C > (cf <= 2 ? 160 : 32) || a.C % 8 != 0 || a.Co % 4 != 0 || a.KH != 1 || a.KW != 1 || a.stride != 1 ||
        a.pad != 0 || a.softmax || a.splits != 1)
        return hipErrorInvalidValue;
    switch (dt) {
    case DT_F16:  return launch_pw_dt<_Float16>(cf, a, grid_blocks, s);
    case DT_BF16: return launch_pw_dt<__bf16>(cf, a, grid_blocks, s);
    default:      return hipErrorInvalidValue;
    }
}

}  // namespace ppipe
