// Implicit-GEMM convolution on gfx950 matrix cores (MFMA), fp32 accumulation.
//
// One kernel family covers every dense layer of a partition: k x k
// convolutions (stride, zero padding), 1 x 1 convolutions (pointwise,
// projection, strided downsample) and fully connected layers (a 1 x 1
// convolution on a 1 x 1 map, or a valid H x W convolution when the FC input
// is a feature map).  The forward of each such layer is
//     y[m][co] = act( scale[co] * sum_k W[co][k] * X[m][k] + bias[co] + res[m][co] )
// with X the on-the-fly im2col view of the NHWC input.
//
// Mapping to CDNA4:
//  * GEMM rows are output channels (MFMA A operand = packed weights), GEMM
//    columns are output pixels (MFMA B operand = gathered activations), so
//    each lane of a 16x16 accumulator holds 4 consecutive channels of one
//    pixel: the NHWC epilogue stores 8 bytes (16-bit types) per lane.
//  * 16-bit types use v_mfma_f32_16x16x32_{f16,bf16}; fp32 uses
//    v_mfma_f32_16x16x4_f32 (full fp32 products, no reduced-precision path).
//  * Per LDS stage a block stages BM x BK weights and BN x BK activations as
//    16-byte vectors (rows padded by 16 bytes), double buffered: the next
//    stage's global loads are issued before the current stage's MFMAs.
//  * The K order (kh, kw, ci) with ci fastest makes every 16-byte vector of
//    a row one contiguous NHWC load when C is a multiple of the vector width.
//    Layers whose C is not (the 3-channel stem) use a scalar gather through
//    a (kh, kw, ci) lookup table in LDS.
//  * blockIdx.z splits K; with out_mode 1 each split writes raw fp32 sums
//    and a separate pass reduces them and applies the epilogue.
#include "kernels.h"

namespace ppipe {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <typename T> struct Mfma;
template <> struct Mfma<_Float16> {
    static __device__ __forceinline__ void step(const uint4& a, const uint4& b, floatx4& c)
    {
        c = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(halfx8, a),
                                                   __builtin_bit_cast(halfx8, b), c, 0, 0, 0);
    }
};
template <> struct Mfma<__bf16> {
    static __device__ __forceinline__ void step(const uint4& a, const uint4& b, floatx4& c)
    {
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                    __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
};
// fp32: a 16-byte vector holds 4 consecutive k; four K=4 MFMAs consume it.
// Lane group g supplies k = 4g + t to instruction t for both operands, so the
// pairing of A and B elements is the same as a plain dot product over k.
template <> struct Mfma<float> {
    static __device__ __forceinline__ void step(const uint4& a, const uint4& b, floatx4& c)
    {
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    }
};

template <typename T> __device__ __forceinline__ float to_f32(T v) { return (float)v; }

__device__ __forceinline__ float apply_act(float v, int act)
{
    if (act == ACT_RELU) return fmaxf(v, 0.0f);
    if (act == ACT_RELU6) return fminf(fmaxf(v, 0.0f), 6.0f);
    return v;
}

// Load / store 4 consecutive elements of T as one vector access.
template <typename T> struct Vec4;
template <> struct Vec4<float> {
    static __device__ __forceinline__ float4 load(const float* p) { return *(const float4*)p; }
    static __device__ __forceinline__ void store(float* p, float4 v) { *(float4*)p = v; }
};
template <typename T> struct Vec4 {   // 16-bit types
    static __device__ __forceinline__ float4 load(const T* p)
    {
        uint2 u = *(const uint2*)p;
        T e[4];
        __builtin_memcpy(e, &u, 8);
        return make_float4((float)e[0], (float)e[1], (float)e[2], (float)e[3]);
    }
    static __device__ __forceinline__ void store(T* p, float4 v)
    {
        T e[4] = {(T)v.x, (T)v.y, (T)v.z, (T)v.w};
        uint2 u;
        __builtin_memcpy(&u, e, 8);
        *(uint2*)p = u;
    }
};

template <typename T, int BM, int BN, int WM, int WN, int KV, bool GENERIC>
__global__ void __launch_bounds__(WM * WN * 64)
conv_gemm_kernel(ConvGemmArgs a)
{
    constexpr int NT = WM * WN * 64;
    constexpr int EPV = 16 / (int)sizeof(T);   // elements per 16-byte vector
    constexpr int BK = KV * EPV;               // K elements per stage
    constexpr int ROW = KV * 16 + 16;          // LDS row pitch in bytes
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 16, FN = WTN / 16;
    constexpr int A_VECS = BM * KV, B_VECS = BN * KV;
    constexpr int A_PER = (A_VECS + NT - 1) / NT;
    constexpr int B_PER = (B_VECS + NT - 1) / NT;
    constexpr int B_ELEMS = BN * BK;
    constexpr int BE_PER = (B_ELEMS + NT - 1) / NT;
    static_assert(KV % 4 == 0, "a stage holds whole 64-byte MFMA k-steps");
    static_assert(FM >= 1 && FN >= 1 && WTM % 16 == 0 && WTN % 16 == 0, "wave tile");
    static_assert(!GENERIC || NT % BK == 0, "generic gather assigns one k column per thread");

    __shared__ __attribute__((aligned(16))) unsigned char smem[2 * (BM + BN) * ROW];
    __shared__ int ktab[GENERIC ? GEMM_KTAB_MAX : 1];

    const T* __restrict__ X = (const T*)a.x;
    const T* __restrict__ Wt = (const T*)a.w;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int m0 = blockIdx.x * BN, co0 = blockIdx.y * BM;
    const int kc_begin = blockIdx.z * a.chunks_per_split;
    const int kc_end = min(a.total_chunks, kc_begin + a.chunks_per_split);
    const int HoWo = a.Ho * a.Wo;

    if constexpr (GENERIC) {
        for (int k = tid; k < a.Kpad && k < GEMM_KTAB_MAX; k += NT) {
            int t = -1;
            if (k < a.K) {
                int tap = k / a.C, ci = k - tap * a.C;
                int kh = tap / a.KW, kw = tap - kh * a.KW;
                t = kh | (kw << 8) | (ci << 16);
            }
            ktab[k] = t;
        }
        __syncthreads();
    }

    // ---- per-thread load slots (fixed for the whole K loop) ----
    int a_row[A_PER], a_kv[A_PER];
    bool a_ok[A_PER];
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
        int v = tid + i * NT;
        a_row[i] = v / KV;
        a_kv[i] = v % KV;
        a_ok[i] = v < A_VECS && co0 + a_row[i] < a.Co;
    }
    constexpr int BROWS = GENERIC ? BE_PER : B_PER;
    int b_row[BROWS], b_kv[BROWS], b_hi0[BROWS], b_wi0[BROWS];
    size_t b_base[BROWS];
    bool b_ok[BROWS];
#pragma unroll
    for (int i = 0; i < BROWS; ++i) {
        int v = tid + i * NT;
        int r, kv;
        bool inrange;
        if constexpr (GENERIC) {
            r = v / BK;
            kv = v % BK;            // here: k column within the stage
            inrange = v < B_ELEMS;
        } else {
            r = v / KV;
            kv = v % KV;
            inrange = v < B_VECS;
        }
        int m = m0 + r;
        bool ok = inrange && m < a.M;
        int mm = ok ? m : 0;
        int n = mm / HoWo, rem = mm - n * HoWo;
        int ho = rem / a.Wo, wo = rem - ho * a.Wo;
        b_row[i] = r;
        b_kv[i] = kv;
        b_hi0[i] = ho * a.stride - a.pad;
        b_wi0[i] = wo * a.stride - a.pad;
        b_base[i] = (size_t)n * a.H * a.W * a.C;
        b_ok[i] = ok;
    }

    uint4 ra[A_PER];
    uint4 rb[GENERIC ? 1 : B_PER];
    T rbe[GENERIC ? BE_PER : 1];

    auto load_stage = [&](int kc) {
        const int k0 = kc * BK;
#pragma unroll
        for (int i = 0; i < A_PER; ++i) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (a_ok[i])
                v = *(const uint4*)(Wt + (size_t)(co0 + a_row[i]) * a.Kpad + k0 + a_kv[i] * EPV);
            ra[i] = v;
        }
        if constexpr (GENERIC) {
#pragma unroll
            for (int i = 0; i < BE_PER; ++i) {
                T v = (T)0.0f;
                int k = k0 + b_kv[i];
                if (b_ok[i] && k < a.K) {
                    int t = ktab[k];
                    int hi = b_hi0[i] + (t & 0xff), wi = b_wi0[i] + ((t >> 8) & 0xff);
                    if ((unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W)
                        v = X[b_base[i] + ((size_t)hi * a.W + wi) * a.C + (t >> 16)];
                }
                rbe[i] = v;
            }
        } else {
            // the whole stage lies in one (kh, kw) tap: C % BK == 0, or a 1x1 window
            const int tap = k0 / a.C, ci0 = k0 - tap * a.C;
            const int kh = tap / a.KW, kw = tap - kh * a.KW;
#pragma unroll
            for (int i = 0; i < B_PER; ++i) {
                uint4 v = make_uint4(0, 0, 0, 0);
                int ci = ci0 + b_kv[i] * EPV;
                int hi = b_hi0[i] + kh, wi = b_wi0[i] + kw;
                if (b_ok[i] && ci < a.C && (unsigned)hi < (unsigned)a.H &&
                    (unsigned)wi < (unsigned)a.W)
                    v = *(const uint4*)(X + b_base[i] + ((size_t)hi * a.W + wi) * a.C + ci);
                rb[i] = v;
            }
        }
    };
    auto store_stage = [&](int buf) {
        unsigned char* As = smem + buf * (BM + BN) * ROW;
        unsigned char* Bs = As + BM * ROW;
#pragma unroll
        for (int i = 0; i < A_PER; ++i)
            if (tid + i * NT < A_VECS)
                *(uint4*)(As + a_row[i] * ROW + a_kv[i] * 16) = ra[i];
        if constexpr (GENERIC) {
#pragma unroll
            for (int i = 0; i < BE_PER; ++i)
                if (tid + i * NT < B_ELEMS)
                    *(T*)(Bs + b_row[i] * ROW + b_kv[i] * (int)sizeof(T)) = rbe[i];
        } else {
#pragma unroll
            for (int i = 0; i < B_PER; ++i)
                if (tid + i * NT < B_VECS)
                    *(uint4*)(Bs + b_row[i] * ROW + b_kv[i] * 16) = rb[i];
        }
    };

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
            acc[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

    if (kc_begin < kc_end) {
        load_stage(kc_begin);
        store_stage(0);
        __syncthreads();
        int buf = 0;
        for (int kc = kc_begin; kc < kc_end; ++kc) {
            const bool more = kc + 1 < kc_end;
            if (more)
                load_stage(kc + 1);
            const unsigned char* As = smem + buf * (BM + BN) * ROW;
            const unsigned char* Bs = As + BM * ROW;
#pragma unroll
            for (int ks = 0; ks < KV / 4; ++ks) {
                uint4 af[FM], bf[FN];
                const int off = ks * 64 + (lane >> 4) * 16;
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    af[i] = *(const uint4*)(As + (wm * WTM + i * 16 + (lane & 15)) * ROW + off);
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    bf[j] = *(const uint4*)(Bs + (wn * WTN + j * 16 + (lane & 15)) * ROW + off);
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j)
                        Mfma<T>::step(af[i], bf[j], acc[i][j]);
            }
            if (more)
                store_stage(buf ^ 1);
            __syncthreads();
            buf ^= 1;
        }
    }

    // ---- epilogue: lane holds channels co..co+3 of pixel m ----
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int co = co0 + wm * WTM + i * 16 + 4 * (lane >> 4);
        if (co >= a.Co)
            continue;
        float4 sc = make_float4(1.f, 1.f, 1.f, 1.f), bi = make_float4(0.f, 0.f, 0.f, 0.f);
        if (a.out_mode == 0) {
            sc = *(const float4*)(a.scale + co);
            bi = *(const float4*)(a.bias + co);
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int m = m0 + wn * WTN + j * 16 + (lane & 15);
            if (m >= a.M)
                continue;
            const floatx4 c = acc[i][j];
            if (a.out_mode == 1) {
                *(float4*)(a.partial + ((size_t)blockIdx.z * a.M + m) * a.Co + co) =
                    make_float4(c[0], c[1], c[2], c[3]);
                continue;
            }
            float4 v = make_float4(c[0] * sc.x + bi.x, c[1] * sc.y + bi.y,
                                   c[2] * sc.z + bi.z, c[3] * sc.w + bi.w);
            const size_t o = (size_t)m * a.Co + co;
            if (a.res) {
                float4 r = Vec4<T>::load((const T*)a.res + o);
                v.x += r.x; v.y += r.y; v.z += r.z; v.w += r.w;
            }
            v.x = apply_act(v.x, a.act); v.y = apply_act(v.y, a.act);
            v.z = apply_act(v.z, a.act); v.w = apply_act(v.w, a.act);
            Vec4<T>::store((T*)a.y + o, v);
        }
    }
}

// ---- split-K reduction + epilogue ----
template <typename T>
__global__ void __launch_bounds__(256)
splitk_epilogue_kernel(const float* __restrict__ partial, int splits, int M, int Co,
                       const float* __restrict__ scale, const float* __restrict__ bias,
                       const T* __restrict__ res, int act, T* __restrict__ y)
{
    const size_t nvec = (size_t)M * Co / 4;
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= nvec)
        return;
    const float4* p = (const float4*)partial;
    float4 s = p[i];
    for (int sp = 1; sp < splits; ++sp) {
        float4 t = p[(size_t)sp * nvec + i];
        s.x += t.x; s.y += t.y; s.z += t.z; s.w += t.w;
    }
    const int co = (int)((i * 4) % (size_t)Co);
    const float4 sc = *(const float4*)(scale + co);
    const float4 bi = *(const float4*)(bias + co);
    float4 v = make_float4(s.x * sc.x + bi.x, s.y * sc.y + bi.y, s.z * sc.z + bi.z,
                           s.w * sc.w + bi.w);
    if (res) {
        float4 r = Vec4<T>::load(res + i * 4);
        v.x += r.x; v.y += r.y; v.z += r.z; v.w += r.w;
    }
    v.x = apply_act(v.x, act); v.y = apply_act(v.y, act);
    v.z = apply_act(v.z, act); v.w = apply_act(v.w, act);
    Vec4<T>::store(y + i * 4, v);
}

// ---- split-K reduction + bias + softmax, one block per row ----
__device__ __forceinline__ float wave_max(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v += __shfl_xor(v, o, 64);
    return v;
}

__global__ void __launch_bounds__(256)
splitk_softmax_kernel(const float* __restrict__ partial, int splits, int M, int O,
                      const float* __restrict__ bias, float* __restrict__ out)
{
    __shared__ float z[SOFTMAX_MAX_O];
    __shared__ float red[4];
    const int m = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float mx = -INFINITY;
    for (int o = tid; o < O; o += 256) {
        float s = bias ? bias[o] : 0.0f;
        for (int sp = 0; sp < splits; ++sp)
            s += partial[((size_t)sp * M + m) * O + o];
        z[o] = s;
        mx = fmaxf(mx, s);
    }
    mx = wave_max(mx);
    if (lane == 0)
        red[wave] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    __syncthreads();
    float sum = 0.0f;
    for (int o = tid; o < O; o += 256) {
        float e = expf(z[o] - mx);
        z[o] = e;
        sum += e;
    }
    sum = wave_sum(sum);
    if (lane == 0)
        red[wave] = sum;
    __syncthreads();
    const float inv = 1.0f / (red[0] + red[1] + red[2] + red[3]);
    for (int o = tid; o < O; o += 256)
        out[(size_t)m * O + o] = z[o] * inv;
}

// ---- host-side launchers ----
GemmCfgInfo gemm_cfg_info(int cfg)
{
    switch (cfg) {
    case GEMM_128x128: return {128, 128, 256, 4};
    case GEMM_64x64:   return {64, 64, 256, 4};
    case GEMM_64x16:   return {64, 16, 256, 4};
    default:           return {0, 0, 0, 0};
    }
}

template <typename T, int BM, int BN, int WM, int WN, int KV>
static hipError_t launch_t(bool generic, const ConvGemmArgs& a, int splits, hipStream_t s)
{
    dim3 grid((a.M + BN - 1) / BN, (a.Co + BM - 1) / BM, splits);
    dim3 block(WM * WN * 64);
    if (generic)
        hipLaunchKernelGGL((conv_gemm_kernel<T, BM, BN, WM, WN, KV, true>), grid, block, 0, s, a);
    else
        hipLaunchKernelGGL((conv_gemm_kernel<T, BM, BN, WM, WN, KV, false>), grid, block, 0, s, a);
    return hipGetLastError();
}

template <typename T>
static hipError_t launch_cfg(int cfg, bool generic, const ConvGemmArgs& a, int splits,
                             hipStream_t s)
{
    switch (cfg) {
    case GEMM_128x128: return launch_t<T, 128, 128, 2, 2, 4>(generic, a, splits, s);
    case GEMM_64x64:   return launch_t<T, 64, 64, 2, 2, 4>(generic, a, splits, s);
    case GEMM_64x16:   return launch_t<T, 64, 16, 4, 1, 4>(generic, a, splits, s);
    default:           return hipErrorInvalidValue;
    }
}

hipError_t launch_conv_gemm(int dt, int cfg, bool generic, const ConvGemmArgs& a,
                            int splits, hipStream_t s)
{
    switch (dt) {
    case DT_F32:  return launch_cfg<float>(cfg, generic, a, splits, s);
    case DT_F16:  return launch_cfg<_Float16>(cfg, generic, a, splits, s);
    case DT_BF16: return launch_cfg<__bf16>(cfg, generic, a, splits, s);
    default:      return hipErrorInvalidValue;
    }
}

static const char* dt_name(int dt)
{
    return dt == DT_F32 ? "f32" : dt == DT_F16 ? "f16" : "bf16";
}

const char* conv_gemm_name(int dt, int cfg, bool generic)
{
    static char names[3][GEMM_NCFG][2][64];
    char* n = names[dt][cfg][generic ? 1 : 0];
    if (!n[0]) {
        GemmCfgInfo c = gemm_cfg_info(cfg);
        snprintf(n, 64, "conv_gemm<%s,%dx%d,kv%d%s>", dt_name(dt), c.bm, c.bn, c.kv,
                 generic ? ",gather" : "");
    }
    return n;
}

hipError_t launch_splitk_epilogue(int dt, const float* partial, int splits, int M, int Co,
                                  const float* scale, const float* bias, const void* res,
                                  int act, void* y, hipStream_t s)
{
    const size_t nvec = (size_t)M * Co / 4;
    dim3 grid((unsigned)((nvec + 255) / 256)), block(256);
    switch (dt) {
    case DT_F32:
        hipLaunchKernelGGL(splitk_epilogue_kernel<float>, grid, block, 0, s, partial, splits,
                           M, Co, scale, bias, (const float*)res, act, (float*)y);
        break;
    case DT_F16:
        hipLaunchKernelGGL(splitk_epilogue_kernel<_Float16>, grid, block, 0, s, partial,
                           splits, M, Co, scale, bias, (const _Float16*)res, act,
                           (_Float16*)y);
        break;
    case DT_BF16:
        hipLaunchKernelGGL(splitk_epilogue_kernel<__bf16>, grid, block, 0, s, partial,
                           splits, M, Co, scale, bias, (const __bf16*)res, act, (__bf16*)y);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

const char* splitk_epilogue_name(int dt)
{
    static const char* n[3] = {"splitk_epilogue<f32>", "splitk_epilogue<f16>",
                               "splitk_epilogue<bf16>"};
    return n[dt];
}

hipError_t launch_splitk_softmax(const float* partial, int splits, int M, int O,
                                 const float* bias, float* out, hipStream_t s)
{
    hipLaunchKernelGGL(splitk_softmax_kernel, dim3(M), dim3(256), 0, s, partial, splits, M,
                       O, bias, out);
    return hipGetLastError();
}

const char* splitk_softmax_name() { return "splitk_softmax<f32>"; }

}  // namespace ppipe
