// Memory-bound layers on NHWC activations: depthwise convolution, max pooling
// and global average pooling.
//
// Each thread owns one 16-byte channel vector (8 x 16-bit or 4 x fp32) of one
// output pixel, so consecutive lanes read and write consecutive 16-byte
// chunks of the channel dimension (fully coalesced global_load_dwordx4 /
// global_store_dwordx4).  Arithmetic is fp32; results are rounded once to
// the storage type.  Window taps that repeat across neighbouring pixels are
// served by L1/L2; HBM sees each input byte about once.
#include "kernels.h"

#include <cstdlib>
#include <type_traits>

namespace ppipe {

template <typename T> struct Vec16 {  // 16-bit element types: 8 per vector
    static constexpr int N = 8;
    static __device__ __forceinline__ void load(const T* p, float* f)
    {
        uint4 u = *(const uint4*)p;
        T e[8];
        __builtin_memcpy(e, &u, 16);
#pragma unroll
        for (int i = 0; i < 8; ++i) f[i] = (float)e[i];
    }
    static __device__ __forceinline__ void store(T* p, const float* f)
    {
        T e[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) e[i] = (T)f[i];
        uint4 u;
        __builtin_memcpy(&u, e, 16);
        *(uint4*)p = u;
    }
};
template <> struct Vec16<float> {
    static constexpr int N = 4;
    static __device__ __forceinline__ void load(const float* p, float* f)
    {
        float4 v = *(const float4*)p;
        f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w;
    }
    static __device__ __forceinline__ void store(float* p, const float* f)
    {
        *(float4*)p = make_float4(f[0], f[1], f[2], f[3]);
    }
};

__device__ __forceinline__ float act_f(float v, int act)
{
    if (act == ACT_RELU) return fmaxf(v, 0.0f);
    if (act == ACT_RELU6) return fminf(fmaxf(v, 0.0f), 6.0f);
    return v;
}

// y[n][ho][wo][c] = act(scale[c] * sum_{kh,kw} x[n][ho*s-p+kh][wo*s-p+kw][c] * w[kh][kw][c] + bias[c])
//
// 3x3 depthwise, stride S: each thread owns one 16-byte channel vector of PW
// consecutive output pixels of one row, so an input column is loaded once for
// every output that uses it and the nine weight vectors once per PW outputs.
// 16-bit types multiply packed: one v_dot2 per output element and tap takes
// the activation word as loaded (two channels) and a weight word with the
// other channel's half zeroed, so activations are never unpacked.
// All loads are buffer loads issued without branches: taps outside the image
// use an offset beyond the buffer and read zeros.  Consecutive lanes take
// consecutive channel vectors (coalesced 16-byte accesses).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t dw_rsrc(const void* p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                             0x00020000);
}
__device__ __forceinline__ uint4 dw_load(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
// Block index with the grid spread over the 8 XCDs in contiguous ranges (the
// hardware deals block b to XCD b % 8): neighbouring output rows, whose input
// windows overlap, run on one XCD and share its L2 instead of each XCD
// fetching the overlapping rows again.
__device__ __forceinline__ uint32_t xcd_block(uint32_t b, uint32_t G)
{
    constexpr uint32_t XCDS = 8;
    const uint32_t xcd = b % XCDS, slot = b / XCDS, per = G / XCDS, rem = G % XCDS;
    return xcd * per + (xcd < rem ? xcd : rem) + slot;
}

// Every kernel argument into scalar registers in one batch of loads (a
// kernel-argument read costs ~0.25 us; left to itself the compiler issues
// them in dependent batches), with the block index and grid size passed
// through so that no argument-dependent work is scheduled before it.
#define PPIPE_ARGS_NOW(B, G, ...) asm volatile("" : "+s"(B), "+s"(G) : __VA_ARGS__)

template <typename T>
__device__ __forceinline__ void unpack16(const uint4& u, float* f)
{
    if constexpr (sizeof(T) == 4) {
        f[0] = __uint_as_float(u.x); f[1] = __uint_as_float(u.y);
        f[2] = __uint_as_float(u.z); f[3] = __uint_as_float(u.w);
    } else {
        T e[8];
        __builtin_memcpy(e, &u, 16);
#pragma unroll
        for (int i = 0; i < 8; ++i) f[i] = (float)e[i];
    }
}

// acc + the product of the low (HI = false) or high 16-bit element of two
// packed pairs, with the other element's weight zero: one v_dot2 instruction
// in place of an unpack and an FMA.  The product of two 16-bit values is
// exact in fp32 and the zero term adds nothing, so this rounds once, as an
// FMA does.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
template <typename T>
__device__ __forceinline__ float dot2_acc(uint32_t x, uint32_t w, float acc)
{
    if constexpr (std::is_same<T, __bf16>::value)
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, x),
                                               __builtin_bit_cast(bf16x2_t, w), acc, false);
    else
        return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2_t, x),
                                      __builtin_bit_cast(f16x2_t, w), acc, false);
}

template <typename T, int S, int PW>
__global__ void __launch_bounds__(256)
dwconv3_kernel(const T* __restrict__ x, const T* __restrict__ w, const float* __restrict__ scale,
               const float* __restrict__ bias, T* __restrict__ y, int N, int H, int W, int C,
               int Ho, int Wo, int pad, int act)
{
    constexpr int V = Vec16<T>::N;
    constexpr int ESZ = (int)sizeof(T);
    constexpr int NCOL = (PW - 1) * S + 3;     // input columns one row of PW outputs reads
    constexpr uint32_t OOB = 0x80000000u;
    const int CV = C / V;
    uint32_t bid = blockIdx.x, grid = gridDim.x;
    PPIPE_ARGS_NOW(bid, grid, "s"(x), "s"(w), "s"(scale), "s"(bias), "s"(y), "s"(N), "s"(H),
                   "s"(W), "s"(C), "s"(Ho), "s"(Wo), "s"(pad), "s"(act));
    const int WQ = (Wo + PW - 1) / PW;
    const uint32_t total = (uint32_t)N * Ho * WQ * CV;
    const uint32_t idx = xcd_block(bid, grid) * 256u + threadIdx.x;
    if (idx >= total)
        return;
    const int cv = (int)(idx % CV);
    uint32_t t = idx / CV;
    const int wq = (int)(t % WQ);
    t /= WQ;
    const int ho = (int)(t % Ho);
    const int n = (int)(t / Ho);
    const int c = cv * V, wo0 = wq * PW;
    const auto xr = dw_rsrc(x, (uint32_t)N * H * W * C * ESZ);
    const auto wr = dw_rsrc(w, 9u * C * ESZ);

    uint4 wk[9];
#pragma unroll
    for (int q = 0; q < 9; ++q)
        wk[q] = dw_load(wr, (uint32_t)(q * C + c) * ESZ);

    float acc[PW][V];
#pragma unroll
    for (int p = 0; p < PW; ++p)
#pragma unroll
        for (int i = 0; i < V; ++i) acc[p][i] = 0.0f;

    const int wi0 = wo0 * S - pad;
    // byte offset of tap (kh, j) = base + kh * rstride + j * cstride (32-bit
    // wrap-around arithmetic; taps outside the image take OOB instead)
    const uint32_t cstride = (uint32_t)C * ESZ, rstride = (uint32_t)W * cstride;
    const uint32_t base = (uint32_t)((n * H + ho * S - pad) * W + wi0) * cstride + (uint32_t)c * ESZ;
    uint32_t colok = 0;   // bit j: input column wi0 + j inside the image
#pragma unroll
    for (int j = 0; j < NCOL; ++j)
        colok |= ((unsigned)(wi0 + j) < (unsigned)W ? 1u : 0u) << j;
#pragma unroll
    for (int kh = 0; kh < 3; ++kh) {
        const int hi = ho * S - pad + kh;
        const bool hok = (unsigned)hi < (unsigned)H;
        const uint32_t row = base + (uint32_t)kh * rstride;
        uint4 xc[NCOL];
#pragma unroll
        for (int j = 0; j < NCOL; ++j) {
            const bool ok = hok && ((colok >> j) & 1u);
            xc[j] = dw_load(xr, ok ? row + (uint32_t)j * cstride : OOB);
        }
#pragma unroll
        for (int kw = 0; kw < 3; ++kw) {
            if constexpr (sizeof(T) == 2) {
                // word k of a vector holds channels 2k (low half) and 2k + 1
                const uint4 wv = wk[kh * 3 + kw];
                const uint32_t ww[4] = {wv.x, wv.y, wv.z, wv.w};
                uint32_t wlo[4], whi[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    wlo[k] = ww[k] & 0x0000ffffu;
                    whi[k] = ww[k] & 0xffff0000u;
                }
#pragma unroll
                for (int p = 0; p < PW; ++p) {
                    const uint4 xv = xc[p * S + kw];
                    const uint32_t xw[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        acc[p][2 * k] = dot2_acc<T>(xw[k], wlo[k], acc[p][2 * k]);
                        acc[p][2 * k + 1] = dot2_acc<T>(xw[k], whi[k], acc[p][2 * k + 1]);
                    }
                }
            } else {
                float wf[V];
                unpack16<T>(wk[kh * 3 + kw], wf);
#pragma unroll
                for (int p = 0; p < PW; ++p) {
                    float xf[V];
                    unpack16<T>(xc[p * S + kw], xf);
#pragma unroll
                    for (int i = 0; i < V; ++i) acc[p][i] = fmaf(xf[i], wf[i], acc[p][i]);
                }
            }
        }
    }
    float sc[V], bi[V];
#pragma unroll
    for (int i = 0; i < V; ++i) {
        sc[i] = scale[c + i];
        bi[i] = bias[c + i];
    }
    // the activation as one clamp: [-inf, inf], [0, inf] or [0, 6]
    const float lo = act == ACT_NONE ? -INFINITY : 0.0f;
    const float hi6 = act == ACT_RELU6 ? 6.0f : INFINITY;
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        if (wo0 + p >= Wo)
            break;
        float o[V];
#pragma unroll
        for (int i = 0; i < V; ++i)
            o[i] = __builtin_amdgcn_fmed3f(fmaf(acc[p][i], sc[i], bi[i]), lo, hi6);
        Vec16<T>::store(y + ((size_t)(n * Ho + ho) * Wo + wo0 + p) * C + c, o);
    }
}

template <typename T>
__global__ void __launch_bounds__(256)
maxpool_kernel(const T* __restrict__ x, T* __restrict__ y, int N, int H, int W, int C, int Ho,
               int Wo, int k, int stride, int pad)
{
    constexpr int V = Vec16<T>::N;
    const int CV = C / V;
    uint32_t bid = blockIdx.x, grid = gridDim.x;
    PPIPE_ARGS_NOW(bid, grid, "s"(x), "s"(y), "s"(N), "s"(H), "s"(W), "s"(C), "s"(Ho), "s"(Wo),
                   "s"(k), "s"(stride), "s"(pad));
    const size_t total = (size_t)N * Ho * Wo * CV;
    const size_t idx = (size_t)xcd_block(bid, grid) * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const int cv = (int)(idx % CV);
    size_t p = idx / CV;
    const int wo = (int)(p % Wo);
    p /= Wo;
    const int ho = (int)(p % Ho);
    const int n = (int)(p / Ho);
    const int c = cv * V;
    float m[V];
#pragma unroll
    for (int i = 0; i < V; ++i) m[i] = -INFINITY;
    for (int kh = 0; kh < k; ++kh) {
        const int hi = ho * stride - pad + kh;
        if ((unsigned)hi >= (unsigned)H)
            continue;
        for (int kw = 0; kw < k; ++kw) {
            const int wi = wo * stride - pad + kw;
            if ((unsigned)wi >= (unsigned)W)
                continue;
            float v[V];
            Vec16<T>::load(x + (((size_t)n * H + hi) * W + wi) * C + c, v);
#pragma unroll
            for (int i = 0; i < V; ++i) m[i] = fmaxf(m[i], v[i]);
        }
    }
    Vec16<T>::store(y + (((size_t)n * Ho + ho) * Wo + wo) * C + c, m);
}

// Max pooling with a fixed K x K window and stride S: the K*K tap loads are
// buffer loads issued together, without branches (taps outside the image
// load at an offset past the buffer and are then replaced by -inf), so a
// thread's loads are in flight at once instead of one loop trip at a time.
template <typename T, int K, int S>
__global__ void __launch_bounds__(256)
maxpool_fixed_kernel(const T* __restrict__ x, T* __restrict__ y, int N, int H, int W, int C,
                     int Ho, int Wo, int pad)
{
    constexpr int V = Vec16<T>::N;
    constexpr int ESZ = (int)sizeof(T);
    constexpr uint32_t OOB = 0x80000000u;
    const int CV = C / V;
    uint32_t bid = blockIdx.x, grid = gridDim.x;
    PPIPE_ARGS_NOW(bid, grid, "s"(x), "s"(y), "s"(N), "s"(H), "s"(W), "s"(C), "s"(Ho), "s"(Wo),
                   "s"(pad));
    const uint32_t total = (uint32_t)N * Ho * Wo * CV;
    const uint32_t idx = xcd_block(bid, grid) * 256u + threadIdx.x;
    if (idx >= total)
        return;
    const int cv = (int)(idx % CV);
    uint32_t t = idx / CV;
    const int wo = (int)(t % Wo);
    t /= Wo;
    const int ho = (int)(t % Ho);
    const int n = (int)(t / Ho);
    const int c = cv * V;
    const auto xr = dw_rsrc(x, (uint32_t)N * H * W * C * ESZ);
    const uint32_t cstride = (uint32_t)C * ESZ, rstride = (uint32_t)W * cstride;
    const int hi0 = ho * S - pad, wi0 = wo * S - pad;
    const uint32_t base = (uint32_t)((n * H + hi0) * W + wi0) * cstride + (uint32_t)c * ESZ;
    uint4 v[K * K];
    uint32_t okm = 0;   // bit kh * K + kw: the tap is inside the image
#pragma unroll
    for (int kh = 0; kh < K; ++kh)
#pragma unroll
        for (int kw = 0; kw < K; ++kw) {
            const bool ok = (unsigned)(hi0 + kh) < (unsigned)H && (unsigned)(wi0 + kw) < (unsigned)W;
            okm |= (ok ? 1u : 0u) << (kh * K + kw);
            v[kh * K + kw] = dw_load(xr, ok ? base + (uint32_t)kh * rstride + (uint32_t)kw * cstride
                                            : OOB);
        }
    float m[V];
#pragma unroll
    for (int i = 0; i < V; ++i) m[i] = -INFINITY;
#pragma unroll
    for (int q = 0; q < K * K; ++q) {
        float f[V];
        unpack16<T>(v[q], f);
        const bool ok = (okm >> q) & 1u;
#pragma unroll
        for (int i = 0; i < V; ++i) m[i] = fmaxf(m[i], ok ? f[i] : -INFINITY);
    }
    Vec16<T>::store(y + ((size_t)(n * Ho + ho) * Wo + wo) * C + c, m);
}

// Global average pool: a block owns 16 channel vectors (128 or 64 channels)
// of one image; its 16 thread rows split the H*W pixels (every 16th pixel per
// thread, loads issued four at a time), so every pixel row of the block is
// one contiguous 256-byte read, and the 16 partial sums are added through LDS
// in a fixed order.
template <typename T>
__global__ void __launch_bounds__(256)
gap_kernel(const T* __restrict__ x, T* __restrict__ y, int N, int HW, int C)
{
    constexpr int V = Vec16<T>::N;
    constexpr int ESZ = (int)sizeof(T);
    constexpr uint32_t OOB = 0x80000000u;
    __shared__ float part[16][16][V + 1];
    uint32_t bid = blockIdx.x, grid = gridDim.x;
    PPIPE_ARGS_NOW(bid, grid, "s"(x), "s"(y), "s"(N), "s"(HW), "s"(C));
    const int CV = C / V;
    const int cg = (CV + 15) / 16;
    const int cv = (int)bid % cg * 16 + (threadIdx.x & 15);
    const int n = (int)bid / cg;
    const int pr = threadIdx.x >> 4;    // pixel row 0..15
    const auto xr = dw_rsrc(x, (uint32_t)N * HW * C * ESZ);
    float s[V];
#pragma unroll
    for (int i = 0; i < V; ++i) s[i] = 0.0f;
    if (cv < CV) {
        const uint32_t base = (uint32_t)(((size_t)n * HW * C + (size_t)cv * V) * ESZ);
        for (int t0 = pr; t0 < HW; t0 += 64) {
            uint4 u[4];
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                const int t = t0 + 16 * d;
                u[d] = dw_load(xr, t < HW ? base + (uint32_t)(t * C * ESZ) : OOB);
            }
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                if (t0 + 16 * d >= HW)
                    break;
                float v[V];
                unpack16<T>(u[d], v);
#pragma unroll
                for (int i = 0; i < V; ++i) s[i] += v[i];
            }
        }
    }
#pragma unroll
    for (int i = 0; i < V; ++i) part[pr][threadIdx.x & 15][i] = s[i];
    __syncthreads();
    if (pr == 0 && cv < CV) {
        const float inv = 1.0f / (float)HW;
        float o[V];
#pragma unroll
        for (int i = 0; i < V; ++i) {
            float t = 0.0f;
            for (int r = 0; r < 16; ++r) t += part[r][threadIdx.x][i];
            o[i] = t * inv;
        }
        Vec16<T>::store(y + (size_t)n * C + cv * V, o);
    }
}

// One thread per pixel: C channels in, Cp out (zero tail); a 16-byte store
// when the padded pixel is exactly one vector.
template <typename T>
__global__ void __launch_bounds__(256)
pad_channels_kernel(const T* __restrict__ x, T* __restrict__ y, size_t npix, int C, int Cp)
{
    const size_t p = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= npix)
        return;
    const T* xp = x + p * C;
    if (Cp == Vec16<T>::N) {
        float v[Vec16<T>::N];
#pragma unroll
        for (int c = 0; c < Vec16<T>::N; ++c) v[c] = c < C ? (float)xp[c] : 0.0f;
        Vec16<T>::store(y + p * Cp, v);
    } else {
        for (int c = 0; c < Cp; ++c) y[p * Cp + c] = c < C ? xp[c] : (T)0.0f;
    }
}

template <typename T>
__global__ void __launch_bounds__(256) fill_uniform_kernel(T* p, size_t n, uint32_t seed)
{
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n)
        return;
    uint32_t h = (uint32_t)i * 0x9E3779B1u ^ seed;
    h ^= h >> 16; h *= 0x85EBCA6Bu; h ^= h >> 13; h *= 0xC2B2AE35u; h ^= h >> 16;
    p[i] = (T)((float)(h >> 8) * (1.0f / 16777216.0f));
}

// Cache sweep: reads a buffer (grid-stride, 16 bytes per thread per step)
// and writes one 16-byte result per thread at its end, so that the data of a
// following launch is no longer in L2 or in the memory-side cache and the
// sweep leaves almost no dirty lines behind to be written back during it.
constexpr unsigned SWEEP_BLOCKS = 4096;
__global__ void __launch_bounds__(256) sweep_kernel(const uint4* __restrict__ a,
                                                    uint4* __restrict__ res, size_t n)
{
    uint4 acc = make_uint4(0u, 0u, 0u, 0u);
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) {
        const uint4 v = a[i];
        acc.x ^= v.x; acc.y ^= v.y; acc.z ^= v.z; acc.w ^= v.w;
    }
    res[(size_t)blockIdx.x * 256 + threadIdx.x] = acc;
}

// Element-wise conversion between storage types (partition-boundary
// quantisation), 4 elements per thread; the last thread takes the tail.
// Narrowing rounds to nearest even (overflow to +-inf, subnormals kept).
template <typename Ti, typename To>
__global__ void __launch_bounds__(256) cast_kernel(const Ti* __restrict__ x, To* __restrict__ y,
                                                   size_t n)
{
    const size_t i = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (i >= n)
        return;
#pragma unroll
    for (int q = 0; q < 4; ++q)
        if (i + q < n)
            y[i + q] = (To)(float)x[i + q];
}

static unsigned blocks_for(size_t n) { return (unsigned)((n + 255) / 256); }

template <typename Ti>
static hipError_t launch_cast_to(const void* x, int out_dt, void* y, size_t n, hipStream_t s)
{
    const dim3 grid(blocks_for((n + 3) / 4));
    switch (out_dt) {
    case DT_F32:
        PPIPE_LAUNCH((cast_kernel<Ti, float>), grid, dim3(256), 0, s, (const Ti*)x, (float*)y, n);
        break;
    case DT_F16:
        PPIPE_LAUNCH((cast_kernel<Ti, _Float16>), grid, dim3(256), 0, s, (const Ti*)x,
                     (_Float16*)y, n);
        break;
    case DT_BF16:
        PPIPE_LAUNCH((cast_kernel<Ti, __bf16>), grid, dim3(256), 0, s, (const Ti*)x,
                     (__bf16*)y, n);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_cast(const void* x, int in_dt, void* y, int out_dt, size_t n, hipStream_t s)
{
    if (n == 0)
        return hipSuccess;
    switch (in_dt) {
    case DT_F32:  return launch_cast_to<float>(x, out_dt, y, n, s);
    case DT_F16:  return launch_cast_to<_Float16>(x, out_dt, y, n, s);
    case DT_BF16: return launch_cast_to<__bf16>(x, out_dt, y, n, s);
    default:      return hipErrorInvalidValue;
    }
}

hipError_t launch_cache_sweep(void* buf, size_t bytes, hipStream_t s)
{
    const size_t res = (size_t)SWEEP_BLOCKS * 256 * 16;   // one 16-byte result per thread
    if (bytes < 2 * res)
        return hipErrorInvalidValue;
    const size_t n = (bytes - res) / 16;
    PPIPE_LAUNCH(sweep_kernel, dim3(SWEEP_BLOCKS), dim3(256), 0, s, (const uint4*)buf,
                 (uint4*)((char*)buf + (bytes - res) / 16 * 16), n);
    return hipGetLastError();
}

#define PPIPE_DISPATCH(dt, KERNEL_CALL)                                   \
    switch (dt) {                                                         \
    case DT_F32:  { typedef float T; KERNEL_CALL; break; }                \
    case DT_F16:  { typedef _Float16 T; KERNEL_CALL; break; }             \
    case DT_BF16: { typedef __bf16 T; KERNEL_CALL; break; }               \
    default: return hipErrorInvalidValue;                                 \
    }

hipError_t launch_dwconv(int dt, const void* x, const void* w, const float* scale,
                         const float* bias, void* y, int N, int H, int W, int C, int Ho,
                         int Wo, int k, int stride, int pad, int act, int pw_force,
                         hipStream_t s)
{
    if (k != 3 || (stride != 1 && stride != 2))
        return hipErrorInvalidValue;
    const int cv = C / (16 / dtype_size(dt));
    // outputs per thread along a row: 4 at stride 1, 2 at stride 2
    // (pw_force = 2 or 4 overrides the stride-1 choice for tuning sweeps)
    int pw = stride == 1 ? 4 : 2;
    if (stride == 1 && (pw_force == 2 || pw_force == 4))
        pw = pw_force;
    const size_t total = (size_t)N * Ho * ((Wo + pw - 1) / pw) * cv;
    if (total >= (1u << 31) || (double)N * H * W * C * dtype_size(dt) >= 2147483648.0)
        return hipErrorInvalidValue;
#define PPIPE_DW(S_, PW_)                                                                         \
    PPIPE_DISPATCH(dt, PPIPE_LAUNCH((dwconv3_kernel<T, S_, PW_>), dim3(blocks_for(total)),        \
                                    dim3(256), 0, s, (const T*)x, (const T*)w, scale, bias,       \
                                    (T*)y, N, H, W, C, Ho, Wo, pad, act))
    if (stride == 1 && pw == 4) {
        PPIPE_DW(1, 4);
    } else if (stride == 1) {
        PPIPE_DW(1, 2);
    } else {
        PPIPE_DW(2, 2);
    }
#undef PPIPE_DW
    return hipGetLastError();
}

hipError_t launch_maxpool(int dt, const void* x, void* y, int N, int H, int W, int C,
                          int Ho, int Wo, int k, int stride, int pad, hipStream_t s)
{
    const size_t total = (size_t)N * Ho * Wo * C / (16 / dtype_size(dt));
    const bool fits32 = total < (1u << 31) && (double)N * H * W * C * dtype_size(dt) < 2147483648.0;
    if (fits32 && k == 2 && stride == 2) {
        PPIPE_DISPATCH(dt, PPIPE_LAUNCH((maxpool_fixed_kernel<T, 2, 2>), dim3(blocks_for(total)),
                                        dim3(256), 0, s, (const T*)x, (T*)y, N, H, W, C, Ho, Wo,
                                        pad));
    } else if (fits32 && k == 3 && stride == 2) {
        PPIPE_DISPATCH(dt, PPIPE_LAUNCH((maxpool_fixed_kernel<T, 3, 2>), dim3(blocks_for(total)),
                                        dim3(256), 0, s, (const T*)x, (T*)y, N, H, W, C, Ho, Wo,
                                        pad));
    } else {
        PPIPE_DISPATCH(dt, PPIPE_LAUNCH(maxpool_kernel<T>, dim3(blocks_for(total)),
                                        dim3(256), 0, s, (const T*)x, (T*)y, N, H, W, C,
                                        Ho, Wo, k, stride, pad));
    }
    return hipGetLastError();
}

hipError_t launch_gap(int dt, const void* x, void* y, int N, int HW, int C, hipStream_t s)
{
    const int CV = C / (16 / dtype_size(dt));
    const unsigned blocks = (unsigned)N * ((CV + 15) / 16);
    if ((double)N * HW * C * dtype_size(dt) >= 2147483648.0)   // 32-bit buffer offsets
        return hipErrorInvalidValue;
    PPIPE_DISPATCH(dt, PPIPE_LAUNCH(gap_kernel<T>, dim3(blocks), dim3(256), 0, s,
                                          (const T*)x, (T*)y, N, HW, C));
    return hipGetLastError();
}

hipError_t launch_pad_channels(int dt, const void* x, void* y, size_t npix, int C, int Cp,
                               hipStream_t s)
{
    PPIPE_DISPATCH(dt, PPIPE_LAUNCH(pad_channels_kernel<T>, dim3(blocks_for(npix)),
                                          dim3(256), 0, s, (const T*)x, (T*)y, npix, C, Cp));
    return hipGetLastError();
}

const char* pad_channels_name(int dt)
{
    static const char* n[3] = {"pad_channels<f32>", "pad_channels<f16>", "pad_channels<bf16>"};
    return n[dt];
}

hipError_t launch_fill_uniform(int dt, void* p, size_t n, uint32_t seed, hipStream_t s)
{
    PPIPE_DISPATCH(dt, PPIPE_LAUNCH(fill_uniform_kernel<T>, dim3(blocks_for(n)),
                                          dim3(256), 0, s, (T*)p, n, seed));
    return hipGetLastError();
}

static const char* dtn(int dt) { return dt == DT_F32 ? "f32" : dt == DT_F16 ? "f16" : "bf16"; }

const char* dwconv_name(int dt, int k)
{
    static char n[3][48];
    if (!n[dt][0]) snprintf(n[dt], 48, "dwconv%dx%d<%s>", k, k, dtn(dt));
    return n[dt];
}
const char* maxpool_name(int dt)
{
    static char n[3][32];
    if (!n[dt][0]) snprintf(n[dt], 32, "maxpool<%s>", dtn(dt));
    return n[dt];
}
const char* gap_name(int dt)
{
    static char n[3][32];
    if (!n[dt][0]) snprintf(n[dt], 32, "global_avgpool<%s>", dtn(dt));
    return n[dt];
}

}  // namespace ppipe
