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
//  * A stage is BM x BK weights plus BN x BK activations (BK = 128 bytes of
//    K per row), staged through LDS (rows padded by 16 bytes) with two LDS
//    buffers.  Global loads run DEPTH stages ahead in a ring of register sets
//    so that DEPTH stages are in flight per block; the small-M layers of a
//    partition are latency-bound and this is what keeps HBM busy.
//  * The K order (kh, kw, ci) with ci fastest makes every 16-byte vector of
//    a row one contiguous NHWC load when C is a multiple of the vector width.
//    Layers whose C is not (the 3-channel stem) gather scalars through a
//    (kh, kw, ci) lookup table in LDS.
//  * The 1-D grid is remapped so that the blocks the hardware deals to one
//    XCD (round-robin over 8) take a contiguous range of tiles: blocks that
//    read the same weight slice (or the same activation rows) share that
//    XCD's L2 instead of fetching it once per XCD.
//  * Layers with few output pixels (small batch, 7x7 / 14x14 maps, fully
//    connected layers) use a second kernel, see conv_gemm_skinny below.
#include "kernels.h"

#include <mutex>
#include <type_traits>

namespace ppipe {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int NUM_XCD = 8;

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

// The activation as one clamp (v_med3_f32): [-inf, inf], [0, inf] or [0, 6].
__device__ __forceinline__ float apply_act(float v, int act)
{
    const float lo = act == ACT_NONE ? -INFINITY : 0.0f;
    const float hi = act == ACT_RELU6 ? 6.0f : INFINITY;
    return __builtin_amdgcn_fmed3f(v, lo, hi);
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

// c ? v : 0 per component.  A conditional expression on uint4 (a class type)
// is lowered as a select between two addresses, which forces both operands
// into scratch memory; scalar selects keep everything in registers.
__device__ __forceinline__ uint4 keep_if(bool c, const uint4& v)
{
    return make_uint4(c ? v.x : 0u, c ? v.y : 0u, c ? v.z : 0u, c ? v.w : 0u);
}

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).  Keeps
// register-ring indices constant so the ring never lands in scratch memory.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f)
{
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

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

// Epilogue of one accumulator fragment row: channels co..co+3 of pixel m.
template <typename T>
__device__ __forceinline__ void store_out4(const ConvGemmArgs& a, int co, int m, floatx4 c)
{
    const float4 sc = *(const float4*)(a.scale + co);
    const float4 bi = *(const float4*)(a.bias + co);
    float4 v = make_float4(c[0] * sc.x + bi.x, c[1] * sc.y + bi.y, c[2] * sc.z + bi.z,
                           c[3] * sc.w + bi.w);
    const size_t o = (size_t)m * a.Co + co;
    if (a.softmax) {
        *(float4*)(a.logits + o) = v;
        return;
    }
    if (a.res) {
        float4 r = Vec4<T>::load((const T*)a.res + o);
        v.x += r.x; v.y += r.y; v.z += r.z; v.w += r.w;
    }
    v.x = apply_act(v.x, a.act); v.y = apply_act(v.y, a.act);
    v.z = apply_act(v.z, a.act); v.w = apply_act(v.w, a.act);
    Vec4<T>::store((T*)a.y + o, v);
}

// Epilogue of VE consecutive output channels co.. of pixel m from fp32 sums v
// (VE = 4, or 8 for 16-bit types: one 16-byte vector).
template <typename T, int VE>
__device__ __forceinline__ void store_outv(const ConvGemmArgs& a, int co, int m, const float* v)
{
    static_assert(VE == 4 || (VE == 8 && sizeof(T) == 2), "vector width");
    float o[VE];
#pragma unroll
    for (int q = 0; q < VE; q += 4) {
        const float4 sc = *(const float4*)(a.scale + co + q);
        const float4 bi = *(const float4*)(a.bias + co + q);
        o[q] = v[q] * sc.x + bi.x;
        o[q + 1] = v[q + 1] * sc.y + bi.y;
        o[q + 2] = v[q + 2] * sc.z + bi.z;
        o[q + 3] = v[q + 3] * sc.w + bi.w;
    }
    const size_t off = (size_t)m * a.Co + co;
    if (a.softmax) {
#pragma unroll
        for (int q = 0; q < VE; q += 4)
            *(float4*)(a.logits + off + q) = make_float4(o[q], o[q + 1], o[q + 2], o[q + 3]);
        return;
    }
    if constexpr (VE == 8) {
        if (a.res) {
            const uint4 u = *(const uint4*)((const T*)a.res + off);
            T r[8];
            __builtin_memcpy(r, &u, 16);
#pragma unroll
            for (int q = 0; q < 8; ++q) o[q] += (float)r[q];
        }
        T e[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) e[q] = (T)apply_act(o[q], a.act);
        uint4 u;
        __builtin_memcpy(&u, e, 16);
        *(uint4*)((T*)a.y + off) = u;
    } else {
        float4 w = make_float4(o[0], o[1], o[2], o[3]);
        if (a.res) {
            const float4 r = Vec4<T>::load((const T*)a.res + off);
            w.x += r.x; w.y += r.y; w.z += r.z; w.w += r.w;
        }
        w.x = apply_act(w.x, a.act); w.y = apply_act(w.y, a.act);
        w.z = apply_act(w.z, a.act); w.w = apply_act(w.w, a.act);
        Vec4<T>::store((T*)a.y + off, w);
    }
}

// Finish `rows` staged pixel rows of a BM-channel tile (fp32, row pitch LROW
// floats): VE channels per thread, consecutive threads along a row.  With
// K splits the raw sums go to the split's partial slice.
template <typename T, int VE, int BM, int LROW, int NT>
__device__ __forceinline__ void epi_rows(const ConvGemmArgs& a, const float* ep, int rows,
                                         int m_base, int co0, int split, int tid)
{
    constexpr int VPR = BM / VE;
    for (int v = tid; v < rows * VPR; v += NT) {
        const int row = v / VPR, c = (v - row * VPR) * VE;
        const int m = m_base + row, co = co0 + c;
        if (m >= a.M || co >= a.Co)
            continue;
        float x[VE];
#pragma unroll
        for (int q = 0; q < VE; q += 4) {
            const floatx4 t = *(const floatx4*)(ep + row * LROW + c + q);
            x[q] = t[0]; x[q + 1] = t[1]; x[q + 2] = t[2]; x[q + 3] = t[3];
        }
        if (a.splits > 1) {
#pragma unroll
            for (int q = 0; q < VE; q += 4)
                *(float4*)(a.partial + ((size_t)split * a.M + m) * a.Co + co + q) =
                    make_float4(x[q], x[q + 1], x[q + 2], x[q + 3]);
        } else {
            store_outv<T, VE>(a, co, m, x);
        }
    }
}

// Tile index -> (m tile, co tile) after spreading the 1-D grid over the XCDs
// in contiguous ranges (the hardware deals block b to XCD b % 8).
// bid, G: the block's index among the G blocks of this problem (a paired
// launch runs two problems in one grid).
__device__ __forceinline__ int3 tile_of_block(const ConvGemmArgs& a, int bid, int G)
{
    const int xcd = bid % NUM_XCD, slot = bid / NUM_XCD;
    const int per = G / NUM_XCD, rem = G % NUM_XCD;
    int lin = xcd * per + min(xcd, rem) + slot;
    const int tiles = a.tiles_m * a.tiles_co;
    const int split = lin / tiles;
    lin -= split * tiles;
    const int fast = a.co_fastest ? a.tiles_co : a.tiles_m;
    const int q = lin / fast, r = lin - q * fast;
    return a.co_fastest ? make_int3(q, r, split) : make_int3(r, q, split);   // (m tile, co tile, split)
}
__device__ __forceinline__ int3 tile_of_block(const ConvGemmArgs& a)
{
    return tile_of_block(a, (int)blockIdx.x, (int)gridDim.x);
}

// ---- buffer loads -------------------------------------------------------
// Operands are read through buffer resources: a lane whose byte offset is at
// or beyond the array size gets zeros from the hardware range check.  Zero
// padding taps, ragged tile rows and the K tail are therefore plain loads at
// offset OOB, with no branch and no select in the main loop.
constexpr uint32_t OOB = 0x80000000u;
constexpr int RSRC_FLAGS = 0x00020000;   // raw buffer, 32-bit data format

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                             RSRC_FLAGS);
}
__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
// Position of a K step in (kh, kw, ci) order, wave-uniform, advanced by a
// fixed number of channels; steps never straddle a tap (C is a multiple of the
// step, or the window is 1x1 and the tail is cut by the channel test).
struct TapCursor {
    int ci, kw, kh;
    __device__ __forceinline__ void start(int k0, int C, int KW)
    {
        const int tap = k0 / C;
        ci = k0 - tap * C;
        kh = tap / KW;
        kw = tap - kh * KW;
    }
    __device__ __forceinline__ void advance(int step, int C, int KW)
    {
        ci += step;
        if (ci >= C) {
            ci = 0;
            if (++kw == KW) {
                kw = 0;
                ++kh;
            }
        }
    }
};

// One output pixel (GEMM column) as seen by the gather: byte offset of its
// window origin and which kernel rows / columns fall inside the image.
struct PixelRow {
    int off;          // bytes of x[n][ho*s - p][wo*s - p][0] (may be negative)
    uint32_t hmask;   // bit kh set: 0 <= ho*s - p + kh < H
    uint32_t wmask;   // bit kw set: 0 <= wo*s - p + kw < W
};

__device__ __forceinline__ PixelRow pixel_row(const ConvGemmArgs& a, int m, int esz)
{
    PixelRow p{0, 0u, 0u};
    if (m >= a.M)
        return p;
    const int HoWo = a.Ho * a.Wo;
    const int n = m / HoWo, rm = m - n * HoWo;
    const int ho = rm / a.Wo, wo = rm - ho * a.Wo;
    const int hi0 = ho * a.stride - a.pad, wi0 = wo * a.stride - a.pad;
    p.off = (((n * a.H + hi0) * a.W + wi0) * a.C) * esz;
    for (int kh = 0; kh < a.KH; ++kh)
        if ((unsigned)(hi0 + kh) < (unsigned)a.H) p.hmask |= 1u << kh;
    for (int kw = 0; kw < a.KW; ++kw)
        if ((unsigned)(wi0 + kw) < (unsigned)a.W) p.wmask |= 1u << kw;
    return p;
}

// LDS-staged implicit GEMM for layers with many output pixels.
// TAPV: the channel count is a multiple of the vector width but not of the
// stage, so each 16-byte vector of a stage may sit in a different (kh, kw)
// tap; a per-block table in LDS maps vector index -> (kh, kw, ci).  Layers
// with fewer channels than a vector (3-channel stems) get their channels
// zero-padded by a prologue kernel and take this path.
template <typename T, int BM, int BN, int WM, int WN, int KV, int DEPTH, bool TAPV>
__global__ void __launch_bounds__(WM * WN * 64)
conv_gemm_kernel(ConvGemmArgs a)
{
    constexpr int NT = WM * WN * 64;
    constexpr int ESZ = (int)sizeof(T);
    constexpr int EPV = 16 / ESZ;              // elements per 16-byte vector
    constexpr int BK = KV * EPV;               // K elements per stage
    constexpr int ROW = KV * 16 + 16;          // LDS row pitch in bytes
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 16, FN = WTN / 16;
    constexpr int A_VECS = BM * KV, B_VECS = BN * KV;
    constexpr int A_PER = (A_VECS + NT - 1) / NT;
    constexpr int B_PER = (B_VECS + NT - 1) / NT;
    constexpr int STAGE = (BM + BN) * ROW;
    static_assert(KV % 4 == 0, "a stage holds whole 64-byte MFMA k-steps");
    static_assert(FM >= 1 && FN >= 1 && WTM % 16 == 0 && WTN % 16 == 0, "wave tile");
    static_assert(DEPTH == 2, "the LDS pipeline keeps two register sets in flight");

    __shared__ __attribute__((aligned(16))) unsigned char smem[2 * STAGE];
    __shared__ int vtab[TAPV ? GEMM_VTAB_MAX : 1];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int3 tt = tile_of_block(a);
    const int m0 = tt.x * BN, co0 = tt.y * BM;
    const int kc_begin = tt.z * a.chunks_per_split;
    const int kc_end = min(a.total_chunks, kc_begin + a.chunks_per_split);
    const int nst = kc_end - kc_begin;
    const auto wsrc = make_rsrc(a.w, (uint32_t)a.Co * a.Kpad * ESZ);
    const auto xsrc = make_rsrc(a.x, (uint32_t)a.N * a.H * a.W * a.C * ESZ);

    if constexpr (TAPV) {
        // vector q covers k = [q * EPV, q * EPV + EPV): one tap, channels ci..ci+EPV
        for (int q = tid; q < a.Kpad / EPV && q < GEMM_VTAB_MAX; q += NT) {
            int e = -1;
            const int k = q * EPV;
            if (k < a.K) {
                const int tap = k / a.C, ci = k - tap * a.C;
                const int kh = tap / a.KW, kw = tap - kh * a.KW;
                e = kh | (kw << 8) | (ci << 16);
            }
            vtab[q] = e;
        }
        __syncthreads();
    }

    // ---- per-thread load slots, fixed for the whole K loop ----
    uint32_t a_off[A_PER];
    int a_lds[A_PER];
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
        const int v = tid + i * NT, row = v / KV, kv = v % KV;
        const bool ok = v < A_VECS && co0 + row < a.Co;
        a_off[i] = ok ? (uint32_t)(((co0 + row) * a.Kpad + kv * EPV) * ESZ) : OOB;
        a_lds[i] = row * ROW + kv * 16;
    }
    PixelRow b_px[B_PER];
    int b_k[B_PER], b_lds[B_PER];
#pragma unroll
    for (int i = 0; i < B_PER; ++i) {
        const int v = tid + i * NT, r = v / KV, kv = v % KV;
        b_px[i] = pixel_row(a, v < B_VECS ? m0 + r : a.M, ESZ);
        b_k[i] = kv;
        b_lds[i] = BM * ROW + r * ROW + kv * 16;
    }

    // register ring: two sets, DEPTH stages in flight
    uint4 ra0[A_PER], ra1[A_PER], rb0[B_PER], rb1[B_PER];
    TapCursor cur;              // (kh, kw, ci) of the next stage to load
    int lst = kc_begin;         // its stage index
    cur.start(kc_begin * BK, a.C, a.KW);

    auto load_stage = [&](uint4 (&sa)[A_PER], uint4 (&sb)[B_PER]) {
        const uint32_t k0b = (uint32_t)(lst * BK * ESZ);
#pragma unroll
        for (int i = 0; i < A_PER; ++i)
            sa[i] = buf_load16(wsrc, a_off[i] + k0b);
        if constexpr (TAPV) {
#pragma unroll
            for (int i = 0; i < B_PER; ++i) {
                const int e = vtab[lst * KV + b_k[i]];
                const int kh = e & 0xff, kw = (e >> 8) & 0xff, ci = e >> 16;
                const bool ok = e >= 0 && ((b_px[i].hmask >> kh) & (b_px[i].wmask >> kw) & 1u);
                sb[i] = buf_load16(
                    xsrc, ok ? (uint32_t)(b_px[i].off + ((kh * a.W + kw) * a.C + ci) * ESZ) : OOB);
            }
        } else {
            const int tap_off = ((cur.kh * a.W + cur.kw) * a.C + cur.ci) * ESZ;
            const int cleft = a.C - cur.ci;
#pragma unroll
            for (int i = 0; i < B_PER; ++i) {
                const bool ok = ((b_px[i].hmask >> cur.kh) & (b_px[i].wmask >> cur.kw) & 1u) &&
                                b_k[i] * EPV < cleft;
                sb[i] = buf_load16(xsrc, ok ? (uint32_t)(b_px[i].off + tap_off + b_k[i] * 16) : OOB);
            }
        }
        if (lst < kc_end - 1) { // past the last stage the same stage is reloaded
            ++lst;
            cur.advance(BK, a.C, a.KW);
        }
    };
    auto store_stage = [&](unsigned char* S, const uint4 (&sa)[A_PER], const uint4 (&sb)[B_PER]) {
#pragma unroll
        for (int i = 0; i < A_PER; ++i)
            if (tid + i * NT < A_VECS)
                *(uint4*)(S + a_lds[i]) = sa[i];
#pragma unroll
        for (int i = 0; i < B_PER; ++i)
            if (tid + i * NT < B_VECS)
                *(uint4*)(S + b_lds[i]) = sb[i];
    };

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
            acc[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

    // fragment read offsets within a stage
    int fa[FM], fb[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[i] = (wm * WTM + i * 16 + (lane & 15)) * ROW + (lane >> 4) * 16;
#pragma unroll
    for (int j = 0; j < FN; ++j)
        fb[j] = BM * ROW + (wn * WTN + j * 16 + (lane & 15)) * ROW + (lane >> 4) * 16;

    // One pipeline step on stage s: refill the register set that held stage s
    // (it went to LDS last step) with stage s + 2, run the MFMAs on LDS buffer
    // s & 1, then move the other set (stage s + 1) into the other LDS buffer.
    // A macro over two named sets keeps every register index a constant.
#define PPIPE_STEP(s, A0, B0, A1, B1)                                                            \
    do {                                                                                          \
        load_stage(A0, B0);                                                                       \
        const unsigned char* S = smem + ((s) & 1) * STAGE;                                        \
        _Pragma("unroll") for (int ks = 0; ks < KV / 4; ++ks) {                                   \
            uint4 af[FM], bf[FN];                                                                 \
            _Pragma("unroll") for (int i = 0; i < FM; ++i)                                        \
                af[i] = *(const uint4*)(S + fa[i] + ks * 64);                                     \
            _Pragma("unroll") for (int j = 0; j < FN; ++j)                                        \
                bf[j] = *(const uint4*)(S + fb[j] + ks * 64);                                     \
            _Pragma("unroll") for (int i = 0; i < FM; ++i)                                        \
                _Pragma("unroll") for (int j = 0; j < FN; ++j)                                    \
                    Mfma<T>::step(af[i], bf[j], acc[i][j]);                                       \
        }                                                                                         \
        if ((s) + 1 < nst)                                                                        \
            store_stage(smem + (((s) + 1) & 1) * STAGE, A1, B1);                                  \
        __syncthreads();                                                                          \
    } while (0)
    if (nst > 0) {
        load_stage(ra0, rb0);
        load_stage(ra1, rb1);
        store_stage(smem, ra0, rb0);
        __syncthreads();
        for (int s0 = 0; s0 < nst; s0 += 2) {
            PPIPE_STEP(s0, ra0, rb0, ra1, rb1);
            if (s0 + 1 < nst)
                PPIPE_STEP(s0 + 1, ra1, rb1, ra0, rb0);
        }
    }
#undef PPIPE_STEP

    // ---- epilogue: lane holds channels co..co+3 of pixel m ----
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int co = co0 + wm * WTM + i * 16 + 4 * (lane >> 4);
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int m = m0 + wn * WTN + j * 16 + (lane & 15);
            if (co >= a.Co || m >= a.M)
                continue;
            if (a.splits > 1) {   // raw sums; splitk_reduce applies the epilogue
                const floatx4 c = acc[i][j];
                *(float4*)(a.partial + ((size_t)tt.z * a.M + m) * a.Co + co) =
                    make_float4(c[0], c[1], c[2], c[3]);
            } else {
                store_out4<T>(a, co, m, acc[i][j]);
            }
        }
    }
}

// ---- DMA-staged variant -------------------------------------------------
// Operand tiles go from global memory straight into LDS with buffer loads in
// LDS mode (no register staging), into a ring of NS stages.  With NS = 2 the
// next stage loads while the MFMAs consume the current one; with NS >= 3 the
// loop is software-pipelined (NS - 2 stages in flight, the fragment reads of
// stage s pending while the MFMAs of stage s - 1 run).  A stage row is 128 bytes of K
// with no padding; 16-byte vector kv of row r sits at slot kv ^ dma_swz(r).
// The MFMA fragment reads take vector kv of 16 consecutive rows; XOR with the
// row's low three bits makes these 16-byte reads free of LDS bank conflicts
// on gfx950 (measured with the SQ_LDS_BANK_CONFLICT counter; plain rows
// conflict on every read).
__device__ __forceinline__ int dma_swz(int r) { return r & 7; }

// One 16-byte load per lane from a buffer resource into LDS: lane L writes
// bytes [lds + 16 L, lds + 16 L + 16); lanes whose offset is beyond the
// resource range write zeros.  Written as inline assembly so that the compiler
// does not insert a full wait for all LDS loads before every LDS read; the
// kernel waits on the vector memory counter itself (dma_wait).  M0 carries the
// LDS address and needs one wait state before the load.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :: "s"(lds), "v"(voff), "s"(r) : "memory");
}
// Workgroup barrier without the memory fence of __syncthreads (which waits
// for every outstanding LDS read first).  Used where the LDS data a barrier
// protects was written by LDS-direct loads each wave already waited for, and
// the only reads still in flight target a stage no load overwrites next.
__device__ __forceinline__ void bare_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Wait until at most N of this wave's vector memory operations are pending
// (they complete in issue order).
template <int N>
__device__ __forceinline__ void dma_wait()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}
// Wait until every LDS read this wave issued has returned its data.
__device__ __forceinline__ void lds_read_drain() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }


// ---- prefetched single-pass epilogue (LDS-staged kernels) ----------------
// Dynamic LDS of a staged kernel: the stage ring, or the whole fp32
// [pixel][channel] accumulator tile (rows padded by 4 floats) when that is
// larger, so the epilogue stages the tile in one pass.
constexpr int gemm_lds_bytes(int BM, int BN, int NS)
{
    return NS * (BM + BN) * 128 > BN * (BM + 4) * 4 ? NS * (BM + BN) * 128 : BN * (BM + 4) * 4;
}

// Epilogue operands of one thread.  A thread finishes the same EPV channels
// (co0 + c, c fixed by the thread index) of NV pixel rows of the tile, so its
// scale, shift and residual vectors are all known when the K loop ends: their
// loads go out together, before the tile is staged, instead of one dependent
// chain per pass.
template <typename T, int BM, int BN, int NT>
struct EpiPre {
    static constexpr int ESZ = (int)sizeof(T);
    static constexpr int EPV = 16 / ESZ;
    static constexpr int VPR = BM / EPV;          // 16-byte vectors per staged pixel row
    static constexpr int NV = BN * VPR / NT;      // vectors per thread
    static_assert(NT % VPR == 0 && (BN * VPR) % NT == 0, "fixed channel group per thread");
    floatx4 sc[EPV / 4], bi[EPV / 4];
    uint4 res[NV];

    __device__ __forceinline__ void load(const ConvGemmArgs& a, int m0, int co0, int tid)
    {
        const int co = co0 + (tid % VPR) * EPV;
        const bool cok = co < a.Co;                // Co % EPV == 0: the whole vector is in range
        const auto sr = make_rsrc(a.scale, (uint32_t)a.Co * 4);
        const auto br = make_rsrc(a.bias, (uint32_t)a.Co * 4);
#pragma unroll
        for (int q = 0; q < EPV / 4; ++q) {
            sc[q] = __builtin_bit_cast(floatx4, buf_load16(sr, cok ? (uint32_t)(co + 4 * q) * 4 : OOB));
            bi[q] = __builtin_bit_cast(floatx4, buf_load16(br, cok ? (uint32_t)(co + 4 * q) * 4 : OOB));
        }
        if (a.res) {
            const auto rr = make_rsrc(a.res, (uint32_t)((size_t)a.M * a.Co * ESZ));
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                const int m = m0 + (tid + k * NT) / VPR;
                res[k] = buf_load16(rr, cok && m < a.M ? (uint32_t)(((size_t)m * a.Co + co) * ESZ) : OOB);
            }
        }
    }

    // The tile is staged in ep ([pixel][channel] fp32, LROW floats a row).
    template <int LROW>
    __device__ __forceinline__ void finish(const ConvGemmArgs& a, const float* ep, int m0, int co0,
                                           int tid) const
    {
        const int c = (tid % VPR) * EPV, co = co0 + c;
        if (co >= a.Co)
            return;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int row = (tid + k * NT) / VPR, m = m0 + row;
            if (m >= a.M)
                break;                            // rows grow with k
            float o[EPV];
#pragma unroll
            for (int q = 0; q < EPV / 4; ++q) {
                const floatx4 x = *(const floatx4*)(ep + row * LROW + c + 4 * q);
#pragma unroll
                for (int j = 0; j < 4; ++j) o[4 * q + j] = x[j] * sc[q][j] + bi[q][j];
            }
            if (a.res) {
                T r[EPV];
                __builtin_memcpy(r, &res[k], 16);
#pragma unroll
                for (int j = 0; j < EPV; ++j) o[j] += (float)r[j];
            }
            T e[EPV];
#pragma unroll
            for (int j = 0; j < EPV; ++j) e[j] = (T)apply_act(o[j], a.act);
            uint4 u;
            __builtin_memcpy(&u, e, 16);
            *(uint4*)((T*)a.y + (size_t)m * a.Co + co) = u;
        }
    }
};

template <typename T, int BM, int BN, int WM, int WN, int NS, bool TAPV>
__device__ __forceinline__ void conv_gemm_dma_body(const ConvGemmArgs& a, int bid, int G)
{
    constexpr int NW = WM * WN;
    constexpr int ESZ = (int)sizeof(T);
    constexpr int EPV = 16 / ESZ;
    constexpr int KV = 8;                      // 16-byte vectors of K per row per stage
    constexpr int BK = KV * EPV;
    constexpr int ROW = KV * 16;
    constexpr int STAGE = (BM + BN) * ROW;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 16, FN = WTN / 16;
    constexpr int PER_A = BM / (8 * NW), PER_B = BN / (8 * NW);   // loads per lane per stage
    constexpr int PER = PER_A + PER_B;
    static_assert(BM % (8 * NW) == 0 && BN % (8 * NW) == 0, "whole 8-row groups per wave");
    static_assert(NS >= 2 && (NS == 2 || (NS - 3) * PER < 64), "ring depth");
    static_assert(FM >= 1 && FN >= 1 && WTM % 16 == 0 && WTN % 16 == 0, "wave tile");

    extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
    __shared__ int vtab[TAPV ? GEMM_VTAB_MAX : 1];
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)dyn_smem;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM, wn = wave / WM;
    const int3 tt = tile_of_block(a, bid, G);
    const int m0 = tt.x * BN, co0 = tt.y * BM;
    const int kc_begin = tt.z * a.chunks_per_split;
    const int kc_end = min(a.total_chunks, kc_begin + a.chunks_per_split);
    const int nst = kc_end - kc_begin;
    const auto wsrc = make_rsrc(a.w, (uint32_t)a.Co * a.Kpad * ESZ);
    const auto xsrc = make_rsrc(a.x, (uint32_t)a.N * a.H * a.W * a.C * ESZ);
    // plain tiles (no K split, no softmax logits, whole 16-byte channel
    // vectors) take the one-pass epilogue
    const bool fast_epi = a.splits == 1 && !a.softmax && a.Co % EPV == 0;

    if constexpr (TAPV) {
        for (int q = tid; q < a.Kpad / EPV && q < GEMM_VTAB_MAX; q += NW * 64) {
            int e = -1;
            const int k = q * EPV;
            if (k < a.K) {
                const int tap = k / a.C, ci = k - tap * a.C;
                const int kh = tap / a.KW, kw = tap - kh * a.KW;
                e = kh | (kw << 8) | (ci << 16);
            }
            vtab[q] = e;
        }
        __syncthreads();
    }

    // Load slots: load i of wave w fills rows 8 (i NW + w) .. + 8 of its
    // operand; lane L covers row + L / 8, slot L % 8.
    const int lr = lane >> 3, lp = lane & 7;
    uint32_t a_off[PER_A];
#pragma unroll
    for (int i = 0; i < PER_A; ++i) {
        const int row = 8 * (i * NW + wave) + lr;
        const int kv = lp ^ dma_swz(row);
        a_off[i] = co0 + row < a.Co ? (uint32_t)(((co0 + row) * a.Kpad + kv * EPV) * ESZ) : OOB;
    }
    PixelRow b_px[PER_B];
    int b_k[PER_B];
#pragma unroll
    for (int i = 0; i < PER_B; ++i) {
        const int row = 8 * (i * NW + wave) + lr;
        b_px[i] = pixel_row(a, m0 + row, ESZ);
        b_k[i] = lp ^ dma_swz(row);
    }

    TapCursor cur;
    int lst = kc_begin;       // next stage to load
    cur.start(kc_begin * BK, a.C, a.KW);
    // Stages past the end of this block's K range load nothing (offset OOB)
    // so that every step issues the same number of loads.
    auto issue = [&](uint32_t slot) {
        const bool live = lst < kc_end;
        const uint32_t k0b = (uint32_t)(lst * BK * ESZ);
#pragma unroll
        for (int i = 0; i < PER_A; ++i)
            dma16(wsrc, live ? a_off[i] + k0b : OOB, slot + (i * NW + wave) * 8 * ROW);
        const uint32_t bslot = slot + BM * ROW;
        if constexpr (TAPV) {
#pragma unroll
            for (int i = 0; i < PER_B; ++i) {
                const int e = live ? vtab[lst * KV + b_k[i]] : -1;
                const int kh = e & 0xff, kw = (e >> 8) & 0xff, ci = e >> 16;
                const bool ok = e >= 0 && ((b_px[i].hmask >> kh) & (b_px[i].wmask >> kw) & 1u);
                dma16(xsrc, ok ? (uint32_t)(b_px[i].off + ((kh * a.W + kw) * a.C + ci) * ESZ) : OOB,
                      bslot + (i * NW + wave) * 8 * ROW);
            }
        } else {
            const int tap_off = ((cur.kh * a.W + cur.kw) * a.C + cur.ci) * ESZ;
            const int cleft = a.C - cur.ci;
#pragma unroll
            for (int i = 0; i < PER_B; ++i) {
                const bool ok = live &&
                                ((b_px[i].hmask >> cur.kh) & (b_px[i].wmask >> cur.kw) & 1u) &&
                                b_k[i] * EPV < cleft;
                dma16(xsrc, ok ? (uint32_t)(b_px[i].off + tap_off + b_k[i] * 16) : OOB,
                      bslot + (i * NW + wave) * 8 * ROW);
            }
        }
        if (live) {
            ++lst;
            cur.advance(BK, a.C, a.KW);
        }
    };

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
            acc[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

    // fragment offsets within a stage for MFMA k-steps 0 and 1 (vector g and g + 4)
    const int sw = (lane >> 4) ^ dma_swz(lane & 15);
    int fa[FM], fb[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[i] = (wm * WTM + i * 16 + (lane & 15)) * ROW + sw * 16;
#pragma unroll
    for (int j = 0; j < FN; ++j) fb[j] = (BM + wn * WTN + j * 16 + (lane & 15)) * ROW + sw * 16;

    // Software pipeline: the MFMAs of stage s - 1 run from registers while the
    // fragment reads of stage s are in flight, and loads run NS - 2 stages
    // ahead.  Step s waits for stage s, then refills the slot of stage s - 2
    // (every wave finished its MFMAs on that stage before the barrier).  Two
    // named fragment sets, loop unrolled by two, keep register indices constant.
    uint4 xa0[KV / 4][FM], xb0[KV / 4][FN], xa1[KV / 4][FM], xb1[KV / 4][FN];
#define PPIPE_READ(S, XA, XB)                                                                     \
    do {                                                                                          \
        _Pragma("unroll") for (int ks = 0; ks < KV / 4; ++ks) {                                   \
            _Pragma("unroll") for (int i = 0; i < FM; ++i)                                        \
                XA[ks][i] = *(const uint4*)((S) + (fa[i] ^ (ks * 64)));                           \
            _Pragma("unroll") for (int j = 0; j < FN; ++j)                                        \
                XB[ks][j] = *(const uint4*)((S) + (fb[j] ^ (ks * 64)));                           \
        }                                                                                         \
    } while (0)
#define PPIPE_MMA(XA, XB)                                                                         \
    do {                                                                                          \
        _Pragma("unroll") for (int ks = 0; ks < KV / 4; ++ks)                                     \
            _Pragma("unroll") for (int i = 0; i < FM; ++i)                                        \
                _Pragma("unroll") for (int j = 0; j < FN; ++j)                                    \
                    Mfma<T>::step(XA[ks][i], XB[ks][j], acc[i][j]);                               \
    } while (0)
#define PPIPE_DSTEP(s, XA, XB, YA, YB)                                                            \
    do {                                                                                          \
        dma_wait<(NS - 3) * PER>();   /* this wave's loads of stage s have landed */              \
        bare_barrier();               /* ... and every wave's; stage s - 2 is consumed */         \
        issue(lds0 + wr * STAGE);                                                                 \
        PPIPE_READ(dyn_smem + rd * STAGE, XA, XB);                                                \
        if ((s) > 0) {                                                                            \
            PPIPE_MMA(YA, YB);                                                                    \
            /* the reads of stage s all go out before the products of s - 1 */                   \
            __builtin_amdgcn_sched_group_barrier(0x100, (KV / 4) * (FM + FN), 0);                 \
            __builtin_amdgcn_sched_group_barrier(0x008, (KV / 4) * FM * FN, 0);                   \
        }                                                                                         \
        rd = rd + 1 == NS ? 0 : rd + 1;                                                           \
        wr = wr + 1 == NS ? 0 : wr + 1;                                                           \
    } while (0)
    if constexpr (NS == 2) {
// Two stages: the load of stage s + 1 runs while the MFMAs consume
        // stage s; fragment reads and MFMAs of a stage run back to back.  The
        // lowest register pressure and LDS footprint of the variants, for
        // layers with several blocks per CU.
        if (nst > 0) {
            issue(lds0);
            for (int s = 0; s < nst; ++s) {
                dma_wait<0>();     // this wave's loads of stage s have landed
                bare_barrier();    // ... and every wave's; stage s - 1 is consumed (its
                                   // fragments fed this wave's MFMAs)
                issue(lds0 + ((s + 1) & 1) * STAGE);
                const unsigned char* S = dyn_smem + (s & 1) * STAGE;
                // Every fragment read of the stage goes out before its first
                // MFMA, so the products of k-step 0 run while the reads of
                // k-step 1 are in flight (left to itself the compiler reuses
                // a few registers and waits on each read in turn).
                uint4 af[KV / 4][FM], bf[KV / 4][FN];
#pragma unroll
                for (int ks = 0; ks < KV / 4; ++ks) {
#pragma unroll
                    for (int i = 0; i < FM; ++i) af[ks][i] = *(const uint4*)(S + (fa[i] ^ (ks * 64)));
#pragma unroll
                    for (int j = 0; j < FN; ++j) bf[ks][j] = *(const uint4*)(S + (fb[j] ^ (ks * 64)));
                }
#pragma unroll
                for (int ks = 0; ks < KV / 4; ++ks)
#pragma unroll
                    for (int i = 0; i < FM; ++i)
#pragma unroll
                        for (int j = 0; j < FN; ++j)
                            Mfma<T>::step(af[ks][i], bf[ks][j], acc[i][j]);
                __builtin_amdgcn_sched_group_barrier(0x100, (KV / 4) * (FM + FN), 0);   // LDS reads
                __builtin_amdgcn_sched_group_barrier(0x008, (KV / 4) * FM * FN, 0);     // then MFMAs
            }
            dma_wait<0>();   // the empty tail load
        }
    } else if (nst > 0) {
#pragma unroll
        for (int p = 0; p < NS - 2; ++p)
            issue(lds0 + p * STAGE);
        int rd = 0, wr = NS - 2;   // slot of stage s; slot that receives stage s + NS - 2
        int s = 0;
        for (; s + 1 < nst; s += 2) {
            PPIPE_DSTEP(s, xa0, xb0, xa1, xb1);
            PPIPE_DSTEP(s + 1, xa1, xb1, xa0, xb0);
        }
        if (s < nst) {
            PPIPE_DSTEP(s, xa0, xb0, xa1, xb1);
            PPIPE_MMA(xa0, xb0);
        } else {
            PPIPE_MMA(xa1, xb1);
        }
        dma_wait<0>();   // the empty tail loads
    }
#undef PPIPE_DSTEP
#undef PPIPE_MMA
#undef PPIPE_READ

    // ---- epilogue staged through LDS ----
    // The accumulators go to a [pixel][channel] fp32 tile in the (now idle)
    // stage ring, then each thread finishes VE consecutive channels of one
    // pixel: scale, bias, residual and activation read and write whole
    // 16-byte vectors along the NHWC rows.  Plain tiles are staged in one
    // pass (the launch provides LDS for the whole tile), their operand loads
    // issued before the staging; split-K partials, softmax logits and ragged
    // channel vectors take passes of CH pixel rows.
    constexpr int LROW = BM + 4;   // floats per staged pixel row (padding spreads banks)
    if (fast_epi) {
        // the epilogue's loads go out first and land while the tile is staged
        EpiPre<T, BM, BN, NW * 64> epre;
        epre.load(a, m0, co0, tid);
        float* ept = (float*)dyn_smem;
        __syncthreads();
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
                *(floatx4*)(ept + (wn * WTN + j * 16 + (lane & 15)) * LROW + wm * WTM + i * 16 +
                            4 * (lane >> 4)) = acc[i][j];
        __syncthreads();
        epre.template finish<LROW>(a, ept, m0, co0, tid);
        return;
    }
    constexpr int CH0 = NS * STAGE / (LROW * 4);
    constexpr int CH = CH0 >= BN ? BN : CH0 / WTN * WTN;
    static_assert(CH >= WTN, "the ring holds at least one wave column of the tile");
    float* ep = (float*)dyn_smem;
#pragma unroll
    for (int p0 = 0; p0 < BN; p0 += CH) {
        __syncthreads();
        const int wc = wn * WTN;
        if (wc >= p0 && wc < p0 + CH) {
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    *(floatx4*)(ep + (wc - p0 + j * 16 + (lane & 15)) * LROW + wm * WTM + i * 16 +
                                4 * (lane >> 4)) = acc[i][j];
        }
        __syncthreads();
        const int rows = min(CH, BN - p0);
        if (a.Co % EPV == 0)
            epi_rows<T, EPV, BM, LROW, NW * 64>(a, ep, rows, m0 + p0, co0, tt.z, tid);
        else
            epi_rows<T, 4, BM, LROW, NW * 64>(a, ep, rows, m0 + p0, co0, tt.z, tid);
    }
}

template <typename T, int BM, int BN, int WM, int WN, int NS, bool TAPV>
__global__ void __launch_bounds__(WM * WN * 64)
conv_gemm_dma(ConvGemmArgs a)
{
    const int3 g = load_args_now(a, (int)blockIdx.x, (int)gridDim.x);
    conv_gemm_dma_body<T, BM, BN, WM, WN, NS, TAPV>(a, g.x, g.y);
}

// Warp-specialised variant of the 16-bit 128 x 128 eight-wave tile (plain
// taps, one K split, the one-pass epilogue): NP more waves issue every
// LDS-direct load and the eight MFMA waves only read fragments and multiply,
// so the loads of later stages no longer wait in the MFMA waves' instruction
// stream.  One barrier per stage: before barrier s the load waves have waited
// for stage s and the MFMA waves have drained their reads of stage s - 1;
// after it the load waves refill the slot of stage s - 1 with stage
// s + NS - 1.  Every wave passes the same nst + 1 barriers of the K loop and
// the two of the epilogue.
template <typename T, int BM, int BN, int WM, int WN, int NS, int NP>
__global__ void __launch_bounds__((WM * WN + NP) * 64)
conv_gemm_ws(ConvGemmArgs a)
{
    constexpr int NW = WM * WN;
    constexpr int ESZ = (int)sizeof(T);
    static_assert(ESZ == 2, "16-bit operands");
    constexpr int EPV = 16 / ESZ;
    constexpr int KV = 8, BK = KV * EPV, ROW = KV * 16;
    constexpr int STAGE = (BM + BN) * ROW;
    constexpr int WTM = BM / WM, WTN = BN / WN, FM = WTM / 16, FN = WTN / 16;
    constexpr int PA = BM / (8 * NP), PB = BN / (8 * NP), PP = PA + PB;   // loads per load wave and stage
    static_assert(BM % (8 * NP) == 0 && BN % (8 * NP) == 0, "whole 8-row groups per load wave");
    static_assert(NS >= 3 && (NS - 2) * PP < 64, "ring depth");

    extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)dyn_smem;
    const int3 g = load_args_now(a, (int)blockIdx.x, (int)gridDim.x);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int3 tt = tile_of_block(a, g.x, g.y);
    const int m0 = tt.x * BN, co0 = tt.y * BM;
    const int nst = a.total_chunks;                 // one K split

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
            acc[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
    const int wm = wave % WM, wn = (wave / WM) % WN;

    if (wave >= NW) {
        // ---- load waves: load i of load wave w fills rows 8 (i NP + w) .. + 8
        const int pw = wave - NW;
        const auto wsrc = make_rsrc(a.w, (uint32_t)a.Co * a.Kpad * ESZ);
        const auto xsrc = make_rsrc(a.x, (uint32_t)a.N * a.H * a.W * a.C * ESZ);
        const int lr = lane >> 3, lp = lane & 7;
        uint32_t a_off[PA];
#pragma unroll
        for (int i = 0; i < PA; ++i) {
            const int row = 8 * (i * NP + pw) + lr;
            const int kv = lp ^ dma_swz(row);
            a_off[i] = co0 + row < a.Co ? (uint32_t)(((co0 + row) * a.Kpad + kv * EPV) * ESZ) : OOB;
        }
        PixelRow b_px[PB];
        int b_k[PB];
#pragma unroll
        for (int i = 0; i < PB; ++i) {
            const int row = 8 * (i * NP + pw) + lr;
            b_px[i] = pixel_row(a, m0 + row, ESZ);
            b_k[i] = lp ^ dma_swz(row);
        }
        TapCursor cur;
        int lst = 0;
        cur.start(0, a.C, a.KW);
        // a stage past the end of K loads nothing (offset OOB): every call issues PP loads
        auto issue = [&](uint32_t slot) {
            const bool live = lst < nst;
            const uint32_t k0b = (uint32_t)(lst * BK * ESZ);
#pragma unroll
            for (int i = 0; i < PA; ++i)
                dma16(wsrc, live ? a_off[i] + k0b : OOB, slot + (i * NP + pw) * 8 * ROW);
            const uint32_t bslot = slot + BM * ROW;
            const int tap_off = ((cur.kh * a.W + cur.kw) * a.C + cur.ci) * ESZ;
            const int cleft = a.C - cur.ci;
#pragma unroll
            for (int i = 0; i < PB; ++i) {
                const bool ok = live &&
                                ((b_px[i].hmask >> cur.kh) & (b_px[i].wmask >> cur.kw) & 1u) &&
                                b_k[i] * EPV < cleft;
                dma16(xsrc, ok ? (uint32_t)(b_px[i].off + tap_off + b_k[i] * 16) : OOB,
                      bslot + (i * NP + pw) * 8 * ROW);
            }
            if (live) {
                ++lst;
                cur.advance(BK, a.C, a.KW);
            }
        };
#pragma unroll
        for (int p = 0; p < NS - 1; ++p)
            issue(lds0 + p * STAGE);
        int wr = NS - 1;   // slot that receives stage s + NS - 1
        for (int s = 0; s < nst; ++s) {
            dma_wait<(NS - 2) * PP>();   // stage s has landed (s + 1 .. s + NS - 2 may not)
            bare_barrier();              // barrier s
            issue(lds0 + wr * STAGE);    // the slot of stage s - 1
            wr = wr + 1 == NS ? 0 : wr + 1;
        }
        dma_wait<0>();   // the tail loads (zeros past K) have landed before the ring is reused
    } else {
        // ---- MFMA waves
        const int sw = (lane >> 4) ^ dma_swz(lane & 15);
        int fa[FM], fb[FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) fa[i] = (wm * WTM + i * 16 + (lane & 15)) * ROW + sw * 16;
#pragma unroll
        for (int j = 0; j < FN; ++j) fb[j] = (BM + wn * WTN + j * 16 + (lane & 15)) * ROW + sw * 16;
        int rd = 0;
        for (int s = 0; s < nst; ++s) {
            bare_barrier();   // barrier s: stage s has landed
            const unsigned char* S = dyn_smem + rd * STAGE;
            uint4 af[KV / 4][FM], bf[KV / 4][FN];
#pragma unroll
            for (int ks = 0; ks < KV / 4; ++ks) {
#pragma unroll
                for (int i = 0; i < FM; ++i) af[ks][i] = *(const uint4*)(S + (fa[i] ^ (ks * 64)));
#pragma unroll
                for (int j = 0; j < FN; ++j) bf[ks][j] = *(const uint4*)(S + (fb[j] ^ (ks * 64)));
            }
#pragma unroll
            for (int ks = 0; ks < KV / 4; ++ks)
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j)
                        Mfma<T>::step(af[ks][i], bf[ks][j], acc[i][j]);
            __builtin_amdgcn_sched_group_barrier(0x100, (KV / 4) * (FM + FN), 0);   // LDS reads
            __builtin_amdgcn_sched_group_barrier(0x008, (KV / 4) * FM * FN, 0);     // then MFMAs
            lds_read_drain();   // this wave's reads of stage s are done before barrier s + 1
            rd = rd + 1 == NS ? 0 : rd + 1;
        }
    }
    bare_barrier();   // the loop's last barrier: every read done, every load landed

    // ---- one-pass epilogue by the MFMA waves; the load waves take its barriers
    constexpr int LROW = BM + 4;
    EpiPre<T, BM, BN, NW * 64> epre;
    if (wave < NW)
        epre.load(a, m0, co0, tid);
    float* ept = (float*)dyn_smem;
    __syncthreads();
    if (wave < NW) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
                *(floatx4*)(ept + (wn * WTN + j * 16 + (lane & 15)) * LROW + wm * WTM + i * 16 +
                            4 * (lane >> 4)) = acc[i][j];
    }
    __syncthreads();
    if (wave < NW)
        epre.template finish<LROW>(a, ept, m0, co0, tid);
}

// Two independent layers of one tile configuration in one launch: blocks
// [0, n0) compute problem 0, the rest problem 1 (a residual block's first
// convolution and its downsample projection, which read the same input).
struct ConvGemmPair {
    ConvGemmArgs a[2];
    int n0;
};
template <typename T, int BM, int BN, int WM, int WN, int NS>
__global__ void __launch_bounds__(WM * WN * 64)
conv_gemm_dma_pair(ConvGemmPair p)
{
    const int bid = (int)blockIdx.x;
    const int q = bid < p.n0 ? 0 : 1;   // block-uniform: one inlined body
    conv_gemm_dma_body<T, BM, BN, WM, WN, NS, false>(p.a[q], q ? bid - p.n0 : bid,
                                                      q ? (int)gridDim.x - p.n0 : p.n0);
}

// ---- 32x32 matrix-instruction variant -------------------------------------
// Same LDS-direct operand staging, tile map and epilogue as conv_gemm_dma,
// but each wave owns a 64x64 (or larger) tile computed with
// v_mfma_f32_32x32x16_{f16,bf16}.  A wave tile of 64x64 reads 4 KB of
// fragments per 16-deep k-step for four 32-cycle products (32 B per clock per
// SIMD), a third less LDS read traffic per FLOP than the 64x32 wave tile of
// the 16x16 kernel.  Fragments are double-buffered per k-step: the reads of
// k-step t + 1 are in flight while the products of k-step t run, and the
// first reads of the next stage go out right after its barrier, before the
// last products of the current stage.
//
// Fragment layout of the 32x32x16 instruction (both operands): lane L
// supplies row L % 32 of its 32-row slice and the 8 consecutive k of half
// L / 32 of the 16-deep step, one 16-byte LDS read.  The accumulator of lane
// L holds column (pixel) L % 32 and rows (channels) 8q + 4 (L / 32) + r in
// element 4q + r.
typedef float floatx16 __attribute__((ext_vector_type(16)));

template <typename T> struct Mfma32;
template <> struct Mfma32<_Float16> {
    static __device__ __forceinline__ void step(const uint4& a, const uint4& b, floatx16& c)
    {
        c = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(halfx8, a),
                                                   __builtin_bit_cast(halfx8, b), c, 0, 0, 0);
    }
};
template <> struct Mfma32<__bf16> {
    static __device__ __forceinline__ void step(const uint4& a, const uint4& b, floatx16& c)
    {
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                    __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
};

// Wait until this wave's LDS reads have all returned.
__device__ __forceinline__ void lds_wait_all() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Stage-row swizzle of the 32x32 layout: vector kv of row r sits at slot
// kv ^ mx_swz(r).  A 32x32x16 fragment read takes 32 consecutive rows at two
// slots; with kv ^ (r & 7) alone, rows r and r + 8 collide (two-way bank
// conflicts on every read, measured with SQ_LDS_BANK_CONFLICT: 4 of the 8
// cycles of a 1 KB read), and flipping bit 0 for rows 8..15 of every 16
// removes them (a conflict-free 16-byte read of 64 lanes takes 4 cycles).
__device__ __forceinline__ int mx_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

template <typename T, int BM, int BN, int WM, int WN, int NS, bool TAPV>
__device__ __forceinline__ void conv_gemm_mx_body(const ConvGemmArgs& a, int bid, int G)
{
    static_assert(sizeof(T) == 2, "16-bit operands only");
    constexpr int NW = WM * WN;
    constexpr int ESZ = 2;
    constexpr int EPV = 8;
    constexpr int KV = 8;                      // 16-byte vectors of K per row per stage
    constexpr int BK = KV * EPV;               // 64 K elements per stage
    constexpr int ROW = KV * 16;
    constexpr int STAGE = (BM + BN) * ROW;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int KS = KV / 2;                 // 16-deep k-steps per stage
    constexpr int PER_A = BM / (8 * NW), PER_B = BN / (8 * NW);
    constexpr int PER = PER_A + PER_B;
    static_assert(BM % (8 * NW) == 0 && BN % (8 * NW) == 0, "whole 8-row groups per wave");
    static_assert(NS >= 2 && (NS - 2) * PER < 64, "ring depth");
    static_assert(FM >= 1 && FN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile");

    extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
    __shared__ int vtab[TAPV ? GEMM_VTAB_MAX : 1];
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)dyn_smem;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM, wn = wave / WM;
    const int3 tt = tile_of_block(a, bid, G);
    const int m0 = tt.x * BN, co0 = tt.y * BM;
    const int kc_begin = tt.z * a.chunks_per_split;
    const int kc_end = min(a.total_chunks, kc_begin + a.chunks_per_split);
    const int nst = kc_end - kc_begin;
    const auto wsrc = make_rsrc(a.w, (uint32_t)a.Co * a.Kpad * ESZ);
    const auto xsrc = make_rsrc(a.x, (uint32_t)a.N * a.H * a.W * a.C * ESZ);
    // plain tiles (no K split, no softmax logits, whole 16-byte channel
    // vectors) take the one-pass epilogue
    const bool fast_epi = a.splits == 1 && !a.softmax && a.Co % EPV == 0;

    if constexpr (TAPV) {
        for (int q = tid; q < a.Kpad / EPV && q < GEMM_VTAB_MAX; q += NW * 64) {
            int e = -1;
            const int k = q * EPV;
            if (k < a.K) {
                const int tap = k / a.C, ci = k - tap * a.C;
                const int kh = tap / a.KW, kw = tap - kh * a.KW;
                e = kh | (kw << 8) | (ci << 16);
            }
            vtab[q] = e;
        }
        __syncthreads();
    }

    // load slots: load i of wave w fills rows 8 (i NW + w) .. + 8 of its
    // operand; lane L covers row + L / 8, slot L % 8 (holding vector slot ^ mx_swz(row))
    const int lr = lane >> 3, lp = lane & 7;
    uint32_t a_off[PER_A];
#pragma unroll
    for (int i = 0; i < PER_A; ++i) {
        const int row = 8 * (i * NW + wave) + lr;
        const int kv = lp ^ mx_swz(row);
        a_off[i] = co0 + row < a.Co ? (uint32_t)(((co0 + row) * a.Kpad + kv * EPV) * ESZ) : OOB;
    }
    PixelRow b_px[PER_B];
    int b_k[PER_B];
#pragma unroll
    for (int i = 0; i < PER_B; ++i) {
        const int row = 8 * (i * NW + wave) + lr;
        b_px[i] = pixel_row(a, m0 + row, ESZ);
        b_k[i] = lp ^ mx_swz(row);
    }

    TapCursor cur;
    int lst = kc_begin;
    cur.start(kc_begin * BK, a.C, a.KW);
    auto issue = [&](uint32_t slot) {
        const bool live = lst < kc_end;
        const uint32_t k0b = (uint32_t)(lst * BK * ESZ);
#pragma unroll
        for (int i = 0; i < PER_A; ++i)
            dma16(wsrc, live ? a_off[i] + k0b : OOB, slot + (i * NW + wave) * 8 * ROW);
        const uint32_t bslot = slot + BM * ROW;
        if constexpr (TAPV) {
#pragma unroll
            for (int i = 0; i < PER_B; ++i) {
                const int e = live ? vtab[lst * KV + b_k[i]] : -1;
                const int kh = e & 0xff, kw = (e >> 8) & 0xff, ci = e >> 16;
                const bool ok = e >= 0 && ((b_px[i].hmask >> kh) & (b_px[i].wmask >> kw) & 1u);
                dma16(xsrc, ok ? (uint32_t)(b_px[i].off + ((kh * a.W + kw) * a.C + ci) * ESZ) : OOB,
                      bslot + (i * NW + wave) * 8 * ROW);
            }
        } else {
            const int tap_off = ((cur.kh * a.W + cur.kw) * a.C + cur.ci) * ESZ;
            const int cleft = a.C - cur.ci;
#pragma unroll
            for (int i = 0; i < PER_B; ++i) {
                const bool ok = live &&
                                ((b_px[i].hmask >> cur.kh) & (b_px[i].wmask >> cur.kw) & 1u) &&
                                b_k[i] * EPV < cleft;
                dma16(xsrc, ok ? (uint32_t)(b_px[i].off + tap_off + b_k[i] * 16) : OOB,
                      bslot + (i * NW + wave) * 8 * ROW);
            }
        }
        if (live) {
            ++lst;
            cur.advance(BK, a.C, a.KW);
        }
    };

    floatx16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

    // fragment offsets within a stage at k-step 0; k-step t reads offset ^ (t * 32)
    // (rows of a fragment start at multiples of 32, so mx_swz(row) = mx_swz(lane % 32))
    const int sw = ((lane >> 5) ^ mx_swz(lane & 31)) << 4;
    int fa[FM], fb[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[i] = (wm * WTM + i * 32 + (lane & 31)) * ROW + sw;
#pragma unroll
    for (int j = 0; j < FN; ++j) fb[j] = (BM + wn * WTN + j * 32 + (lane & 31)) * ROW + sw;

    uint4 xa0[FM], xb0[FN], xa1[FM], xb1[FN];
#define PPIPE_MXREAD(S, T_, XA, XB)                                                               \
    do {                                                                                          \
        _Pragma("unroll") for (int i = 0; i < FM; ++i)                                            \
            XA[i] = *(const uint4*)((S) + (fa[i] ^ ((T_) << 5)));                                 \
        _Pragma("unroll") for (int j = 0; j < FN; ++j)                                            \
            XB[j] = *(const uint4*)((S) + (fb[j] ^ ((T_) << 5)));                                 \
    } while (0)
#define PPIPE_MXMMA(XA, XB)                                                                       \
    do {                                                                                          \
        _Pragma("unroll") for (int i = 0; i < FM; ++i)                                            \
            _Pragma("unroll") for (int j = 0; j < FN; ++j)                                        \
                Mfma32<T>::step(XA[i], XB[j], acc[i][j]);                                         \
    } while (0)

    if (nst > 0) {
#pragma unroll
        for (int p = 0; p < NS - 1; ++p)
            issue(lds0 + p * STAGE);
        dma_wait<(NS - 2) * PER>();    // stage 0 of this wave
        bare_barrier();                // ... and of every wave
        int rd = 0;                    // slot of stage s
        PPIPE_MXREAD(dyn_smem, 0, xa0, xb0);
        for (int s = 0; s < nst; ++s) {
            // every wave finished reading stage s - 1 before the barrier above:
            // its slot takes stage s + NS - 1
            issue(lds0 + (rd == 0 ? NS - 1 : rd - 1) * STAGE);
            const unsigned char* S = dyn_smem + rd * STAGE;
#pragma unroll
            for (int t = 0; t < KS; t += 2) {
                PPIPE_MXREAD(S, t + 1, xa1, xb1);
                PPIPE_MXMMA(xa0, xb0);
                __builtin_amdgcn_sched_group_barrier(0x100, FM + FN, 0);   // reads of t + 1
                __builtin_amdgcn_sched_group_barrier(0x008, FM * FN, 0);   // then products of t
                if (t + 2 < KS) {
                    PPIPE_MXREAD(S, t + 2, xa0, xb0);
                    PPIPE_MXMMA(xa1, xb1);
                    __builtin_amdgcn_sched_group_barrier(0x100, FM + FN, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, FM * FN, 0);
                }
            }
            // last k-step of stage s: its fragments are in xa1/xb1.  All of
            // this wave's reads of stage s have returned (lgkmcnt 0) and its
            // loads of stage s + 1 have landed; after the barrier every wave's
            // have, so stage s + 1's first fragments can be read while the
            // last products of stage s run.
            lds_wait_all();
            if (s + 1 < nst) {
                dma_wait<(NS - 2) * PER>();
                bare_barrier();
                rd = rd + 1 == NS ? 0 : rd + 1;
                PPIPE_MXREAD(dyn_smem + rd * STAGE, 0, xa0, xb0);
            }
            PPIPE_MXMMA(xa1, xb1);
        }
        dma_wait<0>();   // the empty tail loads
    }
#undef PPIPE_MXMMA
#undef PPIPE_MXREAD

    // ---- epilogue staged through LDS: [pixel][channel] fp32 tile ----
    constexpr int LROW = BM + 4;
    if (fast_epi) {   // one pass, operands loaded first (as in conv_gemm_dma_body)
        EpiPre<T, BM, BN, NW * 64> epre;
        epre.load(a, m0, co0, tid);
        float* ept = (float*)dyn_smem;
        __syncthreads();
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const floatx4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1],
                                       acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
                    *(floatx4*)(ept + (wn * WTN + j * 32 + (lane & 31)) * LROW + wm * WTM +
                                i * 32 + 8 * q + 4 * (lane >> 5)) = v;
                }
        __syncthreads();
        epre.template finish<LROW>(a, ept, m0, co0, tid);
        return;
    }
    constexpr int CH0 = NS * STAGE / (LROW * 4);
    constexpr int CH = CH0 >= BN ? BN : CH0 / WTN * WTN;
    static_assert(CH >= WTN, "the ring holds at least one wave column of the tile");
    float* ep = (float*)dyn_smem;
#pragma unroll
    for (int p0 = 0; p0 < BN; p0 += CH) {
        __syncthreads();
        const int wc = wn * WTN;
        if (wc >= p0 && wc < p0 + CH) {
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const floatx4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1],
                                           acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
                        *(floatx4*)(ep + (wc - p0 + j * 32 + (lane & 31)) * LROW + wm * WTM +
                                    i * 32 + 8 * q + 4 * (lane >> 5)) = v;
                    }
        }
        __syncthreads();
        const int rows = min(CH, BN - p0);
        if (a.Co % EPV == 0)
            epi_rows<T, EPV, BM, LROW, NW * 64>(a, ep, rows, m0 + p0, co0, tt.z, tid);
        else
            epi_rows<T, 4, BM, LROW, NW * 64>(a, ep, rows, m0 + p0, co0, tt.z, tid);
    }
}

template <typename T, int BM, int BN, int WM, int WN, int NS, bool TAPV>
__global__ void __launch_bounds__(WM * WN * 64)
conv_gemm_mx(ConvGemmArgs a)
{
    const int3 g = load_args_now(a, (int)blockIdx.x, (int)gridDim.x);
    conv_gemm_mx_body<T, BM, BN, WM, WN, NS, TAPV>(a, g.x, g.y);
}

// Split-K reduction: one thread per 4 output channels of one pixel, partials
// summed in split order (bitwise deterministic), then the layer epilogue.  A
// load past the last split reads zeros through the range check and is not
// added.
template <typename T>
__global__ void __launch_bounds__(256) splitk_reduce_kernel(ConvGemmArgs a)
{
    const int3 g = load_args_now(a, (int)blockIdx.x, (int)gridDim.x);
    const uint32_t nvec = (uint32_t)a.M * a.Co / 4;
    const uint32_t i = (uint32_t)g.x * 256u + threadIdx.x;
    if (i >= nvec)
        return;
    const int co = (int)((i * 4u) % (uint32_t)a.Co);
    const int m = (int)((i * 4u) / (uint32_t)a.Co);
    // The epilogue's operands and the partials of up to 16 splits are all
    // requested before the first addition, so a small grid (few pixels, many
    // splits) waits for memory about once rather than once per few splits.
    // The sum still runs in split order.
    const float4 sc = *(const float4*)(a.scale + co);
    const float4 bi = *(const float4*)(a.bias + co);
    const size_t o = (size_t)m * a.Co + co;
    float4 r = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (a.res)
        r = Vec4<T>::load((const T*)a.res + o);
    const auto src = make_rsrc(a.partial, (uint32_t)a.splits * nvec * 16u);
    const uint32_t plane = nvec * 16u;
    constexpr int G = 16;
    floatx4 t = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int sp0 = 0; sp0 < a.splits; sp0 += G) {
        uint4 u[G];
#pragma unroll
        for (int d = 0; d < G; ++d)
            u[d] = buf_load16(src, sp0 + d < a.splits ? (uint32_t)(sp0 + d) * plane + i * 16u : OOB);
#pragma unroll
        for (int d = 0; d < G; ++d) {
            if (sp0 + d == 0)
                t = __builtin_bit_cast(floatx4, u[0]);
            else if (sp0 + d < a.splits)
                t += __builtin_bit_cast(floatx4, u[d]);
        }
    }
    float4 v = make_float4(t[0] * sc.x + bi.x, t[1] * sc.y + bi.y, t[2] * sc.z + bi.z,
                           t[3] * sc.w + bi.w);
    if (a.softmax) {
        *(float4*)(a.logits + o) = v;
        return;
    }
    if (a.res) {
        v.x += r.x; v.y += r.y; v.z += r.z; v.w += r.w;
    }
    v.x = apply_act(v.x, a.act); v.y = apply_act(v.y, a.act);
    v.z = apply_act(v.z, a.act); v.w = apply_act(v.w, a.act);
    Vec4<T>::store((T*)a.y + o, v);
}

// Skinny implicit GEMM for layers with few output pixels.
//
// A block of WK waves owns one (16*FM) x (16*FN) output tile; wave w reduces
// a contiguous slice of the K steps (a K step is 64 bytes of every operand
// row: one 16x16x32 MFMA for 16-bit types, four 16x16x4 for fp32).  Each MFMA
// operand fragment is one 16-byte buffer load per lane straight from global
// memory: row (lane % 16) of the weights or of the gathered activations, at
// k offset 16 * (lane / 16) bytes, so there is no LDS staging and no block
// barrier in the K loop.  Loads run DEPTH steps ahead in a register ring.
// The WK partial tiles are summed through LDS in wave order, deterministically.
template <typename T, int FM, int FN, int WK, int DEPTH>
__global__ void __launch_bounds__(WK * 64)
conv_gemm_skinny(ConvGemmArgs a)
{
    constexpr int ESZ = (int)sizeof(T);
    constexpr int EPV = 16 / ESZ;
    constexpr int KS = 4 * EPV;               // K elements per step
    constexpr int NF = FM + FN;
    __shared__ floatx4 red[WK][FM * FN][64];

    const int lane = threadIdx.x & 63;
    // wave-uniform: keeps the K-step and tap arithmetic on the scalar unit
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 4, r = lane & 15;
    const int3 bg = load_args_now(a, (int)blockIdx.x, (int)gridDim.x);
    const int3 tt = tile_of_block(a, bg.x, bg.y);
    const int m0 = tt.x * 16 * FN, co0 = tt.y * 16 * FM;
    const auto wsrc = make_rsrc(a.w, (uint32_t)a.Co * a.Kpad * ESZ);
    const auto xsrc = make_rsrc(a.x, (uint32_t)a.N * a.H * a.W * a.C * ESZ);

    // this wave's K steps [u0, u1)
    const int U = a.total_chunks;
    const int u0 = (int)((long)U * wave / WK), u1 = (int)((long)U * (wave + 1) / WK);

    uint32_t a_off[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int co = co0 + i * 16 + r;
        a_off[i] = co < a.Co ? (uint32_t)((co * a.Kpad + g * EPV) * ESZ) : OOB;
    }
    PixelRow px[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        px[j] = pixel_row(a, m0 + j * 16 + r, ESZ);
        px[j].off += g * 16;
    }
    const int gk = g * EPV;     // this lane's first channel within a step

    TapCursor cur;
    int lu = u0;
    cur.start(u0 * KS, a.C, a.KW);
    auto load = [&](uint4 (&v)[NF]) {
        const uint32_t k0b = (uint32_t)(lu * KS * ESZ);
#pragma unroll
        for (int i = 0; i < FM; ++i)
            v[i] = buf_load16(wsrc, a_off[i] + k0b);
        const int tap_off = ((cur.kh * a.W + cur.kw) * a.C + cur.ci) * ESZ;
        const bool chan_ok = gk < a.C - cur.ci;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const bool ok = chan_ok && ((px[j].hmask >> cur.kh) & (px[j].wmask >> cur.kw) & 1u);
            v[FM + j] = buf_load16(xsrc, ok ? (uint32_t)(px[j].off + tap_off) : OOB);
        }
        if (lu < u1 - 1) {
            ++lu;
            cur.advance(KS, a.C, a.KW);
        }
    };

    floatx4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
            acc[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
    auto compute = [&](const uint4 (&v)[NF]) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
                Mfma<T>::step(v[i], v[FM + j], acc[i][j]);
    };

    uint4 ring[DEPTH][NF];
    if (u0 < u1) {
        static_for<0, DEPTH>([&](auto dc) { load(ring[decltype(dc)::value]); });
        int u = u0;
        for (; u + DEPTH <= u1; u += DEPTH) {
            static_for<0, DEPTH>([&](auto dc) {
                constexpr int d = decltype(dc)::value;
                compute(ring[d]);
                load(ring[d]);
            });
        }
        static_for<0, DEPTH>([&](auto dc) {
            constexpr int d = decltype(dc)::value;
            if (u + d < u1)
                compute(ring[d]);
        });
    }

    // ---- reduce the WK partial tiles in wave order, then the epilogue ----
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
            red[wave][i * FN + j][lane] = acc[i][j];
    __syncthreads();
    for (int f = wave; f < FM * FN; f += WK) {
        floatx4 t = red[0][f][lane];
        for (int w = 1; w < WK; ++w)
            t += red[w][f][lane];
        const int i = f / FN, j = f - (f / FN) * FN;
        const int co = co0 + i * 16 + 4 * g;
        const int m = m0 + j * 16 + r;
        if (co < a.Co && m < a.M)
            store_out4<T>(a, co, m, t);
    }
}

// Softmax of each row, one block of 256 threads per row with the row held in
// registers (VPT values per thread).  With K splits the block first sums the
// raw partial rows in split order and applies the FC epilogue (scale, bias),
// so the reduction and the softmax are one launch.
template <int VPT>
__global__ void __launch_bounds__(256)
softmax_rows_kernel(const float* __restrict__ z, int splits, const float* __restrict__ scale,
                    const float* __restrict__ bias, int M, int O, float* __restrict__ out)
{
    __shared__ float red[2][4];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int m = blockIdx.x;
    const size_t plane = (size_t)M * O;
    // Split sums in split order; the loads of up to eight splits (the first
    // included) are issued before their additions, through the buffer range
    // check (past the row or the last split: zeros, not added), so that the
    // row's memory latency is paid once per eight splits.
    constexpr int G = VPT <= 8 ? 8 : 2;
    const auto zs = make_rsrc(z, (uint32_t)((size_t)splits * plane * 4));
    float v[VPT];
    for (int sp0 = 0; sp0 < splits; sp0 += G) {
        float u[G][VPT];
#pragma unroll
        for (int d = 0; d < G; ++d)
#pragma unroll
            for (int q = 0; q < VPT; ++q) {
                const int o = t + q * 256;
                const uint32_t off = sp0 + d < splits && o < O
                                         ? (uint32_t)(((sp0 + d) * plane + (size_t)m * O + o) * 4)
                                         : OOB;
                u[d][q] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(zs, off, 0, 0));
            }
#pragma unroll
        for (int d = 0; d < G; ++d)
#pragma unroll
            for (int q = 0; q < VPT; ++q) {
                if (sp0 + d == 0)
                    v[q] = u[0][q];
                else if (sp0 + d < splits)
                    v[q] += u[d][q];
            }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int q = 0; q < VPT; ++q) {
        const int o = t + q * 256;
        if (o < O) {
            if (scale) v[q] = v[q] * scale[o] + bias[o];
            mx = fmaxf(mx, v[q]);
        }
    }
    mx = wave_max(mx);
    if (lane == 0) red[0][wave] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
    float sum = 0.0f;
#pragma unroll
    for (int q = 0; q < VPT; ++q) {
        const int o = t + q * 256;
        v[q] = o < O ? expf(v[q] - mx) : 0.0f;
        sum += v[q];
    }
    sum = wave_sum(sum);
    if (lane == 0) red[1][wave] = sum;
    __syncthreads();
    const float inv = 1.0f / (red[1][0] + red[1][1] + red[1][2] + red[1][3]);
#pragma unroll
    for (int q = 0; q < VPT; ++q) {
        const int o = t + q * 256;
        if (o < O) out[(size_t)m * O + o] = v[q] * inv;
    }
}

// ---- host-side launchers ----
GemmCfgInfo gemm_cfg_info(int cfg)
{
    switch (cfg) {
    case GEMM_128x128:  return {128, 128, 8, false};
    case GEMM_64x64:    return {64, 64, 8, false};
    case GEMM_64x128:   return {64, 128, 8, false};
    case GEMM_SK_32x32: return {32, 32, 4, true};
    case GEMM_SK_32x16: return {32, 16, 4, true};
    case GEMM_SK_16x32: return {16, 32, 4, true};
    case GEMM_SK_16x16: return {16, 16, 4, true};
    case GEMM_128x128_8W: return {128, 128, 8, false};
    case GEMM_128x64:   return {128, 64, 8, false};
    case GEMM_DMA_64x64_S2: return {64, 64, 8, false, 2, 4};
    case GEMM_DMA_64x64_S3: return {64, 64, 8, false, 3, 4};
    case GEMM_DMA_128x128_8W_S2: return {128, 128, 8, false, 2, 8};
    case GEMM_PW:       return {16, 16, 4, false, 0, 4};
    case GEMM_STEM:     return {16, 16, 4, false, 0, 4};
    case GEMM_DMA_128x128_8W_S3: return {128, 128, 8, false, 3, 8};
    case GEMM_DMA_64x64_8W_S2: return {64, 64, 8, false, 2, 8};
    case GEMM_DMA_64x64_8W_S3: return {64, 64, 8, false, 3, 8};
    case GEMM_DMA_64x64_8W_S4: return {64, 64, 8, false, 4, 8};
    case GEMM_DMA_64x64_8W_S6: return {64, 64, 8, false, 6, 8};
    case GEMM_DMA_64x128_8W_S2: return {64, 128, 8, false, 2, 8};
    case GEMM_DMA_64x256_8W_S2: return {64, 256, 8, false, 2, 8};
    case GEMM_MX_128x128_S2: return {128, 128, 8, false, 2, 4, 32};
    case GEMM_MX_128x128_S3: return {128, 128, 8, false, 3, 4, 32};
    case GEMM_MX_128x128_S4: return {128, 128, 8, false, 4, 4, 32};
    case GEMM_MX_256x128_S2: return {256, 128, 8, false, 2, 8, 32};
    case GEMM_MX_128x256_S2: return {128, 256, 8, false, 2, 8, 32};
    case GEMM_MX_256x128_S3: return {256, 128, 8, false, 3, 8, 32};
    case GEMM_MX_128x128_8W_S2: return {128, 128, 8, false, 2, 8, 32};
    case GEMM_MX_128x128_8W_S3: return {128, 128, 8, false, 3, 8, 32};
    case GEMM_DMA_64x64_2W_S2: return {64, 64, 8, false, 2, 2};
    case GEMM_DMA_64x64_1W_S2: return {64, 64, 8, false, 2, 1};
    case GEMM_DMA_64x64_2W_S3: return {64, 64, 8, false, 3, 2};
    case GEMM_DMA_128x128_8W_S4: return {128, 128, 8, false, 4, 8};
    default:            return {0, 0, 0, false};
    }
}

template <typename T, int BM, int BN, int WM, int WN, int KV, int DEPTH>
static hipError_t launch_lds(bool tapv, const ConvGemmArgs& a, hipStream_t s)
{
    dim3 grid((unsigned)(a.tiles_m * a.tiles_co * a.splits));
    dim3 block(WM * WN * 64);
    if (tapv)
        PPIPE_LAUNCH((conv_gemm_kernel<T, BM, BN, WM, WN, KV, DEPTH, true>), grid, block,
                           0, s, a);
    else
        PPIPE_LAUNCH((conv_gemm_kernel<T, BM, BN, WM, WN, KV, DEPTH, false>), grid, block,
                           0, s, a);
    return hipGetLastError();
}

template <typename T, int BM, int BN, int WM, int WN, int NS, bool TAPV>
static hipError_t launch_dma_one(const ConvGemmArgs& a, hipStream_t s)
{
    constexpr int bytes = gemm_lds_bytes(BM, BN, NS);
    static const hipError_t attr = hipFuncSetAttribute(
        (const void*)conv_gemm_dma<T, BM, BN, WM, WN, NS, TAPV>,
        hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (attr != hipSuccess)
        return attr;
    PPIPE_LAUNCH((conv_gemm_dma<T, BM, BN, WM, WN, NS, TAPV>),
                       dim3((unsigned)(a.tiles_m * a.tiles_co * a.splits)), dim3(WM * WN * 64),
                       bytes, s, a);
    return hipGetLastError();
}

template <typename T, int BM, int BN, int WM, int WN, int NS>
static hipError_t launch_dma_pair(const ConvGemmArgs& a0, const ConvGemmArgs& a1, hipStream_t s)
{
    constexpr int bytes = gemm_lds_bytes(BM, BN, NS);
    static const hipError_t attr = hipFuncSetAttribute(
        (const void*)conv_gemm_dma_pair<T, BM, BN, WM, WN, NS>,
        hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (attr != hipSuccess)
        return attr;
    ConvGemmPair p;
    p.a[0] = a0;
    p.a[1] = a1;
    p.n0 = a0.tiles_m * a0.tiles_co * a0.splits;
    const int n1 = a1.tiles_m * a1.tiles_co * a1.splits;
    PPIPE_LAUNCH((conv_gemm_dma_pair<T, BM, BN, WM, WN, NS>), dim3((unsigned)(p.n0 + n1)),
                 dim3(WM * WN * 64), bytes, s, p);
    return hipGetLastError();
}

template <typename T, int BM, int BN, int WM, int WN, int NS, bool TAPV>
static hipError_t launch_mx_one(const ConvGemmArgs& a, hipStream_t s)
{
    if constexpr (sizeof(T) != 2) {
        return hipErrorInvalidValue;   // 32x32x16 instructions take 16-bit operands
    } else {
        constexpr int bytes = gemm_lds_bytes(BM, BN, NS);
        static const hipError_t attr = hipFuncSetAttribute(
            (const void*)conv_gemm_mx<T, BM, BN, WM, WN, NS, TAPV>,
            hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
        if (attr != hipSuccess)
            return attr;
        PPIPE_LAUNCH((conv_gemm_mx<T, BM, BN, WM, WN, NS, TAPV>),
                     dim3((unsigned)(a.tiles_m * a.tiles_co * a.splits)), dim3(WM * WN * 64),
                     bytes, s, a);
        return hipGetLastError();
    }
}

template <typename T, int BM, int BN, int WM, int WN, int NS>
static hipError_t launch_mx(bool tapv, const ConvGemmArgs& a, hipStream_t s)
{
    return tapv ? launch_mx_one<T, BM, BN, WM, WN, NS, true>(a, s)
                : launch_mx_one<T, BM, BN, WM, WN, NS, false>(a, s);
}

template <typename T, int BM, int BN, int WM, int WN, int NS>
static hipError_t launch_dma(bool tapv, const ConvGemmArgs& a, hipStream_t s)
{
    return tapv ? launch_dma_one<T, BM, BN, WM, WN, NS, true>(a, s)
                : launch_dma_one<T, BM, BN, WM, WN, NS, false>(a, s);
}

template <typename T, int BM, int BN, int WM, int WN, int NS, int NP>
static hipError_t launch_ws(const ConvGemmArgs& a, hipStream_t s)
{
    constexpr int bytes = gemm_lds_bytes(BM, BN, NS);
    static const hipError_t attr = hipFuncSetAttribute(
        (const void*)conv_gemm_ws<T, BM, BN, WM, WN, NS, NP>,
        hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (attr != hipSuccess)
        return attr;
    PPIPE_LAUNCH((conv_gemm_ws<T, BM, BN, WM, WN, NS, NP>), dim3((unsigned)(a.tiles_m * a.tiles_co)),
                 dim3((WM * WN + NP) * 64), bytes, s, a);
    return hipGetLastError();
}

template <typename T, int FM, int FN>
static hipError_t launch_skinny(int wk, const ConvGemmArgs& a, hipStream_t s)
{
    dim3 grid((unsigned)(a.tiles_m * a.tiles_co));
    switch (wk) {
    case 4:
        PPIPE_LAUNCH((conv_gemm_skinny<T, FM, FN, 4, 8>), grid, dim3(256), 0, s, a);
        break;
    case 8:
        PPIPE_LAUNCH((conv_gemm_skinny<T, FM, FN, 8, 8>), grid, dim3(512), 0, s, a);
        break;
    case 16:   // 1024 threads: only the 16x16 tile fits the register file
        if constexpr (FM * FN == 1) {
            PPIPE_LAUNCH((conv_gemm_skinny<T, FM, FN, 16, 8>), grid, dim3(1024), 0, s, a);
            break;
        }
        return hipErrorInvalidValue;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename T>
static hipError_t launch_cfg(int cfg, int wk, bool tapv, const ConvGemmArgs& a,
                             hipStream_t s)
{
    if (gemm_cfg_info(cfg).skinny && tapv)
        return hipErrorInvalidValue;
    switch (cfg) {
    case GEMM_128x128:  return launch_lds<T, 128, 128, 2, 2, 8, 2>(tapv, a, s);
    case GEMM_64x64:    return launch_lds<T, 64, 64, 2, 2, 8, 2>(tapv, a, s);
    case GEMM_64x128:   return launch_lds<T, 64, 128, 2, 2, 8, 2>(tapv, a, s);
    case GEMM_SK_32x32: return launch_skinny<T, 2, 2>(wk, a, s);
    case GEMM_SK_32x16: return launch_skinny<T, 2, 1>(wk, a, s);
    case GEMM_SK_16x32: return launch_skinny<T, 1, 2>(wk, a, s);
    case GEMM_SK_16x16: return launch_skinny<T, 1, 1>(wk, a, s);
    case GEMM_128x128_8W: return launch_lds<T, 128, 128, 2, 4, 8, 2>(tapv, a, s);
    case GEMM_128x64:   return launch_lds<T, 128, 64, 2, 2, 8, 2>(tapv, a, s);
    case GEMM_DMA_64x64_S2: return launch_dma<T, 64, 64, 2, 2, 2>(tapv, a, s);
    case GEMM_DMA_64x64_S3: return launch_dma<T, 64, 64, 2, 2, 3>(tapv, a, s);
    case GEMM_DMA_128x128_8W_S2: return launch_dma<T, 128, 128, 2, 4, 2>(tapv, a, s);
    case GEMM_DMA_128x128_8W_S3: return launch_dma<T, 128, 128, 2, 4, 3>(tapv, a, s);
    case GEMM_DMA_64x64_8W_S2: return launch_dma<T, 64, 64, 2, 4, 2>(tapv, a, s);
    case GEMM_DMA_64x64_8W_S3: return launch_dma<T, 64, 64, 2, 4, 3>(tapv, a, s);
    case GEMM_DMA_64x64_8W_S4: return launch_dma<T, 64, 64, 2, 4, 4>(tapv, a, s);
    case GEMM_DMA_64x64_8W_S6: return launch_dma<T, 64, 64, 2, 4, 6>(tapv, a, s);
    case GEMM_DMA_64x128_8W_S2: return launch_dma<T, 64, 128, 2, 4, 2>(tapv, a, s);
    case GEMM_DMA_64x256_8W_S2: return launch_dma<T, 64, 256, 2, 4, 2>(tapv, a, s);
    case GEMM_MX_128x128_S2: return launch_mx<T, 128, 128, 2, 2, 2>(tapv, a, s);
    case GEMM_MX_128x128_S3: return launch_mx<T, 128, 128, 2, 2, 3>(tapv, a, s);
    case GEMM_MX_128x128_S4: return launch_mx<T, 128, 128, 2, 2, 4>(tapv, a, s);
    case GEMM_MX_256x128_S2: return launch_mx<T, 256, 128, 4, 2, 2>(tapv, a, s);
    case GEMM_MX_128x256_S2: return launch_mx<T, 128, 256, 2, 4, 2>(tapv, a, s);
    case GEMM_MX_256x128_S3: return launch_mx<T, 256, 128, 4, 2, 3>(tapv, a, s);
    case GEMM_MX_128x128_8W_S2: return launch_mx<T, 128, 128, 2, 4, 2>(tapv, a, s);
    case GEMM_MX_128x128_8W_S3: return launch_mx<T, 128, 128, 2, 4, 3>(tapv, a, s);
    case GEMM_DMA_64x64_2W_S2: return launch_dma<T, 64, 64, 1, 2, 2>(tapv, a, s);
    case GEMM_DMA_64x64_1W_S2: return launch_dma<T, 64, 64, 1, 1, 2>(tapv, a, s);
    case GEMM_DMA_64x64_2W_S3: return launch_dma<T, 64, 64, 1, 2, 3>(tapv, a, s);
    case GEMM_DMA_128x128_8W_S4:
        if constexpr (sizeof(T) == 2)
            if (!tapv && a.splits == 1 && !a.softmax && a.Co % 8 == 0)
                return launch_ws<T, 128, 128, 2, 4, 4, 8>(a, s);
        return launch_dma<T, 128, 128, 2, 4, 4>(tapv, a, s);
    default:            return hipErrorInvalidValue;
    }
}

template <typename T>
static hipError_t launch_pair_cfg(int cfg, const ConvGemmArgs& a0, const ConvGemmArgs& a1,
                                  hipStream_t s)
{
    switch (cfg) {
    case GEMM_DMA_64x64_S2: return launch_dma_pair<T, 64, 64, 2, 2, 2>(a0, a1, s);
    case GEMM_DMA_64x64_S3: return launch_dma_pair<T, 64, 64, 2, 2, 3>(a0, a1, s);
    case GEMM_DMA_128x128_8W_S2: return launch_dma_pair<T, 128, 128, 2, 4, 2>(a0, a1, s);
    case GEMM_DMA_128x128_8W_S3: return launch_dma_pair<T, 128, 128, 2, 4, 3>(a0, a1, s);
    case GEMM_DMA_64x64_8W_S2: return launch_dma_pair<T, 64, 64, 2, 4, 2>(a0, a1, s);
    case GEMM_DMA_64x64_8W_S3: return launch_dma_pair<T, 64, 64, 2, 4, 3>(a0, a1, s);
    case GEMM_DMA_64x64_8W_S4: return launch_dma_pair<T, 64, 64, 2, 4, 4>(a0, a1, s);
    case GEMM_DMA_64x64_8W_S6: return launch_dma_pair<T, 64, 64, 2, 4, 6>(a0, a1, s);
    case GEMM_DMA_64x128_8W_S2: return launch_dma_pair<T, 64, 128, 2, 4, 2>(a0, a1, s);
    case GEMM_DMA_64x256_8W_S2: return launch_dma_pair<T, 64, 256, 2, 4, 2>(a0, a1, s);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_conv_gemm_pair(int dt, int cfg, const ConvGemmArgs& a0, const ConvGemmArgs& a1,
                                 hipStream_t s)
{
    if (gemm_cfg_info(cfg).dma == 0 || a0.splits != 1 || a1.splits != 1 || a0.softmax ||
        a1.softmax)
        return hipErrorInvalidValue;
    switch (dt) {
    case DT_F32:  return launch_pair_cfg<float>(cfg, a0, a1, s);
    case DT_F16:  return launch_pair_cfg<_Float16>(cfg, a0, a1, s);
    case DT_BF16: return launch_pair_cfg<__bf16>(cfg, a0, a1, s);
    default:      return hipErrorInvalidValue;
    }
}

hipError_t launch_conv_gemm(int dt, int cfg, int wk, bool tapv, const ConvGemmArgs& a,
                            hipStream_t s)
{
    if (cfg == GEMM_PW)
        return tapv ? hipErrorInvalidValue : launch_pointwise(dt, wk, a, a.grid_blocks, s);
    if (cfg == GEMM_STEM)
        return tapv ? hipErrorInvalidValue : launch_stem(dt, wk, a, a.grid_blocks, s);
    switch (dt) {
    case DT_F32:  return launch_cfg<float>(cfg, wk, tapv, a, s);
    case DT_F16:  return launch_cfg<_Float16>(cfg, wk, tapv, a, s);
    case DT_BF16: return launch_cfg<__bf16>(cfg, wk, tapv, a, s);
    default:      return hipErrorInvalidValue;
    }
}

hipError_t launch_softmax_rows(const float* z, int splits, const float* scale, const float* bias,
                               int M, int O, float* out, hipStream_t s)
{
    static_assert(SOFTMAX_MAX_O <= 256 * 32, "row fits the register array");
    if (O <= 1024)
        PPIPE_LAUNCH(softmax_rows_kernel<4>, dim3(M), dim3(256), 0, s, z, splits, scale,
                           bias, M, O, out);
    else if (O <= 2048)
        PPIPE_LAUNCH(softmax_rows_kernel<8>, dim3(M), dim3(256), 0, s, z, splits, scale,
                           bias, M, O, out);
    else if (O <= SOFTMAX_MAX_O)
        PPIPE_LAUNCH(softmax_rows_kernel<32>, dim3(M), dim3(256), 0, s, z, splits, scale,
                           bias, M, O, out);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

const char* softmax_rows_name() { return "softmax_rows<f32>"; }

hipError_t launch_splitk_reduce(int dt, const ConvGemmArgs& a, hipStream_t s)
{
    const size_t nvec = (size_t)a.M * a.Co / 4;
    if ((double)a.splits * nvec * 16.0 >= 2147483648.0)   // 32-bit buffer offsets
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)((nvec + 255) / 256)), block(256);
    switch (dt) {
    case DT_F32:
        PPIPE_LAUNCH(splitk_reduce_kernel<float>, grid, block, 0, s, a);
        break;
    case DT_F16:
        PPIPE_LAUNCH(splitk_reduce_kernel<_Float16>, grid, block, 0, s, a);
        break;
    case DT_BF16:
        PPIPE_LAUNCH(splitk_reduce_kernel<__bf16>, grid, block, 0, s, a);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

const char* splitk_reduce_name(int dt)
{
    static const char* n[3] = {"splitk_reduce<f32>", "splitk_reduce<f16>", "splitk_reduce<bf16>"};
    return n[dt];
}

static const char* dt_name(int dt)
{
    return dt == DT_F32 ? "f32" : dt == DT_F16 ? "f16" : "bf16";
}

const char* conv_gemm_name(int dt, int cfg, int wk, bool tapv)
{
    static char names[3][GEMM_NCFG][SKINNY_MAX_WAVES + 1][2][64];
    static std::mutex mu;   // entries are written once, on first use, under the lock
    std::lock_guard<std::mutex> lk(mu);
    const GemmCfgInfo c = gemm_cfg_info(cfg);
    const int w = c.skinny || cfg == GEMM_PW || cfg == GEMM_STEM ? wk : 0;
    char* n = names[dt][cfg][w][tapv ? 1 : 0];
    if (!n[0]) {
        if (cfg == GEMM_PW)
            snprintf(n, 64, "pw_conv<%s,cf%d>", dt_name(dt), wk);
        else if (cfg == GEMM_STEM)
            snprintf(n, 64, "stem_conv<%s,cf%d>", dt_name(dt), wk);
        else if (c.skinny)
            snprintf(n, 64, "conv_gemm_skinny<%s,%dx%d,waves%d>", dt_name(dt), c.bm, c.bn, wk);
        else if (c.dma && c.mfma == 32)
            snprintf(n, 64, "conv_gemm_mx<%s,%dx%d,%dw,dma%d%s>", dt_name(dt), c.bm, c.bn,
                     c.waves, c.dma, tapv ? ",tapv" : "");
        else if (c.dma)
            snprintf(n, 64, "conv_gemm<%s,%dx%d,kv%d%s,dma%d%s>", dt_name(dt), c.bm, c.bn, c.kv,
                     c.waves == 8 ? ",8w" : c.waves == 2 ? ",2w" : c.waves == 1 ? ",1w" : "",
                     c.dma, tapv ? ",tapv" : "");
        else
            snprintf(n, 64, "conv_gemm<%s,%dx%d,kv%d%s%s>", dt_name(dt), c.bm, c.bn, c.kv,
                     cfg == GEMM_128x128_8W ? ",8w" : "", tapv ? ",tapv" : "");
    }
    return n;
}

}  // namespace ppipe
