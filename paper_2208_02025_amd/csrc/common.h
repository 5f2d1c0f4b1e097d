// Internal helpers shared by the gfx950 kernels and the host dispatch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ollie {

typedef uint16_t bf16_t;                                         // raw bfloat16 bits
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));       // MFMA operand (8 x bf16)
typedef float f32x4 __attribute__((ext_vector_type(4)));         // 16x16 MFMA accumulator
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));      // 16-byte raw chunk

// float -> bfloat16 bits, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ bf16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu))
        return (bf16_t)((u >> 16) | 0x0040u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
}

__device__ __forceinline__ float bf2f(bf16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// Store helpers for fp32 / bf16 outputs.
template <typename T> struct Out;
template <> struct Out<float> {
    static __device__ __forceinline__ void put(float* p, float v) { *p = v; }
    static __device__ __forceinline__ void put4(float* p, f32x4 v) {
        *reinterpret_cast<f32x4*>(p) = v;
    }
};
template <> struct Out<bf16_t> {
    static __device__ __forceinline__ void put(bf16_t* p, float v) { *p = f2bf(v); }
    static __device__ __forceinline__ void put4(bf16_t* p, f32x4 v) {
        uint32_t lo = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
        uint32_t hi = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
        *reinterpret_cast<uint2*>(p) = make_uint2(lo, hi);
    }
};

// Load helpers: 4 consecutive values widened to fp32.
template <typename T> struct In;
template <> struct In<float> {
    static __device__ __forceinline__ float get(const float* p) { return *p; }
    static __device__ __forceinline__ f32x4 get4(const float* p) {
        return *reinterpret_cast<const f32x4*>(p);
    }
};
template <> struct In<bf16_t> {
    static __device__ __forceinline__ float get(const bf16_t* p) { return bf2f(*p); }
    static __device__ __forceinline__ f32x4 get4(const bf16_t* p) {
        uint2 u = *reinterpret_cast<const uint2*>(p);
        f32x4 r;
        r[0] = __uint_as_float(u.x << 16);
        r[1] = __uint_as_float(u.x & 0xffff0000u);
        r[2] = __uint_as_float(u.y << 16);
        r[3] = __uint_as_float(u.y & 0xffff0000u);
        return r;
    }
};

// Element-wise tail of a convolution-family operator: + bias[k] + residual[pixel][k],
// then ReLU, in fp32 right before the store (a null pointer drops its term).
struct Epi {
    const void* bias;
    const void* res;
    int bias_bf16, res_bf16, relu;
};
__device__ __forceinline__ float epi_load(const void* p, int bf16, int64_t i) {
    return bf16 ? bf2f(reinterpret_cast<const bf16_t*>(p)[i])
                : reinterpret_cast<const float*>(p)[i];
}
__device__ __forceinline__ f32x4 epi_load4(const void* p, int bf16, int64_t i) {
    return bf16 ? In<bf16_t>::get4(reinterpret_cast<const bf16_t*>(p) + i)
                : In<float>::get4(reinterpret_cast<const float*>(p) + i);
}
// ReLU that keeps a NaN a NaN (x < 0 is false for NaN)
__device__ __forceinline__ float relu_f(float x) { return x < 0.f ? 0.f : x; }
// v = out[oi + j] for channels k + j, j = 0..3 (oi, k multiples of 4)
__device__ __forceinline__ f32x4 epi_apply4(const Epi& e, f32x4 v, int64_t oi, int64_t k) {
    if (e.bias) v += epi_load4(e.bias, e.bias_bf16, k);
    if (e.res) v += epi_load4(e.res, e.res_bf16, oi);
    if (e.relu) {
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = relu_f(v[j]);
    }
    return v;
}
__device__ __forceinline__ float epi_apply(const Epi& e, float v, int64_t oi, int64_t k) {
    if (e.bias) v += epi_load(e.bias, e.bias_bf16, k);
    if (e.res) v += epi_load(e.res, e.res_bf16, oi);
    return e.relu ? relu_f(v) : v;
}

// ------------------------------------------------- shared GEMM-tile building blocks
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kTileK = 64;                 // bf16 k-tile depth (128 bytes per row)
constexpr int kTileChunks = kTileK / 8;    // 16-byte chunks per tile row

// LDS slot of logical 16-byte chunk `ch` of tile row `row`: an XOR swizzle that makes
// the 16-row ds_read_b128 fragment reads of an MFMA operand bank-conflict free.
__device__ __forceinline__ int tile_swz(int row, int ch) {
    return row * kTileChunks + (ch ^ (row & 7));
}

// The same for a k-tile of BK bf16 (BK/8 chunks per row): 128-byte rows use the chunk
// XOR (row & 7); 64-byte rows pair up rows and XOR (row/2 & 3), so the eight rows that
// one ds_read_b128 phase touches still land on disjoint banks.
template <int BK>
__device__ __forceinline__ int tile_swz_k(int row, int ch) {
    static_assert(BK == 32 || BK == 64, "k-tile depth");
    if constexpr (BK == 64) return row * 8 + (ch ^ (row & 7));
    else return row * 4 + (ch ^ ((row >> 1) & 3));
}

// One 16-byte-per-lane copy global->LDS through a raw buffer load: lane L's chunk at
// byte offset voff + soff of `base` lands at dst + 16 L.  An offset at or beyond
// `nbytes` reads zeros.  (Kept out of templates: the buffer-resource type inside a
// kernel template stops the host pass from emitting that kernel's launch stub.)
__device__ __forceinline__ void buffer_copy16(const void* base, int nbytes, uint32_t voff,
                                              int soff, lds_void* dst) {
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, nbytes, 0x00020000);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, soff, 0, 0);
}

// s_waitcnt with only the vector-memory counter constrained (expcnt, lgkmcnt at max).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// ---------------------------------------------------------------- launchers
// Each returns the hipError_t of the launch.

// `tile` / `shape` arguments: a forced tile configuration of the kernel (tuning sweeps
// and tests), or -1 for the automatic choice.
hipError_t launch_gemm_nt(int64_t m, int64_t n, int64_t k, const void* a, const void* b,
                          void* y, int in_bf16, int y_bf16, int tile, hipStream_t stream);

struct ConvGeom {
    int64_t n, c, h, w, k, r, s, ho, wo;
    int32_t sh, sw, ph, pw, dh, dw;
};

hipError_t launch_eop_gather(const ConvGeom& g, int transposed, const void* y, int y_bf16,
                             void* out, int out_bf16, const Epi& epi, hipStream_t stream);

// The R x S -> 3x3 derived form's two eOperators (the 3x3 stage's OffsetAdd and the
// block OffsetAdd) fused into one OffsetAdd over the split form's scope
// Y [n*h*w][9*ceil(R/3)*ceil(S/3)*K] (g: the original stride-1 convolution).
hipError_t launch_eop_split3_chain(const ConvGeom& g, const void* y, int y_bf16, void* out,
                                   int out_bf16, const Epi& epi, hipStream_t stream);

// Fused GEMM + eOperator (output-stationary), bf16 operands.  form: the derived
// program evaluated -- the forward convolution, the transposed convolution, or a
// stride-1 dilated convolution as dil_h*dil_w non-dilated convolutions over the
// residue sub-images of the input.  Returns hipErrorInvalidValue when the shape is
// outside what the fused kernel supports.
enum ConvForm { kForward = 0, kTransposed = 1, kResidues = 2 };
bool conv_fused_supported(const ConvGeom& g, int form);
hipError_t launch_conv_fused(const ConvGeom& g, int form, const void* x, const void* wt,
                             void* out, int out_bf16, const Epi& epi, int tile,
                             hipStream_t stream);

// Weight blocks of the R x S -> 3x3 derived form: W3 [3][3][ceil(R/3)*ceil(S/3)*K][C]
// from Wt [R][S][K][C] (g.r, g.s, g.k, g.c), zero where a block overhangs the kernel.
hipError_t launch_split_weights_3x3(const ConvGeom& g, const void* wt, void* w3, int bf16,
                                    hipStream_t stream);

struct BandGeom {
    int64_t b, l, d, w;
    int32_t dil;
    float scale;
};

hipError_t launch_band_g2bmm(const BandGeom& g, const void* q, const void* k, float* s,
                             hipStream_t stream);
hipError_t launch_band_softmax(const BandGeom& g, const float* s, void* p, int mask,
                               hipStream_t stream);
hipError_t launch_band_gbmm(const BandGeom& g, const void* p, const void* v, void* o,
                            int o_bf16, hipStream_t stream);
hipError_t launch_band_fused(const BandGeom& g, const void* q, const void* k, const void* v,
                             void* o, int o_bf16, int mask, int shape, hipStream_t stream);

}  // namespace ollie
