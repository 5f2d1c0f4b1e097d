// eOperator stage of the derived convolution forms: a memory-bound gather-sum over
// the instantiated scope Y [n*h*w][r*s*k].
//
//   forward (OffsetAdd, section 2; dilated form via the tap spacing):
//     out[n][ho][wo][k] = sum_{r,s} [0 <= hi < h][0 <= wi < w] Y[(n*h+hi)*w+wi][(r*S+s)*K+k]
//     hi = ho*sh - ph + r*dh,  wi = wo*sw - pw + s*dw
//   transposed (selective add, section 6.3):
//     th = ho + ph - r*dh >= 0, th % sh == 0, hi = th / sh < h  (likewise along w)
//
// Taps outside the image are never read (boundary tightening, section 4.2), so each
// element of Y is read at most once.  An element-wise tail (bias, residual, ReLU) is
// applied to the sum before the store: OffsetAdd fused with the element-wise operators
// that follow it (section 6.3).  One thread owns VEC consecutive output channels
// of one output pixel; a wavefront covers 64*VEC contiguous channels, so every tap
// is one contiguous, coalesced read of a K-vector.
#include "common.h"

namespace ollie {

namespace {

template <typename YT, typename OT, int VEC, bool TRANSPOSED>
__global__ __launch_bounds__(256) void eop_gather_kernel(const YT* __restrict__ Y,
                                                         OT* __restrict__ out, ConvGeom g,
                                                         int64_t total, Epi epi) {
    const int64_t item = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (item >= total) return;
    const int kv = (int)(g.k / VEC);
    const int ho_n = (int)g.ho, wo_n = (int)g.wo;
    // total < 2^31 (checked on the host), so 32-bit index arithmetic is exact here
    const int it = (int)item;
    const int k = (it % kv) * VEC;
    int pix = it / kv;
    const int wo = pix % wo_n;
    pix /= wo_n;
    const int ho = pix % ho_n;
    const int n = pix / ho_n;
    const int H = (int)g.h, W = (int)g.w, R = (int)g.r, S = (int)g.s, K = (int)g.k;
    const int64_t nc = (int64_t)R * S * K;

    float acc[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = 0.f;

    for (int r = 0; r < R; ++r) {
        int hi;
        if (TRANSPOSED) {
            int th = ho + g.ph - r * g.dh;
            if (th < 0 || th % g.sh != 0) continue;
            hi = th / g.sh;
            if (hi >= H) continue;
        } else {
            hi = ho * g.sh - g.ph + r * g.dh;
            if (hi < 0 || hi >= H) continue;
        }
        for (int s = 0; s < S; ++s) {
            int wi;
            if (TRANSPOSED) {
                int tw = wo + g.pw - s * g.dw;
                if (tw < 0 || tw % g.sw != 0) continue;
                wi = tw / g.sw;
                if (wi >= W) continue;
            } else {
                wi = wo * g.sw - g.pw + s * g.dw;
                if (wi < 0 || wi >= W) continue;
            }
            const int64_t row = ((int64_t)n * H + hi) * W + wi;
            const YT* src = Y + row * nc + (int64_t)(r * S + s) * K + k;
            if (VEC == 4) {
                f32x4 v = In<YT>::get4(src);
#pragma unroll
                for (int e = 0; e < VEC; ++e) acc[e] += v[e];
            } else {
#pragma unroll
                for (int e = 0; e < VEC; ++e) acc[e] += In<YT>::get(src + e);
            }
        }
    }
    const int64_t oi = (((int64_t)n * ho_n + ho) * wo_n + wo) * K + k;
    OT* dst = out + oi;
    if (VEC == 4) {
        f32x4 v = {acc[0], acc[1], acc[2], acc[3]};
        Out<OT>::put4(dst, epi_apply4(epi, v, oi, k));
    } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            Out<OT>::put(dst + e, epi_apply(epi, acc[e], oi + e, k + e));
    }
}

template <typename YT, typename OT, int VEC>
hipError_t go(const ConvGeom& g, int transposed, const void* y, void* out, const Epi& epi,
              hipStream_t st) {
    int64_t total = g.n * g.ho * g.wo * (g.k / VEC);
    if (total == 0) return hipSuccess;
    dim3 grid((unsigned)((total + 255) / 256));
    if (transposed)
        hipLaunchKernelGGL((eop_gather_kernel<YT, OT, VEC, true>), grid, dim3(256), 0, st,
                           (const YT*)y, (OT*)out, g, total, epi);
    else
        hipLaunchKernelGGL((eop_gather_kernel<YT, OT, VEC, false>), grid, dim3(256), 0, st,
                           (const YT*)y, (OT*)out, g, total, epi);
    return hipGetLastError();
}

template <typename YT, typename OT>
hipError_t pick_vec(const ConvGeom& g, int transposed, const void* y, void* out,
                    const Epi& epi, hipStream_t st) {
    if ((g.k & 3) == 0) return go<YT, OT, 4>(g, transposed, y, out, epi, st);
    return go<YT, OT, 1>(g, transposed, y, out, epi, st);
}

}  // namespace

hipError_t launch_eop_gather(const ConvGeom& g, int transposed, const void* y, int y_bf16,
                             void* out, int out_bf16, const Epi& epi, hipStream_t stream) {
    if (y_bf16)
        return out_bf16 ? pick_vec<bf16_t, bf16_t>(g, transposed, y, out, epi, stream)
                        : pick_vec<bf16_t, float>(g, transposed, y, out, epi, stream);
    return out_bf16 ? pick_vec<float, bf16_t>(g, transposed, y, out, epi, stream)
                    : pick_vec<float, float>(g, transposed, y, out, epi, stream);
}

}  // namespace ollie
