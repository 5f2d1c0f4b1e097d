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
//
// Latency: a thread's taps are independent loads, so the common shapes take a kernel
// that computes every candidate tap's address first and issues all of the loads
// before the first add (a tap that is outside the image reads a valid address and
// is dropped by a select), keeping MT*MT 16-byte loads per thread in flight instead
// of one.  Candidates per axis: all R (S) taps of the forward form; for the
// transposed form the taps r with (ho + ph - r*dh) divisible by sh, an arithmetic
// progression r0, r0 + sh/gcd(sh,dh), ...  Large grids (over 2^20 threads, dozens of
// waves per CU) already cover the latency with resident waves; there the loop kernel,
// whose loads stream through Y in a more orderly way, measured ~3% faster.
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

// First candidate and step of the taps along one axis for output coordinate `o`
// (see the header comment); `cnt` candidates r0 + i*step, i < cnt, lie in [0, R).
__device__ __forceinline__ void axis_taps(int o, int stride, int pad, int dil, int R,
                                          int step, bool transposed, int& r0, int& cnt) {
    if (!transposed) {
        r0 = 0;
        cnt = R;
        return;
    }
    const int t0 = o + pad;
    r0 = R;
    for (int r = 0; r < step && r < R; ++r)
        if ((t0 - r * dil) % stride == 0) {
            r0 = r;
            break;
        }
    cnt = r0 < R ? (R - 1 - r0) / step + 1 : 0;
}

template <typename YT, typename OT, bool TRANSPOSED, int MT>
__global__ __launch_bounds__(256) void eop_taps_kernel(const YT* __restrict__ Y,
                                                       OT* __restrict__ out, ConvGeom g,
                                                       int64_t total, int step_h, int step_w,
                                                       Epi epi) {
    const int64_t item = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (item >= total) return;
    const int kv = (int)(g.k / 4);
    const int ho_n = (int)g.ho, wo_n = (int)g.wo;
    // total < 2^31 (checked on the host), so 32-bit index arithmetic is exact here
    const int it = (int)item;
    const int k = (it % kv) * 4;
    int pix = it / kv;
    const int wo = pix % wo_n;
    pix /= wo_n;
    const int ho = pix % ho_n;
    const int n = pix / ho_n;
    const int H = (int)g.h, W = (int)g.w, R = (int)g.r, S = (int)g.s, K = (int)g.k;
    const int64_t nc = (int64_t)R * S * K;

    int r0, cr, s0, cs;
    axis_taps(ho, g.sh, g.ph, g.dh, R, step_h, TRANSPOSED, r0, cr);
    axis_taps(wo, g.sw, g.pw, g.dw, S, step_w, TRANSPOSED, s0, cs);
    // candidate input rows/columns and their validity
    int hi[MT], wi[MT];
    bool vh[MT], vw[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        const int r = r0 + t * step_h, s = s0 + t * step_w;
        if (TRANSPOSED) {
            hi[t] = (ho + g.ph - r * g.dh) / g.sh;   // exact: divisibility holds by construction
            wi[t] = (wo + g.pw - s * g.dw) / g.sw;
            vh[t] = t < cr && ho + g.ph - r * g.dh >= 0 && hi[t] < H;
            vw[t] = t < cs && wo + g.pw - s * g.dw >= 0 && wi[t] < W;
        } else {
            hi[t] = ho * g.sh - g.ph + r * g.dh;
            wi[t] = wo * g.sw - g.pw + s * g.dw;
            vh[t] = t < cr && hi[t] >= 0 && hi[t] < H;
            vw[t] = t < cs && wi[t] >= 0 && wi[t] < W;
        }
    }
    f32x4 v[MT][MT];
#pragma unroll
    for (int a = 0; a < MT; ++a)
#pragma unroll
        for (int b = 0; b < MT; ++b) {
            const bool ok = vh[a] && vw[b];
            const int r = r0 + a * step_h, s = s0 + b * step_w;
            const int64_t row = ((int64_t)n * H + hi[a]) * W + wi[b];
            // an invalid tap reads element 0 of Y (always there) and is discarded below
            const YT* src = ok ? Y + row * nc + (int64_t)(r * S + s) * K + k : Y;
            v[a][b] = In<YT>::get4(src);
        }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int a = 0; a < MT; ++a)
#pragma unroll
        for (int b = 0; b < MT; ++b)
            if (vh[a] && vw[b]) acc += v[a][b];
    const int64_t oi = (((int64_t)n * ho_n + ho) * wo_n + wo) * K + k;
    Out<OT>::put4(out + oi, epi_apply4(epi, acc, oi, k));
}

// The two consecutive eOperators of the R x S -> 3x3 derived form fused into one
// (eOperator fusion, section 5.4).  That form computes Y = X * W3^T with the split
// weights W3[r'][s'][(a*nbs + b)*K + k] = Wt[3a + r'][3b + s'][k], then
//   Z[n][i][j][(a,b),k] = sum_{r',s'} Y[(n, i - ph - er + r', j - pw - es + s')][(r'*3+s')*nbr*nbs*K + (a,b)*K + k]
//   out[n][ho][wo][k]   = sum_{a,b} Z[n][ho + er + 3a][wo + es + 3b][(a,b),k].
// Substituting the first into the second (the shifts er, es cancel) gives one
// OffsetAdd over Y:
//   out[n][ho][wo][k] = sum_{a,b,r',s'} [0 <= hi < h][0 <= wi < w]
//                       Y[(n*h + hi)*w + wi][((r'*3 + s')*nbr*nbs + a*nbs + b)*K + k]
//   hi = ho - ph + 3a + r',  wi = wo - pw + 3b + s'.
// Taps of the relaxed kernel (3a + r' >= R or 3b + s' >= S) have zero weights, so their
// partials are zero and are not read (boundary tightening): the loop runs over the R x S
// taps r = 3a + r', s = 3b + s'.  Y is read once and Z never exists.  Stride 1,
// dilation 1 (the form's domain).
template <typename YT, typename OT, int VEC>
__global__ __launch_bounds__(256) void eop_split3_chain_kernel(const YT* __restrict__ Y,
                                                               OT* __restrict__ out, ConvGeom g,
                                                               int64_t total, Epi epi) {
    const int64_t item = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (item >= total) return;
    const int kv = (int)(g.k / VEC);
    const int ho_n = (int)g.ho, wo_n = (int)g.wo;
    const int it = (int)item;   // total < 2^31 (checked on the host)
    const int k = (it % kv) * VEC;
    int pix = it / kv;
    const int wo = pix % wo_n;
    pix /= wo_n;
    const int ho = pix % ho_n;
    const int n = pix / ho_n;
    const int H = (int)g.h, W = (int)g.w, R = (int)g.r, S = (int)g.s, K = (int)g.k;
    const int nbs = (S + 2) / 3, nb = ((R + 2) / 3) * nbs;
    const int64_t nc = (int64_t)9 * nb * K;   // row length of Y

    float acc[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = 0.f;
    for (int r = 0; r < R; ++r) {
        const int hi = ho - g.ph + r;
        if (hi < 0 || hi >= H) continue;
        const int a = r / 3, rr = r - 3 * a;
        for (int s = 0; s < S; ++s) {
            const int wi = wo - g.pw + s;
            if (wi < 0 || wi >= W) continue;
            const int b = s / 3, ss = s - 3 * b;
            const int64_t row = ((int64_t)n * H + hi) * W + wi;
            const YT* src = Y + row * nc + ((int64_t)(rr * 3 + ss) * nb + a * nbs + b) * K + k;
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

template <typename YT, typename OT>
hipError_t go_chain(const ConvGeom& g, const void* y, void* out, const Epi& epi,
                    hipStream_t st) {
    const bool v4 = (g.k & 3) == 0;
    const int64_t total = g.n * g.ho * g.wo * (v4 ? g.k / 4 : g.k);
    if (total == 0) return hipSuccess;
    const dim3 grid((unsigned)((total + 255) / 256));
    if (v4)
        hipLaunchKernelGGL((eop_split3_chain_kernel<YT, OT, 4>), grid, dim3(256), 0, st,
                           (const YT*)y, (OT*)out, g, total, epi);
    else
        hipLaunchKernelGGL((eop_split3_chain_kernel<YT, OT, 1>), grid, dim3(256), 0, st,
                           (const YT*)y, (OT*)out, g, total, epi);
    return hipGetLastError();
}

int gcd_int(int a, int b) {
    while (b) {
        const int t = a % b;
        a = b;
        b = t;
    }
    return a;
}

// Candidates per axis of the unrolled kernel, or 0 when the shape takes the loop kernel.
int tap_slots(const ConvGeom& g, int transposed, int& step_h, int& step_w) {
    if (g.n * g.ho * g.wo * (g.k / 4) > (int64_t(1) << 20)) return 0;
    step_h = transposed ? (int)(g.sh / gcd_int((int)g.sh, (int)g.dh)) : 1;
    step_w = transposed ? (int)(g.sw / gcd_int((int)g.sw, (int)g.dw)) : 1;
    const int ch = (int)((g.r + step_h - 1) / step_h), cw = (int)((g.s + step_w - 1) / step_w);
    const int c = ch > cw ? ch : cw;
    return c <= 2 ? 2 : c <= 3 ? 3 : 0;
}

template <typename YT, typename OT, bool TR, int MT>
hipError_t go_taps(const ConvGeom& g, const void* y, void* out, const Epi& epi, int step_h,
                   int step_w, hipStream_t st) {
    const int64_t total = g.n * g.ho * g.wo * (g.k / 4);
    if (total == 0) return hipSuccess;
    hipLaunchKernelGGL((eop_taps_kernel<YT, OT, TR, MT>), dim3((unsigned)((total + 255) / 256)),
                       dim3(256), 0, st, (const YT*)y, (OT*)out, g, total, step_h, step_w, epi);
    return hipGetLastError();
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
    if ((g.k & 3) == 0) {
        int step_h, step_w;
        const int mt = tap_slots(g, transposed, step_h, step_w);
        if (mt == 2)
            return transposed ? go_taps<YT, OT, true, 2>(g, y, out, epi, step_h, step_w, st)
                              : go_taps<YT, OT, false, 2>(g, y, out, epi, step_h, step_w, st);
        if (mt == 3)
            return transposed ? go_taps<YT, OT, true, 3>(g, y, out, epi, step_h, step_w, st)
                              : go_taps<YT, OT, false, 3>(g, y, out, epi, step_h, step_w, st);
        return go<YT, OT, 4>(g, transposed, y, out, epi, st);
    }
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

hipError_t launch_eop_split3_chain(const ConvGeom& g, const void* y, int y_bf16, void* out,
                                   int out_bf16, const Epi& epi, hipStream_t stream) {
    if (y_bf16)
        return out_bf16 ? go_chain<bf16_t, bf16_t>(g, y, out, epi, stream)
                        : go_chain<bf16_t, float>(g, y, out, epi, stream);
    return out_bf16 ? go_chain<float, bf16_t>(g, y, out, epi, stream)
                    : go_chain<float, float>(g, y, out, epi, stream);
}

}  // namespace ollie
