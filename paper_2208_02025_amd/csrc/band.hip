// Banded dilated batched matmul: G2BMM (Table 2 iterator groups: bm in all tensors,
// w in weight+output, k in input+weight), row softmax, and the band-times-dense
// product, for head dimension 64.
//
// Dilation removal (section 6.4): with row i = dil*i' + rho the key of band entry j is
//   t = i + (j - w)*dil = dil*(i' + j - w) + rho,
// a NON-dilated band t' = i' + j - w on the residue-rho subsequence.  Every kernel
// works on one (batch, residue, 64-query tile) of that subsequence, so keys and
// values are read as contiguous 64-row blocks of the strided view (no copy is made).
//
// Work split inside a 256-thread workgroup: wave wv owns the 16 queries
// q0 + 16*wv .. +15 and, for each 64-key block, computes the transposed score block
// S^T[t][q] = K[t] . Q[q] with v_mfma_f32_16x16x32_bf16 (A operand = key rows,
// B operand = query rows).  Lane l then holds the scores of query q0+16*wv+l%16 for
// keys 16*ft + 4*(l/16) + v (ft, v in 0..3) -- every value of a lane belongs to one
// query, so softmax statistics stay per lane until a final 4-lane reduction.
//
// For P*V the contraction runs over keys.  The MFMA's k-slots are assigned so that
// lane group g = l/16 of a 32-key half h supplies keys 32h + {4g..4g+3, 16+4g..16+4g+3}:
// exactly the keys the lane already holds in registers.  The V^T operand is read from
// an LDS copy of the value block stored transposed, with the same key order.
#include "common.h"

namespace ollie {

namespace {

constexpr int kD = 64;        // head dimension
constexpr int kT = 64;        // queries per tile and keys per block
constexpr int kVtLd = kT + 4; // row stride (elements) of the transposed V block in LDS

struct Tile {
    int64_t b;      // batch index
    int rho;        // residue
    int64_t lr;     // length of the residue subsequence
    int64_t q0;     // first query (subsequence index) of the tile
};

__device__ __forceinline__ bool tile_of(const BandGeom& g, Tile& t) {
    t.b = blockIdx.z;
    t.rho = blockIdx.y;
    t.lr = (g.l - t.rho + g.dil - 1) / g.dil;
    t.q0 = (int64_t)blockIdx.x * kT;
    return t.q0 < t.lr;
}

// Global row (in [b][l]) of subsequence index tq.
__device__ __forceinline__ int64_t grow(const BandGeom& g, const Tile& t, int64_t tq) {
    return t.b * g.l + tq * g.dil + t.rho;
}

__device__ __forceinline__ int kswz(int row, int ch) { return row * 8 + (ch ^ (row & 7)); }

// Cooperative load of 64 key rows [t0, t0+64) into LDS (16-byte chunks, XOR swizzle);
// rows outside [0, lr) are zero.
__device__ __forceinline__ void load_k_block(const BandGeom& g, const Tile& t,
                                             const bf16_t* __restrict__ K, int64_t t0,
                                             u32x4* lk) {
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        int idx = threadIdx.x + e * 256;
        int row = idx >> 3, ch = idx & 7;
        int64_t tt = t0 + row;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (tt >= 0 && tt < t.lr)
            v = *reinterpret_cast<const u32x4*>(K + grow(g, t, tt) * kD + ch * 8);
        lk[kswz(row, ch)] = v;
    }
}

// Cooperative load of 64 value rows into LDS, transposed: vt[e][t].
__device__ __forceinline__ void load_vt_block(const BandGeom& g, const Tile& t,
                                              const bf16_t* __restrict__ V, int64_t t0,
                                              bf16_t* vt) {
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        int idx = threadIdx.x + e * 256;
        int row = idx >> 3, ch = idx & 7;
        int64_t tt = t0 + row;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (tt >= 0 && tt < t.lr)
            v = *reinterpret_cast<const u32x4*>(V + grow(g, t, tt) * kD + ch * 8);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            vt[(ch * 8 + 2 * i) * kVtLd + row] = (bf16_t)(v[i] & 0xffffu);
            vt[(ch * 8 + 2 * i + 1) * kVtLd + row] = (bf16_t)(v[i] >> 16);
        }
    }
}

// The wave's two Q fragments (d halves) for query q (zero outside [0, lr)).
__device__ __forceinline__ void load_q_frags(const BandGeom& g, const Tile& t,
                                             const bf16_t* __restrict__ Q, int64_t q,
                                             bf16x8 qf[2]) {
    const int grp = (threadIdx.x & 63) >> 4;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
        u32x4 v = {0u, 0u, 0u, 0u};
        if (q < t.lr) v = *reinterpret_cast<const u32x4*>(Q + grow(g, t, q) * kD + kk * 32 + grp * 8);
        qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
}

// s[ft] = S^T block for keys 16*ft + 4*grp + v of the LDS block and the lane's query.
__device__ __forceinline__ void score_block(const u32x4* lk, const bf16x8 qf[2], f32x4 s[4]) {
    const int lane = threadIdx.x & 63;
    const int grp = lane >> 4;
#pragma unroll
    for (int ft = 0; ft < 4; ++ft) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        const int row = ft * 16 + (lane & 15);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            bf16x8 kf = __builtin_bit_cast(bf16x8, lk[kswz(row, kk * 4 + grp)]);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[kk], acc, 0, 0, 0);
        }
        s[ft] = acc;
    }
}

// o[eb] += V^T[16*eb + l%16][keys] * P^T[keys][query]; p holds the lane's 16 probabilities
// (p[ft][v] for key 16*ft + 4*grp + v).
__device__ __forceinline__ void pv_block(const bf16_t* vt, const f32x4 p[4], f32x4 o[4]) {
    const int lane = threadIdx.x & 63;
    const int grp = lane >> 4;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        bf16_t pb[8];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            pb[v] = f2bf(p[2 * h][v]);
            pb[4 + v] = f2bf(p[2 * h + 1][v]);
        }
        bf16x8 pf = __builtin_bit_cast(bf16x8, pb);
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) {
            const bf16_t* row = vt + (eb * 16 + (lane & 15)) * kVtLd + h * 32 + 4 * grp;
            uint2 lo = *reinterpret_cast<const uint2*>(row);
            uint2 hi = *reinterpret_cast<const uint2*>(row + 16);
            u32x4 u = {lo.x, lo.y, hi.x, hi.y};
            o[eb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, u), pf,
                                                            o[eb], 0, 0, 0);
        }
    }
}

// --------------------------------------------------------------------- G2BMM
__global__ __launch_bounds__(256) void band_g2bmm_kernel(BandGeom g, const bf16_t* __restrict__ Q,
                                                        const bf16_t* __restrict__ K,
                                                        float* __restrict__ S) {
    __shared__ u32x4 lk[kT * 8];
    Tile t;
    if (!tile_of(g, t)) return;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, grp = lane >> 4;
    const int64_t q = t.q0 + wv * 16 + (lane & 15);
    const int64_t nb = 2 * g.w + 1;
    bf16x8 qf[2];
    load_q_frags(g, t, Q, q, qf);
    const int nblk = (int)((kT + 2 * g.w + kT - 1) / kT);
    float* srow = S + (q < t.lr ? grow(g, t, q) : 0) * nb;
    for (int kb = 0; kb < nblk; ++kb) {
        const int64_t t0 = t.q0 - g.w + (int64_t)kb * kT;
        __syncthreads();
        load_k_block(g, t, K, t0, lk);
        __syncthreads();
        f32x4 s[4];
        score_block(lk, qf, s);
        if (q >= t.lr) continue;
#pragma unroll
        for (int ft = 0; ft < 4; ++ft)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                int64_t j = t0 + ft * 16 + 4 * grp + v - q + g.w;
                if (j >= 0 && j < nb) srow[j] = g.scale * s[ft][v];
            }
    }
}

// ------------------------------------------------------------------- softmax
// One wavefront per row; NCH chunks of 64 band entries per lane held in registers.
template <int NCH>
__global__ __launch_bounds__(256) void band_softmax_kernel(BandGeom g, const float* __restrict__ S,
                                                          bf16_t* __restrict__ P, int mask) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= g.b * g.l) return;
    const int64_t i = row % g.l;
    const int nb = (int)(2 * g.w + 1);
    const float* s = S + row * nb;
    bf16_t* p = P + row * nb;
    float x[NCH];
    float m = -INFINITY;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        int j = lane + c * 64;
        float val = -INFINITY;
        if (j < nb) {
            val = s[j];
            if (mask) {
                int64_t tt = i + (int64_t)(j - g.w) * g.dil;
                if (tt < 0 || tt >= g.l) val = -INFINITY;
            }
        }
        x[c] = val;
        m = fmaxf(m, val);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        x[c] = __expf(x[c] - m);
        sum += x[c];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
    const float inv = 1.f / sum;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        int j = lane + c * 64;
        if (j < nb) p[j] = f2bf(x[c] * inv);
    }
}

// ---------------------------------------------------------------------- GBMM
template <typename OT>
__global__ __launch_bounds__(256) void band_gbmm_kernel(BandGeom g, const bf16_t* __restrict__ P,
                                                       const bf16_t* __restrict__ V,
                                                       OT* __restrict__ O) {
    __shared__ bf16_t vt[kD * kVtLd];
    Tile t;
    if (!tile_of(g, t)) return;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, grp = lane >> 4;
    const int64_t q = t.q0 + wv * 16 + (lane & 15);
    const int64_t nb = 2 * g.w + 1;
    const bf16_t* prow = P + (q < t.lr ? grow(g, t, q) : 0) * nb;
    const int nblk = (int)((kT + 2 * g.w + kT - 1) / kT);
    f32x4 o[4];
#pragma unroll
    for (int eb = 0; eb < 4; ++eb) o[eb] = (f32x4){0.f, 0.f, 0.f, 0.f};
    for (int kb = 0; kb < nblk; ++kb) {
        const int64_t t0 = t.q0 - g.w + (int64_t)kb * kT;
        __syncthreads();
        load_vt_block(g, t, V, t0, vt);
        __syncthreads();
        f32x4 p[4];
#pragma unroll
        for (int ft = 0; ft < 4; ++ft)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                int64_t j = t0 + ft * 16 + 4 * grp + v - q + g.w;
                p[ft][v] = (q < t.lr && j >= 0 && j < nb) ? bf2f(prow[j]) : 0.f;
            }
        pv_block(vt, p, o);
    }
    if (q >= t.lr) return;
    OT* orow = O + grow(g, t, q) * kD;
#pragma unroll
    for (int eb = 0; eb < 4; ++eb) Out<OT>::put4(orow + eb * 16 + 4 * grp, o[eb]);
}

// --------------------------------------------------------------------- fused
// G2BMM -> online softmax -> GBMM in one pass over the key blocks of the band;
// scores and probabilities stay in registers.
template <typename OT>
__global__ __launch_bounds__(256) void band_fused_kernel(BandGeom g, const bf16_t* __restrict__ Q,
                                                        const bf16_t* __restrict__ K,
                                                        const bf16_t* __restrict__ V,
                                                        OT* __restrict__ O, int mask) {
    __shared__ u32x4 lk[kT * 8];
    __shared__ bf16_t vt[kD * kVtLd];
    Tile t;
    if (!tile_of(g, t)) return;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, grp = lane >> 4;
    const int64_t q = t.q0 + wv * 16 + (lane & 15);
    const float sl2 = g.scale * 1.4426950408889634f;   // scale * log2(e)
    bf16x8 qf[2];
    load_q_frags(g, t, Q, q, qf);
    const int nblk = (int)((kT + 2 * g.w + kT - 1) / kT);
    f32x4 o[4];
#pragma unroll
    for (int eb = 0; eb < 4; ++eb) o[eb] = (f32x4){0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY;   // running max of the query's scores (log2 units)
    float l_run = 0.f;         // this lane's share of the running denominator
    for (int kb = 0; kb < nblk; ++kb) {
        const int64_t t0 = t.q0 - g.w + (int64_t)kb * kT;
        __syncthreads();
        load_k_block(g, t, K, t0, lk);
        load_vt_block(g, t, V, t0, vt);
        __syncthreads();
        f32x4 s[4];
        score_block(lk, qf, s);
        float mb = -INFINITY;
#pragma unroll
        for (int ft = 0; ft < 4; ++ft)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                int64_t tt = t0 + ft * 16 + 4 * grp + v;
                int64_t dj = tt - q;   // j - w
                bool live = dj >= -g.w && dj <= g.w && (!mask || (tt >= 0 && tt < t.lr));
                float x = live ? s[ft][v] * sl2 : -INFINITY;
                s[ft][v] = x;
                mb = fmaxf(mb, x);
            }
        mb = fmaxf(mb, __shfl_xor(mb, 16));
        mb = fmaxf(mb, __shfl_xor(mb, 32));
        const float m_new = fmaxf(m_run, mb);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float corr = exp2f(m_run - m_use);
        m_run = m_new;
        float ls = 0.f;
#pragma unroll
        for (int ft = 0; ft < 4; ++ft)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float pv = exp2f(s[ft][v] - m_use);
                s[ft][v] = pv;
                ls += pv;
            }
        l_run = l_run * corr + ls;
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) o[eb] *= corr;
        pv_block(vt, s, o);
    }
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
    if (q >= t.lr) return;
    const float inv = 1.f / l_run;
    OT* orow = O + grow(g, t, q) * kD;
#pragma unroll
    for (int eb = 0; eb < 4; ++eb) Out<OT>::put4(orow + eb * 16 + 4 * grp, o[eb] * inv);
}

dim3 tile_grid(const BandGeom& g) {
    int64_t l0 = (g.l + g.dil - 1) / g.dil;   // longest residue subsequence (rho = 0)
    return dim3((unsigned)((l0 + kT - 1) / kT), (unsigned)g.dil, (unsigned)g.b);
}

}  // namespace

hipError_t launch_band_g2bmm(const BandGeom& g, const void* q, const void* k, float* s,
                             hipStream_t stream) {
    hipLaunchKernelGGL(band_g2bmm_kernel, tile_grid(g), dim3(256), 0, stream, g,
                       (const bf16_t*)q, (const bf16_t*)k, s);
    return hipGetLastError();
}

hipError_t launch_band_softmax(const BandGeom& g, const float* s, void* p, int mask,
                               hipStream_t stream) {
    const int64_t nb = 2 * g.w + 1;
    const int nch = (int)((nb + 63) / 64);
    dim3 grid((unsigned)((g.b * g.l + 3) / 4));
#define OLLIE_SOFTMAX(N)                                                                     \
    hipLaunchKernelGGL(band_softmax_kernel<N>, grid, dim3(256), 0, stream, g, s, (bf16_t*)p, \
                       mask)
    if (nch <= 1) OLLIE_SOFTMAX(1);
    else if (nch <= 2) OLLIE_SOFTMAX(2);
    else if (nch <= 4) OLLIE_SOFTMAX(4);
    else if (nch <= 9) OLLIE_SOFTMAX(9);
    else if (nch <= 16) OLLIE_SOFTMAX(16);
    else return hipErrorInvalidValue;
#undef OLLIE_SOFTMAX
    return hipGetLastError();
}

hipError_t launch_band_gbmm(const BandGeom& g, const void* p, const void* v, void* o,
                            int o_bf16, hipStream_t stream) {
    if (o_bf16)
        hipLaunchKernelGGL(band_gbmm_kernel<bf16_t>, tile_grid(g), dim3(256), 0, stream, g,
                           (const bf16_t*)p, (const bf16_t*)v, (bf16_t*)o);
    else
        hipLaunchKernelGGL(band_gbmm_kernel<float>, tile_grid(g), dim3(256), 0, stream, g,
                           (const bf16_t*)p, (const bf16_t*)v, (float*)o);
    return hipGetLastError();
}

hipError_t launch_band_fused(const BandGeom& g, const void* q, const void* k, const void* v,
                             void* o, int o_bf16, int mask, hipStream_t stream) {
    if (o_bf16)
        hipLaunchKernelGGL(band_fused_kernel<bf16_t>, tile_grid(g), dim3(256), 0, stream, g,
                           (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, (bf16_t*)o,
                           mask);
    else
        hipLaunchKernelGGL(band_fused_kernel<float>, tile_grid(g), dim3(256), 0, stream, g,
                           (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, (float*)o,
                           mask);
    return hipGetLastError();
}

}  // namespace ollie
