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
// keys 16*ft + 4*(l/16) + v (ft, v in 0..3): every value of a lane belongs to one
// query, so softmax statistics stay per lane until a final 4-lane reduction.
//
// For P*V the contraction runs over keys.  The MFMA's k-slots are assigned so that
// lane group g = l/16 of a 32-key half h supplies keys 32h + {4g..4g+3, 16+4g..16+4g+3}:
// exactly the keys the lane already holds in registers.  The V^T operand comes from a
// row-major LDS copy of the value block through ds_read_b64_tr_b16, whose lane i of
// each 16-lane group receives element i%4 of the 8-byte rows addressed by lanes
// i/4 + 4j (j = 0..3): lanes address rows (keys) and 4-column slices, the hardware
// returns one column (value dimension) across four keys.
#include <stdlib.h>

#include <type_traits>

#include "common.h"

namespace ollie {

namespace {

constexpr int kD = 64;        // head dimension
constexpr int kT = 64;        // queries per tile and keys per block
constexpr int kVLd = kD + 8;  // row stride (elements) of the value block in LDS

typedef short s16x4 __attribute__((ext_vector_type(4)));

struct Tile {
    int b;      // batch index
    int rho;    // residue
    int lr;     // length of the residue subsequence
    int q0;     // first query (subsequence index) of the tile
};

// Tiles are numbered (tile, residue, batch) with the tile fastest.  Workgroup ids are
// dealt round-robin to the 8 XCDs; remap them so each XCD owns a contiguous run of
// tiles of the same sequences, whose key/value blocks then stay in that XCD's L2.
__device__ __forceinline__ bool tile_of(const BandGeom& g, int ntx, Tile& t) {
    const int nblk = gridDim.x;
    const int bid = blockIdx.x;
    const int id = (nblk & 7) == 0 ? (bid & 7) * (nblk >> 3) + (bid >> 3) : bid;
    t.q0 = (id % ntx) * kT;
    const int r = id / ntx;
    t.rho = r % g.dil;
    t.b = r / g.dil;
    t.lr = ((int)g.l - t.rho + g.dil - 1) / g.dil;
    return t.q0 < t.lr;
}

// Row (in [b][l]) of element tq of the tile's subsequence, and its element offset in a
// [b][l][64] tensor.
__device__ __forceinline__ int64_t row_index(const BandGeom& g, const Tile& t, int tq) {
    return (int64_t)t.b * g.l + (int64_t)tq * g.dil + t.rho;
}
__device__ __forceinline__ int64_t row_off(const BandGeom& g, const Tile& t, int tq) {
    return row_index(g, t, tq) * kD;
}

__device__ __forceinline__ int kswz(int row, int ch) { return row * 8 + (ch ^ (row & 7)); }

// Register staging of one 64-row block of K (and V): 2 x 16 bytes per thread each.
struct KVRegs {
    u32x4 k[2];
    u32x4 v[2];
};

template <bool WITH_K, bool WITH_V>
__device__ __forceinline__ void gload_block(const BandGeom& g, const Tile& t,
                                            const bf16_t* __restrict__ K,
                                            const bf16_t* __restrict__ V, int t0, KVRegs& r) {
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const int idx = threadIdx.x + e * 256;
        const int row = idx >> 3, ch = idx & 7;
        const int tt = t0 + row;
        u32x4 kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
        if (tt >= 0 && tt < t.lr) {
            const int64_t off = row_off(g, t, tt) + ch * 8;
            if (WITH_K) kv = *reinterpret_cast<const u32x4*>(K + off);
            if (WITH_V) vv = *reinterpret_cast<const u32x4*>(V + off);
        }
        r.k[e] = kv;
        r.v[e] = vv;
    }
}

// K block: 16-byte chunks with an XOR swizzle (conflict-free ds_read_b128 fragments).
// V block: plain rows padded to kVLd elements (read through the transposing load).
template <bool WITH_K, bool WITH_V>
__device__ __forceinline__ void lstore_block(const KVRegs& r, u32x4* lk, bf16_t* lv) {
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const int idx = threadIdx.x + e * 256;
        const int row = idx >> 3, ch = idx & 7;
        if (WITH_K) lk[kswz(row, ch)] = r.k[e];
        if (WITH_V) *reinterpret_cast<u32x4*>(lv + row * kVLd + ch * 8) = r.v[e];
    }
}

// The lane's two Q fragments (d halves) for query q (zero outside [0, lr)).
__device__ __forceinline__ void load_q_frags(const BandGeom& g, const Tile& t,
                                             const bf16_t* __restrict__ Q, int q,
                                             bf16x8 qf[2]) {
    const int grp = (threadIdx.x & 63) >> 4;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
        u32x4 v = {0u, 0u, 0u, 0u};
        if (q < t.lr)
            v = *reinterpret_cast<const u32x4*>(Q + row_off(g, t, q) + kk * 32 + grp * 8);
        qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
}

// s[ft][v] = K[16*ft + 4*grp + v] . Q[query of the lane] over the LDS key block.
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

__device__ __forceinline__ s16x4 tr_read(const bf16_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(p));
}

// o[eb] (rows e = 16*eb + 4*grp + v, column = the lane's query) += V^T * P^T over the
// block's 64 keys; p[ft][v] is the lane's probability for key 16*ft + 4*grp + v.
__device__ __forceinline__ void pv_block(const bf16_t* lv, const f32x4 p[4], f32x4 o[4]) {
    const int lane = threadIdx.x & 63;
    const int grp = lane >> 4;
    const int li = lane & 15;
    const int col = 4 * (li & 3);      // this lane addresses a 4-column slice ...
    const int krow = li >> 2;          // ... of key row 32h + 4*grp + krow (+16)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        bf16x8 pf;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            pf[v] = (__bf16)p[2 * h][v];
            pf[4 + v] = (__bf16)p[2 * h + 1][v];
        }
        const bf16_t* base = lv + (32 * h + 4 * grp + krow) * kVLd + col;
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) {
            s16x4 lo = tr_read(base + eb * 16);
            s16x4 hi = tr_read(base + 16 * kVLd + eb * 16);
            s16x4 both[2] = {lo, hi};
            bf16x8 vf = __builtin_bit_cast(bf16x8, both);
            o[eb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o[eb], 0, 0, 0);
        }
    }
}

__device__ __forceinline__ int n_key_blocks(const BandGeom& g) {
    return (kT + 2 * (int)g.w + kT - 1) / kT;
}

// --------------------------------------------------------------------- G2BMM
__global__ __launch_bounds__(256) void band_g2bmm_kernel(BandGeom g, int ntx,
                                                        const bf16_t* __restrict__ Q,
                                                        const bf16_t* __restrict__ K,
                                                        float* __restrict__ S) {
    __shared__ u32x4 lk[kT * 8];
    Tile t;
    if (!tile_of(g, ntx, t)) return;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, grp = lane >> 4;
    const int q = t.q0 + wv * 16 + (lane & 15);
    const int w = (int)g.w, nb = 2 * w + 1;
    bf16x8 qf[2];
    load_q_frags(g, t, Q, q, qf);
    const int nblk = n_key_blocks(g);
    float* srow = S + (q < t.lr ? row_index(g, t, q) : 0) * nb;
    KVRegs r;
    for (int kb = 0; kb < nblk; ++kb) {
        const int t0 = t.q0 - w + kb * kT;
        gload_block<true, false>(g, t, K, nullptr, t0, r);
        __syncthreads();
        lstore_block<true, false>(r, lk, nullptr);
        __syncthreads();
        f32x4 s[4];
        score_block(lk, qf, s);
        if (q >= t.lr) continue;
#pragma unroll
        for (int ft = 0; ft < 4; ++ft)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int j = t0 + ft * 16 + 4 * grp + v - q + w;
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
    const int i = (int)(row % g.l);
    const int w = (int)g.w, nb = 2 * w + 1, L = (int)g.l;
    const float* s = S + row * nb;
    bf16_t* p = P + row * nb;
    float x[NCH];
    float m = -INFINITY;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int j = lane + c * 64;
        float val = -INFINITY;
        if (j < nb) {
            val = s[j];
            if (mask) {
                const int64_t tt = (int64_t)i + (int64_t)(j - w) * g.dil;
                if (tt < 0 || tt >= L) val = -INFINITY;
            }
        }
        x[c] = val;
        m = fmaxf(m, val);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    const float ml2 = m * 1.4426950408889634f;
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        x[c] = __builtin_amdgcn_exp2f(x[c] * 1.4426950408889634f - ml2);
        sum += x[c];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
    const float inv = 1.f / sum;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int j = lane + c * 64;
        if (j < nb) p[j] = f2bf(x[c] * inv);
    }
}

// ---------------------------------------------------------------------- GBMM
template <typename OT>
__global__ __launch_bounds__(256) void band_gbmm_kernel(BandGeom g, int ntx,
                                                       const bf16_t* __restrict__ P,
                                                       const bf16_t* __restrict__ V,
                                                       OT* __restrict__ O) {
    __shared__ __attribute__((aligned(16))) bf16_t lv[kT * kVLd];
    Tile t;
    if (!tile_of(g, ntx, t)) return;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, grp = lane >> 4;
    const int q = t.q0 + wv * 16 + (lane & 15);
    const int w = (int)g.w, nb = 2 * w + 1;
    const bf16_t* prow = P + (q < t.lr ? row_index(g, t, q) : 0) * nb;
    const int nblk = n_key_blocks(g);
    f32x4 o[4];
#pragma unroll
    for (int eb = 0; eb < 4; ++eb) o[eb] = (f32x4){0.f, 0.f, 0.f, 0.f};
    KVRegs r;
    for (int kb = 0; kb < nblk; ++kb) {
        const int t0 = t.q0 - w + kb * kT;
        gload_block<false, true>(g, t, nullptr, V, t0, r);
        __syncthreads();
        lstore_block<false, true>(r, nullptr, lv);
        __syncthreads();
        f32x4 p[4];
#pragma unroll
        for (int ft = 0; ft < 4; ++ft)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int j = t0 + ft * 16 + 4 * grp + v - q + w;
                p[ft][v] = (q < t.lr && j >= 0 && j < nb) ? bf2f(prow[j]) : 0.f;
            }
        pv_block(lv, p, o);
    }
    if (q >= t.lr) return;
    OT* orow = O + row_off(g, t, q);
#pragma unroll
    for (int eb = 0; eb < 4; ++eb) Out<OT>::put4(orow + eb * 16 + 4 * grp, o[eb]);
}

// --------------------------------------------------------------------- fused
// G2BMM -> online softmax -> GBMM in one pass over the key blocks of the band; scores
// and probabilities stay in registers, K/V blocks are double-buffered in LDS (the next
// block's global loads are in flight while the current one is computed).
//
// Each wave owns QH 16-query groups; with QH = 2 every K and V fragment read from LDS
// feeds two MFMAs (at the cost of occupancy).  Softmax bookkeeping per query, in log2 units
// (x = scale*log2(e)*score): a running reference m, and the denominator and O both
// accumulated unnormalised by MFMA -- the denominator as the product of an all-ones
// operand with the same bf16 probabilities that multiply V, so O and its normaliser
// see identical rounding.  m is raised only when a block's maximum exceeds it by more
// than kLazy, so most blocks need no rescaling and every exp2 argument stays <= kLazy.
// The scale enters as one FMA per score; a negative scale is handled by negating the
// query fragments (an exact sign flip of bf16) and using |scale|.
template <typename OT, bool MASK, int QH>
__global__ __launch_bounds__(256, QH == 1 ? 4 : 2) void band_fused_kernel(BandGeom g, int ntx,
                                                        const bf16_t* __restrict__ Q,
                                                        const bf16_t* __restrict__ K,
                                                        const bf16_t* __restrict__ V,
                                                        OT* __restrict__ O) {
    constexpr float kLazy = 8.f;
    constexpr int kQPW = 16 * QH;        // queries per wave
    constexpr int kFT = kQPW * 4;        // queries per tile (4 waves)
    __shared__ u32x4 lk[2][kT * 8];
    __shared__ __attribute__((aligned(16))) bf16_t lv[2][kT * kVLd];
    // tile geometry (kFT queries per tile)
    Tile t;
    {
        const int nblk_all = gridDim.x;
        const int bid = blockIdx.x;
        const int id = (nblk_all & 7) == 0 ? (bid & 7) * (nblk_all >> 3) + (bid >> 3) : bid;
        t.q0 = (id % ntx) * kFT;
        const int r = id / ntx;
        t.rho = r % g.dil;
        t.b = r / g.dil;
        t.lr = ((int)g.l - t.rho + g.dil - 1) / g.dil;
        if (t.q0 >= t.lr) return;
    }
    // the wave index through readfirstlane: every per-wave block test below is then a
    // scalar branch rather than an exec-masked one
    const int lane = threadIdx.x & 63, grp = lane >> 4;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int w = (int)g.w;
    const int qa = t.q0 + wv * kQPW;      // the wave's first query
    // byte addresses of the lanes 16 and 32 apart, for the 4-lane row reductions
    const int xor16 = (lane ^ 16) << 2, xor32 = (lane ^ 32) << 2;
    const float sl2 = fabsf(g.scale) * 1.4426950408889634f;
    const uint32_t qflip = g.scale < 0.f ? 0x80008000u : 0u;

    bf16x8 qf[QH][2];
#pragma unroll
    for (int hq = 0; hq < QH; ++hq) {
        const int q = qa + hq * 16 + (lane & 15);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if (q < t.lr)
                v = *reinterpret_cast<const u32x4*>(Q + row_off(g, t, q) + kk * 32 + grp * 8);
            v ^= (u32x4){qflip, qflip, qflip, qflip};
            qf[hq][kk] = __builtin_bit_cast(bf16x8, v);
        }
    }
    const int span = kFT + 2 * w;
    const int nblk = (span + kT - 1) / kT;

    f32x4 o[QH][4], lsum[QH];
#pragma unroll
    for (int hq = 0; hq < QH; ++hq) {
        lsum[hq] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) o[hq][eb] = (f32x4){0.f, 0.f, 0.f, 0.f};
    }
    float m_run[QH];
#pragma unroll
    for (int hq = 0; hq < QH; ++hq) m_run[hq] = -INFINITY;
    const bf16x8 ones = __builtin_bit_cast(bf16x8, (u32x4){0x3f803f80u, 0x3f803f80u,
                                                          0x3f803f80u, 0x3f803f80u});

    // this thread's two 16-byte chunks of every K/V block: rows r0 and r0 + 32
    const int r0 = threadIdx.x >> 3, ch = threadIdx.x & 7;
    const int64_t row_step = (int64_t)kT * g.dil * kD;          // 64 subsequence rows
    const int64_t half_step = (int64_t)32 * g.dil * kD;
    int tt0 = t.q0 - w + r0;                                     // subsequence row of chunk 0
    int64_t off0 = ((int64_t)t.b * g.l + t.rho) * kD + (int64_t)tt0 * g.dil * kD + ch * 8;
    KVRegs r;
    int blk0 = t.q0 - w;                                         // first key of the next block
    auto gload = [&]() {
        if (blk0 >= 0 && blk0 + kT <= t.lr) {                    // whole block in range
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                r.k[e] = *reinterpret_cast<const u32x4*>(K + off0 + e * half_step);
                r.v[e] = *reinterpret_cast<const u32x4*>(V + off0 + e * half_step);
            }
        } else {
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const int tt = tt0 + 32 * e;
                u32x4 kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
                if (tt >= 0 && tt < t.lr) {
                    kv = *reinterpret_cast<const u32x4*>(K + off0 + e * half_step);
                    vv = *reinterpret_cast<const u32x4*>(V + off0 + e * half_step);
                }
                r.k[e] = kv;
                r.v[e] = vv;
            }
        }
        tt0 += kT;
        off0 += row_step;
        blk0 += kT;
    };
    gload();
    lstore_block<true, true>(r, lk[0], lv[0]);
    __syncthreads();

    for (int kb = 0; kb < nblk; ++kb) {
        const int cur = kb & 1;
        const int t0 = t.q0 - w + kb * kT;
        if (kb + 1 < nblk) gload();
        const bool any = t0 + kT - 1 >= qa - w && t0 <= qa + kQPW - 1 + w;
        if (any) {
            // per query half: does the block meet its band, and is it entirely inside?
            f32x4 s[QH][4];
            const u32x4* lkc = lk[cur];
            bf16x8 kf[4][2];          // all key fragments first, then the MFMAs
#pragma unroll
            for (int ft = 0; ft < 4; ++ft) {
                const int row = ft * 16 + (lane & 15);
                kf[ft][0] = __builtin_bit_cast(bf16x8, lkc[kswz(row, grp)]);
                kf[ft][1] = __builtin_bit_cast(bf16x8, lkc[kswz(row, 4 + grp)]);
            }
#pragma unroll
            for (int ft = 0; ft < 4; ++ft)
#pragma unroll
                for (int hq = 0; hq < QH; ++hq) {
                    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[ft][0], qf[hq][0], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[ft][1], qf[hq][1], acc, 0, 0, 0);
                    s[hq][ft] = acc;
                }
            bf16x8 pf[QH][2];
            // Softmax of one 16-query half: block max (4-lane reduction), lazy rescale,
            // then p = exp2(score * scale * log2(e) - m) packed to bf16.  Full blocks and
            // masked blocks run separate copies, so no mask arithmetic reaches full blocks.
            auto soft = [&](int hq, auto masked) {
                constexpr bool M = decltype(masked)::value;
                const int q = qa + hq * 16 + (lane & 15);
                float mb = -INFINITY;
#pragma unroll
                for (int ft = 0; ft < 4; ++ft)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        if constexpr (M) {
                            const int tt = t0 + ft * 16 + 4 * grp + v;
                            const int dj = tt - q;
                            bool l = dj >= -w && dj <= w;
                            if (MASK) l = l && tt >= 0 && tt < t.lr;
                            if (!l) s[hq][ft][v] = -INFINITY;
                        }
                        mb = fmaxf(mb, s[hq][ft][v]);
                    }
                mb = fmaxf(mb, __int_as_float(__builtin_amdgcn_ds_bpermute(xor16, __float_as_int(mb))));
                mb = fmaxf(mb, __int_as_float(__builtin_amdgcn_ds_bpermute(xor32, __float_as_int(mb))));
                const float mbx = mb * sl2;               // block max in log2 units
                const bool need = mbx > m_run[hq] + kLazy;
                if (__any(need)) {
                    const float m_new = need ? mbx : m_run[hq];
                    const float corr = __builtin_amdgcn_exp2f(m_run[hq] - m_new);
                    lsum[hq] *= corr;
#pragma unroll
                    for (int eb = 0; eb < 4; ++eb) o[hq][eb] *= corr;
                    m_run[hq] = m_new;
                }
                const float nm = m_run[hq] == -INFINITY ? 0.f : -m_run[hq];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    bf16x8 pv;
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[hq][2 * h][v], sl2, nm));
                        float p1 =
                            __builtin_amdgcn_exp2f(__builtin_fmaf(s[hq][2 * h + 1][v], sl2, nm));
                        if constexpr (M) {   // -inf * 0 (scale 0) must still give p = 0
                            p0 = s[hq][2 * h][v] == -INFINITY ? 0.f : p0;
                            p1 = s[hq][2 * h + 1][v] == -INFINITY ? 0.f : p1;
                        }
                        pv[v] = (__bf16)p0;
                        pv[4 + v] = (__bf16)p1;
                    }
                    pf[hq][h] = pv;
                }
            };
#pragma unroll
            for (int hq = 0; hq < QH; ++hq) {
                const int qh = qa + hq * 16;              // first query of this half
                bool full = t0 - (qh + 15) >= -w && t0 + kT - 1 - qh <= w;
                if (MASK) full = full && t0 >= 0 && t0 + kT <= t.lr;
                if (full) soft(hq, std::false_type{});
                else soft(hq, std::true_type{});
            }
            // O^T += V^T P^T and the denominator += 1^T P^T, over the block's keys
            const int li = lane & 15;
            const bf16_t* base = lv[cur] + (4 * grp + (li >> 2)) * kVLd + 4 * (li & 3);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
#pragma unroll
                for (int eb = 0; eb < 4; ++eb) {
                    const bf16_t* p = base + 32 * h * kVLd + eb * 16;
                    s16x4 both[2] = {tr_read(p), tr_read(p + 16 * kVLd)};
                    const bf16x8 vf = __builtin_bit_cast(bf16x8, both);
#pragma unroll
                    for (int hq = 0; hq < QH; ++hq)
                        o[hq][eb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[hq][h],
                                                                            o[hq][eb], 0, 0, 0);
                }
#pragma unroll
                for (int hq = 0; hq < QH; ++hq)
                    lsum[hq] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[hq][h],
                                                                       lsum[hq], 0, 0, 0);
            }
        }
        if (kb + 1 < nblk) lstore_block<true, true>(r, lk[cur ^ 1], lv[cur ^ 1]);
        __syncthreads();
    }
#pragma unroll
    for (int hq = 0; hq < QH; ++hq) {
        const int q = qa + hq * 16 + (lane & 15);
        if (q >= t.lr) continue;
        const float inv = 1.f / lsum[hq][0];
        OT* orow = O + row_off(g, t, q);
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) Out<OT>::put4(orow + eb * 16 + 4 * grp, o[hq][eb] * inv);
    }
}

struct Grid {
    dim3 grid;
    int ntx;
};

Grid tile_grid(const BandGeom& g) {
    const int64_t l0 = (g.l + g.dil - 1) / g.dil;   // longest residue subsequence (rho = 0)
    const int ntx = (int)((l0 + kT - 1) / kT);
    return {dim3((unsigned)(ntx * g.dil * g.b)), ntx};
}

}  // namespace

hipError_t launch_band_g2bmm(const BandGeom& g, const void* q, const void* k, float* s,
                             hipStream_t stream) {
    Grid gr = tile_grid(g);
    hipLaunchKernelGGL(band_g2bmm_kernel, gr.grid, dim3(256), 0, stream, g, gr.ntx,
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
    Grid gr = tile_grid(g);
    if (o_bf16)
        hipLaunchKernelGGL(band_gbmm_kernel<bf16_t>, gr.grid, dim3(256), 0, stream, g, gr.ntx,
                           (const bf16_t*)p, (const bf16_t*)v, (bf16_t*)o);
    else
        hipLaunchKernelGGL(band_gbmm_kernel<float>, gr.grid, dim3(256), 0, stream, g, gr.ntx,
                           (const bf16_t*)p, (const bf16_t*)v, (float*)o);
    return hipGetLastError();
}

hipError_t launch_band_fused(const BandGeom& g, const void* q, const void* k, const void* v,
                             void* o, int o_bf16, int mask, hipStream_t stream) {
    // OLLIE_BAND_QH (1 or 2) overrides the queries-per-wave choice, for tuning sweeps
    static const int qh_env = [] {
        const char* e = getenv("OLLIE_BAND_QH");
        return e ? atoi(e) : 0;
    }();
    const int qh = qh_env == 2 ? 2 : 1;
    const int64_t l0 = (g.l + g.dil - 1) / g.dil;
    const int ntx = (int)((l0 + 64 * qh - 1) / (64 * qh));
    const dim3 grid((unsigned)(ntx * g.dil * g.b));
#define OLLIE_FUSED(OT, M, QH)                                                                \
    hipLaunchKernelGGL((band_fused_kernel<OT, M, QH>), grid, dim3(256), 0, stream, g, ntx,     \
                       (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, (OT*)o)
#define OLLIE_FUSED_QH(OT, M) \
    do { if (qh == 2) OLLIE_FUSED(OT, M, 2); else OLLIE_FUSED(OT, M, 1); } while (0)
    if (o_bf16) {
        if (mask) OLLIE_FUSED_QH(bf16_t, true);
        else OLLIE_FUSED_QH(bf16_t, false);
    } else {
        if (mask) OLLIE_FUSED_QH(float, true);
        else OLLIE_FUSED_QH(float, false);
    }
#undef OLLIE_FUSED_QH
#undef OLLIE_FUSED
    return hipGetLastError();
}

}  // namespace ollie
