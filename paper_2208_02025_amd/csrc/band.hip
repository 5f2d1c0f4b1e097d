// Banded dilated batched matmul: G2BMM (Table 2 iterator groups: bm in all tensors,
// w in weight+output, k in input+weight), row softmax, and the band-times-dense
// product, for head dimension 64.
//
// Dilation removal (section 6.4): with row i = dil*i' + rho the key of band entry j is
//   t = i + (j - w)*dil = dil*(i' + j - w) + rho,
// a NON-dilated band t' = i' + j - w on the residue-rho subsequence.  Every kernel
// works on one (batch, residue, query tile) of that subsequence (64 or 128 queries),
// so keys and values are read as contiguous 64-row blocks of the strided view (no copy
// is made).
//
// Work split: a wave owns one or more groups of 16 consecutive queries q0' .. q0' + 15
// and, for each 64-key block, computes the transposed score block
// S^T[t][q] = K[t] . Q[q] with v_mfma_f32_16x16x32_bf16 (A operand = key rows,
// B operand = query rows).  Lane l then holds the scores of query q0' + l%16 for
// keys 16*ft + 4*(l/16) + v (ft, v in 0..3): every value of a lane belongs to one
// query, so softmax statistics stay per lane until a final 4-lane reduction.
//
// For P*V the contraction runs over keys.  The MFMA's k-slots are assigned so that
// lane group g = l/16 of a 32-key half h supplies keys 32h + {4g..4g+3, 16+4g..16+4g+3}:
// in the fused kernel exactly the keys the lane already holds in registers (the staged
// GBMM takes the same entries from its P rows).  The V^T operand comes from a
// row-major LDS copy of the value block through ds_read_b64_tr_b16, whose lane i of
// each 16-lane group receives element i%4 of the 8-byte rows addressed by lanes
// i/4 + 4j (j = 0..3): lanes address rows (keys) and 4-column slices, the hardware
// returns one column (value dimension) across four keys.
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
template <int FT = kT>   // queries per tile
__device__ __forceinline__ bool tile_of(const BandGeom& g, int ntx, Tile& t) {
    const int nblk = gridDim.x;
    const int bid = blockIdx.x;
    const int id = (nblk & 7) == 0 ? (bid & 7) * (nblk >> 3) + (bid >> 3) : bid;
    t.q0 = (id % ntx) * FT;
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

// Register staging of one 64-row block of K (and V), 512 16-byte chunks each: 2 per
// thread of a 256-thread workgroup (NT = 256), 1 per thread of a 512-thread one.
struct KVRegs {
    u32x4 k[2];
    u32x4 v[2];
};

template <bool WITH_K, bool WITH_V, int NT = 256>
__device__ __forceinline__ void gload_block(const BandGeom& g, const Tile& t,
                                            const bf16_t* __restrict__ K,
                                            const bf16_t* __restrict__ V, int t0, KVRegs& r) {
    static_assert(NT == 256 || NT == 512, "workgroup size");
#pragma unroll
    for (int e = 0; e < 512 / NT; ++e) {
        const int idx = threadIdx.x + e * NT;
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
template <bool WITH_K, bool WITH_V, int NT = 256>
__device__ __forceinline__ void lstore_block(const KVRegs& r, u32x4* lk, bf16_t* lv) {
#pragma unroll
    for (int e = 0; e < 512 / NT; ++e) {
        const int idx = threadIdx.x + e * NT;
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

template <int FT = kT>   // key blocks that meet the band of a tile of FT queries
__device__ __forceinline__ int n_key_blocks(const BandGeom& g) {
    return (FT + 2 * (int)g.w + kT - 1) / kT;
}

// Ordering of one wave's accesses to its own LDS patch: a wave's LDS instructions
// complete in issue order, so the compiler only has to keep them in program order.
__device__ __forceinline__ void wave_lds_order() {
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
}

// --------------------------------------------------------------------- G2BMM
// Each wave owns 16 queries.  For one query a key block's 64 scores are 64 consecutive
// band entries j = key - query + w of its S row, i.e. one run [a, a + 64) of S (a row
// base plus the block's first j); runs of different rows start at any 4-byte offset.
// The scores pass through a per-wave LDS patch so that S is written in aligned 16-byte
// chunks: at a block the wave stores the 16 chunks of each row starting at a rounded
// down to a multiple of 4.  The first chunk's entries below a came from the previous
// block (kept in the patch's 4-entry carry), the entries above the last chunk leave
// with the next block (or the final flush).  Chunks that reach past a row's ends
// [0, 2w] are stored entry by entry, the rest as one 16-byte store each: every
// instruction writes four 256-byte runs.
constexpr int kSLd = kT + 4;   // patch row: 4 carried scores, then the block's 64
template <int NW>   // waves per workgroup: a tile of 16*NW queries
__global__ __launch_bounds__(64 * NW) void band_g2bmm_kernel(BandGeom g, int ntx,
                                                            const bf16_t* __restrict__ Q,
                                                            const bf16_t* __restrict__ K,
                                                            float* __restrict__ S) {
    constexpr int NT = 64 * NW, FT = 16 * NW;
    __shared__ u32x4 lk[kT * 8];
    __shared__ __attribute__((aligned(16))) float ls[NW][16 * kSLd];
    Tile t;
    if (!tile_of<FT>(g, ntx, t)) return;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, grp = lane >> 4;
    const int qw = t.q0 + wv * 16;                  // the wave's first query
    const int w = (int)g.w, nb = 2 * w + 1;
    bf16x8 qf[2];
    load_q_frags(g, t, Q, qw + (lane & 15), qf);
    const int nblk = n_key_blocks<FT>(g);
    float* patch = ls[wv];
    // chunk-store slots: instruction n, lane -> row rr = 4n + lane/16, chunk c = lane%16
    const int cc = lane & 15;
    int64_t rbase[4];                               // S offset of row rr (-1: no row)
#pragma unroll
    for (int n = 0; n < 4; ++n) {
        const int qq = qw + 4 * n + (lane >> 4);
        rbase[n] = qq < t.lr ? row_index(g, t, qq) * nb : -1;
    }
    KVRegs r;
    gload_block<true, false, NT>(g, t, K, nullptr, t.q0 - w, r);
    for (int kb = 0; kb < nblk; ++kb) {
        const int t0 = t.q0 - w + kb * kT;
        __syncthreads();
        lstore_block<true, false, NT>(r, lk, nullptr);
        __syncthreads();
        // the next key block's loads overlap this block's scores and stores
        if (kb + 1 < nblk) gload_block<true, false, NT>(g, t, K, nullptr, t0 + kT, r);
        f32x4 s[4];
        score_block(lk, qf, s);
#pragma unroll
        for (int ft = 0; ft < 4; ++ft)   // query lane%16, keys 16ft + 4grp .. +3
            *reinterpret_cast<f32x4*>(patch + (lane & 15) * kSLd + 4 + ft * 16 + 4 * grp) =
                s[ft] * g.scale;
        wave_lds_order();
#pragma unroll
        for (int n = 0; n < 4; ++n) {
            if (rbase[n] < 0) continue;
            const int rr = 4 * n + (lane >> 4);
            const int js = t0 - (qw + rr) + w;      // j of the block's first key
            const int64_t a = rbase[n] + js;
            const int64_t x0 = (a & ~int64_t(3)) + 4 * cc;
            const int j0 = (int)(x0 - rbase[n]);
            const float* src = patch + rr * kSLd + 4 + (int)(x0 - a);
            if (j0 >= 0 && j0 + 3 < nb) {
                const f32x4 v = {src[0], src[1], src[2], src[3]};
                *reinterpret_cast<f32x4*>(S + x0) = v;
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (j0 + e >= 0 && j0 + e < nb) S[x0 + e] = src[e];
            }
        }
        wave_lds_order();
        // carry: the block's last 4 scores of each row (lane -> row lane/4, entry lane%4)
        patch[(lane >> 2) * kSLd + (lane & 3)] = patch[(lane >> 2) * kSLd + kT + (lane & 3)];
        wave_lds_order();
    }
    // flush: the entries of the last block above its last stored chunk (lane -> row
    // lane/4, entry lane%4 of the chunk after it)
    const int rr = lane >> 2;
    const int qq = qw + rr;
    if (qq < t.lr) {
        const int64_t rb = row_index(g, t, qq) * nb;
        const int js = t.q0 - w + (nblk - 1) * kT - qq + w;
        const int64_t a = rb + js;
        const int64_t x = (a & ~int64_t(3)) + kT + (lane & 3);
        const int j = (int)(x - rb);
        if (x < a + kT && j >= 0 && j < nb) S[x] = patch[rr * kSLd + 4 + (int)(x - a)];
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
// The probabilities of a block come in the way the G2BMM's scores leave: for one query
// the block's 64 keys are the run [a, a + 64) of its P row, fetched as aligned 16-byte
// chunks (8 entries) into a per-wave LDS patch.  Slot 0 of a patch row holds the chunk
// containing a (the previous block's last chunk, carried), slots 1..8 the next eight
// chunks, loaded for this block during the previous one: every load instruction reads
// eight 128-byte runs.  Entries outside the row [0, 2w] enter the patch as zeros.  A
// lane then takes its MFMA operand, the four entries at a + 32h + 16f + 4grp .. +3, from
// three patch dwords shifted by 0 or 16 bits.
constexpr int kPSlots = 9;   // 16-byte slots per patch row

// Entries [x0, x0 + 8) of the P row based at rb (zero outside [0, nb)).
__device__ __forceinline__ u32x4 load_p_chunk(const bf16_t* __restrict__ P, int64_t rb,
                                              int64_t x0, int nb) {
    const int j0 = (int)(x0 - rb);
    if (j0 >= 0 && j0 + 7 < nb) return *reinterpret_cast<const u32x4*>(P + x0);
    uint32_t e[8];
#pragma unroll
    for (int v = 0; v < 8; ++v) e[v] = (j0 + v >= 0 && j0 + v < nb) ? (uint32_t)P[x0 + v] : 0u;
    return (u32x4){e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                   e[6] | (e[7] << 16)};
}

template <typename OT, int NW>   // NW waves per workgroup: a tile of 16*NW queries
__global__ __launch_bounds__(64 * NW) void band_gbmm_kernel(BandGeom g, int ntx,
                                                           const bf16_t* __restrict__ P,
                                                           const bf16_t* __restrict__ V,
                                                           OT* __restrict__ O) {
    constexpr int NT = 64 * NW, FT = 16 * NW;
    constexpr int kRows = 16;                       // P rows (queries) per wave
    constexpr int kLoads = kRows * 8 / 64;          // chunk loads per lane per block
    __shared__ __attribute__((aligned(16))) bf16_t lv[kT * kVLd];
    __shared__ u32x4 lp[NW][kRows * kPSlots];
    Tile t;
    if (!tile_of<FT>(g, ntx, t)) return;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, grp = lane >> 4, li = lane & 15;
    const int qw = t.q0 + wv * kRows;
    const int w = (int)g.w, nb = 2 * w + 1;
    const int nblk = n_key_blocks<FT>(g);
    u32x4* patch = lp[wv];
    // chunk-load slots: instruction n, lane -> row rr = 8n + lane/8, chunk c = lane%8
    const int cc = lane & 7;
    int64_t rbase[kLoads];                          // P offset of row rr (-1: no row)
#pragma unroll
    for (int n = 0; n < kLoads; ++n) {
        const int qq = qw + 8 * n + (lane >> 3);
        rbase[n] = qq < t.lr ? row_index(g, t, qq) * nb : -1;
    }
    // aligned start of block kb's run for slot row rr (the chunk in slot 0)
    auto chunk0 = [&](int n, int kb) -> int64_t {
        const int rr = 8 * n + (lane >> 3);
        const int js = t.q0 - w + kb * kT - (qw + rr) + w;
        return (rbase[n] + js) & ~int64_t(7);
    };
    // slots 1..8 of block kb
    auto load_p = [&](int kb, u32x4 (&pc)[kLoads]) {
#pragma unroll
        for (int n = 0; n < kLoads; ++n)
            pc[n] = rbase[n] < 0 ? (u32x4){0u, 0u, 0u, 0u}
                                 : load_p_chunk(P, rbase[n], chunk0(n, kb) + 8 + 8 * cc, nb);
    };
    // slot 0 of block 0 (lanes with chunk index 0 of each row)
    if (cc == 0) {
#pragma unroll
        for (int n = 0; n < kLoads; ++n)
            patch[(8 * n + (lane >> 3)) * kPSlots] =
                rbase[n] < 0 ? (u32x4){0u, 0u, 0u, 0u}
                             : load_p_chunk(P, rbase[n], chunk0(n, 0), nb);
    }
    // the lane's operand offset in its patch row: a - chunk0 (0..7) in entries
    const int q = qw + li;
    const int64_t ra = q < t.lr ? row_index(g, t, q) * nb + (t.q0 - w) - q + w : 0;
    const int o0 = (int)(ra & 7);
    const int col = 4 * (li & 3), krow = li >> 2;
    f32x4 o[4];
#pragma unroll
    for (int eb = 0; eb < 4; ++eb) o[eb] = (f32x4){0.f, 0.f, 0.f, 0.f};
    KVRegs r;
    u32x4 pc[kLoads];
    gload_block<false, true, NT>(g, t, nullptr, V, t.q0 - w, r);
    load_p(0, pc);
    const uint32_t* prow = reinterpret_cast<const uint32_t*>(patch + li * kPSlots);
    for (int kb = 0; kb < nblk; ++kb) {
        const int t0 = t.q0 - w + kb * kT;
        __syncthreads();
        lstore_block<false, true, NT>(r, nullptr, lv);
#pragma unroll
        for (int n = 0; n < kLoads; ++n) patch[(8 * n + (lane >> 3)) * kPSlots + 1 + cc] = pc[n];
        __syncthreads();
        // the next block's value and probability loads overlap this block's products
        if (kb + 1 < nblk) {
            gload_block<false, true, NT>(g, t, nullptr, V, t0 + kT, r);
            load_p(kb + 1, pc);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            uint32_t pu[4];
#pragma unroll
            for (int f = 0; f < 2; ++f) {
                const int e = o0 + 32 * h + 16 * f + 4 * grp;   // patch entry of the run
                const int d = e >> 1, sh = (e & 1) * 16;
                const uint32_t d0 = prow[d], d1 = prow[d + 1], d2 = prow[d + 2];
                pu[2 * f] = __builtin_amdgcn_alignbit(d1, d0, sh);
                pu[2 * f + 1] = __builtin_amdgcn_alignbit(d2, d1, sh);
            }
            const u32x4 pv = {pu[0], pu[1], pu[2], pu[3]};
            const bf16x8 pf = __builtin_bit_cast(bf16x8, pv);
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
        wave_lds_order();
        // carry: slot 8 becomes the next block's slot 0 (one lane per row)
        if (lane < kRows) patch[lane * kPSlots] = patch[lane * kPSlots + 8];
    }
    if (q >= t.lr) return;
    OT* orow = O + row_off(g, t, q);
#pragma unroll
    for (int eb = 0; eb < 4; ++eb) Out<OT>::put4(orow + eb * 16 + 4 * grp, o[eb]);
}

// --------------------------------------------------------------------- fused
// G2BMM -> online softmax -> GBMM in one pass over the key blocks of the band; scores
// and probabilities stay in registers.  A wave owns 32 queries (two 16-query halves hq),
// a workgroup 128.  Key/value blocks of 64 rows reach LDS by direct global->LDS copies
// (global_load_lds_dwordx4) into a ring of kSlots blocks, issued kSlots - 1 blocks
// ahead.  The kernel is latency-bound, so it is sized for occupancy rather than
// intra-wave overlap: with two slots (32 KB of LDS per workgroup) and <= 128 VGPRs,
// four workgroups share a CU and four waves each SIMD, whose independent block
// iterations hide each other's LDS, MFMA and exp2 latencies.
//
// Softmax bookkeeping per query, in log2 units (x = scale*log2(e)*score): a running
// reference m, and the denominator and O both accumulated unnormalised by MFMA -- the
// denominator as the product of an all-ones operand with the same bf16 probabilities
// that multiply V, so O and its normaliser see identical rounding.  m is raised only
// when a score exceeds it by more than kLazy; the test uses each lane's own maximum,
// and only when it fires is the row maximum formed across the row's 4 lanes.  The
// scale enters as one FMA per score; a negative scale is handled by negating the query
// fragments (an exact sign flip of bf16) and using |scale|.  Band and range masks are
// applied in place, only on blocks that cross an edge.
//
// LDS slot layout: 512 16-byte chunks of K, then 512 of V; chunk c of key row r sits
// at r*8 + (c ^ (r & 7)) (an XOR swizzle: the 16-lane fragment reads of K and the
// transposing reads of V then spread over all bank groups).  A DMA instruction writes
// 64 consecutive chunks in lane order, so the swizzle is applied to the source
// address.  Keys outside the subsequence read a 16-byte zero chunk.
constexpr int kSlotChunks = 2 * kT * 8;
__device__ __align__(16) uint32_t kBandZero[4];

// ds_read_b64_tr_b16 as inline assembly, at LDS byte address addr + OFF.  The
// compiler's own form of this load is treated as possibly reading the destination of
// any global->LDS copy still in flight and waits for all of them (vmcnt(0)), which
// would drain the prefetch ring every block; the ring schedule (vmcnt + barrier before
// a slot is read) already guarantees the block is resident.  The compiler does not
// track this load: its results pass through lds_wait() before any use.
template <int OFF>
__device__ __forceinline__ s16x4 tr_read_raw(uint32_t addr) {
    s16x4 r;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
    return r;
}
// Waits for every outstanding LDS read; the listed registers are tied to the wait, so
// no use of them can be scheduled before it.
__device__ __forceinline__ void lds_wait(bf16x8 (&a)[4]) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]));
}

__device__ __forceinline__ void block_sync() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <typename OT, bool MASK, int kSlots, int NW, bool BUF, int HQ>
__global__ __launch_bounds__(64 * NW, HQ <= 2 ? 4 : 2) void band_fused_kernel(BandGeom g, int ntx,
                                                           const bf16_t* __restrict__ Q,
                                                           const bf16_t* __restrict__ K,
                                                           const bf16_t* __restrict__ V,
                                                           OT* __restrict__ O) {
    // The reference moves only when a score exceeds it by more than kLazy (log2 units), so
    // p <= 2^kLazy: with at most 2w+1 terms per row, O and its normaliser stay far inside
    // the fp32 range, and bf16 p keeps its relative precision at any magnitude.  A wide
    // margin means the reference settles after the first block and rescaling is rare.
    constexpr float kLazy = 64.f;
    constexpr int kQW = 16 * HQ;          // queries per wave (HQ groups of 16)
    constexpr int kFT = NW * kQW;         // queries per tile (NW waves)
    constexpr int kPass = 64 / (NW * 8);  // copy instructions per lane per 64-row block
    __shared__ u32x4 lds[kSlots * kSlotChunks];
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
    const int lane = threadIdx.x & 63, grp = lane >> 4, li = lane & 15;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int w = (int)g.w;
    const int qa = t.q0 + wv * kQW;
    const int xor16 = (lane ^ 16) << 2, xor32 = (lane ^ 32) << 2;
    // scale * log2(e), kept >= the smallest normal float: with scale 0 every score then
    // maps to exp2(~0) = 1 exactly, and a masked score (-inf) still maps to 0
    const float sl2 = fmaxf(fabsf(g.scale) * 1.4426950408889634f, 1.17549435e-38f);
    const uint32_t qflip = g.scale < 0.f ? 0x80008000u : 0u;

    bf16x8 qf[HQ][2];
#pragma unroll
    for (int hq = 0; hq < HQ; ++hq) {
        const int q = qa + hq * 16 + li;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if (q < t.lr)
                v = *reinterpret_cast<const u32x4*>(Q + row_off(g, t, q) + kk * 32 + grp * 8);
            v ^= (u32x4){qflip, qflip, qflip, qflip};
            qf[hq][kk] = __builtin_bit_cast(bf16x8, v);
        }
    }
    const int nblk = (kFT + 2 * w + kT - 1) / kT;
    // this wave's key blocks: those that meet the band of one of its queries
    const int lo = wv * kQW / kT;
    const int hi = min(nblk - 1, (wv * kQW + kQW - 1 + 2 * w) / kT);

    // DMA sources of this lane: key rows dr + e*NW*8 of each block, chunk dch, as byte
    // offsets from the start of the residue subsequence (uniform base pointers)
    const int dr = wv * 8 + (lane >> 3);
    const int dch = (lane & 7) ^ ((lane >> 3) & 7);
    const int64_t seq0 = ((int64_t)t.b * g.l + t.rho) * kD;
    const char* kseq = reinterpret_cast<const char*>(K + seq0);
    const char* vseq = reinterpret_cast<const char*>(V + seq0);
    const uint32_t row_bytes = (uint32_t)g.dil * kD * 2;
    const char* zero = reinterpret_cast<const char*>(kBandZero);
    const int tt0 = t.q0 - w + dr;                   // key of row dr of block 0
    // buffer form: byte offsets from the start of the residue subsequence; a key before
    // it (negative offset, >= 2^31 as unsigned) or after it lies outside the buffer's
    // range and reads zeros, so every block takes the same two loads per pass.  The
    // launch takes this form only when every such offset fits in 32 bits.
    const int nrec = BUF ? (t.lr - 1) * (int)row_bytes + kD * 2 : 0;
    const int voff0 = BUF ? tt0 * (int)row_bytes + dch * 16 : 0;
    auto dma = [&](int kb) {
        u32x4* slot = lds + (kb % kSlots) * kSlotChunks;
        if constexpr (BUF) {
#pragma unroll
            for (int e = 0; e < kPass; ++e) {
                const uint32_t o2 = (uint32_t)(voff0 + (kb * kT + e * NW * 8) * (int)row_bytes);
                buffer_copy16(kseq, nrec, o2, 0, (lds_void*)(slot + (e * NW + wv) * 64));
                buffer_copy16(vseq, nrec, o2, 0, (lds_void*)(slot + 512 + (e * NW + wv) * 64));
            }
            return;
        }
        // 64-bit form: a subsequence may span more than 4 GiB
        const int tt = tt0 + kb * kT;
        if (t.q0 - w + kb * kT >= 0 && t.q0 - w + kb * kT + kT <= t.lr) {   // interior block
            const int64_t off = (int64_t)tt * row_bytes + dch * 16;
#pragma unroll
            for (int e = 0; e < kPass; ++e) {
                const int64_t o2 = off + (int64_t)(e * NW * 8) * row_bytes;
                __builtin_amdgcn_global_load_lds((const void*)(kseq + o2),
                                                 (lds_void*)(slot + (e * NW + wv) * 64), 16, 0,
                                                 0);
                __builtin_amdgcn_global_load_lds((const void*)(vseq + o2),
                                                 (lds_void*)(slot + 512 + (e * NW + wv) * 64),
                                                 16, 0, 0);
            }
        } else {
#pragma unroll
            for (int e = 0; e < kPass; ++e) {
                const int te = tt + NW * 8 * e;
                const bool ok = te >= 0 && te < t.lr;
                const int64_t o2 = (int64_t)te * row_bytes + dch * 16;
                __builtin_amdgcn_global_load_lds((const void*)(ok ? kseq + o2 : zero),
                                                 (lds_void*)(slot + (e * NW + wv) * 64), 16, 0,
                                                 0);
                __builtin_amdgcn_global_load_lds((const void*)(ok ? vseq + o2 : zero),
                                                 (lds_void*)(slot + 512 + (e * NW + wv) * 64),
                                                 16, 0, 0);
            }
        }
    };
    // LDS byte offsets (within a slot) of this lane's fragment reads
    //   K fragment (ft, kk): key row 16ft + li, chunk 4kk + grp
    //   V^T fragment (h, eb, i): key row 32h + 16i + 4grp + li/4, 8 bytes at column
    //   16eb + 4(li%4), i.e. chunk 2eb + (li/2)%2, byte 8(li%2) of it
    int koff[2], voff[4];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) koff[kk] = (li * 8 + ((4 * kk + grp) ^ (li & 7))) * 16;
    {
        const int vr = 4 * grp + (li >> 2);
#pragma unroll
        for (int eb = 0; eb < 4; ++eb)
            voff[eb] = kT * 8 * 16 + (vr * 8 + ((2 * eb + ((li >> 1) & 1)) ^ (vr & 7))) * 16 +
                       8 * (li & 1);
    }
    const char* lds_b = reinterpret_cast<const char*>(lds);
    const uint32_t lds_a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)lds;
    // waits until at most `later` blocks (2*kPass copies each per lane) are in flight
    auto wait_blocks = [](int later) {
        static_assert(kSlots >= 2 && kSlots <= 6, "slot count");
        constexpr int kC = 2 * kPass;
        if (later >= 3 && kSlots >= 6) wait_vmcnt<3 * kC>();
        else if (later >= 2 && kSlots >= 5) wait_vmcnt<2 * kC>();
        else if (later >= 1) wait_vmcnt<kC>();
        else wait_vmcnt<0>();
    };

    f32x4 o[HQ][4], lsum[HQ];
    float m_run[HQ];
#pragma unroll
    for (int hq = 0; hq < HQ; ++hq) {
        lsum[hq] = (f32x4){0.f, 0.f, 0.f, 0.f};
        m_run[hq] = -INFINITY;
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) o[hq][eb] = (f32x4){0.f, 0.f, 0.f, 0.f};
    }
    const bf16x8 ones = __builtin_bit_cast(bf16x8, (u32x4){0x3f803f80u, 0x3f803f80u,
                                                          0x3f803f80u, 0x3f803f80u});

    auto read_k = [&](int kb, bf16x8 (&kf)[4][2]) {
        const char* sb = lds_b + (kb % kSlots) * kSlotChunks * 16;
#pragma unroll
        for (int ft = 0; ft < 4; ++ft)
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
                kf[ft][kk] = *reinterpret_cast<const bf16x8*>(sb + koff[kk] + ft * 16 * 128);
    };
    auto scores = [&](const bf16x8 (&kf)[4][2], f32x4 (&s)[HQ][4]) {
#pragma unroll
        for (int ft = 0; ft < 4; ++ft)
#pragma unroll
            for (int hq = 0; hq < HQ; ++hq) {
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[ft][0], qf[hq][0], acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[ft][1], qf[hq][1], acc, 0, 0, 0);
                s[hq][ft] = acc;
            }
    };

    // One block iteration: scores, softmax and P*V of block kb.
    auto step = [&](int kb) {
        const int t0 = t.q0 - w + kb * kT;
        f32x4 s[HQ][4];
        {
            bf16x8 kf[4][2];
            read_k(kb, kf);
            scores(kf, s);
        }
        bool full = t0 >= qa + kQW - 1 - w && t0 + kT - 1 <= qa + w;
        if (MASK) full = full && t0 >= 0 && t0 + kT <= t.lr;
        if (!full) {                               // band (and range) mask, in place
#pragma unroll
            for (int hq = 0; hq < HQ; ++hq) {
                const int base = t0 + 4 * grp - (qa + hq * 16 + li) + w;
#pragma unroll
                for (int ft = 0; ft < 4; ++ft)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        bool ok = (unsigned)(base + ft * 16 + v) <= (unsigned)(2 * w);
                        if (MASK) {
                            const int tt = t0 + ft * 16 + 4 * grp + v;
                            ok = ok && tt >= 0 && tt < t.lr;
                        }
                        s[hq][ft][v] = ok ? s[hq][ft][v] : -INFINITY;
                    }
            }
        }
        float mb[HQ];
#pragma unroll
        for (int hq = 0; hq < HQ; ++hq) {
            mb[hq] = -INFINITY;
#pragma unroll
            for (int ft = 0; ft < 4; ++ft)
#pragma unroll
                for (int v = 0; v < 4; ++v) mb[hq] = fmaxf(mb[hq], s[hq][ft][v]);
        }
        // lazy reference update; the row maximum (4 lanes) only when a lane asks for it
        bool up = false;
#pragma unroll
        for (int hq = 0; hq < HQ; ++hq) up = up || mb[hq] * sl2 > m_run[hq] + kLazy;
        if (__any(up)) {
#pragma unroll
            for (int hq = 0; hq < HQ; ++hq) {
                float m = mb[hq];
                m = fmaxf(m, __int_as_float(__builtin_amdgcn_ds_bpermute(xor16, __float_as_int(m))));
                m = fmaxf(m, __int_as_float(__builtin_amdgcn_ds_bpermute(xor32, __float_as_int(m))));
                const float mbx = m * sl2;
                const float m_new = mbx > m_run[hq] + kLazy ? mbx : m_run[hq];
                const float corr =
                    m_new == m_run[hq] ? 1.f : __builtin_amdgcn_exp2f(m_run[hq] - m_new);
                lsum[hq] *= corr;
#pragma unroll
                for (int eb = 0; eb < 4; ++eb) o[hq][eb] *= corr;
                m_run[hq] = m_new;
            }
        }
        bf16x8 pf[HQ][2];
#pragma unroll
        for (int hq = 0; hq < HQ; ++hq) {
            const float nm = m_run[hq] == -INFINITY ? 0.f : -m_run[hq];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                bf16x8 pv;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    pv[v] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[hq][2 * h][v], sl2, nm));
                    pv[4 + v] =
                        (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[hq][2 * h + 1][v], sl2, nm));
                }
                pf[hq][h] = pv;
            }
        }
        // P*V per 32-key half h: V^T fragments from key rows 32h and 32h + 16 of the slot
        const uint32_t vb = lds_a + (kb % kSlots) * kSlotChunks * 16;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            bf16x8 vf[4];
#pragma unroll
            for (int eb = 0; eb < 4; ++eb) {
                const uint32_t a = vb + voff[eb] + h * 32 * 128;
                s16x4 r[2] = {tr_read_raw<0>(a), tr_read_raw<16 * 128>(a)};
                vf[eb] = __builtin_bit_cast(bf16x8, r);
            }
            lds_wait(vf);
#pragma unroll
            for (int eb = 0; eb < 4; ++eb)
#pragma unroll
                for (int hq = 0; hq < HQ; ++hq)
                    o[hq][eb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[eb], pf[hq][h],
                                                                        o[hq][eb], 0, 0, 0);
#pragma unroll
            for (int hq = 0; hq < HQ; ++hq)
                lsum[hq] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[hq][h], lsum[hq],
                                                                   0, 0, 0);
        }
    };
    // prologue: blocks 0 .. kSlots-2 in flight, block 0 resident before the loop
#pragma unroll
    for (int b = 0; b < kSlots - 1; ++b)
        if (b < nblk) dma(b);
    wait_blocks(min(nblk - 1, kSlots - 2));
    block_sync();
    for (int kb = 0; kb < nblk; ++kb) {
        if (kb + kSlots - 1 < nblk) dma(kb + kSlots - 1);
        if (kb >= lo && kb <= hi) step(kb);          // the block meets the wave's band
        // block kb + 1 is read by the next iteration: its copies must have landed; those
        // of the blocks after it may still be in flight
        wait_blocks(min(nblk - 1, kb + kSlots - 1) - (kb + 1));
        block_sync();
    }
#pragma unroll
    for (int hq = 0; hq < HQ; ++hq) {
        const int q = qa + hq * 16 + li;
        if (q >= t.lr) continue;
        const float inv = 1.f / lsum[hq][0];
        OT* orow = O + row_off(g, t, q);
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) Out<OT>::put4(orow + eb * 16 + 4 * grp, o[hq][eb] * inv);
    }
}

// Half-block form of the fused kernel: the same tiles, ring and softmax bookkeeping as
// band_fused_kernel with four waves of 32 queries, but every 64-key block is evaluated
// as two 32-key halves, each scores -> softmax -> P*V on its own.  That halves the
// score and key-fragment registers live at once (in zero mode five workgroups per CU
// fit: 96 VGPRs, 5 x 32 KB of LDS; the range masks of mask mode need three to stay out
// of scratch memory), and a half
// that lies outside the band of every query of the wave
// is skipped (the band of 32 queries spans 32 + 2w keys: 17 halves instead of the 18
// of nine whole blocks when w = 256).  The softmax denominator is accumulated on the
// VALU by v_dot2_f32_bf16 of the same bf16 probabilities that multiply V (per lane over
// the lane's keys, summed over the row's four lanes at the end), which replaces the
// all-ones MFMAs.
template <typename OT, bool MASK, bool BUF>
__global__ __launch_bounds__(256, MASK ? 3 : 5) void band_fused_half_kernel(BandGeom g, int ntx,
                                                                 const bf16_t* __restrict__ Q,
                                                                 const bf16_t* __restrict__ K,
                                                                 const bf16_t* __restrict__ V,
                                                                 OT* __restrict__ O) {
    constexpr float kLazy = 64.f;
    constexpr int NW = 4, HQ = 2, kSlots = 2;
    constexpr int kQW = 16 * HQ;          // queries per wave
    constexpr int kFT = NW * kQW;         // queries per tile
    constexpr int kPass = 64 / (NW * 8);  // copy instructions per lane per 64-row block
    __shared__ u32x4 lds[kSlots * kSlotChunks];
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
    const int lane = threadIdx.x & 63, grp = lane >> 4, li = lane & 15;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int w = (int)g.w;
    const int qa = t.q0 + wv * kQW;
    const int xor16 = (lane ^ 16) << 2, xor32 = (lane ^ 32) << 2;
    const float sl2 = fmaxf(fabsf(g.scale) * 1.4426950408889634f, 1.17549435e-38f);
    const uint32_t qflip = g.scale < 0.f ? 0x80008000u : 0u;

    bf16x8 qf[HQ][2];
#pragma unroll
    for (int hq = 0; hq < HQ; ++hq) {
        const int q = qa + hq * 16 + li;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if (q < t.lr)
                v = *reinterpret_cast<const u32x4*>(Q + row_off(g, t, q) + kk * 32 + grp * 8);
            v ^= (u32x4){qflip, qflip, qflip, qflip};
            qf[hq][kk] = __builtin_bit_cast(bf16x8, v);
        }
    }
    const int nblk = (kFT + 2 * w + kT - 1) / kT;

    const int dr = wv * 8 + (lane >> 3);
    const int dch = (lane & 7) ^ ((lane >> 3) & 7);
    const int64_t seq0 = ((int64_t)t.b * g.l + t.rho) * kD;
    const char* kseq = reinterpret_cast<const char*>(K + seq0);
    const char* vseq = reinterpret_cast<const char*>(V + seq0);
    const uint32_t row_bytes = (uint32_t)g.dil * kD * 2;
    const char* zero = reinterpret_cast<const char*>(kBandZero);
    const int tt0 = t.q0 - w + dr;
    const int nrec = BUF ? (t.lr - 1) * (int)row_bytes + kD * 2 : 0;
    const int voff0 = BUF ? tt0 * (int)row_bytes + dch * 16 : 0;
    auto dma = [&](int kb) {
        u32x4* slot = lds + (kb % kSlots) * kSlotChunks;
        if constexpr (BUF) {
#pragma unroll
            for (int e = 0; e < kPass; ++e) {
                const uint32_t o2 = (uint32_t)(voff0 + (kb * kT + e * NW * 8) * (int)row_bytes);
                buffer_copy16(kseq, nrec, o2, 0, (lds_void*)(slot + (e * NW + wv) * 64));
                buffer_copy16(vseq, nrec, o2, 0, (lds_void*)(slot + 512 + (e * NW + wv) * 64));
            }
            return;
        }
        const int tt = tt0 + kb * kT;
        if (t.q0 - w + kb * kT >= 0 && t.q0 - w + kb * kT + kT <= t.lr) {
            const int64_t off = (int64_t)tt * row_bytes + dch * 16;
#pragma unroll
            for (int e = 0; e < kPass; ++e) {
                const int64_t o2 = off + (int64_t)(e * NW * 8) * row_bytes;
                __builtin_amdgcn_global_load_lds((const void*)(kseq + o2),
                                                 (lds_void*)(slot + (e * NW + wv) * 64), 16, 0,
                                                 0);
                __builtin_amdgcn_global_load_lds((const void*)(vseq + o2),
                                                 (lds_void*)(slot + 512 + (e * NW + wv) * 64),
                                                 16, 0, 0);
            }
        } else {
#pragma unroll
            for (int e = 0; e < kPass; ++e) {
                const int te = tt + NW * 8 * e;
                const bool ok = te >= 0 && te < t.lr;
                const int64_t o2 = (int64_t)te * row_bytes + dch * 16;
                __builtin_amdgcn_global_load_lds((const void*)(ok ? kseq + o2 : zero),
                                                 (lds_void*)(slot + (e * NW + wv) * 64), 16, 0,
                                                 0);
                __builtin_amdgcn_global_load_lds((const void*)(ok ? vseq + o2 : zero),
                                                 (lds_void*)(slot + 512 + (e * NW + wv) * 64),
                                                 16, 0, 0);
            }
        }
    };
    int koff[2], voff[4];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) koff[kk] = (li * 8 + ((4 * kk + grp) ^ (li & 7))) * 16;
    {
        const int vr = 4 * grp + (li >> 2);
#pragma unroll
        for (int eb = 0; eb < 4; ++eb)
            voff[eb] = kT * 8 * 16 + (vr * 8 + ((2 * eb + ((li >> 1) & 1)) ^ (vr & 7))) * 16 +
                       8 * (li & 1);
    }
    const char* lds_b = reinterpret_cast<const char*>(lds);
    const uint32_t lds_a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)lds;
    auto wait_blocks = [](int later) {
        constexpr int kC = 2 * kPass;
        if (later >= 1) wait_vmcnt<kC>();
        else wait_vmcnt<0>();
    };

    f32x4 o[HQ][4];
    float lsum[HQ], m_run[HQ];
#pragma unroll
    for (int hq = 0; hq < HQ; ++hq) {
        lsum[hq] = 0.f;
        m_run[hq] = -INFINITY;
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) o[hq][eb] = (f32x4){0.f, 0.f, 0.f, 0.f};
    }
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 ones2 = {(__bf16)1.0f, (__bf16)1.0f};

    // One 32-key half h of block kb: keys t0 + 32h + 16f + 4grp + v (f, v in 0..3/0..1)
    auto half = [&](int kb, int h) {
        const int t0 = t.q0 - w + kb * kT;
        const int th = t0 + 32 * h;
        f32x4 s[HQ][2];
        {
            const char* sb = lds_b + (kb % kSlots) * kSlotChunks * 16 + h * 32 * 128;
#pragma unroll
            for (int f = 0; f < 2; ++f) {
                const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(sb + koff[0] + f * 16 * 128);
                const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(sb + koff[1] + f * 16 * 128);
#pragma unroll
                for (int hq = 0; hq < HQ; ++hq) {
                    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qf[hq][0], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qf[hq][1], acc, 0, 0, 0);
                    s[hq][f] = acc;
                }
            }
        }
        bool full = th >= qa + kQW - 1 - w && th + 31 <= qa + w;
        if (MASK) full = full && th >= 0 && th + 32 <= t.lr;
        if (!full) {
#pragma unroll
            for (int hq = 0; hq < HQ; ++hq) {
                const int base = th + 4 * grp - (qa + hq * 16 + li) + w;
#pragma unroll
                for (int f = 0; f < 2; ++f)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        bool ok = (unsigned)(base + f * 16 + v) <= (unsigned)(2 * w);
                        if (MASK) {
                            const int tt = th + f * 16 + 4 * grp + v;
                            ok = ok && tt >= 0 && tt < t.lr;
                        }
                        s[hq][f][v] = ok ? s[hq][f][v] : -INFINITY;
                    }
            }
        }
        float mb[HQ];
#pragma unroll
        for (int hq = 0; hq < HQ; ++hq) {
            mb[hq] = -INFINITY;
#pragma unroll
            for (int f = 0; f < 2; ++f)
#pragma unroll
                for (int v = 0; v < 4; ++v) mb[hq] = fmaxf(mb[hq], s[hq][f][v]);
        }
        bool up = false;
#pragma unroll
        for (int hq = 0; hq < HQ; ++hq) up = up || mb[hq] * sl2 > m_run[hq] + kLazy;
        if (__any(up)) {
#pragma unroll
            for (int hq = 0; hq < HQ; ++hq) {
                float m = mb[hq];
                m = fmaxf(m, __int_as_float(__builtin_amdgcn_ds_bpermute(xor16, __float_as_int(m))));
                m = fmaxf(m, __int_as_float(__builtin_amdgcn_ds_bpermute(xor32, __float_as_int(m))));
                const float mbx = m * sl2;
                const float m_new = mbx > m_run[hq] + kLazy ? mbx : m_run[hq];
                const float corr =
                    m_new == m_run[hq] ? 1.f : __builtin_amdgcn_exp2f(m_run[hq] - m_new);
                lsum[hq] *= corr;
#pragma unroll
                for (int eb = 0; eb < 4; ++eb) o[hq][eb] *= corr;
                m_run[hq] = m_new;
            }
        }
        bf16x8 pf[HQ];
#pragma unroll
        for (int hq = 0; hq < HQ; ++hq) {
            const float nm = m_run[hq] == -INFINITY ? 0.f : -m_run[hq];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                pf[hq][v] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[hq][0][v], sl2, nm));
                pf[hq][4 + v] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[hq][1][v], sl2, nm));
            }
            // (pairs formed from the elements: a bit_cast of the vector's dword e to a
            // bf16 pair was compiled as dword 0 for every e)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bf16x2 pr = {pf[hq][2 * e], pf[hq][2 * e + 1]};
                lsum[hq] = __builtin_amdgcn_fdot2_f32_bf16(pr, ones2, lsum[hq], false);
            }
        }
        const uint32_t a0 = lds_a + (kb % kSlots) * kSlotChunks * 16 + h * 32 * 128;
        bf16x8 vf[4];
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) {
            const uint32_t a = a0 + voff[eb];
            s16x4 r[2] = {tr_read_raw<0>(a), tr_read_raw<16 * 128>(a)};
            vf[eb] = __builtin_bit_cast(bf16x8, r);
        }
        lds_wait(vf);
#pragma unroll
        for (int eb = 0; eb < 4; ++eb)
#pragma unroll
            for (int hq = 0; hq < HQ; ++hq)
                o[hq][eb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[eb], pf[hq], o[hq][eb], 0,
                                                                    0, 0);
    };
    // the wave's band spans keys qa - w .. qa + kQW - 1 + w (subsequence indices)
    const int klo = qa - w, khi = qa + kQW - 1 + w;
#pragma unroll
    for (int b = 0; b < kSlots - 1; ++b)
        if (b < nblk) dma(b);
    wait_blocks(min(nblk - 1, kSlots - 2));
    block_sync();
    for (int kb = 0; kb < nblk; ++kb) {
        if (kb + kSlots - 1 < nblk) dma(kb + kSlots - 1);
        const int t0 = t.q0 - w + kb * kT;
#pragma unroll
        for (int h = 0; h < 2; ++h)
            if (t0 + 32 * h + 31 >= klo && t0 + 32 * h <= khi) half(kb, h);
        wait_blocks(min(nblk - 1, kb + kSlots - 1) - (kb + 1));
        block_sync();
    }
#pragma unroll
    for (int hq = 0; hq < HQ; ++hq) {
        float tot = lsum[hq];
        tot += __int_as_float(__builtin_amdgcn_ds_bpermute(xor16, __float_as_int(tot)));
        tot += __int_as_float(__builtin_amdgcn_ds_bpermute(xor32, __float_as_int(tot)));
        const int q = qa + hq * 16 + li;
        if (q >= t.lr) continue;
        const float inv = 1.f / tot;
        OT* orow = O + row_off(g, t, q);
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) Out<OT>::put4(orow + eb * 16 + 4 * grp, o[hq][eb] * inv);
    }
}

struct Grid {
    dim3 grid;
    int ntx;
};

// Waves per workgroup of the staged G2BMM and GBMM (tiles of 16 queries per wave).
// Eight G2BMM waves share each key block (each key row is read by 5 tiles instead of
// 9 at the Longformer band); the GBMM measured slower with eight.
constexpr int kG2bmmWaves = 8;
constexpr int kGbmmWaves = 4;

Grid tile_grid(const BandGeom& g, int ft = kT) {
    const int64_t l0 = (g.l + g.dil - 1) / g.dil;   // longest residue subsequence (rho = 0)
    const int ntx = (int)((l0 + ft - 1) / ft);
    return {dim3((unsigned)(ntx * g.dil * g.b)), ntx};
}

}  // namespace

hipError_t launch_band_g2bmm(const BandGeom& g, const void* q, const void* k, float* s,
                             hipStream_t stream) {
    constexpr int NW = kG2bmmWaves;
    Grid gr = tile_grid(g, 16 * NW);
    hipLaunchKernelGGL(band_g2bmm_kernel<NW>, gr.grid, dim3(64 * NW), 0, stream, g, gr.ntx,
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
    constexpr int NW = kGbmmWaves;
    Grid gr = tile_grid(g, 16 * NW);
    if (o_bf16)
        hipLaunchKernelGGL((band_gbmm_kernel<bf16_t, NW>), gr.grid, dim3(64 * NW), 0, stream, g,
                           gr.ntx, (const bf16_t*)p, (const bf16_t*)v, (bf16_t*)o);
    else
        hipLaunchKernelGGL((band_gbmm_kernel<float, NW>), gr.grid, dim3(64 * NW), 0, stream, g,
                           gr.ntx, (const bf16_t*)p, (const bf16_t*)v, (float*)o);
    return hipGetLastError();
}

template <int NW, int HQ>
hipError_t launch_fused_nw(const BandGeom& g, const void* q, const void* k, const void* v,
                           void* o, int o_bf16, int mask, hipStream_t stream) {
    const int64_t l0 = (g.l + g.dil - 1) / g.dil;
    const int ntx = (int)((l0 + 16 * HQ * NW - 1) / (16 * HQ * NW));
    const dim3 grid((unsigned)(ntx * g.dil * g.b));
    // buffer-load copies need every key offset of a subsequence, including the band's
    // reach before and after it, inside +-2^31 bytes
    const bool buf = (l0 + g.w + 4 * kT) * g.dil * kD * 2 < (int64_t(1) << 31);
#define OLLIE_FUSED(OT, M, B)                                                                \
    hipLaunchKernelGGL((band_fused_kernel<OT, M, 2, NW, B, HQ>), grid, dim3(64 * NW), 0, stream, \
                       g, ntx, (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, (OT*)o)
#define OLLIE_FUSED_B(OT, M)            \
    if (buf) OLLIE_FUSED(OT, M, true);  \
    else OLLIE_FUSED(OT, M, false)
    if (o_bf16) {
        if (mask) OLLIE_FUSED_B(bf16_t, true);
        else OLLIE_FUSED_B(bf16_t, false);
    } else {
        if (mask) OLLIE_FUSED_B(float, true);
        else OLLIE_FUSED_B(float, false);
    }
#undef OLLIE_FUSED_B
#undef OLLIE_FUSED
    return hipGetLastError();
}

hipError_t launch_fused_half(const BandGeom& g, const void* q, const void* k, const void* v,
                             void* o, int o_bf16, int mask, hipStream_t stream) {
    const int64_t l0 = (g.l + g.dil - 1) / g.dil;
    const int ntx = (int)((l0 + 127) / 128);
    const dim3 grid((unsigned)(ntx * g.dil * g.b));
    const bool buf = (l0 + g.w + 4 * kT) * g.dil * kD * 2 < (int64_t(1) << 31);
#define OLLIE_HALF(OT, M, B)                                                                 \
    hipLaunchKernelGGL((band_fused_half_kernel<OT, M, B>), grid, dim3(256), 0, stream, g, ntx, \
                       (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, (OT*)o)
#define OLLIE_HALF_B(OT, M)            \
    if (buf) OLLIE_HALF(OT, M, true);  \
    else OLLIE_HALF(OT, M, false)
    if (o_bf16) {
        if (mask) OLLIE_HALF_B(bf16_t, true);
        else OLLIE_HALF_B(bf16_t, false);
    } else {
        if (mask) OLLIE_HALF_B(float, true);
        else OLLIE_HALF_B(float, false);
    }
#undef OLLIE_HALF_B
#undef OLLIE_HALF
    return hipGetLastError();
}

// Wave shapes: 0 = four waves of 32 queries (the default: measured faster than eight
// waves, which have half the copies per query but the same occupancy and twice the LDS
// per workgroup), 1 = four waves of 64 queries, 2 = two waves of 64 queries (half the
// LDS reads per score, two waves per SIMD), 3 = four waves of 32 queries over 32-key
// halves (band_fused_half_kernel).  `shape` (0..3, from the caller's flags; -1 =
// automatic) overrides the choice for tuning sweeps and tests.
hipError_t launch_band_fused(const BandGeom& g, const void* q, const void* k, const void* v,
                             void* o, int o_bf16, int mask, int shape, hipStream_t stream) {
    const int cfg = shape < 0 ? 0 : shape;
    if (cfg == 3) return launch_fused_half(g, q, k, v, o, o_bf16, mask, stream);
    if (cfg == 1) return launch_fused_nw<4, 4>(g, q, k, v, o, o_bf16, mask, stream);
    if (cfg == 2) return launch_fused_nw<2, 4>(g, q, k, v, o, o_bf16, mask, stream);
    return launch_fused_nw<4, 2>(g, q, k, v, o, o_bf16, mask, stream);
}

}  // namespace ollie
