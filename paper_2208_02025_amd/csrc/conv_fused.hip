// Fused GEMM + eOperator for the derived convolution forms (expression fusion, §4.1).
//
// Substituting the GEMM scope Y[m][(r,s,k)] = sum_c X[m][c] Wt[r][s][k][c] into the
// OffsetAdd eOperator (section 2) -- or into the selective add of the strided
// transposed convolution (section 6.3) -- gives one expression per output element:
//   out[o][k] = sum_{taps (r,s) valid for o} sum_c X[in(o,r,s)][c] * Wt[r][s][k][c]
// i.e. one contraction over (tap, c) whose A operand is X gathered through the
// eOperator's index map.  This kernel evaluates that fused expression output-stationary:
// a tile of output pixels x output channels accumulates over taps and channel blocks in
// MFMA registers, so Y never exists, not even on chip.  An element-wise tail (bias,
// residual, ReLU) is applied to the accumulators before the store.
//
// Output pixels are grouped into classes that share their tap list:
//   forward conv:     one class; input row hi = stride*ho - pad + r*dil (per-pixel
//                     validity against the image bounds handles the zero padding);
//   transposed conv:  one class per output residue (ho % stride, wo % stride); a tap
//                     belongs to the class iff (ho + pad - r*dil) is divisible by the
//                     stride, and then hi = ho/stride + (ho%stride + pad - r*dil)/stride.
//                     Each class contracts over its own taps only, so no partial that the
//                     selective add would drop is ever computed;
//   dilated conv as residue sub-images (stride 1, section 6.2): one class per output
//                     residue (ho % dil, wo % dil), a non-dilated convolution over the
//                     input sub-image of the matching residue (alpha = gamma = dil).
// All cases are  hi = alpha*i + beta_tap,  ho = oh0 + gamma*i  over class coordinates i.
//
// Main loop: the bf16 DMA pipeline of the GEMM stage (global_load_lds_dwordx4 into an
// XOR-swizzled LDS ring, v_mfma_f32_16x16x32_bf16).  A rows are gathered per tap; rows
// whose input pixel lies in the zero padding fetch a 16-byte zero chunk instead.
#include "common.h"

namespace ollie {

namespace {

constexpr int kMaxCls = 16;

__device__ __align__(16) uint32_t kZeroChunk[4];   // 16 zero bytes (zero-initialised)

// The taps of one class along one axis: kernel indices r0 + i*rstep and input offsets
// b0 + i*bstep, i < n (an arithmetic progression in every form below).
struct AxisTaps {
    int r0, rstep, b0, bstep, n;
};

struct FusedPlan {
    int n, c, h, w, k, ho, wo, s;
    int alpha_h, alpha_w;     // input coordinate = alpha * class coordinate + b_tap
    int gam_h, gam_w;         // output coordinate = o0 + gamma * class coordinate
    int tiles_n;              // output-channel tiles
    int ncls;
    int x_bytes, w_bytes;     // sizes of X and Wt (buffer-load form: both < 2^31)
    int cls_tile0[kMaxCls + 1];   // first workgroup tile of each class
    int cls_hc[kMaxCls], cls_wc[kMaxCls], cls_oh0[kMaxCls], cls_ow0[kMaxCls];
    AxisTaps cls_th[kMaxCls], cls_tw[kMaxCls];   // a class's taps: th x tw, r-major
};

// Which tile of which class a workgroup owns.  Consecutive workgroup ids go to
// different XCDs, so ids are regrouped to give each XCD a contiguous range of tiles.
struct TileId {
    int cls, m0, k0, mc, plane, wc;
};
__device__ __forceinline__ TileId tile_of(const FusedPlan& P, int bm, int bn) {
    const int nblk = gridDim.x;
    const int bid = blockIdx.x;
    const int id = (nblk & 7) == 0 ? (bid & 7) * (nblk >> 3) + (bid >> 3) : bid;
    int cls = 0;
    while (cls + 1 < P.ncls && id >= P.cls_tile0[cls + 1]) ++cls;
    const int local = id - P.cls_tile0[cls];
    TileId t;
    t.cls = cls;
    t.m0 = (local / P.tiles_n) * bm;
    t.k0 = (local % P.tiles_n) * bn;
    t.wc = P.cls_wc[cls];
    t.plane = P.cls_hc[cls] * t.wc;
    t.mc = P.n * t.plane;                 // output pixels of this class
    return t;
}

// Global->LDS copies of one k-tile (64 channels) of the operand tiles: BM rows of X
// gathered through the class's index map and BN rows of Wt, 16-byte chunks written to
// the XOR-swizzled LDS layout (the swizzle is applied to the source chunk, since one
// copy instruction writes 64 lanes x 16 bytes contiguously).  Lane L of wave v copies
// chunk L%8 of rows (i*NW + v)*8 + L/8.
//
// BUF: through buffer loads with 32-bit byte offsets.  A row whose input pixel lies in
// the zero padding gets an offset beyond the buffer's range, for which the load
// returns zeros, so a k-tile costs one add per row; the validity test runs once per
// tap.  Otherwise through 64-bit pointers, a padding row reading a 16-byte zero chunk.
template <int NW, int BM, int BN, bool BUF>
struct TileCopy {
    static constexpr int NT = 64 * NW;
    static constexpr int A = BM * kTileChunks / NT, B = BN * kTileChunks / NT;
    static constexpr int LOADS = A + B;
    static_assert((BM * kTileChunks) % NT == 0 && (BN * kTileChunks) % NT == 0, "whole loads");
    static constexpr uint32_t kOut = 0x80000000u;   // beyond any buffer of < 2^31 bytes

    const bf16_t* X;
    const bf16_t* Wt;
    int x_bytes, w_bytes;
    int H, W, C, K, kc_n, wave, lane, cho;
    int hi0[A], wi0[A], rowpix[A];   // class coordinates (scaled) and base pixel of each row
    uint32_t vbase[A];               // byte offset of the row's tap pixel (+chunk), or kOut
    int wofs[B];                     // byte offset of the Wt row (+chunk) at tap 0, channel 0
    int wrow[B];                     // output channel of each Wt row
    AxisTaps th, tw;                 // the class's taps
    int ri, si, kc;                  // k-tile the next issue() copies: tap (ri, si), channels kc
    int left;                        // k-tiles not yet copied (the last one repeats after)
    int bh, bw, rs;

    __device__ __forceinline__ void init(const FusedPlan& P, const TileId& t, const bf16_t* x,
                                         const bf16_t* wt) {
        X = x; Wt = wt;
        H = P.h; W = P.w; C = P.c; K = P.k; kc_n = P.c / kTileK;
        lane = threadIdx.x & 63;
        wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        cho = ((lane & 7) ^ ((lane >> 3) & 7)) * 8;   // swizzled source chunk (elements)
        x_bytes = P.x_bytes; w_bytes = P.w_bytes;
#pragma unroll
        for (int i = 0; i < A; ++i) {
            const int m = t.m0 + (i * NW + wave) * 8 + (lane >> 3);
            const int mm = m < t.mc ? m : 0;
            const int nn = mm / t.plane, rem = mm - nn * t.plane;
            const int ii = rem / t.wc, jj = rem - ii * t.wc;
            // an out-of-range row reads zeros: its coordinates are pushed off the image
            hi0[i] = m < t.mc ? P.alpha_h * ii : -(1 << 28);
            wi0[i] = P.alpha_w * jj;
            rowpix[i] = m < t.mc ? (nn * H + hi0[i]) * W + wi0[i] : 0;   // read only if valid
        }
#pragma unroll
        for (int i = 0; i < B; ++i) {
            int kk = t.k0 + (i * NW + wave) * 8 + (lane >> 3);
            kk = kk < K ? kk : K - 1;
            wrow[i] = kk;
            wofs[i] = (kk * C + cho) * 2;
        }
        th = P.cls_th[t.cls]; tw = P.cls_tw[t.cls];
        ri = 0; si = 0; kc = 0;
        left = th.n * tw.n * kc_n;
        set_tap(P);
    }
    // tap quantities from scalar arithmetic (no table reads inside the main loop)
    __device__ __forceinline__ void set_tap(const FusedPlan& P) {
        bh = th.b0 + ri * th.bstep;
        bw = tw.b0 + si * tw.bstep;
        rs = (th.r0 + ri * th.rstep) * P.s + tw.r0 + si * tw.rstep;
        if constexpr (BUF) {
            const int shift = bh * W + bw;
#pragma unroll
            for (int i = 0; i < A; ++i) {
                const bool ok = (unsigned)(hi0[i] + bh) < (unsigned)H &&
                                (unsigned)(wi0[i] + bw) < (unsigned)W;
                vbase[i] = ok ? (uint32_t)(((rowpix[i] + shift) * C + cho) * 2) : kOut;
            }
        }
    }
    // copies the current k-tile into `slot` and advances to the next one; past the last
    // k-tile it copies the last one again (the callers issue a fixed number of copies
    // per iteration, so the copy counters need no branches)
    __device__ __forceinline__ void issue(const FusedPlan& P, u32x4* slot) {
        copy(slot);
        advance(P);
    }
    __device__ __forceinline__ void copy(u32x4* slot) {
        if constexpr (BUF) {
            const int kofs = kc * kTileK * 2;
            const int wsoff = rs * K * C * 2 + kofs;
#pragma unroll
            for (int i = 0; i < A; ++i)
                buffer_copy16(X, x_bytes, vbase[i] + kofs, 0,
                              (lds_void*)(slot + (i * NW + wave) * 64));
#pragma unroll
            for (int i = 0; i < B; ++i)
                buffer_copy16(Wt, w_bytes, wofs[i], wsoff,
                              (lds_void*)(slot + BM * kTileChunks + (i * NW + wave) * 64));
        } else {
            const bf16_t* zero = reinterpret_cast<const bf16_t*>(kZeroChunk);
#pragma unroll
            for (int i = 0; i < A; ++i) {
                const int hi = hi0[i] + bh, wi = wi0[i] + bw;
                const bool ok = (unsigned)hi < (unsigned)H && (unsigned)wi < (unsigned)W;
                const bf16_t* p =
                    ok ? X + (int64_t)(rowpix[i] + bh * W + bw) * C + kc * kTileK + cho : zero;
                __builtin_amdgcn_global_load_lds((const void*)p,
                                                 (lds_void*)(slot + (i * NW + wave) * 64), 16, 0,
                                                 0);
            }
#pragma unroll
            for (int i = 0; i < B; ++i)
                __builtin_amdgcn_global_load_lds(
                    (const void*)(Wt + ((int64_t)rs * K + wrow[i]) * C + kc * kTileK + cho),
                    (lds_void*)(slot + BM * kTileChunks + (i * NW + wave) * 64), 16, 0, 0);
        }
    }
    // moves to the next k-tile (the last one stays current once reached)
    __device__ __forceinline__ void advance(const FusedPlan& P) {
        if (--left <= 0) return;
        if (++kc == kc_n) {
            kc = 0;
            if (++si == tw.n) {
                si = 0;
                ++ri;
            }
            set_tap(P);
        }
    }
};

// Output tile store: acc[i][j][v] = out[pixel of class row m][k] with
//   m = m0 + wm*WM + j*16 + lane%16,  k = k0 + wn*WN + i*16 + 4*(lane/16) + v,
// after the element-wise tail.
template <int FM, int FN, int WM, int WN, typename OT>
__device__ __forceinline__ void store_tile(const FusedPlan& P, const TileId& t, int wm, int wn,
                                           f32x4 (&acc)[FN][FM], OT* __restrict__ out,
                                           const Epi& epi) {
    const int lane = threadIdx.x & 63;
    const int K = P.k;
    const bool vec_ok = (K & 3) == 0;
    const int oh0 = P.cls_oh0[t.cls], ow0 = P.cls_ow0[t.cls];
#pragma unroll
    for (int j = 0; j < FM; ++j) {
        const int m = t.m0 + wm * WM + j * 16 + (lane & 15);
        if (m >= t.mc) continue;
        const int nn = m / t.plane, rem = m - nn * t.plane;
        const int ii = rem / t.wc, jj = rem - ii * t.wc;
        const int64_t opix =
            ((int64_t)nn * P.ho + oh0 + P.gam_h * ii) * P.wo + ow0 + P.gam_w * jj;
        OT* orow = out + opix * K;
#pragma unroll
        for (int i = 0; i < FN; ++i) {
            const int k = t.k0 + wn * WN + i * 16 + 4 * (lane >> 4);
            if (vec_ok && k + 3 < K) {
                Out<OT>::put4(orow + k, epi_apply4(epi, acc[i][j], opix * K + k, k));
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    if (k + v < K)
                        Out<OT>::put(orow + k + v,
                                     epi_apply(epi, acc[i][j][v], opix * K + k + v, k + v));
            }
        }
    }
}

// NW = 4 or 8 waves over the tile, several workgroups per CU.  Eight waves keep twice
// as many global->LDS copies in flight per workgroup, which is what bounds the small
// shapes.  KS = 1: the waves tile the output 2 x NW/2.  KS = 2: the two halves of the
// waves take the two 32-deep halves of every k-tile over the same 2 x NW/4 output
// tiling, and the halves' accumulators are summed through LDS at the end; per MFMA the
// larger wave blocks read 3/8 fewer LDS bytes, at two waves per SIMD.
template <int BM, int BN, int NSTAGE, typename OT, int NW, bool BUF, int KS = 1>
__global__ __launch_bounds__(64 * NW, NSTAGE * (BM + BN) * kTileChunks * 16 <= 80 * 1024 ? 2 : 1)
void conv_fused_kernel(const bf16_t* __restrict__ X, const bf16_t* __restrict__ Wt,
                       OT* __restrict__ out, FusedPlan P, Epi epi) {
    static_assert(KS == 1 || KS == 2, "k split");
    constexpr int NWO = NW / KS;                 // waves over the output tile
    constexpr int WM = BM / 2, WN = BN / (NWO / 2);
    constexpr int FM = WM / 16, FN = WN / 16;
    constexpr int STAGE_CHUNKS = (BM + BN) * kTileChunks;
    constexpr int RED_CHUNKS = KS == 2 ? NWO * FN * FM * 64 : 0;   // f32x4 partial sums
    constexpr int LDS_CHUNKS =
        NSTAGE * STAGE_CHUNKS > RED_CHUNKS ? NSTAGE * STAGE_CHUNKS : RED_CHUNKS;
    using Copy = TileCopy<NW, BM, BN, BUF>;
    constexpr int LOADS = Copy::LOADS;
    static_assert(FM >= 1 && FN >= 1, "wave tile");
    __shared__ u32x4 lds[LDS_CHUNKS];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int kh = wave / NWO;                   // k half (KS = 2)
    const int wo = wave % NWO;
    const int wm = wo / (NWO / 2), wn = wo % (NWO / 2);
    const TileId t = tile_of(P, BM, BN);
    const int total = P.cls_th[t.cls].n * P.cls_tw[t.cls].n * (P.c / kTileK);
    Copy cp;
    cp.init(P, t, X, Wt);

    f32x4 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};

    // every iteration issues one k-tile of copies (repeats of the last one near the end
    // land in slots nobody reads again), so the copy counter waits are constant
#pragma unroll
    for (int s = 0; s < NSTAGE - 1; ++s) cp.issue(P, lds + s * STAGE_CHUNKS);
    for (int it = 0; it < total; ++it) {
        wait_vmcnt<(NSTAGE - 2) * LOADS>();
        __builtin_amdgcn_s_barrier();   // tile `it` is in LDS everywhere; `it - 1` is consumed
        cp.copy(lds + ((it + NSTAGE - 1) % NSTAGE) * STAGE_CHUNKS);
        const u32x4* la = lds + (it % NSTAGE) * STAGE_CHUNKS;
        const u32x4* lb = la + BM * kTileChunks;
#pragma unroll
        for (int k2 = 0; k2 < kTileK / 32 / KS; ++k2) {
            const int kk = KS == 2 ? kh : k2;
            const int ch = kk * 4 + (lane >> 4);
            bf16x8 fa[FN], fb[FM];
#pragma unroll
            for (int i = 0; i < FN; ++i)
                fa[i] = __builtin_bit_cast(bf16x8,
                                           lb[tile_swz(wn * WN + i * 16 + (lane & 15), ch)]);
#pragma unroll
            for (int j = 0; j < FM; ++j)
                fb[j] = __builtin_bit_cast(bf16x8,
                                           la[tile_swz(wm * WM + j * 16 + (lane & 15), ch)]);
#pragma unroll
            for (int i = 0; i < FN; ++i)
#pragma unroll
                for (int j = 0; j < FM; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j],
                                                                        0, 0, 0);
        }
        cp.advance(P);
    }
    wait_vmcnt<0>();   // no copy into LDS may still be in flight when the workgroup ends
    if constexpr (KS == 2) {
        // the second k half hands its partial sums to the first through LDS
        __syncthreads();   // every wave is done with the copy ring
        f32x4* red = reinterpret_cast<f32x4*>(lds) + wo * FN * FM * 64 + lane;
        if (kh == 1) {
#pragma unroll
            for (int i = 0; i < FN; ++i)
#pragma unroll
                for (int j = 0; j < FM; ++j) red[(i * FM + j) * 64] = acc[i][j];
        }
        __syncthreads();
        if (kh == 1) return;
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
            for (int j = 0; j < FM; ++j) acc[i][j] += red[(i * FM + j) * 64];
    }
    store_tile<FM, FN, WM, WN, OT>(P, t, wm, wn, acc, out, epi);
}

// Software-pipelined form for large tiles: four waves (2 x 2), each owning a
// (BM/2) x (BN/2) block of the output tile, one workgroup per CU.  The larger wave
// block halves the LDS bytes read per MFMA compared with eight waves on the same tile,
// and the schedule keeps the LDS reads, the global->LDS copies and the MFMAs of one wave
// overlapped instead of letting barrier-aligned waves alternate between them:
//   * the operand fragments of the next k/32 sub-step are read from LDS while the
//     MFMAs of the current one run (two fragment sets in registers);
//   * one barrier per k-tile, between the two sub-steps: after it the slot of the
//     current k-tile is free (every wave has its fragments in registers) and is
//     refilled with the k-tile NS ahead, so NS k-tiles of copies are in flight.
template <int BM, int BN, int NS, typename OT>
__global__ __launch_bounds__(256, 1)
void conv_fused_pipe_kernel(const bf16_t* __restrict__ X, const bf16_t* __restrict__ Wt,
                            OT* __restrict__ out, FusedPlan P, Epi epi) {
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int FM = WM / 16, FN = WN / 16;
    constexpr int STAGE_CHUNKS = (BM + BN) * kTileChunks;
    using Copy = TileCopy<4, BM, BN, true>;
    constexpr int LOADS = Copy::LOADS;
    static_assert(FM >= 1 && FN >= 1 && NS >= 2, "tile");
    __shared__ u32x4 lds[NS * STAGE_CHUNKS];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const TileId t = tile_of(P, BM, BN);
    const int total = P.cls_th[t.cls].n * P.cls_tw[t.cls].n * (P.c / kTileK);
    Copy cp;
    cp.init(P, t, X, Wt);

    struct Frag { bf16x8 a[FN], b[FM]; };
    auto read = [&](int stage, int sub, Frag& f) {
        const u32x4* la = lds + (stage % NS) * STAGE_CHUNKS;
        const u32x4* lb = la + BM * kTileChunks;
        const int ch = sub * 4 + (lane >> 4);
#pragma unroll
        for (int i = 0; i < FN; ++i)
            f.a[i] = __builtin_bit_cast(bf16x8, lb[tile_swz(wn * WN + i * 16 + (lane & 15), ch)]);
#pragma unroll
        for (int j = 0; j < FM; ++j)
            f.b[j] = __builtin_bit_cast(bf16x8, la[tile_swz(wm * WM + j * 16 + (lane & 15), ch)]);
    };

    f32x4 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};
    auto mma = [&](const Frag& f) {
#pragma unroll
        for (int j = 0; j < FM; ++j)
#pragma unroll
            for (int i = 0; i < FN; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.a[i], f.b[j], acc[i][j],
                                                                    0, 0, 0);
    };

    // one k-tile of copies per iteration, repeats of the last k-tile near the end (into
    // slots nobody reads again), so the copy counter waits are constant
#pragma unroll
    for (int s = 0; s < NS; ++s) cp.issue(P, lds + s * STAGE_CHUNKS);
    wait_vmcnt<(NS - 1) * LOADS>();
    __builtin_amdgcn_s_barrier();
    Frag F, G;
    read(0, 0, F);
    for (int it = 0; it < total - 1; ++it) {
        read(it, 1, G);
        mma(F);
        // the reads of G go out first, the MFMAs on F cover their latency
        __builtin_amdgcn_sched_group_barrier(0x100, FM + FN, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, FM * FN, 0);
        // before k-tile it+1 is read: its copies have landed (only those of the later
        // k-tiles may still be in flight), and this wave's reads of slot it are done
        __builtin_amdgcn_sched_barrier(0);    // nothing moves across the barrier
        wait_vmcnt<(NS - 2) * LOADS>();
        __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        cp.copy(lds + (it % NS) * STAGE_CHUNKS);
        read(it + 1, 0, F);
        mma(G);
        // reads of F first, then the copies spread between the MFMAs on G
        __builtin_amdgcn_sched_group_barrier(0x100, FM + FN, 0);
#pragma unroll
        for (int q = 0; q < LOADS; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, (FM * FN) / LOADS, 0);
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - ((FM * FN) / LOADS) * LOADS, 0);
        cp.advance(P);
    }
    if (total > 0) {   // the last k-tile: no reads of a next one
        read(total - 1, 1, G);
        mma(F);
        mma(G);
    }
    wait_vmcnt<0>();   // no copy into LDS may still be in flight when the workgroup ends
    store_tile<FM, FN, WM, WN, OT>(P, t, wm, wn, acc, out, epi);
}

// Row-window form for classes whose taps along w step by one class column (the residue
// form, and stride-1 undilated convolutions): the A operand of the taps (r, s) of one
// kernel row r is, for every s, the same window of input rows shifted by s columns.
// So a k-tile stage covers one (kernel row r, 64 channels) pair: the window of the
// tile's class rows, TH rows of (wc + S - 1) input pixels, is copied once and read at
// column offsets s = 0..S-1 by the MFMA fragments, next to the S weight slices of that
// kernel row.  Against per-tap copies of the 192 gathered rows this moves 40% fewer
// bytes from L2 per MFMA, which is what bounds the large dilated layer.
//
// Fixed shape: 192 x 128 output tile, 8 waves (2 x 4, each 96 x 32), two 80 KB stages
// (one workgroup per CU).  Needs wc % 16 == 0 (a 16-pixel MFMA fragment stays in one
// class row), 192 % wc == 0 (the tile is TH = 192 / wc whole class rows; a tile may
// straddle two images) and S <= 3.  The sum runs over taps in the order (r, channels,
// s), a different summation order from the per-tap forms.
constexpr int kWinBM = 192, kWinBN = 128, kWinArows = 256, kWinS = 3;

template <typename OT>
__global__ __launch_bounds__(512, 1)
void conv_window_kernel(const bf16_t* __restrict__ X, const bf16_t* __restrict__ Wt,
                        OT* __restrict__ out, FusedPlan P, Epi epi) {
    constexpr int NW = 8, BM = kWinBM, BN = kWinBN;
    constexpr int WM = BM / 2, WN = BN / 4, FM = WM / 16, FN = WN / 16;
    constexpr int A_CHUNKS = kWinArows * kTileChunks;
    constexpr int STAGE_CHUNKS = A_CHUNKS + kWinS * BN * kTileChunks;
    constexpr int A_MAX = kWinArows / (8 * NW);          // window copy instructions per wave
    constexpr int B_LOADS = kWinS * BN / (8 * NW);       // weight copy instructions per wave
    __shared__ u32x4 lds[2 * STAGE_CHUNKS];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave / 4, wn = wave % 4;
    const TileId t = tile_of(P, BM, BN);
    const AxisTaps th = P.cls_th[t.cls], tw = P.cls_tw[t.cls];
    const int ns = tw.n;                       // taps along w (1..3)
    const int wrow = t.wc + ns - 1;            // window row length (input pixels)
    const int thr = BM / t.wc;                 // class rows per tile
    const int g0 = t.m0 / t.wc;                // first class row (over images)
    const int hc = t.plane / t.wc;
    const int nrows = P.n * hc;                // class rows over all images
    const int H = P.h, W = P.w, C = P.c, K = P.k;
    const int kc_n = C / kTileK;
    const int total = th.n * kc_n;
    const int nA = (thr * wrow + 7) / 8;       // window copy instructions in all
    const int cho = ((lane & 7) ^ ((lane >> 3) & 7)) * 8;

    // window rows of this lane: input pixel base (tap row 0) and its validity
    int wpix[A_MAX], whi[A_MAX], wwi[A_MAX];
#pragma unroll
    for (int i = 0; i < A_MAX; ++i) {
        const int q = (i * NW + wave) * 8 + (lane >> 3);
        const int ii = q / wrow, jj = q - ii * wrow;
        const int g = g0 + ii;
        const int nn = g / hc, ci = g - nn * hc;
        const bool rowok = ii < thr && g < nrows;
        whi[i] = rowok ? P.alpha_h * ci + th.b0 : -(1 << 28);
        wwi[i] = P.alpha_w * jj + tw.b0;
        wpix[i] = rowok ? (nn * H + whi[i]) * W + wwi[i] : 0;
    }
    // weight rows of this lane: slice s = q / BN, output channel k0 + q % BN
    int wofs[B_LOADS];
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i) {
        const int q = (i * NW + wave) * 8 + (lane >> 3);
        int kk = t.k0 + q % BN;
        kk = kk < K ? kk : K - 1;
        wofs[i] = (kk * C + cho) * 2;
    }
    // fragment rows: output pixel m' = wm*WM + j*16 + lane%16 of the tile sits at window
    // row (m' / wc) * wrow + m' % wc for s = 0
    int arow[FM];
#pragma unroll
    for (int j = 0; j < FM; ++j) {
        const int mm = wm * WM + j * 16 + (lane & 15);
        arow[j] = (mm / t.wc) * wrow + mm % t.wc;
    }

    uint32_t wv[A_MAX];      // window offsets of the current kernel row
    int cur_r = -1;
    auto copy = [&](int stage, u32x4* slot) {
        const int r = stage / kc_n, kc = stage - r * kc_n;
        if (r != cur_r) {
            cur_r = r;
            const int dh = r * th.bstep;
#pragma unroll
            for (int i = 0; i < A_MAX; ++i) {
                const bool ok = (unsigned)(whi[i] + dh) < (unsigned)H &&
                                (unsigned)wwi[i] < (unsigned)W;
                wv[i] = ok ? (uint32_t)(((wpix[i] + dh * W) * C + cho) * 2) : 0x80000000u;
            }
        }
        const int kofs = kc * kTileK * 2;
#pragma unroll
        for (int i = 0; i < A_MAX; ++i)
            if (i * NW + wave < nA)
                buffer_copy16(X, P.x_bytes, wv[i] + kofs, 0,
                              (lds_void*)(slot + (i * NW + wave) * 64));
        const int rk = th.r0 + r * th.rstep;
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
            const int sl = ((i * NW + wave) * 8) / BN;           // weight slice (uniform)
            const int s2 = sl < ns ? sl : ns - 1;
            const int rs = rk * P.s + tw.r0 + s2 * tw.rstep;
            buffer_copy16(Wt, P.w_bytes, wofs[i], rs * K * C * 2 + kofs,
                          (lds_void*)(slot + A_CHUNKS + (i * NW + wave) * 64));
        }
    };

    f32x4 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};

    if (total > 0) copy(0, lds);
    for (int it = 0; it < total; ++it) {
        wait_vmcnt<0>();
        __builtin_amdgcn_s_barrier();   // stage `it` is in LDS everywhere; `it - 1` is consumed
        if (it + 1 < total) copy(it + 1, lds + ((it + 1) & 1) * STAGE_CHUNKS);
        const u32x4* la = lds + (it & 1) * STAGE_CHUNKS;
        const u32x4* lb = la + A_CHUNKS;
        for (int sl = 0; sl < ns; ++sl) {
#pragma unroll
            for (int kk = 0; kk < kTileK / 32; ++kk) {
                const int ch = kk * 4 + (lane >> 4);
                bf16x8 fa[FN], fb[FM];
#pragma unroll
                for (int i = 0; i < FN; ++i)
                    fa[i] = __builtin_bit_cast(
                        bf16x8, lb[tile_swz(sl * BN + wn * WN + i * 16 + (lane & 15), ch)]);
#pragma unroll
                for (int j = 0; j < FM; ++j)
                    fb[j] = __builtin_bit_cast(bf16x8, la[tile_swz(arow[j] + sl, ch)]);
#pragma unroll
                for (int i = 0; i < FN; ++i)
#pragma unroll
                    for (int j = 0; j < FM; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j],
                                                                            acc[i][j], 0, 0, 0);
            }
        }
    }
    store_tile<FM, FN, WM, WN, OT>(P, t, wm, wn, acc, out, epi);
}

// Host-side plan: classes, their taps, and the tile count for a BM x BN tiling.
//
// Taps along one axis of a class, as (kernel index, input offset) pairs in increasing
// kernel index; false if they do not form an arithmetic progression (never the case
// for the forms below, checked anyway).
bool axis_taps(const int* r, const int* b, int n, AxisTaps& a) {
    a = AxisTaps{0, 1, 0, 0, n};
    if (n == 0) return true;
    a.r0 = r[0]; a.b0 = b[0];
    if (n > 1) { a.rstep = r[1] - r[0]; a.bstep = b[1] - b[0]; }
    for (int i = 0; i < n; ++i)
        if (r[i] != a.r0 + i * a.rstep || b[i] != a.b0 + i * a.bstep) return false;
    return true;
}

// One axis of a class with output residue `a` (0 for the forward form):
//   forward:     all taps, input offset -pad + r*dil  (input = stride*i + offset);
//   residues:    all taps, offset a - pad + r*dil     (input = dil*i + offset);
//   transposed:  the taps with (a + pad - r*dil) divisible by the stride, offset
//                (a + pad - r*dil) / stride         (input = i + offset).
bool class_axis(int form, int a, int64_t ksize, int stride, int pad, int dil, AxisTaps& t) {
    if (ksize > 64) return false;
    int r[64], b[64], n = 0;
    for (int k = 0; k < (int)ksize; ++k) {
        if (form == kForward) {
            r[n] = k; b[n++] = -pad + k * dil;
        } else if (form == kResidues) {
            r[n] = k; b[n++] = a - pad + k * dil;
        } else {
            const int th = a + pad - k * dil;
            if (((th % stride) + stride) % stride != 0) continue;
            r[n] = k; b[n++] = th / stride;   // exact: th is a multiple of the stride
        }
    }
    return axis_taps(r, b, n, t);
}

bool make_plan(const ConvGeom& g, int form, FusedPlan& P) {
    P = FusedPlan{};
    P.n = (int)g.n; P.c = (int)g.c; P.h = (int)g.h; P.w = (int)g.w; P.k = (int)g.k;
    P.ho = (int)g.ho; P.wo = (int)g.wo; P.s = (int)g.s;
    const int64_t xb = g.n * g.h * g.w * g.c * 2, wb = g.r * g.s * g.k * g.c * 2;
    P.x_bytes = xb < (int64_t(1) << 31) && wb < (int64_t(1) << 31) ? (int)xb : 0;
    P.w_bytes = P.x_bytes ? (int)wb : 0;
    // classes: output residues modulo gamma (the stride of the transposed form, the
    // dilation of the residue form (section 6.2), 1 for the forward form)
    int gh = 1, gw = 1;
    if (form == kResidues) {
        if (g.sh != 1 || g.sw != 1) return false;
        gh = g.dh; gw = g.dw;
        P.alpha_h = g.dh; P.alpha_w = g.dw;
    } else if (form == kForward) {
        P.alpha_h = g.sh; P.alpha_w = g.sw;
    } else {
        gh = g.sh; gw = g.sw;
        P.alpha_h = 1; P.alpha_w = 1;
    }
    if ((int64_t)gh * gw > kMaxCls) return false;
    P.gam_h = gh; P.gam_w = gw;
    int ncls = 0;
    for (int ah = 0; ah < gh; ++ah)
        for (int aw = 0; aw < gw; ++aw) {
            const int hc = ah < g.ho ? (int)((g.ho - ah + gh - 1) / gh) : 0;
            const int wc = aw < g.wo ? (int)((g.wo - aw + gw - 1) / gw) : 0;
            if (hc == 0 || wc == 0) continue;
            P.cls_hc[ncls] = hc; P.cls_wc[ncls] = wc;
            P.cls_oh0[ncls] = ah; P.cls_ow0[ncls] = aw;
            if (!class_axis(form, ah, g.r, g.sh, g.ph, g.dh, P.cls_th[ncls]) ||
                !class_axis(form, aw, g.s, g.sw, g.pw, g.dw, P.cls_tw[ncls]))
                return false;
            ++ncls;
        }
    P.ncls = ncls;
    return ncls > 0;
}

int64_t plan_tiles(FusedPlan& P, int bm, int bn) {
    P.tiles_n = (P.k + bn - 1) / bn;
    int64_t t = 0;
    for (int c = 0; c < P.ncls; ++c) {
        P.cls_tile0[c] = (int)t;
        const int64_t mc = (int64_t)P.n * P.cls_hc[c] * P.cls_wc[c];
        t += ((mc + bm - 1) / bm) * P.tiles_n;
    }
    P.cls_tile0[P.ncls] = (int)t;
    return t;
}

template <int BM, int BN, int NS, typename OT, int NW, bool BUF = true, int KS = 1>
hipError_t go(FusedPlan& P, const void* x, const void* wt, void* out, const Epi& epi,
              hipStream_t st) {
    const int64_t tiles = plan_tiles(P, BM, BN);
    if (tiles == 0) return hipSuccess;
    hipLaunchKernelGGL((conv_fused_kernel<BM, BN, NS, OT, NW, BUF, KS>), dim3((unsigned)tiles),
                       dim3(64 * NW), 0, st, (const bf16_t*)x, (const bf16_t*)wt, (OT*)out, P,
                       epi);
    return hipGetLastError();
}

template <int BM, int BN, int NS, typename OT>
hipError_t go_pipe(FusedPlan& P, const void* x, const void* wt, void* out, const Epi& epi,
                   hipStream_t st) {
    const int64_t tiles = plan_tiles(P, BM, BN);
    if (tiles == 0) return hipSuccess;
    hipLaunchKernelGGL((conv_fused_pipe_kernel<BM, BN, NS, OT>), dim3((unsigned)tiles),
                       dim3(256), 0, st, (const bf16_t*)x, (const bf16_t*)wt, (OT*)out, P, epi);
    return hipGetLastError();
}

// Whether every class fits the row-window kernel.
bool window_ok(const FusedPlan& P) {
    for (int c = 0; c < P.ncls; ++c) {
        const AxisTaps& tw = P.cls_tw[c];
        const int wc = P.cls_wc[c];
        if (wc % 16 != 0 || kWinBM % wc != 0 || tw.n < 1 || tw.n > kWinS) return false;
        if (tw.n > 1 && tw.bstep != P.alpha_w) return false;
        if ((kWinBM / wc) * (wc + tw.n - 1) > kWinArows) return false;
    }
    return true;
}

template <typename OT>
hipError_t go_window(FusedPlan& P, const void* x, const void* wt, void* out, const Epi& epi,
                     hipStream_t st) {
    const int64_t tiles = plan_tiles(P, kWinBM, kWinBN);
    if (tiles == 0) return hipSuccess;
    hipLaunchKernelGGL((conv_window_kernel<OT>), dim3((unsigned)tiles), dim3(512), 0, st,
                       (const bf16_t*)x, (const bf16_t*)wt, (OT*)out, P, epi);
    return hipGetLastError();
}

// Tile shapes: 0 = 192x128 with 8 waves (one workgroup per CU), 1 = 128x128 with 8 waves
// (two per CU), 2 = 64x128 with 4 waves, 3 = 64x64 with 8 waves and a 4-stage copy ring;
// 4-8 = the software-pipelined four-wave form with 192x128, 128x128, 64x64, 128x64 and
// 256x128 tiles; 9 = the row-window kernel (192x128); 10-12 = the eight-wave kernel with
// the k-tile split between the two halves of the waves, 192x128, 128x128 and 64x64
// (4-stage ring).  Automatic choice: 10 when there is ~one 192x128 tile per CU, else 1
// or 2 at that count, else 12 (measured fastest on the CSRNet, ResNet and DCGAN layers:
// 65-68 vs 68-69 us for 0, 12.2 vs 13.8 us and 11.3 vs 12.9 us for 6).  The row-window
// kernel copies 35% fewer bytes on the CSRNet layer in the residue form but measured no
// faster than 0 there (its copies overlap less with the MFMA work), so it is selected
// only on request.  `forced` (0..14, from the caller's flags; -1 = automatic) overrides
// the choice for tuning sweeps and tests; 9 falls back to the automatic choice where
// the row-window form does not apply.
template <typename OT>
hipError_t dispatch(FusedPlan& P, const void* x, const void* wt, void* out, const Epi& epi,
                    int forced, hipStream_t st) {
    // tensors of 2 GiB or more: 64-bit addressing (buffer offsets are 32-bit)
    if (P.x_bytes == 0 || P.w_bytes == 0) return go<128, 128, 2, OT, 8, false>(P, x, wt, out, epi, st);
    int cfg = forced;
    if (cfg == 9 && !window_ok(P)) cfg = -1;
    if (cfg < 0 || cfg > 14) {
        FusedPlan tmp = P;
        // k-tiles of the longest class contraction
        int steps = 0;
        for (int c = 0; c < P.ncls; ++c) {
            const int n = P.cls_th[c].n * P.cls_tw[c].n * (P.c / kTileK);
            steps = n > steps ? n : steps;
        }
        // output-channel tiles no wider than K (a wider tile multiplies padding)
        if (P.k <= 32 && plan_tiles(tmp, 128, 32) >= 240) cfg = 13;
        else if (P.k <= 64) cfg = 12;
        // a short contraction: the k split's final reduction does not pay
        else if (steps < 16 && plan_tiles(tmp, 128, 128) >= 240) cfg = 1;
        else if (plan_tiles(tmp, 192, 128) >= 240) cfg = 10;
        else if (plan_tiles(tmp, 128, 128) >= 240) cfg = 1;
        else if (plan_tiles(tmp, 64, 128) >= 240) cfg = 2;
        else cfg = 12;
    }
    switch (cfg) {
    case 0: return go<192, 128, 2, OT, 8>(P, x, wt, out, epi, st);
    case 1: return go<128, 128, 2, OT, 8>(P, x, wt, out, epi, st);
    case 2: return go<64, 128, 2, OT, 4>(P, x, wt, out, epi, st);
    case 3: return go<64, 64, 4, OT, 8>(P, x, wt, out, epi, st);
    case 4: return go_pipe<192, 128, 3, OT>(P, x, wt, out, epi, st);
    case 5: return go_pipe<128, 128, 3, OT>(P, x, wt, out, epi, st);
    case 6: return go_pipe<64, 64, 4, OT>(P, x, wt, out, epi, st);
    case 7: return go_pipe<128, 64, 4, OT>(P, x, wt, out, epi, st);
    case 8: return go_pipe<256, 128, 3, OT>(P, x, wt, out, epi, st);
    case 9: return go_window<OT>(P, x, wt, out, epi, st);
    case 10: return go<192, 128, 2, OT, 8, true, 2>(P, x, wt, out, epi, st);
    case 11: return go<128, 128, 2, OT, 8, true, 2>(P, x, wt, out, epi, st);
    case 12: return go<64, 64, 4, OT, 8, true, 2>(P, x, wt, out, epi, st);
    case 13: return go<128, 32, 4, OT, 4>(P, x, wt, out, epi, st);
    case 14: return go<256, 32, 3, OT, 4>(P, x, wt, out, epi, st);
    // the small shapes run right after other kernels have evicted their operands: a
    // 4-deep copy ring hides the longer cold loads (measured in the benchmark step)
    default: return go_pipe<64, 64, 4, OT>(P, x, wt, out, epi, st);
    }
}

}  // namespace

bool conv_fused_supported(const ConvGeom& g, int form) {
    if (g.c % kTileK != 0) return false;
    FusedPlan P;
    return make_plan(g, form, P);
}

hipError_t launch_conv_fused(const ConvGeom& g, int form, const void* x, const void* wt,
                             void* out, int out_bf16, const Epi& epi, int tile,
                             hipStream_t stream) {
    FusedPlan P;
    if (g.c % kTileK != 0 || !make_plan(g, form, P)) return hipErrorInvalidValue;
    return out_bf16 ? dispatch<bf16_t>(P, x, wt, out, epi, tile, stream)
                    : dispatch<float>(P, x, wt, out, epi, tile, stream);
}

}  // namespace ollie
