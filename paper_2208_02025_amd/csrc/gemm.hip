// GEMM stage of the derived convolution forms: the matched Matmul scope
//   Y[m][n] = sum_kk A[m][kk] * B[n][kk]
// with A = X viewed as A'[m][c] (Eq. 3) and B = Wt viewed as K'^T[n][c] (Eq. 4).
// Both operands are K-contiguous ("NT"), which is the natural operand order of the
// CDNA matrix cores: every lane feeds one row and 8 consecutive k of each operand.
//
// bf16 main path (k % 64 == 0): v_mfma_f32_16x16x32_bf16 with fp32 accumulation.
//   * 64-deep k-tiles of both operands are copied global -> LDS by
//     global_load_lds_dwordx4 (no register staging).  One such instruction writes
//     64 lanes x 16 bytes contiguously at the wave-uniform LDS base, so the 16-byte
//     chunk XOR swizzle (conflict-free ds_read_b128 fragments) is applied on the
//     source side: the lane that fills LDS chunk slot p of row r fetches logical
//     chunk p ^ (r & 7).
//   * NSTAGE LDS buffers form a ring; loads for k-tile kt + NSTAGE - 1 are in flight
//     while k-tile kt is multiplied, with explicit vmcnt waits.
//   * Rows past m or n are clamped to the last valid row (their products only reach
//     rows/columns of Y that are never stored).
// bf16 fallback (any k % 8 == 0): register-staged double-buffered 128x128 tiles.
// fp32 path: v_mfma_f32_16x16x4_f32 (small problems; any k).
//
// The MFMA is issued as D = Wt-tile x X-tile^T so that each lane ends up holding four
// consecutive output columns n of one row m: the epilogue writes 16-byte vectors.
#include <stdlib.h>

#include "common.h"

namespace ollie {

namespace {

constexpr int kBK = kTileK;
constexpr int kChunks = kTileChunks;

__device__ __forceinline__ int swz(int row, int ch) { return tile_swz(row, ch); }

// XCD-aware tile order: consecutive workgroup ids are dealt round-robin to the 8 XCDs.
// Remap so that each XCD receives a contiguous range of tiles (which then share
// operand rows in its own L2), and walk tiles in groups of `group_m` tile-rows so
// that a group's B columns stay hot.
__device__ __forceinline__ void tile_of(int bid, int nblk, int tiles_m, int tiles_n,
                                        int& tm, int& tn) {
    int id = bid;
    if ((nblk & 7) == 0) {
        int per = nblk >> 3;
        id = (bid & 7) * per + (bid >> 3);
    }
    const int group_m = 8;
    int group = id / (group_m * tiles_n);
    int first_m = group * group_m;
    int gsize = tiles_m - first_m < group_m ? tiles_m - first_m : group_m;
    int in_group = id - group * group_m * tiles_n;
    tm = first_m + in_group % gsize;
    tn = in_group / gsize;
}

// Epilogue: acc[i][j][v] = Y[m][n], m = m0 + row0 + j*16 + lane%16,
//                                    n = n0 + col0 + i*16 + 4*(lane/16) + v.
template <int FM, int FN, typename YT>
__device__ __forceinline__ void store_tile(YT* __restrict__ Y, const f32x4 (&acc)[FN][FM],
                                           int64_t M, int64_t N, int64_t mb, int64_t nb) {
    const int lane = threadIdx.x & 63;
    const bool vec_ok = (N & 3) == 0;
#pragma unroll
    for (int j = 0; j < FM; ++j) {
        const int64_t m = mb + j * 16 + (lane & 15);
        if (m >= M) continue;
#pragma unroll
        for (int i = 0; i < FN; ++i) {
            const int64_t n = nb + i * 16 + 4 * (lane >> 4);
            YT* dst = Y + m * N + n;
            if (vec_ok && n + 3 < N) {
                Out<YT>::put4(dst, acc[i][j]);
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    if (n + v < N) Out<YT>::put(dst + v, acc[i][j][v]);
            }
        }
    }
}

// ------------------------------------------------------------------ main bf16 path
template <int BM, int BN, int BK, int NSTAGE, typename YT>
__global__ __launch_bounds__(256, (NSTAGE * (BM + BN) * BK * 2 <= 80 * 1024) ? 2 : 1)
void gemm_nt_bf16_dma_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ B,
                             YT* __restrict__ Y, int64_t M, int64_t N, int64_t K, int tiles_m,
                             int tiles_n) {
    constexpr int WM = BM / 2, WN = BN / 2;        // wave sub-tile (2 x 2 waves)
    constexpr int FM = WM / 16, FN = WN / 16;      // 16x16 MFMA blocks per wave
    constexpr int CPR = BK / 8;                    // 16-byte chunks per tile row
    constexpr int RPI = 64 / CPR;                  // tile rows per wave-wide DMA instruction
    constexpr int ROWS = BM + BN;                  // tile rows per stage (A rows, then B rows)
    constexpr int STAGE_CHUNKS = ROWS * CPR;
    constexpr int LOADS = STAGE_CHUNKS / 256;      // DMA instructions per wave per stage
    static_assert(STAGE_CHUNKS % 256 == 0, "stage must be a whole number of wave loads");
    __shared__ u32x4 lds[NSTAGE * STAGE_CHUNKS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    int tm, tn;
    tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
    const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;

    // Per-lane source rows for this wave's DMA instructions.  Instruction i of wave w
    // fills LDS chunk slots [(i*4 + w)*64, +64): rows (i*4+w)*RPI + lane/CPR, slot lane%CPR.
    const bf16_t* src[LOADS];
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
        const int row = (i * 4 + wave) * RPI + lane / CPR;
        const int slot = lane % CPR;
        // the lane filling slot `slot` of `row` fetches the chunk the swizzle puts there
        int ch = 0;
#pragma unroll
        for (int c = 0; c < CPR; ++c)
            if (tile_swz_k<BK>(row, c) - row * CPR == slot) ch = c;
        const bf16_t* p;
        if (row < BM) {
            int64_t gm = m0 + row;
            gm = gm < M ? gm : M - 1;
            p = A + gm * K + ch * 8;
        } else {
            int64_t gn = n0 + (row - BM);
            gn = gn < N ? gn : N - 1;
            p = B + gn * K + ch * 8;
        }
        src[i] = p;
    }
    auto issue = [&](int kt, int buf) {
        const int64_t koff = (int64_t)kt * BK;
#pragma unroll
        for (int i = 0; i < LOADS; ++i)
            __builtin_amdgcn_global_load_lds(
                (const void*)(src[i] + koff),
                (lds_void*)(lds + buf * STAGE_CHUNKS + (i * 4 + wave) * 64), 16, 0, 0);
    };

    f32x4 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};

    const int ktiles = (int)(K / BK);
#pragma unroll
    for (int s = 0; s < NSTAGE - 1; ++s)
        if (s < ktiles) issue(s, s);

    for (int kt = 0; kt < ktiles; ++kt) {
        // k-tile kt has landed once at most (NSTAGE-2) later tiles' loads are pending
        if (kt + NSTAGE - 2 < ktiles) wait_vmcnt<(NSTAGE - 2) * LOADS>();
        else wait_vmcnt<0>();
        __builtin_amdgcn_s_barrier();   // every wave's part of tile kt is in LDS; tile kt-1 is consumed
        if (kt + NSTAGE - 1 < ktiles) issue(kt + NSTAGE - 1, (kt + NSTAGE - 1) % NSTAGE);
        const u32x4* la = lds + (kt % NSTAGE) * STAGE_CHUNKS;
        const u32x4* lb = la + BM * CPR;
#pragma unroll
        for (int kk = 0; kk < BK / 32; ++kk) {
            const int ch = kk * 4 + (lane >> 4);
            bf16x8 fa[FN], fb[FM];
#pragma unroll
            for (int i = 0; i < FN; ++i)
                fa[i] = __builtin_bit_cast(
                    bf16x8, lb[tile_swz_k<BK>(wn * WN + i * 16 + (lane & 15), ch)]);
#pragma unroll
            for (int j = 0; j < FM; ++j)
                fb[j] = __builtin_bit_cast(
                    bf16x8, la[tile_swz_k<BK>(wm * WM + j * 16 + (lane & 15), ch)]);
#pragma unroll
            for (int i = 0; i < FN; ++i)
#pragma unroll
                for (int j = 0; j < FM; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j],
                                                                        0, 0, 0);
        }
    }
    store_tile<FM, FN, YT>(Y, acc, M, N, m0 + wm * WM, n0 + wn * WN);
}

// --------------------------------------------------------- persistent bf16 path
// One workgroup per CU walks a strided list of tiles.  The LDS ring runs across tile
// boundaries: the first k-tiles of the next tile are already in flight while the
// current tile finishes, and its Y stores drain under the next tile's loads and MFMAs.
// The vmcnt bookkeeping assumes vector-memory operations retire in issue order: at
// iteration `it` the wait allows exactly the loads issued for later k-tiles plus the
// stores of an epilogue issued after k-tile `it`'s loads.  Interior tiles store with a
// fixed instruction count; a tile with ragged rows or columns waits for everything.
template <int BM, int BN, int NSTAGE, int WAVES_M, int WAVES_N, typename YT>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N, 1) void gemm_nt_bf16_persistent_kernel(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ B, YT* __restrict__ Y,
    int64_t M, int64_t N, int64_t K, int tiles_m, int tiles_n) {
    constexpr int NW = WAVES_M * WAVES_N;
    constexpr int NT = 64 * NW;
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int FM = WM / 16, FN = WN / 16;
    constexpr int ROWS = BM + BN;
    constexpr int STAGE_CHUNKS = ROWS * kChunks;
    constexpr int LOADS = STAGE_CHUNKS / NT;          // DMA instructions per wave per stage
    constexpr int A_LOADS = BM * kChunks / NT;        // the first A_LOADS of them fetch A rows
    constexpr int STORES = FM * FN;                   // store instructions of an interior epilogue
    static_assert(STAGE_CHUNKS % NT == 0 && (BM * kChunks) % NT == 0, "whole wave loads");
    // waits allow at most 63 outstanding operations; a larger count is clamped, which
    // only makes the wait stricter (operations retire in order)
    constexpr int W_LS = LOADS * (NSTAGE - 2) + STORES < 63 ? LOADS * (NSTAGE - 2) + STORES : 63;
    constexpr int W_L = LOADS * (NSTAGE - 2) < 63 ? LOADS * (NSTAGE - 2) : 63;
    constexpr int W_S = STORES < 63 ? STORES : 63;
    __shared__ u32x4 lds[NSTAGE * STAGE_CHUNKS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int ntiles = tiles_m * tiles_n;
    const int G = gridDim.x;
    const int w = blockIdx.x;
    // XCD-compact assignment: at round i, the G/8 workgroups of one XCD take a
    // contiguous run of the grouped tile order.
    const int slot = (G & 7) == 0 ? (w & 7) * (G >> 3) + (w >> 3) : w;
    const int my_tiles = slot < ntiles ? (ntiles - 1 - slot) / G + 1 : 0;
    const int ktiles = (int)(K / kBK);
    const int total = my_tiles * ktiles;

    auto coords = [&](int i, int64_t& m0, int64_t& n0) {
        // grouped order only (the XCD spreading is already in `slot`)
        const int id = i * G + slot;
        const int group_m = 8;
        const int group = id / (group_m * tiles_n);
        const int first_m = group * group_m;
        const int gsize = tiles_m - first_m < group_m ? tiles_m - first_m : group_m;
        const int in_group = id - group * group_m * tiles_n;
        m0 = (int64_t)(first_m + in_group % gsize) * BM;
        n0 = (int64_t)(in_group / gsize) * BN;
    };
    auto issue = [&](int it) {
        const int ti = it / ktiles, kt = it - ti * ktiles;
        int64_t m0, n0;
        coords(ti, m0, n0);
        const int buf = it % NSTAGE;
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int seg = i * NW + wave;
            const int row = seg * 8 + (lane >> 3);
            const int ch = (lane & 7) ^ (row & 7);
            const bf16_t* p;
            if (i < A_LOADS) {
                int64_t gm = m0 + row;
                gm = gm < M ? gm : M - 1;
                p = A + gm * K;
            } else {
                int64_t gn = n0 + (row - BM);
                gn = gn < N ? gn : N - 1;
                p = B + gn * K;
            }
            __builtin_amdgcn_global_load_lds((const void*)(p + (int64_t)kt * kBK + ch * 8),
                                             (lds_void*)(lds + buf * STAGE_CHUNKS + seg * 64),
                                             16, 0, 0);
        }
    };

    f32x4 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int s = 0; s < NSTAGE - 1; ++s)
        if (s < total) issue(s);

    int last_epi = -1000;       // iteration whose epilogue was the most recent
    bool last_epi_edge = false;
    for (int it = 0; it < total; ++it) {
        // loads issued after k-tile it's: min(NSTAGE-2, total-1-it) stages; stores after
        // it: an epilogue at iteration e in [it-NSTAGE+1, it-1]
        const int later = (total - 1 - it) < (NSTAGE - 2) ? (total - 1 - it) : (NSTAGE - 2);
        const bool epi = last_epi >= it - NSTAGE + 1;
        if (epi && last_epi_edge) {
            wait_vmcnt<0>();
        } else if constexpr (NSTAGE == 3) {
            if (later == 1) {
                if (epi) wait_vmcnt<W_LS>();
                else wait_vmcnt<W_L>();
            } else {
                if (epi) wait_vmcnt<W_S>();
                else wait_vmcnt<0>();
            }
        } else {
            static_assert(NSTAGE == 2, "two or three stages");
            if (epi) wait_vmcnt<W_S>();
            else wait_vmcnt<0>();
        }
        __builtin_amdgcn_s_barrier();
        if (it + NSTAGE - 1 < total) issue(it + NSTAGE - 1);
        const u32x4* la = lds + (it % NSTAGE) * STAGE_CHUNKS;
        const u32x4* lb = la + BM * kChunks;
#pragma unroll
        for (int kk = 0; kk < kBK / 32; ++kk) {
            const int ch = kk * 4 + (lane >> 4);
            bf16x8 fa[FN], fb[FM];
#pragma unroll
            for (int i = 0; i < FN; ++i)
                fa[i] = __builtin_bit_cast(bf16x8, lb[swz(wn * WN + i * 16 + (lane & 15), ch)]);
#pragma unroll
            for (int j = 0; j < FM; ++j)
                fb[j] = __builtin_bit_cast(bf16x8, la[swz(wm * WM + j * 16 + (lane & 15), ch)]);
#pragma unroll
            for (int i = 0; i < FN; ++i)
#pragma unroll
                for (int j = 0; j < FM; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j],
                                                                        0, 0, 0);
        }
        if ((it + 1) % ktiles == 0) {
            int64_t m0, n0;
            coords(it / ktiles, m0, n0);
            const bool interior = m0 + BM <= M && n0 + BN <= N && (N & 3) == 0;
            const int64_t mb = m0 + wm * WM, nb = n0 + wn * WN;
            if (interior) {
#pragma unroll
                for (int j = 0; j < FM; ++j) {
                    const int64_t m = mb + j * 16 + (lane & 15);
#pragma unroll
                    for (int i = 0; i < FN; ++i)
                        Out<YT>::put4(Y + m * N + nb + i * 16 + 4 * (lane >> 4), acc[i][j]);
                }
            } else {
                store_tile<FM, FN, YT>(Y, acc, M, N, mb, nb);
            }
            last_epi = it;
            last_epi_edge = !interior;
#pragma unroll
            for (int i = 0; i < FN; ++i)
#pragma unroll
                for (int j = 0; j < FM; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};
        }
    }
}

// -------------------------------------------------------- register-staged bf16 fallback
template <int BM, int BN, typename YT>
__global__ __launch_bounds__(256) void gemm_nt_bf16_kernel(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ B, YT* __restrict__ Y,
    int64_t M, int64_t N, int64_t K, int tiles_m, int tiles_n) {
    constexpr int WM = BM / 2, WN = BN / 2;        // wave sub-tile (2 x 2 waves)
    constexpr int FM = WM / 16, FN = WN / 16;      // 16x16 MFMA blocks per wave
    constexpr int A_PER = BM * kChunks / 256;      // 16-byte global loads per thread
    constexpr int B_PER = BN * kChunks / 256;
    __shared__ u32x4 lds[2][(BM + BN) * kChunks];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    int tm, tn;
    tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
    const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;

    u32x4 ra[A_PER], rb[B_PER];
    auto gload = [&](int64_t k0) {
#pragma unroll
        for (int i = 0; i < A_PER; ++i) {
            int idx = tid + i * 256;
            int row = idx / kChunks, ch = idx % kChunks;
            int64_t gm = m0 + row, gk = k0 + ch * 8;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (gm < M && gk < K) v = *reinterpret_cast<const u32x4*>(A + gm * K + gk);
            ra[i] = v;
        }
#pragma unroll
        for (int i = 0; i < B_PER; ++i) {
            int idx = tid + i * 256;
            int row = idx / kChunks, ch = idx % kChunks;
            int64_t gn = n0 + row, gk = k0 + ch * 8;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (gn < N && gk < K) v = *reinterpret_cast<const u32x4*>(B + gn * K + gk);
            rb[i] = v;
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_PER; ++i) {
            int idx = tid + i * 256;
            lds[buf][swz(idx / kChunks, idx % kChunks)] = ra[i];
        }
#pragma unroll
        for (int i = 0; i < B_PER; ++i) {
            int idx = tid + i * 256;
            lds[buf][BM * kChunks + swz(idx / kChunks, idx % kChunks)] = rb[i];
        }
    };

    f32x4 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};

    const int ktiles = (int)((K + kBK - 1) / kBK);
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < ktiles; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < ktiles) gload((int64_t)(kt + 1) * kBK);
#pragma unroll
        for (int kk = 0; kk < kBK / 32; ++kk) {
            const int ch = kk * 4 + (lane >> 4);
            bf16x8 fa[FN], fb[FM];
#pragma unroll
            for (int i = 0; i < FN; ++i) {
                int row = wn * WN + i * 16 + (lane & 15);
                fa[i] = __builtin_bit_cast(bf16x8, lds[cur][BM * kChunks + swz(row, ch)]);
            }
#pragma unroll
            for (int j = 0; j < FM; ++j) {
                int row = wm * WM + j * 16 + (lane & 15);
                fb[j] = __builtin_bit_cast(bf16x8, lds[cur][swz(row, ch)]);
            }
#pragma unroll
            for (int i = 0; i < FN; ++i)
#pragma unroll
                for (int j = 0; j < FM; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j],
                                                                        0, 0, 0);
        }
        if (kt + 1 < ktiles) lstore(cur ^ 1);
        __syncthreads();
    }
    store_tile<FM, FN, YT>(Y, acc, M, N, m0 + wm * WM, n0 + wn * WN);
}

// fp32 operands: 64x64 tile, 16-deep k-tile, scalar staged loads (any shape).
template <typename YT>
__global__ __launch_bounds__(256) void gemm_nt_f32_kernel(
    const float* __restrict__ A, const float* __restrict__ B, YT* __restrict__ Y,
    int64_t M, int64_t N, int64_t K, int tiles_m, int tiles_n) {
    constexpr int BM = 64, BN = 64, BKF = 16, LD = BKF + 1;
    __shared__ float la[BM * LD];
    __shared__ float lb[BN * LD];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
    const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};

    for (int64_t k0 = 0; k0 < K; k0 += BKF) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            int idx = tid + e * 256;
            int row = idx / BKF, kk = idx % BKF;
            int64_t gk = k0 + kk;
            int64_t gm = m0 + row, gn = n0 + row;
            la[row * LD + kk] = (gm < M && gk < K) ? A[gm * K + gk] : 0.f;
            lb[row * LD + kk] = (gn < N && gk < K) ? B[gn * K + gk] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < BKF / 4; ++ks) {
            int kk = ks * 4 + (lane >> 4);
            float fa[2], fb[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) fa[i] = lb[(wn * 32 + i * 16 + (lane & 15)) * LD + kk];
#pragma unroll
            for (int j = 0; j < 2; ++j) fb[j] = la[(wm * 32 + j * 16 + (lane & 15)) * LD + kk];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i], fb[j], acc[i][j],
                                                                     0, 0, 0);
        }
        __syncthreads();
    }
    store_tile<2, 2, YT>(Y, acc, M, N, m0 + wm * 32, n0 + wn * 32);
}

template <int BM, int BN, int BK, int NSTAGE, typename YT>
hipError_t go_dma(int64_t m, int64_t n, int64_t k, const void* a, const void* b, void* y,
                  hipStream_t stream) {
    int tiles_m = (int)((m + BM - 1) / BM), tiles_n = (int)((n + BN - 1) / BN);
    hipLaunchKernelGGL((gemm_nt_bf16_dma_kernel<BM, BN, BK, NSTAGE, YT>), dim3(tiles_m * tiles_n),
                       dim3(256), 0, stream, (const bf16_t*)a, (const bf16_t*)b, (YT*)y, m, n, k,
                       tiles_m, tiles_n);
    return hipGetLastError();
}

int num_cus() {
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (!cached[dev]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        cached[dev] = n;
    }
    return cached[dev];
}

template <int BM, int BN, int NSTAGE, int WAVES_M, int WAVES_N, typename YT>
hipError_t go_persistent(int64_t m, int64_t n, int64_t k, const void* a, const void* b, void* y,
                         hipStream_t stream) {
    const int tiles_m = (int)((m + BM - 1) / BM), tiles_n = (int)((n + BN - 1) / BN);
    const int ntiles = tiles_m * tiles_n;
    const int cus = num_cus();
    const int grid = ntiles < cus ? ntiles : cus;
    hipLaunchKernelGGL((gemm_nt_bf16_persistent_kernel<BM, BN, NSTAGE, WAVES_M, WAVES_N, YT>),
                       dim3(grid), dim3(64 * WAVES_M * WAVES_N), 0, stream, (const bf16_t*)a,
                       (const bf16_t*)b, (YT*)y, m, n, k, tiles_m, tiles_n);
    return hipGetLastError();
}

// Tile configuration of the DMA kernels: 0 = 256x128, 3 stages (one workgroup per CU);
// 1 = 128x128, 3 stages (one per CU); 2 = 128x128, 2 stages (two per CU);
// 3 = persistent 256x256, 2 stages, 8 waves; 4 = persistent 256x128, 3 stages, 4 waves;
// 5 = 128x256 and 6 = 256x128 with 32-deep k-tiles, 3 stages (two workgroups per CU);
// 7 = 128x128, 32-deep k-tiles, 4 stages.
// OLLIE_GEMM_CONFIG (0..7) overrides the shape-based choice, for tuning sweeps.
int pick_config(int64_t m, int64_t n) {
    static const int forced = [] {
        const char* e = getenv("OLLIE_GEMM_CONFIG");
        return e ? atoi(e) : -1;
    }();
    if (forced >= 0 && forced <= 7) return forced;
    const int64_t t128 = ((m + 127) / 128) * ((n + 127) / 128);
    if (t128 > 256) return 2;           // two workgroups per CU hide each other's latency
    return 1;
}

template <typename YT>
hipError_t go_bf16(int64_t m, int64_t n, int64_t k, const void* a, const void* b, void* y,
                   hipStream_t stream) {
    if (k % kBK == 0) {
        int cfg = pick_config(m, n);
        if (cfg >= 3 && k / kBK < 2) cfg = 2;    // the cross-tile ring needs >= 2 k-tiles
        switch (cfg) {
        case 3: return go_persistent<256, 256, 2, 2, 4, YT>(m, n, k, a, b, y, stream);
        case 4: return go_persistent<256, 128, 3, 2, 2, YT>(m, n, k, a, b, y, stream);
        case 0: return go_dma<256, 128, 64, 3, YT>(m, n, k, a, b, y, stream);
        case 1: return go_dma<128, 128, 64, 3, YT>(m, n, k, a, b, y, stream);
        case 5: return go_dma<128, 256, 32, 3, YT>(m, n, k, a, b, y, stream);
        case 6: return go_dma<256, 128, 32, 3, YT>(m, n, k, a, b, y, stream);
        case 7: return go_dma<128, 128, 32, 4, YT>(m, n, k, a, b, y, stream);
        default: return go_dma<128, 128, 64, 2, YT>(m, n, k, a, b, y, stream);
        }
    }
    int tiles_m = (int)((m + 127) / 128), tiles_n = (int)((n + 127) / 128);
    hipLaunchKernelGGL((gemm_nt_bf16_kernel<128, 128, YT>), dim3(tiles_m * tiles_n), dim3(256),
                       0, stream, (const bf16_t*)a, (const bf16_t*)b, (YT*)y, m, n, k, tiles_m,
                       tiles_n);
    return hipGetLastError();
}

template <typename YT>
hipError_t go_f32(int64_t m, int64_t n, int64_t k, const void* a, const void* b, void* y,
                  hipStream_t stream) {
    int tiles_m = (int)((m + 63) / 64), tiles_n = (int)((n + 63) / 64);
    hipLaunchKernelGGL((gemm_nt_f32_kernel<YT>), dim3(tiles_m * tiles_n), dim3(256), 0, stream,
                       (const float*)a, (const float*)b, (YT*)y, m, n, k, tiles_m, tiles_n);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_nt(int64_t m, int64_t n, int64_t k, const void* a, const void* b,
                          void* y, int in_bf16, int y_bf16, hipStream_t stream) {
    if (in_bf16)
        return y_bf16 ? go_bf16<bf16_t>(m, n, k, a, b, y, stream)
                      : go_bf16<float>(m, n, k, a, b, y, stream);
    return y_bf16 ? go_f32<bf16_t>(m, n, k, a, b, y, stream)
                  : go_f32<float>(m, n, k, a, b, y, stream);
}

}  // namespace ollie
