// GEMM stage of the derived convolution forms: the matched Matmul scope
//   Y[m][n] = sum_kk A[m][kk] * B[n][kk]
// with A = X viewed as A'[m][c] (Eq. 3) and B = Wt viewed as K'^T[n][c] (Eq. 4).
// Both operands are K-contiguous ("NT"), which is the natural operand order of the
// CDNA matrix cores: every lane feeds one row and 8 consecutive k of each operand.
//
// bf16 path: v_mfma_f32_16x16x32_bf16, fp32 accumulation, LDS-staged double-buffered
// 64-deep k-tiles with an XOR swizzle of 16-byte chunks (conflict-free ds_read_b128).
// fp32 path: v_mfma_f32_16x16x4_f32 (small problems; any k).
//
// The MFMA is issued as D = Wt-tile x X-tile^T so that each lane ends up holding four
// consecutive output columns n of one row m: the epilogue writes 16-byte vectors.
#include "common.h"

namespace ollie {

namespace {

constexpr int kBK = 64;            // bf16 k-tile depth (128 bytes per row)
constexpr int kChunks = kBK / 8;   // 16-byte chunks per tile row

__device__ __forceinline__ int swz(int row, int ch) {
    return row * kChunks + (ch ^ (row & 7));
}

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
    const int wave = tid >> 6;
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

    // acc[i][j][v] = Y[m][n] with m = m0 + wm*WM + j*16 + lane%16,
    //                              n = n0 + wn*WN + i*16 + 4*(lane/16) + v.
    const bool vec_ok = (N & 3) == 0;
#pragma unroll
    for (int j = 0; j < FM; ++j) {
        int64_t m = m0 + wm * WM + j * 16 + (lane & 15);
        if (m >= M) continue;
#pragma unroll
        for (int i = 0; i < FN; ++i) {
            int64_t n = n0 + wn * WN + i * 16 + 4 * (lane >> 4);
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
    const int wave = tid >> 6;
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
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        int64_t m = m0 + wm * 32 + j * 16 + (lane & 15);
        if (m >= M) continue;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            int64_t n = n0 + wn * 32 + i * 16 + 4 * (lane >> 4);
#pragma unroll
            for (int v = 0; v < 4; ++v)
                if (n + v < N) Out<YT>::put(Y + m * N + n + v, acc[i][j][v]);
        }
    }
}

template <int BM, int BN, typename YT>
hipError_t go_bf16(int64_t m, int64_t n, int64_t k, const void* a, const void* b, void* y,
                   hipStream_t stream) {
    int tiles_m = (int)((m + BM - 1) / BM), tiles_n = (int)((n + BN - 1) / BN);
    hipLaunchKernelGGL((gemm_nt_bf16_kernel<BM, BN, YT>), dim3(tiles_m * tiles_n), dim3(256),
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
        return y_bf16 ? go_bf16<128, 128, bf16_t>(m, n, k, a, b, y, stream)
                      : go_bf16<128, 128, float>(m, n, k, a, b, y, stream);
    return y_bf16 ? go_f32<bf16_t>(m, n, k, a, b, y, stream)
                  : go_f32<float>(m, n, k, a, b, y, stream);
}

}  // namespace ollie
