// Weight side of the derived form that evaluates an R x S convolution as a 3x3 one
// (the Conv5x5 -> Conv3x3 transformation, section 6 and Table 3).  The kernel's tap
// range is relaxed to whole 3x3 blocks (boundary relaxing, section 4.2, with zero
// weights in the added taps), the tap index is substituted as r = 3a + r',
// s = 3b + s' (variable substitution), and the blocks (a, b) become output-channel
// groups of one 3x3 weight:
//   W3[r'][s'][(a*nbs + b)*K + k][c] = Wt[3a + r'][3b + s'][k][c], 0 outside R x S.
// Like the layout change of the weights themselves, this depends on the weights only
// (compile-time evaluation, section 5.4); it is one element-wise pass.
#include "common.h"

namespace ollie {

namespace {

template <typename T>
__global__ __launch_bounds__(256) void split_weights_3x3_kernel(const T* __restrict__ wt,
                                                                T* __restrict__ w3, int R, int S,
                                                                int K, int C, int nbs,
                                                                int64_t total) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const int c = (int)(i % C);
    int64_t t = i / C;
    const int k3 = (int)(total / ((int64_t)9 * C));     // nbr * nbs * K
    const int kk = (int)(t % k3);
    t /= k3;
    const int s = (int)(t % 3), r = (int)(t / 3);
    const int k = kk % K, blk = kk / K;
    const int rr = 3 * (blk / nbs) + r, ss = 3 * (blk % nbs) + s;
    T v;
    if (rr < R && ss < S) v = wt[(((int64_t)rr * S + ss) * K + k) * C + c];
    else v = T(0);
    w3[i] = v;
}

template <typename T>
hipError_t go(const ConvGeom& g, const void* wt, void* w3, hipStream_t st) {
    const int nbr = (int)((g.r + 2) / 3), nbs = (int)((g.s + 2) / 3);
    const int64_t total = (int64_t)9 * nbr * nbs * g.k * g.c;
    hipLaunchKernelGGL(split_weights_3x3_kernel<T>, dim3((unsigned)((total + 255) / 256)),
                       dim3(256), 0, st, (const T*)wt, (T*)w3, (int)g.r, (int)g.s, (int)g.k,
                       (int)g.c, nbs, total);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_split_weights_3x3(const ConvGeom& g, const void* wt, void* w3, int bf16,
                                    hipStream_t stream) {
    return bf16 ? go<bf16_t>(g, wt, w3, stream) : go<float>(g, wt, w3, stream);
}

}  // namespace ollie
