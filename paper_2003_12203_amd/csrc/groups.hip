// Grouped convolution (Sec. 5.2): filter block m convolves only with the channel
// group m / (M/G) of every feature-map block.  The convolution runs on the
// block-diagonal expansion of W, a dense [M][C][R][S] that is zero outside each
// filter's channel group: the same outputs, and its Cw1 = sum_m W_m, Cw2 =
// sum_m (m + wbase) W_m are exactly the grouped checksums of Sec. 5.2 (the
// per-group filter sums side by side over the channels), so every checksum kernel
// works unchanged.  The matrix work is that of the dense layer, G times the
// grouped one.
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

template <typename T>
__global__ __launch_bounds__(kThreads) void expand_groups_kernel(const T *__restrict__ W, T *__restrict__ Wf, Geom g) {
    const long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (i >= (long long)g.M * g.K) return;
    const int m = (int)(i / g.K);
    const int k = (int)(i - (long long)m * g.K);
    const int RS = g.R * g.S;
    const int c = k / RS, rs = k - c * RS;
    const int c0 = group_first_channel(g, m);
    Wf[i] = c >= c0 && c < c0 + g.Cg ? W[(long long)m * g.Kg + (long long)(c - c0) * RS + rs] : T(0);
}

}  // namespace

const void *dense_weights(const Plan &pl, const void *W, void *ws, hipStream_t st, hipError_t *err) {
    *err = hipSuccess;
    if (pl.g.G == 1) return W;
    void *Wf = static_cast<char *>(ws) + pl.off_wfull;
    const long long n = (long long)pl.g.M * pl.g.K;
    const unsigned blocks = (unsigned)((n + kThreads - 1) / kThreads);
    if (pl.g.dtype == FTCNN_F32)
        expand_groups_kernel<float><<<blocks, kThreads, 0, st>>>(static_cast<const float *>(W),
                                                                 static_cast<float *>(Wf), pl.g);
    else
        expand_groups_kernel<uint16_t><<<blocks, kThreads, 0, st>>>(static_cast<const uint16_t *>(W),
                                                                    static_cast<uint16_t *>(Wf), pl.g);
    *err = hipGetLastError();
    return Wf;
}

}  // namespace ftcnn
