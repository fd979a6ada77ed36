// The operations between two protected convolution layers of a network (the
// AlexNet, VGG-19 and Darknet-19 stacks of Sec. 6): ReLU, then k x k max pooling
// at stride s with no padding.  Y[n][c][i][j] = max over the window at
// (s*i, s*j) of relu(X), relu(v) = v > 0 ? v : +0 (NaN and both zeros give +0),
// so every output is one of the input values or +0: exact in either dtype.
//
// Memory-bound: each output reads its k x k window (for 3x3/2, neighbouring
// windows share a row and a column, which the caches serve) and is written once.
// Plain ReLU (k = s = 1) moves 16-byte units.
#include <algorithm>

#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

__device__ inline float relu_f(float v) { return v > 0.0f ? v : 0.0f; }

template <typename T> __device__ inline float val(const T *p, long long i) { return Elem<T>::load(p, i); }

// k = s = 1: 16-byte units where the whole tensor allows, else one element per thread.
template <typename T, int VEC>
__global__ __launch_bounds__(kThreads) void relu_kernel(const T *X, T *Y, long long n) {
    const long long stride = (long long)gridDim.x * kThreads;
    for (long long u = (long long)blockIdx.x * kThreads + threadIdx.x; u * VEC < n; u += stride) {
        if constexpr (VEC > 1) {
            union { uint4 q; T e[VEC]; } a;
            a.q = reinterpret_cast<const uint4 *>(X)[u];
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                if constexpr (sizeof(T) == 4) {
                    a.e[v] = relu_f(a.e[v]);
                } else {
                    // bf16 bits: positive (sign clear, not NaN) values stay, the rest become +0
                    const uint16_t b = a.e[v];
                    a.e[v] = (b & 0x8000u) == 0 && (b & 0x7FFFu) <= 0x7F80u ? b : uint16_t(0);
                }
            }
            reinterpret_cast<uint4 *>(Y)[u] = a.q;
        } else {
            Elem<T>::store(Y, u, relu_f(val(X, u)));
        }
    }
}

// One output element per thread; consecutive threads take consecutive j.
template <typename T, int K, int S>
__global__ __launch_bounds__(kThreads) void pool_kernel(const T *__restrict__ X, T *__restrict__ Y, int H, int W,
                                                        int Ho, int Wo, long long total) {
    const long long stride = (long long)gridDim.x * kThreads;
    for (long long o = (long long)blockIdx.x * kThreads + threadIdx.x; o < total; o += stride) {
        const int j = (int)(o % Wo);
        const long long t = o / Wo;
        const int i = (int)(t % Ho);
        const long long nc = t / Ho;
        const T *src = X + nc * H * (long long)W + (long long)(S * i) * W + S * j;
        float m = 0.0f;   // relu(v) >= +0, so +0 is the identity of the max
#pragma unroll
        for (int a = 0; a < K; ++a)
#pragma unroll
            for (int b = 0; b < K; ++b) {
                const float v = relu_f(val(src, (long long)a * W + b));
                m = v > m ? v : m;
            }
        Elem<T>::store(Y, o, m);
    }
}

template <typename T>
hipError_t run_link(const T *X, T *Y, int n, int c, int h, int w, int k, int s, hipStream_t st) {
    const long long cap = 8LL * 256 * 16;   // grid-stride: enough workgroups to fill every CU
    if (k == 1) {
        const long long total = (long long)n * c * h * w;
        constexpr int VEC = 16 / sizeof(T);
        const bool vec = total % VEC == 0 && reinterpret_cast<uintptr_t>(X) % 16 == 0 &&
                         reinterpret_cast<uintptr_t>(Y) % 16 == 0;
        const long long units = vec ? total / VEC : total;
        const unsigned blocks = (unsigned)std::min(cap, (units + kThreads - 1) / kThreads);
        if (vec) relu_kernel<T, VEC><<<blocks, kThreads, 0, st>>>(X, Y, total);
        else relu_kernel<T, 1><<<blocks, kThreads, 0, st>>>(X, Y, total);
        return hipGetLastError();
    }
    const int Ho = (h - k) / s + 1, Wo = (w - k) / s + 1;
    const long long total = (long long)n * c * Ho * Wo;
    const unsigned blocks = (unsigned)std::min(cap, (total + kThreads - 1) / kThreads);
    if (k == 2) pool_kernel<T, 2, 2><<<blocks, kThreads, 0, st>>>(X, Y, h, w, Ho, Wo, total);
    else pool_kernel<T, 3, 2><<<blocks, kThreads, 0, st>>>(X, Y, h, w, Ho, Wo, total);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_relu_pool(ftcnn_dtype dt, const void *X, void *Y, int n, int c, int h, int w, int k, int s,
                            hipStream_t st) {
    if (dt == FTCNN_F32)
        return run_link(static_cast<const float *>(X), static_cast<float *>(Y), n, c, h, w, k, s, st);
    return run_link(static_cast<const uint16_t *>(X), static_cast<uint16_t *>(Y), n, c, h, w, k, s, st);
}

}  // namespace ftcnn
