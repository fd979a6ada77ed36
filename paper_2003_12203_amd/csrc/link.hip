// The operations between two protected convolution layers of a network (the
// AlexNet, VGG-19 and Darknet-19 stacks of Sec. 6): ReLU, then k x k max pooling
// at stride s with no padding.  Y[n][c][i][j] = max over the window at
// (s*i, s*j) of relu(X), relu(v) = v > 0 ? v : +0 (NaN and both zeros give +0),
// so every output is one of the input values or +0: exact in either dtype.
//
// Memory-bound: each output reads its k x k window (for 3x3/2, neighbouring
// windows share a row and a column, which the caches serve) and is written once.
// Plain ReLU (k = s = 1) moves 16-byte units.  The encoding variants also produce
// the next layer's input checksums from the values they write, so that layer's
// channels-last copy has nothing to encode.
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

// With the input checksums of the next layer (Sec. 3.2) encoded from the values written:
// Cd1[c][p] = sum_n Y[n][c][p], Cd2[c][p] = sum_n (n + wbase) Y[n][c][p] in float64.  A
// workgroup owns kEncPos units of positions (VEC consecutive positions of one channel, or one
// pooled position) and kEncGroups threads share each unit: thread group q walks the images
// n = q, q + kEncGroups, ..., four in flight, and the groups' sums are added in group order
// through LDS, so the result is the same on every run.  Consecutive threads take consecutive
// units, so every image's loads and stores are coalesced runs.
constexpr int kEncGroups = 4;
constexpr int kEncPos = kThreads / kEncGroups;

template <int VEC>
__device__ inline void enc_finish(double (&a1)[VEC], double (&a2)[VEC], double (*red)[kEncGroups][kEncPos],
                                  bool ok, long long base, double *cd1, double *cd2) {
    const int pl = threadIdx.x % kEncPos, q = threadIdx.x / kEncPos;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        red[0][q][pl] = a1[v];
        red[1][q][pl] = a2[v];
        __syncthreads();
        if (q == 0 && ok) {
            double s1 = red[0][0][pl], s2 = red[1][0][pl];
#pragma unroll
            for (int k = 1; k < kEncGroups; ++k) {
                s1 += red[0][k][pl];
                s2 += red[1][k][pl];
            }
            cd1[base + v] = s1;
            cd2[base + v] = s2;
        }
        __syncthreads();
    }
}

template <typename T, int VEC>
__global__ __launch_bounds__(kThreads) void relu_enc_kernel(const T *X, T *Y, int N, int C, int HW, int wbase,
                                                            double *__restrict__ cd1, double *__restrict__ cd2) {
    __shared__ double red[2][kEncGroups][kEncPos];
    const int units = HW / VEC;
    const int pl = threadIdx.x % kEncPos, q = threadIdx.x / kEncPos;
    const long long u = (long long)blockIdx.x * kEncPos + pl;
    const bool ok = u < (long long)C * units;
    const long long base = ok ? (u / units) * HW + (u % units) * VEC : 0;   // c * HW + first position
    const long long chw = (long long)C * HW;
    double a1[VEC], a2[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) a1[v] = a2[v] = 0.0;
    if (ok) {
        for (int n0 = q; n0 < N; n0 += 4 * kEncGroups) {
            union { uint4 q; T e[VEC]; } x[4];
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int n = n0 + b * kEncGroups;
                const long long off = (long long)(n < N ? n : n0) * chw + base;
                if constexpr (VEC > 1) {
                    x[b].q = *reinterpret_cast<const uint4 *>(X + off);
                } else {
                    x[b].e[0] = X[off];
                }
            }
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int n = n0 + b * kEncGroups;
                if (n >= N) break;
                const double wn = (double)(n + wbase);
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    float y;
                    if constexpr (sizeof(T) == 4) {
                        y = relu_f(x[b].e[v]);
                        x[b].e[v] = y;
                    } else {
                        // bf16 bits: positive (sign clear, not NaN) values stay, the rest become +0
                        const uint16_t bb = x[b].e[v];
                        const uint16_t r = (bb & 0x8000u) == 0 && (bb & 0x7FFFu) <= 0x7F80u ? bb : uint16_t(0);
                        x[b].e[v] = r;
                        y = bf16_bits_to_f32(r);
                    }
                    a1[v] += (double)y;
                    a2[v] = fma(wn, (double)y, a2[v]);
                }
                const long long off = (long long)n * chw + base;
                if constexpr (VEC > 1) {
                    *reinterpret_cast<uint4 *>(Y + off) = x[b].q;
                } else {
                    Y[off] = x[b].e[0];
                }
            }
        }
    }
    enc_finish<VEC>(a1, a2, red, ok, base, cd1, cd2);
}

template <typename T, int K, int S>
__global__ __launch_bounds__(kThreads) void pool_enc_kernel(const T *__restrict__ X, T *__restrict__ Y, int N, int C,
                                                            int H, int W, int Ho, int Wo, int wbase,
                                                            double *__restrict__ cd1, double *__restrict__ cd2) {
    __shared__ double red[2][kEncGroups][kEncPos];
    const int pl = threadIdx.x % kEncPos, q = threadIdx.x / kEncPos;
    const long long o = (long long)blockIdx.x * kEncPos + pl;   // (c, i, j)
    const long long plane = (long long)Ho * Wo;
    const bool ok = o < (long long)C * plane;
    double a1[1] = {0.0}, a2[1] = {0.0};
    if (ok) {
        const int j = (int)(o % Wo);
        const long long t = o / Wo;
        const int i = (int)(t % Ho);
        const long long c = t / Ho;
        const long long in0 = c * H * (long long)W + (long long)(S * i) * W + S * j;
        const long long chw = (long long)C * H * W, cpl = (long long)C * plane;
        for (int n0 = q; n0 < N; n0 += 4 * kEncGroups) {
            float m[4];
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int n = n0 + b * kEncGroups;
                const T *src = X + (long long)(n < N ? n : n0) * chw + in0;
                float mb = 0.0f;   // relu(v) >= +0
#pragma unroll
                for (int a = 0; a < K; ++a)
#pragma unroll
                    for (int r = 0; r < K; ++r) {
                        const float v = relu_f(val(src, (long long)a * W + r));
                        mb = v > mb ? v : mb;
                    }
                m[b] = mb;
            }
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int n = n0 + b * kEncGroups;
                if (n >= N) break;
                Elem<T>::store(Y, (long long)n * cpl + o, m[b]);
                a1[0] += (double)m[b];
                a2[0] = fma((double)(n + wbase), (double)m[b], a2[0]);
            }
        }
    }
    enc_finish<1>(a1, a2, red, ok, o, cd1, cd2);
}

template <typename T>
hipError_t run_link_enc(const T *X, T *Y, int n, int c, int h, int w, int k, int s, int wbase, double *cd1,
                        double *cd2, hipStream_t st) {
    if (k == 1) {
        const int HW = h * w;
        constexpr int VEC = 16 / sizeof(T);
        const bool vec = HW % VEC == 0 && reinterpret_cast<uintptr_t>(X) % 16 == 0 &&
                         reinterpret_cast<uintptr_t>(Y) % 16 == 0;
        const long long units = (long long)c * (vec ? HW / VEC : HW);
        const unsigned blocks = (unsigned)((units + kEncPos - 1) / kEncPos);
        if (vec) relu_enc_kernel<T, VEC><<<blocks, kThreads, 0, st>>>(X, Y, n, c, HW, wbase, cd1, cd2);
        else relu_enc_kernel<T, 1><<<blocks, kThreads, 0, st>>>(X, Y, n, c, HW, wbase, cd1, cd2);
        return hipGetLastError();
    }
    const int Ho = (h - k) / s + 1, Wo = (w - k) / s + 1;
    const long long total = (long long)c * Ho * Wo;
    const unsigned blocks = (unsigned)((total + kEncPos - 1) / kEncPos);
    if (k == 2) pool_enc_kernel<T, 2, 2><<<blocks, kThreads, 0, st>>>(X, Y, n, c, h, w, Ho, Wo, wbase, cd1, cd2);
    else pool_enc_kernel<T, 3, 2><<<blocks, kThreads, 0, st>>>(X, Y, n, c, h, w, Ho, Wo, wbase, cd1, cd2);
    return hipGetLastError();
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

hipError_t launch_relu_pool_encode(ftcnn_dtype dt, const void *X, void *Y, int n, int c, int h, int w, int k, int s,
                                   int wbase, double *cd1, double *cd2, hipStream_t st) {
    if (dt == FTCNN_F32)
        return run_link_enc(static_cast<const float *>(X), static_cast<float *>(Y), n, c, h, w, k, s, wbase, cd1, cd2,
                            st);
    return run_link_enc(static_cast<const uint16_t *>(X), static_cast<uint16_t *>(Y), n, c, h, w, k, s, wbase, cd1,
                        cd2, st);
}

hipError_t launch_relu_pool(ftcnn_dtype dt, const void *X, void *Y, int n, int c, int h, int w, int k, int s,
                            hipStream_t st) {
    if (dt == FTCNN_F32)
        return run_link(static_cast<const float *>(X), static_cast<float *>(Y), n, c, h, w, k, s, st);
    return run_link(static_cast<const uint16_t *>(X), static_cast<uint16_t *>(Y), n, c, h, w, k, s, st);
}

}  // namespace ftcnn
