// Input checksums (Sec. 3.2): C1 = sum_r X_r and C2 = sum_r (r + wbase) X_r over
// the leading block index of X [rows][cols] (D over images, W over filters).
//
// A streaming column reduction: consecutive lanes own consecutive columns, so
// every row is read with full-width coalesced 16-byte loads, and each lane keeps
// its running sums in float64 registers.  Rows are split across a second grid
// dimension when there are too few columns to fill the chip; the split partials
// are combined in a fixed order, so the result is deterministic.
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

template <typename T, int VEC> struct Vec;
template <> struct Vec<float, 1> {
    __device__ static void load(const float *p, float (&v)[1]) { v[0] = *p; }
};
template <> struct Vec<float, 4> {
    __device__ static void load(const float *p, float (&v)[4]) {
        const float4 q = *reinterpret_cast<const float4 *>(p);
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
    }
};
template <> struct Vec<uint16_t, 1> {
    __device__ static void load(const uint16_t *p, float (&v)[1]) { v[0] = bf16_bits_to_f32(*p); }
};
template <> struct Vec<uint16_t, 8> {
    __device__ static void load(const uint16_t *p, float (&v)[8]) {
        const uint4 q = *reinterpret_cast<const uint4 *>(p);
        const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = __builtin_bit_cast(float, w[i] << 16);
            v[2 * i + 1] = __builtin_bit_cast(float, w[i] & 0xFFFF0000u);
        }
    }
};

template <typename T, int VEC>
__global__ __launch_bounds__(kThreads) void encode_partial(const T *__restrict__ X, long long rows,
                                                           long long cols, int wbase,
                                                           double *__restrict__ c1,
                                                           double *__restrict__ c2,
                                                           double *__restrict__ part) {
    const long long col = ((long long)blockIdx.x * kThreads + threadIdx.x) * VEC;
    if (col >= cols) return;
    const int splits = gridDim.y;
    const long long rps = (rows + splits - 1) / splits;
    const long long r0 = (long long)blockIdx.y * rps;
    const long long r1 = r0 + rps < rows ? r0 + rps : rows;

    double s1[VEC], s2[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) s1[v] = s2[v] = 0.0;

    constexpr int UNR = VEC == 1 ? 16 : 8;  // loads in flight per lane
    long long r = r0;
    for (; r + UNR <= r1; r += UNR) {
        float x[UNR][VEC];
#pragma unroll
        for (int u = 0; u < UNR; ++u) Vec<T, VEC>::load(X + (r + u) * cols + col, x[u]);
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const double wgt = (double)(r + u + wbase);
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                const double e = (double)x[u][v];
                s1[v] += e;
                s2[v] = fma(wgt, e, s2[v]);
            }
        }
    }
    for (; r < r1; ++r) {
        float x[VEC];
        Vec<T, VEC>::load(X + r * cols + col, x);
        const double wgt = (double)(r + wbase);
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            s1[v] += (double)x[v];
            s2[v] = fma(wgt, (double)x[v], s2[v]);
        }
    }
    if (splits == 1) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            c1[col + v] = s1[v];
            c2[col + v] = s2[v];
        }
    } else {
        double *p1 = part + (size_t)blockIdx.y * 2 * cols;
        double *p2 = p1 + cols;
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            p1[col + v] = s1[v];
            p2[col + v] = s2[v];
        }
    }
}

__global__ __launch_bounds__(kThreads) void encode_combine(const double *__restrict__ part,
                                                           long long cols, int splits,
                                                           double *__restrict__ c1,
                                                           double *__restrict__ c2) {
    const long long col = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (col >= cols) return;
    double s1 = 0.0, s2 = 0.0;
    for (int s = 0; s < splits; ++s) {
        s1 += part[(size_t)s * 2 * cols + col];
        s2 += part[(size_t)s * 2 * cols + cols + col];
    }
    c1[col] = s1;
    c2[col] = s2;
}

template <typename T, int VEC>
hipError_t run(const T *X, long long rows, long long cols, int splits, int wbase, double *c1,
               double *c2, double *part, hipStream_t st) {
    const long long threads = (cols + VEC - 1) / VEC;
    dim3 grid((unsigned)((threads + kThreads - 1) / kThreads), (unsigned)splits);
    encode_partial<T, VEC><<<grid, kThreads, 0, st>>>(X, rows, cols, wbase, c1, c2, part);
    if (splits > 1)
        encode_combine<<<(unsigned)((cols + kThreads - 1) / kThreads), kThreads, 0, st>>>(
            part, cols, splits, c1, c2);
    return hipGetLastError();
}

// The bias sums of Sec. 5.1, c1 = sum_m b[m] and c2 = sum_m (m + wbase) b[m]: one
// workgroup, strided per-thread sums added by a fixed tree (deterministic).
__global__ __launch_bounds__(kThreads) void bias_sums_kernel(const float *__restrict__ b, int M, int wbase,
                                                             double *c1, double *c2) {
    __shared__ double red[2][kThreads];
    const int t = threadIdx.x;
    double s1 = 0.0, s2 = 0.0;
    for (int m = t; m < M; m += kThreads) {
        const double v = (double)b[m];
        s1 += v;
        s2 = fma((double)(m + wbase), v, s2);
    }
    red[0][t] = s1;
    red[1][t] = s2;
    for (int h = kThreads / 2; h > 0; h >>= 1) {
        __syncthreads();
        if (t < h) {
            red[0][t] += red[0][t + h];
            red[1][t] += red[1][t + h];
        }
    }
    if (t == 0) {
        *c1 = red[0][0];
        *c2 = red[1][0];
    }
}

// Columns whose re-encoded Cw1 differs bitwise from the stored one: one workgroup, strided
// per-thread counts added by a fixed tree.
__global__ __launch_bounds__(kThreads) void count_mismatch_kernel(const double *__restrict__ fresh,
                                                                  const double *__restrict__ cw1, long long K,
                                                                  int32_t *out) {
    __shared__ int red[kThreads];
    const int t = threadIdx.x;
    int c = 0;
    for (long long k = t; k < K; k += kThreads)
        c += __double_as_longlong(fresh[k]) != __double_as_longlong(cw1[k]) ? 1 : 0;
    red[t] = c;
    for (int h = kThreads / 2; h > 0; h >>= 1) {
        __syncthreads();
        if (t < h) red[t] += red[t + h];
    }
    if (t == 0) *out = red[0];
}

}  // namespace

hipError_t launch_check_weights(const Plan &pl, const void *W, const double *cw1, int32_t *mismatches, void *ws,
                                hipStream_t st) {
    double *fresh = reinterpret_cast<double *>(static_cast<char *>(ws) + pl.off_wchk);
    const hipError_t e = launch_encode(pl, 1, W, fresh, fresh + pl.g.K, ws, st);
    if (e != hipSuccess) return e;
    count_mismatch_kernel<<<1, kThreads, 0, st>>>(fresh, cw1, pl.g.K, mismatches);
    return hipGetLastError();
}

hipError_t launch_bias_sums(const Plan &pl, const float *bias, double *c1, double *c2, hipStream_t st) {
    bias_sums_kernel<<<1, kThreads, 0, st>>>(bias, pl.g.M, pl.g.wbase, c1, c2);
    return hipGetLastError();
}

hipError_t launch_encode(const Plan &pl, int which, const void *X, double *c1, double *c2,
                         void *ws, hipStream_t st) {
    const Geom &g = pl.g;
    const long long rows = which == 0 ? g.N : g.M;
    const long long cols = which == 0 ? g.CHW : (long long)g.K;
    const int splits = which == 0 ? pl.enc_splits_d : pl.enc_splits_w;
    double *part = reinterpret_cast<double *>(static_cast<char *>(ws) + pl.off_enc);
    const uintptr_t a = reinterpret_cast<uintptr_t>(X);
    if (g.dtype == FTCNN_F32) {
        const float *x = static_cast<const float *>(X);
        if (cols % 4 == 0 && a % 16 == 0) return run<float, 4>(x, rows, cols, splits, g.wbase, c1, c2, part, st);
        return run<float, 1>(x, rows, cols, splits, g.wbase, c1, c2, part, st);
    }
    const uint16_t *x = static_cast<const uint16_t *>(X);
    if (cols % 8 == 0 && a % 16 == 0) return run<uint16_t, 8>(x, rows, cols, splits, g.wbase, c1, c2, part, st);
    return run<uint16_t, 1>(x, rows, cols, splits, g.wbase, c1, c2, part, st);
}

}  // namespace ftcnn
