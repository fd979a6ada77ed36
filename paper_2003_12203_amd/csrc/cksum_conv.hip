// Output checksums as convolutions of checksum blocks (Sec. 3.2), in float64:
//   Co5 = Cd1 (x) Cw1, Co6 = Cd1 (x) Cw2, Co7 = Cd2 (x) Cw1        [E][F]
//   Co1 = Cd1 (x) W_m, Co3 = Cd2 (x) W_m                            [M][E][F]
//   Co2 = D_n (x) Cw1, Co4 = D_n (x) Cw2                            [N][E][F]
// One output element is a K = C*R*S dot product over a window.  With enough
// channels a wave shares one element (lanes stride over channels, then a fixed
// butterfly reduction); otherwise one lane computes a whole element.
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

__device__ inline double wave_sum(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

template <typename T> __device__ inline double ld(const T *p, long long i);
template <> __device__ inline double ld<double>(const double *p, long long i) { return p[i]; }
template <> __device__ inline double ld<float>(const float *p, long long i) { return (double)p[i]; }
template <> __device__ inline double ld<uint16_t>(const uint16_t *p, long long i) {
    return (double)bf16_bits_to_f32(p[i]);
}

// Sum over channels c = c0, c0 + cstep, ... of the window products
// a1 * b1, a1 * b2 and a2 * b1 at output position (x, y).
template <typename TA, typename TB>
__device__ inline void window3(const Geom &g, const TA *a1, const TA *a2, const TB *b1, const TB *b2,
                               int x, int y, int c0, int cstep, double &s11, double &s12, double &s21) {
    const long long HW = (long long)g.H * g.W;
    const int RS = g.R * g.S;
    for (int c = c0; c < g.C; c += cstep) {
        for (int r = 0; r < g.R; ++r) {
            const int ih = g.U * x + r - g.P;
            if (ih < 0 || ih >= g.H) continue;
            for (int s = 0; s < g.S; ++s) {
                const int iw = g.U * y + s - g.P;
                if (iw < 0 || iw >= g.W) continue;
                const long long ia = c * HW + (long long)ih * g.W + iw;
                const long long ib = (long long)c * RS + r * g.S + s;
                const double x1 = ld(a1, ia), w1 = ld(b1, ib);
                s11 = fma(x1, w1, s11);
                if (b2) s12 = fma(x1, ld(b2, ib), s12);
                if (a2) s21 = fma(ld(a2, ia), w1, s21);
            }
        }
    }
}

// Co5, Co6, Co7 at every position.  TPP threads share one position and stride
// over the flat k = (c, r, s) index; their partial sums meet in a fixed
// butterfly (and, for TPP = 256, in wave order through LDS).
template <int TPP>
__global__ __launch_bounds__(kThreads) void coc_kernel(Geom g, const double *__restrict__ cd1,
                                                       const double *__restrict__ cd2,
                                                       const double *__restrict__ cw1,
                                                       const double *__restrict__ cw2, double *co5,
                                                       double *co6, double *co7) {
    constexpr int G = TPP < 64 ? TPP : 64;  // lanes combined by shuffles
    const int lane = threadIdx.x % TPP;
    const int p = blockIdx.x * (kThreads / TPP) + threadIdx.x / TPP;
    double s11 = 0.0, s12 = 0.0, s21 = 0.0;
    if (p < g.EF) {
        const int x = p / g.F, y = p - (p / g.F) * g.F;
        const int RS = g.R * g.S;
        for (int k = lane; k < g.K; k += TPP) {
            const int c = k / RS, rem = k - c * RS, r = rem / g.S, s = rem - r * g.S;
            const int ih = g.U * x + r - g.P, iw = g.U * y + s - g.P;
            if (ih < 0 || ih >= g.H || iw < 0 || iw >= g.W) continue;
            const long long ia = ((long long)c * g.H + ih) * g.W + iw;
            const double x1 = cd1[ia];
            // cw1 is NULL when only Co6 (= Cd1 (x) Cw2) is asked for
            const double w1 = cw1 ? cw1[k] : 0.0;
            s11 = fma(x1, w1, s11);
            if (cw2) s12 = fma(x1, cw2[k], s12);
            if (cd2) s21 = fma(cd2[ia], w1, s21);
        }
    }
#pragma unroll
    for (int o = G / 2; o > 0; o >>= 1) {
        s11 += __shfl_xor(s11, o, 64);
        s12 += __shfl_xor(s12, o, 64);
        s21 += __shfl_xor(s21, o, 64);
    }
    if constexpr (TPP == kThreads) {
        __shared__ double red[3][kThreads / 64];
        const int w = threadIdx.x / 64;
        if ((threadIdx.x & 63) == 0) {
            red[0][w] = s11;
            red[1][w] = s12;
            red[2][w] = s21;
        }
        __syncthreads();
        s11 = ((red[0][0] + red[0][1]) + red[0][2]) + red[0][3];
        s12 = ((red[1][0] + red[1][1]) + red[1][2]) + red[1][3];
        s21 = ((red[2][0] + red[2][1]) + red[2][2]) + red[2][3];
    }
    if (p < g.EF && lane == 0) {
        if (co5) co5[p] = s11;
        if (co6) co6[p] = s12;
        if (co7) co7[p] = s21;
    }
}

// Co1[m] = Cd1 (x) W_m and Co3[m] = Cd2 (x) W_m: element (m, p).
template <typename T, bool WAVE>
__global__ __launch_bounds__(kThreads) void row_kernel(Geom g, const double *__restrict__ cd1,
                                                       const double *__restrict__ cd2,
                                                       const T *__restrict__ W, double *co1,
                                                       double *co3) {
    const int per_block = WAVE ? kThreads / 64 : kThreads;
    const long long task = (long long)blockIdx.x * per_block + (WAVE ? threadIdx.x / 64 : threadIdx.x);
    if (task >= (long long)g.M * g.EF) return;
    const int m = (int)(task / g.EF), p = (int)(task - (long long)(task / g.EF) * g.EF);
    const int lane = WAVE ? (threadIdx.x & 63) : 0;
    const int x = p / g.F, y = p - (p / g.F) * g.F;
    const T *Wm = W + (long long)m * g.K;
    double s11 = 0.0, s12 = 0.0, s21 = 0.0;
    window3<double, T>(g, cd1, cd2, Wm, (const T *)nullptr, x, y, lane, WAVE ? 64 : 1, s11, s12, s21);
    if (WAVE) {
        s11 = wave_sum(s11);
        s21 = wave_sum(s21);
    }
    if (lane == 0) {
        if (co1) co1[task] = s11;
        if (co3) co3[task] = s21;
    }
}

// Co2[n] = D_n (x) Cw1 and Co4[n] = D_n (x) Cw2: element (n, p).
template <typename T, bool WAVE>
__global__ __launch_bounds__(kThreads) void col_kernel(Geom g, const T *__restrict__ D,
                                                       const double *__restrict__ cw1,
                                                       const double *__restrict__ cw2, double *co2,
                                                       double *co4) {
    const int per_block = WAVE ? kThreads / 64 : kThreads;
    const long long task = (long long)blockIdx.x * per_block + (WAVE ? threadIdx.x / 64 : threadIdx.x);
    if (task >= (long long)g.N * g.EF) return;
    const int n = (int)(task / g.EF), p = (int)(task - (long long)(task / g.EF) * g.EF);
    const int lane = WAVE ? (threadIdx.x & 63) : 0;
    const int x = p / g.F, y = p - (p / g.F) * g.F;
    const T *Dn = D + (long long)n * g.CHW;
    double s11 = 0.0, s12 = 0.0, s21 = 0.0;
    window3<T, double>(g, Dn, (const T *)nullptr, cw1, cw2, x, y, lane, WAVE ? 64 : 1, s11, s12, s21);
    if (WAVE) {
        s11 = wave_sum(s11);
        s12 = wave_sum(s12);
    }
    if (lane == 0) {
        if (co2) co2[task] = s11;
        if (co4) co4[task] = s12;
    }
}

inline unsigned blocks_for(long long tasks, bool wave) {
    const long long per = wave ? kThreads / 64 : kThreads;
    return (unsigned)((tasks + per - 1) / per);
}

template <typename T>
hipError_t run_rows_cols(const Geom &g, uint32_t which, const void *D, const void *W,
                         const ftcnn_checksums &ck, hipStream_t st, bool wave) {
    if (which & (FTCNN_CO1 | FTCNN_CO3)) {
        const long long tasks = (long long)g.M * g.EF;
        double *o1 = (which & FTCNN_CO1) ? ck.co1 : nullptr;
        double *o3 = (which & FTCNN_CO3) ? ck.co3 : nullptr;
        if (wave)
            row_kernel<T, true><<<blocks_for(tasks, true), kThreads, 0, st>>>(g, ck.cd1, ck.cd2,
                                                                              (const T *)W, o1, o3);
        else
            row_kernel<T, false><<<blocks_for(tasks, false), kThreads, 0, st>>>(g, ck.cd1, ck.cd2,
                                                                                (const T *)W, o1, o3);
    }
    if (which & (FTCNN_CO2 | FTCNN_CO4)) {
        const long long tasks = (long long)g.N * g.EF;
        double *o2 = (which & FTCNN_CO2) ? ck.co2 : nullptr;
        double *o4 = (which & FTCNN_CO4) ? ck.co4 : nullptr;
        if (wave)
            col_kernel<T, true><<<blocks_for(tasks, true), kThreads, 0, st>>>(g, (const T *)D, ck.cw1,
                                                                              ck.cw2, o2, o4);
        else
            col_kernel<T, false><<<blocks_for(tasks, false), kThreads, 0, st>>>(g, (const T *)D, ck.cw1,
                                                                                ck.cw2, o2, o4);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_checksum_conv(const Plan &pl, uint32_t which, const void *D, const void *W,
                                const ftcnn_checksums &ck, hipStream_t st) {
    const Geom &g = pl.g;
    const bool wave = g.C >= 32;
    if (which & (FTCNN_CO5 | FTCNN_CO6 | FTCNN_CO7)) {
        double *o5 = (which & FTCNN_CO5) ? ck.co5 : nullptr;
        double *o6 = (which & FTCNN_CO6) ? ck.co6 : nullptr;
        double *o7 = (which & FTCNN_CO7) ? ck.co7 : nullptr;
        const double *cw1 = (o5 || o7) ? ck.cw1 : nullptr;
        const double *cw2 = o6 ? ck.cw2 : nullptr;
        const double *cd2 = o7 ? ck.cd2 : nullptr;
#define COC(TPP)                                                                                    \
    coc_kernel<TPP><<<(unsigned)((g.EF + kThreads / TPP - 1) / (kThreads / TPP)), kThreads, 0, st>>>( \
        g, ck.cd1, cd2, cw1, cw2, o5, o6, o7)
        if (g.K <= 64) COC(16);
        else if (g.EF <= 4096) COC(256);
        else COC(64);
#undef COC
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (g.dtype == FTCNN_F32) return run_rows_cols<float>(g, which, D, W, ck, st, wave);
    return run_rows_cols<uint16_t>(g, which, D, W, ck, st, wave);
}

}  // namespace ftcnn
