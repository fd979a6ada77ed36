// Channels-last copies for the convolution's vector-gather path: the same
// tensors as eq. (1) uses, in another order,
//   Dt[n][h][w][c] = D[n][c][h][w],   Wt[m][r][s][c] = W[m][c][r][s],
// so that the K = (r, s, c) run of one pixel is contiguous in memory and the
// im2col gather becomes 16-byte loads.
//
// The copy of D also encodes the input checksums of Sec. 3.2,
//   Cd1 = sum_n D_n,   Cd2 = sum_n (n + wbase) D_n,
// from the values it moves, so D is read once for both.  A workgroup owns a
// 32-channel x 32-position tile of the feature maps and walks a range of
// images in order, keeping the running float64 sums of its tile in registers;
// layers with few tiles split the images into ranges (one partial pair per
// range, combined in a fixed order by the convolution launch that follows).
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

constexpr int TT = 32;   // transpose tile: 32 channels x 32 positions, through LDS

template <typename T> __device__ inline double widen(T v) {
    if constexpr (sizeof(T) == 4) return (double)v;
    else return (double)bf16_bits_to_f32(v);
}

template <typename T, bool ENC>
__global__ __launch_bounds__(kThreads) void prep_kernel(const T *__restrict__ D, const T *__restrict__ W,
                                                        T *__restrict__ Dt, T *__restrict__ Wt, Geom g,
                                                        double *cd1, double *cd2, long long split_stride,
                                                        int tr_blocks, int hw_tiles, int c_tiles, int ns) {
    __shared__ T tile[kPrepBatch][TT][TT + 1];
    int b = blockIdx.x;
    const int HW = g.H * g.W;
    if (b < tr_blocks) {
        const int tiles = hw_tiles * c_tiles;
        const int split = b / tiles, rest = b - split * tiles;
        const int ht = rest % hw_tiles, ct = rest / hw_tiles;
        const int n0 = (int)((long long)split * g.N / ns), n1 = (int)((long long)(split + 1) * g.N / ns);
        const int tx = threadIdx.x % TT, ty = threadIdx.x / TT;   // 32 x 8 threads
        const int hw_in = ht * TT + tx;                            // this thread's load column
        const bool in_ok = hw_in < HW;
        const T *src = D + (long long)(ct * TT + ty) * HW + (in_ok ? hw_in : 0);
        double a1[TT / 8], a2[TT / 8];
#pragma unroll
        for (int q = 0; q < TT / 8; ++q) a1[q] = a2[q] = 0.0;
        // kPrepBatch images per round: all their loads in flight at once, one LDS tile each
        for (int nb = n0; nb < n1; nb += kPrepBatch) {
            T v[kPrepBatch][TT / 8];
#pragma unroll
            for (int j = 0; j < kPrepBatch; ++j) {
                const int n = nb + j < n1 ? nb + j : n1 - 1;   // a short last round re-reads a row it ignores
#pragma unroll
                for (int q = 0; q < TT / 8; ++q) v[j][q] = src[(long long)n * g.CHW + (long long)(8 * q) * HW];
            }
            if (nb > n0) __syncthreads();   // the previous round's tiles are read
#pragma unroll
            for (int j = 0; j < kPrepBatch; ++j) {
                if (nb + j >= n1) break;
                if constexpr (ENC) {
                    const double wgt = (double)(nb + j + g.wbase);
#pragma unroll
                    for (int q = 0; q < TT / 8; ++q) {
                        const double x = widen(v[j][q]);
                        a1[q] += x;
                        a2[q] = fma(wgt, x, a2[q]);
                    }
                }
#pragma unroll
                for (int q = 0; q < TT / 8; ++q) tile[j][ty + 8 * q][tx] = v[j][q];
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kPrepBatch; ++j) {
                if (nb + j >= n1) break;
                T *dst = Dt + (long long)(nb + j) * g.CHW;
#pragma unroll
                for (int q = 0; q < TT / 8; ++q) {   // rows of positions, coalesced along c
                    const int hw = ht * TT + ty + 8 * q;
                    if (hw < HW) dst[(long long)hw * g.C + ct * TT + tx] = tile[j][tx][ty + 8 * q];
                }
            }
        }
        if constexpr (ENC) {
            if (in_ok) {
                double *o1 = cd1 + (long long)split * split_stride, *o2 = cd2 + (long long)split * split_stride;
#pragma unroll
                for (int q = 0; q < TT / 8; ++q) {
                    const long long col = (long long)(ct * TT + ty + 8 * q) * HW + hw_in;
                    o1[col] = a1[q];
                    o2[col] = a2[q];
                }
            }
        }
        return;
    }
    b -= tr_blocks;
    // weights: one element of Wt per thread, written in order
    const long long i = (long long)b * kThreads + threadIdx.x;
    if (i >= (long long)g.M * g.K) return;
    const int m = (int)(i / g.K), k = (int)(i - (long long)m * g.K);
    const int rs = k / g.C, c = k - rs * g.C;
    Wt[i] = W[(long long)m * g.K + (long long)c * (g.R * g.S) + rs];
}

template <typename T>
hipError_t run(const Plan &pl, const void *D, const void *W, double *cd1, double *cd2, void *ws, hipStream_t st) {
    const Geom &g = pl.g;
    char *w = static_cast<char *>(ws);
    T *Dt = reinterpret_cast<T *>(w + pl.off_dt);
    T *Wt = reinterpret_cast<T *>(w + pl.off_wt);
    const long long HW = (long long)g.H * g.W;
    const long long hw_tiles = (HW + TT - 1) / TT, c_tiles = g.C / TT;
    // without the encode every round of images is a workgroup of its own
    const int ns = cd1 ? pl.prep_ns : (g.N + kPrepBatch - 1) / kPrepBatch;
    const long long tr = (long long)ns * c_tiles * hw_tiles;
    const long long wb = ((long long)g.M * g.K + kThreads - 1) / kThreads;
    const long long grid = tr + wb;
    if (grid > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    double *o1 = cd1, *o2 = cd2;
    long long stride = 0;
    if (cd1 && ns > 1) {
        // image-split partials [ns][2][Ch*H*W], combined by the convolution launch
        o1 = reinterpret_cast<double *>(w + pl.off_encp);
        o2 = o1 + g.CHW;
        stride = 2 * g.CHW;
    }
    if (cd1)
        prep_kernel<T, true><<<(unsigned)grid, kThreads, 0, st>>>(static_cast<const T *>(D), static_cast<const T *>(W),
                                                                  Dt, Wt, g, o1, o2, stride, (int)tr, (int)hw_tiles,
                                                                  (int)c_tiles, ns);
    else
        prep_kernel<T, false><<<(unsigned)grid, kThreads, 0, st>>>(static_cast<const T *>(D),
                                                                   static_cast<const T *>(W), Dt, Wt, g, nullptr,
                                                                   nullptr, 0, (int)tr, (int)hw_tiles, (int)c_tiles,
                                                                   ns);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_prep(const Plan &pl, const void *D, const void *W, double *cd1, double *cd2, void *ws,
                       hipStream_t st) {
    if (pl.g.dtype == FTCNN_F32) return run<float>(pl, D, W, cd1, cd2, ws, st);
    return run<uint16_t>(pl, D, W, cd1, cd2, ws, st);
}

}  // namespace ftcnn
