// Channels-last copies for the convolution's vector-gather path: the same
// tensors as eq. (1) uses, in another order,
//   Dt[n][h][w][c] = D[n][c][h][w],   Wt[m][r][s][c] = W[m][c][r][s],
// so that the K = (r, s, c) run of one pixel is contiguous in memory and the
// im2col gather becomes 16-byte loads.  Workgroups of the same launch can also
// encode the input checksums Cd1, Cd2 of D (Sec. 3.2), which read D in its own
// order.  Pure data movement: no value is changed.
#include "ftcnn_internal.h"
#include "encode_block.h"

namespace ftcnn {
namespace {

constexpr int TT = 32;   // transpose tile: 32 channels x 32 positions, through LDS

template <typename T>
__global__ __launch_bounds__(kThreads) void prep_kernel(const T *__restrict__ D, const T *__restrict__ W,
                                                        T *__restrict__ Dt, T *__restrict__ Wt, Geom g,
                                                        double *cd1, double *cd2, int enc_blocks, int enc_vec,
                                                        int tr_blocks, int hw_tiles, int c_tiles) {
    __shared__ T tile[TT][TT + 1];
    int b = blockIdx.x;
    if (b < enc_blocks) {
        if (enc_vec) encode_block<T, kThreads, kEncVec>(D, g, b, cd1, cd2);
        else encode_block<T, kThreads, 1>(D, g, b, cd1, cd2);
        return;
    }
    b -= enc_blocks;
    const int HW = g.H * g.W;
    if (b < tr_blocks) {
        const int ht = b % hw_tiles, rest = b / hw_tiles;
        const int ct = rest % c_tiles, n = rest / c_tiles;
        const int tx = threadIdx.x % TT, ty = threadIdx.x / TT;   // 32 x 8 threads
        const T *src = D + (long long)n * g.CHW;
#pragma unroll
        for (int q = 0; q < TT / 8; ++q) {   // rows of channels, coalesced along h*w
            const int c = ct * TT + ty + 8 * q, hw = ht * TT + tx;
            tile[ty + 8 * q][tx] = hw < HW ? src[(long long)c * HW + hw] : T(0);
        }
        __syncthreads();
        T *dst = Dt + (long long)n * g.CHW;
#pragma unroll
        for (int q = 0; q < TT / 8; ++q) {   // rows of positions, coalesced along c
            const int hw = ht * TT + ty + 8 * q, c = ct * TT + tx;
            if (hw < HW) dst[(long long)hw * g.C + c] = tile[tx][ty + 8 * q];
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
    long long enc = 0;
    int enc_vec = 0;
    if (cd1) {
        enc_vec = g.CHW % kEncVec == 0 && reinterpret_cast<uintptr_t>(D) % (kEncVec * sizeof(T)) == 0;
        const long long per = (long long)kThreads * (enc_vec ? kEncVec : 1);
        enc = (g.CHW + per - 1) / per;
    }
    const long long HW = (long long)g.H * g.W;
    const long long hw_tiles = (HW + TT - 1) / TT, c_tiles = g.C / TT;
    const long long tr = (long long)g.N * c_tiles * hw_tiles;
    const long long wb = ((long long)g.M * g.K + kThreads - 1) / kThreads;
    const long long grid = enc + tr + wb;
    if (grid > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    prep_kernel<T><<<(unsigned)grid, kThreads, 0, st>>>(static_cast<const T *>(D), static_cast<const T *>(W), Dt, Wt,
                                                        g, cd1, cd2, (int)enc, enc_vec, (int)tr, (int)hw_tiles,
                                                        (int)c_tiles);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_prep(const Plan &pl, const void *D, const void *W, double *cd1, double *cd2, void *ws,
                       hipStream_t st) {
    if (pl.g.dtype == FTCNN_F32) return run<float>(pl, D, W, cd1, cd2, ws, st);
    return run<uint16_t>(pl, D, W, cd1, cd2, ws, st);
}

}  // namespace ftcnn
