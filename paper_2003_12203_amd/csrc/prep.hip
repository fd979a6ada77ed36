// Channels-last copies for the convolution's vector-gather path: the same
// tensors as eq. (1) uses, in another order,
//   Dt[n][h][w][c] = D[n][c][h][w],   Wt[m][r][s][c] = W[m][c][r][s],
// so that the K = (r, s, c) run of one pixel is contiguous in memory and the
// im2col gather becomes 16-byte loads.
//
// The copy of D also encodes the input checksums of Sec. 3.2,
//   Cd1 = sum_n D_n,   Cd2 = sum_n (n + wbase) D_n,
// from the values it moves, so D is read once for both.  A workgroup owns a
// 32-channel x 128-byte tile of the feature maps and walks a range of images
// in order, keeping the running float64 sums of its tile in registers;
// layers with few tiles split the images into ranges (one partial pair per
// range, combined in a fixed order by the convolution launch that follows).
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

// Transpose tile: TC channels x TH positions per image, TH = 8 vectors of
// 16 bytes (32 fp32 or 64 bf16 positions) and TC = 32 channels, or 64 for bf16
// when the channel count allows (a stored position is then one 128-byte line).
// Every thread loads TC/32 16-byte runs of positions (one channel each) per
// image and stores TC/32 16-byte runs of channels (one position each).
template <typename T, int TC_> struct PrepT {
    static constexpr int TC = TC_;
    static constexpr int VEC = 16 / sizeof(T);          // elements per 16-byte vector
    static constexpr int TH = 8 * VEC;                   // positions per tile
    static constexpr int LDT = TH + 4 / sizeof(T);       // LDS row, padded by one word
    static constexpr int RPT = TC / 32;                  // channel rows per thread
    static constexpr int BATCH = kPrepBatch * 32 / TC;   // images per round (one LDS tile each)
    static constexpr int LDS_ELEMS = BATCH * TC * LDT;
};

template <typename T> __device__ inline double widen(T v) {
    if constexpr (sizeof(T) == 4) return (double)v;
    else return (double)bf16_bits_to_f32(v);
}

template <typename T, int V> union VecT {
    uint4 q;
    T e[V];
};

template <typename T, bool ENC, int TC>
__global__ __launch_bounds__(kThreads) void prep_kernel(const T *__restrict__ D, const T *__restrict__ W,
                                                        T *__restrict__ Dt, T *__restrict__ Wt, Geom g,
                                                        double *cd1, double *cd2, long long split_stride,
                                                        int tr_blocks, int hw_tiles, int c_tiles, int ns, int vec_ok,
                                                        uint4 *__restrict__ zero16) {
    using P = PrepT<T, TC>;
    constexpr int VEC = P::VEC, TH = P::TH, LDT = P::LDT, RPT = P::RPT, BATCH = P::BATCH;
    __shared__ T tile[BATCH][TC][LDT];
    int b = blockIdx.x;
    const int HW = g.H * g.W;
    if (b < tr_blocks) {
        const int tiles = hw_tiles * c_tiles;
        const int split = b / tiles, rest = b - split * tiles;
        const int ht = rest % hw_tiles, ct = rest / hw_tiles;
        const int n0 = (int)((long long)split * g.N / ns), n1 = (int)((long long)(split + 1) * g.N / ns);
        // load role: channel rows cr + 32 q, positions hw0 .. hw0 + VEC
        const int cr = threadIdx.x / 8, vq = threadIdx.x % 8;
        const int hw0 = ht * TH + vq * VEC;
        const T *src = D + (long long)(ct * TC + cr) * HW + hw0;
        // store role: positions hs + 32 q... (of the tile), channels cg*VEC .. cg*VEC + VEC
        constexpr int CG = TC / VEC;
        constexpr int HS = kThreads / CG;                  // positions stored per pass
        const int hs = threadIdx.x / CG, cg = threadIdx.x % CG;
        double a1[RPT][VEC], a2[RPT][VEC];
#pragma unroll
        for (int q = 0; q < RPT; ++q)
#pragma unroll
            for (int v = 0; v < VEC; ++v) a1[q][v] = a2[q][v] = 0.0;
        // one round: BATCH images, one LDS tile each; the loads of the next round are issued
        // before this round goes through LDS, so two rounds of loads are in flight
        auto load_round = [&](int nb, VecT<T, VEC>(&x)[BATCH][RPT]) {
#pragma unroll
            for (int j = 0; j < BATCH; ++j) {
                const int n = nb + j < n1 ? nb + j : n1 - 1;   // past the range: re-read a row, ignored
#pragma unroll
                for (int q = 0; q < RPT; ++q) {
                    const T *p = src + (long long)n * g.CHW + (long long)(32 * q) * HW;
                    if (vec_ok) {
                        // H*W is a multiple of VEC and D is 16-byte aligned
                        x[j][q].q = hw0 < HW ? *reinterpret_cast<const uint4 *>(p) : make_uint4(0, 0, 0, 0);
                    } else {
#pragma unroll
                        for (int v = 0; v < VEC; ++v) x[j][q].e[v] = hw0 + v < HW ? p[v] : T(0);
                    }
                }
            }
        };
        auto do_round = [&](int nb, VecT<T, VEC>(&x)[BATCH][RPT]) {
            __syncthreads();   // the previous round's tiles are read
#pragma unroll
            for (int j = 0; j < BATCH; ++j) {
                if (nb + j >= n1) break;
#pragma unroll
                for (int q = 0; q < RPT; ++q) {
                    if constexpr (ENC) {
                        const double wgt = (double)(nb + j + g.wbase);
#pragma unroll
                        for (int v = 0; v < VEC; ++v) {
                            const double xv = widen(x[j][q].e[v]);
                            a1[q][v] += xv;
                            a2[q][v] = fma(wgt, xv, a2[q][v]);
                        }
                    }
#pragma unroll
                    for (int v = 0; v < VEC; ++v) tile[j][cr + 32 * q][vq * VEC + v] = x[j][q].e[v];
                }
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < BATCH; ++j) {
                if (nb + j >= n1) break;
#pragma unroll
                for (int h = hs; h < TH; h += HS) {
                    const int hw_s = ht * TH + h;
                    if (hw_s >= HW) break;
                    VecT<T, VEC> y;
#pragma unroll
                    for (int v = 0; v < VEC; ++v) y.e[v] = tile[j][cg * VEC + v][h];
                    *reinterpret_cast<uint4 *>(Dt + ((long long)(nb + j) * HW + hw_s) * g.C + ct * TC + cg * VEC) = y.q;
                }
            }
        };
        VecT<T, VEC> xa[BATCH][RPT], xb[BATCH][RPT];
        if (n0 < n1) load_round(n0, xa);
        for (int nb = n0; nb < n1; nb += 2 * BATCH) {
            if (nb + BATCH < n1) load_round(nb + BATCH, xb);
            do_round(nb, xa);
            if (nb + BATCH >= n1) break;
            if (nb + 2 * BATCH < n1) load_round(nb + 2 * BATCH, xa);
            do_round(nb + BATCH, xb);
        }
        if constexpr (ENC) {
            double *o1 = cd1 + (long long)split * split_stride, *o2 = cd2 + (long long)split * split_stride;
#pragma unroll
            for (int q = 0; q < RPT; ++q) {
                const long long col = (long long)(ct * TC + cr + 32 * q) * HW + hw0;
#pragma unroll
                for (int v = 0; v < VEC; ++v)
                    if (hw0 + v < HW) {
                        o1[col + v] = a1[q][v];
                        o2[col + v] = a2[q][v];
                    }
            }
        }
        return;
    }
    // weights: one workgroup per filter m; its [C][R*S] row goes through LDS in channel chunks and
    // comes out as [R*S][C] (coalesced reads of W, runs of channels written to Wt)
    const int m = b - tr_blocks;
    if (m >= g.M) return;
    if (m == 0 && threadIdx.x < 16) zero16[threadIdx.x] = make_uint4(0, 0, 0, 0);
    T *stage = &tile[0][0][0];
    const int RS = g.R * g.S;
    const int cch = P::LDS_ELEMS / RS < g.C ? (P::LDS_ELEMS / RS > 0 ? P::LDS_ELEMS / RS : 1) : g.C;
    const T *wm = W + (long long)m * g.K;
    T *wtm = Wt + (long long)m * g.K;
    for (int c0 = 0; c0 < g.C; c0 += cch) {
        const int nc = cch < g.C - c0 ? cch : g.C - c0;
        __syncthreads();
        for (int e = threadIdx.x; e < nc * RS; e += kThreads) stage[e] = wm[(long long)c0 * RS + e];
        __syncthreads();
        for (int e = threadIdx.x; e < nc * RS; e += kThreads) {
            const int rs = e / nc, c = e - (e / nc) * nc;
            wtm[(long long)rs * g.C + c0 + c] = stage[c * RS + rs];
        }
    }
}

template <typename T, int TC>
hipError_t run_tc(const Plan &pl, const void *D, const void *W, double *cd1, double *cd2, void *ws, hipStream_t st) {
    using P = PrepT<T, TC>;
    const Geom &g = pl.g;
    char *w = static_cast<char *>(ws);
    T *Dt = reinterpret_cast<T *>(w + pl.off_dt);
    T *Wt = reinterpret_cast<T *>(w + pl.off_wt);
    uint4 *zero16 = reinterpret_cast<uint4 *>(w + pl.off_zero);
    const long long HW = (long long)g.H * g.W;
    const long long hw_tiles = (HW + P::TH - 1) / P::TH, c_tiles = g.C / TC;
    // without the encode every round of images is a workgroup of its own
    const int ns = cd1 ? pl.prep_ns : (g.N + P::BATCH - 1) / P::BATCH;
    const int vec_ok = HW % P::VEC == 0 && reinterpret_cast<uintptr_t>(D) % 16 == 0;
    const long long tr = (long long)ns * c_tiles * hw_tiles;
    const long long grid = tr + g.M;
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
        prep_kernel<T, true, TC><<<(unsigned)grid, kThreads, 0, st>>>(static_cast<const T *>(D),
                                                                      static_cast<const T *>(W), Dt, Wt, g, o1, o2,
                                                                      stride, (int)tr, (int)hw_tiles, (int)c_tiles, ns,
                                                                      vec_ok, zero16);
    else
        prep_kernel<T, false, TC><<<(unsigned)grid, kThreads, 0, st>>>(static_cast<const T *>(D),
                                                                       static_cast<const T *>(W), Dt, Wt, g, nullptr,
                                                                       nullptr, 0, (int)tr, (int)hw_tiles,
                                                                       (int)c_tiles, ns, vec_ok, zero16);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_prep(const Plan &pl, const void *D, const void *W, double *cd1, double *cd2, void *ws,
                       hipStream_t st) {
    if (pl.g.dtype == FTCNN_F32) return run_tc<float, 32>(pl, D, W, cd1, cd2, ws, st);
    if (prep_tile_channels(pl.g) == 64) return run_tc<uint16_t, 64>(pl, D, W, cd1, cd2, ws, st);
    return run_tc<uint16_t, 32>(pl, D, W, cd1, cd2, ws, st);
}

}  // namespace ftcnn
