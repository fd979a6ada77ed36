// Channels-last copies for the convolution's vector-gather path: the same
// tensors as eq. (1) uses, in another order,
//   Dt[n][h][w][c] = D[n][c][h][w],   Wt[m][r][s][c] = W[m][c][r][s],
// so that the K = (r, s, c) run of one pixel is contiguous in memory and the
// im2col gather becomes 16-byte loads.
//
// The copy of D also encodes the input checksums of Sec. 3.2,
//   Cd1 = sum_n D_n,   Cd2 = sum_n (n + wbase) D_n,
// from the values it moves, so D is read once for both.  A workgroup owns a
// tile of 32 (or 64) channels x TH positions of the feature maps and walks a
// range of images in order, keeping the running float64 sums of its tile in
// registers; layers with few tiles split the images into ranges (one partial
// pair per range, combined in a fixed order by the convolution launch that
// follows).
//
// Every global access is a 16-byte vector.  A channel row of the tile is read
// as eight aligned vectors.  When H*W is a multiple of the vector the row
// segment starts on a vector and the tile is eight vectors wide; otherwise it
// starts s elements into its first vector (s depends on the channel and the
// tile, not on the image, because Ch*H*W is a multiple of the vector) and the
// tile is seven vectors wide, the eighth covering the shift.
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

// Transpose tile: TC channels x TH positions per image.  ROW = 8 vectors are
// loaded per channel row; TC = 32 channels, or 64 for bf16 when the channel
// count allows (a stored position is then one 128-byte line).  Every thread
// loads TC/32 vectors (one channel row each) per image and stores TC/32 vectors
// of channels (one position each).
template <typename T, int TC_, bool SHIFT_> struct PrepT {
    static constexpr int TC = TC_;
    static constexpr bool SHIFT = SHIFT_;
    static constexpr int VEC = 16 / sizeof(T);          // elements per 16-byte vector
    static constexpr int ROW = 8 * VEC;                  // elements loaded per channel row
    static constexpr int TH = (SHIFT ? 7 : 8) * VEC;     // positions per tile
    static constexpr int LDT = ROW + 4 / sizeof(T);      // LDS row, padded by one word
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

// vec_d / vec_w: D / W is 16-byte aligned (else element loads; the layout is
// the same with shift 0, which a tile of seven vectors also covers).
template <typename T, bool ENC, int TC, bool SHIFT>
__global__ __launch_bounds__(kThreads) void prep_kernel(const T *__restrict__ D, const T *__restrict__ W,
                                                        T *__restrict__ Dt, T *__restrict__ Wt, Geom g,
                                                        double *cd1, double *cd2, long long split_stride,
                                                        int tr_blocks, int hw_tiles, int c_tiles, int ns, int vec_d,
                                                        int vec_w, uint4 *__restrict__ zero16, int *__restrict__ skcnt,
                                                        int skcnt_n) {
    using P = PrepT<T, TC, SHIFT>;
    constexpr int VEC = P::VEC, TH = P::TH, LDT = P::LDT, RPT = P::RPT, BATCH = P::BATCH;
    __shared__ T tile[BATCH][TC][LDT];
    int b = blockIdx.x;
    const int HW = g.H * g.W;
    if (b < tr_blocks) {
        const int tiles = hw_tiles * c_tiles;
        const int split = b / tiles, rest = b - split * tiles;
        const int ht = rest % hw_tiles, ct = rest / hw_tiles;
        const int n0 = (int)((long long)split * g.N / ns), n1 = (int)((long long)(split + 1) * g.N / ns);
        const int p0 = ht * TH;
        const int pend = p0 + TH < HW ? p0 + TH : HW;   // the tile's positions are [p0, pend)
        const int hmod = HW & (VEC - 1);
        // shift of channel row r of the tile: where position p0 sits in its vector
        auto shift = [&](int r) { return vec_d ? ((r & (VEC - 1)) * hmod + p0) & (VEC - 1) : 0; };
        // load role: channel rows cr + 32 q, vector vq of the row; its first element is at
        // position rel[q] of the row
        const int cr = threadIdx.x / 8, vq = threadIdx.x % 8;
        int rel[RPT];
        const T *src[RPT];
#pragma unroll
        for (int q = 0; q < RPT; ++q) {
            rel[q] = p0 - shift(cr + 32 * q) + vq * VEC;
            src[q] = D + (long long)(ct * TC + cr + 32 * q) * HW + rel[q];
        }
        // store role: positions hs + HS i of the tile, channels cg*VEC .. cg*VEC + VEC
        constexpr int CG = TC / VEC;
        constexpr int HS = kThreads / CG;                  // positions stored per pass
        const int hs = threadIdx.x / CG, cg = threadIdx.x % CG;
        int sv[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) sv[v] = shift(v);
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
                    const T *p = src[q] + (long long)n * g.CHW;
                    if (vec_d) {
                        // an aligned vector that overlaps the tile's part of the row lies inside D
                        x[j][q].q = rel[q] < pend ? *reinterpret_cast<const uint4 *>(p) : make_uint4(0, 0, 0, 0);
                    } else {
#pragma unroll
                        for (int v = 0; v < VEC; ++v) x[j][q].e[v] = rel[q] + v < pend ? p[v] : T(0);
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
                    uint32_t *row = reinterpret_cast<uint32_t *>(&tile[j][cr + 32 * q][vq * VEC]);
                    row[0] = x[j][q].q.x;
                    row[1] = x[j][q].q.y;
                    row[2] = x[j][q].q.z;
                    row[3] = x[j][q].q.w;
                }
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < BATCH; ++j) {
                if (nb + j >= n1) break;
#pragma unroll
                for (int h = hs; h < TH; h += HS) {
                    if (p0 + h >= HW) break;
                    VecT<T, VEC> y;
#pragma unroll
                    for (int v = 0; v < VEC; ++v) y.e[v] = tile[j][cg * VEC + v][h + sv[v]];
                    *reinterpret_cast<uint4 *>(Dt + ((long long)(nb + j) * HW + p0 + h) * g.C + ct * TC + cg * VEC) = y.q;
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
            // element v of the thread's vector is position rel + v of its row; each position of the
            // tile is in exactly one vector of the row
            double *o1 = cd1 + (long long)split * split_stride, *o2 = cd2 + (long long)split * split_stride;
#pragma unroll
            for (int q = 0; q < RPT; ++q) {
                const long long row = (long long)(ct * TC + cr + 32 * q) * HW;
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    const int p = rel[q] + v;
                    if (p >= p0 && p < pend) {
                        o1[row + p] = a1[q][v];
                        o2[row + p] = a2[q][v];
                    }
                }
            }
        }
        return;
    }
    // weights: one workgroup per filter m; its [C][R*S] row goes through LDS in channel chunks
    // (whole-vector loads of W) and comes out as [R*S][C] (vectors of VEC channels written to Wt)
    const int m = b - tr_blocks;
    if (m >= g.M) return;
    if (m == 0 && threadIdx.x < 16) zero16[threadIdx.x] = make_uint4(0, 0, 0, 0);
    // the convolution's stream-K arrival counts, spread over the weight workgroups
    for (int i = m * kThreads + threadIdx.x; i < skcnt_n; i += g.M * kThreads) skcnt[i] = 0;
    T *stage = &tile[0][0][0];
    const int RS = g.R * g.S;
    const T *wm = W + (long long)m * g.K;
    T *wtm = Wt + (long long)m * g.K;
    if (vec_w && VEC * RS <= P::LDS_ELEMS) {
        // chunks of a multiple of VEC channels: every chunk starts on a vector of W and of Wt
        int cch = (P::LDS_ELEMS / RS) / VEC * VEC;
        cch = cch < VEC ? VEC : (cch > g.C ? g.C : cch);
        for (int c0 = 0; c0 < g.C; c0 += cch) {
            const int nc = cch < g.C - c0 ? cch : g.C - c0;
            const int nvec = nc * RS / VEC;
            const uint4 *wv = reinterpret_cast<const uint4 *>(wm + (long long)c0 * RS);
            __syncthreads();
            for (int i0 = 0; i0 < nvec; i0 += 4 * kThreads) {
                uint4 x[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int i = i0 + u * kThreads + threadIdx.x;
                    x[u] = i < nvec ? wv[i] : make_uint4(0, 0, 0, 0);
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int i = i0 + u * kThreads + threadIdx.x;
                    if (i < nvec) *reinterpret_cast<uint4 *>(stage + (long long)i * VEC) = x[u];
                }
            }
            __syncthreads();
            const int cv_n = nc / VEC;
            for (int o = threadIdx.x; o < nvec; o += kThreads) {
                const int rs = o / cv_n, cv = o - (o / cv_n) * cv_n;
                VecT<T, VEC> y;
#pragma unroll
                for (int v = 0; v < VEC; ++v) y.e[v] = stage[(cv * VEC + v) * RS + rs];
                *reinterpret_cast<uint4 *>(wtm + (long long)rs * g.C + c0 + cv * VEC) = y.q;
            }
        }
        return;
    }
    const int cch = P::LDS_ELEMS / RS < g.C ? (P::LDS_ELEMS / RS > 0 ? P::LDS_ELEMS / RS : 1) : g.C;
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

template <typename T, int TC, bool SHIFT>
hipError_t run_tc(const Plan &pl, const void *D, const void *W, double *cd1, double *cd2, void *ws, hipStream_t st) {
    using P = PrepT<T, TC, SHIFT>;
    const Geom &g = pl.g;
    char *w = static_cast<char *>(ws);
    T *Dt = reinterpret_cast<T *>(w + pl.off_dt);
    T *Wt = reinterpret_cast<T *>(w + pl.off_wt);
    uint4 *zero16 = reinterpret_cast<uint4 *>(w + pl.off_zero);
    int *skcnt = reinterpret_cast<int *>(w + pl.off_skcnt);
    if (pl.sk_counters > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    const int skcnt_n = (int)pl.sk_counters;
    const long long HW = (long long)g.H * g.W;
    const long long hw_tiles = (HW + P::TH - 1) / P::TH, c_tiles = g.C / TC;
    // without the encode every round of images is a workgroup of its own
    const int ns = cd1 ? pl.prep_ns : (g.N + P::BATCH - 1) / P::BATCH;
    // Ch*H*W and K are multiples of 32 on these layers, so aligned bases keep every vector aligned
    const int vec_d = reinterpret_cast<uintptr_t>(D) % 16 == 0;
    const int vec_w = reinterpret_cast<uintptr_t>(W) % 16 == 0;
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
        prep_kernel<T, true, TC, SHIFT><<<(unsigned)grid, kThreads, 0, st>>>(
            static_cast<const T *>(D), static_cast<const T *>(W), Dt, Wt, g, o1, o2, stride, (int)tr, (int)hw_tiles,
            (int)c_tiles, ns, vec_d, vec_w, zero16, skcnt, skcnt_n);
    else
        prep_kernel<T, false, TC, SHIFT><<<(unsigned)grid, kThreads, 0, st>>>(
            static_cast<const T *>(D), static_cast<const T *>(W), Dt, Wt, g, nullptr, nullptr, 0, (int)tr,
            (int)hw_tiles, (int)c_tiles, ns, vec_d, vec_w, zero16, skcnt, skcnt_n);
    return hipGetLastError();
}

template <typename T, int TC>
hipError_t run_shift(const Plan &pl, const void *D, const void *W, double *cd1, double *cd2, void *ws,
                     hipStream_t st) {
    if (((long long)pl.g.H * pl.g.W) % (16 / sizeof(T)) == 0) return run_tc<T, TC, false>(pl, D, W, cd1, cd2, ws, st);
    return run_tc<T, TC, true>(pl, D, W, cd1, cd2, ws, st);
}

}  // namespace

hipError_t launch_prep(const Plan &pl, const void *D, const void *W, double *cd1, double *cd2, void *ws,
                       hipStream_t st) {
    if (pl.g.dtype == FTCNN_F32) return run_shift<float, 32>(pl, D, W, cd1, cd2, ws, st);
    if (prep_tile_channels(pl.g) == 64) return run_shift<uint16_t, 64>(pl, D, W, cd1, cd2, ws, st);
    return run_shift<uint16_t, 32>(pl, D, W, cd1, cd2, ws, st);
}

}  // namespace ftcnn
