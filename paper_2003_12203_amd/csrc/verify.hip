// CoC-D detection (Sec. 3.6, Sec. 4.3).  With O viewed as [N*M][E*F], every
// output position p sums its column:
//   So5 = sum_{n,m} O,  So6 = sum (m + wbase) O,  So7 = sum (n + wbase) O,
//   Q5  = sqrt(sum O^2)  (the scale of the tolerance),
// and p is flagged when Co5 - So5 is non-finite or beyond the tolerance.
//
// Stage 1 streams O once with coalesced 16-byte loads: consecutive lanes own
// consecutive columns; small E*F layers stack several row groups in one block,
// combined through LDS in a fixed order.  Row ranges are split over a second
// grid dimension so the chip stays full; stage 2 adds the split partials in a
// fixed order (deterministic), applies the test and counts the flags.
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

template <typename T, int VEC> struct VLoad;
template <> struct VLoad<float, 1> {
    __device__ static void load(const float *p, float (&v)[1]) { v[0] = *p; }
};
template <> struct VLoad<float, 4> {
    __device__ static void load(const float *p, float (&v)[4]) {
        const float4 q = *reinterpret_cast<const float4 *>(p);
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
    }
};
template <> struct VLoad<uint16_t, 1> {
    __device__ static void load(const uint16_t *p, float (&v)[1]) { v[0] = bf16_bits_to_f32(*p); }
};
template <> struct VLoad<uint16_t, 8> {
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
__global__ __launch_bounds__(kThreads) void verify_partial(const T *__restrict__ O, Geom g, int ctt,
                                                           double *__restrict__ part,
                                                           ftcnn_report *rep, int cap) {
    __shared__ double red[kThreads][VEC];
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) reset_report(rep, cap);

    const int rpi = kThreads / ctt;                 // row groups per block
    const int t = threadIdx.x;
    const int cg = t % ctt, rg = t / ctt;
    const long long rows = (long long)g.N * g.M;
    const int splits = gridDim.y;
    const long long rps = (rows + splits - 1) / splits;
    const long long r0 = (long long)blockIdx.y * rps;
    const long long r1 = r0 + rps < rows ? r0 + rps : rows;
    const int col = (blockIdx.x * ctt + cg) * VEC;
    const bool active = rg < rpi && col < g.EF;

    // acc[0..3] = So5, So6, So7 and the sum of squares, per column
    double acc[4][VEC];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[a][v] = 0.0;

    if (active) {
        // row r = n*M + m; rows advance by rpi, so (n, m) advance by (dn, dm) with one carry
        const int dn = rpi / g.M, dm = rpi - (rpi / g.M) * g.M;
        long long r = r0 + rg;
        int n = (int)(r / g.M), m = (int)(r - (long long)n * g.M);
        constexpr int UNR = VEC == 1 ? 16 : 8;  // loads in flight per lane
        for (; r + (UNR - 1) * rpi < r1; r += UNR * rpi) {
            float x[UNR][VEC];
#pragma unroll
            for (int u = 0; u < UNR; ++u) VLoad<T, VEC>::load(O + (r + u * rpi) * g.EF + col, x[u]);
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                const double wn = (double)(n + g.wbase);
                const double wm = (double)(m + g.wbase);
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    const double e = (double)x[u][v];
                    acc[0][v] += e;
                    acc[1][v] = fma(wm, e, acc[1][v]);
                    acc[2][v] = fma(wn, e, acc[2][v]);
                    acc[3][v] = fma(e, e, acc[3][v]);
                }
                n += dn;
                m += dm;
                if (m >= g.M) { m -= g.M; ++n; }
            }
        }
        for (; r < r1; r += rpi) {
            float x[VEC];
            VLoad<T, VEC>::load(O + r * g.EF + col, x);
            const double wn = (double)(n + g.wbase);
            const double wm = (double)(m + g.wbase);
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                const double e = (double)x[v];
                acc[0][v] += e;
                acc[1][v] = fma(wm, e, acc[1][v]);
                acc[2][v] = fma(wn, e, acc[2][v]);
                acc[3][v] = fma(e, e, acc[3][v]);
            }
            n += dn;
            m += dm;
            if (m >= g.M) { m -= g.M; ++n; }
        }
    }
    if (rpi > 1) {  // fold the row groups of this block, in row-group order
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            __syncthreads();
#pragma unroll
            for (int v = 0; v < VEC; ++v) red[t][v] = acc[a][v];
            __syncthreads();
            if (rg == 0)
                for (int j = 1; j < rpi; ++j)
#pragma unroll
                    for (int v = 0; v < VEC; ++v) acc[a][v] += red[t + j * ctt][v];
        }
    }
    if (!active || rg != 0) return;
    double *p = part + (size_t)blockIdx.y * 4 * g.EF + col;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        if (col + v >= g.EF) break;
#pragma unroll
        for (int a = 0; a < 4; ++a) p[(size_t)a * g.EF + v] = acc[a][v];
    }
}

// TPP lanes (a power of two <= 64, aligned inside a wave) share one position:
// lane j adds splits j, j + TPP, ... in order, then a fixed butterfly combines
// the lanes.
template <int TPP>
__global__ __launch_bounds__(kThreads) void verify_final(Geom g, int splits, const double *__restrict__ part,
                                                         const double *__restrict__ co5, double *so5,
                                                         double *so6, double *so7, double *q5,
                                                         int *__restrict__ flags, double scale,
                                                         const double *__restrict__ cb, ftcnn_report *rep) {
    const int lane = threadIdx.x % TPP;
    const int p = blockIdx.x * (kThreads / TPP) + threadIdx.x / TPP;
    double a = 0.0, b = 0.0, c = 0.0, d = 0.0;
    if (p < g.EF) {
        for (int s = lane; s < splits; s += TPP) {
            const double *ps = part + (size_t)s * 4 * g.EF + p;
            a += ps[0];
            b += ps[g.EF];
            c += ps[2 * (size_t)g.EF];
            d += ps[3 * (size_t)g.EF];
        }
    }
#pragma unroll
    for (int o = TPP / 2; o > 0; o >>= 1) {
        a += __shfl_xor(a, o, 64);
        b += __shfl_xor(b, o, 64);
        c += __shfl_xor(c, o, 64);
        d += __shfl_xor(d, o, 64);
    }
    int flag = 0;
    if (p < g.EF && lane == 0) {
        const double q = sqrt(d);
        so5[p] = a;
        so6[p] = b;
        so7[p] = c;
        q5[p] = q;
        // with a bias, So5 less its share N * sum_m bias[m] (Sec. 5.1) is what Co5 predicts
        const double share = cb ? (double)g.N * cb[0] : 0.0;
        flag = is_bad(co5[p] - (a - share), q, scale) ? 1 : 0;
        flags[p] = flag;
    }
    const int cnt = __syncthreads_count(flag);
    if (threadIdx.x == 0 && cnt) {
        atomicAdd(&rep->n_flagged, cnt);
        atomicMax(&rep->detected, 1);
    }
}

template <typename T, int VEC>
hipError_t run_partial(const Plan &pl, const T *O, double *part, ftcnn_report *rep, int cap, hipStream_t st) {
    const Geom &g = pl.g;
    const int cols_v = (g.EF + VEC - 1) / VEC;
    const int ctt = cols_v < kThreads ? cols_v : kThreads;
    const int col_blocks = (cols_v + ctt - 1) / ctt;
    dim3 grid((unsigned)col_blocks, (unsigned)pl.ver_splits);
    verify_partial<T, VEC><<<grid, kThreads, 0, st>>>(O, g, ctt, part, rep, cap);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_verify_partial(const Plan &pl, const void *O, ftcnn_report *rep, int cap, void *ws,
                                 hipStream_t st) {
    const Geom &g = pl.g;
    double *part = reinterpret_cast<double *>(static_cast<char *>(ws) + pl.off_ver);
    const bool al = reinterpret_cast<uintptr_t>(O) % 16 == 0;
    if (g.dtype == FTCNN_F32) {
        const float *o = static_cast<const float *>(O);
        return (g.EF % 4 == 0 && al) ? run_partial<float, 4>(pl, o, part, rep, cap, st)
                                     : run_partial<float, 1>(pl, o, part, rep, cap, st);
    }
    const uint16_t *o = static_cast<const uint16_t *>(O);
    return (g.EF % 8 == 0 && al) ? run_partial<uint16_t, 8>(pl, o, part, rep, cap, st)
                                 : run_partial<uint16_t, 1>(pl, o, part, rep, cap, st);
}

hipError_t launch_verify(const Plan &pl, const void *O, const ftcnn_checksums &ck,
                         const ftcnn_policy &pol, ftcnn_report *rep, int cap, void *ws,
                         hipStream_t st) {
    const Geom &g = pl.g;
    char *w = static_cast<char *>(ws);
    double *part = reinterpret_cast<double *>(w + pl.off_ver);
    int *flags = reinterpret_cast<int *>(w + pl.off_flags);
    hipError_t e = launch_verify_partial(pl, O, rep, cap, ws, st);
    if (e != hipSuccess) return e;
    const double scale = tol_scale(g, pol.kappa);
    const int sp = pl.ver_splits;
#define FINAL(TPP)                                                                                     \
    verify_final<TPP><<<(unsigned)((g.EF + kThreads / TPP - 1) / (kThreads / TPP)), kThreads, 0, st>>>( \
        g, sp, part, ck.co5, ck.so5, ck.so6, ck.so7, ck.q5, flags, scale, ck.bias ? ck.cb : nullptr, rep)
    if (sp <= 1) FINAL(1);
    else if (sp <= 4) FINAL(4);
    else if (sp <= 16) FINAL(16);
    else FINAL(64);
#undef FINAL
    return hipGetLastError();
}

}  // namespace ftcnn
