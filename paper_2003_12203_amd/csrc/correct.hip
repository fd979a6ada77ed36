// Correction module of the multischeme workflow (Sec. 4.3, Fig. 7), one launch.
//
// Every scheme of Sec. 3 compares checksums element by element inside the
// output blocks (Level 2 of Sec. 3.2), so each flagged position p is repaired
// independently.  One workgroup takes one flagged position at a time and runs
// the whole chain there:
//
//   CoC  (Sec. 3.6)   i = (Co7-So7)/(Co5-So5), j = (Co6-So6)/(Co5-So5)
//   RC   (Sec. 3.4)   per mismatching column m: i = (Co3-So3)/(Co1-So1)
//   ClC  (Sec. 3.5)   per mismatching row n:    j = (Co4-So4)/(Co2-So2)
//   FC   (Sec. 3.3, 4.1.5) row/column mismatch sets; Co6/Co5 or Co7/Co5
//                     locate the column or row when Co1 or Co2 is blind
//
// The row and column checksums Co1..Co4 are computed lazily and only at p
// (K-long float64 dot products against checksum blocks), which is the whole
// cost of a scheme under Level-2 independence.  A scheme's repairs are undone
// unless Co5, Co6 and Co7 agree with the re-summed output afterwards.  When a
// weighted checksum agrees while Co5 does not, the checksums themselves are
// suspect (Sec. 4.1.4): Co5..Co7 are re-derived from D and W at p, and if O
// agrees with them the position is closed without a repair.
//
// Every sum is a fixed-shape reduction (per-thread serial, then a wave
// butterfly, then the four waves in order), so a rerun gives identical bits.
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

constexpr int KC = 512;  // k per staged window chunk

struct Sh {
    double red[8][4];
    double win1[KC], win2[KC];
    int off[KC];
    int flagbuf[kThreads];
    int list[kThreads];
    double colist[kThreads][3];   // Co5, Co6, Co7 of the listed positions
    int nlist, slot;
    int nfix, fail, cnt_m, cnt_n, one_m, one_n;
    double bcast[4];
};

template <typename T> struct Ctx {
    Geom g;
    const T *D, *W;
    T *O;
    const double *cd1, *cd2, *cw1, *cw2, *co5g, *co6g, *co7g;
    double scale, eta;
    int wb, rc_on, clc_on, recompute;
    double *co1m, *d1, *d3, *q1;   // per filter m at the current position
    double *co2n, *d2, *d4, *q2;   // per image n at the current position
    int *fix_n, *fix_m;
    uint32_t *fix_old;
    ftcnn_report *rep;
    // bias (Sec. 5.1): NULL, or [M] with cb = {sum_m bias[m], sum_m (m + wbase) bias[m]};
    // wn = sum_n (n + wbase)
    const float *bias;
    const double *cb;
    double wn;
};

// The bias shares of Table 5 (Sec. 5.1) moved to the checksum side: the checksums stay
// those of the convolution, and every comparison with a summation of the biased output
// (or repair from one) uses Co plus the share that the summation carries.
template <typename T> __device__ inline double bias_of(const Ctx<T> &c, int m) {
    return c.bias ? (double)c.bias[m] : 0.0;
}
template <typename T> __device__ inline void add_bias_shares(const Ctx<T> &c, double (&co)[3]) {
    if (!c.bias) return;
    const double b1 = c.cb[0], b2 = c.cb[1];
    co[0] += (double)c.g.N * b1;   // So5 carries N sum_m bias[m]
    co[1] += (double)c.g.N * b2;   // So6 carries N sum_m (m + wbase) bias[m]
    co[2] += c.wn * b1;            // So7 carries sum_n (n + wbase) sum_m bias[m]
}

__device__ inline double wave_sum(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

template <int NV> __device__ inline void bsum(double (&v)[NV], Sh &sh) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] = wave_sum(v[i]);
    __syncthreads();
    if (lane == 0)
#pragma unroll
        for (int i = 0; i < NV; ++i) sh.red[i][wave] = v[i];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] = ((sh.red[i][0] + sh.red[i][1]) + sh.red[i][2]) + sh.red[i][3];
}

template <typename T> __device__ inline double ldo(const T *p, long long i) {
    return (double)Elem<T>::load(p, i);
}
template <typename T> __device__ inline uint32_t bits_of(const T *p, long long i);
template <> __device__ inline uint32_t bits_of<float>(const float *p, long long i) {
    return __builtin_bit_cast(uint32_t, p[i]);
}
template <> __device__ inline uint32_t bits_of<uint16_t>(const uint16_t *p, long long i) { return p[i]; }
template <typename T> __device__ inline void put_bits(T *p, long long i, uint32_t b);
template <> __device__ inline void put_bits<float>(float *p, long long i, uint32_t b) {
    p[i] = __builtin_bit_cast(float, b);
}
template <> __device__ inline void put_bits<uint16_t>(uint16_t *p, long long i, uint32_t b) { p[i] = (uint16_t)b; }
template <typename T> __device__ inline void store_val(T *p, long long i, double v) {
    Elem<T>::store(p, i, (float)v);
}
// The value store_val leaves in memory, widened back to float64.
template <typename T> __device__ inline double stored_value(double v) {
    if constexpr (sizeof(T) == 4) return (double)(float)v;
    else return (double)bf16_bits_to_f32(f32_to_bf16_bits((float)v));
}

template <typename T> __device__ inline long long oidx(const Ctx<T> &c, int n, int m, int p) {
    return ((long long)n * c.g.M + m) * c.g.EF + p;
}

// Visits every block (n, m) of position p: thread t takes the elements
// e = n*M + m = t, t + kThreads, ..., with (n, m) advanced incrementally and
// eight loads in flight, and calls f(n, m, value) in that order.
template <typename T, typename F> __device__ inline void for_blocks(const Ctx<T> &c, int p, F &&f) {
    const Geom &g = c.g;
    const int nm = g.N * g.M;
    const int dn = kThreads / g.M, dm = kThreads - dn * g.M;
    int e = threadIdx.x;
    int n = e / g.M, m = e - n * g.M;
    const T *col = c.O + p;
    const long long step = (long long)kThreads * g.EF;
    long long off = (long long)e * g.EF;
    constexpr int U = 8;
    for (; e + (U - 1) * kThreads < nm; e += U * kThreads) {
        double v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = ldo(col, off + u * step);
        off += U * step;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            f(n, m, v[u]);
            n += dn;
            m += dm;
            if (m >= g.M) { m -= g.M; ++n; }
        }
    }
    for (; e < nm; e += kThreads, off += step) {
        f(n, m, ldo(col, off));
        n += dn;
        m += dm;
        if (m >= g.M) { m -= g.M; ++n; }
    }
}

// So5, So6, So7 and their Q (root sums of squares of the weighted terms) at p.
template <typename T> __device__ void sums6(const Ctx<T> &c, int p, Sh &sh, double (&s)[6]) {
    double v[6] = {0, 0, 0, 0, 0, 0};
    const double wb = (double)c.wb;
    for_blocks(c, p, [&](int n, int m, double o) {
        const double t6 = ((double)m + wb) * o, t7 = ((double)n + wb) * o;
        v[0] += o;
        v[1] += t6;
        v[2] += t7;
        v[3] = fma(o, o, v[3]);
        v[4] = fma(t6, t6, v[4]);
        v[5] = fma(t7, t7, v[5]);
    });
    bsum<6>(v, sh);
    s[0] = v[0]; s[1] = v[1]; s[2] = v[2];
    s[3] = sqrt(v[3]); s[4] = sqrt(v[4]); s[5] = sqrt(v[5]);
}

template <typename T>
__device__ bool consistent(const Ctx<T> &c, int p, Sh &sh, const double (&co)[3]) {
    double s[6];
    sums6(c, p, sh, s);
    return !is_bad(co[0] - s[0], s[3], c.scale) && !is_bad(co[1] - s[1], s[4], c.scale) &&
           !is_bad(co[2] - s[2], s[5], c.scale);
}

__device__ inline int legal(double r, int hi, double eta) {
    if (!isfinite(r)) return -1;
    const double i = rint(r);
    if (fabs(r - i) > eta || i < 0.0 || i >= (double)hi) return -1;
    return (int)i;
}

// Offsets of the window of position (x, y) for k in [k0, k0 + KC): -1 where the
// tap falls into the zero padding (or past K).
template <typename T> __device__ void stage_offsets(const Ctx<T> &c, int x, int y, int k0, Sh &sh) {
    const Geom &g = c.g;
    for (int kk = threadIdx.x; kk < KC; kk += kThreads) {
        const int k = k0 + kk;
        int off = -1;
        if (k < g.K) {
            const int RS = g.R * g.S;
            const int ch = k / RS, rem = k - ch * RS, r = rem / g.S, s = rem - r * g.S;
            const int ih = g.U * x + r - g.P, iw = g.U * y + s - g.P;
            if (ih >= 0 && ih < g.H && iw >= 0 && iw < g.W) off = (ch * g.H + ih) * g.W + iw;
        }
        sh.off[kk] = off;
    }
}

// Eq. (1) for one element, serially in k order (the RECOMPUTE repair); on a grouped layer over
// the filter's channel group (Sec. 5.2), W being [M][Cg][R][S].
template <typename T> __device__ double element(const Ctx<T> &c, int n, int m, int x, int y) {
    const Geom &g = c.g;
    const T *Dn = c.D + (long long)n * g.CHW + (long long)group_first_channel(g, m) * g.H * g.W;
    const T *Wm = c.W + (long long)m * g.Kg;
    double acc = 0.0;
    int k = 0;
    for (int ch = 0; ch < g.Cg; ++ch)
        for (int r = 0; r < g.R; ++r)
            for (int s = 0; s < g.S; ++s, ++k) {
                const int ih = g.U * x + r - g.P, iw = g.U * y + s - g.P;
                if (ih < 0 || ih >= g.H || iw < 0 || iw >= g.W) continue;
                acc = fma(ldo(Dn, ((long long)ch * g.H + ih) * g.W + iw), ldo(Wm, k), acc);
            }
    return acc + bias_of(c, m);
}

// Per filter m at p: Co1 = Cd1 (x) W_m, Co3 = Cd2 (x) W_m, and the
// differences to So1 = sum_n O_nm, So3 = sum_n (n + wbase) O_nm.
template <typename T> __device__ void row_arrays(const Ctx<T> &c, int p, int x, int y, Sh &sh) {
    const Geom &g = c.g;
    for (int m = threadIdx.x; m < g.M; m += kThreads) c.co1m[m] = c.d3[m] = 0.0;
    for (int k0 = 0; k0 < g.K; k0 += KC) {
        __syncthreads();
        stage_offsets(c, x, y, k0, sh);
        __syncthreads();
        for (int kk = threadIdx.x; kk < KC; kk += kThreads) {
            const int off = sh.off[kk];
            sh.win1[kk] = off >= 0 ? c.cd1[off] : 0.0;
            sh.win2[kk] = off >= 0 ? c.cd2[off] : 0.0;
        }
        __syncthreads();
        const int kend = g.K - k0 < KC ? g.K - k0 : KC;
        for (int m = threadIdx.x; m < g.M; m += kThreads) {
            double a1 = c.co1m[m], a3 = c.d3[m];
            // filter m's taps in the dense k = (c, r, s) order are the contiguous run of its channel
            // group (the whole K when ungrouped); W holds them from m * Kg
            const int kg0 = group_first_channel(g, m) * g.R * g.S;
            const int lo = kg0 - k0 > 0 ? kg0 - k0 : 0;
            const int hi = kg0 + g.Kg - k0 < kend ? kg0 + g.Kg - k0 : kend;
            const T *wr = c.W + (long long)m * g.Kg + (k0 - kg0);
            for (int kk = lo; kk < hi; ++kk) {
                const double w = ldo(wr, kk);
                a1 = fma(sh.win1[kk], w, a1);
                a3 = fma(sh.win2[kk], w, a3);
            }
            c.co1m[m] = a1;
            c.d3[m] = a3;
        }
    }
    for (int m = threadIdx.x; m < g.M; m += kThreads) {
        double s1 = 0.0, s3 = 0.0, q = 0.0;
#pragma unroll 8
        for (int n = 0; n < g.N; ++n) {
            const double o = ldo(c.O, oidx(c, n, m, p));
            s1 += o;
            s3 = fma((double)(n + c.wb), o, s3);
            q = fma(o, o, q);
        }
        // So1[m] carries N bias[m] and So3[m] sum_n (n + wbase) bias[m] (Sec. 5.1); co1m keeps the
        // shifted Co1, so the repairs from it give biased values
        const double bm = bias_of(c, m);
        c.co1m[m] += (double)g.N * bm;
        c.d1[m] = c.co1m[m] - s1;
        c.d3[m] = c.d3[m] + c.wn * bm - s3;
        c.q1[m] = sqrt(q);
    }
    __syncthreads();
}

// Per image n at p: Co2 = D_n (x) Cw1, Co4 = D_n (x) Cw2, and the differences
// to So2 = sum_m O_nm, So4 = sum_m (m + wbase) O_nm.
template <typename T> __device__ void col_arrays(const Ctx<T> &c, int p, int x, int y, Sh &sh) {
    const Geom &g = c.g;
    for (int n = threadIdx.x; n < g.N; n += kThreads) c.co2n[n] = c.d4[n] = 0.0;
    for (int k0 = 0; k0 < g.K; k0 += KC) {
        __syncthreads();
        stage_offsets(c, x, y, k0, sh);
        for (int kk = threadIdx.x; kk < KC; kk += kThreads) {
            const int k = k0 + kk;
            sh.win1[kk] = k < g.K ? c.cw1[k] : 0.0;
            sh.win2[kk] = k < g.K ? c.cw2[k] : 0.0;
        }
        __syncthreads();
        const int kend = g.K - k0 < KC ? g.K - k0 : KC;
        for (int n = threadIdx.x; n < g.N; n += kThreads) {
            double a2 = c.co2n[n], a4 = c.d4[n];
            const T *dn = c.D + (long long)n * g.CHW;
            for (int kk = 0; kk < kend; ++kk) {
                const int off = sh.off[kk];
                if (off < 0) continue;
                const double d = ldo(dn, off);
                a2 = fma(d, sh.win1[kk], a2);
                a4 = fma(d, sh.win2[kk], a4);
            }
            c.co2n[n] = a2;
            c.d4[n] = a4;
        }
    }
    for (int n = threadIdx.x; n < g.N; n += kThreads) {
        double s2 = 0.0, s4 = 0.0, q = 0.0;
#pragma unroll 8
        for (int m = 0; m < g.M; ++m) {
            const double o = ldo(c.O, oidx(c, n, m, p));
            s2 += o;
            s4 = fma((double)(m + c.wb), o, s4);
            q = fma(o, o, q);
        }
        // So2[n] carries sum_m bias[m] and So4[n] sum_m (m + wbase) bias[m] (Sec. 5.1)
        if (c.bias) {
            c.co2n[n] += c.cb[0];
            c.d4[n] += c.cb[1];
        }
        c.d2[n] = c.co2n[n] - s2;
        c.d4[n] = c.d4[n] - s4;
        c.q2[n] = sqrt(q);
    }
    __syncthreads();
}

// Mismatch sets: counts, and the member when there is exactly one.
template <typename T> __device__ void row_set(const Ctx<T> &c, Sh &sh) {
    if (threadIdx.x == 0) sh.cnt_m = 0, sh.one_m = -1;
    __syncthreads();
    for (int m = threadIdx.x; m < c.g.M; m += kThreads)
        if (is_bad(c.d1[m], c.q1[m], c.scale)) {
            atomicAdd(&sh.cnt_m, 1);
            atomicMax(&sh.one_m, m);
        }
    __syncthreads();
}
template <typename T> __device__ void col_set(const Ctx<T> &c, Sh &sh) {
    if (threadIdx.x == 0) sh.cnt_n = 0, sh.one_n = -1;
    __syncthreads();
    for (int n = threadIdx.x; n < c.g.N; n += kThreads)
        if (is_bad(c.d2[n], c.q2[n], c.scale)) {
            atomicAdd(&sh.cnt_n, 1);
            atomicMax(&sh.one_n, n);
        }
    __syncthreads();
}

// Apply one repair (called by the thread that owns it).
template <typename T> __device__ void repair(const Ctx<T> &c, Sh &sh, int n, int m, int p, double v) {
    const long long i = oidx(c, n, m, p);
    const int slot = atomicAdd(&sh.nfix, 1);
    c.fix_n[slot] = n;
    c.fix_m[slot] = m;
    c.fix_old[slot] = bits_of(c.O, i);
    store_val(c.O, i, v);
}

template <typename T> __device__ void undo(const Ctx<T> &c, Sh &sh, int p) {
    __syncthreads();
    for (int s = threadIdx.x; s < sh.nfix; s += kThreads)
        put_bits(c.O, oidx(c, c.fix_n[s], c.fix_m[s], p), c.fix_old[s]);
    __syncthreads();
}

// Keep the repairs if the CoC checksums agree afterwards, else undo them.
template <typename T> __device__ bool settle(const Ctx<T> &c, Sh &sh, int p, const double (&co)[3]) {
    __syncthreads();
    if (sh.nfix == 0) return false;
    if (consistent(c, p, sh, co)) return true;
    undo(c, sh, p);
    return false;
}

// Repair (i, m) for every m of the row mismatch set from Co1 (exclusive sum over n != i).
template <typename T> __device__ void fix_row_members(const Ctx<T> &c, Sh &sh, int p, int x, int y, int i) {
    for (int m = threadIdx.x; m < c.g.M; m += kThreads) {
        if (!is_bad(c.d1[m], c.q1[m], c.scale)) continue;
        double v;
        if (c.recompute) {
            v = element(c, i, m, x, y);
        } else {
            double s = 0.0;
            for (int n = 0; n < c.g.N; ++n)
                if (n != i) s += ldo(c.O, oidx(c, n, m, p));
            v = c.co1m[m] - s;
        }
        repair(c, sh, i, m, p, v);
    }
}

// Repair (n, j) for every n of the column mismatch set from Co2 (exclusive sum over m != j).
template <typename T> __device__ void fix_col_members(const Ctx<T> &c, Sh &sh, int p, int x, int y, int j) {
    for (int n = threadIdx.x; n < c.g.N; n += kThreads) {
        if (!is_bad(c.d2[n], c.q2[n], c.scale)) continue;
        double v;
        if (c.recompute) {
            v = element(c, n, j, x, y);
        } else {
            double s = 0.0;
            for (int m = 0; m < c.g.M; ++m)
                if (m != j) s += ldo(c.O, oidx(c, n, m, p));
            v = c.co2n[n] - s;
        }
        repair(c, sh, n, j, p, v);
    }
}

template <typename T> __device__ void begin_scheme(Sh &sh) {
    __syncthreads();
    if (threadIdx.x == 0) sh.nfix = 0, sh.fail = 0;
    __syncthreads();
}

template <typename T>
__device__ bool scheme_coc(const Ctx<T> &c, Sh &sh, int p, int x, int y, const double (&co)[3],
                           const double (&d)[3]) {
    const double ri = d[2] / d[0] - (double)c.wb, rj = d[1] / d[0] - (double)c.wb;
    const int i = legal(ri, c.g.N, c.eta), j = legal(rj, c.g.M, c.eta);
    if (i < 0 || j < 0) return false;
    begin_scheme<T>(sh);
    // one pass over the other blocks at p: their sums give the repair (the exclusive sum of R7)
    // and, with the repaired value added, the re-summed checksums of the consistency check
    const double wb = (double)c.wb;
    double e[6] = {0, 0, 0, 0, 0, 0};
    for_blocks(c, p, [&](int n, int m, double o) {
        if (n != i || m != j) {
            const double t6 = ((double)m + wb) * o, t7 = ((double)n + wb) * o;
            e[0] += o;
            e[1] += t6;
            e[2] += t7;
            e[3] = fma(o, o, e[3]);
            e[4] = fma(t6, t6, e[4]);
            e[5] = fma(t7, t7, e[5]);
        }
    });
    bsum<6>(e, sh);
    double v;
    if (c.recompute) {
        double a[1] = {0.0};
        // over filter j's channel group on a grouped layer (Sec. 5.2)
        const T *Dn = c.D + (long long)i * c.g.CHW + (long long)group_first_channel(c.g, j) * c.g.H * c.g.W;
        const T *Wm = c.W + (long long)j * c.g.Kg;
        for (int k = threadIdx.x; k < c.g.Kg; k += kThreads) {
            const int RS = c.g.R * c.g.S;
            const int ch = k / RS, rem = k - ch * RS, r = rem / c.g.S, s = rem - r * c.g.S;
            const int ih = c.g.U * x + r - c.g.P, iw = c.g.U * y + s - c.g.P;
            if (ih >= 0 && ih < c.g.H && iw >= 0 && iw < c.g.W)
                a[0] = fma(ldo(Dn, ((long long)ch * c.g.H + ih) * c.g.W + iw), ldo(Wm, k), a[0]);
        }
        bsum<1>(a, sh);
        v = a[0] + bias_of(c, j);
    } else {
        v = co[0] - e[0];
    }
    if (threadIdx.x == 0) repair(c, sh, i, j, p, v);
    __syncthreads();
    // the value as stored, and the checksums of the position re-summed with it
    const double o = stored_value<T>(v);
    const double t6 = ((double)j + wb) * o, t7 = ((double)i + wb) * o;
    const double s0 = e[0] + o, s1 = e[1] + t6, s2 = e[2] + t7;
    const double q5 = sqrt(fma(o, o, e[3])), q6 = sqrt(fma(t6, t6, e[4])), q7 = sqrt(fma(t7, t7, e[5]));
    if (!is_bad(co[0] - s0, q5, c.scale) && !is_bad(co[1] - s1, q6, c.scale) && !is_bad(co[2] - s2, q7, c.scale))
        return true;
    undo(c, sh, p);
    return false;
}

template <typename T>
__device__ bool scheme_rc(const Ctx<T> &c, Sh &sh, int p, int x, int y, const double (&co)[3]) {
    row_arrays(c, p, x, y, sh);
    row_set(c, sh);
    if (sh.cnt_m == 0) return false;
    begin_scheme<T>(sh);
    // every mismatching column must locate a legal row before anything is repaired
    for (int m = threadIdx.x; m < c.g.M; m += kThreads)
        if (is_bad(c.d1[m], c.q1[m], c.scale) && legal(c.d3[m] / c.d1[m] - (double)c.wb, c.g.N, c.eta) < 0)
            atomicOr(&sh.fail, 1);
    __syncthreads();
    if (sh.fail) return false;
    for (int m = threadIdx.x; m < c.g.M; m += kThreads) {
        if (!is_bad(c.d1[m], c.q1[m], c.scale)) continue;
        const int i = legal(c.d3[m] / c.d1[m] - (double)c.wb, c.g.N, c.eta);
        double v;
        if (c.recompute) {
            v = element(c, i, m, x, y);
        } else {
            double s = 0.0;
            for (int n = 0; n < c.g.N; ++n)
                if (n != i) s += ldo(c.O, oidx(c, n, m, p));
            v = c.co1m[m] - s;
        }
        repair(c, sh, i, m, p, v);
    }
    return settle(c, sh, p, co);
}

template <typename T>
__device__ bool scheme_clc(const Ctx<T> &c, Sh &sh, int p, int x, int y, const double (&co)[3]) {
    col_arrays(c, p, x, y, sh);
    col_set(c, sh);
    if (sh.cnt_n == 0) return false;
    begin_scheme<T>(sh);
    for (int n = threadIdx.x; n < c.g.N; n += kThreads)
        if (is_bad(c.d2[n], c.q2[n], c.scale) && legal(c.d4[n] / c.d2[n] - (double)c.wb, c.g.M, c.eta) < 0)
            atomicOr(&sh.fail, 1);
    __syncthreads();
    if (sh.fail) return false;
    for (int n = threadIdx.x; n < c.g.N; n += kThreads) {
        if (!is_bad(c.d2[n], c.q2[n], c.scale)) continue;
        const int j = legal(c.d4[n] / c.d2[n] - (double)c.wb, c.g.M, c.eta);
        double v;
        if (c.recompute) {
            v = element(c, n, j, x, y);
        } else {
            double s = 0.0;
            for (int m = 0; m < c.g.M; ++m)
                if (m != j) s += ldo(c.O, oidx(c, n, m, p));
            v = c.co2n[n] - s;
        }
        repair(c, sh, n, j, p, v);
    }
    return settle(c, sh, p, co);
}

template <typename T>
__device__ bool scheme_fc(const Ctx<T> &c, Sh &sh, int p, int x, int y, const double (&co)[3],
                          const double (&d)[3], bool have_rows, bool have_cols) {
    if (!have_rows) row_arrays(c, p, x, y, sh);
    if (!have_cols) col_arrays(c, p, x, y, sh);
    row_set(c, sh);
    col_set(c, sh);
    const int nm = sh.cnt_m, nn = sh.cnt_n;
    begin_scheme<T>(sh);
    if (nn == 1 && nm > 0) {                 // one row of blocks (Fig. 5a)
        fix_row_members(c, sh, p, x, y, sh.one_n);
    } else if (nm == 1 && nn > 0) {          // one column of blocks (Fig. 5b)
        fix_col_members(c, sh, p, x, y, sh.one_m);
    } else if (nm == 0 && nn > 0) {          // Co1 blind: column from Co6/Co5 (Fig. 5d)
        const int j = legal(d[1] / d[0] - (double)c.wb, c.g.M, c.eta);
        if (j < 0) return false;
        fix_col_members(c, sh, p, x, y, j);
    } else if (nn == 0 && nm > 0) {          // Co2 blind: row from Co7/Co5 (Fig. 5c)
        const int i = legal(d[2] / d[0] - (double)c.wb, c.g.N, c.eta);
        if (i < 0) return false;
        fix_row_members(c, sh, p, x, y, i);
    } else {
        return false;
    }
    return settle(c, sh, p, co);
}

// Co5..Co7 at p from checksums re-encoded out of D and W (Sec. 4.1.4).
template <typename T> __device__ void fresh_coc(const Ctx<T> &c, int x, int y, Sh &sh, double (&f)[3]) {
    const Geom &g = c.g;
    double v[3] = {0.0, 0.0, 0.0};
    for (int k = threadIdx.x; k < g.K; k += kThreads) {
        const int RS = g.R * g.S;
        const int ch = k / RS, rem = k - ch * RS, r = rem / g.S, s = rem - r * g.S;
        const int ih = g.U * x + r - g.P, iw = g.U * y + s - g.P;
        if (ih < 0 || ih >= g.H || iw < 0 || iw >= g.W) continue;
        const long long off = ((long long)ch * g.H + ih) * g.W + iw;
        double a1 = 0.0, a2 = 0.0, b1 = 0.0, b2 = 0.0;
#pragma unroll 8
        for (int n = 0; n < g.N; ++n) {
            const double dv = ldo(c.D, (long long)n * g.CHW + off);
            a1 += dv;
            a2 = fma((double)(n + c.wb), dv, a2);
        }
        // Cw1, Cw2 at k: the filters whose channel group holds channel ch (all of them when
        // ungrouped; Sec. 5.2), each read at its own offset in W [M][Cg][R][S]
        const int grp = ch / g.Cg;
        const long long kl = (long long)k - (long long)grp * g.Cg * RS;
#pragma unroll 8
        for (int m = grp * g.Mg; m < (grp + 1) * g.Mg; ++m) {
            const double wv = ldo(c.W, (long long)m * g.Kg + kl);
            b1 += wv;
            b2 = fma((double)(m + c.wb), wv, b2);
        }
        v[0] = fma(a1, b1, v[0]);
        v[1] = fma(a1, b2, v[1]);
        v[2] = fma(a2, b1, v[2]);
    }
    bsum<3>(v, sh);
    f[0] = v[0]; f[1] = v[1]; f[2] = v[2];
}

template <typename T> __device__ void record(const Ctx<T> &c, Sh &sh, int scheme, int x, int y) {
    __syncthreads();
    if (threadIdx.x == 0) {
        const int nf = scheme == FTCNN_SCHEME_UNRESOLVED || scheme == FTCNN_SCHEME_CKSUM ? 0 : sh.nfix;
        const int base = nf ? atomicAdd(&c.rep->n_fixes, nf) : 0;
        for (int s = 0; s < nf; ++s)
            if (base + s < c.rep->cap_fixes) {
                ftcnn_fix fx;
                fx.n = c.fix_n[s];
                fx.m = c.fix_m[s];
                fx.x = x;
                fx.y = y;
                fx.scheme = scheme;
                c.rep->fixes[base + s] = fx;
            }
        atomicAdd(&c.rep->resolved_by[scheme], 1);
        atomicMax(&c.rep->status, scheme == FTCNN_SCHEME_UNRESOLVED ? FTCNN_STATUS_NEEDS_RECOMPUTE
                                                                    : FTCNN_STATUS_CORRECTED);
    }
    __syncthreads();
}

template <typename T> __device__ void resolve(const Ctx<T> &c, Sh &sh, int p, const double (&co_in)[3]) {
    const int x = p / c.g.F, y = p - (p / c.g.F) * c.g.F;
    double co[3] = {co_in[0], co_in[1], co_in[2]};
    double s[6];
    sums6(c, p, sh, s);
    double d[3] = {co[0] - s[0], co[1] - s[1], co[2] - s[2]};
    const bool agree = !is_bad(d[0], s[3], c.scale) || !is_bad(d[1], s[4], c.scale) ||
                       !is_bad(d[2], s[5], c.scale);
    if (agree) {  // an inconsistent pattern among Co5/Co6/Co7: suspect the checksums
        double f[3];
        fresh_coc(c, x, y, sh, f);
        add_bias_shares(c, f);
        co[0] = f[0]; co[1] = f[1]; co[2] = f[2];
        if (!is_bad(co[0] - s[0], s[3], c.scale) && !is_bad(co[1] - s[1], s[4], c.scale) &&
            !is_bad(co[2] - s[2], s[5], c.scale)) {
            begin_scheme<T>(sh);
            record(c, sh, FTCNN_SCHEME_CKSUM, x, y);
            return;
        }
        d[0] = co[0] - s[0]; d[1] = co[1] - s[1]; d[2] = co[2] - s[2];
    }
    if (scheme_coc(c, sh, p, x, y, co, d)) return record(c, sh, FTCNN_SCHEME_COC, x, y);
    bool have_rows = false, have_cols = false;
    if (c.rc_on) {
        have_rows = true;
        if (scheme_rc(c, sh, p, x, y, co)) return record(c, sh, FTCNN_SCHEME_RC, x, y);
    }
    if (c.clc_on) {
        have_cols = true;
        if (scheme_clc(c, sh, p, x, y, co)) return record(c, sh, FTCNN_SCHEME_CLC, x, y);
    }
    if (scheme_fc(c, sh, p, x, y, co, d, have_rows, have_cols)) return record(c, sh, FTCNN_SCHEME_FC, x, y);
    begin_scheme<T>(sh);
    record(c, sh, FTCNN_SCHEME_UNRESOLVED, x, y);
}

// Point the per-position arrays of c at this workgroup's slice of scratch.
template <typename T> __device__ inline void bind_scratch(Ctx<T> &c, double *mine) {
    const Geom &g = c.g;
    const int L = g.M > g.N ? g.M : g.N;
    c.co1m = mine;
    c.d1 = c.co1m + g.M;
    c.d3 = c.d1 + g.M;
    c.q1 = c.d3 + g.M;
    c.co2n = c.q1 + g.M;
    c.d2 = c.co2n + g.N;
    c.d4 = c.d2 + g.N;
    c.q2 = c.d4 + g.N;
    c.fix_old = reinterpret_cast<uint32_t *>(c.q2 + g.N);
    c.fix_n = reinterpret_cast<int *>(c.fix_old + L);
    c.fix_m = c.fix_n + L;
}

template <typename T>
__global__ __launch_bounds__(kThreads) void correct_kernel(Ctx<T> c, const int *__restrict__ flags,
                                                           double *scratch, size_t stride, int chunk) {
    if (c.rep->detected == 0) return;
    __shared__ Sh sh;
    const Geom &g = c.g;
    bind_scratch(c, scratch + stride * blockIdx.x);
    // positions are dealt in chunks of `chunk` (<= kThreads) so that flagged
    // positions of small layers still spread over many workgroups
    for (int base = blockIdx.x * chunk; base < g.EF; base += gridDim.x * chunk) {
        const int p = base + threadIdx.x;
        sh.flagbuf[threadIdx.x] = (threadIdx.x < chunk && p < g.EF) ? flags[p] : 0;
        __syncthreads();
        if (threadIdx.x == 0) {
            int n = 0;
            for (int t = 0; t < chunk; ++t)
                if (sh.flagbuf[t]) sh.list[n++] = base + t;
            sh.nlist = n;
        }
        __syncthreads();
        const int cnt = sh.nlist;
        for (int i = 0; i < cnt; ++i) {
            const int p = sh.list[i];
            double co[3] = {c.co5g[p], c.co6g[p], c.co7g[p]};
            add_bias_shares(c, co);
            resolve(c, sh, p, co);
        }
        __syncthreads();
    }
}

// Co5 = Cd1 (x) Cw1, Co6 = Cd1 (x) Cw2, Co7 = Cd2 (x) Cw1 at position (x, y)
// (Sec. 3.2): this lane's share of the K taps, k = lane, lane + TPP, ...,
// with (ch, r, s) advanced incrementally.
template <typename T, int TPP>
__device__ inline void coc_taps(const Ctx<T> &c, int lane, int x, int y, double &c5, double &c6, double &c7) {
    const Geom &g = c.g;
    const int RS = g.R * g.S;
    int ch = lane / RS, rem = lane - ch * RS;
    int r = rem / g.S, s = rem - r * g.S;
    const int dch = TPP / RS, drem = TPP - dch * RS, dr = drem / g.S, ds = drem - dr * g.S;
    const int ih0 = g.U * x - g.P, iw0 = g.U * y - g.P;
    // branch-free taps, eight in flight: a tap past K or in the zero padding reads element 0
    // and selects 0 (the taps are added in the order k = lane, lane + TPP, ...)
    constexpr int U = 8;
    for (int k = lane; k < g.K; k += U * TPP) {
        double d1[U], d2[U], w1[U], w2[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kk = k + u * TPP;
            const int ih = ih0 + r, iw = iw0 + s;
            ok[u] = kk < g.K && ((unsigned)ih < (unsigned)g.H) & ((unsigned)iw < (unsigned)g.W);
            const long long off = ok[u] ? ((long long)ch * g.H + ih) * g.W + iw : 0;
            const int kw = kk < g.K ? kk : 0;
            d1[u] = c.cd1[off];
            d2[u] = c.cd2[off];
            w1[u] = c.cw1[kw];
            w2[u] = c.cw2[kw];
            s += ds;
            r += dr;
            ch += dch;
            if (s >= g.S) { s -= g.S; ++r; }
            if (r >= g.R) { r -= g.R; ++ch; }
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u]) {
                c5 = fma(d1[u], w1[u], c5);
                c6 = fma(d1[u], w2[u], c6);
                c7 = fma(d2[u], w1[u], c7);
            }
    }
}

// Final stage of the detection (the split partials of each position summed in a
// fixed order, then the CoC-D test) with the correction chain run in the same
// workgroup for every position it flags.  A clean layer pays nothing for the
// correction module, and no separate launch is needed.  With COC the same
// lanes also produce Co5..Co7 of their position and store them: from the
// channel-range partials the convolution launch left (rep->reserved[1] of
// them), or else from the taps of Cd and Cw.
//
// TPP threads share a position, and consecutive threads take consecutive
// positions (thread t: position t % per, lane t / per), so every load of a
// partial slice is a coalesced run; the lanes of a position are then added in a
// fixed order (exchanges inside each wave, then the four waves).
template <typename T, int TPP, bool COC>
__global__ __launch_bounds__(kThreads) void verify_correct_kernel(Ctx<T> c, int splits, const double *__restrict__ part,
                                                                  const double *__restrict__ copart, int max_groups,
                                                                  double *co5, double *co6, double *co7,
                                                                  double *so5, double *so6, double *so7, double *q5,
                                                                  int *__restrict__ flags, double *scratch,
                                                                  size_t stride, int nslots) {
    __shared__ Sh sh;
    constexpr int NV = COC ? 7 : 4;
    __shared__ double red[TPP > 1 ? NV : 1][TPP > 1 ? 4 * (kThreads / TPP) : 1];
    const Geom &g = c.g;
    constexpr int per = kThreads / TPP;
    const int slot = threadIdx.x % per, lane = threadIdx.x / per;
    const int p = blockIdx.x * per + slot;
    double v[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] = 0.0;
    if (p < g.EF) {
        // the So partials first: their loads do not wait on the report word that counts the Co
        // partials.  Four slices of loads in flight, added in slice order.
        for (int s0 = lane; s0 < splits; s0 += 4 * TPP) {
            double x[4][4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int s = s0 + u * TPP;
                const double *ps = part + (size_t)(s < splits ? s : 0) * 4 * g.EF + p;
#pragma unroll
                for (int i = 0; i < 4; ++i) x[u][i] = ps[i * (size_t)g.EF];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (s0 + u * TPP < splits)
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] += x[u][i];
        }
        if constexpr (COC) {
            // slices written by the convolution launch that reset this report (never more than
            // the workspace holds)
            const int groups = min(c.rep->reserved[1], max_groups);
            if (groups > 0) {
                for (int s0 = lane; s0 < groups; s0 += 4 * TPP) {
                    double x[4][3];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int s = s0 + u * TPP;
                        const double *ps = copart + (size_t)(s < groups ? s : 0) * 3 * g.EF + p;
                        x[u][0] = ps[0];
                        x[u][1] = ps[g.EF];
                        x[u][2] = ps[2 * (size_t)g.EF];
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        if (s0 + u * TPP < groups) {
                            v[4] += x[u][0];
                            v[5] += x[u][1];
                            v[6] += x[u][2];
                        }
                }
            } else {
                const int x = p / g.F;
                coc_taps<T, TPP>(c, lane, x, p - x * g.F, v[4], v[5], v[6]);
            }
        }
    }
    if constexpr (TPP > 1) {
        // the TPP lanes of a position are the threads t = slot (mod per): inside a wave they are
        // folded by exchanges at distances per, 2 per, ..., 32, then the four waves' sums are
        // added in wave order (a fixed order: the same sums on every run)
        static_assert(kThreads == 256 && TPP >= 4, "four waves, at most 64 positions a workgroup");
#pragma unroll
        for (int o = per; o < 64; o <<= 1)
#pragma unroll
            for (int i = 0; i < NV; ++i) v[i] += __shfl_xor(v[i], o, 64);
        const int wv = threadIdx.x >> 6, wl = threadIdx.x & 63;
        if (wl < per)
#pragma unroll
            for (int i = 0; i < NV; ++i) red[i][wv * per + wl] = v[i];
        __syncthreads();
#pragma unroll
        for (int i = 0; i < NV; ++i)
            v[i] = ((red[i][slot] + red[i][per + slot]) + red[i][2 * per + slot]) + red[i][3 * per + slot];
    }
    double a = v[0], b = v[1], cc = v[2], d = v[3];
    double c5 = 0.0, c6 = 0.0, c7 = 0.0;
    if constexpr (COC) {
        c5 = v[4];
        c6 = v[5];
        c7 = v[6];
    }
    int flag = 0;
    if (p < g.EF && lane == 0) {
        if constexpr (COC) {
            co5[p] = c5;
            co6[p] = c6;
            co7[p] = c7;
        } else {
            c5 = c.co5g[p];
            c6 = c.co6g[p];
            c7 = c.co7g[p];
        }
        const double q = sqrt(d);
        so5[p] = a;
        so6[p] = b;
        so7[p] = cc;
        q5[p] = q;
        // the checksums as the summations of the biased output see them (Sec. 5.1)
        double cs[3] = {c5, c6, c7};
        add_bias_shares(c, cs);
        flag = is_bad(cs[0] - a, q, c.scale) ? 1 : 0;
        flags[p] = flag;
        sh.flagbuf[slot] = flag;
        sh.colist[slot][0] = cs[0];
        sh.colist[slot][1] = cs[1];
        sh.colist[slot][2] = cs[2];
    }
    const int cnt = __syncthreads_count(flag);
    if (cnt == 0) return;
    if (threadIdx.x == 0) {
        atomicAdd(&c.rep->n_flagged, cnt);
        atomicMax(&c.rep->detected, 1);
        // compact the flagged slots in place (slot t moves to n <= t)
        int n = 0;
        for (int t = 0; t < per; ++t)
            if (blockIdx.x * per + t < g.EF && sh.flagbuf[t]) {
                sh.list[n] = blockIdx.x * per + t;
                sh.colist[n][0] = sh.colist[t][0];
                sh.colist[n][1] = sh.colist[t][1];
                sh.colist[n][2] = sh.colist[t][2];
                ++n;
            }
        sh.nlist = n;
        // a scratch slice for this workgroup's chain, taken from the report's slot counter
        sh.slot = atomicAdd(&c.rep->reserved[0], 1);
    }
    __syncthreads();
    const int nl = sh.nlist;
    if (sh.slot >= nslots) {
        // more flagged workgroups than scratch slices: leave these positions to recomputation
        for (int i = 0; i < nl; ++i) {
            begin_scheme<T>(sh);
            const int p = sh.list[i];
            record(c, sh, FTCNN_SCHEME_UNRESOLVED, p / g.F, p - (p / g.F) * g.F);
        }
        return;
    }
    bind_scratch(c, scratch + stride * sh.slot);
    for (int i = 0; i < nl; ++i) {
        const double co[3] = {sh.colist[i][0], sh.colist[i][1], sh.colist[i][2]};
        resolve(c, sh, sh.list[i], co);
    }
}

template <typename T>
Ctx<T> make_ctx(const Plan &pl, const void *D, const void *W, void *O, const ftcnn_checksums &ck,
                const ftcnn_policy &pol, ftcnn_report *rep) {
    Ctx<T> c{};
    c.g = pl.g;
    c.D = static_cast<const T *>(D);
    c.W = static_cast<const T *>(W);
    c.O = static_cast<T *>(O);
    c.cd1 = ck.cd1; c.cd2 = ck.cd2; c.cw1 = ck.cw1; c.cw2 = ck.cw2;
    c.co5g = ck.co5; c.co6g = ck.co6; c.co7g = ck.co7;
    c.scale = tol_scale(pl.g, pol.kappa);
    c.eta = pol.eta;
    c.wb = pl.g.wbase;
    c.rc_on = pol.rc_on;
    c.clc_on = pol.clc_on;
    c.recompute = pol.repair == FTCNN_REPAIR_RECOMPUTE;
    c.rep = rep;
    c.bias = ck.bias;
    c.cb = ck.bias ? ck.cb : nullptr;
    c.wn = (double)pl.g.N * (double)pl.g.wbase + (double)pl.g.N * ((double)pl.g.N - 1.0) / 2.0;
    return c;
}

template <typename T>
hipError_t run_fused(const Plan &pl, const void *D, const void *W, void *O, const ftcnn_checksums &ck,
                     const ftcnn_policy &pol, ftcnn_report *rep, void *ws, size_t off_part, int sp, bool coc,
                     hipStream_t st) {
    const Ctx<T> c = make_ctx<T>(pl, D, W, O, ck, pol, rep);
    char *w = static_cast<char *>(ws);
    const double *part = reinterpret_cast<const double *>(w + off_part);
    int *flags = reinterpret_cast<int *>(w + pl.off_flags);
    double *scratch = reinterpret_cast<double *>(w + pl.off_corr);
    // Co5..Co7 of a channels-last layer come as partial slices from the convolution launch
    // (the kernel checks rep->reserved[1] and falls back to the taps)
    const int taps = coc ? (pl.co_in_conv ? pl.co.groups * pl.prep_ns : pl.g.K) : 0;
    const int tpp = final_tpp(sp, taps, pl.g.EF);
    const double *copart = reinterpret_cast<const double *>(w + pl.off_copart);
    const int max_groups = pl.co_in_conv ? pl.co.groups * pl.prep_ns : 0;
    const unsigned blocks = (unsigned)((pl.g.EF + kThreads / tpp - 1) / (kThreads / tpp));
#define VC(TPP, COC)                                                                                            \
    verify_correct_kernel<T, TPP, COC><<<blocks, kThreads, 0, st>>>(c, sp, part, copart, max_groups, ck.co5,       \
                                                                    ck.co6, ck.co7,                              \
                                                                    ck.so5, ck.so6, ck.so7, ck.q5, flags,        \
                                                                    scratch, pl.corr_stride, pl.corr_slots)
    if (coc) {
        if (tpp == 1) VC(1, true);
        else if (tpp == 4) VC(4, true);
        else if (tpp == 16) VC(16, true);
        else if (tpp == 64) VC(64, true);
        else VC(kThreads, true);
    } else {
        if (tpp == 1) VC(1, false);
        else if (tpp == 4) VC(4, false);
        else if (tpp == 16) VC(16, false);
        else if (tpp == 64) VC(64, false);
        else VC(kThreads, false);
    }
#undef VC
    return hipGetLastError();
}

template <typename T>
hipError_t run(const Plan &pl, const void *D, const void *W, void *O, const ftcnn_checksums &ck,
               const ftcnn_policy &pol, ftcnn_report *rep, void *ws, hipStream_t st) {
    Ctx<T> c{};
    c.g = pl.g;
    c.D = static_cast<const T *>(D);
    c.W = static_cast<const T *>(W);
    c.O = static_cast<T *>(O);
    c.cd1 = ck.cd1; c.cd2 = ck.cd2; c.cw1 = ck.cw1; c.cw2 = ck.cw2;
    c.co5g = ck.co5; c.co6g = ck.co6; c.co7g = ck.co7;
    c.scale = tol_scale(pl.g, pol.kappa);
    c.eta = pol.eta;
    c.wb = pl.g.wbase;
    c.rc_on = pol.rc_on;
    c.clc_on = pol.clc_on;
    c.recompute = pol.repair == FTCNN_REPAIR_RECOMPUTE;
    c.rep = rep;
    c.bias = ck.bias;
    c.cb = ck.bias ? ck.cb : nullptr;
    c.wn = (double)pl.g.N * (double)pl.g.wbase + (double)pl.g.N * ((double)pl.g.N - 1.0) / 2.0;
    char *w = static_cast<char *>(ws);
    const int *flags = reinterpret_cast<const int *>(w + pl.off_flags);
    double *scratch = reinterpret_cast<double *>(w + pl.off_corr);
    int chunk = (pl.g.EF + pl.corr_blocks - 1) / pl.corr_blocks;
    chunk = chunk < 1 ? 1 : (chunk > kThreads ? kThreads : chunk);
    correct_kernel<T><<<(unsigned)pl.corr_blocks, kThreads, 0, st>>>(c, flags, scratch, pl.corr_stride, chunk);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_correct(const Plan &pl, const void *D, const void *W, void *O,
                          const ftcnn_checksums &ck, const ftcnn_policy &pol, ftcnn_report *rep,
                          void *ws, hipStream_t st) {
    if (pl.g.dtype == FTCNN_F32) return run<float>(pl, D, W, O, ck, pol, rep, ws, st);
    return run<uint16_t>(pl, D, W, O, ck, pol, rep, ws, st);
}

hipError_t launch_verify_correct(const Plan &pl, const void *D, const void *W, void *O,
                                 const ftcnn_checksums &ck, const ftcnn_policy &pol, ftcnn_report *rep,
                                 int cap, void *ws, hipStream_t st) {
    hipError_t e = launch_verify_partial(pl, O, rep, cap, ws, st);
    if (e != hipSuccess) return e;
    if (pl.g.dtype == FTCNN_F32)
        return run_fused<float>(pl, D, W, O, ck, pol, rep, ws, pl.off_ver, pl.ver_splits, false, st);
    return run_fused<uint16_t>(pl, D, W, O, ck, pol, rep, ws, pl.off_ver, pl.ver_splits, false, st);
}

hipError_t launch_verify_correct_sums(const Plan &pl, const void *D, const void *W, void *O,
                                      const ftcnn_checksums &ck, const ftcnn_policy &pol, ftcnn_report *rep,
                                      bool coc, void *ws, hipStream_t st) {
    if (pl.g.dtype == FTCNN_F32)
        return run_fused<float>(pl, D, W, O, ck, pol, rep, ws, pl.off_sums, pl.sum_splits, coc, st);
    return run_fused<uint16_t>(pl, D, W, O, ck, pol, rep, ws, pl.off_sums, pl.sum_splits, coc, st);
}

}  // namespace ftcnn
