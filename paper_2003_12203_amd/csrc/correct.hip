// Correction module of the multischeme workflow (Sec. 4.3, Fig. 7).
//
// Every scheme of Sec. 3 compares checksums element by element inside the
// output blocks (Level 2 of Sec. 3.2), so each flagged position p is repaired
// independently, through the chain:
//
//   CoC  (Sec. 3.6)   i = (Co7-So7)/(Co5-So5), j = (Co6-So6)/(Co5-So5)
//   RC   (Sec. 3.4)   per mismatching column m: i = (Co3-So3)/(Co1-So1)
//   ClC  (Sec. 3.5)   per mismatching row n:    j = (Co4-So4)/(Co2-So2)
//   FC   (Sec. 3.3, 4.1.5) row/column mismatch sets; Co6/Co5 or Co7/Co5
//                     locate the column or row when Co1 or Co2 is blind
//
// Two launches.  The launch that flags a position (the final detection launch, or
// the standalone correction launch) only hands it over, with its checksums, to
// the wide stage: one more launch that does nothing when no position is handed
// over.  Its workgroups compute, for every handed position, one work item per
// filter m (Co1, Co3 over the filter's taps, and So1, So3 and two sums of squares
// over the images) and one per image n (Co2, Co4 over the image's window, and
// So2, So4 and a sum of squares over the filters): K-long float64 dot products
// against checksum blocks, M + N of them a position, the whole cost of a scheme
// under Level-2 independence, each item one wave's.  The last workgroup to finish
// takes the decisions of every scheme from those sums: So5..So7 and their Q are
// sums of the per-filter sums (Co5 = sum_m Co1[m], Co6 = sum_m (m + wbase)
// Co1[m], Co7 = sum_m Co3[m], Sec. 3.2), so no workgroup walks all N x M blocks
// of a position.  A scheme's repairs are undone unless Co5, Co6 and Co7 agree
// with the re-summed output afterwards (the repaired filters re-summed over the
// images).  When a weighted checksum agrees while Co5 does not, the checksums
// themselves are suspect (Sec. 4.1.4): Co5..Co7 are re-derived from D and W at p,
// and if O agrees with them the position is closed without a repair.
//
// Every sum is a fixed-shape reduction (per-lane serial, then a wave butterfly,
// then the four waves in order), so a rerun gives identical bits.
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

struct Sh {
    double red[8][4];
    double unit_rows[4][kRowSums];   // a filter unit's results, stored to global memory by thread 0
    int slot;
    int nfix, fail, cnt_m, cnt_n, one_m, one_n;
    double bcast[4];
};

template <typename T> struct Ctx {
    Geom g;
    const T *D, *W;
    T *O;
    const double *cd1, *cd2, *cw1, *cw2, *co5g, *co6g, *co7g;
    const double *so5g, *so6g, *so7g, *q5g;   // the detection's sums (the standalone launch; may be NULL)
    double scale, eta;
    int wb, rc_on, clc_on, recompute;
    double *co1m, *d1, *d3, *q1;   // per filter m at the current position
    double *co2n, *d2, *d4, *q2;   // per image n at the current position
    int *fix_n, *fix_m;
    uint32_t *fix_old;
    int *colmark;   // [M]: filters with a repair at the current position (zero between schemes)
    ftcnn_report *rep;
    // bias (Sec. 5.1): NULL, or [M] with cb = {sum_m bias[m], sum_m (m + wbase) bias[m]};
    // wn = sum_n (n + wbase)
    const float *bias;
    const double *cb;
    double wn;
    // the wide stage's sums for the current position: per filter (kRowSums each), per image
    // (kColSums each), and Co5..Co7 re-encoded from D and W (NULL unless computed)
    const double *pre_rows, *pre_cols, *pre_fresh;
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
template <typename T> __device__ inline long long oidx(const Ctx<T> &c, int n, int m, int p) {
    return ((long long)n * c.g.M + m) * c.g.EF + p;
}

__device__ inline int legal(double r, int hi, double eta) {
    if (!isfinite(r)) return -1;
    const double i = rint(r);
    if (fabs(r - i) > eta || i < 0.0 || i >= (double)hi) return -1;
    return (int)i;
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

// Per filter m at p, from the wide stage's sums: Co1 = Cd1 (x) W_m, Co3 = Cd2 (x) W_m and the
// differences to So1 = sum_n O_nm, So3 = sum_n (n + wbase) O_nm.  So1[m] carries N bias[m] and
// So3[m] sum_n (n + wbase) bias[m] (Sec. 5.1); co1m keeps the shifted Co1, so the repairs from it
// give biased values.
template <typename T> __device__ void row_arrays(const Ctx<T> &c) {
    const Geom &g = c.g;
    for (int m = threadIdx.x; m < g.M; m += kThreads) {
        const double *r = c.pre_rows + kRowSums * (size_t)m;
        const double bm = bias_of(c, m);
        c.co1m[m] = r[0] + (double)g.N * bm;
        c.d1[m] = c.co1m[m] - r[2];
        c.d3[m] = r[1] + c.wn * bm - r[3];
        c.q1[m] = sqrt(r[4]);
    }
    __syncthreads();
}

// Per image n at p, from the wide stage's sums: Co2 = D_n (x) Cw1, Co4 = D_n (x) Cw2 and the
// differences to So2 = sum_m O_nm, So4 = sum_m (m + wbase) O_nm, which carry sum_m bias[m] and
// sum_m (m + wbase) bias[m] (Sec. 5.1).
template <typename T> __device__ void col_arrays(const Ctx<T> &c) {
    const Geom &g = c.g;
    const double b1 = c.bias ? c.cb[0] : 0.0, b2 = c.bias ? c.cb[1] : 0.0;
    for (int n = threadIdx.x; n < g.N; n += kThreads) {
        const double *r = c.pre_cols + kColSums * (size_t)n;
        c.co2n[n] = r[0] + b1;
        c.d2[n] = c.co2n[n] - r[2];
        c.d4[n] = r[1] + b2 - r[3];
        c.q2[n] = sqrt(r[4]);
    }
    __syncthreads();
}

// sum_{n != i} O[n][m][p] in index order, eight loads in flight.
template <typename T> __device__ double excl_sum_n(const Ctx<T> &c, int m, int p, int i) {
    const long long step = (long long)c.g.M * c.g.EF;
    const T *b = c.O + (long long)m * c.g.EF + p;
    double s = 0.0;
    int n = 0;
    for (; n + 8 <= c.g.N; n += 8) {
        double v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = ldo(b, (long long)(n + u) * step);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (n + u != i) s += v[u];
    }
    for (; n < c.g.N; ++n)
        if (n != i) s += ldo(b, (long long)n * step);
    return s;
}
// sum_{m != j} O[n][m][p] by one wave (M can be large): lane l takes m = l, l + 64, ... with
// eight loads in flight, then a butterfly; every lane returns the sum.
template <typename T> __device__ double wave_excl_sum_m(const Ctx<T> &c, int n, int p, int j, int lane) {
    const long long step = c.g.EF;
    const T *b = c.O + (long long)n * c.g.M * c.g.EF + p;
    double s = 0.0;
    int m = lane;
    for (; m + 7 * 64 < c.g.M; m += 8 * 64) {
        double v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = ldo(b, (long long)(m + u * 64) * step);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (m + u * 64 != j) s += v[u];
    }
    for (; m < c.g.M; m += 64)
        if (m != j) s += ldo(b, (long long)m * step);
    return wave_sum(s);
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

// Sums over the images of filter m's blocks at p, in image order with eight loads in flight:
// o, (n + wbase) o, o^2 and ((n + wbase) o)^2.
template <typename T> __device__ void column_sums(const Ctx<T> &c, int m, int p, double (&v)[4]) {
    const long long step = (long long)c.g.M * c.g.EF;
    const T *b = c.O + (long long)m * c.g.EF + p;
    const double wb = (double)c.wb;
    v[0] = v[1] = v[2] = v[3] = 0.0;
    auto add = [&](int n, double o) {
        const double t = ((double)n + wb) * o;
        v[0] += o;
        v[1] = fma((double)n + wb, o, v[1]);
        v[2] = fma(o, o, v[2]);
        v[3] = fma(t, t, v[3]);
    };
    int n = 0;
    for (; n + 8 <= c.g.N; n += 8) {
        double o[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) o[u] = ldo(b, (long long)(n + u) * step);
#pragma unroll
        for (int u = 0; u < 8; ++u) add(n + u, o[u]);
    }
    for (; n < c.g.N; ++n) add(n, ldo(b, (long long)n * step));
}

// So5, So6, So7 and their Q at p (Sec. 3.6) from per-filter sums: the wide stage's, or a fresh
// pass over the images for the filters marked in colmark (those with a repair).  Co5 =
// sum_m Co1[m], Co6 = sum_m (m + wbase) Co1[m] and Co7 = sum_m Co3[m] (Sec. 3.2) hold for the
// summations alike, so no pass over all N x M blocks is needed.
template <typename T> __device__ void position_sums(const Ctx<T> &c, Sh &sh, int p, bool marks, double (&s)[6]) {
    const Geom &g = c.g;
    const double wb = (double)c.wb;
    double v[6] = {0, 0, 0, 0, 0, 0};
    for (int m = threadIdx.x; m < g.M; m += kThreads) {
        double col[4];
        if (marks && c.colmark[m]) {
            column_sums(c, m, p, col);
        } else {
            const double *r = c.pre_rows + kRowSums * (size_t)m;
            col[0] = r[2]; col[1] = r[3]; col[2] = r[4]; col[3] = r[5];
        }
        const double wm = (double)m + wb;
        v[0] += col[0];
        v[1] = fma(wm, col[0], v[1]);
        v[2] += col[1];
        v[3] += col[2];
        v[4] = fma(wm * wm, col[2], v[4]);
        v[5] += col[3];
    }
    bsum<6>(v, sh);
    s[0] = v[0]; s[1] = v[1]; s[2] = v[2];
    s[3] = sqrt(v[3]); s[4] = sqrt(v[4]); s[5] = sqrt(v[5]);
}

// Keep the repairs if the CoC checksums agree afterwards, else undo them.
template <typename T> __device__ bool settle(const Ctx<T> &c, Sh &sh, int p, const double (&co)[3]) {
    __syncthreads();
    if (sh.nfix == 0) return false;
    for (int s = threadIdx.x; s < sh.nfix; s += kThreads) c.colmark[c.fix_m[s]] = 1;
    __syncthreads();
    double v[6];
    position_sums(c, sh, p, true, v);
    for (int s = threadIdx.x; s < sh.nfix; s += kThreads) c.colmark[c.fix_m[s]] = 0;
    __syncthreads();
    if (!is_bad(co[0] - v[0], v[3], c.scale) && !is_bad(co[1] - v[1], v[4], c.scale) &&
        !is_bad(co[2] - v[2], v[5], c.scale))
        return true;
    undo(c, sh, p);
    return false;
}

// Repair (i, m) for every m of the row mismatch set from Co1 (exclusive sum over n != i).
template <typename T> __device__ void fix_row_members(const Ctx<T> &c, Sh &sh, int p, int x, int y, int i) {
    for (int m = threadIdx.x; m < c.g.M; m += kThreads) {
        if (!is_bad(c.d1[m], c.q1[m], c.scale)) continue;
        const double v = c.recompute ? element(c, i, m, x, y) : c.co1m[m] - excl_sum_n(c, m, p, i);
        repair(c, sh, i, m, p, v);
    }
}

// Repair (n, j) for every n of the column mismatch set from Co2 (exclusive sum over m != j).
// (one wave per image n of the set; its lane 0 repairs)
template <typename T> __device__ void fix_col_members(const Ctx<T> &c, Sh &sh, int p, int x, int y, int j) {
    const int lane = threadIdx.x & 63;
    for (int n = threadIdx.x >> 6; n < c.g.N; n += kThreads / 64) {
        if (!is_bad(c.d2[n], c.q2[n], c.scale)) continue;
        const double ex = c.recompute ? 0.0 : wave_excl_sum_m(c, n, p, j, lane);
        if (lane == 0) repair(c, sh, n, j, p, c.recompute ? element(c, n, j, x, y) : c.co2n[n] - ex);
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
    // the exclusive sum of R7: the other filters' sums, then filter j's blocks but (i, j)
    double a[1] = {0.0};
    if (c.recompute) {
        // Eq. (1) over filter j's channel group on a grouped layer (Sec. 5.2), by the workgroup
        const T *Dn = c.D + (long long)i * c.g.CHW + (long long)group_first_channel(c.g, j) * c.g.H * c.g.W;
        const T *Wm = c.W + (long long)j * c.g.Kg;
        for (int k = threadIdx.x; k < c.g.Kg; k += kThreads) {
            const int RS = c.g.R * c.g.S;
            const int ch = k / RS, rem = k - ch * RS, r = rem / c.g.S, s = rem - r * c.g.S;
            const int ih = c.g.U * x + r - c.g.P, iw = c.g.U * y + s - c.g.P;
            if (ih >= 0 && ih < c.g.H && iw >= 0 && iw < c.g.W)
                a[0] = fma(ldo(Dn, ((long long)ch * c.g.H + ih) * c.g.W + iw), ldo(Wm, k), a[0]);
        }
    } else {
        for (int m = threadIdx.x; m < c.g.M; m += kThreads)
            if (m != j) a[0] += c.pre_rows[kRowSums * (size_t)m + 2];
    }
    bsum<1>(a, sh);
    if (threadIdx.x == 0) {
        const double v = c.recompute ? a[0] + bias_of(c, j) : co[0] - (a[0] + excl_sum_n(c, j, p, i));
        repair(c, sh, i, j, p, v);
    }
    return settle(c, sh, p, co);
}

template <typename T>
__device__ bool scheme_rc(const Ctx<T> &c, Sh &sh, int p, int x, int y, const double (&co)[3]) {
    row_arrays(c);
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
        const double v = c.recompute ? element(c, i, m, x, y) : c.co1m[m] - excl_sum_n(c, m, p, i);
        repair(c, sh, i, m, p, v);
    }
    return settle(c, sh, p, co);
}

template <typename T>
__device__ bool scheme_clc(const Ctx<T> &c, Sh &sh, int p, int x, int y, const double (&co)[3]) {
    col_arrays(c);
    col_set(c, sh);
    if (sh.cnt_n == 0) return false;
    begin_scheme<T>(sh);
    for (int n = threadIdx.x; n < c.g.N; n += kThreads)
        if (is_bad(c.d2[n], c.q2[n], c.scale) && legal(c.d4[n] / c.d2[n] - (double)c.wb, c.g.M, c.eta) < 0)
            atomicOr(&sh.fail, 1);
    __syncthreads();
    if (sh.fail) return false;
    // one wave per image n of the set; its lane 0 repairs
    const int lane = threadIdx.x & 63;
    for (int n = threadIdx.x >> 6; n < c.g.N; n += kThreads / 64) {
        if (!is_bad(c.d2[n], c.q2[n], c.scale)) continue;
        const int j = legal(c.d4[n] / c.d2[n] - (double)c.wb, c.g.M, c.eta);
        const double ex = c.recompute ? 0.0 : wave_excl_sum_m(c, n, p, j, lane);
        if (lane == 0) repair(c, sh, n, j, p, c.recompute ? element(c, n, j, x, y) : c.co2n[n] - ex);
    }
    return settle(c, sh, p, co);
}

template <typename T>
__device__ bool scheme_fc(const Ctx<T> &c, Sh &sh, int p, int x, int y, const double (&co)[3],
                          const double (&d)[3], bool have_rows, bool have_cols) {
    if (!have_rows) row_arrays(c);
    if (!have_cols) col_arrays(c);
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

template <typename T> __device__ void unresolved(const Ctx<T> &c, Sh &sh, int x, int y) {
    begin_scheme<T>(sh);
    record(c, sh, FTCNN_SCHEME_UNRESOLVED, x, y);
}

// The chain at one handed-over position, from the wide stage's sums in c.pre_*: CoC, RC, ClC,
// FC, else recomputation (Sec. 4.3), after the suspect-checksum test of Sec. 4.1.4.
template <typename T>
__device__ __attribute__((always_inline)) void decide(const Ctx<T> &c, Sh &sh, int p, const double (&co_in)[3]) {
    const int x = p / c.g.F, y = p - (p / c.g.F) * c.g.F;
    double co[3] = {co_in[0], co_in[1], co_in[2]};
    double s[6];
    position_sums(c, sh, p, false, s);
    double d[3] = {co[0] - s[0], co[1] - s[1], co[2] - s[2]};
    const bool agree = !is_bad(d[0], s[3], c.scale) || !is_bad(d[1], s[4], c.scale) ||
                       !is_bad(d[2], s[5], c.scale);
    if (agree) {  // an inconsistent pattern among Co5/Co6/Co7: suspect the checksums
        // the flagging launch asks for the fresh checksums whenever a weighted checksum can
        // agree (see may_agree), so they are here
        if (!c.pre_fresh) return unresolved(c, sh, x, y);
        double f[3] = {c.pre_fresh[0], c.pre_fresh[1], c.pre_fresh[2]};
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
    unresolved(c, sh, x, y);
}

// Whether a weighted checksum can agree at a flagged position (the suspect-checksum case): from
// the detection's So5..So7 and Q5 alone, since Q6 <= (M - 1 + wbase) Q5 and Q7 <= (N - 1 + wbase) Q5.
// A loose bound (it errs towards yes): it only decides whether the wide stage re-encodes Co5..Co7.
__device__ inline int may_agree(const Geom &g, double scale, const double (&cs)[3], double so5, double so6,
                                double so7, double q5) {
    const double d1 = cs[1] - so6, d2 = cs[2] - so7, d0 = cs[0] - so5;
    const double slack = 1.0 + 1e-6;
    const double b6 = scale * ((double)g.M - 1.0 + (double)g.wbase) * q5 * slack;
    const double b7 = scale * ((double)g.N - 1.0 + (double)g.wbase) * q5 * slack;
    if (!isfinite(b6) || !isfinite(b7)) return 1;
    return (isfinite(d1) && fabs(d1) <= b6) || (isfinite(d2) && fabs(d2) <= b7) ||
           (isfinite(d0) && fabs(d0) <= scale * q5 * slack);
}

// Hand position p over to the wide stage (one thread).  The list has room for every position of
// the layer, each flagged once per call; should the report's counter not have been cleared, the
// position is left to recomputation.
__device__ inline void hand_over(const Geom &g, ftcnn_report *rep, Pending *pend, int p, int mode,
                                 const double (&co)[3]) {
    const int idx = atomicAdd(&rep->reserved[0], 1);
    if (idx < g.EF) {
        Pending &e = pend[idx];
        e.p = p;
        e.mode = mode;
        e.co[0] = co[0];
        e.co[1] = co[1];
        e.co[2] = co[2];
    } else {
        atomicAdd(&rep->resolved_by[FTCNN_SCHEME_UNRESOLVED], 1);
        atomicMax(&rep->status, FTCNN_STATUS_NEEDS_RECOMPUTE);
    }
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
    c.colmark = c.fix_m + L;
}

// The standalone correction launch: hands every position the detection flagged over to the wide
// stage (nothing to do when nothing was detected).
template <typename T>
__global__ __launch_bounds__(kThreads) void correct_kernel(Ctx<T> c, const int *__restrict__ flags, Pending *pend,
                                                           int *wide_done) {
    if (blockIdx.x == 0 && threadIdx.x <= kDoneGroups) wide_done[kDoneStride * threadIdx.x] = 0;  // the wide stage's count
    if (c.rep->detected == 0) return;
    const Geom &g = c.g;
    const bool sums = c.so5g && c.so6g && c.so7g && c.q5g;
    for (int p = blockIdx.x * kThreads + threadIdx.x; p < g.EF; p += gridDim.x * kThreads) {
        if (!flags[p]) continue;
        double co[3] = {c.co5g[p], c.co6g[p], c.co7g[p]};
        add_bias_shares(c, co);
        const int mode = sums ? may_agree(g, c.scale, co, c.so5g[p], c.so6g[p], c.so7g[p], c.q5g[p]) : 1;
        hand_over(g, c.rep, pend, p, mode, co);
    }
}

// The wide stage of the chain (one launch after the flagging one; nothing to do when no position
// was handed over).  Work items of a handed-over position p: one per filter m (Co1 = Cd1 (x) W_m
// and Co3 = Cd2 (x) W_m over the filter's taps, and So1, So3 and the sums of o^2 and of
// ((n + wbase) o)^2 over the images at p) and one per image n (Co2 = D_n (x) Cw1, Co4 = D_n (x) Cw2, and So2, So4 and the sum of
// squares over the filters); each item is one wave's, its lanes taking every 64th term in order and
// folding them by a fixed butterfly.  For suspect checksums (mode 1), Co5..Co7 re-encoded from D
// and W are summed over kFreshRanges fixed ranges of taps, the ranges then added in range order.
// The items of the first kMaxPending positions are spread over every wave of the launch, and the
// last workgroup to finish (a completion counter, no waiting) takes their decisions; a workgroup
// takes any further position whole, items and decisions.  Either way a position's sums have the
// same bits.
__device__ inline long long tap_offset(const Geom &g, int x, int y, int k) {
    const int RS = g.R * g.S;
    const int ch = k / RS, rem = k - ch * RS, r = rem / g.S, s = rem - r * g.S;
    const int ih = g.U * x + r - g.P, iw = g.U * y + s - g.P;
    return (ih >= 0 && ih < g.H && iw >= 0 && iw < g.W) ? ((long long)ch * g.H + ih) * g.W + iw : -1;
}

// The window of position p in Cd1 and Cd2 for every tap k, and whether the tap is inside the input
// (a tap in the zero padding holds 0 and is skipped), staged in shared memory by the workgroup for
// its filter items.  Thread t takes the taps t, t + 256, ..., ten in flight.
struct Window {
    double *c1, *c2;
    unsigned char *in;
};
template <typename T> __device__ void stage_window(const Ctx<T> &c, int p, const Window &w) {
    const Geom &g = c.g;
    const int x = p / g.F, y = p - x * g.F;
    const int RS = g.R * g.S;
    const int dch = kThreads / RS, drem = kThreads - dch * RS, dr = drem / g.S, ds = drem - dr * g.S;
    const int ih0 = g.U * x - g.P, iw0 = g.U * y - g.P;
    int ch = threadIdx.x / RS, rem = threadIdx.x - ch * RS;
    int r = rem / g.S, s = rem - r * g.S;
    constexpr int U = 10;
    __syncthreads();
    for (int k = threadIdx.x; k < g.K; k += U * kThreads) {
        double a[U], b[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int ih = ih0 + r, iw = iw0 + s;
            ok[u] = k + u * kThreads < g.K && ((unsigned)ih < (unsigned)g.H) & ((unsigned)iw < (unsigned)g.W);
            const long long off = ok[u] ? ((long long)ch * g.H + ih) * g.W + iw : 0;
            a[u] = c.cd1[off];
            b[u] = c.cd2[off];
            s += ds;
            r += dr;
            ch += dch;
            if (s >= g.S) { s -= g.S; ++r; }
            if (r >= g.R) { r -= g.R; ++ch; }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kk = k + u * kThreads;
            if (kk < g.K) {
                w.c1[kk] = ok[u] ? a[u] : 0.0;
                w.c2[kk] = ok[u] ? b[u] : 0.0;
                w.in[kk] = ok[u];
            }
        }
    }
    __syncthreads();
}

// Filter unit u of position p: filters m = 4u + w, one a wave w: Co1 = Cd1 (x) W_m and
// Co3 = Cd2 (x) W_m over the filter's taps (its channel group, Sec. 5.2), So1, So3, sum o^2 and
// sum ((n + wbase) o)^2 over the images; the kRowSums sums of each filter go to rows_q (thread 0
// stores them: every store the wide stage publishes is thread 0's).  Lane l takes the taps
// k = l, l + 64, ... in order, a tap in the zero padding skipped (its weight not used).  With the
// window in shared memory, W is read in batches of kWBatch taps a lane, the next batch loaded
// while the current one is used, and the first batch (and the first 64 blocks of O) loaded before
// the window is staged (stage: the workgroup stages it here); without it, Cd1 and Cd2 are read
// straight.
constexpr int kWBatch = 24;
template <typename T>
__device__ __attribute__((always_inline)) void load_wbatch(const T *wr, int k, int kg, float (&w)[kWBatch]) {
#pragma unroll
    for (int u = 0; u < kWBatch; ++u) {
        const int kk = k + u * 64;
        w[u] = (float)ldo(wr, kk < kg ? kk : 0);
    }
}
__device__ __attribute__((always_inline)) void use_wbatch(const float (&w)[kWBatch], int k, int kg, int kg0, const Window &win, double &a,
                                  double &b) {
#pragma unroll
    for (int u = 0; u < kWBatch; ++u) {
        const int kk = k + u * 64;
        if (kk < kg) {
            const double wv = win.in[kg0 + kk] ? (double)w[u] : 0.0;
            a = fma(win.c1[kg0 + kk], wv, a);
            b = fma(win.c2[kg0 + kk], wv, b);
        }
    }
}

template <typename T>
__device__ void filter_unit(const Ctx<T> &c, Sh &sh, int p, int u, bool stage, const Window &win, double *rows_q) {
    const Geom &g = c.g;
    const int x = p / g.F, y = p - x * g.F;
    const double wb = (double)c.wb;
    const int RS = g.R * g.S;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int m = 4 * u + wave;
    const bool live = m < g.M;
    const int mm = live ? m : g.M - 1;   // a wave past the last filter repeats it, results unused
    const int cg0 = group_first_channel(g, mm), kg0 = cg0 * RS;
    const T *wr = c.W + (long long)mm * g.Kg;
    const double o0 = lane < g.N ? ldo(c.O, oidx(c, lane, mm, p)) : 0.0;
    double a = 0.0, b = 0.0;
    if (win.c1) {
        constexpr int B = kWBatch * 64;
        float w0[kWBatch], w1[kWBatch];
        load_wbatch(wr, lane, g.Kg, w0);
        if (stage) stage_window(c, p, win);
        for (int k = lane;;) {
            if (k + B < g.Kg) load_wbatch(wr, k + B, g.Kg, w1);
            use_wbatch(w0, k, g.Kg, kg0, win, a, b);
            k += B;
            if (k >= g.Kg) break;
            if (k + B < g.Kg) load_wbatch(wr, k + B, g.Kg, w0);
            use_wbatch(w1, k, g.Kg, kg0, win, a, b);
            k += B;
            if (k >= g.Kg) break;
        }
    } else {
        const int ih0 = g.U * x - g.P, iw0 = g.U * y - g.P;
        for (int k = lane; k < g.Kg; k += 64) {
            const int ch = k / RS, rem = k - ch * RS, r = rem / g.S, s = rem - r * g.S;
            const int ih = ih0 + r, iw = iw0 + s;
            const double w = ldo(wr, k);
            if ((unsigned)ih < (unsigned)g.H && (unsigned)iw < (unsigned)g.W) {
                const long long off = ((long long)(cg0 + ch) * g.H + ih) * g.W + iw;
                a = fma(c.cd1[off], w, a);
                b = fma(c.cd2[off], w, b);
            } else {
                a = fma(0.0, 0.0, a);
                b = fma(0.0, 0.0, b);
            }
        }
    }
    double s1 = 0.0, s2 = 0.0, sq = 0.0, tq = 0.0;
#pragma unroll 4
    for (int n = lane; n < g.N; n += 64) {
        const double o = n == lane ? o0 : ldo(c.O, oidx(c, n, mm, p));
        const double t = ((double)n + wb) * o;
        s1 += o;
        s2 = fma((double)n + wb, o, s2);
        sq = fma(o, o, sq);
        tq = fma(t, t, tq);
    }
    a = wave_sum(a);
    b = wave_sum(b);
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    sq = wave_sum(sq);
    tq = wave_sum(tq);
    if (lane == 0 && live) {
        double *r = sh.unit_rows[wave];
        r[0] = a;
        r[1] = b;
        r[2] = s1;
        r[3] = s2;
        r[4] = sq;
        r[5] = tq;
    }
    __syncthreads();
    if (threadIdx.x == 0)
        for (int w = 0; w < 4 && 4 * u + w < g.M; ++w)
            for (int i = 0; i < kRowSums; ++i) rows_q[(size_t)(4 * u + w) * kRowSums + i] = sh.unit_rows[w][i];
    __syncthreads();
}

// Image n at position p, by the whole workgroup: Co2 = D_n (x) Cw1, Co4 = D_n (x) Cw2 over all K
// taps, and So2, So4 and sum o^2 over the filters; thread 0 stores the kColSums sums at out.
// Thread t takes the taps k = t, t + 256, ... in order (eight in flight) and the filters
// m = t, t + 256, ...; the threads' sums are then folded in a fixed order.
template <typename T> __device__ void image_item(const Ctx<T> &c, Sh &sh, int p, int n, double *out) {
    const Geom &g = c.g;
    const int x = p / g.F, y = p - x * g.F;
    const double wb = (double)c.wb;
    const int RS = g.R * g.S;
    const int dch = kThreads / RS, drem = kThreads - dch * RS, dr = drem / g.S, ds = drem - dr * g.S;
    const int ih0 = g.U * x - g.P, iw0 = g.U * y - g.P;
    const int t0 = threadIdx.x;
    int ch = t0 / RS, rem = t0 - ch * RS;
    int r = rem / g.S, s = rem - r * g.S;
    const T *dn = c.D + (long long)n * g.CHW;
    constexpr int U = 8;
    double v[5] = {0.0, 0.0, 0.0, 0.0, 0.0};
    for (int k = t0; k < g.K; k += U * kThreads) {
        double dv[U], w1[U], w2[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kk = k + u * kThreads;
            const int ih = ih0 + r, iw = iw0 + s;
            ok[u] = kk < g.K && ((unsigned)ih < (unsigned)g.H) & ((unsigned)iw < (unsigned)g.W);
            const int kw = kk < g.K ? kk : 0;
            dv[u] = ldo(dn, ok[u] ? ((long long)ch * g.H + ih) * g.W + iw : 0);
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
                v[0] = fma(dv[u], w1[u], v[0]);
                v[1] = fma(dv[u], w2[u], v[1]);
            }
    }
#pragma unroll 4
    for (int m = t0; m < g.M; m += kThreads) {
        const double o = ldo(c.O, oidx(c, n, m, p));
        v[2] += o;
        v[3] = fma((double)m + wb, o, v[3]);
        v[4] = fma(o, o, v[4]);
    }
    bsum<5>(v, sh);
    if (threadIdx.x == 0)
        for (int i = 0; i < 5; ++i) out[i] = v[i];
}

// Work units of a position: unit u < ceil(M / 4) is filters 4u .. 4u + 3 (one a wave), unit
// ceil(M / 4) + n is image n.
__device__ inline int filter_units(const Geom &g) { return (g.M + 3) / 4; }
__device__ inline int position_units(const Geom &g) { return filter_units(g) + g.N; }

template <typename T>
__device__ __attribute__((always_inline)) void run_unit(const Ctx<T> &c, Sh &sh, int p, int u, bool stage,
                                                        double *rows_q, double *cols_q, const Window &win) {
    const Geom &g = c.g;
    const int nf = filter_units(g);
    if (u < nf) {
        filter_unit(c, sh, p, u, stage, win, rows_q);
    } else {
        image_item(c, sh, p, u - nf, cols_q + (size_t)(u - nf) * kColSums);
    }
}

// Co5..Co7 at (x, y) from checksums re-encoded out of D and W (Sec. 4.1.4) over the taps of range
// b of kFreshRanges, by the whole workgroup: wave w takes the taps k0 + w, k0 + w + 4, ...; for a
// tap its lanes sum D over the images and W over the filters of the tap's channel group (folded by
// a butterfly), and the tap's products are added in the wave's tap order; then the four waves'
// sums in wave order.
template <typename T>
__device__ __attribute__((always_inline)) void fresh_range(const Ctx<T> &c, int x, int y, int b, Sh &sh, double (&v)[3]) {
    const Geom &g = c.g;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const double wb = (double)c.wb;
    const long long k0 = (long long)g.K * b / kFreshRanges, k1 = (long long)g.K * (b + 1) / kFreshRanges;
    const int RS = g.R * g.S;
    double acc[3] = {0.0, 0.0, 0.0};
    for (long long k = k0 + wave; k < k1; k += 4) {
        const long long off = tap_offset(g, x, y, (int)k);
        if (off < 0) continue;   // the same for every lane of the wave
        double a1 = 0.0, a2 = 0.0, b1 = 0.0, b2 = 0.0;
#pragma unroll 4
        for (int n = lane; n < g.N; n += 64) {
            const double dv = ldo(c.D, (long long)n * g.CHW + off);
            a1 += dv;
            a2 = fma((double)n + wb, dv, a2);
        }
        const int grp = (int)(k / RS) / g.Cg;
        const long long kl = k - (long long)grp * g.Cg * RS;
#pragma unroll 8
        for (int m = grp * g.Mg + lane; m < (grp + 1) * g.Mg; m += 64) {
            const double wv = ldo(c.W, (long long)m * g.Kg + kl);
            b1 += wv;
            b2 = fma((double)m + wb, wv, b2);
        }
        a1 = wave_sum(a1);
        a2 = wave_sum(a2);
        b1 = wave_sum(b1);
        b2 = wave_sum(b2);
        acc[0] = fma(a1, b1, acc[0]);
        acc[1] = fma(a1, b2, acc[1]);
        acc[2] = fma(a2, b1, acc[2]);
    }
    __syncthreads();
    if (lane == 0)
        for (int i = 0; i < 3; ++i) sh.red[i][wave] = acc[i];
    __syncthreads();
    for (int i = 0; i < 3; ++i) v[i] = ((sh.red[i][0] + sh.red[i][1]) + sh.red[i][2]) + sh.red[i][3];
}

// Whether this workgroup is the last of the launch to get here (every workgroup calls it once):
// its own group's counter first, and the last of each group in the top counter.  Every store the
// stage publishes is thread 0's, so thread 0's fence makes them visible to the last workgroup.
__device__ inline bool last_to_finish(int *done, Sh &sh, int blk, int nblk) {
    __syncthreads();
    if (threadIdx.x == 0) {
        __threadfence();
        const int grp = blk % kDoneGroups;
        const int members = (nblk - grp + kDoneGroups - 1) / kDoneGroups;
        int last = 0;
        if (atomicAdd(&done[kDoneStride * (1 + grp)], 1) == members - 1) {
            __threadfence();
            const int groups = nblk < kDoneGroups ? nblk : kDoneGroups;
            last = atomicAdd(&done[0], 1) == groups - 1;
        }
        sh.slot = last;
    }
    __syncthreads();
    if (sh.slot) __threadfence();
    return sh.slot != 0;
}

// The wide stage as workgroup blk of nblk (a launch of its own, or the helpers of the fused final
// launch).
struct WideArgs {
    unsigned char *corr;
    CorrLayout L;
    size_t stride;
    int use_win, cache_rows;
};

template <typename T>
__device__ __attribute__((always_inline)) void wide_body(Ctx<T> c, const WideArgs &wa, int blk, int nblk) {
    unsigned char *corr = wa.corr;
    const CorrLayout &L = wa.L;
    const size_t stride = wa.stride;
    const int use_win = wa.use_win, cache_rows = wa.cache_rows;
    const int np = min(c.rep->reserved[0], c.g.EF);
    if (np <= 0) return;
    __shared__ Sh sh;
    const Geom &g = c.g;
    const Pending *pend = reinterpret_cast<const Pending *>(corr + L.pend);
    double *rows = reinterpret_cast<double *>(corr + L.rows);
    double *cols = reinterpret_cast<double *>(corr + L.cols);
    double *fresh = reinterpret_cast<double *>(corr + L.fresh);
    int *done = reinterpret_cast<int *>(corr + L.done);
    const int nb = min(np, kMaxPending);
    bind_scratch(c, reinterpret_cast<double *>(corr + L.chain) + stride * blk);
    for (int m = threadIdx.x; m < g.M; m += kThreads) c.colmark[m] = 0;
    // the window of the position whose filters this workgroup is on (shared memory, when it fits)
    extern __shared__ double win_sm[];
    Window win{nullptr, nullptr, nullptr};
    if (use_win) win = Window{win_sm, win_sm + g.K, reinterpret_cast<unsigned char *>(win_sm + 2 * (size_t)g.K)};
    int staged = -1;
    // the shared batch: its units in contiguous runs, one run a workgroup; then its fresh
    // checksum ranges
    const int pu = position_units(g), nf = filter_units(g);
    const long long total = (long long)nb * pu;
    const long long run = (total + nblk - 1) / nblk;
    for (long long it = (long long)blk * run; it < total && it < (long long)(blk + 1) * run; ++it) {
        const int q = (int)(it / pu), u = (int)(it - (long long)q * pu);
        const int p = pend[q].p;
        const bool stage = win.c1 && u < nf && staged != q;
        if (stage) staged = q;
        run_unit(c, sh, p, u, stage, rows + (size_t)q * g.M * kRowSums, cols + (size_t)q * g.N * kColSums, win);
    }
    for (int q = 0; q < nb && blk < kFreshRanges; ++q) {
        if (pend[q].mode != 1) continue;
        const int p = pend[q].p, x = p / g.F;
        double v[3];
        fresh_range(c, x, p - x * g.F, blk, sh, v);
        if (threadIdx.x == 0) {
            double *f = fresh + ((size_t)q * kFreshRanges + blk) * 3;
            f[0] = v[0];
            f[1] = v[1];
            f[2] = v[2];
        }
    }
    // then the positions past the shared batch, one workgroup each on its own slabs; the last
    // workgroup to finish (a completion counter, no waiting) then takes the shared batch's decisions
    double *myrows = rows + (size_t)(kMaxPending + blk) * g.M * kRowSums;
    double *mycols = cols + (size_t)(kMaxPending + blk) * g.N * kColSums;
    bool batch = false;
    for (int q = kMaxPending + blk;; q += batch ? 1 : nblk) {
        if (!batch && q >= np) {
            if (!last_to_finish(done, sh, blk, nblk)) return;
            batch = true;
            q = 0;
        }
        if (batch && q >= nb) break;
        const Pending e = pend[q];
        const int x = e.p / g.F, y = e.p - (e.p / g.F) * g.F;
        if (!batch) {
            staged = -1;
            for (int u = 0; u < pu; ++u) run_unit(c, sh, e.p, u, win.c1 && u == 0, myrows, mycols, win);
            if (e.mode == 1) {
                double f[3] = {0.0, 0.0, 0.0};
                for (int b = 0; b < kFreshRanges; ++b) {
                    double v[3];
                    fresh_range(c, x, y, b, sh, v);
                    f[0] += v[0];
                    f[1] += v[1];
                    f[2] += v[2];
                }
                if (threadIdx.x == 0) sh.bcast[0] = f[0], sh.bcast[1] = f[1], sh.bcast[2] = f[2];
            }
            c.pre_rows = myrows;
            c.pre_cols = mycols;
        } else {
            if (e.mode == 1 && threadIdx.x == 0) {
                double f0 = 0.0, f1 = 0.0, f2 = 0.0;
                for (int b = 0; b < kFreshRanges; ++b) {
                    const double *f = fresh + ((size_t)q * kFreshRanges + b) * 3;
                    f0 += f[0];
                    f1 += f[1];
                    f2 += f[2];
                }
                sh.bcast[0] = f0;
                sh.bcast[1] = f1;
                sh.bcast[2] = f2;
            }
            c.pre_rows = rows + (size_t)q * g.M * kRowSums;
            c.pre_cols = cols + (size_t)q * g.N * kColSums;
        }
        __threadfence_block();
        __syncthreads();
        c.pre_fresh = e.mode == 1 ? sh.bcast : nullptr;
        if (cache_rows) {
            // the decisions read the per-filter sums several times: from shared memory (the
            // window's space, not needed again for this position)
            const int nr = g.M * kRowSums;
            for (int i = threadIdx.x; i < nr; i += 8 * kThreads) {
                double v[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) v[k] = i + k * kThreads < nr ? c.pre_rows[i + k * kThreads] : 0.0;
#pragma unroll
                for (int k = 0; k < 8; ++k)
                    if (i + k * kThreads < nr) win_sm[i + k * kThreads] = v[k];
            }
            __syncthreads();
            c.pre_rows = win_sm;
            staged = -1;
        }
        decide(c, sh, e.p, e.co);
        __syncthreads();
    }
    // every workgroup has read the count: clear it for the next call on this report
    if (threadIdx.x == 0) c.rep->reserved[0] = 0;
}

template <typename T>
__global__ __launch_bounds__(kThreads) void wide_kernel(Ctx<T> c, WideArgs wa) {
    wide_body(c, wa, (int)blockIdx.x, (int)gridDim.x);
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
// fixed order, then the CoC-D test); every position it flags is handed over to
// the wide stage, with its checksums, by the thread that flags it.  With COC the same
// lanes also produce Co5..Co7 of their position and store them: from the
// channel-range partials the convolution launch left (rep->reserved[1] of
// them), or else from the taps of Cd and Cw.
//
// TPP threads share a position, and consecutive threads take consecutive
// positions (thread t: position t % per, lane t / per), so every load of a
// partial slice is a coalesced run; the lanes of a position are then added in a
// fixed order (exchanges inside each wave, then the four waves).
struct DetectArgs {
    int splits, max_groups;
    const double *part, *copart;
    double *co5, *co6, *co7, *so5, *so6, *so7, *q5;
    int *flags;
    Pending *pend;
    int *wide_done;
};

// Detection block blk.
template <typename T, int TPP, bool COC>
__device__ __attribute__((always_inline)) void detect_block(const Ctx<T> &c, const DetectArgs &da, int blk) {
    const int splits = da.splits, max_groups = da.max_groups;
    const double *__restrict__ part = da.part;
    const double *__restrict__ copart = da.copart;
    double *co5 = da.co5, *co6 = da.co6, *co7 = da.co7, *so5 = da.so5, *so6 = da.so6, *so7 = da.so7, *q5 = da.q5;
    int *__restrict__ flags = da.flags;
    Pending *pend = da.pend;
    if (blk == 0 && threadIdx.x <= kDoneGroups) da.wide_done[kDoneStride * threadIdx.x] = 0;  // the wide stage's count
    constexpr int NV = COC ? 7 : 4;
    __shared__ double red[TPP > 1 ? NV : 1][TPP > 1 ? 4 * (kThreads / TPP) : 1];
    const Geom &g = c.g;
    constexpr int per = kThreads / TPP;
    const int slot = threadIdx.x % per, lane = threadIdx.x / per;
    const int p = blk * per + slot;
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
        if (flag) hand_over(g, c.rep, pend, p, may_agree(g, c.scale, cs, a, b, cc, q), cs);
    }
    const int cnt = __syncthreads_count(flag);
    if (cnt > 0 && threadIdx.x == 0) {
        atomicAdd(&c.rep->n_flagged, cnt);
        atomicMax(&c.rep->detected, 1);
    }
}

template <typename T, int TPP, bool COC>
__global__ __launch_bounds__(kThreads) void verify_correct_kernel(Ctx<T> c, DetectArgs da) {
    detect_block<T, TPP, COC>(c, da, (int)blockIdx.x);
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
    c.so5g = ck.so5; c.so6g = ck.so6; c.so7g = ck.so7; c.q5g = ck.q5;
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

// The wide stage's launch arguments: the window of a position, and the decisions' per-filter sums,
// in shared memory when they fit beside a second workgroup's.
inline WideArgs wide_args(const Plan &pl, void *ws, size_t *lds) {
    WideArgs wa;
    wa.corr = static_cast<unsigned char *>(ws) + pl.off_corr;
    wa.L = corr_layout(pl.g, pl.corr_stride);
    wa.stride = pl.corr_stride;
    const size_t win_bytes = (2 * sizeof(double) + 1) * (size_t)pl.g.K;
    const size_t row_bytes = sizeof(double) * kRowSums * (size_t)pl.g.M;
    wa.use_win = win_bytes <= kWindowBytes;
    wa.cache_rows = row_bytes <= kWindowBytes;
    *lds = std::max(wa.use_win ? win_bytes : 0, wa.cache_rows ? row_bytes : 0);
    return wa;
}

// The wide stage after a flagging launch: wide_grid workgroups that return at once unless
// positions were handed over.
template <typename T>
hipError_t launch_wide(const Plan &pl, const Ctx<T> &c, void *ws, hipStream_t st) {
    size_t lds = 0;
    const WideArgs wa = wide_args(pl, ws, &lds);
    wide_kernel<T><<<(unsigned)wide_grid(pl.g), kThreads, lds, st>>>(c, wa);
    return hipGetLastError();
}

template <typename T>
hipError_t run_fused(const Plan &pl, const void *D, const void *W, void *O, const ftcnn_checksums &ck,
                     const ftcnn_policy &pol, ftcnn_report *rep, void *ws, size_t off_part, int sp, bool coc,
                     hipStream_t st) {
    Ctx<T> c = make_ctx<T>(pl, D, W, O, ck, pol, rep);
    char *w = static_cast<char *>(ws);
    const CorrLayout L = corr_layout(pl.g, pl.corr_stride);
    DetectArgs da;
    da.splits = sp;
    da.part = reinterpret_cast<const double *>(w + off_part);
    da.flags = reinterpret_cast<int *>(w + pl.off_flags);
    da.pend = reinterpret_cast<Pending *>(w + pl.off_corr + L.pend);
    da.wide_done = reinterpret_cast<int *>(w + pl.off_corr + L.done);
    // Co5..Co7 of a channels-last layer come as partial slices from the convolution launch
    // (the kernel checks rep->reserved[1] and falls back to the taps)
    const int taps = coc ? (pl.co_in_conv ? pl.co.groups * pl.prep_ns : pl.g.K) : 0;
    const int tpp = final_tpp(sp, taps, pl.g.EF);
    da.copart = reinterpret_cast<const double *>(w + pl.off_copart);
    da.max_groups = pl.co_in_conv ? pl.co.groups * pl.prep_ns : 0;
    da.co5 = ck.co5; da.co6 = ck.co6; da.co7 = ck.co7;
    da.so5 = ck.so5; da.so6 = ck.so6; da.so7 = ck.so7; da.q5 = ck.q5;
    const unsigned blocks = (unsigned)((pl.g.EF + kThreads / tpp - 1) / (kThreads / tpp));
#define VC(TPP, COC) verify_correct_kernel<T, TPP, COC><<<blocks, kThreads, 0, st>>>(c, da)
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
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_wide<T>(pl, c, ws, st);
}

template <typename T>
hipError_t run(const Plan &pl, const void *D, const void *W, void *O, const ftcnn_checksums &ck,
               const ftcnn_policy &pol, ftcnn_report *rep, void *ws, hipStream_t st) {
    Ctx<T> c = make_ctx<T>(pl, D, W, O, ck, pol, rep);
    char *w = static_cast<char *>(ws);
    const int *flags = reinterpret_cast<const int *>(w + pl.off_flags);
    const CorrLayout L = corr_layout(pl.g, pl.corr_stride);
    Pending *pend = reinterpret_cast<Pending *>(w + pl.off_corr + L.pend);
    int *wide_done = reinterpret_cast<int *>(w + pl.off_corr + L.done);
    const unsigned blocks = (unsigned)std::min<long long>(pl.corr_blocks, (pl.g.EF + kThreads - 1) / kThreads);
    correct_kernel<T><<<blocks, kThreads, 0, st>>>(c, flags, pend, wide_done);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_wide<T>(pl, c, ws, st);
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
