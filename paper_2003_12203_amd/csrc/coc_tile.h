// Work that extra workgroups of the convolution launch do beside its
// matrix-core tiles when the layer's input checksums were encoded by the
// channels-last copy that precedes it (Sec. 3.2):
//
//   combine   Cd1, Cd2 = the image-split partial sums of that copy, added in
//             split order (only when the images were split);
//   CoC       the checksum-of-checksum products of Sec. 3.2 at every output
//             position, Co5 = Cd1 (x) Cw1, Co6 = Cd1 (x) Cw2, Co7 = Cd2 (x) Cw1,
//             as partial products over ranges of input channels and, when the
//             images were split, over the image ranges (the products are linear
//             in Cd1 and Cd2, so each image range's partial checksums give their
//             share); the final detection launch adds the slices in order.
//
// A CoC workgroup owns a tile of output positions, one channel range and one
// image range (or the combined Cd when the images were not split).  For
// each group of cc channels it stages the tile's input window of Cd1 and Cd2
// (float64, zero outside the feature map) in LDS, then every thread evaluates
// the R x S taps of its own position from there: each checksum element is read
// from memory once per tile instead of once per tap.
#pragma once

#include "ftcnn_internal.h"

namespace ftcnn {

// Sources of Cd1 and Cd2 for the extra workgroups: final arrays (ns = 1) or
// image-split partials [ns][2][Ch*H*W] (p2 = p1 + Ch*H*W, stride = 2*Ch*H*W).
struct CdSrc {
    const double *p1, *p2;
    long long stride;
    int ns;
};

// One combine workgroup: 2*NT consecutive elements of Cd1 and Cd2, each the sum of
// its ns image-range partials added in range order; four ranges of loads (sixteen
// values a thread) are in flight at a time.
template <int NT>
__device__ inline void combine_block(const Geom &g, const CdSrc &src, double *__restrict__ cd1,
                                     double *__restrict__ cd2, int blk) {
    const long long base = (long long)blk * 2 * NT + threadIdx.x;
    long long idx[2];
    bool in[2];
    double a[2][2] = {{0.0, 0.0}, {0.0, 0.0}};
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        idx[e] = base + e * NT;
        in[e] = idx[e] < g.CHW;
        if (!in[e]) idx[e] = 0;
    }
    for (int s0 = 0; s0 < src.ns; s0 += 4) {
        double x[4][2][2];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const long long off = (long long)(s0 + u < src.ns ? s0 + u : 0) * src.stride;
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                x[u][e][0] = src.p1[off + idx[e]];
                x[u][e][1] = src.p2[off + idx[e]];
            }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (s0 + u < src.ns)
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    a[e][0] += x[u][e][0];
                    a[e][1] += x[u][e][1];
                }
    }
#pragma unroll
    for (int e = 0; e < 2; ++e)
        if (in[e]) {
            cd1[idx[e]] = a[e][0];
            cd2[idx[e]] = a[e][1];
        }
}

// One CoC workgroup (blk < tiles * groups * ns), using lds (cc channels of
// coc_channel_bytes).  Writes slice (group * ns + split) of copart
// [groups * ns][3][E*F]: the share of Co5, Co6, Co7 at the tile's positions of
// one channel range and one image range.  Each thread sums its taps in the fixed
// order (channel, r, s).  The window is staged eight elements a thread at a
// time (sixteen loads in flight), with the Cw1, Cw2 taps of the channels beside it.
template <int NT>
__device__ inline void coc_block(const Geom &g, const CocTile &ct, const CdSrc &src, const double *__restrict__ cw1,
                                 const double *__restrict__ cw2, double *__restrict__ copart, int blk,
                                 double *lds) {
    const int tile = blk % ct.tiles, gs = blk / ct.tiles;
    const int grp = gs / src.ns, split = gs - grp * src.ns;
    const double *p1 = src.p1 + (long long)split * src.stride, *p2 = src.p2 + (long long)split * src.stride;
    const int bx = tile / ct.tiles_x, by = tile - (tile / ct.tiles_x) * ct.tiles_x;
    const int x0 = bx * ct.ty, y0 = by * ct.tx;
    const int rows = ct.ty < g.E - x0 ? ct.ty : g.E - x0;
    const int cols = ct.tx < g.F - y0 ? ct.tx : g.F - y0;
    const int PH = (rows - 1) * g.U + g.R, PW = (cols - 1) * g.U + g.S;
    const int plane = PH * PW;
    const int c0 = (int)((long long)grp * g.C / ct.groups), c1 = (int)((long long)(grp + 1) * g.C / ct.groups);
    const int t = threadIdx.x;
    const int tyi = t / ct.tx, txi = t - (t / ct.tx) * ct.tx;
    const bool mine = tyi < rows && txi < cols;
    const int ih0 = g.U * x0 - g.P, iw0 = g.U * y0 - g.P;
    const int RS = g.R * g.S;
    double *s1 = lds, *s2 = lds + (size_t)ct.cc * plane;
    double *w1s = s2 + (size_t)ct.cc * plane, *w2s = w1s + (size_t)ct.cc * RS;
    // staging walk: element e = (c * PH + i) * PW + j of the window; a thread starts at e = t and
    // steps by NT, carrying (c, i, j) along instead of dividing
    const int sj = NT % PW, srow = NT / PW, si = srow % PH, sc = srow / PH;
    const int tj0 = t % PW, trow0 = t / PW, ti0 = trow0 % PH, tc0 = trow0 / PH;
    double c5 = 0.0, c6 = 0.0, c7 = 0.0;
    for (int cb = c0; cb < c1; cb += ct.cc) {
        const int nc = ct.cc < c1 - cb ? ct.cc : c1 - cb;
        const int total = nc * plane;
        __syncthreads();   // the previous group's window is no longer read
        int c = tc0, i = ti0, j = tj0;
        for (int e0 = 0; e0 < total; e0 += 8 * NT) {
            double a1[8], a2[8];
            bool ok[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int ih = ih0 + i, iw = iw0 + j;
                ok[u] = c < nc && (unsigned)ih < (unsigned)g.H && (unsigned)iw < (unsigned)g.W;
                const long long idx = ok[u] ? ((long long)(cb + c) * g.H + ih) * g.W + iw : 0;
                a1[u] = p1[idx];
                a2[u] = p2[idx];
                j += sj;
                i += si;
                c += sc;
                if (j >= PW) { j -= PW; ++i; }
                if (i >= PH) { i -= PH; ++c; }
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int e = e0 + u * NT + t;
                if (e < total) {
                    s1[e] = ok[u] ? a1[u] : 0.0;
                    s2[e] = ok[u] ? a2[u] : 0.0;
                }
            }
        }
        for (int e = t; e < nc * RS; e += NT) {
            w1s[e] = cw1[(long long)cb * RS + e];
            w2s[e] = cw2[(long long)cb * RS + e];
        }
        __syncthreads();
        if (mine) {
            const int base = tyi * g.U * PW + txi * g.U;
            for (int cc = 0; cc < nc; ++cc) {
                const double *r1 = s1 + cc * plane + base, *r2 = s2 + cc * plane + base;
                const double *v1 = w1s + cc * RS, *v2 = w2s + cc * RS;
                for (int r = 0; r < g.R; ++r) {
#pragma unroll 4
                    for (int s = 0; s < g.S; ++s) {
                        const double d1 = r1[r * PW + s], d2 = r2[r * PW + s];
                        const double w1 = v1[r * g.S + s], w2 = v2[r * g.S + s];
                        c5 = fma(d1, w1, c5);
                        c6 = fma(d1, w2, c6);
                        c7 = fma(d2, w1, c7);
                    }
                }
            }
        }
    }
    if (mine) {
        const int p = (x0 + tyi) * g.F + y0 + txi;
        double *o = copart + (size_t)gs * 3 * g.EF + p;
        o[0] = c5;
        o[g.EF] = c6;
        o[2 * (size_t)g.EF] = c7;
    }
}

}  // namespace ftcnn
