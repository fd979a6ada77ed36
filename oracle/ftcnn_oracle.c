/*
 * CPU oracle for checksum-protected convolution (FT-CNN, Zhao et al.,
 * arXiv 2003.12203).  TEST INFRASTRUCTURE ONLY: this file is built into
 * oracle/liboracle.so and is loaded by the tests, by the smoke check and by
 * the benchmark's CPU-baseline leg, never by the product path.  It shares no
 * code, header or constant with the HIP library.
 *
 * Plain, slow, obviously correct loops in float64.  Inputs arrive as float64
 * arrays (fp32 and bf16 values widen to float64 exactly).  OpenMP splits the
 * outermost (image, filter) loop; every output element is still produced by
 * one thread in the fixed (channel, row, column) order of eq. (1).
 */
#include <stdint.h>
#include <stddef.h>

/* Output extent of one spatial axis.  Eq. (1) gives E = (H - R + U) / U with
 * no padding; with zero padding P on both sides this is
 * floor((H + 2P - R) / U) + 1 (a zero border keeps the operation linear). */
int or_out_extent(int h, int r, int u, int p)
{
    int span = h + 2 * p - r;
    if (span < 0 || u <= 0) return 0;
    return span / u + 1;
}

/* Eq. (1) without bias, with zero padding:
 *   O[n][m][x][y] = sum_k sum_i sum_j D[n][k][U*x+i-P][U*y+j-P] * W[m][k][i][j]
 * D is [N][C][H][Wd], W is [M][C][R][S], O is [N][M][E][F], all float64.
 * The same routine evaluates the paper's block operator (x) on checksum blocks
 * (Sec. 3.2: every output checksum is a convolution of checksum blocks), by
 * passing N = 1 and/or M = 1. */
void or_conv(const double *D, const double *W, int N, int C, int H, int Wd,
             int M, int R, int S, int U, int P, double *O)
{
    const int E = or_out_extent(H, R, U, P);
    const int F = or_out_extent(Wd, S, U, P);
    long nm;
#pragma omp parallel for schedule(dynamic, 1)
    for (nm = 0; nm < (long)N * M; ++nm) {
        const int n = (int)(nm / M), m = (int)(nm % M);
        const double *Dn = D + (size_t)n * C * H * Wd;
        const double *Wm = W + (size_t)m * C * R * S;
        double *Onm = O + ((size_t)n * M + m) * E * F;
        for (int x = 0; x < E; ++x)
            for (int y = 0; y < F; ++y) {
                double acc = 0.0;
                for (int k = 0; k < C; ++k)
                    for (int i = 0; i < R; ++i) {
                        const int ih = U * x + i - P;
                        if (ih < 0 || ih >= H) continue;
                        for (int j = 0; j < S; ++j) {
                            const int iw = U * y + j - P;
                            if (iw < 0 || iw >= Wd) continue;
                            acc += Dn[((size_t)k * H + ih) * Wd + iw] *
                                   Wm[((size_t)k * R + i) * S + j];
                        }
                    }
                Onm[(size_t)x * F + y] = acc;
            }
    }
}

/* Eq. (1) evaluated at a list of output coordinates pts[q] = (n, m, x, y).
 * Used to check full-size layers element by element. */
void or_conv_points(const double *D, const double *W, int N, int C, int H, int Wd,
                    int M, int R, int S, int U, int P,
                    const int32_t *pts, long npts, double *out)
{
    (void)N; (void)M;
    long q;
#pragma omp parallel for schedule(static)
    for (q = 0; q < npts; ++q) {
        const int n = pts[4 * q + 0], m = pts[4 * q + 1];
        const int x = pts[4 * q + 2], y = pts[4 * q + 3];
        const double *Dn = D + (size_t)n * C * H * Wd;
        const double *Wm = W + (size_t)m * C * R * S;
        double acc = 0.0;
        for (int k = 0; k < C; ++k)
            for (int i = 0; i < R; ++i) {
                const int ih = U * x + i - P;
                if (ih < 0 || ih >= H) continue;
                for (int j = 0; j < S; ++j) {
                    const int iw = U * y + j - P;
                    if (iw < 0 || iw >= Wd) continue;
                    acc += Dn[((size_t)k * H + ih) * Wd + iw] * Wm[((size_t)k * R + i) * S + j];
                }
            }
        out[q] = acc;
    }
}

/* Sec. 3.2, input checksums: for a stack of `rows` blocks X_0..X_{rows-1},
 * each of `cols` elements,
 *   C1 = sum_r X_r          C2 = sum_r (r + base) * X_r
 * The paper's definition uses base 0 (Cd2 = sum_n n*D_n, Cw2 = sum_m m*W_m). */
void or_block_sums(const double *X, long rows, long cols, double base,
                   double *C1, double *C2)
{
    long c;
#pragma omp parallel for schedule(static)
    for (c = 0; c < cols; ++c) {
        double s1 = 0.0, s2 = 0.0;
        for (long r = 0; r < rows; ++r) {
            const double v = X[(size_t)r * cols + c];
            s1 += v;
            s2 += ((double)r + base) * v;
        }
        C1[c] = s1;
        C2[c] = s2;
    }
}

/* Number of OpenMP threads the loops above use (1 when built without OpenMP). */
int or_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
