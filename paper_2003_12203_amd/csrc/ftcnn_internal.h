// Internal definitions of the HIP library: layer geometry, launch plan,
// workspace layout and small device helpers.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "ftcnn.h"

namespace ftcnn {

// Layer geometry in the paper's notation (Sec. 2.1, Table 1), with zero padding.
struct Geom {
    int N, C, H, W;       // D [N][C][H][W]
    int M, R, S;          // W [M][C][R][S]
    int U, P;             // stride, padding
    int E, F;             // output extent
    int K;                // C*R*S: one dot product of eq. (1)
    int EF;               // output positions per block
    long long CHW;        // elements of one feature-map block D_n
    long long P_total;    // N*E*F: GEMM columns of the implicit-GEMM convolution
    int dtype, wbase;
    // G groups (Sec. 5.2): W is [M][Cg][R][S] with Cg = C/G, Kg = Cg*R*S per filter; filter m
    // meets channels [group_first_channel(m), + Cg).  K = C*R*S is the dense reduction of the
    // block-diagonal expansion of W that the convolution runs on.  G = 1: Cg = C, Kg = K.
    int G, Cg, Mg, Kg;
};
__host__ __device__ inline int group_first_channel(const Geom &g, int m) { return (m / g.Mg) * g.Cg; }

// Tiling of the Co5..Co7 products computed by extra workgroups of the
// convolution launch (channels-last layers): output tiles of tx columns (of F)
// by ty rows (of E), cc channels staged in LDS per step, the channels split
// into `groups` ranges and, when the input checksums come as ns image-range
// partials, one workgroup per range as well (groups * ns partial slices);
// comb_blocks workgroups combine those partials into Cd1, Cd2.
struct CocTile {
    int tx, ty, cc;
    int tiles_x, tiles;
    int groups;
    int comb_blocks;
    int ns;
};
// LDS one channel of a CoC workgroup takes: its input window of Cd1 and Cd2 for a
// ty x tx tile of output positions, and its R*S taps of Cw1 and Cw2 (float64)
inline size_t coc_channel_bytes(const Geom &g, int ty, int tx) {
    const size_t window = (size_t)((ty - 1) * g.U + g.R) * ((tx - 1) * g.U + g.S);
    return 2 * sizeof(double) * (window + (size_t)g.R * g.S);
}

// Split counts and workspace offsets shared by every call on one layer.
struct Plan {
    Geom g;
    int enc_splits_d, enc_splits_w;   // row splits of the input-checksum reductions
    int ver_splits;                   // row splits of the verification reduction
    int ver_cols_per_block;           // columns handled by one verify block
    int corr_blocks;                  // workgroups of the standalone correction kernel
    int sum_splits;                   // partial-sum slices written by the convolution epilogue
    bool nhwc;                        // the convolution reads channels-last copies of D and W
    int prep_ns;                      // image ranges of the encode fused into the channels-last copy
    bool co_in_conv;                  // Co5..Co7 partials computed by workgroups of the convolution launch
    CocTile co;                       // their tiling (co_in_conv)
    size_t off_flags, off_enc, off_ver, off_sums, off_corr, off_dt, off_wt, off_encp, off_copart, off_zero,
        off_wchk, off_wfull, bytes;
    int sk_smax;                      // stream-K workgroups the scratch has room for (0: none)
    size_t off_skpart, off_skcnt;     // their partial accumulators, and one arrival count per tile
    long long sk_counters;
    size_t corr_stride;               // doubles of the decision stage's per-position arrays
};

constexpr int kThreads = 256;

// The correction's wide stage (the Sec. 4.3 chain): flagged positions are handed over as Pending
// records (room for every position of the layer).  The stage's workgroups spread the row and
// column checksums Co1..Co4 and the per-filter and per-image summations of the first kMaxPending
// of them (and, for possibly suspect checksums, Co5..Co7 re-encoded from D and W over
// kFreshRanges ranges of taps) over the whole launch, and the last of them takes those positions'
// decisions; any further position is taken whole by one workgroup.
constexpr int kMaxPending = 64;
constexpr int kFreshRanges = 256;
constexpr int kRowSums = 6;   // per filter: Co1, Co3 (without bias), So1, So3, sum o^2, sum ((n + wbase) o)^2
constexpr int kColSums = 5;   // per image: Co2, Co4 (without bias), So2, So4, sum o^2
struct Pending {
    int p, mode;     // position; mode 1: a weighted checksum may agree (re-encode Co5..Co7)
    double co[3];    // Co5..Co7 at p as the summations see them (bias shares added)
};
// Workgroups of the wide stage: one per work unit of a position (four filters, or one image), at
// least kFreshRanges, at most 1024.
inline int wide_grid(const Geom &g) {
    const long long need = ((long long)g.M + 3) / 4 + g.N;
    return (int)(need < kFreshRanges ? kFreshRanges : (need > 1024 ? 1024 : need));
}
// Largest window of Cd1 and Cd2 at one position (2 K doubles and K flags) that the wide stage
// stages in shared memory, so that two of its workgroups still share a compute unit.
constexpr size_t kWindowBytes = 79 << 10;
// The wide stage's completion count: kDoneGroups counters (workgroup b counts in b % kDoneGroups),
// the last arrival of each then in one more, so that no single counter takes every arrival.
// Counters sit kDoneStride ints (4 KiB) apart, the top one first.
constexpr int kDoneGroups = 32;
constexpr int kDoneStride = 1024;
// Byte offsets inside the correction scratch (the workspace at Plan::off_corr).
struct CorrLayout {
    size_t done, pend, rows, cols, fresh, chain, bytes;
};
inline CorrLayout corr_layout(const Geom &g, size_t chain_doubles) {
    auto a256 = [](size_t b) { return (b + 255) & ~size_t(255); };
    const size_t blocks = (size_t)wide_grid(g);
    const size_t slabs = (size_t)kMaxPending + blocks;   // the shared batch, then one per workgroup
    CorrLayout L{};
    size_t off = 0;
    L.done = off;  off += a256(sizeof(int) * kDoneStride * (kDoneGroups + 1));
    L.pend = off;  off += a256(sizeof(Pending) * (size_t)g.EF);
    L.rows = off;  off += a256(sizeof(double) * kRowSums * (size_t)g.M * slabs);
    L.cols = off;  off += a256(sizeof(double) * kColSums * (size_t)g.N * slabs);
    L.fresh = off; off += a256(sizeof(double) * 3 * (size_t)kFreshRanges * kMaxPending);
    L.chain = off; off += a256(sizeof(double) * chain_doubles * blocks);
    L.bytes = off;
    return L;
}
// Bytes of the static device scratch that ftcnn_protected_conv_noalloc uses in place of a workspace.
constexpr size_t kStaticScratchBytes = size_t(128) << 20;
constexpr int kPrepBatch = 8;   // images per load round of the channels-last copy
constexpr int kMaxFaults = 64;
constexpr double kUAcc = 5.9604644775390625e-08;   // 2^-24, fp32 accumulation unit roundoff
constexpr double kUOutBf16 = 3.90625e-03;          // 2^-8, bf16 storage unit roundoff

// ---- element access -------------------------------------------------------

__host__ __device__ inline float bf16_bits_to_f32(uint16_t b) {
    return __builtin_bit_cast(float, (uint32_t)b << 16);
}

__host__ __device__ inline uint16_t f32_to_bf16_bits(float f) {
    uint32_t u = __builtin_bit_cast(uint32_t, f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)0x7FC0;
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// The same rounding (nearest, ties to even) in one gfx950 instruction (v_cvt_pk_bf16_f32),
// for the output stores of the kernels; a NaN becomes a quiet NaN.
__device__ inline uint16_t f32_to_bf16_rne(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

template <typename T> struct Elem;
template <> struct Elem<float> {
    __device__ static float load(const float *p, long long i) { return p[i]; }
    __device__ static void store(float *p, long long i, float v) { p[i] = v; }
};
template <> struct Elem<uint16_t> {
    __device__ static float load(const uint16_t *p, long long i) { return bf16_bits_to_f32(p[i]); }
    __device__ static void store(uint16_t *p, long long i, float v) { p[i] = f32_to_bf16_rne(v); }
};

// ---- faults planted for testing (the paper's source-level injection, Sec. 6.1)

// A fault list passed by value in kernel arguments.
struct FaultList {
    ftcnn_fault f[kMaxFaults];
    int n;
};

// One fault applied to a stored output pattern: kind 0 flips a bit of the
// pattern, kind 1 adds a value, kind 2 stores a value (rounded to the dtype).
__device__ inline float fault_apply(float v, const ftcnn_fault &f) {
    if (f.kind == 0) return __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, v) ^ (1u << f.bit));
    return (float)(f.kind == 1 ? (double)v + f.value : f.value);
}
__device__ inline uint16_t fault_apply(uint16_t b, const ftcnn_fault &f) {
    if (f.kind == 0) return (uint16_t)(b ^ (1u << f.bit));
    return f32_to_bf16_bits((float)(f.kind == 1 ? (double)bf16_bits_to_f32(b) + f.value : f.value));
}

// A fresh report: nothing detected, cap_fixes recorded.
__device__ inline void reset_report(ftcnn_report *rep, int cap) {
    rep->detected = 0;
    rep->n_flagged = 0;
    rep->status = FTCNN_STATUS_CLEAN;
    for (int i = 0; i < 7; ++i) rep->resolved_by[i] = 0;
    rep->n_fixes = 0;
    rep->cap_fixes = cap;
    rep->reserved[0] = rep->reserved[1] = 0;
}

// ---- tolerance (the shared reading of "not equal") ------------------------

__host__ __device__ inline double tol_scale(const Geom &g, double kappa) {
    const double u_out = g.dtype == FTCNN_BF16 ? kUOutBf16 : 0.0;
    return kappa * (kUAcc * sqrt((double)g.Kg) + u_out);   // Kg: the dot length of one output
}

__device__ inline bool is_bad(double d, double q, double scale) {
    return !isfinite(d) || fabs(d) > scale * q;
}

// ---- instrumentation ------------------------------------------------------

// Events the caller asked to have recorded around the next launch of the
// convolution kernel on this thread (ftcnn_set_kernel_events); cleared once used.
struct KernelEvents {
    hipEvent_t before, after;
};
KernelEvents &kernel_events();

// ---- launches (one per kernel family; defined in the .hip files) ----------

hipError_t launch_encode(const Plan &pl, int which, const void *X, double *c1, double *c2,
                         void *ws, hipStream_t st);
// bias: NULL, or fp32 [M] added to every O[n][m] before rounding (Sec. 5.1).
hipError_t launch_conv(const Plan &pl, const void *D, const void *W, void *O, hipStream_t st,
                       const float *bias = nullptr);
// Grouped layers (G > 1, Sec. 5.2): the block-diagonal expansion of W ([M][Cg][R][S]) into the
// dense [M][C][R][S] at pl.off_wfull, zeros outside each filter's channel group; returns W itself
// when G = 1.  Its Cw1, Cw2 are the grouped checksums of Sec. 5.2.
const void *dense_weights(const Plan &pl, const void *W, void *ws, hipStream_t st, hipError_t *err);
// ReLU then k x k / s max pooling between two layers of a network (k = s = 1: ReLU only)
hipError_t launch_relu_pool(ftcnn_dtype dt, const void *X, void *Y, int n, int c, int h, int w, int k, int s,
                            hipStream_t st);
// ... and the next layer's Cd1, Cd2 [c][h'][w'] from the values written
hipError_t launch_relu_pool_encode(ftcnn_dtype dt, const void *X, void *Y, int n, int c, int h, int w, int k, int s,
                                   int wbase, double *cd1, double *cd2, hipStream_t st);
// Re-encode Cw1, Cw2 of W into the workspace (pl.off_wchk) and count the columns whose Cw1
// differs bitwise from cw1 into *mismatches (Sec. 4.1.2).
hipError_t launch_check_weights(const Plan &pl, const void *W, const double *cw1, int32_t *mismatches, void *ws,
                                hipStream_t st);
// c1 = sum_m bias[m], c2 = sum_m (m + wbase) bias[m] (Sec. 5.1), one double each.
hipError_t launch_bias_sums(const Plan &pl, const float *bias, double *c1, double *c2, hipStream_t st);
// The convolution with the CoC-D summations in its epilogue: every tile also
// writes its (So5, So6, So7, sum of squares) partials for the pixels it owns to
// the workspace (pl.sum_splits slices, layout of the verification partials) and
// the report is reset.  With ck->cd1 and cd2 set, Cd1 and Cd2 are encoded in
// the same pass (by the channels-last copy, or by extra workgroups of the
// convolution launch); on pl.co_in_conv layers with ck->cw1 and cw2 set too,
// extra workgroups of the convolution launch also compute the Co5..Co7
// partials (pl.co.groups slices at pl.off_copart), and rep->reserved[1] records
// how many.  faults (at most kMaxFaults, host array) are planted in the stored
// values before they are summed.
hipError_t launch_conv_sums(const Plan &pl, const void *D, const void *W, void *O, const ftcnn_checksums *ck,
                            ftcnn_report *rep, int cap, const ftcnn_fault *faults, int nf, void *ws,
                            hipStream_t st, bool cd_given = false);
// The convolution kernel chosen for this layer (ftcnn_conv_tile): tile rows, pixels, chunk depth,
// main-loop kind, channels-last, grouped channel skip.
void conv_tile_info(const Geom &g, bool nhwc, int out[6]);
// Rows of C per workgroup tile of the convolution chosen for this layer.
int conv_tile_m(const Geom &g, bool nhwc);
// Threads per workgroup and dynamic LDS bytes of the convolution chosen for this layer.
void conv_tile_shape(const Geom &g, bool nhwc, int *threads, size_t *lds_bytes);
// Stream-K scratch of a layer's channels-last convolution: at most smax workgroups, part_bytes of
// partial accumulators, one int counter per tile (all zero when its kernel has no stream-K form).
// Sized for kSkComputeUnits compute units; a device with more runs at most smax workgroups.
constexpr int kSkComputeUnits = 256;
void conv_sk_space(const Geom &g, bool nhwc, int *smax, size_t *part_bytes, long long *counters);
// Stream-K workgroups the plan's channels-last convolution launches on the current device (0: one
// workgroup per tile).
struct Plan;
int conv_stream_k(const Plan &pl);
// Layers whose convolution reads channels-last copies (pl.nhwc): Ch a multiple of 32 (and
// kernels of at most 4096 taps, whose weight rows the copy stages in LDS).
inline bool nhwc_layer(const Geom &g) { return g.C % 32 == 0 && g.R * g.S <= 4096; }
// Positions per tile of the channels-last copy (128 bytes of one channel) and channels per
// tile (64 for bf16 when that still leaves 512 tiles: a stored position is then one 128-byte
// line).
// positions per tile of the channels-last copy: eight 16-byte vectors of a channel row, or seven
// when H*W is not a multiple of the vector (each row segment then starts inside a vector)
inline int prep_tile_positions(const Geom &g) {
    const int vec = g.dtype == FTCNN_F32 ? 4 : 8;
    return ((long long)g.H * g.W) % vec == 0 ? 8 * vec : 7 * vec;
}
inline int prep_tile_channels(const Geom &g) {
    const long long hw_tiles = ((long long)g.H * g.W + prep_tile_positions(g) - 1) / prep_tile_positions(g);
    return g.dtype == FTCNN_BF16 && g.C % 64 == 0 && (g.C / 64) * hw_tiles >= 512 ? 64 : 32;
}
// Dt = D in [n][h][w][c] order and Wt = W in [m][r][s][c] order into the workspace
// (pl.off_dt, pl.off_wt); with cd1 and cd2 set, the copy of D also encodes them
// (directly when pl.prep_ns == 1, else as image-split partials at pl.off_encp
// that the convolution launch combines into cd1 and cd2).
hipError_t launch_prep(const Plan &pl, const void *D, const void *W, double *cd1, double *cd2, void *ws,
                       hipStream_t st);
// The convolution alone through the path ftcnn_conv_fwd_sums takes (channels-last
// copies for pl.nhwc layers): O bitwise equal to that of launch_conv_sums.
hipError_t launch_conv_ws(const Plan &pl, const void *D, const void *W, void *O, void *ws, hipStream_t st,
                          const float *bias = nullptr);
hipError_t launch_checksum_conv(const Plan &pl, uint32_t which, const void *D, const void *W,
                                const ftcnn_checksums &ck, hipStream_t st);
hipError_t launch_verify(const Plan &pl, const void *O, const ftcnn_checksums &ck,
                         const ftcnn_policy &pol, ftcnn_report *rep, int cap, void *ws,
                         hipStream_t st);
hipError_t launch_correct(const Plan &pl, const void *D, const void *W, void *O,
                          const ftcnn_checksums &ck, const ftcnn_policy &pol, ftcnn_report *rep,
                          void *ws, hipStream_t st);
hipError_t launch_verify_partial(const Plan &pl, const void *O, ftcnn_report *rep, int cap, void *ws,
                                 hipStream_t st);
hipError_t launch_verify_correct(const Plan &pl, const void *D, const void *W, void *O,
                                 const ftcnn_checksums &ck, const ftcnn_policy &pol, ftcnn_report *rep,
                                 int cap, void *ws, hipStream_t st);
// Final detection stage and correction over the partials the convolution epilogue wrote;
// with coc, Co5..Co7 are computed in the same launch from Cd1, Cd2, Cw1, Cw2.
hipError_t launch_verify_correct_sums(const Plan &pl, const void *D, const void *W, void *O,
                                      const ftcnn_checksums &ck, const ftcnn_policy &pol, ftcnn_report *rep,
                                      bool coc, void *ws, hipStream_t st);

// Threads that share one position in the final verification stage (1, 4, 16,
// 64 or a whole workgroup; the float64 split partials of that position, and the
// K taps of its Co5..Co7 when those are computed there too, are spread over
// them): at most about 24 partial rows or taps per thread, and enough threads
// in the grid (32K) to keep every CU's loads in flight.
inline int final_tpp(int splits, int taps, long long positions) {
    const long long w = (long long)splits + taps;
    int t = 1;
    while (t < kThreads && w > 24LL * t) t *= 4;
    while (t < kThreads && (long long)t * positions < 32768) t *= 4;
    return t > kThreads ? kThreads : t;
}
hipError_t launch_inject(const Plan &pl, void *O, const ftcnn_fault *f, int nf, hipStream_t st);
// Device address of the static scratch (kStaticScratchBytes, 256-byte aligned) on `device`; looked up
// once per device with that device current, then cached.
hipError_t static_scratch(int device, void **ptr);

}  // namespace ftcnn
