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
};

// Split counts and workspace offsets shared by every call on one layer.
struct Plan {
    Geom g;
    int enc_splits_d, enc_splits_w;   // row splits of the input-checksum reductions
    int ver_splits;                   // row splits of the verification reduction
    int ver_cols_per_block;           // columns handled by one verify block
    int corr_blocks;                  // workgroups of the correction kernel
    int corr_slots;                   // per-workgroup scratch slices (correction or fused verification)
    size_t off_flags, off_enc, off_ver, off_corr, bytes;
    size_t corr_stride;               // doubles of scratch per correction workgroup
};

constexpr int kThreads = 256;
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

template <typename T> struct Elem;
template <> struct Elem<float> {
    __device__ static float load(const float *p, long long i) { return p[i]; }
    __device__ static void store(float *p, long long i, float v) { p[i] = v; }
};
template <> struct Elem<uint16_t> {
    __device__ static float load(const uint16_t *p, long long i) { return bf16_bits_to_f32(p[i]); }
    __device__ static void store(uint16_t *p, long long i, float v) { p[i] = f32_to_bf16_bits(v); }
};

// ---- tolerance (the shared reading of "not equal") ------------------------

__host__ __device__ inline double tol_scale(const Geom &g, double kappa) {
    const double u_out = g.dtype == FTCNN_BF16 ? kUOutBf16 : 0.0;
    return kappa * (kUAcc * sqrt((double)g.K) + u_out);
}

__device__ inline bool is_bad(double d, double q, double scale) {
    return !isfinite(d) || fabs(d) > scale * q;
}

// ---- launches (one per kernel family; defined in the .hip files) ----------

hipError_t launch_encode(const Plan &pl, int which, const void *X, double *c1, double *c2,
                         void *ws, hipStream_t st);
hipError_t launch_conv(const Plan &pl, const void *D, const void *W, void *O, hipStream_t st);
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

// Threads that share one position in the final verification stage (a power of
// two; the float64 split partials of that position are spread over them).
inline int final_tpp(int splits) { return splits <= 1 ? 1 : splits <= 4 ? 4 : splits <= 16 ? 16 : 64; }
hipError_t launch_inject(const Plan &pl, void *O, const ftcnn_fault *f, int nf, hipStream_t st);

}  // namespace ftcnn
