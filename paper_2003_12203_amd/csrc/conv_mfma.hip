// The layer's convolution, eq. (1), as an implicit GEMM on the CDNA4 matrix cores.
//
//   C[m][p] = sum_k A[m][k] * B[k][p]
//   A = W viewed as [M][K] (already row-major, K = C*R*S ordered (c, r, s)),
//   B = im2col(D): B[k][p] = D[n][c][U*x + r - P][U*y + s - P] (zero outside),
//   p = (n, x, y) runs over the N*E*F output pixels, and C[m][p] is O[n][m][x][y].
//
// A workgroup computes a TM x TP tile of C with WM x WP waves; every wave owns
// FM x FP blocks of 32x32 accumulators.  The K loop walks chunks of TK: the next
// chunk is fetched from global memory into registers (A with 16-byte loads, B as
// a per-pixel im2col gather whose addresses are coalesced along p) while the
// matrix cores work on the current chunk from LDS; LDS is double buffered, so one
// barrier per chunk suffices.  Lanes of a 32x32 MFMA own one output pixel each,
// so the epilogue writes whole 128-byte runs of O.  Workgroup ids are remapped so
// that the M tiles of one pixel tile land on the same XCD (its L2 then serves the
// repeated im2col reads of D).
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

// Map the hardware workgroup id onto a logical tile so that each XCD (ids are
// dealt round-robin over 8 XCDs) receives a contiguous run of logical tiles.
__device__ inline int xcd_tile(int bid, int total) {
    const int q = total / 8, rem = total % 8, x = bid % 8;
    return x * q + (x < rem ? x : rem) + bid / 8;
}

// Element-type traits: fp32 uses v_mfma_f32_32x32x2_f32 (2 k per instruction),
// bf16 uses v_mfma_f32_32x32x16_bf16 (16 k per instruction).
struct F32T {
    using T = float;
    static constexpr int TK = 16;      // k per chunk
    static constexpr int LDK = 20;     // LDS row stride in elements (16 + 4 pad)
    static constexpr int VEC = 4;      // elements per 16-byte A load
};
struct BF16T {
    using T = uint16_t;
    static constexpr int TK = 32;
    static constexpr int LDK = 40;     // 32 + 8 pad (80-byte rows)
    static constexpr int VEC = 8;
};

template <typename Tr, int WM, int WP, int FM, int FP>
struct Cfg {
    using T = typename Tr::T;
    static constexpr int NT = 64 * WM * WP;
    static constexpr int TM = WM * FM * 32;
    static constexpr int TP = WP * FP * 32;
    static constexpr int TK = Tr::TK;
    static constexpr int LDK = Tr::LDK;
    static constexpr int VEC = Tr::VEC;
    static constexpr int A_SLOTS = TM * TK / VEC;                    // 16-byte slots of the A tile
    static constexpr int A_PER = (A_SLOTS + NT - 1) / NT;
    static constexpr int KG = NT / TP;                               // threads per pixel along k
    static constexpr int KR = TK / KG;                               // k per thread in the gather
    static_assert(NT % TP == 0 && TK % KG == 0 && KR % VEC == 0, "tile shape");
    static constexpr size_t LDS_BYTES = 2ull * (TM + TP) * LDK * sizeof(T);
    static_assert(LDS_BYTES <= 65536, "tile exceeds the default LDS allocation");
};

// 16 bytes of elements, moved between global memory, registers and LDS as one unit.
template <typename T, int VEC> union Pack {
    uint4 q;
    T e[VEC];
};

template <typename C>
__device__ inline void load_a(const typename C::T *__restrict__ Wt, const Geom &g, int m0, int kbase,
                              int tid, bool kvec, Pack<typename C::T, C::VEC> (&ra)[C::A_PER]) {
    using T = typename C::T;
#pragma unroll
    for (int i = 0; i < C::A_PER; ++i) {
        const int slot = tid + i * C::NT;
        const int row = slot / (C::TK / C::VEC);
        const int kq = slot % (C::TK / C::VEC);
        const int m = m0 + row;
        const int k = kbase + kq * C::VEC;
        if (slot < C::A_SLOTS && m < g.M && k < g.K) {
            const T *src = Wt + (long long)m * g.K + k;
            if (kvec && k + C::VEC <= g.K) {
                ra[i].q = *reinterpret_cast<const uint4 *>(src);
            } else {
#pragma unroll
                for (int v = 0; v < C::VEC; ++v) ra[i].e[v] = (k + v < g.K) ? src[v] : T(0);
            }
        } else {
            ra[i].q = make_uint4(0u, 0u, 0u, 0u);
        }
    }
}

template <typename C>
__device__ inline void load_b(const typename C::T *__restrict__ Dt, const Geom &g, int kstart,
                              bool pvalid, long long dbase, int ih0, int iw0,
                              Pack<typename C::T, C::VEC> (&rb)[C::KR / C::VEC]) {
    using T = typename C::T;
    const int RS = g.R * g.S;
    int c = kstart / RS;
    int rem = kstart - c * RS;
    int r = rem / g.S;
    int s = rem - r * g.S;
    const long long HW = (long long)g.H * g.W;
#pragma unroll
    for (int j = 0; j < C::KR; ++j) {
        const int ih = ih0 + r, iw = iw0 + s;
        const bool ok = pvalid && (kstart + j < g.K) && ih >= 0 && ih < g.H && iw >= 0 && iw < g.W;
        rb[j / C::VEC].e[j % C::VEC] = ok ? Dt[dbase + c * HW + (long long)ih * g.W + iw] : T(0);
        if (++s == g.S) {
            s = 0;
            if (++r == g.R) { r = 0; ++c; }
        }
    }
}

template <typename C>
__device__ inline void store_lds(typename C::T *As, typename C::T *Bs, int tid,
                                 const Pack<typename C::T, C::VEC> (&ra)[C::A_PER],
                                 const Pack<typename C::T, C::VEC> (&rb)[C::KR / C::VEC], int bp, int bkg) {
#pragma unroll
    for (int i = 0; i < C::A_PER; ++i) {
        const int slot = tid + i * C::NT;
        if (slot < C::A_SLOTS) {
            const int row = slot / (C::TK / C::VEC);
            const int kq = slot % (C::TK / C::VEC);
            *reinterpret_cast<uint4 *>(&As[row * C::LDK + kq * C::VEC]) = ra[i].q;
        }
    }
#pragma unroll
    for (int j = 0; j < C::KR; j += C::VEC)
        *reinterpret_cast<uint4 *>(&Bs[bp * C::LDK + bkg * C::KR + j]) = rb[j / C::VEC].q;
}

// One chunk of MFMAs from LDS.  Within a chunk, lanes 0-31 take the first half
// of the k range and lanes 32-63 the second half; A and B use the same
// assignment, so every k of the chunk is summed exactly once.
template <int FM, int FP>
__device__ inline void mma_f32(const float *As, const float *Bs, int lane, int arow0, int brow0,
                               floatx16 (&acc)[FM][FP]) {
    const int l32 = lane & 31, h = lane >> 5;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        floatx4 a[FM], b[FP];
#pragma unroll
        for (int i = 0; i < FM; ++i)
            a[i] = *reinterpret_cast<const floatx4 *>(&As[(arow0 + i * 32 + l32) * F32T::LDK + h * 8 + q * 4]);
#pragma unroll
        for (int j = 0; j < FP; ++j)
            b[j] = *reinterpret_cast<const floatx4 *>(&Bs[(brow0 + j * 32 + l32) * F32T::LDK + h * 8 + q * 4]);
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FP; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][t], b[j][t], acc[i][j], 0, 0, 0);
    }
}

template <int FM, int FP>
__device__ inline void mma_bf16(const uint16_t *As, const uint16_t *Bs, int lane, int arow0, int brow0,
                                floatx16 (&acc)[FM][FP]) {
    const int l32 = lane & 31, h = lane >> 5;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        bf16x8 a[FM], b[FP];
#pragma unroll
        for (int i = 0; i < FM; ++i)
            a[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8 *>(
                                                  &As[(arow0 + i * 32 + l32) * BF16T::LDK + h * 16 + q * 8]));
#pragma unroll
        for (int j = 0; j < FP; ++j)
            b[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8 *>(
                                                  &Bs[(brow0 + j * 32 + l32) * BF16T::LDK + h * 16 + q * 8]));
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FP; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
}

template <typename Tr, int WM, int WP, int FM, int FP>
__global__ __launch_bounds__(64 * WM * WP) void conv_kernel(const typename Tr::T *__restrict__ D,
                                                            const typename Tr::T *__restrict__ Wt,
                                                            typename Tr::T *__restrict__ O, Geom g,
                                                            int tiles_m, int tiles_total, int kvec) {
    using C = Cfg<Tr, WM, WP, FM, FP>;
    using T = typename C::T;
    extern __shared__ __align__(16) unsigned char smem[];
    T *As0 = reinterpret_cast<T *>(smem);
    T *Bs0 = As0 + 2 * C::TM * C::LDK;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wp = wave / WM;
    const int tile = xcd_tile(blockIdx.x, tiles_total);
    const int m0 = (tile % tiles_m) * C::TM;
    const long long p0 = (long long)(tile / tiles_m) * C::TP;

    // this thread's im2col pixel (fixed over the K loop)
    const int bp = tid % C::TP, bkg = tid / C::TP;
    const long long pg = p0 + bp;
    const bool pvalid = pg < g.P_total;
    long long dbase = 0;
    int ih0 = 0, iw0 = 0;
    if (pvalid) {
        const long long n = pg / g.EF;
        const int pix = (int)(pg - n * g.EF);
        const int x = pix / g.F, y = pix - (pix / g.F) * g.F;
        dbase = n * g.CHW;
        ih0 = g.U * x - g.P;
        iw0 = g.U * y - g.P;
    }

    floatx16 acc[FM][FP];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FP; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

    Pack<T, C::VEC> ra[C::A_PER];
    Pack<T, C::VEC> rb[C::KR / C::VEC];
    const int nchunks = (g.K + C::TK - 1) / C::TK;
    load_a<C>(Wt, g, m0, 0, tid, kvec != 0, ra);
    load_b<C>(D, g, bkg * C::KR, pvalid, dbase, ih0, iw0, rb);
    store_lds<C>(As0, Bs0, tid, ra, rb, bp, bkg);
    __syncthreads();

    const int arow0 = wm * FM * 32, brow0 = wp * FP * 32;
    for (int kc = 0; kc < nchunks; ++kc) {
        const int buf = kc & 1;
        const bool more = kc + 1 < nchunks;
        if (more) {
            const int kb = (kc + 1) * C::TK;
            load_a<C>(Wt, g, m0, kb, tid, kvec != 0, ra);
            load_b<C>(D, g, kb + bkg * C::KR, pvalid, dbase, ih0, iw0, rb);
        }
        const T *As = As0 + buf * C::TM * C::LDK;
        const T *Bs = Bs0 + buf * C::TP * C::LDK;
        if constexpr (sizeof(T) == 4)
            mma_f32<FM, FP>(reinterpret_cast<const float *>(As), reinterpret_cast<const float *>(Bs),
                            lane, arow0, brow0, acc);
        else
            mma_bf16<FM, FP>(reinterpret_cast<const uint16_t *>(As), reinterpret_cast<const uint16_t *>(Bs),
                             lane, arow0, brow0, acc);
        if (more) store_lds<C>(As0 + (buf ^ 1) * C::TM * C::LDK, Bs0 + (buf ^ 1) * C::TP * C::LDK, tid, ra,
                               rb, bp, bkg);
        __syncthreads();
    }

    // epilogue: lane owns pixel (lane & 31) of each 32-wide block
    const int l32 = lane & 31, h = lane >> 5;
#pragma unroll
    for (int j = 0; j < FP; ++j) {
        const long long pgo = p0 + brow0 + j * 32 + l32;
        if (pgo >= g.P_total) continue;
        const long long n = pgo / g.EF;
        const long long ob = n * g.M * (long long)g.EF + (pgo - n * g.EF);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int m = m0 + arow0 + i * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
                if (m < g.M) Elem<T>::store(O, ob + (long long)m * g.EF, acc[i][j][e]);
            }
    }
}

template <typename Tr, int WM, int WP, int FM, int FP>
hipError_t run_conv(const Geom &g, const void *D, const void *W, void *O, hipStream_t st) {
    using C = Cfg<Tr, WM, WP, FM, FP>;
    using T = typename C::T;
    const int tiles_m = (g.M + C::TM - 1) / C::TM;
    const long long tiles_p = (g.P_total + C::TP - 1) / C::TP;
    const long long total = tiles_p * tiles_m;
    if (total > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    const int kvec = (g.K % C::VEC == 0 && reinterpret_cast<uintptr_t>(W) % 16 == 0) ? 1 : 0;
    conv_kernel<Tr, WM, WP, FM, FP><<<(unsigned)total, C::NT, C::LDS_BYTES, st>>>(static_cast<const T *>(D), static_cast<const T *>(W),
                                                       static_cast<T *>(O), g, tiles_m, (int)total, kvec);
    return hipGetLastError();
}

}  // namespace

// Tile choice per layer: the filter tile follows M (small-M layers would waste
// most of a 128-row tile); pixel tiles are as wide as the register budget allows.
hipError_t launch_conv(const Plan &pl, const void *D, const void *W, void *O, hipStream_t st) {
    const Geom &g = pl.g;
    if (g.dtype == FTCNN_F32) {
        if (g.M <= 32) return run_conv<F32T, 1, 4, 1, 2>(g, D, W, O, st);
        if (g.M <= 64) return run_conv<F32T, 1, 4, 2, 2>(g, D, W, O, st);
        if (g.M <= 96) return run_conv<F32T, 1, 4, 3, 2>(g, D, W, O, st);
        return run_conv<F32T, 2, 2, 2, 2>(g, D, W, O, st);
    }
    if (g.M <= 32) return run_conv<BF16T, 1, 4, 1, 2>(g, D, W, O, st);
    if (g.M <= 64) return run_conv<BF16T, 1, 4, 2, 2>(g, D, W, O, st);
    return run_conv<BF16T, 2, 2, 2, 2>(g, D, W, O, st);
}

}  // namespace ftcnn
