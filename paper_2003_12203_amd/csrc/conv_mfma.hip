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
#include <type_traits>

#include "ftcnn_internal.h"
#include "encode_block.h"
#include "coc_tile.h"

namespace ftcnn {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

// A 16-byte unit, or zeros: the selects work on whole 32-bit words.
__device__ inline uint4 keep_or_zero(bool ok, uint4 v) {
    return make_uint4(ok ? v.x : 0u, ok ? v.y : 0u, ok ? v.z : 0u, ok ? v.w : 0u);
}

// Map the hardware workgroup id onto a logical tile so that each XCD (ids are
// dealt round-robin over 8 XCDs) receives a contiguous run of logical tiles.
__device__ inline int xcd_tile(int bid, int total) {
    const int q = total / 8, rem = total % 8, x = bid % 8;
    return x * q + (x < rem ? x : rem) + bid / 8;
}

// Element-type traits: fp32 uses v_mfma_f32_32x32x2_f32 (2 k per instruction),
// bf16 uses v_mfma_f32_32x32x16_bf16 (16 k per instruction).  TK_ is the k
// extent of one LDS chunk; rows are padded by 16 bytes against bank conflicts.
template <int TK_> struct F32T {
    using T = float;
    static constexpr int TK = TK_;
    static constexpr int LDK = TK_ + 4;
    static constexpr int VEC = 4;      // elements per 16-byte load
};
template <int TK_> struct BF16T {
    using T = uint16_t;
    static constexpr int TK = TK_;
    static constexpr int LDK = TK_ + 8;
    static constexpr int VEC = 8;
};

// DSTAGES > 0: the direct-to-LDS loop with that many stages of (TM + TP) rows of 128 bytes.
template <typename Tr, int WM, int WP, int FM, int FP, bool KVEC_ = true, int DSTAGES = 0>
struct Cfg {
    using T = typename Tr::T;
    static constexpr bool KVEC = KVEC_;   // W rows 16-byte aligned: whole-slot weight loads
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
    static_assert(KR <= 64 && A_PER * VEC <= 64, "gather masks are at most 64-bit");
    // one bit per gathered element of a thread
    using Mask = typename std::conditional<(KR > 32 || A_PER * VEC > 32), uint64_t, uint32_t>::type;
    static constexpr size_t LDS_BYTES = DSTAGES > 0 ? (size_t)DSTAGES * (TM + TP) * 128
                                                    : 2ull * (TM + TP) * LDK * sizeof(T);
    static_assert(LDS_BYTES <= 160 * 1024, "tile exceeds the LDS of a CU");
};

// 16 bytes of elements, moved between global memory, registers and LDS as one unit.
template <typename T, int VEC> union Pack {
    uint4 q;
    T e[VEC];
};

// Per-lane constants of the A (weights) gather: which 16-byte slots of the
// TM x TK tile this lane moves, and where each slot's row starts in W.
template <typename C> struct ASlots {
    int base[C::A_PER];   // element offset of the slot's first k in W, -1 if the row is past M
    int kq[C::A_PER];     // k offset of the slot inside the chunk
};

template <typename C>
__device__ inline void a_slots(const Geom &g, int m0, int tid, ASlots<C> &as) {
#pragma unroll
    for (int i = 0; i < C::A_PER; ++i) {
        const int slot = tid + i * C::NT;
        const int row = slot / (C::TK / C::VEC);
        const int m = m0 + row;
        as.kq[i] = (slot % (C::TK / C::VEC)) * C::VEC;
        as.base[i] = (slot < C::A_SLOTS && m < g.M) ? m * g.K + as.kq[i] : -1;
    }
}

// Loads are unconditional (a masked lane reads element 0 and discards it), so
// the whole gather is straight-line code the scheduler can interleave with MFMAs.
// The masks are applied only when the registers go to LDS (after the MFMAs of
// the current chunk), so no wait for these loads sits in front of the MFMAs.
template <typename C>
__device__ inline typename C::Mask load_a(const typename C::T *__restrict__ Wt, const Geom &g, int kbase, bool,
                                          const ASlots<C> &as, Pack<typename C::T, C::VEC> (&ra)[C::A_PER]) {
    using M = typename C::Mask;
    M mask = 0;
#pragma unroll
    for (int i = 0; i < C::A_PER; ++i) {
        const int k = kbase + as.kq[i];
        if constexpr (C::KVEC) {
            // W rows start on 16-byte boundaries (K % VEC == 0, aligned base): index
            // through a uint4 pointer so the load is one global_load_dwordx4
            const bool ok = (as.base[i] >= 0) & (k < g.K);
            const uint4 *w4 = reinterpret_cast<const uint4 *>(Wt);
            // an invalid slot (k >= K or a row past M) reads element 0 and keeps zeros
            ra[i].q = keep_or_zero(ok, w4[ok ? (as.base[i] + kbase) / C::VEC : 0]);
            mask |= (ok ? ((M(1) << C::VEC) - M(1)) : M(0)) << (i * C::VEC);
        } else {
#pragma unroll
            for (int v = 0; v < C::VEC; ++v) {
                const bool ok = (as.base[i] >= 0) & (k + v < g.K);
                ra[i].e[v] = Wt[ok ? as.base[i] + kbase + v : 0];
                mask |= (ok ? M(1) : M(0)) << (i * C::VEC + v);
            }
        }
    }
    return mask;
}

// The im2col gather of B: this lane's pixel is fixed (lane_base = n*C*H*W +
// ih0*W + iw0); the run of KR consecutive k is the same for the whole wave, so
// (c, r, s) and the k part of the offset live in scalar registers.
template <typename C>
__device__ inline typename C::Mask load_b(const typename C::T *__restrict__ Dt, const Geom &g, int kstart_lane,
                                          bool pvalid, int lane_base, int ih0, int iw0,
                                          Pack<typename C::T, C::VEC> (&rb)[C::KR / C::VEC]) {
    using M = typename C::Mask;
    M mask = 0;
    using T = typename C::T;
    const int kstart = __builtin_amdgcn_readfirstlane(kstart_lane);
    const int RS = g.R * g.S;
    int c = kstart / RS;
    const int rem = kstart - c * RS;
    int r = rem / g.S;
    int s = rem - r * g.S;
    const int HW = g.H * g.W;
    int koff = c * HW + r * g.W + s;
    const int wrap_s = g.W - g.S, wrap_r = HW - g.R * g.W;
    // bf16: the loads go through a buffer descriptor of D, and an element outside the image, past K
    // or of a pixel past the end takes an offset past the buffer, whose load returns zero: no
    // validity bits and no 64-bit address per element (2 N C H W bytes < 2^32: make_plan keeps
    // N C H W below 2^31)
    [[maybe_unused]] __amdgpu_buffer_rsrc_t rd;
    if constexpr (sizeof(T) == 2)
        rd = __builtin_amdgcn_make_buffer_rsrc(const_cast<T *>(Dt), (short)0,
                                               (int)(unsigned)(2ull * (unsigned long long)g.N * (unsigned long long)g.CHW),
                                               0x00020000);
#pragma unroll
    for (int j = 0; j < C::KR; ++j) {
        const int ih = ih0 + r, iw = iw0 + s;
        // bitwise, not short-circuit: no branches in the gather
        const bool ok = pvalid & (kstart + j < g.K) & ((unsigned)ih < (unsigned)g.H) &
                        ((unsigned)iw < (unsigned)g.W);
        if constexpr (sizeof(T) == 2) {
            rb[j / C::VEC].e[j % C::VEC] =
                __builtin_amdgcn_raw_buffer_load_b16(rd, ok ? 2u * (unsigned)(lane_base + koff) : 0xFFFFFFFEu, 0, 0);
        } else {
            rb[j / C::VEC].e[j % C::VEC] = Dt[ok ? lane_base + koff : 0];
            mask |= (ok ? M(1) : M(0)) << j;
        }
        // advance (c, r, s) by one k with selects (scalar registers)
        ++s;
        ++koff;
        const bool ws = s == g.S;
        s = ws ? 0 : s;
        koff += ws ? wrap_s : 0;
        r += ws ? 1 : 0;
        const bool wr = r == g.R;
        r = wr ? 0 : r;
        koff += wr ? wrap_r : 0;
        c += wr ? 1 : 0;
    }
    if constexpr (sizeof(T) == 2) return ~M(0);   // every invalid element is a zero already
    return mask;
}

// NOMASK: the gathers zeroed every invalid element already (channels-last layers
// with 16-byte weight rows), so the registers go to LDS as they are.
template <typename C, bool NOMASK = false>
__device__ inline void store_lds(typename C::T *As, typename C::T *Bs, int tid,
                                 Pack<typename C::T, C::VEC> (&ra)[C::A_PER], typename C::Mask amask,
                                 Pack<typename C::T, C::VEC> (&rb)[C::KR / C::VEC], typename C::Mask bmask,
                                 int bp, int bkg) {
    using T = typename C::T;
#pragma unroll
    for (int i = 0; i < C::A_PER; ++i) {
        const int slot = tid + i * C::NT;
        if (C::A_SLOTS % C::NT == 0 || slot < C::A_SLOTS) {
            if constexpr (!NOMASK) {
#pragma unroll
                for (int v = 0; v < C::VEC; ++v)
                    ra[i].e[v] = ((amask >> (i * C::VEC + v)) & 1) ? ra[i].e[v] : T(0);
            }
            const int row = slot / (C::TK / C::VEC);
            const int kq = slot % (C::TK / C::VEC);
            *reinterpret_cast<uint4 *>(&As[row * C::LDK + kq * C::VEC]) = ra[i].q;
        }
    }
    if constexpr (!NOMASK) {
#pragma unroll
        for (int j = 0; j < C::KR; ++j)
            rb[j / C::VEC].e[j % C::VEC] = ((bmask >> j) & 1) ? rb[j / C::VEC].e[j % C::VEC] : T(0);
    }
#pragma unroll
    for (int j = 0; j < C::KR; j += C::VEC)
        *reinterpret_cast<uint4 *>(&Bs[bp * C::LDK + bkg * C::KR + j]) = rb[j / C::VEC].q;
}

// One chunk of MFMAs from LDS.  Within a chunk, lanes 0-31 take the first half
// of the k range and lanes 32-63 the second half; A and B use the same
// assignment, so every k of the chunk is summed exactly once.
template <int TK, int FM, int FP>
__device__ inline void mma_f32(const float *As, const float *Bs, int lane, int arow0, int brow0,
                               floatx16 (&acc)[FM][FP]) {
    constexpr int LDK = F32T<TK>::LDK;
    const int l32 = lane & 31, h = lane >> 5;
#pragma unroll
    for (int q = 0; q < TK / 8; ++q) {
        floatx4 a[FM], b[FP];
#pragma unroll
        for (int i = 0; i < FM; ++i)
            a[i] = *reinterpret_cast<const floatx4 *>(&As[(arow0 + i * 32 + l32) * LDK + h * (TK / 2) + q * 4]);
#pragma unroll
        for (int j = 0; j < FP; ++j)
            b[j] = *reinterpret_cast<const floatx4 *>(&Bs[(brow0 + j * 32 + l32) * LDK + h * (TK / 2) + q * 4]);
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FP; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][t], b[j][t], acc[i][j], 0, 0, 0);
    }
}

template <int TK, int FM, int FP>
__device__ inline void mma_bf16(const uint16_t *As, const uint16_t *Bs, int lane, int arow0, int brow0,
                                floatx16 (&acc)[FM][FP]) {
    constexpr int LDK = BF16T<TK>::LDK;
    const int l32 = lane & 31, h = lane >> 5;
#pragma unroll
    for (int q = 0; q < TK / 16; ++q) {
        bf16x8 a[FM], b[FP];
#pragma unroll
        for (int i = 0; i < FM; ++i)
            a[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8 *>(
                                                  &As[(arow0 + i * 32 + l32) * LDK + h * (TK / 2) + q * 8]));
#pragma unroll
        for (int j = 0; j < FP; ++j)
            b[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8 *>(
                                                  &Bs[(brow0 + j * 32 + l32) * LDK + h * (TK / 2) + q * 8]));
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FP; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
}

// One chunk of MFMAs from LDS for either element type.
template <typename C, int FM, int FP>
__device__ inline void mma_chunk(const typename C::T *As, const typename C::T *Bs, int lane, int arow0, int brow0,
                                 floatx16 (&acc)[FM][FP]) {
    if constexpr (sizeof(typename C::T) == 4)
        mma_f32<C::TK, FM, FP>(reinterpret_cast<const float *>(As), reinterpret_cast<const float *>(Bs), lane, arow0,
                               brow0, acc);
    else
        mma_bf16<C::TK, FM, FP>(reinterpret_cast<const uint16_t *>(As), reinterpret_cast<const uint16_t *>(Bs), lane,
                                arow0, brow0, acc);
}

// The B gather from channels-last Dt[n][h][w][c] with K in (r, s, c) order: a
// thread's run of KR consecutive k lies inside one (r, s) (Ch is a multiple of
// the chunk), so it is KR contiguous elements of one input pixel, loaded as
// 16-byte units; the padding test is one test for the whole run.
template <typename C>
__device__ inline typename C::Mask load_b_nhwc(const typename C::T *__restrict__ Dt, const Geom &g, int kstart_lane,
                                       bool pvalid, int img_base, int ih0, int iw0,
                                       Pack<typename C::T, C::VEC> (&rb)[C::KR / C::VEC]) {
    const int kstart = __builtin_amdgcn_readfirstlane(kstart_lane);
    const int rs = kstart / g.C, c0 = kstart - rs * g.C;
    const int r = rs / g.S, s = rs - r * g.S;
    const int ih = ih0 + r, iw = iw0 + s;
    const bool ok = pvalid & (kstart < g.K) & ((unsigned)ih < (unsigned)g.H) & ((unsigned)iw < (unsigned)g.W);
    // a multiple of KR: 16-byte aligned; a run outside the image reads element 0 and keeps zeros
    const uint4 *src = reinterpret_cast<const uint4 *>(Dt + (ok ? img_base + (ih * g.W + iw) * g.C + c0 : 0));
#pragma unroll
    for (int i = 0; i < C::KR / C::VEC; ++i) rb[i].q = keep_or_zero(ok, src[i]);
    using M = typename C::Mask;
    constexpr M all = C::KR == 8 * (int)sizeof(M) ? ~M(0) : ((M(1) << C::KR) - M(1));
    return ok ? all : 0u;
}

// Chunks of K on channels-last operands, each TK consecutive channels of one tap (r, s), walked
// with the channel blocks outer and the taps inner: the input window of one block of channels is
// read for all R*S taps of a tile while it is still in the L2 of the tile's XCD (with the taps
// outer, a tile's window over all channels was evicted before the next tap came back to it).
// The state is wave-uniform and advances by additions only (scalar registers, no divisions).
struct TapWalk {
    int r, s, c0;        // the chunk: tap (r, s), channels [c0, c0 + TK)
    __device__ inline void next(const Geom &g, int tk) {
        ++s;
        if (s == g.S) {
            s = 0;
            ++r;
            if (r == g.R) {
                r = 0;
                c0 += tk;
            }
        }
    }
    __device__ inline int kb(const Geom &g) const { return (r * g.S + s) * g.C + c0; }
};
// The TapWalk state of chunk j (chunks of tk channels, channel blocks outer, taps inner).
__device__ inline TapWalk tap_at(const Geom &g, int j, int tk) {
    const int rs_n = g.R * g.S, blk = j / rs_n, rs = j - blk * rs_n, r = rs / g.S;
    return TapWalk{r, rs - r * g.S, blk * tk};
}

// A 16-byte unit in global memory (address space 1): loads through it are global loads that the
// compiler knows cannot alias the thread's private arrays, which then stay in registers.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4 glb_u32x4;
__device__ inline uint4 load16(uintptr_t a) {
    return __builtin_bit_cast(uint4, *reinterpret_cast<const glb_u32x4 *>(a));
}

// The gathers of one chunk for the TapWalk loops, as raw 16-byte loads: a slot outside the
// operands (a weight row past M, a tap in the zero padding) loads from the 256-byte zero page
// instead, so no select waits on the loaded data and the loads stay in flight across the MFMAs
// of the current chunk.  Addresses are selected as integers (a pointer select becomes a branch).
template <typename C>
__device__ inline void load_a_tap(const typename C::T *__restrict__ Wt, int kb, const ASlots<C> &as, uintptr_t zpa,
                                  Pack<typename C::T, C::VEC> (&ra)[C::A_PER]) {
#pragma unroll
    for (int i = 0; i < C::A_PER; ++i) {
        const uintptr_t src = as.base[i] >= 0 ? reinterpret_cast<uintptr_t>(Wt + as.base[i] + kb) : zpa;
        ra[i].q = load16(src);
    }
}

// The B gather: the thread's KR channels of its pixel's input at tap (r, s).  pix_off = image
// base + (ih0 W + iw0) C + the thread's channel offset in the chunk.
template <typename C>
__device__ inline void load_b_tap(const typename C::T *__restrict__ Dt, const Geom &g, const TapWalk &t, bool pvalid,
                                  int pix_off, int ih0, int iw0, uintptr_t zpa,
                                  Pack<typename C::T, C::VEC> (&rb)[C::KR / C::VEC]) {
    const bool ok = pvalid & ((unsigned)(ih0 + t.r) < (unsigned)g.H) & ((unsigned)(iw0 + t.s) < (unsigned)g.W);
    const int off = pix_off + (t.r * g.W + t.s) * g.C + t.c0;
    const uintptr_t src = ok ? reinterpret_cast<uintptr_t>(Dt + off) : zpa;
#pragma unroll
    for (int i = 0; i < C::KR / C::VEC; ++i) rb[i].q = load16(src + 16 * i);
}

// Stateful form of the B gather, so that its elements can be issued one at a
// time between MFMAs: (c, r, s) and the k offset advance in scalar registers.
template <typename C> struct BGather {
    int kstart, c, r, s, koff;
    typename C::Mask mask;
    __device__ inline void begin(const Geom &g, int kstart_lane) {
        kstart = __builtin_amdgcn_readfirstlane(kstart_lane);
        const int RS = g.R * g.S;
        c = kstart / RS;
        const int rem = kstart - c * RS;
        r = rem / g.S;
        s = rem - r * g.S;
        koff = c * g.H * g.W + r * g.W + s;
        mask = 0;
    }
    __device__ inline void element(const typename C::T *__restrict__ Dt, const Geom &g, int j, bool pvalid,
                                   int lane_base, int ih0, int iw0, Pack<typename C::T, C::VEC> (&rb)[C::KR / C::VEC]) {
        const int ih = ih0 + r, iw = iw0 + s;
        const bool ok = pvalid & (kstart + j < g.K) & ((unsigned)ih < (unsigned)g.H) &
                        ((unsigned)iw < (unsigned)g.W);
        rb[j / C::VEC].e[j % C::VEC] = Dt[ok ? lane_base + koff : 0];
        mask |= (ok ? typename C::Mask(1) : typename C::Mask(0)) << j;
        ++s;
        ++koff;
        const bool ws = s == g.S;
        s = ws ? 0 : s;
        koff += ws ? g.W - g.S : 0;
        r += ws ? 1 : 0;
        const bool wr = r == g.R;
        r = wr ? 0 : r;
        koff += wr ? g.H * g.W - g.R * g.W : 0;
        c += wr ? 1 : 0;
    }
};

// One fp32 chunk with the next chunk's gather woven in: after every k-step
// (FM x FP MFMAs) the wave issues its share of the gather, so the vector ALU
// and the load pipeline run while the matrix core works.  sched_barrier(0)
// keeps the compiler from regrouping the two streams.
template <typename C, int FM, int FP, bool NEXT>
__device__ inline void chunk_f32(const float *As, const float *Bs, int lane, int arow0, int brow0,
                                 floatx16 (&acc)[FM][FP], const typename C::T *__restrict__ Dt,
                                 const typename C::T *__restrict__ Wt, const Geom &g, int kb_next, bool kvec,
                                 const ASlots<C> &as, Pack<typename C::T, C::VEC> (&ra)[C::A_PER], typename C::Mask &amask,
                                 BGather<C> &bg, int bkg, bool pvalid, int lane_base, int ih0, int iw0,
                                 Pack<typename C::T, C::VEC> (&rb)[C::KR / C::VEC]) {
    constexpr int TK = C::TK, LDK = C::LDK, STEPS = TK / 2;
    const int l32 = lane & 31, h = lane >> 5;
    floatx4 a[TK / 8][FM], b[TK / 8][FP];
#pragma unroll
    for (int q = 0; q < TK / 8; ++q) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
            a[q][i] = *reinterpret_cast<const floatx4 *>(&As[(arow0 + i * 32 + l32) * LDK + h * (TK / 2) + q * 4]);
#pragma unroll
        for (int j = 0; j < FP; ++j)
            b[q][j] = *reinterpret_cast<const floatx4 *>(&Bs[(brow0 + j * 32 + l32) * LDK + h * (TK / 2) + q * 4]);
    }
    if constexpr (NEXT) {
        amask = load_a<C>(Wt, g, kb_next, kvec, as, ra);
        bg.begin(g, kb_next + bkg * C::KR);
    }
#pragma unroll
    for (int t = 0; t < STEPS; ++t) {
        const int q = t / 4, tt = t % 4;
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FP; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[q][i][tt], b[q][j][tt], acc[i][j], 0, 0, 0);
        if constexpr (NEXT) {
            __builtin_amdgcn_sched_barrier(0);
            const int E0 = t * C::KR / STEPS, E1 = (t + 1) * C::KR / STEPS;  // folded by unrolling
#pragma unroll
            for (int e = E0; e < E1; ++e) bg.element(Dt, g, e, pvalid, lane_base, ih0, iw0, rb);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
}

// ---- direct-to-LDS main loop (bf16, channels-last, 64-deep chunks) ----------
//
// global_load_lds_dwordx4 moves 16 bytes per lane from global memory straight
// into LDS: lane L of a wave lands at the instruction's LDS base + 16*L (the
// base is wave-uniform), while every lane picks its own global address.  The
// tiles are kept as rows of 64 bf16 (128 bytes, eight 16-byte chunks) with
// chunk c of row r stored at position c ^ ((r >> 1) & 7), so one instruction
// fills eight whole rows, and a 16-byte fragment read of 16 consecutive rows
// (what the LDS serves in one cycle: 256 bytes over 64 banks) touches 16
// distinct 16-byte bank groups: rows 2i and 2i + 1 share a position but lie in
// different halves of a 256-byte line.  (The row's own low bits, c ^ (r & 7),
// put rows r and r + 8 on the same banks: two cycles a read, as the bank
// conflict counter showed.)  Two LDS stages: chunk k + 2 is requested into the stage of
// chunk k as soon as every wave has read chunk k, so a chunk's loads have a
// whole chunk of MFMAs to land.  Waits on the loads are explicit (vmcnt), and
// the barriers carry compiler-only fences: a memory fence would make the
// compiler wait for every load in flight, the next chunk's included.

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) const void glb_cvoid_t;

// s_waitcnt: at most V vector-memory operations of this wave outstanding.
template <int V> __device__ inline void wait_vmcnt() {
    static_assert(V >= 0 && V < 64, "vmcnt is six bits");
    __builtin_amdgcn_s_waitcnt((V & 15) | (0x7 << 4) | (0xF << 8) | ((V >> 4) << 14));
}
// s_waitcnt: no LDS operation of this wave outstanding.
__device__ inline void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }
// Workgroup barrier that orders LDS accesses around it in the compiler only.
__device__ inline void lds_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// One chunk of MFMAs from a swizzled stage.  The fragments of k-step q + 1 are
// read while the MFMAs of step q run (sched_barrier keeps the two groups
// apart), so no MFMA waits on the read right before it.
template <typename C, int FM, int FP>
__device__ inline void mma_chunk_swz(const unsigned char *As, const unsigned char *Bs, int lane, int arow0, int brow0,
                                     floatx16 (&acc)[FM][FP]) {
    const int l32 = lane & 31, h = lane >> 5, sw = (l32 >> 1) & 7;
    const unsigned char *arow = As + (arow0 + l32) * 128, *brow = Bs + (brow0 + l32) * 128;
    bf16x8 a[2][FM], b[2][FP];
    auto load = [&](int q, int slot) {
        const int pos = ((4 * h + q) ^ sw) * 16;
#pragma unroll
        for (int i = 0; i < FM; ++i)
            a[slot][i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8 *>(arow + i * 32 * 128 + pos));
#pragma unroll
        for (int j = 0; j < FP; ++j)
            b[slot][j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8 *>(brow + j * 32 * 128 + pos));
    };
    load(0, 0);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if (q + 1 < 4) load(q + 1, (q + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FP; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[q & 1][i], b[q & 1][j], acc[i][j], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// A raw buffer descriptor over [base, base + bytes) (stride 0, the data-format word of gfx9
// buffer resources), and a 16-byte load through it straight into LDS: lane L writes lds + 16 L.
__device__ inline __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, bytes, 0x00020000);
}
__device__ inline void buffer_load_lds16(__amdgpu_buffer_rsrc_t r, unsigned char *lds, unsigned voff, unsigned soff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t *)lds, 16, voff, soff, 0, 0);
}

// s_waitcnt vmcnt for a count known only at run time (the chunks still in flight behind the one
// about to be consumed): at most STAGES - 1 chunks of NI loads each.
template <int NI, int STAGES> __device__ inline void wait_chunks_behind(int behind) {
    if constexpr (STAGES > 2) {
        if (behind >= 2) {
            wait_vmcnt<2 * NI>();
            return;
        }
    }
    if (behind >= 1) wait_vmcnt<NI>();
    else wait_vmcnt<0>();
}

// The whole K loop of one tile, with buffer loads straight into LDS (buffer_load_dwordx4 ... lds:
// lane L of a wave lands at the LDS base + 16 L, the base wave-uniform).  Two buffer descriptors:
// the weights Wt, and the zero page followed by Dt (256 zero bytes in front of the channels-last
// input in the workspace).  A weight slot's offset is fixed for the tile (rows past M read row
// M - 1: their outputs are never stored) and the chunk's k goes into the scalar offset; an input
// slot's offset is its pixel's base plus the chunk's tap offset, or 0 (the zero page) for a tap in
// the padding.  So a chunk costs a few vector instructions per input slot and none per weight
// slot.  Chunks follow TapWalk (channel blocks of 64 outer, taps inner) through a ring of STAGES
// LDS stages: chunk k + STAGES - 1 is requested as soon as every wave has read chunk k - 1's
// stage, so a chunk's loads have STAGES - 1 chunks of MFMAs to land.  Needs Ch % 64 == 0.
template <typename C, int FM, int FP, int STAGES>
__device__ inline void dma_mainloop(const uint16_t *__restrict__ Wt, const Geom &g, int m0, long long p0,
                                    const unsigned char *zp_dt, unsigned char *smem, floatx16 (&acc)[FM][FP],
                                    int tid, int arow0, int brow0, int k0, int kn) {
    constexpr int NW = C::NT / 64;
    constexpr int NIA = C::TM / (8 * NW), NIB = C::TP / (8 * NW), NI = NIA + NIB;
    static_assert(C::TM % (8 * NW) == 0 && C::TP % (8 * NW) == 0 && (STAGES - 1) * NI < 64, "DMA tile shape");
    constexpr int STAGE_A = C::TM * 128, STAGE = (C::TM + C::TP) * 128;
    const int lane = tid & 63, w = tid >> 6;
    const int lr = lane >> 3;              // row of the instruction's eight
    // the global chunk this lane loads (its LDS chunk is lane & 7) for an instruction whose eight
    // rows start at a multiple of 16 (sw = 0) or 8 mod 16 (sw = 4): row r's swizzle is (r >> 1) & 7
    auto cg = [&](int sw) { return (lane & 7) ^ ((sw + (lr >> 1)) & 7); };
    const __amdgpu_buffer_rsrc_t rw = buffer_rsrc(Wt, (int)((long long)g.M * g.K * 2));
    const __amdgpu_buffer_rsrc_t rd = buffer_rsrc(zp_dt, (int)(256 + (long long)g.N * g.CHW * 2));
    unsigned a_off[NIA];
#pragma unroll
    for (int j = 0; j < NIA; ++j) {
        int m = m0 + (j * NW + w) * 8 + lr;
        m = m < g.M ? m : g.M - 1;
        a_off[j] = (unsigned)(m * g.K + cg(4 * ((j * NW + w) & 1)) * 8) * 2u;
    }
    unsigned b_off[NIB];
    int b_ih[NIB], b_iw[NIB];
#pragma unroll
    for (int j = 0; j < NIB; ++j) {
        long long pg = p0 + (j * NW + w) * 8 + lr;
        pg = pg < g.P_total ? pg : g.P_total - 1;   // columns past the end are never stored
        const int n = (int)(pg / g.EF);
        const int pix = (int)(pg - (long long)n * g.EF);
        const int x = pix / g.F, y = pix - (pix / g.F) * g.F;
        b_ih[j] = g.U * x - g.P;
        b_iw[j] = g.U * y - g.P;
        // 32-bit wrap-around arithmetic: the sum with a valid tap's offset is the element's offset
        b_off[j] = 256u + 2u * (unsigned)(n * (int)g.CHW + (b_ih[j] * g.W + b_iw[j]) * g.C +
                                          cg(4 * ((j * NW + w) & 1)) * 8);
    }
    // part q (of 4) of a chunk's loads: every fourth weight and input slot
    auto issue_part = [&](const TapWalk &t, unsigned char *base, int q) {
        const unsigned soff_a = 2u * (unsigned)t.kb(g);
        const unsigned tap = 2u * (unsigned)((t.r * g.W + t.s) * g.C + t.c0);
#pragma unroll
        for (int j = q; j < NIA; j += 4) {
            buffer_load_lds16(rw, base + (j * NW + w) * 8 * 128, a_off[j], soff_a);
        }
#pragma unroll
        for (int j = q; j < NIB; j += 4) {
            const bool ok = ((unsigned)(b_ih[j] + t.r) < (unsigned)g.H) & ((unsigned)(b_iw[j] + t.s) < (unsigned)g.W);
            buffer_load_lds16(rd, base + STAGE_A + (j * NW + w) * 8 * 128, ok ? b_off[j] + tap : 0u, 0u);
        }
    };
    // chunks [k0, k0 + nch) of the tile's K (kn < 0: all of them)
    const int nch = kn >= 0 ? kn : g.R * g.S * (g.C / 64);
    TapWalk ti = tap_at(g, k0, 64);
#pragma unroll
    for (int st = 0; st + 1 < STAGES; ++st) {
        if (st < nch) {
#pragma unroll
            for (int q = 0; q < 4; ++q) issue_part(ti, smem + st * STAGE, q);
            ti.next(g, 64);
        }
    }
    for (int kc = 0; kc < nch; ++kc) {
        // this wave's loads of chunk kc have landed when at most the later chunks' are in flight
        const int behind = nch - 1 - kc < STAGES - 2 ? nch - 1 - kc : STAGES - 2;
        wait_chunks_behind<NI, STAGES>(behind);
        lds_barrier();                        // ... and every wave's; every wave is done with chunk kc - 1
        // chunk kc + STAGES - 1 goes into the stage chunk kc - 1 used, all of it before this
        // chunk's MFMAs (spreading the requests between the k-steps measured slower)
        if (kc + STAGES - 1 < nch) {
            unsigned char *nbase = smem + ((kc + STAGES - 1) % STAGES) * STAGE;
#pragma unroll
            for (int q = 0; q < 4; ++q) issue_part(ti, nbase, q);
            ti.next(g, 64);
        }
        const unsigned char *st = smem + (kc % STAGES) * STAGE;
        mma_chunk_swz<C, FM, FP>(st, st + STAGE_A, lane, arow0, brow0, acc);
        wait_lgkm0();
    }
}

// Epilogue arguments.  EPI 0: plain store.  EPI 1: the CoC-D summations of
// every stored value as well (Sec. 3.6): for each pixel p of the tile, the tile's
// rows give sum O, sum (m + wbase) O, (n + wbase) sum O and sum O^2, written as
// slice (tile_m * N + n) of a [slices][4][E*F] float64 array; block 0 resets the
// report.  EPI 2: EPI 1 with faults planted in the stored values first.
// With EPI 1 and 2, aux_groups groups of eight consecutive workgroup ids (one per
// XCD) may do other work of the protected layer instead of a tile, memory-bound work
// that runs beside the matrix-bound tiles of the same launch:
//   aux_kind 1: encode the input checksums Cd1, Cd2 of D (Sec. 3.2), in the first
//               groups of the grid (they read D as the first tiles do);
//   aux_kind 2: combine the image-split partials of Cd1, Cd2 left by the
//               channels-last copy, and compute the Co5..Co7 partial products
//               (coc_tile.h), in the last groups, after the tile_groups groups of
//               tiles, where they fill the slots the tiles' last round leaves.
struct NoFaults {};
// Stream-K schedule of the channels-last loops (S > 0): the launch has S workgroups (after the
// extra ones), as many as are resident at once.  The first dp_waves x S tiles run whole, tile
// r S + w being workgroup w's r-th, so that the workgroups resident together work on neighbouring
// tiles, as in the plain grid.  The last one to two waves' tiles (T of them) are shared evenly:
// workgroup w runs their iterations [w U / S, (w + 1) U / S) of the U = T x nch (tile, chunk)
// pairs in tile order.  A tile whose chunks span several workgroups is summed by the last of them
// to arrive: each writes its partial accumulators to a slot (0: the workgroup's first shared
// segment, 1: its last), counts itself in cnt[tile], and the last adds the slots in chunk order (a
// fixed order, whichever workgroup is last) before the epilogue.
struct SkArgs {
    float *part;    // [S][2][TM * TP]
    int *cnt;       // [tiles], zero at the launch (the channels-last copy clears it); left zero
    int S;          // 0: one tile per workgroup
    int nch;        // chunks per tile
    int dp_waves;   // waves of whole tiles before the shared ones
};
template <int EPI> struct Epi {
    double *part;
    ftcnn_report *rep;
    int cap;
    int aux_kind, aux_blocks, aux_groups;
    int tile_groups;     // groups of eight tile workgroups in front of the aux_kind 2 ones
    double *cd1, *cd2;   // kind 1: encoded here; kind 2: written by the combine workgroups
    int enc_vec;         // kind 1: 16-byte loads
    CdSrc src;           // kind 2
    const double *cw1, *cw2;
    double *copart;
    CocTile co;
    int co_slices;       // Co partial slices this launch writes (recorded in rep->reserved[1])
    typename std::conditional<EPI == 2, FaultList, NoFaults>::type fl;
    const float *bias;   // NULL, or [M] added to every stored value of filter m (Sec. 5.1)
};
template <> struct Epi<0> {
    const float *bias;
};

template <typename T> struct Bits;
template <> struct Bits<float> {
    using B = float;   // an fp32 output is stored as computed
    __device__ static B make(float v) { return v; }
    __device__ static float value(B b) { return b; }
};
template <> struct Bits<uint16_t> {
    using B = uint16_t;
    __device__ static B make(float v) { return f32_to_bf16_rne(v); }
    __device__ static float value(B b) { return bf16_bits_to_f32(b); }
};

template <typename Tr, int WM, int WP, int FM, int FP, int WEAVE, bool KVEC, int EPI, bool NHWC, bool GRP = false,
          bool SK = false>
__global__ __launch_bounds__(64 * WM * WP) void conv_kernel(const typename Tr::T *__restrict__ D,
                                                            const typename Tr::T *__restrict__ Wt,
                                                            typename Tr::T *__restrict__ O, Geom g,
                                                            int tiles_m, int tiles_total, int m_major,
                                                            const void *zp, Epi<EPI> ep, SkArgs sk) {
    using C = Cfg<Tr, WM, WP, FM, FP, KVEC, (WEAVE >= 3 ? WEAVE - 1 : 0)>;
    using T = typename C::T;
    extern __shared__ __align__(16) unsigned char smem[];
    T *As0 = reinterpret_cast<T *>(smem);
    T *Bs0 = As0 + 2 * C::TM * C::LDK;

    const int tid = threadIdx.x;
    int bid = blockIdx.x;
    if constexpr (EPI != 0) {
        if (bid == 0 && tid == 0) {
            reset_report(ep.rep, ep.cap);
            ep.rep->reserved[1] = ep.co_slices;
        }
        if (ep.aux_groups > 0) {
            int ab = -1;   // this workgroup's index among the extra ones
            if (ep.aux_kind == 2) {
                if ((bid >> 3) >= ep.tile_groups) ab = bid - 8 * ep.tile_groups;
            } else if ((bid >> 3) < ep.aux_groups) {
                ab = bid;
            } else {
                bid -= 8 * ep.aux_groups;   // keeps bid % 8, hence the XCD the tile order assumes
            }
            if (ab >= 0) {
                const int bid = ab;
                if (bid < ep.aux_blocks) {
                    if (ep.aux_kind == 1) {
                        if (ep.enc_vec) encode_block<T, C::NT, kEncVec>(D, g, bid, ep.cd1, ep.cd2);
                        else encode_block<T, C::NT, 1>(D, g, bid, ep.cd1, ep.cd2);
                    } else if (bid < ep.co.comb_blocks) {
                        combine_block<C::NT>(g, ep.src, ep.cd1, ep.cd2, bid);
                    } else {
                        coc_block<C::NT>(g, ep.co, ep.src, ep.cw1, ep.cw2, ep.copart, bid - ep.co.comb_blocks,
                                         reinterpret_cast<double *>(smem));
                    }
                }
                return;
            }
        }
    }
    constexpr bool DMA = NHWC && WEAVE >= 3 && sizeof(T) == 2 && C::TK == 64;
    // the stream-K form (a separate kernel: the whole-tile kernels keep their registers) of the
    // loops that can run a range of a tile's chunks (channels-last, dense)
    constexpr bool SKOK = SK && NHWC && !GRP && WEAVE != 2;
    constexpr bool skm = SKOK;
    long long sk_it = 0, sk_end = 0, sk_u = 0, sk_i0 = 0;
    int wl = 0, dp = 0;
    if (skm) {
        if (bid >= sk.S) return;
        // contiguous tiles and iteration ranges per XCD, as the tile order below
        wl = xcd_tile(bid, sk.S);
        sk_i0 = (long long)sk.dp_waves * sk.S * sk.nch;   // the first shared iteration
        sk_u = (long long)tiles_total * sk.nch - sk_i0;
        sk_it = sk_i0 + (long long)wl * sk_u / sk.S;
        sk_end = sk_i0 + (long long)(wl + 1) * sk_u / sk.S;
    } else if (bid >= tiles_total) {
        return;
    }
    bool first_seg = true;    // the next shared segment is this workgroup's first
    bool first_iter = true;
    const Geom &g_all = g;
    for (;;) {
    // In the stream-K kernel the thread index and the geometry are passed through empty asm at
    // every segment, so that nothing derived from them is hoisted out of the segment loop and
    // held (in registers, or spilled) across the main loop and the epilogue.
    int tid;
    Geom g = g_all;
    if constexpr (SK) {
        asm volatile("v_mov_b32 %0, %1" : "=v"(tid) : "v"((int)threadIdx.x));
        asm volatile("" : "+s"(g.N), "+s"(g.C), "+s"(g.H), "+s"(g.W), "+s"(g.M), "+s"(g.R), "+s"(g.S));
        asm volatile("" : "+s"(g.U), "+s"(g.P), "+s"(g.E), "+s"(g.F), "+s"(g.K), "+s"(g.EF));
        asm volatile("" : "+s"(g.CHW), "+s"(g.P_total), "+s"(g.wbase));
    } else {
        tid = threadIdx.x;
    }
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wp = wave / WM;
    // the segment: chunks [k0, k0 + kn) of one tile (kn < 0: the whole tile)
    int tile, k0 = 0, kn = -1;
    if (skm) {
        if (dp < sk.dp_waves) {
            tile = dp * sk.S + wl;
            kn = sk.nch;
        } else {
            if (sk_it >= sk_end) break;
            tile = (int)(sk_it / sk.nch);
            k0 = (int)(sk_it - (long long)tile * sk.nch);
            kn = (int)(sk_end - sk_it < (long long)(sk.nch - k0) ? sk_end - sk_it : (long long)(sk.nch - k0));
        }
        if (!first_iter) __syncthreads();   // every wave is done with the last segment's LDS
    } else {
        // logical tile order: pixel-major keeps the M tiles of one pixel tile on one
        // XCD (its L2 serves the repeated D reads); M-major keeps one slab of W
        // resident per XCD instead (preferred when W is larger than an XCD's L2)
        tile = xcd_tile(bid, tiles_total);
    }
    const int tiles_p = tiles_total / tiles_m;
    const int mt = m_major ? tile / tiles_p : tile % tiles_m;
    const int pt = m_major ? tile % tiles_p : tile / tiles_m;
    const int m0 = mt * C::TM;
    const long long p0 = (long long)pt * C::TP;

    // this thread's im2col pixel (fixed over the K loop)
    const int bp = tid % C::TP, bkg = tid / C::TP;
    const long long pg = p0 + bp;
    const bool pvalid = pg < g.P_total;
    int lane_base = 0, ih0 = 0, iw0 = 0;
    if (pvalid) {
        const int n = (int)(pg / g.EF);
        const int pix = (int)(pg - (long long)n * g.EF);
        const int x = pix / g.F, y = pix - (pix / g.F) * g.F;
        ih0 = g.U * x - g.P;
        iw0 = g.U * y - g.P;
        // channels-last: the image's base in Dt; otherwise the pixel's first tap in D
        lane_base = NHWC ? n * (int)g.CHW : n * (int)g.CHW + ih0 * g.W + iw0;
    }
    ASlots<C> as;
    a_slots<C>(g, m0, tid, as);

    floatx16 acc[FM][FP];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FP; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

    const int arow0 = wm * FM * 32, brow0 = wp * FP * 32;
    Pack<T, C::VEC> ra[C::A_PER];
    Pack<T, C::VEC> rb[C::KR / C::VEC];
    const int nchunks = (g.K + C::TK - 1) / C::TK;
    // grouped layers (Sec. 5.2) run on the block-diagonal expansion of W: a tile whose filters all
    // lie in one group needs only the chunks of K = (r, s, c) with c in that group's channels (the
    // others multiply zeros), and the channels-last loop below walks just those
    constexpr bool KSKIP = GRP && NHWC && !DMA && WEAVE != 2;   // a separate kernel: dense loops unchanged
    int nch = nchunks, cpr = 0, cg0 = 0;
    if constexpr (KSKIP) {
        const int mlast = (m0 + C::TM < g.M ? m0 + C::TM : g.M) - 1;
        if (g.G > 1 && g.Cg % C::TK == 0 && m0 / g.Mg == mlast / g.Mg) {
            cpr = g.Cg / C::TK;
            cg0 = group_first_channel(g, m0);
            nch = g.R * g.S * cpr;
        }
    }
    auto kbase = [&](int j) {
        if (KSKIP && cpr > 0) {
            const int rs = j / cpr;
            return rs * g.C + cg0 + (j - rs * cpr) * C::TK;
        }
        return j * C::TK;
    };
    typename C::Mask amask = 0, bmask = 0;
    // channels-last loops other than the two-in-flight one: chunks walked by TapWalk, channel
    // blocks [cg0, cg0 + TK * (nch / (R S))) outer, taps inner
    constexpr bool TAPS = NHWC && !DMA && WEAVE != 2;
    TapWalk tw{0, 0, 0};
    int pix_off = 0;
    const uintptr_t zpa = reinterpret_cast<uintptr_t>(zp);   // 256 zero bytes (channels-last layers)
    if constexpr (TAPS) {
        tw.c0 = cg0;
        if (!(KSKIP && cpr > 0)) nch = g.R * g.S * (g.C / C::TK);
        pix_off = lane_base + (ih0 * g.W + iw0) * g.C + bkg * C::KR;
        if (SKOK && kn >= 0) {
            tw = tap_at(g, k0, C::TK);
            nch = kn;
        }
    }
    if constexpr (!DMA) {
        if constexpr (TAPS) {
            load_a_tap<C>(Wt, tw.kb(g), as, zpa, ra);
            load_b_tap<C>(D, g, tw, pvalid, pix_off, ih0, iw0, zpa, rb);
        } else {
            amask = load_a<C>(Wt, g, kbase(0), KVEC, as, ra);
            bmask = NHWC ? load_b_nhwc<C>(D, g, kbase(0) + bkg * C::KR, pvalid, lane_base, ih0, iw0, rb)
                         : load_b<C>(D, g, bkg * C::KR, pvalid, lane_base, ih0, iw0, rb);
        }
        store_lds<C, NHWC>(As0, Bs0, tid, ra, amask, rb, bmask, bp, bkg);
        __syncthreads();
    }

    if constexpr (DMA) {
        // D is the channels-last copy, which the workspace keeps right behind the zero page zp
        dma_mainloop<C, FM, FP, WEAVE - 1>(reinterpret_cast<const uint16_t *>(Wt), g, m0, p0,
                                           static_cast<const unsigned char *>(zp), smem, acc, tid, arow0, brow0,
                                           k0, kn);
    } else if constexpr (NHWC && WEAVE == 2) {
        // channels-last, two chunks in flight: chunk kc + 2 is loaded into one register set
        // while chunk kc is consumed from LDS, and chunk kc + 1 (loaded a whole chunk earlier,
        // in the other set) then goes to the other LDS buffer, so the stores wait only on loads
        // issued two chunks back.  Unrolled by two so that each register set keeps its
        // registers; loads past the last chunk are fully masked (in-bounds, no effect).
        Pack<T, C::VEC> ra2[C::A_PER];
        Pack<T, C::VEC> rb2[C::KR / C::VEC];
        typename C::Mask amask2 = load_a<C>(Wt, g, C::TK, KVEC, as, ra2);
        typename C::Mask bmask2 = load_b_nhwc<C>(D, g, C::TK + bkg * C::KR, pvalid, lane_base, ih0, iw0, rb2);
        T *A0 = As0, *A1 = As0 + C::TM * C::LDK, *B0 = Bs0, *B1 = Bs0 + C::TP * C::LDK;
        // no exit inside the body (a chunk past the end is stored as zeros and never used), so the
        // accumulators stay in one set of registers
        int kc = 0;
        for (; kc + 1 < nchunks; kc += 2) {
            amask = load_a<C>(Wt, g, (kc + 2) * C::TK, KVEC, as, ra);
            bmask = load_b_nhwc<C>(D, g, (kc + 2) * C::TK + bkg * C::KR, pvalid, lane_base, ih0, iw0, rb);
            mma_chunk<C, FM, FP>(A0, B0, lane, arow0, brow0, acc);
            store_lds<C, NHWC>(A1, B1, tid, ra2, amask2, rb2, bmask2, bp, bkg);
            __syncthreads();
            amask2 = load_a<C>(Wt, g, (kc + 3) * C::TK, KVEC, as, ra2);
            bmask2 = load_b_nhwc<C>(D, g, (kc + 3) * C::TK + bkg * C::KR, pvalid, lane_base, ih0, iw0, rb2);
            mma_chunk<C, FM, FP>(A1, B1, lane, arow0, brow0, acc);
            store_lds<C, NHWC>(A0, B0, tid, ra, amask, rb, bmask, bp, bkg);
            __syncthreads();
        }
        if (kc < nchunks) mma_chunk<C, FM, FP>(A0, B0, lane, arow0, brow0, acc);   // odd count: the last chunk
    } else if constexpr (NHWC) {
        // channels-last: a whole chunk's gather is a few 16-byte loads per thread, issued
        // before this chunk's MFMAs and stored after them.  The scheduling fences keep the
        // compiler from sinking the loads next to their stores: they then have the whole
        // chunk of MFMAs to land instead of a few.
        for (int kc = 0; kc + 1 < nch; ++kc) {
            const int buf = kc & 1;
            tw.next(g, C::TK);
            load_a_tap<C>(Wt, tw.kb(g), as, zpa, ra);
            load_b_tap<C>(D, g, tw, pvalid, pix_off, ih0, iw0, zpa, rb);
            __builtin_amdgcn_sched_barrier(0);
            mma_chunk<C, FM, FP>(As0 + buf * C::TM * C::LDK, Bs0 + buf * C::TP * C::LDK, lane, arow0, brow0, acc);
            __builtin_amdgcn_sched_barrier(0);
            store_lds<C, NHWC>(As0 + (buf ^ 1) * C::TM * C::LDK, Bs0 + (buf ^ 1) * C::TP * C::LDK, tid, ra, amask, rb,
                         bmask, bp, bkg);
            __syncthreads();
        }
        mma_chunk<C, FM, FP>(As0 + ((nch - 1) & 1) * C::TM * C::LDK, Bs0 + ((nch - 1) & 1) * C::TP * C::LDK,
                             lane, arow0, brow0, acc);
    } else if constexpr (WEAVE == 2 && sizeof(T) == 4) {
        // two chunks in flight: while a chunk is consumed from one LDS buffer, the gather of the
        // chunk two ahead is woven between its MFMAs into one register set, and the other set
        // (the next chunk, loaded a whole chunk earlier) goes to the other buffer at the end, so
        // no load latency is waited on.  The loop is unrolled by two so that each register set
        // keeps its registers; chunks past the last one are fully masked (zeros, no effect).
        Pack<T, C::VEC> ra2[C::A_PER];
        Pack<T, C::VEC> rb2[C::KR / C::VEC];
        typename C::Mask amask2 = load_a<C>(Wt, g, C::TK, KVEC, as, ra2);
        BGather<C> bg, bg2;
        bg2.mask = load_b<C>(D, g, C::TK + bkg * C::KR, pvalid, lane_base, ih0, iw0, rb2);
        const float *A0 = reinterpret_cast<const float *>(As0), *A1 = A0 + C::TM * C::LDK;
        const float *B0 = reinterpret_cast<const float *>(Bs0), *B1 = B0 + C::TP * C::LDK;
        for (int kc = 0; kc < nchunks; kc += 2) {
            chunk_f32<C, FM, FP, true>(A0, B0, lane, arow0, brow0, acc, D, Wt, g, (kc + 2) * C::TK, KVEC, as, ra,
                                       amask, bg, bkg, pvalid, lane_base, ih0, iw0, rb);
            store_lds<C>(As0 + C::TM * C::LDK, Bs0 + C::TP * C::LDK, tid, ra2, amask2, rb2, bg2.mask, bp, bkg);
            __syncthreads();
            chunk_f32<C, FM, FP, true>(A1, B1, lane, arow0, brow0, acc, D, Wt, g, (kc + 3) * C::TK, KVEC, as, ra2,
                                       amask2, bg2, bkg, pvalid, lane_base, ih0, iw0, rb2);
            if (kc + 2 >= nchunks) break;
            store_lds<C>(As0, Bs0, tid, ra, amask, rb, bg.mask, bp, bkg);
            __syncthreads();
        }
    } else if constexpr (WEAVE == 1 && sizeof(T) == 4) {
        // every chunk but the last: the next chunk's gather is woven between this chunk's MFMAs
        BGather<C> bg;
        for (int kc = 0; kc + 1 < nchunks; ++kc) {
            const int buf = kc & 1;
            chunk_f32<C, FM, FP, true>(reinterpret_cast<const float *>(As0 + buf * C::TM * C::LDK),
                                       reinterpret_cast<const float *>(Bs0 + buf * C::TP * C::LDK), lane, arow0,
                                       brow0, acc, D, Wt, g, (kc + 1) * C::TK, KVEC, as, ra, amask, bg, bkg,
                                       pvalid, lane_base, ih0, iw0, rb);
            store_lds<C>(As0 + (buf ^ 1) * C::TM * C::LDK, Bs0 + (buf ^ 1) * C::TP * C::LDK, tid, ra, amask, rb,
                         bg.mask, bp, bkg);
            __syncthreads();
        }
        chunk_f32<C, FM, FP, false>(reinterpret_cast<const float *>(As0 + ((nchunks - 1) & 1) * C::TM * C::LDK),
                                    reinterpret_cast<const float *>(Bs0 + ((nchunks - 1) & 1) * C::TP * C::LDK),
                                    lane, arow0, brow0, acc, D, Wt, g, 0, KVEC, as, ra, amask, bg, bkg, pvalid,
                                    lane_base, ih0, iw0, rb);
    } else {
        auto mma = [&](int buf) {
            const T *As = As0 + buf * C::TM * C::LDK;
            const T *Bs = Bs0 + buf * C::TP * C::LDK;
            if constexpr (sizeof(T) == 4)
                mma_f32<C::TK, FM, FP>(reinterpret_cast<const float *>(As), reinterpret_cast<const float *>(Bs),
                                       lane, arow0, brow0, acc);
            else
                mma_bf16<C::TK, FM, FP>(reinterpret_cast<const uint16_t *>(As),
                                        reinterpret_cast<const uint16_t *>(Bs), lane, arow0, brow0, acc);
        };
        // every chunk but the last: fetch the next one while the MFMAs consume this one
        for (int kc = 0; kc + 1 < nchunks; ++kc) {
            const int buf = kc & 1;
            const int kb = (kc + 1) * C::TK;
            amask = load_a<C>(Wt, g, kb, KVEC, as, ra);
            bmask = load_b<C>(D, g, kb + bkg * C::KR, pvalid, lane_base, ih0, iw0, rb);
            mma(buf);
            store_lds<C>(As0 + (buf ^ 1) * C::TM * C::LDK, Bs0 + (buf ^ 1) * C::TP * C::LDK, tid, ra, amask, rb,
                         bmask, bp, bkg);
            __syncthreads();
        }
        mma((nchunks - 1) & 1);
    }

    if constexpr (SKOK) {
        if (kn >= 0 && kn < sk.nch) {
            // a part of the tile: publish it; the last of the tile's workgroups sums them all
            const long long ib = (long long)tile * sk.nch;
            // the workgroup whose range holds iteration i
            auto owner = [&](long long i) { return (int)(((i - sk_i0 + 1) * sk.S - 1) / sk_u); };
            const int w0 = owner(ib), w1 = owner(ib + sk.nch - 1);
            constexpr int NR = FM * FP * 16;   // accumulators per thread; slot layout [NR][NT]
            float *mine = sk.part + ((size_t)wl * 2 + (first_seg ? 0 : 1)) * (size_t)(C::TM * C::TP);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FP; ++j) {
#pragma unroll
                    for (int e = 0; e < 16; ++e)
                        __hip_atomic_store(mine + ((i * FP + j) * 16 + e) * C::NT + tid, acc[i][j][e],
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __builtin_amdgcn_sched_barrier(0);   // a few store addresses live at a time
                }
            // The parts go to memory with device-coherent stores (they bypass the XCD's L2), so
            // once every wave has seen its stores complete, one device-scope count publishes the
            // whole part: no L2 write-back is needed.  Every wave is past the main loop: the first
            // word of LDS carries the verdict.
            int *sk_last = reinterpret_cast<int *>(smem);
            wait_vmcnt<0>();
            __syncthreads();
            if (tid == 0)
                *sk_last = __hip_atomic_fetch_add(sk.cnt + tile, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                           w1 - w0;
            __syncthreads();
            const bool last = *sk_last != 0;
            if (!last) {
                sk_it += kn;
                first_seg = false;
                first_iter = false;
                continue;
            }
            // the other parts, read with device-coherent loads after the count said they are all there
            if (tid == 0) __hip_atomic_store(sk.cnt + tile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            // the tile's parts in chunk order (this workgroup's own from its slot too): part w lies
            // in slot 0 of workgroup w when its range starts inside this tile, else in its slot 1
            // (its last segment).  Sixteen loads at a time, so the sums need few registers beyond
            // the accumulators.
            static_assert(NR * C::NT == C::TM * C::TP, "slot size");
            for (int w = w0; w <= w1; ++w) {
                const int slot = sk_i0 + (long long)w * sk_u / sk.S >= ib ? 0 : 1;
                const float *src = sk.part + ((size_t)w * 2 + slot) * (size_t)(C::TM * C::TP) + tid;
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FP; ++j) {
                        float v[16];
#pragma unroll
                        for (int e = 0; e < 16; ++e)
                            v[e] = __hip_atomic_load(src + ((i * FP + j) * 16 + e) * C::NT, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
                        for (int e = 0; e < 16; ++e) acc[i][j][e] = w == w0 ? v[e] : acc[i][j][e] + v[e];
                        __builtin_amdgcn_sched_barrier(0);
                    }
            }
        }
    }

    // epilogue: lane owns pixel (lane & 31) of each 32-wide block; register e of
    // block (i, j) is row 8*(e/4) + 4*(lane/32) + e%4 of that block
    const int l32 = lane & 31, h = lane >> 5;
    // the tile's bias rows (Sec. 5.1), staged in LDS once the main loop is done: read in the store
    // loops below from LDS, whose wait never holds on the tile's own output stores
    const bool hb = ep.bias != nullptr;
    constexpr size_t kBiasOff = EPI == 0 ? 0 : (size_t)WM * 3 * C::TP * sizeof(double);
    static_assert(kBiasOff + C::TM * sizeof(float) <= C::LDS_BYTES, "bias rows fit LDS");
    float *bias_s = reinterpret_cast<float *>(smem + kBiasOff);
    if (hb) {
        __syncthreads();   // every wave is done with the operand tiles
        for (int t = tid; t < C::TM; t += C::NT) bias_s[t] = m0 + t < g.M ? ep.bias[m0 + t] : 0.0f;
        __syncthreads();
    }
    if constexpr (EPI == 0) {
        if (!hb) {
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
        } else {
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
                        const int mt_row = arow0 + i * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
                        const int m = m0 + mt_row;
                        if (m < g.M) Elem<T>::store(O, ob + (long long)m * g.EF, acc[i][j][e] + bias_s[mt_row]);
                    }
            }
        }
    } else {
        using Bt = Bits<T>;
        // faults inside this tile (a uniform test; usually none)
        bool planted = false;
        if constexpr (EPI == 2) {
            for (int f = 0; f < ep.fl.n; ++f) {
                const ftcnn_fault &q = ep.fl.f[f];
                const long long pf = (long long)q.n * g.EF + (long long)q.x * g.F + q.y;
                planted |= q.m >= m0 && q.m < m0 + C::TM && pf >= p0 && pf < p0 + C::TP;
            }
        }
        if constexpr (WM > 1) __syncthreads();  // the LDS tiles are free: reuse them for the cross-wave fold
        double *red = reinterpret_cast<double *>(smem);   // [WM][3][TP]
        const double wb = (double)g.wbase;
        // per-column state; rows are visited one register at a time (row-dependent
        // values are then live only briefly, which keeps the kernel's register
        // budget, and so the main loop's occupancy, close to the plain store's)
        const int mrow = m0 + arow0 + 4 * h;
        T *obase[FP];
        long long pcol[FP];
        bool cval[FP];
        double s1[FP], s6[FP], sq[FP];
#pragma unroll
        for (int j = 0; j < FP; ++j) {
            const long long pgo = p0 + brow0 + j * 32 + l32;
            cval[j] = pgo < g.P_total;
            const long long n = cval[j] ? pgo / g.EF : 0;
            pcol[j] = pgo;
            obase[j] = O + (n * g.M + mrow) * (long long)g.EF + (pgo - n * g.EF);
            s1[j] = s6[j] = sq[j] = 0.0;
        }
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            if constexpr (sizeof(T) == 2) {
                // bf16 outputs: the 16 rows of a block are first summed in fp32, then added in
                // fp64.  Every term is exact in fp32 (8-bit values, weights m + wbase below 2^16),
                // so the only roundings are the 15 additions of a run: at most 15 * 2^-24 of the
                // run's sum of magnitudes, far inside the bf16 tolerance (whose output unit is
                // 2^-8), and none at all while the partial sums stay integers below 2^24.  The
                // fp64 arithmetic per element would otherwise cost as much as a third of the
                // matrix-core time on short-K layers.
                float f1[FP], f6[FP], fq[FP];
#pragma unroll
                for (int j = 0; j < FP; ++j) f1[j] = f6[j] = fq[j] = 0.0f;
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int mo = i * 32 + 8 * (e >> 2) + (e & 3);   // row offset from mrow
                    const int m = mrow + mo;
                    const bool mok = m < g.M;
                    const float wm = (float)(m + g.wbase);
                    const float bm = hb ? bias_s[m - m0] : 0.0f;
#pragma unroll
                    for (int j = 0; j < FP; ++j) {
                        const typename Bt::B b = Bt::make(hb ? acc[i][j][e] + bm : acc[i][j][e]);
                        if (cval[j] && mok) {
                            const float v = Bt::value(b);
                            f1[j] += v;
                            f6[j] = fmaf(wm, v, f6[j]);
                            fq[j] = fmaf(v, v, fq[j]);
                            obase[j][(long long)mo * g.EF] = b;
                        }
                    }
                }
#pragma unroll
                for (int j = 0; j < FP; ++j) {
                    s1[j] += (double)f1[j];
                    s6[j] += (double)f6[j];
                    sq[j] += (double)fq[j];
                }
            } else {
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int mo = i * 32 + 8 * (e >> 2) + (e & 3);   // row offset from mrow
                    const int m = mrow + mo;
                    const bool mok = m < g.M;
                    const double wm = (double)m + wb;
                    const float bm = hb ? bias_s[m - m0] : 0.0f;
#pragma unroll
                    for (int j = 0; j < FP; ++j) {
                        const typename Bt::B b = Bt::make(hb ? acc[i][j][e] + bm : acc[i][j][e]);
                        if (cval[j] && mok) {
                            const double v = (double)Bt::value(b);
                            s1[j] += v;
                            s6[j] = fma(wm, v, s6[j]);
                            sq[j] = fma(v, v, sq[j]);
                            obase[j][(long long)mo * g.EF] = b;
                        }
                    }
                }
            }
        }
#pragma unroll
        for (int j = 0; j < FP; ++j) {
            // rows 4..7 of every 8 sit in the other half-wave: both halves end with the same sums
            const double a1 = s1[j] + __shfl_xor(s1[j], 32, 64);
            const double a6 = s6[j] + __shfl_xor(s6[j], 32, 64);
            const double aq = sq[j] + __shfl_xor(sq[j], 32, 64);
            const int cl = brow0 + j * 32 + l32;
            if (WM == 1) {
                if (h == 0 && cval[j]) {
                    const long long pgo = pcol[j];
                    const long long n = pgo / g.EF;
                    double *dst = ep.part + ((size_t)mt * g.N + n) * 4 * g.EF + (pgo - n * g.EF);
                    dst[0] = a1;
                    dst[g.EF] = a6;
                    dst[2 * (size_t)g.EF] = ((double)n + wb) * a1;
                    dst[3 * (size_t)g.EF] = aq;
                }
            } else if (h == 0) {
                red[(wm * 3 + 0) * C::TP + cl] = a1;
                red[(wm * 3 + 1) * C::TP + cl] = a6;
                red[(wm * 3 + 2) * C::TP + cl] = aq;
            }
        }
        if constexpr (WM > 1) {
            __syncthreads();
            for (int cl = tid; cl < C::TP; cl += C::NT) {
                const long long pgo = p0 + cl;
                if (pgo >= g.P_total) continue;
                double s1 = 0.0, s6 = 0.0, sq = 0.0;
#pragma unroll
                for (int w = 0; w < WM; ++w) {
                    s1 += red[(w * 3 + 0) * C::TP + cl];
                    s6 += red[(w * 3 + 1) * C::TP + cl];
                    sq += red[(w * 3 + 2) * C::TP + cl];
                }
                const long long n = pgo / g.EF;
                double *dst = ep.part + ((size_t)mt * g.N + n) * 4 * g.EF + (pgo - n * g.EF);
                dst[0] = s1;
                dst[g.EF] = s6;
                dst[2 * (size_t)g.EF] = ((double)n + wb) * s1;
                dst[3 * (size_t)g.EF] = sq;
            }
        }
        if constexpr (EPI == 2) {
            // the planted faults of this tile, in list order, on the values as stored: each one
            // rewrites its element of O and moves the tile's partial sums of that pixel by the
            // change it made (one thread, after every store of the tile is done)
            if (planted) {
                __syncthreads();
                if (tid == 0) {
                    for (int f = 0; f < ep.fl.n; ++f) {
                        const ftcnn_fault &q = ep.fl.f[f];
                        const long long pf = (long long)q.n * g.EF + (long long)q.x * g.F + q.y;
                        if (!(q.m >= m0 && q.m < m0 + C::TM && pf >= p0 && pf < p0 + C::TP)) continue;
                        const long long pos = pf - (long long)q.n * g.EF;
                        T *o = O + ((long long)q.n * g.M + q.m) * g.EF + pos;
                        const typename Bt::B b = *o, b2 = fault_apply(b, q);
                        *o = b2;
                        const double v = (double)Bt::value(b), v2 = (double)Bt::value(b2), d = v2 - v;
                        double *dst = ep.part + ((size_t)mt * g.N + q.n) * 4 * g.EF + pos;
                        dst[0] += d;
                        dst[g.EF] += ((double)q.m + wb) * d;
                        dst[2 * (size_t)g.EF] += ((double)q.n + wb) * d;
                        dst[3 * (size_t)g.EF] += v2 * v2 - v * v;
                    }
                }
            }
        }
    }
    if (!skm) break;
    first_iter = false;
    if (dp < sk.dp_waves) {
        ++dp;
    } else {
        sk_it += kn;
        first_seg = false;
    }
    }   // segments
}

// Stream-K workgroups of a tile configuration on the current device: the workgroups that are
// resident at once (the least over the three epilogues, so that the protected kernel and its
// plain twin split K at the same places and store the same bits), at most smax, a multiple of 8.
template <typename Tr, int WM, int WP, int FM, int FP, int WEAVE, bool KVEC, bool NHWC>
int sk_workgroups(int smax) {
    using C = Cfg<Tr, WM, WP, FM, FP, KVEC, (WEAVE >= 3 ? WEAVE - 1 : 0)>;
    static const int per_cu = [] {
        int lo = 1 << 30;
        const void *k[3] = {
            reinterpret_cast<const void *>(conv_kernel<Tr, WM, WP, FM, FP, WEAVE, KVEC, 0, NHWC, false, true>),
            reinterpret_cast<const void *>(conv_kernel<Tr, WM, WP, FM, FP, WEAVE, KVEC, 1, NHWC, false, true>),
            reinterpret_cast<const void *>(conv_kernel<Tr, WM, WP, FM, FP, WEAVE, KVEC, 2, NHWC, false, true>)};
        const void *w[3] = {
            reinterpret_cast<const void *>(conv_kernel<Tr, WM, WP, FM, FP, WEAVE, KVEC, 0, NHWC>),
            reinterpret_cast<const void *>(conv_kernel<Tr, WM, WP, FM, FP, WEAVE, KVEC, 1, NHWC>),
            reinterpret_cast<const void *>(conv_kernel<Tr, WM, WP, FM, FP, WEAVE, KVEC, 2, NHWC>)};
        int whole = 1 << 30;
        size_t spill = 0, spill_whole = 0;
        for (int i = 0; i < 6; ++i) {
            const void *f = i < 3 ? k[i] : w[i - 3];
            if (C::LDS_BYTES > 65536 &&
                hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS_BYTES) != hipSuccess)
                return 0;
            int nb = 0;
            if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, f, C::NT, C::LDS_BYTES) != hipSuccess) return 0;
            hipFuncAttributes fa;
            if (hipFuncGetAttributes(&fa, f) != hipSuccess) return 0;
            if (i < 3) {
                lo = nb < lo ? nb : lo;
                spill = fa.localSizeBytes > spill ? fa.localSizeBytes : spill;
            } else {
                whole = nb < whole ? nb : whole;
                spill_whole = fa.localSizeBytes > spill_whole ? fa.localSizeBytes : spill_whole;
            }
        }
        if (spill > spill_whole) return 0;   // registers spilled to scratch: slower than any balance
        // the stream-K kernels hold more registers; where that costs resident workgroups, the
        // balance they bring does not pay for it
        if (lo < whole) return 0;
        return lo;
    }();
    int dev = 0, cus = 0;
    if (per_cu <= 0 || hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    long long S = (long long)per_cu * cus;
    S = S < smax ? S : smax;
    return (int)(S / 8 * 8);
}

// Stream-K pays (the partial writes and the last workgroup's sums of a split tile) where a plain
// grid of whole tiles would leave its last round of S resident workgroups partly idle, and where
// every workgroup still has a long run of chunks.
inline bool use_stream_k(long long tiles, int S, int nch) {
    if (tiles * nch < 32LL * S) return false;   // under 32 chunks a workgroup
    const long long rounds = (tiles + S - 1) / S;
    return tiles * 100 < rounds * S * 90;       // the whole-tile grid would use < 90 % of its slots
}

// The stream-K workgroups of a layer's channels-last fp32 convolution on the current device, or 0
// for one workgroup per tile.  The bf16 loops run whole tiles: on VGG-19 bf16 the stream-K form of
// the direct-to-LDS 128 x 128 tile was 5-8 % slower where its balance should have helped, and the
// 256 x 256 tile (eight waves, at most 256 registers each) spills in that form.
template <typename Tr, int WM, int WP, int FM, int FP, int WEAVE, bool KVEC, bool NHWC>
int sk_decide(const Geom &g, int smax) {
    using C = Cfg<Tr, WM, WP, FM, FP, KVEC, (WEAVE >= 3 ? WEAVE - 1 : 0)>;
    if constexpr (!(NHWC && WEAVE != 2 && sizeof(typename C::T) == 4)) {
        return 0;
    } else {
        if (smax <= 0 || g.G > 1 || g.C % C::TK != 0) return 0;
        const int nch = g.R * g.S * (g.C / C::TK);
        const long long tiles = ((g.P_total + C::TP - 1) / C::TP) * (long long)((g.M + C::TM - 1) / C::TM);
        const int S = sk_workgroups<Tr, WM, WP, FM, FP, WEAVE, KVEC, NHWC>(smax);
        return S > 0 && use_stream_k(tiles, S, nch) ? S : 0;
    }
}

template <typename Tr, int WM, int WP, int FM, int FP, int WEAVE, bool KVEC, int EPI, bool NHWC, bool GRP = false>
hipError_t launch_one(const Geom &g, const void *D, const void *W, void *O, hipStream_t st, int m_major,
                      const void *zp, const Epi<EPI> &ep, const SkArgs &skin) {
    using C = Cfg<Tr, WM, WP, FM, FP, KVEC, (WEAVE >= 3 ? WEAVE - 1 : 0)>;
    using T = typename C::T;
    static_assert(EPI == 0 || (size_t)WM * 3 * C::TP * sizeof(double) <= C::LDS_BYTES, "epilogue fold fits LDS");
    const int tiles_m = (g.M + C::TM - 1) / C::TM;
    const long long tiles_p = (g.P_total + C::TP - 1) / C::TP;
    const long long total = tiles_p * tiles_m;
    Epi<EPI> e = ep;
    SkArgs sk{nullptr, nullptr, 0, 0, 0};
    if constexpr (NHWC && !GRP && WEAVE != 2) {
        if (skin.S > 0 && skin.part && skin.cnt) {
            const int S = sk_decide<Tr, WM, WP, FM, FP, WEAVE, KVEC, NHWC>(g, skin.S);
            if (S > 0) {
                // whole-tile waves but for the last one to two, whose tiles are shared
                const long long waves = (total + S - 1) / S;
                sk = SkArgs{skin.part, skin.cnt, S, g.R * g.S * (g.C / C::TK), (int)(waves > 2 ? waves - 2 : 0)};
            }
        }
    }
    long long grid = sk.S > 0 ? sk.S : total;
    if constexpr (EPI != 0) {
        if (e.aux_kind == 1) {
            e.enc_vec = g.CHW % kEncVec == 0 && reinterpret_cast<uintptr_t>(D) % (kEncVec * sizeof(T)) == 0;
            const long long per = (long long)C::NT * (e.enc_vec ? kEncVec : 1);
            const long long eb = (g.CHW + per - 1) / per;
            if (eb > 0x7FFFFFFFLL) return hipErrorInvalidValue;
            e.aux_blocks = (int)eb;
        }
        if (e.aux_kind == 2 && e.co_slices > 0 && (size_t)e.co.cc * coc_channel_bytes(g, e.co.ty, e.co.tx) > C::LDS_BYTES)
            return hipErrorInvalidValue;   // the plan sized the CoC window for this tile's LDS
        if (e.aux_kind != 0 && e.aux_blocks > 0) {
            // the encode first (it reads D beside the first tiles); the Co5..Co7 work after the
            // tiles, in the slots their last round leaves (in front of them it held back the first
            // tiles: VGG-19 bf16 v6 197 -> 190 us, VGG-19 fp32 overhead 4.4 -> 3.2 %)
            e.aux_groups = (e.aux_blocks + 7) / 8;
            e.tile_groups = (int)((grid + 7) / 8);
            grid = 8 * (e.aux_groups + (grid + 7) / 8);
        } else {
            e.aux_groups = 0;
        }
    }
    if (grid > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    auto kern = conv_kernel<Tr, WM, WP, FM, FP, WEAVE, KVEC, EPI, NHWC, GRP>;
    if constexpr (C::LDS_BYTES > 65536) {
        static const hipError_t attr = hipFuncSetAttribute(
            reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS_BYTES);
        if (attr != hipSuccess) return attr;
    }
    if constexpr (NHWC && !GRP && WEAVE != 2) {
        if (sk.S > 0) {
            kern = conv_kernel<Tr, WM, WP, FM, FP, WEAVE, KVEC, EPI, NHWC, GRP, true>;
            if constexpr (C::LDS_BYTES > 65536) {
                static const hipError_t attr_sk = hipFuncSetAttribute(
                    reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                    (int)C::LDS_BYTES);
                if (attr_sk != hipSuccess) return attr_sk;
            }
        }
    }
    KernelEvents &ev = kernel_events();
    if (ev.before) {
        const hipError_t r = hipEventRecord(ev.before, st);
        if (r != hipSuccess) return r;
    }
    kern<<<(unsigned)grid, C::NT, C::LDS_BYTES, st>>>(static_cast<const T *>(D),
                                                               static_cast<const T *>(W), static_cast<T *>(O), g,
                                                               tiles_m, (int)total, m_major, zp, e, sk);
    const hipError_t r = hipGetLastError();
    if (r != hipSuccess) return r;
    if (ev.after) {
        const hipError_t r2 = hipEventRecord(ev.after, st);
        if (r2 != hipSuccess) return r2;
    }
    ev.before = ev.after = nullptr;
    return hipSuccess;
}

// One tile configuration, dispatched on the weight alignment and the epilogue.
template <typename Tr, int WM, int WP, int FM, int FP, int WEAVE> struct Tile {
    static constexpr int TM = WM * FM * 32;
    static constexpr int TP = WP * FP * 32;
    static constexpr int TK = Tr::TK;
    static constexpr int WEAVE_KIND = WEAVE;
    static constexpr int NT = Cfg<Tr, WM, WP, FM, FP>::NT;
    static constexpr size_t LDS_BYTES = Cfg<Tr, WM, WP, FM, FP, true, (WEAVE >= 3 ? WEAVE - 1 : 0)>::LDS_BYTES;
    // stream-K workgroups of the channels-last form on the current device (0: whole tiles)
    static int stream_k(const Geom &g, int smax) {
        if constexpr (WEAVE == 2) return 0;
        else return sk_decide<Tr, WM, WP, FM, FP, WEAVE, true, true>(g, smax);
    }
    static constexpr bool SK_FORM = WEAVE != 2 && sizeof(typename Tr::T) == 4;
    // NCHW: D and W as given; NHWC: the channels-last copies Dt and Wt (always aligned, K % VEC == 0)
    template <int EPI>
    static hipError_t run(const Geom &g, const void *D, const void *W, void *O, hipStream_t st, const Epi<EPI> &ep,
                          bool nhwc = false, const void *zp = nullptr, const SkArgs &sk = SkArgs{nullptr, nullptr, 0, 0, 0}) {
        const SkArgs none{nullptr, nullptr, 0, 0};
        if constexpr (WEAVE >= 3) {
            // direct-to-LDS tiles exist for channels-last operands only, with the copy of D right
            // behind the zero page (one buffer descriptor reaches both)
            if (!nhwc || !zp || static_cast<const char *>(zp) + 256 != static_cast<const char *>(D))
                return hipErrorInvalidValue;
            return launch_one<Tr, WM, WP, FM, FP, WEAVE, true, EPI, true>(g, D, W, O, st, 0, zp, ep, sk);
        } else {
            if constexpr (WEAVE != 2) {
                if (nhwc && g.G > 1)   // grouped: the loop that skips other groups' channels
                    return launch_one<Tr, WM, WP, FM, FP, WEAVE, true, EPI, true, true>(g, D, W, O, st, 0, zp, ep,
                                                                                        none);
            }
            if (nhwc) return launch_one<Tr, WM, WP, FM, FP, WEAVE, true, EPI, true>(g, D, W, O, st, 0, zp, ep, sk);
            const bool kvec = g.K % Tr::VEC == 0 && reinterpret_cast<uintptr_t>(W) % 16 == 0;
            if (kvec) return launch_one<Tr, WM, WP, FM, FP, WEAVE, true, EPI, false>(g, D, W, O, st, 0, zp, ep, none);
            return launch_one<Tr, WM, WP, FM, FP, WEAVE, false, EPI, false>(g, D, W, O, st, 0, zp, ep, none);
        }
    }
};

// Tile choice per layer, from sweeps over the workload shapes on MI355X.  The
// filter tile follows M so small-M layers waste no MFMA rows; for larger M the
// biggest tile that still leaves about two workgroups per CU wins.  For bf16
// (eight times the fp32 matrix rate per instruction), channels-last layers with
// 64-channel multiples take direct-to-LDS loads (WEAVE 3): 64 x 128 tiles for
// M <= 64, 256 x 256 tiles (eight waves of 128 x 64) for M >= 256 where there
// are enough of them, 128 x 64 where 128 x 128 tiles would not fill the compute
// units, 128 x 128 elsewhere; the other channels-last layers keep
// two chunks in flight (WEAVE 2), and the rest take 64 x 256, 256 x 256 or
// 128 x 128 tiles with register-staged loads.
long long n_tiles(const Geom &g, int tm, int tp) {
    return ((g.P_total + tp - 1) / tp) * (long long)((g.M + tm - 1) / tm);
}

using F32_M32 = Tile<F32T<16>, 1, 4, 1, 2, true>;
using F32_M64 = Tile<F32T<16>, 2, 2, 1, 2, true>;
using F32_64x256 = Tile<F32T<16>, 1, 4, 2, 2, true>;   // channels-last M <= 64: 64 x 64 a wave
using F32_M96 = Tile<F32T<16>, 1, 4, 3, 1, true>;   // 96 x 128: AlexNet conv1 gets 1513 tiles, 3 full rounds
using F32_128x128 = Tile<F32T<16>, 2, 2, 2, 2, true>;
using F32_128x128_K32 = Tile<F32T<32>, 2, 2, 2, 2, true>;   // 32-deep chunks: half the barriers
using F32_128x64 = Tile<F32T<32>, 2, 2, 2, 1, true>;
using F32_64x64 = Tile<F32T<32>, 2, 2, 1, 1, true>;
using BF16_M32 = Tile<BF16T<32>, 1, 4, 1, 2, 0>;
using BF16_M64 = Tile<BF16T<32>, 1, 4, 2, 2, 2>;
using BF16_128x128_K64 = Tile<BF16T<64>, 2, 2, 2, 2, 2>;
using BF16_256x256 = Tile<BF16T<32>, 2, 2, 4, 4, 2>;
using BF16_DMA_128x128 = Tile<BF16T<64>, 2, 2, 2, 2, 3>;
// four waves of 64 x 32, a 48 KB ring (three workgroups a compute unit): for layers with fewer
// 128 x 128 tiles than compute units (VGG-19 v13-v16 and ResNet-18 layer4, 196 tiles: 63.5 -> 55.5
// us a layer unprotected); where it only adds a partly filled round it is slower (ResNet-18 l3
// 49 -> 62 us, l2 62 -> 65 us)
using BF16_DMA_128x64 = Tile<BF16T<64>, 2, 2, 2, 1, 3>;
// M <= 64: four waves of 64 x 32, a 48 KB ring, three workgroups a compute unit (against 64 x 256
// tiles of four 64 x 64 waves, two a compute unit: ResNet-18 l1 89 -> 79 us, VGG-19 v2 299 -> 287 us
// with the channels-last copy; 64 x 64 tiles of two waves, 64 x 128 of two waves and deeper rings
// were slower)
using BF16_DMA_64x128 = Tile<BF16T<64>, 1, 4, 2, 1, 3>;
// eight waves of 128 x 64 (two a SIMD, accumulators in 128 registers a lane): against four waves
// of 128 x 128 (one a SIMD) 5-8 % faster on VGG-19 bf16 v5-v12, which also beat 128 x 128 tiles
using BF16_DMA_256x256 = Tile<BF16T<64>, 2, 4, 4, 2, 3>;

// Calls f(TileType{}) for the tile this layer uses (nhwc: the launch reads the
// channels-last copies).
template <typename Fn>
auto with_tile(const Geom &g, bool nhwc, Fn &&f) {
    if (g.dtype == FTCNN_F32) {
        if (g.M <= 32) return f(F32_M32{});
        // on channels-last layers a wave of the 64 x 256 tile holds 64 x 64 outputs, as in the
        // 128 x 128 tile (VGG-19 v2 1309 -> 1284 us, Darknet-19 c2 349 -> 334 us protected)
        if (g.M <= 64) return nhwc ? f(F32_64x256{}) : f(F32_M64{});
        if (g.M <= 96) return f(F32_M96{});
        // grouped layers: rows of tiles inside one group, so that every tile skips the other
        // groups' channels (192 filters a group: 64-row tiles)
        if (g.G > 1 && g.Mg % 128 != 0 && g.Mg % 64 == 0) return f(F32_64x64{});
        // dense channels-last layers whose tiles the stream-K schedule shares out evenly (at the two
        // workgroups a compute unit that these tiles keep on 256 compute units) lose nothing to the
        // last round of tiles: there the larger tile is the faster one per output (VGG-19 v5-v9:
        // 128 x 128 3-5 % faster than 128 x 64; v13-v16, Darknet-19 c9-c18 and AlexNet conv5:
        // 128 x 64 6-9 % faster than 64 x 64 or 128 x 128)
        if (nhwc && g.G == 1) {
            auto shared = [&](long long tiles, int tk) {
                return g.C % tk == 0 && use_stream_k(tiles, 2 * kSkComputeUnits, g.R * g.S * (g.C / tk));
            };
            // with 512 or more channels the 32-deep chunks pay (VGG-19 v10-v12 1013 -> 986 us; on
            // v3-v8, 64 to 256 channels, they were up to 2.6 % slower)
            if (n_tiles(g, 128, 128) >= 600 && shared(n_tiles(g, 128, 128), 16))
                return g.C >= 512 ? f(F32_128x128_K32{}) : f(F32_128x128{});
            if (n_tiles(g, 128, 64) >= 256 && shared(n_tiles(g, 128, 64), 32)) return f(F32_128x64{});
        }
        // the tile with the least predicted time: the padded outputs (tiles x TM x TP), plus half of
        // the idle slots in the last round of 256 tiles, at the tile's own rate per output
        // (128 x 128 : 128 x 64 : 64 x 64 = 1 : 0.972 : 0.925).  The one-half and the rates are
        // fitted to VGG-19 (224^2 .. 14^2, batch 32) and Darknet-19 (104^2 .. 13^2, batch 16),
        // where they pick the fastest of the three on every layer or one within 1%; 128 x 128
        // needs at least 600 tiles and 128 x 64 one a compute unit (fewer hide too little latency)
        const auto cost = [](long long tiles, double tile_outputs, double rate) {
            const long long slots = (tiles + 255) / 256 * 256;
            return ((double)tiles + 0.5 * (double)(slots - tiles)) * tile_outputs / rate;
        };
        const long long t128 = n_tiles(g, 128, 128), t12864 = n_tiles(g, 128, 64);
        const double c64 = cost(n_tiles(g, 64, 64), 64.0 * 64.0, 0.925);
        const double c12864 = t12864 >= 256 ? cost(t12864, 128.0 * 64.0, 0.972) : 1e300;
        const double c128 = t128 >= 600 ? cost(t128, 128.0 * 128.0, 1.0) : 1e300;
        if (c128 <= c12864 && c128 <= c64) return f(F32_128x128{});
        if (c12864 <= c64) return f(F32_128x64{});
        return f(F32_64x64{});
    }
    // direct-to-LDS loads reach the operands through 32-bit buffer offsets
    const bool dma = nhwc && g.C % 64 == 0 && (long long)g.M * g.K * 2 < (1LL << 31) &&
                     256 + (long long)g.N * g.CHW * 2 < (1LL << 31);
    if (g.M <= 32) return f(BF16_M32{});
    // M <= 64 with 64-channel multiples: direct-to-LDS 64 x 128 (against register-staged loads,
    // VGG-19 v2 384 -> 308 us and ResNet-18 l1 109 -> 90 us for the convolution alone, before the
    // tile went from 64 x 256 to 64 x 128)
    if (g.M <= 64) return dma ? f(BF16_DMA_64x128{}) : f(BF16_M64{});
    if (dma) {
        // 256 x 256 where M is large and there are enough such tiles
        if (g.M >= 256 && n_tiles(g, 256, 256) >= 192) return f(BF16_DMA_256x256{});
        if (n_tiles(g, 128, 128) < 256) return f(BF16_DMA_128x64{});
        return f(BF16_DMA_128x128{});
    }
    if (g.M >= 256 && n_tiles(g, 256, 256) >= 192) return f(BF16_256x256{});
    return f(BF16_128x128_K64{});
}

}  // namespace

void conv_tile_info(const Geom &g, bool nhwc, int out[6]) {
    with_tile(g, nhwc, [&](auto t) {
        using Tt = decltype(t);
        out[0] = Tt::TM;
        out[1] = Tt::TP;
        out[2] = Tt::TK;
        out[3] = Tt::WEAVE_KIND;
        out[4] = nhwc ? 1 : 0;
        out[5] = (nhwc && g.G > 1 && Tt::WEAVE_KIND != 2 && Tt::WEAVE_KIND != 3) ? 1 : 0;
        return 0;
    });
}

int conv_tile_m(const Geom &g, bool nhwc) {
    return with_tile(g, nhwc, [](auto t) { return decltype(t)::TM; });
}

hipError_t launch_conv(const Plan &pl, const void *D, const void *W, void *O, hipStream_t st, const float *bias) {
    const Epi<0> ep{bias};
    return with_tile(pl.g, false, [&](auto t) { return decltype(t)::run(pl.g, D, W, O, st, ep); });
}

void conv_sk_space(const Geom &g, bool nhwc, int *smax, size_t *part_bytes, long long *counters) {
    *smax = 0;
    *part_bytes = 0;
    *counters = 0;
    if (!nhwc || g.G > 1) return;
    with_tile(g, true, [&](auto t) {
        using Tt = decltype(t);
        if constexpr (Tt::SK_FORM) {
            // room for every workgroup the LDS of kSkComputeUnits compute units could hold
            const int waves = Tt::NT / 64;
            long long per_cu = 160LL * 1024 / (long long)Tt::LDS_BYTES;
            per_cu = per_cu < 32 / waves ? per_cu : 32 / waves;
            *smax = (int)(per_cu * kSkComputeUnits / 8 * 8);
            *part_bytes = (size_t)*smax * 2 * Tt::TM * Tt::TP * sizeof(float);
            *counters = n_tiles(g, Tt::TM, Tt::TP);
        }
        return 0;
    });
}

int conv_stream_k(const Plan &pl) {
    if (!pl.nhwc || pl.sk_smax <= 0) return 0;
    return with_tile(pl.g, true, [&](auto t) { return decltype(t)::stream_k(pl.g, pl.sk_smax); });
}

void conv_tile_shape(const Geom &g, bool nhwc, int *threads, size_t *lds_bytes) {
    with_tile(g, nhwc, [&](auto t) {
        *threads = decltype(t)::NT;
        *lds_bytes = decltype(t)::LDS_BYTES;
        return 0;
    });
}

// The stream-K scratch of the plan (none when the plan has no room for it).
SkArgs sk_args(const Plan &pl, void *ws) {
    if (pl.sk_smax <= 0) return SkArgs{nullptr, nullptr, 0, 0, 0};
    char *w = static_cast<char *>(ws);
    return SkArgs{reinterpret_cast<float *>(w + pl.off_skpart), reinterpret_cast<int *>(w + pl.off_skcnt), pl.sk_smax, 0,
                  0};
}

hipError_t launch_conv_sums(const Plan &pl, const void *D, const void *W, void *O, const ftcnn_checksums *ck,
                            ftcnn_report *rep, int cap, const ftcnn_fault *faults, int nf, void *ws,
                            hipStream_t st, bool cd_given) {
    char *w = static_cast<char *>(ws);
    double *cd1 = ck ? ck->cd1 : nullptr, *cd2 = ck ? ck->cd2 : nullptr;
    const void *Dc = D, *Wc = W;
    const void *zp = pl.nhwc ? w + pl.off_zero : nullptr;   // zeroed by the channels-last copy
    int aux_kind = 0, aux_blocks = 0, co_slices = 0;
    CdSrc src{cd1, cd2, 0, 1};
    if (pl.nhwc) {
        // channels-last copies; the copy of D also encodes Cd1, Cd2 (if asked and not given)
        const hipError_t e = cd_given ? launch_prep(pl, D, W, nullptr, nullptr, ws, st)
                                      : launch_prep(pl, D, W, cd1, cd2, ws, st);
        if (e != hipSuccess) return e;
        Dc = w + pl.off_dt;
        Wc = w + pl.off_wt;
        if (cd1) {
            // given checksums are whole: no image-range partials to combine
            const int ns = cd_given ? 1 : pl.prep_ns;
            if (ns > 1) {
                const double *p1 = reinterpret_cast<const double *>(w + pl.off_encp);
                src = CdSrc{p1, p1 + pl.g.CHW, 2 * pl.g.CHW, ns};
            }
            const bool coc = pl.co_in_conv && ck->cw1 && ck->cw2;
            const int comb = ns > 1 ? pl.co.comb_blocks : 0;
            aux_blocks = comb + (coc ? pl.co.tiles * pl.co.groups * ns : 0);
            aux_kind = aux_blocks > 0 ? 2 : 0;
            co_slices = coc ? pl.co.groups * ns : 0;
        }
    } else if (cd1 && !cd_given) {
        aux_kind = 1;   // encode workgroups; their count follows the tile's threads
    }
    CocTile co = pl.co;
    if (!(pl.nhwc && pl.prep_ns > 1) || cd_given) co.comb_blocks = 0;
    double *part = reinterpret_cast<double *>(w + pl.off_sums);
    double *copart = reinterpret_cast<double *>(w + pl.off_copart);
    const double *cw1 = ck ? ck->cw1 : nullptr, *cw2 = ck ? ck->cw2 : nullptr;
    const float *bias = ck ? ck->bias : nullptr;
    if (nf == 0) {
        Epi<1> ep{part, rep, cap, aux_kind, aux_blocks, 0, 0, cd1, cd2, 0, src, cw1, cw2, copart, co, co_slices, {}, bias};
        return with_tile(pl.g, pl.nhwc,
                         [&](auto t) { return decltype(t)::run(pl.g, Dc, Wc, O, st, ep, pl.nhwc, zp, sk_args(pl, ws)); });
    }
    Epi<2> ep{part, rep, cap, aux_kind, aux_blocks, 0, 0, cd1, cd2, 0, src, cw1, cw2, copart, co, co_slices, {}, bias};
    for (int i = 0; i < nf; ++i) ep.fl.f[i] = faults[i];
    ep.fl.n = nf;
    return with_tile(pl.g, pl.nhwc,
                     [&](auto t) { return decltype(t)::run(pl.g, Dc, Wc, O, st, ep, pl.nhwc, zp, sk_args(pl, ws)); });
}

hipError_t launch_conv_ws(const Plan &pl, const void *D, const void *W, void *O, void *ws, hipStream_t st,
                          const float *bias) {
    if (!pl.nhwc) return launch_conv(pl, D, W, O, st, bias);
    const hipError_t e = launch_prep(pl, D, W, nullptr, nullptr, ws, st);
    if (e != hipSuccess) return e;
    char *w = static_cast<char *>(ws);
    const Epi<0> ep{bias};
    return with_tile(pl.g, true, [&](auto t) {
        return decltype(t)::run(pl.g, w + pl.off_dt, w + pl.off_wt, O, st, ep, true, w + pl.off_zero, sk_args(pl, ws));
    });
}

}  // namespace ftcnn
