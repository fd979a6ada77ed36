/*
 * ftcnn.h — checksum-protected convolution on AMD MI355X (gfx950).
 *
 * Implements the algorithm-based fault tolerance of FT-CNN (Zhao et al.,
 * "FT-CNN: Algorithm-Based Fault Tolerance for Convolutional Neural
 * Networks", arXiv 2003.12203) for one convolution layer:
 *
 *   encode    input checksums Cd1, Cd2 of D and Cw1, Cw2 of W     (Sec. 3.2)
 *   conv_fwd  the layer itself, O = D (x) W                       (Sec. 2.1, eq. 1)
 *   checksum  output checksums Co1..Co7 as convolutions of        (Sec. 3.2)
 *   _conv     checksum blocks
 *   verify    CoC-D detection: So5 = sum_{n,m} O_nm against Co5    (Sec. 3.6, Sec. 4.3)
 *   correct   the correction chain CoC -> RC -> ClC -> FC          (Sec. 3.3-3.6, 4.1, 4.3)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every tensor pointer is a DEVICE pointer owned by the caller.  The
 *   library never allocates, frees or retains device memory; scratch comes
 *   from a caller-supplied workspace of ftcnn_workspace_bytes() bytes
 *   (256-byte aligned).
 * - Layouts are dense row-major: D [n][ch][h][w], W [m][ch/groups][r][s]
 *   (W [m][ch][r][s] when groups = 1), O [n][m][E][F] with
 *   E = floor((h + 2*pad - r)/stride) + 1 and
 *   F = floor((w + 2*pad - s)/stride) + 1.  D, W and O share the dtype of the
 *   descriptor (fp32, or bf16 as raw 16-bit patterns); accumulation is fp32 in
 *   the convolution and fp64 everywhere on the checksum side, except that a
 *   bf16 layer's convolution epilogue adds each run of 16 filters of a pixel in
 *   fp32 (every term exact; at most 15 roundings of 2^-24 a run) before fp64.
 * - Checksum arrays are float64: Cd1, Cd2 [ch][h][w]; Cw1, Cw2 [ch][r][s];
 *   Co5, Co6, Co7, So5, So6, So7, Q5 [E][F]; Co1, Co3 [m][E][F];
 *   Co2, Co4 [n][E][F].
 * - Block index weights: Cd2 = sum_n (n + wbase) D_n, Cw2 = sum_m (m + wbase) W_m,
 *   and the weighted summations use the same weights.  wbase = 0 is the
 *   paper's definition (Sec. 3.2).
 * - Calls taking a stream are asynchronous on it and never synchronize it.
 *   The shape and size queries are host-only.
 * - Return value: FTCNN_OK (0) or a negative FTCNN_E_* code; on error the
 *   stream receives no work and ftcnn_last_error() describes the failure.
 *   A detected soft error is NOT an error: it is reported in ftcnn_report.
 * - Functions are thread-safe for distinct streams and distinct buffers.
 *   Calls sharing a workspace or report must be ordered on one stream.
 */
#ifndef FTCNN_H
#define FTCNN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    FTCNN_OK = 0,
    FTCNN_E_ARG = -1,          /* null pointer or inconsistent argument          */
    FTCNN_E_SHAPE = -2,        /* non-positive or oversized dimension            */
    FTCNN_E_DTYPE = -3,        /* dtype not FTCNN_F32 / FTCNN_BF16               */
    FTCNN_E_WORKSPACE = -4,    /* workspace missing or misaligned                */
    FTCNN_E_HIP = -5,          /* kernel launch failed                           */
    FTCNN_E_UNSUPPORTED = -6   /* a combination that is not built, e.g. a grouped
                                  layer without a workspace, a pooling window
                                  other than 1/1, 2/2 and 3/2                     */
};

typedef enum { FTCNN_F32 = 0, FTCNN_BF16 = 1 } ftcnn_dtype;

/* One convolution layer (notation of Sec. 2.1, Table 1: N, Ch, H, M, R, U). */
typedef struct {
    int32_t n, ch, h, w;     /* D [n][ch][h][w]                                  */
    int32_t m, r, s;         /* W [m][ch/groups][r][s]                           */
    int32_t stride, pad;     /* U of eq. (1); zero padding on every side         */
    int32_t groups;          /* G >= 1 dividing ch and m (Sec. 5.2): filter m
                                sees channels [(m / (m_total/G)) * ch/G, + ch/G).
                                G > 1 needs the workspace in every call that
                                reads W (the convolution runs on the
                                block-diagonal expansion of W kept there):
                                ftcnn_conv_fwd and Co1/Co3 of
                                ftcnn_checksum_conv return FTCNN_E_UNSUPPORTED */
    int32_t dtype;           /* ftcnn_dtype of D, W and O                        */
    int32_t wbase;           /* block index weight offset, 0 or 1                */
} ftcnn_conv_desc;

/* Device pointers to the float64 checksum arrays of one layer (Sec. 3.2).
 * A call reads or writes only the members its description names; the others
 * may be NULL.  The struct itself lives in host memory. */
typedef struct {
    double *cd1, *cd2;              /* [ch][h][w]   input checksums of D   */
    double *cw1, *cw2;              /* [ch][r][s]   input checksums of W   */
    double *co5, *co6, *co7;        /* [E][F]       checksum of checksums  */
    double *so5, *so6, *so7, *q5;   /* [E][F]       summations of O, and sqrt(sum O^2) */
    double *co1, *co3;              /* [m][E][F]    row checksums          */
    double *co2, *co4;              /* [n][E][F]    column checksums       */
    /* Optional bias (Sec. 5.1): bias[m] (fp32, for either layer dtype) is added to every
     * element of O[n][m] by the calls that compute O with the checksums (ftcnn_conv_fwd_sums,
     * ftcnn_protected_conv); cb = {sum_m bias[m], sum_m (m + wbase) bias[m]}, from
     * ftcnn_encode(which = 2), once per layer.  The checksums Co1..Co7 stay those of the
     * convolution; every detection and correction call given a non-NULL bias subtracts the
     * bias share of Table 5 from each summation before comparing it (N bias[m] from So1[m],
     * (sum_n (n + wbase)) bias[m] from So3[m], cb[0] from So2[n], cb[1] from So4[n],
     * N cb[0] from So5, N cb[1] from So6, (sum_n (n + wbase)) cb[0] from So7), and a
     * recomputed element includes its bias.  NULL bias: no bias (cb unused). */
    const float *bias;              /* [m]                                  */
    double *cb;                     /* [2]                                  */
} ftcnn_checksums;

/* Correction schemes, as recorded per repaired element and per position. */
enum {
    FTCNN_SCHEME_NONE = 0,
    FTCNN_SCHEME_COC = 1,          /* checksum-of-checksum, Sec. 3.6          */
    FTCNN_SCHEME_RC = 2,           /* row checksum, Sec. 3.4                  */
    FTCNN_SCHEME_CLC = 3,          /* column checksum, Sec. 3.5               */
    FTCNN_SCHEME_FC = 4,           /* full checksum, Sec. 3.3 and Sec. 4.1.5  */
    FTCNN_SCHEME_CKSUM = 5,        /* the checksums were corrupt, Sec. 4.1.4  */
    FTCNN_SCHEME_UNRESOLVED = 6    /* left for recomputation, Sec. 4.1.1      */
};

enum {
    FTCNN_STATUS_CLEAN = 0,            /* nothing detected                        */
    FTCNN_STATUS_CORRECTED = 1,        /* every flagged position resolved         */
    FTCNN_STATUS_NEEDS_RECOMPUTE = 2,  /* some position unresolved: rerun the layer */
    FTCNN_STATUS_RECOMPUTED = 3,       /* set by a caller that reran and re-verified */
    FTCNN_STATUS_FAILED = 4            /* set by a caller whose rerun still mismatches */
};

typedef struct { int32_t n, m, x, y, scheme; } ftcnn_fix;

/* Detection and correction report, in device memory (updated with device
 * atomics).  ftcnn_verify() resets it; ftcnn_correct() fills in the repairs.
 * fixes[] is in no particular order; n_fixes counts every repair even past
 * cap_fixes. */
typedef struct {
    int32_t detected;          /* CoC-D verdict for the layer                     */
    int32_t n_flagged;         /* positions p with Co5 - So5 beyond tolerance     */
    int32_t status;            /* FTCNN_STATUS_*                                  */
    int32_t resolved_by[7];    /* positions per FTCNN_SCHEME_*                    */
    int32_t n_fixes;
    int32_t cap_fixes;
    int32_t reserved[2];       /* internal to the library (zeroed with the report)  */
    ftcnn_fix fixes[];
} ftcnn_report;

/* Tolerance and workflow policy.  A checksum difference d at one element is
 * bad when it is non-finite or |d| > kappa * (2^-24 sqrt(ch*r*s) + u_out) * Q,
 * Q being the root sum of squares of the weighted terms of the summation and
 * u_out = 0 (fp32) or 2^-8 (bf16).  A located index is legal when its ratio is
 * within eta of an integer inside the index range.  rc_on / clc_on enable the
 * RC and ClC stages per layer (Sec. 4.3). */
enum { FTCNN_REPAIR_CHECKSUM = 0, FTCNN_REPAIR_RECOMPUTE = 1 };
typedef struct {
    int32_t rc_on, clc_on;
    int32_t repair;            /* FTCNN_REPAIR_*: exclusive checksum sum, or eq. (1) again */
    int32_t reserved;
    double kappa, eta;         /* defaults 16 and 0.1                             */
} ftcnn_policy;

/* A fault planted for testing (the paper's source-level injection, Sec. 6.1)
 * at output element (n, m, x, y): kind 0 flips bit `bit` of the stored fp32 or
 * bf16 pattern, kind 1 adds `value`, kind 2 stores `value` (both rounded to
 * the dtype). */
typedef struct { int32_t n, m, x, y, kind, bit; double value; } ftcnn_fault;

/* ---- host-only queries -------------------------------------------------- */

/* E and F of eq. (1) with zero padding.  Returns FTCNN_E_SHAPE when either is < 1. */
int ftcnn_out_shape(const ftcnn_conv_desc *desc, int32_t *E, int32_t *F);

/* Bytes of workspace every call on this layer may use (0 on a bad descriptor). */
size_t ftcnn_workspace_bytes(const ftcnn_conv_desc *desc);

/* Bytes of an ftcnn_report holding cap_fixes repairs. */
size_t ftcnn_report_bytes(int32_t cap_fixes);

/* Description of the last error on the calling thread ("" if none). */
const char *ftcnn_last_error(void);

/* INSTRUMENTATION (host-only, no device work; not an operation of the paper): the
 * convolution kernel this layer's calls launch.  path 0: ftcnn_conv_fwd and
 * ftcnn_conv_fwd_bias without a workspace (D and W read as given); path 1: every call
 * that takes a workspace (ftcnn_conv_fwd_ws, ftcnn_conv_fwd_sums, ftcnn_protected_conv,
 * ...).  out[0] = filters (rows of W) per workgroup tile, out[1] = output pixels per tile,
 * out[2] = k per LDS chunk, out[3] = main loop (0 register-staged gather, 1 gather woven
 * between the matrix-core instructions, 2 two chunks in flight, 3 direct-to-LDS loads),
 * out[4] = 1 when the convolution reads channels-last copies, out[5] = 1 when its tiles
 * skip the channels of other groups (grouped layers).  Lets a test check that it covers
 * every kernel a set of layers runs. */
int ftcnn_conv_tile(const ftcnn_conv_desc *desc, int32_t path, int32_t out[6]);

/* INSTRUMENTATION (host query of the current device, no device work): *workgroups = the
 * stream-K workgroups of the convolution launched by the calls that take a workspace (path 1
 * of ftcnn_conv_tile), or 0 when it runs one workgroup per output tile.  Stream-K is a
 * schedule, not another operation: every workgroup takes an equal run of the layer's
 * (tile, chunk of K) pairs, and a tile whose chunks span several workgroups is summed by the
 * last of them to finish, in chunk order (so the protected convolution and its unprotected
 * twin store the same bits).  It is used for dense channels-last fp32 layers whose tile count
 * would leave the last round of resident workgroups less than 90 % busy. */
int ftcnn_conv_stream_k(const ftcnn_conv_desc *desc, int32_t *workgroups);

/* ---- device work -------------------------------------------------------- */

/* Sec. 3.2 input checksums.  which = 0: X is D, c1 = Cd1 = sum_n D_n and
 * c2 = Cd2 = sum_n (n + wbase) D_n, each [ch][h][w].  which = 1: X is W,
 * c1 = Cw1, c2 = Cw2, each [ch][r][s] (computed once per layer, before the
 * application, Sec. 4.2).  which = 2: X is a bias (float [m]), c1 = sum_m bias[m]
 * and c2 = sum_m (m + wbase) bias[m], one double each (the precomputed bias sums
 * of Sec. 5.1).  float64 accumulation; deterministic. */
int ftcnn_encode(const ftcnn_conv_desc *desc, int32_t which, const void *X,
                 double *c1, double *c2, void *workspace, hipStream_t stream);

/* Weights in memory (Sec. 4.1.2): a soft error in W shows as a difference between Cw1
 * re-encoded from the current W and cw1 encoded before the application (ftcnn_encode,
 * which = 1); the remedy is to reload W.  The re-encode runs the same deterministic kernels,
 * so intact weights reproduce cw1 bit for bit and the comparison is exact.  *mismatches
 * (device int32) receives the number of columns (c, r, s) whose sums differ: 0 when W is
 * intact.  Uses the workspace. */
int ftcnn_check_weights(const ftcnn_conv_desc *desc, const void *W, const double *cw1, int32_t *mismatches,
                        void *workspace, hipStream_t stream);

/* Eq. (1) without bias, with zero padding: O[n][m][x][y] = sum_{k,i,j}
 * D[n][k][Ux+i-P][Uy+j-P] W[m][k][i][j].  Implicit GEMM on the matrix cores,
 * fp32 accumulation, O rounded to the layer dtype (nearest even). */
int ftcnn_conv_fwd(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                   hipStream_t stream);

/* Eq. (1) plus a bias (Sec. 5.1): O[n][m][x][y] = (eq. (1)) + bias[m], added to the fp32
 * accumulator before O is rounded to the layer dtype.  bias: device, fp32 [m].  With a
 * workspace (ftcnn_workspace_bytes) the convolution runs through the kernels of the
 * protected path (channels-last copies on layers whose ch is a multiple of 32), so O is
 * bitwise that of ftcnn_conv_fwd_sums with the same bias; with NULL, through those of
 * ftcnn_conv_fwd. */
int ftcnn_conv_fwd_bias(const ftcnn_conv_desc *desc, const void *D, const void *W, const float *bias,
                        void *O, void *workspace, hipStream_t stream);

/* Output checksums of Sec. 3.2, as convolutions of checksum blocks, float64:
 *   FTCNN_CO1 | FTCNN_CO3: Co1 = Cd1 (x) W, Co3 = Cd2 (x) W   (reads cd1/cd2, W)
 *   FTCNN_CO2 | FTCNN_CO4: Co2 = D (x) Cw1, Co4 = D (x) Cw2   (reads D, cw1/cw2)
 *   FTCNN_CO5..7:          Co5 = Cd1 (x) Cw1, Co6 = Cd1 (x) Cw2, Co7 = Cd2 (x) Cw1
 * CoC-D needs only Co5; the correction chain computes what else it needs at
 * the flagged positions by itself, so the full Co1..Co4 arrays are optional. */
enum { FTCNN_CO1 = 1u << 0, FTCNN_CO2 = 1u << 1, FTCNN_CO3 = 1u << 2, FTCNN_CO4 = 1u << 3,
       FTCNN_CO5 = 1u << 4, FTCNN_CO6 = 1u << 5, FTCNN_CO7 = 1u << 6 };
int ftcnn_checksum_conv(const ftcnn_conv_desc *desc, uint32_t which, const void *D,
                        const void *W, const ftcnn_checksums *ck, hipStream_t stream);

/* CoC-D detection (Sec. 3.6, Sec. 4.3).  Reads O and ck->co5; writes
 * ck->so5, so6, so7, q5 and a per-position flag map into the workspace;
 * resets *rep (cap_fixes recorded) and sets rep->detected and rep->n_flagged. */
int ftcnn_verify(const ftcnn_conv_desc *desc, const void *O, const ftcnn_checksums *ck,
                 const ftcnn_policy *policy, ftcnn_report *rep, int32_t cap_fixes,
                 void *workspace, hipStream_t stream);

/* Correction module (Sec. 4.3): two device-gated launches that do nothing
 * unless rep->detected.  Every flagged position runs CoC, then RC and ClC if
 * enabled, then FC (with the fallbacks of Sec. 4.1.5), each scheme undone
 * unless Co5..Co7 agree with the re-summed output afterwards.  Repairs O in
 * place.  Positions where a weighted checksum agrees while Co5 does not are
 * re-checked against checksums re-encoded from D and W (Sec. 4.1.4).  The first
 * launch hands the flagged positions over; the second computes the row and
 * column checksums Co1..Co4 and the per-filter and per-image summations at
 * them over the whole device, and its last workgroup takes every decision.
 * Reads D, W, ck->cd1/cd2/cw1/cw2/co5/co6/co7, ck->so5/so6/so7/q5 when set (as
 * ftcnn_verify leaves them) and the verify flag map in the workspace.  Leaves
 * status NEEDS_RECOMPUTE if any position is unresolved; the caller then reruns
 * ftcnn_conv_fwd and ftcnn_verify (Sec. 4.1.1). */
int ftcnn_correct(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                  const ftcnn_checksums *ck, const ftcnn_policy *policy, ftcnn_report *rep,
                  void *workspace, hipStream_t stream);

/* ftcnn_verify and ftcnn_correct in two launches: the final detection stage
 * hands every position it flags to the correction's second launch, which does
 * nothing when none was flagged, so a clean layer pays one empty launch for the
 * correction module.  Same inputs, outputs and report as the two calls in
 * sequence. */
int ftcnn_verify_correct(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                         const ftcnn_checksums *ck, const ftcnn_policy *policy, ftcnn_report *rep,
                         int32_t cap_fixes, void *workspace, hipStream_t stream);

/* Eq. (1) as ftcnn_conv_fwd, through the path the protected calls below use:
 * for layers with ch a multiple of 32, D and W are first copied channels-last
 * into the workspace (D as [n][h][w][ch], W as [m][r][s][ch]) so that the
 * convolution gathers 16-byte runs; K is then summed in (r, s, ch) order, so
 * O may differ from ftcnn_conv_fwd's in the last bits (both are eq. (1) with
 * fp32 accumulation).  O is bitwise that of ftcnn_conv_fwd_sums.  Other layers
 * take ftcnn_conv_fwd's kernel.  Needs the workspace of ftcnn_workspace_bytes. */
int ftcnn_conv_fwd_ws(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                      void *workspace, hipStream_t stream);

/* Eq. (1) as ftcnn_conv_fwd_ws (same kernels, bitwise the same O), with the
 * CoC-D summations of Sec. 3.6 computed in the epilogue from the values as
 * stored: every workgroup tile writes, for each of its output pixels, the
 * partial So5, So6, So7 and sum of squares over its filters into the
 * workspace, so detection never re-reads O.  Also resets *rep (cap_fixes
 * recorded).  Follow it with ftcnn_verify_correct_sums on the same workspace
 * and report.
 * ck: may be NULL.  When ck->cd1 and ck->cd2 are set, Cd1 and Cd2 are encoded
 * from D as ftcnn_encode(which = 0) does (Sec. 3.2): by the channels-last copy
 * of D as it moves the values, or by extra workgroups beside the matrix-core
 * tiles.  When ck->cw1 and ck->cw2 (the encoded W) are set as well, layers
 * with ch a multiple of 32 also compute the products Co5, Co6, Co7 of Sec. 3.2
 * in extra workgroups of the convolution launch, as per-channel-range partials
 * in the workspace that ftcnn_verify_correct_sums(which = CO5|CO6|CO7) adds up.
 * Other members are not used.
 * faults / nf: TEST ONLY, NULL / 0 otherwise.  A HOST array of at most 64
 * faults planted in the output values before they are summed and stored, as
 * a fault of the convolution's own arithmetic would appear (Sec. 6.1).
 * Checks every fault as ftcnn_inject does. */
int ftcnn_conv_fwd_sums(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                        const ftcnn_checksums *ck, ftcnn_report *rep, int32_t cap_fixes,
                        const ftcnn_fault *faults, int32_t nf, void *workspace, hipStream_t stream);

/* ftcnn_conv_fwd_sums for a layer whose input checksums are already encoded:
 * ck->cd1 and ck->cd2 (required) hold Cd1, Cd2 of D as inputs, for instance from
 * ftcnn_relu_pool_encode of the layer before (Sec. 3.2), and are not written.  The
 * channels-last copy of D then only copies, and no encode or combine workgroups run;
 * everything else is as ftcnn_conv_fwd_sums (same O, same sums, Co5..Co7 partials when
 * ck->cw1 and ck->cw2 are set).  Follow it with ftcnn_verify_correct_sums. */
int ftcnn_conv_fwd_sums_given(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                              const ftcnn_checksums *ck, ftcnn_report *rep, int32_t cap_fixes,
                              const ftcnn_fault *faults, int32_t nf, void *workspace, hipStream_t stream);

/* ftcnn_verify_correct over the partial sums that ftcnn_conv_fwd_sums left in
 * the workspace (one launch; O is read only at flagged positions).  The
 * report must be the one ftcnn_conv_fwd_sums reset.  which = 0: Co5..Co7 are
 * read from ck (ftcnn_checksum_conv ran before); which = FTCNN_CO5 |
 * FTCNN_CO6 | FTCNN_CO7: the same launch produces them at every position
 * first, adding the partial products ftcnn_conv_fwd_sums computed (when it
 * did) or else evaluating them from ck->cd1, cd2, cw1, cw2, and stores them in
 * ck->co5, co6, co7.  Writes ck->so5, so6, so7, q5 and the flag map; same
 * decisions and repairs as ftcnn_verify_correct. */
int ftcnn_verify_correct_sums(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                              const ftcnn_checksums *ck, const ftcnn_policy *policy, ftcnn_report *rep,
                              uint32_t which, void *workspace, hipStream_t stream);

/* The whole path of one protected layer on one stream:
 * conv_fwd_sums (with the encode of Cd1, Cd2, and Co5..Co7 on channels-last
 * layers) -> verify_correct_sums (with Co5..Co7): two launches, three for
 * channels-last layers.  ck->cw1/cw2 must hold the encoded W (ftcnn_encode with
 * which = 1); ck->cd1, cd2, co5..co7, so5..so7 and q5 are written. */
int ftcnn_protected_conv(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                         const ftcnn_checksums *ck, const ftcnn_policy *policy,
                         ftcnn_report *rep, int32_t cap_fixes, void *workspace,
                         hipStream_t stream);

/* ftcnn_protected_conv for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the same two or three
 * launches with no workspace argument.  Scratch comes from a static device array of the
 * library, 128 MiB on each device, which that device holds from the first call there until
 * the process ends; nothing is allocated or freed by the call.  The call uses the plan of
 * ftcnn_protected_conv when that plan's workspace (ftcnn_workspace_bytes) fits the array, and
 * otherwise the plan without channels-last copies, whose convolution gathers from D as given
 * (the same results within the output tolerance; K summed in (ch, r, s) order); a layer that
 * needs more than 128 MiB even then is rejected with FTCNN_E_WORKSPACE before any launch.
 * The device is the stream's (the current device for the NULL stream).  Every call on one
 * device shares that device's array and leaves its contents behind; calls whose work overlaps
 * on one device (other streams, other threads) race on it and must be ordered by the caller.
 * Arguments, outputs and report as ftcnn_protected_conv. */
int ftcnn_protected_conv_noalloc(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                                 const ftcnn_checksums *ck, const ftcnn_policy *policy,
                                 ftcnn_report *rep, int32_t cap_fixes, hipStream_t stream);

/* INSTRUMENTATION (measurement, not an operation of the paper): the next call
 * on the calling thread that launches the convolution kernel (ftcnn_conv_fwd,
 * ftcnn_conv_fwd_ws, ftcnn_conv_fwd_sums, ftcnn_protected_conv) records
 * `before` on its stream immediately before that launch and `after`
 * immediately after it, so that their elapsed time is the kernel's alone (the
 * channels-last copy and the other launches of the call fall outside); the
 * hook is then cleared.  Either may be NULL.  The events must be created by
 * the caller (with timing enabled) on the device of that stream. */
int ftcnn_set_kernel_events(hipEvent_t before, hipEvent_t after);

/* Between two protected layers of a network (AlexNet, VGG-19 and Darknet-19 in
 * Sec. 6): Y = k x k / s max pooling (no padding) of relu(X), relu(v) = v > 0 ? v : +0
 * (NaN and both zeros give +0).  X [n][c][h][w] and Y [n][c][(h-k)/s+1][(w-k)/s+1]
 * are device tensors of the dtype (FTCNN_F32 or FTCNN_BF16); every output is an input
 * value or +0, so the result is exact.  (k, s) is (1, 1) (ReLU only; X == Y allowed),
 * (2, 2) or (3, 2) (X and Y must not overlap), else FTCNN_E_UNSUPPORTED.  The next
 * layer then encodes its Cd1, Cd2 from Y, the corrected output of this layer after
 * these operations. */
int ftcnn_relu_pool(int32_t dtype, int32_t n, int32_t c, int32_t h, int32_t w, int32_t k, int32_t s,
                    const void *X, void *Y, hipStream_t stream);

/* ftcnn_relu_pool, and with it the input checksums of the layer that reads Y
 * (Sec. 3.2): cd1[c][i][j] = sum_n Y[n][c][i][j] and cd2[c][i][j] = sum_n (n + wbase)
 * Y[n][c][i][j], float64 device arrays of c * ((h-k)/s+1) * ((w-k)/s+1) elements, the
 * images added in order.  Y is the corrected output of one layer after the operations
 * between layers, so the next layer's checksums come from the values it will read, in the
 * pass that writes them; pass them to that layer's ftcnn_conv_fwd_sums_given.  wbase is
 * 0 or 1 (the next layer's descriptor's). */
int ftcnn_relu_pool_encode(int32_t dtype, int32_t n, int32_t c, int32_t h, int32_t w, int32_t k, int32_t s,
                           int32_t wbase, const void *X, void *Y, double *cd1, double *cd2,
                           hipStream_t stream);

/* TEST ONLY: corrupt stored outputs, reproducing the paper's source-level
 * fault injection (Sec. 6.1).  faults is a HOST array of at most 64 entries
 * (ftcnn_fault above), applied in order.  Positions must be in range. */
int ftcnn_inject(const ftcnn_conv_desc *desc, void *O, const ftcnn_fault *faults, int32_t nf,
                 hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* FTCNN_H */
