// The C ABI of include/ftcnn.h: argument checks, the per-layer launch plan and
// the workspace layout.  All device work is enqueued by the launch_* functions.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

thread_local char g_err[512] = "";
thread_local KernelEvents g_events{nullptr, nullptr};

int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int hip_fail(hipError_t e, const char *where) {
    return fail(FTCNN_E_HIP, "%s: %s", where, hipGetErrorString(e));
}

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

long long ceil_div(long long a, long long b) { return (a + b - 1) / b; }

int clampi(long long v, long long lo, long long hi) { return (int)(v < lo ? lo : (v > hi ? hi : v)); }

// Row splits for a column reduction of [rows][cols]: enough workgroups to fill
// the chip, but every split keeps at least `min_rows` rows.
int row_splits(long long rows, long long col_blocks, long long target_blocks, long long min_rows) {
    const long long want = ceil_div(target_blocks, col_blocks);
    const long long cap = rows / min_rows > 1 ? rows / min_rows : 1;
    return clampi(want, 1, cap);
}

// allow_nhwc = false: every convolution gathers from D as given (no channels-last copies in
// the workspace), a plan with a smaller workspace for layers that would otherwise copy.
int make_plan(const ftcnn_conv_desc *d, Plan *pl, bool allow_nhwc = true, bool allow_sk = true) {
    if (!d) return fail(FTCNN_E_ARG, "null descriptor");
    if (d->groups < 1 || d->ch % d->groups != 0 || d->m % d->groups != 0)
        return fail(FTCNN_E_SHAPE, "groups = %d must divide ch = %d and m = %d", d->groups, d->ch, d->m);
    if (d->dtype != FTCNN_F32 && d->dtype != FTCNN_BF16) return fail(FTCNN_E_DTYPE, "dtype %d", d->dtype);
    if (d->wbase != 0 && d->wbase != 1) return fail(FTCNN_E_ARG, "wbase %d (0 or 1)", d->wbase);
    if (d->n < 1 || d->ch < 1 || d->h < 1 || d->w < 1 || d->m < 1 || d->r < 1 || d->s < 1 ||
        d->stride < 1 || d->pad < 0)
        return fail(FTCNN_E_SHAPE, "non-positive dimension");
    Geom &g = pl->g;
    g.N = d->n; g.C = d->ch; g.H = d->h; g.W = d->w;
    g.M = d->m; g.R = d->r; g.S = d->s; g.U = d->stride; g.P = d->pad;
    const long long hs = (long long)d->h + 2LL * d->pad - d->r, ws = (long long)d->w + 2LL * d->pad - d->s;
    if (hs < 0 || ws < 0) return fail(FTCNN_E_SHAPE, "kernel larger than the padded input");
    g.E = (int)(hs / d->stride + 1);
    g.F = (int)(ws / d->stride + 1);
    const long long K = (long long)d->ch * d->r * d->s;
    const long long EF = (long long)g.E * g.F;
    const long long CHW = (long long)d->ch * d->h * d->w;
    if (K > (1LL << 30) || EF > (1LL << 30) || CHW > (1LL << 30) || d->m > (1 << 20) || d->n > (1 << 20) ||
        (long long)d->n * d->m > (1LL << 30) || (long long)d->n * CHW >= (1LL << 31) ||
        (long long)d->m * K >= (1LL << 31))
        return fail(FTCNN_E_SHAPE, "dimension beyond the supported range");
    // the bf16 epilogue adds the weighted terms (m + wbase) o of a pixel in fp32 runs; they are exact
    // (8-bit significands times weights below 2^16), which bounds the runs' rounding
    if (d->dtype == FTCNN_BF16 && (long long)d->m + d->wbase > (1LL << 16))
        return fail(FTCNN_E_UNSUPPORTED, "bf16 layers take at most 65536 - wbase filters");
    g.K = (int)K;
    g.EF = (int)EF;
    g.CHW = CHW;
    g.P_total = (long long)g.N * EF;
    g.dtype = d->dtype;
    g.wbase = d->wbase;
    g.G = d->groups;
    g.Cg = d->ch / d->groups;
    g.Mg = d->m / d->groups;
    g.Kg = g.Cg * d->r * d->s;

    const int vec = g.dtype == FTCNN_F32 ? 4 : 8;
    // input checksums
    pl->enc_splits_d = row_splits(g.N, ceil_div(ceil_div(CHW, vec), kThreads), 512, 8);
    pl->enc_splits_w = row_splits(g.M, ceil_div(ceil_div(K, vec), kThreads), 512, 8);
    // verification
    const long long cols_v = ceil_div(EF, EF % vec == 0 ? vec : 1);
    const long long ctt = cols_v < kThreads ? cols_v : kThreads;
    pl->ver_cols_per_block = (int)ctt;
    // enough blocks to fill the chip, while the float64 split partials stay a few percent of O
    const long long rows_o = (long long)g.N * g.M;
    const long long o_bytes = rows_o * EF * (g.dtype == FTCNN_F32 ? 4 : 2);
    const long long part_budget = o_bytes / 20 > (4LL << 20) ? o_bytes / 20 : (4LL << 20);
    const long long part_cap = part_budget / (32 * EF);
    pl->ver_splits = row_splits(rows_o, ceil_div(cols_v, ctt), 1024, 32);
    if (pl->ver_splits > part_cap) pl->ver_splits = part_cap > 1 ? (int)part_cap : 1;
    pl->nhwc = allow_nhwc && nhwc_layer(g);
    // summations fused into the convolution epilogue: one slice per (filter tile, image)
    pl->sum_splits = (int)(ceil_div(g.M, conv_tile_m(g, pl->nhwc)) * g.N);
    // correction: the standalone launch hands the flagged positions over from at most corr_blocks
    // workgroups; every path leaves the chain to the wide stage, whose scratch is laid out by
    // corr_layout
    pl->corr_blocks = 256;
    const long long L = g.M > g.N ? g.M : g.N;
    pl->corr_stride = (size_t)((4LL * g.M + 4LL * g.N + 2 * L + 31) / 32 * 32);

    size_t off = 0;
    pl->off_flags = off;
    off += align256(sizeof(int) * (size_t)EF);
    pl->off_enc = off;
    const size_t enc_d = pl->enc_splits_d > 1 ? 2ull * pl->enc_splits_d * CHW * sizeof(double) : 0;
    const size_t enc_w = pl->enc_splits_w > 1 ? 2ull * pl->enc_splits_w * K * sizeof(double) : 0;
    off += align256(enc_d > enc_w ? enc_d : enc_w);
    pl->off_ver = off;
    off += align256(4ull * pl->ver_splits * EF * sizeof(double));
    pl->off_sums = off;
    off += align256(4ull * pl->sum_splits * EF * sizeof(double));
    // channels-last copies of D and W for the vector-gather convolution; the copy of D encodes
    // Cd1, Cd2 too, over image ranges when the layer has few tiles: enough ranges for about 1024
    // workgroups, with at least 16 images (fp32) or 32 (bf16) a range, so that the float64 partial
    // pairs (16 bytes per element of Cd) cost at most a quarter of D's traffic, and at most 16
    const size_t es = g.dtype == FTCNN_F32 ? 4 : 2;
    pl->prep_ns = 1;
    pl->co_in_conv = false;
    pl->co = CocTile{1, 1, 1, 1, 1, 1, 0, 1};
    if (pl->nhwc) {
        const long long tiles = (long long)(g.C / prep_tile_channels(g)) * ceil_div((long long)g.H * g.W, prep_tile_positions(g));
        const int min_imgs = g.dtype == FTCNN_F32 ? 16 : 32;   // a multiple of both image batches
        long long most = g.N / min_imgs;
        most = most > 16 ? 16 : (most < 1 ? 1 : most);
        pl->prep_ns = clampi(ceil_div(1024, tiles), 1, most);
        // Co5..Co7 in extra workgroups of the convolution launch, in its threads and LDS, where
        // they hide behind the matrix-core tiles: on layers with many taps to evaluate (E*F*K of
        // at least 1M; one pass per image range when the input checksums come split) and on
        // every layer whose input checksums are whole.  On the others (small and split) the
        // final launch evaluates the taps itself.
        int nt = 0;
        size_t lds = 0;
        conv_tile_shape(g, true, &nt, &lds);
        CocTile &co = pl->co;
        co.tx = g.F >= 24 ? 32 : (g.F >= 12 ? 16 : 8);
        co.ty = nt / co.tx < g.E ? nt / co.tx : g.E;
        while (co.ty > 1 && coc_channel_bytes(g, co.ty, co.tx) > lds) co.ty /= 2;
        if ((pl->prep_ns == 1 || EF * K >= (1LL << 20)) && coc_channel_bytes(g, co.ty, co.tx) <= lds) {
            pl->co_in_conv = true;
            const size_t cc = lds / coc_channel_bytes(g, co.ty, co.tx);
            co.cc = (int)(cc < 8 ? cc : 8);
            co.tiles_x = (int)ceil_div(g.F, co.tx);
            co.tiles = (int)(ceil_div(g.E, co.ty) * co.tiles_x);
            co.groups = clampi(ceil_div(768, co.tiles), 1, ceil_div(g.C, co.cc));
        }
        co.ns = pl->prep_ns;
        co.comb_blocks = pl->prep_ns > 1 ? (int)ceil_div(CHW, 2LL * nt) : 0;
    }
    // 256 zero bytes for loads that fall outside the operands (written by the copy), directly in
    // front of Dt: the direct-to-LDS loads reach both through one buffer descriptor
    pl->off_zero = off;
    off += pl->nhwc ? 256 : 0;
    pl->off_dt = off;
    off += pl->nhwc ? align256((size_t)g.N * CHW * es) : 0;
    pl->off_wt = off;
    off += pl->nhwc ? align256((size_t)g.M * K * es) : 0;
    pl->off_encp = off;
    off += pl->prep_ns > 1 ? align256(2ull * pl->prep_ns * CHW * sizeof(double)) : 0;
    pl->off_copart = off;
    off += pl->co_in_conv ? align256(3ull * pl->co.groups * pl->prep_ns * EF * sizeof(double)) : 0;
    pl->off_corr = off;
    off += align256(corr_layout(g, pl->corr_stride).bytes);
    pl->off_wchk = off;   // Cw1, Cw2 re-encoded by ftcnn_check_weights
    off += align256(2 * sizeof(double) * (size_t)K);
    pl->off_wfull = off;  // grouped layers: the block-diagonal expansion of W
    off += g.G > 1 ? align256((size_t)g.M * K * es) : 0;
    // the stream-K partials and per-tile counts of the channels-last convolution (the counts are
    // cleared by the channels-last copy that runs before every such convolution)
    pl->sk_smax = 0;
    pl->sk_counters = 0;
    pl->off_skpart = pl->off_skcnt = off;
    if (pl->nhwc && allow_sk) {
        int smax = 0;
        size_t pbytes = 0;
        long long counters = 0;
        conv_sk_space(g, true, &smax, &pbytes, &counters);
        if (smax > 0) {
            pl->sk_smax = smax;
            pl->sk_counters = counters;
            pl->off_skpart = off;
            off += align256(pbytes);
            pl->off_skcnt = off;
            off += align256((size_t)counters * sizeof(int));
        }
    }
    pl->bytes = off;
    return FTCNN_OK;
}

int check_ws(const Plan &pl, const void *ws) {
    if (!ws) return fail(FTCNN_E_WORKSPACE, "null workspace (%zu bytes needed)", pl.bytes);
    if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(FTCNN_E_WORKSPACE, "workspace not 256-byte aligned");
    return FTCNN_OK;
}

#define FT_TRY(expr)                  \
    do {                              \
        const int _rc = (expr);       \
        if (_rc != FTCNN_OK) return _rc; \
    } while (0)

#define FT_HIP(expr, where)                          \
    do {                                             \
        const hipError_t _e = (expr);                \
        if (_e != hipSuccess) return hip_fail(_e, where); \
    } while (0)

// The weights the convolution and the weight encode run on: W itself, or on grouped layers its
// block-diagonal expansion in the workspace (which those layers therefore always need).
int weights_for_conv(const Plan &pl, const void *W, void *ws, hipStream_t st, const void **out) {
    if (pl.g.G > 1) FT_TRY(check_ws(pl, ws));
    hipError_t e;
    *out = dense_weights(pl, W, ws, st, &e);
    FT_HIP(e, "grouped weights");
    return FTCNN_OK;
}


int check_policy(const ftcnn_policy *p) {
    if (!p) return fail(FTCNN_E_ARG, "null policy");
    if (!(p->kappa > 0.0) || !(p->eta >= 0.0 && p->eta < 0.5))
        return fail(FTCNN_E_ARG, "policy needs kappa > 0 and 0 <= eta < 0.5");
    if (p->repair != FTCNN_REPAIR_CHECKSUM && p->repair != FTCNN_REPAIR_RECOMPUTE)
        return fail(FTCNN_E_ARG, "policy repair %d", p->repair);
    return FTCNN_OK;
}

int do_encode(const Plan &pl, int which, const void *X, double *c1, double *c2, void *ws, hipStream_t st) {
    if (which < 0 || which > 2) return fail(FTCNN_E_ARG, "encode which = %d (0 = D, 1 = W, 2 = bias)", which);
    if (!X || !c1 || !c2) return fail(FTCNN_E_ARG, "encode: null pointer");
    if (which == 2) {
        FT_HIP(launch_bias_sums(pl, static_cast<const float *>(X), c1, c2, st), "encode bias");
        return FTCNN_OK;
    }
    const int splits = which == 0 ? pl.enc_splits_d : pl.enc_splits_w;
    if (splits > 1) FT_TRY(check_ws(pl, ws));
    if (which == 1) FT_TRY(weights_for_conv(pl, X, ws, st, &X));   // grouped: Sec. 5.2's Cw1, Cw2
    FT_HIP(launch_encode(pl, which, X, c1, c2, ws, st), "encode");
    return FTCNN_OK;
}

int do_conv(const Plan &pl, const void *D, const void *W, void *O, hipStream_t st) {
    if (!D || !W || !O) return fail(FTCNN_E_ARG, "conv_fwd: null pointer");
    if (pl.g.G > 1)
        return fail(FTCNN_E_UNSUPPORTED, "conv_fwd: grouped layers run through ftcnn_conv_fwd_ws (W is expanded in the workspace)");
    FT_HIP(launch_conv(pl, D, W, O, st), "conv_fwd");
    return FTCNN_OK;
}

int do_cksum(const Plan &pl, uint32_t which, const void *D, const void *W, const ftcnn_checksums *ck,
             hipStream_t st) {
    if (!ck) return fail(FTCNN_E_ARG, "checksum_conv: null checksums");
    if (which & ~0x7Fu) return fail(FTCNN_E_ARG, "checksum_conv: unknown bits 0x%x", which);
    if ((which & (FTCNN_CO5 | FTCNN_CO6)) && !ck->cd1) return fail(FTCNN_E_ARG, "Co5/Co6 need cd1");
    if ((which & (FTCNN_CO5 | FTCNN_CO7)) && !ck->cw1) return fail(FTCNN_E_ARG, "Co5/Co7 need cw1");
    if ((which & FTCNN_CO6) && !ck->cw2) return fail(FTCNN_E_ARG, "Co6 needs cw2");
    if ((which & FTCNN_CO7) && !ck->cd2) return fail(FTCNN_E_ARG, "Co7 needs cd2");
    if ((which & FTCNN_CO7) && !(which & FTCNN_CO5) && !ck->cd1) return fail(FTCNN_E_ARG, "Co7 needs cd1");
    if ((which & FTCNN_CO5) && !ck->co5) return fail(FTCNN_E_ARG, "null co5");
    if ((which & FTCNN_CO6) && !ck->co6) return fail(FTCNN_E_ARG, "null co6");
    if ((which & FTCNN_CO7) && !ck->co7) return fail(FTCNN_E_ARG, "null co7");
    if ((which & (FTCNN_CO1 | FTCNN_CO3)) && (!W || !ck->cd1 || !ck->cd2))
        return fail(FTCNN_E_ARG, "Co1/Co3 need W, cd1 and cd2");
    if ((which & (FTCNN_CO2 | FTCNN_CO4)) && (!D || !ck->cw1 || !ck->cw2))
        return fail(FTCNN_E_ARG, "Co2/Co4 need D, cw1 and cw2");
    if ((which & (FTCNN_CO1 | FTCNN_CO3)) && pl.g.G > 1)
        return fail(FTCNN_E_UNSUPPORTED, "Co1/Co3 of a grouped layer: the correction computes them where flagged");
    if (((which & FTCNN_CO1) && !ck->co1) || ((which & FTCNN_CO3) && !ck->co3) ||
        ((which & FTCNN_CO2) && !ck->co2) || ((which & FTCNN_CO4) && !ck->co4))
        return fail(FTCNN_E_ARG, "checksum_conv: null output array");
    FT_HIP(launch_checksum_conv(pl, which, D, W, *ck, st), "checksum_conv");
    return FTCNN_OK;
}

// A bias takes its precomputed sums (ftcnn_encode, which = 2) into every check.
int check_bias(const ftcnn_checksums *ck) {
    if (ck && ck->bias && !ck->cb) return fail(FTCNN_E_ARG, "a bias needs its sums cb (ftcnn_encode which = 2)");
    return FTCNN_OK;
}

int do_verify(const Plan &pl, const void *O, const ftcnn_checksums *ck, const ftcnn_policy *pol,
              ftcnn_report *rep, int32_t cap, void *ws, hipStream_t st) {
    FT_TRY(check_policy(pol));
    if (!O || !ck || !rep) return fail(FTCNN_E_ARG, "verify: null pointer");
    FT_TRY(check_bias(ck));
    if (!ck->co5 || !ck->so5 || !ck->so6 || !ck->so7 || !ck->q5)
        return fail(FTCNN_E_ARG, "verify needs co5, so5, so6, so7 and q5");
    if (cap < 0) return fail(FTCNN_E_ARG, "negative cap_fixes");
    FT_TRY(check_ws(pl, ws));
    FT_HIP(launch_verify(pl, O, *ck, *pol, rep, cap, ws, st), "verify");
    return FTCNN_OK;
}

int do_verify_correct(const Plan &pl, const void *D, const void *W, void *O, const ftcnn_checksums *ck,
                      const ftcnn_policy *pol, ftcnn_report *rep, int32_t cap, void *ws, hipStream_t st) {
    FT_TRY(check_policy(pol));
    if (!D || !W || !O || !ck || !rep) return fail(FTCNN_E_ARG, "verify_correct: null pointer");
    FT_TRY(check_bias(ck));
    if (!ck->co5 || !ck->so5 || !ck->so6 || !ck->so7 || !ck->q5)
        return fail(FTCNN_E_ARG, "verify needs co5, so5, so6, so7 and q5");
    if (!ck->cd1 || !ck->cd2 || !ck->cw1 || !ck->cw2 || !ck->co6 || !ck->co7)
        return fail(FTCNN_E_ARG, "correct needs cd1, cd2, cw1, cw2, co5, co6 and co7");
    if (cap < 0) return fail(FTCNN_E_ARG, "negative cap_fixes");
    FT_TRY(check_ws(pl, ws));
    FT_HIP(launch_verify_correct(pl, D, W, O, *ck, *pol, rep, cap, ws, st), "verify_correct");
    return FTCNN_OK;
}

int check_faults(const Geom &g, const ftcnn_fault *faults, int nf, const char *who) {
    if (nf > 0 && !faults) return fail(FTCNN_E_ARG, "%s: null fault list", who);
    if (nf < 0 || nf > kMaxFaults) return fail(FTCNN_E_ARG, "%s: %d faults (at most %d)", who, nf, kMaxFaults);
    const int bits = g.dtype == FTCNN_F32 ? 32 : 16;
    for (int i = 0; i < nf; ++i) {
        const ftcnn_fault &f = faults[i];
        if (f.n < 0 || f.n >= g.N || f.m < 0 || f.m >= g.M || f.x < 0 || f.x >= g.E || f.y < 0 || f.y >= g.F)
            return fail(FTCNN_E_ARG, "%s: fault %d out of range", who, i);
        if (f.kind < 0 || f.kind > 2 || (f.kind == 0 && (f.bit < 0 || f.bit >= bits)))
            return fail(FTCNN_E_ARG, "%s: fault %d has kind %d bit %d", who, i, f.kind, f.bit);
    }
    return FTCNN_OK;
}

int do_conv_sums(const Plan &pl, const void *D, const void *W, void *O, const ftcnn_checksums *ck,
                 ftcnn_report *rep, int32_t cap, const ftcnn_fault *faults, int32_t nf, void *ws, hipStream_t st,
                 bool cd_given = false) {
    if (!D || !W || !O || !rep) return fail(FTCNN_E_ARG, "conv_fwd_sums: null pointer");
    if (cd_given && (!ck || !ck->cd1 || !ck->cd2))
        return fail(FTCNN_E_ARG, "conv_fwd_sums_given: ck->cd1 and ck->cd2 hold the given checksums");
    if (cap < 0) return fail(FTCNN_E_ARG, "negative cap_fixes");
    const double *cd1 = ck ? ck->cd1 : nullptr, *cd2 = ck ? ck->cd2 : nullptr;
    if ((cd1 == nullptr) != (cd2 == nullptr)) return fail(FTCNN_E_ARG, "conv_fwd_sums: cd1 and cd2 go together");
    if (ck && ((ck->cw1 == nullptr) != (ck->cw2 == nullptr)))
        return fail(FTCNN_E_ARG, "conv_fwd_sums: cw1 and cw2 go together");
    FT_TRY(check_faults(pl.g, faults, nf, "conv_fwd_sums"));
    FT_TRY(check_ws(pl, ws));
    FT_TRY(weights_for_conv(pl, W, ws, st, &W));
    FT_HIP(launch_conv_sums(pl, D, W, O, ck, rep, cap, faults, nf, ws, st, cd_given), "conv_fwd_sums");
    return FTCNN_OK;
}

int do_verify_correct_sums(const Plan &pl, const void *D, const void *W, void *O, const ftcnn_checksums *ck,
                           const ftcnn_policy *pol, ftcnn_report *rep, uint32_t which, void *ws, hipStream_t st) {
    FT_TRY(check_policy(pol));
    if (!D || !W || !O || !ck || !rep) return fail(FTCNN_E_ARG, "verify_correct_sums: null pointer");
    FT_TRY(check_bias(ck));
    const uint32_t coc = FTCNN_CO5 | FTCNN_CO6 | FTCNN_CO7;
    if (which != 0 && which != coc)
        return fail(FTCNN_E_ARG, "verify_correct_sums: which must be 0 or CO5|CO6|CO7 (0x%x)", which);
    if (!ck->co5 || !ck->so5 || !ck->so6 || !ck->so7 || !ck->q5)
        return fail(FTCNN_E_ARG, "verify needs co5, so5, so6, so7 and q5");
    if (!ck->cd1 || !ck->cd2 || !ck->cw1 || !ck->cw2 || !ck->co6 || !ck->co7)
        return fail(FTCNN_E_ARG, "correct needs cd1, cd2, cw1, cw2, co5, co6 and co7");
    FT_TRY(check_ws(pl, ws));
    FT_HIP(launch_verify_correct_sums(pl, D, W, O, *ck, *pol, rep, which == coc, ws, st), "verify_correct_sums");
    return FTCNN_OK;
}

int do_correct(const Plan &pl, const void *D, const void *W, void *O, const ftcnn_checksums *ck,
               const ftcnn_policy *pol, ftcnn_report *rep, void *ws, hipStream_t st) {
    FT_TRY(check_policy(pol));
    if (!D || !W || !O || !ck || !rep) return fail(FTCNN_E_ARG, "correct: null pointer");
    FT_TRY(check_bias(ck));
    if (!ck->cd1 || !ck->cd2 || !ck->cw1 || !ck->cw2 || !ck->co5 || !ck->co6 || !ck->co7)
        return fail(FTCNN_E_ARG, "correct needs cd1, cd2, cw1, cw2, co5, co6 and co7");
    FT_TRY(check_ws(pl, ws));
    FT_HIP(launch_correct(pl, D, W, O, *ck, *pol, rep, ws, st), "correct");
    return FTCNN_OK;
}

}  // namespace

KernelEvents &kernel_events() { return g_events; }

}  // namespace ftcnn

using namespace ftcnn;

// Arguments of the operations between layers (ftcnn_relu_pool and its encoding form).
int check_link(int32_t dtype, int32_t n, int32_t c, int32_t h, int32_t w, int32_t k, int32_t s, const void *X,
               const void *Y, const char *what) {
    if (dtype != FTCNN_F32 && dtype != FTCNN_BF16) return fail(FTCNN_E_DTYPE, "%s: dtype %d", what, dtype);
    if (n <= 0 || c <= 0 || h <= 0 || w <= 0) return fail(FTCNN_E_SHAPE, "%s: non-positive dimension", what);
    if (!((k == 1 && s == 1) || (k == 2 && s == 2) || (k == 3 && s == 2)))
        return fail(FTCNN_E_UNSUPPORTED, "%s: window %d stride %d (1/1, 2/2 and 3/2 are built)", what, k, s);
    if (h < k || w < k) return fail(FTCNN_E_SHAPE, "%s: %dx%d map smaller than the %dx%d window", what, h, w, k, k);
    if ((long long)n * c * h * w > (1LL << 40)) return fail(FTCNN_E_SHAPE, "%s: tensor too large", what);
    if (!X || !Y) return fail(FTCNN_E_ARG, "%s: null pointer", what);
    if (k > 1) {
        // pooling reads windows of X while writing Y: the two must not overlap
        const long long es = dtype == FTCNN_F32 ? 4 : 2;
        const char *x0 = static_cast<const char *>(X), *y0 = static_cast<const char *>(Y);
        const long long xb = (long long)n * c * h * w * es;
        const long long yb = (long long)n * c * ((h - k) / s + 1) * ((w - k) / s + 1) * es;
        if (x0 < y0 + yb && y0 < x0 + xb) return fail(FTCNN_E_ARG, "%s: X and Y overlap", what);
    }
    return FTCNN_OK;
}

extern "C" {

const char *ftcnn_last_error(void) { return g_err; }

int ftcnn_set_kernel_events(hipEvent_t before, hipEvent_t after) {
    g_events.before = before;
    g_events.after = after;
    return FTCNN_OK;
}

int ftcnn_out_shape(const ftcnn_conv_desc *desc, int32_t *E, int32_t *F) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    if (E) *E = pl.g.E;
    if (F) *F = pl.g.F;
    return FTCNN_OK;
}

size_t ftcnn_workspace_bytes(const ftcnn_conv_desc *desc) {
    Plan pl;
    if (make_plan(desc, &pl) != FTCNN_OK) return 0;
    return pl.bytes;
}

int ftcnn_conv_tile(const ftcnn_conv_desc *desc, int32_t path, int32_t out[6]) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    if (!out) return fail(FTCNN_E_ARG, "conv_tile: null output");
    if (path != 0 && path != 1) return fail(FTCNN_E_ARG, "conv_tile: path %d (0 or 1)", path);
    int o[6];
    conv_tile_info(pl.g, path == 1 && pl.nhwc, o);
    for (int i = 0; i < 6; ++i) out[i] = o[i];
    return FTCNN_OK;
}

int ftcnn_conv_stream_k(const ftcnn_conv_desc *desc, int32_t *workgroups) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    if (!workgroups) return fail(FTCNN_E_ARG, "conv_stream_k: null output");
    *workgroups = conv_stream_k(pl);
    return FTCNN_OK;
}

size_t ftcnn_report_bytes(int32_t cap_fixes) {
    return sizeof(ftcnn_report) + (size_t)(cap_fixes > 0 ? cap_fixes : 0) * sizeof(ftcnn_fix);
}

int ftcnn_encode(const ftcnn_conv_desc *desc, int32_t which, const void *X, double *c1, double *c2,
                 void *workspace, hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    return do_encode(pl, which, X, c1, c2, workspace, stream);
}

int ftcnn_conv_fwd(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O, hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    return do_conv(pl, D, W, O, stream);
}

int ftcnn_checksum_conv(const ftcnn_conv_desc *desc, uint32_t which, const void *D, const void *W,
                        const ftcnn_checksums *ck, hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    return do_cksum(pl, which, D, W, ck, stream);
}

int ftcnn_verify(const ftcnn_conv_desc *desc, const void *O, const ftcnn_checksums *ck,
                 const ftcnn_policy *policy, ftcnn_report *rep, int32_t cap_fixes, void *workspace,
                 hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    return do_verify(pl, O, ck, policy, rep, cap_fixes, workspace, stream);
}

int ftcnn_correct(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                  const ftcnn_checksums *ck, const ftcnn_policy *policy, ftcnn_report *rep,
                  void *workspace, hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    return do_correct(pl, D, W, O, ck, policy, rep, workspace, stream);
}

int ftcnn_protected_conv(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                         const ftcnn_checksums *ck, const ftcnn_policy *policy, ftcnn_report *rep,
                         int32_t cap_fixes, void *workspace, hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    FT_TRY(check_policy(policy));
    if (!ck || !D || !W || !O || !rep) return fail(FTCNN_E_ARG, "protected_conv: null pointer");
    FT_TRY(check_ws(pl, workspace));
    if (!ck->cd1 || !ck->cd2) return fail(FTCNN_E_ARG, "protected_conv needs cd1 and cd2");
    FT_TRY(do_conv_sums(pl, D, W, O, ck, rep, cap_fixes, nullptr, 0, workspace, stream));
    return do_verify_correct_sums(pl, D, W, O, ck, policy, rep, FTCNN_CO5 | FTCNN_CO6 | FTCNN_CO7, workspace,
                                  stream);
}

int ftcnn_protected_conv_noalloc(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                                 const ftcnn_checksums *ck, const ftcnn_policy *policy, ftcnn_report *rep,
                                 int32_t cap_fixes, hipStream_t stream) {
    // the plan of ftcnn_protected_conv when its workspace fits the static scratch, else that plan
    // without the stream-K scratch (whole tiles per workgroup: K split at other places), else the
    // plan without channels-last copies (K summed in (c, r, s) order instead of (r, s, c)); the
    // last two give the same results within the output tolerance
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    if (pl.bytes > kStaticScratchBytes) FT_TRY(make_plan(desc, &pl, true, false));
    if (pl.bytes > kStaticScratchBytes) {
        FT_TRY(make_plan(desc, &pl, false));
        if (pl.bytes > kStaticScratchBytes)
            return fail(FTCNN_E_WORKSPACE, "protected_conv_noalloc: the layer needs %zu bytes of scratch, the "
                        "static scratch holds %zu", pl.bytes, kStaticScratchBytes);
    }
    FT_TRY(check_policy(policy));
    if (!ck || !D || !W || !O || !rep) return fail(FTCNN_E_ARG, "protected_conv_noalloc: null pointer");
    if (!ck->cd1 || !ck->cd2) return fail(FTCNN_E_ARG, "protected_conv_noalloc needs cd1 and cd2");
    int dev = 0;
    if (stream) FT_HIP(hipStreamGetDevice(stream, &dev), "protected_conv_noalloc: stream device");
    else FT_HIP(hipGetDevice(&dev), "protected_conv_noalloc: current device");
    void *ws = nullptr;
    FT_HIP(static_scratch(dev, &ws), "protected_conv_noalloc: static scratch");
    FT_TRY(do_conv_sums(pl, D, W, O, ck, rep, cap_fixes, nullptr, 0, ws, stream));
    return do_verify_correct_sums(pl, D, W, O, ck, policy, rep, FTCNN_CO5 | FTCNN_CO6 | FTCNN_CO7, ws, stream);
}

int ftcnn_check_weights(const ftcnn_conv_desc *desc, const void *W, const double *cw1, int32_t *mismatches,
                        void *workspace, hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    if (!W || !cw1 || !mismatches) return fail(FTCNN_E_ARG, "check_weights: null pointer");
    FT_TRY(check_ws(pl, workspace));
    FT_TRY(weights_for_conv(pl, W, workspace, stream, &W));
    FT_HIP(launch_check_weights(pl, W, cw1, mismatches, workspace, stream), "check_weights");
    return FTCNN_OK;
}

int ftcnn_conv_fwd_bias(const ftcnn_conv_desc *desc, const void *D, const void *W, const float *bias,
                        void *O, void *workspace, hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    if (!D || !W || !O || !bias) return fail(FTCNN_E_ARG, "conv_fwd_bias: null pointer");
    if (workspace) {
        FT_TRY(check_ws(pl, workspace));
        FT_TRY(weights_for_conv(pl, W, workspace, stream, &W));
        FT_HIP(launch_conv_ws(pl, D, W, O, workspace, stream, bias), "conv_fwd_bias");
    } else {
        if (pl.g.G > 1) return fail(FTCNN_E_UNSUPPORTED, "conv_fwd_bias: a grouped layer needs the workspace");
        FT_HIP(launch_conv(pl, D, W, O, stream, bias), "conv_fwd_bias");
    }
    return FTCNN_OK;
}

int ftcnn_conv_fwd_ws(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O, void *workspace,
                      hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    if (!D || !W || !O) return fail(FTCNN_E_ARG, "conv_fwd_ws: null pointer");
    FT_TRY(check_ws(pl, workspace));
    FT_TRY(weights_for_conv(pl, W, workspace, stream, &W));
    FT_HIP(launch_conv_ws(pl, D, W, O, workspace, stream), "conv_fwd_ws");
    return FTCNN_OK;
}

int ftcnn_conv_fwd_sums(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                        const ftcnn_checksums *ck, ftcnn_report *rep, int32_t cap_fixes, const ftcnn_fault *faults,
                        int32_t nf, void *workspace, hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    return do_conv_sums(pl, D, W, O, ck, rep, cap_fixes, faults, nf, workspace, stream);
}

int ftcnn_conv_fwd_sums_given(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                              const ftcnn_checksums *ck, ftcnn_report *rep, int32_t cap_fixes,
                              const ftcnn_fault *faults, int32_t nf, void *workspace, hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    return do_conv_sums(pl, D, W, O, ck, rep, cap_fixes, faults, nf, workspace, stream, true);
}

int ftcnn_verify_correct_sums(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                              const ftcnn_checksums *ck, const ftcnn_policy *policy, ftcnn_report *rep,
                              uint32_t which, void *workspace, hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    return do_verify_correct_sums(pl, D, W, O, ck, policy, rep, which, workspace, stream);
}

int ftcnn_verify_correct(const ftcnn_conv_desc *desc, const void *D, const void *W, void *O,
                         const ftcnn_checksums *ck, const ftcnn_policy *policy, ftcnn_report *rep,
                         int32_t cap_fixes, void *workspace, hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    return do_verify_correct(pl, D, W, O, ck, policy, rep, cap_fixes, workspace, stream);
}

int ftcnn_inject(const ftcnn_conv_desc *desc, void *O, const ftcnn_fault *faults, int32_t nf,
                 hipStream_t stream) {
    Plan pl;
    FT_TRY(make_plan(desc, &pl));
    if (!O) return fail(FTCNN_E_ARG, "inject: null pointer");
    FT_TRY(check_faults(pl.g, faults, nf, "inject"));
    if (nf == 0) return FTCNN_OK;
    FT_HIP(launch_inject(pl, O, faults, nf, stream), "inject");
    return FTCNN_OK;
}

int ftcnn_relu_pool(int32_t dtype, int32_t n, int32_t c, int32_t h, int32_t w, int32_t k, int32_t s, const void *X,
                    void *Y, hipStream_t stream) {
    const int rc = check_link(dtype, n, c, h, w, k, s, X, Y, "relu_pool");
    if (rc != FTCNN_OK) return rc;
    FT_HIP(launch_relu_pool((ftcnn_dtype)dtype, X, Y, n, c, h, w, k, s, stream), "relu_pool");
    return FTCNN_OK;
}

int ftcnn_relu_pool_encode(int32_t dtype, int32_t n, int32_t c, int32_t h, int32_t w, int32_t k, int32_t s,
                           int32_t wbase, const void *X, void *Y, double *cd1, double *cd2, hipStream_t stream) {
    if (!cd1 || !cd2) return fail(FTCNN_E_ARG, "relu_pool_encode: null checksum pointer");
    if (wbase != 0 && wbase != 1) return fail(FTCNN_E_ARG, "relu_pool_encode: wbase must be 0 or 1");
    const int rc = check_link(dtype, n, c, h, w, k, s, X, Y, "relu_pool_encode");
    if (rc != FTCNN_OK) return rc;
    FT_HIP(launch_relu_pool_encode((ftcnn_dtype)dtype, X, Y, n, c, h, w, k, s, wbase, cd1, cd2, stream),
           "relu_pool_encode");
    return FTCNN_OK;
}

}  // extern "C"
