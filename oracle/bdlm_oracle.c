/*
 * bdlm_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 CPU reference for the block-restricted bidirectional
 * Mamba scan of BDLM Mamba-H ("Training Hybrid Block Diffusion Language Models
 * with Partial Bidirectionality").  Only the test suite, the smoke check and
 * the benchmark's CPU-baseline leg may load this library.  It shares no
 * source, header, table or helper with the HIP library; the product path never
 * calls it.
 *
 * What is computed, and where the paper defines it:
 *   - selective state-space update  s_i = A_i s_{i-1} + B_i x_i,
 *     y_i = C_i s_i + D x_i                        (Sec. 3, Eq. mamba-scan-background)
 *     read in the Mamba-2 form the paper's mixers use (App. C): per head a
 *     scalar A_h, token decay a_t = exp(dt_t * A_h), input B_t scaled by dt_t.
 *   - forward boundary state s_k = F_fwd(clean prefix)   (Sec. 4, Eq. boundary-state)
 *   - active block: forward scan continued from s_k, reverse scan of the
 *     reversed block from a zero state, outputs summed    (Sec. 4, Eq. partial-reverse)
 *   - block finalisation appends the clean block's forward state to the
 *     cache                                               (Sec. 3 BDLM cache; Sec. 4.1)
 *   - full-window bidirectional scan (DiffuMamba-style contrast: forward and
 *     reverse over the whole window, both from zero)      (Sec. 4, Sec. 5.1)
 *   - the convolution part of the Mamba boundary state: a width-4 depthwise
 *     causal convolution with SiLU over the x, B, C channels (App. C: Mamba
 *     convolution width 4), continued from the cached last three input rows in
 *     the forward branch and zero-padded inside the block in the reverse branch
 *     (Sec. 2 and Sec. 4, Eq. partial-reverse: the cached boundary state carries
 *     the convolution rows as well as the SSM state, and the right-to-left scan
 *     never reads tokens outside the block being denoised)
 *   - the gated RMS normalisation that follows the scan in a Mamba-2 mixer
 *     (App. C: the paper's Mamba layers are Mamba-2 mixers; the paper gives no
 *     formula, so the Mamba-2 mixer's output path is taken as written there:
 *     gate by SiLU(z), then normalise over channel groups, then scale)
 *
 * Every function takes the same stored bytes the GPU reads (fp32 or bf16
 * activations, fp32 per-head A / D / D_rev) and decodes them exactly to
 * double.  States are double.  Loops follow the recurrence token by token;
 * no blocking, no fusion.  The (batch, head) loop may run on several OpenMP
 * threads: each (batch, head) pair is independent, so the result does not
 * depend on the thread count.
 *
 * Layouts (row-major, contiguous):
 *   x    [batch][len][nheads][headdim]      dt [batch][len][nheads]
 *   Bm,Cm[batch][len][ngroups][dstate]      A, D, D_rev [nheads] fp32
 *   h    [nslots][nheads][headdim][dstate]  double
 *   y    [batch][len][nheads][headdim]      double
 * Head h reads group g = h / (nheads / ngroups).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_DTYPE_F32 0
#define OR_DTYPE_BF16 1
#define OR_DTYPE_F64 2   /* already-decoded values, e.g. convolution outputs */

#define OR_OK 0
#define OR_ERR_ARG (-1)
#define OR_ERR_OFFSET (-2)
#define OR_ERR_SLOT (-3)

typedef struct {
    int64_t batch, nheads, headdim, dstate, ngroups, len;
    int32_t in_dtype;
} or_shape;

/* Exact decode of one stored activation to double. */
static double rd(const void *base, int64_t i, int dtype)
{
    if (dtype == OR_DTYPE_BF16) {
        uint32_t bits = (uint32_t)((const uint16_t *)base)[i] << 16;
        float f;
        memcpy(&f, &bits, sizeof f);
        return (double)f;
    }
    if (dtype == OR_DTYPE_F64) return ((const double *)base)[i];
    return (double)((const float *)base)[i];
}

static int shape_ok(const or_shape *s)
{
    if (s->batch < 0 || s->len < 0) return 0;
    if (s->nheads <= 0 || s->headdim <= 0 || s->dstate <= 0 || s->ngroups <= 0) return 0;
    if (s->nheads % s->ngroups) return 0;
    if (s->in_dtype != OR_DTYPE_F32 && s->in_dtype != OR_DTYPE_BF16 &&
        s->in_dtype != OR_DTYPE_F64)
        return 0;
    return 1;
}

/* Index helpers for the layouts above. */
static int64_t ix_x(const or_shape *s, int64_t b, int64_t t, int64_t h, int64_t p)
{
    return ((b * s->len + t) * s->nheads + h) * s->headdim + p;
}
static int64_t ix_dt(const or_shape *s, int64_t b, int64_t t, int64_t h)
{
    return (b * s->len + t) * s->nheads + h;
}
static int64_t ix_bc(const or_shape *s, int64_t b, int64_t t, int64_t g, int64_t n)
{
    return ((b * s->len + t) * s->ngroups + g) * s->dstate + n;
}

/*
 * One token of the selective update on a headdim x dstate state S, then the
 * readout.  S <- a S + dt * x (outer) B ;  out[p] = sum_n S[p][n] C[n] + skip * x[p].
 * Used for both scan directions: the reverse direction feeds tokens in
 * reversed order and each token keeps its own (x, dt, B, C), which is what
 * rev(F(rev(block))) means.
 */
static void token_update(const or_shape *s, double *S, int64_t b, int64_t t, int64_t h,
                         int64_t g, const void *x, const void *dt, double A_h,
                         const void *Bm, const void *Cm, double skip, double *out)
{
    const int64_t P = s->headdim, N = s->dstate;
    const int dty = s->in_dtype;
    const double dtv = rd(dt, ix_dt(s, b, t, h), dty);
    const double a = exp(dtv * A_h);
    for (int64_t p = 0; p < P; ++p) {
        const double xv = rd(x, ix_x(s, b, t, h, p), dty);
        double acc = 0.0;
        for (int64_t n = 0; n < N; ++n) {
            const double bv = rd(Bm, ix_bc(s, b, t, g, n), dty);
            S[p * N + n] = a * S[p * N + n] + dtv * xv * bv;
            acc += S[p * N + n] * rd(Cm, ix_bc(s, b, t, g, n), dty);
        }
        if (out) out[p] = acc + skip * xv;
    }
}

/*
 * Active-block step (Eq. partial-reverse), all (batch, head) pairs.
 *   y_fwd = F_fwd(block; s_k)     forward scan from the cached state of the
 *                                  batch row's slot (slot_idx[b], or b)
 *   y_rev = rev(F_rev(rev(block))) reverse scan from zero, block-local
 *   y     = y_fwd + y_rev
 * The cache is read only.  y_fwd / y_rev may be NULL.  If h_out is non-NULL
 * it receives the forward state after the last block token for every batch
 * row, laid out [batch][nheads][headdim][dstate] (what a commit would store).
 */
int bdlm_oracle_block_step(const or_shape *s, const void *x, const void *dt, const float *A,
                           const void *Bm, const void *Cm, const float *D, const float *D_rev,
                           const double *h_pool, int64_t nslots, const int32_t *slot_idx,
                           double *y, double *y_fwd, double *y_rev, double *h_out)
{
    if (!s || !shape_ok(s) || !x || !dt || !A || !Bm || !Cm || !D || !D_rev || !h_pool || !y)
        return OR_ERR_ARG;
    const int64_t Bt = s->batch, L = s->len, H = s->nheads, P = s->headdim, N = s->dstate;
    const int64_t hpg = H / s->ngroups;
    for (int64_t b = 0; b < Bt; ++b) {
        const int64_t slot = slot_idx ? slot_idx[b] : b;
        if (slot < 0 || slot >= nslots) return OR_ERR_SLOT;
    }
    int err = OR_OK;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t b = 0; b < Bt; ++b) {
        for (int64_t h = 0; h < H; ++h) {
            const int64_t slot = slot_idx ? slot_idx[b] : b;
            const int64_t g = h / hpg;
            double *S = (double *)malloc(sizeof(double) * P * N);
            double *R = (double *)malloc(sizeof(double) * P * N);
            double *yf = (double *)malloc(sizeof(double) * L * P);
            double *yr = (double *)malloc(sizeof(double) * L * P);
            if (!S || !R || !yf || !yr) {
#pragma omp atomic write
                err = OR_ERR_ARG;
                free(S); free(R); free(yf); free(yr);
                continue;
            }
            /* forward: continue from the cached boundary state */
            memcpy(S, h_pool + (slot * H + h) * P * N, sizeof(double) * P * N);
            for (int64_t t = 0; t < L; ++t)
                token_update(s, S, b, t, h, g, x, dt, (double)A[h], Bm, Cm, (double)D[h],
                             yf + t * P);
            /* reverse: the flipped block from a zero state (nothing outside the block) */
            memset(R, 0, sizeof(double) * P * N);
            for (int64_t t = L - 1; t >= 0; --t)
                token_update(s, R, b, t, h, g, x, dt, (double)A[h], Bm, Cm, (double)D_rev[h],
                             yr + t * P);
            for (int64_t t = 0; t < L; ++t)
                for (int64_t p = 0; p < P; ++p) {
                    const int64_t o = ix_x(s, b, t, h, p);
                    y[o] = yf[t * P + p] + yr[t * P + p];
                    if (y_fwd) y_fwd[o] = yf[t * P + p];
                    if (y_rev) y_rev[o] = yr[t * P + p];
                }
            if (h_out) memcpy(h_out + (b * H + h) * P * N, S, sizeof(double) * P * N);
            free(S); free(R); free(yf); free(yr);
        }
    }
    return err;
}

/*
 * Block finalisation: the clean block's forward scan from the cached state
 * replaces that state (the cache now summarises prefix ++ block), and the
 * slot's bookkeeping advances by one block of len tokens.  If y_clean is
 * non-NULL it receives the layer output on the clean block, computed as the
 * active-block step above from the state before the update.
 * Every row's slot must hold exactly expected_block_index committed blocks
 * (a negative value skips that check) and no slot may appear twice; on any
 * violation nothing is modified.
 */
int bdlm_oracle_commit(const or_shape *s, const void *x, const void *dt, const float *A,
                       const void *Bm, const void *Cm, const float *D, const float *D_rev,
                       double *h_pool, int64_t nslots, const int32_t *slot_idx,
                       int64_t *n_committed, int64_t *n_blocks, int64_t expected_block_index,
                       double *y_clean)
{
    if (!s || !shape_ok(s) || !h_pool || !n_committed || !n_blocks) return OR_ERR_ARG;
    const int64_t Bt = s->batch, H = s->nheads, P = s->headdim, N = s->dstate;
    for (int64_t b = 0; b < Bt; ++b) {
        const int64_t slot = slot_idx ? slot_idx[b] : b;
        if (slot < 0 || slot >= nslots) return OR_ERR_SLOT;
        for (int64_t c = 0; c < b; ++c)
            if ((slot_idx ? slot_idx[c] : c) == slot) return OR_ERR_SLOT;
        if (expected_block_index >= 0 && n_blocks[slot] != expected_block_index)
            return OR_ERR_OFFSET;
    }
    double *hn = (double *)malloc(sizeof(double) * (Bt > 0 ? Bt : 1) * H * P * N);
    double *yc = (double *)malloc(sizeof(double) * (Bt > 0 ? Bt : 1) * s->len * H * P + 8);
    if (!hn || !yc) { free(hn); free(yc); return OR_ERR_ARG; }
    int rc = bdlm_oracle_block_step(s, x, dt, A, Bm, Cm, D, D_rev, h_pool, nslots, slot_idx,
                                    yc, NULL, NULL, hn);
    if (rc == OR_OK) {
        for (int64_t b = 0; b < Bt; ++b) {
            const int64_t slot = slot_idx ? slot_idx[b] : b;
            memcpy(h_pool + slot * H * P * N, hn + b * H * P * N, sizeof(double) * H * P * N);
            n_committed[slot] += s->len;
            n_blocks[slot] += 1;
        }
        if (y_clean) memcpy(y_clean, yc, sizeof(double) * Bt * s->len * H * P);
    }
    free(hn);
    free(yc);
    return rc;
}

/*
 * Forward-only scan over a sequence of len tokens, continuing each batch
 * row's state h[b] in place ([batch][nheads][headdim][dstate]).  This is how
 * a clean prefix is summarised into its boundary state (Eq. boundary-state).
 * If y is non-NULL it receives the forward outputs (skip term D included).
 */
int bdlm_oracle_scan_forward(const or_shape *s, const void *x, const void *dt, const float *A,
                             const void *Bm, const void *Cm, const float *D, double *h,
                             double *y)
{
    if (!s || !shape_ok(s) || !x || !dt || !A || !Bm || !Cm || !D || !h) return OR_ERR_ARG;
    const int64_t Bt = s->batch, L = s->len, H = s->nheads, P = s->headdim, N = s->dstate;
    const int64_t hpg = H / s->ngroups;
    int err = OR_OK;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t b = 0; b < Bt; ++b) {
        for (int64_t hh = 0; hh < H; ++hh) {
            double *out = (double *)malloc(sizeof(double) * P);
            if (!out) {
#pragma omp atomic write
                err = OR_ERR_ARG;
                continue;
            }
            double *S = h + (b * H + hh) * P * N;
            for (int64_t t = 0; t < L; ++t) {
                token_update(s, S, b, t, hh, hh / hpg, x, dt, (double)A[hh], Bm, Cm,
                             (double)D[hh], out);
                if (y)
                    for (int64_t p = 0; p < P; ++p) y[ix_x(s, b, t, hh, p)] = out[p];
            }
            free(out);
        }
    }
    return err;
}

/*
 * Full-window bidirectional scan (the DiffuMamba-style contrast): forward
 * over all len tokens from zero plus reverse over all len tokens from zero,
 * summed.  Identical to bdlm_oracle_block_step with a zero cache and the whole
 * window as one block; kept as its own entry so tests can state that.
 */
int bdlm_oracle_full_window(const or_shape *s, const void *x, const void *dt, const float *A,
                            const void *Bm, const void *Cm, const float *D, const float *D_rev,
                            double *y)
{
    if (!s || !shape_ok(s)) return OR_ERR_ARG;
    const int64_t Bt = s->batch, H = s->nheads, P = s->headdim, N = s->dstate;
    double *zero = (double *)calloc((size_t)((Bt > 0 ? Bt : 1) * H * P * N), sizeof(double));
    if (!zero) return OR_ERR_ARG;
    int rc = bdlm_oracle_block_step(s, x, dt, A, Bm, Cm, D, D_rev, zero, Bt > 0 ? Bt : 1, NULL,
                                    y, NULL, NULL, NULL);
    free(zero);
    return rc;
}

/*
 * The convolution of the Mamba mixer over one block, per batch row b and channel c
 * of xBC (channels: x head-major h*headdim + p, then B g*dstate + n, then C), with
 * pre-convolution inputs u[t] (decoded from the stored bytes), weights w[c][0..3]
 * (w[c][3] multiplies the current token) and bias bc[c]:
 *
 *   forward  xf[t] = silu(bc + sum_k w[k] u[t - 3 + k]),  u[-3..-1] = cache rows 0..2
 *   reverse  xr[t] = silu(bc + sum_k w[k] u[t + 3 - k]),  u[L..L+2] = 0
 *
 * The reverse line is the causal convolution of the flipped block from zeros,
 * flipped back: the reverse branch stays inside the block.  silu(v) = v / (1 + e^-v).
 * cache   [nslots][3][channels] double, row 0 the oldest input; with commit != 0
 *         the rows become the last three rows of (cache rows ++ block).
 * Outputs (double, layouts of x / B / C): xf, bf, cf (forward), xr, br, cr (reverse);
 * any may be NULL.  slot_idx as for bdlm_oracle_block_step; with commit the slots
 * must be distinct.
 */
static double silu(double v) { return v / (1.0 + exp(-v)); }

int bdlm_oracle_conv(const or_shape *s, const void *x, const void *Bm, const void *Cm,
                     const float *w, const float *bias, double *cache, int64_t nslots,
                     const int32_t *slot_idx, int commit, double *xf, double *bf, double *cf,
                     double *xr, double *br, double *cr)
{
    if (!shape_ok(s) || !w || !bias || !cache || nslots <= 0) return OR_ERR_ARG;
    const int64_t L = s->len, HP = s->nheads * s->headdim, GN = s->ngroups * s->dstate;
    const int64_t ch = HP + 2 * GN;
    for (int64_t b = 0; b < s->batch; ++b) {
        const int64_t sl = slot_idx ? slot_idx[b] : b;
        if (sl < 0 || sl >= nslots) return OR_ERR_SLOT;
        if (commit && slot_idx)
            for (int64_t b2 = 0; b2 < b; ++b2)
                if (slot_idx[b2] == sl) return OR_ERR_SLOT;
    }
    double *u = malloc((size_t)(L + 6) * sizeof(double));
    if (!u) return OR_ERR_ARG;
    for (int64_t b = 0; b < s->batch; ++b) {
        const int64_t sl = slot_idx ? slot_idx[b] : b;
        double *crow = cache + sl * 3 * ch;
        for (int64_t c = 0; c < ch; ++c) {
            /* u[0..2] cache rows, u[3..L+2] the block, u[L+3..L+5] zeros */
            for (int k = 0; k < 3; ++k) u[k] = crow[k * ch + c];
            double *of, *orv;
            int64_t oi;
            const void *src;
            if (c < HP) {
                const int64_t h = c / s->headdim, p = c % s->headdim;
                src = x;
                of = xf;
                orv = xr;
                oi = ix_x(s, b, 0, h, p);
                for (int64_t t = 0; t < L; ++t) u[3 + t] = rd(x, ix_x(s, b, t, h, p), s->in_dtype);
            } else {
                const int64_t j = (c - HP) % GN, g = j / s->dstate, n = j % s->dstate;
                src = c < HP + GN ? Bm : Cm;
                of = c < HP + GN ? bf : cf;
                orv = c < HP + GN ? br : cr;
                oi = ix_bc(s, b, 0, g, n);
                for (int64_t t = 0; t < L; ++t) u[3 + t] = rd(src, ix_bc(s, b, t, g, n), s->in_dtype);
            }
            for (int k = 0; k < 3; ++k) u[L + 3 + k] = 0.0;
            /* token stride of this channel's output layout */
            const int64_t ts = c < HP ? s->nheads * s->headdim : s->ngroups * s->dstate;
            for (int64_t t = 0; t < L; ++t) {
                double vf = bias[c], vr = bias[c];
                for (int k = 0; k < 4; ++k) {
                    vf += (double)w[c * 4 + k] * u[3 + t - 3 + k];
                    vr += (double)w[c * 4 + k] * u[3 + t + 3 - k];
                }
                if (of) of[oi + t * ts] = silu(vf);
                if (orv) orv[oi + t * ts] = silu(vr);
            }
            if (commit)
                for (int k = 0; k < 3; ++k) crow[k * ch + c] = u[L + k];
        }
    }
    free(u);
    return OR_OK;
}

/*
 * Gated RMS normalisation of the mixer output (Mamba-2 mixer, App. C):
 *
 *   g[c]   = y[c] * silu(z[c])
 *   out[c] = w[c] * g[c] / sqrt(ms(group of c) + eps),
 *   ms(G)  = (1 / |G|) * sum over c' in G of g[c']^2
 *
 * per token, over nch = nheads * headdim channels (head-major) split into ngroups
 * groups of nch / ngroups consecutive channels.  y double [ntok][nch]; z stored
 * (zdtype) [ntok][nch]; w fp32 [nch]; out double [ntok][nch].
 */
int bdlm_oracle_gated_rmsnorm(int64_t ntok, int64_t nch, int64_t ngroups, const double *y,
                              const void *z, int zdtype, const float *w, double eps, double *out)
{
    if (ntok < 0 || nch <= 0 || ngroups <= 0 || nch % ngroups != 0 || !y || !z || !w || !out)
        return OR_ERR_ARG;
    const int64_t gs = nch / ngroups;
    double *g = malloc((size_t)nch * sizeof(double));
    if (!g) return OR_ERR_ARG;
    for (int64_t t = 0; t < ntok; ++t) {
        for (int64_t c = 0; c < nch; ++c) g[c] = y[t * nch + c] * silu(rd(z, t * nch + c, zdtype));
        for (int64_t k = 0; k < ngroups; ++k) {
            double ss = 0.0;
            for (int64_t c = k * gs; c < (k + 1) * gs; ++c) ss += g[c] * g[c];
            const double r = 1.0 / sqrt(ss / (double)gs + eps);
            for (int64_t c = k * gs; c < (k + 1) * gs; ++c) out[t * nch + c] = (double)w[c] * g[c] * r;
        }
    }
    free(g);
    return OR_OK;
}

int bdlm_oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Thread count of the OpenMP loops over (batch, head) from now on; n <= 0 changes
 * nothing.  Timing only: every result is the same at any thread count. */
void bdlm_oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
