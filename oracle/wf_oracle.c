/*
 * CPU oracle for spatial autoregressive context-model decoding and encoding.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  It shares no code,
 * header, table or constant with the GPU path and never imports it.
 *
 * What it computes (paper, Sec. III-A, Eq. 2-4, and Appendix A, Def. 1): the
 * latent grid is decoded one latent at a time in a given topological order of
 * the dependency DAG (raster order by default, Eq. 2).  For each latent the
 * context is a (2R+1)x(2R+1) causal masked convolution (Def. 1: the R rows
 * above within horizontal offset R, and the R latents to the left; R = 2, the
 * 5x5 mask, unless `radius` says otherwise), then the
 * entropy-parameter network maps [hyperprior params ; context] to the
 * distribution parameters (Sec. II-B, Eq. 1).  Decoding writes y_hat = s + mu
 * for the given integer symbol s; encoding quantises s = round(y - mu) and
 * writes the same y_hat.  Because the per-latent function only reads latents
 * that precede it in every topological order, any such order gives the same
 * bits (Sec. III-A); the wavefront order of Sec. III-B is one of them.
 *
 * Arithmetic: every dot product is accumulated in fp64 starting from the
 * bias, and every stored vector is rounded to fp32.  In bf16 mode every weight
 * is rounded to bf16 (round half to even), and every activation operand
 * (gathered taps, hyperprior params, context, hidden activations) is carried
 * as the sum of two bf16 values, hi = bf16(x) and lo = bf16(x - hi), which
 * holds x to about 2^-17 relative; biases and the parameter epilogue stay
 * fp32.  (Rounding the activations to one bf16 each makes the decode
 * ill-conditioned: a 1e-6 difference in accumulation order re-rounds a tap by
 * a whole bf16 step and the change spreads along the wavefront, so two
 * correct evaluations no longer agree to 1e-2.)
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *  - out-of-image taps contribute zero (Def. 1 keeps only in-image edges);
 *  - the conv is a cross-correlation with bias: tap (dy,dx) uses
 *    weight[o][c][dy+R][dx+R] of a [2M][M][2R+1][2R+1] weight;
 *  - the network input is [psi ; ctx]; activation is LeakyReLU;
 *  - output channels are [mean | scale] for one Gaussian, and
 *    [weight | mean | scale] (component-major blocks of M) for a 3-component
 *    mixture; mixture weights are a softmax over the 3 logits per channel and
 *    the dequantisation offset is the mixture mean;
 *  - scale = max(raw scale, table[0]); index = number of the first L-1 table
 *    entries strictly below the scale;
 *  - the quantiser rounds half to even.
 *
 * Context approximation (Sec. III-D, Fig. 3), when group > 1: the wavefronts
 * t = lambda*i + j (lambda = 3, or 2 for the relaxed mask; Sec. III-B) are
 * taken N = group at a time, and all latents of group floor(t / N) are
 * evaluated together.  A tap of the same group is not yet decoded; it is
 * replaced, channel by channel, by the mean of the latent's in-image taps of
 * earlier groups, or by zero when there is none (the paper fills with zero
 * when nothing is known).  Out-of-image taps stay zero.  Reading taken where
 * the paper says "local neighborhood": the taps of the causal mask.  The
 * per-latent function then reads only latents of earlier groups, all of which
 * precede it in raster order, so a raster pass computes the grouped decode.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "wf_rans.h"

typedef struct {
    int32_t H, W, M, B, K;      /* rows, cols, channels, images, mixture comps */
    int32_t d1, d2;             /* hidden widths of the parameter network     */
    int32_t relaxed;            /* 1: drop taps (-1,+2) and (-2,+2)           */
    int32_t bf16;               /* 1: bf16 weights, activations as bf16 pairs */
    float slope;                /* LeakyReLU negative slope                   */
    const float *ctx_w;         /* [2M][M][5][5]                              */
    const float *ctx_b;         /* [2M]                                       */
    const float *w1, *b1;       /* [d1][4M], [d1]                             */
    const float *w2, *b2;       /* [d2][d1], [d2]                             */
    const float *w3, *b3;       /* [n3][d2], [n3]; n3 = 2M (K=1) or 9M (K=3)  */
    const float *table;         /* [L], strictly increasing                   */
    int32_t L;
    int32_t group;              /* 0 or 1: exact; N > 1: groups of N wavefronts */
    int32_t radius;             /* mask radius R (0 means 2); ctx_w is [2M][M][2R+1][2R+1] */
} oracle_model;

typedef struct {
    float *y_hat;               /* [B][H][W][M]                               */
    float *mean;                /* [B][H][W][M]  (mixture mean when K=3)      */
    float *scale;               /* [B][H][W][K][M]                            */
    int32_t *idx;               /* [B][H][W][K][M]                            */
    float *weight;              /* [B][H][W][K][M] or NULL                    */
    float *comp_mean;           /* [B][H][W][K][M] or NULL                    */
} oracle_out;

/* Round an fp32 value to the nearest bf16 (ties to even), returned as fp32. */
static float to_bf16(float v)
{
    uint32_t u;
    memcpy(&u, &v, 4);
    if ((u & 0x7f800000u) == 0x7f800000u) { /* inf / nan: truncate */
        u &= 0xffff0000u;
    } else {
        uint32_t lsb = (u >> 16) & 1u;
        u += 0x7fffu + lsb;
        u &= 0xffff0000u;
    }
    memcpy(&v, &u, 4);
    return v;
}

/* A weight operand: rounded to bf16 in bf16 mode. */
static double weight_op(const oracle_model *m, float w)
{
    return (double)(m->bf16 ? to_bf16(w) : w);
}

/* An activation operand: hi + lo, two bf16 values, in bf16 mode (x - hi is
 * exact in fp32, and so is hi + lo). */
static double act_op(const oracle_model *m, float x)
{
    if (!m->bf16) return (double)x;
    float hi = to_bf16(x);
    float lo = to_bf16(x - hi);
    return (double)hi + (double)lo;
}

static int radius_of(const oracle_model *m)
{
    return m->radius > 0 ? m->radius : 2;
}

/* Is the causal tap (dy,dx) part of the mask?  The (2R+1)^2 causal mask keeps
 * rows dy = -R..-1 with any dx in [-R,R], and dy = 0 with dx in [-R,-1]. */
static int tap_in_mask(const oracle_model *m, int dy, int dx)
{
    const int R = radius_of(m);
    if (dy < -R || dy > 0 || dx < -R || dx > R) return 0;
    if (dy == 0 && dx >= 0) return 0;
    if (m->relaxed && dx == 2 && (dy == -1 || dy == -2)) return 0;
    return 1;
}

/* Weight of output oc, input channel c, tap (dy,dx). */
static float conv_weight(const oracle_model *m, int oc, int c, int dy, int dx)
{
    const int R = radius_of(m), k = 2 * R + 1;
    return m->ctx_w[(((size_t)oc * m->M + c) * k + (dy + R)) * k + (dx + R)];
}

/* The least shear of the mask (Sec. III-B): R + 1, or 2 for the relaxed 5x5 mask. */
static int shear_of(const oracle_model *m)
{
    return m->relaxed ? 2 : radius_of(m) + 1;
}

/* Status of tap (dy,dx) of latent (i,j): 0 outside the image, 1 decoded
 * before the latent's group (its value is used), 2 in the latent's own group
 * (filled).  Without grouping every in-image tap has status 1. */
static int tap_status(const oracle_model *m, int i, int j, int dy, int dx)
{
    int ii = i + dy, jj = j + dx;
    if (ii < 0 || ii >= m->H || jj < 0 || jj >= m->W) return 0;
    if (m->group <= 1) return 1;
    int lam = shear_of(m);
    int g = (lam * i + j) / m->group;
    int gt = (lam * ii + jj) / m->group;
    return gt < g ? 1 : 2;
}

/* Exported for the tests: tap_status of the model's grid and grouping. */
int oracle_tap_status(const oracle_model *m, int i, int j, int dy, int dx)
{
    return m ? tap_status(m, i, j, dy, dx) : -1;
}

static float lrelu(const oracle_model *m, float v)
{
    return v >= 0.0f ? v : m->slope * v;
}

static size_t n3_of(const oracle_model *m)
{
    return (size_t)(m->K == 1 ? 2 : 9) * (size_t)m->M;
}

/*
 * The per-latent function: distribution parameters of latent (b,i,j) from the
 * current reconstruction y_hat and the hyperprior params psi.  Writes
 * mu[M], sigma[K*M], index[K*M], weight[K*M], cmean[K*M] (component-major).
 * scratch must hold 5M + d1 + d2 + n3 floats.
 */
static void latent_params(const oracle_model *m, const float *y_hat,
                          const float *psi, int b, int i, int j,
                          float *mu, float *sigma, int32_t *index,
                          float *weight, float *cmean, float *scratch)
{
    const int M = m->M, H = m->H, W = m->W;
    float *h0 = scratch;              /* [4M] = [psi ; ctx] */
    float *h1 = h0 + 4 * M;           /* [d1] */
    float *h2 = h1 + m->d1;           /* [d2] */
    float *o = h2 + m->d2;            /* [n3] */
    const size_t lat = ((size_t)b * H + i) * W + j;

    /* Grouped decode: the fill value of same-group taps, per channel, the
     * mean of the decoded in-image taps (zero when there is none). */
    float *fill = o + n3_of(m);       /* [M] */
    if (m->group > 1) {
        int known = 0;
        for (int c = 0; c < M; ++c) fill[c] = 0.0f;
        double *sum = calloc((size_t)M, sizeof(double));
        const int R = radius_of(m);
        for (int dy = -R; dy <= 0; ++dy)
            for (int dx = -R; dx <= R; ++dx) {
                if (!tap_in_mask(m, dy, dx) || tap_status(m, i, j, dy, dx) != 1) continue;
                const float *src = y_hat + (((size_t)b * H + i + dy) * W + j + dx) * M;
                for (int c = 0; c < M; ++c) sum[c] += (double)src[c];
                ++known;
            }
        if (known > 0)
            for (int c = 0; c < M; ++c) fill[c] = (float)(sum[c] / known);
        free(sum);
    }

    /* Context: the masked conv evaluated at (i,j), Def. 1 / Sec. III-C. */
    const int R = radius_of(m);
    for (int oc = 0; oc < 2 * M; ++oc) {
        double acc = (double)m->ctx_b[oc];
        for (int dy = -R; dy <= 0; ++dy) {
            for (int dx = -R; dx <= R; ++dx) {
                if (!tap_in_mask(m, dy, dx)) continue;
                int st = tap_status(m, i, j, dy, dx);
                if (st == 0) continue;
                const float *src = st == 1 ? y_hat + (((size_t)b * H + i + dy) * W + j + dx) * M : fill;
                for (int c = 0; c < M; ++c)
                    acc += weight_op(m, conv_weight(m, oc, c, dy, dx)) * act_op(m, src[c]);
            }
        }
        h0[2 * M + oc] = (float)acc;
    }
    for (int c = 0; c < 2 * M; ++c) h0[c] = psi[lat * 2 * M + c];

    /* Entropy-parameter network: three 1x1 layers. */
    for (int n = 0; n < m->d1; ++n) {
        double acc = (double)m->b1[n];
        for (int k = 0; k < 4 * M; ++k)
            acc += weight_op(m, m->w1[(size_t)n * 4 * M + k]) * act_op(m, h0[k]);
        h1[n] = lrelu(m, (float)acc);
    }
    for (int n = 0; n < m->d2; ++n) {
        double acc = (double)m->b2[n];
        for (int k = 0; k < m->d1; ++k)
            acc += weight_op(m, m->w2[(size_t)n * m->d1 + k]) * act_op(m, h1[k]);
        h2[n] = lrelu(m, (float)acc);
    }
    const size_t n3 = n3_of(m);
    for (size_t n = 0; n < n3; ++n) {
        double acc = (double)m->b3[n];
        for (int k = 0; k < m->d2; ++k)
            acc += weight_op(m, m->w3[n * m->d2 + k]) * act_op(m, h2[k]);
        o[n] = (float)acc;
    }

    /* Parameter epilogue. */
    const int K = m->K;
    for (int c = 0; c < M; ++c) {
        if (K == 1) {
            mu[c] = o[c];
            sigma[c] = o[M + c];
            weight[c] = 1.0f;
            cmean[c] = o[c];
        } else {
            double lg[3], mx = -INFINITY, den = 0.0, mix = 0.0;
            for (int k = 0; k < 3; ++k) {
                lg[k] = (double)o[(size_t)k * M + c];
                if (lg[k] > mx) mx = lg[k];
            }
            for (int k = 0; k < 3; ++k) den += exp(lg[k] - mx);
            for (int k = 0; k < 3; ++k) {
                double wk = exp(lg[k] - mx) / den;
                float mk = o[(size_t)(3 + k) * M + c];
                weight[k * M + c] = (float)wk;
                cmean[k * M + c] = mk;
                sigma[k * M + c] = o[(size_t)(6 + k) * M + c];
                mix += wk * (double)mk;
            }
            mu[c] = (float)mix;
        }
    }
    for (int q = 0; q < K * M; ++q) {
        float s = sigma[q] > m->table[0] ? sigma[q] : m->table[0];
        int32_t cnt = 0;
        for (int l = 0; l < m->L - 1; ++l)
            if (m->table[l] < s) ++cnt;
        sigma[q] = s;
        index[q] = cnt;
    }
}

static size_t scratch_floats(const oracle_model *m)
{
    return (size_t)5 * m->M + m->d1 + m->d2 + n3_of(m);
}

static void store_params(const oracle_model *m, const oracle_out *out, size_t lat,
                         const float *mu, const float *sigma, const int32_t *index,
                         const float *weight, const float *cmean)
{
    const size_t M = m->M, KM = (size_t)m->K * m->M;
    if (out->mean) memcpy(out->mean + lat * M, mu, M * sizeof(float));
    if (out->scale) memcpy(out->scale + lat * KM, sigma, KM * sizeof(float));
    if (out->idx) memcpy(out->idx + lat * KM, index, KM * sizeof(int32_t));
    if (out->weight) memcpy(out->weight + lat * KM, weight, KM * sizeof(float));
    if (out->comp_mean) memcpy(out->comp_mean + lat * KM, cmean, KM * sizeof(float));
}

/*
 * Sequential decode (y_in == NULL) or encode (y_in != NULL) of all B*H*W
 * latents, in the order given by order[] (indices b*H*W + i*W + j); order ==
 * NULL means raster order (Eq. 2).  Decode reads sym; encode writes sym.
 * y_hat is zeroed first.  Returns 0, or -1 on a bad argument or allocation.
 */
int oracle_run(const oracle_model *m, const float *psi, int32_t *sym,
               const float *y_in, const int64_t *order, int64_t n_order,
               const oracle_out *out)
{
    if (!m || !psi || !sym || !out || !out->y_hat) return -1;
    if (m->K != 1 && m->K != 3) return -1;
    const size_t M = m->M;
    const size_t total = (size_t)m->B * m->H * m->W;
    if (order && n_order != (int64_t)total) return -1;
    float *scratch = malloc(scratch_floats(m) * sizeof(float));
    float *mu = malloc(M * sizeof(float));
    float *sigma = malloc(3 * M * sizeof(float));
    float *weight = malloc(3 * M * sizeof(float));
    float *cmean = malloc(3 * M * sizeof(float));
    int32_t *index = malloc(3 * M * sizeof(int32_t));
    if (!scratch || !mu || !sigma || !weight || !cmean || !index) {
        free(scratch); free(mu); free(sigma); free(weight); free(cmean); free(index);
        return -1;
    }
    memset(out->y_hat, 0, total * M * sizeof(float));
    int rc = 0;
    for (size_t n = 0; n < total; ++n) {
        size_t lat = order ? (size_t)order[n] : n;
        if (lat >= total) { rc = -1; break; }
        int b = (int)(lat / ((size_t)m->H * m->W));
        int i = (int)((lat / m->W) % m->H);
        int j = (int)(lat % m->W);
        latent_params(m, out->y_hat, psi, b, i, j, mu, sigma, index, weight, cmean, scratch);
        store_params(m, out, lat, mu, sigma, index, weight, cmean);
        for (size_t c = 0; c < M; ++c) {
            float s;
            if (y_in) {
                float r = y_in[lat * M + c] - mu[c];
                s = nearbyintf(r);          /* default mode: ties to even */
                sym[lat * M + c] = (int32_t)s;
            } else {
                s = (float)sym[lat * M + c];
            }
            out->y_hat[lat * M + c] = s + mu[c];
        }
    }
    free(scratch); free(mu); free(sigma); free(weight); free(cmean); free(index);
    return rc;
}

/*
 * Decode with the symbols taken from rANS streams (wf_rans.c): in raster
 * order, each latent's parameters give its scale indices, and with them the
 * next symbol of the stream of its (image, grid row, channel) is decoded
 * before y_hat = s + mean is written (K = 1: the Gaussian of the scale
 * level; K = 3: the mixture of the three components, wf_rans.c).  sym_out
 * receives the decoded symbols.  Returns 0, or -1 on a bad argument or a malformed stream.
 */
int oracle_run_bits(const oracle_model *m, const float *psi, const uint32_t *bits,
                    const uint32_t *offsets, int32_t *sym_out, const oracle_out *out)
{
    if (!m || !psi || !bits || !offsets || !sym_out || !out || !out->y_hat) return -1;
    if (m->K != 1 && m->K != 3) return -1;
    const int K = m->K;
    const size_t M = m->M;
    const size_t total = (size_t)m->B * m->H * m->W;
    const size_t nstreams = (size_t)m->B * m->H * M;
    rans_tables t;
    mix_tables mt;
    if (K == 1 ? rans_tables_build(m->table, m->L, &t) : mix_tables_build(m->table, m->L, &mt)) return -1;
    float *scratch = malloc(scratch_floats(m) * sizeof(float));
    float *mu = malloc(M * sizeof(float));
    float *sigma = malloc(K * M * sizeof(float));
    float *weight = malloc(K * M * sizeof(float));
    float *cmean = malloc(K * M * sizeof(float));
    int32_t *index = malloc(K * M * sizeof(int32_t));
    rans_dec *dec = malloc(nstreams * sizeof(rans_dec));
    int rc = 0;
    if (!scratch || !mu || !sigma || !weight || !cmean || !index || !dec) rc = -1;
    for (size_t k = 0; k < nstreams && !rc; ++k)
        if (rans_dec_init(&dec[k], bits + offsets[k], (int64_t)offsets[k + 1] - offsets[k])) rc = -1;
    if (!rc) memset(out->y_hat, 0, total * M * sizeof(float));
    for (size_t lat = 0; lat < total && !rc; ++lat) {
        int b = (int)(lat / ((size_t)m->H * m->W));
        int i = (int)((lat / m->W) % m->H);
        int j = (int)(lat % m->W);
        latent_params(m, out->y_hat, psi, b, i, j, mu, sigma, index, weight, cmean, scratch);
        store_params(m, out, lat, mu, sigma, index, weight, cmean);
        for (size_t c = 0; c < M; ++c) {
            rans_dec *d = &dec[((size_t)b * m->H + i) * M + c];
            int32_t s;
            if (K == 1) {
                if (rans_dec_symbol(d, &t, index[c], &s)) { rc = -1; break; }
            } else {
                /* the mixture of the channel's three components */
                const float w3[3] = {weight[c], weight[M + c], weight[2 * M + c]};
                const float m3[3] = {cmean[c], cmean[M + c], cmean[2 * M + c]};
                const int32_t l3[3] = {index[c], index[M + c], index[2 * M + c]};
                mix_param p;
                if (mix_params(&mt, w3, m3, mu[c], l3, &p) || mix_dec_symbol(d, &mt, &p, &s)) { rc = -1; break; }
            }
            sym_out[lat * M + c] = s;
            out->y_hat[lat * M + c] = (float)s + mu[c];
        }
    }
    free(scratch); free(mu); free(sigma); free(weight); free(cmean); free(index); free(dec);
    if (K == 1) rans_tables_free(&t);
    else mix_tables_free(&mt);
    return rc;
}

/*
 * Teacher-forced evaluation: the per-latent parameters computed from a GIVEN
 * reconstruction y_hat (nothing is written to it), at the n listed latents
 * (all B*H*W latents in raster order when lats == NULL).  Output row q of
 * each out array belongs to lats[q].  out->y_hat is not used.
 */
int oracle_eval(const oracle_model *m, const float *y_hat, const float *psi,
                const int64_t *lats, int64_t n, const oracle_out *out)
{
    if (!m || !y_hat || !psi || !out) return -1;
    if (m->K != 1 && m->K != 3) return -1;
    const size_t M = m->M;
    const size_t total = (size_t)m->B * m->H * m->W;
    if (!lats) n = (int64_t)total;
    float *scratch = malloc(scratch_floats(m) * sizeof(float));
    float *mu = malloc(M * sizeof(float));
    float *sigma = malloc(3 * M * sizeof(float));
    float *weight = malloc(3 * M * sizeof(float));
    float *cmean = malloc(3 * M * sizeof(float));
    int32_t *index = malloc(3 * M * sizeof(int32_t));
    if (!scratch || !mu || !sigma || !weight || !cmean || !index) {
        free(scratch); free(mu); free(sigma); free(weight); free(cmean); free(index);
        return -1;
    }
    int rc = 0;
    for (int64_t q = 0; q < n; ++q) {
        size_t lat = lats ? (size_t)lats[q] : (size_t)q;
        if (lat >= total) { rc = -1; break; }
        int b = (int)(lat / ((size_t)m->H * m->W));
        int i = (int)((lat / m->W) % m->H);
        int j = (int)(lat % m->W);
        latent_params(m, y_hat, psi, b, i, j, mu, sigma, index, weight, cmean, scratch);
        store_params(m, out, (size_t)q, mu, sigma, index, weight, cmean);
    }
    free(scratch); free(mu); free(sigma); free(weight); free(cmean); free(index);
    return rc;
}
