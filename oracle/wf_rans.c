/*
 * rANS entropy coding of the quantised latents of a mean-scale Gaussian
 * entropy model -- the oracle's side.  TEST INFRASTRUCTURE ONLY (see
 * oracle/__init__.py); it shares no code with the GPU path.
 *
 * The paper pairs the wavefront decode with rANS (Sec. III-C, "Tensorized
 * rANS"): once the per-latent parameters are known, each symbol is coded
 * with the discretised Gaussian of its scale (Sec. II-A: the latents are
 * coded losslessly with an entropy coder under the predicted distribution).
 * The coder here is Duda's range variant of asymmetric numeral systems,
 * written from its definition: a 64-bit state x in [2^31, 2^63), 32-bit
 * renormalisation words and probabilities quantised to 2^-16 (the state's
 * lower bound is 2^15 times the probability scale, so rounding the state
 * costs almost nothing; a 32-bit state over 16-bit words lost 0.05 bits per
 * symbol).
 *
 *   push(x, f, c):  if x >= f * 2^47: emit the low 32 bits, x >>= 32;
 *                   x = floor(x / f) * 2^16 + (x mod f) + c
 *   pop(x):         slot = x mod 2^16; the symbol u with c_u <= slot < c_u + f_u;
 *                   x = f_u * floor(x / 2^16) + slot - c_u;
 *                   if x < 2^31: x = x * 2^32 + next word
 *
 * Tables (one per level l of the scale table; the level is the symbol's scale
 * index, and the coding scale is the level's value T_l, the upper end of the
 * scales that share the index):
 *   n_l = max(1, ceil(6 T_l)), symbols s in [-n_l, n_l] (u = s + n_l) and an
 *   escape u = 2 n_l + 1 for |s| > n_l;
 *   p(s) = the Gaussian mass of [s - 1/2, s + 1/2] (zero mean, scale T_l),
 *   written with erfc of a = (|s| - 1/2) / (T_l sqrt 2), b = (|s| + 1/2) / (T_l sqrt 2):
 *     p(0) = 1 - erfc(b),  p(s != 0) = (erfc(a) - erfc(b)) / 2,
 *     p(escape) = erfc((n_l + 1/2) / (T_l sqrt 2));
 *   f_u = 1 + floor(p_u (2^16 - (2 n_l + 2))), and what is left of 2^16
 *   goes to s = 0 (the mode); c_u = sum of f below u.
 * An escaped symbol is followed by e = 2(|s| - n_l - 1) + (s < 0) in 15-bit
 * chunks, low chunk first, each coded uniformly (f = 1 of 2^16) as a 16-bit
 * value whose top bit says that another chunk follows.
 *
 * Streams: one per (image b, grid row i, channel c), index k = (b H + i) M + c,
 * holding the row's symbols in column order j = 0..W-1 (the order in which a
 * wavefront decode reaches them: one per step).  A stream is the final state
 * (high word, low word) followed by the renormalisation words in the order the
 * decoder reads them, all 32-bit; offsets[k] is its first word, offsets[B H M]
 * the total.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "wf_rans.h"

#define PREC_BITS 16
#define PREC_TOTAL (1u << PREC_BITS)
#define STATE_LOW (1ull << 31)
#define TAIL_SIGMAS 6.0

static int support_of(float scale)
{
    double n = ceil(TAIL_SIGMAS * (double)scale);
    if (n < 1.0) n = 1.0;
    if (n > 1.0e6) n = 1.0e6;
    return (int)n;
}

/* Gaussian mass of symbol u of a level with support n and scale sigma. */
static double mass_of(int u, int n, double sigma)
{
    const double r = sigma * sqrt(2.0);
    if (u == 2 * n + 1) return erfc(((double)n + 0.5) / r);
    const int s = abs(u - n);
    const double b = ((double)s + 0.5) / r;
    if (s == 0) return 1.0 - erfc(b);
    const double a = ((double)s - 0.5) / r;
    return 0.5 * (erfc(a) - erfc(b));
}

int rans_tables_build(const float *table, int L, rans_tables *t)
{
    memset(t, 0, sizeof(*t));
    if (!table || L < 1) return -1;
    t->L = L;
    t->n = malloc((size_t)L * sizeof(int32_t));
    t->base = malloc(((size_t)L + 1) * sizeof(int64_t));
    if (!t->n || !t->base) { rans_tables_free(t); return -1; }
    int64_t total = 0;
    for (int l = 0; l < L; ++l) {
        t->n[l] = support_of(table[l]);
        t->base[l] = total;
        total += 2 * (int64_t)t->n[l] + 3;
    }
    t->base[L] = total;
    t->cum = malloc((size_t)total * sizeof(uint32_t));
    if (!t->cum) { rans_tables_free(t); return -1; }
    for (int l = 0; l < L; ++l) {
        const int n = t->n[l], K = 2 * n + 2;
        const double sigma = (double)table[l];
        const double R = (double)(PREC_TOTAL - (uint32_t)K);
        uint32_t *f = malloc((size_t)K * sizeof(uint32_t));
        if (!f) { rans_tables_free(t); return -1; }
        uint32_t sum = 0;
        for (int u = 0; u < K; ++u) {
            f[u] = 1u + (uint32_t)floor(mass_of(u, n, sigma) * R);
            sum += f[u];
        }
        f[n] += PREC_TOTAL - sum;
        uint32_t *c = t->cum + t->base[l];
        c[0] = 0;
        for (int u = 0; u < K; ++u) c[u + 1] = c[u] + f[u];
        free(f);
    }
    return 0;
}

void rans_tables_free(rans_tables *t)
{
    free(t->n); free(t->base); free(t->cum);
    memset(t, 0, sizeof(*t));
}

/* ---- encoder: words are emitted in reverse decode order ---------------- */

typedef struct {
    uint64_t x;
    uint32_t *buf;     /* emitted words, in emission order */
    int64_t n, cap;
    int overflow;
} rans_enc;

static void enc_push(rans_enc *e, uint32_t cum, uint32_t freq)
{
    uint64_t x = e->x;
    if (x >= ((uint64_t)freq << 47)) {
        if (e->n < e->cap) e->buf[e->n] = (uint32_t)(x & 0xffffffffu);
        else e->overflow = 1;
        e->n++;
        x >>= 32;
    }
    x = ((x / freq) << PREC_BITS) + (x % freq) + cum;
    e->x = x;
}

/* Push symbol s of level l (escape chunks first: the decoder reads them
 * after the escape symbol). */
static void enc_symbol(rans_enc *e, const rans_tables *t, int l, int32_t s)
{
    const int n = t->n[l];
    const uint32_t *c = t->cum + t->base[l];
    int u;
    if (s >= -n && s <= n) {
        u = s + n;
    } else {
        u = 2 * n + 1;
        const int64_t mag = s < 0 ? -(int64_t)s : (int64_t)s;
        const uint64_t ev = 2u * (uint64_t)(mag - n - 1) + (s < 0 ? 1u : 0u);
        uint32_t chunk[5];
        int nc = 0;
        uint64_t v = ev;
        do {
            chunk[nc++] = (uint32_t)(v & 0x7fffu);
            v >>= 15;
        } while (v);
        for (int q = 0; q < nc - 1; ++q) chunk[q] |= 0x8000u;
        for (int q = nc - 1; q >= 0; --q) enc_push(e, chunk[q], 1);
    }
    enc_push(e, c[u], c[u + 1] - c[u]);
}

/* Encode all streams.  sym, idx: [B][H][W][M].  Returns the total word count
 * (written to offsets[B H M]), or -1 on a bad argument or when `bits` (cap
 * words) is too small; with bits == NULL only the offsets are computed. */
int64_t oracle_rans_encode(const int32_t *sym, const int32_t *idx, int B, int H, int W, int M,
                           const float *table, int L, uint32_t *bits, int64_t cap, uint32_t *offsets)
{
    if (!sym || !idx || !table || !offsets || B < 1 || H < 1 || W < 1 || M < 1) return -1;
    rans_tables t;
    if (rans_tables_build(table, L, &t)) return -1;
    const int64_t per = 2 + 4 * (int64_t)W;   /* words a stream can emit at most */
    uint32_t *tmp = malloc((size_t)per * sizeof(uint32_t));
    if (!tmp) { rans_tables_free(&t); return -1; }
    int64_t pos = 0;
    int bad = 0;
    for (int b = 0; b < B && !bad; ++b)
        for (int i = 0; i < H && !bad; ++i)
            for (int ch = 0; ch < M && !bad; ++ch) {
                const int64_t k = ((int64_t)b * H + i) * M + ch;
                rans_enc e = {STATE_LOW, tmp, 0, per, 0};
                for (int j = W - 1; j >= 0; --j) {
                    const size_t q = (((size_t)b * H + i) * W + j) * M + ch;
                    const int l = idx[q];
                    if (l < 0 || l >= L) { bad = 1; break; }
                    enc_symbol(&e, &t, l, sym[q]);
                }
                if (bad || e.overflow || pos + 2 + e.n > (int64_t)UINT32_MAX) { bad = 1; break; }
                offsets[k] = (uint32_t)pos;
                if (bits && pos + 2 + e.n <= cap) {
                    bits[pos] = (uint32_t)(e.x >> 32);
                    bits[pos + 1] = (uint32_t)(e.x & 0xffffffffu);
                    for (int64_t q = 0; q < e.n; ++q) bits[pos + 2 + q] = tmp[e.n - 1 - q];
                } else if (bits) {
                    bad = 1;
                }
                pos += 2 + e.n;
            }
    free(tmp);
    rans_tables_free(&t);
    if (bad) return -1;
    offsets[(int64_t)B * H * M] = (uint32_t)pos;
    return pos;
}

/* ---- decoder ------------------------------------------------------------ */

int rans_dec_init(rans_dec *d, const uint32_t *w, int64_t n_words)
{
    if (n_words < 2) return -1;
    d->x = ((uint64_t)w[0] << 32) | w[1];
    d->w = w + 2;
    d->end = w + n_words;
    return d->x >= STATE_LOW ? 0 : -1;
}

static int dec_pop(rans_dec *d, const uint32_t *c, int K, int *u_out)
{
    const uint32_t slot = d->x & (PREC_TOTAL - 1u);
    int u;
    if (!c) {
        u = (int)slot;                       /* uniform chunk */
        d->x = d->x >> PREC_BITS;
    } else {
        int lo = 0, hi = K - 1;              /* largest u with c[u] <= slot */
        while (lo < hi) {
            const int mid = (lo + hi + 1) / 2;
            if (c[mid] <= slot) lo = mid;
            else hi = mid - 1;
        }
        u = lo;
        d->x = (c[u + 1] - c[u]) * (d->x >> PREC_BITS) + slot - c[u];
    }
    if (d->x < STATE_LOW) {
        if (d->w >= d->end) return -1;
        d->x = (d->x << 32) | *d->w++;
    }
    *u_out = u;
    return 0;
}

int rans_dec_symbol(rans_dec *d, const rans_tables *t, int level, int32_t *s)
{
    if (level < 0 || level >= t->L) return -1;
    const int n = t->n[level];
    int u;
    if (dec_pop(d, t->cum + t->base[level], 2 * n + 2, &u)) return -1;
    if (u <= 2 * n) {
        *s = u - n;
        return 0;
    }
    uint64_t ev = 0;
    for (int q = 0; q < 5; ++q) {
        int chunk;
        if (dec_pop(d, NULL, 0, &chunk)) return -1;
        ev |= (uint64_t)(chunk & 0x7fff) << (15 * q);
        if (!(chunk & 0x8000)) {
            const int64_t mag = (int64_t)(ev >> 1) + n + 1;
            *s = (int32_t)((ev & 1u) ? -mag : mag);
            return 0;
        }
    }
    return -1;
}

/* Decode all streams with given scale indices (teacher-forced): sym_out and
 * idx [B][H][W][M].  Returns 0, or -1 on a malformed stream. */
int oracle_rans_decode(const uint32_t *bits, const uint32_t *offsets, const int32_t *idx, int B, int H,
                       int W, int M, const float *table, int L, int32_t *sym_out)
{
    if (!bits || !offsets || !idx || !table || !sym_out) return -1;
    rans_tables t;
    if (rans_tables_build(table, L, &t)) return -1;
    int rc = 0;
    for (int b = 0; b < B && !rc; ++b)
        for (int i = 0; i < H && !rc; ++i)
            for (int ch = 0; ch < M && !rc; ++ch) {
                const int64_t k = ((int64_t)b * H + i) * M + ch;
                rans_dec d;
                if (rans_dec_init(&d, bits + offsets[k], (int64_t)offsets[k + 1] - offsets[k])) { rc = -1; break; }
                for (int j = 0; j < W; ++j) {
                    const size_t q = (((size_t)b * H + i) * W + j) * M + ch;
                    if (rans_dec_symbol(&d, &t, idx[q], &sym_out[q])) { rc = -1; break; }
                }
            }
    rans_tables_free(&t);
    return rc;
}

/* The tables of a scale table: n [L], base [L+1], and (when cum != NULL and
 * base[L] <= cap) the cumulative frequencies.  Returns base[L] or -1. */
int64_t oracle_rans_tables(const float *table, int L, int32_t *n, int64_t *base, uint32_t *cum, int64_t cap)
{
    rans_tables t;
    if (rans_tables_build(table, L, &t)) return -1;
    const int64_t total = t.base[L];
    if (n) memcpy(n, t.n, (size_t)L * sizeof(int32_t));
    if (base) memcpy(base, t.base, ((size_t)L + 1) * sizeof(int64_t));
    if (cum && total <= cap) memcpy(cum, t.cum, (size_t)total * sizeof(uint32_t));
    rans_tables_free(&t);
    return total;
}

/* ---- mixture model (K = 3) ----------------------------------------------
 * The Cheng2020-style entropy model gives each latent channel a mixture of
 * three Gaussians (weights w_k, means mu_k, scales sigma_k); the symbol is
 * s = round(y - mu) with mu = sum_k w_k mu_k, the mixture mean, and its
 * probability is the mixture mass of [s - 1/2, s + 1/2] around mu:
 *   p(s) = sum_k w_k (Phi((s + 1/2 - d_k) / sigma_k) - Phi((s - 1/2 - d_k) / sigma_k)),
 * d_k = mu_k - mu.  Encoder and decoder must build bit-identical frequency
 * tables for every latent, so the real parameters are first quantised, in
 * fp32 as the decode holds them, and the rest is integer arithmetic:
 *   weights  v_k = 1 + floor(w_k 4093) (w_k 4093 clamped to [0, 4093]), then
 *            4096 - sum v added to the largest v_k (the first of equals);
 *   offsets  q_k = rint(16 d_k) clamped to [-2^14, 2^14] (sixteenths of a
 *            symbol; NaN goes to -2^14);
 *   scales   the component's scale level l_k, coded at the level's value T_l.
 * Per level: X_l = 16 (n_l + 1), n_l the one-Gaussian support, and an
 * integer CDF over sixteenths
 *   G_l(x) = floor(2^20 Phi(x / (16 T_l)) + 1/2) for |x| < X_l,
 *            0 for x <= -X_l, 2^20 for x >= X_l.
 * Mixture CDF at the upper edge of symbol s (F_tot = 2^32):
 *   F(s) = sum_k v_k G_{l_k}(16 s + 8 - q_k).
 * Support s_lo = min_k floor((q_k - X_k) / 16), s_hi = max_k ceil((q_k + X_k) / 16),
 * S = s_hi - s_lo + 1, and
 *   cum(s) = (s - s_lo) + floor(F(s - 1) (2^16 - S - 1) / 2^32),  s_lo <= s <= s_hi + 1,
 * so every symbol has frequency >= 1 and cum(s_hi + 1) = 2^16 - 1: the last
 * slot (frequency 1) is the escape for a symbol outside [s_lo, s_hi],
 * followed by e = 2 (s_lo - 1 - s) + 1 below the support or
 * e = 2 (s - s_hi - 1) above it, in 15-bit chunks as for one Gaussian.  The
 * decoder finds s by bisection on cum.
 */
#define MIX_FINE 16
#define MIX_QMAX (1 << 14)
#define MIX_WSUM 4096u
#define MIX_CDF_BITS 20
#define MIX_MAX_SYMBOLS (1 << 15)

int mix_tables_build(const float *table, int L, mix_tables *t)
{
    memset(t, 0, sizeof(*t));
    if (!table || L < 1) return -1;
    t->L = L;
    t->X = malloc((size_t)L * sizeof(int32_t));
    t->base = malloc(((size_t)L + 1) * sizeof(int64_t));
    if (!t->X || !t->base) { mix_tables_free(t); return -1; }
    int64_t total = 0;
    for (int l = 0; l < L; ++l) {
        t->X[l] = MIX_FINE * (support_of(table[l]) + 1);
        t->base[l] = total;
        total += 2 * (int64_t)t->X[l] + 1;
    }
    t->base[L] = total;
    t->G = malloc((size_t)total * sizeof(uint32_t));
    if (!t->G) { mix_tables_free(t); return -1; }
    for (int l = 0; l < L; ++l) {
        const double scale = MIX_FINE * (double)table[l] * sqrt(2.0);
        uint32_t *g = t->G + t->base[l];
        for (int x = -t->X[l]; x <= t->X[l]; ++x) {
            /* Phi(z) = erfc(-z / sqrt 2) / 2 */
            const double phi = 0.5 * erfc(-(double)x / scale);
            g[x + t->X[l]] = (uint32_t)floor(phi * (double)(1u << MIX_CDF_BITS) + 0.5);
        }
    }
    return 0;
}

void mix_tables_free(mix_tables *t)
{
    free(t->X); free(t->base); free(t->G);
    memset(t, 0, sizeof(*t));
}

static uint64_t mix_G(const mix_tables *t, int l, int64_t x)
{
    const int64_t X = t->X[l];
    if (x <= -X) return 0;
    if (x >= X) return 1u << MIX_CDF_BITS;
    return t->G[t->base[l] + x + X];
}

static int64_t floor_div16(int64_t a) { return a >= 0 ? a / MIX_FINE : -((-a + MIX_FINE - 1) / MIX_FINE); }

int mix_params(const mix_tables *t, const float *w, const float *cm, float mu, const int32_t *lvl, mix_param *p)
{
    uint32_t sum = 0;
    int top = 0;
    for (int k = 0; k < 3; ++k) {
        if (lvl[k] < 0 || lvl[k] >= t->L) return -1;
        p->l[k] = lvl[k];
        float wf = w[k] * 4093.0f;
        if (!(wf >= 0.0f)) wf = 0.0f;
        if (wf > 4093.0f) wf = 4093.0f;
        p->v[k] = 1u + (uint32_t)floorf(wf);
        sum += p->v[k];
        if (p->v[k] > p->v[top]) top = k;
        float d = rintf((cm[k] - mu) * (float)MIX_FINE);
        if (!(fabsf(d) <= (float)MIX_QMAX)) d = d > 0.0f ? (float)MIX_QMAX : -(float)MIX_QMAX;
        p->q[k] = (int32_t)d;
    }
    p->v[top] += MIX_WSUM - sum;
    int64_t lo = INT64_MAX, hi = INT64_MIN;
    for (int k = 0; k < 3; ++k) {
        const int64_t X = t->X[p->l[k]];
        const int64_t a = floor_div16(p->q[k] - X), b = -floor_div16(-(p->q[k] + X));
        if (a < lo) lo = a;
        if (b > hi) hi = b;
    }
    if (hi - lo + 1 > MIX_MAX_SYMBOLS) return -1;
    p->lo = (int32_t)lo;
    p->hi = (int32_t)hi;
    return 0;
}

/* F(s): the mixture CDF at the upper edge of symbol s, in units of 2^-32. */
static uint64_t mix_F(const mix_tables *t, const mix_param *p, int64_t s)
{
    uint64_t f = 0;
    for (int k = 0; k < 3; ++k) f += (uint64_t)p->v[k] * mix_G(t, p->l[k], MIX_FINE * s + MIX_FINE / 2 - p->q[k]);
    return f;
}

uint32_t mix_cum(const mix_tables *t, const mix_param *p, int64_t s)
{
    const uint64_t S = (uint64_t)((int64_t)p->hi - p->lo + 1);
    const uint64_t R = PREC_TOTAL - S - 1u;
    return (uint32_t)((uint64_t)(s - p->lo) + ((mix_F(t, p, s - 1) * R) >> 32));
}

static void mix_enc_symbol(rans_enc *e, const mix_tables *t, const mix_param *p, int32_t s)
{
    if (s >= p->lo && s <= p->hi) {
        const uint32_t c0 = mix_cum(t, p, s), c1 = mix_cum(t, p, (int64_t)s + 1);
        enc_push(e, c0, c1 - c0);
        return;
    }
    const uint64_t ev = s < p->lo ? 2u * (uint64_t)((int64_t)p->lo - 1 - s) + 1u
                                  : 2u * (uint64_t)((int64_t)s - p->hi - 1);
    uint32_t chunk[5];
    int nc = 0;
    uint64_t v = ev;
    do {
        chunk[nc++] = (uint32_t)(v & 0x7fffu);
        v >>= 15;
    } while (v);
    for (int q = 0; q < nc - 1; ++q) chunk[q] |= 0x8000u;
    for (int q = nc - 1; q >= 0; --q) enc_push(e, chunk[q], 1);
    enc_push(e, PREC_TOTAL - 1u, 1);
}

int mix_dec_symbol(rans_dec *d, const mix_tables *t, const mix_param *p, int32_t *s)
{
    const uint32_t slot = (uint32_t)(d->x & (PREC_TOTAL - 1u));
    int chunk;
    if (slot == PREC_TOTAL - 1u) {
        /* escape: frequency 1 at the last slot */
        d->x = d->x >> PREC_BITS;
        if (d->x < STATE_LOW) {
            if (d->w >= d->end) return -1;
            d->x = (d->x << 32) | *d->w++;
        }
        uint64_t ev = 0;
        for (int q = 0; q < 5; ++q) {
            if (dec_pop(d, NULL, 0, &chunk)) return -1;
            ev |= (uint64_t)(chunk & 0x7fff) << (15 * q);
            if (!(chunk & 0x8000)) {
                const int64_t v = (ev & 1u) ? (int64_t)p->lo - 1 - (int64_t)(ev >> 1) : (int64_t)p->hi + 1 + (int64_t)(ev >> 1);
                if (v < INT32_MIN || v > INT32_MAX) return -1;
                *s = (int32_t)v;
                return 0;
            }
        }
        return -1;
    }
    int64_t lo = p->lo, hi = p->hi;   /* the largest s with cum(s) <= slot */
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo + 1) / 2;
        if (mix_cum(t, p, mid) <= slot) lo = mid;
        else hi = mid - 1;
    }
    const uint32_t c0 = mix_cum(t, p, lo), c1 = mix_cum(t, p, lo + 1);
    d->x = (uint64_t)(c1 - c0) * (d->x >> PREC_BITS) + slot - c0;
    if (d->x < STATE_LOW) {
        if (d->w >= d->end) return -1;
        d->x = (d->x << 32) | *d->w++;
    }
    *s = (int32_t)lo;
    return 0;
}

/* The parameters of channel c of latent lat: weight, cmean, idx [lat][3][M], mean [lat][M]. */
static int mix_params_at(const mix_tables *t, const float *weight, const float *cmean, const float *mean,
                         const int32_t *idx, size_t lat, int M, int c, mix_param *p)
{
    float w[3], cm[3];
    int32_t l[3];
    for (int k = 0; k < 3; ++k) {
        const size_t q = (lat * 3 + k) * (size_t)M + c;
        w[k] = weight[q];
        cm[k] = cmean[q];
        l[k] = idx[q];
    }
    return mix_params(t, w, cm, mean[lat * (size_t)M + c], l, p);
}

int64_t oracle_mix_encode(const int32_t *sym, const float *weight, const float *cmean, const float *mean,
                          const int32_t *idx, int B, int H, int W, int M, const float *table, int L,
                          uint32_t *bits, int64_t cap, uint32_t *offsets)
{
    if (!sym || !weight || !cmean || !mean || !idx || !table || !offsets || B < 1 || H < 1 || W < 1 || M < 1)
        return -1;
    mix_tables t;
    if (mix_tables_build(table, L, &t)) return -1;
    const int64_t per = 2 + 4 * (int64_t)W;
    uint32_t *tmp = malloc((size_t)per * sizeof(uint32_t));
    if (!tmp) { mix_tables_free(&t); return -1; }
    int64_t pos = 0;
    int bad = 0;
    for (int b = 0; b < B && !bad; ++b)
        for (int i = 0; i < H && !bad; ++i)
            for (int ch = 0; ch < M && !bad; ++ch) {
                const int64_t k = ((int64_t)b * H + i) * M + ch;
                rans_enc e = {STATE_LOW, tmp, 0, per, 0};
                for (int j = W - 1; j >= 0; --j) {
                    const size_t lat = ((size_t)b * H + i) * W + j;
                    mix_param p;
                    if (mix_params_at(&t, weight, cmean, mean, idx, lat, M, ch, &p)) { bad = 1; break; }
                    mix_enc_symbol(&e, &t, &p, sym[lat * M + ch]);
                }
                if (bad || e.overflow || pos + 2 + e.n > (int64_t)UINT32_MAX) { bad = 1; break; }
                offsets[k] = (uint32_t)pos;
                if (bits && pos + 2 + e.n <= cap) {
                    bits[pos] = (uint32_t)(e.x >> 32);
                    bits[pos + 1] = (uint32_t)(e.x & 0xffffffffu);
                    for (int64_t q = 0; q < e.n; ++q) bits[pos + 2 + q] = tmp[e.n - 1 - q];
                } else if (bits) {
                    bad = 1;
                }
                pos += 2 + e.n;
            }
    free(tmp);
    mix_tables_free(&t);
    if (bad) return -1;
    offsets[(int64_t)B * H * M] = (uint32_t)pos;
    return pos;
}

int oracle_mix_decode(const uint32_t *bits, const uint32_t *offsets, const float *weight, const float *cmean,
                      const float *mean, const int32_t *idx, int B, int H, int W, int M, const float *table, int L,
                      int32_t *sym_out)
{
    if (!bits || !offsets || !weight || !cmean || !mean || !idx || !table || !sym_out) return -1;
    mix_tables t;
    if (mix_tables_build(table, L, &t)) return -1;
    int rc = 0;
    for (int b = 0; b < B && !rc; ++b)
        for (int i = 0; i < H && !rc; ++i)
            for (int ch = 0; ch < M && !rc; ++ch) {
                const int64_t k = ((int64_t)b * H + i) * M + ch;
                rans_dec d;
                if (rans_dec_init(&d, bits + offsets[k], (int64_t)offsets[k + 1] - offsets[k])) { rc = -1; break; }
                for (int j = 0; j < W; ++j) {
                    const size_t lat = ((size_t)b * H + i) * W + j;
                    mix_param p;
                    if (mix_params_at(&t, weight, cmean, mean, idx, lat, M, ch, &p) ||
                        mix_dec_symbol(&d, &t, &p, &sym_out[lat * M + ch])) { rc = -1; break; }
                }
            }
    mix_tables_free(&t);
    return rc;
}

/* The level tables (X [L], base [L+1], G [base[L]] when G != NULL and fits cap). */
int64_t oracle_mix_tables(const float *table, int L, int32_t *X, int64_t *base, uint32_t *G, int64_t cap)
{
    mix_tables t;
    if (mix_tables_build(table, L, &t)) return -1;
    const int64_t total = t.base[L];
    if (X) memcpy(X, t.X, (size_t)L * sizeof(int32_t));
    if (base) memcpy(base, t.base, ((size_t)L + 1) * sizeof(int64_t));
    if (G && total <= cap) memcpy(G, t.G, (size_t)total * sizeof(uint32_t));
    mix_tables_free(&t);
    return total;
}

/* One latent channel's quantised parameters and cumulative frequencies:
 * v, q, l [3], lo_hi [2], cum [S + 1] (cum[u] = cum(lo + u); when it fits cap).
 * Returns S, or -1. */
int oracle_mix_latent(const float *table, int L, const float *w, const float *cm, float mu, const int32_t *lvl,
                      uint32_t *v, int32_t *q, int32_t *lo_hi, uint32_t *cum, int64_t cap)
{
    mix_tables t;
    if (mix_tables_build(table, L, &t)) return -1;
    mix_param p;
    int rc = mix_params(&t, w, cm, mu, lvl, &p);
    if (!rc) {
        const int64_t S = (int64_t)p.hi - p.lo + 1;
        for (int k = 0; k < 3; ++k) { v[k] = p.v[k]; q[k] = p.q[k]; }
        lo_hi[0] = p.lo;
        lo_hi[1] = p.hi;
        if (cum && S + 1 <= cap)
            for (int64_t u = 0; u <= S; ++u) cum[u] = mix_cum(&t, &p, p.lo + u);
        rc = (int)S;
    }
    mix_tables_free(&t);
    return rc;
}

