/*
 * rANS entropy coding of the symbols of a mean-scale Gaussian entropy model
 * (the oracle's side; TEST INFRASTRUCTURE ONLY, see wf_rans.c).
 */
#ifndef WF_RANS_H
#define WF_RANS_H

#include <stdint.h>

/* Per-level tables of one scale table. */
typedef struct {
    int L;
    int32_t *n;       /* [L] support half-width of each level                  */
    int64_t *base;    /* [L+1] first entry of each level's cumulative array    */
    uint32_t *cum;    /* [base[L]] cumulative frequencies, 2n+3 per level      */
} rans_tables;

int rans_tables_build(const float *table, int L, rans_tables *t);
void rans_tables_free(rans_tables *t);

/* Decoder state of one stream. */
typedef struct {
    uint64_t x;
    const uint32_t *w;    /* next word */
    const uint32_t *end;  /* one past the stream's last word */
} rans_dec;

/* Start decoding the stream of `n_words` words at `w`; -1 if too short. */
int rans_dec_init(rans_dec *d, const uint32_t *w, int64_t n_words);
/* Decode one symbol at scale level `level`; -1 on a malformed stream. */
int rans_dec_symbol(rans_dec *d, const rans_tables *t, int level, int32_t *s);

/* Mixture model (K = 3): per-level integer CDFs on sixteenths of a symbol. */
typedef struct {
    int L;
    int32_t *X;       /* [L] half-width of each level's table, in sixteenths    */
    int64_t *base;    /* [L+1] first entry of each level                        */
    uint32_t *G;      /* [base[L]] G_l(x) for x = -X_l..X_l                      */
} mix_tables;

/* Quantised parameters of one latent channel. */
typedef struct {
    uint32_t v[3];    /* weights, summing to 4096                               */
    int32_t q[3];     /* component mean minus mixture mean, in sixteenths       */
    int32_t l[3];     /* scale levels                                           */
    int32_t lo, hi;   /* coded symbols s_lo..s_hi (others escape)               */
} mix_param;

int mix_tables_build(const float *table, int L, mix_tables *t);
void mix_tables_free(mix_tables *t);
int mix_params(const mix_tables *t, const float *w, const float *cm, float mu, const int32_t *lvl, mix_param *p);
uint32_t mix_cum(const mix_tables *t, const mix_param *p, int64_t s);
int mix_dec_symbol(rans_dec *d, const mix_tables *t, const mix_param *p, int32_t *s);

#endif
