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

#endif
