/* avsg_oracle.h — plain CPU reference of the AVSG per-decode-step operator.
 *
 * TEST INFRASTRUCTURE ONLY.  This header and avsg_oracle.c exist to check the
 * GPU implementation; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load them.  They share no code, header, table or helper
 * with the GPU library.
 *
 * Everything here is written from the AVSG paper (Accelerated Vectorized Sparse
 * Gather, arXiv 2609.37538): Section 3 (method), Appendix B (Probe, UpdateState,
 * CollectDead, life-cycle update, MTP-aware processing), Appendix D (core
 * binding strategies) and Appendix F (metadata decode chain).
 */
#ifndef AVSG_ORACLE_H
#define AVSG_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t batch;     /* B: requests */
    int32_t topk;      /* K: selected indices per query token */
    int32_t n_q;       /* N_q = N_mtp + 1 query tokens per request per step */
    int32_t slots;     /* S = 2^m slots per request (Section 3.2) */
    int32_t retry;     /* R: probe retry budget, R+1 buckets per chain */
    int32_t max_life;  /* L: lifetime a hit or a new slot is set to */
    uint32_t a1, a2;   /* the two distinct primes of the probe (Eq. 9) */
} avsg_ref_config;

typedef struct {
    uint64_t hits, misses;
    uint64_t lost_exhausted;   /* misses whose install chain found no reusable bucket */
    uint64_t lost_collision;   /* misses whose mapping was overwritten in the same scatter */
    uint64_t alloc_decays;     /* unit decays done by the allocation loop */
    uint64_t revivals;         /* hits on a slot whose lifetime was negative */
    uint64_t invalidations;    /* cached ids cleared by speculative invalidation */
    int32_t max_step_alloc_decays; /* largest allocation-decay count of one request-step */
    int32_t pad;
} avsg_ref_counters;

typedef struct avsg_ref_state avsg_ref_state;

/* Status: 0 ok, negative on a bad configuration (same meaning as the codes of
 * the GPU library, but defined independently). */
avsg_ref_state *avsg_ref_create(const avsg_ref_config *cfg, int32_t *status);
void avsg_ref_destroy(avsg_ref_state *st);

/* One decode step (Algorithm 4) for all requests.
 *   X         [B][n_q][K] selected indices (host)
 *   verified  [B] verified context length N per request, or NULL (no
 *             speculative invalidation)
 *   O         [B][n_q][K] out: slot of every selected index
 *   n         [B][n_q]    out: miss count of every token
 *   miss_x, miss_o [B][n_q*K] out: each request's transfer list, ordered by
 *             token then by position inside the token; entries past the
 *             request's miss total are left untouched
 *   Gather (Stage Two) runs when n_streams > 0: for stream s and request r the
 *   host rows start at host[s*B + r] and the device-buffer image at
 *   buf[s*B + r]; rows are row_bytes[s] long.  rows[r] bounds the ids of r.
 * Returns 0, or -5 if an id lies outside [0, rows[r]) when rows is given. */
int32_t avsg_ref_step(avsg_ref_state *st, const int32_t *X, const int64_t *verified,
                      int32_t *O, int32_t *n, int32_t *miss_x, int32_t *miss_o,
                      int32_t n_streams, const void *const *host, void *const *buf,
                      const int64_t *row_bytes, const int64_t *rows, int32_t nthreads);

/* Selection check (Section 3.2 "Problem formulation": every token contributes
 * a top-K list of K selected positions of its request's context).  For each
 * token row X[r][g] (row index r * n_q + g): verdict = 1 if some index lies
 * outside [0, rows[r]), plus 2 if some index inside [0, rows[r]) occurs more
 * than once in the row, else 0. */
void avsg_ref_validate(const int32_t *X, int32_t B, int32_t n_q, int32_t K, const int64_t *rows,
                       int32_t *verdict);

/* Canonical table view of request r: c_j and the packed metadata word q_j. */
void avsg_ref_export(const avsg_ref_state *st, int32_t r, int32_t *c, uint32_t *q);
/* Replace request r's table (used to set up hand-made states in tests). */
void avsg_ref_import(avsg_ref_state *st, int32_t r, const int32_t *c, const uint32_t *q);
void avsg_ref_stats(const avsg_ref_state *st, int32_t r, avsg_ref_counters *out);

/* Metadata word helpers (Eq. 2, Eq. 3, Appendix F), for tests. */
uint32_t avsg_ref_pack(int32_t m, int32_t lifetime, int32_t invalid, int64_t fingerprint,
                       int64_t slot);
void avsg_ref_decode(int32_t m, uint32_t q, int32_t *lifetime, int32_t *invalid,
                     int64_t *fingerprint, int64_t *slot);
int64_t avsg_ref_phi(int32_t m, int64_t x);

/* Probe of one index against request r's current table (Eq. 8-11). */
void avsg_ref_probe(const avsg_ref_state *st, int32_t r, int32_t x, int32_t *hit, int32_t *h);

/* Scalar dual-pointer (sort-merge) matching baseline, buffer of S = K slots. */
typedef struct avsg_ref_dp avsg_ref_dp;
avsg_ref_dp *avsg_ref_dp_create(int32_t batch, int32_t topk);
void avsg_ref_dp_destroy(avsg_ref_dp *dp);
/* One step, one query token per request.  Same output layout as
 * avsg_ref_step with n_q = 1; the transfer list is in increasing id order. */
int32_t avsg_ref_dp_step(avsg_ref_dp *dp, const int32_t *X, int32_t *O, int32_t *n,
                         int32_t *miss_x, int32_t *miss_o, int32_t n_streams,
                         const void *const *host, void *const *buf, const int64_t *row_bytes,
                         int32_t nthreads);
void avsg_ref_dp_export(const avsg_ref_dp *dp, int32_t r, int32_t *cached);

/* Stage Two work assignment over C workers (Appendix D).
 * Balanced miss list (Eq. 6): begin[c] for c = 0..C, worker c owns
 *   list entries [begin[c], begin[c+1]).
 * Request level (Eq. 13): positions[c] assigned to worker c. */
void avsg_ref_partition_balanced(int64_t n_miss, int32_t C, int64_t *begin);
void avsg_ref_partition_request(int32_t B, int32_t C, int32_t n_q, int32_t K,
                                int64_t *positions);
/* Equal top-K position ranges (Eq. 14): begin[c] for c = 0..C over N_g*K. */
void avsg_ref_partition_position(int64_t n_positions, int32_t C, int64_t *begin);

#ifdef __cplusplus
}
#endif
#endif
