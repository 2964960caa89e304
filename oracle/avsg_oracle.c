/* avsg_oracle.c — plain CPU reference of the AVSG per-decode-step operator.
 *
 * TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the
 * benchmark's CPU-baseline leg are the only users.  Nothing here is shared with
 * the GPU library.
 *
 * The code is written from the AVSG paper (arXiv 2609.37538), in its order
 * and notation, with scalar loops and no blocking or fusion:
 *   - Section 3.2: Hash-State table, Eq. 1 (hit indicator), Eq. 2 (metadata
 *     word layout), Eq. 3 (packed mapping), Eq. 4 (reusable predicate);
 *   - Sections 3.3 and 3.5 (Algorithms 1-3): per token, each index is looked
 *     up (Eq. 8-11) and a hit renews its slot; the misses get the smallest
 *     reclaimable slots (Eq. 12) after as much ageing as needed, and each is
 *     linked to the first reusable bucket of its chain;
 *   - Section 3.6 (Algorithm 4): a request's tokens in order on one table,
 *     then speculative invalidation;
 *   - Section 3.4 and Appendix D: Stage Two and the S1/S2/S3 assignments
 *     (Eq. 5, 6, 13, 14);
 *   - Appendix F: metadata decode chain (Eq. 16-18).
 *
 * Readings where the paper leaves a choice (each is listed with its reason in
 * the design notes of the repository):
 *   - initial table: every c_j = -1, every lifetime -1, every bucket invalid
 *     with fingerprint 0 and slot 0;
 *   - a decay never takes a lifetime below -1 (only the sign of a lifetime is
 *     ever observed, and the 8-bit field must not wrap);
 *   - a lifetime write changes only the lifetime byte, a mapping install only
 *     the low 24 bits of the word (the install keeps the lifetime);
 *   - the reusable predicate of UpdateState reads the table as it is before
 *     that call's writes;
 *   - of several misses installing into one bucket, the one with the largest
 *     miss rank keeps the bucket (a sequential scatter in rank order);
 *   - phi(x) = x mod F is the non-negative remainder, so phi(-1) = F - 1;
 *   - speculative invalidation runs after Stage Two, as in Algorithm 4.
 */
#include "avsg_oracle.h"

#include <stdlib.h>
#include <string.h>

struct avsg_ref_state {
    avsg_ref_config cfg;
    int32_t m;       /* slot bit width, S = 2^m */
    int64_t S;       /* slots */
    int64_t F;       /* representable fingerprints, 2^23 / S */
    int32_t *c;      /* [B][S] cached selected index of slot j */
    uint32_t *q;     /* [B][S] metadata word of entry j (Eq. 2) */
    avsg_ref_counters *stats; /* [B] */
};

/* ------------------------------------------------------------------ */
/* Metadata word (Eq. 2, Eq. 3, Appendix F).  2FS = 2^24, FS = 2^23.   */
/* ------------------------------------------------------------------ */
#define TWO_FS 16777216LL
#define FS_ 8388608LL

static int64_t math_mod(int64_t a, int64_t n) { return ((a % n) + n) % n; }

/* u_h = q_h mod 2FS */
static int64_t field_u(uint32_t q) { return (int64_t)q % TWO_FS; }
/* b_h = floor(u_h / FS) */
static int32_t field_invalid(uint32_t q) { return (int32_t)(field_u(q) / FS_); }
/* o_h = u_h mod S */
static int64_t field_slot(const avsg_ref_state *st, uint32_t q) { return field_u(q) % st->S; }
/* phi_h = floor((u_h mod FS) / S) */
static int64_t field_phi(const avsg_ref_state *st, uint32_t q) {
    return (field_u(q) % FS_) / st->S;
}
/* lifetime: the top 8 bits, read as a two's-complement byte */
static int32_t field_life(uint32_t q) {
    int64_t v = (int64_t)q / TWO_FS; /* 0..255 */
    return (int32_t)(v >= 128 ? v - 256 : v);
}
/* Eq. 3: q = 2FS*l + FS*b + phi_hat + o, taken modulo 2^32 */
static uint32_t pack_word(const avsg_ref_state *st, int32_t l, int32_t b, int64_t phi, int64_t o) {
    int64_t v = TWO_FS * (int64_t)l + FS_ * (int64_t)b + phi * st->S + o;
    return (uint32_t)(uint64_t)v;
}
static uint32_t with_life(uint32_t q, int32_t l) {
    int64_t v = TWO_FS * (int64_t)l + field_u(q);
    return (uint32_t)(uint64_t)v;
}
/* phi(x) = x mod F;  phi_hat(x) = phi(x) * S  (Section 3.3) */
static int64_t phi_of(const avsg_ref_state *st, int64_t x) { return math_mod(x, st->F); }

/* ------------------------------------------------------------------ */
/* configuration                                                       */
/* ------------------------------------------------------------------ */
static int is_prime_u32(uint32_t v) {
    if (v < 2) return 0;
    if (v % 2 == 0) return v == 2;
    for (uint64_t d = 3; d * d <= v; d += 2)
        if (v % d == 0) return 0;
    return 1;
}

avsg_ref_state *avsg_ref_create(const avsg_ref_config *cfg, int32_t *status) {
    int32_t s = 0;
    if (!cfg || cfg->batch < 1 || cfg->topk < 1 || cfg->n_q < 1) s = -1;
    else if (cfg->slots < 2 || (cfg->slots & (cfg->slots - 1)) != 0 || cfg->slots > (1 << 23)) s = -2;
    else if ((int64_t)cfg->slots < (int64_t)cfg->n_q * cfg->topk) s = -3; /* Eq. 7 */
    else if (cfg->retry < 0 || cfg->max_life < 1 || cfg->max_life > 127 || cfg->a1 == cfg->a2 ||
             !is_prime_u32(cfg->a1) || !is_prime_u32(cfg->a2))
        s = -4;
    if (status) *status = s;
    if (s) return NULL;
    avsg_ref_state *st = (avsg_ref_state *)calloc(1, sizeof(*st));
    st->cfg = *cfg;
    st->S = cfg->slots;
    st->m = 0;
    while ((1LL << st->m) < st->S) st->m++;
    st->F = (1LL << 23) / st->S;
    size_t n = (size_t)cfg->batch * (size_t)st->S;
    st->c = (int32_t *)malloc(n * sizeof(int32_t));
    st->q = (uint32_t *)malloc(n * sizeof(uint32_t));
    st->stats = (avsg_ref_counters *)calloc((size_t)cfg->batch, sizeof(avsg_ref_counters));
    /* initial table: empty slots, dead lifetimes, invalid buckets */
    for (size_t j = 0; j < n; ++j) {
        st->c[j] = -1;
        st->q[j] = pack_word(st, -1, 1, 0, 0);
    }
    return st;
}

void avsg_ref_destroy(avsg_ref_state *st) {
    if (!st) return;
    free(st->c);
    free(st->q);
    free(st->stats);
    free(st);
}

/* ------------------------------------------------------------------ */
/* one request's table                                                 */
/* ------------------------------------------------------------------ */
typedef struct {
    const avsg_ref_state *st;
    int32_t *c;   /* this request's c_j */
    uint32_t *q;  /* this request's q_j */
} table_view;

static int64_t initial_bucket(const avsg_ref_state *st, int32_t x) { /* Eq. 9 */
    return (int64_t)(((uint64_t)st->cfg.a1 * (uint64_t)(int64_t)x) % (uint64_t)st->S);
}
static int64_t stride_of(const avsg_ref_state *st, int32_t x) { /* Eq. 9, odd stride */
    return (int64_t)(((uint64_t)st->cfg.a2 * (uint64_t)(int64_t)x) % (uint64_t)st->S) | 1;
}

/* The lookup of one selected index (Eq. 8-11): walks x's chain of R+1
 * buckets and stops at the first bucket whose slot field names a slot that
 * caches x.  Returns the hit flag m; *h_out is the matching bucket on a hit,
 * the last bucket examined on a miss.  Reads slot fields and ids only. */
static int32_t find_index(const table_view *t, int32_t x, int64_t *h_out) {
    const avsg_ref_state *st = t->st;
    const int64_t d = stride_of(st, x);
    int64_t h = initial_bucket(st, x);
    int32_t hit = 0;
    for (int32_t r = 0; r <= st->cfg.retry; ++r) {
        if (r > 0) h = (h + d) % st->S;                 /* Eq. 11: only an unresolved probe moves on */
        hit = (t->c[(int64_t)t->q[h] % st->S] == x);    /* Eq. 10 */
        if (hit) break;
    }
    *h_out = h;
    return hit;
}

/* One unit of ageing for every slot, never below -1 (reading I4). */
static void age_table(table_view *t) {
    for (int64_t j = 0; j < t->st->S; ++j) {
        int32_t l = field_life(t->q[j]);
        t->q[j] = with_life(t->q[j], l > -1 ? l - 1 : -1);
    }
}

/* The reclaimable slots (Eq. 12): every slot whose lifetime is negative, in
 * increasing slot order.  Returns how many there are. */
static int64_t list_dead(const table_view *t, int32_t *dead) {
    int64_t n = 0;
    for (int64_t j = 0; j < t->st->S; ++j)
        if (field_life(t->q[j]) < 0) dead[n++] = (int32_t)j;
    return n;
}

/* Eq. 4: a bucket may take a new mapping when its own mapping is invalid,
 * when the slot it names is inactive, or when its stored fingerprint is no
 * longer that of the slot's occupant. */
static int bucket_reusable(const table_view *t, uint32_t qh) {
    const avsg_ref_state *st = t->st;
    const int64_t o = field_slot(st, qh);
    const int invalid = field_invalid(qh) != 0;
    const int inactive = field_life(t->q[o]) < 0;
    const int stale = field_phi(st, qh) != phi_of(st, t->c[o]);
    return invalid || inactive || stale;
}

/* The install bucket of a missed index: the first reusable bucket among the
 * R+1 of its chain (the chain of Eq. 9, 11), in *h_out.  Returns 0 when all
 * R+1 buckets hold live mappings (the index is cached but not mapped). */
static int find_install_bucket(const table_view *t, int32_t x, int64_t *h_out) {
    const avsg_ref_state *st = t->st;
    const int64_t d = stride_of(st, x);
    int64_t h = initial_bucket(st, x);
    for (int32_t r = 0; r <= st->cfg.retry; ++r) {
        if (r > 0) h = (h + d) % st->S;
        if (bucket_reusable(t, t->q[h])) {
            *h_out = h;
            return 1;
        }
    }
    *h_out = h;
    return 0;
}

typedef struct {
    int32_t *pending;   /* [K] positions of the token's misses, increasing */
    int32_t *dead;      /* [S] reclaimable slots */
    int32_t *found;     /* [K] the miss found an install bucket */
    int64_t *bucket;    /* [K] its install bucket */
} token_scratch;

/* Token g of one request (Section 3.3 with the lifetime rules of Section 3.5;
 * Algorithm 1, whose lifetime steps Algorithm 3 restates, and Algorithm 2 for
 * the installs).  Writes the token's slots into o[K], its misses (index,
 * slot), in increasing position, into miss_x / miss_o, and returns their
 * number n_g. */
static int64_t run_token(table_view *t, int32_t g, const int32_t *x, int32_t *o, int32_t *miss_x,
                         int32_t *miss_o, token_scratch *w, avsg_ref_counters *stats,
                         int32_t *step_decays) {
    const avsg_ref_state *st = t->st;
    const int32_t K = st->cfg.topk, L = st->cfg.max_life;

    /* the request's first token ages every slot once (global pre-decay) */
    if (g == 0) age_table(t);

    /* each index on its own: a hit renews its slot's lifetime to L.  The
     * lookup reads slot fields and ids, the renewal writes a lifetime byte
     * only (reading I5), so renewing before the next lookup changes nothing */
    int64_t n_g = 0;
    for (int32_t i = 0; i < K; ++i) {
        int64_t h;
        if (find_index(t, x[i], &h)) {
            const int64_t slot = field_slot(st, t->q[h]);
            if (field_life(t->q[slot]) < 0) stats->revivals++;   /* reading I9 */
            t->q[slot] = with_life(t->q[slot], L);
            o[i] = (int32_t)slot;
        } else {
            w->pending[n_g++] = i;
        }
    }
    stats->hits += (uint64_t)(K - n_g);
    stats->misses += (uint64_t)n_g;
    if (n_g == 0) return 0;   /* reading I11 */

    /* enough reclaimable slots for the misses: further unit ageing of every
     * slot until there are (Eq. 12) */
    int64_t n_dead = list_dead(t, w->dead);
    while (n_dead < n_g) {
        age_table(t);
        (*step_decays)++;
        stats->alloc_decays++;
        n_dead = list_dead(t, w->dead);
    }

    /* every miss's install bucket is chosen on the table as it is before any
     * of this token's writes (reading I6) */
    for (int64_t k = 0; k < n_g; ++k)
        w->found[k] = find_install_bucket(t, x[w->pending[k]], &w->bucket[k]);

    /* the k-th miss (by position) takes the k-th smallest reclaimable slot
     * (reading I10): the slot caches the index with lifetime L, and a found
     * bucket is linked to it with the index's fingerprint (Eq. 3, keeping the
     * bucket's own lifetime, reading I5).  A later miss linking the same bucket
     * replaces an earlier one (reading I7). */
    for (int64_t k = 0; k < n_g; ++k) {
        const int32_t xk = x[w->pending[k]];
        const int32_t slot = w->dead[k];
        t->c[slot] = xk;
        t->q[slot] = with_life(t->q[slot], L);
        if (w->found[k]) {
            const int64_t h = w->bucket[k];
            t->q[h] = pack_word(st, field_life(t->q[h]), 0, phi_of(st, xk), slot);
        }
        o[w->pending[k]] = slot;
        miss_x[k] = xk;
        miss_o[k] = slot;
    }
    /* installs that did not stick: no reusable bucket, or a later miss took it */
    for (int64_t k = 0; k < n_g; ++k) {
        if (!w->found[k]) stats->lost_exhausted++;
        else if (field_slot(st, t->q[w->bucket[k]]) != miss_o[k]) stats->lost_collision++;
    }
    return n_g;
}

/* Stage One for request r: its tokens in order on the shared table
 * (Algorithm 4); the transfer list is the tokens' misses in order. */
static void stage_one(avsg_ref_state *st, int32_t r, const int32_t *X, int32_t *O, int32_t *n,
                      int32_t *miss_x, int32_t *miss_o) {
    const int32_t K = st->cfg.topk, Nq = st->cfg.n_q;
    const int64_t S = st->S;
    table_view t = {st, st->c + (size_t)r * S, st->q + (size_t)r * S};
    token_scratch w;
    w.pending = (int32_t *)malloc(sizeof(int32_t) * K);
    w.dead = (int32_t *)malloc(sizeof(int32_t) * S);
    w.found = (int32_t *)malloc(sizeof(int32_t) * K);
    w.bucket = (int64_t *)malloc(sizeof(int64_t) * K);
    avsg_ref_counters *stats = &st->stats[r];
    int32_t step_decays = 0;
    int64_t listed = 0;
    const size_t lbase = (size_t)r * Nq * K;
    for (int32_t g = 0; g < Nq; ++g) {
        const size_t xo = ((size_t)r * Nq + g) * K;
        const int64_t n_g = run_token(&t, g, X + xo, O + xo, miss_x + lbase + listed,
                                      miss_o + lbase + listed, &w, stats, &step_decays);
        n[(size_t)r * Nq + g] = (int32_t)n_g;
        listed += n_g;
    }
    if (step_decays > stats->max_step_alloc_decays) stats->max_step_alloc_decays = step_decays;
    free(w.pending); free(w.dead); free(w.found); free(w.bucket);
}

/* Stage Two: copy every listed miss from its host row to its buffer slot. */
static void stage_two(int32_t B, int32_t r, int64_t per_req, int64_t total, const int32_t *miss_x,
                      const int32_t *miss_o, int32_t n_streams, const void *const *host,
                      void *const *buf, const int64_t *row_bytes) {
    for (int32_t s = 0; s < n_streams; ++s) {
        const uint8_t *src = (const uint8_t *)host[(size_t)s * B + r];
        uint8_t *dst = (uint8_t *)buf[(size_t)s * B + r];
        const int64_t rb = row_bytes[s];
        for (int64_t k = 0; k < total; ++k) {
            const size_t e = (size_t)r * per_req + k;
            memcpy(dst + (int64_t)miss_o[e] * rb, src + (int64_t)miss_x[e] * rb, (size_t)rb);
        }
    }
}

int32_t avsg_ref_step(avsg_ref_state *st, const int32_t *X, const int64_t *verified, int32_t *O,
                      int32_t *n, int32_t *miss_x, int32_t *miss_o, int32_t n_streams,
                      const void *const *host, void *const *buf, const int64_t *row_bytes,
                      const int64_t *rows, int32_t nthreads) {
    const int32_t B = st->cfg.batch, K = st->cfg.topk, Nq = st->cfg.n_q;
    const int64_t per_req = (int64_t)Nq * K;
    if (rows) {
        for (int32_t r = 0; r < B; ++r)
            for (int64_t i = 0; i < per_req; ++i) {
                int32_t x = X[(size_t)r * per_req + i];
                if (x < 0 || x >= rows[r]) return -5;
            }
    }
    if (nthreads < 1) nthreads = 1;
    /* Stage One (all tokens of every request, requests independent) */
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
    for (int32_t r = 0; r < B; ++r) stage_one(st, r, X, O, n, miss_x, miss_o);
    /* Stage Two */
    if (n_streams > 0) {
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
        for (int32_t r = 0; r < B; ++r) {
            int64_t total = 0;
            for (int32_t g = 0; g < Nq; ++g) total += n[(size_t)r * Nq + g];
            stage_two(B, r, per_req, total, miss_x, miss_o, n_streams, host, buf, row_bytes);
        }
    }
    /* end of step: speculative invalidation (c_j >= N -> -1) */
    if (verified) {
        for (int32_t r = 0; r < B; ++r) {
            int32_t *c = st->c + (size_t)r * st->S;
            for (int64_t j = 0; j < st->S; ++j)
                if ((int64_t)c[j] >= verified[r]) {
                    c[j] = -1;
                    st->stats[r].invalidations++;
                }
        }
    }
    return 0;
}

static int cmp_i32(const void *a, const void *b) {
    const int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

void avsg_ref_validate(const int32_t *X, int32_t B, int32_t n_q, int32_t K, const int64_t *rows,
                       int32_t *verdict) {
    int32_t *in_range = (int32_t *)malloc(sizeof(int32_t) * (size_t)K);
    for (int64_t row = 0; row < (int64_t)B * n_q; ++row) {
        const int32_t *x = X + (size_t)row * K;
        const int64_t n_rows = rows[row / n_q];
        int32_t v = 0, n = 0;
        for (int32_t i = 0; i < K; ++i) {
            if (x[i] < 0 || (int64_t)x[i] >= n_rows) v |= 1;
            else in_range[n++] = x[i];
        }
        /* a repeated index sits next to its copy once the row is sorted */
        qsort(in_range, (size_t)n, sizeof(int32_t), cmp_i32);
        for (int32_t i = 1; i < n; ++i)
            if (in_range[i] == in_range[i - 1]) v |= 2;
        verdict[row] = v;
    }
    free(in_range);
}

void avsg_ref_export(const avsg_ref_state *st, int32_t r, int32_t *c, uint32_t *q) {
    memcpy(c, st->c + (size_t)r * st->S, sizeof(int32_t) * (size_t)st->S);
    memcpy(q, st->q + (size_t)r * st->S, sizeof(uint32_t) * (size_t)st->S);
}

void avsg_ref_import(avsg_ref_state *st, int32_t r, const int32_t *c, const uint32_t *q) {
    memcpy(st->c + (size_t)r * st->S, c, sizeof(int32_t) * (size_t)st->S);
    memcpy(st->q + (size_t)r * st->S, q, sizeof(uint32_t) * (size_t)st->S);
}

void avsg_ref_stats(const avsg_ref_state *st, int32_t r, avsg_ref_counters *out) {
    *out = st->stats[r];
}

/* ------------------------------------------------------------------ */
/* exported word helpers                                               */
/* ------------------------------------------------------------------ */
static avsg_ref_state word_ctx(int32_t m) {
    avsg_ref_state st;
    memset(&st, 0, sizeof(st));
    st.m = m;
    st.S = 1LL << m;
    st.F = (1LL << 23) / st.S;
    return st;
}

uint32_t avsg_ref_pack(int32_t m, int32_t lifetime, int32_t invalid, int64_t fingerprint,
                       int64_t slot) {
    avsg_ref_state st = word_ctx(m);
    return pack_word(&st, lifetime, invalid, fingerprint, slot);
}

void avsg_ref_decode(int32_t m, uint32_t q, int32_t *lifetime, int32_t *invalid,
                     int64_t *fingerprint, int64_t *slot) {
    avsg_ref_state st = word_ctx(m);
    *lifetime = field_life(q);
    *invalid = field_invalid(q);
    *fingerprint = field_phi(&st, q);
    *slot = field_slot(&st, q);
}

int64_t avsg_ref_phi(int32_t m, int64_t x) {
    avsg_ref_state st = word_ctx(m);
    return phi_of(&st, x);
}

void avsg_ref_probe(const avsg_ref_state *st, int32_t r, int32_t x, int32_t *hit, int32_t *h) {
    table_view t = {st, st->c + (size_t)r * st->S, st->q + (size_t)r * st->S};
    int64_t hh;
    *hit = find_index(&t, x, &hh);
    *h = (int32_t)hh;
}

/* ------------------------------------------------------------------ */
/* scalar dual-pointer matching (the sort-merge baseline, S = K)       */
/* ------------------------------------------------------------------ */
struct avsg_ref_dp {
    int32_t B, K;
    int32_t *cached; /* [B][K] id held by slot j, -1 when empty */
};

typedef struct {
    int32_t id, pos;
} id_pos;

static int cmp_id_pos(const void *a, const void *b) {
    const id_pos *x = (const id_pos *)a, *y = (const id_pos *)b;
    if (x->id != y->id) return x->id < y->id ? -1 : 1;
    return x->pos < y->pos ? -1 : (x->pos > y->pos);
}

avsg_ref_dp *avsg_ref_dp_create(int32_t batch, int32_t topk) {
    if (batch < 1 || topk < 1) return NULL;
    avsg_ref_dp *dp = (avsg_ref_dp *)calloc(1, sizeof(*dp));
    dp->B = batch;
    dp->K = topk;
    dp->cached = (int32_t *)malloc(sizeof(int32_t) * (size_t)batch * topk);
    for (size_t j = 0; j < (size_t)batch * topk; ++j) dp->cached[j] = -1;
    return dp;
}

void avsg_ref_dp_destroy(avsg_ref_dp *dp) {
    if (!dp) return;
    free(dp->cached);
    free(dp);
}

static int32_t dp_request(avsg_ref_dp *dp, int32_t r, const int32_t *x, int32_t *o,
                          int32_t *miss_x, int32_t *miss_o) {
    const int32_t K = dp->K;
    int32_t *cached = dp->cached + (size_t)r * K;
    id_pos *cs = (id_pos *)malloc(sizeof(id_pos) * K);
    id_pos *xs = (id_pos *)malloc(sizeof(id_pos) * K);
    char *used = (char *)calloc((size_t)K, 1);
    int32_t nc = 0;
    for (int32_t j = 0; j < K; ++j)
        if (cached[j] >= 0) { cs[nc].id = cached[j]; cs[nc].pos = j; nc++; }
    for (int32_t i = 0; i < K; ++i) { xs[i].id = x[i]; xs[i].pos = i; }
    qsort(cs, (size_t)nc, sizeof(id_pos), cmp_id_pos);
    qsort(xs, (size_t)K, sizeof(id_pos), cmp_id_pos);
    /* the two-pointer merge: equal ids keep their slot, the rest miss */
    int32_t p = 0, nm = 0;
    for (int32_t qi = 0; qi < K;) {
        if (p < nc && cs[p].id < xs[qi].id) {
            p++;
        } else if (p < nc && cs[p].id == xs[qi].id) {
            o[xs[qi].pos] = cs[p].pos;
            used[cs[p].pos] = 1;
            p++;
            qi++;
        } else {
            xs[nm++] = xs[qi];   /* compacted in increasing id order (nm <= qi) */
            qi++;
        }
    }
    /* freed slots in increasing slot order go to the misses in increasing id order */
    int32_t k = 0;
    for (int32_t j = 0; j < K && k < nm; ++j) {
        if (used[j]) continue;
        o[xs[k].pos] = j;
        cached[j] = xs[k].id;
        miss_x[k] = xs[k].id;
        miss_o[k] = j;
        k++;
    }
    free(cs); free(xs); free(used);
    return nm;
}

int32_t avsg_ref_dp_step(avsg_ref_dp *dp, const int32_t *X, int32_t *O, int32_t *n,
                         int32_t *miss_x, int32_t *miss_o, int32_t n_streams,
                         const void *const *host, void *const *buf, const int64_t *row_bytes,
                         int32_t nthreads) {
    const int32_t B = dp->B, K = dp->K;
    if (nthreads < 1) nthreads = 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
    for (int32_t r = 0; r < B; ++r) {
        const size_t off = (size_t)r * K;
        n[r] = dp_request(dp, r, X + off, O + off, miss_x + off, miss_o + off);
    }
    if (n_streams > 0) {
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
        for (int32_t r = 0; r < B; ++r)
            stage_two(B, r, K, n[r], miss_x, miss_o, n_streams, host, buf, row_bytes);
    }
    return 0;
}

void avsg_ref_dp_export(const avsg_ref_dp *dp, int32_t r, int32_t *cached) {
    memcpy(cached, dp->cached + (size_t)r * dp->K, sizeof(int32_t) * (size_t)dp->K);
}

/* ------------------------------------------------------------------ */
/* Stage Two work assignment (Appendix D)                              */
/* ------------------------------------------------------------------ */
void avsg_ref_partition_balanced(int64_t n_miss, int32_t C, int64_t *begin) {
    /* Eq. 6: consecutive misses, floor or ceil of N_miss / C per worker */
    for (int32_t c = 0; c <= C; ++c) begin[c] = (int64_t)(((__int128)c * n_miss) / C);
}

void avsg_ref_partition_request(int32_t B, int32_t C, int32_t n_q, int32_t K, int64_t *positions) {
    /* Eq. 13: one extra request on each of the first B mod C workers */
    const int32_t rB = B % C;
    for (int32_t c = 0; c < C; ++c)
        positions[c] = (int64_t)(B / C + (c < rB ? 1 : 0)) * n_q * K;
}

void avsg_ref_partition_position(int64_t n_positions, int32_t C, int64_t *begin) {
    /* Eq. 14: near-equal contiguous ranges of the flattened positions */
    for (int32_t c = 0; c <= C; ++c) begin[c] = (int64_t)(((__int128)c * n_positions) / C);
}
