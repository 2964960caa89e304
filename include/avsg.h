/* avsg.h — C ABI of the MI355X (gfx950) implementation of AVSG's per-decode-step
 * sparse-gather operator (Accelerated Vectorized Sparse Gather, arXiv 2609.37538).
 *
 * Per decode step, for every request r of a batch of B requests and every one
 * of its N_q query tokens (the initial token plus N_mtp speculative ones,
 * Section 3.2 "Problem formulation"), the operator takes the K token indices the
 * sparse-attention indexer selected and
 *   1. matches them against the request's persistent S-slot Hash-State table
 *      (Section 3.2, Eq. 1-4; Probe, Eq. 8-11),
 *   2. reserves slots for the misses with lifetime-based eviction
 *      (Section 3.3 Algorithm 1, Section 3.5, CollectDead Eq. 12, Algorithms 2-3),
 *   3. shares those reservations across the N_q tokens of the step
 *      (Section 3.6, Algorithm 4), and
 *   4. copies only the missed rows from host memory into the reserved slots of
 *      the device buffer, with the miss list split evenly over all workers
 *      (Section 3.4, Eq. 5-6).
 * At the end of the step every cached index >= the verified context length N
 * is cleared (speculative invalidation, Section 3.6 and Algorithm 4).
 *
 * Conventions for every entry point:
 *   - Memory is owned by the caller: pinned host rows, the device workspace,
 *     the device buffers and the step outputs.  The handle owns host-side
 *     bookkeeping and HIP events only.
 *   - "device" pointers are HIP device memory of the current device; "host"
 *     pointers are ordinary host memory unless stated otherwise.
 *   - Calls return an avsg_status; they never throw and never abort.  A
 *     negative status leaves the handle usable; avsg_last_error() gives detail.
 *   - avsg_step is asynchronous on the given stream.  Calls on one handle are
 *     not thread-safe and must be ordered by the caller.
 *   - Nothing here allocates device memory except avsg_host_alloc (pinned host
 *     memory) and the HIP events/staging kept by a handle; avsg_step_static
 *     allocates nothing at all.
 */
#ifndef AVSG_H
#define AVSG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t avsg_status;

#define AVSG_OK 0
#define AVSG_E_INVAL (-1)       /* null pointer, non-positive size, bad mode */
#define AVSG_E_NOTPOW2 (-2)     /* S is not a power of two in [2, 2^23] */
#define AVSG_E_CAPACITY (-3)    /* S < N_q * K (Eq. 7), or 9*S + 12*K bytes beyond one workgroup's LDS
                                   (or, resident reuse, no room beside the table for a map of 1.5*N_q*K
                                   words and S fan words) */
#define AVSG_E_RANGE (-4)       /* R < 0, L outside [1, 127], a1/a2 not distinct primes, row size */
#define AVSG_E_BADINDEX (-5)    /* validate mode: a selected index outside [0, rows of its request), or an
                                   index repeated within one token's top-K list */
#define AVSG_E_HIP (-6)         /* a HIP runtime call failed */
#define AVSG_E_INTERNAL (-7)    /* broken internal invariant */
#define AVSG_E_UNSUPPORTED (-8) /* valid but unsupported combination (e.g. dual-pointer with N_q > 1) */

/* Stage One matching algorithm. */
#define AVSG_MATCH_HASH 0     /* vectorized open-addressing hash matching (Section 3.3) */
#define AVSG_MATCH_DUALPTR 1  /* scalar dual-pointer sort-merge baseline, needs S == K (Appendix C) */

/* Stage Two work assignment (Appendix D). */
#define AVSG_GATHER_BALANCED 0 /* S3: the miss list split into floor/ceil(N_miss/C) consecutive misses per worker (Eq. 6) */
#define AVSG_GATHER_REQUEST 1  /* S1: one worker per request (Eq. 13) */
#define AVSG_GATHER_SDMA 2     /* comparator: the miss list is read back and every missed row is one hipMemcpyAsync on the copy engines */
#define AVSG_GATHER_NONE 3     /* Stage One only (matching measured alone) */
#define AVSG_GATHER_POSITION 4 /* S2: the N_g*K selected positions split into C near-equal ranges, hits issue nothing (Eq. 14) */
#define AVSG_GATHER_PIPELINED 5 /* Stage One and Stage Two in one launch: each token's misses are queued in
                                   chunks as soon as they are reserved and copied by every CU (hash matching,
                                   batch <= CU count) */
#define AVSG_GATHER_RESIDENT 6  /* Stage Two that moves over the host link only the misses whose row is not
                                   yet on the device (hash matching only).  A miss whose index is still cached
                                   by a slot of the same request outside this step's reservations (its mapping
                                   was lost to an exhausted probe chain or a bucket collision, so the probe of
                                   Eq. 8-11 cannot find it) is copied from that slot; a miss that repeats a
                                   miss of another token of the step (same index) is written by that index's
                                   host copy, which fills up to two such repeats (further repeats, from four
                                   tokens on, are copied from its slot).  Host rows go in 6-row tiles claimed
                                   by every CU.  Slots, counts, tables and buffer
                                   contents are identical to AVSG_GATHER_BALANCED.  Relies on the same
                                   property as a hit: a cached row below the verified length does not change
                                   on the host. */
#define AVSG_GATHER_EARLY 7     /* resident reuse whose host reads start before Stage One (hash matching
                                   only).  An index that no slot of its request holds when the step begins
                                   misses where it first occurs (Eq. 10 needs c[o] == x) and is in no slot
                                   outside the step's reservations afterwards, so Stage Two reads its row from
                                   the host whatever slots Stage One picks.  A first kernel lists those indices
                                   (at most four positions each); in the next launch workgroups beside the
                                   matching ones copy their rows while Stage One runs, straight into the slots
                                   of their positions once a request's O is written, else into HBM staging
                                   that a third kernel moves to the slots.  The matching workgroup plans and
                                   copies the rest as AVSG_GATHER_RESIDENT does.  Slots, counts, tables and
                                   buffer contents are identical to AVSG_GATHER_BALANCED. */

#define AVSG_GATHER_AUTO 8      /* AVSG_GATHER_RESIDENT when a step looks up at least 8192 indices
                                   (B*N_q*K) with hash matching and the resident plan fits beside the
                                   table, else AVSG_GATHER_BALANCED: below that size the plan costs more
                                   than the host rows it saves (measured crossover between 4096 and 8192
                                   lookups per step).  Resolved once, at create; avsg_resolve_config
                                   tells which. */

#define AVSG_MAX_STREAMS 2

/* Bytes of the library's own static device array behind avsg_step_static (one
 * array per GPU the library runs on, held until the process ends). */
#define AVSG_STATIC_SCRATCH_BYTES ((size_t)32 << 20)

typedef struct avsg_config {
    int32_t batch;      /* B >= 1 */
    int32_t topk;       /* K >= 1, selected indices per query token */
    int32_t n_q;        /* N_q = N_mtp + 1 in [1, 127] query tokens per request per step */
    int32_t slots;      /* S = 2^m, 2 <= S <= 2^23, S >= N_q*K (Eq. 7) */
    int32_t retry;      /* R >= 0; probes examine R+1 buckets (default 3) */
    int32_t max_life;   /* L in [1, 127]; lifetime of a hit or new slot (default 16) */
    uint32_t a1, a2;    /* distinct primes setting initial bucket and stride (Eq. 9) */
    int32_t n_streams;  /* 1 (KV rows) or 2 (KV rows + indexer-key rows) */
    int32_t gather_workers; /* C, workgroups of the balanced gather; 0 = one per CU */
    int64_t row_bytes[AVSG_MAX_STREAMS]; /* bytes per row of each stream, multiple of 4 */
    int32_t match_mode;  /* AVSG_MATCH_* */
    int32_t gather_mode; /* AVSG_GATHER_* */
    /* AVSG_GATHER_EARLY only (0 = default for both): */
    int32_t early_staging_rows; /* rows of HBM staging for rows fetched before their slots are known:
                                   0 = min(B*N_q*K, 16384), -1 = none (such rows are read from the host
                                   again after Stage One), else the count */
    int32_t early_direct;       /* 0 = a fetched row goes straight into its slots once they are known;
                                   -1 = every early row goes through staging (measurement and tests) */
    int32_t validate;   /* 1 = check the selections of every step before any table write: an index
                           outside [0, rows of its request) or repeated within one token's top-K list
                           (Section 3.2 "Problem formulation": a token's K selected indices) makes
                           avsg_step return AVSG_E_BADINDEX with the tables untouched; costs one
                           check kernel and one read-back (and a host synchronization) per step.
                           0 = no check: out-of-range indices are counted and skipped (bad_indices),
                           repeated indices are the caller's error. */
} avsg_config;

/* Cumulative counters since create (or the last avsg_reset_stats). */
typedef struct avsg_stats_t {
    uint64_t steps;           /* avsg_step calls */
    uint64_t lookups;         /* selected indices looked up: steps * B * N_q * K */
    uint64_t hits;            /* lookups that found their index resident */
    uint64_t misses;          /* lookups that reserved a slot and caused a copy */
    uint64_t bytes_moved;     /* payload bytes written into the buffers: misses * row bytes, all streams */
    uint64_t lost_exhausted;  /* misses whose R+1 install probes found no reusable bucket */
    uint64_t lost_collision;  /* misses whose bucket install lost to a larger miss rank */
    uint64_t alloc_decays;    /* unit decays done by the allocation loop (Algorithm 1) */
    uint64_t revivals;        /* hits on a slot whose lifetime was negative */
    uint64_t invalidations;   /* cached indices cleared by speculative invalidation */
    uint64_t bad_indices;     /* selected indices outside [0, rows) (skipped by the copy) */
    uint64_t resident_rows;   /* AVSG_GATHER_RESIDENT: misses filled from a slot that already held the row */
    uint64_t duplicate_rows;  /* AVSG_GATHER_RESIDENT: misses filled from a same-step miss of the same index */
    uint64_t host_bytes;      /* payload bytes read over the host link, all streams */
    int32_t max_step_alloc_decays; /* largest allocation-decay count of one request-step */
    int32_t queue_timeouts;   /* pipelined step: consumers that gave up waiting (0 in correct operation) */
    uint64_t copy_calls;      /* AVSG_GATHER_SDMA: runtime copy calls issued (one per step when the HIP
                                 runtime in the process has the batched copy call, else one per row) */
    uint64_t early_rows;      /* AVSG_GATHER_EARLY: host rows fetched before Stage One (one per index) */
    uint64_t early_staged_rows;   /* of those, rows parked in staging until their slots were known */
    uint64_t early_deferred_rows; /* of those, rows read after Stage One because staging was full */
} avsg_stats_t;

typedef struct avsg_handle avsg_handle;

/* Validate a configuration without touching the device: AVSG_OK or the status
 * avsg_create would return for it (AVSG_E_INVAL, AVSG_E_NOTPOW2,
 * AVSG_E_CAPACITY, AVSG_E_RANGE, AVSG_E_UNSUPPORTED).  The rules are the
 * parameters of Section 3.2 (S = 2^m with m slot bits, Eq. 2; a1 and a2 two
 * distinct primes; the retry budget R; the lifetime L of an 8-bit field,
 * Section 3.5) and the capacity rule S >= N_q * K of Eq. 7. */
avsg_status avsg_check_config(const avsg_config *cfg);

/* The configuration a handle of cfg runs: cfg with AVSG_GATHER_AUTO replaced by
 * the transfer it selects (a call of this library's own).  Returns the status
 * avsg_check_config gives cfg; *out is written only on AVSG_OK. */
avsg_status avsg_resolve_config(const avsg_config *cfg, avsg_config *out);

/* A call of this library's own with no counterpart in the paper (which keeps
 * the table in each core's on-chip buffer): size in bytes of the device
 * workspace that avsg_create needs for cfg
 * (per-request tables of 8*S bytes, transfer lists of 8*N_q*K bytes, a hit
 * mask of N_q*K bytes, counters and pointer tables; with AVSG_GATHER_RESIDENT
 * or AVSG_GATHER_EARLY three more lists of 8*N_q*K bytes and fan slot pairs
 * of 8*N_q*K bytes per request;
 * with AVSG_GATHER_EARLY also early keys, positions and finish entries of
 * 36*N_q*K bytes per request and the staging rows (early_staging_rows, by
 * default min(B*N_q*K, 16384), times the row bytes of every stream); with
 * AVSG_GATHER_PIPELINED a chunk queue of 16 bytes per 32 misses).  Returns 0
 * for an invalid cfg. */
size_t avsg_workspace_bytes(const avsg_config *cfg);

/* Create a handle and reset every table to empty (c_j = -1, lifetime -1, every
 * bucket invalid) on `stream`: one Hash-State table of S entries E_j = (c_j,
 * q_j) per request, shared by the request's N_q tokens (Section 3.2 "Problem
 * formulation" and "Hash-State table", Eq. 2), with S >= N_q * K (Eq. 7).
 *   host_rows        [n_streams*B] host row arrays, entry s*B + r is row 0 of
 *                    request r in stream s; each row is row_bytes[s] long.  The
 *                    memory must be pinned and mapped for the device
 *                    (avsg_host_alloc or hipHostMalloc), 16-byte aligned when
 *                    row_bytes[s] is a multiple of 16.  Row x of request r is
 *                    the KV (or indexer-key) entry of token position x.
 *   rows_per_request [B] host array: number of rows of each request (ids must
 *                    lie in [0, rows)).
 *   d_workspace      device memory of avsg_workspace_bytes(cfg) bytes, 256-byte
 *                    aligned; owned by the caller and used exclusively by this
 *                    handle until avsg_destroy.
 *   d_buffers        [n_streams*B] device buffers, entry s*B + r holds S rows of
 *                    row_bytes[s] bytes (slot o at offset o*row_bytes[s]).
 *   stream           hipStream_t (NULL = default stream).
 * Errors: AVSG_E_INVAL, AVSG_E_NOTPOW2, AVSG_E_CAPACITY, AVSG_E_RANGE,
 * AVSG_E_UNSUPPORTED, AVSG_E_HIP.  On error *out is NULL. */
avsg_status avsg_create(const avsg_config *cfg, const void *const *host_rows,
                        const int64_t *rows_per_request, void *d_workspace, size_t workspace_bytes,
                        void *const *d_buffers, void *stream, avsg_handle **out);

/* One decode step (Algorithm 4) for the whole batch, enqueued on `stream`.
 *   d_topk          device int32 [B][N_q][K]: selected indices; the indices of
 *                   one token must be distinct (a DSA top-K list is).
 *   d_verified_len  device int64 [B]: verified context length N of each
 *                   request; cached indices >= N are cleared at the end of the
 *                   step.  NULL disables the invalidation.
 *   d_slots         device int32 [B][N_q][K] out: buffer slot of every index
 *                   (the matrix O of Algorithm 4).
 *   d_miss_counts   device int32 [B][N_q] out: miss count n_g of every token.
 * When the step's kernels finish, every slot named in d_slots holds the row of
 * its index in every stream.  Indices outside [0, rows) are counted in
 * bad_indices and not copied.  The current HIP device must be the one that
 * was current at avsg_create.  With timing off, a step of any transfer but
 * the copy-engine one (which waits on the host) can be captured into a HIP
 * graph (stream capture): it enqueues kernels only, keeps every piece of step
 * state in the workspace (step stamps advance on the device), and each replay
 * is the next decode step on whatever d_topk then holds.
 * With cfg.validate = 1 the step first checks every token's K indices (in
 * [0, rows) and distinct within the token, the input of Section 3.2 "Problem
 * formulation"), reads the verdict back (a host synchronization; such a step
 * cannot be captured) and returns AVSG_E_BADINDEX, naming the first bad
 * request and token in avsg_last_error, before any table is written.
 * Errors: AVSG_E_INVAL (null pointer, other device), AVSG_E_BADINDEX
 * (validate mode), AVSG_E_HIP. */
avsg_status avsg_step(avsg_handle *h, const int32_t *d_topk, const int64_t *d_verified_len,
                      int32_t *d_slots, int32_t *d_miss_counts, void *stream);

/* Cumulative counters.  Synchronizes with the handle's last stream.  steps
 * and lookups count avsg_step calls on the host, so replays of a captured
 * step are not in them; every other counter is kept on the device and
 * includes them.  hits and misses count the hit indicator m_i of Eq. 1 over
 * every selected index (hit rate = hits / lookups; a later token's hit on a
 * slot an earlier token of the same step reserved counts as a hit,
 * Section 3.6); misses also equal the transfers N_miss of Section 3.4. */
avsg_status avsg_stats(avsg_handle *h, avsg_stats_t *out);

/* The same counters for request r alone (lookups = steps * N_q * K), for
 * per-request hit rates such as the request-averaged rate the paper reports
 * over real requests (Appendix A).  queue_timeouts and copy_calls (counted for
 * the whole handle) are 0.  Synchronizes with the
 * handle's last stream.  Errors: AVSG_E_INVAL (r outside [0, B)), AVSG_E_HIP. */
avsg_status avsg_request_stats(avsg_handle *h, int32_t r, avsg_stats_t *out);
avsg_status avsg_reset_stats(avsg_handle *h, void *stream);

/* Return request r's table to the initial empty state (a new request takes
 * over the batch position), enqueued on `stream`: the cold start of Section
 * 3.6, after which the request's first token misses every index and later
 * tokens of the same step reuse its reservations.  The buffers are untouched. */
avsg_status avsg_reset_request(avsg_handle *h, int32_t r, void *stream);

/* Canonical table view of request r, copied to host memory (synchronous):
 * c_out[S] cached indices, q_out[S] metadata words in the layout of Eq. 2
 * (lifetime byte | invalid bit | fingerprint | slot).  Hash mode only. */
avsg_status avsg_export_state(avsg_handle *h, int32_t r, int32_t *c_out, uint32_t *q_out);

/* Replace request r's table with c_in[S] / q_in[S] in the layout of Eq. 2 (as
 * avsg_export_state returns them; Section 3.2 "Hash-State table"), copied
 * from host memory and synchronized on `stream` before returning: restores a
 * checkpointed table, or hands a request's table to another handle of the
 * same configuration.  Every lifetime byte must lie in [-1, L] (a lifetime the
 * method can reach; Section 3.5); other fields are taken as they are.  The
 * buffers are untouched: they must hold the rows the imported table names.
 * Errors: AVSG_E_INVAL, AVSG_E_RANGE (a lifetime outside [-1, L]),
 * AVSG_E_UNSUPPORTED (dual-pointer matching), AVSG_E_HIP. */
avsg_status avsg_import_state(avsg_handle *h, int32_t r, const int32_t *c_in, const uint32_t *q_in,
                              void *stream);

/* Transfer list of request r from the last step, copied to host memory
 * (synchronous): n_out receives the request's miss total, x_out/o_out
 * (capacity N_q*K each) the index and slot of every miss, ordered by token,
 * then by position inside the token (increasing index order for dual-pointer). */
avsg_status avsg_export_misses(avsg_handle *h, int32_t r, int32_t *n_out, int32_t *x_out,
                               int32_t *o_out);

/* Stage Two plan of request r from the last step (AVSG_GATHER_RESIDENT, or
 * AVSG_GATHER_EARLY, whose plan leaves out the misses of early-fetched
 * indices), copied to host memory (synchronous); every list keeps
 * transfer-list order and has capacity N_q*K:
 *   n_host, host_x[k], host_o[k],  misses copied from host row host_x[k] into
 *   host_fan[2k], host_fan[2k+1]   slot host_o[k], and also into slots
 *                                  host_fan[2k] and host_fan[2k+1] where they
 *                                  are not -1 (the two largest repeat
 *                                  destinations of the index, larger first;
 *                                  host_fan has capacity 2*N_q*K);
 *   n_res, res_src[k], res_dst[k]  misses whose row is already in slot
 *                                  res_src[k] (the largest slot outside this
 *                                  step's reservations that caches the index
 *                                  below the verified length): copied slot to
 *                                  slot, alongside the host copies;
 *   n_rep, rep_src[k], rep_dst[k]  further repeats of an index missed by four
 *                                  or more tokens of the step: copied from the
 *                                  largest slot this step reserved for it, after
 *                                  the host copies.
 * Errors: AVSG_E_INVAL, AVSG_E_UNSUPPORTED (another gather mode), AVSG_E_HIP. */
avsg_status avsg_export_plan(avsg_handle *h, int32_t r, int32_t *n_host, int32_t *host_x,
                             int32_t *host_o, int32_t *host_fan, int32_t *n_res, int32_t *res_src,
                             int32_t *res_dst, int32_t *n_rep, int32_t *rep_src, int32_t *rep_dst);

/* Early list of request r from the last step (AVSG_GATHER_EARLY only), copied
 * to host memory (synchronous): *n_out indices x_out[k] (capacity N_q*K) whose
 * rows were fetched before Stage One, in the kernel's order (a hash order),
 * and pos_out[4*k .. 4*k+3] the flat positions g*K + i of x_out[k] among the
 * step's selections, in no particular order, -1 padded.
 * Errors: AVSG_E_INVAL, AVSG_E_UNSUPPORTED (another gather mode), AVSG_E_HIP. */
avsg_status avsg_export_early(avsg_handle *h, int32_t r, int32_t *n_out, int32_t *x_out,
                              int32_t *pos_out);

/* Per-step kernel timing with HIP events recorded on the step's stream.
 * avsg_set_timing(h, 1) starts recording (and clears the record);
 * avsg_timing copies up to `cap` recorded steps (synchronizing):
 * match_ms[i] is the duration of step i's matching kernel, gather_ms[i] that
 * of its main Stage Two kernel (or copies), and tail_ms[i] (may be NULL) the
 * rest of Stage Two: the repeat copies of AVSG_GATHER_RESIDENT with four or
 * more tokens per step, 0 otherwise.  AVSG_GATHER_EARLY: match_ms is the early
 * list kernel, gather_ms the launch that matches and copies, tail_ms the
 * finishing kernel. */
avsg_status avsg_set_timing(avsg_handle *h, int32_t enable);
avsg_status avsg_timing(avsg_handle *h, float *match_ms, float *gather_ms, float *tail_ms,
                        int32_t cap, int32_t *n_out);

avsg_status avsg_destroy(avsg_handle *h);

/* For callers that cannot allocate memory -- code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc: one decode step like
 * avsg_step, without a handle or a caller workspace.  The tables, transfer
 * lists, plan lists, counters and pointer tables live in the library's own
 * static device array of AVSG_STATIC_SCRATCH_BYTES on the current GPU; the
 * call makes no hipMalloc, hipFree or other allocating call.
 *   cfg, host_rows, rows_per_request, d_buffers   as for avsg_create (host_rows
 *                    pinned and device-mapped; the host arrays are read during
 *                    the call only);
 *   d_topk, d_verified_len, d_slots, d_miss_counts, stream   as for avsg_step;
 *   cold_start       nonzero: every table starts empty (and the counters at
 *                    zero) before this step; 0: the step continues from the
 *                    tables the previous call on this GPU left, which must have
 *                    succeeded with the same configuration.
 * Every call on a GPU shares that GPU's array, which keeps the last call's
 * contents: calls on one GPU must be ordered on one stream, and calls that
 * overlap (two streams, two host threads) race.
 * Hash matching with AVSG_GATHER_BALANCED, _REQUEST, _POSITION, _RESIDENT or
 * _NONE, and dual-pointer matching with _BALANCED, _REQUEST or _NONE.
 * Errors: AVSG_E_INVAL (null pointer, misaligned rows, a continuing call after
 * another configuration or a failed call), AVSG_E_NOTPOW2, AVSG_E_RANGE,
 * AVSG_E_CAPACITY (avsg_workspace_bytes(cfg) above AVSG_STATIC_SCRATCH_BYTES,
 * or the LDS limit), AVSG_E_UNSUPPORTED (validate mode or another transfer),
 * AVSG_E_HIP; each error is described on stderr. */
avsg_status avsg_step_static(const avsg_config *cfg, const void *const *host_rows,
                             const int64_t *rows_per_request, void *const *d_buffers,
                             const int32_t *d_topk, const int64_t *d_verified_len, int32_t *d_slots,
                             int32_t *d_miss_counts, int32_t cold_start, void *stream);

const char *avsg_strerror(avsg_status s);
const char *avsg_last_error(const avsg_handle *h);

/* Pinned, device-mapped host memory for the host rows (hipHostMalloc with
 * hipHostMallocMapped, plus hipHostMallocNonCoherent when coherent == 0 so the
 * device may cache reads).  Free with avsg_host_free. */
avsg_status avsg_host_alloc(size_t bytes, int32_t coherent, void **out);
avsg_status avsg_host_free(void *p);

/* Measured hipMemcpyAsync host-to-device bandwidth from pinned `host` to
 * `device` (`bytes` each), median of `iters` timed copies after one warm-up,
 * in GB/s (1e9 B/s).  Synchronous. */
avsg_status avsg_h2d_peak(const void *host, void *device, size_t bytes, int32_t iters,
                          void *stream, double *gbps);

/* Number of compute units of the current device (the default C). */
int32_t avsg_device_cus(void);

#ifdef __cplusplus
}
#endif
#endif /* AVSG_H */
