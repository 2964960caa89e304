/* C caller of the library: a small two-stream MTP workload stepped through
 * the C ABI (include/avsg.h, device memory from hipMalloc, host rows from
 * avsg_host_alloc) and through the CPU oracle's C interface on the same
 * inputs.  After every step the slots, the miss counts and every byte of both
 * streams' buffers must be equal.
 *
 *   usage: c_abi_parity GATHER_MODE        prints "ok ..." and exits 0 on success
 *
 * Selections: token 0 keeps each index of the previous step's token 0 with
 * probability 0.85 and draws the rest uniformly from the unused positions;
 * token 1 replaces about 10% of token 0's indices with unused positions.
 * Host row bytes are a fixed function of (stream, request, position, byte). */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "avsg.h"
#include "avsg_oracle.h"

enum { B = 3, K = 200, NQ = 2, S = 1024, T = 10, NSTREAMS = 2 };
static const int64_t kCtx = 4000;
static const int64_t kRowBytes[NSTREAMS] = {1152, 132};

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) {
  rng = rng * 6364136223846793005ull + 1442695040888963407ull;
  return (uint32_t)(rng >> 33);
}

#define HIP_OK(call)                                                         \
  do {                                                                       \
    hipError_t e_ = (call);                                                  \
    if (e_ != hipSuccess) {                                                  \
      fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));      \
      exit(2);                                                               \
    }                                                                        \
  } while (0)

#define AVSG_OK_(call)                                                       \
  do {                                                                       \
    avsg_status s_ = (call);                                                 \
    if (s_ != AVSG_OK) {                                                     \
      fprintf(stderr, "%s failed: %s\n", #call, avsg_strerror(s_));          \
      exit(2);                                                               \
    }                                                                        \
  } while (0)

/* draw an index in [0, kCtx) not marked in `used`, and mark it */
static int32_t fresh(uint8_t *used) {
  for (;;) {
    int32_t x = (int32_t)(next_u32() % (uint32_t)kCtx);
    if (!used[x]) {
      used[x] = 1;
      return x;
    }
  }
}

static void select_step(int t, int32_t *X /* [B][NQ][K] */, int32_t *prev /* [B][K] */) {
  uint8_t *used = malloc((size_t)kCtx);
  for (int r = 0; r < B; ++r) {
    int32_t *x0 = X + (size_t)r * NQ * K, *x1 = x0 + K;
    memset(used, 0, (size_t)kCtx);
    for (int i = 0; i < K; ++i) {
      if (t > 0 && next_u32() % 100 < 85) {
        x0[i] = prev[r * K + i];
        used[x0[i]] = 1;
      } else {
        x0[i] = -1;
      }
    }
    for (int i = 0; i < K; ++i)
      if (x0[i] < 0) x0[i] = fresh(used);
    for (int i = 0; i < K; ++i) x1[i] = (next_u32() % 10 == 0) ? fresh(used) : x0[i];
    memcpy(prev + r * K, x0, sizeof(int32_t) * K);
  }
  free(used);
}

int main(int argc, char **argv) {
  const int mode = argc > 1 ? atoi(argv[1]) : AVSG_GATHER_BALANCED;
  HIP_OK(hipSetDevice(0));
  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));

  avsg_config cfg;
  memset(&cfg, 0, sizeof(cfg));
  cfg.batch = B;
  cfg.topk = K;
  cfg.n_q = NQ;
  cfg.slots = S;
  cfg.retry = 1;
  cfg.max_life = 8;
  cfg.a1 = 2654435761u;
  cfg.a2 = 2246822519u;
  cfg.n_streams = NSTREAMS;
  cfg.row_bytes[0] = kRowBytes[0];
  cfg.row_bytes[1] = kRowBytes[1];
  cfg.match_mode = AVSG_MATCH_HASH;
  cfg.gather_mode = mode;
  AVSG_OK_(avsg_check_config(&cfg));

  /* host rows (pinned, mapped) and the oracle's buffer images */
  void *host[NSTREAMS];
  const void *host_rows[NSTREAMS * B];
  uint8_t *images[NSTREAMS];
  void *image_rows[NSTREAMS * B];
  int64_t rows[B];
  for (int r = 0; r < B; ++r) rows[r] = kCtx;
  for (int s = 0; s < NSTREAMS; ++s) {
    const size_t bytes = (size_t)B * kCtx * kRowBytes[s];
    AVSG_OK_(avsg_host_alloc(bytes, 0, &host[s]));
    uint8_t *h = host[s];
    for (size_t i = 0; i < bytes; ++i) h[i] = (uint8_t)(i * 2654435761u >> 13) ^ (uint8_t)(s * 91);
    images[s] = calloc((size_t)B * S * kRowBytes[s], 1);
    for (int r = 0; r < B; ++r) {
      host_rows[s * B + r] = h + (size_t)r * kCtx * kRowBytes[s];
      image_rows[s * B + r] = images[s] + (size_t)r * S * kRowBytes[s];
    }
  }

  /* device memory owned by this caller */
  const size_t ws_bytes = avsg_workspace_bytes(&cfg);
  void *ws, *bufs[NSTREAMS], *d_x, *d_slots, *d_counts;
  void *buf_rows[NSTREAMS * B];
  HIP_OK(hipMalloc(&ws, ws_bytes));
  for (int s = 0; s < NSTREAMS; ++s) {
    HIP_OK(hipMalloc(&bufs[s], (size_t)B * S * kRowBytes[s]));
    HIP_OK(hipMemset(bufs[s], 0, (size_t)B * S * kRowBytes[s]));   /* the oracle's images start at zero */
    for (int r = 0; r < B; ++r) buf_rows[s * B + r] = (uint8_t *)bufs[s] + (size_t)r * S * kRowBytes[s];
  }
  HIP_OK(hipMalloc(&d_x, sizeof(int32_t) * B * NQ * K));
  HIP_OK(hipMalloc(&d_slots, sizeof(int32_t) * B * NQ * K));
  HIP_OK(hipMalloc(&d_counts, sizeof(int32_t) * B * NQ));

  avsg_handle *h = NULL;
  AVSG_OK_(avsg_create(&cfg, host_rows, rows, ws, ws_bytes, buf_rows, stream, &h));

  avsg_ref_config rc = {B, K, NQ, S, cfg.retry, cfg.max_life, cfg.a1, cfg.a2};
  int32_t st = 0;
  avsg_ref_state *ref = avsg_ref_create(&rc, &st);
  if (!ref) {
    fprintf(stderr, "oracle config refused (%d)\n", st);
    return 2;
  }

  static int32_t X[B * NQ * K], prev[B * K], O[B * NQ * K], O_ref[B * NQ * K];
  static int32_t n[B * NQ], n_ref[B * NQ], mx[B * NQ * K], mo[B * NQ * K];
  uint8_t *got = malloc((size_t)B * S * kRowBytes[0]);
  int failures = 0;
  for (int t = 0; t < T && !failures; ++t) {
    select_step(t, X, prev);
    HIP_OK(hipMemcpy(d_x, X, sizeof(X), hipMemcpyHostToDevice));
    AVSG_OK_(avsg_step(h, d_x, NULL, d_slots, d_counts, stream));
    if (avsg_ref_step(ref, X, NULL, O_ref, n_ref, mx, mo, NSTREAMS, host_rows, image_rows, kRowBytes, rows,
                      1) != 0) {
      fprintf(stderr, "oracle step %d failed\n", t);
      return 2;
    }
    HIP_OK(hipStreamSynchronize(stream));
    HIP_OK(hipMemcpy(O, d_slots, sizeof(O), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(n, d_counts, sizeof(n), hipMemcpyDeviceToHost));
    if (memcmp(O, O_ref, sizeof(O)) != 0) {
      fprintf(stderr, "step %d: slots differ\n", t);
      failures++;
    }
    if (memcmp(n, n_ref, sizeof(n)) != 0) {
      fprintf(stderr, "step %d: miss counts differ\n", t);
      failures++;
    }
    for (int s = 0; s < NSTREAMS; ++s) {
      const size_t bytes = (size_t)B * S * kRowBytes[s];
      HIP_OK(hipMemcpy(got, bufs[s], bytes, hipMemcpyDeviceToHost));
      if (memcmp(got, images[s], bytes) != 0) {
        fprintf(stderr, "step %d stream %d: buffers differ\n", t, s);
        failures++;
      }
    }
  }
  /* handover to a validating handle */
  avsg_config cfg2 = cfg;
  cfg2.validate = 1;
  const size_t ws2_bytes = avsg_workspace_bytes(&cfg2);
  void *ws2, *bufs2[NSTREAMS], *buf2_rows[NSTREAMS * B];
  HIP_OK(hipMalloc(&ws2, ws2_bytes));
  for (int s = 0; s < NSTREAMS; ++s) {
    const size_t bytes = (size_t)B * S * kRowBytes[s];
    HIP_OK(hipMalloc(&bufs2[s], bytes));
    HIP_OK(hipMemcpy(bufs2[s], bufs[s], bytes, hipMemcpyDeviceToDevice));
    for (int r = 0; r < B; ++r) buf2_rows[s * B + r] = (uint8_t *)bufs2[s] + (size_t)r * S * kRowBytes[s];
  }
  avsg_handle *h2 = NULL;
  AVSG_OK_(avsg_create(&cfg2, host_rows, rows, ws2, ws2_bytes, buf2_rows, stream, &h2));
  static int32_t tc[S], tc2[S];
  static uint32_t q1[S], q2[S];
  for (int r = 0; r < B && !failures; ++r) {
    AVSG_OK_(avsg_export_state(h, r, tc, q1));
    AVSG_OK_(avsg_import_state(h2, r, tc, q1, stream));
    AVSG_OK_(avsg_export_state(h2, r, tc2, q2));
    if (memcmp(tc, tc2, sizeof(tc)) != 0 || memcmp(q1, q2, sizeof(q1)) != 0) {
      fprintf(stderr, "request %d: imported table differs from the exported one\n", r);
      failures++;
    }
  }
  for (int t = T; t < T + 2 && !failures; ++t) {
    select_step(t, X, prev);
    if (t == T) {
      /* a repeated index inside token 1 of request 2: refused before any write */
      static int32_t Xd[B * NQ * K];
      memcpy(Xd, X, sizeof(X));
      Xd[(2 * NQ + 1) * K + 7] = Xd[(2 * NQ + 1) * K + 3];
      HIP_OK(hipMemcpy(d_x, Xd, sizeof(Xd), hipMemcpyHostToDevice));
      const avsg_status bad = avsg_step(h2, d_x, NULL, d_slots, d_counts, stream);
      if (bad != AVSG_E_BADINDEX || strstr(avsg_last_error(h2), "request 2 token 1") == NULL) {
        fprintf(stderr, "validate: status %d (%s), expected AVSG_E_BADINDEX for request 2 token 1\n", bad,
                avsg_last_error(h2));
        failures++;
      }
      for (int r = 0; r < B; ++r) {
        AVSG_OK_(avsg_export_state(h, r, tc, q1));
        AVSG_OK_(avsg_export_state(h2, r, tc2, q2));
        if (memcmp(tc, tc2, sizeof(tc)) != 0 || memcmp(q1, q2, sizeof(q1)) != 0) {
          fprintf(stderr, "validate: request %d's table changed by a refused step\n", r);
          failures++;
        }
      }
    }
    HIP_OK(hipMemcpy(d_x, X, sizeof(X), hipMemcpyHostToDevice));
    AVSG_OK_(avsg_step(h2, d_x, NULL, d_slots, d_counts, stream));
    if (avsg_ref_step(ref, X, NULL, O_ref, n_ref, mx, mo, NSTREAMS, host_rows, image_rows, kRowBytes, rows,
                      1) != 0) {
      fprintf(stderr, "oracle step %d failed\n", t);
      return 2;
    }
    HIP_OK(hipStreamSynchronize(stream));
    HIP_OK(hipMemcpy(O, d_slots, sizeof(O), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(n, d_counts, sizeof(n), hipMemcpyDeviceToHost));
    if (memcmp(O, O_ref, sizeof(O)) != 0 || memcmp(n, n_ref, sizeof(n)) != 0) {
      fprintf(stderr, "step %d after the handover: slots or counts differ\n", t);
      failures++;
    }
    for (int s = 0; s < NSTREAMS; ++s) {
      const size_t bytes = (size_t)B * S * kRowBytes[s];
      HIP_OK(hipMemcpy(got, bufs2[s], bytes, hipMemcpyDeviceToHost));
      if (memcmp(got, images[s], bytes) != 0) {
        fprintf(stderr, "step %d after the handover, stream %d: buffers differ\n", t, s);
        failures++;
      }
    }
  }
  AVSG_OK_(avsg_destroy(h2));
  for (int s = 0; s < NSTREAMS; ++s) HIP_OK(hipFree(bufs2[s]));
  HIP_OK(hipFree(ws2));

  avsg_stats_t stats;
  AVSG_OK_(avsg_stats(h, &stats));
  AVSG_OK_(avsg_destroy(h));
  avsg_ref_destroy(ref);
  free(got);
  for (int s = 0; s < NSTREAMS; ++s) {
    free(images[s]);
    HIP_OK(hipFree(bufs[s]));
    AVSG_OK_(avsg_host_free(host[s]));
  }
  HIP_OK(hipFree(ws));
  HIP_OK(hipFree(d_x));
  HIP_OK(hipFree(d_slots));
  HIP_OK(hipFree(d_counts));
  HIP_OK(hipStreamDestroy(stream));
  if (failures) return 1;
  printf("ok mode %d steps %d (+2 after a validated handover) hits %llu misses %llu\n", mode, T,
         (unsigned long long)stats.hits,
         (unsigned long long)stats.misses);
  return 0;
}
