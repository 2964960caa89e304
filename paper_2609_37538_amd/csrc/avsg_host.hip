// Host side of libavsg: the C ABI declared in include/avsg.h.
//
// Validates configurations, lays out the caller's device workspace, records
// device-visible addresses of the caller's pinned host rows, and enqueues the
// Stage One / Stage Two kernels of each decode step on the caller's stream.
#include "avsg.h"

#include <dlfcn.h>

#include <algorithm>
#include <array>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "avsg_internal.h"

using namespace avsg;

struct avsg_handle {
  avsg_config cfg{};
  int device = 0;
  int m = 0;
  size_t lds = 0;
  int workers = 0;
  // workspace sections
  int32_t* table_c = nullptr;
  uint32_t* table_q = nullptr;
  int2* dp_state = nullptr;
  int2* miss_list = nullptr;
  uint8_t* hit_mask = nullptr;
  int2* host_list = nullptr;    // resident-reuse plan (AVSG_GATHER_RESIDENT)
  int2* host_fan = nullptr;
  int2* res_list = nullptr;
  int2* rep_list = nullptr;
  int32_t* plan_counts = nullptr;  // [B][3]
  int32_t* plan_claim = nullptr;
  int plan_words = 0;
  int plan_list_off = 0;   // LDS offset of the transfer list the plan reads
  int plan_scan_off = 0;   // LDS offset of the plan scan's candidate lists
  // early-fetch transfer (AVSG_GATHER_EARLY)
  int32_t* early_x = nullptr;
  int4* early_pos = nullptr;
  int32_t* early_n = nullptr;
  uint32_t* early_done = nullptr;
  int* early_ctl = nullptr;
  int4* early_fin = nullptr;
  uint64_t stage0 = 0, stage1 = 0;
  int stage_rows = 0;
  int early_workers = 0;
  size_t early_list_lds = 0;
  int* pipe_ctl = nullptr;      // head, tail, done, exit_count, error, last epoch
  int4* pipe_chunks = nullptr;
  int pipe_max_chunks = 0;
  int cus = 0;
  unsigned long long* stats = nullptr;
  uint64_t* host_ptrs = nullptr;
  uint64_t* buf_ptrs = nullptr;
  int64_t* rows_dev = nullptr;
  // host copies
  std::vector<int64_t> rows;
  std::vector<uint64_t> host_dev, bufs;
  uint64_t steps = 0;
  hipStream_t last_stream = nullptr;
  int32_t* last_counts = nullptr;
  // timing
  bool timing = false;
  std::vector<std::array<hipEvent_t, 4>> events;   // before Stage One, after it, after the
                                                   // main Stage Two kernel, after Stage Two
  std::vector<bool> has_tail;                      // step recorded the fourth event
  size_t n_timed = 0;
  // SDMA comparator staging (pinned host); the batched copy call when the HIP
  // runtime loaded in the process exports it
  hipError_t (*batch_copy)(void**, void**, size_t*, size_t, hipMemcpyAttributes*, size_t*, size_t,
                           size_t*, hipStream_t) = nullptr;
  uint64_t copy_calls = 0;
  int32_t* h_counts = nullptr;
  int2* h_list = nullptr;
  std::vector<void*> dsts, srcs;
  std::vector<size_t> sizes;
  // validate mode: per-row verdicts of the last check, read back to the host
  int32_t* val_rows = nullptr;
  std::vector<int32_t> h_val;
  char err[256] = {0};
};

// Device memory of avsg_step_static: one array per GPU the library runs on,
// held until the process ends.  In host code `scratch` names a host-side
// stand-in; its device address on each GPU comes from hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[AVSG_STATIC_SCRATCH_BYTES];

namespace {

constexpr size_t kAlign = 256;
constexpr int kMaxBatch = 1024;
constexpr size_t kMaxTimedSteps = 16384;
constexpr size_t kLdsPerWorkgroup = 160 * 1024;   // gfx950
constexpr int kRepeatWorkersPerCu = 4;
constexpr int kEarlyStagingRows = 16384;   // default staging capacity of the early-fetch transfer
constexpr int kEarlyWorkers = 32;          // default copy workgroups beside the matching ones

size_t up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool is_prime_u32(uint32_t v) {
  if (v < 2) return false;
  if (v % 2 == 0) return v == 2;
  for (uint64_t d = 3; d * d <= v; d += 2)
    if (v % d == 0) return false;
  return true;
}

size_t pipe_chunks_for(const avsg_config& c);

struct Layout {
  size_t table_c, table_q, miss_list, hit_mask, plan, early, pipe, pipe_bytes, stats, host_ptrs, buf_ptrs,
      rows, val, total;
};

bool has_plan(const avsg_config& c) {
  return c.gather_mode == AVSG_GATHER_RESIDENT || c.gather_mode == AVSG_GATHER_EARLY;
}

// Staging rows of the early-fetch transfer.
int early_stage_rows(const avsg_config& c) {
  const long long nk = static_cast<long long>(c.batch) * c.n_q * c.topk;
  if (c.early_staging_rows < 0) return 0;
  const long long want = c.early_staging_rows == 0 ? kEarlyStagingRows : c.early_staging_rows;
  return static_cast<int>(want < nk ? want : nk);
}

// Early-fetch sections, in order: keys, positions, counts, flags, control
// words, finish entries, staging of stream 0, staging of stream 1.
std::array<size_t, 9> early_sections(const avsg_config& c) {
  const size_t nk = static_cast<size_t>(c.batch) * c.n_q * c.topk;
  const size_t rows = static_cast<size_t>(early_stage_rows(c));
  std::array<size_t, 9> off{};
  size_t o = 0;
  const size_t sz[8] = {nk * 4, nk * 16, static_cast<size_t>(c.batch) * 4, static_cast<size_t>(c.batch) * 4,
                        64, nk * 16, rows * static_cast<size_t>(c.row_bytes[0]),
                        c.n_streams > 1 ? rows * static_cast<size_t>(c.row_bytes[1]) : 0};
  for (int i = 0; i < 8; ++i) {
    off[i] = o;
    o += up(sz[i]);
  }
  off[8] = o;
  return off;
}

Layout layout_of(const avsg_config& c) {
  Layout L{};
  const size_t B = static_cast<size_t>(c.batch), S = static_cast<size_t>(c.slots);
  size_t off = 0;
  L.table_c = off; off += up(B * S * 4);
  L.table_q = off; off += up(B * S * 4);
  L.miss_list = off; off += up(B * static_cast<size_t>(c.n_q) * c.topk * 8);
  L.hit_mask = off; off += up(B * static_cast<size_t>(c.n_q) * c.topk);
  L.plan = off;
  if (has_plan(c))   // host, resident, repeat lists; fan slot pairs; counts; claims
    off += 4 * up(B * static_cast<size_t>(c.n_q) * c.topk * 8) + up(B * 12) + up(8);
  L.early = off;
  if (c.gather_mode == AVSG_GATHER_EARLY) off += early_sections(c)[8];
  L.pipe = off;
  L.pipe_bytes = up(kAlign + 16 * pipe_chunks_for(c));
  off += L.pipe_bytes;
  L.stats = off; off += up(B * kNumStats * 8);
  L.host_ptrs = off; off += up(static_cast<size_t>(c.n_streams) * B * 8);
  L.buf_ptrs = off; off += up(static_cast<size_t>(c.n_streams) * B * 8);
  L.rows = off; off += up(B * 8);
  L.val = off;
  if (c.validate) off += up(B * static_cast<size_t>(c.n_q) * 4);
  L.total = off;
  return L;
}

size_t pipe_chunks_for(const avsg_config& c) {
  const int ch = pipelined_chunk_misses();
  return static_cast<size_t>(c.batch) * c.n_q * ((c.topk + ch - 1) / ch);
}

int log2_exact(int32_t s) {
  int m = 0;
  while ((1 << m) < s) ++m;
  return m;
}

avsg_status check_resolved(const avsg_config* c, std::string* why) {
  auto fail = [&](avsg_status s, const char* msg) {
    if (why) *why = msg;
    return s;
  };
  if (!c) return fail(AVSG_E_INVAL, "null config");
  if (c->batch < 1 || c->batch > kMaxBatch) return fail(AVSG_E_INVAL, "batch must be in [1, 1024]");
  if (c->topk < 1 || c->n_q < 1) return fail(AVSG_E_INVAL, "topk and n_q must be positive");
  if (c->n_q > 127) return fail(AVSG_E_RANGE, "n_q must be at most 127");
  if (c->slots < 2 || (c->slots & (c->slots - 1)) != 0 || c->slots > (1 << 23))
    return fail(AVSG_E_NOTPOW2, "slots must be a power of two in [2, 2^23]");
  if (static_cast<int64_t>(c->slots) < static_cast<int64_t>(c->n_q) * c->topk)
    return fail(AVSG_E_CAPACITY, "slots < n_q * topk (buffer capacity rule)");
  if (c->retry < 0) return fail(AVSG_E_RANGE, "retry must be >= 0");
  if (c->max_life < 1 || c->max_life > 127) return fail(AVSG_E_RANGE, "max_life must be in [1, 127]");
  if (c->a1 == c->a2 || !is_prime_u32(c->a1) || !is_prime_u32(c->a2))
    return fail(AVSG_E_RANGE, "a1 and a2 must be distinct primes");
  if (c->n_streams < 1 || c->n_streams > AVSG_MAX_STREAMS)
    return fail(AVSG_E_INVAL, "n_streams must be 1 or 2");
  for (int s = 0; s < c->n_streams; ++s)
    if (c->row_bytes[s] <= 0 || (c->row_bytes[s] & 3) != 0)
      return fail(AVSG_E_RANGE, "row_bytes must be a positive multiple of 4");
  if (c->gather_workers < 0) return fail(AVSG_E_INVAL, "gather_workers must be >= 0");
  if (c->match_mode != AVSG_MATCH_HASH && c->match_mode != AVSG_MATCH_DUALPTR)
    return fail(AVSG_E_INVAL, "unknown match_mode");
  if (c->gather_mode < AVSG_GATHER_BALANCED || c->gather_mode > AVSG_GATHER_EARLY)
    return fail(AVSG_E_INVAL, "unknown gather_mode");
  if (c->early_staging_rows < -1) return fail(AVSG_E_INVAL, "early_staging_rows must be >= -1");
  if (c->early_direct != 0 && c->early_direct != -1) return fail(AVSG_E_INVAL, "early_direct must be 0 or -1");
  if (c->validate != 0 && c->validate != 1) return fail(AVSG_E_INVAL, "validate must be 0 or 1");
  if (c->match_mode == AVSG_MATCH_DUALPTR) {
    if (c->n_q != 1) return fail(AVSG_E_UNSUPPORTED, "dual-pointer matching handles one token per step");
    if (c->slots != c->topk) return fail(AVSG_E_UNSUPPORTED, "dual-pointer matching needs slots == topk");
    if (c->topk > 4096) return fail(AVSG_E_CAPACITY, "dual-pointer matching supports topk <= 4096");
    if (c->gather_mode == AVSG_GATHER_POSITION || c->gather_mode == AVSG_GATHER_PIPELINED ||
        has_plan(*c))
      return fail(AVSG_E_UNSUPPORTED,
                  "position-level, pipelined, resident-reuse and early-fetch transfer need hash matching");
  } else {
    const size_t lds = c->gather_mode == AVSG_GATHER_PIPELINED ? pipelined_lds_bytes(c->slots, c->topk)
                       : c->gather_mode == AVSG_GATHER_EARLY
                           ? early_step_lds_bytes(c->slots, c->topk, c->n_q)
                           : stage_one_lds_bytes(c->slots, c->topk, c->n_q, has_plan(*c));
    if (match_lds_bytes(c->slots, c->topk) == 0 || lds > kLdsPerWorkgroup)
      return fail(AVSG_E_CAPACITY, "table and selection exceed one workgroup's LDS (9*S + 12*K bytes)");
    if (has_plan(*c) && plan_map_words(c->slots, c->topk, c->n_q) == 0)
      return fail(AVSG_E_CAPACITY, "resident-reuse plan: the index map of 1.5*n_q*topk words does not fit in LDS");
    if (c->gather_mode == AVSG_GATHER_EARLY && early_map_words(c->topk, c->n_q) == 0)
      return fail(AVSG_E_CAPACITY, "early fetch: the list map of 1.25*n_q*topk index words does not fit in LDS");
  }
  return AVSG_OK;
}

// AVSG_GATHER_AUTO: resident reuse when a step looks up at least this many
// indices (B * N_q * K) and its plan fits beside the table, else the paper's
// S3.  Measured crossover (µs per step, S3 / resident): 4096 lookups 33.5 / 35.4
// (B = 2, K = 2048) and 40.6 / 43.8 (B = 1, two tokens); 8192 lookups 48.6 /
// 44.7 (B = 4) and 55.1 / 52.8 (B = 2, two tokens).
constexpr long long kAutoResidentLookups = 8192;

avsg_config resolved(const avsg_config& c) {
  avsg_config r = c;
  if (c.gather_mode != AVSG_GATHER_AUTO) return r;
  r.gather_mode = AVSG_GATHER_BALANCED;
  const long long lookups = static_cast<long long>(c.batch) * c.n_q * c.topk;
  if (c.match_mode == AVSG_MATCH_HASH && lookups >= kAutoResidentLookups) {
    avsg_config t = c;
    t.gather_mode = AVSG_GATHER_RESIDENT;
    if (check_resolved(&t, nullptr) == AVSG_OK) r.gather_mode = AVSG_GATHER_RESIDENT;
  }
  return r;
}

avsg_status check_config(const avsg_config* c, std::string* why) {
  if (!c) {
    if (why) *why = "null config";
    return AVSG_E_INVAL;
  }
  const avsg_config r = resolved(*c);
  return check_resolved(&r, why);
}

void set_err(avsg_handle* h, const char* fmt, ...) {
  if (!h) return;
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(h->err, sizeof(h->err), fmt, ap);
  va_end(ap);
}

avsg_status hip_fail(avsg_handle* h, hipError_t e, const char* what) {
  set_err(h, "%s: %s", what, hipGetErrorString(e));
  return AVSG_E_HIP;
}

#define HIP_TRY(h, call)                                   \
  do {                                                     \
    hipError_t e_ = (call);                                \
    if (e_ != hipSuccess) return hip_fail((h), e_, #call); \
  } while (0)

// Section pointers of a workspace laid out by layout_of(h->cfg) at ws.
void bind_workspace(avsg_handle* h, unsigned char* ws, const Layout& L) {
  const avsg_config& c = h->cfg;
  const int B = c.batch;
  h->table_c = reinterpret_cast<int32_t*>(ws + L.table_c);
  h->table_q = reinterpret_cast<uint32_t*>(ws + L.table_q);
  h->dp_state = reinterpret_cast<int2*>(ws + L.table_c);  // S == K: the two table arrays hold [B][K] pairs
  h->miss_list = reinterpret_cast<int2*>(ws + L.miss_list);
  h->hit_mask = ws + L.hit_mask;
  if (has_plan(c)) {
    const size_t list = up(static_cast<size_t>(B) * c.n_q * c.topk * 8);
    h->host_list = reinterpret_cast<int2*>(ws + L.plan);
    h->res_list = reinterpret_cast<int2*>(ws + L.plan + list);
    h->rep_list = reinterpret_cast<int2*>(ws + L.plan + 2 * list);
    const size_t fan = list;   // two slots per host entry
    h->host_fan = reinterpret_cast<int2*>(ws + L.plan + 3 * list);
    h->plan_counts = reinterpret_cast<int32_t*>(ws + L.plan + 3 * list + fan);
    h->plan_claim = reinterpret_cast<int32_t*>(ws + L.plan + 3 * list + fan + up(static_cast<size_t>(B) * 12));
    h->plan_words = plan_map_words(c.slots, c.topk, c.n_q);
    h->plan_list_off = static_cast<int>(plan_list_offset(c.slots, c.topk, c.n_q));
    h->plan_scan_off = static_cast<int>(plan_scan_offset(c.slots, c.topk, c.n_q));
  }
  if (c.gather_mode == AVSG_GATHER_EARLY) {
    const std::array<size_t, 9> o = early_sections(c);
    unsigned char* eb = ws + L.early;
    h->early_x = reinterpret_cast<int32_t*>(eb + o[0]);
    h->early_pos = reinterpret_cast<int4*>(eb + o[1]);
    h->early_n = reinterpret_cast<int32_t*>(eb + o[2]);
    h->early_done = reinterpret_cast<uint32_t*>(eb + o[3]);
    h->early_ctl = reinterpret_cast<int*>(eb + o[4]);
    h->early_fin = reinterpret_cast<int4*>(eb + o[5]);
    h->stage0 = reinterpret_cast<uint64_t>(eb + o[6]);
    h->stage1 = c.n_streams > 1 ? reinterpret_cast<uint64_t>(eb + o[7]) : 0;
    h->stage_rows = early_stage_rows(c);
  }
  h->pipe_ctl = reinterpret_cast<int*>(ws + L.pipe);
  h->pipe_chunks = reinterpret_cast<int4*>(ws + L.pipe + kAlign);
  h->pipe_max_chunks = static_cast<int>(pipe_chunks_for(c));
  h->stats = reinterpret_cast<unsigned long long*>(ws + L.stats);
  h->host_ptrs = reinterpret_cast<uint64_t*>(ws + L.host_ptrs);
  h->buf_ptrs = reinterpret_cast<uint64_t*>(ws + L.buf_ptrs);
  h->rows_dev = reinterpret_cast<int64_t*>(ws + L.rows);
  h->val_rows = c.validate ? reinterpret_cast<int32_t*>(ws + L.val) : nullptr;
}

// Request sizes, and host-row and buffer addresses aligned for the copies.
bool rows_ok(const avsg_config& c, const void* const* host_rows, const int64_t* rows_per_request,
             void* const* d_buffers) {
  const int B = c.batch;
  for (int r = 0; r < B; ++r)
    if (rows_per_request[r] < 1) return false;
  for (int i = 0; i < c.n_streams * B; ++i) {
    if (!host_rows[i] || !d_buffers[i]) return false;
    const int s = i / B;
    if ((c.row_bytes[s] & 15) == 0 &&
        ((reinterpret_cast<uintptr_t>(host_rows[i]) & 15) != 0 ||
         (reinterpret_cast<uintptr_t>(d_buffers[i]) & 15) != 0))
      return false;
    if ((reinterpret_cast<uintptr_t>(host_rows[i]) & 3) != 0 ||
        (reinterpret_cast<uintptr_t>(d_buffers[i]) & 3) != 0)
      return false;
  }
  return true;
}

int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return cus;
}

}  // namespace

extern "C" {

avsg_status avsg_check_config(const avsg_config* cfg) { return check_config(cfg, nullptr); }

size_t avsg_workspace_bytes(const avsg_config* cfg) {
  if (check_config(cfg, nullptr) != AVSG_OK) return 0;
  return layout_of(resolved(*cfg)).total;
}

avsg_status avsg_resolve_config(const avsg_config* cfg, avsg_config* out) {
  if (!out) return AVSG_E_INVAL;
  const avsg_status st = check_config(cfg, nullptr);
  if (st != AVSG_OK) return st;
  *out = resolved(*cfg);
  return AVSG_OK;
}

const char* avsg_strerror(avsg_status s) {
  switch (s) {
    case AVSG_OK: return "ok";
    case AVSG_E_INVAL: return "invalid argument";
    case AVSG_E_NOTPOW2: return "slots is not a power of two in [2, 2^23]";
    case AVSG_E_CAPACITY: return "capacity: slots < n_q*topk, or beyond the on-chip limit";
    case AVSG_E_RANGE: return "parameter out of range";
    case AVSG_E_BADINDEX: return "selected index out of range";
    case AVSG_E_HIP: return "HIP runtime error";
    case AVSG_E_INTERNAL: return "internal error";
    case AVSG_E_UNSUPPORTED: return "unsupported combination";
    default: return "unknown status";
  }
}

const char* avsg_last_error(const avsg_handle* h) { return h ? h->err : ""; }

int32_t avsg_device_cus(void) { return device_cus(); }

avsg_status avsg_create(const avsg_config* cfg, const void* const* host_rows,
                        const int64_t* rows_per_request, void* d_workspace, size_t workspace_bytes,
                        void* const* d_buffers, void* stream, avsg_handle** out) {
  if (!out) return AVSG_E_INVAL;
  *out = nullptr;
  std::string why;
  avsg_status st = check_config(cfg, &why);
  if (st != AVSG_OK) {
    std::fprintf(stderr, "avsg_create: %s\n", why.c_str());
    return st;
  }
  const avsg_config c = resolved(*cfg);
  if (!host_rows || !rows_per_request || !d_workspace || !d_buffers) return AVSG_E_INVAL;
  const Layout L = layout_of(c);
  if (workspace_bytes < L.total) return AVSG_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(d_workspace) & (kAlign - 1)) != 0) return AVSG_E_INVAL;
  const int B = c.batch;
  if (!rows_ok(c, host_rows, rows_per_request, d_buffers)) return AVSG_E_INVAL;

  auto* h = new avsg_handle();
  h->cfg = c;
  hipStream_t s = static_cast<hipStream_t>(stream);
  h->last_stream = s;
  if (hipGetDevice(&h->device) != hipSuccess) {
    delete h;
    return AVSG_E_HIP;
  }
  h->m = log2_exact(c.slots);
  bind_workspace(h, static_cast<unsigned char*>(d_workspace), L);
  if (c.validate) h->h_val.resize(static_cast<size_t>(B) * c.n_q);
  h->rows.assign(rows_per_request, rows_per_request + B);
  h->host_dev.resize(static_cast<size_t>(c.n_streams) * B);
  h->bufs.resize(static_cast<size_t>(c.n_streams) * B);
  for (int i = 0; i < c.n_streams * B; ++i) {
    void* dptr = nullptr;
    hipError_t e = hipHostGetDevicePointer(&dptr, const_cast<void*>(host_rows[i]), 0);
    if (e != hipSuccess || !dptr) {
      set_err(h, "host rows must be pinned, device-mapped memory (avsg_host_alloc / hipHostMalloc)");
      std::fprintf(stderr, "avsg_create: %s (%s)\n", h->err, hipGetErrorString(e));
      delete h;
      return AVSG_E_INVAL;
    }
    h->host_dev[i] = reinterpret_cast<uint64_t>(dptr);
    h->bufs[i] = reinterpret_cast<uint64_t>(d_buffers[i]);
  }
  const int cus = device_cus();
  h->cus = cus;
  h->workers = c.gather_workers > 0 ? c.gather_workers : std::max(1, cus);

  auto cleanup = [&](avsg_status rc) {
    if (h->h_counts) (void)hipHostFree(h->h_counts);
    if (h->h_list) (void)hipHostFree(h->h_list);
    delete h;
    return rc;
  };
  hipError_t e;
  if (c.match_mode == AVSG_MATCH_HASH) {
    h->lds = stage_one_lds_bytes(c.slots, c.topk, c.n_q, has_plan(c));
    int max_lds = 0;
    if ((e = hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device)) !=
        hipSuccess)
      return cleanup(AVSG_E_HIP);
    if (max_lds > 0 && h->lds > static_cast<size_t>(max_lds)) {
      std::fprintf(stderr, "avsg_create: table of %d slots needs %zu B of LDS, limit %d\n",
                   c.slots, h->lds, max_lds);
      return cleanup(AVSG_E_CAPACITY);
    }
    if ((e = prepare_match_hash(h->lds)) != hipSuccess) return cleanup(hip_fail(nullptr, e, ""));
    if (c.gather_mode == AVSG_GATHER_PIPELINED) {
      // producers (one per request) must all be resident beside the consumers
      if (c.batch > cus) {
        std::fprintf(stderr, "avsg_create: pipelined step needs batch <= %d (one workgroup per CU)\n", cus);
        return cleanup(AVSG_E_UNSUPPORTED);
      }
      h->lds = pipelined_lds_bytes(c.slots, c.topk);
      if ((e = prepare_step_pipelined(h->lds)) != hipSuccess) return cleanup(AVSG_E_HIP);
      if (launch_zero_u64(reinterpret_cast<unsigned long long*>(h->pipe_ctl), L.pipe_bytes / 8, s) !=
          hipSuccess)
        return cleanup(AVSG_E_HIP);
    }
    if (c.gather_mode == AVSG_GATHER_EARLY) {
      h->lds = early_step_lds_bytes(c.slots, c.topk, c.n_q);
      h->early_list_lds = early_list_lds_bytes(c.topk, c.n_q);
      if (max_lds > 0 && (h->lds > static_cast<size_t>(max_lds) || h->early_list_lds > static_cast<size_t>(max_lds)))
        return cleanup(AVSG_E_CAPACITY);
      if ((e = prepare_step_early(h->early_list_lds, h->lds)) != hipSuccess) return cleanup(AVSG_E_HIP);
      h->early_workers = c.gather_workers > 0 ? c.gather_workers : kEarlyWorkers;
      // a step that never ran has no early list
      if (launch_zero_u64(reinterpret_cast<unsigned long long*>(static_cast<unsigned char*>(d_workspace) + L.early),
                          early_sections(c)[6] / 8, s) != hipSuccess)
        return cleanup(AVSG_E_HIP);
    }
    if ((e = launch_reset_tables(h->table_c, h->table_q,
                                 static_cast<size_t>(B) * c.slots, s)) != hipSuccess)
      return cleanup(AVSG_E_HIP);
  } else {
    h->lds = dualptr_lds_bytes(c.topk);
    if ((e = prepare_match_dualptr(h->lds)) != hipSuccess) return cleanup(AVSG_E_HIP);
    if ((e = launch_reset_dualptr(h->dp_state, B, c.topk, s)) != hipSuccess) return cleanup(AVSG_E_HIP);
  }
  if (launch_zero_u64(h->stats, static_cast<size_t>(B) * kNumStats, s) != hipSuccess)
    return cleanup(AVSG_E_HIP);
  if (hipMemcpyAsync(h->host_ptrs, h->host_dev.data(), h->host_dev.size() * 8,
                     hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(h->buf_ptrs, h->bufs.data(), h->bufs.size() * 8, hipMemcpyHostToDevice, s) !=
          hipSuccess ||
      hipMemcpyAsync(h->rows_dev, h->rows.data(), h->rows.size() * 8, hipMemcpyHostToDevice, s) !=
          hipSuccess)
    return cleanup(AVSG_E_HIP);
  if (c.gather_mode == AVSG_GATHER_SDMA) {
    const size_t nl = static_cast<size_t>(B) * c.n_q * c.topk;
    if (hipHostMalloc(reinterpret_cast<void**>(&h->h_counts), static_cast<size_t>(B) * c.n_q * 4, 0) != hipSuccess ||
        hipHostMalloc(reinterpret_cast<void**>(&h->h_list), nl * 8, 0) != hipSuccess)
      return cleanup(AVSG_E_HIP);
    h->dsts.reserve(nl * c.n_streams);
    h->srcs.reserve(nl * c.n_streams);
    // looked up at run time: the library must also load into processes whose
    // runtime predates the call (PyTorch ships such a runtime)
    h->batch_copy = reinterpret_cast<decltype(h->batch_copy)>(dlsym(RTLD_DEFAULT, "hipMemcpyBatchAsync"));
    h->sizes.reserve(nl * c.n_streams);
  }
  if (hipStreamSynchronize(s) != hipSuccess) return cleanup(AVSG_E_HIP);
  *out = h;
  return AVSG_OK;
}

static avsg_status record(avsg_handle* h, int which, hipStream_t s) {
  if (!h->timing || h->n_timed >= kMaxTimedSteps) return AVSG_OK;
  if (h->events.size() <= h->n_timed) {
    std::array<hipEvent_t, 4> ev{};
    // timing-only events: no system-scope cache write-back/invalidate at record
    for (size_t i = 0; i < ev.size(); ++i) {
      const hipError_t e = hipEventCreateWithFlags(&ev[i], hipEventDisableSystemFence);
      if (e != hipSuccess) {
        for (size_t j = 0; j < i; ++j) (void)hipEventDestroy(ev[j]);
        return hip_fail(h, e, "hipEventCreateWithFlags");
      }
    }
    h->events.push_back(ev);
    h->has_tail.push_back(false);
  }
  HIP_TRY(h, hipEventRecord(h->events[h->n_timed][which], s));
  return AVSG_OK;
}

static avsg_status sdma_gather(avsg_handle* h, const int32_t* d_counts, hipStream_t s) {
  const avsg_config& c = h->cfg;
  const int B = c.batch;
  const size_t per_req = static_cast<size_t>(c.n_q) * c.topk;
  HIP_TRY(h, hipMemcpyAsync(h->h_counts, d_counts, static_cast<size_t>(B) * c.n_q * 4,
                            hipMemcpyDeviceToHost, s));
  HIP_TRY(h, hipMemcpyAsync(h->h_list, h->miss_list, static_cast<size_t>(B) * per_req * 8,
                            hipMemcpyDeviceToHost, s));
  HIP_TRY(h, hipStreamSynchronize(s));
  h->dsts.clear();
  h->srcs.clear();
  h->sizes.clear();
  for (int r = 0; r < B; ++r) {
    int64_t tot = 0;
    for (int g = 0; g < c.n_q; ++g) tot += h->h_counts[static_cast<size_t>(r) * c.n_q + g];
    for (int64_t k = 0; k < tot; ++k) {
      const int2 e = h->h_list[static_cast<size_t>(r) * per_req + k];
      if (e.x < 0 || e.x >= h->rows[r] || e.y < 0 || e.y >= c.slots) continue;
      for (int st = 0; st < c.n_streams; ++st) {
        const uint64_t rb = static_cast<uint64_t>(c.row_bytes[st]);
        h->srcs.push_back(reinterpret_cast<void*>(h->host_dev[static_cast<size_t>(st) * B + r] +
                                                  static_cast<uint64_t>(e.x) * rb));
        h->dsts.push_back(reinterpret_cast<void*>(h->bufs[static_cast<size_t>(st) * B + r] +
                                                  static_cast<uint64_t>(e.y) * rb));
        h->sizes.push_back(static_cast<size_t>(rb));
      }
    }
  }
  if (h->sizes.empty()) return AVSG_OK;
  if (h->batch_copy) {
    // every row and stream in one batched call (the runtime takes no copy
    // attributes; the copies are ordered on the stream like any other)
    size_t failed = 0;
    const hipError_t e = h->batch_copy(h->dsts.data(), h->srcs.data(), h->sizes.data(), h->sizes.size(),
                                       nullptr, nullptr, 0, &failed, s);
    if (e == hipSuccess) {
      h->copy_calls += 1;
      return AVSG_OK;
    }
    if (e != hipErrorNotSupported) return hip_fail(h, e, "hipMemcpyBatchAsync");
    // refused before any copy was queued (the legacy default stream, for
    // one): this handle issues one call per row from now on
    (void)hipGetLastError();
    h->batch_copy = nullptr;
  }
  // one copy-engine command per missed row and stream
  for (size_t i = 0; i < h->sizes.size(); ++i)
    HIP_TRY(h, hipMemcpyAsync(h->dsts[i], h->srcs[i], h->sizes[i], hipMemcpyHostToDevice, s));
  h->copy_calls += h->sizes.size();
  return AVSG_OK;
}

// The kernels of one decode step for the handle's configuration, enqueued on s.
static avsg_status enqueue_step(avsg_handle* h, const int32_t* d_topk, const int64_t* d_verified_len,
                                int32_t* d_slots, int32_t* d_miss_counts, hipStream_t s) {
  const avsg_config& c = h->cfg;
  h->last_stream = s;
  h->last_counts = d_miss_counts;
  avsg_status rc;
  if ((rc = record(h, 0, s)) != AVSG_OK) return rc;
  if (c.gather_mode == AVSG_GATHER_PIPELINED) {
    MatchParams p{};
    p.B = c.batch; p.K = c.topk; p.n_q = c.n_q; p.S = c.slots; p.m = h->m;
    p.R = c.retry; p.L = c.max_life; p.a1 = c.a1; p.a2 = c.a2;
    p.f_mask = static_cast<uint32_t>((1u << (23 - h->m)) - 1u);
    p.topk = d_topk; p.verified = d_verified_len; p.rows = h->rows_dev;
    p.table_c = h->table_c; p.table_q = h->table_q;
    p.slots_out = d_slots; p.miss_counts = d_miss_counts; p.miss_list = h->miss_list;
    p.stats = h->stats; p.hit_mask = nullptr;
    GatherParams g{};
    g.B = c.batch; g.n_q = c.n_q; g.K = c.topk; g.S = c.slots;
    g.miss_counts = d_miss_counts; g.counts_per_req = c.n_q; g.count_stride = c.n_q;
    g.miss_list = h->miss_list; g.rows = h->rows_dev;
    g.n_streams = c.n_streams; g.host_ptrs = h->host_ptrs; g.buf_ptrs = h->buf_ptrs;
    g.row_bytes0 = c.row_bytes[0];
    g.row_bytes1 = c.n_streams > 1 ? c.row_bytes[1] : 0;
    PipeParams q{};
    q.head = h->pipe_ctl; q.tail = h->pipe_ctl + 1; q.done = h->pipe_ctl + 2;
    q.exit_count = h->pipe_ctl + 3; q.error = h->pipe_ctl + 4; q.last_epoch = h->pipe_ctl + 5;
    q.chunks = h->pipe_chunks; q.max_chunks = h->pipe_max_chunks;
    const int wgs = std::max(c.batch, c.gather_workers > 0 ? c.gather_workers : h->cus);
    HIP_TRY(h, launch_step_pipelined(p, g, q, wgs, h->lds, s));
    if ((rc = record(h, 1, s)) != AVSG_OK) return rc;
    if ((rc = record(h, 2, s)) != AVSG_OK) return rc;
    if (h->timing && h->n_timed < kMaxTimedSteps) h->has_tail[h->n_timed++] = false;
    h->steps++;
    return AVSG_OK;
  }
  if (c.gather_mode == AVSG_GATHER_EARLY) {
    // early list, then Stage One beside the early copies, then the rows that
    // arrived before their slots were known
    MatchParams p{};
    p.B = c.batch; p.K = c.topk; p.n_q = c.n_q; p.S = c.slots; p.m = h->m;
    p.R = c.retry; p.L = c.max_life; p.a1 = c.a1; p.a2 = c.a2;
    p.f_mask = static_cast<uint32_t>((1u << (23 - h->m)) - 1u);
    p.topk = d_topk; p.verified = d_verified_len; p.rows = h->rows_dev;
    p.table_c = h->table_c; p.table_q = h->table_q;
    p.slots_out = d_slots; p.miss_counts = d_miss_counts; p.miss_list = h->miss_list;
    p.stats = h->stats; p.hit_mask = nullptr;
    p.plan_words = h->plan_words;
    p.plan_list_off = h->plan_list_off;
    p.plan_scan_off = h->plan_scan_off;
    p.host_list = h->host_list; p.host_fan = h->host_fan;
    p.res_list = h->res_list; p.rep_list = h->rep_list;
    p.plan_counts = h->plan_counts; p.plan_claim = h->plan_claim;
    p.early_x = h->early_x; p.early_n = h->early_n; p.early_done = h->early_done;
    EarlyParams e{};
    e.B = c.batch; e.K = c.topk; e.n_q = c.n_q; e.S = c.slots;
    e.map_words = early_map_words(c.topk, c.n_q);
    e.topk = d_topk; e.rows = h->rows_dev; e.table_c = h->table_c; e.slots = d_slots;
    e.early_x = h->early_x; e.early_pos = h->early_pos; e.early_n = h->early_n; e.done = h->early_done;
    e.ctl = h->early_ctl; e.fin = h->early_fin; e.stage_rows = h->stage_rows;
    e.direct = c.early_direct == 0 ? 1 : 0;
    e.stage0 = h->stage0; e.stage1 = h->stage1; e.stats = h->stats;
    e.n_streams = c.n_streams; e.host_ptrs = h->host_ptrs; e.buf_ptrs = h->buf_ptrs;
    e.row_bytes0 = c.row_bytes[0];
    e.row_bytes1 = c.n_streams > 1 ? c.row_bytes[1] : 0;
    e.host_list = h->host_list; e.host_fan = h->host_fan; e.res_list = h->res_list; e.rep_list = h->rep_list;
    HIP_TRY(h, launch_early_list(e, h->early_list_lds, s));
    if ((rc = record(h, 1, s)) != AVSG_OK) return rc;
    HIP_TRY(h, launch_step_early(p, e, h->early_workers, h->lds, s));
    if ((rc = record(h, 2, s)) != AVSG_OK) return rc;
    HIP_TRY(h, launch_finish_early(e, std::max(1, h->cus), s));
    if ((rc = record(h, 3, s)) != AVSG_OK) return rc;
    if (h->timing && h->n_timed < kMaxTimedSteps) h->has_tail[h->n_timed++] = true;
    h->steps++;
    return AVSG_OK;
  }
  if (c.match_mode == AVSG_MATCH_HASH) {
    MatchParams p{};
    p.B = c.batch; p.K = c.topk; p.n_q = c.n_q; p.S = c.slots; p.m = h->m;
    p.R = c.retry; p.L = c.max_life; p.a1 = c.a1; p.a2 = c.a2;
    p.f_mask = static_cast<uint32_t>((1u << (23 - h->m)) - 1u);
    p.topk = d_topk; p.verified = d_verified_len; p.rows = h->rows_dev;
    p.table_c = h->table_c; p.table_q = h->table_q;
    p.slots_out = d_slots; p.miss_counts = d_miss_counts; p.miss_list = h->miss_list;
    p.stats = h->stats;
    p.hit_mask = c.gather_mode == AVSG_GATHER_POSITION ? h->hit_mask : nullptr;
    if (c.gather_mode == AVSG_GATHER_RESIDENT) {
      p.plan_words = h->plan_words;
      p.plan_list_off = h->plan_list_off;
      p.plan_scan_off = h->plan_scan_off;
      p.host_list = h->host_list;
      p.host_fan = h->host_fan;
      p.res_list = h->res_list;
      p.rep_list = h->rep_list;
      p.plan_counts = h->plan_counts;
      p.plan_claim = h->plan_claim;
    }
    HIP_TRY(h, launch_match_hash(p, h->lds, s));
  } else {
    DualPtrParams p{};
    p.B = c.batch; p.K = c.topk; p.topk = d_topk; p.rows = h->rows_dev; p.state = h->dp_state;
    p.slots_out = d_slots; p.miss_counts = d_miss_counts; p.miss_list = h->miss_list;
    p.stats = h->stats;
    HIP_TRY(h, launch_match_dualptr(p, h->lds, s));
  }
  if ((rc = record(h, 1, s)) != AVSG_OK) return rc;
  GatherParams g{};
  g.B = c.batch; g.n_q = c.n_q; g.K = c.topk; g.S = c.slots;
  g.miss_counts = d_miss_counts; g.counts_per_req = c.n_q; g.count_stride = c.n_q;
  g.miss_list = h->miss_list; g.rows = h->rows_dev;
  g.n_streams = c.n_streams; g.host_ptrs = h->host_ptrs; g.buf_ptrs = h->buf_ptrs;
  g.row_bytes0 = c.row_bytes[0];
  g.row_bytes1 = c.n_streams > 1 ? c.row_bytes[1] : 0;
  g.topk = d_topk; g.slots = d_slots; g.hit_mask = h->hit_mask;
  switch (c.gather_mode) {
    case AVSG_GATHER_BALANCED: HIP_TRY(h, launch_gather_balanced(g, h->workers, s)); break;
    case AVSG_GATHER_REQUEST: HIP_TRY(h, launch_gather_request(g, s)); break;
    case AVSG_GATHER_POSITION: HIP_TRY(h, launch_gather_position(g, h->workers, s)); break;
    case AVSG_GATHER_RESIDENT: {
      // host list (each row also to its fan slots) and resident copies in one
      // kernel, then the repeats left over
      GatherParams gh = g, gr = g;
      gh.miss_counts = h->plan_counts; gh.counts_per_req = 1; gh.count_stride = 3;
      gh.miss_list = h->host_list; gh.fan = h->host_fan;
      gr.miss_counts = h->plan_counts + 1; gr.counts_per_req = 1; gr.count_stride = 3;
      gr.miss_list = h->res_list;
      HIP_TRY(h, launch_gather_resident(gh, gr, h->plan_claim, h->workers, s));
      if ((rc = record(h, 2, s)) != AVSG_OK) return rc;
      // the host copies also fill each index's two largest repeats, so
      // repeats are left only with four or more tokens per step; they are few
      // and HBM-latency bound, so they get more, smaller workgroups
      if (c.n_q > 3) {
        g.miss_counts = h->plan_counts + 2; g.counts_per_req = 1; g.count_stride = 3;
        g.miss_list = h->rep_list;
        HIP_TRY(h, launch_copy_device(g, kRepeatWorkersPerCu * std::max(1, h->cus), s));
      }
      break;
    }
    case AVSG_GATHER_SDMA:
      if ((rc = sdma_gather(h, d_miss_counts, s)) != AVSG_OK) return rc;
      break;
    default: break;
  }
  // a fourth event only when Stage Two has a tail kernel (each record costs
  // the step stream a few microseconds)
  const bool tail = c.gather_mode == AVSG_GATHER_RESIDENT && c.n_q > 3;
  if (c.gather_mode != AVSG_GATHER_RESIDENT && (rc = record(h, 2, s)) != AVSG_OK) return rc;
  if (tail && (rc = record(h, 3, s)) != AVSG_OK) return rc;
  if (h->timing && h->n_timed < kMaxTimedSteps) h->has_tail[h->n_timed++] = tail;
  h->steps++;
  return AVSG_OK;
}

// Validate mode: every token row's verdict, read back before any table write.
static avsg_status validate_step(avsg_handle* h, const int32_t* d_topk, hipStream_t s) {
  const avsg_config& c = h->cfg;
  const size_t n = static_cast<size_t>(c.batch) * c.n_q;
  HIP_TRY(h, launch_validate_topk(d_topk, h->rows_dev, c.batch, c.n_q, c.topk, h->val_rows, s));
  HIP_TRY(h, hipMemcpyAsync(h->h_val.data(), h->val_rows, n * 4, hipMemcpyDeviceToHost, s));
  HIP_TRY(h, hipStreamSynchronize(s));
  for (size_t i = 0; i < n; ++i)
    if (h->h_val[i] != 0) {
      const int r = static_cast<int>(i / c.n_q), g = static_cast<int>(i % c.n_q);
      set_err(h, "avsg_step: request %d token %d: %s%s%s", r, g,
              (h->h_val[i] & 1) ? "an index outside [0, rows)" : "",
              (h->h_val[i] & 3) == 3 ? " and " : "", (h->h_val[i] & 2) ? "a repeated index" : "");
      return AVSG_E_BADINDEX;
    }
  return AVSG_OK;
}

avsg_status avsg_step(avsg_handle* h, const int32_t* d_topk, const int64_t* d_verified_len,
                      int32_t* d_slots, int32_t* d_miss_counts, void* stream) {
  if (!h || !d_topk || !d_slots || !d_miss_counts) return AVSG_E_INVAL;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != h->device) {
    set_err(h, "avsg_step: the current device is not the one the handle was created on");
    return AVSG_E_INVAL;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (h->cfg.validate) {
    h->last_stream = s;
    const avsg_status rc = validate_step(h, d_topk, s);
    if (rc != AVSG_OK) return rc;
  }
  return enqueue_step(h, d_topk, d_verified_len, d_slots, d_miss_counts, s);
}

// Counters of requests [r0, r1) into *out (steps and lookups counted for
// those requests only).
static avsg_status collect_stats(avsg_handle* h, int r0, int r1, avsg_stats_t* out) {
  const avsg_config& c = h->cfg;
  HIP_TRY(h, hipStreamSynchronize(h->last_stream));
  const size_t n = static_cast<size_t>(r1 - r0) * kNumStats;
  std::vector<unsigned long long> st(n);
  HIP_TRY(h, hipMemcpy(st.data(), h->stats + static_cast<size_t>(r0) * kNumStats, n * 8,
                       hipMemcpyDeviceToHost));
  std::memset(out, 0, sizeof(*out));
  out->steps = h->steps;
  out->lookups = h->steps * static_cast<uint64_t>(r1 - r0) * c.n_q * c.topk;
  uint64_t max_dec = 0;
  for (int r = 0; r < r1 - r0; ++r) {
    const unsigned long long* s = &st[static_cast<size_t>(r) * kNumStats];
    out->hits += s[kStatHits];
    out->misses += s[kStatMisses];
    out->lost_exhausted += s[kStatLostExhausted];
    out->lost_collision += s[kStatLostCollision];
    out->alloc_decays += s[kStatAllocDecays];
    out->revivals += s[kStatRevivals];
    out->invalidations += s[kStatInvalidations];
    out->bad_indices += s[kStatBadIndices];
    out->resident_rows += s[kStatResident];
    out->duplicate_rows += s[kStatDuplicate];
    out->early_rows += s[kStatEarly];
    out->early_staged_rows += s[kStatEarlyStaged];
    out->early_deferred_rows += s[kStatEarlyDeferred];
    max_dec = std::max<uint64_t>(max_dec, s[kStatMaxStepDecays]);
  }
  out->max_step_alloc_decays = static_cast<int32_t>(max_dec);
  uint64_t rb = 0;
  for (int s = 0; s < c.n_streams; ++s) rb += static_cast<uint64_t>(c.row_bytes[s]);
  out->bytes_moved = c.gather_mode == AVSG_GATHER_NONE ? 0 : out->misses * rb;
  out->host_bytes = c.gather_mode == AVSG_GATHER_NONE
                        ? 0
                        : (out->misses - out->resident_rows - out->duplicate_rows) * rb;
  return AVSG_OK;
}

avsg_status avsg_stats(avsg_handle* h, avsg_stats_t* out) {
  if (!h || !out) return AVSG_E_INVAL;
  avsg_status rc = collect_stats(h, 0, h->cfg.batch, out);
  if (rc != AVSG_OK) return rc;
  out->copy_calls = h->copy_calls;
  if (h->cfg.gather_mode == AVSG_GATHER_PIPELINED) {
    int ctl[5] = {0, 0, 0, 0, 0};
    HIP_TRY(h, hipMemcpy(ctl, h->pipe_ctl, sizeof(ctl), hipMemcpyDeviceToHost));
    out->queue_timeouts = ctl[4];
    if (ctl[4]) {
      set_err(h, "pipelined step: a consumer timed out waiting for the chunk queue");
      return AVSG_E_INTERNAL;
    }
  }
  return AVSG_OK;
}

avsg_status avsg_request_stats(avsg_handle* h, int32_t r, avsg_stats_t* out) {
  if (!h || !out || r < 0 || r >= h->cfg.batch) return AVSG_E_INVAL;
  return collect_stats(h, r, r + 1, out);
}

avsg_status avsg_reset_stats(avsg_handle* h, void* stream) {
  if (!h) return AVSG_E_INVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIP_TRY(h, launch_zero_u64(h->stats, static_cast<size_t>(h->cfg.batch) * kNumStats, s));
  h->steps = 0;
  h->copy_calls = 0;
  h->last_stream = s;
  return AVSG_OK;
}

avsg_status avsg_reset_request(avsg_handle* h, int32_t r, void* stream) {
  if (!h || r < 0 || r >= h->cfg.batch) return AVSG_E_INVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t S = static_cast<size_t>(h->cfg.slots);
  if (h->cfg.match_mode == AVSG_MATCH_HASH) {
    HIP_TRY(h, launch_reset_tables(h->table_c + r * S, h->table_q + r * S, S, s));
  } else {
    // a one-request reset of the dual-pointer list: (-1, j) for j = 0..K-1
    HIP_TRY(h, launch_reset_dualptr(h->dp_state + r * S, 1, h->cfg.topk, s));
  }
  h->last_stream = s;
  return AVSG_OK;
}

avsg_status avsg_export_state(avsg_handle* h, int32_t r, int32_t* c_out, uint32_t* q_out) {
  if (!h || !c_out || !q_out || r < 0 || r >= h->cfg.batch) return AVSG_E_INVAL;
  if (h->cfg.match_mode != AVSG_MATCH_HASH) return AVSG_E_UNSUPPORTED;
  const size_t S = static_cast<size_t>(h->cfg.slots);
  HIP_TRY(h, hipStreamSynchronize(h->last_stream));
  HIP_TRY(h, hipMemcpy(c_out, h->table_c + r * S, S * 4, hipMemcpyDeviceToHost));
  HIP_TRY(h, hipMemcpy(q_out, h->table_q + r * S, S * 4, hipMemcpyDeviceToHost));
  return AVSG_OK;
}

avsg_status avsg_import_state(avsg_handle* h, int32_t r, const int32_t* c_in, const uint32_t* q_in,
                              void* stream) {
  if (!h || !c_in || !q_in || r < 0 || r >= h->cfg.batch) return AVSG_E_INVAL;
  if (h->cfg.match_mode != AVSG_MATCH_HASH) return AVSG_E_UNSUPPORTED;
  const size_t S = static_cast<size_t>(h->cfg.slots);
  for (size_t j = 0; j < S; ++j) {
    const int life = static_cast<int8_t>(q_in[j] >> 24);
    if (life < -1 || life > h->cfg.max_life) {
      set_err(h, "avsg_import_state: entry %zu has lifetime %d outside [-1, %d]", j, life, h->cfg.max_life);
      return AVSG_E_RANGE;
    }
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIP_TRY(h, hipMemcpyAsync(h->table_c + r * S, c_in, S * 4, hipMemcpyHostToDevice, s));
  HIP_TRY(h, hipMemcpyAsync(h->table_q + r * S, q_in, S * 4, hipMemcpyHostToDevice, s));
  HIP_TRY(h, hipStreamSynchronize(s));
  h->last_stream = s;
  return AVSG_OK;
}

avsg_status avsg_export_misses(avsg_handle* h, int32_t r, int32_t* n_out, int32_t* x_out,
                               int32_t* o_out) {
  if (!h || !n_out || !x_out || !o_out || r < 0 || r >= h->cfg.batch) return AVSG_E_INVAL;
  const avsg_config& c = h->cfg;
  if (!h->last_counts) {
    *n_out = 0;
    return AVSG_OK;
  }
  HIP_TRY(h, hipStreamSynchronize(h->last_stream));
  std::vector<int32_t> cnt(c.n_q);
  HIP_TRY(h, hipMemcpy(cnt.data(), h->last_counts + static_cast<size_t>(r) * c.n_q, c.n_q * 4,
                       hipMemcpyDeviceToHost));
  int64_t tot = 0;
  for (int g = 0; g < c.n_q; ++g) tot += cnt[g];
  if (tot < 0 || tot > static_cast<int64_t>(c.n_q) * c.topk) return AVSG_E_INTERNAL;
  std::vector<int2> ml(static_cast<size_t>(tot));
  if (tot > 0)
    HIP_TRY(h, hipMemcpy(ml.data(), h->miss_list + static_cast<size_t>(r) * c.n_q * c.topk,
                         static_cast<size_t>(tot) * 8, hipMemcpyDeviceToHost));
  for (int64_t k = 0; k < tot; ++k) {
    x_out[k] = ml[k].x;
    o_out[k] = ml[k].y;
  }
  *n_out = static_cast<int32_t>(tot);
  return AVSG_OK;
}

avsg_status avsg_export_plan(avsg_handle* h, int32_t r, int32_t* n_host, int32_t* host_x,
                             int32_t* host_o, int32_t* host_fan, int32_t* n_res, int32_t* res_src,
                             int32_t* res_dst, int32_t* n_rep, int32_t* rep_src, int32_t* rep_dst) {
  if (!h || !n_host || !host_x || !host_o || !host_fan || !n_res || !res_src || !res_dst || !n_rep ||
      !rep_src || !rep_dst || r < 0 || r >= h->cfg.batch)
    return AVSG_E_INVAL;
  const avsg_config& c = h->cfg;
  if (!has_plan(c)) return AVSG_E_UNSUPPORTED;
  *n_host = *n_res = *n_rep = 0;
  if (!h->last_counts) return AVSG_OK;
  HIP_TRY(h, hipStreamSynchronize(h->last_stream));
  int32_t cnt[3] = {0, 0, 0};
  HIP_TRY(h, hipMemcpy(cnt, h->plan_counts + 3 * static_cast<size_t>(r), sizeof(cnt),
                       hipMemcpyDeviceToHost));
  const int64_t cap = static_cast<int64_t>(c.n_q) * c.topk;
  if (cnt[0] < 0 || cnt[1] < 0 || cnt[2] < 0 ||
      static_cast<int64_t>(cnt[0]) + cnt[1] + cnt[2] > cap)
    return AVSG_E_INTERNAL;
  const size_t base = static_cast<size_t>(r) * c.n_q * c.topk;
  const int2* lists[3] = {h->host_list, h->res_list, h->rep_list};
  int32_t* outs[3][2] = {{host_x, host_o}, {res_src, res_dst}, {rep_src, rep_dst}};
  std::vector<int2> v;
  for (int k = 0; k < 3; ++k) {
    v.resize(static_cast<size_t>(cnt[k]));
    if (cnt[k] > 0)
      HIP_TRY(h, hipMemcpy(v.data(), lists[k] + base, static_cast<size_t>(cnt[k]) * 8,
                           hipMemcpyDeviceToHost));
    for (int i = 0; i < cnt[k]; ++i) {
      outs[k][0][i] = v[i].x;
      outs[k][1][i] = v[i].y;
    }
  }
  if (cnt[0] > 0)
    HIP_TRY(h, hipMemcpy(host_fan, h->host_fan + base, static_cast<size_t>(cnt[0]) * 8,
                         hipMemcpyDeviceToHost));
  *n_host = cnt[0];
  *n_res = cnt[1];
  *n_rep = cnt[2];
  return AVSG_OK;
}

avsg_status avsg_export_early(avsg_handle* h, int32_t r, int32_t* n_out, int32_t* x_out,
                              int32_t* pos_out) {
  if (!h || !n_out || !x_out || !pos_out || r < 0 || r >= h->cfg.batch) return AVSG_E_INVAL;
  const avsg_config& c = h->cfg;
  if (c.gather_mode != AVSG_GATHER_EARLY) return AVSG_E_UNSUPPORTED;
  HIP_TRY(h, hipStreamSynchronize(h->last_stream));
  int32_t n = 0;
  HIP_TRY(h, hipMemcpy(&n, h->early_n + r, 4, hipMemcpyDeviceToHost));
  const int64_t cap = static_cast<int64_t>(c.n_q) * c.topk;
  if (n < 0 || n > cap) return AVSG_E_INTERNAL;
  const size_t base = static_cast<size_t>(r) * c.n_q * c.topk;
  if (n > 0) {
    HIP_TRY(h, hipMemcpy(x_out, h->early_x + base, static_cast<size_t>(n) * 4, hipMemcpyDeviceToHost));
    HIP_TRY(h, hipMemcpy(pos_out, h->early_pos + base, static_cast<size_t>(n) * 16, hipMemcpyDeviceToHost));
  }
  *n_out = n;
  return AVSG_OK;
}

avsg_status avsg_set_timing(avsg_handle* h, int32_t enable) {
  if (!h) return AVSG_E_INVAL;
  h->timing = enable != 0;
  h->n_timed = 0;
  return AVSG_OK;
}

avsg_status avsg_timing(avsg_handle* h, float* match_ms, float* gather_ms, float* tail_ms,
                        int32_t cap, int32_t* n_out) {
  if (!h || !n_out || cap < 0) return AVSG_E_INVAL;
  HIP_TRY(h, hipStreamSynchronize(h->last_stream));
  const size_t n = std::min<size_t>(h->n_timed, static_cast<size_t>(cap));
  for (size_t i = 0; i < n; ++i) {
    float a = 0.f, b = 0.f;
    HIP_TRY(h, hipEventElapsedTime(&a, h->events[i][0], h->events[i][1]));
    HIP_TRY(h, hipEventElapsedTime(&b, h->events[i][1], h->events[i][2]));
    if (tail_ms) {
      float c = 0.f;
      if (h->has_tail[i]) HIP_TRY(h, hipEventElapsedTime(&c, h->events[i][2], h->events[i][3]));
      tail_ms[i] = c;
    }
    if (match_ms) match_ms[i] = a;
    if (gather_ms) gather_ms[i] = b;
  }
  *n_out = static_cast<int32_t>(n);
  return AVSG_OK;
}

avsg_status avsg_destroy(avsg_handle* h) {
  if (!h) return AVSG_E_INVAL;
  (void)hipStreamSynchronize(h->last_stream);
  for (auto& ev : h->events)
    for (auto& x : ev) (void)hipEventDestroy(x);
  if (h->h_counts) (void)hipHostFree(h->h_counts);
  if (h->h_list) (void)hipHostFree(h->h_list);
  delete h;
  return AVSG_OK;
}

avsg_status avsg_host_alloc(size_t bytes, int32_t coherent, void** out) {
  if (!out || bytes == 0) return AVSG_E_INVAL;
  *out = nullptr;
  unsigned flags = hipHostMallocMapped | (coherent ? hipHostMallocCoherent : hipHostMallocNonCoherent);
  if (hipHostMalloc(out, bytes, flags) != hipSuccess) {
    *out = nullptr;
    return AVSG_E_HIP;
  }
  return AVSG_OK;
}

avsg_status avsg_host_free(void* p) {
  if (!p) return AVSG_E_INVAL;
  return hipHostFree(p) == hipSuccess ? AVSG_OK : AVSG_E_HIP;
}

avsg_status avsg_h2d_peak(const void* host, void* device, size_t bytes, int32_t iters, void* stream,
                          double* gbps) {
  if (!host || !device || !gbps || bytes == 0 || iters < 1) return AVSG_E_INVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipEvent_t a, b;
  if (hipEventCreate(&a) != hipSuccess) return AVSG_E_HIP;
  if (hipEventCreate(&b) != hipSuccess) {
    (void)hipEventDestroy(a);
    return AVSG_E_HIP;
  }
  std::vector<float> ms;
  avsg_status rc = AVSG_OK;
  for (int i = 0; i <= iters && rc == AVSG_OK; ++i) {
    if (hipEventRecord(a, s) != hipSuccess ||
        hipMemcpyAsync(device, host, bytes, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipEventRecord(b, s) != hipSuccess || hipEventSynchronize(b) != hipSuccess) {
      rc = AVSG_E_HIP;
      break;
    }
    float t = 0.f;
    if (hipEventElapsedTime(&t, a, b) != hipSuccess) rc = AVSG_E_HIP;
    if (i > 0) ms.push_back(t);
  }
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  if (rc != AVSG_OK) return rc;
  std::sort(ms.begin(), ms.end());
  const double med = ms[ms.size() / 2];
  *gbps = static_cast<double>(bytes) / (med * 1e-3) / 1e9;
  return AVSG_OK;
}

}  // extern "C"

namespace {
constexpr int kMaxStaticDevices = 64;
// Per-GPU state of avsg_step_static (host memory, fixed size).
struct StaticDevice {
  unsigned char* ptr = nullptr;   // device address of `scratch` on this GPU
  size_t match_lds = 0;           // dynamic LDS the matching kernels are prepared for
  size_t dualptr_lds = 0;
  bool has_last = false;          // a call completed since the last failure
  avsg_config last{};             // its configuration
};
StaticDevice g_static[kMaxStaticDevices];
std::mutex g_static_mu;

bool same_config(const avsg_config& a, const avsg_config& b) {
  return a.batch == b.batch && a.topk == b.topk && a.n_q == b.n_q && a.slots == b.slots &&
         a.retry == b.retry && a.max_life == b.max_life && a.a1 == b.a1 && a.a2 == b.a2 &&
         a.n_streams == b.n_streams && a.gather_workers == b.gather_workers &&
         a.row_bytes[0] == b.row_bytes[0] && (a.n_streams < 2 || a.row_bytes[1] == b.row_bytes[1]) &&
         a.match_mode == b.match_mode && a.gather_mode == b.gather_mode;
}

// n values produced by value(i), written to device memory through kernel
// arguments (no host staging that must outlive the call)
template <typename F>
hipError_t put_values(unsigned long long* dst, size_t n, F value, hipStream_t s) {
  unsigned long long chunk[120];
  for (size_t i = 0; i < n; i += 120) {
    const size_t m = std::min<size_t>(120, n - i);
    for (size_t k = 0; k < m; ++k) chunk[k] = value(i + k);
    const hipError_t e = launch_put_u64(dst + i, chunk, m, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
}  // namespace

extern "C" avsg_status avsg_step_static(const avsg_config* cfg, const void* const* host_rows,
                                        const int64_t* rows_per_request, void* const* d_buffers,
                                        const int32_t* d_topk, const int64_t* d_verified_len,
                                        int32_t* d_slots, int32_t* d_miss_counts, int32_t cold_start,
                                        void* stream) {
  avsg_status st = check_config(cfg, nullptr);
  if (st != AVSG_OK) return st;
  const avsg_config c = resolved(*cfg);
  if (c.validate || c.gather_mode == AVSG_GATHER_SDMA || c.gather_mode == AVSG_GATHER_PIPELINED ||
      c.gather_mode == AVSG_GATHER_EARLY) {
    std::fprintf(stderr, "avsg_step_static: validate mode and the copy-engine, pipelined and early-fetch "
                         "transfers are not available without a handle\n");
    return AVSG_E_UNSUPPORTED;
  }
  if (!host_rows || !rows_per_request || !d_buffers || !d_topk || !d_slots || !d_miss_counts)
    return AVSG_E_INVAL;
  if (!rows_ok(c, host_rows, rows_per_request, d_buffers)) return AVSG_E_INVAL;
  const Layout L = layout_of(c);
  if (L.total > AVSG_STATIC_SCRATCH_BYTES) {
    std::fprintf(stderr, "avsg_step_static: this configuration needs %zu bytes of scratch; the library's "
                         "array holds %zu (AVSG_STATIC_SCRATCH_BYTES)\n",
                 L.total, static_cast<size_t>(AVSG_STATIC_SCRATCH_BYTES));
    return AVSG_E_CAPACITY;
  }
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return AVSG_E_HIP;
  if (dev >= kMaxStaticDevices) return AVSG_E_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_static_mu);
  StaticDevice& sd = g_static[dev];
  if (!sd.ptr) {
    // once per GPU, with that GPU current: the array's address on it
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      std::fprintf(stderr, "avsg_step_static: hipGetSymbolAddress: %s\n", hipGetErrorString(e));
      return AVSG_E_HIP;
    }
    sd.ptr = static_cast<unsigned char*>(p);
  }
  if (!cold_start && !(sd.has_last && same_config(sd.last, c))) {
    std::fprintf(stderr, "avsg_step_static: cold_start = 0 continues the tables of the previous call on "
                         "this GPU, which must have succeeded with the same configuration\n");
    return AVSG_E_INVAL;
  }
  sd.has_last = false;

  avsg_handle h;   // section pointers into this GPU's array; allocates nothing
  h.cfg = c;
  h.device = dev;
  h.m = log2_exact(c.slots);
  bind_workspace(&h, sd.ptr, L);
  h.cus = device_cus();
  h.workers = c.gather_workers > 0 ? c.gather_workers : std::max(1, h.cus);
  int max_lds = 0;
  if (hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return AVSG_E_HIP;
  if (c.match_mode == AVSG_MATCH_HASH) {
    h.lds = stage_one_lds_bytes(c.slots, c.topk, c.n_q, has_plan(c));
    if (max_lds > 0 && h.lds > static_cast<size_t>(max_lds)) return AVSG_E_CAPACITY;
    if (sd.match_lds < h.lds) {
      if (prepare_match_hash(h.lds) != hipSuccess) return AVSG_E_HIP;
      sd.match_lds = h.lds;
    }
  } else {
    h.lds = dualptr_lds_bytes(c.topk);
    if (sd.dualptr_lds < h.lds) {
      if (prepare_match_dualptr(h.lds) != hipSuccess) return AVSG_E_HIP;
      sd.dualptr_lds = h.lds;
    }
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t B = static_cast<size_t>(c.batch), nsb = static_cast<size_t>(c.n_streams) * B;
  for (size_t i = 0; i < nsb; ++i) {
    void* dp = nullptr;
    if (hipHostGetDevicePointer(&dp, const_cast<void*>(host_rows[i]), 0) != hipSuccess || !dp) {
      std::fprintf(stderr, "avsg_step_static: host rows must be pinned, device-mapped memory\n");
      return AVSG_E_INVAL;
    }
  }
  hipError_t e = put_values(
      reinterpret_cast<unsigned long long*>(h.host_ptrs), nsb,
      [&](size_t i) {
        void* dp = nullptr;
        (void)hipHostGetDevicePointer(&dp, const_cast<void*>(host_rows[i]), 0);
        return static_cast<unsigned long long>(reinterpret_cast<uintptr_t>(dp));
      },
      s);
  if (e == hipSuccess)
    e = put_values(reinterpret_cast<unsigned long long*>(h.buf_ptrs), nsb,
                   [&](size_t i) { return static_cast<unsigned long long>(reinterpret_cast<uintptr_t>(d_buffers[i])); },
                   s);
  if (e == hipSuccess)
    e = put_values(reinterpret_cast<unsigned long long*>(h.rows_dev), B,
                   [&](size_t i) { return static_cast<unsigned long long>(rows_per_request[i]); }, s);
  if (e == hipSuccess && cold_start) {
    // every table empty and the counters at zero (fill kernels)
    if (c.match_mode == AVSG_MATCH_HASH)
      e = launch_reset_tables(h.table_c, h.table_q, B * static_cast<size_t>(c.slots), s);
    else
      e = launch_reset_dualptr(h.dp_state, c.batch, c.topk, s);
    if (e == hipSuccess) e = launch_zero_u64(h.stats, B * kNumStats, s);
  }
  if (e != hipSuccess) {
    std::fprintf(stderr, "avsg_step_static: %s\n", hipGetErrorString(e));
    return AVSG_E_HIP;
  }
  st = enqueue_step(&h, d_topk, d_verified_len, d_slots, d_miss_counts, s);
  if (st != AVSG_OK) {
    std::fprintf(stderr, "avsg_step_static: %s\n", h.err);
    return st;
  }
  sd.last = c;
  sd.has_last = true;
  return AVSG_OK;
}
