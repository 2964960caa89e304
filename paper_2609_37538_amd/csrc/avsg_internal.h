// Internal declarations shared by the translation units of libavsg (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace avsg {

// Threads of one matching workgroup (one request per workgroup).
constexpr int kMatchThreads = 1024;
// Threads of one gather workgroup.
constexpr int kGatherThreads = 256;
// Misses staged per gather tile.
constexpr int kGatherTile = 64;
// XCDs of an MI355X (gfx950): 8 accelerator dies of 32 CUs, each with its own L2.
constexpr int kXcds = 8;

// Per-request device counters (uint64 each, cumulative).
enum StatIndex : int {
  kStatHits = 0,
  kStatMisses,
  kStatLostExhausted,
  kStatLostCollision,
  kStatAllocDecays,
  kStatRevivals,
  kStatInvalidations,
  kStatBadIndices,
  kStatMaxStepDecays,
  kStatResident,
  kStatDuplicate,
  kStatEarly,          // rows fetched before Stage One (early-fetch transfer)
  kStatEarlyStaged,    // of those, rows parked in HBM staging until their slots were known
  kStatEarlyDeferred,  // of those, rows read from the host only after Stage One (staging full)
  kNumStats
};

// Word written to every bucket/slot by a reset: lifetime -1, invalid, fp 0, slot 0.
constexpr uint32_t kEmptyWord = 0xFF800000u;

struct MatchParams {
  int32_t B, K, n_q, S, m, R, L;
  uint32_t a1, a2;
  uint32_t f_mask;              // F - 1, F = 2^(23-m)
  const int32_t* topk;          // [B][n_q][K]
  const int64_t* verified;      // [B] or nullptr
  const int64_t* rows;          // [B]
  int32_t* table_c;             // [B][S]
  uint32_t* table_q;            // [B][S]
  int32_t* slots_out;           // [B][n_q][K]
  int32_t* miss_counts;         // [B][n_q]
  int2* miss_list;              // [B][n_q*K]  (index, slot)
  unsigned long long* stats;    // [B][kNumStats]
  uint8_t* hit_mask;            // [B][n_q][K] 1 = hit, or nullptr (not written)
  // Stage Two plan of the resident-reuse gather (written when plan_words > 0)
  int32_t plan_words;           // words of the end-of-step index map in LDS
  int32_t plan_list_off;        // LDS byte offset of the step's transfer list kept as 16-bit slots
  int32_t plan_scan_off;        // LDS byte offset of the scan's per-wave candidate lists (0: none)
  int2* host_list;              // [B][n_q*K] (index, slot) copied from the host
  int2* host_fan;               // [B][n_q*K] the two further slots a host entry is also copied to (-1: none)
  int2* res_list;               // [B][n_q*K] (source slot, slot): row already resident
  int2* rep_list;               // [B][n_q*K] (source slot, slot): repeat of a host entry
  int32_t* plan_counts;         // [B][3] host, resident, repeat entries
  int32_t* plan_claim;          // [2] resident and host rows claimed by the gather (reset here)
  // early-fetch transfer (nullptr otherwise): the keys fetched before Stage
  // One leave the plan, and each request flags when its O is final
  const int32_t* early_x;       // [B][n_q*K] early keys of each request
  const int32_t* early_n;       // [B] number of early keys
  uint32_t* early_done;         // [B] 1 once the request's slots are written
};

struct GatherParams {
  int32_t B, n_q, K, S;
  // entry counts of request r: miss_counts[r * count_stride + g], g < counts_per_req
  const int32_t* miss_counts;
  int32_t counts_per_req, count_stride;
  const int2* miss_list;        // [B][n_q*K] (index or source slot, slot)
  const int2* fan;              // [B][n_q*K] two further destination slots per entry (-1: none), or nullptr
  const int64_t* rows;          // [B]
  int32_t n_streams;
  const uint64_t* host_ptrs;    // [n_streams][B] device-visible addresses of host row 0
  const uint64_t* buf_ptrs;     // [n_streams][B] device buffer base addresses
  int64_t row_bytes0, row_bytes1;
  // position-level assignment only
  const int32_t* topk;          // [B][n_q][K]
  const int32_t* slots;         // [B][n_q][K]
  const uint8_t* hit_mask;      // [B][n_q][K]
};

// Device-wide chunk queue of the pipelined step (workspace resident).
struct PipeParams {
  int* head;          // next queue entry to claim
  int* tail;          // queue entries reserved by producers
  int* done;          // requests whose Stage One has finished
  int* exit_count;    // workgroups that have left
  int* error;         // set when a consumer gave up waiting
  int* last_epoch;    // stamp of the last finished step (advanced on the device)
  int4* chunks;       // [max_chunks] (request, first miss, count, epoch)
  int max_chunks;
  int epoch;          // this step's stamp, never 0 (set by the kernel from last_epoch)
};

// Early-fetch transfer: the rows of indices that no slot held when the step
// began are read from the host while Stage One runs (workspace resident).
struct EarlyParams {
  int32_t B, K, n_q, S;
  uint32_t map_words;           // LDS map of the list kernel
  const int32_t* topk;          // [B][n_q][K]
  const int64_t* rows;          // [B]
  const int32_t* table_c;       // [B][S] cached indices as the step begins
  const int32_t* slots;         // [B][n_q][K] O of this step
  int32_t* early_x;             // [B][n_q*K] early keys
  int4* early_pos;              // [B][n_q*K] flat positions g*K+i of each key, -1 padded
  int32_t* early_n;             // [B]
  uint32_t* done;               // [B] O final (set by the matching workgroups)
  int* ctl;                     // [0] rows claimed, [1] staging rows claimed, [2] finish entries
  int4* fin;                    // [B*n_q*K] (request, key, staging row or -1, 0) left to finish
  int32_t stage_rows;           // staging capacity in rows (0: none)
  int32_t direct;               // write rows straight into known slots
  uint64_t stage0, stage1;      // staging bases per stream
  unsigned long long* stats;    // [B][kNumStats]
  int32_t n_streams;
  const uint64_t* host_ptrs;    // [n_streams][B]
  const uint64_t* buf_ptrs;     // [n_streams][B]
  int64_t row_bytes0, row_bytes1;
  // the matching workgroup's own lists (resident-reuse plan of the rest)
  const int2* host_list;
  const int2* host_fan;
  const int2* res_list;
  const int2* rep_list;
};

struct DualPtrParams {
  int32_t B, K;
  const int32_t* topk;          // [B][K]
  const int64_t* rows;          // [B]
  int2* state;                  // [B][K] (cached id, slot) sorted by id
  int32_t* slots_out;           // [B][K]
  int32_t* miss_counts;         // [B]
  int2* miss_list;              // [B][K]
  unsigned long long* stats;    // [B][kNumStats]
};

// LDS bytes of the matching kernel for (S, K); 0 if K exceeds the supported
// indices per thread.
size_t match_lds_bytes(int S, int K);
// threads of the matching workgroup for (S, K)
int match_threads(int S, int K);
size_t dualptr_lds_bytes(int K);

hipError_t launch_match_hash(const MatchParams& p, size_t lds, hipStream_t s);
hipError_t prepare_match_hash(size_t lds);
hipError_t launch_reset_tables(int32_t* c, uint32_t* q, size_t n, hipStream_t s);
hipError_t launch_zero_u64(unsigned long long* p, size_t n, hipStream_t s);
// validate mode: verdict[B * n_q] per token row (1 index out of range, 2 index
// repeated, 3 both, 0 valid); K <= 8192
hipError_t launch_validate_topk(const int32_t* topk, const int64_t* rows, int B, int n_q, int K,
                                int32_t* verdict, hipStream_t s);
// n 64-bit values from host memory to device memory through kernel arguments
// (the host array may be reused as soon as the call returns)
hipError_t launch_put_u64(unsigned long long* dst, const unsigned long long* v, size_t n, hipStream_t s);
hipError_t launch_gather_balanced(const GatherParams& p, int workers, hipStream_t s);
hipError_t launch_gather_request(const GatherParams& p, hipStream_t s);
hipError_t launch_gather_position(const GatherParams& p, int workers, hipStream_t s);
// device-to-device row copies: miss_list entries are (source slot, slot)
hipError_t launch_copy_device(const GatherParams& p, int workers, hipStream_t s);
// resident-reuse Stage Two: host entries, then resident copies, both claimed
// tile by tile; `dev` describes the resident list, `claim` the two counters
hipError_t launch_gather_resident(const GatherParams& host, const GatherParams& dev, int* claim,
                                  int workers, hipStream_t s);
// words of the end-of-step index map the matching kernel can hold for (S, K, n_q);
// 0 when the plan does not fit in the kernel's LDS
int plan_map_words(int S, int K, int n_q);
// LDS byte offset of the transfer list the matching kernel keeps for the plan
size_t plan_list_offset(int S, int K, int n_q);
size_t plan_scan_offset(int S, int K, int n_q);
// dynamic LDS of the matching workgroup for (S, K, n_q), with room for the
// end-of-step plan when `plan`; 0 when it does not fit
size_t stage_one_lds_bytes(int S, int K, int n_q, bool plan);
int pipelined_chunk_misses();
size_t pipelined_lds_bytes(int S, int K);
hipError_t prepare_step_pipelined(size_t lds);
hipError_t launch_step_pipelined(const MatchParams& mp, const GatherParams& gp, const PipeParams& q,
                                 int workgroups, size_t lds, hipStream_t s);
// early-fetch step: list kernel (one workgroup per request), matching +
// early copies in one launch (B matching workgroups + `workers` copiers), then
// the finishing kernel for rows fetched before their slots were known
uint32_t early_map_words(int K, int n_q);
size_t early_list_lds_bytes(int K, int n_q);
size_t early_step_lds_bytes(int S, int K, int n_q);
hipError_t prepare_step_early(size_t list_lds, size_t step_lds);
hipError_t launch_early_list(const EarlyParams& e, size_t lds, hipStream_t s);
hipError_t launch_step_early(const MatchParams& mp, const EarlyParams& e, int workers, size_t lds,
                             hipStream_t s);
hipError_t launch_finish_early(const EarlyParams& e, int workers, hipStream_t s);
hipError_t launch_match_dualptr(const DualPtrParams& p, size_t lds, hipStream_t s);
hipError_t prepare_match_dualptr(size_t lds);
hipError_t launch_reset_dualptr(int2* state, int B, int K, hipStream_t s);

}  // namespace avsg
