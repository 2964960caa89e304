// Stage One of AVSG on gfx950: vectorized open-addressing hash matching,
// lifetime-based slot reservation and shared MTP reservations.
//
// One workgroup of 1024 threads (16 wave64s; 256 threads for tables of at
// most 1024 slots and 512 indices per token) owns one request.  The request's
// Hash-State table (Section 3.2: cached index c_j and metadata word q_j, Eq. 2)
// is staged from HBM into LDS as three arrays -- c[S] (int32), the low 24 bits
// of q (invalid | fingerprint | slot) and the lifetime byte -- so lifetime
// updates and mapping installs never share an LDS word.
//
// The first token's decay of every lifetime (Algorithm 1's global pre-decay) is
// applied to the lifetime bytes as they are staged in.  Per query token
// (Algorithm 1; tokens run in order on the shared table, Algorithm 4):
//   A  every index is probed by its own lane (Probe, Eq. 8-11; a lane's
//      chains advance together, the reads of two rounds issued at once);
//      hits refresh their slot's lifetime to L and
//      write their slot; misses are ranked in index order by wave ballots;
//   B  misses are compacted into dense LDS arrays (index, position); each
//      thread loads the lifetimes it owns (a contiguous run) as whole words
//      and counts its dead slots; a wave scan gives dead ranks;
//   C  if fewer than n_g slots are dead, the decay loop of Algorithm 1 is
//      evaluated as counts of lifetimes below k and all k* decays are applied
//      at once; the first n_g dead slots in increasing order (CollectDead,
//      Eq. 12) become o^miss;
//   D  the misses, one per lane, walk their reusable chains (Eq. 4) on the
//      table as it was before this token's writes (UpdateState, Algorithm 2);
//   E  each miss takes its slot (c = index, lifetime = L) and bids for its
//      bucket with an LDS atomic max on (marker | token | o^miss | fingerprint),
//      so a later token, then the largest miss rank, keeps a contended bucket
//      (a sequential scatter); a bucket holding a bid is read as a valid
//      mapping by every later reader and is rewritten in the canonical Eq. 3
//      layout when the table goes back to HBM.
// After the last token, speculative invalidation (c_j >= N -> -1) is fused
// into the write back.  With the resident-reuse gather the workgroup then
// plans Stage Two (plan_request): which misses need the host link and which
// can be filled from a slot that already holds their row.
#include "match_body.h"

namespace avsg {
namespace {

struct NoPublish {
  __device__ __forceinline__ void operator()(int, int, int) const {}
};

template <int IPT, int NT, int SPT>
__global__ __launch_bounds__(NT) void match_hash_kernel(MatchParams p) {
  extern __shared__ __align__(16) unsigned char lds[];
  NoPublish none;
  match_request<IPT, NT, SPT>(p, static_cast<int>(blockIdx.x), lds, none);
}

__global__ void reset_tables_kernel(int32_t* c, uint32_t* q, size_t n) {
  for (size_t j = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; j < n;
       j += static_cast<size_t>(gridDim.x) * blockDim.x) {
    c[j] = -1;
    q[j] = kEmptyWord;
  }
}

__global__ void zero_u64_kernel(unsigned long long* p, size_t n) {
  for (size_t j = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; j < n;
       j += static_cast<size_t>(gridDim.x) * blockDim.x)
    p[j] = 0ull;
}

constexpr int kSmallThreads = 256;
constexpr int kValidateThreads = 256;

// Selection check of the validate mode, one workgroup per token row (request
// r = row / n_q): every index must lie in [0, rows_r) and appear once in the
// row (a token's top-K list holds K distinct indices).  An LDS set of P >= 2K
// words (index + 1, 0 = empty, linear probing) finds repeats.  verdict[row] =
// 1 if an index is out of range, | 2 if an index repeats, 0 if the row is
// valid.
__global__ __launch_bounds__(kValidateThreads) void validate_topk_kernel(const int32_t* topk,
                                                                         const int64_t* rows, int K,
                                                                         int n_q, uint32_t P,
                                                                         int32_t* verdict) {
  extern __shared__ uint32_t seen[];   // [P]
  __shared__ int flags;
  const int row = static_cast<int>(blockIdx.x), tid = static_cast<int>(threadIdx.x);
  const int64_t rows_r = rows[row / n_q];
  for (uint32_t j = tid; j < P; j += kValidateThreads) seen[j] = 0u;
  if (tid == 0) flags = 0;
  __syncthreads();
  const int32_t* x = topk + static_cast<size_t>(row) * K;
  int f = 0;
  for (int i = tid; i < K; i += kValidateThreads) {
    const int32_t v = x[i];
    if (v < 0 || static_cast<int64_t>(v) >= rows_r) {
      f |= 1;
      continue;
    }
    const uint32_t key = static_cast<uint32_t>(v) + 1u;
    uint32_t h = (static_cast<uint32_t>(v) * 0x9E3779B1u) & (P - 1u);
    for (uint32_t t = 0; t < P; ++t) {   // at most K keys in P >= 2K words: an empty word is reached
      const uint32_t w = atomicCAS(&seen[h], 0u, key);
      if (w == 0u) break;
      if (w == key) {
        f |= 2;
        break;
      }
      h = (h + 1u) & (P - 1u);
    }
  }
  if (f) atomicOr(&flags, f);
  __syncthreads();
  if (tid == 0) verdict[row] = flags;
}

// Values written by one launch of put_u64_kernel; the chunk travels in the
// kernel arguments, so a caller's host array needs to live only for the launch
// call.
constexpr int kPutWords = 120;
struct PutChunk {
  unsigned long long* dst;
  int32_t n;
  int32_t pad;
  unsigned long long v[kPutWords];
};

__global__ void put_u64_kernel(PutChunk c) {
  for (int i = static_cast<int>(threadIdx.x); i < c.n; i += static_cast<int>(blockDim.x)) c.dst[i] = c.v[i];
}

}  // namespace

uint32_t validate_set_words(int K) {
  uint32_t P = 1;
  while (P < 2u * static_cast<uint32_t>(K)) P <<= 1;
  return P;
}

hipError_t launch_validate_topk(const int32_t* topk, const int64_t* rows, int B, int n_q, int K,
                                int32_t* verdict, hipStream_t s) {
  const uint32_t P = validate_set_words(K);
  const size_t lds = 4 * static_cast<size_t>(P);
  if (lds > 64 * 1024) return hipErrorInvalidValue;
  hipLaunchKernelGGL(validate_topk_kernel, dim3(static_cast<unsigned>(B) * static_cast<unsigned>(n_q)),
                     dim3(kValidateThreads), lds, s, topk, rows, K, n_q, P, verdict);
  return hipGetLastError();
}

hipError_t launch_put_u64(unsigned long long* dst, const unsigned long long* v, size_t n, hipStream_t s) {
  for (size_t i = 0; i < n; i += kPutWords) {
    PutChunk c{};
    c.dst = dst + i;
    c.n = static_cast<int32_t>(n - i < static_cast<size_t>(kPutWords) ? n - i : kPutWords);
    for (int k = 0; k < c.n; ++k) c.v[k] = v[i + k];
    hipLaunchKernelGGL(put_u64_kernel, dim3(1), dim3(128), 0, s, c);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Threads of the matching workgroup for (S, K): a table of at most 1024 slots
// with at most 512 indices per token runs on four waves (each thread owns at
// most four lifetimes and two indices; fewer waves wait at every barrier),
// anything larger on sixteen.  Measured at batch 1 and 64: S = K = 256 15.3
// against 17.4 µs, S = K = 512 17.2 against 17.9 µs; at S = 4096, K = 512
// four waves are slower (12.2 against 10.9 µs: sixteen lifetimes per thread).
int match_threads(int S, int K) {
  return (S <= 1024 && K <= 2 * kSmallThreads) ? kSmallThreads : kMatchThreads;
}

static int ipt_for(int S, int K) {
  const int nt = match_threads(S, K);
  return (K + nt - 1) / nt;
}

size_t match_lds_bytes(int S, int K) {
  const int ipt = ipt_for(S, K);
  if (ipt < 1 || ipt > kMaxIPT || S > kMaxSPT * match_threads(S, K)) return 0;
  return 8 * static_cast<size_t>(S) + align16(S) + 12 * static_cast<size_t>(K) +
         4 * static_cast<size_t>(kScratchInts);
}

// LDS of one workgroup (gfx950), the bound of the end-of-step plan's map.
constexpr size_t kWorkgroupLds = 160 * 1024;

// The plan's LDS: c[] (4 S bytes, padded to 16) stays, then the reservation
// bitmap, P map words, P fan words and its counters.  Where there is room, the
// step's transfer list (2 bytes per entry, n_q K entries at most) is kept at
// the end, past both the token loop's arrays and the plan's words, and behind
// it the scan's candidate lists (kPlanScanList 16-bit slots per wave);
// otherwise the plan reads the list back from device memory, or walks each
// lane's candidates in that lane.
static size_t plan_list_bytes(int K, int n_q) { return align16(2 * static_cast<size_t>(n_q) * K); }

static size_t plan_scan_bytes(int S, int K) {
  return align16(2 * static_cast<size_t>(kPlanScanList) * (match_threads(S, K) / 64));
}

static size_t plan_words_end(int S, long long P) {
  return align16(4 * static_cast<size_t>(S)) + 4 * plan_state_words(S, static_cast<int>(P));
}

// P for `words` free LDS words (map and fan words take P each): a power of
// two where one fits, else a multiple of four; at most four words per key and
// at least 1.5 (the map is at most two-thirds full); 0 if that does not fit
static long long plan_words_for(long long words, long long keys) {
  const long long need = (3 * keys + 1) / 2;
  long long P = (4 * keys < words / 2 ? 4 * keys : words / 2) & ~3ll;
  long long pow2 = 1;
  while (2 * pow2 <= P) pow2 *= 2;
  P = pow2 >= need ? pow2 : P;
  return P >= need ? P : 0;
}

struct PlanLayout {
  int P;             // map words (0: no plan fits)
  size_t list_off;   // LDS offset of the kept transfer list (0: none)
  size_t scan_off;   // LDS offset of the scan's candidate lists (0: none)
  size_t total;      // LDS bytes of the matching workgroup
};

// Tried in order: the list and the candidate lists, the list alone, neither.
static PlanLayout plan_layout(int S, int K, int n_q) {
  const size_t m = match_lds_bytes(S, K);
  if (m == 0 || n_q < 1 || S > 32768) return {0, 0, 0, 0};   // kept slots and fan fields are 16-bit values
  const size_t A = align16(4 * static_cast<size_t>(S));
  const long long keys = static_cast<long long>(n_q) * K;
  const long long fixed = plan_bitmap_words(S) + kPlanMiscWords;   // besides map and fan words
  const size_t list = plan_list_bytes(K, n_q), scan = plan_scan_bytes(S, K);
  for (int with_scan = 1; with_scan >= 0; --with_scan) {
    const size_t extra = list + (with_scan ? scan : 0);
    if (align16(m) + extra > kWorkgroupLds) continue;
    const long long P = plan_words_for(static_cast<long long>((kWorkgroupLds - extra - A) / 4) - fixed, keys);
    if (P == 0) continue;
    const size_t e = plan_words_end(S, P), off = align16(m > e ? m : e);
    return {static_cast<int>(P), off, with_scan ? off + list : 0, off + extra};
  }
  const long long P = plan_words_for(static_cast<long long>((kWorkgroupLds - A) / 4) - fixed, keys);
  if (P == 0) return {0, 0, 0, 0};
  const size_t e = plan_words_end(S, P);
  return {static_cast<int>(P), 0, 0, m > e ? m : e};
}

int plan_map_words(int S, int K, int n_q) { return plan_layout(S, K, n_q).P; }

size_t plan_list_offset(int S, int K, int n_q) { return plan_layout(S, K, n_q).list_off; }

size_t plan_scan_offset(int S, int K, int n_q) { return plan_layout(S, K, n_q).scan_off; }

size_t stage_one_lds_bytes(int S, int K, int n_q, bool plan) {
  const size_t m = match_lds_bytes(S, K);
  if (m == 0 || !plan) return m;
  return plan_layout(S, K, n_q).total;
}

// The instantiations: lifetimes per thread S / NT is a power of two up to 16
// with 1024 threads (S <= 16384) and up to 4 with 256 (S <= 1024).
template <int IPT, int NT>
static const void* match_kernel_for(int spt) {
  switch (spt) {
    case 1: return reinterpret_cast<const void*>(&match_hash_kernel<IPT, NT, 1>);
    case 2: return reinterpret_cast<const void*>(&match_hash_kernel<IPT, NT, 2>);
    case 4: return reinterpret_cast<const void*>(&match_hash_kernel<IPT, NT, 4>);
    default: break;
  }
  if constexpr (NT == kMatchThreads) {
    if (spt == 8) return reinterpret_cast<const void*>(&match_hash_kernel<IPT, NT, 8>);
    if (spt == 16) return reinterpret_cast<const void*>(&match_hash_kernel<IPT, NT, 16>);
  }
  return nullptr;
}

static const void* match_kernel(int S, int K) {
  const int nt = match_threads(S, K), ipt = ipt_for(S, K), spt = S >= nt ? S / nt : 1;
  if (nt == kSmallThreads) {
    switch (ipt) {
      case 1: return match_kernel_for<1, kSmallThreads>(spt);
      case 2: return match_kernel_for<2, kSmallThreads>(spt);
      default: return nullptr;
    }
  }
  switch (ipt) {
    case 1: return match_kernel_for<1, kMatchThreads>(spt);
    case 2: return match_kernel_for<2, kMatchThreads>(spt);
    case 3: return match_kernel_for<3, kMatchThreads>(spt);
    case 4: return match_kernel_for<4, kMatchThreads>(spt);
    default: return nullptr;
  }
}

hipError_t prepare_match_hash(size_t lds) {
  static const int spts[] = {1, 2, 4, 8, 16};
  for (int ipt = 1; ipt <= kMaxIPT; ++ipt)
    for (int spt : spts) {
      const void* k[2] = {nullptr, nullptr};
      switch (ipt) {
        case 1: k[0] = match_kernel_for<1, kMatchThreads>(spt); k[1] = match_kernel_for<1, kSmallThreads>(spt); break;
        case 2: k[0] = match_kernel_for<2, kMatchThreads>(spt); k[1] = match_kernel_for<2, kSmallThreads>(spt); break;
        case 3: k[0] = match_kernel_for<3, kMatchThreads>(spt); break;
        case 4: k[0] = match_kernel_for<4, kMatchThreads>(spt); break;
        default: break;
      }
      for (const void* f : k) {
        if (!f) continue;
        const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (e != hipSuccess) return e;
      }
    }
  return hipSuccess;
}

hipError_t launch_match_hash(const MatchParams& p, size_t lds, hipStream_t s) {
  const void* f = match_kernel(p.S, p.K);
  if (!f) return hipErrorInvalidValue;
  MatchParams args = p;
  void* argv[] = {&args};
  return hipLaunchKernel(f, dim3(p.B), dim3(match_threads(p.S, p.K)), argv, lds, s);
}

hipError_t launch_reset_tables(int32_t* c, uint32_t* q, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(reset_tables_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, c, q, n);
  return hipGetLastError();
}

hipError_t launch_zero_u64(unsigned long long* p, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(zero_u64_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace avsg
