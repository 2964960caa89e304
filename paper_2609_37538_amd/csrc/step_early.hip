// Early-fetch decode step on gfx950: the host link starts before Stage One.
//
// An index that no slot of its request holds when the step begins must miss
// where it first occurs (the hit test of Eq. 10 needs c[o] == x) and can be
// in no slot outside the step's reservations afterwards, so the paper's Stage
// Two reads its row from the host whatever slots Stage One picks.  Such rows
// are fetched while Stage One runs, in three launches on one stream, none of
// which waits on another workgroup:
//   1. early_list_kernel (one workgroup per request): the distinct valid
//      indices of the step's tokens that no slot holds, each listed at most
//      four times, with their flat positions g*K + i;
//   2. step_early_kernel: workgroups 0..B-1 run Stage One for their request
//      (the matching kernel's code), raise a flag once the request's O is
//      written, plan the remaining misses (resident-reuse plan without the
//      early keys) and copy them; the other workgroups claim tiles of early
//      rows across the batch and copy each row straight into the slots of its
//      positions when its request's flag is up, else into HBM staging;
//   3. finish_early_kernel: rows parked in staging (or, when staging was
//      full, read from the host now) go to their slots.
// Slots, counts, tables and buffer bytes are those of the paper's Stage Two.
#include "gather_body.h"
#include "match_body.h"

namespace avsg {
namespace {

constexpr uint32_t kEarlyCached = 0x80000000u;   // some slot holds the key
constexpr uint32_t kEarlyKey = 0x40000000u;      // the word is an early key
constexpr uint32_t kEarlyCount = 0x3FFFFFFFu;    // positions counted while listing
constexpr int kEarlyMaxPos = 4;                  // positions kept per key (an int4)
#ifndef AVSG_EARLY_TILE
#define AVSG_EARLY_TILE 64
#endif
#ifndef AVSG_EARLY_UNROLL
#define AVSG_EARLY_UNROLL 2
#endif
constexpr int kEarlyTile = AVSG_EARLY_TILE;      // early rows per claimed tile
constexpr int kEarlyUnroll = AVSG_EARLY_UNROLL;  // loads in flight per lane of a copy workgroup
constexpr int kListTile = 64;                    // rows per tile of the matching workgroup's lists
constexpr int kEarlyMaxBatch = 1024;

struct NoPublish {
  __device__ __forceinline__ void operator()(int, int, int) const {}
};

__device__ __forceinline__ int load_agent(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Home word of index x in a map of P words (multiplicative hash).
__device__ __forceinline__ uint32_t early_home(int32_t x, uint32_t P) {
  return static_cast<uint32_t>((static_cast<uint64_t>(static_cast<uint32_t>(x) * 0x9E3779B1u) * P) >> 32);
}

// Word holding key x, or -1 (linear probing; the map always has an empty word).
__device__ __forceinline__ int early_find(const int32_t* skey, uint32_t P, int32_t x) {
  uint32_t h = early_home(x, P);
  for (uint32_t t = 0; t < P; ++t) {
    const int32_t k = skey[h];
    if (k == x) return static_cast<int>(h);
    if (k == -1) return -1;
    h = (h + 1u == P) ? 0u : h + 1u;
  }
  return -1;
}

// ---- 1. the early list of one request ---------------------------------------
// LDS: key[P] (index or -1) and meta[P]: while listing, the number of
// positions of the key plus kEarlyCached; once compacted, kEarlyKey | list
// index << 8, with the low byte counting the positions written.  The step's
// selections and the request's cached indices are loaded into registers
// together at the start (kListPX positions and kListPC slots per thread per
// round; larger requests take more rounds).
constexpr int kListPX = 8;
constexpr int kListPC = 8;

template <int NT>
__global__ __launch_bounds__(NT) void early_list_kernel(EarlyParams e) {
  extern __shared__ __align__(16) unsigned char lds[];
  constexpr int MW = NT / 64;
  const uint32_t P = e.map_words;
  int32_t* skey = reinterpret_cast<int32_t*>(lds);
  uint32_t* smeta = reinterpret_cast<uint32_t*>(skey + P);
  int* swc = reinterpret_cast<int*>(smeta + P);   // [MW] keys per wave
  const int r = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
  const int nk = e.n_q * e.K, S = e.S;
  const size_t lb = static_cast<size_t>(r) * nk;
  const int32_t* xr = e.topk + lb;
  const int32_t* cr = e.table_c + static_cast<size_t>(r) * S;
  const int64_t rows_r = e.rows[r];
  auto valid = [&](int32_t x) { return x >= 0 && static_cast<int64_t>(x) < rows_r; };

  int32_t xs[kListPX], cs[kListPC];
#pragma unroll
  for (int u = 0; u < kListPX; ++u) xs[u] = u * NT + tid < nk ? xr[u * NT + tid] : -1;
#pragma unroll
  for (int u = 0; u < kListPC; ++u) cs[u] = u * NT + tid < S ? cr[u * NT + tid] : -1;

  // the step's flags and counters start over (the previous step's kernels
  // have finished: same stream)
  if (tid == 0) {
    e.done[r] = 0u;
    if (r == 0) {
      e.ctl[0] = 0;
      e.ctl[1] = 0;
      e.ctl[2] = 0;
    }
  }
  for (uint32_t h = tid; h < P; h += NT) {
    skey[h] = -1;
    smeta[h] = 0u;
  }
  __syncthreads();

  // one word per distinct valid index, counting its positions
  auto insert = [&](int32_t x) {
    uint32_t h = early_home(x, P);
    for (uint32_t t = 0; t < P; ++t) {
      const int32_t old = atomicCAS(&skey[h], -1, x);
      if (old == -1 || old == x) {
        atomicAdd(&smeta[h], 1u);
        return;
      }
      h = (h + 1u == P) ? 0u : h + 1u;
    }
  };
#pragma unroll
  for (int u = 0; u < kListPX; ++u)
    if (valid(xs[u])) insert(xs[u]);
  for (int pos = kListPX * NT + tid; pos < nk; pos += NT)
    if (valid(xr[pos])) insert(xr[pos]);
  __syncthreads();

  // indices that some slot holds as the step begins
  auto mark = [&](int32_t c) {
    if (!valid(c)) return;
    const int h = early_find(skey, P, c);
    if (h >= 0) atomicOr(&smeta[h], kEarlyCached);
  };
#pragma unroll
  for (int u = 0; u < kListPC; ++u) mark(cs[u]);
  for (int j = kListPC * NT + tid; j < S; j += NT) mark(cr[j]);
  __syncthreads();

  // compact the keys nobody holds (listed at most four times): each thread
  // takes a contiguous run of map words, one prefix over the workgroup
  const uint32_t run = (P + NT - 1) / NT;
  const uint32_t h0 = tid * run, h1 = h0 + run < P ? h0 + run : P;
  auto is_key = [&](uint32_t h) {
    const uint32_t m = smeta[h];
    return skey[h] != -1 && !(m & kEarlyCached) && (m & kEarlyCount) <= kEarlyMaxPos;
  };
  int mine = 0;
  for (uint32_t h = h0; h < h1; ++h) mine += is_key(h) ? 1 : 0;
  const int incl = wave_inclusive_scan(mine, lane);
  if (lane == 63) swc[wave] = incl;
  __syncthreads();
  int idx = incl - mine, total = 0;
  for (int w = 0; w < MW; ++w) {
    idx += (w < wave) ? swc[w] : 0;
    total += swc[w];
  }
  for (uint32_t h = h0; h < h1; ++h) {
    if (!is_key(h)) continue;
    const int cnt = static_cast<int>(smeta[h] & kEarlyCount);
    e.early_x[lb + idx] = skey[h];
    int* pp = reinterpret_cast<int*>(e.early_pos + lb + idx);
    for (int k = cnt; k < kEarlyMaxPos; ++k) pp[k] = -1;   // the listed positions fill the rest
    smeta[h] = kEarlyKey | (static_cast<uint32_t>(idx) << 8);
    ++idx;
  }
  __syncthreads();

  // the positions of each key (their order inside a key does not matter)
  auto place = [&](int32_t x, int pos) {
    if (!valid(x)) return;
    const int h = early_find(skey, P, x);
    if (h < 0) return;
    const uint32_t m = smeta[h];
    if (!(m & kEarlyKey)) return;
    const int k = static_cast<int>(atomicAdd(&smeta[h], 1u) & 0xFFu);
    if (k < kEarlyMaxPos) reinterpret_cast<int*>(e.early_pos + lb + ((m >> 8) & 0x3FFFFFu))[k] = pos;
  };
#pragma unroll
  for (int u = 0; u < kListPX; ++u) place(xs[u], u * NT + tid);
  for (int pos = kListPX * NT + tid; pos < nk; pos += NT) place(xr[pos], pos);
  if (tid == 0) {
    e.early_n[r] = total;
    if (total) atomicAdd(&e.stats[static_cast<size_t>(r) * kNumStats + kStatEarly],
                         static_cast<unsigned long long>(total));
  }
}

// ---- copies ------------------------------------------------------------------
// Rows i < tn: copy chunks * sizeof(V) bytes from src[i] (0 skips the row) to
// every nonzero d[k * T + i], k < ND, by NT lanes (this one is `self`) each
// with U loads in flight.
template <typename V, int U, int NT, int ND>
__device__ __forceinline__ void copy_rows_to(const uint64_t* src, const uint64_t* d, int T, int tn,
                                             int chunks, int self) {
  const int total = tn * chunks;
  for (int q0 = self; q0 < total; q0 += NT * U) {
    V v[U];
    int row[U];
    uint64_t off[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int q = q0 + u * NT;
      row[u] = -1;
      if (q < total) {
        const int i = q / chunks;
        off[u] = static_cast<uint64_t>(q - i * chunks) * sizeof(V);
        const uint64_t s = src[i];
        if (s) {
          v[u] = *reinterpret_cast<const V*>(s + off[u]);
          row[u] = i;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (row[u] < 0) continue;
#pragma unroll
      for (int k = 0; k < ND; ++k) {
        const uint64_t a = d[k * T + row[u]];
        if (a) *reinterpret_cast<V*>(a + off[u]) = v[u];
      }
    }
  }
}

template <int U, int NT, int ND>
__device__ __forceinline__ void copy_tile(const EarlyParams& e, const uint64_t* src0, const uint64_t* d0,
                                          const uint64_t* src1, const uint64_t* d1, int T, int tn, int self) {
  if ((e.row_bytes0 & 15) == 0)
    copy_rows_to<u32x4, U, NT, ND>(src0, d0, T, tn, static_cast<int>(e.row_bytes0 / 16), self);
  else
    copy_rows_to<uint32_t, U, NT, ND>(src0, d0, T, tn, static_cast<int>(e.row_bytes0 / 4), self);
  if (e.n_streams > 1) {
    if ((e.row_bytes1 & 15) == 0)
      copy_rows_to<u32x4, U, NT, ND>(src1, d1, T, tn, static_cast<int>(e.row_bytes1 / 16), self);
    else
      copy_rows_to<uint32_t, U, NT, ND>(src1, d1, T, tn, static_cast<int>(e.row_bytes1 / 4), self);
  }
}

// Destinations of early key k of request r: the distinct slots of its
// positions (every position of an early key ends with its row), written to
// dst[0..3] of stream 0 and dstb[0..3] of stream 1 (0 = unused).  Slot loads
// bypass the L1: O was written by another workgroup of this launch.
__device__ __forceinline__ void early_dests(const EarlyParams& e, int r, int k, bool agent, uint64_t* d0,
                                            uint64_t* d1, int T) {
  const size_t lb = static_cast<size_t>(r) * e.n_q * e.K;
  const int4 pv = e.early_pos[lb + k];
  const int pos[kEarlyMaxPos] = {pv.x, pv.y, pv.z, pv.w};
  int o[kEarlyMaxPos];
#pragma unroll
  for (int j = 0; j < kEarlyMaxPos; ++j) {
    o[j] = -1;
    if (pos[j] >= 0) o[j] = agent ? load_agent(e.slots + lb + pos[j]) : e.slots[lb + pos[j]];
    if (o[j] < 0 || o[j] >= e.S) o[j] = -1;
  }
#pragma unroll
  for (int j = 0; j < kEarlyMaxPos; ++j) {
    bool seen = false;
#pragma unroll
    for (int i = 0; i < j; ++i) seen |= o[i] == o[j];
    const bool use = o[j] >= 0 && !seen;
    d0[j * T] = use ? e.buf_ptrs[r] + static_cast<uint64_t>(o[j]) * e.row_bytes0 : 0;
    if (e.n_streams > 1)
      d1[j * T] = use ? e.buf_ptrs[e.B + r] + static_cast<uint64_t>(o[j]) * e.row_bytes1 : 0;
  }
}

// Exclusive prefix of count[0..B) into pre[0..B] (pre[B] = total); NT threads.
template <int NT>
__device__ void prefix_counts(const int32_t* count, int B, long long* pre, long long* wtot) {
  const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
  const int per = (B + NT - 1) / NT;
  const int r0 = tid * per;
  long long local = 0;
  for (int k = 0; k < per; ++k)
    if (r0 + k < B) local += count[r0 + k];
  long long incl = local;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const long long t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  if (lane == 63) wtot[wave] = incl;
  __syncthreads();
  long long base = incl - local;
  for (int w = 0; w < wave; ++w) base += wtot[w];
  for (int k = 0; k < per; ++k)
    if (r0 + k < B) {
      pre[r0 + k] = base;
      base += count[r0 + k];
    }
  if (tid == NT - 1) pre[B] = base;
  __syncthreads();
}

// Early rows in claimed tiles across the batch.  A row whose request has its
// slots goes straight to them; any other row goes to HBM staging (or, when
// staging is full, is left to the finishing kernel) with a finish entry.
template <int NT>
__device__ void early_copy(const EarlyParams& e, unsigned char* lds) {
  constexpr int T = kEarlyTile;
  long long* pre = reinterpret_cast<long long*>(lds);                 // [B + 1]
  long long* wtot = pre + kEarlyMaxBatch + 1;                         // [NT / 64]
  uint64_t* src0 = reinterpret_cast<uint64_t*>(wtot + NT / 64);       // [T]
  uint64_t* d0 = src0 + T;                                            // [4][T]
  uint64_t* src1 = d0 + kEarlyMaxPos * T;                             // [T]
  uint64_t* d1 = src1 + T;                                            // [4][T]
  int* sh = reinterpret_cast<int*>(d1 + kEarlyMaxPos * T);            // [4]
  prefix_counts<NT>(e.early_n, e.B, pre, wtot);
  const long long N = pre[e.B];
  const int tid = threadIdx.x;
  for (;;) {
    if (tid == 0) {
      sh[0] = atomicAdd(&e.ctl[0], T);
      sh[1] = 0;
    }
    __syncthreads();
    const long long t0 = sh[0];
    if (t0 >= N) break;
    const int tn = static_cast<int>(N - t0 < T ? N - t0 : T);
    int r = 0, k = 0, park = -1;
    bool direct = false;
    if (tid < tn) {
      const long long j = t0 + tid;
      r = find_request(pre, e.B, j);
      k = static_cast<int>(j - pre[r]);
      direct = e.direct && __hip_atomic_load(e.done + r, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) != 0u;
      if (!direct) park = atomicAdd(&sh[1], 1);
    }
    __syncthreads();
    if (tid == 0 && sh[1] > 0) {
      sh[2] = atomicAdd(&e.ctl[1], sh[1]);
      sh[3] = atomicAdd(&e.ctl[2], sh[1]);
    }
    __syncthreads();
    if (tid < tn) {
      const size_t lb = static_cast<size_t>(r) * e.n_q * e.K;
      const int32_t x = e.early_x[lb + k];
      src0[tid] = e.host_ptrs[r] + static_cast<uint64_t>(x) * e.row_bytes0;
      if (e.n_streams > 1) src1[tid] = e.host_ptrs[e.B + r] + static_cast<uint64_t>(x) * e.row_bytes1;
      if (direct) {
        early_dests(e, r, k, true, d0 + tid, d1 + tid, T);
      } else {
        const int srow = sh[2] + park;
        const bool staged = srow < e.stage_rows;
        e.fin[sh[3] + park] = make_int4(r, k, staged ? srow : -1, 0);
        unsigned long long* st = e.stats + static_cast<size_t>(r) * kNumStats;
        atomicAdd(&st[staged ? kStatEarlyStaged : kStatEarlyDeferred], 1ull);
        if (!staged) src0[tid] = src1[tid] = 0;
        for (int q = 0; q < kEarlyMaxPos; ++q) d0[q * T + tid] = d1[q * T + tid] = 0;
        if (staged) {
          d0[tid] = e.stage0 + static_cast<uint64_t>(srow) * e.row_bytes0;
          if (e.n_streams > 1) d1[tid] = e.stage1 + static_cast<uint64_t>(srow) * e.row_bytes1;
        }
      }
    }
    __syncthreads();
    copy_tile<kEarlyUnroll, NT, kEarlyMaxPos>(e, src0, d0, src1, d1, T, tn, tid);
    __syncthreads();
  }
}

// The matching workgroup's own rows of request r after its plan: host entries
// (each also to its fan slots) and resident copies, then the repeats, which
// read slots the host copies just wrote.
template <int NT>
__device__ void copy_request_lists(const EarlyParams& e, int r, const int* counts, unsigned char* lds) {
  constexpr int T = kListTile;
  uint64_t* src0 = reinterpret_cast<uint64_t*>(lds);
  uint64_t* dst0 = src0 + T;
  uint64_t* dx0 = dst0 + T;
  uint64_t* dy0 = dx0 + T;
  uint64_t* src1 = dy0 + T;
  uint64_t* dst1 = src1 + T;
  uint64_t* dx1 = dst1 + T;
  uint64_t* dy1 = dx1 + T;
  const size_t lb = static_cast<size_t>(r) * e.n_q * e.K;
  const int64_t rows_r = e.rows[r];
  const uint64_t b0 = e.buf_ptrs[r], b1 = e.n_streams > 1 ? e.buf_ptrs[e.B + r] : 0;
  const uint64_t h0 = e.host_ptrs[r], h1 = e.n_streams > 1 ? e.host_ptrs[e.B + r] : 0;
  const int tid = threadIdx.x;
  // list 0: host entries, 1: resident, 2: repeats
  for (int list = 0; list < 3; ++list) {
    if (list == 2) {
      // the repeats' sources are slots this workgroup's host copies wrote
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      __syncthreads();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    const int n = list == 0 ? counts[0] : list == 1 ? counts[1] : counts[2];
    const int2* l = (list == 0 ? e.host_list : list == 1 ? e.res_list : e.rep_list) + lb;
    for (int t0 = 0; t0 < n; t0 += T) {
      const int tn = n - t0 < T ? n - t0 : T;
      if (tid < tn) {
        const int2 v = l[t0 + tid];
        const bool dst_ok = v.y >= 0 && v.y < e.S;
        bool ok;
        uint64_t s0, s1;
        if (list == 0) {
          ok = dst_ok && v.x >= 0 && static_cast<int64_t>(v.x) < rows_r;
          s0 = h0 + static_cast<uint64_t>(v.x) * e.row_bytes0;
          s1 = h1 + static_cast<uint64_t>(v.x) * e.row_bytes1;
        } else {
          ok = dst_ok && v.x >= 0 && v.x < e.S;
          s0 = b0 + static_cast<uint64_t>(v.x) * e.row_bytes0;
          s1 = b1 + static_cast<uint64_t>(v.x) * e.row_bytes1;
        }
        int2 fan = list == 0 ? e.host_fan[lb + t0 + tid] : make_int2(-1, -1);
        if (fan.x < 0 || fan.x >= e.S) fan.x = -1;
        if (fan.y < 0 || fan.y >= e.S) fan.y = -1;
        src0[tid] = ok ? s0 : 0;
        dst0[tid] = b0 + static_cast<uint64_t>(v.y) * e.row_bytes0;
        dx0[tid] = fan.x >= 0 ? b0 + static_cast<uint64_t>(fan.x) * e.row_bytes0 : 0;
        dy0[tid] = fan.y >= 0 ? b0 + static_cast<uint64_t>(fan.y) * e.row_bytes0 : 0;
        if (e.n_streams > 1) {
          src1[tid] = ok ? s1 : 0;
          dst1[tid] = b1 + static_cast<uint64_t>(v.y) * e.row_bytes1;
          dx1[tid] = fan.x >= 0 ? b1 + static_cast<uint64_t>(fan.x) * e.row_bytes1 : 0;
          dy1[tid] = fan.y >= 0 ? b1 + static_cast<uint64_t>(fan.y) * e.row_bytes1 : 0;
        }
      }
      __syncthreads();
      if ((e.row_bytes0 & 15) == 0)
        copy_rows<u32x4, 1, NT>(src0, dst0, tn, static_cast<int>(e.row_bytes0 / 16), dx0, dy0);
      else
        copy_rows<uint32_t, 1, NT>(src0, dst0, tn, static_cast<int>(e.row_bytes0 / 4), dx0, dy0);
      if (e.n_streams > 1) {
        if ((e.row_bytes1 & 15) == 0)
          copy_rows<u32x4, 1, NT>(src1, dst1, tn, static_cast<int>(e.row_bytes1 / 16), dx1, dy1);
        else
          copy_rows<uint32_t, 1, NT>(src1, dst1, tn, static_cast<int>(e.row_bytes1 / 4), dx1, dy1);
      }
      __syncthreads();
    }
  }
}

// ---- 2. Stage One beside the early copies ----------------------------------
template <int IPT, int NT>
__global__ __launch_bounds__(NT) void step_early_kernel(MatchParams mp, EarlyParams e) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (static_cast<int>(blockIdx.x) < mp.B) {
    const int r = static_cast<int>(blockIdx.x);
    NoPublish none;
    int counts[3] = {0, 0, 0};
    match_request<IPT, NT, 0>(mp, r, lds, none, counts);
    __syncthreads();
    copy_request_lists<NT>(e, r, counts, lds);
  } else {
    early_copy<NT>(e, lds);
  }
}

// ---- 3. rows fetched before their slots were known --------------------------
__global__ __launch_bounds__(GT) void finish_early_kernel(EarlyParams e) {
  constexpr int T = TILE;
  __shared__ uint64_t src0[T], d0[kEarlyMaxPos * T], src1[T], d1[kEarlyMaxPos * T];
  const long long N = e.ctl[2];
  const long long C = gridDim.x, w = blockIdx.x;
  const long long a = (w * N) / C, b = ((w + 1) * N) / C;   // Eq. 6 split of the entries
  for (long long t0 = a; t0 < b; t0 += T) {
    const int tn = static_cast<int>(b - t0 < T ? b - t0 : T);
    const int i = threadIdx.x;
    if (i < tn) {
      const int4 f = e.fin[t0 + i];
      const int r = f.x, k = f.y, srow = f.z;
      const size_t lb = static_cast<size_t>(r) * e.n_q * e.K;
      if (srow >= 0) {
        src0[i] = e.stage0 + static_cast<uint64_t>(srow) * e.row_bytes0;
        src1[i] = e.stage1 + static_cast<uint64_t>(srow) * e.row_bytes1;
      } else {
        const int32_t x = e.early_x[lb + k];
        src0[i] = e.host_ptrs[r] + static_cast<uint64_t>(x) * e.row_bytes0;
        src1[i] = e.n_streams > 1 ? e.host_ptrs[e.B + r] + static_cast<uint64_t>(x) * e.row_bytes1 : 0;
      }
      early_dests(e, r, k, false, d0 + i, d1 + i, T);
    }
    __syncthreads();
    copy_tile<kUnroll, GT, kEarlyMaxPos>(e, src0, d0, src1, d1, T, tn, threadIdx.x);
    __syncthreads();
  }
}

constexpr int kSmallThreads = 256;

template <int NT>
size_t early_copy_lds() {
  return 8 * (kEarlyMaxBatch + 1 + NT / 64) + 8 * 2 * (1 + kEarlyMaxPos) * kEarlyTile + 16;
}

}  // namespace

uint32_t early_map_words(int K, int n_q) {
  const long long nk = static_cast<long long>(K) * n_q;
  const long long limit = (160 * 1024 - 64 * 4) / 8;   // two words per map entry, wave counts
  long long P = 2 * nk;
  if (P > limit) P = limit;
  if (P * 4 < 5 * nk) return 0;                          // keep the map at most 80% full
  return static_cast<uint32_t>(P);
}

size_t early_list_lds_bytes(int K, int n_q) {
  const uint32_t P = early_map_words(K, n_q);
  return P ? 8 * static_cast<size_t>(P) + 4 * (kMatchThreads / 64) : 0;
}

size_t early_step_lds_bytes(int S, int K, int n_q) {
  const size_t m = stage_one_lds_bytes(S, K, n_q, true);
  if (m == 0) return 0;
  const size_t copier = match_threads(S, K) == kSmallThreads ? early_copy_lds<kSmallThreads>()
                                                             : early_copy_lds<kMatchThreads>();
  const size_t lists = 8 * 8 * kListTile;
  size_t v = m > copier ? m : copier;
  return v > lists ? v : lists;
}

hipError_t prepare_step_early(size_t list_lds, size_t step_lds) {
  const void* list_kernels[] = {reinterpret_cast<const void*>(&early_list_kernel<kMatchThreads>)};
  for (const void* k : list_kernels) {
    const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(list_lds));
    if (e != hipSuccess) return e;
  }
  const void* step_kernels[] = {
      reinterpret_cast<const void*>(&step_early_kernel<1, kMatchThreads>),
      reinterpret_cast<const void*>(&step_early_kernel<2, kMatchThreads>),
      reinterpret_cast<const void*>(&step_early_kernel<3, kMatchThreads>),
      reinterpret_cast<const void*>(&step_early_kernel<4, kMatchThreads>),
      reinterpret_cast<const void*>(&step_early_kernel<1, kSmallThreads>),
      reinterpret_cast<const void*>(&step_early_kernel<2, kSmallThreads>)};
  for (const void* k : step_kernels) {
    const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(step_lds));
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_early_list(const EarlyParams& e, size_t lds, hipStream_t s) {
  if (e.B > kEarlyMaxBatch || e.map_words == 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(early_list_kernel<kMatchThreads>, dim3(e.B), dim3(kMatchThreads), lds, s, e);
  return hipGetLastError();
}

hipError_t launch_step_early(const MatchParams& mp, const EarlyParams& e, int workers, size_t lds,
                             hipStream_t s) {
  if (e.B > kEarlyMaxBatch || workers < 1) return hipErrorInvalidValue;
  const dim3 grid(mp.B + workers);
  const int nt = match_threads(mp.S, mp.K);
  const int ipt = (mp.K + nt - 1) / nt;
  if (nt == kSmallThreads) {
    switch (ipt) {
      case 1: hipLaunchKernelGGL((step_early_kernel<1, kSmallThreads>), grid, dim3(nt), lds, s, mp, e); break;
      case 2: hipLaunchKernelGGL((step_early_kernel<2, kSmallThreads>), grid, dim3(nt), lds, s, mp, e); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  switch (ipt) {
    case 1: hipLaunchKernelGGL((step_early_kernel<1, kMatchThreads>), grid, dim3(nt), lds, s, mp, e); break;
    case 2: hipLaunchKernelGGL((step_early_kernel<2, kMatchThreads>), grid, dim3(nt), lds, s, mp, e); break;
    case 3: hipLaunchKernelGGL((step_early_kernel<3, kMatchThreads>), grid, dim3(nt), lds, s, mp, e); break;
    case 4: hipLaunchKernelGGL((step_early_kernel<4, kMatchThreads>), grid, dim3(nt), lds, s, mp, e); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_finish_early(const EarlyParams& e, int workers, hipStream_t s) {
  if (workers < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(finish_early_kernel, dim3(workers), dim3(GT), 0, s, e);
  return hipGetLastError();
}

}  // namespace avsg
