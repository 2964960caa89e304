// Device code of Stage Two shared by the gather kernels and the pipelined
// step kernel (see gather.hip for the work assignments).
#pragma once

#include "avsg_internal.h"

namespace avsg {
namespace {


constexpr int GT = kGatherThreads;
constexpr int TILE = kGatherTile;
constexpr int kMaxBatch = 1024;
constexpr int kUnroll = 4;

__device__ __forceinline__ int lane_index() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

// Exclusive prefix of the per-request miss totals into pre[0..B] (pre[B] = N).
__device__ inline void request_prefix(const GatherParams& p, long long* pre, long long* wtot) {
  const int tid = threadIdx.x, lane = lane_index(), wave = tid >> 6;
  const int per = (p.B + GT - 1) / GT;
  const int r0 = tid * per;
  long long local = 0;
  for (int k = 0; k < per; ++k) {
    const int r = r0 + k;
    if (r < p.B) {
      long long t = 0;
      for (int g = 0; g < p.counts_per_req; ++g)
        t += p.miss_counts[static_cast<size_t>(r) * p.count_stride + g];
      pre[r + 1] = t;
      local += t;
    }
  }
  long long incl = local;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    long long t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  if (lane == 63) wtot[wave] = incl;
  __syncthreads();
  long long base = incl - local;
  for (int w = 0; w < wave; ++w) base += wtot[w];
  for (int k = 0; k < per; ++k) {
    const int r = r0 + k;
    if (r < p.B) {
      const long long t = pre[r + 1];
      base += t;
      pre[r + 1] = base;
    }
  }
  if (tid == 0) pre[0] = 0;
  __syncthreads();
}

// First tiles of the resident-reuse gather: workgroup w < ch copies tile
// w div B of request w mod B's host list before any prefix is known.  Request
// r has nfirst(r) such workgroups; its n host entries go to them in tiles of
// ceil(n / nfirst) rows, at least one and at most T0, so few entries still
// spread over many CUs (one workgroup reads ~2.5 GB/s from the host).  No
// request gets first tiles when one would get more than eight (ch > 8 B):
// with 192 such workgroups, twelve per request (16 requests) made the step
// slower than none, six (32 requests) and three (64) faster.
__device__ __forceinline__ bool first_tiles_on(int B, int ch) { return ch <= 8 * B; }
__device__ __forceinline__ long long first_tiles(int r, int B, int ch) {
  return first_tiles_on(B, ch) && r < ch ? (ch - 1 - r) / B + 1 : 0;
}
__device__ __forceinline__ long long first_tile_rows(long long n, long long nfirst, int T0) {
  const long long t = nfirst > 0 ? (n + nfirst - 1) / nfirst : 1;
  return t < 1 ? 1 : (t > T0 ? T0 : t);
}

// Prefixes for the resident-reuse gather: of the host entries that remain
// after each request's first tiles (pre_a; cov[r] = the entries of request r
// the first tiles copy) and of the resident entries (pre_b), B + 1 entries
// each.  With at most GT requests thread r's two counts are ha and hb, which
// the caller requested before its first tile so the loads overlap it.
// wtot: 2 * GT / 64 entries.
__device__ inline void request_prefix_resid(const GatherParams& pa, long long* pre_a, long long* cov,
                                            const GatherParams& pb, long long* pre_b, long long* wtot,
                                            int ch, int T0, long long ha, long long hb) {
  const int tid = threadIdx.x, lane = lane_index(), wave = tid >> 6;
  constexpr int NW = GT / 64;
  const int per = (pa.B + GT - 1) / GT;
  const int r0 = tid * per;
  long long la = 0, lb = 0;
  for (int k = 0; k < per; ++k) {
    const int r = r0 + k;
    if (r < pa.B) {
      long long ta = per == 1 ? ha : pa.miss_counts[static_cast<size_t>(r) * pa.count_stride];
      const long long tb = per == 1 ? hb : pb.miss_counts[static_cast<size_t>(r) * pb.count_stride];
      const long long nfirst = first_tiles(r, pa.B, ch);
      const long long span = nfirst * first_tile_rows(ta, nfirst, T0);
      const long long c = ta < span ? ta : span;
      cov[r] = c;
      ta -= c;
      pre_a[r + 1] = ta;
      pre_b[r + 1] = tb;
      la += ta;
      lb += tb;
    }
  }
  long long ia = la, ib = lb;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const long long ta = __shfl_up(ia, off, 64), tb = __shfl_up(ib, off, 64);
    if (lane >= off) {
      ia += ta;
      ib += tb;
    }
  }
  if (lane == 63) {
    wtot[wave] = ia;
    wtot[NW + wave] = ib;
  }
  __syncthreads();
  long long ba = ia - la, bb = ib - lb;
  for (int w = 0; w < wave; ++w) {
    ba += wtot[w];
    bb += wtot[NW + w];
  }
  for (int k = 0; k < per; ++k) {
    const int r = r0 + k;
    if (r < pa.B) {
      ba += pre_a[r + 1];
      bb += pre_b[r + 1];
      pre_a[r + 1] = ba;
      pre_b[r + 1] = bb;
    }
  }
  if (tid == 0) {
    pre_a[0] = 0;
    pre_b[0] = 0;
  }
  __syncthreads();
}

__device__ __forceinline__ int find_request(const long long* pre, int B, long long j) {
  int lo = 0, hi = B;  // pre[lo] <= j < pre[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (pre[mid] <= j) lo = mid;
    else hi = mid;
  }
  return lo;
}

// A 16-byte vector as a clang vector type: arrays of it stay in registers
// (HIP's uint4 is a union-based struct that is kept in scratch memory here).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Rows i < tn: copy chunks * sizeof(V) bytes from src[i] to dst[i] (src[i] == 0
// skips the row), and also to dstx[i] and dsty[i] where those are given and
// nonzero, with NT threads each keeping U loads in flight.
template <typename V, int U = kUnroll, int NT = GT>
__device__ __forceinline__ void copy_rows(const uint64_t* src, const uint64_t* dst, int tn,
                                          int chunks, const uint64_t* dstx = nullptr,
                                          const uint64_t* dsty = nullptr) {
  const int total = tn * chunks;
  for (int q0 = threadIdx.x; q0 < total; q0 += NT * U) {
    V v[U];
    uint64_t da[U], xa[U], ya[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int q = q0 + u * NT;
      da[u] = 0;
      xa[u] = 0;
      ya[u] = 0;
      if (q < total) {
        const int i = q / chunks;
        const int ch = q - i * chunks;
        const uint64_t s = src[i];
        if (s) {
          const uint64_t off = static_cast<uint64_t>(ch) * sizeof(V);
          v[u] = *reinterpret_cast<const V*>(s + off);
          da[u] = dst[i] + off;
          if (dstx && dstx[i]) xa[u] = dstx[i] + off;
          if (dsty && dsty[i]) ya[u] = dsty[i] + off;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (da[u]) *reinterpret_cast<V*>(da[u]) = v[u];
      if (xa[u]) *reinterpret_cast<V*>(xa[u]) = v[u];
      if (ya[u]) *reinterpret_cast<V*>(ya[u]) = v[u];
    }
  }
}

__device__ inline void copy_tile_rows(const GatherParams& p, int tn, uint64_t* src0, uint64_t* dst0,
                               uint64_t* src1, uint64_t* dst1) {
  __syncthreads();
  if ((p.row_bytes0 & 15) == 0)
    copy_rows<u32x4>(src0, dst0, tn, static_cast<int>(p.row_bytes0 / 16));
  else
    copy_rows<uint32_t>(src0, dst0, tn, static_cast<int>(p.row_bytes0 / 4));
  if (p.n_streams > 1) {
    if ((p.row_bytes1 & 15) == 0)
      copy_rows<u32x4>(src1, dst1, tn, static_cast<int>(p.row_bytes1 / 16));
    else
      copy_rows<uint32_t>(src1, dst1, tn, static_cast<int>(p.row_bytes1 / 4));
  }
  __syncthreads();
}

// Copy entries [a, b) of the batch-wide list.  kDevice: an entry is (source
// slot, slot) of the request's own buffers; otherwise (host row, slot), and
// with p.fan and staging for it (dstx0/1, dsty0/1), the row also goes to the
// entry's fan slots.  Entry j of the batch-wide list is entry cov[r] + j -
// pre[r] of request r's list (cov: rows of each request left out of the
// batch-wide list, or none); with fixed_r >= 0, [a, b) are entries of request
// fixed_r's own list and pre is not read.
template <bool kDevice>
__device__ __forceinline__ void copy_range(const GatherParams& p, const long long* pre, long long a, long long b,
                           uint64_t* src0, uint64_t* dst0, uint64_t* src1, uint64_t* dst1,
                           uint64_t* dstx0 = nullptr, uint64_t* dstx1 = nullptr,
                           uint64_t* dsty0 = nullptr, uint64_t* dsty1 = nullptr,
                           const long long* cov = nullptr, int fixed_r = -1) {
  const size_t per_req = static_cast<size_t>(p.n_q) * p.K;
  for (long long t0 = a; t0 < b; t0 += TILE) {
    const int tn = static_cast<int>((b - t0) < TILE ? (b - t0) : TILE);
    for (int i = threadIdx.x; i < tn; i += GT) {
      const long long j = t0 + i;
      const int r = fixed_r >= 0 ? fixed_r : find_request(pre, p.B, j);
      const long long k = fixed_r >= 0 ? j : (cov ? cov[r] : 0) + j - pre[r];   // entry of request r
      const size_t at = static_cast<size_t>(r) * per_req + static_cast<size_t>(k);
      const int2 e = p.miss_list[at];
      const bool ok = e.x >= 0 && e.y >= 0 && e.y < p.S &&
                      (kDevice ? e.x < p.S : static_cast<int64_t>(e.x) < p.rows[r]);
      const uint64_t base0 = kDevice ? p.buf_ptrs[r] : p.host_ptrs[r];
      src0[i] = ok ? base0 + static_cast<uint64_t>(e.x) * p.row_bytes0 : 0;
      dst0[i] = p.buf_ptrs[r] + static_cast<uint64_t>(e.y) * p.row_bytes0;
      int2 fan = make_int2(-1, -1);
      if (dstx0) {
        fan = p.fan[at];
        if (fan.x < 0 || fan.x >= p.S) fan.x = -1;
        if (fan.y < 0 || fan.y >= p.S) fan.y = -1;
        dstx0[i] = fan.x >= 0 ? p.buf_ptrs[r] + static_cast<uint64_t>(fan.x) * p.row_bytes0 : 0;
        dsty0[i] = fan.y >= 0 ? p.buf_ptrs[r] + static_cast<uint64_t>(fan.y) * p.row_bytes0 : 0;
      }
      if (p.n_streams > 1) {
        const uint64_t base1 = kDevice ? p.buf_ptrs[p.B + r] : p.host_ptrs[p.B + r];
        src1[i] = ok ? base1 + static_cast<uint64_t>(e.x) * p.row_bytes1 : 0;
        dst1[i] = p.buf_ptrs[p.B + r] + static_cast<uint64_t>(e.y) * p.row_bytes1;
        if (dstx1) {
          dstx1[i] = fan.x >= 0 ? p.buf_ptrs[p.B + r] + static_cast<uint64_t>(fan.x) * p.row_bytes1 : 0;
          dsty1[i] = fan.y >= 0 ? p.buf_ptrs[p.B + r] + static_cast<uint64_t>(fan.y) * p.row_bytes1 : 0;
        }
      }
    }
    __syncthreads();
    if ((p.row_bytes0 & 15) == 0)
      copy_rows<u32x4>(src0, dst0, tn, static_cast<int>(p.row_bytes0 / 16), dstx0, dsty0);
    else
      copy_rows<uint32_t>(src0, dst0, tn, static_cast<int>(p.row_bytes0 / 4), dstx0, dsty0);
    if (p.n_streams > 1) {
      if ((p.row_bytes1 & 15) == 0)
        copy_rows<u32x4>(src1, dst1, tn, static_cast<int>(p.row_bytes1 / 16), dstx1, dsty1);
      else
        copy_rows<uint32_t>(src1, dst1, tn, static_cast<int>(p.row_bytes1 / 4), dstx1, dsty1);
    }
    __syncthreads();
  }
}

}  // namespace
}  // namespace avsg
