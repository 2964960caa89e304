// Stage Two of AVSG on gfx950: miss-only copy of host rows into reserved slots.
//
// The miss list is ordered by (request, token, miss rank) (Section 3.4).  The
// balanced kernel (S3, Eq. 6) runs C workgroups; workgroup w takes the
// consecutive misses [floor(w N / C), floor((w+1) N / C)) of the batch-wide list
// of N misses, so any two workgroups differ by at most one row.  The request
// kernel (S1, Eq. 13) runs one workgroup per request.  Inside a workgroup a
// tile of misses is staged in LDS as (source, destination) address pairs, and
// the lanes copy the rows with 16-byte loads from pinned, device-mapped host
// memory (4-byte loads for rows that are not a multiple of 16 bytes, such as
// the 132-byte indexer-key rows), several loads in flight per lane.  The
// position kernel (S2, Eq. 14) splits the flattened N_g*K selected positions
// into C near-equal contiguous ranges; hit positions issue no copy but still
// occupy their worker's share.
#include "avsg_internal.h"

namespace avsg {
namespace {

constexpr int NT = kGatherThreads;
constexpr int TILE = kGatherTile;
constexpr int kMaxBatch = 1024;
constexpr int kUnroll = 4;

__device__ __forceinline__ int lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

// Exclusive prefix of the per-request miss totals into pre[0..B] (pre[B] = N).
__device__ void request_prefix(const GatherParams& p, long long* pre, long long* wtot) {
  const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
  const int per = (p.B + NT - 1) / NT;
  const int r0 = tid * per;
  long long local = 0;
  for (int k = 0; k < per; ++k) {
    const int r = r0 + k;
    if (r < p.B) {
      long long t = 0;
      for (int g = 0; g < p.n_q; ++g) t += p.miss_counts[static_cast<size_t>(r) * p.n_q + g];
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

__device__ __forceinline__ int find_request(const long long* pre, int B, long long j) {
  int lo = 0, hi = B;  // pre[lo] <= j < pre[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (pre[mid] <= j) lo = mid;
    else hi = mid;
  }
  return lo;
}

template <typename V>
__device__ __forceinline__ void copy_rows(const uint64_t* src, const uint64_t* dst, int tn,
                                          int chunks) {
  const int total = tn * chunks;
  for (int q0 = threadIdx.x; q0 < total; q0 += NT * kUnroll) {
    V v[kUnroll];
    uint64_t da[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int q = q0 + u * NT;
      da[u] = 0;
      if (q < total) {
        const int i = q / chunks;
        const int ch = q - i * chunks;
        const uint64_t s = src[i];
        if (s) {
          v[u] = *reinterpret_cast<const V*>(s + static_cast<uint64_t>(ch) * sizeof(V));
          da[u] = dst[i] + static_cast<uint64_t>(ch) * sizeof(V);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (da[u]) *reinterpret_cast<V*>(da[u]) = v[u];
  }
}

__device__ void copy_tile_rows(const GatherParams& p, int tn, uint64_t* src0, uint64_t* dst0,
                               uint64_t* src1, uint64_t* dst1) {
  __syncthreads();
  if ((p.row_bytes0 & 15) == 0)
    copy_rows<uint4>(src0, dst0, tn, static_cast<int>(p.row_bytes0 / 16));
  else
    copy_rows<uint32_t>(src0, dst0, tn, static_cast<int>(p.row_bytes0 / 4));
  if (p.n_streams > 1) {
    if ((p.row_bytes1 & 15) == 0)
      copy_rows<uint4>(src1, dst1, tn, static_cast<int>(p.row_bytes1 / 16));
    else
      copy_rows<uint32_t>(src1, dst1, tn, static_cast<int>(p.row_bytes1 / 4));
  }
  __syncthreads();
}

// Copy misses [a, b) of the batch-wide list.
__device__ void copy_range(const GatherParams& p, const long long* pre, long long a, long long b,
                           uint64_t* src0, uint64_t* dst0, uint64_t* src1, uint64_t* dst1) {
  const size_t per_req = static_cast<size_t>(p.n_q) * p.K;
  for (long long t0 = a; t0 < b; t0 += TILE) {
    const int tn = static_cast<int>((b - t0) < TILE ? (b - t0) : TILE);
    for (int i = threadIdx.x; i < tn; i += NT) {
      const long long j = t0 + i;
      const int r = find_request(pre, p.B, j);
      const int2 e = p.miss_list[static_cast<size_t>(r) * per_req + static_cast<size_t>(j - pre[r])];
      const bool ok = e.x >= 0 && static_cast<int64_t>(e.x) < p.rows[r] && e.y >= 0 && e.y < p.S;
      src0[i] = ok ? p.host_ptrs[r] + static_cast<uint64_t>(e.x) * p.row_bytes0 : 0;
      dst0[i] = p.buf_ptrs[r] + static_cast<uint64_t>(e.y) * p.row_bytes0;
      if (p.n_streams > 1) {
        src1[i] = ok ? p.host_ptrs[p.B + r] + static_cast<uint64_t>(e.x) * p.row_bytes1 : 0;
        dst1[i] = p.buf_ptrs[p.B + r] + static_cast<uint64_t>(e.y) * p.row_bytes1;
      }
    }
    __syncthreads();
    if ((p.row_bytes0 & 15) == 0)
      copy_rows<uint4>(src0, dst0, tn, static_cast<int>(p.row_bytes0 / 16));
    else
      copy_rows<uint32_t>(src0, dst0, tn, static_cast<int>(p.row_bytes0 / 4));
    if (p.n_streams > 1) {
      if ((p.row_bytes1 & 15) == 0)
        copy_rows<uint4>(src1, dst1, tn, static_cast<int>(p.row_bytes1 / 16));
      else
        copy_rows<uint32_t>(src1, dst1, tn, static_cast<int>(p.row_bytes1 / 4));
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(NT) void gather_balanced_kernel(GatherParams p) {
  __shared__ long long pre[kMaxBatch + 1];
  __shared__ long long wtot[NT / 64];
  __shared__ uint64_t src0[TILE], dst0[TILE], src1[TILE], dst1[TILE];
  request_prefix(p, pre, wtot);
  const long long N = pre[p.B];
  const long long C = gridDim.x, w = blockIdx.x;
  const long long a = (w * N) / C;          // Eq. 6: consecutive, floor/ceil(N/C) each
  const long long b = ((w + 1) * N) / C;
  copy_range(p, pre, a, b, src0, dst0, src1, dst1);
}

__global__ __launch_bounds__(NT) void gather_position_kernel(GatherParams p) {
  __shared__ uint64_t src0[TILE], dst0[TILE], src1[TILE], dst1[TILE];
  const long long per_req = static_cast<long long>(p.n_q) * p.K;
  const long long P = per_req * p.B;
  const long long C = gridDim.x, w = blockIdx.x;
  const long long a = (w * P) / C;          // Eq. 14: near-equal ranges of positions
  const long long b = ((w + 1) * P) / C;
  for (long long t0 = a; t0 < b; t0 += TILE) {
    const int tn = static_cast<int>((b - t0) < TILE ? (b - t0) : TILE);
    for (int i = threadIdx.x; i < tn; i += NT) {
      const long long pos = t0 + i;
      const int r = static_cast<int>(pos / per_req);
      const int32_t x = p.topk[pos];
      const int32_t o = p.slots[pos];
      const bool miss = p.hit_mask[pos] == 0;
      const bool ok = miss && x >= 0 && static_cast<int64_t>(x) < p.rows[r] && o >= 0 && o < p.S;
      src0[i] = ok ? p.host_ptrs[r] + static_cast<uint64_t>(x) * p.row_bytes0 : 0;
      dst0[i] = p.buf_ptrs[r] + static_cast<uint64_t>(o) * p.row_bytes0;
      if (p.n_streams > 1) {
        src1[i] = ok ? p.host_ptrs[p.B + r] + static_cast<uint64_t>(x) * p.row_bytes1 : 0;
        dst1[i] = p.buf_ptrs[p.B + r] + static_cast<uint64_t>(o) * p.row_bytes1;
      }
    }
    copy_tile_rows(p, tn, src0, dst0, src1, dst1);
  }
}

__global__ __launch_bounds__(NT) void gather_request_kernel(GatherParams p) {
  __shared__ long long pre[kMaxBatch + 1];
  __shared__ long long wtot[NT / 64];
  __shared__ uint64_t src0[TILE], dst0[TILE], src1[TILE], dst1[TILE];
  request_prefix(p, pre, wtot);
  const int r = blockIdx.x;                 // Eq. 13: one worker per request
  copy_range(p, pre, pre[r], pre[r + 1], src0, dst0, src1, dst1);
}

}  // namespace

hipError_t launch_gather_balanced(const GatherParams& p, int workers, hipStream_t s) {
  if (p.B > kMaxBatch || workers < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_balanced_kernel, dim3(workers), dim3(NT), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_gather_position(const GatherParams& p, int workers, hipStream_t s) {
  if (workers < 1 || !p.hit_mask || !p.topk || !p.slots) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_position_kernel, dim3(workers), dim3(NT), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_gather_request(const GatherParams& p, hipStream_t s) {
  if (p.B > kMaxBatch) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_request_kernel, dim3(p.B), dim3(NT), 0, s, p);
  return hipGetLastError();
}

}  // namespace avsg
