// Stage Two of AVSG on gfx950: miss-only copy of host rows into reserved slots.
//
// The miss list is ordered by (request, token, miss rank) (Section 3.4).  The
// balanced kernel (S3, Eq. 6) runs C workers; worker w takes the consecutive
// misses [floor(w N / C), floor((w+1) N / C)) of the batch-wide list of N
// misses, so any two workers differ by at most one row, and consecutive
// workers run on one XCD (xcd_worker).  The request
// kernel (S1, Eq. 13) runs one workgroup per request.  Inside a workgroup a
// tile of misses is staged in LDS as (source, destination) address pairs, and
// the lanes copy the rows with 16-byte loads from pinned, device-mapped host
// memory (4-byte loads for rows that are not a multiple of 16 bytes, such as
// the 132-byte indexer-key rows), several loads in flight per lane.  The
// position kernel (S2, Eq. 14) splits the flattened N_g*K selected positions
// into C near-equal contiguous ranges; hit positions issue no copy but still
// occupy their worker's share.  With the resident-reuse plan of the matching
// kernel, the resident kernel copies the host list (each row also to its two
// fan slots) and the rows already in the device buffer; with four or more
// tokens per step the device-copy kernel then fills the repeats left over.
#include "gather_body.h"

namespace avsg {
namespace {

// Worker index of workgroup b among C workers.  The dispatcher deals
// workgroups to the eight XCDs of the chip round-robin (workgroup b to XCD
// b mod 8), and each XCD has its own L2; consecutive workers get consecutive
// stretches of the miss list, which hold the same request's tokens, so they
// go to one XCD: a row that several tokens of a step miss (a lost install) is
// then read over the host link once and served from that XCD's L2 after.
// A bijection of [0, C) for any C; the split of Eq. 6 and Eq. 14 is unchanged.
__device__ __forceinline__ long long xcd_worker(long long b, long long C) {
  constexpr long long X = kXcds;
  const long long x = b % X, q = C / X, rem = C % X;
  return x * q + (x < rem ? x : rem) + b / X;
}

__global__ __launch_bounds__(GT) void gather_balanced_kernel(GatherParams p) {
  __shared__ long long pre[kMaxBatch + 1];
  __shared__ long long wtot[GT / 64];
  __shared__ uint64_t src0[TILE], dst0[TILE], src1[TILE], dst1[TILE];
  request_prefix(p, pre, wtot);
  const long long N = pre[p.B];
  const long long C = gridDim.x, w = xcd_worker(blockIdx.x, C);
  const long long a = (w * N) / C;          // Eq. 6: consecutive, floor/ceil(N/C) each
  const long long b = ((w + 1) * N) / C;
  copy_range<false>(p, pre, a, b, src0, dst0, src1, dst1);
}

// Resident-reuse Stage Two over two lists: host rows (each also written to
// its fan slots, the two largest repeats of its index in the step), and rows
// already in a slot of the same request (not written this step).  The last
// quarter of the workgroups starts with the resident list and the others
// with the host list, so the HBM copies run while the host link is busy (the
// link saturates with far fewer workgroups); each group then moves to the
// other list.  A host-first workgroup's first tile is a stretch of one
// request's own host list (first_tiles; none when a request would get more
// than eight of them), which needs no batch-wide prefix, so
// host reads start one list read after the launch; the rest of the host list
// goes in claimed tiles.  Tile i of the resident list first goes to the i-th
// resident-first workgroup, later tiles are claimed.  Claimed tiles (an atomic
// counter) let the workgroups that finish first take more (a CU's host-read
// rate varies up to 2x across the chip; they end the kernel more evenly than a
// static Eq. 6 split).  A resident list shorter than one full tile per
// workgroup of its group is cut into tiles of ceil(n / group) rows.
// claim[0] and claim[1] count the claimed resident and host rows; the
// matching kernel resets both.
constexpr int kHostTile = 6;

// Rows per tile of a list of n entries shared by `group` workgroups.
__device__ __forceinline__ int tile_rows(long long n, int group, int max_rows) {
  const long long t = (n + group - 1) / group;
  return t < 1 ? 1 : (t > max_rows ? max_rows : static_cast<int>(t));
}

// Copy tiles of T entries of a list of n entries: `first` (or none, -1) then
// claimed tiles, which start at row `base`.
template <bool kDevice>
__device__ void copy_tiles(const GatherParams& p, const long long* pre, long long n, int T, long long first,
                           long long base, int* counter, long long* next, uint64_t* src0,
                           uint64_t* dst0, uint64_t* src1, uint64_t* dst1, uint64_t* dstx0 = nullptr,
                           uint64_t* dstx1 = nullptr, uint64_t* dsty0 = nullptr, uint64_t* dsty1 = nullptr,
                           const long long* cov = nullptr) {
  long long t0 = first;
  for (;;) {
    if (t0 < 0) {
      if (threadIdx.x == 0) *next = base + atomicAdd(counter, T);
      __syncthreads();
      t0 = *next;
      __syncthreads();
    }
    if (t0 >= n) break;
    copy_range<kDevice>(p, pre, t0, t0 + T < n ? t0 + T : n, src0, dst0, src1, dst1, dstx0, dstx1, dsty0,
                        dsty1, cov);
    t0 = -1;
  }
}

__global__ __launch_bounds__(GT) void gather_resident_kernel(GatherParams hp, GatherParams rp,
                                                              int* claim) {
  __shared__ long long pre_h[kMaxBatch + 1], pre_r[kMaxBatch + 1], cov[kMaxBatch];
  __shared__ long long wtot[2 * (GT / 64)];
  __shared__ uint64_t src0[TILE], dst0[TILE], src1[TILE], dst1[TILE], dstx0[TILE], dstx1[TILE], dsty0[TILE],
      dsty1[TILE];
  __shared__ long long next;
  const int C = static_cast<int>(gridDim.x), w = static_cast<int>(blockIdx.x);
  const int cr = C / 4;                  // workgroups that start with the resident list (may be 0)
  const int ch = C - cr;                 // >= 1
  const int B = hp.B;
  // the counts of the prefixes below are requested before the first tile, so
  // their latency overlaps it
  long long ha = 0, hb = 0;
  if (B <= GT && static_cast<int>(threadIdx.x) < B) {
    ha = hp.miss_counts[static_cast<size_t>(threadIdx.x) * hp.count_stride];
    hb = rp.miss_counts[static_cast<size_t>(threadIdx.x) * rp.count_stride];
  }
  if (w < ch && first_tiles_on(B, ch)) {
    // first tile, before any prefix: entries [k T, (k+1) T) of request
    // w mod B's host list, k = w div B (the host link starts one list read
    // after the launch)
    const int r = w % B, k = w / B;
    const long long cnt = hp.miss_counts[static_cast<size_t>(r) * hp.count_stride];
    const long long T = first_tile_rows(cnt, first_tiles(r, B, ch), kHostTile);
    const long long lo = static_cast<long long>(k) * T;
    const long long hi = lo + T < cnt ? lo + T : cnt;
    if (lo < hi)
      copy_range<false>(hp, nullptr, lo, hi, src0, dst0, src1, dst1, dstx0, dstx1, dsty0, dsty1, nullptr, r);
  }
  // the rest of the host list, batch-wide, in claimed tiles (every group),
  // and the resident list (tile i of it first to the i-th resident-first
  // workgroup, the rest claimed)
  request_prefix_resid(hp, pre_h, cov, rp, pre_r, wtot, ch, kHostTile, ha, hb);
  const long long N = pre_h[B], R = pre_r[rp.B];
  const int tr = tile_rows(R, cr > 0 ? cr : ch, TILE);
  const long long res_base = static_cast<long long>(cr) * tr;
  if (w >= ch) {
    const long long i = C - 1 - w;       // 0 .. cr-1
    copy_tiles<true>(rp, pre_r, R, tr, i * tr, res_base, claim, &next, src0, dst0, src1, dst1);
    copy_tiles<false>(hp, pre_h, N, kHostTile, -1, 0, claim + 1, &next, src0, dst0, src1, dst1,
                      dstx0, dstx1, dsty0, dsty1, cov);
  } else {
    copy_tiles<false>(hp, pre_h, N, kHostTile, -1, 0, claim + 1, &next, src0, dst0, src1, dst1,
                      dstx0, dstx1, dsty0, dsty1, cov);
    copy_tiles<true>(rp, pre_r, R, tr, -1, res_base, claim, &next, src0, dst0, src1, dst1);
  }
}

// Device-to-device row copies (source slot -> slot) over the same balanced
// split; runs after the host copies of the step, so every source holds its row.
__global__ __launch_bounds__(GT) void copy_device_kernel(GatherParams p) {
  __shared__ long long pre[kMaxBatch + 1];
  __shared__ long long wtot[GT / 64];
  __shared__ uint64_t src0[TILE], dst0[TILE], src1[TILE], dst1[TILE];
  request_prefix(p, pre, wtot);
  const long long N = pre[p.B];
  const long long C = gridDim.x, w = blockIdx.x;
  const long long a = (w * N) / C;
  const long long b = ((w + 1) * N) / C;
  copy_range<true>(p, pre, a, b, src0, dst0, src1, dst1);
}

__global__ __launch_bounds__(GT) void gather_position_kernel(GatherParams p) {
  __shared__ uint64_t src0[TILE], dst0[TILE], src1[TILE], dst1[TILE];
  const long long per_req = static_cast<long long>(p.n_q) * p.K;
  const long long P = per_req * p.B;
  const long long C = gridDim.x, w = xcd_worker(blockIdx.x, C);
  const long long a = (w * P) / C;          // Eq. 14: near-equal ranges of positions
  const long long b = ((w + 1) * P) / C;
  for (long long t0 = a; t0 < b; t0 += TILE) {
    const int tn = static_cast<int>((b - t0) < TILE ? (b - t0) : TILE);
    for (int i = threadIdx.x; i < tn; i += GT) {
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

__global__ __launch_bounds__(GT) void gather_request_kernel(GatherParams p) {
  __shared__ long long pre[kMaxBatch + 1];
  __shared__ long long wtot[GT / 64];
  __shared__ uint64_t src0[TILE], dst0[TILE], src1[TILE], dst1[TILE];
  request_prefix(p, pre, wtot);
  const int r = blockIdx.x;                 // Eq. 13: one worker per request
  copy_range<false>(p, pre, pre[r], pre[r + 1], src0, dst0, src1, dst1);
}

}  // namespace

hipError_t launch_gather_balanced(const GatherParams& p, int workers, hipStream_t s) {
  if (p.B > kMaxBatch || workers < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_balanced_kernel, dim3(workers), dim3(GT), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_copy_device(const GatherParams& p, int workers, hipStream_t s) {
  if (workers < 1 || p.B > kMaxBatch) return hipErrorInvalidValue;
  hipLaunchKernelGGL(copy_device_kernel, dim3(workers), dim3(GT), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_gather_resident(const GatherParams& host, const GatherParams& dev, int* claim,
                                  int workers, hipStream_t s) {
  if (workers < 1 || host.B > kMaxBatch || !claim || !host.fan) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_resident_kernel, dim3(workers), dim3(GT), 0, s, host, dev, claim);
  return hipGetLastError();
}

hipError_t launch_gather_position(const GatherParams& p, int workers, hipStream_t s) {
  if (workers < 1 || !p.hit_mask || !p.topk || !p.slots) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_position_kernel, dim3(workers), dim3(GT), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_gather_request(const GatherParams& p, hipStream_t s) {
  if (p.B > kMaxBatch) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_request_kernel, dim3(p.B), dim3(GT), 0, s, p);
  return hipGetLastError();
}

}  // namespace avsg
