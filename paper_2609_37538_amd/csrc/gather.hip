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
// occupy their worker's share.  With the resident-reuse plan of the matching
// kernel, the resident kernel copies the host list and the rows already in the
// device buffer, and the device-copy kernel then fills repeats of this step's
// host rows.
#include "gather_body.h"

namespace avsg {
namespace {

__global__ __launch_bounds__(GT) void gather_balanced_kernel(GatherParams p) {
  __shared__ long long pre[kMaxBatch + 1];
  __shared__ long long wtot[GT / 64];
  __shared__ uint64_t src0[TILE], dst0[TILE], src1[TILE], dst1[TILE];
  request_prefix(p, pre, wtot);
  const long long N = pre[p.B];
  const long long C = gridDim.x, w = blockIdx.x;
  const long long a = (w * N) / C;          // Eq. 6: consecutive, floor/ceil(N/C) each
  const long long b = ((w + 1) * N) / C;
  copy_range<false>(p, pre, a, b, src0, dst0, src1, dst1);
}

// Resident-reuse Stage Two: workgroups claim 32-row tiles of the host list
// with an atomic counter (the host-read rate of a CU varies up to 2x across
// the chip, so claimed tiles end the kernel more evenly than a static Eq. 6
// split: 0.6% faster at 64 requests), then 64-row tiles of the resident list
// (rows already in a slot of the same request, not written this step) until
// none is left.  claim[0] counts resident rows, claim[1] host rows; the
// matching kernel resets both.
constexpr int kHostClaim = 32;

__global__ __launch_bounds__(GT) void gather_resident_kernel(GatherParams hp, GatherParams rp,
                                                              int* claim) {
  __shared__ long long pre[kMaxBatch + 1];
  __shared__ long long wtot[GT / 64];
  __shared__ uint64_t src0[TILE], dst0[TILE], src1[TILE], dst1[TILE];
  __shared__ long long next;
  request_prefix(hp, pre, wtot);
  const long long N = pre[hp.B];
  for (;;) {
    if (threadIdx.x == 0) next = atomicAdd(claim + 1, kHostClaim);
    __syncthreads();
    const long long t0 = next;
    if (t0 >= N) break;
    copy_range<false>(hp, pre, t0, t0 + kHostClaim < N ? t0 + kHostClaim : N, src0, dst0, src1, dst1);
  }
  __syncthreads();
  request_prefix(rp, pre, wtot);
  const long long R = pre[rp.B];
  for (;;) {
    if (threadIdx.x == 0) next = atomicAdd(claim, TILE);
    __syncthreads();
    const long long t0 = next;
    if (t0 >= R) break;
    copy_range<true>(rp, pre, t0, t0 + TILE < R ? t0 + TILE : R, src0, dst0, src1, dst1);
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
  const long long C = gridDim.x, w = blockIdx.x;
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
  if (workers < 1 || host.B > kMaxBatch || !claim) return hipErrorInvalidValue;
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
