// Pipelined decode step on gfx950: Stage One and Stage Two in one launch.
//
// The paper leaves overlapping state maintenance with the transfer as future
// work (decoupled state update with latency hiding).  Here one 1024-thread
// workgroup runs per CU.  Workgroups 0..B-1 first run Stage One for their
// request (the same code as the matching kernel); after each token they
// publish that token's transfer-list entries as chunks of kChunk misses in a
// device-wide queue, stamped with the step's epoch (one more than the last
// step's, kept in device memory, so a captured step replayed from a HIP graph
// stamps every replay anew).  Every workgroup -- the
// producers once their request is matched -- then claims chunks with an
// atomic counter and copies them, so copying starts after the first token of
// the first requests instead of after the whole batch is matched.  Work is
// balanced dynamically: any two workgroups' shares differ by at most a chunk.
//
// Progress does not depend on scheduling: producers never wait, consumers wait
// only for producers, and producers have the lowest workgroup ids.  Every
// poll of a consumer counts against a fixed bound: past it the consumer sets
// an error flag and leaves rather than hang; a producer whose chunks do not
// fit in the queue sets the same flag.  The last workgroup to leave resets the queue for the next step.
#include "gather_body.h"
#include "match_body.h"

namespace avsg {
namespace {

#ifndef AVSG_PIPE_CHUNK
#define AVSG_PIPE_CHUNK 32
#endif
constexpr int kChunk = AVSG_PIPE_CHUNK;     // misses per queue entry (at most 1024)
static_assert(kChunk >= 1 && kChunk <= kMatchThreads, "one staging thread per miss of a chunk");
constexpr unsigned kSpinLimit = 1u << 24;   // polls before a consumer gives up

// Loads and stores coherent at device scope without fencing the whole L2.
__device__ __forceinline__ int load_agent(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_agent(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int2 load_agent2(const int2* p) {
  const unsigned long long v = __hip_atomic_load(reinterpret_cast<const unsigned long long*>(p),
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_int2(static_cast<int>(v & 0xFFFFFFFFull), static_cast<int>(v >> 32));
}

struct QueuePublish {
  PipeParams q;
  // called by every thread of the producer workgroup after a token's
  // transfer-list entries [first, first + count) of request r are written
  __device__ void operator()(int r, int first, int count) const {
    // the dense miss lanes (threads below count) wrote the entries: their
    // waves make them visible at device scope before the queue entry is set
    if ((static_cast<int>(threadIdx.x) & ~63) < count) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (threadIdx.x == 0) {
      const int nch = (count + kChunk - 1) / kChunk;
      const int base = atomicAdd(q.tail, nch);
      // a queue sized below a step's chunks is a broken invariant: report it
      // (consumers waiting for the dropped chunks then time out and leave)
      if (base + nch > q.max_chunks) atomicExch(q.error, 1);
      for (int c = 0; c < nch && base + c < q.max_chunks; ++c) {
        int4* e = q.chunks + base + c;
        store_agent(&e->x, r);
        store_agent(&e->y, first + c * kChunk);
        store_agent(&e->z, min(kChunk, count - c * kChunk));
      }
      for (int c = 0; c < nch && base + c < q.max_chunks; ++c)
        __hip_atomic_store(&q.chunks[base + c].w, q.epoch, __ATOMIC_RELEASE,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
  }
};

__device__ __forceinline__ void consume(const GatherParams& gp, const PipeParams& q, unsigned char* lds) {
  uint64_t* src0 = reinterpret_cast<uint64_t*>(lds);
  uint64_t* dst0 = src0 + kChunk;
  uint64_t* src1 = dst0 + kChunk;
  uint64_t* dst1 = src1 + kChunk;
  int* sh = reinterpret_cast<int*>(dst1 + kChunk);
  const size_t per_req = static_cast<size_t>(gp.n_q) * gp.K;
  for (;;) {
    if (threadIdx.x == 0) {
      const int i = atomicAdd(q.head, 1);
      int stop = 0, r = 0, off = 0, cnt = 0;
      for (unsigned spins = 0;; ++spins) {
        if (i < q.max_chunks && load_agent(&q.chunks[i].w) == q.epoch) {
          r = load_agent(&q.chunks[i].x);
          off = load_agent(&q.chunks[i].y);
          cnt = load_agent(&q.chunks[i].z);
          break;
        }
        if (load_agent(q.done) == gp.B) {
          // every producer's tail update precedes its done increment
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
          if (i >= load_agent(q.tail)) {
            stop = 1;
            break;
          }
          // else entry i is published but not yet visible here: keep polling,
          // under the same bound
        }
        if (spins > kSpinLimit) {
          atomicExch(q.error, 1);
          stop = 1;
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
      sh[0] = stop;
      sh[1] = r;
      sh[2] = off;
      sh[3] = cnt;
    }
    __syncthreads();
    const int stop = sh[0], r = sh[1], off = sh[2];
    if (stop) break;
    const bool entry_ok = r >= 0 && r < gp.B && off >= 0 && sh[3] >= 0 && sh[3] <= kChunk &&
                          static_cast<size_t>(off) + sh[3] <= per_req;
    const int cnt = entry_ok ? sh[3] : 0;
    if (threadIdx.x < cnt) {
      const int2 e = load_agent2(gp.miss_list + static_cast<size_t>(r) * per_req + off + threadIdx.x);
      const bool ok = e.x >= 0 && static_cast<int64_t>(e.x) < gp.rows[r] && e.y >= 0 && e.y < gp.S;
      const int i = threadIdx.x;
      src0[i] = ok ? gp.host_ptrs[r] + static_cast<uint64_t>(e.x) * gp.row_bytes0 : 0;
      dst0[i] = ok ? gp.buf_ptrs[r] + static_cast<uint64_t>(e.y) * gp.row_bytes0 : 0;
      if (gp.n_streams > 1) {
        src1[i] = ok ? gp.host_ptrs[gp.B + r] + static_cast<uint64_t>(e.x) * gp.row_bytes1 : 0;
        dst1[i] = ok ? gp.buf_ptrs[gp.B + r] + static_cast<uint64_t>(e.y) * gp.row_bytes1 : 0;
      }
    }
    __syncthreads();
    // every thread of the workgroup copies, one 16-byte (or 4-byte) load in
    // flight each: the fused kernel's register budget is set by Stage One
    if ((gp.row_bytes0 & 15) == 0)
      copy_rows<u32x4, 1, kMatchThreads>(src0, dst0, cnt, static_cast<int>(gp.row_bytes0 / 16));
    else
      copy_rows<uint32_t, 1, kMatchThreads>(src0, dst0, cnt, static_cast<int>(gp.row_bytes0 / 4));
    if (gp.n_streams > 1) {
      if ((gp.row_bytes1 & 15) == 0)
        copy_rows<u32x4, 1, kMatchThreads>(src1, dst1, cnt, static_cast<int>(gp.row_bytes1 / 16));
      else
        copy_rows<uint32_t, 1, kMatchThreads>(src1, dst1, cnt, static_cast<int>(gp.row_bytes1 / 4));
    }
    __syncthreads();
  }
}

template <int IPT>
__global__ __launch_bounds__(kMatchThreads) void step_pipelined_kernel(MatchParams mp, GatherParams gp,
                                                                       PipeParams q) {
  extern __shared__ __align__(16) unsigned char lds[];
  // every workgroup reads the last stamp before any can leave, and only the
  // last to leave advances it
  q.epoch = load_agent(q.last_epoch) + 1;
  if (q.epoch <= 0) q.epoch = 1;
  if (static_cast<int>(blockIdx.x) < mp.B) {
    QueuePublish pub{q};
    match_request<IPT, kMatchThreads, 0>(mp, static_cast<int>(blockIdx.x), lds, pub);
    __syncthreads();
    if (threadIdx.x == 0) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      atomicAdd(q.done, 1);
    }
  }
  consume(gp, q, lds);
  if (threadIdx.x == 0) {
    __threadfence();
    if (atomicAdd(q.exit_count, 1) == static_cast<int>(gridDim.x) - 1) {
      // every other workgroup has left: reset the queue for the next step
      *q.head = 0;
      *q.tail = 0;
      *q.done = 0;
      *q.last_epoch = q.epoch;
      __threadfence();
      *q.exit_count = 0;
    }
  }
}

}  // namespace

int pipelined_chunk_misses() { return kChunk; }

size_t pipelined_lds_bytes(int S, int K) {
  const size_t m = match_lds_bytes(S, K);
  const size_t c = 4 * kChunk * sizeof(uint64_t) + 4 * sizeof(int);
  return m > c ? m : c;
}

hipError_t prepare_step_pipelined(size_t lds) {
  hipError_t e;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(&step_pipelined_kernel<1>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(&step_pipelined_kernel<2>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(&step_pipelined_kernel<3>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&step_pipelined_kernel<4>),
                             hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
}

hipError_t launch_step_pipelined(const MatchParams& mp, const GatherParams& gp, const PipeParams& q,
                                 int workgroups, size_t lds, hipStream_t s) {
  if (workgroups < mp.B) return hipErrorInvalidValue;
  const dim3 grid(workgroups), block(kMatchThreads);
  switch ((mp.K + kMatchThreads - 1) / kMatchThreads) {
    case 1: hipLaunchKernelGGL(step_pipelined_kernel<1>, grid, block, lds, s, mp, gp, q); break;
    case 2: hipLaunchKernelGGL(step_pipelined_kernel<2>, grid, block, lds, s, mp, gp, q); break;
    case 3: hipLaunchKernelGGL(step_pipelined_kernel<3>, grid, block, lds, s, mp, gp, q); break;
    case 4: hipLaunchKernelGGL(step_pipelined_kernel<4>, grid, block, lds, s, mp, gp, q); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace avsg
