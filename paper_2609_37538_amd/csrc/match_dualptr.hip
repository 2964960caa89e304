// Baseline Stage One: scalar dual-pointer (sort-merge) matching with S = K.
//
// The paper's comparison point (Section 2, Appendix C) keeps exactly K cached
// ids, sorts the requested ids, and merges the two sorted lists with two
// pointers: equal ids keep their slot, the other requested ids miss and take
// the freed slots.  Here one workgroup per request sorts the selection
// cooperatively in LDS (bitonic), a single lane performs the two-pointer merge
// (the scalar part the paper measures), and the freed slots are compacted in
// increasing slot order and handed to the misses in increasing id order.  The
// request's cached list is kept sorted by id between steps, so only the
// selection needs sorting.
#include "avsg_internal.h"

namespace avsg {
namespace {

constexpr int NT = 1024;
constexpr int NW = NT / 64;

__device__ __forceinline__ int lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

__host__ __device__ inline int next_pow2(int v) {
  int p = 1;
  while (p < v) p <<= 1;
  return p;
}

__global__ __launch_bounds__(NT) void match_dualptr_kernel(DualPtrParams p) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int K = p.K;
  const int Kp = next_pow2(K);
  unsigned long long* key = reinterpret_cast<unsigned long long*>(lds);       // [Kp] (id, pos)
  int2* cs = reinterpret_cast<int2*>(key + Kp);                                 // [K] cached (id, slot)
  int2* missv = cs + K;                                                         // [K] misses (id, pos)
  int32_t* os = reinterpret_cast<int32_t*>(missv + K);                          // [K] slot per position
  int32_t* freed = os + K;                                                      // [K]
  unsigned char* used = reinterpret_cast<unsigned char*>(freed + K);            // [K]
  int32_t* sw = reinterpret_cast<int32_t*>(used + ((K + 15) & ~15));           // scratch

  const int r = blockIdx.x, tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
  const int32_t* x = p.topk + static_cast<size_t>(r) * K;
  int2* st = p.state + static_cast<size_t>(r) * K;
  const int64_t rows_r = p.rows[r];

  int bad = 0;
  for (int i = tid; i < Kp; i += NT) {
    if (i < K) {
      const int32_t xi = x[i];
      if (xi < 0 || static_cast<int64_t>(xi) >= rows_r) bad++;
      key[i] = (static_cast<unsigned long long>(static_cast<uint32_t>(xi)) << 32) |
               static_cast<uint32_t>(i);
      cs[i] = st[i];
      used[i] = 0;
    } else {
      key[i] = ~0ull;
    }
  }
  __syncthreads();
  // bitonic sort of the selection by (id, position)
  for (int size = 2; size <= Kp; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = tid; t < Kp / 2; t += NT) {
        const int i = 2 * stride * (t / stride) + (t % stride);
        const int j = i + stride;
        const bool asc = (i & size) == 0;
        const unsigned long long a = key[i], b = key[j];
        if ((a > b) == asc) {
          key[i] = b;
          key[j] = a;
        }
      }
      __syncthreads();
    }
  }
  // the scalar two-pointer merge
  if (tid == 0) {
    int pc = 0, nm = 0;
    for (int q = 0; q < K;) {
      const int32_t xid = static_cast<int32_t>(key[q] >> 32);
      const int32_t pos = static_cast<int32_t>(key[q] & 0xFFFFFFFFu);
      const int2 c = pc < K ? cs[pc] : make_int2(0x7FFFFFFF, 0);
      if (pc < K && c.x < xid) {
        pc++;
      } else if (pc < K && c.x == xid) {
        os[pos] = c.y;
        used[c.y] = 1;
        pc++;
        q++;
      } else {
        missv[nm++] = make_int2(xid, pos);
        q++;
      }
    }
    sw[0] = nm;
  }
  __syncthreads();
  const int nm = sw[0];
  // freed slots in increasing slot order
  const int per = (K + NT - 1) / NT;
  const int j0 = tid * per;
  int cnt = 0;
  for (int e = 0; e < per; ++e) {
    const int j = j0 + e;
    cnt += (j < K && !used[j]) ? 1 : 0;
  }
  int incl = cnt;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  if (lane == 63) sw[1 + wave] = incl;
  __syncthreads();
  int rk = incl - cnt;
  for (int w = 0; w < wave; ++w) rk += sw[1 + w];
  for (int e = 0; e < per; ++e) {
    const int j = j0 + e;
    if (j < K && !used[j]) freed[rk++] = j;
  }
  __syncthreads();
  int2* ml = p.miss_list + static_cast<size_t>(r) * K;
  for (int k = tid; k < nm; k += NT) {
    const int2 mv = missv[k];
    const int slot = freed[k];
    os[mv.y] = slot;
    ml[k] = make_int2(mv.x, slot);
  }
  __syncthreads();
  int32_t* og = p.slots_out + static_cast<size_t>(r) * K;
  for (int i = tid; i < K; i += NT) {
    og[i] = os[i];
    const int32_t xid = static_cast<int32_t>(key[i] >> 32);
    const int32_t pos = static_cast<int32_t>(key[i] & 0xFFFFFFFFu);
    st[i] = make_int2(xid, os[pos]);   // new cached list, sorted by id
  }
  // counters
  int b = bad;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) b += __shfl_xor(b, off, 64);
  if (lane == 0) sw[1 + NW + wave] = b;
  __syncthreads();
  if (tid == 0) {
    int tb = 0;
    for (int w = 0; w < NW; ++w) tb += sw[1 + NW + w];
    p.miss_counts[r] = nm;
    unsigned long long* s = p.stats + static_cast<size_t>(r) * kNumStats;
    s[kStatHits] += static_cast<unsigned long long>(K - nm);
    s[kStatMisses] += static_cast<unsigned long long>(nm);
    s[kStatBadIndices] += static_cast<unsigned long long>(tb);
  }
}

__global__ void reset_dualptr_kernel(int2* state, int B, int K) {
  const size_t n = static_cast<size_t>(B) * K;
  for (size_t j = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; j < n;
       j += static_cast<size_t>(gridDim.x) * blockDim.x)
    state[j] = make_int2(-1, static_cast<int>(j % K));
}

}  // namespace

size_t dualptr_lds_bytes(int K) {
  const size_t Kp = static_cast<size_t>(next_pow2(K));
  return 8 * Kp + 8 * static_cast<size_t>(K) * 2 + 4 * static_cast<size_t>(K) * 2 +
         ((static_cast<size_t>(K) + 15) & ~size_t(15)) + 4 * (1 + 2 * NW + 8);
}

hipError_t prepare_match_dualptr(size_t lds) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&match_dualptr_kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
}

hipError_t launch_match_dualptr(const DualPtrParams& p, size_t lds, hipStream_t s) {
  hipLaunchKernelGGL(match_dualptr_kernel, dim3(p.B), dim3(NT), lds, s, p);
  return hipGetLastError();
}

hipError_t launch_reset_dualptr(int2* state, int B, int K, hipStream_t s) {
  const size_t n = static_cast<size_t>(B) * K;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(reset_dualptr_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s,
                     state, B, K);
  return hipGetLastError();
}

}  // namespace avsg
