// Stage One of AVSG on gfx950: vectorized open-addressing hash matching,
// lifetime-based slot reservation and shared MTP reservations.
//
// One workgroup of 1024 threads (16 wave64s) owns one request.  The request's
// Hash-State table (Section 3.2: cached index c_j and metadata word q_j, Eq. 2)
// is staged from HBM into LDS as three arrays -- c[S] (int32), the low 24 bits
// of q (invalid | fingerprint | slot) and the lifetime byte -- so that lifetime
// and mapping updates never touch the same LDS word.  Every selected index is
// probed by its own lane (Probe, Eq. 8-11); misses are compacted in index order
// with wave ballots and a workgroup prefix; the dead-slot list of CollectDead
// (Eq. 12) is produced the same way; the allocation decay loop of Algorithm 1
// is evaluated as counts of lifetimes below k, so all k* unit decays are
// applied in one sweep; UpdateState (Algorithm 2) reads the reusable predicate
// (Eq. 4) on the pre-write table and installs mappings with an LDS atomic max
// so that the miss with the largest rank keeps a contended bucket
// deterministically.  The N_q tokens of a request run in order on the same
// LDS table (Algorithm 4); speculative invalidation is fused into the write
// back to HBM.
#include "avsg_internal.h"

namespace avsg {
namespace {

constexpr int NT = kMatchThreads;
constexpr int NW = NT / 64;
constexpr int kMaxIPT = 4;           // up to K = 4096 indices per token
constexpr int kScratchInts = 2 * kMaxIPT * NW + NW + 4 + 16;

__device__ __forceinline__ int lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}
// number of set bits of `mask` at lanes below this lane
__device__ __forceinline__ int bits_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}
__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
__device__ __forceinline__ int wave_inclusive_scan(int v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int t = __shfl_up(v, off, 64);
    if (lane >= off) v += t;
  }
  return v;
}

__host__ __device__ constexpr size_t align16(size_t v) { return (v + 15) & ~size_t(15); }

template <int IPT>
__global__ __launch_bounds__(NT) void match_hash_kernel(MatchParams p) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int S = p.S, K = p.K, R = p.R;
  const uint32_t smask = static_cast<uint32_t>(S - 1);
  int32_t* sc = reinterpret_cast<int32_t*>(lds);
  uint32_t* smap = reinterpret_cast<uint32_t*>(lds + 4 * static_cast<size_t>(S));
  int8_t* slife = reinterpret_cast<int8_t*>(lds + 8 * static_cast<size_t>(S));
  int32_t* somiss = reinterpret_cast<int32_t*>(lds + 8 * static_cast<size_t>(S) + align16(S));
  int32_t* swc = somiss + K;                 // [2][IPT][NW] miss counts per wave
  int32_t* sdead = swc + 2 * kMaxIPT * NW;   // [NW] dead counts per wave
  int32_t* sred = sdead + NW;                // [3] rotating reduction slots
  int32_t* sstat = sred + 4;                 // [8] counter reduction

  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = lane_id();

  int32_t* gc = p.table_c + static_cast<size_t>(r) * S;
  uint32_t* gq = p.table_q + static_cast<size_t>(r) * S;
  for (int j = tid; j < S; j += NT) {
    const uint32_t q = gq[j];
    sc[j] = gc[j];
    smap[j] = q & 0xFFFFFFu;
    slife[j] = static_cast<int8_t>(q >> 24);
  }
  if (tid < 4) sred[tid] = 0;
  if (tid < 8) sstat[tid] = 0;

  const int SPT = (S + NT - 1) / NT;  // lifetimes owned by this thread: [j0, j0 + SPT)
  const int j0 = tid * SPT;
  const int64_t rows_r = p.rows[r];
  const int64_t n_verified = p.verified ? p.verified[r] : INT64_MAX;
  const uint32_t a1 = p.a1, a2 = p.a2, fmask = p.f_mask;
  const int m = p.m, L = p.L;

  int st_hits = 0, st_miss = 0, st_exh = 0, st_col = 0, st_rev = 0, st_bad = 0;
  int step_decays = 0;
  int listed = 0;
  int red_it = 0;
  __syncthreads();

  for (int g = 0; g < p.n_q; ++g) {
    // Pass 1 (refresh): the first token decays every lifetime by one.
    if (g == 0) {
      for (int e = 0; e < SPT; ++e) {
        const int j = j0 + e;
        if (j < S) {
          const int l = slife[j];
          slife[j] = static_cast<int8_t>(l > -1 ? l - 1 : -1);
        }
      }
      __syncthreads();
    }
    const size_t row = static_cast<size_t>(r) * p.n_q + g;
    const int32_t* xg = p.topk + row * K;
    int32_t* og = p.slots_out + row * K;
    int32_t* wc = swc + (g & 1) * kMaxIPT * NW;

    int32_t xv[IPT];
    bool hit[IPT], act[IPT];
    int rank[IPT];
#pragma unroll
    for (int u = 0; u < IPT; ++u) {
      const int i = u * NT + tid;
      act[u] = i < K;
      const int32_t x = act[u] ? xg[i] : 0;
      xv[u] = x;
      bool h_ok = false;
      if (act[u]) {
        if (x < 0 || static_cast<int64_t>(x) >= rows_r) st_bad++;
        const uint32_t ux = static_cast<uint32_t>(x);
        uint32_t h = (a1 * ux) & smask;              // initial bucket (Eq. 9)
        const uint32_t d = ((a2 * ux) & smask) | 1u;  // odd stride (Eq. 9)
        int o = 0;
        for (int rd = 0; rd <= R; ++rd) {
          o = static_cast<int>(smap[h] & smask);      // candidate slot (Eq. 10)
          if (sc[o] == x) {
            h_ok = true;
            break;
          }
          h = (h + d) & smask;                        // unresolved probes advance (Eq. 11)
        }
        if (h_ok) {
          if (slife[o] < 0) st_rev++;
          slife[o] = static_cast<int8_t>(L);          // refresh the hit slot
          og[i] = o;                                  // Pass 2: o[m] = o^match
          st_hits++;
        }
      }
      hit[u] = h_ok;
      if (p.hit_mask && act[u]) p.hit_mask[row * K + i] = h_ok ? 1 : 0;
      const uint64_t mm = __ballot(act[u] && !h_ok);
      if (lane == 0) wc[u * NW + wave] = __popcll(mm);
      rank[u] = bits_below(mm);
    }
    __syncthreads();

    // Pass 2 (classify): miss ranks in index order and the miss count n_g.
    int n_g = 0;
#pragma unroll
    for (int u = 0; u < IPT; ++u) {
      int tot = 0, before = 0;
      for (int w = 0; w < NW; ++w) {
        const int c = wc[u * NW + w];
        tot += c;
        before += (w < wave) ? c : 0;
      }
      rank[u] += n_g + before;
      n_g += tot;
    }
    if (tid == 0) p.miss_counts[row] = n_g;

    if (n_g > 0) {
      // Pass 3 (allocate).  The decay loop of Algorithm 1 stops at the first
      // k with #{j : lifetime_j - k < 0} >= n_g; count lifetimes below k.
      int kstar = 0;
      for (int k = 0;; ++k) {
        int cnt = 0;
        for (int e = 0; e < SPT; ++e) {
          const int j = j0 + e;
          cnt += (j < S && slife[j] < k) ? 1 : 0;
        }
        cnt = wave_sum(cnt);
        const int slot = red_it % 3;
        if (lane == 0 && cnt) atomicAdd(&sred[slot], cnt);
        if (tid == 0) sred[(red_it + 1) % 3] = 0;
        red_it++;
        __syncthreads();
        if (sred[slot] >= n_g || k > L) {
          kstar = k;
          break;
        }
      }
      if (kstar > 0) {
        for (int e = 0; e < SPT; ++e) {
          const int j = j0 + e;
          if (j < S) {
            const int l = slife[j] - kstar;
            slife[j] = static_cast<int8_t>(l < -1 ? -1 : l);
          }
        }
        step_decays += kstar;
      }
      // CollectDead (Eq. 12): dead slots in increasing order; o^miss = e[:n_g].
      int dcnt = 0;
      for (int e = 0; e < SPT; ++e) {
        const int j = j0 + e;
        dcnt += (j < S && slife[j] < 0) ? 1 : 0;
      }
      const int incl = wave_inclusive_scan(dcnt, lane);
      if (lane == 63) sdead[wave] = incl;
      __syncthreads();
      int drank = incl - dcnt;
      for (int w = 0; w < wave; ++w) drank += sdead[w];
      if (drank < n_g) {
        for (int e = 0; e < SPT && drank < n_g; ++e) {
          const int j = j0 + e;
          if (j < S && slife[j] < 0) somiss[drank++] = j;
        }
      }
      __syncthreads();

      // UpdateState (Algorithm 2): reusable chains on the pre-write table.
      uint32_t hk[IPT];
      bool vk[IPT];
      int onew[IPT];
#pragma unroll
      for (int u = 0; u < IPT; ++u) {
        hk[u] = 0;
        vk[u] = false;
        onew[u] = 0;
        if (act[u] && !hit[u]) {
          onew[u] = somiss[rank[u]] & static_cast<int>(smask);
          const uint32_t ux = static_cast<uint32_t>(xv[u]);
          uint32_t h = (a1 * ux) & smask;
          const uint32_t d = ((a2 * ux) & smask) | 1u;
          bool v = false;
          for (int rd = 0; rd <= R; ++rd) {
            const uint32_t qh = smap[h];
            const uint32_t o2 = qh & smask;
            const bool invalid = (qh >> 23) & 1u;
            const uint32_t fph = (qh >> m) & fmask;
            if (invalid || slife[o2] < 0 || fph != (static_cast<uint32_t>(sc[o2]) & fmask)) {
              v = true;   // reusable (Eq. 4)
              break;
            }
            if (rd < R) h = (h + d) & smask;
          }
          hk[u] = h;
          vk[u] = v;
        }
      }
      __syncthreads();
      // every miss owns its slot; reusable probes bid for their bucket
      const size_t lbase = static_cast<size_t>(r) * p.n_q * K + listed;
#pragma unroll
      for (int u = 0; u < IPT; ++u) {
        if (act[u] && !hit[u]) {
          const int i = u * NT + tid;
          sc[onew[u]] = xv[u];
          slife[onew[u]] = static_cast<int8_t>(L);
          if (vk[u]) atomicMax(&smap[hk[u]], 0x80000000u | static_cast<uint32_t>(onew[u]));
          og[i] = onew[u];                              // o[not m] = o^miss
          p.miss_list[lbase + rank[u]] = make_int2(xv[u], onew[u]);
          st_miss++;
        }
      }
      __syncthreads();
      // the largest bid (largest o^miss = largest miss rank) installs its mapping
#pragma unroll
      for (int u = 0; u < IPT; ++u) {
        if (act[u] && !hit[u]) {
          if (vk[u]) {
            const uint32_t bid = 0x80000000u | static_cast<uint32_t>(onew[u]);
            if (smap[hk[u]] == bid)
              smap[hk[u]] = ((static_cast<uint32_t>(xv[u]) & fmask) << m) |
                            static_cast<uint32_t>(onew[u]);
            else
              st_col++;
          } else {
            st_exh++;
          }
        }
      }
      __syncthreads();
      listed += n_g;
    }
  }

  // End of step: speculative invalidation fused into the write back.
  int st_inv = 0;
  for (int j = tid; j < S; j += NT) {
    int32_t c = sc[j];
    if (static_cast<int64_t>(c) >= n_verified) {
      c = -1;
      st_inv++;
    }
    gc[j] = c;
    gq[j] = (static_cast<uint32_t>(static_cast<uint8_t>(slife[j])) << 24) | (smap[j] & 0xFFFFFFu);
  }

  int vals[7] = {st_hits, st_miss, st_exh, st_col, st_rev, st_inv, st_bad};
#pragma unroll
  for (int k = 0; k < 7; ++k) {
    const int v = wave_sum(vals[k]);
    if (lane == 0 && v) atomicAdd(&sstat[k], v);
  }
  __syncthreads();
  if (tid == 0) {
    unsigned long long* st = p.stats + static_cast<size_t>(r) * kNumStats;
    st[kStatHits] += static_cast<unsigned long long>(sstat[0]);
    st[kStatMisses] += static_cast<unsigned long long>(sstat[1]);
    st[kStatLostExhausted] += static_cast<unsigned long long>(sstat[2]);
    st[kStatLostCollision] += static_cast<unsigned long long>(sstat[3]);
    st[kStatRevivals] += static_cast<unsigned long long>(sstat[4]);
    st[kStatInvalidations] += static_cast<unsigned long long>(sstat[5]);
    st[kStatBadIndices] += static_cast<unsigned long long>(sstat[6]);
    st[kStatAllocDecays] += static_cast<unsigned long long>(step_decays);
    if (static_cast<unsigned long long>(step_decays) > st[kStatMaxStepDecays])
      st[kStatMaxStepDecays] = static_cast<unsigned long long>(step_decays);
  }
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

int ipt_for(int K) { return (K + NT - 1) / NT; }

}  // namespace

size_t match_lds_bytes(int S, int K) {
  const int ipt = ipt_for(K);
  if (ipt < 1 || ipt > kMaxIPT) return 0;
  return 8 * static_cast<size_t>(S) + align16(S) + 4 * static_cast<size_t>(K) +
         4 * static_cast<size_t>(kScratchInts);
}

hipError_t prepare_match_hash(size_t lds) {
  hipError_t e;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(&match_hash_kernel<1>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(&match_hash_kernel<2>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(&match_hash_kernel<3>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&match_hash_kernel<4>),
                             hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
}

hipError_t launch_match_hash(const MatchParams& p, size_t lds, hipStream_t s) {
  const dim3 grid(p.B), block(NT);
  switch (ipt_for(p.K)) {
    case 1: hipLaunchKernelGGL(match_hash_kernel<1>, grid, block, lds, s, p); break;
    case 2: hipLaunchKernelGGL(match_hash_kernel<2>, grid, block, lds, s, p); break;
    case 3: hipLaunchKernelGGL(match_hash_kernel<3>, grid, block, lds, s, p); break;
    case 4: hipLaunchKernelGGL(match_hash_kernel<4>, grid, block, lds, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
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
