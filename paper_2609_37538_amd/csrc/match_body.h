// Device code of Stage One shared by the matching kernel and the pipelined
// step kernel (see match_hash.hip for the phases).
#pragma once

#include "avsg_internal.h"

namespace avsg {
namespace {


// A workgroup has NT threads (1024, or 256 for small tables); the LDS
// bookkeeping below is sized for the largest workgroup.
constexpr int kMaxWaves = kMatchThreads / 64;
constexpr int kMaxIPT = 4;                 // up to 4 NT indices per token
constexpr int kMaxSPT = 16;                // up to 16 NT slots
constexpr int kScratchInts = 2 * kMaxIPT * kMaxWaves + kMaxWaves + 4;
constexpr uint32_t kBid = 0x80000000u;     // marks a bucket written by an install bid

// 16-byte vectors as clang vector types (kept in registers)
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}
// number of set bits of `mask` at lanes below this lane
__device__ __forceinline__ int bits_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}
// Inclusive prefix sum over the 64 lanes of a wave, register to register
// with DPP: shifts by 1, 2, 4 and 8 lanes inside each 16-lane row (a lane
// whose source lies outside its row adds 0), then the last lane of row 0 is
// broadcast into row 1 and of row 2 into row 3, and the last lane of row 1
// (by then the total of rows 0-1) into rows 2 and 3.  Every lane of the wave
// must be active.
__device__ __forceinline__ int wave_inclusive_scan(int v, int /*lane*/) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);   // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);   // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);   // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);   // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);   // row_bcast:15 into rows 1, 3
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);   // row_bcast:31 into rows 2, 3
  return v;
}
// Sum over the 64 lanes of a wave, in every lane (every lane active).
__device__ __forceinline__ int wave_sum(int v) {
  return __builtin_amdgcn_readlane(wave_inclusive_scan(v, 0), 63);
}
// Orders this wave's LDS accesses before and after it for the compiler (the
// hardware runs one wave's LDS instructions in order): lanes that read what
// other lanes of the wave wrote call it in between.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}
// Index of this thread's wave, held in a scalar register.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6); }
// Per-wave values cnt[0..nw) (nw <= 64) as seen by wave `wave`: the sum over
// the waves before it and over all of them.  Lane w reads cnt[w] and a wave
// scan adds them up, so the sums take one LDS read (every lane active).
struct WavePrefix {
  int before, total;
};
__device__ __forceinline__ WavePrefix wave_prefix(const int* cnt, int nw, int wave) {
  const int lane = lane_id();
  const int incl = wave_inclusive_scan(lane < nw ? cnt[lane] : 0, lane);
  WavePrefix r;
  r.total = __builtin_amdgcn_readlane(incl, 63);
  r.before = wave > 0 ? __builtin_amdgcn_readlane(incl, wave - 1) : 0;
  return r;
}

__host__ __device__ constexpr size_t align16(size_t v) { return (v + 15) & ~size_t(15); }

// The low 32 bits of the product of the low 24 bits of a and b, as the
// full-rate v_mul_u32_u24 (a uniform).  Written as that one instruction since
// the compiler otherwise folds the masks around a 24-bit multiply into a
// quarter-rate 32-bit one.
__device__ __forceinline__ uint32_t mul24(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_mul_u32_u24 %0, %1, %2" : "=v"(r) : "s"(a), "v"(b));
  return r;
}
// the same with a divergent first operand
__device__ __forceinline__ uint32_t mul24v(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_mul_u32_u24 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// Bucket words in LDS keep the fields of Eq. 3 with the slot above the
// fingerprint: invalid << 23 | slot << (23 - m) | fingerprint, or, for an
// install bid, kBid | token << 24 | slot << (23 - m) | fingerprint (bit 23
// clear: a bid is a valid mapping).  Both forms decode alike; the table in
// HBM keeps the Eq. 3 order (invalid | fingerprint | slot), converted as it
// is staged in and written back.
struct Word {
  uint32_t m, smask, fmask;
  __device__ __forceinline__ uint32_t slot(uint32_t w) const { return (w >> (23 - m)) & smask; }
  __device__ __forceinline__ bool invalid(uint32_t w) const { return (w >> 23) & 1u; }
  __device__ __forceinline__ uint32_t fp(uint32_t w) const { return w & fmask; }
  // the low 24 bits of Eq. 3 from an LDS word
  __device__ __forceinline__ uint32_t canonical(uint32_t w) const {
    return (w & 0x800000u) | (fp(w) << m) | slot(w);
  }
  // an LDS word from the low 24 bits of Eq. 3
  __device__ __forceinline__ uint32_t staged(uint32_t q) const {
    return (q & 0x800000u) | ((q & smask) << (23 - m)) | ((q >> m) & fmask);
  }
};

// The lifetimes a thread owns (spt consecutive slots), four to a register as
// biased bytes v = lifetime + 1 in [0, 128] (0 = dead); bytes past spt hold
// 0xFF and never count as below any k <= 128.  Counting and decaying work on
// two 16-bit lanes per word: (v + 256 - k) has bit 8 set exactly when v >= k.
struct Own {
  static constexpr uint32_t kLo = 0x00FF00FFu, kOne = 0x00010001u, kBias = 0x01000100u;
  uint32_t w[kMaxSPT / 4];
  uint32_t pad;   // bytes of w[0] past spt (spt < 4), kept at 0xFF
  __device__ __forceinline__ int get(int e) const {
    return static_cast<int>((w[e >> 2] >> (8 * (e & 3))) & 0xFFu) - 1;
  }
  __device__ __forceinline__ void set(int e, int life) {
    const uint32_t sh = 8 * (e & 3);
    w[e >> 2] = (w[e >> 2] & ~(0xFFu << sh)) | (static_cast<uint32_t>(life + 1) << sh);
  }
  // two's-complement lifetime bytes <-> biased bytes, four at a time
  static __device__ __forceinline__ uint32_t bias(uint32_t raw) {
    return ((raw & 0x7F7F7F7Fu) + 0x01010101u) ^ (raw & 0x80808080u);
  }
  static __device__ __forceinline__ uint32_t unbias(uint32_t b) {
    return ((b | 0x80808080u) - 0x01010101u) ^ ((b ^ 0xFEFEFEFEu) & 0x80808080u);
  }
  // one decay, never below -1, of four two's-complement lifetime bytes:
  // (v + 127) has bit 7 set exactly when the biased byte v is at least 1
  static __device__ __forceinline__ uint32_t decay1(uint32_t raw) {
    const uint32_t v = bias(raw);
    return unbias(v - (((v + 0x7F7F7F7Fu) & 0x80808080u) >> 7));
  }
  __device__ __forceinline__ void load(const int8_t* slife, int j0, int spt) {
#pragma unroll
    for (int k = 0; k < kMaxSPT / 4; ++k) w[k] = 0xFFFFFFFFu;
    pad = spt >= 4 ? 0u : 0xFFFFFFFFu << (8 * spt);
    if (spt >= 4) {
      const uint32_t* p = reinterpret_cast<const uint32_t*>(slife + j0);
#pragma unroll
      for (int k = 0; k < kMaxSPT / 4; ++k)
        if (k < spt / 4) w[k] = bias(p[k]);
    } else {
#pragma unroll
      for (int e = 0; e < 3; ++e)
        if (e < spt) set(e, slife[j0 + e]);
    }
  }
  __device__ __forceinline__ void store(int8_t* slife, int j0, int spt) const {
    if (spt >= 4) {
      uint32_t* p = reinterpret_cast<uint32_t*>(slife + j0);
#pragma unroll
      for (int k = 0; k < kMaxSPT / 4; ++k)
        if (k < spt / 4) p[k] = unbias(w[k]);
    } else {
#pragma unroll
      for (int e = 0; e < 3; ++e)
        if (e < spt) slife[j0 + e] = static_cast<int8_t>(get(e));
    }
  }
  // number of owned lifetimes below k (0 <= k <= 128)
  __device__ __forceinline__ int count_below(int k, int spt) const {
    const uint32_t kk = static_cast<uint32_t>(k + 1) * kOne;
    int at_least = 0, n = 0;
#pragma unroll
    for (int i = 0; i < kMaxSPT / 4; ++i)
      if (i < (spt + 3) / 4) {
        const uint32_t te = ((w[i] & kLo) + kBias) - kk;
        const uint32_t to = (((w[i] >> 8) & kLo) + kBias) - kk;
        at_least += __popc(((te >> 8) & kOne) | (((to >> 8) & kOne) << 1));
        n += 4;
      }
    return n - at_least;
  }
  // decay by k (1 <= k <= 128), never below -1
  __device__ __forceinline__ void decay(int k, int spt) {
    const uint32_t kk = static_cast<uint32_t>(k) * kOne;
#pragma unroll
    for (int i = 0; i < kMaxSPT / 4; ++i)
      if (i < (spt + 3) / 4) {
        const uint32_t te = ((w[i] & kLo) + kBias) - kk;
        const uint32_t to = (((w[i] >> 8) & kLo) + kBias) - kk;
        const uint32_t me = ((te >> 8) & kOne) * 0xFFu, mo = ((to >> 8) & kOne) * 0xFFu;
        w[i] = (te & me) | ((to & mo) << 8);
      }
    w[0] |= pad;
  }
};

// Words of LDS bookkeeping of the end-of-step plan besides the reservation
// bitmap, the index map and its fan words: per-wave counts of the three lists
// for two compaction rounds, plus totals.
constexpr int kPlanMiscWords = 6 * kMaxWaves + 4;
// 16-bit entries of a wave's list of scan candidates: a wave appends at most
// 64 to fewer than 64 pending ones before it walks 64 of them.
constexpr int kPlanScanList = 128;
// Words of the plan's reservation bitmap for S slots, padded to a multiple of
// four so that the map behind it starts 16-byte aligned.
__host__ __device__ constexpr int plan_bitmap_words(int S) { return (((S + 31) >> 5) + 3) & ~3; }
// All LDS words of the plan past c[]: the reservation bitmap, P map words, P
// fan words and the counters.
__host__ __device__ constexpr size_t plan_state_words(int S, int P) {
  return static_cast<size_t>(plan_bitmap_words(S)) + 2 * static_cast<size_t>(P) + kPlanMiscWords;
}
// A map word, from the high bits down; atomicMax on words of one index
// orders them by (resident, slot).
constexpr uint32_t kPlanResident = 0x80000000u;   // names a slot outside this step's reservations
constexpr uint32_t kPlanEarly = 0x40000000u;      // the word's index was fetched before Stage One
constexpr uint32_t kPlanTag = 0x3F000000u;        // six bits of a second hash of the word's index
constexpr uint32_t kPlanSlot = 0x00FFFFFEu;       // slot + 1, shifted up by one
constexpr uint32_t kPlanDisp = 0x00000001u;       // another index whose home is this word sits further on
__device__ __forceinline__ uint32_t plan_val(int slot) { return (static_cast<uint32_t>(slot) + 1u) << 1; }
__device__ __forceinline__ int plan_slot(uint32_t w) { return static_cast<int>((w & kPlanSlot) >> 1) - 1; }

// Home word and tag of index x in the plan's map of P words (P < 2^16), from
// one multiplicative hash of the low 24 bits of x, h = x * 0x9E3779 mod 2^32:
// the home is floor((h >> 16) * P / 2^16) (the top p bits of h when P = 2^p)
// and the tag bits 8..13 of h.  Both multiplies are full-rate 24-bit ones.
// The tag is kept in the map word so that a probe passes over most foreign
// words without reading the slot they name.  Indices that share their low 24
// bits share a home and a tag; the slot's index, read through c[], tells them
// apart.
struct PlanHash {
  uint32_t P;
  __device__ __forceinline__ explicit PlanHash(uint32_t words) : P(words) {}
  __device__ __forceinline__ uint32_t hash(int32_t x) const { return mul24(0x9E3779u, static_cast<uint32_t>(x)); }
  __device__ __forceinline__ uint32_t home(uint32_t h) const { return mul24(P, h >> 16) >> 16; }
  __device__ __forceinline__ uint32_t tag(uint32_t h) const { return ((h >> 8) & 0x3Fu) << 24; }
  __device__ __forceinline__ uint32_t next(uint32_t h) const { return h + 1u == P ? 0u : h + 1u; }
};

// A fan word: the two largest bids (slot + 1, nonzero, below 2^16), the larger
// in the low 16 bits, 0 = no bid.  Bids of one word are distinct slots.
__device__ __forceinline__ void fan_bid(uint32_t* w, uint32_t v) {
  uint32_t cur = *w;
  for (;;) {
    const uint32_t a = cur & 0xFFFFu, b = cur >> 16;
    uint32_t nw;
    if (v > a) nw = v | (a << 16);
    else if (v > b) nw = a | (v << 16);
    else return;   // not among the two largest
    const uint32_t prev = atomicCAS(w, cur, nw);
    if (prev == cur) return;
    cur = prev;
  }
}
// The two fan slots of a fan word (-1 = none).
__device__ __forceinline__ int2 fan_slots(uint32_t w) {
  return make_int2(static_cast<int>(w & 0xFFFFu) - 1, static_cast<int>(w >> 16) - 1);
}

// Position of index x's word in the map (its word in *word), or -1.
__device__ __forceinline__ int plan_lookup(const uint32_t* smp, const int32_t* sc, const PlanHash& ph,
                                           int32_t x, uint32_t* word) {
  const uint32_t hx = ph.hash(x), tag = ph.tag(hx);
  uint32_t h = ph.home(hx);
  for (uint32_t t = 0; t < ph.P; ++t) {
    const uint32_t w = smp[h];
    if (w == 0u) break;
    if ((w & kPlanTag) == tag && sc[plan_slot(w)] == x) {
      *word = w;
      return static_cast<int>(h);
    }
    h = ph.next(h);
  }
  return -1;
}

// Stage Two plan of the resident-reuse gather, after the step's table write
// back (every LDS array but c[] and the slot list is free, and the write back
// has cleared the plan's words).  Each of the step's listed misses (index x,
// slot o) becomes
//   a resident copy from the largest slot outside this step's reservations
//   that still caches x below the verified length (its row arrived in an
//   earlier step and cannot have changed), or else
//   a repeat copy from the largest slot this step reserved for x, when that is
//   not o (a later token missed x again after its install was lost), or else
//   a host copy.
// A host entry also writes its row to the two largest repeat destinations of
// its index (its fan slots: the second and third largest slots reserved for
// the index), so with up to three tokens per step no repeat is left for a
// later copy.  The lists keep transfer-list order.  LDS: a map of P words,
// open addressing with linear probing keyed by the index a word names through
// c[]; a word is (resident bit | early bit | tag | slot + 1), 0 = free, and
// atomicMax makes every choice deterministic; beside it P fan words, one per
// map word: the two largest repeat destinations of the word's index as two
// 16-bit fields of slot + 1 (larger in the low field, 0 = none; a table holds
// at most 2^14 slots), kept by a compare-and-swap loop, so the result does not
// depend on the order of the bids.  A word's lowest bit marks that an index whose home is that word
// sits further on (it may also be set on a word whose own index took a
// larger slot; that only costs the scan below a probe).  The map holds at
// most N_q * K keys and P >= 1.5 N_q K, so every probe sequence ends at a
// free word.  The transfer list is read from the
// slot list the token loop kept in LDS where there was room (entry e is slot
// o = slist[e], index c[o]: no reserved slot is reassigned within a step),
// else from device memory.
// rows_u / lim_u: an index x is valid when (uint32)x < rows_u, and a cached
// index qualifies as a resident source when (uint32)x < lim_u (both bounds
// clamped to 2^31, so negative indices fail).
template <int NT>
__device__ __forceinline__ void plan_request(const MatchParams& p, const int r, unsigned char* lds,
                                             const int listed, const uint32_t rows_u, const uint32_t lim_u,
                                             int* counts_out) {
  constexpr int MT = NT, MW = NT / 64;
  const int S = p.S;
  const int32_t* sc = reinterpret_cast<const int32_t*>(lds);
  uint32_t* sres = reinterpret_cast<uint32_t*>(lds + align16(4 * static_cast<size_t>(S)));  // reserved-slot bitmap
  const int nb = plan_bitmap_words(S);
  const uint32_t P = static_cast<uint32_t>(p.plan_words);   // a multiple of 4
  const PlanHash ph(P);
  uint32_t* smp = sres + nb;                                        // [P] index map
  uint32_t* sfan = smp + P;                                         // [P] fan word of each map word
  int* scnt = reinterpret_cast<int*>(sfan + P);                     // [kPlanMiscWords]
  const uint16_t* slist = reinterpret_cast<const uint16_t*>(lds + p.plan_list_off);
  const int tid = threadIdx.x, wave = wave_id(), lane = lane_id();
  const size_t lb = static_cast<size_t>(r) * p.n_q * p.K;
  const int2* ml = p.miss_list + lb;
  // entry e of the transfer list: (index, slot)
  auto entry = [&](int e) __attribute__((always_inline)) {
    if (p.plan_list_off == 0) return ml[e];
    const int o = slist[e];
    return make_int2(sc[o], o);
  };
  if (r == 0 && tid == 0) {
    p.plan_claim[0] = 0;
    p.plan_claim[1] = 0;
  }

  // (1) mark this step's reservations; one map word per distinct valid index
  // with its largest reserved slot, and the second and third largest in its
  // fan word
  for (int e = tid; e < listed; e += MT) {
    const int2 v = entry(e);
    const int32_t x = v.x, o = v.y;
    atomicOr(&sres[o >> 5], 1u << (o & 31));
    if (static_cast<uint32_t>(x) >= rows_u) continue;
    const uint32_t hx = ph.hash(x), tag = ph.tag(hx);
    const uint32_t val = tag | plan_val(o);
    uint32_t h = ph.home(hx);
    for (uint32_t t = 0; t < P; ++t) {
      const uint32_t w = atomicCAS(&smp[h], 0u, val);
      if (w == 0u) break;
      if ((w & kPlanTag) == tag && sc[plan_slot(w)] == x) {
        // the largest reserved slot of the index (the mark bit is set with it
        // since a mark already on the word must not be lost); whichever of
        // the old and the new slot is smaller bids for the fan word: every
        // slot of the index but the largest bids once, and the word keeps the
        // two largest bids
        const uint32_t old = atomicMax(&smp[h], val | kPlanDisp);
        const int other = (old & kPlanSlot) < (val & kPlanSlot) ? plan_slot(old) : o;
        fan_bid(&sfan[h], static_cast<uint32_t>(other) + 1u);
        break;
      }
      if (t == 0) atomicOr(&smp[h], kPlanDisp);   // another index holds the home word
      h = ph.next(h);
    }
  }
  __syncthreads();

  // (2) slots outside the reservations that cache one of those indices.  A
  // first pass reads kScan slots per thread (their LDS reads in flight
  // together) and keeps, as bits, the slots that may cache a key: qualified,
  // not reserved, and the home word of their index holds a word with the
  // index's tag or one marked as the home of an index placed further on.
  // Every slot that caches a key passes (its key sits at its home word or
  // further on from a marked home); only those walk a probe sequence, in a
  // second pass.  A key is often cached in several slots outside the
  // reservations (copies left by lost installs), so most candidates bid.
  constexpr int kScan = 8;
  // the walk of one candidate slot j: find its index's word, bid the slot
  auto walk = [&](int j) __attribute__((always_inline)) {
    const int32_t x = sc[j];
    const uint32_t hx = ph.hash(x), tag = ph.tag(hx);
    uint32_t h = ph.home(hx);
    for (uint32_t t = 0; t < P; ++t) {
      const uint32_t w = smp[h];
      if (w == 0u) break;
      if ((w & kPlanTag) == tag && sc[plan_slot(w)] == x) {
        // the marks are final by now: keep the word's own
        atomicMax(&smp[h], kPlanResident | tag | plan_val(j) | (w & kPlanDisp));
        break;
      }
      h = ph.next(h);
    }
  };
  // a wave's candidates are appended to its list in LDS and walked 64 at a
  // time, one per lane, where the layout has room for the lists; otherwise
  // each lane walks its own
  uint16_t* wl = p.plan_scan_off ? reinterpret_cast<uint16_t*>(lds + p.plan_scan_off) + wave * kPlanScanList
                                 : nullptr;
  int pending = 0;   // entries in the wave's list (the same in every lane)
  for (int j0 = tid; j0 < S; j0 += kScan * MT) {
    int32_t xs[kScan];
    uint32_t cand = 0u;
#pragma unroll
    for (int u = 0; u < kScan; ++u) {
      const int j = j0 + u * MT;
      xs[u] = sc[j < S ? j : S - 1];
    }
#pragma unroll
    for (int u = 0; u < kScan; ++u) {
      const int j = j0 + u * MT < S ? j0 + u * MT : S - 1;
      const uint32_t hx = ph.hash(xs[u]);
      const uint32_t w = smp[ph.home(hx)];
      const uint32_t rb = sres[j >> 5] >> (j & 31);
      const bool ok = j0 + u * MT < S && static_cast<uint32_t>(xs[u]) < lim_u && !(rb & 1u) && w != 0u &&
                      ((w & kPlanTag) == ph.tag(hx) || (w & kPlanDisp));
      cand |= ok ? (1u << u) : 0u;
    }
    if (wl) {
#pragma unroll
      for (int u = 0; u < kScan; ++u) {
        const bool c = (cand >> u) & 1u;
        const uint64_t mk = __ballot(c);
        if (c) wl[pending + bits_below(mk)] = static_cast<uint16_t>(j0 + u * MT);
        pending += __popcll(mk);
        if (pending >= 64) {
          wave_sync();
          walk(wl[lane]);
          pending -= 64;
          const int rest = lane < pending ? wl[64 + lane] : 0;
          wave_sync();
          if (lane < pending) wl[lane] = static_cast<uint16_t>(rest);
        }
      }
    } else {
      while (cand) {
        const int u = __builtin_ctz(cand);
        cand &= cand - 1u;
        walk(j0 + u * MT);
      }
    }
  }
  if (wl) {
    wave_sync();
    if (lane < pending) walk(wl[lane]);
  }
  __syncthreads();

  // (2b) early-fetch transfer: the indices whose rows were requested from the
  // host before Stage One (no slot held them when the step began) leave the
  // plan; every position of such an index is written by that fetch
  if (p.early_x) {
    const int ne = p.early_n[r];
    const int32_t* ex = p.early_x + lb;
    for (int k = tid; k < ne; k += MT) {
      uint32_t w = 0u;
      const int hw = plan_lookup(smp, sc, ph, ex[k], &w);
      if (hw >= 0) atomicOr(&smp[hw], kPlanEarly);
    }
    __syncthreads();
  }

  // classify one entry: kind 0 host, 1 resident, 2 repeat (src = source
  // slot), 4 / 5 first / further miss of an early-fetched index, -1 past the
  // list; hw = the map position of the entry's index (returned by value:
  // out-parameters would put these locals on the stack)
  struct Entry {
    int kind, src, hw;
    int2 v;
  };
  auto classify = [&](int e) __attribute__((always_inline)) {
    Entry c{-1, 0, -1, make_int2(0, 0)};
    if (e >= listed) return c;
    c.v = entry(e);
    const int o = c.v.y;
    c.kind = 0;
    if (static_cast<uint32_t>(c.v.x) >= rows_u) return c;
    uint32_t w = 0u;
    c.hw = plan_lookup(smp, sc, ph, c.v.x, &w);
    if (c.hw < 0) return c;
    const int src = plan_slot(w);
    if (w & kPlanEarly) {
      c.kind = src != o ? 5 : 4;   // fetched early; 5 = a further miss of it
    } else if (w & kPlanResident) {
      c.kind = 1;
      c.src = src;
    } else if (src != o) {
      c.kind = 2;
      c.src = src;
    }
    return c;
  };

  // (3) classify the first round's entries (kept for the compaction)
  const Entry first = classify(tid);

  // (4) compact the three lists in transfer-list order; host entries carry
  // their two fan slots, repeats that are in the fan word leave the repeat list
  int n_list[3] = {0, 0, 0}, n_rep = 0;
  for (int e0 = 0, it = 0; e0 < listed; e0 += MT, ++it) {
    Entry c = it == 0 ? first : classify(e0 + tid);
    int2 fan = make_int2(-1, -1);
    if (c.kind == 0 && c.hw >= 0) fan = fan_slots(sfan[c.hw]);
    if (c.kind == 2) {
      ++n_rep;
      const int2 f = fan_slots(sfan[c.hw]);
      if (f.x == c.v.y || f.y == c.v.y) c.kind = 3;   // written by the host copy
    }
    if (c.kind == 5) ++n_rep;             // filled by the early fetch's copy of its index
    const int kind = c.kind;
    uint64_t mk[3];
    int* wc = scnt + (it & 1) * 3 * MW;
#pragma unroll
    for (int k = 0; k < 3; ++k) mk[k] = __ballot(kind == k);
    // host and resident counts share a word (16 bits each: at most MT entries)
    if (lane == 0) {
      wc[wave] = __popcll(mk[0]) | (__popcll(mk[1]) << 16);
      wc[MW + wave] = __popcll(mk[2]);
    }
    __syncthreads();
    const WavePrefix p01 = wave_prefix(wc, MW, wave), p2 = wave_prefix(wc + MW, MW, wave);
    const int before[3] = {p01.before & 0xFFFF, p01.before >> 16, p2.before};
    const int total[3] = {p01.total & 0xFFFF, p01.total >> 16, p2.total};
    if (kind == 0) {
      const size_t at = lb + n_list[0] + before[0] + bits_below(mk[0]);
      p.host_list[at] = c.v;
      p.host_fan[at] = fan;
    } else if (kind == 1) {
      p.res_list[lb + n_list[1] + before[1] + bits_below(mk[1])] = make_int2(c.src, c.v.y);
    } else if (kind == 2) {
      p.rep_list[lb + n_list[2] + before[2] + bits_below(mk[2])] = make_int2(c.src, c.v.y);
    }
#pragma unroll
    for (int k = 0; k < 3; ++k) n_list[k] += total[k];
  }
  n_rep = wave_sum(n_rep);
  if (counts_out) {
    counts_out[0] = n_list[0];
    counts_out[1] = n_list[1];
    counts_out[2] = n_list[2];
  }
  unsigned long long* st = p.stats + static_cast<size_t>(r) * kNumStats;
  if (lane == 0 && n_rep) atomicAdd(&st[kStatDuplicate], static_cast<unsigned long long>(n_rep));
  if (tid == 0) {
    int32_t* pc = p.plan_counts + 3 * static_cast<size_t>(r);
    pc[0] = n_list[0];
    pc[1] = n_list[1];
    pc[2] = n_list[2];
    if (n_list[1]) atomicAdd(&st[kStatResident], static_cast<unsigned long long>(n_list[1]));
  }
}

// Stage One for request r (Algorithm 4's token loop) in workgroup-owned LDS.
// After each token with misses, publish(r, first, count) is called by every
// thread once the token's transfer-list entries are written (a no-op for the
// plain matching kernel).  SPT is the number of lifetimes a thread owns
// (S / NT, at least 1) when known at compile time, so that the loops over them
// unroll without scalar conditions; 0 takes it from S at run time.
template <int IPT, int NT, int SPT, typename Publish>
__device__ __forceinline__ void match_request(const MatchParams& p, const int r, unsigned char* lds,
                              Publish& publish, int* plan_counts = nullptr) {
  constexpr int MT = NT, MW = NT / 64;
  static_assert(NT % 64 == 0 && NT <= kMatchThreads, "whole waves, at most the largest workgroup");
  // probe and chain rounds whose LDS reads are issued together: all R + 1 = 4
  // of the default retry count with up to two indices per thread, one at a
  // time with more (whose registers would otherwise spill)
  constexpr int kChainBatch = IPT <= 2 ? 4 : 1;
  // with two or more lifetimes per thread the table has exactly SPT * NT slots
  const int S = SPT >= 2 ? SPT * MT : p.S, K = p.K, R = p.R;
  const uint32_t smask = static_cast<uint32_t>(S - 1);
  const Word W{static_cast<uint32_t>(p.m), smask, p.f_mask};
  int32_t* sc = reinterpret_cast<int32_t*>(lds);
  uint32_t* smap = reinterpret_cast<uint32_t*>(lds + 4 * static_cast<size_t>(S));
  int8_t* slife = reinterpret_cast<int8_t*>(lds + 8 * static_cast<size_t>(S));
  int32_t* somiss = reinterpret_cast<int32_t*>(lds + 8 * static_cast<size_t>(S) + align16(S));
  int32_t* smx = somiss + K;                 // [K] dense miss indices
  int32_t* smp = smx + K;                    // [K] dense miss positions
  int32_t* swc = smp + K;                    // [2][IPT][MW] miss counts per wave
  int32_t* sdead = swc + 2 * kMaxIPT * MW;   // [MW] dead counts per wave
  int32_t* sred = sdead + MW;                // [4] rotating reduction slots
  // the step's transfer list as slots, kept for the Stage Two plan
  uint16_t* slist = reinterpret_cast<uint16_t*>(lds + p.plan_list_off);

  const int tid = threadIdx.x;
  const int wave = wave_id();
  const int lane = lane_id();

  // the first token's indices are requested before the table, so the two
  // memory latencies overlap
  int32_t xv[IPT];
  {
    const int32_t* xg = p.topk + static_cast<size_t>(r) * p.n_q * K;
#pragma unroll
    for (int u = 0; u < IPT; ++u) {
      const int i = u * MT + tid;
      xv[u] = i < K ? xg[i] : 0;
    }
  }

  int32_t* gc = p.table_c + static_cast<size_t>(r) * S;
  uint32_t* gq = p.table_q + static_cast<size_t>(r) * S;
  // stage-in: 16-byte loads of 4 entries, the loads of two blocks issued
  // before their LDS stores (all of a thread's blocks when the lifetimes per
  // thread are known: S = SPT * NT).  The first token's decay of every
  // lifetime (the global pre-decay of Algorithm 1) is applied as the
  // lifetimes come in.
  auto stage_block = [&](int b, const i32x4 c, const u32x4 q) __attribute__((always_inline)) {
    reinterpret_cast<i32x4*>(sc)[b] = c;
    reinterpret_cast<u32x4*>(smap)[b] = u32x4{W.staged(q.x), W.staged(q.y), W.staged(q.z), W.staged(q.w)};
    reinterpret_cast<uint32_t*>(slife)[b] =
        Own::decay1((q.x >> 24) | ((q.y >> 24) << 8) | ((q.z >> 24) << 16) | (q.w & 0xFF000000u));
  };
  // with the lifetimes per thread known, a thread keeps the index blocks it
  // staged in, and the write back stores only those that changed
  i32x4 cb[SPT >= 4 ? SPT / 4 : 1];
  if constexpr (SPT >= 4) {
    constexpr int NB = SPT / 4;
    u32x4 qb[NB];
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      cb[k] = reinterpret_cast<const i32x4*>(gc)[tid + k * MT];
      qb[k] = reinterpret_cast<const u32x4*>(gq)[tid + k * MT];
    }
#pragma unroll
    for (int k = 0; k < NB; ++k) stage_block(tid + k * MT, cb[k], qb[k]);
  } else if ((S & (4 * MT - 1)) == 0) {
    for (int b = tid; b < S / 4; b += 2 * MT) {
      const i32x4 c0 = reinterpret_cast<const i32x4*>(gc)[b];
      const u32x4 q0 = reinterpret_cast<const u32x4*>(gq)[b];
      const bool two = b + MT < S / 4;
      i32x4 c1 = 0;
      u32x4 q1 = 0u;
      if (two) {
        c1 = reinterpret_cast<const i32x4*>(gc)[b + MT];
        q1 = reinterpret_cast<const u32x4*>(gq)[b + MT];
      }
      stage_block(b, c0, q0);
      if (two) stage_block(b + MT, c1, q1);
    }
  } else {
    for (int j = tid; j < S; j += MT) {
      const uint32_t q = gq[j];
      sc[j] = gc[j];
      smap[j] = W.staged(q);
      const int life = static_cast<int8_t>(q >> 24);
      slife[j] = static_cast<int8_t>(life > -1 ? life - 1 : -1);
    }
  }
  if (tid < 4) sred[tid] = 0;

  // lifetimes owned by this thread: [j0, j0 + spt) if it owns any (tid < S).
  // spt is uniform, so the Own loops branch on scalars; only tables smaller
  // than a workgroup leave threads without lifetimes.
  const int spt = SPT > 0 ? SPT : (S >= MT ? S / MT : 1);
  const bool owns = tid < S;
  const int j0 = owns ? tid * spt : 0;
  const int64_t rows_r = p.rows[r];
  const int64_t n_verified = p.verified ? p.verified[r] : INT64_MAX;
  // 32-bit forms of the bounds: x is a valid index when (uint32)x < rows_u
  // (negative x fail), a cached index lies below the verified length when
  // (uint32)x < ver_u, and c >= N (speculative invalidation) is decided on
  // int32 c with the two out-of-range cases of N taken apart
  auto clamp_u = [](int64_t v) { return static_cast<uint32_t>(v <= 0 ? 0 : (v > 0x80000000ll ? 0x80000000ll : v)); };
  const uint32_t rows_u = clamp_u(rows_r);
  const uint32_t lim_u = rows_u < clamp_u(n_verified) ? rows_u : clamp_u(n_verified);
  const bool inv_all = n_verified <= static_cast<int64_t>(INT32_MIN);
  const bool inv_none = n_verified > static_cast<int64_t>(INT32_MAX);
  const int32_t ver32 = (inv_all || inv_none) ? 0 : static_cast<int32_t>(n_verified);
  auto invalidated = [&](int32_t c) { return inv_all || (!inv_none && c >= ver32); };
  const uint32_t a1 = p.a1, a2 = p.a2, fmask = p.f_mask;
  // (a x) mod S from the low 24 bits of a mod S and of x (S divides 2^24):
  // the full-rate 24-bit multiply gives the low 32 bits of their product
  const uint32_t a1m = a1 & smask, a2m = a2 & smask;
  const int m = p.m, L = p.L;

  int st_hits = 0, st_miss = 0, st_exh = 0, st_col = 0, st_rev = 0, st_bad = 0;
  int step_decays = 0;
  int listed = 0;
  int red_it = 0;
  // bids of the previous token, checked after the next barrier
  uint32_t bid_h[IPT], bid_v[IPT];
#pragma unroll
  for (int u = 0; u < IPT; ++u) {
    bid_v[u] = 0u;
    bid_h[u] = 0u;
  }

  __syncthreads();

  // the first token's global pre-decay (every lifetime down by one) was
  // applied by the stage-in
  for (int g = 0; g < p.n_q; ++g) {
    const size_t row = static_cast<size_t>(r) * p.n_q + g;
    int32_t* og = p.slots_out + row * K;
    int32_t* wc = swc + (g & 1) * kMaxIPT * MW;

    // ---- A: probe, refresh hits, rank misses ------------------------------
    uint32_t hh[IPT], dd[IPT];
    int oo[IPT];
    bool act[IPT], found[IPT];
#pragma unroll
    for (int u = 0; u < IPT; ++u) {
      act[u] = u * MT + tid < K;
      const uint32_t ux = static_cast<uint32_t>(xv[u]);
      hh[u] = mul24(a1m, ux) & smask;          // initial bucket (Eq. 9)
      dd[u] = (mul24(a2m, ux) & smask) | 1u;   // odd stride (Eq. 9)
      found[u] = false;
      oo[u] = 0;
      if (act[u] && static_cast<uint32_t>(xv[u]) >= rows_u) st_bad++;
    }
    // the buckets of kChainBatch consecutive rounds depend only on the index,
    // so their words and then their slots' ids are read together: two LDS
    // round trips per batch instead of two per round; the first round whose
    // slot holds the index decides, as in the round-by-round probe
    for (int rd0 = 0; rd0 <= R; rd0 += kChainBatch) {
      // every round of the batch is read, also rounds past R (their buckets
      // are valid addresses and their words are ignored), so the reads carry
      // no conditions and go out together
      uint32_t qw[IPT][kChainBatch];
      int32_t cv[IPT][kChainBatch];
#pragma unroll
      for (int u = 0; u < IPT; ++u)
#pragma unroll
        for (int b = 0; b < kChainBatch; ++b) qw[u][b] = smap[(hh[u] + b * dd[u]) & smask];
#pragma unroll
      for (int u = 0; u < IPT; ++u)
#pragma unroll
        for (int b = 0; b < kChainBatch; ++b) cv[u][b] = sc[W.slot(qw[u][b])];   // Eq. 10
      // the decision takes selects and bitwise tests only: a branch on a
      // round's test would let the compiler move that round's reads behind it
      bool pending = false;
#pragma unroll
      for (int u = 0; u < IPT; ++u) {
        // the first round of the batch whose slot holds the index
        uint32_t wf = 0u;
        bool hit = false;
#pragma unroll
        for (int b = kChainBatch - 1; b >= 0; --b) {
          const bool m = (cv[u][b] == xv[u]) & (rd0 + b <= R);
          hit = hit | m;
          wf = m ? qw[u][b] : wf;
        }
        const bool open = act[u] & !found[u];
        oo[u] = (open & hit) ? static_cast<int>(W.slot(wf)) : oo[u];
        found[u] = found[u] | (open & hit);
        // unresolved probes advance (Eq. 11)
        hh[u] = (open & !hit) ? (hh[u] + kChainBatch * dd[u]) & smask : hh[u];
        pending = pending | (open & !hit & (rd0 + kChainBatch <= R));
      }
      if (!__ballot(pending)) break;
    }
    int rank[IPT];
    // per-wave miss counts, two indices per word (16 bits each)
    int packed[2] = {0, 0};
#pragma unroll
    for (int u = 0; u < IPT; ++u) {
      const int i = u * MT + tid;
      if (found[u]) {
        if (slife[oo[u]] < 0) st_rev++;
        slife[oo[u]] = static_cast<int8_t>(L);   // refresh the hit slot
        og[i] = oo[u];                           // a hit's output slot
        st_hits++;
      }
      if (p.hit_mask && act[u]) p.hit_mask[row * K + i] = found[u] ? 1 : 0;
      const uint64_t mm = __ballot(act[u] && !found[u]);
      packed[u >> 1] |= __popcll(mm) << (16 * (u & 1));
      rank[u] = bits_below(mm);
    }
    if (lane == 0) {
      wc[wave] = packed[0];
      if (IPT > 2) wc[MW + wave] = packed[1];
    }
    // installs of the previous token that lost their bucket
#pragma unroll
    for (int u = 0; u < IPT; ++u)
      if (bid_v[u]) {
        if (smap[bid_h[u]] != bid_v[u]) st_col++;
        bid_v[u] = 0u;
      }
    __syncthreads();

    // ---- B: classify, compact misses, count dead slots ---------------------
    int n_g = 0;
    {
      const WavePrefix pf[2] = {wave_prefix(wc, MW, wave),
                                IPT > 2 ? wave_prefix(wc + MW, MW, wave) : WavePrefix{0, 0}};
#pragma unroll
      for (int u = 0; u < IPT; ++u) {
        const int sh = 16 * (u & 1);
        rank[u] += n_g + ((pf[u >> 1].before >> sh) & 0xFFFF);
        n_g += (pf[u >> 1].total >> sh) & 0xFFFF;
      }
    }
    if (tid == 0) {
      p.miss_counts[row] = n_g;
      st_miss += n_g;
    }
#pragma unroll
    for (int u = 0; u < IPT; ++u)
      if (act[u] && !found[u]) {
        smx[rank[u]] = xv[u];
        smp[rank[u]] = u * MT + tid;
      }
    Own own;
    if (owns) own.load(slife, j0, spt);
    int dcnt = owns ? own.count_below(0, spt) : 0;
    int incl = wave_inclusive_scan(dcnt, lane);
    if (lane == 63) sdead[wave] = incl;
    // prefetch the next token's indices
    if (g + 1 < p.n_q) {
      const int32_t* xg = p.topk + (row + 1) * K;
#pragma unroll
      for (int u = 0; u < IPT; ++u) {
        const int i = u * MT + tid;
        xv[u] = i < K ? xg[i] : 0;
      }
    }
    __syncthreads();

    if (n_g > 0) {
      // ---- C: enough dead slots (decay loop of Algorithm 1), CollectDead --
      const WavePrefix pd = wave_prefix(sdead, MW, wave);
      const int dead = pd.total;
      int wbase = pd.before;
      if (dead < n_g) {
        // smallest k with #{lifetime_j < k} >= n_g; k = L + 1 always suffices
        int kstar = 1;
        for (int k = 1;; ++k) {
          const int cnt = wave_sum(owns ? own.count_below(k, spt) : 0);
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
        if (owns) {
          own.decay(kstar, spt);
          own.store(slife, j0, spt);
        }
        step_decays += kstar;
        dcnt = owns ? own.count_below(0, spt) : 0;
        incl = wave_inclusive_scan(dcnt, lane);
        if (lane == 63) sdead[wave] = incl;   // every wave read sdead before the loop's barrier
        __syncthreads();
        wbase = wave_prefix(sdead, MW, wave).before;
      }
      int drank = wbase + incl - dcnt;
      if (drank < n_g) {
#pragma unroll
        for (int e = 0; e < kMaxSPT; ++e)
          if (owns && e < spt && own.get(e) < 0 && drank < n_g) somiss[drank++] = j0 + e;
      }
      __syncthreads();

      // ---- D: reusable chains on the pre-write table (Algorithm 2) ---------
      int32_t mt[IPT], mo[IPT], mp[IPT];
      uint32_t mh[IPT], md[IPT];
      bool mact[IPT], mv[IPT];
#pragma unroll
      for (int u = 0; u < IPT; ++u) {
        // the misses are ranks 0..n_g-1, one per lane: reads are issued for
        // whole waves (a lane past n_g reads a valid entry and ignores it)
        const int k = u * MT + tid;
        const int kr = k < n_g ? k : 0;
        mact[u] = k < n_g;
        mv[u] = false;
        mt[u] = 0;
        mp[u] = 0;
        mo[u] = 0;
        if (u * MT + wave * 64 < n_g) {   // the wave holds a miss
          mt[u] = smx[kr];
          mp[u] = smp[kr];
          mo[u] = somiss[kr] & static_cast<int>(smask);
        }
        const uint32_t ux = static_cast<uint32_t>(mt[u]);
        mh[u] = mul24(a1m, ux) & smask;
        md[u] = (mul24(a2m, ux) & smask) | 1u;
      }
      // a batch of rounds at a time, as in the probe: every word of the batch,
      // then the lifetime and id of each word's slot, then the first
      // reusable bucket in round order
      for (int rd0 = 0; rd0 <= R; rd0 += kChainBatch) {
        uint32_t qw[IPT][kChainBatch];
        int lf[IPT][kChainBatch];
        int32_t cv[IPT][kChainBatch];
        // every lane of a wave that holds a miss reads every round of the
        // batch (the buckets and slots are valid whatever the lane holds;
        // rounds past R are read and ignored), so the reads go out together
#pragma unroll
        for (int u = 0; u < IPT; ++u) {
#pragma unroll
          for (int b = 0; b < kChainBatch; ++b) {
            qw[u][b] = 0u;
            lf[u][b] = 0;
            cv[u][b] = 0;
          }
          if (u * MT + wave * 64 < n_g) {
#pragma unroll
            for (int b = 0; b < kChainBatch; ++b) qw[u][b] = smap[(mh[u] + b * md[u]) & smask];
          }
        }
#pragma unroll
        for (int u = 0; u < IPT; ++u)
          if (u * MT + wave * 64 < n_g) {
#pragma unroll
            for (int b = 0; b < kChainBatch; ++b) {
              const uint32_t o2 = W.slot(qw[u][b]);
              lf[u][b] = slife[o2];
              cv[u][b] = sc[o2];
            }
          }
        bool pending = false;
#pragma unroll
        for (int u = 0; u < IPT; ++u) {
          if (!mact[u] || mv[u]) continue;
          int first = -1;
#pragma unroll
          for (int b = kChainBatch - 1; b >= 0; --b)
            // reusable (Eq. 4): invalid, pointed slot inactive, or stale fingerprint
            if (rd0 + b <= R && (W.invalid(qw[u][b]) || lf[u][b] < 0 ||
                                 W.fp(qw[u][b]) != (static_cast<uint32_t>(cv[u][b]) & fmask)))
              first = b;
          if (first >= 0) {
            mv[u] = true;
            mh[u] = (mh[u] + mul24v(static_cast<uint32_t>(first), md[u])) & smask;
          } else {
            mh[u] = (mh[u] + kChainBatch * md[u]) & smask;
            pending = pending || rd0 + kChainBatch <= R;
          }
        }
        if (!__ballot(pending)) break;
      }
      __syncthreads();

      // ---- E: take the slots, bid for buckets, emit outputs ---------------
      const size_t lbase = static_cast<size_t>(r) * p.n_q * K + listed;
#pragma unroll
      for (int u = 0; u < IPT; ++u) {
        if (!mact[u]) continue;
        const int k = u * MT + tid;
        sc[mo[u]] = mt[u];
        slife[mo[u]] = static_cast<int8_t>(L);
        og[mp[u]] = mo[u];                                   // a miss's output slot
        p.miss_list[lbase + k] = make_int2(mt[u], mo[u]);
        if (p.plan_list_off > 0) slist[listed + k] = static_cast<uint16_t>(mo[u]);
        if (mv[u]) {
          const uint32_t bid = kBid | (static_cast<uint32_t>(g) << 24) |
                               (static_cast<uint32_t>(mo[u]) << (23 - m)) |
                               (static_cast<uint32_t>(mt[u]) & fmask);
          atomicMax(&smap[mh[u]], bid);
          bid_h[u] = mh[u];
          bid_v[u] = bid;
        } else {
          st_exh++;
        }
      }
      publish(r, listed, n_g);
      listed += n_g;
      __syncthreads();
    }
  }

  // installs of the last token that lost their bucket: of the bids it made,
  // all but one per bucket it bid for (the write back counts the buckets
  // whose word is a bid of the last token; the sum over the workgroup is what
  // matters, not which thread counts)
#pragma unroll
  for (int u = 0; u < IPT; ++u)
    if (bid_v[u]) st_col++;
  const uint32_t last_bid = kBid | (static_cast<uint32_t>(p.n_q - 1) << 24);
  auto last_token_bid = [&](uint32_t w) { return (w & 0xFF000000u) == last_bid ? 1 : 0; };

  // every slot of the request's O is written: an early-fetch worker may now
  // copy rows straight into them (each wave's stores are made visible at
  // device scope before the flag)
  if (p.early_done) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (tid == 0) __hip_atomic_store(p.early_done + r, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  }

  // End of step: speculative invalidation fused into the write back.  With a
  // Stage Two plan to follow, each thread also clears the plan's LDS words
  // that it has just read (bucket words and lifetimes), and the threads share
  // the rest of the plan's words, which the write back does not read.
  const bool plan = p.plan_words > 0;
  int st_inv = 0;
  auto write_block = [&](int b, i32x4 c, bool store_c) __attribute__((always_inline)) {
      const u32x4 m = reinterpret_cast<const u32x4*>(smap)[b];
      const uint32_t l = reinterpret_cast<const uint32_t*>(slife)[b];
      if (plan) {
        reinterpret_cast<u32x4*>(smap)[b] = 0u;
        reinterpret_cast<uint32_t*>(slife)[b] = 0u;
      }
      st_col -= last_token_bid(m.x) + last_token_bid(m.y) + last_token_bid(m.z) + last_token_bid(m.w);
      u32x4 q;
      q.x = (l << 24) | W.canonical(m.x);
      q.y = ((l << 16) & 0xFF000000u) | W.canonical(m.y);
      q.z = ((l << 8) & 0xFF000000u) | W.canonical(m.z);
      q.w = (l & 0xFF000000u) | W.canonical(m.w);
      if (store_c) reinterpret_cast<i32x4*>(gc)[b] = c;
      reinterpret_cast<u32x4*>(gq)[b] = q;
  };
  if constexpr (SPT >= 4) {
#pragma unroll
    for (int k = 0; k < SPT / 4; ++k) {
      const int b = tid + k * MT;
      i32x4 c = reinterpret_cast<const i32x4*>(sc)[b];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (invalidated(c[e])) {
          c[e] = -1;
          st_inv++;
        }
      const bool same = c.x == cb[k].x && c.y == cb[k].y && c.z == cb[k].z && c.w == cb[k].w;
      write_block(b, c, !same);
    }
  } else if ((S & (4 * MT - 1)) == 0) {
    // four entries per 16-byte store
    for (int b = tid; b < S / 4; b += MT) {
      i32x4 c = reinterpret_cast<const i32x4*>(sc)[b];
      const u32x4 m = reinterpret_cast<const u32x4*>(smap)[b];
      const uint32_t l = reinterpret_cast<const uint32_t*>(slife)[b];
      if (plan) {
        reinterpret_cast<u32x4*>(smap)[b] = 0u;
        reinterpret_cast<uint32_t*>(slife)[b] = 0u;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (invalidated(c[e])) {
          c[e] = -1;
          st_inv++;
        }
      st_col -= last_token_bid(m.x) + last_token_bid(m.y) + last_token_bid(m.z) + last_token_bid(m.w);
      u32x4 q;
      q.x = (l << 24) | W.canonical(m.x);
      q.y = ((l << 16) & 0xFF000000u) | W.canonical(m.y);
      q.z = ((l << 8) & 0xFF000000u) | W.canonical(m.z);
      q.w = (l & 0xFF000000u) | W.canonical(m.w);
      reinterpret_cast<i32x4*>(gc)[b] = c;
      reinterpret_cast<u32x4*>(gq)[b] = q;
    }
  } else {
    for (int j = tid; j < S; j += MT) {
      int32_t c = sc[j];
      const uint32_t m = smap[j];
      const uint8_t l = static_cast<uint8_t>(slife[j]);
      if (plan) {
        smap[j] = 0u;
        slife[j] = 0;
      }
      if (invalidated(c)) {
        c = -1;
        st_inv++;
      }
      st_col -= last_token_bid(m);
      gc[j] = c;
      gq[j] = (static_cast<uint32_t>(l) << 24) | W.canonical(m);
    }
  }
  if (plan) {
    // plan words past the bucket words and lifetimes (16-byte aligned ends)
    const size_t from = 8 * static_cast<size_t>(S) + align16(S);
    const size_t to = align16(4 * static_cast<size_t>(S)) + 4 * plan_state_words(S, p.plan_words);
    for (size_t o = from + 16 * static_cast<size_t>(tid); o < to; o += 16 * static_cast<size_t>(MT))
      *reinterpret_cast<u32x4*>(lds + o) = 0u;
  }

  // counters: each wave adds its sums with atomics that return nothing.  Two
  // counters share a wave sum, 16 bits each: a thread's counts are at most
  // IPT * n_q (<= 508) and its collision count at least -spt (the last
  // token's winning buckets among the words it wrote back), which the bias
  // spt lifts to zero, so every sum stays below 2^16.
  {
    unsigned long long* st = p.stats + static_cast<size_t>(r) * kNumStats;
    const int s0 = wave_sum(st_hits | (st_exh << 16));
    const int s1 = wave_sum(st_rev | (st_bad << 16));
    const int s2 = wave_sum((st_col + spt) | (st_inv << 16));
    const int vals[6] = {s0 & 0xFFFF, s0 >> 16, (s2 & 0xFFFF) - 64 * spt, s1 & 0xFFFF, s2 >> 16, s1 >> 16};
    const StatIndex idx[6] = {kStatHits, kStatLostExhausted, kStatLostCollision,
                              kStatRevivals, kStatInvalidations, kStatBadIndices};
    if (lane == 0) {
#pragma unroll
      for (int k = 0; k < 6; ++k)
        if (vals[k]) atomicAdd(&st[idx[k]], static_cast<unsigned long long>(static_cast<long long>(vals[k])));
    }
    if (tid == 0) {
      if (st_miss) atomicAdd(&st[kStatMisses], static_cast<unsigned long long>(st_miss));
      if (step_decays) {
        atomicAdd(&st[kStatAllocDecays], static_cast<unsigned long long>(step_decays));
        atomicMax(&st[kStatMaxStepDecays], static_cast<unsigned long long>(step_decays));
      }
    }
  }
  if (plan) {
    __syncthreads();   // the plan's words are clear
    plan_request<NT>(p, r, lds, listed, rows_u, lim_u, plan_counts);
  }
}

}  // namespace
}  // namespace avsg
