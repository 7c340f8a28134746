// Workgroup-wide exact top-m selection (radix select on order-preserving keys).
//
// Selects the `need` elements of a source that rank first by (key descending,
// position ascending) and hands each selected position to put(slot, pos), with
// consecutive slots counted from sh.emitted (set by the caller).
//
// With BUCKET (for sets whose scores straddle zero and crowd a few exponents,
// where radix digits taken from the top key bits pile most elements into a
// handful of bins and the histogram atomics on one LDS address serialise):
//   1 the key range [kmin, kmax] (one reduction);
//   2 a 256-bin histogram of the VALUE, linearly bucketed over that range
//     (a monotone map, so buckets keep the order), finds the bucket b* that
//     holds the need-th element.
// Then (over b*, or over all elements without BUCKET):
//   3 the key bits shared by every element are skipped (AND / OR reduction)
//     and 8-bit radix passes over the rest find the threshold key;
//   4 if the threshold key is shared by more elements than remain to be taken,
//     4 passes over the positions of the tied elements pick the lowest ones;
//   5 every element above the threshold (and the chosen ties) is emitted.
// Positions must be distinct non-negative int32.
//
// A source provides visit(f), calling f(key, pos) for each of the calling
// thread's elements; every thread of the workgroup calls it.  Sources may keep
// their elements in registers, LDS or global memory.
#pragma once

#include "device_common.h"
#include "dpp.h"

namespace pivot {

// Appends the calling lanes whose `take` is set through ONE atomic on the LDS
// counter per wave (not one per lane: lanes of a wave appending to the same
// counter would serialise on it); f(slot) runs on the taking lanes.  Must be
// reached by all lanes of the wave that may take.
template <class F>
__device__ __forceinline__ void wave_append(bool take, int32_t* counter, F f) {
  const uint64_t bal = __ballot(take);
  if (bal == 0) return;
  const int leader = __ffsll((unsigned long long)bal) - 1;
  int base = 0;
  if ((int)(threadIdx.x & 63) == leader) base = atomicAdd(counter, (int)__popcll((unsigned long long)bal));
  base = __shfl(base, leader, 64);
  if (take)
    f(base + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u)));
}

struct SelectShared {
  uint32_t hist[256];
  uint32_t wsum[16];
  uint32_t wand[16], wor[16];
  uint32_t digit, before, equal;
  int32_t emitted;
};

// Inclusive prefix sum over the 64 lanes of a wave: row shifts within each
// row of 16 lanes, then row broadcasts of lanes 15 and 31 (DPP: no LDS round
// trips, unlike a shuffle ladder).
__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, true);   // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, true);   // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, true);   // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, true);   // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);  // row_bcast:15 -> rows 1, 3
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);  // row_bcast:31 -> rows 2, 3
  return x;
}

// Find the digit d (of `bins`) where the running count crosses `rem`, scanning
// digits downwards (desc) or upwards (!desc).  Threads take the digits in scan
// order, bins/THREADS consecutive ones each (one, or none, when bins is
// smaller): with DESC thread 0 holds the highest digits, so one ascending
// scan over the lanes and waves serves both directions.  Writes sh.digit,
// sh.before (count strictly before d in scan order) and sh.equal (count at
// d).  Contains workgroup barriers.
template <int THREADS, bool DESC>
__device__ __forceinline__ void find_digit(const uint32_t* hist, SelectShared& sh, uint32_t rem, int bins) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int per = bins / THREADS;  // bins is a multiple of THREADS, or smaller
  const int cnt = per > 0 ? per : (tid < bins ? 1 : 0);
  const int first = per > 0 ? (DESC ? bins - 1 - per * tid : per * tid) : (DESC ? bins - 1 - tid : tid);
  auto digit = [&](int k) { return DESC ? first - k : first + k; };  // k-th digit of this thread in scan order
  uint32_t tot = 0;
  for (int k = 0; k < cnt; ++k) tot += hist[digit(k)];
  const uint32_t s = wave_incl_sum(tot);
  if (lane == 63) sh.wsum[wv] = s;
  __syncthreads();
  uint32_t before = s - tot;
  for (int w = 0; w < wv; ++w) before += sh.wsum[w];
  for (int k = 0; k < cnt; ++k) {
    const uint32_t h = hist[digit(k)];
    if (before < rem && rem <= before + h) {
      sh.digit = digit(k);
      sh.before = before;
      sh.equal = h;
    }
    before += h;
  }
  __syncthreads();
}

// Inverse of float_key (zero comes back as +0).
__device__ __forceinline__ float key_float(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// Workgroup reduction of (min, max) or (and, or) pairs through sh.wand / sh.wor.
template <int THREADS, bool MINMAX>
__device__ __forceinline__ void block_pair_reduce(uint32_t& a, uint32_t& o, SelectShared& sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  a = wave_total_at63(a, ~0u, [](uint32_t x, uint32_t y) { return MINMAX ? min(x, y) : (x & y); });
  o = wave_total_at63(o, 0u, [](uint32_t x, uint32_t y) { return MINMAX ? max(x, y) : (x | y); });
  if (lane == 63) {
    sh.wand[wv] = a;
    sh.wor[wv] = o;
  }
  __syncthreads();
  for (int w = 0; w < THREADS / 64; ++w) {
    a = MINMAX ? min(a, sh.wand[w]) : (a & sh.wand[w]);
    o = MINMAX ? max(o, sh.wor[w]) : (o | sh.wor[w]);
  }
  __syncthreads();
}

template <int THREADS, bool BUCKET, class Src, class Put>
__device__ void block_select(const Src& src, uint32_t need, SelectShared& sh, Put put) {
  const int tid = threadIdx.x;
  if (need == 0) return;
  uint32_t kmin = ~0u, kmax = 0u;
  if constexpr (BUCKET) {
    src.visit([&](uint32_t key, int32_t) {
      kmin = min(kmin, key);
      kmax = max(kmax, key);
    });
    block_pair_reduce<THREADS, true>(kmin, kmax, sh);
  }
  // value buckets: bucket(key) is monotone in the key
  const float fmin = key_float(kmin);
  const float scale = 256.0f / (key_float(kmax) - fmin);
  const bool bucketed = BUCKET && kmin != kmax && scale > 0.0f && scale < __builtin_inff();
  auto bucket = [&](uint32_t key) { return min(255, (int)((key_float(key) - fmin) * scale)); };
  uint32_t rem = need, equal = 0xFFFFFFFFu;  // equal: keys at the threshold (unknown: take the tie passes)
  int bsel = 0;
  if (bucketed) {
    for (int i = tid; i < 256; i += THREADS) sh.hist[i] = 0;
    __syncthreads();
    src.visit([&](uint32_t key, int32_t) { atomicAdd(&sh.hist[bucket(key)], 1u); });
    __syncthreads();
    find_digit<THREADS, true>(sh.hist, sh, rem, 256);
    bsel = (int)sh.digit;
    rem -= sh.before;
    equal = sh.equal;
    __syncthreads();
  }
  auto member = [&](uint32_t key) { return !bucketed || bucket(key) == bsel; };
  // bits shared by the members of the bucket
  uint32_t a = ~0u, o = 0u;
  src.visit([&](uint32_t key, int32_t) {
    if (member(key)) {
      a &= key;
      o |= key;
    }
  });
  block_pair_reduce<THREADS, false>(a, o, sh);
  const uint32_t diff = a ^ o;
  int low = diff ? 32 - __clz(diff) : 0;  // key bits [0, low) still to resolve
  uint32_t fixed = low == 32 ? 0u : ~((1u << low) - 1u);
  uint32_t prefix = a & fixed;
  while (low > 0) {
    const int w = low < 8 ? low : 8, shift = low - w;
    const uint32_t dmask = (1u << w) - 1u;
    for (int i = tid; i < 256; i += THREADS) sh.hist[i] = 0;
    __syncthreads();
    src.visit([&](uint32_t key, int32_t) {
      if ((key & fixed) == prefix && member(key)) atomicAdd(&sh.hist[(key >> shift) & dmask], 1u);
    });
    __syncthreads();
    find_digit<THREADS, true>(sh.hist, sh, rem, 256);
    rem -= sh.before;
    equal = sh.equal;
    prefix |= sh.digit << shift;
    fixed |= dmask << shift;
    low = shift;
    __syncthreads();
  }
  const uint32_t T = prefix;
  const bool all_ties = (rem == equal);
  uint32_t ipref = 0, imask = 0;
  if (!all_ties) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += THREADS) sh.hist[i] = 0;
      __syncthreads();
      src.visit([&](uint32_t key, int32_t pos) {
        const uint32_t p = (uint32_t)pos;
        if (key == T && (p & imask) == ipref) atomicAdd(&sh.hist[(p >> shift) & 255u], 1u);
      });
      __syncthreads();
      find_digit<THREADS, false>(sh.hist, sh, rem, 256);
      rem -= sh.before;
      ipref |= sh.digit << shift;
      imask |= 255u << shift;
      __syncthreads();
    }
  }
  src.visit([&](uint32_t key, int32_t pos) {
    const bool take = key > T || (key == T && (all_ties || (uint32_t)pos <= ipref));
    wave_append(take, &sh.emitted, [&](int slot) { put(slot, pos); });
  });
  __syncthreads();
}

// Fast exact top-`need` of a source whose keys spread over a range of values
// (a candidate set): one reduction for the key range, one pass over an
// NB-bin histogram of the value bucketed linearly over that range (a
// monotone map), and one pass that emits every element of the buckets above
// the one holding the need-th element and lists that bucket's members in
// LDS; each listed member then counts the members ranking above it (key
// descending, position ascending).  Returns false, having emitted nothing,
// when the keys are all equal or the bucket holds more than kBucketList
// elements; the caller then uses block_select().  NB: about one bin per
// element keeps the bucket short for long-tailed sets.
// hist: NB LDS words; lkey / lpos: kBucketList LDS entries (they may alias
// hist: the histogram is dead by the time the list is written); lcount: an
// LDS word.
constexpr int kBucketList = 256;

// bucket_select's emission pass: elements of buckets above bsel go out
// through put (one LDS atomic per wave and element, wave_append), members of
// bucket bsel go to list(key, pos).  Sources with a faster form overload it
// (found by argument-dependent lookup).
template <class Src, class Bk, class Put, class List>
__device__ __forceinline__ void emit_bucket(const Src& src, Bk bucket, int bsel, SelectShared& sh, Put put,
                                            List list) {
  src.visit([&](uint32_t key, int32_t pos) {
    const int bk = bucket(key);
    wave_append(bk > bsel, &sh.emitted, [&](int slot) { put(slot, pos); });
    if (bk == bsel) list(key, pos);
  });
}

// bucket_select's last step: the in_b elements listed in LDS (lkey, lpos)
// share the bucket holding the need-th element, and rem of them are still
// wanted.  Each listed element's rank is the number of listed elements
// ranking above it (key descending, position ascending); those with
// rank < rem go out through put.  Ends with a workgroup barrier.
template <int THREADS, class Put>
__device__ __forceinline__ void rank_listed(uint32_t in_b, uint32_t rem, const uint32_t* lkey, const int32_t* lpos,
                                            SelectShared& sh, Put put) {
  const int tid = threadIdx.x;
  // rank of each listed member = members ranking above it; G threads share a
  // member (THREADS >= kBucketList >= in_b), each counting over a part of the
  // list with 8 loads issued before the compares, then summed across lanes
  constexpr int G = THREADS / kBucketList;
  static_assert(G >= 1 && (G & (G - 1)) == 0 && G <= 64, "threads per listed member");
  {
    const int t = tid / G, part = tid % G;
    const bool mine = t < (int)in_b;
    uint32_t key = 0, rank = 0;
    int32_t pos = 0;
    if (mine) {
      key = lkey[t];
      pos = lpos[t];
      const int span = ((int)in_b + G - 1) / G;
      const int u1 = min((int)in_b, (part + 1) * span);
      int u = part * span;
      for (; u + 8 <= u1; u += 8) {
        uint32_t ku[8];
        int32_t pu[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          ku[j] = lkey[u + j];
          pu[j] = lpos[u + j];
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) rank += (ku[j] > key) || (ku[j] == key && pu[j] < pos);
      }
      for (; u < u1; ++u) {
        const uint32_t ku = lkey[u];
        rank += (ku > key) || (ku == key && lpos[u] < pos);
      }
    }
#pragma unroll
    for (int o = 1; o < G; o <<= 1) rank += __shfl_xor(rank, o, 64);
    wave_append(mine && part == 0 && rank < rem, &sh.emitted, [&](int slot) { put(slot, pos); });
  }
  __syncthreads();
}

template <int THREADS, int NB = 4096, class Src, class Put>
__device__ bool bucket_select(const Src& src, uint32_t need, uint32_t* hist, uint32_t* lkey, int32_t* lpos,
                              int32_t* lcount, SelectShared& sh, Put put) {
  const int tid = threadIdx.x;
  uint32_t kmin = ~0u, kmax = 0u;
  src.visit([&](uint32_t key, int32_t) {
    kmin = min(kmin, key);
    kmax = max(kmax, key);
  });
  block_pair_reduce<THREADS, true>(kmin, kmax, sh);
  static_assert(NB % THREADS == 0 || NB < THREADS, "bins per thread");
  const float fmin = key_float(kmin);
  const float scale = (float)NB / (key_float(kmax) - fmin);
  if (kmin == kmax || !(scale > 0.0f && scale < __builtin_inff())) return false;
  auto bucket = [&](uint32_t key) { return min(NB - 1, (int)((key_float(key) - fmin) * scale)); };
  for (int k = tid; k < NB; k += THREADS) hist[k] = 0;
  if (tid == 0) *lcount = 0;
  __syncthreads();
  src.visit([&](uint32_t key, int32_t) { atomicAdd(&hist[bucket(key)], 1u); });
  __syncthreads();
  find_digit<THREADS, true>(hist, sh, need, NB);
  const int bsel = (int)sh.digit;
  const uint32_t rem = need - sh.before, in_b = sh.equal;
  __syncthreads();
  if (in_b > (uint32_t)kBucketList) return false;
  emit_bucket(src, bucket, bsel, sh, put, [&](uint32_t key, int32_t pos) {  // a few elements: a plain LDS atomic
    const int c = atomicAdd(lcount, 1);
    lkey[c] = key;
    lpos[c] = pos;
  });
  __syncthreads();
  rank_listed<THREADS>(in_b, rem, lkey, lpos, sh, put);
  return true;
}

// Elements e = tid, tid + THREADS, ... < count of (key[], pos[]) arrays.
template <int THREADS>
struct ArraySource {
  const uint32_t* key;
  const int32_t* pos;
  int count;
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
    for (int e = threadIdx.x; e < count; e += THREADS) f(key[e], pos[e]);
  }
};

// Two-level exact top-m of a source with n elements (n > m): a 4096-bin
// histogram of the top 12 key bits finds the bin b1 holding the m-th key;
// keys above b1 are emitted at once and b1's keys are compacted into LDS
// (at most CAP), where block_select() resolves the rest.  If b1 holds more
// than CAP keys, block_select() runs over the whole source instead.
template <int CAP>
struct TwoLevelShared {
  uint32_t hist[4096];
  uint32_t ckey[CAP];
  int32_t cpos[CAP];
  SelectShared sel;
  uint32_t b1, above, in_b1;
  int32_t ncand, lcount;
};

template <int THREADS, int CAP, class Src, class Put>
__device__ void two_level_select(const Src& src, uint32_t m, TwoLevelShared<CAP>& sh, Put put) {
  const int tid = threadIdx.x;
  uint32_t* hist = sh.hist;
  for (int k = tid; k < 4096; k += THREADS) hist[k] = 0;
  if (tid == 0) sh.ncand = 0;
  __syncthreads();
  src.visit([&](uint32_t key, int32_t) { atomicAdd(&hist[key >> 20], 1u); });
  __syncthreads();
  find_digit<THREADS, true>(hist, sh.sel, m, 4096);  // the bin holding the m-th key
  const uint32_t b1 = sh.sel.digit, above = sh.sel.before, in_b1 = sh.sel.equal;
  __syncthreads();
  if (in_b1 <= (uint32_t)CAP) {
    src.visit([&](uint32_t key, int32_t pos) {
      const uint32_t top = key >> 20;
      wave_append(top > b1, &sh.sel.emitted, [&](int slot) { put(slot, pos); });
      if (top == b1) {  // rare: a plain LDS atomic
        const int c = atomicAdd(&sh.ncand, 1);
        sh.ckey[c] = key;
        sh.cpos[c] = pos;
      }
    });
    __syncthreads();
    ArraySource<THREADS> cand{sh.ckey, sh.cpos, sh.ncand};
    // the histogram is free again: it serves the bucket pass and its list
    if (!bucket_select<THREADS>(cand, m - above, hist, hist, reinterpret_cast<int32_t*>(hist + kBucketList),
                                &sh.lcount, sh.sel, put))
      block_select<THREADS, false>(cand, m - above, sh.sel, put);
  } else {
    block_select<THREADS, false>(src, m, sh.sel, put);
  }
}

}  // namespace pivot
