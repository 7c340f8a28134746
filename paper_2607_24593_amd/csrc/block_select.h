// Workgroup-wide exact top-m selection (radix select on order-preserving keys).
//
// Selects the `need` elements of a source that rank first by (key descending,
// position ascending) and hands each selected position to `emit`.  The key is
// resolved in 4 histogram passes (12, 8, 8, 4 bits); if the m-th key is shared
// by more elements than remain to be taken, 4 more passes over the positions
// of the tied elements pick the lowest ones.  A final pass emits every element
// above the threshold.  Positions must be distinct non-negative int32.
//
// A source provides visit(f), calling f(key, pos) for each of the calling
// thread's elements; every thread of the workgroup calls it.  Sources may keep
// their elements in registers, LDS or global memory.
#pragma once

#include "device_common.h"

namespace pivot {

struct SelectShared {
  uint32_t hist[4096];
  uint32_t wsum[16];
  uint32_t digit, before, equal;
  int32_t emitted;
};

// Find the digit d (of `bins`) where the running count crosses `rem`, scanning
// digits downwards (desc) or upwards (!desc); every thread owns bins/THREADS
// consecutive digits.  Writes sh.digit, sh.before (count strictly before d in
// scan order) and sh.equal (count at d).  Contains workgroup barriers.
template <int THREADS, bool DESC>
__device__ __forceinline__ void find_digit(SelectShared& sh, uint32_t rem, int bins) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int per = bins / THREADS;  // bins is a multiple of THREADS, or smaller
  const int lo = per > 0 ? per * tid : tid;
  const int cnt = per > 0 ? per : (tid < bins ? 1 : 0);
  uint32_t tot = 0;
  for (int k = 0; k < cnt; ++k) tot += sh.hist[lo + k];
  uint32_t s = tot;  // inclusive scan over lanes in scan order
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t t = DESC ? __shfl_down(s, o, 64) : __shfl_up(s, o, 64);
    if (DESC ? (lane + o < 64) : (lane >= o)) s += t;
  }
  if (DESC ? lane == 0 : lane == 63) sh.wsum[wv] = s;
  __syncthreads();
  uint32_t before = s - tot;
  if (DESC) {
    for (int w = wv + 1; w < THREADS / 64; ++w) before += sh.wsum[w];
  } else {
    for (int w = 0; w < wv; ++w) before += sh.wsum[w];
  }
  for (int kk = 0; kk < cnt; ++kk) {
    const int k = DESC ? cnt - 1 - kk : kk;
    const uint32_t h = sh.hist[lo + k];
    if (before < rem && rem <= before + h) {
      sh.digit = lo + k;
      sh.before = before;
      sh.equal = h;
    }
    before += h;
  }
  __syncthreads();
}

// Key digits, most significant first: 12 bits (sign, exponent, 3 mantissa
// bits: spreads typical scores over many bins, so the histogram atomics rarely
// collide), then 8, 8, 4.  Positions use 8-bit digits.
template <int THREADS, class Src, class Emit>
__device__ void block_select(const Src& src, uint32_t need, SelectShared& sh, Emit emit) {
  constexpr int kShift[4] = {20, 12, 4, 0};
  constexpr int kBits[4] = {12, 8, 8, 4};
  const int tid = threadIdx.x;
  if (need == 0) return;
  uint32_t prefix = 0, mask = 0, rem = need, equal = 0;
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = kShift[pass], bins = 1 << kBits[pass];
    const uint32_t dmask = (uint32_t)bins - 1;
    for (int i = tid; i < bins; i += THREADS) sh.hist[i] = 0;
    __syncthreads();
    src.visit([&](uint32_t key, int32_t) {
      if ((key & mask) == prefix) atomicAdd(&sh.hist[(key >> shift) & dmask], 1u);
    });
    __syncthreads();
    find_digit<THREADS, true>(sh, rem, bins);
    rem -= sh.before;
    equal = sh.equal;
    prefix |= sh.digit << shift;
    mask |= dmask << shift;
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
      find_digit<THREADS, false>(sh, rem, 256);
      rem -= sh.before;
      ipref |= sh.digit << shift;
      imask |= 255u << shift;
      __syncthreads();
    }
  }
  src.visit([&](uint32_t key, int32_t pos) {
    if (key > T || (key == T && (all_ties || (uint32_t)pos <= ipref))) emit(pos);
  });
  __syncthreads();
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
  uint32_t ckey[CAP];
  int32_t cpos[CAP];
  SelectShared sel;  // its 4096-bin histogram also serves the first level
  uint32_t b1, above, in_b1;
  int32_t ncand;
};

template <int THREADS, int CAP, class Src, class Emit>
__device__ void two_level_select(const Src& src, uint32_t m, TwoLevelShared<CAP>& sh, Emit emit) {
  const int tid = threadIdx.x;
  uint32_t* hist = sh.sel.hist;
  for (int k = tid; k < 4096; k += THREADS) hist[k] = 0;
  if (tid == 0) sh.ncand = 0;
  __syncthreads();
  src.visit([&](uint32_t key, int32_t) { atomicAdd(&hist[key >> 20], 1u); });
  __syncthreads();
  find_digit<THREADS, true>(sh.sel, m, 4096);  // the bin holding the m-th key
  const uint32_t b1 = sh.sel.digit, above = sh.sel.before, in_b1 = sh.sel.equal;
  __syncthreads();
  if (in_b1 <= (uint32_t)CAP) {
    src.visit([&](uint32_t key, int32_t pos) {
      const uint32_t top = key >> 20;
      if (top > b1) {
        emit(pos);
      } else if (top == b1) {
        const int c = atomicAdd(&sh.ncand, 1);
        sh.ckey[c] = key;
        sh.cpos[c] = pos;
      }
    });
    __syncthreads();
    ArraySource<THREADS> cand{sh.ckey, sh.cpos, sh.ncand};
    block_select<THREADS>(cand, m - above, sh.sel, emit);
  } else {
    block_select<THREADS>(src, m, sh.sel, emit);
  }
}

}  // namespace pivot
