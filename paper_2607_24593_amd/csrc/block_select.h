// Workgroup-wide exact top-m selection (radix select on order-preserving keys).
//
// Selects the `need` elements of a source that rank first by (key descending,
// position ascending) and hands each selected position to `emit`.  The key is
// resolved 8 bits at a time (4 histogram passes); if the m-th key is shared by
// more elements than remain to be taken, 4 more passes over the positions of
// the tied elements pick the lowest ones.  A final pass emits every element
// above the threshold.  Positions must be distinct non-negative int32.
//
// A source provides visit(f), calling f(key, pos) for each of the calling
// thread's elements; every thread of the workgroup calls it.  Sources may keep
// their elements in registers, LDS or global memory.
#pragma once

#include "device_common.h"

namespace pivot {

struct SelectShared {
  uint32_t hist[256];
  uint32_t digit, before, equal;
  int32_t emitted;
};

// One wave (the workgroup's first) finds the digit d where the running count
// crosses `rem`, scanning digits downwards (desc) or upwards (!desc).  Writes
// sh.digit, sh.before (count strictly before d in scan order), sh.equal (count at d).
template <bool DESC>
__device__ __forceinline__ void find_digit(SelectShared& sh, uint32_t rem) {
  const int lane = threadIdx.x & 63;
  if (threadIdx.x >= 64) return;
  uint32_t v[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = sh.hist[4 * lane + i];
  const uint32_t tot = v[0] + v[1] + v[2] + v[3];
  uint32_t s = tot;  // inclusive scan in scan order
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t t = DESC ? __shfl_down(s, o, 64) : __shfl_up(s, o, 64);
    bool ok = DESC ? (lane + o < 64) : (lane >= o);
    if (ok) s += t;
  }
  uint32_t before = s - tot;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int i = DESC ? 3 - k : k;
    if (before < rem && rem <= before + v[i]) {
      sh.digit = 4 * lane + i;
      sh.before = before;
      sh.equal = v[i];
    }
    before += v[i];
  }
}

template <int THREADS, class Src, class Emit>
__device__ void block_select(const Src& src, uint32_t need, SelectShared& sh, Emit emit) {
  const int tid = threadIdx.x;
  if (need == 0) return;
  uint32_t prefix = 0, mask = 0, rem = need, equal = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < 256; i += THREADS) sh.hist[i] = 0;
    __syncthreads();
    src.visit([&](uint32_t key, int32_t) {
      if ((key & mask) == prefix) atomicAdd(&sh.hist[(key >> shift) & 255u], 1u);
    });
    __syncthreads();
    find_digit<true>(sh, rem);
    __syncthreads();
    rem -= sh.before;
    equal = sh.equal;
    prefix |= sh.digit << shift;
    mask |= 255u << shift;
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
      find_digit<false>(sh, rem);
      __syncthreads();
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
  uint32_t hist[4096];
  uint32_t ckey[CAP];
  int32_t cpos[CAP];
  SelectShared sel;
  uint32_t wsum[16];
  uint32_t b1, above, in_b1;
  int32_t ncand;
};

template <int THREADS, int CAP, class Src, class Emit>
__device__ void two_level_select(const Src& src, uint32_t m, TwoLevelShared<CAP>& sh, Emit emit) {
  const int tid = threadIdx.x;
  for (int k = tid; k < 4096; k += THREADS) sh.hist[k] = 0;
  if (tid == 0) sh.ncand = 0;
  __syncthreads();
  src.visit([&](uint32_t key, int32_t) { atomicAdd(&sh.hist[key >> 20], 1u); });
  __syncthreads();
  {  // bin where the count from the top crosses m: each thread owns 4096/THREADS bins
    constexpr int PER = 4096 / THREADS;
    const int lane = tid & 63, wv = tid >> 6;
    uint32_t tot = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) tot += sh.hist[PER * tid + k];
    uint32_t s = tot;  // inclusive suffix sum within the wave (lanes >= lane)
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      uint32_t t = __shfl_down(s, o, 64);
      if (lane + o < 64) s += t;
    }
    if (lane == 0) sh.wsum[wv] = s;
    __syncthreads();
    uint32_t above = s - tot;
    for (int w = wv + 1; w < THREADS / 64; ++w) above += sh.wsum[w];
#pragma unroll
    for (int k = PER - 1; k >= 0; --k) {
      const uint32_t h = sh.hist[PER * tid + k];
      if (above < m && m <= above + h) {
        sh.b1 = PER * tid + k;
        sh.above = above;
        sh.in_b1 = h;
      }
      above += h;
    }
  }
  __syncthreads();
  const uint32_t b1 = sh.b1, above = sh.above, in_b1 = sh.in_b1;
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
