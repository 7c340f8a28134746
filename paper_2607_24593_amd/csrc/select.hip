// Per-row top-m selection over score rows of fp32, or of bf16 (the rows the
// fp8 path writes; every bf16 value widens exactly to the fp32 it selects
// on), for the TopK of Sec. 3.1 and of Eqs. 6-7: one 512-thread workgroup per row (1024 threads when a launch
// holds at most 256 long rows), or, for such a launch given scratch (decode),
// the split select described below.
//
// Long rows (n >= kSampleMinLen) are read once when the expected number of
// compacted keys fits in LDS:
//   1 sample   every stride-th 256-byte chunk of the row (at most 8192
//              fp32 or 16384 bf16 scores) is held in registers; two histogram passes over the
//              sample (top 12, then next 8 key bits) find a 20-bit prefix
//              `thr` such that at least ts sampled keys have prefix >= thr,
//              where ts is the sample's expected share of m plus four
//              standard deviations;
//   2 compact  one pass over the row appends every key with prefix >= thr to
//              LDS (at most CAP: 4096 for m <= 2048, else 8000; each wave
//              fills its own CAP / waves entries, slots from a ballot prefix)
//              (a row whose ts, scaled to the whole row, would fill more
//              than 80% of CAP skips the sample and takes the two-pass path);
//   3 select   if the pass found at least m keys (and no wave more than its
//              share of CAP),
//              they include every key >= the m-th largest of the row, ties
//              included, so block_select() over them is exact; otherwise the
//              row takes the two-pass path below.
// Few long rows (decode) with a scratch buffer: step 1 runs in
// topk_thr_kernel (one workgroup per row writes the row's threshold), step 2
// in topk_slice_kernel on P workgroups per row (each compacts 1/P of the row
// into scratch), step 3 in topk_merge_kernel, which gathers the row's
// compacted keys into LDS; one workgroup per row could not pull its row fast
// enough on its own.
// Other rows: two_level_select() (block_select.h) over the row in global
// memory: pass 1 builds a 4096-bin histogram of the top 12 key bits, pass 2
// emits the keys above the threshold bin and compacts that bin into LDS, where
// the remaining bits are resolved (ties: lower position); a threshold bin that
// overflows LDS (e.g. many equal scores) selects directly over the row.
// A row with no more than m valid entries returns all of them, then -1.
#include <algorithm>
#include <climits>
#include <cstring>

#include "block_select.h"
#include "launch.h"

namespace pivot {

constexpr int kSelThreads = 512;
constexpr int kSelThreadsWide = 1024;  // few long rows: one workgroup per row must pull the row alone
constexpr int kWideMaxRows = kSplitMaxRows;  // "few": at most one row per CU
// LDS candidates: 16 KiB histogram + 32 KiB -> three workgroups per CU, or
// + 62.5 KiB -> two
constexpr int kSelCapSmall = 4096;
constexpr int kSelCapLarge = 8000;
constexpr int kSelCap16 = 7680;  // bf16 rows: 6-byte candidates, three 512-thread workgroups per CU
constexpr int kSampleMinLen = kSplitMinKeys;  // shorter rows take the two-pass path
constexpr int kChunk4 = 16;           // float4 per sampled chunk (256 bytes)
constexpr int kSampleChunks = 128;    // at most 8192 sampled scores
// split select: scratch entries per row over its P slices (each slice may hold
// twice its even share of the merge capacity), P in [kSplitMinP, kSplitMaxP]
constexpr int kSplitThreads = 256;
constexpr int kSplitSlots = 2 * kSelCapLarge;
constexpr int kSplitMinP = 4, kSplitMaxP = 16;
constexpr int kSplitPerMax = kSplitSlots / kSplitMinP;
constexpr int kSplitTargetBlocks = 1024;

// Elements of a score row (fp32 or bf16, E), visited with 16-byte vector
// loads (U in flight per thread) when aligned.
template <int T, int U, class E>
struct RowSource {
  using SV = ScoreVec<E>;
  static constexpr int N = SV::N;
  const E* row;
  int count;
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
    const int tid = threadIdx.x;
    if ((reinterpret_cast<uintptr_t>(row) & 15u) == 0) {
      const int nv = count / N;
      const uint4* r16 = reinterpret_cast<const uint4*>(row);
      auto each = [&](const uint4& a, int i) {
        float v[N];
        SV::unpack(a, v);
#pragma unroll
        for (int j = 0; j < N; ++j) f(float_key(v[j]), N * i + j);
      };
      int i = tid;
      for (; i + (U - 1) * T < nv; i += U * T) {
        uint4 a[U];
#pragma unroll
        for (int u = 0; u < U; ++u) a[u] = r16[i + u * T];
#pragma unroll
        for (int u = 0; u < U; ++u) each(a[u], i + u * T);
      }
      for (; i < nv; i += T) each(r16[i], i);
      for (int e = N * nv + tid; e < count; e += T) f(float_key(SV::one(row, e)), e);
    } else {
      for (int e = tid; e < count; e += T) f(float_key(SV::one(row, e)), e);
    }
  }
};

// The sampled keys (positions are not needed): V 16-byte vectors of N
// scores per thread.
template <int V, int N>
struct SampleSource {
  uint32_t key[N * V];
  bool ok[V];
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
#pragma unroll
    for (int v = 0; v < V; ++v)
      if (ok[v]) {
#pragma unroll
        for (int j = 0; j < N; ++j) f(key[N * v + j], 0);
      }
  }
};

// 20-bit key prefix of the ts-th largest sampled key (ts <= sampled count);
// hist: 4096 bins of LDS.
template <int T, class Src>
__device__ uint32_t sample_prefix(const Src& src, uint32_t ts, uint32_t* hist, SelectShared& sh) {
  const int tid = threadIdx.x;
  for (int k = tid; k < 4096; k += T) hist[k] = 0;
  __syncthreads();
  src.visit([&](uint32_t key, int32_t) { atomicAdd(&hist[key >> 20], 1u); });
  __syncthreads();
  find_digit<T, true>(hist, sh, ts, 4096);
  const uint32_t d1 = sh.digit, rem = ts - sh.before;
  __syncthreads();
  for (int k = tid; k < 256; k += T) hist[k] = 0;
  __syncthreads();
  src.visit([&](uint32_t key, int32_t) {
    if ((key >> 20) == d1) atomicAdd(&hist[(key >> 12) & 255u], 1u);
  });
  __syncthreads();
  find_digit<T, true>(hist, sh, rem, 256);
  const uint32_t thr = (d1 << 8) | sh.digit;
  __syncthreads();
  return thr;
}

// Steps 1 of the one-read path for a long aligned row: false (before any
// load) when the expected compacted count ts n / s would not leave room for
// its spread in CAP entries; else the threshold score fthr (every key with
// prefix >= thr compares >= fthr as a float).  Uniform over the workgroup.
template <int T, int CAP, class E>
__device__ bool sample_threshold(const E* row, int n, int m, uint32_t* hist, SelectShared& sel, float& fthr) {
  using SVec = ScoreVec<E>;
  constexpr int N = SVec::N;
  constexpr int SV = kSampleChunks * kChunk4 / T;  // sampled 16-byte vectors per thread
  const int tid = threadIdx.x;
  const int nch = n / (N * kChunk4);
  const int stride = max(16, (nch + kSampleChunks - 1) / kSampleChunks);
  const int sch = (nch + stride - 1) / stride;  // chunks 0, stride, 2 stride, ... < nch
  const int s = sch * N * kChunk4;
  const float rm = (float)s * (float)m / (float)n;
  const uint32_t ts = (uint32_t)ceilf(rm + 4.0f * sqrtf(rm)) + 1u;
  if (!(ts < (uint32_t)s && (float)ts * (float)n <= 0.8f * (float)CAP * (float)s)) return false;
  const uint4* r16 = reinterpret_cast<const uint4*>(row);
  SampleSource<SV, N> smp;
#pragma unroll
  for (int v = 0; v < SV; ++v) {
    const int qi = tid + T * v;
    smp.ok[v] = qi < sch * kChunk4;
    const uint4 a = smp.ok[v] ? r16[(int64_t)(qi / kChunk4) * stride * kChunk4 + qi % kChunk4] : make_uint4(0u, 0u, 0u, 0u);
    float x[N];
    SVec::unpack(a, x);
#pragma unroll
    for (int j = 0; j < N; ++j) smp.key[N * v + j] = float_key(x[j]);
  }
  const uint32_t thr = sample_prefix<T>(smp, ts, hist, sel);
  // key >> 12 >= thr  <=>  score >= the smallest score with that prefix
  // (the key map is monotone; -0 and +0 share a key and compare equal)
  fthr = key_float(thr << 12);
  return true;
}

// Step 2 of the one-read path: wave w appends the keys >= fthr it reads to
// its own segment [w SEG, (w + 1) SEG) of (ckey, cpos), a ballot prefix
// giving each lane its slot (no LDS atomics in the stream), then the segments
// are packed to the front.  The loops are uniform over the wave, so the
// running count stays the same in every lane.  Returns the number of keys, or
// CAP + 1 when a segment overflowed.  Aligned rows only.  KT: the stored key,
// the order-preserving uint32 key, or its upper half for bf16 rows (whose
// keys have 16 significant bits, key16_expand() restores them).
template <int T, int U, int CAP, class E, class KT = uint32_t>
__device__ __forceinline__ int stream_compact(const E* row, int n, float fthr, KT* ckey, int32_t* cpos,
                                              int32_t* wcnt) {
  using SV = ScoreVec<E>;
  constexpr int N = SV::N;
  constexpr int NW = T / 64, SEG = CAP / NW, R = (SEG + 63) / 64;
  constexpr int KSHIFT = 32 - 8 * (int)sizeof(KT);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  KT* mk = ckey + wv * SEG;
  int32_t* mp = cpos + wv * SEG;
  int wc = 0;
  auto take = [&](bool valid, float v, int pos) {
    const bool t = valid && v >= fthr;
    const uint64_t bal = __ballot(t);
    if (bal) {
      const int slot =
          wc + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
      if (t && slot < SEG) {
        mk[slot] = (KT)(float_key(v) >> KSHIFT);
        mp[slot] = pos;
      }
      wc += (int)__popcll((unsigned long long)bal);
    }
  };
  const int nv = n / N;
  const uint4* r16 = reinterpret_cast<const uint4*>(row);
  int base = 0;
  for (; base + U * T <= nv; base += U * T) {
    uint4 a[U];
#pragma unroll
    for (int u = 0; u < U; ++u) a[u] = r16[base + u * T + tid];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float x[N];
      SV::unpack(a[u], x);
      const int p = N * (base + u * T + tid);
#pragma unroll
      for (int j = 0; j < N; ++j) take(true, x[j], p + j);
    }
  }
  for (; base < nv; base += T) {
    const int q = base + tid;
    const bool ok = q < nv;
    float x[N];
    SV::unpack(ok ? r16[q] : make_uint4(0u, 0u, 0u, 0u), x);
#pragma unroll
    for (int j = 0; j < N; ++j) take(ok, x[j], N * q + j);
  }
  if (N * nv < n) {  // the n mod N tail
    const int e = N * nv + tid;
    const bool ok = e < n;
    take(ok, ok ? SV::one(row, e) : 0.f, e);
  }
  if (lane == 0) wcnt[wv] = wc;
  __syncthreads();
  int pre = 0, tot = 0;
  bool over = false;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int c = wcnt[w];
    pre += w < wv ? c : 0;
    tot += c;
    over |= c > SEG;
  }
  if (over) return CAP + 1;
  // a segment moves left onto space other waves may still be reading:
  // through registers, with a barrier in between
  KT kk[R];
  int32_t pp[R];
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const int e = lane + 64 * j;
    if (e < wc) {
      kk[j] = mk[e];
      pp[j] = mp[e];
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const int e = lane + 64 * j;
    if (e < wc) {
      ckey[pre + e] = kk[j];
      cpos[pre + e] = pp[j];
    }
  }
  __syncthreads();
  return tot;
}

// Where row (b, i)'s indices go (OutDesc).
struct RowDest {
  int32_t* base;
  int64_t dest0;
  int ndest;
  int ld;
  __device__ RowDest(const OutDesc& od, const SeqTable& st, int b, int i) : base(od.base), ld(od.ld) {
    if (od.fan_g == 0) {
      dest0 = (int64_t)(od.groups ? st.grp0[b] : st.row0[b]) + i;
      ndest = 1;
    } else {
      dest0 = (int64_t)st.row0[b] + (int64_t)i * od.fan_g;
      ndest = min(od.fan_g, st.n_rows[b] - i * od.fan_g);
    }
  }
  __device__ __forceinline__ void operator()(int p, int32_t v) const {
    for (int u = 0; u < ndest; ++u) base[(dest0 + u) * ld + p] = v;
  }
};

// SAMPLE: the launch holds rows long enough for the one-read path (a launch
// of short rows only takes the kernel without it, which keeps the two-pass
// loops as lean as they compile alone).  Register budget: as many 512-thread
// workgroups per CU as LDS allows (three for CAP 4096, else two).
template <int CAP, int T, bool SAMPLE, class E>
__global__ __launch_bounds__(T) __attribute__((amdgpu_waves_per_eu(CAP == kSelCapSmall && T == kSelThreads ? 6 : 4)))
void topk_rows_kernel(const E* __restrict__ scores, int64_t ld, SeqTable st, RowSpace rs, OutDesc od) {
  // 16-byte row loads in flight per thread (the same bytes for bf16 rows,
  // whose vectors hold twice as many scores)
  constexpr int U = T == kSelThreads ? 4 : 8;
  __shared__ TwoLevelShared<CAP> sh;
  const int nrows = rs.i1 - rs.i0;
  const int b = blockIdx.x / nrows;
  const int i = rs.i0 + blockIdx.x % nrows;
  if (!row_active(st, rs, b, i)) return;
  const int tid = threadIdx.x;
  const int64_t n64 = row_limit(st, rs, b, i) + 1;
  const int n = (int)max((int64_t)0, n64);
  const E* row = scores + ((int64_t)b * nrows + (i - rs.i0)) * ld;
  const int m = od.m;
  const RowDest put(od, st, b, i);
  if (n <= m) {
    for (int p = tid; p < m; p += T) put(p, p < n ? p : -1);
    return;
  }
  if (tid == 0) sh.sel.emitted = 0;
  RowSource<T, U, E> src{row, n};
  const bool aligned = (reinterpret_cast<uintptr_t>(row) & 15u) == 0;
  float fthr;
  if (SAMPLE && n >= kSampleMinLen && aligned) {
    if (sample_threshold<T, CAP>(row, n, m, sh.hist, sh.sel, fthr)) {
      __shared__ int32_t wcnt[T / 64];
      const int found = stream_compact<T, U, CAP>(row, n, fthr, sh.ckey, sh.cpos, wcnt);
      if (found >= m && found <= CAP) {
        ArraySource<T> cand{sh.ckey, sh.cpos, found};
        // the sample's histogram is free: it serves the bucket pass and its list
        if (!bucket_select<T>(cand, (uint32_t)m, sh.hist, sh.hist, reinterpret_cast<int32_t*>(sh.hist + kBucketList),
                              &sh.lcount, sh.sel, put))
          block_select<T, false>(cand, (uint32_t)m, sh.sel, put);
        return;
      }
    }
  }
  two_level_select<T>(src, (uint32_t)m, sh, put);
}

// The order-preserving key of a bf16 score from its upper half: the lower
// half of a bf16 value's fp32 key is 0 for +0 and positive values, 0xFFFF for
// negative ones (float_key complements them).
__device__ __forceinline__ uint32_t key16_expand(uint32_t k16) {
  return (k16 << 16) | ((k16 & 0x8000u) ? 0u : 0xFFFFu);
}

// Elements e = tid, tid + THREADS, ... < count of (16-bit key, position) arrays.
template <int THREADS>
struct ArraySource16 {
  const uint16_t* key;
  const int32_t* pos;
  int count;
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
    for (int e = threadIdx.x; e < count; e += THREADS) f(key16_expand(key[e]), pos[e]);
  }
};

// Members of one tied value (equal keys): positions only.
template <int THREADS>
struct TieSource {
  const int32_t* pos;
  int count;
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
    for (int e = threadIdx.x; e < count; e += THREADS) f(0u, pos[e]);
  }
};

// The candidates of stream_compact16 in place: wave w's wcnt[w] entries
// start at w * SEG; element e of the concatenation lies in the segment whose
// prefix count it reaches.
template <int THREADS, int NW, int SEG>
struct SegSource16 {
  const uint16_t* key;
  const int32_t* pos;
  int pre[NW + 1];  // prefix counts of the segments
  __device__ SegSource16(const uint16_t* k, const int32_t* p, const int32_t* wcnt) : key(k), pos(p) {
    pre[0] = 0;  // uniform: scalar registers
#pragma unroll
    for (int w = 0; w < NW; ++w) pre[w + 1] = __builtin_amdgcn_readfirstlane(pre[w] + wcnt[w]);
  }
  __device__ __forceinline__ int count() const { return pre[NW]; }
  __device__ __forceinline__ int index(int e) const {
    int w = 0, base = 0;  // compares, not an indexed read (which would put pre[] in scratch)
#pragma unroll
    for (int k = 1; k < NW; ++k)
      if (e >= pre[k]) {
        w = k;
        base = pre[k];
      }
    return w * SEG + (e - base);
  }
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
    for (int e = threadIdx.x; e < pre[NW]; e += THREADS) {
      const int i = index(e);
      f(key16_expand(key[i]), pos[i]);
    }
  }
};

// LDS of topk_rows16_kernel: one region serves, in turn, the sampling
// histogram (4096 words), the candidates (16-bit keys and int32 positions,
// CAP each) with the exact select's histogram (kNB16 words), or, for a row
// that falls back, the two-level select's buffers (TwoLevelShared<CAP2>).
constexpr int kNB16 = 1024;
template <int CAP>
struct Rows16Lds {
  static constexpr int KEY_BYTES = (2 * CAP + 15) / 16 * 16;
  static constexpr int POS_BYTES = 4 * CAP;
  static constexpr int MAIN = KEY_BYTES + POS_BYTES + 4 * kNB16;
  static constexpr int CAP2 = ((MAIN - (int)sizeof(TwoLevelShared<0>)) / 8) / 64 * 64;
  static constexpr int RAW = MAIN > 4 * 4096 ? MAIN : 4 * 4096;
  static_assert((int)sizeof(TwoLevelShared<CAP2>) <= RAW, "fallback fits the region");
};

// The 16-bit order-preserving keys of the two bf16 scores of a word
// (key16_expand(k) == float_key(score)), without branches: a half with its
// sign bit set is complemented, any other gets its sign bit set; -0 (0x8000)
// then lands on 0x7FFF, one below +0's key 0x8000, and is moved up to it.
__device__ __forceinline__ uint32_t key16_pair(uint32_t w) {
  const uint32_t t = (w >> 15) & 0x00010001u;  // the sign of each half in its bit 0
  const uint32_t k = w ^ (t * 0x7FFFu | 0x80008000u);
  return k + (((k & 0xFFFFu) == 0x7FFFu ? 1u : 0u) | ((k >> 16) == 0x7FFFu ? 0x10000u : 0u));
}

// The 16-bit order key of one bf16 value (key16_pair of one half).
__device__ __forceinline__ uint32_t key16_one(uint32_t h) {
  const uint32_t k = h ^ ((h & 0x8000u) ? 0xFFFFu : 0x8000u);
  return k + (k == 0x7FFFu ? 1u : 0u);
}

// The sampled keys of bf16 rows, packed two per register: V 16-byte vectors
// per thread.
template <int V>
struct SampleSource16 {
  uint32_t pk[4 * V];
  bool ok[V];
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
#pragma unroll
    for (int v = 0; v < V; ++v)
      if (ok[v]) {
#pragma unroll
        for (int j = 0; j < 8; ++j) f(key16_expand((pk[4 * v + j / 2] >> (16 * (j & 1))) & 0xFFFFu), 0);
      }
  }
};

// sample_threshold for bf16 rows with the sample held as packed 16-bit keys,
// at most SCH chunks: 32 (4096 scores, 1/32 of a 131072-score row) for the
// large candidate buffer, where the count above the threshold spreads by ~8%
// of m inside the room CAP leaves; 64 for the small one (m <= 2048), whose
// room is tighter.  base16 receives the 16-bit key below which no kept key
// lies.
template <int T, int CAP, int SCH>
__device__ bool sample_threshold16(const bf16_t* row, int n, int m, uint32_t* hist, SelectShared& sel, float& fthr,
                                   uint32_t& base16) {
  constexpr int N = 8;
  constexpr int SV = (SCH * kChunk4 + T - 1) / T;  // sampled 16-byte vectors per thread
  const int tid = threadIdx.x;
  const int nch = n / (N * kChunk4);
  const int stride = max(16, (nch + SCH - 1) / SCH);
  const int sch = (nch + stride - 1) / stride;
  const int s = sch * N * kChunk4;
  const float rm = (float)s * (float)m / (float)n;
  const uint32_t ts = (uint32_t)ceilf(rm + 4.0f * sqrtf(rm)) + 1u;
  if (!(ts < (uint32_t)s && (float)ts * (float)n <= 0.8f * (float)CAP * (float)s)) return false;
  const uint4* r16 = reinterpret_cast<const uint4*>(row);
  SampleSource16<SV> smp;
#pragma unroll
  for (int v = 0; v < SV; ++v) {
    const int qi = tid + T * v;
    smp.ok[v] = qi < sch * kChunk4;
    const uint4 a = smp.ok[v] ? r16[(int64_t)(qi / kChunk4) * stride * kChunk4 + qi % kChunk4] : make_uint4(0u, 0u, 0u, 0u);
    smp.pk[4 * v + 0] = key16_pair(a.x);
    smp.pk[4 * v + 1] = key16_pair(a.y);
    smp.pk[4 * v + 2] = key16_pair(a.z);
    smp.pk[4 * v + 3] = key16_pair(a.w);
  }
  const uint32_t thr = sample_prefix<T>(smp, ts, hist, sel);
  fthr = key_float(thr << 12);
  base16 = thr >> 4;
  return true;
}

// Step 2 for bf16 rows: stream_compact storing 16-bit keys, with the next U
// vectors' loads issued before the current ones are examined, and every kept
// key counted in `hist` (kNB16 words, zeroed by the caller) at its distance
// above the threshold, bin min(k16 - base16, kNB16 - 1): below the top bin,
// one bin per bf16 value.  The waves' segments stay where they are (counts in
// wcnt; SegSource16 reads them in place).
template <int T, int U, int CAP>
__device__ __forceinline__ int stream_compact16(const bf16_t* row, int n, float fthr, uint32_t base16,
                                                uint16_t* ckey, int32_t* cpos, uint32_t* hist, int32_t* wcnt) {
  static_assert(8 * U <= 32, "one 32-bit mask per batch");
  using SV = ScoreVec<bf16_t>;
  constexpr int N = SV::N;
  constexpr int NW = T / 64, SEG = CAP / NW;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  uint16_t* mk = ckey + wv * SEG;
  int32_t* mp = cpos + wv * SEG;
  int wc = 0;  // keys this wave has kept (the same in every lane)
  // Appends the kept scores of a batch (bit 8 u + j of `bits`: score j of the
  // lane's vector u, which is vector q0 + u T of the row): a wave prefix sum
  // of the lanes' counts gives each lane its first slot, then every lane
  // writes its own keys, vector by vector, a loop over its set bits (rarely
  // more than two per vector).
  auto append = [&](const uint4 (&a)[U], uint32_t bits, int q0) {
    const uint32_t cnt = (uint32_t)__popc(bits);
    const uint32_t incl = wave_incl_sum(cnt);
    int slot = wc + (int)(incl - cnt);
    wc += __builtin_amdgcn_readlane((int)incl, 63);
#pragma unroll
    for (int u = 0; u < U; ++u) {  // a static vector index: its words stay in registers
      uint32_t mu = (bits >> (N * u)) & 0xFFu;
      const uint64_t lo = ((uint64_t)a[u].y << 32) | a[u].x, hi = ((uint64_t)a[u].w << 32) | a[u].z;
      while (mu) {
        const int j = __builtin_ctz(mu);
        mu &= mu - 1;
        const uint32_t h = (uint32_t)(((j & 4) ? hi : lo) >> (16 * (j & 3))) & 0xFFFFu;
        const uint32_t k16 = key16_one(h);
        atomicAdd(&hist[min(k16 - base16, (uint32_t)(kNB16 - 1))], 1u);
        if (slot < SEG) {
          mk[slot] = (uint16_t)k16;
          mp[slot] = N * (q0 + u * T) + j;
        }
        ++slot;
      }
    }
  };
  auto mask_of = [&](const uint4& a, int u) {
    float x[N];
    SV::unpack(a, x);
    uint32_t bits = 0;
#pragma unroll
    for (int j = 0; j < N; ++j) bits |= (x[j] >= fthr ? 1u : 0u) << (N * u + j);
    return bits;
  };
  const int nv = n / N;
  const uint4* r16 = reinterpret_cast<const uint4*>(row);
  int base = 0;
  for (; base + U * T <= nv; base += U * T) {
    uint4 a[U];
#pragma unroll
    for (int u = 0; u < U; ++u) a[u] = r16[base + u * T + tid];
    uint32_t bits = 0;
#pragma unroll
    for (int u = 0; u < U; ++u) bits |= mask_of(a[u], u);
    append(a, bits, base + tid);
  }
  for (; base < nv; base += T) {  // fewer than U T vectors left: one per lane
    const int q = base + tid;
    uint4 a[U];
#pragma unroll
    for (int u = 0; u < U; ++u) a[u] = make_uint4(0u, 0u, 0u, 0u);
    if (q < nv) a[0] = r16[q];
    append(a, q < nv ? mask_of(a[0], 0) : 0u, q);
  }
  if (N * nv < n) {  // the n mod N tail: score e is element e mod N of vector e / N
    const int e = N * nv + tid;
    const bool ok = e < n;
    const int j = e & (N - 1);
    const uint32_t h = ok ? (uint32_t)row[e] : 0u;
    const uint32_t w = (j & 1) ? (h << 16) : h;
    uint4 a[U];
#pragma unroll
    for (int u = 0; u < U; ++u) a[u] = make_uint4(0u, 0u, 0u, 0u);
    a[0] = make_uint4((j >> 1) == 0 ? w : 0u, (j >> 1) == 1 ? w : 0u, (j >> 1) == 2 ? w : 0u, (j >> 1) == 3 ? w : 0u);
    const bool t = ok && __uint_as_float(h << 16) >= fthr;
    append(a, t ? (1u << j) : 0u, e / N);
  }
  if (lane == 0) wcnt[wv] = wc;
  __syncthreads();
  int tot = 0;
  bool over = false;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    tot += wcnt[w];
    over |= wcnt[w] > SEG;
  }
  return over ? CAP + 1 : tot;
}

// Step 3 for bf16 rows, from the histogram the compaction built: b* = the bin
// holding the m-th largest key; every candidate in a higher bin is taken, and
// bin b* (below the top bin) holds one bf16 value, so its members tie and the
// lowest positions among them complete the set.  Returns false, having
// emitted nothing, when b* is the top bin or holds more than kNB16
// members.  lpos: kNB16 LDS words (may alias hist).
template <int T, class Src, class Put>
__device__ bool select16(const Src& cand, uint32_t base16, uint32_t m, uint32_t* hist, int32_t* lpos,
                         int32_t* lcount, SelectShared& sh, Put put) {
  const int tid = threadIdx.x;
  find_digit<T, true>(hist, sh, m, kNB16);  // ends with a barrier
  const uint32_t bsel = sh.digit, rem = m - sh.before, in_b = sh.equal;
  if (bsel == (uint32_t)(kNB16 - 1) || in_b > (uint32_t)kNB16) return false;
  if (tid == 0) *lcount = 0;
  __syncthreads();
  cand.visit([&](uint32_t key, int32_t p) {
    const uint32_t d = min((key >> 16) - base16, (uint32_t)(kNB16 - 1));
    wave_append(d > bsel, &sh.emitted, [&](int slot) { put(slot, p); });
    if (d == bsel) lpos[atomicAdd(lcount, 1)] = p;
  });
  __syncthreads();
  if (in_b <= (uint32_t)kBucketList) {  // rank each tied member by its position
    static_assert(T >= kBucketList, "one thread per tied member");
    const bool mine = tid < (int)in_b;
    const int32_t p = mine ? lpos[tid] : 0;
    uint32_t r = 0;
    if (mine)
      for (int u = 0; u < (int)in_b; ++u) r += (uint32_t)(lpos[u] < p);
    wave_append(mine && r < rem, &sh.emitted, [&](int slot) { put(slot, p); });
    __syncthreads();
  } else {  // many ties: a radix select on their positions (the keys are equal)
    const TieSource<T> ties{lpos, (int)in_b};
    block_select<T, false>(ties, rem, sh, put);
  }
  return true;
}

// topk_rows_kernel's one-read path for bf16 score rows (fp8 inputs) of a
// launch holding rows of 16384+ scores: candidates take 6 bytes (16-bit key,
// int32 position) instead of 8, and the sampling histogram, the candidates
// and the row fallback share one LDS region (they are never live together),
// so three 512-thread workgroups fit a CU instead of two.
template <int CAP, int T>
__global__ __launch_bounds__(T) __attribute__((amdgpu_waves_per_eu(6)))
void topk_rows16_kernel(const bf16_t* __restrict__ scores, int64_t ld, SeqTable st, RowSpace rs, OutDesc od) {
  using Lds = Rows16Lds<CAP>;
  constexpr int U = 4;
  __shared__ __attribute__((aligned(16))) uint8_t raw[Lds::RAW];
  __shared__ SelectShared sel;
  __shared__ int32_t lcount;
  __shared__ int32_t wcnt[T / 64];
  const int nrows = rs.i1 - rs.i0;
  const int b = blockIdx.x / nrows;
  const int i = rs.i0 + blockIdx.x % nrows;
  if (!row_active(st, rs, b, i)) return;
  const int tid = threadIdx.x;
  const int n = (int)max((int64_t)0, row_limit(st, rs, b, i) + 1);
  const bf16_t* row = scores + ((int64_t)b * nrows + (i - rs.i0)) * ld;
  const int m = od.m;
  const RowDest put(od, st, b, i);
  if (n <= m) {
    for (int p = tid; p < m; p += T) put(p, p < n ? p : -1);
    return;
  }
  if (tid == 0) sel.emitted = 0;
  const bool aligned = (reinterpret_cast<uintptr_t>(row) & 15u) == 0;
  uint16_t* ckey = reinterpret_cast<uint16_t*>(raw);
  int32_t* cpos = reinterpret_cast<int32_t*>(raw + Lds::KEY_BYTES);
  uint32_t* hist = reinterpret_cast<uint32_t*>(raw + Lds::KEY_BYTES + Lds::POS_BYTES);
  for (int k = tid; k < kNB16; k += T) hist[k] = 0;  // outside the sampling histogram's words
  float fthr;
  uint32_t base16;
  if (n >= kSampleMinLen && aligned &&
      sample_threshold16<T, CAP, CAP == kSelCapSmall ? 64 : 32>(row, n, m, reinterpret_cast<uint32_t*>(raw), sel,
                                                               fthr, base16)) {
    const int found = stream_compact16<T, U, CAP>(row, n, fthr, base16, ckey, cpos, hist, wcnt);
    if (found >= m && found <= CAP) {
      const SegSource16<T, T / 64, CAP / (T / 64)> cand(ckey, cpos, wcnt);
      if (select16<T>(cand, base16, (uint32_t)m, hist, reinterpret_cast<int32_t*>(hist), &lcount, sel, put))
        return;
      if (!bucket_select<T, kNB16>(cand, (uint32_t)m, hist, hist, reinterpret_cast<int32_t*>(hist + kBucketList),
                                   &lcount, sel, put))
        block_select<T, false>(cand, (uint32_t)m, sel, put);
      return;
    }
  }
  TwoLevelShared<Lds::CAP2>& fb = *reinterpret_cast<TwoLevelShared<Lds::CAP2>*>(raw);
  __syncthreads();  // the region's previous use has ended in every wave
  if (tid == 0) fb.sel.emitted = 0;
  RowSource<T, U, bf16_t> src{row, n};
  two_level_select<T>(src, (uint32_t)m, fb, put);
}

// Split select, step 1: workgroup r writes row r's threshold score to
// thr[r], or NaN when the row takes the two-pass path (n <= m, short or
// unaligned row, sample declined).
template <int CAP, int T, class E>
__global__ __launch_bounds__(T) void topk_thr_kernel(const E* __restrict__ scores, int64_t ld, SeqTable st,
                                                     RowSpace rs, int m, float* __restrict__ thr) {
  __shared__ uint32_t hist[4096];
  __shared__ SelectShared sel;
  const int nrows = rs.i1 - rs.i0;
  const int r = blockIdx.x;
  const int b = r / nrows;
  const int i = rs.i0 + r % nrows;
  if (!row_active(st, rs, b, i)) return;
  const int n = (int)max((int64_t)0, row_limit(st, rs, b, i) + 1);
  const E* row = scores + ((int64_t)b * nrows + (i - rs.i0)) * ld;
  const bool aligned = (reinterpret_cast<uintptr_t>(row) & 15u) == 0;
  float fthr;
  if (n <= m || n < kSampleMinLen || !aligned || !sample_threshold<T, CAP>(row, n, m, hist, sel, fthr))
    fthr = __builtin_nanf("");
  if (threadIdx.x == 0) thr[r] = fthr;
}

// Split select, step 2: workgroup (r, s) compacts the keys >= thr[r] among
// 16-byte vectors [s per_v, (s+1) per_v) of row r (the last slice also takes
// the n mod N tail) into LDS and writes them to cand[(r P + s) per ..] with
// their count in cnt[r P + s]: -1 when the row takes the two-pass path
// (thr[r] is NaN), -2 when the slice held more than `per` keys.
template <class E>
__global__ __launch_bounds__(kSplitThreads) void topk_slice_kernel(const E* __restrict__ scores, int64_t ld,
                                                                   SeqTable st, RowSpace rs, int P, int per,
                                                                   const float* __restrict__ thr,
                                                                   uint2* __restrict__ cand,
                                                                   int32_t* __restrict__ cnt) {
  using SV = ScoreVec<E>;
  constexpr int N = SV::N;
  constexpr int T = kSplitThreads, U = 8;  // 16-byte loads in flight per thread
  __shared__ uint2 lc[kSplitPerMax];
  __shared__ int32_t nc;
  const int nrows = rs.i1 - rs.i0;
  const int r = blockIdx.x, slice = blockIdx.y;
  const int b = r / nrows;
  const int i = rs.i0 + r % nrows;
  if (!row_active(st, rs, b, i)) return;
  const int tid = threadIdx.x;
  const int n = (int)max((int64_t)0, row_limit(st, rs, b, i) + 1);
  const E* row = scores + ((int64_t)b * nrows + (i - rs.i0)) * ld;
  int32_t* my_cnt = cnt + (int64_t)r * P + slice;
  const float fthr = thr[r];
  if (__builtin_isnan(fthr)) {
    if (tid == 0) *my_cnt = -1;
    return;
  }
  if (tid == 0) nc = 0;
  __syncthreads();
  auto take = [&](float v, int pos) {
    if (v >= fthr) {
      const int c = atomicAdd(&nc, 1);
      if (c < per) lc[c] = make_uint2(float_key(v), (uint32_t)pos);
    }
  };
  const int nv = n / N;
  const int per_v = (nv + P - 1) / P;
  const int a_v = slice * per_v, e_v = min(nv, a_v + per_v);
  const uint4* r16 = reinterpret_cast<const uint4*>(row);
  int q = a_v + tid;
  for (; q + (U - 1) * T < e_v; q += U * T) {
    uint4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = r16[q + u * T];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float v[N];
      SV::unpack(x[u], v);
      const int p = N * (q + u * T);
#pragma unroll
      for (int j = 0; j < N; ++j) take(v[j], p + j);
    }
  }
  for (; q < e_v; q += T) {
    float v[N];
    SV::unpack(r16[q], v);
#pragma unroll
    for (int j = 0; j < N; ++j) take(v[j], N * q + j);
  }
  if (slice == P - 1)
    for (int e = N * nv + tid; e < n; e += T) take(SV::one(row, e), e);
  __syncthreads();
  const int c = nc;
  if (tid == 0) *my_cnt = c <= per ? c : -2;
  if (c <= per) {
    uint2* dst = cand + ((int64_t)r * P + slice) * per;
    for (int e = tid; e < c; e += T) dst[e] = lc[e];
  }
}

// Split select, step 3: one workgroup per row gathers the keys its slices
// compacted (when every slice kept its keys and they number m .. CAP) into
// LDS and selects exactly over them; any other row takes the two-pass path.
template <int CAP, int T, class E>
__global__ __launch_bounds__(T) void topk_merge_kernel(const E* __restrict__ scores, int64_t ld, SeqTable st,
                                                       RowSpace rs, OutDesc od, int P, int per,
                                                       const uint2* __restrict__ cand,
                                                       const int32_t* __restrict__ cnt) {
  constexpr int U = 8 * (int)sizeof(E) / 4;  // 16-byte loads in flight (fallback path)
  constexpr int V = (CAP + T - 1) / T;  // gathered keys per thread
  __shared__ TwoLevelShared<CAP> sh;
  __shared__ int32_t pre[kSplitMaxP + 1];
  const int nrows = rs.i1 - rs.i0;
  const int r = blockIdx.x;
  const int b = r / nrows;
  const int i = rs.i0 + r % nrows;
  if (!row_active(st, rs, b, i)) return;
  const int tid = threadIdx.x;
  const int n = (int)max((int64_t)0, row_limit(st, rs, b, i) + 1);
  const E* row = scores + ((int64_t)b * nrows + (i - rs.i0)) * ld;
  const int m = od.m;
  const RowDest put(od, st, b, i);
  if (n <= m) {
    for (int p = tid; p < m; p += T) put(p, p < n ? p : -1);
    return;
  }
  if (tid < 64) {  // the slices' counts, one per lane, and their prefix sums
    const int c = tid < P ? cnt[(int64_t)r * P + tid] : 0;
    int incl = max(c, 0);
#pragma unroll
    for (int o = 1; o < kSplitMaxP; o <<= 1) {
      const int t = __shfl_up(incl, o, 64);
      if (tid >= o) incl += t;
    }
    const bool ok = __ballot(tid < P && c < 0) == 0;
    if (tid < P) pre[tid] = incl - max(c, 0);
    const int tot = __shfl(incl, P - 1, 64);
    if (tid == 0) {
      pre[P] = ok ? tot : -1;
      sh.sel.emitted = 0;
    }
  }
  __syncthreads();
  const int total = pre[P];
  if (total >= m && total <= CAP) {
    // every thread fetches its (at most V) keys at once, then stores them;
    // an element's slice comes from the prefix sums held in registers
    int pr[kSplitMaxP];
#pragma unroll
    for (int k = 0; k < kSplitMaxP; ++k) pr[k] = k < P ? pre[k] : 0x7FFFFFFF;
    uint2 v[V];
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const int e = tid + j * T;
      v[j] = make_uint2(0u, 0u);
      if (e < total) {
        int s = 0, base = 0;
#pragma unroll
        for (int k = 1; k < kSplitMaxP; ++k)
          if (e >= pr[k]) {
            s = k;
            base = pr[k];
          }
        v[j] = cand[((int64_t)r * P + s) * per + (e - base)];
      }
    }
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const int e = tid + j * T;
      if (e < total) {
        sh.ckey[e] = v[j].x;
        sh.cpos[e] = (int32_t)v[j].y;
      }
    }
    __syncthreads();
    ArraySource<T> src{sh.ckey, sh.cpos, total};
    if (!bucket_select<T>(src, (uint32_t)m, sh.hist, sh.hist, reinterpret_cast<int32_t*>(sh.hist + kBucketList),
                          &sh.lcount, sh.sel, put))
      block_select<T, false>(src, (uint32_t)m, sh.sel, put);
    return;
  }
  RowSource<T, U, E> src{row, n};
  two_level_select<T>(src, (uint32_t)m, sh, put);
}

size_t split_scratch_bytes(int64_t rows) {
  return (size_t)rows * ((size_t)kSplitSlots * sizeof(uint2) + (size_t)kSplitMaxP * sizeof(int32_t) + sizeof(float));
}

// Smallest limit of an active row of rs (limits grow with the row index).
static int64_t min_limit(const SeqTable& st, const RowSpace& rs) {
  int64_t lim = INT64_MAX;
  for (int b = 0; b < st.n; ++b) {
    const int cnt = rs.kind == kProxyRows ? (st.n_rows[b] + rs.step - 1) / rs.step : st.n_rows[b];
    int hi = std::min(rs.i1, cnt), lo = rs.i0;
    if (rs.kind == kDenseRows) hi = std::min(hi, st.dense_rows[b]);
    if (rs.kind == kProxyRows) lo = std::max(lo, st.first_proxy[b]);
    if (hi > lo) lim = std::min(lim, (int64_t)st.q_pos0[b] + (int64_t)lo * rs.step);
  }
  return lim;
}

template <class E>
static hipError_t topk_launch(const E* scores, int64_t ld, const SeqTable& st, const RowSpace& rs,
                              const OutDesc& od, int64_t lim_max, void* scratch, size_t scratch_bytes,
                              hipStream_t stream) {
  const int nrows = rs.i1 - rs.i0;
  if (nrows <= 0 || st.n <= 0) return hipSuccess;
  const int64_t blocks = (int64_t)st.n * nrows;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
  if (blocks <= kWideMaxRows && lim_max + 1 >= kSampleMinLen && scratch &&
      scratch_bytes >= split_scratch_bytes(blocks)) {
    // few long rows: P slice workgroups per row, then one merge workgroup
    const int P = (int)std::max<int64_t>(kSplitMinP, std::min<int64_t>(kSplitMaxP, kSplitTargetBlocks / blocks));
    const int per = kSplitSlots / P;
    uint2* cand = reinterpret_cast<uint2*>(scratch);
    int32_t* cnt = reinterpret_cast<int32_t*>(cand + (size_t)blocks * kSplitSlots);
    float* thr = reinterpret_cast<float*>(cnt + (size_t)blocks * kSplitMaxP);
    const dim3 sgrid((unsigned)blocks, (unsigned)P);
    const bool small = od.m <= kSelCapSmall / 2;
    if (small)
      hipLaunchKernelGGL((topk_thr_kernel<kSelCapSmall, kSelThreadsWide, E>), dim3((unsigned)blocks),
                         dim3(kSelThreadsWide), 0, stream, scores, ld, st, rs, od.m, thr);
    else
      hipLaunchKernelGGL((topk_thr_kernel<kSelCapLarge, kSelThreadsWide, E>), dim3((unsigned)blocks),
                         dim3(kSelThreadsWide), 0, stream, scores, ld, st, rs, od.m, thr);
    hipLaunchKernelGGL(topk_slice_kernel<E>, sgrid, dim3(kSplitThreads), 0, stream, scores, ld, st, rs, P, per, thr,
                       cand, cnt);
    if (small)
      hipLaunchKernelGGL((topk_merge_kernel<kSelCapSmall, kSelThreadsWide, E>), dim3((unsigned)blocks),
                         dim3(kSelThreadsWide), 0, stream, scores, ld, st, rs, od, P, per, cand, cnt);
    else
      hipLaunchKernelGGL((topk_merge_kernel<kSelCapLarge, kSelThreadsWide, E>), dim3((unsigned)blocks),
                         dim3(kSelThreadsWide), 0, stream, scores, ld, st, rs, od, P, per, cand, cnt);
    return hipGetLastError();
  }
  if (blocks <= kWideMaxRows && lim_max + 1 >= kSampleMinLen) {
    // few long rows (decode): one wide workgroup per row
    if (od.m <= kSelCapSmall / 2)
      hipLaunchKernelGGL((topk_rows_kernel<kSelCapSmall, kSelThreadsWide, true, E>), dim3((unsigned)blocks),
                         dim3(kSelThreadsWide), 0, stream, scores, ld, st, rs, od);
    else
      hipLaunchKernelGGL((topk_rows_kernel<kSelCapLarge, kSelThreadsWide, true, E>), dim3((unsigned)blocks),
                         dim3(kSelThreadsWide), 0, stream, scores, ld, st, rs, od);
    return hipGetLastError();
  }
  const bool small = od.m <= kSelCapSmall / 2, sample = lim_max + 1 >= kSampleMinLen;
  const dim3 grid((unsigned)blocks), block(kSelThreads);
  if constexpr (sizeof(E) == 2) {  // bf16 rows: 6-byte candidates, three workgroups per CU
    // only when every row takes the sampled path (a short row would fall back
    // to a two-level select with the smaller buffer the shared region leaves)
    if (sample && min_limit(st, rs) + 1 >= kSampleMinLen) {
      if (small)
        hipLaunchKernelGGL((topk_rows16_kernel<kSelCapSmall, kSelThreads>), grid, block, 0, stream, scores, ld, st,
                           rs, od);
      else
        hipLaunchKernelGGL((topk_rows16_kernel<kSelCap16, kSelThreads>), grid, block, 0, stream, scores, ld, st, rs,
                           od);
      return hipGetLastError();
    }
  }
  if (small && sample)
    hipLaunchKernelGGL((topk_rows_kernel<kSelCapSmall, kSelThreads, true, E>), grid, block, 0, stream, scores, ld, st, rs,
                       od);
  else if (small)
    hipLaunchKernelGGL((topk_rows_kernel<kSelCapSmall, kSelThreads, false, E>), grid, block, 0, stream, scores, ld, st,
                       rs, od);
  else if (sample)
    hipLaunchKernelGGL((topk_rows_kernel<kSelCapLarge, kSelThreads, true, E>), grid, block, 0, stream, scores, ld, st, rs,
                       od);
  else
    hipLaunchKernelGGL((topk_rows_kernel<kSelCapLarge, kSelThreads, false, E>), grid, block, 0, stream, scores, ld, st,
                       rs, od);
  return hipGetLastError();
}

hipError_t launch_topk(const void* scores, bool scores_bf16, int64_t ld, const SeqTable& st, const RowSpace& rs,
                       const OutDesc& od, int64_t lim_max, void* scratch, size_t scratch_bytes,
                       hipStream_t stream) {
  if (scores_bf16)
    return topk_launch(static_cast<const bf16_t*>(scores), ld, st, rs, od, lim_max, scratch, scratch_bytes, stream);
  return topk_launch(static_cast<const float*>(scores), ld, st, rs, od, lim_max, scratch, scratch_bytes, stream);
}

__global__ void fill_guardrail_kernel(int32_t* base, int width, SeqTable st, int j0, int32_t value) {
  const int j = j0 + blockIdx.x, b = blockIdx.y;
  if (b >= st.n || j >= st.first_proxy[b]) return;
  int32_t* row = base + ((int64_t)st.grp0[b] + j) * width;
  for (int e = threadIdx.x; e < width; e += blockDim.x) row[e] = value;
}

hipError_t launch_fill_guardrail(int32_t* base, int width, const SeqTable& st, int j0, int j1, int32_t value,
                                 hipStream_t stream) {
  if (j1 <= j0 || st.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_guardrail_kernel, dim3((unsigned)(j1 - j0), (unsigned)st.n), dim3(256), 0, stream, base,
                     width, st, j0, value);
  return hipGetLastError();
}

struct CopyDst {
  int32_t* p[kMaxCopyDst];
  int32_t n;
};

// Grid-stride copy of src[0, n) to every destination; vec: every pointer is
// 16-byte aligned, so the bulk moves as int4.
__global__ __launch_bounds__(256) void copy_fanout_kernel(const int32_t* __restrict__ src, CopyDst dst, int64_t n,
                                                          int vec) {
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t tail = 0;
  if (vec) {
    const int64_t n4 = n / 4;
    const int4* s4 = reinterpret_cast<const int4*>(src);
    for (int64_t j = i0; j < n4; j += step) {
      const int4 v = s4[j];
      for (int d = 0; d < dst.n; ++d) reinterpret_cast<int4*>(dst.p[d])[j] = v;
    }
    tail = 4 * n4;
  }
  for (int64_t e = tail + i0; e < n; e += step) {
    const int32_t v = src[e];
    for (int d = 0; d < dst.n; ++d) dst.p[d][e] = v;
  }
}

hipError_t launch_copy_fanout(const int32_t* src, int32_t* const* dst, int n_dst, int64_t n, hipStream_t stream) {
  if (n <= 0 || n_dst <= 0) return hipSuccess;
  if (n_dst > kMaxCopyDst) return hipErrorInvalidValue;
  CopyDst cd;
  memset(&cd, 0, sizeof cd);
  cd.n = n_dst;
  bool vec = (reinterpret_cast<uintptr_t>(src) & 15u) == 0;
  for (int d = 0; d < n_dst; ++d) {
    cd.p[d] = dst[d];
    vec = vec && (reinterpret_cast<uintptr_t>(dst[d]) & 15u) == 0;
  }
  const int64_t units = vec ? std::max<int64_t>(n / 4, 1) : n;
  const int64_t blocks = std::min<int64_t>((units + 255) / 256, 4096);
  hipLaunchKernelGGL(copy_fanout_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, src, cd, n, (int)vec);
  return hipGetLastError();
}

}  // namespace pivot
