// Per-row top-m selection over fp32 score rows (the TopK of Sec. 3.1 and of
// Eqs. 6-7): one 512-thread workgroup per row.
//
// Long rows (n >= kSampleMinLen) are read once when the expected number of
// compacted keys fits in LDS:
//   1 sample   every stride-th 256-byte chunk of the row (at most 8192
//              scores) is held in registers; two histogram passes over the
//              sample (top 12, then next 8 key bits) find a 20-bit prefix
//              `thr` such that at least ts sampled keys have prefix >= thr,
//              where ts is the sample's expected share of m plus four
//              standard deviations;
//   2 compact  one pass over the row appends every key with prefix >= thr to
//              LDS (at most CAP: 4096 for m <= 2048, else 8000);
//   3 select   if the pass found at least m keys (and no more than CAP),
//              they include every key >= the m-th largest of the row, ties
//              included, so block_select() over them is exact; otherwise the
//              row takes the two-pass path below.
// Other rows: two_level_select() (block_select.h) over the row in global
// memory: pass 1 builds a 4096-bin histogram of the top 12 key bits, pass 2
// emits the keys above the threshold bin and compacts that bin into LDS, where
// the remaining bits are resolved (ties: lower position); a threshold bin that
// overflows LDS (e.g. many equal scores) selects directly over the row.
// A row with no more than m valid entries returns all of them, then -1.
#include <algorithm>

#include "block_select.h"
#include "launch.h"

namespace pivot {

constexpr int kSelThreads = 512;
// LDS candidates: 16 KiB histogram + 32 KiB -> three workgroups per CU, or
// + 62.5 KiB -> two
constexpr int kSelCapSmall = 4096;
constexpr int kSelCapLarge = 8000;
constexpr int kSampleMinLen = 16384;  // shorter rows take the two-pass path
constexpr int kChunk4 = 16;           // float4 per sampled chunk (256 bytes)
constexpr int kSampleChunks = 128;    // at most 8192 sampled scores, 16 per thread
constexpr int kSampleV = kSampleChunks * kChunk4 / kSelThreads;

// Elements of a score row, visited with 16-byte vector loads (four in flight
// per thread) when aligned.
struct RowSource {
  const float* row;
  int count;
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
    constexpr int T = kSelThreads;
    const int tid = threadIdx.x;
    if ((reinterpret_cast<uintptr_t>(row) & 15u) == 0) {
      const int n4 = count >> 2;
      const float4* r4 = reinterpret_cast<const float4*>(row);
      auto each = [&](const float4& a, int i) {
        f(float_key(a.x), 4 * i); f(float_key(a.y), 4 * i + 1);
        f(float_key(a.z), 4 * i + 2); f(float_key(a.w), 4 * i + 3);
      };
      int i = tid;
      for (; i + 3 * T < n4; i += 4 * T) {
        const float4 a = r4[i], b = r4[i + T], c = r4[i + 2 * T], d = r4[i + 3 * T];
        each(a, i); each(b, i + T); each(c, i + 2 * T); each(d, i + 3 * T);
      }
      for (; i < n4; i += T) each(r4[i], i);
      for (int e = 4 * n4 + tid; e < count; e += T) f(float_key(row[e]), e);
    } else {
      for (int e = tid; e < count; e += T) f(float_key(row[e]), e);
    }
  }
};

// The sampled keys (positions are not needed).
struct SampleSource {
  uint32_t key[4 * (kSampleV > 0 ? kSampleV : 1)];
  bool ok[kSampleV];
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
#pragma unroll
    for (int v = 0; v < kSampleV; ++v)
      if (ok[v]) {
        f(key[4 * v], 0); f(key[4 * v + 1], 0); f(key[4 * v + 2], 0); f(key[4 * v + 3], 0);
      }
  }
};

// 20-bit key prefix of the ts-th largest sampled key (ts <= sampled count);
// hist: 4096 bins of LDS.
template <class Src>
__device__ uint32_t sample_prefix(const Src& src, uint32_t ts, uint32_t* hist, SelectShared& sh) {
  const int tid = threadIdx.x;
  for (int k = tid; k < 4096; k += kSelThreads) hist[k] = 0;
  __syncthreads();
  src.visit([&](uint32_t key, int32_t) { atomicAdd(&hist[key >> 20], 1u); });
  __syncthreads();
  find_digit<kSelThreads, true>(hist, sh, ts, 4096);
  const uint32_t d1 = sh.digit, rem = ts - sh.before;
  __syncthreads();
  for (int k = tid; k < 256; k += kSelThreads) hist[k] = 0;
  __syncthreads();
  src.visit([&](uint32_t key, int32_t) {
    if ((key >> 20) == d1) atomicAdd(&hist[(key >> 12) & 255u], 1u);
  });
  __syncthreads();
  find_digit<kSelThreads, true>(hist, sh, rem, 256);
  const uint32_t thr = (d1 << 8) | sh.digit;
  __syncthreads();
  return thr;
}

template <int CAP>
__global__ __launch_bounds__(kSelThreads) void topk_rows_kernel(const float* __restrict__ scores, int64_t ld,
                                                                SeqTable st, RowSpace rs, OutDesc od) {
  __shared__ TwoLevelShared<CAP> sh;
  const int nrows = rs.i1 - rs.i0;
  const int b = blockIdx.x / nrows;
  const int i = rs.i0 + blockIdx.x % nrows;
  if (!row_active(st, rs, b, i)) return;
  const int tid = threadIdx.x;
  const int64_t n64 = row_limit(st, rs, b, i) + 1;
  const int n = (int)max((int64_t)0, n64);
  const float* row = scores + ((int64_t)b * nrows + (i - rs.i0)) * ld;
  const int m = od.m;

  int64_t dest0;
  int ndest;
  if (od.fan_g == 0) {
    dest0 = (int64_t)b * od.per_seq + i;
    ndest = 1;
  } else {
    dest0 = (int64_t)b * od.per_seq + (int64_t)i * od.fan_g;
    ndest = min(od.fan_g, od.fan_n - i * od.fan_g);
  }
  auto put = [&](int p, int32_t v) {
    for (int u = 0; u < ndest; ++u) od.base[(dest0 + u) * m + p] = v;
  };
  if (n <= m) {
    for (int p = tid; p < m; p += kSelThreads) put(p, p < n ? p : -1);
    return;
  }
  if (tid == 0) sh.sel.emitted = 0;
  RowSource src{row, n};
  const bool aligned = (reinterpret_cast<uintptr_t>(row) & 15u) == 0;
  if (n >= kSampleMinLen && aligned) {
    const int nch = n / (4 * kChunk4);
    const int stride = max(16, (nch + kSampleChunks - 1) / kSampleChunks);
    const int sch = (nch + stride - 1) / stride;  // chunks 0, stride, 2 stride, ... < nch
    const float4* r4 = reinterpret_cast<const float4*>(row);
    SampleSource smp;
#pragma unroll
    for (int v = 0; v < kSampleV; ++v) {
      const int qi = tid + kSelThreads * v;
      smp.ok[v] = qi < sch * kChunk4;
      const float4 a = smp.ok[v] ? r4[(int64_t)(qi / kChunk4) * stride * kChunk4 + qi % kChunk4]
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
      smp.key[4 * v] = float_key(a.x);
      smp.key[4 * v + 1] = float_key(a.y);
      smp.key[4 * v + 2] = float_key(a.z);
      smp.key[4 * v + 3] = float_key(a.w);
    }
    const int s = sch * 4 * kChunk4;
    const float rm = (float)s * (float)m / (float)n;
    const uint32_t ts = (uint32_t)ceilf(rm + 4.0f * sqrtf(rm)) + 1u;
    // expected compacted count ts n / s: leave room for its spread
    if (ts < (uint32_t)s && (float)ts * (float)n <= 0.8f * (float)CAP * (float)s) {
      const uint32_t thr = sample_prefix(smp, ts, sh.hist, sh.sel);
      if (tid == 0) sh.ncand = 0;
      __syncthreads();
      src.visit([&](uint32_t key, int32_t pos) {
        if ((key >> 12) >= thr) {  // a few percent of the row: plain LDS atomics
          const int c = atomicAdd(&sh.ncand, 1);
          if (c < CAP) {
            sh.ckey[c] = key;
            sh.cpos[c] = pos;
          }
        }
      });
      __syncthreads();
      const int found = sh.ncand;
      __syncthreads();  // every thread has read the count before it is reused
      if (found >= m && found <= CAP) {
        ArraySource<kSelThreads> cand{sh.ckey, sh.cpos, found};
        block_select<kSelThreads, false>(cand, (uint32_t)m, sh.sel, put);
        return;
      }
    }
  }
  two_level_select<kSelThreads>(src, (uint32_t)m, sh, put);
}

// ---------------------------------------------------------------------------
// Split select: rows too few to fill the GPU with one workgroup each (decode:
// 32-64 rows of 131072 scores) are cut into P slices, each a workgroup.
//   1 split_zero    clear each row's global histogram and counters;
//   2 split_hist    per slice: 4096-bin LDS histogram of the top 12 key bits,
//                   merged into the row's global histogram with atomics;
//   3 split_emit    per slice: find the row's threshold bin b1 from the global
//                   histogram; emit keys above b1 (global counter), append keys
//                   in b1 to the row's candidate buffer;
//   4 split_final   per row: block_select() over the candidates (or, if b1
//                   overflowed the buffer, over the whole row).
// Same result as the one-workgroup path: the set of the m largest keys, ties
// to the lower position.
struct SplitRowHeader {
  int32_t emitted;
  int32_t ncand;
  int32_t pad[62];
};

struct SplitScratch {
  uint32_t* hist;          // [rows, 4096]
  SplitRowHeader* head;    // [rows]
  uint32_t* ckey;          // [rows, cap]
  int32_t* cpos;           // [rows, cap]
  int32_t cap;
};

size_t split_scratch_bytes(int64_t rows, int cap) {
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  return up(rows * 4096 * sizeof(uint32_t)) + up(rows * sizeof(SplitRowHeader)) +
         2 * up(rows * (size_t)cap * sizeof(uint32_t));
}

static SplitScratch carve_split(void* base, int64_t rows, int cap) {
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  uint8_t* p = (uint8_t*)base;
  SplitScratch s;
  s.hist = (uint32_t*)p;
  p += up(rows * 4096 * sizeof(uint32_t));
  s.head = (SplitRowHeader*)p;
  p += up(rows * sizeof(SplitRowHeader));
  s.ckey = (uint32_t*)p;
  p += up(rows * (size_t)cap * sizeof(uint32_t));
  s.cpos = (int32_t*)p;
  s.cap = cap;
  return s;
}

// Row r of a launch: sequence and local index, its length, its output rows.
struct RowRef {
  int b, i;
  int n;
  bool active;
  __device__ RowRef(const SeqTable& st, const RowSpace& rs, int r) {
    const int nrows = rs.i1 - rs.i0;
    b = r / nrows;
    i = rs.i0 + r % nrows;
    active = row_active(st, rs, b, i);
    n = active ? (int)max((int64_t)0, row_limit(st, rs, b, i) + 1) : 0;
  }
};

__device__ __forceinline__ void put_index(const OutDesc& od, int b, int i, int p, int32_t v) {
  int64_t dest0;
  int ndest;
  if (od.fan_g == 0) {
    dest0 = (int64_t)b * od.per_seq + i;
    ndest = 1;
  } else {
    dest0 = (int64_t)b * od.per_seq + (int64_t)i * od.fan_g;
    ndest = min(od.fan_g, od.fan_n - i * od.fan_g);
  }
  for (int u = 0; u < ndest; ++u) od.base[(dest0 + u) * od.m + p] = v;
}

__global__ __launch_bounds__(256) void split_zero_kernel(SplitScratch sc, int rows) {
  const int r = blockIdx.x;
  if (r >= rows) return;
  for (int k = threadIdx.x; k < 4096; k += 256) sc.hist[(int64_t)r * 4096 + k] = 0;
  if (threadIdx.x == 0) {
    sc.head[r].emitted = 0;
    sc.head[r].ncand = 0;
  }
}

__device__ __forceinline__ void slice_of(int n, int P, int part, int& lo, int& hi) {
  const int per = ((n + P - 1) / P + 3) & ~3;  // multiple of 4: aligned vector loads
  lo = min(n, part * per);
  hi = min(n, lo + per);
}

__global__ __launch_bounds__(256) void split_hist_kernel(const float* __restrict__ scores, int64_t ld, SeqTable st,
                                                         RowSpace rs, int m, int P, SplitScratch sc) {
  __shared__ uint32_t hist[4096];
  const int r = blockIdx.y, part = blockIdx.x;
  RowRef rr(st, rs, r);
  if (!rr.active || rr.n <= m) return;
  int lo, hi;
  slice_of(rr.n, P, part, lo, hi);
  for (int k = threadIdx.x; k < 4096; k += 256) hist[k] = 0;
  __syncthreads();
  const float* row = scores + (int64_t)r * ld;
  for (int e = lo + 4 * (int)threadIdx.x; e < hi; e += 1024) {
    if (e + 4 <= hi) {
      const float4 v = *reinterpret_cast<const float4*>(row + e);
      atomicAdd(&hist[float_key(v.x) >> 20], 1u);
      atomicAdd(&hist[float_key(v.y) >> 20], 1u);
      atomicAdd(&hist[float_key(v.z) >> 20], 1u);
      atomicAdd(&hist[float_key(v.w) >> 20], 1u);
    } else {
      for (int x = e; x < hi; ++x) atomicAdd(&hist[float_key(row[x]) >> 20], 1u);
    }
  }
  __syncthreads();
  uint32_t* g = sc.hist + (int64_t)r * 4096;
  for (int k = threadIdx.x; k < 4096; k += 256)
    if (hist[k]) atomicAdd(&g[k], hist[k]);
}

// Threshold bin of row r from its global histogram (every thread gets it).
struct Threshold {
  uint32_t b1, above, in_b1;
};

__device__ Threshold row_threshold(const uint32_t* g, uint32_t m, uint32_t* wsum, Threshold* out) {
  constexpr int PER = 16;  // 4096 bins / 256 threads
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  uint32_t h[PER];
  uint32_t tot = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    h[k] = g[PER * tid + k];
    tot += h[k];
  }
  uint32_t s = tot;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t t = __shfl_down(s, o, 64);
    if (lane + o < 64) s += t;
  }
  if (lane == 0) wsum[wv] = s;
  __syncthreads();
  uint32_t above = s - tot;
  for (int w = wv + 1; w < 4; ++w) above += wsum[w];
#pragma unroll
  for (int k = PER - 1; k >= 0; --k) {
    if (above < m && m <= above + h[k]) *out = Threshold{(uint32_t)(PER * tid + k), above, h[k]};
    above += h[k];
  }
  __syncthreads();
  return *out;
}

__global__ __launch_bounds__(256) void split_emit_kernel(const float* __restrict__ scores, int64_t ld, SeqTable st,
                                                         RowSpace rs, OutDesc od, int P, SplitScratch sc) {
  __shared__ uint32_t wsum[4];
  __shared__ Threshold th;
  __shared__ int32_t n_above, n_equal, base_above, base_equal;
  const int r = blockIdx.y, part = blockIdx.x;
  RowRef rr(st, rs, r);
  if (!rr.active || rr.n <= od.m) return;
  const Threshold t = row_threshold(sc.hist + (int64_t)r * 4096, (uint32_t)od.m, wsum, &th);
  if (t.in_b1 > (uint32_t)sc.cap) return;  // split_final selects over the whole row
  int lo, hi;
  slice_of(rr.n, P, part, lo, hi);
  const float* row = scores + (int64_t)r * ld;
  SplitRowHeader* head = sc.head + r;
  uint32_t* ck = sc.ckey + (int64_t)r * sc.cap;
  int32_t* cp = sc.cpos + (int64_t)r * sc.cap;
  // count this slice's keys above / in the threshold bin, reserve both ranges
  // with one global atomic each, then write (a slice is a few thousand keys,
  // so the second read hits the cache)
  if (threadIdx.x == 0) n_above = n_equal = 0;
  __syncthreads();
  int my_above = 0, my_equal = 0;
  for (int e = lo + (int)threadIdx.x; e < hi; e += 256) {
    const uint32_t top = float_key(row[e]) >> 20;
    my_above += top > t.b1;
    my_equal += top == t.b1;
  }
  if (my_above) atomicAdd(&n_above, my_above);
  if (my_equal) atomicAdd(&n_equal, my_equal);
  __syncthreads();
  if (threadIdx.x == 0) {
    base_above = n_above ? atomicAdd(&head->emitted, n_above) : 0;
    base_equal = n_equal ? atomicAdd(&head->ncand, n_equal) : 0;
    n_above = n_equal = 0;
  }
  __syncthreads();
  for (int e = lo + (int)threadIdx.x; e < hi; e += 256) {
    const uint32_t key = float_key(row[e]);
    const uint32_t top = key >> 20;
    wave_append(top > t.b1, &n_above, [&](int slot) { put_index(od, rr.b, rr.i, base_above + slot, e); });
    wave_append(top == t.b1, &n_equal, [&](int slot) {
      ck[base_equal + slot] = key;
      cp[base_equal + slot] = e;
    });
  }
}

struct GlobalArraySource {
  const uint32_t* key;
  const int32_t* pos;
  int count;
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
    for (int e = threadIdx.x; e < count; e += 256) f(key[e], pos[e]);
  }
};

struct GlobalRowSource {
  const float* row;
  int count;
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
    for (int e = threadIdx.x; e < count; e += 256) f(float_key(row[e]), e);
  }
};

__global__ __launch_bounds__(256) void split_final_kernel(const float* __restrict__ scores, int64_t ld, SeqTable st,
                                                          RowSpace rs, OutDesc od, SplitScratch sc) {
  __shared__ uint32_t wsum[4];
  __shared__ Threshold th;
  __shared__ SelectShared sel;
  const int r = blockIdx.x;
  RowRef rr(st, rs, r);
  if (!rr.active) return;
  const int m = od.m;
  if (rr.n <= m) {
    for (int p = threadIdx.x; p < m; p += 256) put_index(od, rr.b, rr.i, p, p < rr.n ? p : -1);
    return;
  }
  const Threshold t = row_threshold(sc.hist + (int64_t)r * 4096, (uint32_t)m, wsum, &th);
  SplitRowHeader* head = sc.head + r;
  if (threadIdx.x == 0) sel.emitted = (t.in_b1 <= (uint32_t)sc.cap) ? head->emitted : 0;
  __syncthreads();
  auto put = [&](int slot, int32_t p) { put_index(od, rr.b, rr.i, slot, p); };
  if (t.in_b1 <= (uint32_t)sc.cap) {
    GlobalArraySource src{sc.ckey + (int64_t)r * sc.cap, sc.cpos + (int64_t)r * sc.cap, head->ncand};
    block_select<256, false>(src, (uint32_t)m - t.above, sel, put);
  } else {
    GlobalRowSource src{scores + (int64_t)r * ld, rr.n};
    block_select<256, false>(src, (uint32_t)m, sel, put);
  }
}

hipError_t launch_topk(const float* scores, int64_t ld, const SeqTable& st, const RowSpace& rs,
                       const OutDesc& od, void* scratch, size_t scratch_bytes, int64_t lim_max,
                       hipStream_t stream) {
  const int nrows = rs.i1 - rs.i0;
  if (nrows <= 0 || st.n <= 0) return hipSuccess;
  const int64_t blocks = (int64_t)st.n * nrows;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
  if (scratch && blocks <= kSplitMaxRows && lim_max + 1 >= kSplitMinLen &&
      split_scratch_bytes(blocks, kSplitCap) <= scratch_bytes) {
    const int rows = (int)blocks;
    const int P = (int)std::max<int64_t>(1, std::min<int64_t>(64, 2048 / rows));
    SplitScratch sc = carve_split(scratch, rows, kSplitCap);
    hipLaunchKernelGGL(split_zero_kernel, dim3(rows), dim3(256), 0, stream, sc, rows);
    hipLaunchKernelGGL(split_hist_kernel, dim3(P, rows), dim3(256), 0, stream, scores, ld, st, rs, od.m, P, sc);
    hipLaunchKernelGGL(split_emit_kernel, dim3(P, rows), dim3(256), 0, stream, scores, ld, st, rs, od, P, sc);
    hipLaunchKernelGGL(split_final_kernel, dim3(rows), dim3(256), 0, stream, scores, ld, st, rs, od, sc);
    return hipGetLastError();
  }
  if (od.m <= kSelCapSmall / 2)
    hipLaunchKernelGGL(topk_rows_kernel<kSelCapSmall>, dim3((unsigned)blocks), dim3(kSelThreads), 0, stream, scores,
                       ld, st, rs, od);
  else
    hipLaunchKernelGGL(topk_rows_kernel<kSelCapLarge>, dim3((unsigned)blocks), dim3(kSelThreads), 0, stream, scores,
                       ld, st, rs, od);
  return hipGetLastError();
}

__global__ void fill_guardrail_kernel(int32_t* base, int per_seq, int width, SeqTable st, int j0, int32_t value) {
  const int j = j0 + blockIdx.x, b = blockIdx.y;
  if (b >= st.n || j >= st.first_proxy[b]) return;
  int32_t* row = base + ((int64_t)b * per_seq + j) * width;
  for (int e = threadIdx.x; e < width; e += blockDim.x) row[e] = value;
}

hipError_t launch_fill_guardrail(int32_t* base, int per_seq, int width, const SeqTable& st, int j0, int j1,
                                 int32_t value, hipStream_t stream) {
  if (j1 <= j0 || st.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_guardrail_kernel, dim3((unsigned)(j1 - j0), (unsigned)st.n), dim3(256), 0, stream, base,
                     per_seq, width, st, j0, value);
  return hipGetLastError();
}

}  // namespace pivot
