// Per-row top-m selection over fp32 score rows (the TopK of Sec. 3.1 and of
// Eqs. 6-7): one 512-thread workgroup per row.
//
//   pass 1  stream the row (16-B vector loads) into a 4096-bin LDS histogram of
//           the top 12 bits of the order-preserving key; one wave finds the bin
//           b1 holding the m-th largest key;
//   pass 2  stream the row again: keys above b1 are emitted at once, keys in b1
//           are compacted into LDS (at most CAP of them);
//   final   block_select() resolves the remaining bits of b1's candidates in
//           LDS, with ties broken by lower position.
// Rows whose bin b1 holds more than CAP keys (e.g. many equal scores) run
// block_select() directly over the row in global memory instead.
// A row with no more than m valid entries returns all of them, then -1.
#include "block_select.h"
#include "launch.h"

namespace pivot {

constexpr int kSelThreads = 512;
constexpr int kSelCap = 6144;  // LDS: 16 KiB histogram + 48 KiB candidates -> two workgroups per CU

struct TopkShared {
  uint32_t hist[4096];
  uint32_t ckey[kSelCap];
  int32_t cpos[kSelCap];
  SelectShared sel;
  uint32_t b1, above, in_b1;
  int32_t ncand;
};

struct RowSource {
  const float* row;
  int count;
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
    for (int e = threadIdx.x; e < count; e += kSelThreads) f(float_key(row[e]), e);
  }
};

// Visit every element of row[0, n) as (position, key); vector loads when aligned.
template <class F>
__device__ __forceinline__ void for_each_key(const float* row, int n, F f) {
  const int tid = threadIdx.x;
  if ((reinterpret_cast<uintptr_t>(row) & 15u) == 0) {
    const int n4 = n >> 2;
    const float4* r4 = reinterpret_cast<const float4*>(row);
    int i = tid;
    for (; i + kSelThreads < n4; i += 2 * kSelThreads) {
      float4 a = r4[i], b = r4[i + kSelThreads];
      f(4 * i, float_key(a.x)); f(4 * i + 1, float_key(a.y));
      f(4 * i + 2, float_key(a.z)); f(4 * i + 3, float_key(a.w));
      const int j = i + kSelThreads;
      f(4 * j, float_key(b.x)); f(4 * j + 1, float_key(b.y));
      f(4 * j + 2, float_key(b.z)); f(4 * j + 3, float_key(b.w));
    }
    for (; i < n4; i += kSelThreads) {
      float4 a = r4[i];
      f(4 * i, float_key(a.x)); f(4 * i + 1, float_key(a.y));
      f(4 * i + 2, float_key(a.z)); f(4 * i + 3, float_key(a.w));
    }
    for (int e = 4 * n4 + tid; e < n; e += kSelThreads) f(e, float_key(row[e]));
  } else {
    for (int e = tid; e < n; e += kSelThreads) f(e, float_key(row[e]));
  }
}

__global__ __launch_bounds__(kSelThreads) void topk_rows_kernel(const float* __restrict__ scores, int64_t ld,
                                                                SeqTable st, RowSpace rs, OutDesc od) {
  __shared__ TopkShared sh;
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

  for (int k = tid; k < 4096; k += kSelThreads) sh.hist[k] = 0;
  if (tid == 0) {
    sh.sel.emitted = 0;
    sh.ncand = 0;
  }
  __syncthreads();
  for_each_key(row, n, [&](int, uint32_t key) { atomicAdd(&sh.hist[key >> 20], 1u); });
  __syncthreads();
  // bin b1 where the count from the top crosses m (one wave, 64 bins per lane)
  if (tid < 64) {
    uint32_t tot = 0;
    for (int k = 0; k < 64; ++k) tot += sh.hist[64 * tid + k];
    uint32_t s = tot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      uint32_t t = __shfl_down(s, o, 64);
      if (tid + o < 64) s += t;
    }
    uint32_t above = s - tot;
    const uint32_t need = (uint32_t)m;
    for (int k = 63; k >= 0; --k) {
      const uint32_t h = sh.hist[64 * tid + k];
      if (above < need && need <= above + h) {
        sh.b1 = 64 * tid + k;
        sh.above = above;
        sh.in_b1 = h;
      }
      above += h;
    }
  }
  __syncthreads();
  const uint32_t b1 = sh.b1, above = sh.above, in_b1 = sh.in_b1;
  auto emit = [&](int32_t p) { put(atomicAdd(&sh.sel.emitted, 1), p); };

  if (in_b1 <= (uint32_t)kSelCap) {
    for_each_key(row, n, [&](int e, uint32_t key) {
      const uint32_t top = key >> 20;
      if (top > b1) {
        emit(e);
      } else if (top == b1) {
        const int c = atomicAdd(&sh.ncand, 1);
        sh.ckey[c] = key;
        sh.cpos[c] = e;
      }
    });
    __syncthreads();
    ArraySource<kSelThreads> src{sh.ckey, sh.cpos, sh.ncand};
    block_select<kSelThreads>(src, (uint32_t)m - above, sh.sel, emit);
  } else {
    RowSource src{row, n};
    block_select<kSelThreads>(src, (uint32_t)m, sh.sel, emit);
  }
}

hipError_t launch_topk(const float* scores, int64_t ld, const SeqTable& st, const RowSpace& rs,
                       const OutDesc& od, hipStream_t stream) {
  const int nrows = rs.i1 - rs.i0;
  if (nrows <= 0 || st.n <= 0) return hipSuccess;
  const int64_t blocks = (int64_t)st.n * nrows;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(topk_rows_kernel, dim3((unsigned)blocks), dim3(kSelThreads), 0, stream, scores, ld, st, rs,
                     od);
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
