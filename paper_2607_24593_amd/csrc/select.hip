// Per-row top-m selection over fp32 score rows (the TopK of Sec. 3.1 and of
// Eqs. 6-7): one 512-thread workgroup per row.
//
// two_level_select() (block_select.h) over the row in global memory, read with
// 16-byte vector loads: pass 1 builds a 4096-bin histogram of the top 12 key
// bits, pass 2 emits the keys above the threshold bin and compacts that bin
// into LDS, where the remaining bits are resolved (ties: lower position).  Rows
// whose threshold bin overflows LDS (e.g. many equal scores) select directly
// over the row.
// A row with no more than m valid entries returns all of them, then -1.
#include "block_select.h"
#include "launch.h"

namespace pivot {

constexpr int kSelThreads = 512;
constexpr int kSelCap = 6144;  // LDS: 16 KiB histogram + 48 KiB candidates -> two workgroups per CU

// Elements of a score row, visited with 16-byte vector loads when aligned.
struct RowSource {
  const float* row;
  int count;
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
    const int tid = threadIdx.x;
    if ((reinterpret_cast<uintptr_t>(row) & 15u) == 0) {
      const int n4 = count >> 2;
      const float4* r4 = reinterpret_cast<const float4*>(row);
      int i = tid;
      for (; i + kSelThreads < n4; i += 2 * kSelThreads) {
        const float4 a = r4[i], b = r4[i + kSelThreads];
        const int j = i + kSelThreads;
        f(float_key(a.x), 4 * i); f(float_key(a.y), 4 * i + 1);
        f(float_key(a.z), 4 * i + 2); f(float_key(a.w), 4 * i + 3);
        f(float_key(b.x), 4 * j); f(float_key(b.y), 4 * j + 1);
        f(float_key(b.z), 4 * j + 2); f(float_key(b.w), 4 * j + 3);
      }
      for (; i < n4; i += kSelThreads) {
        const float4 a = r4[i];
        f(float_key(a.x), 4 * i); f(float_key(a.y), 4 * i + 1);
        f(float_key(a.z), 4 * i + 2); f(float_key(a.w), 4 * i + 3);
      }
      for (int e = 4 * n4 + tid; e < count; e += kSelThreads) f(float_key(row[e]), e);
    } else {
      for (int e = tid; e < count; e += kSelThreads) f(float_key(row[e]), e);
    }
  }
};

__global__ __launch_bounds__(kSelThreads) void topk_rows_kernel(const float* __restrict__ scores, int64_t ld,
                                                                SeqTable st, RowSpace rs, OutDesc od) {
  __shared__ TwoLevelShared<kSelCap> sh;
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
  two_level_select<kSelThreads>(src, (uint32_t)m, sh, [&](int32_t p) { put(atomicAdd(&sh.sel.emitted, 1), p); });
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
