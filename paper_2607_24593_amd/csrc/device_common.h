// Shared device-side definitions of the gfx950 PIVOT indexer kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pivot {

constexpr int kH = 64;        // indexer heads (the only H this build specialises)
constexpr int kD = 128;       // head dimension
constexpr int kMaxSeq = 64;   // sequences per launch (the host splits larger batches)
constexpr int kWave = 64;     // CDNA wavefront size

enum Dtype : int { kBf16 = 0, kFp8 = 1 };

// Sequences of one launch, passed by value as a kernel argument.  Positions of
// row i of sequence b are q_pos0[b] + i * step (RowSpace.step).
struct SeqTable {
  int32_t n;
  int32_t q_pos0[kMaxSeq];
  int32_t dense_rows[kMaxSeq];   // query rows [0, dense_rows) go through the dense path
  int32_t first_proxy[kMaxSeq];  // groups [first_proxy, n_groups) go through the proxy path
};

// The rows one launch covers: for every sequence b < SeqTable.n, the local rows
// [i0, i1).  Output/score row of (b, i) is b * (i1 - i0) + (i - i0).
struct RowSpace {
  int32_t i0, i1;
  int32_t step;     // position step between consecutive local rows
  int32_t kind;     // kAll, kDenseRows, kProxyRows
};
enum RowKind : int { kAll = 0, kDenseRows = 1, kProxyRows = 2 };

__device__ __forceinline__ bool row_active(const SeqTable& st, const RowSpace& rs, int b, int i) {
  if (b >= st.n || i < rs.i0 || i >= rs.i1) return false;
  if (rs.kind == kDenseRows) return i < st.dense_rows[b];
  if (rs.kind == kProxyRows) return i >= st.first_proxy[b];
  return true;
}

__device__ __forceinline__ int64_t row_limit(const SeqTable& st, const RowSpace& rs, int b, int i) {
  return (int64_t)st.q_pos0[b] + (int64_t)i * rs.step;
}

// Order-preserving map of a float onto uint32 (larger float -> larger key);
// -0 and +0 map to the same key.
__device__ __forceinline__ uint32_t float_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) == 0u) return 0x80000000u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Wavefront reductions (wave64) through cross-lane shuffles.
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

}  // namespace pivot
