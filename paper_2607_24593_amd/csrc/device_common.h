// Shared device-side definitions of the gfx950 PIVOT indexer kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pivot {

constexpr int kH = 64;        // indexer heads (the only H this library specialises)
constexpr int kD = 128;       // head dimension
constexpr int kMaxSeq = 64;   // sequences per launch (the host splits larger batches)
constexpr int kWave = 64;     // CDNA wavefront size

enum Dtype : int { kBf16 = 0, kFp8 = 1 };

// Sequences of one launch, passed by value as a kernel argument.  Positions of
// row i of sequence b are q_pos0[b] + i * step (RowSpace.step).  Sequence b
// owns query rows row0[b] .. row0[b] + n_rows[b] - 1 of the launch's query
// arrays (q, q_scale, w, linear terms, outputs) and groups grp0[b] .. of its
// group arrays (proxies, candidate rows); a padded batch has row0 = b n_q.
struct SeqTable {
  int32_t n;
  int32_t q_pos0[kMaxSeq];
  int32_t dense_rows[kMaxSeq];   // query rows [0, dense_rows) go through the dense path
  int32_t first_proxy[kMaxSeq];  // groups [first_proxy, n_groups) go through the proxy path
  int32_t n_rows[kMaxSeq];       // query rows of the sequence in this call
  int32_t row0[kMaxSeq];
  int32_t grp0[kMaxSeq];
};

// Groups of g consecutive query rows of sequence b (the last may be shorter).
__device__ __forceinline__ int seq_groups(const SeqTable& st, int b, int g) { return (st.n_rows[b] + g - 1) / g; }

// The rows one launch covers: for every sequence b < SeqTable.n, the local rows
// [i0, i1).  Score row of (b, i) is b * (i1 - i0) + (i - i0).  Rows of kind
// kProxyRows are groups (step = g), the others query rows.
struct RowSpace {
  int32_t i0, i1;
  int32_t step;     // position step between consecutive local rows
  int32_t kind;     // kAll, kDenseRows, kProxyRows
};
enum RowKind : int { kAll = 0, kDenseRows = 1, kProxyRows = 2 };

// Rows of sequence b of the RowSpace's kind.
__device__ __forceinline__ int row_count(const SeqTable& st, const RowSpace& rs, int b) {
  return rs.kind == kProxyRows ? seq_groups(st, b, rs.step) : st.n_rows[b];
}

__device__ __forceinline__ bool row_active(const SeqTable& st, const RowSpace& rs, int b, int i) {
  if (b >= st.n || i < rs.i0 || i >= rs.i1 || i >= row_count(st, rs, b)) return false;
  if (rs.kind == kDenseRows) return i < st.dense_rows[b];
  if (rs.kind == kProxyRows) return i >= st.first_proxy[b];
  return true;
}

// Index of row (b, i) in the launch's query (or, for kProxyRows, group) arrays.
__device__ __forceinline__ int64_t row_index(const SeqTable& st, const RowSpace& rs, int b, int i) {
  return (int64_t)(rs.kind == kProxyRows ? st.grp0[b] : st.row0[b]) + i;
}

__device__ __forceinline__ int64_t row_limit(const SeqTable& st, const RowSpace& rs, int b, int i) {
  return (int64_t)st.q_pos0[b] + (int64_t)i * rs.step;
}

// Where key s of sequence b of a launch lives in the key arrays: row
// b * stride + s, or, with a page table, row page * page_size + s mod
// page_size with page = pages[b * max_pages + s / page_size] (clamped into
// the pool, so a bad entry cannot address memory outside it).
struct KeyMap {
  const int32_t* pages;  // dev [sequences, max_pages], or nullptr: contiguous keys
  int64_t stride;        // contiguous: key rows between consecutive sequences
  int32_t max_pages;
  int32_t shift;         // log2(page_size)
  int32_t n_pages;       // pages in the pool
  __device__ __forceinline__ int64_t row(int b, int64_t s) const {
    if (!pages) return (int64_t)b * stride + s;
    const int32_t pg = min(max(pages[(int64_t)b * max_pages + (s >> shift)], 0), n_pages - 1);
    return ((int64_t)pg << shift) | (s & ((1 << shift) - 1));
  }
};

// Order-preserving map of a float onto uint32 (larger float -> larger key);
// -0 and +0 map to the same key.
__device__ __forceinline__ uint32_t float_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) == 0u) return 0x80000000u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// bf16 bits of an fp32 value, rounded to nearest even: gfx950's conversion
// instruction (one VALU operation; the same bits as rounding the upper half
// by hand for every finite value, subnormals and overflow to infinity
// included).
__device__ __forceinline__ uint16_t bf16_rne(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

// Score rows hold fp32 or bf16 values (the fp8 path stores bf16 scores); E is
// float or bf16_t (bf16 bits).  A 16-byte vector holds N scores, widened to
// fp32 exactly (a bf16 value is the high half of an fp32 word).
using bf16_t = uint16_t;
template <class E>
struct ScoreVec;
template <>
struct ScoreVec<float> {
  static constexpr int N = 4;
  __device__ static __forceinline__ void unpack(const uint4& a, float (&v)[4]) {
    v[0] = __uint_as_float(a.x); v[1] = __uint_as_float(a.y);
    v[2] = __uint_as_float(a.z); v[3] = __uint_as_float(a.w);
  }
  __device__ static __forceinline__ float one(const float* row, int64_t e) { return row[e]; }
};
template <>
struct ScoreVec<bf16_t> {
  static constexpr int N = 8;
  __device__ static __forceinline__ void unpack(const uint4& a, float (&v)[8]) {
    v[0] = __uint_as_float(a.x << 16); v[1] = __uint_as_float(a.x & 0xFFFF0000u);
    v[2] = __uint_as_float(a.y << 16); v[3] = __uint_as_float(a.y & 0xFFFF0000u);
    v[4] = __uint_as_float(a.z << 16); v[5] = __uint_as_float(a.z & 0xFFFF0000u);
    v[6] = __uint_as_float(a.w << 16); v[7] = __uint_as_float(a.w & 0xFFFF0000u);
  }
  __device__ static __forceinline__ float one(const bf16_t* row, int64_t e) {
    return __uint_as_float((uint32_t)row[e] << 16);
  }
};

// Wavefront reductions (wave64) through cross-lane shuffles.
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

}  // namespace pivot
