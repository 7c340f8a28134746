// Register-resident query rows and one 16-key MFMA step of the lightning-indexer
// score (Sec. 3.1 Eq. 1; fp8 form of App. A):
//
//   S(row, s) = kscale[s] * sum_j (w[row, j] * qscale[row]) * ReLU(q[row, j] . k[s])
//
// Layout.  The inner products of R query rows x 64 heads against 16 keys form
// a (64 R) x 16 matrix computed as 4R MFMA tiles of 16 (row, head) pairs x 16
// keys, with K = d = 128 (one v_mfma_f32_16x16x128_f8f6f4, or four
// v_mfma_f32_16x16x32_bf16).  The accumulator of a 16x16 MFMA puts tile rows
// 4q .. 4q+3 in lane group q (lanes 16q .. 16q+15), key n in lane 16q + n.
// Tile rows are assigned so that every lane group belongs to ONE query row:
// with G = 4/R lane groups per row, tile j row 4q + i is head
// 4G j + 4 (q mod G) + i of query row q / G.  Each lane therefore folds its
// heads into fp32 sums with no cross-lane traffic; only G > 1 needs log2(G)
// shuffles per 16 keys at the end.
//
// Summation order.  Every tile shape adds a (row, key) pair's 64 heads in the
// same order, so a score has the same bits whichever R computed it (the
// dense, proxy and Refine launches pick R by their row counts): four partial
// sums P_p, p = 0..3, each an FMA chain over heads 16 j + 4 p + i (j, then i,
// ascending), combined as ((P_0 + P_1) + P_2) + P_3; the fp8 linear term is
// added last.  With G lane groups per row a lane holds R = 4 / G of the
// partials (tile j feeds partial j mod R) and shuffles bring in the others.
//
// fp8 epilogue.  With x = q8 . k8 and w' = w * qscale,
//   sum_j w'_j ReLU(x_j) = sum_j (w'_j / 2) |x_j|  +  u . k8,
//   u = sum_j (w'_j / 2) q8_j   (a 128-vector per row),
// because ReLU(x) = (x + |x|) / 2.  The first sum costs one FMA per element
// (|x| is a free source modifier) instead of a max and an FMA.  The second is
// linear in the key: u is stored as four fp8 levels u ~ sum_l sigma_l c_l
// (each level quantises the residual of the previous ones at a scale 16x
// finer, sigma_l = sigma_0 16^-l, so the error is below 2^-19 of max|u|),
// and one more MFMA tile per 16 keys computes c_l . k8 for the R rows'
// levels, combined as sigma_0 (c_0 + 2^-4 c_1 + 2^-8 c_2 + 2^-12 c_3).  bf16 rows use (w/2)|x| + (w/2)x directly (two FMAs).
//
// K split.  Lane l supplies dims 32 (l / 16) .. 32 (l / 16) + 31 of its A row
// and of its B column.  Any assignment of dims to (lane group, register slot)
// gives the same product as long as A and B use the same one.
#pragma once

#include "device_common.h"

namespace pivot {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kLinLevels = 4;
constexpr int kLinBytes = kLinLevels * kD;  // fp8 codes of the four levels of u, per row
// sigma_l / sigma_0 of the levels (powers of two, so the products are exact)
__device__ constexpr float kLinStep[kLinLevels] = {1.0f, 0x1p-4f, 0x1p-8f, 0x1p-12f};

template <int DT>
struct KeyFrag;

// Buffer resource over [base, base + bytes): buffer loads through it are
// range-checked by the hardware (reads past the end return zero).
// A pointer that is the same in every lane, moved to scalar registers (so a
// buffer resource built from it needs no per-lane loop).
template <class P>
__device__ __forceinline__ P* uniform_ptr(P* p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)u);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(u >> 32));
  return reinterpret_cast<P*>(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

template <>
struct KeyFrag<kFp8> {
  v8i v;  // 32 E4M3 codes
  __device__ __forceinline__ void load(const uint8_t* key_row, int kg) {
    const v4i* p = reinterpret_cast<const v4i*>(key_row + 32 * kg);
    v4i lo = p[0], hi = p[1];
    v = v8i{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
  }
  // key at byte offset `row_off` of the resource, this lane's 32 bytes
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t row_off, int kg) {
    v4i lo = __builtin_amdgcn_raw_buffer_load_b128(r, row_off + 32 * kg, 0, 0);
    v4i hi = __builtin_amdgcn_raw_buffer_load_b128(r, row_off + 32 * kg + 16, 0, 0);
    v = v8i{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
  }
};

template <>
struct KeyFrag<kBf16> {
  v4i v[4];  // 4 x 8 bf16
  __device__ __forceinline__ void load(const uint8_t* key_row, int kg) {
    const v4i* p = reinterpret_cast<const v4i*>(key_row + 64 * kg);
#pragma unroll
    for (int s = 0; s < 4; ++s) v[s] = p[s];
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t row_off, int kg) {
#pragma unroll
    for (int s = 0; s < 4; ++s) v[s] = __builtin_amdgcn_raw_buffer_load_b128(r, row_off + 64 * kg + 16 * s, 0, 0);
  }
};

__device__ __forceinline__ v4f mfma_fp8(const v8i& a, const v8i& b) {
  const v4f z = {0.f, 0.f, 0.f, 0.f};
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, z, 0, 0, 0, 0, 0, 0);
}

template <int DT, int R>
struct RowTile {
  static_assert(R == 1 || R == 2 || R == 4, "rows per wave");
  static constexpr int G = 4 / R;        // lane groups per query row
  static constexpr int T = 4 * R;        // MFMA tiles (16 (row, head) pairs each)
  static constexpr int EB = DT == kFp8 ? 1 : 2;
  static constexpr int ROW_BYTES = kH * kD * EB;

  KeyFrag<DT> a[T];   // A operand, same register format as a key fragment
  float wv[T][4];     // w * qscale / 2 (bf16: qscale = 1)
  KeyFrag<kFp8> al;   // fp8: the four levels of u of the wave's rows
  float ls0;          // fp8: sigma_0 of this lane's row (0 in non-owning lane groups)

  // rows[r]: the R query rows' codes; wrow[r]: gates; qscale[r]: per-row scale;
  // lin[r] / lscale[r]: the rows' levels of u and their scales (fp8 only).
  __device__ __forceinline__ void load(const uint8_t* const* rows, const float* const* wrow,
                                       const float* qscale, const uint8_t* const* lin,
                                       const float* const* lscale, int lane) {
    const int lr = lane & 15, kg = lane >> 4;
    const int gq_a = lr >> 2, i_a = lr & 3;
    const uint8_t* arow = rows[gq_a / G];
#pragma unroll
    for (int j = 0; j < T; ++j) {
      const int head = 4 * G * j + 4 * (gq_a % G) + i_a;
      a[j].load(arow + (size_t)head * kD * EB, kg);
    }
    const int gq = kg;
    const int qr = gq / G;
    const float* wr = wrow[qr];
    const float sc = (DT == kFp8) ? qscale[qr] * 0.5f : 0.5f;
#pragma unroll
    for (int j = 0; j < T; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) wv[j][i] = wr[4 * G * j + 4 * (gq % G) + i] * sc;
    if constexpr (DT == kFp8) {
      al.load(lin[gq_a / G] + i_a * kD, kg);
      ls0 = (gq % G) == 0 ? lscale[qr][0] : 0.f;
    }
  }

  // Gate-weighted ReLU sum over all heads of row (lane >> 4) / G for key
  // (lane & 15) of the fragment b, in the lanes that store it (lane group
  // (lane >> 4) % G == 0; the other lane groups of the row lack the fp8
  // linear term).  Tile R j'' + p feeds partial p, j'' ascending.  The fp8
  // 4-row tile keeps its four partials live and visits the tiles in natural
  // order; the other shapes visit them partial by partial, so a partial's
  // FMA chain runs without a break and is folded as soon as it ends (two
  // sums live).  Every shape adds a partial's terms in the same order.
  static constexpr int TPR = T / R;  // tiles per partial
  __device__ __forceinline__ static constexpr int tile_at(int jj) { return R * (jj % TPR) + jj / TPR; }

  // Folds partial p, just finished in `part`, into ((P_0 + P_1) + P_2) + P_3:
  // `hold` carries the running sum, `tot` receives the whole sum with the
  // last partial (valid in the lane groups that store the row).
  __device__ __forceinline__ static void fold(int p, float part, float& hold, float& tot) {
    if constexpr (R == 4) {  // partials in order, one lane
      if (p == 0) hold = part;
      if (p == 1 || p == 2) hold = hold + part;
      if (p == 3) tot = hold + part;
    } else if constexpr (R == 2) {  // lane group parity q holds P_q (p = 0) and P_{2+q} (p = 1)
      // v_permlane16_swap of a value with itself leaves, in every lane, the
      // even lane group's value of the pair in the first result and the odd
      // one's in the second
      const auto e = __builtin_amdgcn_permlane16_swap(__float_as_uint(part), __float_as_uint(part), false, false);
      const float even = __uint_as_float(e[0]), odd = __uint_as_float(e[1]);
      if (p == 0) hold = even + odd;   // P_0 + P_1
      else tot = (hold + even) + odd;  // + P_2, + P_3
    } else {  // lane group q holds P_q; lane group 0 gathers the others
      // after the 16-lane swap: (P_0 | P_2) and (P_1 | P_3) in each half;
      // the 32-lane swaps bring the upper half's values (P_2, P_3) down
      const auto e = __builtin_amdgcn_permlane16_swap(__float_as_uint(part), __float_as_uint(part), false, false);
      const auto h0 = __builtin_amdgcn_permlane32_swap(e[0], e[0], false, false);
      const auto h1 = __builtin_amdgcn_permlane32_swap(e[1], e[1], false, false);
      tot = ((__uint_as_float(e[0]) + __uint_as_float(e[1])) + __uint_as_float(h0[1])) + __uint_as_float(h1[1]);
    }
  }

  __device__ __forceinline__ float score(const KeyFrag<DT>& b) const {
    float part = 0.f, hold = 0.f, tot = 0.f;
    if constexpr (DT == kFp8) {
      // Software pipeline: the MFMA of the tile two ahead is issued before the
      // epilogue of the current one, so the matrix core and the VALU work side
      // by side with three accumulators live.  The scheduling barriers keep
      // the compiler from hoisting all MFMAs ahead (which would need 4 (T+1)
      // accumulator registers and push operands into AGPRs).
      if constexpr (R == 4) {
        // four partial sums live, tiles in natural order (tile j feeds
        // partial j % 4): each partial still sees its tiles and heads in
        // the same order, but consecutive tiles no longer wait on each other
        float ps[4] = {0.f, 0.f, 0.f, 0.f};
        v4f cl = mfma_fp8(al.v, b.v);
        v4f c0 = mfma_fp8(a[0].v, b.v);
        v4f c1 = mfma_fp8(a[1].v, b.v);
#pragma unroll
        for (int jj = 2; jj <= T + 1; ++jj) {
          v4f nxt = c1;
          if (jj < T) nxt = mfma_fp8(a[jj].v, b.v);
          __builtin_amdgcn_sched_barrier(0);
          const int e = jj - 2;
#pragma unroll
          for (int i = 0; i < 4; ++i) ps[e % 4] = fmaf(wv[e][i], fabsf(c0[i]), ps[e % 4]);
          asm volatile("" : "+v"(ps[e % 4]));
          __builtin_amdgcn_sched_barrier(0);
          c0 = c1;
          c1 = nxt;
        }
        tot = ((ps[0] + ps[1]) + ps[2]) + ps[3];
        const float lin = fmaf(cl[3], kLinStep[3], fmaf(cl[2], kLinStep[2], fmaf(cl[1], kLinStep[1], cl[0])));
        return fmaf(ls0, lin, tot);
      }
      v4f cl = mfma_fp8(al.v, b.v);
      v4f c0 = mfma_fp8(a[tile_at(0)].v, b.v);
      v4f c1 = mfma_fp8(a[tile_at(1)].v, b.v);
#pragma unroll
      for (int jj = 2; jj <= T + 1; ++jj) {
        v4f nxt = c1;
        if (jj < T) nxt = mfma_fp8(a[tile_at(jj)].v, b.v);
        __builtin_amdgcn_sched_barrier(0);
        const int e = jj - 2, j = tile_at(e);
#pragma unroll
        for (int i = 0; i < 4; ++i) part = fmaf(wv[j][i], fabsf(c0[i]), part);
        asm volatile("" : "+v"(part));  // pins this epilogue between the barriers
        __builtin_amdgcn_sched_barrier(0);
        if ((e + 1) % TPR == 0) {
          fold(e / TPR, part, hold, tot);
          part = 0.f;
        }
        c0 = c1;
        c1 = nxt;
      }
      // the levels' dot products, finest first scaled in, then sigma_0
      const float lin = fmaf(cl[3], kLinStep[3], fmaf(cl[2], kLinStep[2], fmaf(cl[1], kLinStep[1], cl[0])));
      return fmaf(ls0, lin, tot);
    } else {
#pragma unroll
      for (int jj = 0; jj < T; ++jj) {
        const int j = tile_at(jj);
        v4f c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 4; ++s)
          c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a[j].v[s]),
                                                      __builtin_bit_cast(v8bf, b.v[s]), c, 0, 0, 0);
        // w ReLU(x) = (w/2) |x| + (w/2) x: two FMAs, no max
#pragma unroll
        for (int i = 0; i < 4; ++i) part = fmaf(wv[j][i], c[i], fmaf(wv[j][i], fabsf(c[i]), part));
        if ((jj + 1) % TPR == 0) {
          fold(jj / TPR, part, hold, tot);
          part = 0.f;
        }
      }
      return tot;
    }
  }
};

}  // namespace pivot
