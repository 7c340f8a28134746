// PIVOT-Refine fine step (Sec. 4.4 Eqs. 8-9): every member of a group
// re-scores the group's candidate set C with its own query and gates and keeps
// its own top-k.
//
// One workgroup (4 waves) per group.  Members are taken four at a time: the
// four rows sit in every wave's registers as MFMA A operands (mfma_tile.h) and
// the waves split C into 16-candidate fragments, each lane gathering 32 bytes
// of one candidate key by index.  Scores are kept in LDS as order-preserving
// keys (four rows of |C|), then block_select() takes each member's top-k with
// ties broken by lower position.
#include "block_select.h"
#include "launch.h"
#include "mfma_tile.h"

namespace pivot {

struct CandSource {
  const uint32_t* key;
  const int32_t* pos;
  int count;
  __device__ int n() const { return count; }
  __device__ void get(int e, uint32_t& k, int32_t& p) const {
    k = key[e];
    p = pos[e];
  }
};

template <int DT>
__global__ __launch_bounds__(256) void refine_kernel(const uint8_t* __restrict__ q,
                                                     const float* __restrict__ q_scale,
                                                     const float* __restrict__ w,
                                                     const uint8_t* __restrict__ lin,
                                                     const float* __restrict__ lin_scale, int n_q, int g,
                                                     int n_groups, const uint8_t* __restrict__ k,
                                                     const float* __restrict__ k_scale, int64_t k_seq_stride,
                                                     SeqTable st, int j0, const int32_t* __restrict__ cand, int c,
                                                     int m, int32_t* __restrict__ out_idx) {
  using Tile = RowTile<DT, 4>;
  constexpr int EB = Tile::EB;
  extern __shared__ uint32_t skeys[];  // [4][c]
  __shared__ SelectShared sel;
  const int j = j0 + blockIdx.x, b = blockIdx.y;
  if (b >= st.n || j >= n_groups || j < st.first_proxy[b]) return;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t t0 = (int64_t)st.q_pos0[b] + (int64_t)j * g;
  const int nc = (int)min((int64_t)c, t0 + 1);
  const int gs = min(g, n_q - j * g);
  const int32_t* crow = cand + ((int64_t)b * n_groups + j) * c;
  const int64_t r0 = (int64_t)b * n_q + (int64_t)j * g;
  const uint8_t* kb = k + (int64_t)b * k_seq_stride * kD * EB;
  const float* ksb = (DT == kFp8) ? k_scale + (int64_t)b * k_seq_stride : nullptr;
  const int lr = lane & 15, kg = lane >> 4;

  for (int quad = 0; quad * 4 < gs; ++quad) {
    const int rows_here = min(4, gs - 4 * quad);
    const uint8_t* rows[4];
    const float* wrows[4];
    const uint8_t* lrows[4];
    const float* lsc[4];
    float qs[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = r0 + 4 * quad + min(r, rows_here - 1);
      rows[r] = q + row * Tile::ROW_BYTES;
      wrows[r] = w + row * kH;
      qs[r] = (DT == kFp8) ? q_scale[row] : 1.0f;
      lrows[r] = (DT == kFp8) ? lin + row * kLinBytes : nullptr;
      lsc[r] = (DT == kFp8) ? lin_scale + row * kLinLevels : nullptr;
    }
    Tile tile;
    tile.load(rows, wrows, qs, lrows, lsc, lane);
    const int nfrag = (nc + 15) >> 4;
    int f = wave;
    KeyFrag<DT> cur, nxt;
    int32_t s_cur = 0, s_nxt = 0;
    if (f < nfrag) {
      s_cur = crow[min(16 * f + lr, nc - 1)];
      cur.load(kb + (int64_t)s_cur * kD * EB, kg);
    }
    for (; f < nfrag; f += 4) {
      const int fn = f + 4;
      if (fn < nfrag) {
        s_nxt = crow[min(16 * fn + lr, nc - 1)];
        nxt.load(kb + (int64_t)s_nxt * kD * EB, kg);
      }
      float acc = tile.score(cur);
      asm volatile("" : "+v"(acc));  // keep the epilogue ahead of the store's branch
      const int slot = 16 * f + lr;
      if (slot < nc && kg < rows_here) {
        if constexpr (DT == kFp8) acc *= ksb[s_cur];
        skeys[kg * c + slot] = float_key(acc);
      }
      cur = nxt;
      s_cur = s_nxt;
    }
    __syncthreads();
    for (int r = 0; r < rows_here; ++r) {
      int32_t* orow = out_idx + (r0 + 4 * quad + r) * m;
      if (tid == 0) sel.emitted = 0;
      __syncthreads();
      const int need = min(m, nc);
      CandSource src{skeys + r * c, crow, nc};
      block_select<256>(src, (uint32_t)need, sel, [&](int32_t p) { orow[atomicAdd(&sel.emitted, 1)] = p; });
      for (int p = need + tid; p < m; p += 256) orow[p] = -1;
    }
    __syncthreads();
  }
}

hipError_t launch_refine(int dtype, const void* q, const float* q_scale, const float* w, const uint8_t* lin,
                         const float* lin_scale, int n_q, int g, int n_groups, const void* k,
                         const float* k_scale, int64_t k_seq_stride,
                         const SeqTable& st, int j0, int j1, const int32_t* cand, int c, int m,
                         int32_t* out_idx, hipStream_t stream) {
  if (j1 <= j0 || st.n <= 0) return hipSuccess;
  const size_t lds = (size_t)4 * c * sizeof(uint32_t);
  dim3 grid((unsigned)(j1 - j0), (unsigned)st.n);
  if (dtype == kFp8) {
    (void)hipFuncSetAttribute((const void*)refine_kernel<kFp8>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(refine_kernel<kFp8>, grid, dim3(256), lds, stream, (const uint8_t*)q, q_scale, w, lin, lin_scale,
                       n_q, g, n_groups, (const uint8_t*)k, k_scale, k_seq_stride, st, j0, cand, c, m, out_idx);
  } else {
    (void)hipFuncSetAttribute((const void*)refine_kernel<kBf16>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(refine_kernel<kBf16>, grid, dim3(256), lds, stream, (const uint8_t*)q, q_scale, w, lin, lin_scale,
                       n_q, g, n_groups, (const uint8_t*)k, k_scale, k_seq_stride, st, j0, cand, c, m, out_idx);
  }
  return hipGetLastError();
}

}  // namespace pivot
