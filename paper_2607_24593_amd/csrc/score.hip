// Lightning-indexer scoring kernel for gfx950 (Sec. 3.1 Eq. 1; App. A fp8 form).
//
// One workgroup = 4 waves.  A wave keeps R query rows (all 64 heads x 128
// dims) in registers as MFMA A operands and streams 16-key fragments of the
// sequence's keys straight from global memory (each lane loads 32 contiguous
// bytes; a fragment is one contiguous 2 KiB (fp8) block).  The ReLU, the
// gate-and-scale weighting and the head reduction run in the MFMA epilogue
// (mfma_tile.h), so every (row, key) pair leaves the kernel as one fp32.
//
// Two wave arrangements:
//   rows mode  (>= 16 rows per sequence, prefill): the 4 waves hold 4 different
//              row groups and walk the same keys, so a key fragment is fetched
//              from L2 once and served to 4 waves from the vector L1;
//   keys mode  (< 16 rows per sequence, decode): the 4 waves hold the same rows
//              and split the keys.
// Grid: x = key segment, y = row block.  Linear workgroup ids are dealt to the
// 8 XCDs round robin, so with a segment count that is a multiple of 8 each XCD
// always streams the same 1/8 of the keys and keeps it in its own L2.
#include "launch.h"
#include "mfma_tile.h"

namespace pivot {

template <int DT, int R, bool KSPLIT>
__global__ __launch_bounds__(256) void score_kernel(const uint8_t* __restrict__ q,
                                                    const float* __restrict__ q_scale,
                                                    const float* __restrict__ w,
                                                    const uint8_t* __restrict__ lin,
                                                    const float* __restrict__ lin_scale, int64_t q_seq_rows,
                                                    const uint8_t* __restrict__ k,
                                                    const float* __restrict__ k_scale, int64_t k_seq_stride,
                                                    SeqTable st, RowSpace rs, float* __restrict__ out,
                                                    int64_t ld, int seg_keys) {
  using Tile = RowTile<DT, R>;
  constexpr int EB = Tile::EB;
  constexpr int RB = KSPLIT ? R : 4 * R;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nrows = rs.i1 - rs.i0;
  const int nbps = (nrows + RB - 1) / RB;
  const int b = blockIdx.y / nbps;
  if (b >= st.n) return;
  const int i_w = rs.i0 + (blockIdx.y % nbps) * RB + (KSPLIT ? 0 : wave * R);

  int64_t lim_max = -1;
#pragma unroll
  for (int r = 0; r < R; ++r)
    if (row_active(st, rs, b, i_w + r)) lim_max = max(lim_max, row_limit(st, rs, b, i_w + r));
  const int64_t seg0 = (int64_t)blockIdx.x * seg_keys;
  if (lim_max < seg0) return;  // waves are independent: no workgroup barrier follows
  const int64_t seg1 = min(seg0 + (int64_t)seg_keys, lim_max + 1);

  const uint8_t* rows[R];
  const float* wrows[R];
  const uint8_t* lrows[R];
  const float* lsc[R];
  float qs[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    int64_t i = min((int64_t)(i_w + r), q_seq_rows - 1);
    int64_t row = (int64_t)b * q_seq_rows + i;
    rows[r] = q + row * Tile::ROW_BYTES;
    wrows[r] = w + row * kH;
    qs[r] = (DT == kFp8) ? q_scale[row] : 1.0f;
    lrows[r] = (DT == kFp8) ? lin + row * kLinBytes : nullptr;
    lsc[r] = (DT == kFp8) ? lin_scale + row * kLinLevels : nullptr;
  }
  Tile tile;
  tile.load(rows, wrows, qs, lrows, lsc, lane);

  const uint8_t* kb = k + (int64_t)b * k_seq_stride * kD * EB;
  const float* ksb = (DT == kFp8) ? k_scale + (int64_t)b * k_seq_stride : nullptr;
  const int lr = lane & 15, kg = lane >> 4;
  const int qr = kg / Tile::G;
  const int my_i = i_w + qr;
  const bool writer = (kg % Tile::G) == 0 && row_active(st, rs, b, my_i);
  const int64_t my_lim = row_limit(st, rs, b, my_i);
  float* orow = out + ((int64_t)b * nrows + (my_i - rs.i0)) * ld;

  // Two key fragments alternate: while one is scored the other is loading
  // (the second wave on the SIMD covers the rest of the latency).  Loads past
  // the segment are clamped to a valid key (their data is never used), so no
  // load is conditional.
  const int64_t S = KSPLIT ? 64 : 16;
  int64_t t = seg0 + (KSPLIT ? 16 * wave : 0);
  auto key_at = [&](int64_t base) { return kb + min(base + lr, lim_max) * kD * EB; };
  auto emit = [&](float acc, int64_t base) {
    // keep the epilogue ahead of the store's branch (no sinking into it)
    asm volatile("" : "+v"(acc));
    const int64_t s = base + lr;
    if (writer && s <= my_lim) {
      if constexpr (DT == kFp8) acc *= ksb[s];
      orow[s] = acc;
    }
  };
  KeyFrag<DT> f0, f1;
  f0.load(key_at(t), kg);
  f1.load(key_at(t + S), kg);
  for (; t < seg1; t += 2 * S) {
    emit(tile.score(f0), t);
    f0.load(key_at(t + 2 * S), kg);
    if (t + S >= seg1) break;
    emit(tile.score(f1), t + S);
    f1.load(key_at(t + 3 * S), kg);
  }
}

template <int DT, int R, bool KSPLIT>
static hipError_t run_score(const void* q, const float* qs, const float* w, const uint8_t* lin, const float* lsc,
                            int64_t q_seq_rows, const void* k, const float* ks, int64_t kstride, const SeqTable& st,
                            const RowSpace& rs, int64_t lim_max, float* out, int64_t ld, int seg,
                            hipStream_t stream) {
  constexpr int RB = KSPLIT ? R : 4 * R;
  const int nrows = rs.i1 - rs.i0;
  const int64_t nseg = ((lim_max + 1 + seg - 1) / seg + 7) / 8 * 8;
  const int64_t nblk = (int64_t)st.n * ((nrows + RB - 1) / RB);
  if (nseg > 0x7FFFFFFF || nblk > 65535) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((score_kernel<DT, R, KSPLIT>), dim3((unsigned)nseg, (unsigned)nblk), dim3(256), 0, stream,
                     (const uint8_t*)q, qs, w, lin, lsc, q_seq_rows, (const uint8_t*)k, ks, kstride, st, rs, out,
                     ld, seg);
  return hipGetLastError();
}

hipError_t launch_score(int dtype, const void* q, const float* q_scale, const float* w, const uint8_t* lin,
                        const float* lin_scale, int64_t q_seq_rows, const void* k, const float* k_scale,
                        int64_t k_seq_stride, const SeqTable& st, const RowSpace& rs, int64_t lim_max, float* out,
                        int64_t ld, hipStream_t stream) {
  const int nrows = rs.i1 - rs.i0;
  if (nrows <= 0 || lim_max < 0 || st.n <= 0) return hipSuccess;
  if (dtype == kFp8) {
    if (nrows >= 16)
      return run_score<kFp8, 4, false>(q, q_scale, w, lin, lin_scale, q_seq_rows, k, k_scale, k_seq_stride, st, rs, lim_max,
                                       out, ld, 4096, stream);
    if (nrows == 1)
      return run_score<kFp8, 1, true>(q, q_scale, w, lin, lin_scale, q_seq_rows, k, k_scale, k_seq_stride, st, rs, lim_max,
                                      out, ld, 2048, stream);
    if (nrows == 2)
      return run_score<kFp8, 2, true>(q, q_scale, w, lin, lin_scale, q_seq_rows, k, k_scale, k_seq_stride, st, rs, lim_max,
                                      out, ld, 2048, stream);
    return run_score<kFp8, 4, true>(q, q_scale, w, lin, lin_scale, q_seq_rows, k, k_scale, k_seq_stride, st, rs, lim_max, out,
                                    ld, 2048, stream);
  }
  if (nrows >= 16)
    return run_score<kBf16, 2, false>(q, nullptr, w, nullptr, nullptr, q_seq_rows, k, nullptr, k_seq_stride, st, rs, lim_max,
                                      out, ld, 2048, stream);
  if (nrows == 1)
    return run_score<kBf16, 1, true>(q, nullptr, w, nullptr, nullptr, q_seq_rows, k, nullptr, k_seq_stride, st, rs, lim_max,
                                     out, ld, 2048, stream);
  return run_score<kBf16, 2, true>(q, nullptr, w, nullptr, nullptr, q_seq_rows, k, nullptr, k_seq_stride, st, rs, lim_max, out,
                                   ld, 2048, stream);
}

}  // namespace pivot
