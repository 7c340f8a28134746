// Lightning-indexer scoring kernel for gfx950 (Sec. 3.1 Eq. 1; App. A fp8 form).
//
// One workgroup = 4 waves.  A wave keeps R query rows (all 64 heads x 128
// dims) in registers as MFMA A operands and scores 16-key fragments of the
// sequence's keys against them (a lane takes 32 contiguous bytes of a key
// row per MFMA step; a fragment is one contiguous 2 KiB (fp8) or 4 KiB
// (bf16) block).  The ReLU, the
// gate-and-scale weighting and the head reduction run in the MFMA epilogue
// (mfma_tile.h), so every (row, key) pair leaves the kernel as one fp32, or
// one bf16 (round to nearest even) where the caller asks for bf16 score rows.
//
// Two wave arrangements:
//   rows mode  (>= 16 rows per sequence, prefill): the 4 waves hold 4 different
//              row groups and walk the same keys, so the workgroup fetches
//              each key once into LDS and the 4 waves read it from there;
//   keys mode  (< 16 rows per sequence, decode): the 4 waves hold the same rows
//              and split the keys, each loading its fragments from global
//              memory into registers.
// Grid: rows mode runs a 1-D grid whose linear index is segment * row blocks
// + row block, so consecutive workgroups take the row blocks of one key
// segment: dispatched round-robin over the 8 XCDs, the ~64 workgroups resident
// on an XCD share one or two segments in its L2, and the causal triangle's
// active (row block, segment) pairs still spread evenly over the XCDs
// (pinning segments to XCDs would idle the XCDs that own the late segments of
// short prefixes).  Keys mode runs x = key segment, y = sequence.  The segment
// length adapts to the launch size.
#include <climits>

#include "launch.h"
#include "mfma_tile.h"

namespace pivot {

// A key offset past every paged pool (pools stay below 2^31 bytes): its
// loads read zeros, and adding a fragment's lane offset cannot wrap it.
constexpr uint32_t kDropOffset = 0x80000000u;

// Rows mode stages keys through LDS 8 KiB at a time: 64 fp8 or 32 bf16 keys,
// each row padded by 16 bytes; a thread fetches two 16-byte pieces per stage.
template <int DT>
constexpr int kStageKeys = DT == kFp8 ? 64 : 32;
template <int DT>
constexpr int kPassKeys = 256 * 16 / (kD * (DT == kFp8 ? 1 : 2));  // keys of one 16-byte piece per thread
template <int DT>
constexpr int kPieces = kStageKeys<DT> / kPassKeys<DT>;
template <int DT>
constexpr int kStageSlot = kStageKeys<DT> * (kD * (DT == kFp8 ? 1 : 2) + 16);

// OB16: scores leave as bf16 (RNE) instead of fp32.
template <int DT, int R, bool KSPLIT, bool PAGED, bool OB16>
__global__ __launch_bounds__(256) void score_kernel(const uint8_t* __restrict__ q,
                                                    const float* __restrict__ q_scale,
                                                    const float* __restrict__ w,
                                                    const uint8_t* __restrict__ lin,
                                                    const float* __restrict__ lin_scale,
                                                    const uint8_t* __restrict__ k,
                                                    const float* __restrict__ k_scale, KeyMap km,
                                                    SeqTable st, RowSpace rs, void* __restrict__ out,
                                                    int64_t ld, int seg_keys) {
  constexpr int SE = OB16 ? 2 : 4;  // bytes per score
  using Tile = RowTile<DT, R>;
  constexpr int EB = Tile::EB;
  constexpr int KB = kD * EB;  // bytes per key
  constexpr int RB = KSPLIT ? R : 4 * R;
  // the segment's key scales (fp8); a key index never reaches 4096 (rows
  // mode: at most 64 stages of 64 keys; keys mode: 2048-key segments plus
  // two fragment strides), and 32 spare words keep a stray read inside
  __shared__ float sks[4096 + 32];
  __shared__ __align__(16) uint8_t kst[KSPLIT ? 16 : 3 * kStageSlot<DT>];  // rows mode: staged keys
  __shared__ int32_t spg[PAGED ? 256 : 1];  // the segment's pages (paged keys; a segment of <= 4096 keys
                                            // starts on a page boundary or lies inside one page)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
  const int nrows = rs.i1 - rs.i0;
  const int nbps = (nrows + RB - 1) / RB;
  const uint32_t nblk = (uint32_t)(st.n * nbps);
  const uint32_t yb = KSPLIT ? blockIdx.y : blockIdx.x % nblk;  // row block
  const uint32_t xs = KSPLIT ? blockIdx.x : blockIdx.x / nblk;  // key segment
  const int b = (int)(yb / nbps);
  if (b >= st.n) return;
  const int i_blk = rs.i0 + (int)(yb % nbps) * RB;
  const int64_t seg0 = (int64_t)xs * seg_keys;

  // the workgroup's key range (uniform, so every wave reaches the barrier)
  int64_t lim_blk = -1;
  for (int r = 0; r < RB; ++r)
    if (row_active(st, rs, b, i_blk + r)) lim_blk = max(lim_blk, row_limit(st, rs, b, i_blk + r));
  if (lim_blk < seg0) return;
  const int nseg_keys = (int)(min(seg0 + (int64_t)seg_keys, lim_blk + 1) - seg0);

  const int i_w = i_blk + (KSPLIT ? 0 : wave * R);
  int64_t lim_max = -1;
#pragma unroll
  for (int r = 0; r < R; ++r)
    if (row_active(st, rs, b, i_w + r)) lim_max = max(lim_max, row_limit(st, rs, b, i_w + r));
  // this wave's keys (0: the wave only helps stage the key scales)
  const int nkeys = lim_max < seg0 ? 0 : (int)(min(seg0 + (int64_t)seg_keys, lim_max + 1) - seg0);

  const uint8_t* rows[R];
  const float* wrows[R];
  const uint8_t* lrows[R];
  const float* lsc[R];
  float qs[R];
  const int last = row_count(st, rs, b) - 1;  // >= 0: the workgroup has an active row
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row_index(st, rs, b, min(i_w + r, last));
    rows[r] = q + row * Tile::ROW_BYTES;
    wrows[r] = w + row * kH;
    qs[r] = (DT == kFp8) ? q_scale[row] : 1.0f;
    lrows[r] = (DT == kFp8) ? lin + row * kLinBytes : nullptr;
    lsc[r] = (DT == kFp8) ? lin_scale + row * kLinLevels : nullptr;
  }
  // The segment's key scales, the row tile and the first key fragments are
  // all requested before the one workgroup barrier, the scales first (all 16
  // loads of a thread in flight at once, range-checked), so their latencies
  // overlap and the scales can be written to LDS without waiting for the rest.
  constexpr int KS_PER = 4096 / 256;
  float ksv[KS_PER];
  if constexpr (DT == kFp8 && !PAGED) {
    const __amdgpu_buffer_rsrc_t ksr = buffer_rsrc(k_scale + km.row(b, seg0), (uint32_t)nseg_keys * 4);
#pragma unroll
    for (int u = 0; u < KS_PER; ++u)
      ksv[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ksr, (uint32_t)(tid + 256 * u) * 4u, 0, 0));
  }
  if constexpr (DT == kFp8 && PAGED) {  // gathered through the page table
#pragma unroll
    for (int u = 0; u < KS_PER; ++u) {
      const int e = tid + 256 * u;
      ksv[u] = e < nseg_keys ? k_scale[km.row(b, seg0 + e)] : 0.0f;
    }
  }
  Tile tile;
  tile.load(rows, wrows, qs, lrows, lsc, lane);

  // keys through a range-checked buffer resource with 32-bit offsets: the
  // segment's contiguous keys (reads past the workgroup's last key in rows
  // mode, the wave's in keys mode, return zeros), or the page pool (such keys
  // are sent to kDropOffset)
  const __amdgpu_buffer_rsrc_t kr =
      PAGED ? buffer_rsrc(k, (uint32_t)(((int64_t)km.n_pages << km.shift) * KB))
            : buffer_rsrc(k + km.row(b, seg0) * KB, (uint32_t)(KSPLIT ? nkeys : nseg_keys) * KB);
  // e: key index within the segment; the prologue reads the page table in
  // global memory, the loop the segment's pages staged in LDS
  const int64_t page0 = PAGED ? seg0 >> km.shift : 0;
  if constexpr (PAGED) {
    const int n_ent = (int)(((seg0 + nseg_keys - 1) >> km.shift) - page0 + 1);
    if (tid < n_ent) spg[tid] = min(max(km.pages[(int64_t)b * km.max_pages + page0 + tid], 0), km.n_pages - 1);
  }
  auto key_off0 = [&](int e) -> uint32_t {
    if constexpr (PAGED) return e < nkeys ? (uint32_t)(km.row(b, seg0 + e) * KB) : kDropOffset;
    else return (uint32_t)e * KB;
  };
  auto key_off = [&](int e) -> uint32_t {
    if constexpr (PAGED) {
      if (e >= nkeys) return kDropOffset;
      const int64_t s = seg0 + e;
      return (uint32_t)((((int64_t)spg[(s >> km.shift) - page0] << km.shift) | (s & ((1 << km.shift) - 1))) * KB);
    } else {
      return (uint32_t)e * KB;
    }
  };
  const int lr = lane & 15, kg = lane >> 4;
  const int qr = kg / Tile::G;
  const int my_i = i_w + qr;
  const bool writer = (kg % Tile::G) == 0 && row_active(st, rs, b, my_i);
  const int my_n = (int)min((int64_t)nkeys, row_limit(st, rs, b, my_i) + 1 - seg0);  // keys this row takes
  // Scores leave through a buffer resource over the wave's R output rows:
  // lanes with nothing to store give an offset past its end, which the
  // hardware drops.  Every lane issues the same stores, so the count of
  // outstanding memory operations never depends on the data and the waits
  // before each fragment stay exact.  (The host keeps R * ld * 4 < 2^31.)
  const __amdgpu_buffer_rsrc_t orr =
      buffer_rsrc((uint8_t*)out + (((int64_t)b * nrows + (i_w - rs.i0)) * ld + seg0) * SE,
                  (uint32_t)(((int64_t)(R - 1) * ld + nkeys) * SE));
  const uint32_t my_off = (uint32_t)((int64_t)qr * ld * SE) + (uint32_t)SE * (uint32_t)lr;
  // key base + lr is stored when base < my_lim (the fragment's base is the
  // same in every lane, so the test is one compare against a lane constant)
  const int my_lim = writer ? my_n - lr : INT_MIN;

  auto emit = [&](float acc, int base) {
    if constexpr (DT == kFp8) acc *= sks[base + lr];
    const uint32_t off = base < my_lim ? my_off + (uint32_t)SE * (uint32_t)base : 0xFFFFFFFFu;
    if constexpr (OB16)
      __builtin_amdgcn_raw_buffer_store_b16(bf16_rne(acc), orr, off, 0, 0);
    else
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc), orr, off, 0, 0);
  };
  if constexpr (KSPLIT) {
    // keys mode: each wave walks its own 16-key fragments, three rotating
    // (one scored while the next two load).  The loop body has no exits, so
    // the compiler keeps each reload right after the fragment's last use;
    // fragments past the wave's keys read zeros and their stores are dropped.
    constexpr int S = 64;
    int t = 16 * wave;  // key offset within the segment
    KeyFrag<DT> f0, f1, f2;
    f0.load(kr, key_off0(t + lr), kg);
    f1.load(kr, key_off0(t + S + lr), kg);
    f2.load(kr, key_off0(t + 2 * S + lr), kg);
    if constexpr (DT == kFp8) {
#pragma unroll
      for (int u = 0; u < KS_PER; ++u) sks[tid + 256 * u] = ksv[u];  // zeros past the segment
      __syncthreads();
    } else if constexpr (PAGED) {
      __syncthreads();  // the staged pages
    }
    for (; t < nkeys; t += 3 * S) {
      emit(tile.score(f0), t);
      f0.load(kr, key_off(t + 3 * S + lr), kg);
      emit(tile.score(f1), t + S);
      f1.load(kr, key_off(t + 4 * S + lr), kg);
      emit(tile.score(f2), t + 2 * S);
      f2.load(kr, key_off(t + 5 * S + lr), kg);
    }
  } else {
    // rows mode: the 4 waves score the same keys, so the workgroup fetches
    // each 8 KiB stage of keys once (every thread two 16-byte pieces, the
    // stage one contiguous block) and the waves read their fragments from
    // LDS.  Three LDS slots rotate with one barrier per stage: stage i + 1 is
    // written while stage i is scored, and the slot it overwrites held stage
    // i - 2, which every wave finished before the previous barrier.  Each
    // thread has the next stage's loads in flight while a stage is scored
    // (one register set: more would cost the tile's occupancy of two waves
    // per SIMD).  Key rows sit KB + 16 bytes apart in LDS, so
    // the 16 rows of a fragment start in 16 different 16-byte bank groups.
    // Every wave runs every stage of the workgroup's key range (the barriers
    // are uniform).
    const int nst = (nseg_keys + kStageKeys<DT> - 1) / kStageKeys<DT>;
    const int my_key = tid / (KB / 16), my_piece = tid % (KB / 16);
    uint8_t* const put_at = kst + my_key * (KB + 16) + 16 * my_piece;
    struct Pieces {
      v4i p[kPieces<DT>];
    };
    // prologue fetches (before the first barrier) read the page table in
    // global memory, later ones the copy staged in LDS
    auto fetch = [&](int st_i, bool prologue = false) -> Pieces {
      Pieces r;
#pragma unroll
      for (int h = 0; h < kPieces<DT>; ++h) {
        const int e = st_i * kStageKeys<DT> + h * kPassKeys<DT> + my_key;
        uint32_t off;
        if constexpr (PAGED) {
          if (e >= nseg_keys) {
            off = kDropOffset;
          } else if (prologue) {
            off = (uint32_t)(km.row(b, seg0 + e) * KB);
          } else {
            const int64_t s = seg0 + e;
            off = (uint32_t)((((int64_t)spg[(s >> km.shift) - page0] << km.shift) | (s & ((1 << km.shift) - 1))) * KB);
          }
        } else {
          off = (uint32_t)e * KB;  // past the segment: zeros (range-checked resource)
        }
        r.p[h] = __builtin_amdgcn_raw_buffer_load_b128(kr, off + 16 * my_piece, 0, 0);
      }
      return r;
    };
    auto put = [&](const Pieces& r, int slot) {
#pragma unroll
      for (int h = 0; h < kPieces<DT>; ++h)
        *reinterpret_cast<v4i*>(put_at + slot * kStageSlot<DT> + h * kPassKeys<DT> * (KB + 16)) = r.p[h];
    };
    Pieces r = fetch(0, true);
    if constexpr (DT == kFp8) {
#pragma unroll
      for (int u = 0; u < KS_PER; ++u) sks[tid + 256 * u] = ksv[u];  // zeros past the segment
    }
    put(r, 0);
    r = fetch(1, true);
    __syncthreads();
    // r holds stage i + 1 on entry; stage s sits in slot s % 3
    auto stage = [&](int i, int slot_put, int slot) {
      put(r, slot_put);  // stage i + 1
      r = fetch(i + 2);
      __syncthreads();
      const int t = i * kStageKeys<DT>;
#pragma unroll
      for (int f = 0; f < kStageKeys<DT> / 16; ++f) {
        KeyFrag<DT> fr;
        fr.load(kst + slot * kStageSlot<DT> + (16 * f + lr) * (KB + 16), kg);
        emit(tile.score(fr), t + 16 * f);
      }
    };
    // Every stage issues the same loads and stores (a wave's stages past its
    // own keys are scored too, their stores dropped; rows of a workgroup end
    // within 16 keys of each other), so the compiler's memory-counter waits
    // stay exact across the loop and each staged register waits only for its
    // own load.
    int i = 0;
    for (; i + 3 <= nst; i += 3) {
      stage(i, 1, 0);
      stage(i + 1, 2, 1);
      stage(i + 2, 0, 2);
    }
    if (i < nst) stage(i, 1, 0);
    if (i + 1 < nst) stage(i + 1, 2, 1);
  }
}

// Workgroups one launch should have for the machine to stay busy through the
// causal tail: 256 CUs x 2 resident workgroups x 4 rounds.
constexpr int64_t kTargetWorkgroups = 2048;

template <int DT, int R, bool KSPLIT, bool OB16>
static hipError_t run_score(const void* q, const float* qs, const float* w, const uint8_t* lin, const float* lsc,
                            const void* k, const float* ks, const KeyMap& km, const SeqTable& st,
                            const RowSpace& rs, int64_t lim_max, void* out, int64_t ld, int max_seg,
                            hipStream_t stream) {
  constexpr int RB = KSPLIT ? R : 4 * R;
  const int nrows = rs.i1 - rs.i0;
  const int64_t nblk = (int64_t)st.n * ((nrows + RB - 1) / RB);
  // Longest key segment that still gives kTargetWorkgroups (down to 512 keys);
  // longer segments amortise the row-tile load over more keys.
  int seg = max_seg;  // <= 4096: the key scales of a segment are staged in LDS
  while (seg > 512 && nblk * ((lim_max + seg) / seg) < kTargetWorkgroups) seg >>= 1;
  const int64_t nseg = (lim_max + seg) / seg;
  if (KSPLIT ? (nseg > 0x7FFFFFFF || nblk > 65535) : nseg * nblk > 0x7FFFFFFF)
    return hipErrorInvalidConfiguration;
  const dim3 grid = KSPLIT ? dim3((unsigned)nseg, (unsigned)nblk) : dim3((unsigned)(nseg * nblk));
  if (km.pages)
    hipLaunchKernelGGL((score_kernel<DT, R, KSPLIT, true, OB16>), grid, dim3(256), 0, stream, (const uint8_t*)q, qs,
                       w, lin, lsc, (const uint8_t*)k, ks, km, st, rs, out, ld, seg);
  else
    hipLaunchKernelGGL((score_kernel<DT, R, KSPLIT, false, OB16>), grid, dim3(256), 0, stream, (const uint8_t*)q, qs,
                       w, lin, lsc, (const uint8_t*)k, ks, km, st, rs, out, ld, seg);
  return hipGetLastError();
}

template <bool OB16>
static hipError_t score_fp8(const void* q, const float* q_scale, const float* w, const uint8_t* lin,
                            const float* lin_scale, const void* k, const float* k_scale, const KeyMap& km,
                            const SeqTable& st, const RowSpace& rs, int64_t lim_max, void* out, int64_t ld,
                            hipStream_t stream) {
  const int nrows = rs.i1 - rs.i0;
  if (nrows >= 16)
    return run_score<kFp8, 4, false, OB16>(q, q_scale, w, lin, lin_scale, k, k_scale, km, st, rs, lim_max, out,
                                           ld, 4096, stream);
  if (nrows == 1)
    return run_score<kFp8, 1, true, OB16>(q, q_scale, w, lin, lin_scale, k, k_scale, km, st, rs, lim_max, out,
                                          ld, 2048, stream);
  if (nrows == 2)
    return run_score<kFp8, 2, true, OB16>(q, q_scale, w, lin, lin_scale, k, k_scale, km, st, rs, lim_max, out,
                                          ld, 2048, stream);
  return run_score<kFp8, 4, true, OB16>(q, q_scale, w, lin, lin_scale, k, k_scale, km, st, rs, lim_max, out, ld,
                                        2048, stream);
}

hipError_t launch_score(int dtype, const void* q, const float* q_scale, const float* w, const uint8_t* lin,
                        const float* lin_scale, const void* k, const float* k_scale, const KeyMap& km,
                        const SeqTable& st, const RowSpace& rs, int64_t lim_max, void* out, bool out_bf16,
                        int64_t ld, hipStream_t stream) {
  const int nrows = rs.i1 - rs.i0;
  if (nrows <= 0 || lim_max < 0 || st.n <= 0) return hipSuccess;
  if (dtype == kFp8)
    return out_bf16 ? score_fp8<true>(q, q_scale, w, lin, lin_scale, k, k_scale, km, st, rs, lim_max, out, ld, stream)
                    : score_fp8<false>(q, q_scale, w, lin, lin_scale, k, k_scale, km, st, rs, lim_max, out, ld,
                                       stream);
  if (out_bf16) return hipErrorInvalidValue;  // bf16 inputs keep fp32 scores
  if (nrows >= 16)
    return run_score<kBf16, 2, false, false>(q, nullptr, w, nullptr, nullptr, k, nullptr, km, st, rs, lim_max,
                                             out, ld, 2048, stream);
  if (nrows == 1)
    return run_score<kBf16, 1, true, false>(q, nullptr, w, nullptr, nullptr, k, nullptr, km, st, rs, lim_max,
                                            out, ld, 2048, stream);
  return run_score<kBf16, 2, true, false>(q, nullptr, w, nullptr, nullptr, k, nullptr, km, st, rs, lim_max, out,
                                          ld, 2048, stream);
}

}  // namespace pivot
