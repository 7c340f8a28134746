// PIVOT-Refine fine step (Sec. 4.4 Eqs. 8-9): every member of a group
// re-scores the group's candidate set C with its own query and gates (Eq. 8)
// and keeps its own top-k (Eq. 9).
//
// rescore_kernel: a block of R members of a group (R = 4 for fp8 groups of
// more than two, else 2), held as the A operands of the MFMA row tile
// (mfma_tile.h), scores C in 16-candidate fragments: one wave per block with
// many groups (prefill), or the 4 waves of a workgroup splitting C (decode).  The candidate positions are staged in LDS, so each lane reads
// its position there and gathers 32 bytes of that key (and, for fp8, its
// scale) three fragments ahead of its use.  Scores go to a
// [group, member, |C|] buffer (it stays in the last-level cache for the
// select that follows): bf16 (round to nearest even) for fp8 inputs, like the
// full-prefix score rows, fp32 for bf16 inputs.
//
// topk_short_kernel: one workgroup per (group, member) row of |C| <= 8192
// scores; each thread keeps its share of (key, position) pairs in registers
// (read four at a time: 16-byte position loads, 16- or 8-byte score loads)
// and the bucket select (else block_select()) takes the top-k, ties broken by
// lower position.  The g member rows of a group run as consecutive
// workgroups of one XCD, so the group's candidate positions are read from
// HBM once and then from that XCD's L2.
//
// App. B local window: window_kernel writes the union of the members' windows
// into the candidate row after the proxy's slots.  A candidate row then has
// `width` slots; member t re-scores all of them (empty slots read key 0) and
// its select keeps the slots it may use: position in [0, t], and for a union
// slot of the per-query window also position >= t - W + 1.
#include <algorithm>
#include <climits>

#include "block_select.h"
#include "launch.h"
#include "mfma_tile.h"
#include "pivot.h"

namespace pivot {

constexpr int kMaxCand = 8192;

// WPG: each wave takes its own (group, member block) unit and all of the
// group's candidates (at most kWpgCand), with no workgroup barrier, so a wave
// loads its row tile once per |C| candidates rather than per |C| / 4;
// otherwise the 4 waves of a workgroup share one unit (and slice) and split
// its fragments.
constexpr int kWpgCand = 4096;
// Staged positions run kPosPad entries past a wave's (WPG) or workgroup's
// candidates, holding key 0, so the fetch three fragments ahead (at most
// 5 fragment strides past the loop's last fragment) reads a position without
// clamping its index.
constexpr int kPosPadWpg = 96, kPosPad = 384;

// B32: the keys (and scales) a launch can gather span less than 2^31 bytes,
// so they are read through buffer resources with 32-bit offsets (fewer
// address operations per fragment than 64-bit pointers).
template <int DT, int R, bool OB16, bool WPG, bool B32>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void rescore_kernel(
    const uint8_t* __restrict__ q, const float* __restrict__ q_scale, const float* __restrict__ w,
    const uint8_t* __restrict__ lin, const float* __restrict__ lin_scale, int g,
    const uint8_t* __restrict__ k, const float* __restrict__ k_scale, KeyMap km, SeqTable st, int j0,
    const int32_t* __restrict__ cand, int c, int all_slots, int parts, void* __restrict__ rsc) {
  using Tile = RowTile<DT, R>;
  constexpr uint32_t SE = OB16 ? 2 : 4;  // bytes per stored score
  constexpr int EB = Tile::EB;
  constexpr int PAD = WPG ? kPosPadWpg : kPosPad;
  __shared__ int32_t spos_all[WPG ? 4 * (kWpgCand + kPosPadWpg) : kMaxCand + kPosPad];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
  // members [R blk, R blk + R); candidate fragments of slice `part`
  // WPG: workgroups are dealt round-robin to the 8 XCDs; XCD x % 8 takes a
  // contiguous run of groups (consecutive groups share most candidates, so
  // their gathers hit that XCD's L2); a partial last round keeps its order
  const int nwg = (int)gridDim.x, full = nwg - nwg % 8, bx = (int)blockIdx.x;
  const int wgx = WPG && bx < full ? (bx % 8) * (full / 8) + bx / 8 : bx;
  const int nblk = (g + R - 1) / R, unit = 4 * wgx + wave;
  const int j = j0 + (WPG ? unit / nblk : (int)blockIdx.x), b = blockIdx.y;
  const int blk = WPG ? unit % nblk : (int)blockIdx.z / parts, part = WPG ? 0 : (int)blockIdx.z % parts;
  if (b >= st.n || j >= seq_groups(st, b, g) || j < st.first_proxy[b]) return;
  const int gs = min(g, st.n_rows[b] - j * g);
  if (R * blk >= gs) return;
  int32_t* spos = WPG ? spos_all + wave * (kWpgCand + kPosPadWpg) : spos_all;
  constexpr int ST = WPG ? 64 : 256;  // threads staging the positions
  const int sid = WPG ? lane : tid;
  const int64_t t0 = (int64_t)st.q_pos0[b] + (int64_t)j * g;
  // without a window only the first t0 + 1 slots can hold a position
  const int nc = all_slots ? c : (int)min((int64_t)c, t0 + 1);
  const int rows_here = min(R, gs - R * blk);
  const int64_t grp = (int64_t)st.grp0[b] + j;
  const int32_t* crow = cand + grp * c;
  const int64_t r0 = (int64_t)st.row0[b] + (int64_t)j * g + R * blk;
  // contiguous keys: the sequence's base, staged positions; paged keys: the
  // pool, positions staged as pool rows (empty slots as key 0's row)
  const uint8_t* kb = km.pages ? k : k + km.row(b, 0) * kD * EB;
  const float* ksb = DT == kFp8 ? (km.pages ? k_scale : k_scale + km.row(b, 0)) : nullptr;
  const int lr = lane & 15, kg = lane >> 4;
  const int nfrag_all = (nc + 15) >> 4;
  const int fpp = (nfrag_all + parts - 1) / parts;
  const int fbeg = min(nfrag_all, part * fpp), fend = min(nfrag_all, fbeg + fpp);
  if (fbeg >= fend) return;
  const int cbeg = 16 * fbeg, ncs = min(nc, 16 * fend) - cbeg;  // this slice's candidates
  // positions staged eight per thread at a time: the loads of a batch are
  // issued before the first is used (then, for paged keys, the batch's
  // page-table loads), one or two memory round trips per batch instead of
  // one per element
  for (int e0 = 0; e0 < ncs; e0 += 8 * ST) {
    constexpr int SB = 8;
    int32_t pv[SB];
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const int e = e0 + sid + ST * k;
      pv[k] = e < ncs ? crow[cbeg + e] : 0;
    }
    if (km.pages) {
#pragma unroll
      for (int k = 0; k < SB; ++k)
        if (e0 + sid + ST * k < ncs) pv[k] = (int32_t)km.row(b, max(pv[k], 0));
    }
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const int e = e0 + sid + ST * k;
      if (e < ncs) spos[e] = max(pv[k], 0);  // empty slots (-1): key 0's row
    }
  }
  {
    const int32_t key0 = km.pages ? (int32_t)km.row(b, 0) : 0;
    for (int e = ncs + sid; e < ncs + PAD; e += ST) spos[e] = key0;
  }

  const uint8_t* rows[R];
  const float* wrows[R];
  const uint8_t* lrows[R];
  const float* lsc[R];
  float qs[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = r0 + min(r, rows_here - 1);
    rows[r] = q + row * Tile::ROW_BYTES;
    wrows[r] = w + row * kH;
    qs[r] = (DT == kFp8) ? q_scale[row] : 1.0f;
    lrows[r] = (DT == kFp8) ? lin + row * kLinBytes : nullptr;
    lsc[r] = (DT == kFp8) ? lin_scale + row * kLinLevels : nullptr;
  }
  const int qr = kg / Tile::G;
  const bool writer = (kg % Tile::G) == 0 && qr < rows_here;
  // scores leave through a buffer resource over the block's R member rows;
  // lanes with nothing to store give an offset past its end (dropped), so
  // every lane issues the same memory operations and the waits stay exact
  const __amdgpu_buffer_rsrc_t orr = buffer_rsrc(static_cast<uint8_t*>(rsc) + (grp * g + R * blk) * (int64_t)c * SE,
                                                 (uint32_t)(R * c) * SE);
  const uint32_t my_off = (uint32_t)(qr * c + cbeg + lr) * SE;
  // slot 16 f + lr is stored when 16 f < my_lim (one compare of the
  // fragment's uniform base against a lane constant)
  const int my_lim = writer ? ncs - lr : INT_MIN;
  const int nfrag = fend - fbeg;
  constexpr int S = WPG ? 1 : 4;  // fragment stride between the waves
  auto pos_of = [&](int f) { return spos[16 * f + lr]; };  // past the candidates: key 0
  // the same position read from global memory (before the LDS copy is staged)
  auto pos_glob = [&](int f) {
    const int p = max(crow[cbeg + min(16 * f + lr, ncs - 1)], 0);
    return km.pages ? (int)km.row(b, p) : p;
  };
  auto emit = [&](float acc, float ks, int f) {
    const uint32_t off = 16 * f < my_lim ? my_off + SE * (uint32_t)(16 * f) : 0xFFFFFFFFu;
    if constexpr (OB16)
      __builtin_amdgcn_raw_buffer_store_b16(bf16_rne(acc * ks), orr, off, 0, 0);
    else
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc * ks), orr, off, 0, 0);
  };
  // the rows a launch can gather: the pool (paged) or a sequence's stride
  const int64_t key_rows = km.pages ? ((int64_t)km.n_pages << km.shift) : km.stride;
  const __amdgpu_buffer_rsrc_t krs = buffer_rsrc(kb, B32 ? (uint32_t)(key_rows * kD * EB) : 0u);
  const __amdgpu_buffer_rsrc_t srs = buffer_rsrc(ksb, B32 && DT == kFp8 ? (uint32_t)(key_rows * 4) : 0u);
  auto fetch_at = [&](KeyFrag<DT>& kf, float& sc, int p) {
    if constexpr (B32) {
      sc = DT == kFp8 ? __int_as_float(__builtin_amdgcn_raw_buffer_load_b32(srs, (uint32_t)p * 4u, 0, 0)) : 1.0f;
      kf.load(krs, (uint32_t)p * (uint32_t)(kD * EB), kg);
    } else {
      sc = DT == kFp8 ? ksb[p] : 1.0f;
      kf.load(kb + (int64_t)p * kD * EB, kg);
    }
  };
  auto fetch = [&](KeyFrag<DT>& kf, float& sc, int ff) { fetch_at(kf, sc, pos_of(ff)); };
  // three fragments in flight per wave, with no exits in the loop body:
  // fragments past the end repeat the last candidate and are not stored.
  // The first three are requested before the row tile and the barrier, so
  // their loads overlap the tile's.
  int f = WPG ? 0 : wave;
  KeyFrag<DT> k0, k1, k2;
  float s0, s1, s2;
  fetch_at(k0, s0, pos_glob(f));
  fetch_at(k1, s1, pos_glob(f + S));
  fetch_at(k2, s2, pos_glob(f + 2 * S));
  Tile tile;
  tile.load(rows, wrows, qs, lrows, lsc, lane);
  if constexpr (WPG) {  // this wave's own positions: its LDS writes precede its reads
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  } else {
    __syncthreads();  // candidate positions staged
  }
  for (; f < nfrag; f += 3 * S) {
    emit(tile.score(k0), s0, f);
    fetch(k0, s0, f + 3 * S);
    emit(tile.score(k1), s1, f + S);
    fetch(k1, s1, f + 4 * S);
    emit(tile.score(k2), s2, f + 2 * S);
    fetch(k2, s2, f + 5 * S);
  }
}

// Fused fine step (Eqs. 8-9 in one launch) for fp8 groups of at most four
// members whose candidate rows have no window slots and at most kFuseCand
// entries: one workgroup per group.  The 4 waves split the group's candidate
// fragments (gathered three ahead, as in rescore_kernel) and write the
// members' bf16 scores into LDS; after one barrier wave t selects member t's
// top-m from there, so the scores never leave the CU.  The select keys a
// score as its 16-bit order key plus one (0 marks an unusable slot), each
// lane holding 64 (key, position) pairs in registers, and finds
//   K  = the key with fewer than m entries above it and at least m at or
//        above it (two radix passes, high byte then low byte, over a 256-bin
//        LDS histogram of the wave's own),
//   P  = the smallest position with enough entries of key K at positions
//        <= P to fill the row (bisection over the tied positions, compacted
//        into LDS),
// which picks exactly the top m by (score desc, position asc).
constexpr int kFuseCand = 4096;

template <int R, bool PAGED>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void rescore_select_kernel(
    const uint8_t* __restrict__ q, const float* __restrict__ q_scale, const float* __restrict__ w,
    const uint8_t* __restrict__ lin, const float* __restrict__ lin_scale, int g, const uint8_t* __restrict__ k,
    const float* __restrict__ k_scale, KeyMap km, SeqTable st, int j0, const int32_t* __restrict__ cand, int c,
    int m, int32_t* __restrict__ out_idx) {
  using Tile = RowTile<kFp8, R>;
  constexpr int NV = kFuseCand / 64;  // (key, position) pairs per lane in the select
  __shared__ int32_t spos[kFuseCand];                  // candidate positions
  __shared__ int32_t sprow[PAGED ? kFuseCand : 1];     // their pool rows (paged keys)
  __shared__ uint16_t ssc[R * kFuseCand];              // member scores, bf16 bits
  __shared__ uint32_t shist[4 * 257];                  // each wave's select histogram (+ a sink bin)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // workgroups are dealt round-robin to the 8 XCDs: XCD x % 8 takes a
  // contiguous run of groups (consecutive groups share most candidates, so
  // their gathers hit that XCD's L2); a partial last round keeps its order
  const int nwg = (int)gridDim.x, full = nwg - nwg % 8, bx = (int)blockIdx.x;
  const int j = j0 + (bx < full ? (bx % 8) * (full / 8) + bx / 8 : bx), b = blockIdx.y;
  if (b >= st.n || j >= seq_groups(st, b, g) || j < st.first_proxy[b]) return;
  const int gs = min(g, st.n_rows[b] - j * g);  // members, <= R
  const int64_t t0 = (int64_t)st.q_pos0[b] + (int64_t)j * g;
  const int nc = (int)min((int64_t)c, t0 + 1);  // usable slots: the first min(c, t0 + 1)
  const int32_t* crow = cand + ((int64_t)st.grp0[b] + j) * c;
  const int64_t r0 = (int64_t)st.row0[b] + (int64_t)j * g;
  const uint8_t* kb = PAGED ? k : k + km.row(b, 0) * kD;
  const float* ksb = PAGED ? k_scale : k_scale + km.row(b, 0);

  // positions: all loads of a thread issued before the first store
  {
    constexpr int SB = kFuseCand / 256;
    int32_t pv[SB];
#pragma unroll
    for (int u = 0; u < SB; ++u) pv[u] = tid + 256 * u < nc ? crow[tid + 256 * u] : 0;
#pragma unroll
    for (int u = 0; u < SB; ++u)
      if (tid + 256 * u < nc) {
        spos[tid + 256 * u] = pv[u];
        if constexpr (PAGED) sprow[tid + 256 * u] = (int32_t)km.row(b, max(pv[u], 0));
      }
  }
  const int lr = lane & 15, kg = lane >> 4;
  // key row of slot 16 f + lr (slots past the row repeat its last one;
  // empty slots read key 0), from LDS or, before the barrier, global memory
  auto row_lds = [&](int f) {
    const int e = min(16 * f + lr, nc - 1);
    return PAGED ? sprow[e] : max(spos[e], 0);
  };
  auto row_glob = [&](int f) {
    const int p = max(crow[min(16 * f + lr, nc - 1)], 0);
    return PAGED ? (int)km.row(b, p) : p;
  };
  auto fetch = [&](KeyFrag<kFp8>& kf, float& sc, int row) {
    sc = ksb[row];
    kf.load(kb + (int64_t)row * kD, kg);
  };
  constexpr int S = 4;  // fragment stride between the waves
  const int nfrag = (nc + 15) >> 4;
  int f = wave;
  KeyFrag<kFp8> k0, k1, k2;
  float s0, s1, s2;
  fetch(k0, s0, row_glob(f));
  fetch(k1, s1, row_glob(f + S));
  fetch(k2, s2, row_glob(f + 2 * S));
  const uint8_t* rows[R];
  const float* wrows[R];
  const uint8_t* lrows[R];
  const float* lsc[R];
  float qs[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = r0 + min(r, gs - 1);
    rows[r] = q + row * Tile::ROW_BYTES;
    wrows[r] = w + row * kH;
    qs[r] = q_scale[row];
    lrows[r] = lin + row * kLinBytes;
    lsc[r] = lin_scale + row * kLinLevels;
  }
  Tile tile;
  tile.load(rows, wrows, qs, lrows, lsc, lane);
  const int qr = kg / Tile::G;
  const bool writer = (kg % Tile::G) == 0 && qr < gs;
  uint16_t* my_sc = ssc + qr * kFuseCand;
  auto emit = [&](float acc, float ks, int ff) {
    const int slot = 16 * ff + lr;
    if (writer && slot < nc) my_sc[slot] = bf16_rne(acc * ks);
  };
  __syncthreads();  // positions staged
  for (; f < nfrag; f += 3 * S) {
    emit(tile.score(k0), s0, f);
    fetch(k0, s0, row_lds(f + 3 * S));
    emit(tile.score(k1), s1, f + S);
    fetch(k1, s1, row_lds(f + 4 * S));
    emit(tile.score(k2), s2, f + 2 * S);
    fetch(k2, s2, row_lds(f + 5 * S));
  }
  __syncthreads();  // scores staged

  if (wave >= gs) return;
  int32_t* orow = out_idx + (r0 + wave) * m;
  if (nc <= m) {  // every usable slot is selected
    for (int p = lane; p < m; p += 64) orow[p] = p < nc ? spos[p] : -1;
    return;
  }
  const uint16_t* row_sc = ssc + wave * kFuseCand;
  uint32_t key[NV];
  int32_t pos[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int e = lane + 64 * v;
    const bool in = e < nc;
    const int32_t p = in ? spos[e] : -1;
    const uint32_t k16 = float_key(__uint_as_float((uint32_t)(in ? row_sc[e] : 0) << 16)) >> 16;
    key[v] = p >= 0 ? k16 + 1u : 0u;
    pos[v] = p;
  }
  auto count = [&](auto pred) {
    int n = 0;
#pragma unroll
    for (int v = 0; v < NV; ++v) n += __popcll(__ballot(pred(v)));
    return n;
  };
  // the row's m outputs through a range-checked resource: lanes without an
  // entry store past its end (dropped), so no per-element branches
  const __amdgpu_buffer_rsrc_t orr = buffer_rsrc(orow, (uint32_t)m * 4u);
  auto emit_sel = [&](auto pred, int base) {  // compacts the chosen positions into orow[base ..]
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const bool take = pred(v);
      const uint64_t bal = __ballot(take);
      const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
      __builtin_amdgcn_raw_buffer_store_b32(pos[v], orr, take ? 4u * (uint32_t)(base + below) : 0xFFFFFFFFu, 0, 0);
      base += __popcll(bal);
    }
    return base;
  };
  auto wave_sum = [](int n) {
    for (int o = 32; o > 0; o >>= 1) n += __shfl_xor(n, o, 64);
    return n;
  };
  auto wave_max = [](int32_t x) {
    for (int o = 32; o > 0; o >>= 1) x = max(x, __shfl_xor(x, o, 64));
    return x;
  };
  int n_valid = 0;
#pragma unroll
  for (int v = 0; v < NV; ++v) n_valid += key[v] != 0u ? 1 : 0;
  n_valid = wave_sum(n_valid);
  if (n_valid <= m) {  // every usable candidate, then padding
    const int n = emit_sel([&](int v) { return key[v] != 0u; }, 0);
    for (int p = n + lane; p < m; p += 64) orow[p] = -1;
    return;
  }
  // Two radix passes over a 256-bin histogram of this wave's own (LDS
  // atomics; a wave's LDS operations complete in order): the high byte of
  // k16 = key - 1, then the low byte among keys in the chosen high bin.
  uint32_t* hist = shist + wave * 257;
  auto wave_sync = [] {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };
  // the bin b with count(digit > b) < need <= count(digit >= b); returns b
  // and sets `above` = count(digit > b), `in_bin` = count(digit == b)
  auto pick = [&](int need_here, int& above, int& in_bin) {
    uint32_t h[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) h[i] = hist[4 * lane + i];
    const int blk = (int)(h[0] + h[1] + h[2] + h[3]);
    int suf = blk;  // bins 4 lane .. 255
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_down(suf, o, 64);
      if (lane + o < 64) suf += t;
    }
    int over = suf - blk, bin = -1, ab = 0, ib = 0;  // over: bins above this lane's four
#pragma unroll
    for (int i = 3; i >= 0; --i) {
      if (bin < 0 && over < need_here && over + (int)h[i] >= need_here) {
        bin = 4 * lane + i;
        ab = over;
        ib = (int)h[i];
      }
      over += (int)h[i];
    }
    const uint64_t who = __ballot(bin >= 0);
    const int src = (int)__builtin_ctzll(who);
    above = __shfl(ab, src, 64);
    in_bin = __shfl(ib, src, 64);
    return __shfl(bin, src, 64);
  };
  // (bin 256 takes the entries a pass skips, so every lane adds every time)
#pragma unroll
  for (int i = 0; i < 4; ++i) hist[4 * lane + i] = 0u;
  wave_sync();
#pragma unroll
  for (int v = 0; v < NV; ++v) atomicAdd(&hist[key[v] != 0u ? (key[v] - 1u) >> 8 : 256u], 1u);
  wave_sync();
  int above1, in1;
  const int hb = pick(m, above1, in1);
  wave_sync();
#pragma unroll
  for (int i = 0; i < 4; ++i) hist[4 * lane + i] = 0u;
  wave_sync();
  const uint32_t khb = ((uint32_t)hb << 8) + 1u;  // the high bin's keys: khb .. khb + 255
#pragma unroll
  for (int v = 0; v < NV; ++v) atomicAdd(&hist[key[v] - khb < 256u ? key[v] - khb : 256u], 1u);
  wave_sync();
  int above2, ties;
  const int lb = pick(m - above1, above2, ties);
  const uint32_t K = (uint32_t)((hb << 8) | lb) + 1u;
  const int n_gt = above1 + above2;  // < m entries above K, all taken
  const int need = m - n_gt;         // >= 1 of the `ties` entries of key K
  emit_sel([&](int v) { return key[v] > K; }, 0);
  // from here key[v] holds the position of a tied entry, else INT32_MAX
#pragma unroll
  for (int v = 0; v < NV; ++v) key[v] = key[v] == K ? (uint32_t)pos[v] : 0x7FFFFFFFu;
  int32_t P = 0x7FFFFFFE;  // every tie when they are exactly enough (positions < 2^31 - 1)
  if (ties > need) {
    // the tied positions, compacted into this wave's score row (read into
    // registers above, so free) when they fit, else searched in registers
    int32_t* tl = reinterpret_cast<int32_t*>(ssc + wave * kFuseCand);
    constexpr int kTieCap = kFuseCand / 2 - 1;
    int32_t top = -1;
#pragma unroll
    for (int v = 0; v < NV; ++v) top = max(top, key[v] != 0x7FFFFFFFu ? (int32_t)key[v] : -1);
    top = wave_max(top);
    const bool listed = ties <= kTieCap;
    if (listed) {
      wave_sync();
      int base = 0;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const bool t = key[v] != 0x7FFFFFFFu;
        const uint64_t bal = __ballot(t);
        const int below =
            __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
        tl[t ? base + below : kTieCap] = (int32_t)key[v];  // slot kTieCap: a sink for the others
        base += __popcll(bal);
      }
      wave_sync();
    }
    // P: count(tied, pos <= plo) < need <= count(tied, pos <= phi)
    int64_t plo = -1, phi = top;
    while (phi - plo > 1) {
      const int32_t mid = (int32_t)(plo + ((phi - plo) >> 1));
      int n = 0;
      if (listed) {
        for (int e = lane; e < ties; e += 64) n += tl[e] <= mid;
        n = wave_sum(n);
      } else {
        n = count([&](int v) { return (int32_t)key[v] <= mid; });
      }
      if (n >= need) phi = mid;
      else plo = mid;
    }
    P = (int32_t)phi;
  }
  emit_sel([&](int v) { return (int32_t)key[v] <= P; }, n_gt);
}

// (key, position) pairs held in registers: entry 4 q + u is element
// 4 (tid + T q) + u of the row (loaded four at a time; T threads).
template <int V>
struct RegSource {
  static_assert(V % 4 == 0, "quads of elements");
  uint32_t key[V];
  int32_t pos[V];  // -1: not a candidate of this member
  template <class F>
  __device__ __forceinline__ void visit(F f) const {
#pragma unroll
    for (int v = 0; v < V; ++v)
      if (pos[v] >= 0) f(key[v], pos[v]);
  }
};

// bucket_select's emission for pairs held in registers: the taken entries of
// a lane form a bit mask, the wave reserves its slots with ONE LDS atomic,
// and each entry index then goes out with a ballot prefix (consecutive slots
// per store, as with wave_append, without an atomic per entry).
template <int V, class Bk, class Put, class List>
__device__ __forceinline__ void emit_bucket(const RegSource<V>& src, Bk bucket, int bsel, SelectShared& sh,
                                            Put put, List list) {
  static_assert(V <= 32, "one mask word");
  uint32_t take = 0;
#pragma unroll
  for (int v = 0; v < V; ++v) {
    if (src.pos[v] < 0) continue;
    const int bk = bucket(src.key[v]);
    take |= (bk > bsel ? 1u : 0u) << v;
    if (bk == bsel) list(src.key[v], src.pos[v]);
  }
  int total = 0;
#pragma unroll
  for (int v = 0; v < V; ++v) total += __popcll(__ballot((take >> v) & 1u));
  if (total == 0) return;  // uniform
  int base = 0;
  if ((threadIdx.x & 63) == 0) base = atomicAdd(&sh.emitted, total);
  base = __shfl(base, 0, 64);
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const bool t = (take >> v) & 1u;
    const uint64_t bal = __ballot(t);
    if (t) put(base + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u)),
               src.pos[v]);
    base += __popcll(bal);
  }
}

// Candidate slots a member may use (App. B): slots >= wslot are per-query
// window slots with the lower bound t - W + 1; window == 0 means a plain
// candidate row whose first min(c, t0 + 1) slots are all usable.
struct SlotRule {
  int32_t window;
  int32_t wslot;
};

// Workgroup x of a sequence's g * n row selects -> (group, member): in each
// full chunk of 8 g workgroups, group 8 c + x % 8 takes workgroups x, x + 8,
// .., x + 8 (g - 1) of the chunk, which the round-robin dispatch places on one
// XCD one after another; the partial last chunk is taken in plain order.
__device__ __forceinline__ void member_of(int x, int g, int n, int& j, int& member) {
  const int chunk = 8 * g, full = (g * n) / chunk * chunk;
  if (x < full) {
    const int r = x % chunk;
    j = (x / chunk) * 8 + r % 8;
    member = r / 8;
  } else {
    j = x / g;
    member = x % g;
  }
}

// Up to 16 pairs per thread the select fits 8 waves per SIMD: the compiler is
// held to that occupancy (a few scalar values move to VGPR lanes instead of
// holding it to 7 with their scalar registers).
template <int V, class E, int T>
__global__ __launch_bounds__(T) __attribute__((amdgpu_waves_per_eu(V <= 16 ? 8 : 1))) void topk_short_kernel(const E* __restrict__ rsc,
                                                         const int32_t* __restrict__ cand, int g, SeqTable st,
                                                         int j0, int nj, int c, SlotRule rule, int m,
                                                         int32_t* __restrict__ out_idx) {
  __shared__ SelectShared sel;
  __shared__ uint32_t hist[4 * 256];  // bucket_select's histogram, then its list
  __shared__ int32_t lcount, nvalid_sh;
  int jl, member;
  member_of((int)blockIdx.x, g, nj, jl, member);
  const int j = j0 + jl, b = blockIdx.y;
  if (b >= st.n || j >= seq_groups(st, b, g) || j < st.first_proxy[b]) return;
  const int gs = min(g, st.n_rows[b] - j * g);
  if (member >= gs) return;
  const int tid = threadIdx.x;
  const int64_t t0 = (int64_t)st.q_pos0[b] + (int64_t)j * g;
  const int64_t tt = t0 + member;
  const bool win = rule.window > 0;
  const int nc = win ? c : (int)min((int64_t)c, t0 + 1);
  const int64_t grp = (int64_t)st.grp0[b] + j;
  const E* srow = rsc + (grp * g + member) * (int64_t)c;
  const int32_t* crow = cand + grp * c;
  int32_t* orow = out_idx + ((int64_t)st.row0[b] + (int64_t)j * g + member) * m;

  RegSource<V> src;
  int mine = 0;
  // quads of scores and positions with 16-byte loads when the rows allow it
  const bool vec = (c & 3) == 0 && (reinterpret_cast<uintptr_t>(srow) & (4 * sizeof(E) - 1)) == 0 &&
                   (reinterpret_cast<uintptr_t>(crow) & 15u) == 0;
#pragma unroll
  for (int q4 = 0; q4 < V / 4; ++q4) {
    const int e0 = 4 * (tid + T * q4);
    float kv[4] = {0.f, 0.f, 0.f, 0.f};
    int32_t pv[4] = {-1, -1, -1, -1};
    if (vec) {
      if (e0 < nc) {  // c is a multiple of 4: the quad lies inside the row
        if constexpr (sizeof(E) == 4) {
          const float4 a = *reinterpret_cast<const float4*>(srow + e0);
          kv[0] = a.x; kv[1] = a.y; kv[2] = a.z; kv[3] = a.w;
        } else {
          const uint2 a = *reinterpret_cast<const uint2*>(srow + e0);
          kv[0] = __uint_as_float(a.x << 16); kv[1] = __uint_as_float(a.x & 0xFFFF0000u);
          kv[2] = __uint_as_float(a.y << 16); kv[3] = __uint_as_float(a.y & 0xFFFF0000u);
        }
        const int4 q = *reinterpret_cast<const int4*>(crow + e0);
        pv[0] = q.x; pv[1] = q.y; pv[2] = q.z; pv[3] = q.w;
      }
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (e0 + u < nc) {
          if constexpr (sizeof(E) == 4)
            kv[u] = srow[e0 + u];
          else
            kv[u] = __uint_as_float((uint32_t)srow[e0 + u] << 16);
          pv[u] = crow[e0 + u];
        }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = e0 + u;
      const bool in = e < nc;
      const int32_t p = in ? pv[u] : -1;
      bool ok = in;
      if (win) ok = p >= 0 && p <= tt && !(e >= rule.wslot && p < tt - rule.window + 1);
      src.key[4 * q4 + u] = in ? float_key(kv[u]) : 0u;
      src.pos[4 * q4 + u] = ok ? p : -1;
      mine += ok;
    }
  }
  if (!win) {
    if (nc <= m) {  // every candidate is selected
      for (int p = tid; p < m; p += T) orow[p] = p < nc ? crow[p] : -1;
      return;
    }
  } else {
    if (tid == 0) {
      nvalid_sh = 0;
      sel.emitted = 0;
    }
    __syncthreads();
    atomicAdd(&nvalid_sh, mine);
    __syncthreads();
    const int nvalid = nvalid_sh;
    if (nvalid <= m) {  // every usable slot is selected, then -1 padding
#pragma unroll
      for (int v = 0; v < V; ++v)
        wave_append(src.pos[v] >= 0, &sel.emitted, [&](int slot) { orow[slot] = src.pos[v]; });
      for (int p = nvalid + tid; p < m; p += T) orow[p] = -1;
      return;
    }
    __syncthreads();  // sel.emitted is cleared again below
  }
  if (tid == 0) sel.emitted = 0;
  __syncthreads();
  auto put = [&](int slot, int32_t p) { orow[slot] = p; };
  if (!bucket_select<T, 1024>(src, (uint32_t)m, hist, hist, reinterpret_cast<int32_t*>(hist + kBucketList), &lcount,
                                sel, put)) {
    // block_select() takes its source by reference; handing it a copy keeps
    // `src` itself in registers on the bucket path (a referenced array of 32
    // pairs would otherwise live in scratch memory)
    const RegSource<V> fb = src;
    block_select<T, true>(fb, (uint32_t)m, sel, put);
  }
}

// The member select of bf16 score rows of at most 4096 slots, 16 per thread
// of 256: bucket_select's algorithm (the same NB value buckets over the
// usable slots' range, so the same decisions), with the scores kept as bf16
// pairs in registers (widened exactly on use) rather than as order keys.
// The range, the histogram and the emission form no keys; only the boundary
// bucket's few members get one.  Unusable slots (past the row, or excluded
// by the window rule) are masked: their histogram count goes to a sink bin.
// Each compare's bit mask gives the emission with one LDS atomic per wave.
// Returns false, having emitted nothing, where bucket_select would (equal
// values, a boundary bucket longer than kBucketList).  hist: NB + 1 LDS words.
template <int V, int T, int NB>
__device__ __forceinline__ bool member_select16(const uint32_t (&sc)[V / 2], const int32_t (&pv)[V], uint32_t vmask,
                                                bool full, uint32_t m, uint32_t* hist, int32_t* lcount,
                                                SelectShared& sh, int32_t* __restrict__ orow) {
  static_assert(V <= 32 && V % 2 == 0 && NB % T == 0 && NB >= 2 * kBucketList, "mask word, bins, list");
  const int tid = threadIdx.x, lane = tid & 63;
  auto fv = [&](int v) { return __uint_as_float(v & 1 ? sc[v >> 1] & 0xFFFF0000u : sc[v >> 1] << 16); };
  auto usable = [&](int v) { return ((vmask >> v) & 1u) != 0u; };
  if (tid == 0) sh.emitted = 0;  // ordered before any append by the barriers below
  float lo = __builtin_inff(), hi = -__builtin_inff();
  if (full) {  // uniform
#pragma unroll
    for (int v = 0; v < V; ++v) {
      lo = fminf(lo, fv(v));
      hi = fmaxf(hi, fv(v));
    }
  } else {
#pragma unroll
    for (int v = 0; v < V; ++v) {
      lo = fminf(lo, usable(v) ? fv(v) : __builtin_inff());
      hi = fmaxf(hi, usable(v) ? fv(v) : -__builtin_inff());
    }
  }
  uint32_t kmin = float_key(lo), kmax = float_key(hi);
  block_pair_reduce<T, true>(kmin, kmax, sh);
  const float fmin = key_float(kmin);
  const float scale = (float)NB / (key_float(kmax) - fmin);
  if (kmin == kmax || !(scale > 0.0f && scale < __builtin_inff())) return false;
  auto bucket = [&](float f, float f0, float s) { return min(NB - 1, (int)((f - f0) * s)); };
  for (int k = tid; k < NB; k += T) hist[k] = 0;
  if (tid == 0) *lcount = 0;
  __syncthreads();
  if (full) {
#pragma unroll
    for (int v = 0; v < V; ++v) atomicAdd(&hist[bucket(fv(v), fmin, scale)], 1u);
  } else {
#pragma unroll
    for (int v = 0; v < V; ++v) atomicAdd(&hist[usable(v) ? bucket(fv(v), fmin, scale) : NB], 1u);
  }
  __syncthreads();
  find_digit<T, true>(hist, sh, m, NB);
  const int bsel = (int)sh.digit;
  const uint32_t rem = m - sh.before, in_b = sh.equal;
  __syncthreads();  // the histogram's words become the boundary list
  if (in_b > (uint32_t)kBucketList) return false;
  uint32_t* lkey = hist;
  int32_t* lpos = reinterpret_cast<int32_t*>(hist + kBucketList);
  // The buckets are computed again rather than kept from the histogram pass
  // (sixteen more live registers would cost occupancy); copies of fmin and
  // scale that the compiler cannot see through keep it from reusing them.
  const float fmin2 = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(fmin)));
  const float scale2 = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(scale)));
  uint32_t tb = 0, lb = 0;  // taken (bucket above bsel) and listed (bucket bsel) slots
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const int bk = bucket(fv(v), fmin2, scale2);
    tb |= (bk > bsel ? 1u : 0u) << v;
    lb |= (bk == bsel ? 1u : 0u) << v;
  }
  tb &= vmask;
  lb &= vmask;
  // one LDS atomic per wave for each of the two appends
  const uint32_t nt = wave_incl_sum((uint32_t)__popc(tb)), nl = wave_incl_sum((uint32_t)__popc(lb));
  const uint32_t tt = (uint32_t)__builtin_amdgcn_readlane((int)nt, 63);
  const uint32_t lt = (uint32_t)__builtin_amdgcn_readlane((int)nl, 63);
  int tbase = 0, lbase = 0;
  if (lane == 0) {
    if (tt) tbase = atomicAdd(&sh.emitted, (int)tt);
    if (lt) lbase = atomicAdd(lcount, (int)lt);
  }
  tbase = __builtin_amdgcn_readfirstlane(tbase);
  lbase = __builtin_amdgcn_readfirstlane(lbase);
  const __amdgpu_buffer_rsrc_t orr = buffer_rsrc(orow, m * 4u);  // 32-bit offsets
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const bool t = (tb >> v) & 1u;
    const uint64_t bal = __ballot(t);
    if (t) {
      const int slot = tbase + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                              __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
      __builtin_amdgcn_raw_buffer_store_b32((uint32_t)pv[v], orr, 4 * slot, 0, 0);
    }
    tbase += (int)__popcll(bal);
    const bool l = (lb >> v) & 1u;
    const uint64_t lbal = __ballot(l);
    if (lbal) {  // uniform over the wave, and rare
      if (l) {
        const int slot = lbase + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(lbal >> 32),
                                                                __builtin_amdgcn_mbcnt_lo((uint32_t)lbal, 0u));
        lkey[slot] = float_key(fv(v));
        lpos[slot] = pv[v];
      }
      lbase += (int)__popcll(lbal);
    }
  }
  __syncthreads();
  rank_listed<T>(in_b, rem, lkey, lpos, sh, [&](int slot, int32_t p) { orow[slot] = p; });
  return true;
}

// Member selects of bf16 score rows with |C| <= V x T (4096: the prefill
// Refine shape, 16 per thread of 256; MTP decode, 4 per thread of 1024): the
// workgroup mapping, slot rules and early exits of topk_short_kernel, then
// member_select16, falling back to block_select.
template <int V, int T>
__global__ __launch_bounds__(T) __attribute__((amdgpu_waves_per_eu(8))) void topk_member16_kernel(
    const uint16_t* __restrict__ rsc, const int32_t* __restrict__ cand, int g, SeqTable st, int j0, int nj, int c,
    SlotRule rule, int m, int32_t* __restrict__ out_idx) {
  constexpr int NB = 1024;
  static_assert(V % 4 == 0, "quads of slots");
  __shared__ SelectShared sel;
  __shared__ uint32_t hist[NB + 1];  // the histogram (and a sink bin), then the boundary list
  __shared__ int32_t lcount, nvalid_sh;
  int jl, member;
  member_of((int)blockIdx.x, g, nj, jl, member);
  jl = __builtin_amdgcn_readfirstlane(jl);  // uniform: scalar registers
  member = __builtin_amdgcn_readfirstlane(member);
  const int j = j0 + jl, b = blockIdx.y;
  if (b >= st.n || j >= seq_groups(st, b, g) || j < st.first_proxy[b]) return;
  const int gs = min(g, st.n_rows[b] - j * g);
  if (member >= gs) return;
  const int tid = threadIdx.x;
  const int64_t t0 = (int64_t)st.q_pos0[b] + (int64_t)j * g;
  const int64_t tt = t0 + member;
  const bool win = rule.window > 0;
  const int nc = win ? c : (int)min((int64_t)c, t0 + 1);
  const int64_t grp = (int64_t)st.grp0[b] + j;
  const uint16_t* srow = uniform_ptr(rsc + (grp * g + member) * (int64_t)c);
  const int32_t* crow = uniform_ptr(cand + grp * c);
  int32_t* orow = uniform_ptr(out_idx + ((int64_t)st.row0[b] + (int64_t)j * g + member) * m);

  // quads of scores (8 bytes) and positions (16 bytes) when the rows allow it
  const bool vec = (c & 3) == 0 && (reinterpret_cast<uintptr_t>(srow) & 7u) == 0 &&
                   (reinterpret_cast<uintptr_t>(crow) & 15u) == 0;
  uint32_t sc[V / 2];  // bf16 scores, two per word (the even slot in the low half)
  int32_t pv[V];       // -1: not usable by this member
  uint32_t vmask = 0;
#pragma unroll
  for (int q4 = 0; q4 < V / 4; ++q4) {
    const int e0 = 4 * (tid + T * q4);
    uint32_t s01 = 0, s23 = 0;
    int32_t p4[4] = {-1, -1, -1, -1};
    if (vec) {
      if (e0 < nc) {  // c is a multiple of 4: the quad lies inside the row
        const uint2 a = *reinterpret_cast<const uint2*>(srow + e0);
        s01 = a.x;
        s23 = a.y;
        const int4 q = *reinterpret_cast<const int4*>(crow + e0);
        p4[0] = q.x;
        p4[1] = q.y;
        p4[2] = q.z;
        p4[3] = q.w;
      }
    } else {
      uint32_t h[4] = {0, 0, 0, 0};
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (e0 + u < nc) {
          h[u] = srow[e0 + u];
          p4[u] = crow[e0 + u];
        }
      s01 = h[0] | (h[1] << 16);
      s23 = h[2] | (h[3] << 16);
    }
    sc[2 * q4] = s01;
    sc[2 * q4 + 1] = s23;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = e0 + u;
      const int32_t p = p4[u];
      bool ok = e < nc;
      if (win) ok = ok && p >= 0 && p <= tt && !(e >= rule.wslot && p < tt - rule.window + 1);
      pv[4 * q4 + u] = ok ? p : -1;
      vmask |= (ok ? 1u : 0u) << (4 * q4 + u);
    }
  }
  if (!win) {
    if (nc <= m) {  // every candidate is selected
      for (int p = tid; p < m; p += T) orow[p] = p < nc ? crow[p] : -1;
      return;
    }
  } else {
    if (tid == 0) {
      nvalid_sh = 0;
      sel.emitted = 0;
    }
    __syncthreads();
    atomicAdd(&nvalid_sh, __popc(vmask));
    __syncthreads();
    const int nvalid = nvalid_sh;
    if (nvalid <= m) {  // every usable slot is selected, then -1 padding
#pragma unroll
      for (int v = 0; v < V; ++v)
        wave_append(pv[v] >= 0, &sel.emitted, [&](int slot) { orow[slot] = pv[v]; });
      for (int p = nvalid + tid; p < m; p += T) orow[p] = -1;
      return;
    }
    __syncthreads();  // sel.emitted is cleared again below
  }
  const bool full = !win && nc == V * T;
  if (member_select16<V, T, NB>(sc, pv, vmask, full, (uint32_t)m, hist, &lcount, sel, orow)) return;
  RegSource<V> src;
#pragma unroll
  for (int v = 0; v < V; ++v) {
    src.key[v] = float_key(__uint_as_float(v & 1 ? sc[v >> 1] & 0xFFFF0000u : sc[v >> 1] << 16));
    src.pos[v] = pv[v];
  }
  __syncthreads();
  if (tid == 0) sel.emitted = 0;
  __syncthreads();
  block_select<T, true>(src, (uint32_t)m, sel, [&](int slot, int32_t p) { orow[slot] = p; });
}

// App. B window union: slot0 + u (u < wg) of every candidate row of the
// groups [j0, j1) with j >= first_proxy[b] takes position t0 - W + 1 + u, or
// -1 below 0, past the group's last member, or (dedupe) when it is already
// among the row's first slot0 slots.
__global__ __launch_bounds__(256) void window_kernel(int32_t* __restrict__ cand, int g, SeqTable st, int j0,
                                                     int width, int slot0, int W, int wg, int dedupe) {
  __shared__ uint8_t seen[kMaxCand];
  const int j = j0 + blockIdx.x, b = blockIdx.y;
  if (b >= st.n || j >= seq_groups(st, b, g) || j < st.first_proxy[b]) return;
  const int tid = threadIdx.x;
  const int gs = min(g, st.n_rows[b] - j * g);
  const int64_t t0 = (int64_t)st.q_pos0[b] + (int64_t)j * g;
  const int64_t lo = t0 - W + 1;
  int32_t* row = cand + ((int64_t)st.grp0[b] + j) * width;
  if (dedupe) {
    for (int u = tid; u < wg; u += 256) seen[u] = 0;
    __syncthreads();
    for (int i = tid; i < slot0; i += 256) {
      const int64_t p = row[i];
      if (p >= lo && p < lo + wg) seen[p - lo] = 1;
    }
    __syncthreads();
  }
  for (int u = tid; u < wg; u += 256) {
    const int64_t p = lo + u;
    const bool ok = p >= 0 && p <= t0 + gs - 1 && !(dedupe && seen[u]);
    row[slot0 + u] = ok ? (int32_t)p : -1;
  }
}

hipError_t launch_window(int32_t* cand, int g, const SeqTable& st, int j0, int j1, int width, int slot0, int W,
                         bool dedupe, hipStream_t stream) {
  const int wg = W + g - 1;
  if (j1 <= j0 || st.n <= 0 || W <= 0) return hipSuccess;
  if (width > kMaxCand || slot0 < 0 || slot0 + wg > width) return hipErrorInvalidValue;
  hipLaunchKernelGGL(window_kernel, dim3((unsigned)(j1 - j0), (unsigned)st.n), dim3(256), 0, stream, cand, g, st, j0,
                     width, slot0, W, wg, (int)dedupe);
  return hipGetLastError();
}

// Member selects of groups [j0, j1): one workgroup per (group, member) row,
// x = the sequence's g (j1 - j0) rows in member_of() order; 256 threads, or
// 1024 when the launch has too few rows to fill the GPU (decode), so each
// row's select runs on more threads.
template <class E>
hipError_t launch_short(const E* rescore, const int32_t* cand, int g, const SeqTable& st, int j0, int j1, int c,
                        SlotRule rule, int m, int32_t* out_idx, hipStream_t stream) {
  const int nj = j1 - j0;
  const dim3 sgrid((unsigned)(nj * g), (unsigned)st.n);
  const bool few = (int64_t)nj * g * st.n < 256;
#define PIVOT_SHORT(V, T)                                                                                         \
  hipLaunchKernelGGL((topk_short_kernel<V, E, T>), sgrid, dim3(T), 0, stream, rescore, cand, g, st, j0, nj, c, rule, \
                     m, out_idx)
  if (c <= 1024)
    PIVOT_SHORT(4, 256);
  else if (few && c <= 4096 && sizeof(E) == 2)
    hipLaunchKernelGGL((topk_member16_kernel<4, 1024>), sgrid, dim3(1024), 0, stream,
                       reinterpret_cast<const uint16_t*>(rescore), cand, g, st, j0, nj, c, rule, m, out_idx);
  else if (few && c <= 4096)
    PIVOT_SHORT(4, 1024);
  else if (few)
    PIVOT_SHORT(8, 1024);
  else if (c <= 4096 && sizeof(E) == 2)
    hipLaunchKernelGGL((topk_member16_kernel<16, 256>), sgrid, dim3(256), 0, stream,
                       reinterpret_cast<const uint16_t*>(rescore), cand, g, st, j0, nj, c, rule, m, out_idx);
  else if (c <= 4096)
    PIVOT_SHORT(16, 256);
  else if (c <= 5120)  // c = 4096 plus a window union
    PIVOT_SHORT(20, 256);
  else
    PIVOT_SHORT(32, 256);
#undef PIVOT_SHORT
  return hipGetLastError();
}

hipError_t launch_refine(int dtype, const void* q, const float* q_scale, const float* w, const uint8_t* lin,
                         const float* lin_scale, int g, const void* k, const float* k_scale, const KeyMap& km,
                         const SeqTable& st, int j0, int j1, const int32_t* cand, int c, int W, int wslot, int m,
                         void* rescore, int32_t* out_idx, int path, hipStream_t stream) {
  if (j1 <= j0 || st.n <= 0) return hipSuccess;
  if (c > kMaxCand) return hipErrorInvalidValue;
  // the fused re-score and select on request, where it applies.  Not the
  // default: at two workgroups per CU (the 4-row tile's registers) a group's
  // member selects cannot hide their latency behind other groups' scoring,
  // and the split path (many small select workgroups per CU) is faster.
  const bool fusable = dtype == kFp8 && W == 0 && g <= 4 && c <= kFuseCand;
  if (fusable && path == PIVOT_REFINE_FUSED) {
    const dim3 grid((unsigned)(j1 - j0), (unsigned)st.n);
#define PIVOT_FUSED(RV, PG)                                                                                         \
  hipLaunchKernelGGL((rescore_select_kernel<RV, PG>), grid, dim3(256), 0, stream, (const uint8_t*)q, q_scale, w, lin, \
                     lin_scale, g, (const uint8_t*)k, k_scale, km, st, j0, cand, c, m, out_idx)
    if (g > 2) {
      if (km.pages) PIVOT_FUSED(4, true);
      else PIVOT_FUSED(4, false);
    } else {
      if (km.pages) PIVOT_FUSED(2, true);
      else PIVOT_FUSED(2, false);
    }
#undef PIVOT_FUSED
    return hipGetLastError();
  }
  const SlotRule rule{W, wslot};
  const int all_slots = W > 0;
  // few groups (decode): split the candidates so the launch still fills the GPU;
  // fp8 groups of at most two members take the 2-row tile (half the MFMA work)
  const int R = (dtype == kFp8 && g > 2) ? 4 : 2;
  const int64_t wgs = (int64_t)(j1 - j0) * st.n * ((g + R - 1) / R);
  const int nfrag = (c + 15) / 16;
  // (at least 6 fragments per wave: the loop runs in steps of 3)
  const int parts = (int)std::max<int64_t>(1, std::min<int64_t>(std::max(1, nfrag / 24), (512 + wgs - 1) / wgs));
  // many groups (prefill): one unit per wave when the candidate rows fit its LDS share
  const bool wpg = parts == 1 && c <= kWpgCand;
  const int64_t units = (int64_t)(j1 - j0) * ((g + R - 1) / R);
  const dim3 grid = wpg ? dim3((unsigned)((units + 3) / 4), (unsigned)st.n, 1u)
                        : dim3((unsigned)(j1 - j0), (unsigned)st.n, (unsigned)(((g + R - 1) / R) * parts));
  // 32-bit gather offsets when every gatherable key row lies below 2^31 bytes
  // (a paged pool always does)
  const int eb = dtype == kFp8 ? 1 : 2;
  const bool b32 = km.pages || km.stride * kD * eb < ((int64_t)1 << 31);
#define PIVOT_RESCORE(DTV, RV, OB, WP, KS)                                                                        \
  if (b32)                                                                                                        \
    hipLaunchKernelGGL((rescore_kernel<DTV, RV, OB, WP, true>), grid, dim3(256), 0, stream, (const uint8_t*)q,     \
                       q_scale, w, lin, lin_scale, g, (const uint8_t*)k, KS, km, st, j0, cand, c, all_slots, parts, \
                       rescore);                                                                                  \
  else                                                                                                            \
    hipLaunchKernelGGL((rescore_kernel<DTV, RV, OB, WP, false>), grid, dim3(256), 0, stream, (const uint8_t*)q,    \
                       q_scale, w, lin, lin_scale, g, (const uint8_t*)k, KS, km, st, j0, cand, c, all_slots, parts, \
                       rescore)
  if (dtype == kFp8 && R == 4) {
    if (wpg) PIVOT_RESCORE(kFp8, 4, true, true, k_scale);
    else PIVOT_RESCORE(kFp8, 4, true, false, k_scale);
  } else if (dtype == kFp8) {
    if (wpg) PIVOT_RESCORE(kFp8, 2, true, true, k_scale);
    else PIVOT_RESCORE(kFp8, 2, true, false, k_scale);
  } else {
    if (wpg) PIVOT_RESCORE(kBf16, 2, false, true, nullptr);
    else PIVOT_RESCORE(kBf16, 2, false, false, nullptr);
  }
#undef PIVOT_RESCORE
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (dtype == kFp8) return launch_short(static_cast<const bf16_t*>(rescore), cand, g, st, j0, j1, c, rule, m, out_idx,
                                         stream);
  return launch_short(static_cast<const float*>(rescore), cand, g, st, j0, j1, c, rule, m, out_idx, stream);
}

}  // namespace pivot
