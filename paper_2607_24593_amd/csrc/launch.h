// Host-side launchers of the gfx950 kernels (internal to libpivot.so).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"

namespace pivot {

// Where a row's top-m indices go: row (b, i) writes entries [0, m) of out rows
//   fan_g == 0: (groups ? grp0[b] : row0[b]) + i
//   fan_g  > 0: row0[b] + i * fan_g + u, u < min(fan_g, n_rows[b] - i * fan_g)
// (SeqTable; the fan-out shares a proxy's top-k with the members of its
// group); out rows are ld >= m entries apart (a candidate row keeps window
// slots after m).
struct OutDesc {
  int32_t* base;
  int32_t m;
  int32_t fan_g;
  int32_t groups;
  int32_t ld;
};

// Proxy rows (Eq. 4) of groups [j0, j1) of each sequence (query rows and
// proxies placed as SeqTable says).  all_groups ignores first_proxy.
// agg: PIVOT_AGG_MEAN (Eq. 4), or PIVOT_AGG_FIRST / LAST (that member's row).
// Optional fp8 outputs of the proxy kernel: the linear terms (lin_kernel's
// layout) of each proxy (plin / plsc, indexed like pq) and of each member row
// of the groups it handles (qlin / qlsc, indexed like q); NULL: not written.
struct LinOut {
  uint8_t* plin = nullptr;
  float* plsc = nullptr;
  uint8_t* qlin = nullptr;
  float* qlsc = nullptr;
};
hipError_t launch_proxy(int dtype, const void* q, const float* q_scale, const float* w, int g, const SeqTable& st,
                        int j0, int j1, bool all_groups, int agg, void* pq, float* psc, float* pw, hipStream_t stream,
                        const LinOut& lo = LinOut{});

// The fp8 epilogue's linear term (mfma_tile.h) for flat rows [r0, r1) of an
// fp8 row array: lin [rows, 4 * 128] codes, lin_scale [rows, 4].  The two-set
// form covers two row arrays (e.g. query rows and their proxies) in one launch.
struct LinRows {
  const uint8_t* q = nullptr;
  const float* q_scale = nullptr;
  const float* w = nullptr;
  int64_t r0 = 0, r1 = 0;
  uint8_t* lin = nullptr;
  float* lin_scale = nullptr;
};
hipError_t launch_lin(const LinRows& set0, const LinRows& set1, hipStream_t stream);
hipError_t launch_lin(const void* q, const float* q_scale, const float* w, int64_t r0, int64_t r1, uint8_t* lin,
                      float* lin_scale, hipStream_t stream);

// Score rows rs (row data [rows, H, d] indexed by row_index(), with lin /
// lin_scale rows in the same order for fp8) against each sequence's keys
// 0 .. limit; out [B * (i1 - i0), ld] of fp32, or of bf16 when out_bf16 (fp8
// inputs only).  lim_max: largest limit of any active row.
hipError_t launch_score(int dtype, const void* q, const float* q_scale, const float* w, const uint8_t* lin,
                        const float* lin_scale, const void* k, const float* k_scale, const KeyMap& km,
                        const SeqTable& st, const RowSpace& rs, int64_t lim_max, void* out, bool out_bf16,
                        int64_t ld, hipStream_t stream);

// Top-m of score rows (fp32, or bf16 when scores_bf16): row (b, i) has
// limit + 1 valid entries; lim_max is the largest limit.  Up to 256 long rows
// (decode) are split over several workgroups each when `scratch` holds
// split_scratch_bytes(rows) (else one 1024-thread workgroup each); more rows
// take one 512-thread workgroup each.
hipError_t launch_topk(const void* scores, bool scores_bf16, int64_t ld, const SeqTable& st, const RowSpace& rs,
                       const OutDesc& od, int64_t lim_max, void* scratch, size_t scratch_bytes,
                       hipStream_t stream);
size_t split_scratch_bytes(int64_t rows);
constexpr int kSplitMaxRows = 256;   // launches with more rows do not split
constexpr int kSplitMinKeys = 16384; // nor do launches whose rows are all shorter

// Refine (Eqs. 8-9) for groups [j0, j1) with j >= first_proxy[b]: re-score
// the candidate rows [groups, c] into rescore [groups, g, c] (bf16 scores
// for fp8 inputs, fp32 for bf16 inputs), then
// select top-m.  W = 0: plain rows (the first min(c, t0 + 1) slots hold
// positions).  W > 0 (App. B window): any slot may be empty (-1); member t
// uses positions in [0, t], from slot wslot on also >= t - W + 1.  path: a
// pivot_refine_path (the fused launch needs no `rescore` buffer).
hipError_t launch_refine(int dtype, const void* q, const float* q_scale, const float* w, const uint8_t* lin,
                         const float* lin_scale, int g, const void* k, const float* k_scale, const KeyMap& km,
                         const SeqTable& st, int j0, int j1, const int32_t* cand, int c, int W, int wslot, int m,
                         void* rescore, int32_t* out_idx, int path, hipStream_t stream);

// App. B window union of groups [j0, j1) (j >= first_proxy[b]) into slots
// [slot0, slot0 + W + g - 1) of the [groups, width] candidate rows; dedupe
// empties positions already among the first slot0 slots.
hipError_t launch_window(int32_t* cand, int g, const SeqTable& st, int j0, int j1, int width, int slot0, int W,
                         bool dedupe, hipStream_t stream);

// Fill the group rows (b, j), j < first_proxy[b], j in [j0, j1), of a
// [groups, width] int32 array.
hipError_t launch_fill_guardrail(int32_t* base, int width, const SeqTable& st, int j0, int j1, int32_t value,
                                 hipStream_t stream);

hipError_t launch_encode_e4m3(const float* x, uint8_t* out, int64_t n, hipStream_t stream);

// n int32 of src copied to each of dst[0 .. n_dst) (n_dst <= kMaxCopyDst): one
// read of src, n_dst writes (IndexCache follower layers).
constexpr int kMaxCopyDst = 16;
hipError_t launch_copy_fanout(const int32_t* src, int32_t* const* dst, int n_dst, int64_t n, hipStream_t stream);

}  // namespace pivot
