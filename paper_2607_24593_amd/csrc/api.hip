// C ABI of libpivot.so: argument validation, the group plan of Algorithm 1
// (App. E), workspace carving and the launch sequence on the caller's stream.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <atomic>
#include <mutex>
#include <vector>

#include "launch.h"
#include "mfma_tile.h"
#include "pivot.h"

using namespace pivot;

// Scratch of pivot_group_index_noalloc: one copy per device in the code
// object.  Host code uses the device address hipGetSymbolAddress returns
// (g_scratch_ptr), never this name.
static __device__ __align__(256) uint8_t scratch[PIVOT_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local char g_err[512] = "";

pivot_status fail(pivot_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

pivot_status hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return PIVOT_OK;
  return fail(PIVOT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// ---- optional per-kernel event timing (pivot_profile_begin / _end) ----
struct ProfRecord {
  int kind;
  hipEvent_t start, stop;
};
std::mutex g_prof_mu;
// read without the lock on every launch; written under g_prof_mu
std::atomic<bool> g_prof_on{false};
std::atomic<uint32_t> g_prof_mask{0};  // kernel kinds bracketed while a profile runs
std::vector<ProfRecord> g_prof_recs;
std::vector<hipEvent_t> g_prof_pool;

hipEvent_t prof_event() {
  if (!g_prof_pool.empty()) {
    hipEvent_t e = g_prof_pool.back();
    g_prof_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Run one launcher; with profiling on, bracket it with events on `stream`.
template <class F>
hipError_t timed(int kind, hipStream_t stream, F launch) {
  if (!g_prof_on.load(std::memory_order_relaxed) || !((g_prof_mask.load(std::memory_order_relaxed) >> kind) & 1u))
    return launch();
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof_on.load(std::memory_order_relaxed)) return launch();  // ended meanwhile
  ProfRecord r{kind, prof_event(), prof_event()};
  if (!r.start || !r.stop) return hipErrorOutOfMemory;
  hipError_t e = hipEventRecord(r.start, stream);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(r.stop, stream);
  if (e != hipSuccess) return e;
  g_prof_recs.push_back(r);
  return hipSuccess;
}

constexpr size_t kAlign = 256;
constexpr int64_t kDefaultScoreBytes = int64_t(1) << 30;  // score tiles target ~1 GiB

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
// Score-row stride in floats: a multiple of 64 (256 B), and an odd one, so the
// rows that a workgroup writes in step are spread over memory channels (about
// 1% on the scoring kernel at 131072 keys against the power-of-two stride).
int64_t ld_for(int64_t n) {
  const int64_t u = (n + 63) / 64;
  return (u | 1) * 64;
}
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
// Score rows hold bf16 for fp8 inputs (half the bytes the select streams; the
// rounding, at most 2^-9 relative, is far inside the fp8 score tolerance) and
// fp32 for bf16 inputs.
bool bf16_scores(int dtype) { return dtype == PIVOT_DT_FP8_E4M3; }
int64_t score_eb(int dtype) { return bf16_scores(dtype) ? 2 : 4; }

// The group plan: for each sequence, its query rows and groups, how many
// leading query rows take the dense path (the guardrail of Algorithm 1) and
// from which group on the proxy path runs.
struct Plan {
  int mode = PIVOT_DENSE;  // PIVOT_DENSE, PIVOT_REUSE or PIVOT_REFINE
  int g = 1, c = 0, dense_below = 0;
  int B = 0, topk = 0, dtype = 0, EB = 1;
  int n_q = 0;       // most query rows of a sequence
  int n_groups = 0;  // most groups of a sequence
  int64_t rows_total = 0, groups_total = 0;
  size_t row_bytes = 0;
  std::vector<int32_t> dense_rows, first_proxy, q_pos0, n_k, nq, row0, ng, grp0;
  int dense_hi = 0;       // max dense_rows over sequences
  int proxy_lo = 0;       // min first_proxy over sequences
  bool any_proxy = false;  // some sequence has a group on the proxy path
  int64_t max_nk = 0;
  // keys: contiguous (stride) or paged
  const int32_t* pages = nullptr;
  int32_t max_pages = 0, page_shift = 0, n_pages = 0;
  int64_t k_stride = 0;
  // workspace layout
  size_t off_pq = 0, off_psc = 0, off_pw = 0, off_cand = 0, off_scores = 0, fixed = 0;
  size_t off_qlin = 0, off_qlsc = 0, off_plin = 0, off_plsc = 0;  // fp8 epilogue's linear term
  size_t off_rsc = 0;                                              // Refine member scores
  size_t off_sel = 0, sel_bytes = 0;                               // split select scratch
  bool qlin = false, plin = false;
  // App. B window and the proxy aggregation
  int W = 0, wkind = PIVOT_WINDOW_SHARED, agg = PIVOT_AGG_MEAN;
  int rpath = PIVOT_REFINE_AUTO;  // pivot_refine_path
  int wg = 0;          // window union slots (W + g - 1, or 0)
  int width = 0;       // candidate slots per group
  int proxy_m = 0;     // slots the proxy fills (c, or c - wg for the shared window)
  int scan_shift = 0;  // the proxy scans [0, t0 - scan_shift]
};

bool layout_varlen(const pivot_layout* l) { return l && l->cu_q; }
bool layout_paged(const pivot_layout* l) { return l && l->block_table; }

// Checks that need no plan; `nq` receives each sequence's query rows.
pivot_status check_args(const pivot_args* a, const pivot_layout* l, std::vector<int32_t>& nq) {
  if (!a) return fail(PIVOT_ERR_INVALID_ARG, "args is NULL");
  if (a->dtype != PIVOT_DT_BF16 && a->dtype != PIVOT_DT_FP8_E4M3)
    return fail(PIVOT_ERR_UNSUPPORTED, "dtype %d not supported", a->dtype);
  if (a->heads != kH || a->dim != kD)
    return fail(PIVOT_ERR_UNSUPPORTED, "heads=%d dim=%d: this library specialises H=64, d=128", a->heads, a->dim);
  if (a->batch < 1) return fail(PIVOT_ERR_INVALID_ARG, "batch must be >= 1");
  if (a->topk < 1) return fail(PIVOT_ERR_INVALID_ARG, "topk must be >= 1");
  if (!a->q_pos0 || !a->n_k) return fail(PIVOT_ERR_INVALID_ARG, "q_pos0 and n_k (host arrays) are required");
  nq.assign(a->batch, 0);
  if (layout_varlen(l)) {
    if (l->cu_q[0] != 0) return fail(PIVOT_ERR_INVALID_ARG, "cu_q[0] must be 0");
    for (int b = 0; b < a->batch; ++b) {
      if (l->cu_q[b + 1] < l->cu_q[b]) return fail(PIVOT_ERR_INVALID_ARG, "cu_q must be nondecreasing (at %d)", b);
      nq[b] = l->cu_q[b + 1] - l->cu_q[b];
    }
  } else {
    if (a->n_q < 0) return fail(PIVOT_ERR_INVALID_ARG, "n_q must be >= 0");
    nq.assign(a->batch, a->n_q);
  }
  const bool paged = layout_paged(l);
  const int64_t key_bytes = (int64_t)kD * (a->dtype == PIVOT_DT_FP8_E4M3 ? 1 : 2);
  if (paged) {
    const int P = l->page_size;
    if (P < 16 || P > 65536 || (P & (P - 1)))
      return fail(PIVOT_ERR_INVALID_ARG, "page_size=%d must be a power of two in [16, 65536]", P);
    if (l->max_pages < 1) return fail(PIVOT_ERR_INVALID_ARG, "max_pages must be >= 1");
    if (l->pool_keys < P || l->pool_keys % P)
      return fail(PIVOT_ERR_INVALID_ARG, "pool_keys=%lld must be a positive multiple of page_size",
                  (long long)l->pool_keys);
    if (l->pool_keys * key_bytes > ((int64_t)1 << 31))  // 32-bit buffer offsets with room for a drop offset
      return fail(PIVOT_ERR_UNSUPPORTED, "key pool of %lld keys exceeds 2^31 bytes", (long long)l->pool_keys);
  }
  int64_t total = 0;
  for (int b = 0; b < a->batch; ++b) {
    if (a->q_pos0[b] < 0) return fail(PIVOT_ERR_INVALID_ARG, "q_pos0[%d] < 0", b);
    if ((int64_t)a->q_pos0[b] + nq[b] > a->n_k[b])
      return fail(PIVOT_ERR_INVALID_ARG, "n_k[%d]=%d < q_pos0+n_q=%lld", b, a->n_k[b], (long long)a->q_pos0[b] + nq[b]);
    if (paged) {
      if ((int64_t)a->n_k[b] > (int64_t)l->max_pages * l->page_size)
        return fail(PIVOT_ERR_INVALID_ARG, "n_k[%d]=%d exceeds max_pages*page_size", b, a->n_k[b]);
    } else if (a->n_k[b] > a->k_seq_stride) {
      return fail(PIVOT_ERR_INVALID_ARG, "n_k[%d]=%d exceeds k_seq_stride=%lld", b, a->n_k[b],
                  (long long)a->k_seq_stride);
    }
    if (a->n_k[b] > PIVOT_MAX_KEYS)
      return fail(PIVOT_ERR_UNSUPPORTED, "n_k[%d]=%d exceeds PIVOT_MAX_KEYS=%d", b, a->n_k[b], PIVOT_MAX_KEYS);
    total += nq[b];
  }
  if (total > 0x7FFFFFFF) return fail(PIVOT_ERR_UNSUPPORTED, "more than 2^31 query rows");
  if (total > 0) {
    if (!a->q || !a->w || !a->k || !a->out_idx)
      return fail(PIVOT_ERR_INVALID_ARG, "q, w, k and out_idx are required");
    if (a->dtype == PIVOT_DT_FP8_E4M3 && (!a->q_scale || !a->k_scale))
      return fail(PIVOT_ERR_INVALID_ARG, "fp8 inputs need q_scale and k_scale");
  }
  return PIVOT_OK;
}

// Width of a group's candidate row (App. B): c, plus the window union for the
// per-query window.
int cand_width(int c, int g, int W, int wkind) {
  return (W > 0 && wkind == PIVOT_WINDOW_PER_QUERY) ? c + W + g - 1 : c;
}

// ext_cand: Refine writes its candidate sets to the caller's buffer, so the
// workspace reserves none.
pivot_status make_plan(const pivot_args* a, const pivot_layout* l, int mode, int g, int c, int dense_below,
                       bool ext_cand, Plan& p, int W = 0, int wkind = PIVOT_WINDOW_SHARED,
                       int agg = PIVOT_AGG_MEAN, int rpath = PIVOT_REFINE_AUTO) {
  pivot_status s = check_args(a, l, p.nq);
  if (s != PIVOT_OK) return s;
  if (mode != PIVOT_DENSE && mode != PIVOT_REUSE && mode != PIVOT_REFINE)
    return fail(PIVOT_ERR_INVALID_ARG, "mode %d", mode);
  if (agg != PIVOT_AGG_MEAN && agg != PIVOT_AGG_FIRST && agg != PIVOT_AGG_LAST)
    return fail(PIVOT_ERR_INVALID_ARG, "aggregate %d", agg);
  if (wkind != PIVOT_WINDOW_SHARED && wkind != PIVOT_WINDOW_PER_QUERY)
    return fail(PIVOT_ERR_INVALID_ARG, "window_kind %d", wkind);
  if (W < 0) return fail(PIVOT_ERR_INVALID_ARG, "window must be >= 0");
  if (rpath != PIVOT_REFINE_AUTO && rpath != PIVOT_REFINE_FUSED && rpath != PIVOT_REFINE_SPLIT)
    return fail(PIVOT_ERR_INVALID_ARG, "refine_path %d", rpath);
  if (mode != PIVOT_DENSE) {
    if (g < 1) return fail(PIVOT_ERR_INVALID_ARG, "g must be >= 1");
    if (c < 0) return fail(PIVOT_ERR_INVALID_ARG, "c must be >= 0");
    if (W > 0 && mode != PIVOT_REFINE) return fail(PIVOT_ERR_INVALID_ARG, "the window applies to Refine only");
    if (W > 0 && wkind == PIVOT_WINDOW_SHARED && c < W + g - 1)
      return fail(PIVOT_ERR_INVALID_ARG, "the shared window needs c >= W + g - 1");
    if (W > 0 && wkind == PIVOT_WINDOW_PER_QUERY && W < g)
      return fail(PIVOT_ERR_INVALID_ARG, "the per-query window needs W >= g");
    const int64_t width = mode == PIVOT_REFINE ? (int64_t)cand_width(c, g, W, wkind) : c;
    if (mode == PIVOT_REFINE && width < a->topk)
      return fail(PIVOT_ERR_INVALID_ARG, "Refine needs topk <= candidate slots (%lld)", (long long)width);
    if (mode == PIVOT_REFINE && width > 8192) return fail(PIVOT_ERR_UNSUPPORTED, "Refine supports <= 8192 candidates");
    if (mode == PIVOT_REFINE && g > 65535) return fail(PIVOT_ERR_UNSUPPORTED, "Refine supports g <= 65535");
  } else {
    g = 1;
    c = 0;
    W = 0;
    agg = PIVOT_AGG_MEAN;
  }
  p.W = W;
  p.wkind = wkind;
  p.agg = agg;
  p.rpath = rpath;
  p.wg = W > 0 ? W + g - 1 : 0;
  p.width = mode == PIVOT_REFINE ? cand_width(c, g, W, wkind) : c;
  p.proxy_m = (W > 0 && wkind == PIVOT_WINDOW_SHARED) ? c - p.wg : c;
  p.scan_shift = (W > 0 && wkind == PIVOT_WINDOW_SHARED) ? W : 0;
  p.mode = mode;
  p.g = g;
  p.c = c;
  p.dense_below = (mode == PIVOT_DENSE) ? 0 : (dense_below < 0 ? c : dense_below);
  p.B = a->batch;
  p.topk = a->topk;
  p.dtype = a->dtype;
  p.EB = a->dtype == PIVOT_DT_FP8_E4M3 ? 1 : 2;
  p.row_bytes = (size_t)kH * kD * p.EB;
  p.q_pos0.assign(a->q_pos0, a->q_pos0 + p.B);
  p.n_k.assign(a->n_k, a->n_k + p.B);
  p.dense_rows.resize(p.B);
  p.first_proxy.resize(p.B);
  p.row0.resize(p.B);
  p.ng.resize(p.B);
  p.grp0.resize(p.B);
  p.n_q = 0;
  p.n_groups = 0;
  p.rows_total = 0;
  p.groups_total = 0;
  for (int b = 0; b < p.B; ++b) {
    p.row0[b] = (int32_t)p.rows_total;
    p.grp0[b] = (int32_t)p.groups_total;
    p.ng[b] = (int32_t)cdiv(p.nq[b], g);
    p.rows_total += p.nq[b];
    p.groups_total += p.ng[b];
    p.n_q = std::max(p.n_q, p.nq[b]);
    p.n_groups = std::max(p.n_groups, p.ng[b]);
  }
  if (p.groups_total > 0x7FFFFFFF / std::max(1, p.width))
    return fail(PIVOT_ERR_UNSUPPORTED, "candidate rows exceed 2^31 entries");
  if (layout_paged(l)) {
    p.pages = l->block_table;
    p.max_pages = l->max_pages;
    p.page_shift = __builtin_ctz((unsigned)l->page_size);
    p.n_pages = (int32_t)(l->pool_keys / l->page_size);
  } else {
    p.k_stride = a->k_seq_stride;
  }
  p.dense_hi = 0;
  p.proxy_lo = p.n_groups;
  p.any_proxy = false;
  p.max_nk = 0;
  for (int b = 0; b < p.B; ++b) {
    int J;
    if (mode == PIVOT_DENSE) {
      J = p.ng[b];
    } else {
      const int64_t gap = (int64_t)p.dense_below - p.q_pos0[b];  // groups with t0 < dense_below
      J = gap <= 0 ? 0 : (int)std::min<int64_t>(cdiv(gap, g), p.ng[b]);
    }
    p.first_proxy[b] = J;
    p.dense_rows[b] = (int)std::min<int64_t>((int64_t)J * g, p.nq[b]);
    p.dense_hi = std::max(p.dense_hi, p.dense_rows[b]);
    if (J < p.ng[b]) {
      p.proxy_lo = std::min(p.proxy_lo, J);
      p.any_proxy = mode != PIVOT_DENSE;
    }
    p.max_nk = std::max<int64_t>(p.max_nk, p.n_k[b]);
  }
  if (!p.any_proxy) p.proxy_lo = p.n_groups;
  // workspace layout
  size_t off = 0;
  const size_t ng = (size_t)p.groups_total;
  const bool fp8 = p.dtype == PIVOT_DT_FP8_E4M3;
  const bool proxies = p.any_proxy;
  // query rows need the linear term when scored densely or re-scored by Refine
  p.qlin = fp8 && (p.dense_hi > 0 || (proxies && mode == PIVOT_REFINE));
  p.plin = fp8 && proxies;
  if (p.qlin) {
    const size_t nq = (size_t)p.rows_total;
    p.off_qlin = off;
    off = align_up(off + nq * kLinBytes);
    p.off_qlsc = off;
    off = align_up(off + nq * kLinLevels * sizeof(float));
  }
  if (p.plin) {
    p.off_plin = off;
    off = align_up(off + ng * kLinBytes);
    p.off_plsc = off;
    off = align_up(off + ng * kLinLevels * sizeof(float));
  }
  if (proxies) {
    p.off_pq = off;
    off = align_up(off + ng * p.row_bytes);
    p.off_psc = off;
    off = align_up(off + ng * sizeof(float));
    p.off_pw = off;
    off = align_up(off + ng * kH * sizeof(float));
    if (mode == PIVOT_REFINE) {
      p.off_rsc = off;
      off = align_up(off + ng * (size_t)g * p.width * score_eb(p.dtype));
      p.off_cand = off;
      if (!ext_cand) off = align_up(off + ng * (size_t)p.width * sizeof(int32_t));
    }
  }
  if (p.max_nk >= kSplitMinKeys) {  // few long rows per select launch (decode) split over workgroups
    const int64_t rows = (int64_t)p.B * std::max(p.n_q, p.n_groups);
    p.off_sel = off;
    p.sel_bytes = split_scratch_bytes(std::min<int64_t>(kSplitMaxRows, rows));
    off = align_up(off + p.sel_bytes);
  }
  p.off_scores = off;
  p.fixed = off;
  return PIVOT_OK;
}

// Bytes of scores for the whole call at once, and for the smallest tile.
void score_need(const Plan& p, int64_t& full, int64_t& min_tile) {
  full = 0;
  min_tile = 0;
  const int64_t ld = ld_for(p.max_nk), eb = score_eb(p.dtype);
  if (p.dense_hi > 0) {
    const int64_t rows = (p.B == 1) ? p.dense_hi : (int64_t)p.B * p.dense_hi;
    full = std::max(full, rows * ld * eb);
    min_tile = std::max(min_tile, std::min<int64_t>(16, p.dense_hi) * ld * eb);
  }
  if (p.any_proxy) {
    const int64_t span = p.n_groups - p.proxy_lo;
    const int64_t rows = (p.B == 1) ? span : (int64_t)p.B * span;
    full = std::max(full, rows * ld * eb);
    min_tile = std::max(min_tile, std::min<int64_t>(16, span) * ld * eb);
  }
}

size_t recommended_bytes(const Plan& p) {
  int64_t full, min_tile;
  score_need(p, full, min_tile);
  const int64_t scores = std::min(full, std::max(min_tile, kDefaultScoreBytes));
  return p.fixed + (size_t)scores;
}

// Sequences b0 .. b0 + nb - 1 as one launch sees them: row and group offsets
// relative to the first, so the launch's array pointers start at
// row0[b0] / grp0[b0].  shift: subtracted from the query positions for the
// row limits (the shared window's proxy scans [0, t0 - W]); may make early
// limits negative.
SeqTable table_for(const Plan& p, int b0, int nb, int shift = 0) {
  SeqTable st;
  memset(&st, 0, sizeof st);
  st.n = nb;
  for (int u = 0; u < nb; ++u) {
    st.q_pos0[u] = p.q_pos0[b0 + u] - shift;
    st.dense_rows[u] = p.dense_rows[b0 + u];
    st.first_proxy[u] = p.first_proxy[b0 + u];
    st.n_rows[u] = p.nq[b0 + u];
    st.row0[u] = p.row0[b0 + u] - p.row0[b0];
    st.grp0[u] = p.grp0[b0 + u] - p.grp0[b0];
  }
  return st;
}

// Keys of sequences b0 .. : the key arrays' base and the map of a launch.
struct KeyBase {
  const uint8_t* k;
  const float* ks;
  KeyMap map;
};
KeyBase keys_for(const pivot_args* a, const Plan& p, int b0) {
  KeyBase kb;
  kb.map.max_pages = p.max_pages;
  kb.map.shift = p.page_shift;
  kb.map.n_pages = p.n_pages;
  kb.map.stride = p.k_stride;
  if (p.pages) {  // the pool is shared: only the page table moves
    kb.k = (const uint8_t*)a->k;
    kb.ks = a->k_scale;
    kb.map.pages = p.pages + (size_t)b0 * p.max_pages;
  } else {
    kb.k = (const uint8_t*)a->k + (size_t)b0 * p.k_stride * kD * p.EB;
    kb.ks = a->k_scale ? a->k_scale + (size_t)b0 * p.k_stride : nullptr;
    kb.map.pages = nullptr;
  }
  return kb;
}

// Largest limit of an active row of rs in any sequence of st.
int64_t max_limit(const SeqTable& st, const RowSpace& rs) {
  int64_t lim = -1;
  for (int b = 0; b < st.n; ++b) {
    int hi = std::min(rs.i1, rs.kind == kProxyRows ? (st.n_rows[b] + rs.step - 1) / rs.step : st.n_rows[b]);
    int lo = rs.i0;
    if (rs.kind == kDenseRows) hi = std::min(hi, st.dense_rows[b]);
    if (rs.kind == kProxyRows) lo = std::max(lo, st.first_proxy[b]);
    if (hi > lo) lim = std::max(lim, (int64_t)st.q_pos0[b] + (int64_t)(hi - 1) * rs.step);
  }
  return lim;
}

struct RowData {
  const void* q;
  const float* qs;
  const float* w;
  const uint8_t* lin;  // fp8 only
  const float* lsc;
  bool groups;         // the rows are groups (proxies), else query rows
};

// Score and select rows [lo, hi) of each sequence, tiled to the score budget:
// several whole sequences per tile when they fit, else row tiles of one.
pivot_status run_rows(const pivot_args* a, const Plan& p, int kind, int lo, int hi, int step,
                      const RowData& rd_all, OutDesc od_all, void* scores, int64_t score_bytes,
                      hipStream_t stream, int lim_shift = 0) {
  if (hi <= lo) return PIVOT_OK;
  const int64_t ld_max = ld_for(p.max_nk);
  const int64_t row_bytes = ld_max * score_eb(p.dtype);
  const bool sb16 = bf16_scores(p.dtype);
  int seqs_per_tile, rows_per_tile;
  if (p.B > 1 && score_bytes / (row_bytes * (hi - lo)) >= 1) {
    rows_per_tile = hi - lo;
    seqs_per_tile = (int)std::min<int64_t>(score_bytes / (row_bytes * (hi - lo)), kMaxSeq);
  } else {
    seqs_per_tile = 1;
    int64_t r = score_bytes / row_bytes;
    r = std::max<int64_t>(16, r / 16 * 16);
    rows_per_tile = (int)std::min<int64_t>(r, hi - lo);
  }
  if ((int64_t)seqs_per_tile * rows_per_tile * row_bytes > score_bytes)
    return fail(PIVOT_ERR_WORKSPACE, "workspace too small for one score tile");
  for (int b0 = 0; b0 < p.B; b0 += seqs_per_tile) {
    const int nb = std::min(seqs_per_tile, p.B - b0);
    SeqTable st = table_for(p, b0, nb, lim_shift);
    const size_t r0 = rd_all.groups ? (size_t)p.grp0[b0] : (size_t)p.row0[b0];
    RowData rd = rd_all;
    rd.q = (const uint8_t*)rd_all.q + r0 * p.row_bytes;
    rd.qs = rd_all.qs ? rd_all.qs + r0 : nullptr;
    rd.w = rd_all.w + r0 * kH;
    rd.lin = rd_all.lin ? rd_all.lin + r0 * kLinBytes : nullptr;
    rd.lsc = rd_all.lsc ? rd_all.lsc + r0 * kLinLevels : nullptr;
    const KeyBase kb = keys_for(a, p, b0);
    OutDesc od = od_all;
    od.base = od_all.base + (size_t)(od_all.fan_g == 0 && od_all.groups ? p.grp0[b0] : p.row0[b0]) * od_all.ld;
    for (int i0 = lo; i0 < hi; i0 += rows_per_tile) {
      RowSpace rs{i0, std::min(hi, i0 + rows_per_tile), step, kind};
      const int64_t lim = max_limit(st, rs);
      const int64_t ld = ld_for(std::max<int64_t>(lim, 0) + 1);
      pivot_status s = PIVOT_OK;
      if (lim >= 0)  // no key in reach (shifted limits): the select only pads with -1
        s = hip_check(timed(PIVOT_KERNEL_SCORE, stream, [&] {
                        return launch_score(p.dtype, rd.q, rd.qs, rd.w, rd.lin, rd.lsc, kb.k, kb.ks, kb.map, st, rs,
                                            lim, scores, sb16, ld, stream);
                      }),
                      "score kernel");
      if (s != PIVOT_OK) return s;
      s = hip_check(timed(PIVOT_KERNEL_SELECT, stream,
                          [&] {
                            return launch_topk(scores, sb16, ld, st, rs, od, lim,
                                               p.sel_bytes ? (uint8_t*)a->workspace + p.off_sel : nullptr,
                                               p.sel_bytes, stream);
                          }),
                    "top-k kernel");
      if (s != PIVOT_OK) return s;
    }
  }
  return PIVOT_OK;
}

pivot_status check_workspace(const pivot_args* a, const Plan& p, int64_t& score_bytes) {
  int64_t full, min_tile;
  score_need(p, full, min_tile);
  const size_t need_min = p.fixed + (size_t)min_tile;
  if (need_min > 0) {
    if (!a->workspace) return fail(PIVOT_ERR_WORKSPACE, "workspace is NULL (need >= %zu bytes)", need_min);
    if (reinterpret_cast<uintptr_t>(a->workspace) % kAlign)
      return fail(PIVOT_ERR_INVALID_ARG, "workspace must be %zu-byte aligned", kAlign);
    if (a->workspace_bytes < need_min)
      return fail(PIVOT_ERR_WORKSPACE, "workspace_bytes=%zu < minimum %zu", a->workspace_bytes, need_min);
  }
  score_bytes = (int64_t)(a->workspace_bytes - p.fixed);
  return PIVOT_OK;
}

// Query rows that need the fp8 linear term (mfma_tile.h): the leading dense
// rows of a single sequence, else every row (a batch, or Refine re-scoring
// the members).
int64_t query_lin_rows(const Plan& p) {
  return (p.B == 1 && p.mode != PIVOT_REFINE) ? p.dense_hi : p.rows_total;
}

pivot_status query_lin(const pivot_args* a, const Plan& p, uint8_t* ws, hipStream_t stream) {
  if (!p.qlin) return PIVOT_OK;
  const int64_t rows = query_lin_rows(p);
  return hip_check(timed(PIVOT_KERNEL_LIN, stream, [&] {
                     return launch_lin(a->q, a->q_scale, a->w, 0, rows, ws + p.off_qlin,
                                       reinterpret_cast<float*>(ws + p.off_qlsc), stream);
                   }),
                   "linear-term kernel");
}

pivot_status dense_part(const pivot_args* a, const Plan& p, void* scores, int64_t score_bytes, hipStream_t stream) {
  uint8_t* ws = (uint8_t*)a->workspace;
  const bool fp8 = a->dtype == PIVOT_DT_FP8_E4M3;
  RowData rd{a->q, fp8 ? a->q_scale : nullptr, a->w, fp8 ? ws + p.off_qlin : nullptr,
             fp8 ? reinterpret_cast<const float*>(ws + p.off_qlsc) : nullptr, false};
  OutDesc od{a->out_idx, p.topk, 0, 0, p.topk};
  const int kind = p.mode == PIVOT_DENSE ? kAll : kDenseRows;
  return run_rows(a, p, kind, 0, p.dense_hi, 1, rd, od, scores, score_bytes, stream);
}

// Sizing validates the shape only: the pointers get non-null stand-ins.
pivot_args shape_of(const pivot_args* a) {
  pivot_args shape = *a;
  static const float dummy = 0.f;
  shape.q = shape.k = &dummy;
  shape.w = shape.q_scale = shape.k_scale = &dummy;
  shape.out_idx = reinterpret_cast<int32_t*>(const_cast<float*>(&dummy));
  return shape;
}

pivot_status group_plan(const pivot_args* a, const pivot_layout* l, const pivot_group_opts* o, bool ext_cand,
                        Plan& p) {
  if (!o) return fail(PIVOT_ERR_INVALID_ARG, "opts is NULL");
  if (o->mode != PIVOT_REUSE && o->mode != PIVOT_REFINE) return fail(PIVOT_ERR_INVALID_ARG, "mode %d", o->mode);
  return make_plan(a, l, o->mode, o->g, o->c, o->dense_below, ext_cand, p, o->window, o->window_kind, o->aggregate,
                   o->refine_path);
}

pivot_status dense_index(const pivot_args* a, const pivot_layout* l) {
  Plan p;
  pivot_status s = make_plan(a, l, PIVOT_DENSE, 1, 0, 0, false, p);
  if (s != PIVOT_OK) return s;
  if (p.rows_total == 0) return PIVOT_OK;
  int64_t score_bytes;
  s = check_workspace(a, p, score_bytes);
  if (s != PIVOT_OK) return s;
  void* scores = (uint8_t*)a->workspace + p.off_scores;
  s = query_lin(a, p, (uint8_t*)a->workspace, (hipStream_t)a->stream);
  if (s != PIVOT_OK) return s;
  return dense_part(a, p, scores, score_bytes, (hipStream_t)a->stream);
}

pivot_status group_index(const pivot_args* a, const pivot_layout* l, const pivot_group_opts* o) {
  Plan p;
  pivot_status s = group_plan(a, l, o, o && o->out_cand != nullptr && o->mode == PIVOT_REFINE, p);
  if (s != PIVOT_OK) return s;
  if (p.rows_total == 0) return PIVOT_OK;
  const int mode = p.mode;
  int32_t* out_cand = mode == PIVOT_REFINE ? o->out_cand : nullptr;
  const int width = p.width;
  hipStream_t stream = (hipStream_t)a->stream;
  int64_t score_bytes;
  s = check_workspace(a, p, score_bytes);
  if (s != PIVOT_OK) return s;
  uint8_t* ws = (uint8_t*)a->workspace;
  void* scores = ws + p.off_scores;

  void* pq = ws + p.off_pq;
  float* psc = reinterpret_cast<float*>(ws + p.off_psc);
  float* pw = reinterpret_cast<float*>(ws + p.off_pw);
  int32_t* cand = (mode == PIVOT_REFINE) ? (out_cand ? out_cand : reinterpret_cast<int32_t*>(ws + p.off_cand))
                                         : nullptr;
  const float* qs = p.dtype == PIVOT_DT_FP8_E4M3 ? a->q_scale : nullptr;

  // fp8 linear terms (mfma_tile.h): the proxy kernel writes those of the
  // proxies, and for Refine those of the members it reads, unless some
  // sequence of a batch also has dense rows (then every query row is done by
  // the linear-term kernel, which needs a contiguous range)
  uint8_t* plin = p.plin ? ws + p.off_plin : nullptr;
  float* plsc = p.plin ? reinterpret_cast<float*>(ws + p.off_plsc) : nullptr;
  uint8_t* qlin = p.qlin ? ws + p.off_qlin : nullptr;
  float* qlsc = p.qlin ? reinterpret_cast<float*>(ws + p.off_qlsc) : nullptr;
  const bool member_lin = p.plin && p.qlin && mode == PIVOT_REFINE && (p.B == 1 || p.dense_hi == 0);
  if (p.any_proxy)
    for (int b0 = 0; b0 < p.B; b0 += kMaxSeq) {  // Eq. 4 proxies (or the first / last member)
      const int nb = std::min(kMaxSeq, p.B - b0);
      SeqTable st = table_for(p, b0, nb);
      const size_t qoff = (size_t)p.row0[b0];
      const size_t poff = (size_t)p.grp0[b0];
      LinOut lo;
      if (p.plin) {
        lo.plin = plin + poff * kLinBytes;
        lo.plsc = plsc + poff * kLinLevels;
      }
      if (member_lin) {
        lo.qlin = qlin + qoff * kLinBytes;
        lo.qlsc = qlsc + qoff * kLinLevels;
      }
      s = hip_check(timed(PIVOT_KERNEL_PROXY, stream, [&] {
                      return launch_proxy(p.dtype, (const uint8_t*)a->q + qoff * p.row_bytes,
                                          qs ? qs + qoff : nullptr, a->w + qoff * kH, p.g, st, p.proxy_lo,
                                          p.n_groups, false, p.agg, (uint8_t*)pq + poff * p.row_bytes, psc + poff,
                                          pw + poff * kH, stream, lo);
                    }),
                    "proxy kernel");
      if (s != PIVOT_OK) return s;
    }

  // the remaining query rows' linear terms: the dense rows, or every row
  if (p.qlin) {
    const int64_t rows = member_lin ? (p.B == 1 ? p.dense_hi : 0) : query_lin_rows(p);
    if (rows > 0) {
      s = hip_check(timed(PIVOT_KERNEL_LIN, stream, [&] {
                      return launch_lin(LinRows{(const uint8_t*)a->q, a->q_scale, a->w, 0, rows, qlin, qlsc},
                                        LinRows{}, stream);
                    }),
                    "linear-term kernel");
      if (s != PIVOT_OK) return s;
    }
  }

  s = dense_part(a, p, scores, score_bytes, stream);  // guardrail groups (Algorithm 1)
  if (s != PIVOT_OK) return s;
  if (!p.any_proxy) {
    if (out_cand)
      for (int b0 = 0; b0 < p.B; b0 += kMaxSeq) {
        const int nb = std::min(kMaxSeq, p.B - b0);
        SeqTable st = table_for(p, b0, nb);
        s = hip_check(timed(PIVOT_KERNEL_FILL, stream, [&] {
                        return launch_fill_guardrail(out_cand + (size_t)p.grp0[b0] * width, width, st, 0, p.n_groups,
                                                     -1, stream);
                      }),
                      "fill kernel");
        if (s != PIVOT_OK) return s;
      }
    return PIVOT_OK;
  }

  // Eq. 5 proxy scan, then Eq. 6 (Reuse: top-k shared by the members) or
  // Eq. 7 (Refine: top-c candidates; before a shared window, the top c - W - g + 1
  // over [0, t0 - W])
  RowData rd{pq, p.dtype == PIVOT_DT_FP8_E4M3 ? psc : nullptr, pw, plin, plsc, true};
  OutDesc od = (mode == PIVOT_REUSE) ? OutDesc{a->out_idx, p.topk, p.g, 0, p.topk}
                                     : OutDesc{cand, p.proxy_m, 0, 1, width};
  if (od.m > 0) {
    s = run_rows(a, p, kProxyRows, p.proxy_lo, p.n_groups, p.g, rd, od, scores, score_bytes, stream, p.scan_shift);
    if (s != PIVOT_OK) return s;
  }
  if (mode == PIVOT_REUSE) return PIVOT_OK;

  for (int b0 = 0; b0 < p.B; b0 += kMaxSeq) {  // App. B window, Eqs. 8-9
    const int nb = std::min(kMaxSeq, p.B - b0);
    SeqTable st = table_for(p, b0, nb);
    const size_t qoff = (size_t)p.row0[b0];
    const size_t goff = (size_t)p.grp0[b0];
    int32_t* cb = cand + goff * width;
    if (out_cand) {
      s = hip_check(timed(PIVOT_KERNEL_FILL, stream,
                          [&] { return launch_fill_guardrail(cb, width, st, 0, p.n_groups, -1, stream); }),
                    "fill kernel");
      if (s != PIVOT_OK) return s;
    }
    if (p.W > 0) {
      s = hip_check(timed(PIVOT_KERNEL_FILL, stream, [&] {
                      return launch_window(cb, p.g, st, p.proxy_lo, p.n_groups, width, p.proxy_m, p.W,
                                           p.wkind == PIVOT_WINDOW_PER_QUERY, stream);
                    }),
                    "window kernel");
      if (s != PIVOT_OK) return s;
    }
    const int wslot = p.wkind == PIVOT_WINDOW_PER_QUERY ? p.proxy_m : width;
    const KeyBase kb = keys_for(a, p, b0);
    s = hip_check(timed(PIVOT_KERNEL_REFINE, stream, [&] {
                    return launch_refine(p.dtype, (const uint8_t*)a->q + qoff * p.row_bytes,
                                         qs ? qs + qoff : nullptr, a->w + qoff * kH,
                                         p.qlin ? ws + p.off_qlin + qoff * kLinBytes : nullptr,
                                         p.qlin ? reinterpret_cast<const float*>(ws + p.off_qlsc) + qoff * kLinLevels
                                                : nullptr,
                                         p.g, kb.k, kb.ks, kb.map, st, p.proxy_lo, p.n_groups, cb, width, p.W, wslot,
                                         p.topk, ws + p.off_rsc + goff * p.g * width * score_eb(p.dtype),
                                         a->out_idx + qoff * p.topk, p.rpath, stream);
                  }),
                  "refine kernel");
    if (s != PIVOT_OK) return s;
  }
  return PIVOT_OK;
}

// PIVOT composed with IndexCache over n_layers layers (Sec. 5.1, the +IC rows
// of Table 1): anchors are indexed on their own inputs, each run of followers
// gets the preceding anchor's sets through one fan-out copy.  Everything is
// validated before the first launch.
pivot_status index_layers(const pivot_args* L, int n_layers, int stride, const uint8_t* anchors,
                          const pivot_group_opts* o) {
  if (!L) return fail(PIVOT_ERR_INVALID_ARG, "layers is NULL");
  if (n_layers < 1) return fail(PIVOT_ERR_INVALID_ARG, "n_layers must be >= 1");
  if (!anchors && stride < 1) return fail(PIVOT_ERR_INVALID_ARG, "stride must be >= 1");
  auto anchor = [&](int l) { return anchors ? anchors[l] != 0 : l % stride == 0; };
  if (!anchor(0)) return fail(PIVOT_ERR_INVALID_ARG, "layer 0 must be an anchor");
  if (o && o->out_cand) return fail(PIVOT_ERR_INVALID_ARG, "out_cand must be NULL across layers");
  const pivot_args& a0 = L[0];
  std::vector<int32_t> nq0;
  pivot_status s = check_args(&a0, nullptr, nq0);
  if (s != PIVOT_OK) return s;
  const int64_t rows = (int64_t)a0.batch * a0.n_q;
  for (int l = 1; l < n_layers; ++l) {
    const pivot_args& a = L[l];
    if (a.dtype != a0.dtype || a.heads != a0.heads || a.dim != a0.dim || a.batch != a0.batch || a.n_q != a0.n_q ||
        a.topk != a0.topk || a.k_seq_stride != a0.k_seq_stride)
      return fail(PIVOT_ERR_INVALID_ARG, "layer %d: shape or parameters differ from layer 0", l);
    if (!a.q_pos0 || !a.n_k) return fail(PIVOT_ERR_INVALID_ARG, "layer %d: q_pos0 and n_k are required", l);
    for (int b = 0; b < a0.batch; ++b)
      if (a.q_pos0[b] != a0.q_pos0[b] || a.n_k[b] != a0.n_k[b])
        return fail(PIVOT_ERR_INVALID_ARG, "layer %d: positions of sequence %d differ from layer 0", l, b);
    if (rows > 0 && !a.out_idx) return fail(PIVOT_ERR_INVALID_ARG, "layer %d: out_idx is required", l);
  }
  // every anchor as its own call would see it: layer 0's workspace and stream
  auto as_anchor = [&](int l) {
    pivot_args a = L[l];
    a.workspace = a0.workspace;
    a.workspace_bytes = a0.workspace_bytes;
    a.stream = a0.stream;
    return a;
  };
  // arguments of every anchor first, then the workspace each one needs
  for (int pass = 0; pass < 2; ++pass)
    for (int l = 0; l < n_layers; ++l) {
      if (!anchor(l)) continue;
      const pivot_args a = as_anchor(l);
      Plan p;
      s = o ? group_plan(&a, nullptr, o, false, p) : make_plan(&a, nullptr, PIVOT_DENSE, 1, 0, 0, false, p);
      if (s == PIVOT_OK && pass == 1 && p.rows_total > 0) {
        int64_t score_bytes;
        s = check_workspace(&a, p, score_bytes);
      }
      if (s != PIVOT_OK) {
        char why[sizeof g_err];
        snprintf(why, sizeof why, "%s", g_err);
        return fail(s, "layer %d: %s", l, why);
      }
    }
  if (rows == 0) return PIVOT_OK;
  hipStream_t stream = (hipStream_t)a0.stream;
  const int64_t n = rows * a0.topk;
  int src = 0;
  for (int l = 0; l < n_layers;) {
    if (anchor(l)) {
      const pivot_args a = as_anchor(l);
      s = o ? group_index(&a, nullptr, o) : dense_index(&a, nullptr);
      if (s != PIVOT_OK) return s;
      src = l++;
      continue;
    }
    int e = l;
    while (e < n_layers && !anchor(e)) ++e;
    for (int f = l; f < e; f += kMaxCopyDst) {  // one read of the anchor's sets per launch
      int32_t* dst[kMaxCopyDst];
      const int nd = std::min(kMaxCopyDst, e - f);
      for (int u = 0; u < nd; ++u) dst[u] = L[f + u].out_idx;
      s = hip_check(timed(PIVOT_KERNEL_COPY, stream,
                          [&] { return launch_copy_fanout(L[src].out_idx, dst, nd, n, stream); }),
                    "copy kernel");
      if (s != PIVOT_OK) return s;
    }
    l = e;
  }
  return PIVOT_OK;
}

// ---- the no-alloc variant's scratch address per device ----
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, looked up once per device.
pivot_status static_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_check(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(PIVOT_ERR_UNSUPPORTED, "device %d: scratch tracked for %d devices", dev,
                                                 kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_check(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(PIVOT_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return PIVOT_OK;
}

pivot_status group_index_noalloc(const pivot_args* a, const pivot_group_opts* o) {
  if (!a) return fail(PIVOT_ERR_INVALID_ARG, "args is NULL");
  Plan p;  // the size check comes before any HIP call
  pivot_status s = group_plan(a, nullptr, o, o && o->out_cand != nullptr && o->mode == PIVOT_REFINE, p);
  if (s != PIVOT_OK) return s;
  if (p.rows_total == 0) return PIVOT_OK;
  int64_t full, min_tile;
  score_need(p, full, min_tile);
  const size_t need = p.fixed + (size_t)min_tile;
  if (need > PIVOT_NOALLOC_SCRATCH_BYTES)
    return fail(PIVOT_ERR_WORKSPACE, "the call needs %zu bytes of scratch; the no-alloc scratch holds %zu", need,
                (size_t)PIVOT_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  s = static_scratch(&ws);
  if (s != PIVOT_OK) return s;
  pivot_args b = *a;
  b.workspace = ws;
  b.workspace_bytes = PIVOT_NOALLOC_SCRATCH_BYTES;
  return group_index(&b, nullptr, o);
}

pivot_group_opts plain_opts(int32_t mode, int32_t g, int32_t c, int32_t dense_below, int32_t* out_cand) {
  pivot_group_opts o;
  memset(&o, 0, sizeof o);
  o.mode = mode;
  o.g = g;
  o.c = c;
  o.dense_below = dense_below;
  o.window = 0;
  o.window_kind = PIVOT_WINDOW_SHARED;
  o.aggregate = PIVOT_AGG_MEAN;
  o.out_cand = out_cand;
  return o;
}

}  // namespace

extern "C" {

size_t pivot_workspace_size_layout(const pivot_args* a, const pivot_layout* l, const pivot_group_opts* o) {
  if (!a) return 0;
  pivot_args shape = shape_of(a);
  Plan p;
  if (!o) {
    if (make_plan(&shape, l, PIVOT_DENSE, 1, 0, 0, false, p) != PIVOT_OK) return 0;
    return recommended_bytes(p);
  }
  pivot_group_opts oc = *o;
  oc.out_cand = nullptr;
  if (group_plan(&shape, l, &oc, false, p) != PIVOT_OK) return 0;
  return recommended_bytes(p);
}

size_t pivot_workspace_size(const pivot_args* a, int32_t mode, int32_t g, int32_t c) {
  if (!a) return 0;
  if (mode == PIVOT_DENSE) return pivot_workspace_size_layout(a, nullptr, nullptr);
  const pivot_group_opts o = plain_opts(mode, g, c, c, nullptr);
  return pivot_workspace_size_layout(a, nullptr, &o);
}

int32_t pivot_cand_width(const pivot_group_opts* o) {
  if (!o) return 0;
  return cand_width(o->c, o->g, o->window, o->window_kind);
}

size_t pivot_group_workspace_size(const pivot_args* a, const pivot_group_opts* o) {
  if (!o) return 0;
  return pivot_workspace_size_layout(a, nullptr, o);
}

pivot_status pivot_dense_index(const pivot_args* a) { return dense_index(a, nullptr); }

pivot_status pivot_dense_index_layout(const pivot_args* a, const pivot_layout* l) { return dense_index(a, l); }

pivot_status pivot_group_index(const pivot_args* a, int32_t mode, int32_t g, int32_t c, int32_t dense_below,
                               int32_t* out_cand) {
  const pivot_group_opts o = plain_opts(mode, g, c, dense_below, out_cand);
  return group_index(a, nullptr, &o);
}

pivot_status pivot_group_index_opts(const pivot_args* a, const pivot_group_opts* o) {
  return group_index(a, nullptr, o);
}

pivot_status pivot_group_index_layout(const pivot_args* a, const pivot_layout* l, const pivot_group_opts* o) {
  return group_index(a, l, o);
}

pivot_status pivot_group_index_noalloc(const pivot_args* a, const pivot_group_opts* o) {
  return group_index_noalloc(a, o);
}

pivot_status pivot_index_layers(const pivot_args* layers, int32_t n_layers, int32_t stride, const uint8_t* anchors,
                                const pivot_group_opts* o) {
  return index_layers(layers, n_layers, stride, anchors, o);
}

pivot_status pivot_proxy_rows(int32_t dtype, int32_t heads, int32_t dim, int32_t n_q, int32_t g, const void* q,
                              const float* q_scale, const float* w, void* out_q, float* out_scale, float* out_w,
                              void* stream) {
  if (dtype != PIVOT_DT_BF16 && dtype != PIVOT_DT_FP8_E4M3) return fail(PIVOT_ERR_UNSUPPORTED, "dtype %d", dtype);
  if (heads != kH || dim != kD) return fail(PIVOT_ERR_UNSUPPORTED, "heads=%d dim=%d", heads, dim);
  if (n_q < 0 || g < 1) return fail(PIVOT_ERR_INVALID_ARG, "n_q >= 0 and g >= 1 required");
  if (n_q == 0) return PIVOT_OK;
  if (!q || !w || !out_q || !out_scale || !out_w || (dtype == PIVOT_DT_FP8_E4M3 && !q_scale))
    return fail(PIVOT_ERR_INVALID_ARG, "null pointer");
  SeqTable st;
  memset(&st, 0, sizeof st);
  st.n = 1;
  st.n_rows[0] = n_q;
  const int ng = (int)cdiv(n_q, g);
  return hip_check(launch_proxy(dtype, q, dtype == PIVOT_DT_FP8_E4M3 ? q_scale : nullptr, w, g, st, 0, ng, true,
                                PIVOT_AGG_MEAN, out_q, out_scale, out_w, (hipStream_t)stream),
                   "proxy kernel");
}

pivot_status pivot_score_rows(int32_t dtype, int32_t heads, int32_t dim, int32_t n_rows, const void* q,
                              const float* q_scale, const float* w, const void* k, const float* k_scale,
                              int64_t lim0, int32_t lim_step, float* out, int64_t ld, void* workspace,
                              size_t workspace_bytes, void* stream) {
  if (dtype != PIVOT_DT_BF16 && dtype != PIVOT_DT_FP8_E4M3) return fail(PIVOT_ERR_UNSUPPORTED, "dtype %d", dtype);
  if (heads != kH || dim != kD) return fail(PIVOT_ERR_UNSUPPORTED, "heads=%d dim=%d", heads, dim);
  if (n_rows < 0 || lim0 < 0 || lim_step < 0) return fail(PIVOT_ERR_INVALID_ARG, "negative size");
  if (n_rows == 0) return PIVOT_OK;
  if (!q || !w || !k || !out || (dtype == PIVOT_DT_FP8_E4M3 && (!q_scale || !k_scale)))
    return fail(PIVOT_ERR_INVALID_ARG, "null pointer");
  const int64_t lim_max = lim0 + (int64_t)(n_rows - 1) * lim_step;
  if (lim_max > 0x7FFFFFFE) return fail(PIVOT_ERR_INVALID_ARG, "limits exceed int32 positions");
  if (ld < lim_max + 1) return fail(PIVOT_ERR_INVALID_ARG, "ld=%lld < %lld", (long long)ld, (long long)lim_max + 1);
  if (ld > PIVOT_MAX_KEYS)
    return fail(PIVOT_ERR_UNSUPPORTED, "ld=%lld exceeds PIVOT_MAX_KEYS=%d", (long long)ld, PIVOT_MAX_KEYS);
  const bool fp8 = dtype == PIVOT_DT_FP8_E4M3;
  const size_t lin_off = align_up((size_t)n_rows * kLinBytes);
  const size_t need = fp8 ? lin_off + (size_t)n_rows * kLinLevels * sizeof(float) : 0;
  if (need > 0) {
    if (!workspace || workspace_bytes < need)
      return fail(PIVOT_ERR_WORKSPACE, "score rows need %zu workspace bytes", need);
    if (reinterpret_cast<uintptr_t>(workspace) % kAlign)
      return fail(PIVOT_ERR_INVALID_ARG, "workspace must be %zu-byte aligned", kAlign);
  }
  uint8_t* lin = fp8 ? (uint8_t*)workspace : nullptr;
  float* lsc = fp8 ? reinterpret_cast<float*>((uint8_t*)workspace + lin_off) : nullptr;
  SeqTable st;
  memset(&st, 0, sizeof st);
  st.n = 1;
  st.q_pos0[0] = (int32_t)lim0;
  st.n_rows[0] = n_rows;
  RowSpace rs{0, n_rows, lim_step, kAll};
  if (fp8) {
    pivot_status s = hip_check(launch_lin(q, q_scale, w, 0, n_rows, lin, lsc, (hipStream_t)stream),
                               "linear-term kernel");
    if (s != PIVOT_OK) return s;
  }
  KeyMap km;
  memset(&km, 0, sizeof km);  // one sequence of contiguous keys
  return hip_check(launch_score(dtype, q, fp8 ? q_scale : nullptr, w, lin, lsc, k, fp8 ? k_scale : nullptr, km, st,
                                rs, lim_max, out, false, ld, (hipStream_t)stream),
                   "score kernel");
}

size_t pivot_topk_rows_workspace_size(int32_t n_rows) {
  if (n_rows <= 0 || n_rows > kSplitMaxRows) return 0;
  return split_scratch_bytes(n_rows);
}

pivot_status pivot_topk_rows(int32_t n_rows, const float* scores, int64_t ld, int64_t n0, int32_t n_step, int32_t m,
                             int32_t* out, void* stream) {
  return pivot_topk_rows_ws(n_rows, scores, ld, n0, n_step, m, out, nullptr, 0, stream);
}

pivot_status pivot_topk_rows_bf16(int32_t n_rows, const uint16_t* scores, int64_t ld, int64_t n0, int32_t n_step,
                                  int32_t m, int32_t* out, void* stream) {
  if (n_rows < 0 || n0 < 0 || n_step < 0 || m < 1) return fail(PIVOT_ERR_INVALID_ARG, "bad size");
  if (n_rows == 0) return PIVOT_OK;
  if (!scores || !out) return fail(PIVOT_ERR_INVALID_ARG, "null pointer");
  const int64_t n_max = n0 + (int64_t)(n_rows - 1) * n_step;
  if (n_max > ld) return fail(PIVOT_ERR_INVALID_ARG, "row length %lld exceeds ld", (long long)n_max);
  if (n_max > 0x7FFFFFFE) return fail(PIVOT_ERR_INVALID_ARG, "rows exceed int32 positions");
  SeqTable st;
  memset(&st, 0, sizeof st);
  st.n = 1;
  st.q_pos0[0] = (int32_t)(n0 - 1);
  st.n_rows[0] = n_rows;
  RowSpace rs{0, n_rows, n_step, kAll};
  OutDesc od{out, m, 0, 0, m};
  return hip_check(launch_topk(scores, true, ld, st, rs, od, n_max - 1, nullptr, 0, (hipStream_t)stream),
                   "top-k kernel");
}

pivot_status pivot_topk_rows_ws(int32_t n_rows, const float* scores, int64_t ld, int64_t n0, int32_t n_step,
                                int32_t m, int32_t* out, void* workspace, size_t workspace_bytes, void* stream) {
  if (workspace && reinterpret_cast<uintptr_t>(workspace) % kAlign)
    return fail(PIVOT_ERR_INVALID_ARG, "workspace must be %zu-byte aligned", kAlign);
  if (n_rows < 0 || n0 < 0 || n_step < 0 || m < 1) return fail(PIVOT_ERR_INVALID_ARG, "bad size");
  if (n_rows == 0) return PIVOT_OK;
  if (!scores || !out) return fail(PIVOT_ERR_INVALID_ARG, "null pointer");
  const int64_t n_max = n0 + (int64_t)(n_rows - 1) * n_step;
  if (n_max > ld) return fail(PIVOT_ERR_INVALID_ARG, "row length %lld exceeds ld", (long long)n_max);
  if (n_max > 0x7FFFFFFE) return fail(PIVOT_ERR_INVALID_ARG, "rows exceed int32 positions");
  SeqTable st;
  memset(&st, 0, sizeof st);
  st.n = 1;
  st.q_pos0[0] = (int32_t)(n0 - 1);
  st.n_rows[0] = n_rows;
  RowSpace rs{0, n_rows, n_step, kAll};
  OutDesc od{out, m, 0, 0, m};
  return hip_check(launch_topk(scores, false, ld, st, rs, od, n_max - 1, workspace, workspace ? workspace_bytes : 0,
                               (hipStream_t)stream),
                   "top-k kernel");
}

pivot_status pivot_encode_e4m3(const float* x, uint8_t* out, int64_t n, void* stream) {
  if (n < 0) return fail(PIVOT_ERR_INVALID_ARG, "n < 0");
  if (n == 0) return PIVOT_OK;
  if (!x || !out) return fail(PIVOT_ERR_INVALID_ARG, "null pointer");
  return hip_check(launch_encode_e4m3(x, out, n, (hipStream_t)stream), "encode kernel");
}

pivot_status pivot_profile_begin_kinds(uint32_t kinds) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (g_prof_on) return fail(PIVOT_ERR_INVALID_ARG, "a profile is already running");
  if (kinds == 0 || (kinds >> PIVOT_KERNEL_KINDS) != 0)
    return fail(PIVOT_ERR_INVALID_ARG, "kernel kind mask 0x%x outside 1 .. 0x%x", kinds,
                (1u << PIVOT_KERNEL_KINDS) - 1);
  g_prof_recs.clear();
  g_prof_mask = kinds;
  g_prof_on = true;
  return PIVOT_OK;
}

pivot_status pivot_profile_begin(void) { return pivot_profile_begin_kinds((1u << PIVOT_KERNEL_KINDS) - 1); }

pivot_status pivot_profile_end(pivot_profile* out) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof_on) return fail(PIVOT_ERR_INVALID_ARG, "no profile is running");
  g_prof_on = false;
  pivot_profile acc;
  memset(&acc, 0, sizeof acc);
  pivot_status st = PIVOT_OK;
  for (ProfRecord& r : g_prof_recs) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.stop);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess && st == PIVOT_OK) st = hip_check(e, "profile events");
    acc.launches[r.kind] += 1;
    acc.total_ms[r.kind] += ms;
    g_prof_pool.push_back(r.start);
    g_prof_pool.push_back(r.stop);
  }
  g_prof_recs.clear();
  if (out) *out = acc;
  return st;
}

const char* pivot_status_string(int32_t status) {
  switch (status) {
    case PIVOT_OK: return "ok";
    case PIVOT_ERR_INVALID_ARG: return "invalid argument";
    case PIVOT_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case PIVOT_ERR_WORKSPACE: return "workspace too small";
    case PIVOT_ERR_HIP: return "HIP launch failure";
    default: return "unknown status";
  }
}

const char* pivot_last_error(void) { return g_err; }

const char* pivot_version(void) { return "pivot-gfx950 0.1"; }

}  // extern "C"
