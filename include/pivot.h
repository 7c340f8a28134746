/*
 * pivot.h - C ABI of the MI355X (gfx950) PIVOT indexer library (libpivot.so).
 *
 * The library computes the DeepSeek-Sparse-Attention lightning indexer and the
 * PIVOT grouped replacement for it (PIVOT: Efficient Query-Group Indexing for
 * Token-Level Sparse Attention):
 *
 *   score   I[t,s] = sum_j w[t,j] * ReLU(q[t,j] . k[s])          Sec. 3.1 Eq. (1)
 *           fp8 form: kscale[s] * sum_j (w[t,j] * qscale[t])
 *                              * ReLU(q8[t,j] . k8[s])             App. A
 *   dense   T_t = TopK({I[t,s] : s <= t}, k)                      Sec. 3.1
 *   PIVOT   Algorithm 1 (App. E): groups of g queries (Eqs. 2-3), a proxy per
 *           group (per-head mean, Eq. 4), one proxy scan over s <= t0 (Eq. 5),
 *           then Reuse (proxy top-k shared, Eq. 6) or Refine (proxy top-c
 *           candidates, Eq. 7, re-scored per member, Eqs. 8-9); groups whose
 *           first position t0 is below the guardrail threshold are indexed
 *           densely.
 *
 * Conventions for every entry point:
 *   - positions are 0-based; a query at position t may select any s <= t;
 *   - an index set is k int32 positions in unspecified order; when fewer than
 *     k positions are valid, all of them are returned followed by -1;
 *   - TopK ranks by score, then by lower position among equal scores; with
 *     fp8 inputs the full-prefix scans (dense, and the proxy scan of Reuse /
 *     Refine) and Refine's member re-scores keep their scores in bf16 (round
 *     to nearest even, relative error at most 2^-9, far inside what fp8
 *     inputs resolve) and rank those; bf16 inputs keep fp32 scores;
 *   - "dev" pointers are device memory on the current HIP device, "host"
 *     pointers are host memory read during the call;
 *   - the caller owns every buffer; the library never allocates device memory
 *     and never synchronises the stream; work is enqueued on `stream`
 *     (a hipStream_t, NULL for the null stream);
 *   - every argument is validated before the first launch; a failed call
 *     returns a status and launches nothing; no call aborts or throws;
 *   - v1 supports H = 64 indexer heads of dimension d = 128 (UNSUPPORTED
 *     otherwise); fp8 means OCP E4M3FN (largest finite 448) with fp32
 *     per-token scales; gates w are fp32.
 */
#ifndef PIVOT_H
#define PIVOT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PIVOT_OK = 0,
  PIVOT_ERR_INVALID_ARG = 1,  /* null pointer, inconsistent size or parameter */
  PIVOT_ERR_UNSUPPORTED = 2,  /* shape or dtype this library does not specialise */
  PIVOT_ERR_WORKSPACE = 3,    /* workspace_bytes below pivot_workspace_size() */
  PIVOT_ERR_HIP = 4           /* a HIP launch failed; see pivot_last_error() */
} pivot_status;

typedef enum { PIVOT_DT_BF16 = 0, PIVOT_DT_FP8_E4M3 = 1 } pivot_dtype;

typedef enum { PIVOT_REUSE = 0, PIVOT_REFINE = 1 } pivot_mode;

/* Passed as `mode` to pivot_workspace_size() for a dense call. */
#define PIVOT_DENSE (-1)
/* Keys per sequence (and score row length) this library handles: 2^27.  The
 * scoring kernel addresses four score rows through one 32-bit range. */
#define PIVOT_MAX_KEYS (1 << 27)

/*
 * One indexer call over B sequences.
 *
 * Layouts (row-major, contiguous):
 *   q        dev  [B, n_q, H, d]  bf16 bits or E4M3FN codes
 *   q_scale  dev  [B, n_q]        fp32, fp8 only (NULL for bf16)
 *   w        dev  [B, n_q, H]     fp32 gates
 *   k        dev  [B, k_seq_stride, d]  keys of each sequence, position-major
 *   k_scale  dev  [B, k_seq_stride]     fp32, fp8 only (NULL for bf16)
 *   out_idx  dev  [B, n_q, topk]  int32 result
 *
 * Sequence b holds n_q queries at positions q_pos0[b] .. q_pos0[b]+n_q-1 and
 * keys at positions 0 .. n_k[b]-1, with q_pos0[b] + n_q <= n_k[b] <=
 * k_seq_stride and n_k[b] <= PIVOT_MAX_KEYS (else PIVOT_ERR_UNSUPPORTED).
 * Prefill passes B = 1, q_pos0 = the chunk start and
 * n_k = q_pos0 + n_q; chunks whose start is a multiple of g give groups aligned
 * to absolute positions.  Decode passes n_q = g (the current query and its MTP
 * drafts, Eq. 3) and q_pos0[b] = n_k[b] - g.
 */
typedef struct {
  int32_t dtype;            /* pivot_dtype */
  int32_t heads;            /* H, must be 64 */
  int32_t dim;              /* d, must be 128 */
  int32_t batch;            /* B >= 1 */
  int32_t n_q;              /* queries per sequence in this call, >= 0 */
  const int32_t* q_pos0;    /* host [B] */
  const int32_t* n_k;       /* host [B] */
  const void* q;
  const float* q_scale;
  const float* w;
  const void* k;
  const float* k_scale;
  int64_t k_seq_stride;     /* key rows between consecutive sequences */
  int32_t topk;             /* k >= 1 */
  int32_t* out_idx;
  void* workspace;          /* dev scratch, >= pivot_workspace_size() bytes, 256-B aligned */
  size_t workspace_bytes;
  void* stream;             /* hipStream_t */
} pivot_args;

/*
 * Workspace bytes needed by pivot_dense_index (mode = PIVOT_DENSE) or by
 * pivot_group_index (mode = PIVOT_REUSE / PIVOT_REFINE with g, c and the
 * guardrail at c) for the shapes in `a`; only the host arrays q_pos0 / n_k are
 * read.  Returns 0 if the shapes are invalid.  The score rows (bf16 for fp8
 * inputs, fp32 for bf16 inputs) are tiled so that this size stays near 1 GiB
 * for long prefixes.  Any workspace of at
 * least this size works; smaller ones down to one score tile also work (more
 * tiles), and below that the entry points return PIVOT_ERR_WORKSPACE.
 */
size_t pivot_workspace_size(const pivot_args* a, int32_t mode, int32_t g, int32_t c);

/*
 * Dense lightning indexer (Sec. 3.1 Eq. 1 with the fp8 form of App. A):
 * out_idx[b, i, :] = TopK over s in [0, q_pos0[b] + i] of the score of query
 * (b, i) against key s, k = a->topk.
 */
pivot_status pivot_dense_index(const pivot_args* a);

/*
 * PIVOT (Algorithm 1, App. E).  Groups are runs of g consecutive queries from
 * each sequence's first query in the call (Eq. 2; a decode call with n_q = g is
 * one MTP group, Eq. 3); the last run may be shorter.  For a group with first
 * position t0:
 *   - t0 < dense_below: each member gets its dense index set (the guardrail of
 *     Algorithm 1; pass dense_below = c to follow Algorithm 1, 0 to disable,
 *     a negative value means c);
 *   - otherwise the proxy is the per-head mean of the members' dequantised
 *     queries and of their gates (Eq. 4), stored as a query row (fp8: scale
 *     amax/448 and round-to-nearest-even codes; bf16: round-to-nearest-even);
 *     a group of one is its own proxy.  The proxy scores positions [0, t0]
 *     (Eq. 5).  PIVOT_REUSE gives every member the proxy top-k (Eq. 6);
 *     PIVOT_REFINE keeps the proxy top-c set C (Eq. 7) and gives each member
 *     the top-k of its own scores over C (Eqs. 8-9).
 * Requirements: g >= 1; Refine needs topk <= c <= 8192.
 * out_cand (optional, Refine only): dev int32 [B, ceil(n_q/g), c] receives each
 * group's candidate set (unordered, -1 padded; all -1 for guardrail groups).
 */
pivot_status pivot_group_index(const pivot_args* a, int32_t mode, int32_t g, int32_t c,
                               int32_t dense_below, int32_t* out_cand);

/* App. B's local window: how the window is added to the candidate set. */
typedef enum {
  PIVOT_WINDOW_SHARED = 0,    /* prefill: one set per group holds the window union */
  PIVOT_WINDOW_PER_QUERY = 1  /* decode: each query adds its own window to the pool */
} pivot_window_kind;

/* How a group is collapsed into its proxy query. */
typedef enum {
  PIVOT_AGG_MEAN = 0,   /* the per-head mean of Eq. 4 */
  PIVOT_AGG_FIRST = 1,  /* the group's first member, unchanged */
  PIVOT_AGG_LAST = 2    /* the group's last member, unchanged */
} pivot_aggregate;

/* How Refine runs Eqs. 8-9; every path gives the same top-k sets.
 *   PIVOT_REFINE_SPLIT: re-score every member into the workspace, then one
 *     select launch over the member rows.
 *   PIVOT_REFINE_FUSED: one launch; each group's member scores stay on chip
 *     and its members select there.  Applies to fp8 inputs with g <= 4, no
 *     window and pivot_cand_width() <= 4096; other calls take the split path.
 *   PIVOT_REFINE_AUTO: the faster path for the shapes at hand; currently
 *     always the split one (the fused launch runs two workgroups per CU,
 *     too few to hide its selects' latency). */
typedef enum {
  PIVOT_REFINE_AUTO = 0,
  PIVOT_REFINE_FUSED = 1,
  PIVOT_REFINE_SPLIT = 2
} pivot_refine_path;

typedef struct {
  int32_t mode;         /* PIVOT_REUSE or PIVOT_REFINE */
  int32_t g, c;         /* group size, candidate budget (as pivot_group_index) */
  int32_t dense_below;  /* guardrail threshold (as pivot_group_index) */
  int32_t window;       /* W >= 0, Refine only; 0 = no window */
  int32_t window_kind;  /* pivot_window_kind */
  int32_t aggregate;    /* pivot_aggregate */
  int32_t* out_cand;    /* optional dev int32 [B, ceil(n_q/g), pivot_cand_width()] */
  int32_t refine_path;  /* pivot_refine_path (0 = PIVOT_REFINE_AUTO) */
} pivot_group_opts;

/*
 * PIVOT with the options of App. B and of the aggregation ablation (Sec. 5.4);
 * opts {mode, g, c, dense_below, 0, 0, PIVOT_AGG_MEAN, out_cand,
 * PIVOT_REFINE_AUTO} is exactly pivot_group_index; refine_path picks how
 * Refine runs (pivot_refine_path; any other value is PIVOT_ERR_INVALID_ARG).  With window W > 0 (Refine only), for a group with first
 * position t0 and gs members:
 *   - PIVOT_WINDOW_SHARED (prefill): the union of the members' windows,
 *     positions t0-W+1 .. t0+g-1, takes w = W+g-1 of the c candidate slots
 *     (slots for positions below 0 or past the last member hold -1); the
 *     proxy fills the other c - w slots with its top over [0, t0-W].  Needs
 *     c >= W + g - 1.
 *   - PIVOT_WINDOW_PER_QUERY (decode): the proxy's top-c over [0, t0] is the
 *     pool; the union follows it in W+g-1 more slots, with positions already
 *     in the pool replaced by -1.  Needs W >= g.
 *   Member t re-scores the candidates at positions <= t (and, for a union
 *   slot of the per-query kind, >= t-W+1) and keeps its top-k; fewer valid
 *   candidates than k are padded with -1.
 * Requirements as pivot_group_index, with topk <= pivot_cand_width() <= 8192;
 * other values return PIVOT_ERR_INVALID_ARG (PIVOT_ERR_UNSUPPORTED past 8192).
 * The candidate slots of a group are c + W + g - 1 for PIVOT_WINDOW_PER_QUERY
 * with W > 0, else c (pivot_cand_width(); 0 for a NULL opts).
 * pivot_group_workspace_size: workspace bytes for pivot_group_index_opts with
 * these opts and shapes (dense_below as given), 0 if they are invalid; the
 * rules of pivot_workspace_size apply.  opts is read, never kept.
 */
int32_t pivot_cand_width(const pivot_group_opts* o);
size_t pivot_group_workspace_size(const pivot_args* a, const pivot_group_opts* o);
pivot_status pivot_group_index_opts(const pivot_args* a, const pivot_group_opts* o);

/*
 * Batch layouts beyond the padded, contiguous one of pivot_args: packed
 * variable-length query runs (one per request of a batch) and a paged key
 * cache.  A NULL layout, or one whose two pointers are NULL, is pivot_args'
 * own layout.
 *   cu_q (host [B+1], or NULL): sequence b owns query rows cu_q[b] ..
 *     cu_q[b+1]-1 of the packed q / q_scale / w / out_idx (cu_q[0] = 0,
 *     nondecreasing); a->n_q is ignored.  Groups restart at every sequence's
 *     first query, so no group spans two requests (Sec. 4.1); candidate rows
 *     (out_cand) are packed the same way, sum over b of ceil(n_b / g) rows.
 *   block_table (dev int32 [B, max_pages], or NULL): key s < n_k[b] of
 *     sequence b is row block_table[b * max_pages + s / page_size] *
 *     page_size + s % page_size of k / k_scale, a pool of pool_keys rows;
 *     a->k_seq_stride is ignored.  Entries outside [0, pool_keys / page_size)
 *     are clamped into it (the result is then meaningless, but no access
 *     leaves the pool).  page_size is a power of two in [16, 65536];
 *     pool_keys is a multiple of page_size with pool_keys * bytes-per-key
 *     at most 2^31 (128 B per fp8 key, 256 B per bf16 key); n_k[b] <=
 *     max_pages * page_size.
 * Invalid layouts return PIVOT_ERR_INVALID_ARG (PIVOT_ERR_UNSUPPORTED for a
 * pool past the 2^31-byte limit).  The layout is read, never kept.
 */
typedef struct {
  const int32_t* cu_q;
  const int32_t* block_table;
  int32_t max_pages;
  int32_t page_size;
  int64_t pool_keys;
} pivot_layout;

/*
 * pivot_dense_index and pivot_group_index_opts with a layout.  The workspace
 * size for such a call is pivot_workspace_size_layout(a, l, o) with o the
 * options, or NULL for the dense index.
 */
pivot_status pivot_dense_index_layout(const pivot_args* a, const pivot_layout* l);
pivot_status pivot_group_index_layout(const pivot_args* a, const pivot_layout* l, const pivot_group_opts* o);
size_t pivot_workspace_size_layout(const pivot_args* a, const pivot_layout* l, const pivot_group_opts* o);

/*
 * PIVOT composed with IndexCache (Sec. 5.1 "Baselines"; the +IC rows of
 * Table 1).  IndexCache works on the layer axis (Sec. 2): one layer's index
 * sets T_t serve the layers after it; composed with PIVOT, the layers that do
 * index run PIVOT.
 *   layers[0 .. n_layers-1]: consecutive indexer layers over the same query
 *     and key positions.  Each has its own q, q_scale, w, k, k_scale and
 *     out_idx (layouts as in pivot_args); every other field must equal
 *     layers[0]'s: dtype, heads, dim, batch, n_q, topk, k_seq_stride, and the
 *     contents of q_pos0 and n_k.
 *   Layer l is an anchor when anchors[l] != 0 (anchors: host [n_layers]) or,
 *     with anchors NULL, when l % stride == 0 (stride >= 1).  Layer 0 must be
 *     an anchor.
 *   An anchor layer is indexed as pivot_group_index_opts(&layers[l], o) would
 *     index it (o NULL: as pivot_dense_index, i.e. IndexCache alone).  Every
 *     other layer receives in its out_idx the sets of the nearest anchor
 *     before it; its q, q_scale, w, k and k_scale are not read (they may be
 *     NULL).
 *   All work is enqueued on layers[0].stream in layer order and uses
 *     layers[0].workspace, which needs the bytes of one anchor call,
 *     pivot_workspace_size_layout(&layers[0], NULL, o); the other layers'
 *     workspace and stream fields are ignored.  o->out_cand must be NULL.
 * Every layer is validated before the first launch: a layer that differs from
 * layer 0, a missing pointer, stride < 1 without anchors, n_layers < 1 or an
 * unset anchor 0 return PIVOT_ERR_INVALID_ARG; an anchor's own checks return
 * what its single-layer call would.  A follower costs one copy of the index
 * sets; a run of followers reads the anchor's sets once.
 */
pivot_status pivot_index_layers(const pivot_args* layers, int32_t n_layers, int32_t stride,
                                const uint8_t* anchors, const pivot_group_opts* o);

/*
 * pivot_group_index_opts that allocates nothing, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  a->workspace and a->workspace_bytes are
 * ignored: the call uses a scratch array of PIVOT_NOALLOC_SCRATCH_BYTES that
 * the library holds on each device it runs on (in its code object, until the
 * process ends).  Its address on the current device is looked up on the first
 * call there.  The call itself makes no allocation, frees nothing and
 * synchronises nothing; results are those of pivot_group_index_opts.
 *   - A call whose workspace minimum (fixed regions plus one score tile, see
 *     pivot_group_workspace_size) exceeds the scratch returns
 *     PIVOT_ERR_WORKSPACE before touching the device (e.g. 32 decode
 *     sequences of 131072 keys need ~18 MB; a 2048-query prefill chunk with
 *     g = 4, c = 4096 ~35 MB; an 8192-query chunk does not fit).
 *   - Calls share the device's scratch and each leaves its contents behind;
 *     no region needs to start at zero.  Calls that overlap on one device
 *     (two streams, two threads) race on it: order them on one stream.
 */
#define PIVOT_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
pivot_status pivot_group_index_noalloc(const pivot_args* a, const pivot_group_opts* o);

/*
 * Stage: proxy rows of Eq. 4 for one sequence's queries q [n_q, H, d] /
 * q_scale [n_q] / w [n_q, H] split into runs of g (last may be shorter).
 * Writes out_q [ceil(n_q/g), H, d] (same format as q), out_scale
 * [ceil(n_q/g)] (1.0 for bf16) and out_w [ceil(n_q/g), H].  Dev pointers.
 */
pivot_status pivot_proxy_rows(int32_t dtype, int32_t heads, int32_t dim, int32_t n_q, int32_t g,
                              const void* q, const float* q_scale, const float* w,
                              void* out_q, float* out_scale, float* out_w, void* stream);

/*
 * Stage: score rows (Eq. 1 / App. A).  Row r (r < n_rows) of q [n_rows, H, d],
 * q_scale [n_rows] (fp8) and w [n_rows, H] is scored against keys
 * s = 0 .. lim0 + r * lim_step of k / k_scale (which must hold at least that
 * many keys); out[r * ld + s] receives the fp32 score.  Entries past a row's
 * limit are not written.  Requires ld >= lim0 + (n_rows-1)*lim_step + 1 and
 * ld <= PIVOT_MAX_KEYS (else PIVOT_ERR_UNSUPPORTED).
 * fp8 rows need a workspace of PIVOT_SCORE_ROWS_WORKSPACE(n_rows) bytes
 * (256-B aligned) for the per-row linear term of the epilogue; bf16 needs none.
 */
#define PIVOT_SCORE_ROWS_WORKSPACE(n_rows) \
  ((((size_t)(n_rows) * 512 + 255) / 256) * 256 + (size_t)(n_rows) * 16)
pivot_status pivot_score_rows(int32_t dtype, int32_t heads, int32_t dim, int32_t n_rows,
                              const void* q, const float* q_scale, const float* w,
                              const void* k, const float* k_scale, int64_t lim0, int32_t lim_step,
                              float* out, int64_t ld, void* workspace, size_t workspace_bytes,
                              void* stream);

/*
 * Stage: TopK of fp32 rows.  Row r of scores [n_rows, ld] has its first
 * n0 + r * n_step entries valid; out [n_rows, m] receives their top-m
 * positions (score descending, then position ascending; -0 == +0; -1 padded).
 */
pivot_status pivot_topk_rows(int32_t n_rows, const float* scores, int64_t ld, int64_t n0,
                             int32_t n_step, int32_t m, int32_t* out, void* stream);

/*
 * Stage: pivot_topk_rows over rows of bf16 scores (uint16 bits), the score
 * rows the fp8 index paths rank; ties and padding as pivot_topk_rows.
 */
pivot_status pivot_topk_rows_bf16(int32_t n_rows, const uint16_t* scores, int64_t ld, int64_t n0, int32_t n_step,
                                  int32_t m, int32_t* out, void* stream);

/*
 * Stage: pivot_topk_rows with a device workspace (256-B aligned, or NULL).
 * With at least pivot_topk_rows_workspace_size(n_rows) bytes, a call of at
 * most 256 rows whose longest row has >= 16384 entries splits every row over
 * several workgroups (the decode shape of the index paths); otherwise it
 * runs as pivot_topk_rows.  The result is the same either way.
 * pivot_topk_rows_workspace_size returns 0 for n_rows outside [1, 256].
 */
size_t pivot_topk_rows_workspace_size(int32_t n_rows);
pivot_status pivot_topk_rows_ws(int32_t n_rows, const float* scores, int64_t ld, int64_t n0,
                                int32_t n_step, int32_t m, int32_t* out, void* workspace,
                                size_t workspace_bytes, void* stream);

/*
 * Utility: x [n] fp32 -> E4M3FN codes out [n] with the same conversion the
 * proxy kernel uses (round to nearest even).  Dev pointers.
 */
pivot_status pivot_encode_e4m3(const float* x, uint8_t* out, int64_t n, void* stream);

/*
 * Kernel timing.  Between pivot_profile_begin() and pivot_profile_end() every
 * kernel the library launches is bracketed by two HIP events recorded on the
 * launch's stream.  pivot_profile_end() waits for those events and returns,
 * per kernel kind, the number of launches and the summed event-to-event time;
 * it then stops recording.  Event objects are host-side resources created on
 * first use; no device memory is allocated.  One profile at a time per process.
 * pivot_profile_begin_kinds(mask) brackets only the kinds whose bit
 * (1 << PIVOT_KERNEL_*) is set, so that the events of other kernels add no
 * gaps to a timed run; a mask of 0 or with bits past PIVOT_KERNEL_KINDS is
 * INVALID_ARG.
 */
enum {
  PIVOT_KERNEL_PROXY = 0,   /* proxy aggregation, Eq. 4 */
  PIVOT_KERNEL_SCORE = 1,   /* MFMA scoring, Eq. 1 / Eq. 5 */
  PIVOT_KERNEL_SELECT = 2,  /* row top-k / top-c selection */
  PIVOT_KERNEL_REFINE = 3,  /* Refine gather, re-score and select, Eqs. 8-9 */
  PIVOT_KERNEL_FILL = 4,    /* -1 fill of guardrail candidate rows */
  PIVOT_KERNEL_LIN = 5,     /* per-row linear term of the fp8 score epilogue */
  PIVOT_KERNEL_COPY = 6,    /* index sets copied to IndexCache follower layers */
  PIVOT_KERNEL_KINDS = 7
};

typedef struct {
  int64_t launches[PIVOT_KERNEL_KINDS];
  double total_ms[PIVOT_KERNEL_KINDS];
} pivot_profile;

pivot_status pivot_profile_begin(void);
pivot_status pivot_profile_begin_kinds(uint32_t kinds);
pivot_status pivot_profile_end(pivot_profile* out);

/* Static description of a status code. */
const char* pivot_status_string(int32_t status);

/* Detail of the last failure on the calling thread (empty if none). */
const char* pivot_last_error(void);

/* Library version string. */
const char* pivot_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PIVOT_H */
