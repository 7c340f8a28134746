/*
 * CPU oracle for the PIVOT indexer path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
 * the benchmark's CPU-baseline leg may load this library.  It is a plain, slow
 * restatement of what the method computes, written for a reader to check
 * against the paper by eye; it shares no code with the GPU path.
 *
 * Sources in the paper (PIVOT: Efficient Query-Group Indexing for Token-Level
 * Sparse Attention):
 *   - lightning-indexer score:            Sec. 3.1 Eq. (1); App. A (FP8 form)
 *   - TopK and the index set T_t:         Sec. 3.1; App. A
 *   - prefill / decode grouping:          Sec. 4.1 Eqs. (2), (3)
 *   - proxy query (per-head mean):        Sec. 4.2 Eq. (4)
 *   - proxy scan with cutoff at t0:       Sec. 4.2 Eq. (5)
 *   - Reuse:                              Sec. 4.3 Eq. (6)
 *   - Refine candidate set / re-score /
 *     per-query selection:                Sec. 4.4 Eqs. (7), (8), (9)
 *   - short-group guardrail and the
 *     overall order of the steps:         App. E, Algorithm 1
 *   - local window W (prefill / decode):  App. B
 *   - first / last member as the proxy:   Sec. 5.4 (query aggregation ablation)
 *   - PIVOT composed with IndexCache
 *     (index sets shared across layers):  Sec. 5.1 "Baselines", the +IC rows
 *                                         of Table 1; Sec. 2 (layer axis)
 *
 * Readings where the paper is silent (the same list is kept with the design
 * notes of the repository):
 *   - positions are 0-based and a query at position t may select s <= t;
 *   - TopK orders by (score descending, position ascending); -0 == +0;
 *     fewer than m valid positions -> all of them, padded with -1;
 *   - the proxy of a group covers positions [0, t0], t0 = first member;
 *   - a group of one is its own proxy (the identity stated in App. A);
 *   - the proxy is formed in fp32 from the dequantised members (ascending
 *     member order, correctly rounded divide by |G|) and stored in the query
 *     format: bf16 by RNE, or fp8 E4M3FN with scale amax/448 and RNE codes
 *     saturated to +-448;
 *   - the guardrail of Algorithm 1 (t0 < c -> dense) applies to both variants;
 *     `dense_below` carries its threshold (callers pass c, or 0 to disable);
 *   - local window (Refine only; W = 0 is the plain candidate set):
 *       prefill ("shared"): the union of the members' windows is the w_g =
 *         W + g - 1 positions t0-W+1 .. t0+g-1; the proxy fills the other
 *         c - w_g slots with its top over [0, t0-W] (the positions before the
 *         union); union positions below 0 or past the group's last member are
 *         empty (-1);
 *       decode ("per query"): the pool is the proxy's top-c over [0, t0]; the
 *         union t0-W+1 .. t0+g-1 follows it (c + W + g - 1 slots), with
 *         positions already in the pool emptied; W >= g;
 *       member t re-scores the slots it may use: position <= t, and, for a
 *         union slot of the per-query kind, position >= t - W + 1;
 *   - first / last aggregation: the proxy is that member's row, unchanged;
 *   - IndexCache composition (the paper gives no layer pattern): layers are
 *     taken in order; an anchor layer runs the indexer on its own inputs, and
 *     every other layer takes the index sets of the nearest anchor before it,
 *     unchanged; the first layer is an anchor.
 *
 * Floating point: every score is accumulated in double.  For fp8 inputs the
 * inner products are exact in double (codes are multiples of 2^-9 with
 * magnitude <= 448, so 128-term sums need < 44 significant bits).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { OR_BF16 = 0, OR_FP8 = 1 };
enum { OR_DENSE = 0, OR_REUSE = 1, OR_REFINE = 2 };

/* ------------------------------------------------------------------ codecs */

/* OCP 8-bit floating point, E4M3 "FN" variant: 1 sign, 4 exponent (bias 7),
 * 3 mantissa bits; no infinities; S.1111.111 is NaN; largest finite 448. */
static double e4m3_value[256];
static int codec_ready = 0;

static void build_codecs(void) {
    if (codec_ready) return;
    for (int code = 0; code < 256; ++code) {
        int s = code >> 7, e = (code >> 3) & 15, m = code & 7;
        double v;
        if (e == 15 && m == 7) v = NAN;
        else if (e == 0) v = ldexp((double)m / 8.0, -6);        /* subnormal */
        else v = ldexp(1.0 + (double)m / 8.0, e - 7);           /* normal */
        e4m3_value[code] = s ? -v : v;
    }
    codec_ready = 1;
}

double oracle_e4m3_decode(uint8_t code) { build_codecs(); return e4m3_value[code]; }

/* Round x to the nearest E4M3FN value, ties to the code with even mantissa,
 * saturating magnitudes beyond 448 to 448.  Searches the 127 finite
 * non-negative codes, which are increasing in value. */
uint8_t oracle_e4m3_encode(float x) {
    build_codecs();
    if (isnan(x)) return 0x7F;
    uint8_t sign = signbit(x) ? 0x80 : 0x00;
    double a = fabs((double)x);
    if (a >= 448.0) return sign | 0x7E;
    int lo = 0;                                   /* largest code with value <= a */
    for (int c = 0; c <= 0x7E; ++c) if (e4m3_value[c] <= a) lo = c;
    if (e4m3_value[lo] == a || lo == 0x7E) return sign | (uint8_t)lo;
    int hi = lo + 1;
    double dlo = a - e4m3_value[lo], dhi = e4m3_value[hi] - a;
    int pick = (dlo < dhi) ? lo : (dhi < dlo) ? hi : ((lo & 1) ? hi : lo);
    return sign | (uint8_t)pick;
}

/* bfloat16: the upper 16 bits of an IEEE binary32. */
double oracle_bf16_decode(uint16_t bits) {
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* binary32 -> bfloat16, round to nearest, ties to even. */
uint16_t oracle_bf16_encode(float x) {
    uint32_t u;
    memcpy(&u, &x, 4);
    if (isnan(x)) return (uint16_t)((u >> 16) | 0x40);
    uint32_t keep = u >> 16, rest = u & 0xFFFFu;
    if (rest > 0x8000u || (rest == 0x8000u && (keep & 1u))) keep += 1;
    return (uint16_t)keep;
}

static inline double elem(int fmt, const void* base, int64_t i) {
    return fmt == OR_FP8 ? e4m3_value[((const uint8_t*)base)[i]]
                         : oracle_bf16_decode(((const uint16_t*)base)[i]);
}

/* ------------------------------------------------------------------ score */

/* Eq. (1) in the scaled form of App. A for one (row, key) pair:
 *   S = ks * sum_j (w_j * sq) * ReLU( sum_i q_{j,i} * k_i )
 * q_row: H*d codes of one query (or proxy) row; w_row: H gates; sq, ks: the
 * per-token scales (1 for bf16). */
static double score_pair(int fmt, int H, int d, const void* q_row, double sq,
                         const float* w_row, const void* k_row, double ks) {
    double total = 0.0;
    for (int j = 0; j < H; ++j) {
        double dot = 0.0;
        for (int i = 0; i < d; ++i)
            dot += elem(fmt, q_row, (int64_t)j * d + i) * elem(fmt, k_row, i);
        double relu = dot > 0.0 ? dot : 0.0;
        total += ((double)w_row[j] * sq) * relu;
    }
    return ks * total;
}

typedef struct {
    int fmt, H, d;
    const void* k;          /* key codes of one sequence [n_keys, d] */
    const float* k_scale;   /* [n_keys] or NULL */
} keyset;

static const void* key_row(const keyset* K, int64_t s) {
    size_t b = K->fmt == OR_FP8 ? 1 : 2;
    return (const char*)K->k + (size_t)s * K->d * b;
}

/* Scores of one row against the listed key positions. */
static void score_positions(const keyset* K, const void* q_row, double sq, const float* w_row,
                            const int32_t* pos, int64_t n, double* out) {
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t i = 0; i < n; ++i) {
        int64_t s = pos[i];
        double ks = K->k_scale ? (double)K->k_scale[s] : 1.0;
        out[i] = score_pair(K->fmt, K->H, K->d, q_row, sq, w_row, key_row(K, s), ks);
    }
}

/* ------------------------------------------------------------------ TopK */

typedef struct { double f; int32_t s; } scored;

static int by_score_then_position(const void* pa, const void* pb) {
    const scored* a = (const scored*)pa;
    const scored* b = (const scored*)pb;
    if (a->f > b->f) return -1;       /* higher score first (-0 == +0 here) */
    if (a->f < b->f) return 1;
    return (a->s < b->s) ? -1 : (a->s > b->s) ? 1 : 0;   /* then lower position */
}

/* TopK over a domain: the first min(m, n) positions in (score desc, position
 * asc) order, then -1 up to m.  Returns the number of valid entries. */
static int topk(const double* f, const int32_t* pos, int64_t n, int m, int32_t* out) {
    scored* v = (scored*)malloc(sizeof(scored) * (size_t)(n > 0 ? n : 1));
    for (int64_t i = 0; i < n; ++i) { v[i].f = f[i]; v[i].s = pos[i]; }
    qsort(v, (size_t)n, sizeof(scored), by_score_then_position);
    int take = (int)(n < m ? n : m);
    for (int i = 0; i < take; ++i) out[i] = v[i].s;
    for (int i = take; i < m; ++i) out[i] = -1;
    free(v);
    return take;
}

int oracle_topk(const double* f, const int32_t* pos, int64_t n, int m, int32_t* out) {
    return topk(f, pos, n, m, out);
}

/* ------------------------------------------------------------------ steps */

/* Dense index set of one query at position t: TopK over [0, t]. */
static void dense_row(const keyset* K, const void* q_row, double sq, const float* w_row,
                      int64_t t, int m, int32_t* out) {
    int64_t n = t + 1;
    int32_t* pos = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
    double* f = (double*)malloc(sizeof(double) * (size_t)n);
    for (int64_t s = 0; s < n; ++s) pos[s] = (int32_t)s;
    score_positions(K, q_row, sq, w_row, pos, n, f);
    topk(f, pos, n, m, out);
    free(pos);
    free(f);
}

/* Eq. (4): the group's proxy query.  Members are rows [0, gs) of q / w /
 * q_scale.  Writes the proxy codes (H*d), its scale and its H gates. */
enum { OR_AGG_MEAN = 0, OR_AGG_FIRST = 1, OR_AGG_LAST = 2 };

static void proxy_of_agg(int fmt, int H, int d, const void* q, const float* q_scale,
                         const float* w, int gs, int agg, void* pq, float* psc, float* pw) {
    size_t n = (size_t)H * d, b = fmt == OR_FP8 ? 1 : 2;
    if (gs == 1 || agg != OR_AGG_MEAN) { /* a group of one is its own proxy; first / last member */
        int t = (agg == OR_AGG_LAST) ? gs - 1 : 0;
        memcpy(pq, (const char*)q + (size_t)t * n * b, n * b);
        *psc = (fmt == OR_FP8) ? q_scale[t] : 1.0f;
        memcpy(pw, w + (size_t)t * H, sizeof(float) * (size_t)H);
        return;
    }
    float* mean = (float*)malloc(sizeof(float) * n);
    const float count = (float)gs;
    for (size_t e = 0; e < n; ++e) {
        float sum = 0.0f;
        for (int t = 0; t < gs; ++t) {
            float sq = (fmt == OR_FP8) ? q_scale[t] : 1.0f;
            float x = (float)elem(fmt, q, (int64_t)t * (int64_t)n + (int64_t)e);
            float deq = sq * x;           /* one fp32 rounding */
            sum = sum + deq;              /* fp32, ascending member order */
        }
        mean[e] = sum / count;            /* correctly rounded fp32 divide */
    }
    for (int j = 0; j < H; ++j) {
        float sum = 0.0f;
        for (int t = 0; t < gs; ++t) sum = sum + w[(size_t)t * H + j];
        pw[j] = sum / count;
    }
    if (fmt == OR_BF16) {
        for (size_t e = 0; e < n; ++e) ((uint16_t*)pq)[e] = oracle_bf16_encode(mean[e]);
        *psc = 1.0f;
    } else {
        float amax = 0.0f;
        for (size_t e = 0; e < n; ++e) { float a = fabsf(mean[e]); if (a > amax) amax = a; }
        float sigma = (amax > 0.0f) ? amax / 448.0f : 1.0f;
        for (size_t e = 0; e < n; ++e) ((uint8_t*)pq)[e] = oracle_e4m3_encode(mean[e] / sigma);
        *psc = sigma;
    }
    free(mean);
}

static void proxy_of(int fmt, int H, int d, const void* q, const float* q_scale,
                     const float* w, int gs, void* pq, float* psc, float* pw) {
    proxy_of_agg(fmt, H, d, q, q_scale, w, gs, OR_AGG_MEAN, pq, psc, pw);
}

int oracle_proxy(int fmt, int H, int d, const void* q, const float* q_scale, const float* w,
                 int gs, void* pq, float* psc, float* pw) {
    build_codecs();
    if (gs < 1) return 1;
    proxy_of(fmt, H, d, q, q_scale, w, gs, pq, psc, pw);
    return 0;
}

/* Scores of one row (query or proxy) over positions [0, lim]. */
int oracle_scores(int fmt, int H, int d, const void* q_row, float sq, const float* w_row,
                  const void* k, const float* k_scale, int64_t lim, double* out) {
    build_codecs();
    keyset K = {fmt, H, d, k, fmt == OR_FP8 ? k_scale : NULL};
    int64_t n = lim + 1;
    int32_t* pos = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
    for (int64_t s = 0; s < n; ++s) pos[s] = (int32_t)s;
    score_positions(&K, q_row, fmt == OR_FP8 ? (double)sq : 1.0, w_row, pos, n, out);
    free(pos);
    return 0;
}

/* Scores of one row over an explicit list of positions. */
int oracle_scores_at(int fmt, int H, int d, const void* q_row, float sq, const float* w_row,
                     const void* k, const float* k_scale, const int32_t* pos, int64_t n,
                     double* out) {
    build_codecs();
    keyset K = {fmt, H, d, k, fmt == OR_FP8 ? k_scale : NULL};
    score_positions(&K, q_row, fmt == OR_FP8 ? (double)sq : 1.0, w_row, pos, n, out);
    return 0;
}

/* Eqs. (8)-(9) on a given candidate set: each of the gs member rows re-scores
 * the n_cand candidates and keeps its own top-m. */
int oracle_refine_on(int fmt, int H, int d, const void* q, const float* q_scale, const float* w,
                     int gs, const void* k, const float* k_scale, const int32_t* cand,
                     int64_t n_cand, int m, int32_t* out) {
    build_codecs();
    keyset K = {fmt, H, d, k, fmt == OR_FP8 ? k_scale : NULL};
    size_t rowb = (size_t)H * d * (fmt == OR_FP8 ? 1 : 2);
    double* f = (double*)malloc(sizeof(double) * (size_t)(n_cand > 0 ? n_cand : 1));
    for (int t = 0; t < gs; ++t) {
        const void* qr = (const char*)q + (size_t)t * rowb;
        double sq = fmt == OR_FP8 ? (double)q_scale[t] : 1.0;
        score_positions(&K, qr, sq, w + (size_t)t * H, cand, n_cand, f);
        topk(f, cand, n_cand, m, out + (size_t)t * m);
    }
    free(f);
    return 0;
}

/*
 * Algorithm 1 over the queries of one sequence.
 *
 * Queries are the n_q rows of q / q_scale / w, at positions p0 .. p0+n_q-1;
 * keys are positions 0 .. n_k-1.  Groups are runs of g rows starting at the
 * first row (Eq. (2)); a decode call passes its g MTP queries as one run
 * (Eq. (3)).  mode: 0 dense (every row: TopK over [0, t]), 1 Reuse, 2 Refine.
 * window / window_kind / agg: App. B's local window (0 = none; kind 0 the
 * prefill reading, 1 the decode reading) and the proxy aggregation (0 mean,
 * 1 first member, 2 last member), as read in the header.
 *
 * sel / n_sel: optional list of group indices to compute (others are left
 * untouched); NULL computes every group.  out_idx [n_q, topk]; out_cand
 * [n_groups, width] (Refine only, optional; -1 for guardrail groups), width =
 * c, or c + W + g - 1 for the decode window; out_pq / out_psc / out_pw:
 * optional proxies [n_groups, H*d] / [n_groups] / [n_groups, H] (left
 * untouched for guardrail groups).
 */
int oracle_index_ex(int fmt, int H, int d,
                    const void* q, const float* q_scale, const float* w, int n_q, int64_t p0,
                    const void* k, const float* k_scale, int64_t n_k,
                    int mode, int g, int c, int m, int dense_below,
                    int window, int window_kind, int agg,
                    const int32_t* sel, int n_sel,
                    int32_t* out_idx, int32_t* out_cand,
                    void* out_pq, float* out_psc, float* out_pw) {
    build_codecs();
    if (H < 1 || d < 1 || n_q < 0 || m < 1 || g < 1) return 1;
    if (p0 < 0 || p0 + n_q > n_k) return 1;
    if (fmt == OR_FP8 && (!q_scale || !k_scale)) return 1;
    if (window < 0 || (window > 0 && mode != OR_REFINE)) return 1;
    if (window_kind != 0 && window_kind != 1) return 1;
    if (agg < OR_AGG_MEAN || agg > OR_AGG_LAST) return 1;
    const int W = window;
    const int wg = W > 0 ? W + g - 1 : 0;                   /* the union's slots */
    if (W > 0 && window_kind == 0 && c < wg) return 1;
    if (W > 0 && window_kind == 1 && W < g) return 1;
    const int width = (W > 0 && window_kind == 1) ? c + wg : c;   /* candidate slots */
    if (mode == OR_REFINE && width < m) return 1;
    keyset K = {fmt, H, d, k, fmt == OR_FP8 ? k_scale : NULL};
    size_t b = fmt == OR_FP8 ? 1 : 2;
    size_t rowb = (size_t)H * d * b;
    int n_groups = (n_q + g - 1) / g;
    int count = sel ? n_sel : n_groups;

    void* pq = malloc(rowb);
    float* pw = (float*)malloc(sizeof(float) * (size_t)H);
    for (int gi = 0; gi < count; ++gi) {
        int grp = sel ? sel[gi] : gi;
        if (grp < 0 || grp >= n_groups) { free(pq); free(pw); return 1; }
        int r0 = grp * g;
        int gs = (n_q - r0 < g) ? (n_q - r0) : g;
        int64_t t0 = p0 + r0;
        const char* qg = (const char*)q + (size_t)r0 * rowb;
        const float* sg = fmt == OR_FP8 ? q_scale + r0 : NULL;
        const float* wg_ = w + (size_t)r0 * H;
        int32_t* og = out_idx + (size_t)r0 * m;

        if (mode == OR_DENSE || t0 < dense_below) {          /* dense, or guardrail */
            for (int t = 0; t < gs; ++t)
                dense_row(&K, qg + (size_t)t * rowb, sg ? (double)sg[t] : 1.0, wg_ + (size_t)t * H,
                          t0 + t, m, og + (size_t)t * m);
            if (mode == OR_REFINE && out_cand)
                for (int i = 0; i < width; ++i) out_cand[(size_t)grp * width + i] = -1;
            continue;
        }

        float psc;                                                   /* Eq. (4) */
        proxy_of_agg(fmt, H, d, qg, sg, wg_, gs, agg, pq, &psc, pw);
        if (out_pq) memcpy((char*)out_pq + (size_t)grp * rowb, pq, rowb);
        if (out_psc) out_psc[grp] = psc;
        if (out_pw) memcpy(out_pw + (size_t)grp * H, pw, sizeof(float) * (size_t)H);

        /* Eq. (5), over [0, t0] (or [0, t0-W] before a prefill window) */
        int64_t lim = (W > 0 && window_kind == 0) ? t0 - W : t0;
        int64_t n = lim + 1 > 0 ? lim + 1 : 0;
        int32_t* pos = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
        double* f = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
        for (int64_t s = 0; s < n; ++s) pos[s] = (int32_t)s;
        score_positions(&K, pq, fmt == OR_FP8 ? (double)psc : 1.0, pw, pos, n, f);

        if (mode == OR_REUSE) {                                      /* Eq. (6) */
            topk(f, pos, n, m, og);
            for (int t = 1; t < gs; ++t) memcpy(og + (size_t)t * m, og, sizeof(int32_t) * (size_t)m);
        } else {                                                     /* Eqs. (7)-(9) */
            int32_t* cand = (int32_t*)malloc(sizeof(int32_t) * (size_t)width);
            int proxy_slots = (W > 0 && window_kind == 0) ? c - wg : c;
            if (proxy_slots > 0) topk(f, pos, n, proxy_slots, cand);
            for (int u = 0; u < wg; ++u) {                           /* App. B window union */
                int64_t p = t0 - W + 1 + u;
                int ok = p >= 0 && p <= t0 + gs - 1;
                if (ok && window_kind == 1)                          /* decode: not twice */
                    for (int i = 0; i < c; ++i)
                        if (cand[i] == (int32_t)p) { ok = 0; break; }
                cand[proxy_slots + u] = ok ? (int32_t)p : -1;
            }
            if (out_cand) memcpy(out_cand + (size_t)grp * width, cand, sizeof(int32_t) * (size_t)width);
            int32_t* use = (int32_t*)malloc(sizeof(int32_t) * (size_t)width);
            double* fc = (double*)malloc(sizeof(double) * (size_t)width);
            for (int t = 0; t < gs; ++t) {
                int64_t tt = t0 + t;
                int nu = 0;
                for (int i = 0; i < width; ++i) {
                    int32_t p = cand[i];
                    if (p < 0 || p > tt) continue;
                    if (W > 0 && window_kind == 1 && i >= c && p < tt - W + 1) continue;
                    use[nu++] = p;
                }
                score_positions(&K, qg + (size_t)t * rowb, sg ? (double)sg[t] : 1.0,
                                wg_ + (size_t)t * H, use, nu, fc);
                topk(fc, use, nu, m, og + (size_t)t * m);
            }
            free(fc);
            free(use);
            free(cand);
        }
        free(pos);
        free(f);
    }
    free(pq);
    free(pw);
    return 0;
}

int oracle_index(int fmt, int H, int d,
                 const void* q, const float* q_scale, const float* w, int n_q, int64_t p0,
                 const void* k, const float* k_scale, int64_t n_k,
                 int mode, int g, int c, int m, int dense_below,
                 const int32_t* sel, int n_sel,
                 int32_t* out_idx, int32_t* out_cand,
                 void* out_pq, float* out_psc, float* out_pw) {
    return oracle_index_ex(fmt, H, d, q, q_scale, w, n_q, p0, k, k_scale, n_k, mode, g, c, m, dense_below,
                           0, 0, OR_AGG_MEAN, sel, n_sel, out_idx, out_cand, out_pq, out_psc, out_pw);
}

/*
 * PIVOT composed with IndexCache (Sec. 5.1 "Baselines"; the +IC rows of
 * Table 1).  IndexCache shares index sets along the layer axis (Sec. 2): one
 * layer's T_t serves nearby layers.  Layer l (0 <= l < n_layers) is an anchor
 * when anchor[l] != 0: it runs the indexer (mode as oracle_index: dense, or
 * Algorithm 1 with Reuse / Refine) on its own q[l], q_scale[l], w[l], k[l],
 * k_scale[l].  Any other layer's out_idx[l] [n_q, m] receives the sets of
 * the nearest anchor before it; its inputs are not read.  Layer 0 must be an
 * anchor.  Returns 0, or 1 for rejected arguments.
 */
int oracle_index_layers(int fmt, int H, int d, int n_layers, const uint8_t* anchor,
                        const void* const* q, const float* const* q_scale, const float* const* w,
                        int n_q, int64_t p0, const void* const* k, const float* const* k_scale, int64_t n_k,
                        int mode, int g, int c, int m, int dense_below, int32_t* const* out_idx) {
    if (n_layers < 1 || !anchor || !anchor[0] || n_q < 0 || m < 1) return 1;
    int src = 0;                                  /* the layer whose sets are shared */
    for (int l = 0; l < n_layers; ++l) {
        if (anchor[l]) {
            int rc = oracle_index(fmt, H, d, q[l], q_scale ? q_scale[l] : NULL, w[l], n_q, p0, k[l],
                                  k_scale ? k_scale[l] : NULL, n_k, mode, g, c, m, dense_below, NULL, 0,
                                  out_idx[l], NULL, NULL, NULL, NULL);
            if (rc != 0) return rc;
            src = l;
        } else {
            memcpy(out_idx[l], out_idx[src], sizeof(int32_t) * (size_t)n_q * (size_t)m);
        }
    }
    return 0;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
