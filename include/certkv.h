/*
 * certkv.h -- C ABI of libcertkv.so, the gfx950 (MI355X) implementation of the
 * CertKV one-shot compression pass over a prefilled KV cache.
 *
 * Source of the method: "Beyond Sparse Weights: When Is Attention
 * Compressible?" (arXiv 2608.21541), Section 4 ("CertKV: value-aware
 * compression under exact budgets", subsection "Dispersion-guided allocation
 * with exact slot accounting", Eq. certkv-curve) and the appendix subsection
 * "CertKV: implementation and exact-budget protocol" with its Algorithm 1.
 *
 * The pass, per (layer, sequence) and per KV head h:
 *   score     s_j  = sum over window rows and the GQA group of softmax weights
 *                    (the observation-window scorer the method keeps unchanged)
 *   allocate  a    = (s)_+ / sum (s)_+, keys ordered by s descending (ties: lower
 *                    index first), suffix moments m, W, Q, dispersion curve
 *                    c(b) = sqrt((m Q - |W|^2)_+), then a shared-multiplier
 *                    bisection (T steps) and one-token best-marginal repair to
 *                    an exact real-token budget
 *   select    the top-b_h keys of each head, emitted in ascending position
 *   tail      one synthetic slot per head: the proxy-weighted key and value
 *                    centroid of the evicted keys
 *   compact   a packed cache of b_h kept rows plus the slot row per head
 *
 * Conventions shared by every entry point
 *   - Tensor pointers are DEVICE pointers unless the name ends in _host.
 *   - The caller owns every buffer.  The library never allocates or frees
 *     device memory; scratch space comes from the caller's workspace
 *     (size from certkv_workspace_size) and must not be shared by two calls
 *     that run concurrently.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream)
 *     and the call returns without synchronising.  Argument errors are
 *     reported synchronously before anything is launched; CERTKV_EHIP reports
 *     a failed launch.
 *   - No entry point throws; every one returns a certkv_status.
 *
 * Index conventions
 *   L = num_layers, B = batch, H = num_kv_heads, G = group, d = head_dim,
 *   w = window, Hq = H*G query heads (query head hq belongs to KV head hq/G).
 *   Sequence b owns tokens [cu_seqlens[b], cu_seqlens[b+1]) of the packed token
 *   axis of length T = cu_seqlens[B]; its length is n_b.
 *   A "unit" is one (layer, sequence, KV head); units are numbered
 *   u = (l*B + b)*H + h.
 *   Window row q (0 <= q < w) of sequence b is the query at position
 *   n_b - w + q; with CERTKV_CAUSAL it sees keys j <= n_b - w + q.
 */
#ifndef CERTKV_H
#define CERTKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t certkv_status;
enum {
  CERTKV_OK = 0,
  CERTKV_EINVAL = -1,       /* null pointer, bad size, stride or flag      */
  CERTKV_EUNSUPPORTED = -2, /* head_dim not 64/128, dtype not built, or a  */
                            /* per-head slice spanning 4 GiB or more      */
  CERTKV_EINFEASIBLE = -3,  /* n_keep < 2 or n_keep > n_b (budget algebra), */
                            /* or b_min < w under CERTKV_KEEP_WINDOW       */
  CERTKV_ENONFINITE = -4,   /* written to *dev_status by a kernel that met */
                            /* a non-finite input (never returned by a    */
                            /* call: the launches are asynchronous)        */
  CERTKV_EWORKSPACE = -5,   /* workspace smaller than required             */
  CERTKV_EHIP = -6,         /* a HIP runtime call or launch failed         */
  CERTKV_ERANGE = -7        /* written to *dev_status by certkv_decode     */
                            /* when a packed segment holds more rows than */
                            /* its max_rows bound allowed for              */
};

enum { CERTKV_F32 = 0, CERTKV_BF16 = 1 };

enum {
  CERTKV_CAUSAL = 1u << 0,  /* window rows see only keys at or before them  */
  CERTKV_DRY_RUN = 1u << 1, /* validate arguments, launch nothing           */
  CERTKV_KEEP_WINDOW = 1u << 2, /* the w window keys of each sequence take  */
                            /* ranks 0..w-1 (ascending position), as if     */
                            /* their scores were +infinity, so every head   */
                            /* keeps them; their masses a_j are unchanged.  */
                            /* Budget calls need b_min >= w (else           */
                            /* CERTKV_EINFEASIBLE); a selection budget      */
                            /* below w keeps the first b window keys;       */
                            /* coverage budgets are at least w.  The paper  */
                            /* ranks all n keys (the default); this is the  */
                            /* option of never evicting the window.         */
  /* One-factor ablations of the appendix (one-factor ablations table),
   * each changing one design choice of the default pass:                    */
  CERTKV_STAT_UNCENTERED = 1u << 3, /* curves c(b) = sqrt(m Q), no centering */
  CERTKV_STAT_TAIL_MASS = 1u << 4,  /* curves c(b) = m(b), the tail mass     */
  CERTKV_ALLOC_UNIFORM = 1u << 5,   /* true uniform: b_h = B_real / H        */
  CERTKV_ALLOC_GREEDY = 1u << 6,    /* greedy marginal: no bisection step,   */
                                    /* the repair from b_min (steps ignored) */
  CERTKV_NO_SLOT = 1u << 7          /* no tail-summary row: its live slot is */
                                    /* one more real token per head, B_real  */
                                    /* = H n_keep with 1 <= n_keep <= n - 1; */
                                    /* k*, v* are still formed, the packed   */
                                    /* segments hold the b_h kept rows only  */
  /* The two statistic flags, or the two allocator flags, together are
   * CERTKV_EINVAL. */
};

/* Selection modes of certkv_select. */
enum {
  CERTKV_SELECT_BUDGET = 0,   /* keep the top budgets[u] keys of each unit  */
  CERTKV_SELECT_COVERAGE = 1  /* keep the top k_eta keys, k_eta written out */
};

/* Stage selectors for certkv_workspace_size. */
enum {
  CERTKV_STAGE_SCORE = 1,
  CERTKV_STAGE_ALLOCATE = 2,
  CERTKV_STAGE_SELECT = 3,
  CERTKV_STAGE_TAIL = 4,
  CERTKV_STAGE_COMPACT = 5,
  CERTKV_STAGE_COMPRESS = 6
};

/* A strided [L][tokens][heads][head_dim] tensor.  Strides are in ELEMENTS;
 * the head_dim axis is contiguous.  The pointer must be 16-byte aligned and
 * every stride a multiple of 8 elements.  The rows of one (layer, head,
 * sequence) must span less than 4 GiB ((n_max - 1) * s_token + head_dim
 * elements), else CERTKV_EUNSUPPORTED. */
typedef struct certkv_tensor {
  const void* ptr;
  int64_t s_layer;
  int64_t s_token;
  int64_t s_head;
} certkv_tensor;

typedef struct certkv_problem {
  int32_t num_layers;            /* L >= 1                                    */
  int32_t batch;                 /* B >= 1                                    */
  int32_t num_kv_heads;          /* H, 1..64                                  */
  int32_t group;                 /* G >= 1 query heads per KV head            */
  int32_t head_dim;              /* d: 64 or 128                              */
  int32_t window;                /* w: 1 <= w <= n_b for every sequence       */
  const int64_t* cu_seqlens_host;/* [B+1] host array, cu[0] = 0, increasing   */
  int32_t q_dtype;               /* CERTKV_F32 or CERTKV_BF16                 */
  int32_t kv_dtype;              /* CERTKV_F32 or CERTKV_BF16; equal to q_dtype */
  float softmax_scale;           /* logit scale; 0 selects 1/sqrt(d)          */
  uint32_t flags;                /* CERTKV_CAUSAL | CERTKV_DRY_RUN |
                                    CERTKV_KEEP_WINDOW                        */
  int32_t* dev_status;           /* optional device int32: kernels that meet a
                                    non-finite value (a window row whose
                                    log-sum-exp is not finite, a caller log-sum
                                    that is not finite, or a non-finite
                                    dispersion value) store CERTKV_ENONFINITE
                                    there; nothing else writes it, so the
                                    caller sets it to CERTKV_OK beforehand and
                                    reads it after synchronising.  NULL: no
                                    reporting.  Outputs computed from
                                    non-finite inputs are unspecified. */
} certkv_problem;

/* Outputs of the fused pass.  Layouts:
 *   scores        [L][H][T] fp32, the per-key window mass s_j
 *   budgets       [L*B*H] int32, b_h (real tokens kept per unit)
 *   kept_offsets  [L*B*H+1] int64, start of each unit's run in kept_idx
 *   kept_idx      [sum b_h] int32, kept positions (0-based within the
 *                 sequence), ascending inside each unit
 *   k_star,v_star [L*B*H][d] fp32, the tail-summary slot
 *   tail_mass     [L*B*H] fp64, m_h(b_h), the normalized evicted mass
 *   k_packed,
 *   v_packed      [sum (b_h+1)][d] in kv_dtype: per unit, its kept rows in
 *                 ascending position, then the slot row
 *   pos_packed    [sum (b_h+1)] int32, source position of each packed row,
 *                 -1 for the slot row
 *   packed_offsets[L*B*H+1] int64, start of each unit's packed segment
 *   curves        optional [L][H][T] fp32, c_h(b) for b = 0..n_b-1
 *   perm          optional [L][H][T] int32, key position at each rank
 *   alloc_stats   optional [L*B][3] int64 diagnostics of the allocation per
 *                 (layer, sequence): one-token repairs performed, and the
 *                 bisection and repair durations in 100 MHz clock ticks
 *   kept_mask     optional [L][H][T] uint8, 1 at the kept positions of each
 *                 unit and 0 elsewhere
 *   lse           optional [L][B*w][Hq] fp32, the natural-log log-sum-exp of
 *                 every window row over its visible keys (the caller's lse_in
 *                 when one was given)
 * Every (layer, sequence) block of the packed cache holds exactly
 * H * n_keep_b rows (the matched live-slot budget). */
typedef struct certkv_outputs {
  float* scores;
  int32_t* budgets;
  int64_t* kept_offsets;
  int32_t* kept_idx;
  float* k_star;
  float* v_star;
  double* tail_mass;
  void* k_packed;
  void* v_packed;
  int32_t* pos_packed;
  int64_t* packed_offsets;
  float* curves;
  int32_t* perm;
  int64_t* alloc_stats;
  uint8_t* kept_mask;
  float* lse;
} certkv_outputs;

/* Human-readable name of a status code (static storage). */
const char* certkv_status_string(certkv_status st);

/* Workspace bytes that `stage` needs for problem `p` (0 on invalid input).
 * The workspace must be 256-byte aligned. */
size_t certkv_workspace_size(const certkv_problem* p, int32_t stage);

/* Observation-window scoring (paper appendix, "CertKV: implementation and
 * exact-budget protocol": the unchanged window scorer; Section 3 one-row
 * setup for the 1/sqrt(d) logit scale).
 *   q_win  [L][B*w][Hq][d]: row b*w+q holds window query q of sequence b
 *   k      [L][T][H][d]
 *   lse_in optional [L][B*w][Hq] fp32: the natural-log log-sum-exp of each
 *          window row's logits scale * q . k_j over its visible keys, as an
 *          attention prefill already computes it.  When given, the pass that
 *          forms the row sums is skipped and K is read once; a non-finite
 *          entry is reported through dev_status.  NULL: computed here.
 *   scores [L][H][T] fp32 out: s_j = sum_{g in group(h)} sum_q softmax_j(
 *          scale * q_{g,q} . k_j) over the keys visible to row q
 *   ksum   optional [L*B*H][d] fp64 out: sum_j (s_j)_+ k_j (used by the tail
 *          summary to avoid re-reading evicted keys); NULL to skip.
 *   lse_out optional [L][B*w][Hq] fp32 out: the row log-sum-exp used (natural
 *          log), in lse_in's layout.
 * Softmax rows are normalized in fp32 from bf16 (or fp32) inputs with fp32
 * MFMA accumulation. */
certkv_status certkv_score(const certkv_problem* p, certkv_tensor q_win,
                           certkv_tensor k, const float* lse_in, float* scores,
                           double* ksum, float* lse_out, void* ws,
                           size_t ws_bytes, void* stream);

/* certkv_score without a caller workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops that forbid
 * allocation).  Same arguments, kernels and results as certkv_score; the
 * scoring partials live in a fixed device array of
 * certkv_score_noalloc_max_bytes() bytes (64 MiB) that each device holds
 * from its first call until the process ends.  A problem whose scoring
 * workspace (certkv_workspace_size(p, CERTKV_STAGE_SCORE)) exceeds that
 * returns CERTKV_EWORKSPACE before any launch.  Nothing in the array needs
 * to start at zero, and no call allocates or frees memory; every call on one
 * device shares the array, so calls that overlap on one device (on different
 * streams, or from several threads) race: the caller serializes them. */
size_t certkv_score_noalloc_max_bytes(void);
certkv_status certkv_score_noalloc(const certkv_problem* p,
                                   certkv_tensor q_win, certkv_tensor k,
                                   const float* lse_in, float* scores,
                                   double* ksum, float* lse_out, void* stream);

/* Dispersion curves and budget allocation (paper Section 4.1, Eq.
 * certkv-curve; appendix Algorithm 1, the sort, suffix-scan, bisection and
 * repair steps).
 *   scores      [L][H][T] fp32 in
 *   v           [L][T][H][d]
 *   n_keep_host [B] host: live slots per head incl. the slot, 2 <= n_keep <= n_b
 *   alpha       safeguard fraction (the paper uses 0.2)
 *   steps       bisection steps T (the paper uses 40), 0..200
 *   budgets     [L*B*H] int32 out
 *   perm        optional [L][H][T] int32 out, position at each rank
 *   curves      optional [L][H][T] fp32 out, c(b) for b = 0..n_b-1
 *   vsum        optional [L*B*H][d] fp64 out: sum_j (s_j)_+ v_j
 * Budget algebra per (layer, sequence): B_live = H*n_keep, B_real = B_live-H,
 * b_min = max(1, floor(alpha*B_real/H)), b_h in [b_min, n_b-1],
 * sum_h b_h = B_real.  Ordering: s descending, equal s by ascending position.
 * Integer results are a deterministic function of the fp32 curves: the
 * multiplier bisection evaluates fma(lambda, b, c(b)) in fp64 and takes the
 * smallest b among equal minima. */
certkv_status certkv_allocate(const certkv_problem* p, const float* scores,
                              certkv_tensor v, const int32_t* n_keep_host,
                              double alpha, int32_t steps, int32_t* budgets,
                              int32_t* perm, float* curves, double* vsum,
                              void* ws, size_t ws_bytes, void* stream);

/* Allocation from caller-supplied fp32 curves [L][H][T] (the bisection and
 * repair steps of Algorithm 1 alone).  Same budget algebra and tie rules as
 * certkv_allocate; used to check the integer stage against the oracle fed the
 * very same curves. */
certkv_status certkv_allocate_curves(const certkv_problem* p,
                                     const float* curves,
                                     const int32_t* n_keep_host, double alpha,
                                     int32_t steps, int32_t* budgets, void* ws,
                                     size_t ws_bytes, void* stream);

/* Selection of the kept keys (Algorithm 1, return step: the top-b_h real
 * tokens per head; coverage mode: the budget k_eta of the paper's coverage
 * definition, Section 3, with retained mass retain_mass = 1 - eta).
 *   scores       [L][H][T] fp32 in
 *   budgets_io   [L*B*H] int32: in for CERTKV_SELECT_BUDGET (1..n_b);
 *                out (k_eta) for CERTKV_SELECT_COVERAGE
 *   kept_offsets [L*B*H+1] int64 out
 *   kept_idx     int32 out, capacity kept_capacity entries; needs
 *                sum(budgets) entries, L*H*T in coverage mode
 *   kept_mask    optional [L][H][T] uint8 out: 1 at kept positions, else 0
 * Kept = the first b ranks of the order (s descending, ties by position);
 * positions are written ascending.  Coverage: k_eta = min{k >= 1 :
 * sum_{r<=k} a_(r) >= retain_mass}, the prefix summed in rank order in fp64,
 * n_b if the sum never reaches retain_mass. */
certkv_status certkv_select(const certkv_problem* p, const float* scores,
                            int32_t* budgets_io, int32_t mode,
                            double retain_mass, int64_t* kept_offsets,
                            int32_t* kept_idx, int64_t kept_capacity,
                            uint8_t* kept_mask, void* ws, size_t ws_bytes,
                            void* stream);

/* Tail-summary slot (Section 4.1: the synthetic pair is the key and value
 * centroid of the evicted suffix under r = a/m; Theorem "fixed-row tail
 * factorization" for why the weighted tail sum is the missing quantity).
 *   kept_offsets/kept_idx as produced by certkv_select
 *   ksum, vsum   optional totals from certkv_score / certkv_allocate; when both
 *                are given the evicted sums are formed as total minus kept
 *                (falling back to a direct pass when the evicted mass is under
 *                1/64 of the total); NULL means a direct pass over evicted keys
 *   k_star, v_star [L*B*H][d] fp32 out; tail_mass [L*B*H] fp64 out (m)
 * m = 0 gives k* = v* = 0 (the paper's convention for an empty tail). */
certkv_status certkv_tail_summary(const certkv_problem* p, const float* scores,
                                  certkv_tensor k, certkv_tensor v,
                                  const int64_t* kept_offsets,
                                  const int32_t* kept_idx, const double* ksum,
                                  const double* vsum, float* k_star,
                                  float* v_star, double* tail_mass, void* ws,
                                  size_t ws_bytes, void* stream);

/* Packed cache (appendix "Physical cache capacity": b_h real rows plus one
 * charged slot per head).  Kept rows are exact copies; the slot row is the
 * round-to-nearest-even kv_dtype value of the fp32 k*, v*.
 *   k_packed, v_packed [sum(b_h+1)][d] out; pos_packed out;
 *   packed_offsets [L*B*H+1] out. */
certkv_status certkv_compact(const certkv_problem* p, certkv_tensor k,
                             certkv_tensor v, const int64_t* kept_offsets,
                             const int32_t* kept_idx, const float* k_star,
                             const float* v_star, void* k_packed,
                             void* v_packed, int32_t* pos_packed,
                             int64_t* packed_offsets, void* stream);

/* The whole pass in order (score, allocate, select, tail summary, compact)
 * with one workspace of certkv_workspace_size(p, CERTKV_STAGE_COMPRESS).
 * lse_in is optional, as for certkv_score. */
certkv_status certkv_compress(const certkv_problem* p, certkv_tensor q_win,
                              certkv_tensor k, certkv_tensor v,
                              const float* lse_in, const int32_t* n_keep_host,
                              double alpha, int32_t steps,
                              const certkv_outputs* out, void* ws,
                              size_t ws_bytes, void* stream);

/* Decode over the packed cache (Section 4.1: after eviction each head keeps
 * its b_h real tokens and one charged centroid pair, and a later query
 * attends over these b_h + 1 rows as ordinary keys; the plain slot carries no
 * logit bias).  For the tq new queries of every sequence, query row
 * (t, head h*G + g) of layer l attends over the packed segment of unit
 * (l, b, h):
 *   z_i = scale <q, k_i>, out = sum_i softmax(z)_i v_i, lse = log sum_i e^z_i.
 *   q_new          [L][B*tq][Hq][d] in (kv_dtype), same stride rules as q_win
 *   max_rows       bound on the rows of any head's segment (b_h + 1), or 0 for
 *                  n_b of the longest sequence; it sizes the workspace. A
 *                  longer segment stores CERTKV_ERANGE in *dev_status and its
 *                  rows past the next multiple of 4096 are left out
 *   k_packed, v_packed, packed_offsets  the packed cache of certkv_compact or
 *                  certkv_compress (device)
 *   out            [L][B*tq][Hq][d] fp32 out (contiguous)
 *   lse            optional [L][B*tq][Hq] fp32 out (natural log)
 * Every packed row is visible to every new query (they follow the whole
 * cache).  bf16 caches only (CERTKV_EUNSUPPORTED for fp32); tq * G <= 512.
 * The workspace is certkv_decode_workspace_size(p, tq, max_rows) bytes,
 * 256-byte aligned; a non-finite output sets the status word. */
size_t certkv_decode_workspace_size(const certkv_problem* p, int32_t tq,
                                    int32_t max_rows);
certkv_status certkv_decode(const certkv_problem* p, certkv_tensor q_new,
                            int32_t tq, int32_t max_rows, const void* k_packed,
                            const void* v_packed,
                            const int64_t* packed_offsets, float* out,
                            float* lse, void* ws, size_t ws_bytes,
                            void* stream);

/* Clustered tail summaries (appendix, deterministic output-error bound for
 * clustered tail summaries): per head, the evicted ranks b_h..n-1 in the
 * pass's rank order are cut into m contiguous groups of ceil((n - b_h) / m)
 * ranks (later groups may be short or empty).  Per group g of unit u:
 *   cluster_count [U][m] int32 out   n_g
 *   cluster_k, cluster_v [U][m][d] out in kv_dtype: the unweighted mean key
 *                  and value (fp64 sums), as stored
 *   cluster_rk, cluster_rv [U][m] fp32 out: radii in the sense of the
 *                  cluster-radii equation, >= |k_j - kbar_g| and >= |v_j -
 *                  vbar_g| for every member against the stored means: with
 *                  c_g the mean of every S-th member (S = n_g / 64 clamped to
 *                  [1, 16]), max |x_j - c_g| + |c_g - xbar_g| (triangle
 *                  inequality; one pass over the members), fp64, rounded up
 *   kept_vmax [U] fp32 out: the largest norm of a kept value
 * Inputs: k, v as for certkv_score; perm [L][H][T] the rank order of the
 * pass (certkv_allocate or certkv_outputs.perm); budgets [U] (b_h).
 * The summaries replace the single slot: the problem must carry
 * CERTKV_NO_SLOT (else CERTKV_EINVAL), so that the evicted ranks are counted
 * once.  1 <= m <= 64, else CERTKV_EINVAL.  Allocates nothing. */
certkv_status certkv_cluster_tail(const certkv_problem* p, certkv_tensor k,
                                  certkv_tensor v, const int32_t* perm,
                                  const int32_t* budgets, int32_t m,
                                  void* cluster_k, void* cluster_v,
                                  int32_t* cluster_count, float* cluster_rk,
                                  float* cluster_rv, float* kept_vmax,
                                  void* stream);

/* Decode with clustered tail summaries: as certkv_decode over the kept rows
 * (k_packed, v_packed, packed_offsets: segments of kept rows only, e.g. the
 * packed cache of a CERTKV_NO_SLOT pass), plus per unit the m cluster terms of
 * certkv_cluster_tail: the ratio estimator
 *   out = (sum_S e^l v + sum_g n_g e^lbar_g vbar_g) / Zhat,
 *   lbar_g = scale <q, kbar_g>,  Zhat = sum_S e^l + sum_g n_g e^lbar_g,
 * lse = log Zhat.  bound (optional [L][B*tq][Hq] fp32 out): the runtime
 * certificate with r_g = scale |q| R_g: 3 (D_N + V' D_Z) / Zhat when
 * D_Z <= Zhat / 3, +infinity otherwise.  The segments must hold kept rows
 * only: a problem without CERTKV_NO_SLOT returns CERTKV_EINVAL (a slot row
 * would count the evicted mass a second time beside the cluster terms).
 * bf16 only; the workspace is certkv_decode_workspace_size(p, tq, max_rows). */
certkv_status certkv_decode_clustered(const certkv_problem* p,
                                      certkv_tensor q_new, int32_t tq,
                                      int32_t max_rows, const void* k_packed,
                                      const void* v_packed,
                                      const int64_t* packed_offsets, int32_t m,
                                      const void* cluster_k,
                                      const void* cluster_v,
                                      const int32_t* cluster_count,
                                      const float* cluster_rk,
                                      const float* cluster_rv,
                                      const float* kept_vmax, float* out,
                                      float* lse, float* bound, void* ws,
                                      size_t ws_bytes, void* stream);

/* Per-kernel timing.  While enabled, every kernel the library launches is
 * bracketed by two hipEvents on its launch stream; certkv_profile_read
 * synchronises those events and reports, per kernel name, the launch count
 * and the summed duration in milliseconds.  Returns the number of distinct
 * kernels (at most max_entries are written).  Disabled by default. */
certkv_status certkv_profile_enable(int32_t enable);
int32_t certkv_profile_read(char (*names)[64], int64_t* counts,
                            double* total_ms, int32_t max_entries);
void certkv_profile_reset(void);

#ifdef __cplusplus
}
#endif
#endif /* CERTKV_H */
