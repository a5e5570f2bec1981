/*
 * certkv_oracle.c -- TEST INFRASTRUCTURE.  A plain, slow, fp64 CPU oracle of
 * the CertKV one-shot compression pass.  Only the test suite, the smoke check
 * and the CPU-baseline leg of the benchmark may call it; the product path
 * (libcertkv.so) never does, and the two share no source.
 *
 * Source: "Beyond Sparse Weights: When Is Attention Compressible?"
 * (arXiv 2608.21541).  Every function below names the passage it follows.
 * Arithmetic is IEEE binary64, built with -ffp-contract=off so that every
 * a*b+c is two roundings unless fma() is written out.
 *
 * Readings of points the paper leaves open (each is listed in the design doc):
 *   - GQA: the scores of the query heads of one KV head are summed.
 *   - Causal window rows: row q at position p sees keys j <= p.
 *   - Sort key: the fp32 score s itself, descending; equal s keep ascending
 *     position (the paper's tie rule for orderings).
 *   - lambda_hi = 2 * max over every head and every b in [0, n-1] of c + 1.
 *   - argmin ties go to the smallest b; c(b) + lambda*b is evaluated as the
 *     single-rounding fma(lambda, b, c(b)) on the fp32 curve values.
 *   - Repair adds one token to the head with the smallest marginal
 *     c(b+1) - c(b) (ties: lowest head), or, should the bisection end above
 *     the budget, removes one from the head with the smallest c(b-1) - c(b).
 *   - The slot centroids are direct weighted sums over the evicted keys;
 *     m = 0 gives zero vectors.
 *
 * Parity pins of each function are the tests in tests/test_oracle_pins.py.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORA_OK 0
#define ORA_EINVAL -1
#define ORA_EINFEASIBLE -3
#define ORA_ENONFINITE -4
#define ORA_ENOMEM -7

int ora_curves_stat(int64_t n, int32_t d, const float* s32, const int32_t* perm,
                    const double* v, int32_t stat, double* c, float* c32);
int ora_budget_params_slot(int32_t H, int64_t n, int64_t n_keep, double alpha,
                           int32_t slot, int64_t* B_real, int64_t* b_min);
int ora_allocate_variant(int32_t H, int64_t n, const float* c32, int64_t n_keep,
                         double alpha, int32_t T, int32_t slot, int32_t uniform,
                         int32_t* b, int64_t* repairs, double* lam);
int ora_compress_block_variant(int64_t n, int32_t H, int32_t G, int32_t d, int32_t w,
                               const double* q, const double* k, const double* v,
                               double scale, int32_t causal, int64_t n_keep,
                               double alpha, int32_t T, int32_t keep_window,
                               int32_t variant, const float* s32_in,
                               double* s, float* s32, int32_t* perm, float* c32,
                               int32_t* b, int32_t* kept, int64_t* kept_off,
                               double* kstar, double* vstar, double* m,
                               int64_t* repairs);

/* ------------------------------------------------------------------------ */
/* Scores.  Section 3, one-row setup: A_j = exp(l_j) / sum_t exp(l_t) with
 * l_j = <q, k_j> / sqrt(d).  The window scorer sums the softmax weights of
 * every window row (and here every query head of the group) per key.
 *   q     [M][d]  the M = w*G window rows of one KV head
 *   qpos  [M]     position of each row (causal: keys j <= qpos visible)
 *   k     [n][d]
 *   s     [n]     out, sum over rows of A_{row, j}
 *   lse   [M]     out (may be NULL), natural-log partition function per row */
int ora_scores(int64_t n, int32_t d, int32_t M, const double* q,
               const int64_t* qpos, const double* k, double scale,
               int32_t causal, double* s, double* lse) {
  if (n <= 0 || d <= 0 || M <= 0) return ORA_EINVAL;
  double* logit = (double*)malloc(sizeof(double) * (size_t)n);
  if (!logit) return ORA_ENOMEM;
  for (int64_t j = 0; j < n; ++j) s[j] = 0.0;
  for (int32_t r = 0; r < M; ++r) {
    int64_t visible = n;
    if (causal) {
      visible = qpos[r] + 1;
      if (visible > n) visible = n;
      if (visible < 1) visible = 1;
    }
    const double* qr = q + (size_t)r * d;
    double mx = -INFINITY;
    for (int64_t j = 0; j < visible; ++j) {
      const double* kj = k + (size_t)j * d;
      double dot = 0.0;
      for (int32_t t = 0; t < d; ++t) dot += qr[t] * kj[t];
      logit[j] = scale * dot;
      if (logit[j] > mx) mx = logit[j];
    }
    double z = 0.0;
    for (int64_t j = 0; j < visible; ++j) z += exp(logit[j] - mx);
    for (int64_t j = 0; j < visible; ++j) s[j] += exp(logit[j] - mx) / z;
    if (lse) lse[r] = mx + log(z);
  }
  free(logit);
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Ordering.  Algorithm 1 sorts each head's keys by score descending; the
 * paper orders ties by index (Section 3, the ordering pi of the gap profile).
 * perm[r] = position of the key at rank r (rank 0 = highest score). */
static const float* g_sort_keys; /* qsort has no context argument */

static int cmp_desc_then_index(const void* pa, const void* pb) {
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  float sa = g_sort_keys[a], sb = g_sort_keys[b];
  if (sa > sb) return -1;
  if (sa < sb) return 1;
  return (a < b) ? -1 : (a > b);
}

int ora_order(int64_t n, const float* s32, int32_t* perm) {
  if (n <= 0) return ORA_EINVAL;
  for (int64_t j = 0; j < n; ++j) {
    if (!isfinite(s32[j])) return ORA_ENONFINITE;
    perm[j] = (int32_t)j;
  }
#pragma omp critical(ora_sort)
  {
    g_sort_keys = s32;
    qsort(perm, (size_t)n, sizeof(int32_t), cmp_desc_then_index);
  }
  return ORA_OK;
}

/* Ordering with the observation window kept (the option that never evicts
 * the w window keys, which the unchanged window scorer leaves to the
 * caller): the keys at positions n-w..n-1 take ranks 0..w-1 in ascending
 * position, as if their scores were +infinity; the other keys follow in the
 * plain order (score descending, ties by position).  w = 0 is the plain
 * order. */
int ora_order_window(int64_t n, const float* s32, int64_t w, int32_t* perm) {
  if (n <= 0 || w < 0 || w > n) return ORA_EINVAL;
  for (int64_t j = 0; j < n; ++j)
    if (!isfinite(s32[j])) return ORA_ENONFINITE;
  for (int64_t r = 0; r < w; ++r) perm[r] = (int32_t)(n - w + r);
  int32_t* rest = perm + w;
  for (int64_t j = 0; j < n - w; ++j) rest[j] = (int32_t)j;
  if (n - w > 1) {
#pragma omp critical(ora_sort)
    {
      g_sort_keys = s32;
      qsort(rest, (size_t)(n - w), sizeof(int32_t), cmp_desc_then_index);
    }
  }
  return ORA_OK;
}

/* Normalization, appendix "CertKV: implementation": a_j = (s_j)_+ /
 * sum_i (s_i)_+, normalized directly (no second softmax).  The sum runs in
 * position order.  An all-zero score vector gives the uniform a = 1/n. */
int ora_normalize(int64_t n, const float* s32, double* a) {
  double tot = 0.0;
  for (int64_t j = 0; j < n; ++j) {
    if (!isfinite(s32[j])) return ORA_ENONFINITE;
    double sp = s32[j] > 0.0f ? (double)s32[j] : 0.0;
    tot += sp;
  }
  for (int64_t j = 0; j < n; ++j) {
    double sp = s32[j] > 0.0f ? (double)s32[j] : 0.0;
    a[j] = tot > 0.0 ? sp / tot : 1.0 / (double)n;
  }
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Dispersion curve.  Section 4.1 Eq. certkv-curve and the appendix's suffix
 * moments: over the evicted suffix E(b) = ranks b..n-1 (0-based; the keys
 * ranked after the b kept ones)
 *   m(b) = sum a_j,  W(b) = sum a_j v_j,  Q(b) = sum a_j |v_j|^2,
 *   c(b) = sqrt((m Q - |W|^2)_+),  b = 0..n-1.
 * The sums are accumulated from rank n-1 down to rank 0, one key at a time.
 *   v [n][d] (position-indexed), c [n] fp64 out, c32 [n] fp32 out (either
 *   may be NULL). */
int ora_curves(int64_t n, int32_t d, const float* s32, const int32_t* perm,
               const double* v, double* c, float* c32) {
  return ora_curves_stat(n, d, s32, perm, v, 0, c, c32);
}

/* The statistics of the one-factor ablations (appendix, one-factor ablations
 * table): stat 0 is the centered dispersion above (the default), stat 1 the
 * uncentered dispersion sqrt(m(b) Q(b)) and stat 2 the tail mass m(b), on the
 * same suffix sums. */
int ora_curves_stat(int64_t n, int32_t d, const float* s32, const int32_t* perm,
                    const double* v, int32_t stat, double* c, float* c32) {
  if (stat < 0 || stat > 2) return ORA_EINVAL;
  if (n <= 0 || d <= 0) return ORA_EINVAL;
  double* a = (double*)malloc(sizeof(double) * (size_t)n);
  double* W = (double*)calloc((size_t)d, sizeof(double));
  if (!a || !W) {
    free(a);
    free(W);
    return ORA_ENOMEM;
  }
  int st = ora_normalize(n, s32, a);
  if (st != ORA_OK) {
    free(a);
    free(W);
    return st;
  }
  double m = 0.0, Q = 0.0;
  for (int64_t b = n - 1; b >= 0; --b) {
    int32_t j = perm[b];
    const double* vj = v + (size_t)j * d;
    double vv = 0.0;
    for (int32_t t = 0; t < d; ++t) vv += vj[t] * vj[t];
    m += a[j];
    Q += a[j] * vv;
    for (int32_t t = 0; t < d; ++t) W[t] += a[j] * vj[t];
    double w2 = 0.0;
    for (int32_t t = 0; t < d; ++t) w2 += W[t] * W[t];
    double cb;
    if (stat == 2) {
      cb = m;
    } else {
      double c2 = stat == 1 ? m * Q : m * Q - w2;
      cb = sqrt(c2 > 0.0 ? c2 : 0.0);
    }
    if (c) c[b] = cb;
    if (c32) c32[b] = (float)cb;
  }
  free(a);
  free(W);
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Exact slot accounting, Section 4.1 and the appendix: with n_keep live
 * slots per head, B_live = H n_keep, B_real = B_live - H, b_min =
 * max{1, floor(alpha B_real / H)}; feasible iff 2 <= n_keep <= n. */
int ora_budget_params(int32_t H, int64_t n, int64_t n_keep, double alpha,
                      int64_t* B_real, int64_t* b_min) {
  return ora_budget_params_slot(H, n, n_keep, alpha, 1, B_real, b_min);
}

/* The same algebra with or without the slot.  Without it (the no-slot
 * ablation: the slot's live row goes to one more real token per head) all
 * H n_keep live rows are real: B_real = H n_keep, feasible iff
 * 1 <= n_keep <= n - 1 (a head keeps at most n - 1 keys). */
int ora_budget_params_slot(int32_t H, int64_t n, int64_t n_keep, double alpha,
                           int32_t slot, int64_t* B_real, int64_t* b_min) {
  if (H <= 0 || n <= 0) return ORA_EINVAL;
  if (slot) {
    if (n_keep < 2 || n_keep > n) return ORA_EINFEASIBLE;
  } else {
    if (n_keep < 1 || n_keep > n - 1) return ORA_EINFEASIBLE;
  }
  int64_t br = (int64_t)H * n_keep - (slot ? H : 0);
  int64_t bm = (int64_t)floor(alpha * (double)br / (double)H);
  if (bm < 1) bm = 1;
  if (bm > n - 1 || (int64_t)H * bm > br) return ORA_EINFEASIBLE;
  *B_real = br;
  *b_min = bm;
  return ORA_OK;
}

/* argmin over b in [lo, hi] of fma(lam, b, c(b)), smallest b on ties. */
int64_t ora_argmin_penalized(const float* c32, int64_t lo, int64_t hi,
                             double lam) {
  int64_t best = lo;
  double bestv = fma(lam, (double)lo, (double)c32[lo]);
  for (int64_t b = lo + 1; b <= hi; ++b) {
    double f = fma(lam, (double)b, (double)c32[b]);
    if (f < bestv) {
      bestv = f;
      best = b;
    }
  }
  return best;
}

/* Allocation, Algorithm 1: lambda bisection on the shared multiplier for T
 * steps, b_h = b_h(lambda_hi), then one-token best-marginal repair until
 * sum b_h = B_real.
 *   c32 [H][n] fp32 curves; b [H] out; repairs (may be NULL) out;
 *   lam (may be NULL) out: the final {lambda_lo, lambda_hi}. */
int ora_allocate(int32_t H, int64_t n, const float* c32, int64_t n_keep,
                 double alpha, int32_t T, int32_t* b, int64_t* repairs,
                 double* lam) {
  return ora_allocate_variant(H, n, c32, n_keep, alpha, T, 1, 0, b, repairs, lam);
}

/* The allocators of the one-factor ablations: uniform != 0 gives every head
 * the same B_real / H (which the budget algebra makes whole: n_keep - 1 with
 * the slot, n_keep without); otherwise the Lagrangian allocation with repair
 * above, where T = 0 is the greedy-marginal allocator (every head at b_min,
 * then one token at a time to the smallest marginal). */
int ora_allocate_variant(int32_t H, int64_t n, const float* c32, int64_t n_keep,
                         double alpha, int32_t T, int32_t slot, int32_t uniform,
                         int32_t* b, int64_t* repairs, double* lam) {
  int64_t B_real, b_min;
  int st = ora_budget_params_slot(H, n, n_keep, alpha, slot, &B_real, &b_min);
  if (st != ORA_OK) return st;
  if (uniform) {
    for (int32_t h = 0; h < H; ++h) b[h] = (int32_t)(B_real / H);
    if (repairs) *repairs = 0;
    if (lam) lam[0] = lam[1] = 0.0;
    return ORA_OK;
  }
  double cmax = 0.0;
  for (int32_t h = 0; h < H; ++h)
    for (int64_t j = 0; j < n; ++j) {
      double cj = (double)c32[(size_t)h * n + j];
      if (!isfinite(cj)) return ORA_ENONFINITE;
      if (cj > cmax) cmax = cj;
    }
  double lo = 0.0, hi = 2.0 * cmax + 1.0;
  int64_t* bl = (int64_t*)malloc(sizeof(int64_t) * (size_t)H);
  int64_t* bh = (int64_t*)malloc(sizeof(int64_t) * (size_t)H);
  if (!bl || !bh) {
    free(bl);
    free(bh);
    return ORA_ENOMEM;
  }
  for (int32_t h = 0; h < H; ++h)
    bh[h] = ora_argmin_penalized(c32 + (size_t)h * n, b_min, n - 1, hi);
  for (int32_t t = 0; t < T; ++t) {
    double lam = (lo + hi) / 2.0;
    int64_t sum = 0;
    for (int32_t h = 0; h < H; ++h) {
      bl[h] = ora_argmin_penalized(c32 + (size_t)h * n, b_min, n - 1, lam);
      sum += bl[h];
    }
    if (sum > B_real) {
      lo = lam;
    } else {
      hi = lam;
      for (int32_t h = 0; h < H; ++h) bh[h] = bl[h];
    }
  }
  int64_t sum = 0, nrep = 0;
  for (int32_t h = 0; h < H; ++h) sum += bh[h];
  while (sum < B_real) {
    int32_t best = -1;
    double bestd = 0.0;
    for (int32_t h = 0; h < H; ++h) {
      if (bh[h] >= n - 1) continue;
      const float* ch = c32 + (size_t)h * n;
      double dl = (double)ch[bh[h] + 1] - (double)ch[bh[h]];
      if (best < 0 || dl < bestd) {
        best = h;
        bestd = dl;
      }
    }
    if (best < 0) break; /* cannot happen: B_real <= H (n-1) */
    bh[best] += 1;
    sum += 1;
    ++nrep;
  }
  while (sum > B_real) {
    int32_t best = -1;
    double bestd = 0.0;
    for (int32_t h = 0; h < H; ++h) {
      if (bh[h] <= b_min) continue;
      const float* ch = c32 + (size_t)h * n;
      double dl = (double)ch[bh[h] - 1] - (double)ch[bh[h]];
      if (best < 0 || dl < bestd) {
        best = h;
        bestd = dl;
      }
    }
    if (best < 0) break; /* cannot happen: H b_min <= B_real */
    bh[best] -= 1;
    sum -= 1;
    ++nrep;
  }
  for (int32_t h = 0; h < H; ++h) b[h] = (int32_t)bh[h];
  if (repairs) *repairs = nrep;
  if (lam) {
    lam[0] = lo;
    lam[1] = hi;
  }
  free(bl);
  free(bh);
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Selection, Algorithm 1 return step: the b top-ranked keys, listed by
 * ascending position.  kept [b] out. */
int ora_select(int64_t n, const int32_t* perm, int64_t b, int32_t* kept) {
  if (b < 0 || b > n) return ORA_EINVAL;
  unsigned char* mark = (unsigned char*)calloc((size_t)n, 1);
  if (!mark) return ORA_ENOMEM;
  for (int64_t r = 0; r < b; ++r) mark[perm[r]] = 1;
  int64_t o = 0;
  for (int64_t j = 0; j < n; ++j)
    if (mark[j]) kept[o++] = (int32_t)j;
  free(mark);
  return ORA_OK;
}

/* Coverage budget, Section 3 Eq. coverage-def with retained fraction
 * retain = 1 - eta: the smallest k >= k_min whose top-k mass
 * sum_{r<=k} a_(r), summed in rank order, reaches retain; n if it never
 * does.  k_min = 1 is the definition; k_min = w keeps the whole observation
 * window when it leads the order. */
int ora_coverage(int64_t n, const float* s32, const int32_t* perm,
                 double retain, int64_t k_min, int64_t* k_eta) {
  if (k_min < 1 || k_min > n) return ORA_EINVAL;
  double* a = (double*)malloc(sizeof(double) * (size_t)n);
  if (!a) return ORA_ENOMEM;
  int st = ora_normalize(n, s32, a);
  if (st != ORA_OK) {
    free(a);
    return st;
  }
  double p = 0.0;
  int64_t k = n;
  for (int64_t r = 0; r < n; ++r) {
    p += a[perm[r]];
    if (r + 1 >= k_min && p >= retain) {
      k = r + 1;
      break;
    }
  }
  *k_eta = k;
  free(a);
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Tail summary, Section 4.1: with r_j = a_j / m over the evicted set E,
 * (k*, v*) = E_{j~r}[(k_j, v_j)] and m = sum_E a_j; m = 0 gives zero
 * vectors (appendix, centered-moment envelope: v* = 0 when m = 0).
 *   kept [b] ascending positions; k, v [n][d]; kstar, vstar [d] out. */
int ora_tail(int64_t n, int32_t d, const float* s32, const int32_t* kept,
             int64_t b, const double* k, const double* v, double* kstar,
             double* vstar, double* m_out) {
  double* a = (double*)malloc(sizeof(double) * (size_t)n);
  unsigned char* mark = (unsigned char*)calloc((size_t)n, 1);
  if (!a || !mark) {
    free(a);
    free(mark);
    return ORA_ENOMEM;
  }
  int st = ora_normalize(n, s32, a);
  if (st != ORA_OK) {
    free(a);
    free(mark);
    return st;
  }
  for (int64_t i = 0; i < b; ++i) mark[kept[i]] = 1;
  double m = 0.0;
  for (int32_t t = 0; t < d; ++t) kstar[t] = vstar[t] = 0.0;
  for (int64_t j = 0; j < n; ++j) {
    if (mark[j]) continue;
    m += a[j];
    for (int32_t t = 0; t < d; ++t) {
      kstar[t] += a[j] * k[(size_t)j * d + t];
      vstar[t] += a[j] * v[(size_t)j * d + t];
    }
  }
  for (int32_t t = 0; t < d; ++t) {
    kstar[t] = m > 0.0 ? kstar[t] / m : 0.0;
    vstar[t] = m > 0.0 ? vstar[t] / m : 0.0;
  }
  *m_out = m;
  free(a);
  free(mark);
  return ORA_OK;
}

/* Round an fp32 value to bfloat16, round-to-nearest-even (IEEE 754
 * binary32 -> the upper 16 bits), NaN kept quiet. */
uint16_t ora_f32_to_bf16(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu))
    return (uint16_t)((u >> 16) | 0x0040u);
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

/* ------------------------------------------------------------------------ */
/* Output-error helpers (Section 3.2, Theorem "fixed-row tail
 * factorization"; the worked examples of the oracle-subset and proxy
 * sections of the appendix use the same quantities).
 * For one realized row with weights A [n] and values V [n][d], a kept mask,
 * and a compensation vector u [d] (NULL = none):
 *   err = | sum_{j kept} A_j V_j + u - sum_j A_j V_j |_2.               */
double ora_row_error(int64_t n, int32_t d, const double* A, const double* V,
                     const unsigned char* kept, const double* u) {
  double acc2 = 0.0;
  for (int32_t t = 0; t < d; ++t) {
    double full = 0.0, part = 0.0;
    for (int64_t j = 0; j < n; ++j) {
      full += A[j] * V[(size_t)j * d + t];
      if (kept[j]) part += A[j] * V[(size_t)j * d + t];
    }
    double e = part + (u ? u[t] : 0.0) - full;
    acc2 += e * e;
  }
  return sqrt(acc2);
}

/* ------------------------------------------------------------------------ */
/* One (layer, sequence) block end to end: every KV head through score, order,
 * curves, allocation, selection and tail, heads in parallel (OpenMP) where a
 * stage is per head.  Inputs already in fp64.
 *   q      [w][H*G][d]   window rows of this sequence
 *   k, v   [n][H][d]
 *   s      [H][n] fp64 out; s32 [H][n] fp32 out (the shared scores)
 *   perm   [H][n] out; c32 [H][n] out; b [H] out
 *   kept   [H*n] out, unit h's run at kept_off[h]; kept_off [H+1] out
 *   kstar, vstar [H][d] out; m [H] out
 * When s32_in is not NULL the scoring step is skipped and those fp32 scores
 * are used instead (stage parity: the oracle fed the GPU's scores).
 * keep_window != 0 ranks the w window keys first (ora_order_window), so
 * every head keeps them; it needs b_min >= w. */
int ora_compress_block(int64_t n, int32_t H, int32_t G, int32_t d, int32_t w,
                       const double* q, const double* k, const double* v,
                       double scale, int32_t causal, int64_t n_keep,
                       double alpha, int32_t T, int32_t keep_window,
                       const float* s32_in,
                       double* s, float* s32, int32_t* perm, float* c32,
                       int32_t* b, int32_t* kept, int64_t* kept_off,
                       double* kstar, double* vstar, double* m,
                       int64_t* repairs) {
  return ora_compress_block_variant(n, H, G, d, w, q, k, v, scale, causal, n_keep, alpha, T,
                                    keep_window, 0, s32_in, s, s32, perm, c32, b, kept,
                                    kept_off, kstar, vstar, m, repairs);
}

/* The whole block under a one-factor ablation.  variant bits: 1 uncentered
 * statistic, 2 tail-mass statistic, 4 uniform allocator, 8 greedy-marginal
 * allocator (T = 0), 16 no slot (B_real = H n_keep; the tail summary is still
 * formed, the packed cache would hold no slot row). */
int ora_compress_block_variant(int64_t n, int32_t H, int32_t G, int32_t d, int32_t w,
                               const double* q, const double* k, const double* v,
                               double scale, int32_t causal, int64_t n_keep,
                               double alpha, int32_t T, int32_t keep_window,
                               int32_t variant, const float* s32_in,
                               double* s, float* s32, int32_t* perm, float* c32,
                               int32_t* b, int32_t* kept, int64_t* kept_off,
                               double* kstar, double* vstar, double* m,
                               int64_t* repairs) {
  if (w > n || w <= 0) return ORA_EINVAL;
  if ((variant & 3) == 3 || (variant & 12) == 12 || (variant & ~31)) return ORA_EINVAL;
  const int32_t stat = (variant & 1) ? 1 : (variant & 2) ? 2 : 0;
  const int32_t slot = (variant & 16) ? 0 : 1;
  if (variant & 8) T = 0;
  int32_t M = w * G;
  int err = ORA_OK;
  int64_t B_real, b_min;
  int st = ora_budget_params_slot(H, n, n_keep, alpha, slot, &B_real, &b_min);
  if (st != ORA_OK) return st;
  /* with the window kept, every head must be able to hold it */
  if (keep_window && b_min < w) return ORA_EINFEASIBLE;
#pragma omp parallel for schedule(dynamic, 1)
  for (int32_t h = 0; h < H; ++h) {
    int lerr = ORA_OK;
    double* kh = (double*)malloc(sizeof(double) * (size_t)n * d);
    double* vh = (double*)malloc(sizeof(double) * (size_t)n * d);
    double* qh = (double*)malloc(sizeof(double) * (size_t)M * d);
    int64_t* qpos = (int64_t*)malloc(sizeof(int64_t) * (size_t)M);
    if (!kh || !vh || !qh || !qpos) lerr = ORA_ENOMEM;
    if (lerr == ORA_OK) {
      for (int64_t j = 0; j < n; ++j)
        for (int32_t t = 0; t < d; ++t) {
          kh[(size_t)j * d + t] = k[((size_t)j * H + h) * d + t];
          vh[(size_t)j * d + t] = v[((size_t)j * H + h) * d + t];
        }
      for (int32_t r = 0; r < w; ++r)
        for (int32_t g = 0; g < G; ++g) {
          int32_t row = r * G + g;
          qpos[row] = n - w + r;
          for (int32_t t = 0; t < d; ++t)
            qh[(size_t)row * d + t] =
                q[((size_t)r * H * G + (size_t)h * G + g) * d + t];
        }
      if (s32_in) {
        for (int64_t j = 0; j < n; ++j) {
          s32[(size_t)h * n + j] = s32_in[(size_t)h * n + j];
          s[(size_t)h * n + j] = (double)s32_in[(size_t)h * n + j];
        }
      } else {
        lerr = ora_scores(n, d, M, qh, qpos, kh, scale, causal,
                          s + (size_t)h * n, NULL);
        for (int64_t j = 0; j < n; ++j)
          s32[(size_t)h * n + j] = (float)s[(size_t)h * n + j];
      }
    }
    if (lerr == ORA_OK)
      lerr = ora_order_window(n, s32 + (size_t)h * n, keep_window ? w : 0,
                              perm + (size_t)h * n);
    if (lerr == ORA_OK)
      lerr = ora_curves_stat(n, d, s32 + (size_t)h * n, perm + (size_t)h * n, vh,
                             stat, NULL, c32 + (size_t)h * n);
    free(kh);
    free(vh);
    free(qh);
    free(qpos);
    if (lerr != ORA_OK) {
#pragma omp critical(ora_err)
      err = lerr;
    }
  }
  if (err != ORA_OK) return err;
  err = ora_allocate_variant(H, n, c32, n_keep, alpha, T, slot, (variant & 4) != 0, b,
                             repairs, NULL);
  if (err != ORA_OK) return err;
  kept_off[0] = 0;
  for (int32_t h = 0; h < H; ++h) kept_off[h + 1] = kept_off[h] + b[h];
#pragma omp parallel for schedule(dynamic, 1)
  for (int32_t h = 0; h < H; ++h) {
    int lerr = ora_select(n, perm + (size_t)h * n, b[h], kept + kept_off[h]);
    double* kh = (double*)malloc(sizeof(double) * (size_t)n * d);
    double* vh = (double*)malloc(sizeof(double) * (size_t)n * d);
    if (!kh || !vh) lerr = ORA_ENOMEM;
    if (lerr == ORA_OK) {
      for (int64_t j = 0; j < n; ++j)
        for (int32_t t = 0; t < d; ++t) {
          kh[(size_t)j * d + t] = k[((size_t)j * H + h) * d + t];
          vh[(size_t)j * d + t] = v[((size_t)j * H + h) * d + t];
        }
      lerr = ora_tail(n, d, s32 + (size_t)h * n, kept + kept_off[h], b[h], kh,
                      vh, kstar + (size_t)h * d, vstar + (size_t)h * d, m + h);
    }
    free(kh);
    free(vh);
    if (lerr != ORA_OK) {
#pragma omp critical(ora_err)
      err = lerr;
    }
  }
  return err;
}

int ora_num_threads(void) {
#ifdef _OPENMP
  extern int omp_get_max_threads(void);
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Decode over the packed cache.  Section 4.1: after eviction each head keeps
 * its b_h real tokens and one charged centroid pair (k*, v*), and a later
 * query attends over these b_h + 1 rows as ordinary keys; the plain slot
 * carries no logit bias.  For query row r:
 *   z_i = scale <q_r, k_i>,  out_r = sum_i softmax(z)_i v_i,
 *   lse_r = log sum_i exp z_i  (evaluated with the maximum factored out).
 *   q [m][d], kp [nk][d], vp [nk][d], out [m][d], lse [m] or NULL. */
int ora_decode(int64_t nk, int32_t m, int32_t d, const double* q, const double* kp,
               const double* vp, double scale, double* out, double* lse) {
  if (nk < 1 || m < 0 || d < 1) return ORA_EINVAL;
  double* z = (double*)malloc((size_t)nk * sizeof(double));
  if (!z) return ORA_ENOMEM;
  int err = ORA_OK;
  for (int32_t r = 0; r < m; ++r) {
    double zmax = -INFINITY;
    for (int64_t i = 0; i < nk; ++i) {
      double dot = 0.0;
      for (int32_t t = 0; t < d; ++t) dot += q[(int64_t)r * d + t] * kp[i * d + t];
      z[i] = scale * dot;
      if (isnan(z[i])) err = ORA_ENONFINITE;
      if (z[i] > zmax) zmax = z[i];
    }
    double zsum = 0.0;
    for (int64_t i = 0; i < nk; ++i) zsum += exp(z[i] - zmax);
    for (int32_t t = 0; t < d; ++t) out[(int64_t)r * d + t] = 0.0;
    for (int64_t i = 0; i < nk; ++i) {
      const double a = exp(z[i] - zmax) / zsum;
      for (int32_t t = 0; t < d; ++t) out[(int64_t)r * d + t] += a * vp[i * d + t];
    }
    if (lse) lse[r] = zmax + log(zsum);
  }
  free(z);
  return err;
}

/* Theorem "future-query lift and summary mismatch" (section "Scoped
 * guarantees behind CertKV"): one future query row over the original n keys,
 * split into the retained set S (kept[j] != 0) and the evicted set T, with a
 * slot whose value is v* = sum_T r_j v_j.
 *   A     exact attention over S u T, O = sum_j A_j v_j;
 *   Ahat  attention over S u {slot}, slot logit z* = scale <q, k*>,
 *         Ohat = sum_S Ahat_i v_i + Ahat_* v*.
 *   out[0] p = A(T)      out[1] q = Ahat_*
 *   out[2] ||a - r||_1 with a = A_T / p (0 when p = 0)
 *   out[3] Lambda_T = log sum_T exp z_j (-inf for an empty T)
 *   out[4] z*            out[5] V_max = max_j ||v_j||_2 over S u T
 *   out[6] ||O - Ohat||_2
 * The theorem bounds out[6] by V_max (2 |p - q| + min(p, q) ||a - r||_1) and
 * |p - q| by tanh(|Lambda_T - z*| / 4). */
int ora_lift_terms(int64_t n, int32_t d, const double* q, const double* k, const double* v,
                   const uint8_t* kept, const double* r, const double* kslot,
                   const double* vslot, double scale, double* out) {
  if (n < 1 || d < 1) return ORA_EINVAL;
  double* z = (double*)malloc((size_t)n * sizeof(double));
  double* O = (double*)calloc((size_t)d, sizeof(double));
  double* Oh = (double*)calloc((size_t)d, sizeof(double));
  if (!z || !O || !Oh) {
    free(z);
    free(O);
    free(Oh);
    return ORA_ENOMEM;
  }
  double zs = 0.0;
  for (int32_t t = 0; t < d; ++t) zs += q[t] * kslot[t];
  zs *= scale;
  double zmax = zs, vmax = 0.0;
  for (int64_t j = 0; j < n; ++j) {
    double dot = 0.0, vv = 0.0;
    for (int32_t t = 0; t < d; ++t) {
      dot += q[t] * k[j * d + t];
      vv += v[j * d + t] * v[j * d + t];
    }
    z[j] = scale * dot;
    if (z[j] > zmax) zmax = z[j];
    if (sqrt(vv) > vmax) vmax = sqrt(vv);
  }
  double ZS = 0.0, ZT = 0.0;
  for (int64_t j = 0; j < n; ++j) {
    const double e = exp(z[j] - zmax);
    if (kept[j])
      ZS += e;
    else
      ZT += e;
  }
  const double es = exp(zs - zmax);
  const double Z = ZS + ZT, Zh = ZS + es;
  const double p = ZT / Z, qs = es / Zh;
  double l1 = 0.0;
  for (int64_t j = 0; j < n; ++j) {
    const double e = exp(z[j] - zmax);
    const double A = e / Z;
    for (int32_t t = 0; t < d; ++t) O[t] += A * v[j * d + t];
    if (kept[j]) {
      const double Ah = e / Zh;
      for (int32_t t = 0; t < d; ++t) Oh[t] += Ah * v[j * d + t];
    } else if (p > 0.0) {
      l1 += fabs(A / p - r[j]);
    }
  }
  for (int32_t t = 0; t < d; ++t) Oh[t] += qs * vslot[t];
  double err2 = 0.0;
  for (int32_t t = 0; t < d; ++t) err2 += (O[t] - Oh[t]) * (O[t] - Oh[t]);
  out[0] = p;
  out[1] = qs;
  out[2] = l1;
  out[3] = ZT > 0.0 ? zmax + log(ZT) : -INFINITY;
  out[4] = zs;
  out[5] = vmax;
  out[6] = sqrt(err2);
  free(z);
  free(O);
  free(Oh);
  return ORA_OK;
}

/* ------------------------------------------------------------------------ */
/* Clustered tail summaries (appendix, deterministic output-error bound for
 * clustered tail summaries).  The evicted ranks b..n-1 of one head, in the
 * pass's order, are cut into m contiguous groups of ceil((n - b) / m) ranks
 * (later groups may be short or empty).  Per group g: the count n_g, the
 * representative key and value (the unweighted means, rounded to fp32 and
 * then to bf16 when bf16 != 0, as they would be stored), and radii that the
 * cluster-radii equation admits, i.e. upper bounds of |k_j - kbar_g| and
 * |v_j - vbar_g| over the members: with c_g the mean of every S-th member
 * (ranks r0, r0 + S, ...; S = n_g / 64 clamped to [1, ORA_CLUSTER_SAMPLE],
 * so at least 64 members or all of them),
 *   R_g = max_j |k_j - c_g| + |c_g - kbar_g|   (triangle inequality),
 * likewise rho_g, rounded up to fp32.  Also the largest kept value norm.
 *   perm [n] the rank order; k, v [n][d] position-indexed
 *   kbar, vbar [m][d] out; cnt [m] out; R, rho [m] out; vmax_kept out. */
#define ORA_CLUSTER_SAMPLE 16
static double ora_store_rep(double x, int32_t bf16) {
  float f = (float)x;
  if (!bf16) return (double)f;
  uint32_t b = (uint32_t)ora_f32_to_bf16(f) << 16;
  float y;
  memcpy(&y, &b, 4);
  return (double)y;
}

static float ora_round_up_f32(double x) {
  float f = (float)x;
  if ((double)f < x) f = nextafterf(f, INFINITY);
  return f;
}

int ora_cluster_summaries(int64_t n, int32_t d, const int32_t* perm, int64_t b,
                          const double* k, const double* v, int32_t m, int32_t bf16,
                          double* kbar, double* vbar, int32_t* cnt, float* R, float* rho,
                          float* vmax_kept) {
  if (n <= 0 || d <= 0 || m <= 0 || b < 0 || b > n) return ORA_EINVAL;
  const int64_t E = n - b;
  const int64_t cs = (E + m - 1) / m;
  for (int32_t g = 0; g < m; ++g) {
    int64_t r0 = b + (int64_t)g * cs, r1 = r0 + cs;
    if (r0 > n) r0 = n;
    if (r1 > n) r1 = n;
    cnt[g] = (int32_t)(r1 - r0);
    double* kb = kbar + (size_t)g * d;
    double* vb = vbar + (size_t)g * d;
    for (int32_t t = 0; t < d; ++t) kb[t] = vb[t] = 0.0;
    R[g] = rho[g] = 0.f;
    if (r1 <= r0) continue;
    for (int64_t r = r0; r < r1; ++r) {
      const int32_t j = perm[r];
      for (int32_t t = 0; t < d; ++t) {
        kb[t] += k[(size_t)j * d + t];
        vb[t] += v[(size_t)j * d + t];
      }
    }
    for (int32_t t = 0; t < d; ++t) {
      kb[t] = ora_store_rep(kb[t] / (double)(r1 - r0), bf16);
      vb[t] = ora_store_rep(vb[t] / (double)(r1 - r0), bf16);
    }
    /* provisional centres: the mean of the sampled members */
    double* ck = (double*)calloc((size_t)2 * d, sizeof(double));
    if (!ck) return ORA_ENOMEM;
    double* cv = ck + d;
    int64_t stride = (r1 - r0) / 64;
    if (stride < 1) stride = 1;
    if (stride > ORA_CLUSTER_SAMPLE) stride = ORA_CLUSTER_SAMPLE;
    int64_t ns = 0;
    for (int64_t r = r0; r < r1; r += stride, ++ns) {
      const int32_t j = perm[r];
      for (int32_t t = 0; t < d; ++t) {
        ck[t] += k[(size_t)j * d + t];
        cv[t] += v[(size_t)j * d + t];
      }
    }
    for (int32_t t = 0; t < d; ++t) {
      ck[t] /= (double)ns;
      cv[t] /= (double)ns;
    }
    double rk = 0.0, rv = 0.0;
    for (int64_t r = r0; r < r1; ++r) {
      const int32_t j = perm[r];
      double sk = 0.0, sv = 0.0;
      for (int32_t t = 0; t < d; ++t) {
        const double dk = k[(size_t)j * d + t] - ck[t];
        const double dv = v[(size_t)j * d + t] - cv[t];
        sk += dk * dk;
        sv += dv * dv;
      }
      if (sk > rk) rk = sk;
      if (sv > rv) rv = sv;
    }
    double ek = 0.0, ev = 0.0;
    for (int32_t t = 0; t < d; ++t) {
      ek += (ck[t] - kb[t]) * (ck[t] - kb[t]);
      ev += (cv[t] - vb[t]) * (cv[t] - vb[t]);
    }
    free(ck);
    R[g] = ora_round_up_f32(sqrt(rk) + sqrt(ek));
    rho[g] = ora_round_up_f32(sqrt(rv) + sqrt(ev));
  }
  double vm = 0.0;
  for (int64_t r = 0; r < b; ++r) {
    const int32_t j = perm[r];
    double s2 = 0.0;
    for (int32_t t = 0; t < d; ++t) s2 += v[(size_t)j * d + t] * v[(size_t)j * d + t];
    if (s2 > vm) vm = s2;
  }
  *vmax_kept = ora_round_up_f32(sqrt(vm));
  return ORA_OK;
}

/* The ratio estimator of the clustered-summary theorem and its certificate,
 * for one query q [d]: logits l_j = scale <q, k_j> over the nk kept rows
 * kp, vp [nk][d]; cluster logits lbar_g = scale <q, kbar_g> with weight
 * n_g e^{lbar_g}; r_g = scale |q| R_g (the Cauchy-Schwarz logit radius).
 *   out [d]: Ohat = (sum_S e^l v + sum_g n_g e^lbar vbar) / Zhat
 *   cert[6]: log Zhat, D_Z / Zhat, D_N / Zhat, V'_max, the bound
 *            3 (D_N + V'_max D_Z) / Zhat (+inf unless D_Z <= Zhat / 3), and
 *            the structural form 3 (1 - p_S) max_g e^{r_g} (2 V' (e^{r_g} - 1)
 *            + rho_g). */
int ora_cluster_estimate(int64_t nk, int32_t d, const double* q, const double* kp,
                         const double* vp, int32_t m, const double* kbar, const double* vbar,
                         const int32_t* cnt, const float* R, const float* rho,
                         float vmax_kept, double scale, double* out, double* cert) {
  if (d <= 0 || m < 0 || nk < 0) return ORA_EINVAL;
  double* l = (double*)malloc(sizeof(double) * (size_t)(nk + m + 1));
  if (!l) return ORA_ENOMEM;
  double mx = -INFINITY;
  for (int64_t i = 0; i < nk; ++i) {
    double s = 0.0;
    for (int32_t t = 0; t < d; ++t) s += q[t] * kp[(size_t)i * d + t];
    l[i] = scale * s;
    if (l[i] > mx) mx = l[i];
  }
  for (int32_t g = 0; g < m; ++g) {
    double s = 0.0;
    for (int32_t t = 0; t < d; ++t) s += q[t] * kbar[(size_t)g * d + t];
    l[nk + g] = cnt[g] > 0 ? scale * s + log((double)cnt[g]) : -INFINITY;
    if (l[nk + g] > mx) mx = l[nk + g];
  }
  double Zs = 0.0, Z = 0.0;
  for (int32_t t = 0; t < d; ++t) out[t] = 0.0;
  for (int64_t i = 0; i < nk + m; ++i) {
    if (l[i] == -INFINITY) continue;
    const double w = exp(l[i] - mx);
    Z += w;
    if (i < nk) Zs += w;
    const double* vi = i < nk ? vp + (size_t)i * d : vbar + (size_t)(i - nk) * d;
    for (int32_t t = 0; t < d; ++t) out[t] += w * vi[t];
  }
  for (int32_t t = 0; t < d; ++t) out[t] /= Z;
  double qn = 0.0;
  for (int32_t t = 0; t < d; ++t) qn += q[t] * q[t];
  qn = sqrt(qn);
  double dz = 0.0, dn = 0.0, vmax = (double)vmax_kept, smax = 0.0;
  for (int32_t g = 0; g < m; ++g) {
    if (cnt[g] <= 0) continue;
    double vb = 0.0;
    for (int32_t t = 0; t < d; ++t) vb += vbar[(size_t)g * d + t] * vbar[(size_t)g * d + t];
    vb = sqrt(vb);
    if (vb + (double)rho[g] > vmax) vmax = vb + (double)rho[g];
  }
  for (int32_t g = 0; g < m; ++g) {
    if (cnt[g] <= 0) continue;
    double vb = 0.0;
    for (int32_t t = 0; t < d; ++t) vb += vbar[(size_t)g * d + t] * vbar[(size_t)g * d + t];
    vb = sqrt(vb);
    const double r = scale * qn * (double)R[g];
    const double zg = exp(l[nk + g] - mx) / Z; /* Zhat_g / Zhat */
    const double er = exp(r);
    dz += (er - 1.0) * er * zg;
    dn += er * zg * ((er - 1.0) * vb + (double)rho[g]);
    const double sf = er * (2.0 * vmax * (er - 1.0) + (double)rho[g]);
    if (sf > smax) smax = sf;
  }
  cert[0] = mx + log(Z);
  cert[1] = dz;
  cert[2] = dn;
  cert[3] = vmax;
  cert[4] = dz <= 1.0 / 3.0 ? 3.0 * (dn + vmax * dz) : INFINITY;
  cert[5] = dz <= 1.0 / 3.0 ? 3.0 * (1.0 - Zs / Z) * smax : INFINITY;
  free(l);
  return ORA_OK;
}
