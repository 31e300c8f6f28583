/*
 * SGD-KV CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 implementation of what the SGD-KV hot path computes
 * (Liu et al., "SGD-KV: Summarization Guided KV Cache Compression"):
 *   - head budget allocation (Sec. 3.3, Eq. 2; Appendix A.1, Algorithm 1;
 *     GQA score reduction by max, Appendix A.7),
 *   - SnapKV-style token selection inside each budget (Sec. 3.3 last
 *     paragraph; Sec. 5, "Query-Aware" observation window),
 *   - the per-KV-head compressed cache (Appendix A.2, allocation before the
 *     KV heads are repeated) and decode attention over it.
 *
 * Only the test suite, the smoke entry point and the benchmark's CPU-baseline
 * leg may load this library. The GPU product path never calls it and shares
 * no code, header, table or helper with it.
 *
 * Every routine follows the definition directly: logits are materialised one
 * row at a time, top-k is a full stable sort, decode is a direct loop. All
 * arithmetic is fp64 from exact copies of the inputs. Compile with
 * -ffp-contract=off so that the allocation arithmetic (which decides integers)
 * happens in exactly the order written here.
 *
 * Where the paper is silent or garbled, the readings used are:
 *   - the ABI takes an integer total budget over all kept rows (sink, window
 *     and middle of every head);
 *   - shares are integerised by largest remainder (ties: larger raw score,
 *     then lower flat index) before Algorithm 1's cap and redistribution;
 *   - the cap of Algorithm 1 is applied to the middle part m_h against M;
 *   - redistribution (mode 0) is a greedy fill in descending score order;
 *     mode 1 is the classic proportional water level;
 *   - window-row softmax is causal over keys 0..C-w+i; only keys 0..C-w-1
 *     are scored; the G query heads of a group are averaged;
 *   - scores are average-pooled with an odd kernel, stride 1, zero padding,
 *     divisor always the kernel size;
 *   - top-k ties go to the lower position.
 * End-to-end results are "parity unpinned" against the paper (it prints no
 * numeric worked example of the hot path); each step is pinned by the tests
 * under tests/ against closed forms, invariants and brute force.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_INVALID 1

/* ------------------------------------------------------------------ */
/* GQA reduction of per-query-head summarization scores (Appendix A.7):
 * one score per KV head, the maximum over the G query heads of its group.
 * Query head q belongs to KV head q / G. Layout [L][Hq] -> [L][Hkv].     */
int orc_reduce_group_max(const double* per_q, int L, int Hq, int Hkv, double* out) {
  if (L < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0) return ORC_INVALID;
  int G = Hq / Hkv;
  for (int l = 0; l < L; ++l)
    for (int h = 0; h < Hkv; ++h) {
      double m = per_q[(int64_t)l * Hq + (int64_t)h * G];
      for (int g = 1; g < G; ++g) {
        double v = per_q[(int64_t)l * Hq + (int64_t)h * G + g];
        if (v > m) m = v;
      }
      out[(int64_t)l * Hkv + h] = m;
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Total budget from a ratio R.
 * of_middle = 1: Eq. 2 summed over all heads, R applied to the middle only:
 *                L*H*(s+W) + floor(R*L*H*M).
 * of_middle = 0: R of all rows, floor(R*L*H*C) ("reduce KV memory by up to
 *                75%" at R = 25%).                                         */
int orc_total_from_ratio(double R, int L, int H, int64_t C, int64_t s, int64_t W,
                         int of_middle, int64_t* total) {
  if (!(R >= 0.0 && R <= 1.0) || L < 1 || H < 1 || C < 1 || s < 0 || W < 0 || s + W > C)
    return ORC_INVALID;
  double LH = (double)L * (double)H;
  if (of_middle) {
    int64_t M = C - s - W;
    *total = (int64_t)L * H * (s + W) + (int64_t)floor(R * LH * (double)M);
  } else {
    int64_t t = (int64_t)floor(R * LH * (double)C);
    if (t < (int64_t)L * H * (s + W)) return ORC_INVALID; /* cannot cover sink + window */
    *total = t;
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Budget allocation (Sec. 3.3, Eq. 2 and Appendix A.1, Algorithm 1).
 *
 * sigma[L*H]  raw per-KV-head summarization scores, layer-major, >= 0.
 * Normalisation S_h = sigma_h / sum(sigma) over all L*H heads (Sec. 3.3).
 * Eq. 2 without the reserved rows gives the middle share
 *   x_h = S_h * L*H*R*M = S_h * T,  T = total - L*H*(s+W),
 * computed as (sigma_h / sum(sigma)) * T: the normalised score first, so no
 * intermediate exceeds T whatever the scale of the raw scores.
 * mode 0: integerise, cap every m_h at M, give the excess to the remaining
 *         heads in descending score order, each up to M (Algorithm 1).
 * mode 1: x_h = min(lambda*sigma_h, M) with the exact water level lambda,
 *         then integerise.
 * budgets[h] = s + W + m_h.                                                 */

typedef struct {
  double frac;
  double sigma;
  int64_t idx;
} orc_rank_t;

/* order: frac descending, then sigma descending, then index ascending */
static int orc_cmp_rank(const void* pa, const void* pb) {
  const orc_rank_t* a = (const orc_rank_t*)pa;
  const orc_rank_t* b = (const orc_rank_t*)pb;
  if (a->frac > b->frac) return -1;
  if (a->frac < b->frac) return 1;
  if (a->sigma > b->sigma) return -1;
  if (a->sigma < b->sigma) return 1;
  return (a->idx < b->idx) ? -1 : (a->idx > b->idx);
}

/* Largest-remainder rounding of real shares x[n] (sum = T) to integers m[n]. */
static void orc_integerise(const double* x, const double* sigma, int64_t n, int64_t T, int64_t* m) {
  orc_rank_t* r = (orc_rank_t*)malloc(sizeof(orc_rank_t) * (size_t)n);
  int64_t sum_floor = 0, n_frac = 0;
  for (int64_t h = 0; h < n; ++h) {
    double f = floor(x[h]);
    m[h] = (int64_t)f;
    sum_floor += m[h];
    r[h].frac = x[h] - f;
    r[h].sigma = sigma[h];
    r[h].idx = h;
    if (r[h].frac > 0.0) ++n_frac;
  }
  qsort(r, (size_t)n, sizeof(orc_rank_t), orc_cmp_rank);
  int64_t rem = T - sum_floor;
  /* fp residue guard: hand out at most one unit per fractional head first,
   * then round-robin in the same order (never taken on well-posed inputs). */
  int64_t first = rem < 0 ? 0 : (rem < n_frac ? rem : n_frac);
  for (int64_t k = 0; k < first; ++k) m[r[k].idx] += 1;
  rem -= first;
  for (int64_t k = 0; rem > 0; k = (k + 1) % n, --rem) m[r[k].idx] += 1;
  for (int64_t k = 0; rem < 0; k = (k + 1) % n) {
    int64_t h = r[n - 1 - k].idx;
    if (m[h] > 0) { m[h] -= 1; ++rem; }
  }
  free(r);
}

typedef struct {
  double sigma;
  int64_t idx;
} orc_head_t;

/* sigma descending, index ascending */
static int orc_cmp_head(const void* pa, const void* pb) {
  const orc_head_t* a = (const orc_head_t*)pa;
  const orc_head_t* b = (const orc_head_t*)pb;
  if (a->sigma > b->sigma) return -1;
  if (a->sigma < b->sigma) return 1;
  return (a->idx < b->idx) ? -1 : (a->idx > b->idx);
}

int orc_allocate_budgets(const double* sigma, int L, int H, int64_t C, int64_t s, int64_t W,
                         int64_t total, int mode, int64_t* budgets) {
  if (L < 1 || H < 1 || C < 1 || s < 0 || W < 0 || s + W > C) return ORC_INVALID;
  if (mode != 0 && mode != 1) return ORC_INVALID;
  int64_t n = (int64_t)L * H;
  int64_t M = C - s - W;
  if (total < n * (s + W) || total > n * C) return ORC_INVALID;
  double sum = 0.0;
  for (int64_t h = 0; h < n; ++h) {
    if (!(sigma[h] >= 0.0) || isinf(sigma[h])) return ORC_INVALID;
    sum += sigma[h];
  }
  if (isinf(sum)) return ORC_INVALID;
  int64_t T = total - n * (s + W); /* rows to hand out over the middles */

  double* x = (double*)malloc(sizeof(double) * (size_t)n);
  int64_t* m = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
  double* sg = (double*)malloc(sizeof(double) * (size_t)n);
  for (int64_t h = 0; h < n; ++h) sg[h] = (sum > 0.0) ? sigma[h] : 1.0; /* all-zero -> uniform */
  double sgsum = (sum > 0.0) ? sum : (double)n;

  if (mode == 0) {
    /* Eq. 2 shares, integerised */
    for (int64_t h = 0; h < n; ++h) x[h] = (sg[h] / sgsum) * (double)T;
    orc_integerise(x, sg, n, T, m);
    /* Algorithm 1: excess over the cap, cap, greedy redistribution */
    int64_t E = 0;
    for (int64_t h = 0; h < n; ++h)
      if (m[h] > M) { E += m[h] - M; m[h] = M; }
    orc_head_t* order = (orc_head_t*)malloc(sizeof(orc_head_t) * (size_t)n);
    for (int64_t h = 0; h < n; ++h) { order[h].sigma = sg[h]; order[h].idx = h; }
    qsort(order, (size_t)n, sizeof(orc_head_t), orc_cmp_head);
    for (int64_t k = 0; k < n && E > 0; ++k) {
      int64_t h = order[k].idx;
      int64_t room = M - m[h];
      if (room <= 0) continue;
      int64_t give = room < E ? room : E;
      m[h] += give;
      E -= give;
    }
    free(order);
  } else {
    /* Proportional water level: x_h = min(lambda*sigma_h, M), sum x_h = T.
     * Heads sorted by sigma descending; the first c are capped at M. Take
     * the smallest c with lambda_c*sigma_(c) <= M, where
     * lambda_c = (T - c*M) / (sum of the sigmas not capped).
     * lambda*sigma_h is evaluated as (sigma_h / rest) * left, a fraction of
     * at most 1 times the rows left, so tiny scores cannot overflow it.
     * If every uncapped head has sigma 0, the rows left after the capped
     * heads are split evenly over those heads (a flat water level).       */
    orc_head_t* order = (orc_head_t*)malloc(sizeof(orc_head_t) * (size_t)n);
    for (int64_t h = 0; h < n; ++h) { order[h].sigma = sg[h]; order[h].idx = h; }
    qsort(order, (size_t)n, sizeof(orc_head_t), orc_cmp_head);
    /* sums of sigma over sorted positions k..n-1, added from the smallest */
    double* rest = (double*)malloc(sizeof(double) * (size_t)(n + 1));
    rest[n] = 0.0;
    for (int64_t k = n - 1; k >= 0; --k) rest[k] = rest[k + 1] + order[k].sigma;
    int64_t c = 0;
    double lambda = 0.0;
    int flat = 0;
    double left = (double)T;
    for (c = 0; c < n; ++c) {
      left = (double)T - (double)c * (double)M;
      if (rest[c] <= 0.0) { flat = 1; lambda = left / (double)(n - c); break; }
      if ((order[c].sigma / rest[c]) * left <= (double)M) break;
    }
    for (int64_t k = 0; k < n; ++k) {
      int64_t h = order[k].idx;
      double v = (k < c) ? (double)M : (flat ? lambda : (order[k].sigma / rest[c]) * left);
      x[h] = v > (double)M ? (double)M : v;
    }
    orc_integerise(x, sg, n, T, m);
    /* rounding cannot lift a head above M unless fp residue did; move any
     * such surplus to the next heads in score order */
    int64_t E = 0;
    for (int64_t h = 0; h < n; ++h)
      if (m[h] > M) { E += m[h] - M; m[h] = M; }
    for (int64_t k = 0; k < n && E > 0; ++k) {
      int64_t h = order[k].idx;
      int64_t room = M - m[h];
      int64_t give = room < E ? room : E;
      if (give > 0) { m[h] += give; E -= give; }
    }
    free(rest);
    free(order);
  }
  for (int64_t h = 0; h < n; ++h) budgets[h] = s + W + m[h];
  free(x);
  free(m);
  free(sg);
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Allocation variants of the head-configuration ablation (Appendix A.7,
 * Table 5):
 *   0 PLAIN           orc_allocate_budgets.
 *   1 THR             scores below the mean of all L*H scores become 0 before
 *                     the allocation ("SGD-KV (thr)").
 *   2 REVERSE         the allocation is inverted head by head: a head that
 *                     keeps m_h of its M middle rows keeps M - m_h instead
 *                     ("SGD-KV (Reverse)": 10 % becomes 90 %). The total is
 *                     then L*H*(C + s + W) - total.
 *   3 MIX             the scores are the average of the normalised
 *                     summarization scores and a second normalised score
 *                     vector sigma2 ("SGD-KV + HeadKV" with R2 scores); an
 *                     all-zero vector normalises to uniform.
 *   4 BINARY          the floor(f*n) heads first in (score descending, index
 *                     ascending) order keep all C rows, the others only
 *                     s + W ("DuoAttention (Sum.)"); total is not used.
 *   5 BINARY_REVERSE  the floor(f*n) heads last in that order keep all rows
 *                     ("DuoAttention (Sum., Reverse)", f = 0.75).          */
int orc_allocate_variant(const double* sigma, const double* sigma2, int L, int H, int64_t C, int64_t s,
                         int64_t W, int64_t total, int mode, int variant, double f, int64_t* budgets) {
  if (L < 1 || H < 1 || C < 1 || s < 0 || W < 0 || s + W > C) return ORC_INVALID;
  int64_t n = (int64_t)L * H;
  int64_t M = C - s - W;
  for (int64_t h = 0; h < n; ++h)
    if (!(sigma[h] >= 0.0) || isinf(sigma[h])) return ORC_INVALID;
  if (variant == 0) return orc_allocate_budgets(sigma, L, H, C, s, W, total, mode, budgets);
  if (variant == 1) {
    double sum = 0.0;
    for (int64_t h = 0; h < n; ++h) sum += sigma[h];
    double mean = sum / (double)n;
    double* t = (double*)malloc(sizeof(double) * (size_t)n);
    for (int64_t h = 0; h < n; ++h) t[h] = sigma[h] < mean ? 0.0 : sigma[h];
    int rc = orc_allocate_budgets(t, L, H, C, s, W, total, mode, budgets);
    free(t);
    return rc;
  }
  if (variant == 2) {
    int rc = orc_allocate_budgets(sigma, L, H, C, s, W, total, mode, budgets);
    if (rc != ORC_OK) return rc;
    for (int64_t h = 0; h < n; ++h) budgets[h] = s + W + (M - (budgets[h] - s - W));
    return ORC_OK;
  }
  if (variant == 3) {
    if (!sigma2) return ORC_INVALID;
    double s1 = 0.0, s2 = 0.0;
    for (int64_t h = 0; h < n; ++h) {
      if (!(sigma2[h] >= 0.0) || isinf(sigma2[h])) return ORC_INVALID;
      s1 += sigma[h];
      s2 += sigma2[h];
    }
    if (isinf(s1) || isinf(s2)) return ORC_INVALID;
    double* t = (double*)malloc(sizeof(double) * (size_t)n);
    for (int64_t h = 0; h < n; ++h) {
      double a = s1 > 0.0 ? sigma[h] / s1 : 1.0 / (double)n;
      double b = s2 > 0.0 ? sigma2[h] / s2 : 1.0 / (double)n;
      t[h] = (a + b) / 2.0;
    }
    int rc = orc_allocate_budgets(t, L, H, C, s, W, total, mode, budgets);
    free(t);
    return rc;
  }
  if (variant == 4 || variant == 5) {
    if (!(f >= 0.0 && f <= 1.0)) return ORC_INVALID;
    int64_t k = (int64_t)floor(f * (double)n);
    orc_head_t* order = (orc_head_t*)malloc(sizeof(orc_head_t) * (size_t)n);
    for (int64_t h = 0; h < n; ++h) { order[h].sigma = sigma[h]; order[h].idx = h; }
    qsort(order, (size_t)n, sizeof(orc_head_t), orc_cmp_head);
    for (int64_t h = 0; h < n; ++h) budgets[h] = s + W;
    for (int64_t j = 0; j < k; ++j) budgets[order[variant == 4 ? j : n - 1 - j].idx] = C;
    free(order);
    return ORC_OK;
  }
  return ORC_INVALID;
}

/* ------------------------------------------------------------------ */
/* Observation-window attention (Sec. 3.3 last paragraph, Sec. 5).
 * Window row i of query head q sits at position win0+i and attends causally
 * to the cached keys 0..min(win0+i, C-1):  l_ij = scale * <q_i, k_j>.
 * lse[b,q,i] = log sum_{j <= min(win0+i, C-1)} exp(l_ij).
 * win0 = C-w: the last w prompt tokens (Query-Aware, the default);
 * win0 < C-w: a window before the final question (Query-Unaware);
 * win0 = C:   rows after the prompt that see every cached key (Proxy-Query);
 * the softmax runs over cached keys only.
 * Layouts: q_win [B][Hq][w][d], k [B][Hkv][C][d].                          */
static double orc_dot(const double* a, const double* b, int d) {
  double s = 0.0;
  for (int t = 0; t < d; ++t) s += a[t] * b[t];
  return s;
}

int orc_window_lse(const double* q_win, const double* k, int B, int Hq, int Hkv, int d, int64_t C,
                   int w, int64_t win0, double scale, double* lse) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || d < 1 || w < 1 || win0 < 0 || win0 > C) return ORC_INVALID;
  int G = Hq / Hkv;
  int64_t rows = (int64_t)B * Hq * w;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < rows; ++r) {
    int64_t i = r % w, q = (r / w) % Hq, b = r / ((int64_t)w * Hq);
    int64_t h = q / G;
    const double* qi = q_win + r * d;
    const double* kb = k + ((int64_t)b * Hkv + h) * C * d;
    int64_t last = win0 + i; /* causal: keys 0..last that the cache holds */
    if (last > C - 1) last = C - 1;
    double mx = -INFINITY;
    for (int64_t j = 0; j <= last; ++j) {
      double l = scale * orc_dot(qi, kb + j * d, d);
      if (l > mx) mx = l;
    }
    double z = 0.0;
    for (int64_t j = 0; j <= last; ++j) z += exp(scale * orc_dot(qi, kb + j * d, d) - mx);
    lse[r] = mx + log(z);
  }
  return ORC_OK;
}

/* Cumulative window attention per scored key, averaged over the group:
 *   a[b,h,j] = (1/G) sum_{q in group h} sum_{i<w} exp(l_{q,i,j} - lse[b,q,i]),
 * for the scored keys j in [0, win0) (every window row sees all of them).
 * Output layout [B][Hkv][win0].                                            */
int orc_window_colsum(const double* q_win, const double* k, const double* lse, int B, int Hq,
                      int Hkv, int d, int64_t C, int w, int64_t win0, double scale, double* colsum) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || d < 1 || w < 1 || win0 < 0 || win0 > C) return ORC_INVALID;
  int G = Hq / Hkv;
  int64_t n = win0;
  int64_t cols = (int64_t)B * Hkv * n;
#pragma omp parallel for schedule(static)
  for (int64_t c = 0; c < cols; ++c) {
    int64_t j = c % n, h = (c / n) % Hkv, b = c / (n * Hkv);
    const double* kj = k + (((int64_t)b * Hkv + h) * C + j) * d;
    double acc = 0.0;
    for (int g = 0; g < G; ++g) {
      int64_t q = h * G + g;
      for (int i = 0; i < w; ++i) {
        int64_t r = ((int64_t)b * Hq + q) * w + i;
        acc += exp(scale * orc_dot(q_win + r * d, kj, d) - lse[r]);
      }
    }
    colsum[c] = acc / (double)G;
  }
  return ORC_OK;
}

/* Importance-weighted group aggregation (Appendix A.7, "Ipt." rows of
 * Table 5). With A_g[j] = sum_{i<w} exp(l_{q,i,j} - lse[b,q,i]) the window
 * attention of query head q = h*G + g and sigma_q its summarization score
 * (qscore[Hq], the same for every sequence):
 *   agg 1 (Ipt., max):  a_j = max_g sigma_q * A_g[j]
 *   agg 2 (Ipt., mean): a_j = (1/G) sum_g sigma_q * A_g[j]
 *   agg 3 (Ipt., only): a_j = A_{g*}[j], g* the group's head with the largest
 *                       sigma (ties: lower g); every head inherits its scores.
 * agg 0 is the plain group mean (orc_window_colsum). Output [B][Hkv][win0]. */
int orc_window_colsum_ipt(const double* q_win, const double* k, const double* lse, int B, int Hq,
                          int Hkv, int d, int64_t C, int w, int64_t win0, double scale, const double* qscore,
                          int agg, double* colsum) {
  if (agg == 0) return orc_window_colsum(q_win, k, lse, B, Hq, Hkv, d, C, w, win0, scale, colsum);
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || d < 1 || w < 1 || win0 < 0 || win0 > C || agg < 1 || agg > 3 ||
      !qscore)
    return ORC_INVALID;
  for (int q = 0; q < Hq; ++q)
    if (!(qscore[q] >= 0.0) || isinf(qscore[q])) return ORC_INVALID;
  int G = Hq / Hkv;
  int64_t n = win0;
  int64_t cols = (int64_t)B * Hkv * n;
#pragma omp parallel for schedule(static)
  for (int64_t c = 0; c < cols; ++c) {
    int64_t j = c % n, h = (c / n) % Hkv, b = c / (n * Hkv);
    const double* kj = k + (((int64_t)b * Hkv + h) * C + j) * d;
    int gstar = 0;
    for (int g = 1; g < G; ++g)
      if (qscore[h * G + g] > qscore[h * G + gstar]) gstar = g;
    double out = 0.0;
    for (int g = 0; g < G; ++g) {
      if (agg == 3 && g != gstar) continue;
      int64_t q = h * G + g;
      double A = 0.0;
      for (int i = 0; i < w; ++i) {
        int64_t r = ((int64_t)b * Hq + q) * w + i;
        A += exp(scale * orc_dot(q_win + r * d, kj, d) - lse[r]);
      }
      if (agg == 1) {
        double v = qscore[q] * A;
        out = (g == 0 || v > out) ? v : out;
      } else if (agg == 2) {
        out += qscore[q] * A;
      } else {
        out = A;
      }
    }
    colsum[c] = agg == 2 ? out / (double)G : out;
  }
  return ORC_OK;
}

/* 1-D average pooling along the key axis: odd kernel kp, stride 1, zero
 * padding of r = (kp-1)/2 on both ends, divisor always kp.
 * a and pooled are [rows][n].                                              */
int orc_pool(const double* a, int64_t rows, int64_t n, int kp, double* pooled) {
  if (rows < 0 || n < 0 || kp < 1 || kp % 2 == 0) return ORC_INVALID;
  int64_t r = (kp - 1) / 2;
  for (int64_t row = 0; row < rows; ++row)
    for (int64_t j = 0; j < n; ++j) {
      double s = 0.0;
      for (int64_t t = j - r; t <= j + r; ++t)
        if (t >= 0 && t < n) s += a[row * n + t];
      pooled[row * n + j] = s / (double)kp;
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Token selection inside one head's budget (Sec. 3.3, SnapKV-style).
 * Candidates are the middle positions j in [s, C-W); the m candidates with
 * the largest pooled score are kept, ties to the lower position (a full
 * stable sort by (score desc, position asc)). The kept list is the sink
 * [0,s), the selected positions and the recent window [C-W, C), ascending.
 * pooled holds the scores of positions [0, C-w); W >= w so every candidate
 * has a score. kept receives s + m + W positions.                          */
typedef struct {
  double v;
  int64_t j;
} orc_cand_t;

static int orc_cmp_cand(const void* pa, const void* pb) {
  const orc_cand_t* a = (const orc_cand_t*)pa;
  const orc_cand_t* b = (const orc_cand_t*)pb;
  if (a->v > b->v) return -1;
  if (a->v < b->v) return 1;
  return (a->j < b->j) ? -1 : (a->j > b->j);
}

static int orc_cmp_i32(const void* pa, const void* pb) {
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  return (a > b) - (a < b);
}

int orc_select(const double* pooled, int64_t C, int64_t n_scored, int64_t s, int64_t W, int64_t m,
               int32_t* kept) {
  /* every candidate in [s, C-W) needs a score: C - W <= n_scored */
  if (n_scored < 0 || s < 0 || C - W > n_scored || s + W > C || m < 0 || m > C - s - W) return ORC_INVALID;
  int64_t M = C - s - W;
  orc_cand_t* cand = (orc_cand_t*)malloc(sizeof(orc_cand_t) * (size_t)(M > 0 ? M : 1));
  for (int64_t t = 0; t < M; ++t) { cand[t].j = s + t; cand[t].v = pooled[s + t]; }
  qsort(cand, (size_t)M, sizeof(orc_cand_t), orc_cmp_cand);
  int64_t o = 0;
  for (int64_t j = 0; j < s; ++j) kept[o++] = (int32_t)j;
  for (int64_t t = 0; t < m; ++t) kept[o++] = (int32_t)cand[t].j;
  for (int64_t j = C - W; j < C; ++j) kept[o++] = (int32_t)j;
  qsort(kept, (size_t)o, sizeof(int32_t), orc_cmp_i32);
  free(cand);
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Decode attention over the compressed per-KV-head cache (the cache is
 * allocated before the KV heads are repeated, Appendix A.2).
 * Query head q of sequence b attends to the rows of segment (b, q/G):
 * rows offsets[b*Hkv+h] .. offsets[b*Hkv+h+1]-1 of kc/vc ([rows][d]).
 *   out = sum_r softmax_r(scale*<q,k_r>) v_r,  lse = log sum_r exp(...).
 * An empty segment gives out = 0, lse = -inf.  q/out: [B][Hq][d].          */
int orc_decode(const double* q, const double* kc, const double* vc, const int64_t* offsets, int B,
               int Hq, int Hkv, int d, double scale, double* out, double* lse) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || d < 1) return ORC_INVALID;
  int G = Hq / Hkv;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t bq = 0; bq < (int64_t)B * Hq; ++bq) {
    int64_t b = bq / Hq, qh = bq % Hq, h = qh / G;
    int64_t r0 = offsets[b * Hkv + h], r1 = offsets[b * Hkv + h + 1];
    const double* qv = q + bq * d;
    double* o = out + bq * d;
    for (int t = 0; t < d; ++t) o[t] = 0.0;
    if (r1 <= r0) { lse[bq] = -INFINITY; continue; }
    double mx = -INFINITY;
    for (int64_t r = r0; r < r1; ++r) {
      double l = scale * orc_dot(qv, kc + r * d, d);
      if (l > mx) mx = l;
    }
    double z = 0.0;
    for (int64_t r = r0; r < r1; ++r) {
      double p = exp(scale * orc_dot(qv, kc + r * d, d) - mx);
      z += p;
      for (int t = 0; t < d; ++t) o[t] += p * vc[r * d + t];
    }
    for (int t = 0; t < d; ++t) o[t] /= z;
    lse[bq] = mx + log(z);
  }
  return ORC_OK;
}

/* Decode during generation (the step after compression, Appendix A.2 keeps
 * one cache per KV head): each (b, h) also holds the rows appended since the
 * compression, rows 0..n_new-1 of knew/vnew [B][Hkv][cap][d]. Query head q of
 * sequence b attends to its segment's compressed rows followed by those:
 *   out = sum over both sets of softmax(scale*<q,k>) v,  lse as in orc_decode. */
int orc_decode_append(const double* q, const double* kc, const double* vc, const int64_t* offsets,
                      const double* knew, const double* vnew, int64_t cap, int64_t n_new, int B, int Hq,
                      int Hkv, int d, double scale, double* out, double* lse) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || d < 1 || cap < 0 || n_new < 0 || n_new > cap) return ORC_INVALID;
  int G = Hq / Hkv;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t bq = 0; bq < (int64_t)B * Hq; ++bq) {
    int64_t b = bq / Hq, qh = bq % Hq, h = qh / G;
    int64_t r0 = offsets[b * Hkv + h], r1 = offsets[b * Hkv + h + 1];
    const double* kn = knew + ((int64_t)b * Hkv + h) * cap * d;
    const double* vn = vnew + ((int64_t)b * Hkv + h) * cap * d;
    const double* qv = q + bq * d;
    double* o = out + bq * d;
    for (int t = 0; t < d; ++t) o[t] = 0.0;
    int64_t n = (r1 > r0 ? r1 - r0 : 0) + n_new;
    if (n == 0) { lse[bq] = -INFINITY; continue; }
    double mx = -INFINITY;
    for (int64_t e = 0; e < n; ++e) {
      const double* kr = e < r1 - r0 ? kc + (r0 + e) * d : kn + (e - (r1 - r0 > 0 ? r1 - r0 : 0)) * d;
      double l = scale * orc_dot(qv, kr, d);
      if (l > mx) mx = l;
    }
    double z = 0.0;
    for (int64_t e = 0; e < n; ++e) {
      int64_t nc = r1 - r0 > 0 ? r1 - r0 : 0;
      const double* kr = e < nc ? kc + (r0 + e) * d : kn + (e - nc) * d;
      const double* vr = e < nc ? vc + (r0 + e) * d : vn + (e - nc) * d;
      double p = exp(scale * orc_dot(qv, kr, d) - mx);
      z += p;
      for (int t = 0; t < d; ++t) o[t] += p * vr[t];
    }
    for (int t = 0; t < d; ++t) o[t] /= z;
    lse[bq] = mx + log(z);
  }
  return ORC_OK;
}

int orc_num_threads(void) {
#ifdef _OPENMP
  extern int omp_get_max_threads(void);
  return omp_get_max_threads();
#else
  return 1;
#endif
}
