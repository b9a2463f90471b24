/*
 * confidence_oracle.c -- plain, slow CPU oracle of ActKV's confidence-driven budget
 * allocation (Sec. 6.1 confidence monitor; Alg. 2).
 *
 * TEST INFRASTRUCTURE ONLY, like actkv_oracle.c: only the tests, the package's smoke check
 * and the benchmark's CPU-baseline leg use it, and it shares nothing with the HIP library.
 * Built with -ffp-contract=off: every floating-point operation below is rounded on its own.
 *
 *   token confidence  T = -(1/k) sum_{j<=k} log P(j), P = softmax of one row of logits and
 *                     P(j) its j-th largest probability.  With log P(j) = x_(j) - LSE(x),
 *                     T = LSE(x) - (1/k) sum_{j<=k} x_(j), x_(j) the j-th largest logit.
 *                     fp64 throughout; k larger than the vocabulary takes the whole row.
 *   trace confidence  R'_m = min_{i in [m s, m s + w)} T_i, m = 0 .. floor((n - w) / s) (the
 *                     paper's 1-based windows, 0-based); R = the R'_m with R'_m <= Q_b(R'),
 *                     kept in window order.  Q_b is the b-th percentile by linear
 *                     interpolation between order statistics: pos = (b / 100) (M - 1),
 *                     Q = v_lo + (pos - lo) (v_lo+1 - v_lo), v sorted ascending.
 *   trend             alpha = the least-squares slope of R'_m against m over the retained
 *                     windows: means first, then sum (m - mean m)(R'_m - mean R') over
 *                     sum (m - mean m)^2, every sum in window order, fp64.  Fewer than two
 *                     retained windows (or fewer than w token confidences): alpha = 0.
 *   budget            B' = min(floor(B * scale_up), B_upper) when alpha < 0, else B
 *                     (Alg. 2 step 4; the call is made when compression triggers).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static int cmp_desc(const void* a, const void* b) {
  const double x = *(const double*)a, y = *(const double*)b;
  return x < y ? 1 : (x > y ? -1 : 0);
}

static int cmp_asc(const void* a, const void* b) {
  const double x = *(const double*)a, y = *(const double*)b;
  return x < y ? -1 : (x > y ? 1 : 0);
}

/* out[r] = T of row r of logits ([rows][row_stride] floats, the first `vocab` used). */
int actkv_oracle_token_confidence(const float* logits, int64_t rows, int64_t vocab,
                                  int64_t row_stride, int32_t k, double* out) {
  if (!logits || !out || rows < 0 || vocab <= 0 || row_stride < vocab || k <= 0) return -1;
  const int64_t kk = k < vocab ? k : vocab;
  double* x = (double*)malloc(sizeof(double) * (size_t)vocab);
  if (!x) return -1;
  for (int64_t r = 0; r < rows; ++r) {
    const float* row = logits + r * row_stride;
    double m = -INFINITY;
    for (int64_t v = 0; v < vocab; ++v) {
      x[v] = (double)row[v];
      m = x[v] > m ? x[v] : m;
    }
    double s = 0.0;
    for (int64_t v = 0; v < vocab; ++v) s += exp(x[v] - m);
    const double lse = m + log(s);
    qsort(x, (size_t)vocab, sizeof(double), cmp_desc);
    double top = 0.0;
    for (int64_t j = 0; j < kk; ++j) top += x[j];
    out[r] = lse - top / (double)kk;
  }
  free(x);
  return 0;
}

/*
 * Per request r, conf[offsets[r] .. offsets[r + 1]) is its token-confidence sequence TL.
 * Writes budgets_out[r], slopes[r] (alpha), and when not NULL thresholds[r] (Q_b, NaN with no
 * window) and retained[r] (|R|).
 */
int actkv_oracle_budget_update(const float* conf, const int64_t* offsets, int32_t num_reqs,
                               int32_t window, int32_t stride, double bottom_pct,
                               double scale_up, int32_t budget_upper, const int32_t* budgets_in,
                               int32_t* budgets_out, double* slopes, double* thresholds,
                               int32_t* retained) {
  if (num_reqs < 0 || window <= 0 || stride <= 0 || !(bottom_pct >= 0.0 && bottom_pct <= 100.0) ||
      !(scale_up >= 1.0) || budget_upper < 0 || !offsets || !budgets_in || !budgets_out || !slopes)
    return -1;
  for (int r = 0; r < num_reqs; ++r) {
    const int64_t n = offsets[r + 1] - offsets[r];
    const float* t = conf + offsets[r];
    double alpha = 0.0, q = NAN;
    int32_t kept = 0;
    if (n >= window) {
      /* Step 2: trace-level confidence */
      const int64_t M = (n - window) / stride + 1;
      double* rp = (double*)malloc(sizeof(double) * (size_t)M);
      double* sorted = (double*)malloc(sizeof(double) * (size_t)M);
      for (int64_t m = 0; m < M; ++m) {
        double v = (double)t[m * stride];
        for (int64_t i = m * stride + 1; i < m * stride + window; ++i)
          v = (double)t[i] < v ? (double)t[i] : v;
        rp[m] = v;
        sorted[m] = v;
      }
      qsort(sorted, (size_t)M, sizeof(double), cmp_asc);
      const double pos = (bottom_pct / 100.0) * (double)(M - 1);
      const int64_t lo = (int64_t)floor(pos);
      const double frac = pos - (double)lo;
      q = lo + 1 < M ? sorted[lo] + frac * (sorted[lo + 1] - sorted[lo]) : sorted[lo];
      /* Step 3: least-squares slope over the retained windows, in window order */
      double sx = 0.0, sy = 0.0;
      for (int64_t m = 0; m < M; ++m)
        if (rp[m] <= q) {
          sx += (double)m;
          sy += rp[m];
          ++kept;
        }
      if (kept >= 2) {
        const double mx = sx / (double)kept, my = sy / (double)kept;
        double num = 0.0, den = 0.0;
        for (int64_t m = 0; m < M; ++m)
          if (rp[m] <= q) {
            const double dx = (double)m - mx, dy = rp[m] - my;
            num += dx * dy;
            den += dx * dx;
          }
        alpha = num / den;
      }
      free(rp);
      free(sorted);
    }
    /* Step 4: budget */
    int32_t b = budgets_in[r];
    if (alpha < 0.0) {
      const double grown = floor((double)b * scale_up);
      b = grown < (double)budget_upper ? (int32_t)grown : budget_upper;
    }
    budgets_out[r] = b;
    slopes[r] = alpha;
    if (thresholds) thresholds[r] = q;
    if (retained) retained[r] = kept;
  }
  return 0;
}
