/*
 * actkv_oracle.c -- plain, slow CPU oracle of the ActKV compression step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or calls this file;
 * only the tests, the package's smoke check and the benchmark's CPU-baseline leg do.  It
 * shares no source, header, table or helper with the HIP library: it has its own problem
 * struct, its own bf16 decoding and its own paged addressing.
 *
 * What it computes (ActKV, "Efficient LLM Agents through Action-Guided KV Cache
 * Management"):
 *   scores   -- for every cached entry t of request r and KV head h, the softmax attention
 *               that the action-region queries give it (Sec. 2.3 attention definition;
 *               Sec. 7.1 log-sum-exp and the recovery identity A = exp(s - LSE); Alg. 3).
 *               Aggregation over the query heads of a GQA group and over the action
 *               queries is a SUM, or (Alg. 3 / Sec. 7.1 prose) a max over the group followed
 *               by a mean over the queries.
 *   pool     -- an optional centred 1-D max-pool over token positions (not in the paper;
 *               window 1 means none).
 *   select   -- TopK(score, k = budget) per (request, KV head) (Alg. 1, step 5), ties to
 *               the lower token index, emitted in ascending token order.
 *   lrfu     -- (the eviction policy of Sec. 5.1 / Alg. 1 steps 2-5) a top-p hit mask over the
 *               scores and the attention-aware LRFU keep-score update; selection then
 *               runs on the keep scores.
 *   compact  -- the survivors' K/V rows are written, in ascending token order, into fresh
 *               pages taken from a free list; the block table row is rewritten and the old
 *               pages are returned (the freed-block return of Sec. 7.2);
 *   compact_inplace -- the paper's own in-place compaction (Alg. 4): survivors outside the
 *               last blocks are paired with the evicted slots inside them and copied there.
 *
 * Every floating-point quantity is carried in double (fp64).  The raw per-entry score is
 * rounded once to float at the end; pooling and selection then act on those float values,
 * which is also the precision the selection is decided in on the GPU.
 *
 * Readings where the paper is silent:
 *   - logits are sm_scale * q.k (the paper writes q.k^T with no scale);
 *   - action query j of a request with L cached tokens and n action queries sits at
 *     position L - n + j and, when causal, sees keys t <= L - n + j (itself included);
 *     non-causal queries see all L keys;
 *   - MAX_MEAN with n == 0 queries gives 0.
 *
 * Paged layout (Sec. 2.5): kv is [2][num_pages][page_size][Hkv][D] bf16, K at [0], V at
 * [1]; logical token t of a request lives in physical block bt[t / page_size], slot
 * t % page_size, so its flat slot index is bt[t / page_size] * page_size + t % page_size.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORACLE_AGG_SUM = 0, ORACLE_AGG_MAX_MEAN = 1 };

typedef struct oracle_problem {
  int32_t num_reqs, num_q_heads, num_kv_heads, head_dim, page_size;
  int64_t num_pages;
  int32_t bt_stride;
  const int32_t* seq_lens;   /* [R] */
  const int32_t* q_lens;     /* [R] */
  const int32_t* budgets;    /* [R * Hkv] */
  double sm_scale;
  int32_t pool_window;       /* odd >= 1 */
  int32_t causal;
  int32_t agg;
} oracle_problem;

/* bf16 bit pattern -> value: the 16 bits are the high half of an IEEE float. */
static double bf16_value(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Sec. 2.5 worked example: bt = [17, 9], page_size 2, tokens 0..2 -> slots 34, 35, 18. */
int64_t actkv_oracle_slot(const int32_t* bt_row, int32_t page_size, int64_t t) {
  return (int64_t)bt_row[t / page_size] * page_size + t % page_size;
}

static const uint16_t* kv_row(const oracle_problem* p, const uint16_t* kv, int which,
                              int64_t slot, int h) {
  int64_t plane = p->num_pages * (int64_t)p->page_size;
  return kv + (((int64_t)which * plane + slot) * p->num_kv_heads + h) * p->head_dim;
}

static uint16_t* kv_row_mut(const oracle_problem* p, uint16_t* kv, int which, int64_t slot,
                            int h) {
  int64_t plane = p->num_pages * (int64_t)p->page_size;
  return kv + (((int64_t)which * plane + slot) * p->num_kv_heads + h) * p->head_dim;
}

static int64_t q_offset(const oracle_problem* p, int r) {
  int64_t off = 0;
  for (int i = 0; i < r; ++i) off += p->q_lens[i];
  return off;
}

static int64_t score_offset(const oracle_problem* p, int r) {
  int64_t off = 0;
  for (int i = 0; i < r; ++i) off += (int64_t)p->num_kv_heads * p->seq_lens[i];
  return off;
}

static int64_t kept_offset(const oracle_problem* p, int r, int h) {
  int64_t off = 0;
  for (int i = 0; i < r * p->num_kv_heads + h; ++i) {
    int64_t L = p->seq_lens[i / p->num_kv_heads];
    int64_t b = p->budgets[i];
    off += b < 0 ? 0 : (b > L ? L : b);
  }
  return off;
}

/* Position of action query j (see the readings above); keys t <= position are visible. */
static int64_t last_visible_key(const oracle_problem* p, int r, int j) {
  int64_t L = p->seq_lens[r], n = p->q_lens[r];
  return p->causal ? L - n + j : L - 1;
}

/* s[t] = sm_scale * q . k_t for t = 0..last (Sec. 2.3: q_i K^T, Sec. 7.1: s_ij). */
static void logits_row(const oracle_problem* p, const uint16_t* q_row, const uint16_t* kv,
                       const int32_t* bt_row, int h, int64_t last, double* s) {
  for (int64_t t = 0; t <= last; ++t) {
    const uint16_t* k = kv_row(p, kv, 0, actkv_oracle_slot(bt_row, p->page_size, t), h);
    double dot = 0.0;
    for (int d = 0; d < p->head_dim; ++d) dot += bf16_value(q_row[d]) * bf16_value(k[d]);
    s[t] = p->sm_scale * dot;
  }
}

/* LSE = log sum_t exp(s_t) (Sec. 7.1), evaluated as m + log sum exp(s_t - m). */
static double log_sum_exp(const double* s, int64_t count) {
  double m = -INFINITY;
  for (int64_t t = 0; t < count; ++t) m = s[t] > m ? s[t] : m;
  if (count == 0) return -INFINITY;
  double acc = 0.0;
  for (int64_t t = 0; t < count; ++t) acc += exp(s[t] - m);
  return m + log(acc);
}

static int check_problem(const oracle_problem* p) {
  if (!p || p->num_reqs < 0 || p->num_kv_heads <= 0 || p->num_q_heads <= 0 ||
      p->num_q_heads % p->num_kv_heads || p->head_dim <= 0 || p->page_size <= 0)
    return -1;
  for (int r = 0; r < p->num_reqs; ++r) {
    if (p->seq_lens[r] < 0 || p->q_lens[r] < 0) return -1;
    if (p->causal && p->q_lens[r] > p->seq_lens[r]) return -1;
    if ((p->seq_lens[r] + p->page_size - 1) / p->page_size > p->bt_stride) return -1;
  }
  return 0;
}

/* lse_out[(q_offset(r) + j) * Hq + g] = log sum_{t visible to j} exp(s_t)   (Sec. 7.1). */
int actkv_oracle_lse(const oracle_problem* p, const uint16_t* q, const uint16_t* kv,
                     const int32_t* bt, double* lse_out) {
  if (check_problem(p)) return -1;
  const int Hq = p->num_q_heads, G = p->num_q_heads / p->num_kv_heads, D = p->head_dim;
  for (int r = 0; r < p->num_reqs; ++r) {
    const int64_t qoff = q_offset(p, r);
    const int n = p->q_lens[r];
#pragma omp parallel for schedule(dynamic, 1)
    for (int row = 0; row < n * Hq; ++row) {
      const int j = row / Hq, g = row % Hq;
      const int64_t last = last_visible_key(p, r, j);
      double* s = (double*)malloc(sizeof(double) * (size_t)(last + 1 > 0 ? last + 1 : 1));
      logits_row(p, q + ((qoff + j) * Hq + g) * D, kv, bt + (int64_t)r * p->bt_stride, g / G,
                 last, s);
      lse_out[(qoff + j) * Hq + g] = log_sum_exp(s, last + 1);
      free(s);
    }
  }
  return 0;
}

/*
 * raw_out[score_offset(r) + h * L_r + t]:
 *   SUM:      sum_{g in group(h)} sum_{j : t visible} exp(s_{j,g,t} - LSE_{j,g})
 *   MAX_MEAN: (1/n) sum_{j : t visible} max_{g in group(h)} exp(s_{j,g,t} - LSE_{j,g})
 * LSE is taken from lse_in (float, [sum n][Hq]) when given -- the recovery of Sec. 7.1 --
 * and otherwise computed here from its definition.  Each value is rounded to float once.
 */
int actkv_oracle_scores(const oracle_problem* p, const uint16_t* q, const uint16_t* kv,
                        const int32_t* bt, const float* lse_in, float* raw_out) {
  if (check_problem(p)) return -1;
  const int Hq = p->num_q_heads, Hkv = p->num_kv_heads, G = Hq / Hkv, D = p->head_dim;
#pragma omp parallel for schedule(dynamic, 1)
  for (int rh = 0; rh < p->num_reqs * Hkv; ++rh) {
    const int r = rh / Hkv, h = rh % Hkv;
    const int64_t L = p->seq_lens[r], qoff = q_offset(p, r), soff = score_offset(p, r);
    const int n = p->q_lens[r];
    {
      double* acc = (double*)calloc((size_t)(L > 0 ? L : 1), sizeof(double));
      double* s = (double*)malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
      double* mx = (double*)malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
      for (int j = 0; j < n; ++j) {
        const int64_t last = last_visible_key(p, r, j);
        for (int64_t t = 0; t <= last; ++t) mx[t] = 0.0;
        for (int gi = 0; gi < G; ++gi) {
          const int g = h * G + gi;
          logits_row(p, q + ((qoff + j) * Hq + g) * D, kv, bt + (int64_t)r * p->bt_stride, h,
                     last, s);
          const double lse = lse_in ? (double)lse_in[(qoff + j) * Hq + g]
                                    : log_sum_exp(s, last + 1);
          for (int64_t t = 0; t <= last; ++t) {
            const double a = exp(s[t] - lse);   /* A_{j,t} = exp(s - LSE), Sec. 7.1 */
            if (p->agg == ORACLE_AGG_SUM) acc[t] += a;
            else mx[t] = a > mx[t] ? a : mx[t];
          }
        }
        if (p->agg == ORACLE_AGG_MAX_MEAN)
          for (int64_t t = 0; t <= last; ++t) acc[t] += mx[t];
      }
      for (int64_t t = 0; t < L; ++t) {
        double v = acc[t];
        if (p->agg == ORACLE_AGG_MAX_MEAN) v = n > 0 ? v / n : 0.0;
        raw_out[soff + h * L + t] = (float)v;
      }
      free(acc);
      free(s);
      free(mx);
    }
  }
  return 0;
}

/* pooled[t] = max raw[u] over |u - t| <= w/2, 0 <= u < L, per (request, KV head). */
int actkv_oracle_pool(const oracle_problem* p, const float* raw, float* pooled) {
  if (check_problem(p) || p->pool_window < 1 || p->pool_window % 2 == 0) return -1;
  const int half = p->pool_window / 2;
  for (int r = 0; r < p->num_reqs; ++r) {
    const int64_t L = p->seq_lens[r], soff = score_offset(p, r);
    for (int h = 0; h < p->num_kv_heads; ++h) {
      const float* in = raw + soff + h * L;
      float* out = pooled + soff + h * L;
      for (int64_t t = 0; t < L; ++t) {
        float m = in[t];
        for (int64_t u = t - half; u <= t + half; ++u)
          if (u >= 0 && u < L && in[u] > m) m = in[u];
        out[t] = m;
      }
    }
  }
  return 0;
}

typedef struct { float v; int32_t t; } scored_entry;

/* Descending score, then ascending token index: the order TopK keeps. */
static int by_score_then_index(const void* a, const void* b) {
  const scored_entry* x = (const scored_entry*)a;
  const scored_entry* y = (const scored_entry*)b;
  if (x->v > y->v) return -1;
  if (x->v < y->v) return 1;
  return (x->t > y->t) - (x->t < y->t);
}

static int ascending_int(const void* a, const void* b) {
  int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
  return (x > y) - (x < y);
}

/* kept[kept_offset(r,h) ...] = the min(max(B,0), L) best entries of (r,h), ascending. */
int actkv_oracle_select(const oracle_problem* p, const float* pooled, int32_t* kept) {
  if (check_problem(p)) return -1;
  for (int r = 0; r < p->num_reqs; ++r) {
    const int64_t L = p->seq_lens[r], soff = score_offset(p, r);
    for (int h = 0; h < p->num_kv_heads; ++h) {
      int64_t k = p->budgets[r * p->num_kv_heads + h];
      if (k < 0) return -1;
      if (k > L) k = L;
      scored_entry* e = (scored_entry*)malloc(sizeof(scored_entry) * (size_t)(L > 0 ? L : 1));
      for (int64_t t = 0; t < L; ++t) {
        float v = pooled[soff + h * L + t];
        e[t].v = v == 0.0f ? 0.0f : v;   /* -0 and +0 compare equal; keep one spelling */
        e[t].t = (int32_t)t;
      }
      qsort(e, (size_t)L, sizeof(scored_entry), by_score_then_index);
      int32_t* out = kept + kept_offset(p, r, h);
      for (int64_t i = 0; i < k; ++i) out[i] = e[i].t;
      qsort(out, (size_t)k, sizeof(int32_t), ascending_int);
      free(e);
    }
  }
  return 0;
}

/* Host-side totals of one step: entries kept, fresh pages needed, pages freed. */
int actkv_oracle_totals(const oracle_problem* p, int64_t* num_kept, int64_t* fresh_needed,
                        int64_t* pages_freed) {
  if (check_problem(p)) return -1;
  int64_t nk = 0, fresh = 0, freed = 0;
  for (int r = 0; r < p->num_reqs; ++r) {
    const int64_t L = p->seq_lens[r];
    int64_t kmax = 0, bmin = INT64_MAX;
    for (int h = 0; h < p->num_kv_heads; ++h) {
      int64_t b = p->budgets[r * p->num_kv_heads + h];
      if (b < 0) return -1;
      int64_t k = b > L ? L : b;
      nk += k;
      kmax = k > kmax ? k : kmax;
      bmin = b < bmin ? b : bmin;
    }
    if (bmin >= L) continue;   /* every head keeps everything: request left untouched */
    fresh += (kmax + p->page_size - 1) / p->page_size;
    freed += (L + p->page_size - 1) / p->page_size;
  }
  *num_kept = nk;
  *fresh_needed = fresh;
  *pages_freed = freed;
  return 0;
}

/*
 * Fresh-page compaction.  Requests in order; a request whose every head keeps all its
 * entries is skipped (block table row, pages and lengths untouched).  Otherwise, with
 * X = ceil(max_h k_h / page_size) and Y = ceil(L / page_size):
 *   fresh    = free_pages[off .. off + X), off advancing over the requests in order;
 *   for each head h and j < k_h the K and V rows of token kept[j] are copied bit for bit
 *   to page fresh[j / page_size], slot j % page_size;
 *   freed_out gets the old bt[r, 0 .. Y) (request order);
 *   bt[r, 0 .. X) = fresh, bt[r, X .. Y) = -1;  new_lens[r, h] = k_h.
 * Slots of fresh pages at or beyond k_h (for head h) are not written.
 */
int actkv_oracle_compact(const oracle_problem* p, uint16_t* kv, int32_t* bt,
                         const int32_t* kept, const int32_t* free_pages, int64_t num_free,
                         int32_t* freed_out, int32_t* new_lens) {
  if (check_problem(p)) return -1;
  int64_t nk, need, nfreed;
  if (actkv_oracle_totals(p, &nk, &need, &nfreed)) return -1;
  if (need > num_free) return -2;
  const int Hkv = p->num_kv_heads, D = p->head_dim, BS = p->page_size;
  int64_t fresh_off = 0, freed_off = 0;
  for (int r = 0; r < p->num_reqs; ++r) {
    const int64_t L = p->seq_lens[r];
    int32_t* row = bt + (int64_t)r * p->bt_stride;
    int64_t kmax = 0, bmin = INT64_MAX;
    for (int h = 0; h < Hkv; ++h) {
      int64_t b = p->budgets[r * Hkv + h];
      int64_t k = b > L ? L : b;
      kmax = k > kmax ? k : kmax;
      bmin = b < bmin ? b : bmin;
    }
    if (bmin >= L) {
      for (int h = 0; h < Hkv; ++h) new_lens[r * Hkv + h] = (int32_t)L;
      continue;
    }
    const int64_t X = (kmax + BS - 1) / BS, Y = (L + BS - 1) / BS;
    const int32_t* fresh = free_pages + fresh_off;
    int32_t* old_pages = freed_out + freed_off;
    for (int64_t i = 0; i < Y; ++i) old_pages[i] = row[i];
    for (int h = 0; h < Hkv; ++h) {
      int64_t b = p->budgets[r * Hkv + h];
      int64_t k = b > L ? L : b;
      const int32_t* idx = kept + kept_offset(p, r, h);
      for (int64_t j = 0; j < k; ++j) {
        const int64_t src = actkv_oracle_slot(old_pages, BS, idx[j]);
        const int64_t dst = (int64_t)fresh[j / BS] * BS + j % BS;
        for (int which = 0; which < 2; ++which)
          memcpy(kv_row_mut(p, kv, which, dst, h), kv_row(p, kv, which, src, h),
                 sizeof(uint16_t) * (size_t)D);
      }
      new_lens[r * Hkv + h] = (int32_t)k;
    }
    for (int64_t i = 0; i < Y; ++i) row[i] = i < X ? fresh[i] : -1;
    fresh_off += X;
    freed_off += Y;
  }
  return 0;
}

/*
 * In-place compaction (Alg. 4, Sec. 7.2): the survivors of a request are packed into the
 * request's own last blocks instead of fresh pages.  Requests are handled in order; one
 * whose every head keeps all its entries is left untouched, as above.
 *
 * Definition used here.  Y = ceil(L / BS) blocks hold the request; X = ceil(max_h k_h / BS)
 * of them, the last X, are kept.  Every KV head has its own keep set (its k_h = min(budget,
 * L) kept token indices, ascending), but a block holds every head's row of a slot, so all
 * heads share the same tail: it starts at logical slot Start = (Y - X) * BS, and head h
 * fills [Start, Start + k_h).  Inside that range, a slot already holding a kept entry stays
 * as it is; every other slot of the range -- including slots at or past L in a partly
 * filled last block, which exist but hold no entry -- receives one kept entry from outside
 * the range.  Kept entries outside the range and free slots inside it are paired in
 * ascending order of their logical slots, and each pair copies the K and V rows of head h
 * (physical slots through the request's block-table row as it was before this call).
 * Sources are kept entries and destinations are not, so no copy overwrites a row another
 * copy still reads.
 *
 * Afterwards the block-table row is bt[r, Y - X .. Y) followed by -1 up to Y; the first
 * Y - X blocks go to freed_out (request order); new_lens[r, h] = k_h; new_order (laid out
 * like kept) gets, for every new slot j < k_h, the original token index of the entry now
 * there.  A skipped request keeps new_order = kept.  *num_pairs (if given) counts the
 * copies.  Returns -3 if a head's free slots and outside entries are not equal in number
 * (cannot happen for a valid keep set).
 */
int actkv_oracle_compact_inplace(const oracle_problem* p, uint16_t* kv, int32_t* bt,
                                 const int32_t* kept, int32_t* freed_out, int32_t* new_lens,
                                 int32_t* new_order, int64_t* num_pairs) {
  if (check_problem(p)) return -1;
  const int Hkv = p->num_kv_heads, D = p->head_dim, BS = p->page_size;
  int64_t freed_off = 0, pairs_total = 0;
  for (int r = 0; r < p->num_reqs; ++r) {
    const int64_t L = p->seq_lens[r];
    int32_t* row = bt + (int64_t)r * p->bt_stride;
    int64_t kmax = 0, bmin = INT64_MAX;
    for (int h = 0; h < Hkv; ++h) {
      const int64_t b = p->budgets[r * Hkv + h];
      if (b < 0) return -1;
      const int64_t k = b > L ? L : b;
      kmax = k > kmax ? k : kmax;
      bmin = b < bmin ? b : bmin;
    }
    if (bmin >= L) {
      for (int h = 0; h < Hkv; ++h) {
        new_lens[r * Hkv + h] = (int32_t)L;
        const int64_t ko = kept_offset(p, r, h);
        for (int64_t j = 0; j < L; ++j) new_order[ko + j] = kept[ko + j];
      }
      continue;
    }
    /* the shared tail: the last X of the request's Y blocks */
    const int64_t Y = (L + BS - 1) / BS, X = (kmax + BS - 1) / BS;
    const int64_t start = (Y - X) * BS, slots = Y * BS;
    unsigned char* is_kept = (unsigned char*)malloc((size_t)slots);
    int64_t* outside = (int64_t*)malloc(sizeof(int64_t) * (size_t)(slots > 0 ? slots : 1));
    int64_t* holes = (int64_t*)malloc(sizeof(int64_t) * (size_t)(slots > 0 ? slots : 1));
    for (int h = 0; h < Hkv; ++h) {
      const int64_t b = p->budgets[r * Hkv + h];
      const int64_t k = b > L ? L : b;
      const int64_t end = start + k;
      const int64_t ko = kept_offset(p, r, h);
      memset(is_kept, 0, (size_t)slots);
      for (int64_t j = 0; j < k; ++j) is_kept[kept[ko + j]] = 1;
      /* slots of [start, end): a kept entry already there stays, the rest are holes */
      int64_t n_holes = 0;
      for (int64_t t = start; t < end; ++t) {
        if (is_kept[t]) new_order[ko + (t - start)] = (int32_t)t;
        else holes[n_holes++] = t;
      }
      /* kept entries outside [start, end), ascending */
      int64_t n_out = 0;
      for (int64_t t = 0; t < slots; ++t)
        if (is_kept[t] && (t < start || t >= end)) outside[n_out++] = t;
      if (n_out != n_holes) {
        free(is_kept); free(outside); free(holes);
        return -3;
      }
      /* the i-th outside entry moves into the i-th hole */
      for (int64_t i = 0; i < n_out; ++i) {
        const int64_t ps = actkv_oracle_slot(row, BS, outside[i]);
        const int64_t pd = actkv_oracle_slot(row, BS, holes[i]);
        for (int which = 0; which < 2; ++which)
          memcpy(kv_row_mut(p, kv, which, pd, h), kv_row(p, kv, which, ps, h),
                 sizeof(uint16_t) * (size_t)D);
        new_order[ko + (holes[i] - start)] = (int32_t)outside[i];
      }
      pairs_total += n_out;
      new_lens[r * Hkv + h] = (int32_t)k;
    }
    free(is_kept); free(outside); free(holes);
    /* the freed blocks, then the row: the last X blocks move to the front */
    for (int64_t i = 0; i < Y - X; ++i) freed_out[freed_off + i] = row[i];
    for (int64_t i = 0; i < X; ++i) row[i] = row[Y - X + i];
    for (int64_t i = X; i < Y; ++i) row[i] = -1;
    freed_off += Y - X;
  }
  if (num_pairs) *num_pairs = pairs_total;
  return 0;
}

/* The whole step: scores -> pool -> select -> compact, each as defined above. */
int actkv_oracle_step(const oracle_problem* p, const uint16_t* q, uint16_t* kv, int32_t* bt,
                      const float* lse_in, const int32_t* free_pages, int64_t num_free,
                      float* raw_out, float* pooled_out, int32_t* kept_out,
                      int32_t* freed_out, int32_t* new_lens) {
  int rc = actkv_oracle_scores(p, q, kv, bt, lse_in, raw_out);
  if (!rc) rc = actkv_oracle_pool(p, raw_out, pooled_out);
  if (!rc) rc = actkv_oracle_select(p, pooled_out, kept_out);
  if (!rc) rc = actkv_oracle_compact(p, kv, bt, kept_out, free_pages, num_free, freed_out,
                                     new_lens);
  return rc;
}

/* ---------------------------------------------------------------------------------------
 * Attention-aware LRFU keep scores (Sec. 5.1 keep-score update; Alg. 1 steps 2-5).
 *
 * Hit mask (Alg. 1 step 3, GetHitMask): per (request, KV head), order the entries by score
 * descending (ties: lower token index first) and take the shortest prefix whose running
 * sum reaches top_p times the segment's total.  Those entries are hits.  The running sum
 * and the total are carried in double; a segment whose top_p * total is not positive has
 * no hits.  top_p >= 1 asks for the whole mass: every entry with a positive score is a hit
 * (the same set, without depending on how the running sum rounds against the total).
 * ------------------------------------------------------------------------------------- */
int actkv_oracle_hits(const oracle_problem* p, const float* att, double top_p, uint8_t* hit) {
  if (check_problem(p)) return -1;
  for (int r = 0; r < p->num_reqs; ++r) {
    const int64_t L = p->seq_lens[r], soff = score_offset(p, r);
    for (int h = 0; h < p->num_kv_heads; ++h) {
      const float* a = att + soff + h * L;
      uint8_t* out = hit + soff + h * L;
      double total = 0.0;
      for (int64_t t = 0; t < L; ++t) total += (double)a[t];
      for (int64_t t = 0; t < L; ++t) out[t] = 0;
      const double need = top_p * total;
      if (!(need > 0.0)) continue;
      if (top_p >= 1.0) {
        for (int64_t t = 0; t < L; ++t) out[t] = a[t] > 0.0f;
        continue;
      }
      scored_entry* e = (scored_entry*)malloc(sizeof(scored_entry) * (size_t)(L > 0 ? L : 1));
      for (int64_t t = 0; t < L; ++t) {
        e[t].v = a[t] == 0.0f ? 0.0f : a[t];
        e[t].t = (int32_t)t;
      }
      qsort(e, (size_t)L, sizeof(scored_entry), by_score_then_index);
      double run = 0.0;
      for (int64_t i = 0; i < L && run < need; ++i) {
        out[e[i].t] = 1;
        run += (double)e[i].v;
      }
      free(e);
    }
  }
  return 0;
}

/* Keep-score update (Alg. 1 step 4): KS <- decay * KS, plus the entry's score if it is a
 * hit.  KS is fp32 state; each of the two operations rounds to fp32 (no fused multiply-add),
 * in this order. */
int actkv_oracle_lrfu_update(const oracle_problem* p, const float* att, const uint8_t* hit,
                             float decay, float* ks) {
  if (check_problem(p)) return -1;
  int64_t n = 0;
  for (int r = 0; r < p->num_reqs; ++r) n += (int64_t)p->seq_lens[r] * p->num_kv_heads;
  for (int64_t i = 0; i < n; ++i) {
    volatile float scaled = decay * ks[i];
    volatile float sum = scaled + (hit[i] ? att[i] : 0.0f);
    ks[i] = sum;
  }
  return 0;
}

/* Timing support (not part of what the oracle computes): the OpenMP thread count the
 * parallel loops above use, and setting it (the benchmark times the oracle at one thread
 * and at all host threads). */
#include <omp.h>
int actkv_oracle_get_threads(void) { return omp_get_max_threads(); }
void actkv_oracle_set_threads(int n) { if (n > 0) omp_set_num_threads(n); }
