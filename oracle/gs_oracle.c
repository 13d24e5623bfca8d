/*
 * gs_oracle.c -- plain, slow, obviously correct CPU oracle of the gs-SGD
 * gradient-compression step.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg load this library. The GPU library shares no code, header, table or
 * helper with it, and neither side includes or calls the other.
 *
 * Source: Dai, Diao, Li, Xu, "A Distributed SGD Algorithm with Global Sketching for Deep
 * Learning Training Acceleration" (arXiv 2108.06004).
 *   - Count Sketch of a gradient, S(g) = C g, a linear map, hence S(a+b) = S(a) + S(b)
 *     (Sec. III-A, the Count Sketch paragraph).
 *   - Every worker sketches its own gradient (Alg. 1, sketch step).
 *   - The P sketches are summed along a binomial tree: in each round the even local rank
 *     receives from the next rank and adds, the odd one sends; an odd participant count
 *     lets the highest id pass through (Alg. 1 reduction loop; Sec. III-A, the
 *     non-power-of-two paragraph).
 *   - HEAVYMIX: estimate every coordinate from the merged sketch, pick Top_k, fetch the
 *     exact values of Top_k in a second round (Alg. 2).
 *   - Momentum and error accumulation alongside sketching (Sec. II, sketching paragraph;
 *     error feedback and momentum correction are the related-work methods cited there).
 *
 * Readings where the paper is silent (listed with reasons in the design notes):
 *   accumulate    u <- fl(fl(rho*u) + g), v <- fl(v + u)   (fp32, no fused multiply-add)
 *   bucket hash   h_j(i) = ((a_j*i + b_j) mod p) mod c,  p = 2^31 - 1
 *   sign hash     s_j(i) = +1 if ((a2_j*i + b2_j) mod p) is odd, else -1
 *   sketch cells  summed in double precision, rounded once to fp32
 *   merge, gather binomial-tree order (above), fp32 additions
 *   estimate      median over rows of s_j(i) * S[j][h_j(i)]; even r: fl(fl(m1+m2)*0.5f)
 *   Top_k         the k largest |estimate|, ties to the lower index, returned ascending
 *   HEAVYMIX      as printed, with a fixed pairwise order for the row sums of squares and
 *                 the random fill taken from caller-supplied draws (see ora_heavymix)
 *   sketch state  momentum and error kept in the merged sketch (see ora_sketch_momentum_step)
 *   reset         v (and u when reset_momentum) zeroed at Top_k on every worker
 *
 * Build: gcc -O2 -ffp-contract=off -std=c11 (no -ffast-math). On x86-64 float arithmetic
 * is IEEE binary32 with round-to-nearest-even, so each fl() above is one rounding.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORA_P 2147483647ULL /* the Mersenne prime 2^31 - 1 */

/* ---------------------------------------------------------------------------------- */
/* Hash families (Count Sketch, Sec. III-A). Arguments: 1 <= a < p, 0 <= b < p, 0 <= i < p. */

uint64_t ora_hash_raw(uint32_t a, uint32_t b, int64_t i) {
  /* a < 2^31 and i < 2^31, so a*i + b < 2^63: exact in 64-bit unsigned arithmetic. */
  return ((uint64_t)a * (uint64_t)i + (uint64_t)b) % ORA_P;
}

int64_t ora_bucket(uint32_t a, uint32_t b, int64_t c, int64_t i) {
  return (int64_t)(ora_hash_raw(a, b, i) % (uint64_t)c);
}

int ora_sign(uint32_t a2, uint32_t b2, int64_t i) { return (ora_hash_raw(a2, b2, i) & 1u) ? 1 : -1; }

/* Vector forms for tests: out[t] = bucket / sign of coordinate idx[t]. */
void ora_buckets(uint32_t a, uint32_t b, int64_t c, int64_t n, const int64_t* idx, int64_t* out) {
  for (int64_t t = 0; t < n; ++t) out[t] = ora_bucket(a, b, c, idx[t]);
}
void ora_signs(uint32_t a2, uint32_t b2, int64_t n, const int64_t* idx, int32_t* out) {
  for (int64_t t = 0; t < n; ++t) out[t] = ora_sign(a2, b2, idx[t]);
}
void ora_hash_raws(uint32_t a, uint32_t b, int64_t n, const int64_t* idx, int64_t* out) {
  for (int64_t t = 0; t < n; ++t) out[t] = (int64_t)ora_hash_raw(a, b, idx[t]);
}

/* ---------------------------------------------------------------------------------- */
/* Momentum + error-feedback accumulation (Sec. II sketching paragraph; Alg. 1 starts
 * from a zero state). Elementwise over n = P*d entries: u <- rho*u + g, v <- v + u. */

void ora_accumulate(int64_t n, float rho, const float* g, float* u, float* v) {
  for (int64_t t = 0; t < n; ++t) {
    float m = rho * u[t];
    float un = m + g[t];
    u[t] = un;
    v[t] = v[t] + un;
  }
}

/* ---------------------------------------------------------------------------------- */
/* Count Sketch insertion (Sec. III-A; Alg. 1 sketch step), for every worker:
 *   tables[q][j][col] = sum over i with h_j(i) == col of s_j(i) * v[q][i]
 * summed in double, rounded once. v is [P][d], tables is [P][r][c]. Returns 0, or 1 when
 * the scratch allocation fails. */

int ora_sketch(int32_t P, int64_t d, int32_t r, int64_t c, const uint32_t* ha, const uint32_t* hb,
               const uint32_t* sa, const uint32_t* sb, const float* v, float* tables) {
  double* cell = (double*)calloc((size_t)P * (size_t)r * (size_t)c, sizeof(double));
  if (!cell) return 1;
  for (int32_t j = 0; j < r; ++j) {
    for (int64_t i = 0; i < d; ++i) {
      int64_t col = ora_bucket(ha[j], hb[j], c, i);
      double s = (double)ora_sign(sa[j], sb[j], i);
      for (int32_t q = 0; q < P; ++q) cell[((int64_t)q * r + j) * c + col] += s * (double)v[(int64_t)q * d + i];
    }
  }
  for (int64_t t = 0; t < (int64_t)P * r * c; ++t) tables[t] = (float)cell[t];
  free(cell);
  return 0;
}

/* Selected cells only: out[n][q] = sketch cell (row[n], col[n]) of worker q, computed as
 * above. Used to check full-size tables at sampled cells. Returns 0, or 1 on bad input. */
int ora_sketch_cells(int32_t P, int64_t d, int32_t r, int64_t c, const uint32_t* ha, const uint32_t* hb,
                     const uint32_t* sa, const uint32_t* sb, const float* v, int64_t ncell,
                     const int32_t* row, const int64_t* col, float* out) {
  int64_t* slot = (int64_t*)malloc((size_t)c * sizeof(int64_t));
  double* acc = (double*)calloc((size_t)ncell * (size_t)P, sizeof(double));
  if (!slot || !acc) { free(slot); free(acc); return 1; }
  for (int32_t j = 0; j < r; ++j) {
    int any = 0;
    for (int64_t t = 0; t < c; ++t) slot[t] = -1;
    for (int64_t n = 0; n < ncell; ++n) {
      if (row[n] == j) {
        if (col[n] < 0 || col[n] >= c || slot[col[n]] != -1) { free(slot); free(acc); return 1; }
        slot[col[n]] = n;
        any = 1;
      }
    }
    if (!any) continue;
    for (int64_t i = 0; i < d; ++i) {
      int64_t n = slot[ora_bucket(ha[j], hb[j], c, i)];
      if (n < 0) continue;
      double s = (double)ora_sign(sa[j], sb[j], i);
      for (int32_t q = 0; q < P; ++q) acc[n * P + q] += s * (double)v[(int64_t)q * d + i];
    }
  }
  for (int64_t t = 0; t < ncell * P; ++t) out[t] = (float)acc[t];
  free(slot);
  free(acc);
  return 0;
}

/* ---------------------------------------------------------------------------------- */
/* Binomial-tree reduction (Alg. 1 reduction loop; Sec. III-A, non-power-of-two case).
 * bufs[0..P-1] point at P arrays of n floats. The list L of participating ranks starts as
 * 0..P-1. Each round pairs L[0] with L[1], L[2] with L[3], ...: the first of each pair
 * (even local rank) adds the second's array into its own and stays in the list; an
 * unpaired last rank passes to the next round untouched. When one rank is left (always
 * rank 0) its array holds the sum. The arrays of the other ranks are left as they were
 * after their last round. */

static void tree_reduce(int32_t P, int64_t n, float** bufs, int32_t* L) {
  int32_t m = P;
  for (int32_t t = 0; t < P; ++t) L[t] = t;
  while (m > 1) {
    int32_t next = 0;
    for (int32_t t = 0; t < m; t += 2) {
      if (t + 1 < m) {
        float* dst = bufs[L[t]];
        const float* src = bufs[L[t + 1]];
        for (int64_t e = 0; e < n; ++e) dst[e] = src[e] + dst[e];
      }
      L[next++] = L[t];
    }
    m = next;
  }
}

/* Sum of P floats in tree order. */
float ora_tree_sum(int32_t P, const float* x) {
  float* tmp = (float*)malloc((size_t)P * sizeof(float));
  float** ptr = (float**)malloc((size_t)P * sizeof(float*));
  int32_t* L = (int32_t*)malloc((size_t)P * sizeof(int32_t));
  float res = 0.0f;
  if (tmp && ptr && L) {
    for (int32_t q = 0; q < P; ++q) { tmp[q] = x[q]; ptr[q] = &tmp[q]; }
    tree_reduce(P, 1, ptr, L);
    res = tmp[0];
  }
  free(tmp);
  free(ptr);
  free(L);
  return res;
}

/* merged[j][col] = tree-order sum over q of tables[q][j][col]; tables is [P][rc].
 * Returns 0, or 1 when the scratch allocation fails. */
int ora_merge(int32_t P, int64_t rc, const float* tables, float* merged) {
  float* work = (float*)malloc((size_t)P * (size_t)rc * sizeof(float));
  float** bufs = (float**)malloc((size_t)P * sizeof(float*));
  int32_t* L = (int32_t*)malloc((size_t)P * sizeof(int32_t));
  if (!work || !bufs || !L) { free(work); free(bufs); free(L); return 1; }
  memcpy(work, tables, (size_t)P * (size_t)rc * sizeof(float));
  for (int32_t q = 0; q < P; ++q) bufs[q] = work + (int64_t)q * rc;
  tree_reduce(P, rc, bufs, L);
  memcpy(merged, work, (size_t)rc * sizeof(float));
  free(work);
  free(bufs);
  free(L);
  return 0;
}

/* ---------------------------------------------------------------------------------- */
/* HEAVYMIX query (Alg. 2, first step): the Count Sketch estimate of coordinate i is the
 * median over rows of s_j(i) * S[j][h_j(i)]. The r values are fully sorted (insertion
 * sort); odd r takes the middle one, even r the fp32 mean of the two middle ones. */

static float median_of(int32_t r, float* vals) {
  for (int32_t a = 1; a < r; ++a) {
    float x = vals[a];
    int32_t b = a - 1;
    while (b >= 0 && vals[b] > x) { vals[b + 1] = vals[b]; --b; }
    vals[b + 1] = x;
  }
  if (r & 1) return vals[r / 2];
  float s = vals[r / 2 - 1] + vals[r / 2];
  return s * 0.5f;
}

static float estimate_at(int32_t r, int64_t c, const uint32_t* ha, const uint32_t* hb, const uint32_t* sa,
                         const uint32_t* sb, const float* merged, int64_t i, float* vals) {
  for (int32_t j = 0; j < r; ++j) {
    float cellv = merged[(int64_t)j * c + ora_bucket(ha[j], hb[j], c, i)];
    vals[j] = ora_sign(sa[j], sb[j], i) > 0 ? cellv : -cellv;
  }
  return median_of(r, vals);
}

/* est[i] for every i in [0, d). Returns 0, or 1 on allocation failure. */
int ora_unsketch(int64_t d, int32_t r, int64_t c, const uint32_t* ha, const uint32_t* hb, const uint32_t* sa,
                 const uint32_t* sb, const float* merged, float* est) {
  float* vals = (float*)malloc((size_t)r * sizeof(float));
  if (!vals) return 1;
  for (int64_t i = 0; i < d; ++i) est[i] = estimate_at(r, c, ha, hb, sa, sb, merged, i, vals);
  free(vals);
  return 0;
}

/* est at selected coordinates: out[t] = estimate of coordinate idx[t]. */
int ora_unsketch_at(int32_t r, int64_t c, const uint32_t* ha, const uint32_t* hb, const uint32_t* sa,
                    const uint32_t* sb, const float* merged, int64_t n, const int64_t* idx, float* out) {
  float* vals = (float*)malloc((size_t)r * sizeof(float));
  if (!vals) return 1;
  for (int64_t t = 0; t < n; ++t) out[t] = estimate_at(r, c, ha, hb, sa, sb, merged, idx[t], vals);
  free(vals);
  return 0;
}

/* ---------------------------------------------------------------------------------- */
/* Top_k (Alg. 2, selection; Sec. III-A: the top-k largest elements by magnitude).
 * Sort every coordinate by (|est| descending, index ascending), keep the first k, and
 * return their indices in ascending order. Also returns the k-th key (the smallest kept
 * |est|) through *kth_key when kth_key is not NULL. */

typedef struct { float key; int64_t idx; } ora_kv;

static int cmp_kv(const void* pa, const void* pb) {
  const ora_kv* a = (const ora_kv*)pa;
  const ora_kv* b = (const ora_kv*)pb;
  if (a->key > b->key) return -1;
  if (a->key < b->key) return 1;
  return (a->idx > b->idx) - (a->idx < b->idx);
}

static int cmp_i32(const void* pa, const void* pb) {
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  return (a > b) - (a < b);
}

int ora_topk(int64_t d, int64_t k, const float* est, int32_t* idx_out, float* kth_key) {
  if (k < 1 || k > d) return 1;
  ora_kv* kv = (ora_kv*)malloc((size_t)d * sizeof(ora_kv));
  if (!kv) return 1;
  for (int64_t i = 0; i < d; ++i) {
    float e = est[i];
    kv[i].key = e < 0.0f ? -e : e + 0.0f; /* |e|, with -0 mapped to +0 */
    kv[i].idx = i;
  }
  qsort(kv, (size_t)d, sizeof(ora_kv), cmp_kv);
  for (int64_t t = 0; t < k; ++t) idx_out[t] = (int32_t)kv[t].idx;
  if (kth_key) *kth_key = kv[k - 1].key;
  qsort(idx_out, (size_t)k, sizeof(int32_t), cmp_i32);
  free(kv);
  return 0;
}

/* ---------------------------------------------------------------------------------- */
/* Exact values of Top_k (Alg. 2, second round) and error reset.
 * values[t] = tree-order sum over workers of v[q][idx[t]] (before the reset); then
 * v[q][idx[t]] = 0 and, if reset_momentum, u[q][idx[t]] = 0, for every worker q. */

int ora_gather_reset(int32_t P, int64_t d, int64_t k, const int32_t* idx, int32_t reset_momentum, float* u,
                     float* v, float* values) {
  float* tmp = (float*)malloc((size_t)P * sizeof(float));
  if (!tmp) return 1;
  for (int64_t t = 0; t < k; ++t) {
    int64_t i = idx[t];
    if (i < 0 || i >= d) { free(tmp); return 1; }
    for (int32_t q = 0; q < P; ++q) tmp[q] = v[(int64_t)q * d + i];
    values[t] = ora_tree_sum(P, tmp);
  }
  for (int64_t t = 0; t < k; ++t) {
    int64_t i = idx[t];
    for (int32_t q = 0; q < P; ++q) {
      v[(int64_t)q * d + i] = 0.0f;
      if (reset_momentum) u[(int64_t)q * d + i] = 0.0f;
    }
  }
  free(tmp);
  return 0;
}

/* ---------------------------------------------------------------------------------- */
/* HEAVYMIX as printed (Alg. 2): query every estimate, split the coordinates by the heavy
 * test into H and NH, and take Top_k = H plus a random l-subset of NH, l = k - |H|.
 *
 * The l2-norm-squared estimate: for each row j the sum over columns of S[j][col]^2, the
 * median of these r row sums (even r: fl(fl(m1 + m2) * 0.5)), all in fp64. A square of an
 * fp32 value is exact in fp64; the row sum is taken in a fixed order, a pairwise tree: the
 * c squares, padded with zeros to the next power of two, are added in adjacent pairs, level
 * by level, until one value remains. The fixed order makes the heavy decision below a
 * function of S alone.
 *
 * Heavy test: theta = fl(l2sq / k); i is heavy when est_i^2 >= theta (est_i^2 exact in
 * fp64). The paper's test compares the queried square of the estimate with l2sq / k.
 *
 * Random fill: rnd[i] is the caller's random draw for coordinate i (one uniform 32-bit
 * word each). The fill takes the l non-heavy coordinates with the largest rnd[i] >> 1,
 * ties to the lower index: with independent uniform draws this is a uniformly random
 * l-subset of NH (ties, which need equal 31-bit draws, aside).
 *
 * When |H| >= k (l would be zero or negative) Top_k is the k members of H with the
 * largest |est_i|, ties to the lower index; every member of H outranks every member of
 * NH, so this is the deterministic top-k. Top_k is returned in ascending order. */

/* In-place pairwise (adjacent pairs) tree sum of n = 2^m values; destroys buf. */
static double pairwise_sum(double* buf, int64_t n) {
  for (int64_t w = n; w > 1; w /= 2)
    for (int64_t m = 0; m < w / 2; ++m) buf[m] = buf[2 * m] + buf[2 * m + 1];
  return buf[0];
}

double ora_row_sq_sum(int64_t c, const float* row) {
  int64_t n = 1;
  while (n < c) n *= 2;
  double* buf = (double*)calloc((size_t)n, sizeof(double));
  if (!buf) return -1.0;
  for (int64_t t = 0; t < c; ++t) buf[t] = (double)row[t] * (double)row[t];
  const double s = pairwise_sum(buf, n);
  free(buf);
  return s;
}

double ora_l2sq_estimate(int32_t r, int64_t c, const float* merged) {
  double* rows = (double*)malloc((size_t)r * sizeof(double));
  double res = 0.0;
  if (!rows) return -1.0;
  for (int32_t j = 0; j < r; ++j) rows[j] = ora_row_sq_sum(c, merged + (int64_t)j * c);
  for (int32_t a = 1; a < r; ++a) {
    double x = rows[a];
    int32_t b = a - 1;
    while (b >= 0 && rows[b] > x) { rows[b + 1] = rows[b]; --b; }
    rows[b + 1] = x;
  }
  res = (r & 1) ? rows[r / 2] : 0.5 * (rows[r / 2 - 1] + rows[r / 2]);
  free(rows);
  return res;
}

int64_t ora_heavy_count(int64_t d, int64_t k, const float* est, double l2sq) {
  const double theta = l2sq / (double)k;
  int64_t n = 0;
  for (int64_t i = 0; i < d; ++i) {
    double e = (double)est[i];
    if (e * e >= theta) ++n;
  }
  return n;
}

typedef struct { uint32_t key; int64_t idx; } ora_uk;

static int cmp_uk(const void* pa, const void* pb) {
  const ora_uk* a = (const ora_uk*)pa;
  const ora_uk* b = (const ora_uk*)pb;
  if (a->key > b->key) return -1;
  if (a->key < b->key) return 1;
  return (a->idx > b->idx) - (a->idx < b->idx);
}

int ora_heavymix(int64_t d, int32_t r, int64_t c, int64_t k, const uint32_t* ha, const uint32_t* hb,
                 const uint32_t* sa, const uint32_t* sb, const float* merged, const uint32_t* rnd, float* est,
                 int32_t* idx_out, int64_t* n_heavy, double* l2sq_out) {
  if (k < 1 || k > d) return 1;
  float* es = est ? est : (float*)malloc((size_t)d * sizeof(float));
  ora_kv* heavy = (ora_kv*)malloc((size_t)d * sizeof(ora_kv));
  ora_uk* light = (ora_uk*)malloc((size_t)d * sizeof(ora_uk));
  int rc = (!es || !heavy || !light) ? 1 : 0;
  int64_t nh = 0, nl = 0;
  double l2 = 0.0;
  if (!rc) rc = ora_unsketch(d, r, c, ha, hb, sa, sb, merged, es);
  if (!rc) {
    /* step 1: query the estimates (above); step 2: H and NH */
    l2 = ora_l2sq_estimate(r, c, merged);
    const double theta = l2 / (double)k;
    for (int64_t i = 0; i < d; ++i) {
      const double e = (double)es[i];
      if (e * e >= theta) {
        heavy[nh].key = es[i] < 0.0f ? -es[i] : es[i] + 0.0f;
        heavy[nh].idx = i;
        ++nh;
      } else {
        light[nl].key = rnd[i] >> 1;
        light[nl].idx = i;
        ++nl;
      }
    }
    /* step 3: Top_k = H plus rand_l(NH) */
    int64_t t = 0;
    if (nh >= k) {
      qsort(heavy, (size_t)nh, sizeof(ora_kv), cmp_kv);
      for (; t < k; ++t) idx_out[t] = (int32_t)heavy[t].idx;
    } else {
      for (int64_t m = 0; m < nh; ++m) idx_out[t++] = (int32_t)heavy[m].idx;
      qsort(light, (size_t)nl, sizeof(ora_uk), cmp_uk);
      for (int64_t m = 0; t < k; ++m) idx_out[t++] = (int32_t)light[m].idx;
    }
    qsort(idx_out, (size_t)k, sizeof(int32_t), cmp_i32);
  }
  if (n_heavy) *n_heavy = nh;
  if (l2sq_out) *l2sq_out = l2;
  if (!est) free(es);
  free(heavy);
  free(light);
  return rc;
}

/* ---------------------------------------------------------------------------------- */
/* The weight update (Alg. 1, last step): w <- w - eta * G~, where G~ is zero outside Top_k
 * and holds the selected values there: w[idx[t]] = fl(w[idx[t]] - fl(eta * values[t])). */

int ora_apply_update(int64_t d, int64_t k, const int32_t* idx, const float* values, float lr, float* w) {
  for (int64_t t = 0; t < k; ++t) {
    const int64_t i = idx[t];
    if (i < 0 || i >= d) return 1;
    const float step = lr * values[t];
    w[i] = w[i] - step;
  }
  return 0;
}

/* ---------------------------------------------------------------------------------- */
/* Momentum and error accumulation kept in the sketch (the sketch is linear, so both can be
 * carried inside it: Sec. II, sketching paragraph, after FetchSGD). One step:
 *   S = tree-order merge of the P workers' sketches of g          (Alg. 1 sketch + reduction)
 *   U <- fl(fl(rho * U) + S),  E <- fl(E + U)                       (per cell, fp32, no FMA)
 *   est = median unsketch of E;  Top_k = the k largest |est|, ties to the lower index
 *   values: Delta_i = est_i for i in Top_k (no per-worker vectors hold exact values)
 *   E <- fl(E - D) on every cell D touches, where D = S(Delta) is the sketch of the sparse
 *        selection, each touched cell summed in fp64 and rounded once to fp32
 *   U <- 0 on those cells when reset_momentum (momentum masking)
 * U and E are [r][c], updated in place; merged ([r][c]) receives S; est ([d]) may be NULL.
 * ora_sketch_state_update is the part after the merge, from a given S. */

int ora_sketch_state_update(int64_t d, int32_t r, int64_t c, int64_t k, float rho, int32_t reset_momentum,
                            const uint32_t* ha, const uint32_t* hb, const uint32_t* sa, const uint32_t* sb,
                            const float* merged, float* U, float* E, float* est, int32_t* idx, float* values) {
  const int64_t rc = (int64_t)r * c;
  float* es = est ? est : (float*)malloc((size_t)d * sizeof(float));
  double* acc = (double*)calloc((size_t)rc, sizeof(double));
  unsigned char* touched = (unsigned char*)calloc((size_t)rc, 1);
  int rc_ = (!es || !acc || !touched) ? 1 : 0;
  if (!rc_) {
    for (int64_t e = 0; e < rc; ++e) {
      float m = rho * U[e];
      U[e] = m + merged[e];
      E[e] = E[e] + U[e];
    }
    rc_ = ora_unsketch(d, r, c, ha, hb, sa, sb, E, es);
  }
  if (!rc_) rc_ = ora_topk(d, k, es, idx, NULL);
  if (!rc_) {
    for (int64_t t = 0; t < k; ++t) {
      const int64_t i = idx[t];
      values[t] = es[i];
      for (int32_t j = 0; j < r; ++j) {
        const int64_t cell = (int64_t)j * c + ora_bucket(ha[j], hb[j], c, i);
        acc[cell] += (double)ora_sign(sa[j], sb[j], i) * (double)es[i];
        touched[cell] = 1;
      }
    }
    for (int64_t e = 0; e < rc; ++e) {
      if (!touched[e]) continue;
      E[e] = E[e] - (float)acc[e];
      if (reset_momentum) U[e] = 0.0f;
    }
  }
  if (!est) free(es);
  free(acc);
  free(touched);
  return rc_;
}

int ora_sketch_momentum_step(int32_t P, int64_t d, int32_t r, int64_t c, int64_t k, float rho,
                             int32_t reset_momentum, const uint32_t* ha, const uint32_t* hb, const uint32_t* sa,
                             const uint32_t* sb, const float* g, float* U, float* E, float* merged, float* est,
                             int32_t* idx, float* values) {
  const int64_t rc = (int64_t)r * c;
  float* tb = (float*)malloc((size_t)P * (size_t)rc * sizeof(float));
  int rc_ = tb ? 0 : 1;
  if (!rc_) rc_ = ora_sketch(P, d, r, c, ha, hb, sa, sb, g, tb);
  if (!rc_) rc_ = ora_merge(P, rc, tb, merged);
  if (!rc_) rc_ = ora_sketch_state_update(d, r, c, k, rho, reset_momentum, ha, hb, sa, sb, merged, U, E, est, idx,
                                          values);
  free(tb);
  return rc_;
}

/* ---------------------------------------------------------------------------------- */
/* One full step: accumulate -> sketch -> merge -> estimate -> Top_k -> exact values and
 * reset. g, u, v are [P][d]; u and v are updated in place. tables ([P][r][c]) and est
 * ([d]) may be NULL, in which case scratch is used. Returns 0 on success. */

int ora_step(int32_t P, int64_t d, int32_t r, int64_t c, int64_t k, float rho, int32_t reset_momentum,
             const uint32_t* ha, const uint32_t* hb, const uint32_t* sa, const uint32_t* sb, const float* g,
             float* u, float* v, float* tables, float* merged, float* est, int32_t* idx, float* values) {
  int rc = 0;
  float* tb = tables ? tables : (float*)malloc((size_t)P * (size_t)r * (size_t)c * sizeof(float));
  float* es = est ? est : (float*)malloc((size_t)d * sizeof(float));
  if (!tb || !es) rc = 1;
  if (!rc) ora_accumulate((int64_t)P * d, rho, g, u, v);
  if (!rc) rc = ora_sketch(P, d, r, c, ha, hb, sa, sb, v, tb);
  if (!rc) rc = ora_merge(P, (int64_t)r * c, tb, merged);
  if (!rc) rc = ora_unsketch(d, r, c, ha, hb, sa, sb, merged, es);
  if (!rc) rc = ora_topk(d, k, es, idx, NULL);
  if (!rc) rc = ora_gather_reset(P, d, k, idx, reset_momentum, u, v, values);
  if (!tables) free(tb);
  if (!est) free(es);
  return rc;
}
