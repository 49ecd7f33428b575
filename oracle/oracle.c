/*
 * CPU oracle for the Sparse DNN Challenge inference (Kepner et al., 2019).
 *
 * TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load this library. The product path (the HIP library) never links, loads or calls it, and this
 * file shares no code, header or table with that path.
 *
 * What it computes
 *   Sec. II, batched inference equation:  Y_{l+1} = h(Y_l W_l + B_l), h = ReLU capped at YMAX = 32.
 *   Sec. V, serial reference loop: each layer forms the product Z of the activations and the
 *   weights, adds the bias only to the entries of Z that are nonzero, and clamps the result to
 *   [0, YMAX]. (Sec. II writes B_l as the bias replicated over the nonzero rows of Y_l; for the
 *   nonpositive biases of Table 1 the two readings agree.)
 *   Sec. V, second timed step: the categories are the rows of the final Y with any entry > 0.
 *
 * Two diagnostics beside the result (test infrastructure for judging fp32 against other orders or
 * precisions): the margin, min |z + b| over every layer and every entry whose product z is nonzero,
 * per row and overall (an entry this close to the clamp at 0 may flip under a different rounding);
 * and the smallest row maximum of the final Y over the rows that are categories (how far the
 * weakest category is from being dropped).
 *
 * Precision and order. The paper does not fix a precision (its Matlab listing runs in Matlab's
 * double sparse type); this oracle computes in fp32 with one fixed order so that a correct GPU
 * implementation can match it bit for bit:
 *   z[j] = fmaf(y[k_m], w_m, ... fmaf(y[k_1], w_1, fmaf(y[k_0], w_0, +0.0f)))
 * over the nonzero sources k_0 < k_1 < ... of column j, i.e. ascending source index, one fused
 * multiply-add per term, starting from +0. The bias is one fp32 add, the clamps are exact.
 * Terms with y[k] == 0 are skipped: fmaf(0, w, acc) returns acc exactly for finite w and an
 * accumulator that is never -0 (it starts at +0 and x + (-x) rounds to +0).
 *
 * Rows whose activations are all zero are not processed further: for such a row Z = 0, so the
 * bias is not added and the row stays zero for every later W and b (an exact fact of the
 * recurrence, not an approximation).
 *
 * Layout: weights arrive per layer in CSC (column j lists its sources, ascending); the oracle
 * turns each layer into CSR by source (row k lists the targets j of k) and runs Gustavson's
 * row-by-row product, so for each output the sources are visited in ascending order.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#include <pthread.h>

typedef struct {
  int32_t N;
  int64_t M;
  float ymax;
  float *y;          /* M x N current activations */
  uint8_t *live;     /* row is not all zero */
  double *margin;    /* per row: min |z + b| over all layers and entries with z != 0 */
  int64_t *counts;   /* counts[l] = live rows entering layer l */
  int64_t nlayers, cap;
} oracle_t;

static int64_t count_live(const oracle_t *o) {
  int64_t c = 0;
  for (int64_t i = 0; i < o->M; ++i) c += o->live[i];
  return c;
}

void *oracle_create(int32_t N, int64_t M, float ymax, const float *y0) {
  if (N <= 0 || M < 0 || !(ymax > 0.0f)) return NULL;
  oracle_t *o = (oracle_t *)calloc(1, sizeof(oracle_t));
  if (!o) return NULL;
  o->N = N; o->M = M; o->ymax = ymax;
  size_t n = (size_t)M * (size_t)N;
  o->y = (float *)malloc(sizeof(float) * (n ? n : 1));
  o->live = (uint8_t *)calloc((size_t)(M ? M : 1), 1);
  o->margin = (double *)malloc(sizeof(double) * (size_t)(M ? M : 1));
  o->cap = 64;
  o->counts = (int64_t *)malloc(sizeof(int64_t) * (size_t)o->cap);
  if (!o->y || !o->live || !o->margin || !o->counts) {
    free(o->y); free(o->live); free(o->margin); free(o->counts); free(o);
    return NULL;
  }
  if (n) memcpy(o->y, y0, sizeof(float) * n);
  for (int64_t i = 0; i < M; ++i) {
    const float *r = o->y + (size_t)i * N;
    uint8_t any = 0;
    for (int32_t k = 0; k < N; ++k) any |= (r[k] != 0.0f);
    o->live[i] = any;
    o->margin[i] = INFINITY;
  }
  o->counts[0] = count_live(o);
  o->nlayers = 0;
  return o;
}

void oracle_destroy(void *h) {
  oracle_t *o = (oracle_t *)h;
  if (!o) return;
  free(o->y); free(o->live); free(o->margin); free(o->counts); free(o);
}

typedef struct {
  oracle_t *o;
  const int64_t *rp;   /* CSR by source: targets of k are tj[rp[k] .. rp[k+1]) */
  const int32_t *tj;
  const float *tw;
  const float *bias;
  int64_t r0, r1;
  int rc;
} layer_job;

static void *layer_rows(void *arg) {
  layer_job *J = (layer_job *)arg;
  oracle_t *o = J->o;
  const int32_t N = o->N;
  float *acc = (float *)malloc(sizeof(float) * (size_t)N);
  if (!acc) { J->rc = -2; return NULL; }
  for (int64_t i = J->r0; i < J->r1; ++i) {
    if (!o->live[i]) continue;
    float *y = o->y + (size_t)i * N;
    for (int32_t j = 0; j < N; ++j) acc[j] = 0.0f;
    /* Z = Y W: Gustavson, sources in ascending order */
    for (int32_t k = 0; k < N; ++k) {
      const float yk = y[k];
      if (yk == 0.0f) continue;
      for (int64_t e = J->rp[k]; e < J->rp[k + 1]; ++e) {
        const int32_t j = J->tj[e];
        acc[j] = fmaf(yk, J->tw[e], acc[j]);
      }
    }
    /* bias on the nonzero entries of Z only, then the clamps to [0, YMAX] (Sec. V loop) */
    uint8_t any = 0;
    double m = o->margin[i];
    for (int32_t j = 0; j < N; ++j) {
      const float z = acc[j];
      float out = 0.0f;
      if (z != 0.0f) {
        const float t = z + J->bias[j];
        const double at = fabs((double)t);
        if (at < m) m = at;
        if (t > o->ymax) out = o->ymax;
        else if (t > 0.0f) out = t;
      }
      y[j] = out;
      any |= (out > 0.0f);
    }
    o->margin[i] = m;
    o->live[i] = any;
  }
  free(acc);
  return NULL;
}

/* Apply one layer. col_ptr has N+1 entries indexing row_idx/val (offsets need not start at 0);
   row indices must lie in [0, N). Returns 0, or -1 on malformed input, -2 on allocation failure. */
int oracle_layer(void *h, const int64_t *col_ptr, const int32_t *row_idx, const float *val, const float *bias,
                 int32_t nthreads) {
  oracle_t *o = (oracle_t *)h;
  const int32_t N = o->N;
  const int64_t base = col_ptr[0], nnz = col_ptr[N] - col_ptr[0];
  if (nnz < 0) return -1;
  for (int32_t j = 0; j < N; ++j)
    if (col_ptr[j + 1] < col_ptr[j]) return -1;
  for (int64_t e = 0; e < nnz; ++e)
    if (row_idx[base + e] < 0 || row_idx[base + e] >= N) return -1;

  /* CSC by target -> CSR by source */
  int64_t *rp = (int64_t *)calloc((size_t)N + 1, sizeof(int64_t));
  int32_t *tj = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nnz ? nnz : 1));
  float *tw = (float *)malloc(sizeof(float) * (size_t)(nnz ? nnz : 1));
  int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
  if (!rp || !tj || !tw || !fill) { free(rp); free(tj); free(tw); free(fill); return -2; }
  for (int64_t e = 0; e < nnz; ++e) rp[row_idx[base + e] + 1]++;
  for (int32_t k = 0; k < N; ++k) rp[k + 1] += rp[k];
  for (int32_t k = 0; k < N; ++k) fill[k] = rp[k];
  for (int32_t j = 0; j < N; ++j)
    for (int64_t e = col_ptr[j]; e < col_ptr[j + 1]; ++e) {
      const int32_t k = row_idx[e];
      tj[fill[k]] = j;
      tw[fill[k]] = val[e];
      fill[k]++;
    }

  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if ((int64_t)nthreads > o->M) nthreads = o->M > 0 ? (int32_t)o->M : 1;
  layer_job jobs[256];
  pthread_t th[256];
  for (int t = 0; t < nthreads; ++t) {
    jobs[t].o = o; jobs[t].rp = rp; jobs[t].tj = tj; jobs[t].tw = tw; jobs[t].bias = bias;
    jobs[t].r0 = o->M * t / nthreads; jobs[t].r1 = o->M * (t + 1) / nthreads; jobs[t].rc = 0;
  }
  if (nthreads == 1) {
    layer_rows(&jobs[0]);
  } else {
    for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, layer_rows, &jobs[t]);
    for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  }
  int rc = 0;
  for (int t = 0; t < nthreads; ++t) if (jobs[t].rc) rc = jobs[t].rc;
  free(rp); free(tj); free(tw); free(fill);
  if (rc) return rc;

  if (o->nlayers + 2 > o->cap) {
    int64_t nc = o->cap * 2;
    int64_t *c = (int64_t *)realloc(o->counts, sizeof(int64_t) * (size_t)nc);
    if (!c) return -2;
    o->counts = c; o->cap = nc;
  }
  o->nlayers++;
  o->counts[o->nlayers] = count_live(o);
  return 0;
}

int64_t oracle_num_layers(void *h) { return ((oracle_t *)h)->nlayers; }

int64_t oracle_live_count(void *h) { return count_live((oracle_t *)h); }

/* counts[0..nlayers]: live rows entering each layer, and after the last one. */
void oracle_live_counts(void *h, int64_t *out) {
  oracle_t *o = (oracle_t *)h;
  memcpy(out, o->counts, sizeof(int64_t) * (size_t)(o->nlayers + 1));
}

/* Rows of the current Y with any entry > 0, ascending. ids may be NULL to count only. */
int64_t oracle_categories(void *h, int64_t *ids) {
  oracle_t *o = (oracle_t *)h;
  int64_t c = 0;
  for (int64_t i = 0; i < o->M; ++i) {
    const float *r = o->y + (size_t)i * o->N;
    int pos = 0;
    for (int32_t j = 0; j < o->N && !pos; ++j) pos = r[j] > 0.0f;
    if (pos) { if (ids) ids[c] = i; ++c; }
  }
  return c;
}

void oracle_rows(void *h, const int64_t *ids, int64_t n, float *out) {
  oracle_t *o = (oracle_t *)h;
  for (int64_t q = 0; q < n; ++q) memcpy(out + (size_t)q * o->N, o->y + (size_t)ids[q] * o->N, sizeof(float) * (size_t)o->N);
}

/* Smallest |z + b| seen over entries with z != 0 (per row into per_row if given, M entries). */
double oracle_margin(void *h, double *per_row) {
  oracle_t *o = (oracle_t *)h;
  double m = INFINITY;
  for (int64_t i = 0; i < o->M; ++i) {
    if (per_row) per_row[i] = o->margin[i];
    if (o->margin[i] < m) m = o->margin[i];
  }
  return m;
}

/* Smallest row maximum of the current Y over the rows with any entry > 0 (the categories);
   +infinity when there is none. */
double oracle_min_final_rowmax(void *h) {
  oracle_t *o = (oracle_t *)h;
  double m = INFINITY;
  for (int64_t i = 0; i < o->M; ++i) {
    const float *r = o->y + (size_t)i * o->N;
    float mx = 0.0f;
    for (int32_t j = 0; j < o->N; ++j) mx = r[j] > mx ? r[j] : mx;
    if (mx > 0.0f && (double)mx < m) m = (double)mx;
  }
  return m;
}
