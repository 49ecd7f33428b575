/*
 * Seeded synthetic workloads for the Sparse DNN Challenge inference (Kepner et al., 2019).
 *
 * This file generates INPUTS only: weight-layer sparsity patterns, bias tables and binary input
 * images. It performs none of the inference arithmetic. Both the CPU oracle and the GPU path read
 * what it writes, and nothing here depends on either of them.
 *
 * Random numbers: counter-based. Value i of a stream with 64-bit key k is
 *     mix64(k + (i + 1) * 0x9E3779B97F4A7C15)
 * where mix64 is the SplitMix64 output function (Steele, Lea and Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014). Keys are derived by chaining mix64 over
 * (root seed, purpose, network or input-set id, layer, permutation), so any single layer or image
 * can be regenerated on its own. Bounded integers use Lemire's multiply-and-reject method
 * ("Fast random integer generation in an interval", ACM TOMACS 2019).
 *
 * Weight layers (Sec. III, Tables 1-2: N neurons, 32 connections per neuron): each layer is the
 * union of K random permutation matrices. Permutation a is drawn by Fisher-Yates; a row i whose new
 * target sigma_a(i) repeats one of its earlier targets is repaired by swapping sigma_a(i) with
 * sigma_a(i') for a random partner i' such that both rows end collision-free. The result has
 * exactly K nonzeros in every row and every column and no duplicate (i, j). W(i, sigma_a(i)) is the
 * weight value passed in; the inference code must read it from memory.
 *
 * Input images (Sec. IV: binary R x R images flattened row-major into N = R*R features): the MNIST
 * set is not available, so three synthetic kinds stand in:
 *   kind 0 "strokes": per image a target density d = clip(mean + sd * g, 0.05, 0.40), g an
 *            Irwin-Hall(12) - 6 approximately-normal draw; polyline pen strokes (2-5 segments,
 *            lengths U(0.15R, 0.45R), heading turns U(-60, 60) degrees, round pen of radius
 *            max(1, round(R * U(0.03, 0.06)))) or, with probability 0.2, a filled rotated ellipse
 *            (semi-axes U(0.05R, 0.15R)), stamped until at least d*R*R pixels are set.
 *   kind 1 "bernoulli": every pixel independently 1 with probability p.
 *   kind 2 "mixed": per image a density U(lo, hi), then Bernoulli pixels.
 * Image n of a set depends only on (root, kind, set id, n), so a prefix of a set is the same
 * images as the start of a larger set of the same id.
 *
 * Floating point here is only for drawing shapes; sin/cos are evaluated by a fixed Taylor
 * polynomial (no libm) so the images are identical on every machine with IEEE doubles.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <pthread.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

enum { PURPOSE_PERM = 1, PURPOSE_REPAIR = 2, PURPOSE_INPUT = 3, PURPOSE_RADIX = 4 };

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t stream_value(uint64_t key, uint64_t i) { return mix64(key + (i + 1) * GOLDEN); }

static uint64_t derive_key(uint64_t root, uint64_t purpose, uint64_t a, uint64_t b, uint64_t c) {
  uint64_t k = mix64(root ^ mix64(purpose + GOLDEN));
  k = mix64(k ^ mix64(a + 2 * GOLDEN));
  k = mix64(k ^ mix64(b + 3 * GOLDEN));
  k = mix64(k ^ mix64(c + 4 * GOLDEN));
  return k;
}

/* Lemire: uniform integer in [0, range), range >= 1. Draws stream values *ctr, *ctr+1, ... */
static uint32_t bounded(uint64_t key, uint64_t *ctr, uint32_t range) {
  for (;;) {
    uint64_t x = stream_value(key, (*ctr)++);
    unsigned __int128 m = (unsigned __int128)x * range;
    uint64_t lo = (uint64_t)m;
    if (lo < range) {
      uint64_t t = (0 - (uint64_t)range) % range;
      if (lo < t) continue;
    }
    return (uint32_t)(m >> 64);
  }
}

/* uniform double in [0, 1) */
static inline double unit(uint64_t key, uint64_t *ctr) {
  return (double)(stream_value(key, (*ctr)++) >> 11) * (1.0 / 9007199254740992.0);
}

/* ---------------------------------------------------------------------------------------------- */
/* Weight layers                                                                                   */

/* Fills perm[a*N + i] = sigma_a(i) for a in [0, K). tgt is scratch of N*K int32.
   Returns 0, or -1 if K > N or a repair did not converge. */
static int layer_perms(uint64_t root, uint64_t net, uint64_t layer, int32_t N, int32_t K, int32_t *perm, int32_t *tgt) {
  if (K > N) return -1;
  for (int32_t a = 0; a < K; ++a) {
    int32_t *s = perm + (int64_t)a * N;
    uint64_t key = derive_key(root, PURPOSE_PERM, net, layer, (uint64_t)a);
    for (int32_t i = 0; i < N; ++i) s[i] = i;
    for (int32_t i = N - 1; i >= 1; --i) {
      uint64_t ctr = (uint64_t)i << 8;
      int32_t j = (int32_t)bounded(key, &ctr, (uint32_t)i + 1);
      int32_t t = s[i]; s[i] = s[j]; s[j] = t;
    }
    if (a > 0) {
      uint64_t rkey = derive_key(root, PURPOSE_REPAIR, net, layer, (uint64_t)a);
      uint64_t rctr = 0;
      for (int32_t i = 0; i < N; ++i) {
        const int32_t *ti = tgt + (int64_t)i * K;
        int hit = 0;
        for (int32_t b = 0; b < a; ++b) hit |= (ti[b] == s[i]);
        if (!hit) continue;
        int64_t tries = 0;
        for (;;) {
          if (++tries > 100000) return -1;
          int32_t p = (int32_t)bounded(rkey, &rctr, (uint32_t)N);
          if (p == i) continue;
          const int32_t *tp = tgt + (int64_t)p * K;
          int ok = 1;
          for (int32_t b = 0; b < a && ok; ++b) ok = (ti[b] != s[p]) && (tp[b] != s[i]);
          if (!ok) continue;
          int32_t t = s[i]; s[i] = s[p]; s[p] = t;
          break;
        }
      }
    }
    for (int32_t i = 0; i < N; ++i) tgt[(int64_t)i * K + a] = s[i];
  }
  return 0;
}

int synth_layer_perms(uint64_t root, uint64_t net, uint64_t layer, int32_t N, int32_t K, int32_t *perm) {
  if (N <= 0 || K <= 0) return -1;
  int32_t *tgt = (int32_t *)malloc(sizeof(int32_t) * (size_t)N * (size_t)K);
  if (!tgt) return -2;
  int rc = layer_perms(root, net, layer, N, K, perm, tgt);
  free(tgt);
  return rc;
}

/* One layer in CSC form: column j holds sources {i : sigma_a(i) = j}, sorted ascending.
   col_ptr[j] = base + j*K (so a chunk of layers stays contiguous), row_idx/val of length N*K.
   perm is reused to hold the inverse permutations after the draw. */
static int layer_csc(uint64_t root, uint64_t net, uint64_t layer, int32_t N, int32_t K, float wval, int64_t base,
                     int64_t *col_ptr, int32_t *row_idx, float *val, int32_t *perm, int32_t *tgt) {
  int rc = layer_perms(root, net, layer, N, K, perm, tgt);
  if (rc) return rc;
  /* tgt <- inverse permutations, [a][j] = i with sigma_a(i) = j */
  for (int32_t a = 0; a < K; ++a) {
    const int32_t *s = perm + (int64_t)a * N;
    int32_t *inv = tgt + (int64_t)a * N;
    for (int32_t i = 0; i < N; ++i) inv[s[i]] = i;
  }
  for (int32_t j = 0; j < N; ++j) {
    int32_t *c = row_idx + (int64_t)j * K;
    for (int32_t a = 0; a < K; ++a) c[a] = tgt[(int64_t)a * N + j];
    for (int32_t x = 1; x < K; ++x) { /* insertion sort, K is small */
      int32_t v = c[x], y = x - 1;
      while (y >= 0 && c[y] > v) { c[y + 1] = c[y]; --y; }
      c[y + 1] = v;
    }
    col_ptr[j] = base + (int64_t)j * K;
  }
  col_ptr[N] = base + (int64_t)N * K;
  for (int64_t e = 0; e < (int64_t)N * K; ++e) val[e] = wval;
  return 0;
}

typedef struct {
  uint64_t root, net; int32_t l0, nl, N, K; float wval;
  int64_t *col_ptr; int32_t *row_idx; float *val;
  int next; pthread_mutex_t mu; int rc;
} layers_job;

static void *layers_worker(void *arg) {
  layers_job *J = (layers_job *)arg;
  int32_t *perm = (int32_t *)malloc(sizeof(int32_t) * (size_t)J->N * (size_t)J->K);
  int32_t *tgt = (int32_t *)malloc(sizeof(int32_t) * (size_t)J->N * (size_t)J->K);
  if (!perm || !tgt) { pthread_mutex_lock(&J->mu); J->rc = -2; pthread_mutex_unlock(&J->mu); free(perm); free(tgt); return NULL; }
  for (;;) {
    pthread_mutex_lock(&J->mu);
    int i = J->next++;
    int stop = J->rc != 0;
    pthread_mutex_unlock(&J->mu);
    if (stop || i >= J->nl) break;
    int64_t nnz = (int64_t)J->N * J->K;
    int rc = layer_csc(J->root, J->net, (uint64_t)(J->l0 + i), J->N, J->K, J->wval, (int64_t)i * nnz,
                       J->col_ptr + (int64_t)i * (J->N + 1), J->row_idx + (int64_t)i * nnz, J->val + (int64_t)i * nnz, perm, tgt);
    if (rc) { pthread_mutex_lock(&J->mu); J->rc = rc; pthread_mutex_unlock(&J->mu); }
  }
  free(perm); free(tgt);
  return NULL;
}

/* Layers [l0, l0+nl) of network `net`, in CSC, layer i's offsets continuing layer i-1's:
   col_ptr: nl*(N+1) int64, row_idx: nl*N*K int32, val: nl*N*K float. Returns 0 on success. */
int synth_layers_csc(uint64_t root, uint64_t net, int32_t l0, int32_t nl, int32_t N, int32_t K, float wval,
                     int64_t *col_ptr, int32_t *row_idx, float *val, int32_t nthreads) {
  if (N <= 0 || K <= 0 || K > N || nl < 0 || l0 < 0) return -1;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > nl) nthreads = nl > 0 ? nl : 1;
  layers_job J = {root, net, l0, nl, N, K, wval, col_ptr, row_idx, val, 0, PTHREAD_MUTEX_INITIALIZER, 0};
  pthread_t th[256];
  if (nthreads > 256) nthreads = 256;
  for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, layers_worker, &J);
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  return J.rc;
}

/* ---------------------------------------------------------------------------------------------- */
/* Structured (RadiX-Net style) weight layers                                                      */
/*
 * Sec. III, Fig. 1 and Table 1 describe the challenge's networks: a base DNN from a radix set of D
 * radices 2 (2^D nodes per layer, 2 connections per node), expanded by a Kronecker product with
 * 16 x 16 blocks into N = 16 * 2^D neurons with 32 connections each, then made deep by appending
 * randomly permuted copies of the base DNN. The construction of the base layers belongs to the
 * RadiX-Net paper, which is not at hand; this generator takes the mixed-radix reading: base layer i
 * links node u to u and to u + 2^i (mod 2^D), so that within one copy of D layers every input node
 * reaches every output node by exactly one path. After the Kronecker product neuron 16u + a feeds
 * neuron 16v + b for all a, b whenever u links to v. Copy c (layers cD .. cD + D - 1) is relabelled
 * by a random permutation P_c of the N neurons: W_l(P_c(s), P_c(t)) = B_{l mod D}(s, t). P_c is drawn
 * by Fisher-Yates from the stream of (root, PURPOSE_RADIX, net, c).
 */

/* D with N = 16 * 2^D, or -1 */
static int radix_depth(int32_t N) {
  if (N < 32 || (N & 15) != 0) return -1;
  int32_t nodes = N / 16, d = 0;
  while ((1 << d) < nodes) ++d;
  return (1 << d) == nodes ? d : -1;
}

/* perm[x] = P_c(x) for copy c; returns 0, or -1 if N is not 16 * 2^D with D >= 1 */
int synth_radix_perm(uint64_t root, uint64_t net, uint64_t copy, int32_t N, int32_t *perm) {
  if (radix_depth(N) < 1) return -1;
  uint64_t key = derive_key(root, PURPOSE_RADIX, net, copy, 0);
  for (int32_t i = 0; i < N; ++i) perm[i] = i;
  for (int32_t i = N - 1; i >= 1; --i) {
    uint64_t ctr = (uint64_t)i << 8;
    int32_t j = (int32_t)bounded(key, &ctr, (uint32_t)i + 1);
    int32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t;
  }
  return 0;
}

/* One structured layer in CSC form (sources ascending per column), col_ptr[j] = base + 32 j. perm and
   inv are scratch of N int32 each. */
static int radix_layer_csc(uint64_t root, uint64_t net, uint64_t layer, int32_t N, float wval, int64_t base,
                           int64_t *col_ptr, int32_t *row_idx, float *val, int32_t *perm, int32_t *inv) {
  const int D = radix_depth(N);
  if (D < 1) return -1;
  const uint64_t copy = layer / (uint64_t)D;
  const int32_t i = (int32_t)(layer % (uint64_t)D), nodes = N / 16;
  int rc = synth_radix_perm(root, net, copy, N, perm);
  if (rc) return rc;
  for (int32_t x = 0; x < N; ++x) inv[perm[x]] = x;
  for (int32_t j = 0; j < N; ++j) {
    /* column j is relabelled neuron t = 16 v + b; its base sources are nodes v and v - 2^i */
    const int32_t t = inv[j], v = t / 16;
    const int32_t u[2] = {v, (v - (1 << i) + nodes) % nodes};
    int32_t *c = row_idx + (int64_t)j * 32;
    for (int32_t k = 0; k < 2; ++k)
      for (int32_t a = 0; a < 16; ++a) c[16 * k + a] = perm[16 * u[k] + a];
    for (int32_t x = 1; x < 32; ++x) { /* insertion sort */
      int32_t w = c[x], y = x - 1;
      while (y >= 0 && c[y] > w) { c[y + 1] = c[y]; --y; }
      c[y + 1] = w;
    }
    col_ptr[j] = base + (int64_t)j * 32;
  }
  col_ptr[N] = base + (int64_t)N * 32;
  for (int64_t e = 0; e < (int64_t)N * 32; ++e) val[e] = wval;
  return 0;
}

typedef struct {
  uint64_t root, net; int32_t l0, nl, N; float wval;
  int64_t *col_ptr; int32_t *row_idx; float *val;
  int next; pthread_mutex_t mu; int rc;
} radix_job;

static void *radix_worker(void *arg) {
  radix_job *J = (radix_job *)arg;
  int32_t *perm = (int32_t *)malloc(sizeof(int32_t) * (size_t)J->N);
  int32_t *inv = (int32_t *)malloc(sizeof(int32_t) * (size_t)J->N);
  if (!perm || !inv) { pthread_mutex_lock(&J->mu); J->rc = -2; pthread_mutex_unlock(&J->mu); free(perm); free(inv); return NULL; }
  for (;;) {
    pthread_mutex_lock(&J->mu);
    int i = J->next++;
    int stop = J->rc != 0;
    pthread_mutex_unlock(&J->mu);
    if (stop || i >= J->nl) break;
    int64_t nnz = (int64_t)J->N * 32;
    int rc = radix_layer_csc(J->root, J->net, (uint64_t)(J->l0 + i), J->N, J->wval, (int64_t)i * nnz,
                             J->col_ptr + (int64_t)i * (J->N + 1), J->row_idx + (int64_t)i * nnz, J->val + (int64_t)i * nnz,
                             perm, inv);
    if (rc) { pthread_mutex_lock(&J->mu); J->rc = rc; pthread_mutex_unlock(&J->mu); }
  }
  free(perm); free(inv);
  return NULL;
}

/* Structured layers [l0, l0+nl) of network `net` (N = 16 * 2^D), in the layout of synth_layers_csc
   with K = 32. Returns 0 on success. */
int synth_radix_layers_csc(uint64_t root, uint64_t net, int32_t l0, int32_t nl, int32_t N, float wval,
                           int64_t *col_ptr, int32_t *row_idx, float *val, int32_t nthreads) {
  if (radix_depth(N) < 1 || nl < 0 || l0 < 0) return -1;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > nl) nthreads = nl > 0 ? nl : 1;
  radix_job J = {root, net, l0, nl, N, wval, col_ptr, row_idx, val, 0, PTHREAD_MUTEX_INITIALIZER, 0};
  pthread_t th[256];
  if (nthreads > 256) nthreads = 256;
  for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, radix_worker, &J);
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  return J.rc;
}

/* ---------------------------------------------------------------------------------------------- */
/* Input images                                                                                    */

static const double PI = 3.14159265358979323846;

/* sin/cos by Taylor series after reduction to [-pi, pi]; deterministic, ~1e-15 accurate */
static double dsin(double x) {
  double k = (double)(int64_t)(x / (2 * PI));
  x -= k * 2 * PI;
  if (x > PI) x -= 2 * PI;
  if (x < -PI) x += 2 * PI;
  double term = x, sum = x, x2 = x * x;
  for (int n = 1; n < 14; ++n) { term *= -x2 / ((2.0 * n) * (2.0 * n + 1)); sum += term; }
  return sum;
}
static double dcos(double x) { return dsin(x + PI / 2); }

static inline int64_t iround(double v) { return (int64_t)(v < 0 ? v - 0.5 : v + 0.5); }

/* Set every pixel whose center lies within rad of the segment (x0,y0)-(x1,y1): a pen stroke of
   radius rad (the union of discs centered on the segment). Returns the number of new ones. */
static int64_t stamp_capsule(float *img, int32_t R, double x0, double y0, double x1, double y1, int32_t rad) {
  int64_t added = 0;
  const double dx = x1 - x0, dy = y1 - y0, len2 = dx * dx + dy * dy, r2 = (double)rad * rad;
  int64_t xa = (int64_t)(x0 < x1 ? x0 : x1) - rad - 1, xb = (int64_t)(x0 > x1 ? x0 : x1) + rad + 1;
  int64_t ya = (int64_t)(y0 < y1 ? y0 : y1) - rad - 1, yb = (int64_t)(y0 > y1 ? y0 : y1) + rad + 1;
  if (xa < 0) xa = 0;
  if (ya < 0) ya = 0;
  if (xb > R - 1) xb = R - 1;
  if (yb > R - 1) yb = R - 1;
  for (int64_t y = ya; y <= yb; ++y)
    for (int64_t x = xa; x <= xb; ++x) {
      double t = len2 > 0 ? ((x - x0) * dx + (y - y0) * dy) / len2 : 0.0;
      if (t < 0) t = 0;
      if (t > 1) t = 1;
      const double ex = x - (x0 + t * dx), ey = y - (y0 + t * dy);
      if (ex * ex + ey * ey > r2) continue;
      float *p = img + y * R + x;
      if (*p == 0.0f) { *p = 1.0f; ++added; }
    }
  return added;
}

static void image_strokes(uint64_t key, int32_t R, double mean, double sd, float *img) {
  uint64_t ctr = 0;
  double g = -6.0;
  for (int q = 0; q < 12; ++q) g += unit(key, &ctr);
  double d = mean + sd * g;
  if (d < 0.05) d = 0.05;
  if (d > 0.40) d = 0.40;
  int64_t target = (int64_t)(d * (double)R * (double)R);
  if (target < 1) target = 1;
  int64_t ones = 0;
  for (int shape = 0; shape < 400 && ones < target; ++shape) {
    if (unit(key, &ctr) < 0.2) {
      double cx = R * (0.2 + 0.6 * unit(key, &ctr)), cy = R * (0.2 + 0.6 * unit(key, &ctr));
      double a = R * (0.05 + 0.10 * unit(key, &ctr)), b = R * (0.05 + 0.10 * unit(key, &ctr));
      double th = PI * unit(key, &ctr), c = dcos(th), s = dsin(th);
      int64_t ext = (int64_t)(a > b ? a : b) + 1;
      for (int64_t y = iround(cy) - ext; y <= iround(cy) + ext; ++y)
        for (int64_t x = iround(cx) - ext; x <= iround(cx) + ext; ++x) {
          if (x < 0 || y < 0 || x >= R || y >= R) continue;
          double u = (x - cx) * c + (y - cy) * s, v = -(x - cx) * s + (y - cy) * c;
          if ((u / a) * (u / a) + (v / b) * (v / b) <= 1.0) {
            float *p = img + y * R + x;
            if (*p == 0.0f) { *p = 1.0f; ++ones; }
          }
        }
    } else {
      double x = R * (0.15 + 0.70 * unit(key, &ctr)), y = R * (0.15 + 0.70 * unit(key, &ctr));
      double h = 2 * PI * unit(key, &ctr);
      int32_t rad = (int32_t)iround(R * (0.03 + 0.03 * unit(key, &ctr)));
      if (rad < 1) rad = 1;
      int nseg = 2 + (int)bounded(key, &ctr, 4);
      for (int sgm = 0; sgm < nseg; ++sgm) {
        double len = R * (0.15 + 0.30 * unit(key, &ctr));
        double dx = dcos(h), dy = dsin(h);
        ones += stamp_capsule(img, R, x, y, x + len * dx, y + len * dy, rad);
        x += len * dx; y += len * dy;
        if (x < 0) x = 0;
        if (y < 0) y = 0;
        if (x > R - 1) x = R - 1;
        if (y > R - 1) y = R - 1;
        h += (unit(key, &ctr) * 2.0 - 1.0) * (PI / 3.0);
      }
    }
  }
}

static void image_bernoulli(uint64_t key, int64_t n, double p, float *img) {
  uint64_t ctr = 1; /* value 0 reserved for a per-image density draw */
  for (int64_t i = 0; i < n; ++i) img[i] = unit(key, &ctr) < p ? 1.0f : 0.0f;
}

typedef struct {
  uint64_t root, set; int32_t kind, R; int64_t row0, nrows; double pa, pb; float *out;
  int64_t next; pthread_mutex_t mu;
} inputs_job;

static void make_image(const inputs_job *J, int64_t r) {
  int64_t n = (int64_t)J->R * J->R;
  float *img = J->out + r * n;
  uint64_t idx = (uint64_t)(J->row0 + r);
  uint64_t key = derive_key(J->root, PURPOSE_INPUT, (uint64_t)J->kind, J->set, idx);
  memset(img, 0, sizeof(float) * (size_t)n);
  if (J->kind == 0) {
    image_strokes(key, J->R, J->pa, J->pb, img);
  } else if (J->kind == 1) {
    image_bernoulli(key, n, J->pa, img);
  } else {
    uint64_t c0 = 0;
    double p = J->pa + (J->pb - J->pa) * unit(key, &c0);
    image_bernoulli(key, n, p, img);
  }
}

static void *inputs_worker(void *arg) {
  inputs_job *J = (inputs_job *)arg;
  for (;;) {
    pthread_mutex_lock(&J->mu);
    int64_t r0 = J->next;
    J->next += 16;
    pthread_mutex_unlock(&J->mu);
    if (r0 >= J->nrows) break;
    int64_t r1 = r0 + 16 < J->nrows ? r0 + 16 : J->nrows;
    for (int64_t r = r0; r < r1; ++r) make_image(J, r);
  }
  return NULL;
}

/* Images [row0, row0+nrows) of input set `set`, written densely: out[r*R*R + y*R + x] in {0, 1}.
   kind 0: strokes with density mean pa, sd pb; kind 1: Bernoulli(pa); kind 2: Bernoulli(U(pa, pb)). */
int synth_inputs(uint64_t root, uint64_t set, int32_t kind, int32_t R, int64_t row0, int64_t nrows,
                 double pa, double pb, float *out, int32_t nthreads) {
  if (R <= 0 || nrows < 0 || row0 < 0 || kind < 0 || kind > 2) return -1;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  inputs_job J = {root, set, kind, R, row0, nrows, pa, pb, out, 0, PTHREAD_MUTEX_INITIALIZER};
  pthread_t th[256];
  for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, inputs_worker, &J);
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  return 0;
}

/* Exposed for tests of the generator itself. */
uint64_t synth_stream_value(uint64_t key, uint64_t i) { return stream_value(key, i); }
uint64_t synth_mix64(uint64_t z) { return mix64(z); }
