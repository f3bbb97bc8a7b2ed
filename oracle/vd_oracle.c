/*
 * vd_oracle.c -- plain, slow CPU oracle for paged causal attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the GPU path: it reads bf16 bit patterns and
 * page tables in its own plain layout and computes in IEEE double.
 *
 * What it computes (the problem statement of Appendix A.1 of the paper,
 * "Properties and Logical Inputs", and the causal contract of Section 5.3):
 *
 *   An invocation holds num_seqs requests.  Request r has query length
 *   s_r = cu_q_lens[r+1] - cu_q_lens[r] and key length n_r = context_lens[r],
 *   with 0 < s_r <= n_r.  Its query row i (0 <= i < s_r) stands for logical
 *   position p = n_r - s_r + i.
 *
 *   Logical keys and values come from the physical pool through the request's
 *   page table pi_r:  K[j,:] = Kphys[pi_r(floor(j/P)), kv_head, j mod P, :]
 *   (the pool here is laid out [page][kv_head][slot][d]).
 *
 *   Query head h reads KV head floor(h / (Hq/Hkv)) (contiguous GQA groups;
 *   the paper does not fix the grouping, this is the usual convention).
 *
 *   For each selected row and head:
 *       score_j = scale * sum_d q[d] * K[j,d]           for j = 0..p
 *       w_j     = exp(score_j - max_j score) / sum_j exp(score_j - max_j score)
 *       out[d]  = sum_j w_j * V[j,d]
 *   which is exactly softmax attention restricted to the causal prefix
 *   j <= p (the mask of Appendix A.2 reduces to j <= p because p < n).
 *
 *   Optionally also the row's log-sum-exp (the normaliser the paper's tile
 *   update carries as (m, z), Appendix A.2; the paper does not export it):
 *       lse = log sum_j exp(score_j) = max_j score_j + log sum_j exp(score_j - max)
 *   in natural log, over the same visible keys.
 *
 *   Sliding-window attention (Appendix A.5, "Relational Alignment and
 *   Composition"): with a window size w > 0 shared by the call, key j is
 *   visible to position p only when also j > p - w, so the sums above run
 *   over j = max(0, p - w + 1) .. p.  w = 0 means no window (the full
 *   causal prefix).
 *
 * Every sum runs in ascending index order in double precision.  No blocking,
 * no online softmax, no splitting: the definition written out.
 *
 * Linear layer (the matmul contract of Section 5.4, Fig. 3: the output row
 * of a token depends only on that token's input row and the weights):
 *       c[m][n] = sum_k a[m][k] * b[n][k]      for k = 0..K-1
 *   with a the activations [M][K] and b the weights [N][K] (one row per output
 *   column, as a linear layer stores them), in double, k ascending.
 *
 * Error behaviour: returns 0 on success, a negative code on invalid input
 * (nothing is written to `out` for a rejected call).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#define VDO_OK 0
#define VDO_ERR_ARG (-1)
#define VDO_ERR_LENGTHS (-2)
#define VDO_ERR_PAGE (-3)
#define VDO_ERR_NOMEM (-4)

/* bf16 is the top half of an IEEE binary32; widening is exact. */
static double bf16_to_double(uint16_t bits) {
  uint32_t u = ((uint32_t)bits) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

typedef struct {
  int num_seqs;
  int64_t total_q_tokens;
  int hq, hkv, d, page_size;
  double scale;
  int window; /* 0: full causal prefix; w > 0: keys p - w < j <= p */
  const uint16_t *q;
  const int32_t *cu_q_lens, *context_lens, *page_table;
  int pt_stride;
  const uint16_t *k_pool, *v_pool;
  int64_t num_pages;
  const uint8_t *row_select;
  double *out;
  double *lse; /* optional [T, Hq] */
  /* work queue over (request, q-head) pairs */
  int64_t next_item;
  pthread_mutex_t lock;
} job_t;

/* One (request, query head) pair: every selected row of that request. */
static int run_item(job_t *J, int r, int h, double *score, double *w) {
  const int D = J->d, P = J->page_size;
  const int group = J->hq / J->hkv;
  const int g = h / group;
  const int32_t q0 = J->cu_q_lens[r];
  const int s = J->cu_q_lens[r + 1] - q0;
  const int n = J->context_lens[r];
  const int32_t *pt = J->page_table + (int64_t)r * J->pt_stride;

  for (int i = 0; i < s; ++i) {
    const int64_t t = (int64_t)q0 + i;
    if (J->row_select && !J->row_select[t]) continue;
    const int p = n - s + i; /* logical position of this row */
    /* first visible key: 0, or the start of the sliding window */
    const int lo = (J->window > 0 && p - J->window + 1 > 0) ? p - J->window + 1 : 0;
    const uint16_t *qrow = J->q + (t * J->hq + h) * (int64_t)D;

    /* scores over the visible keys j = lo..p */
    for (int j = lo; j <= p; ++j) {
      const int64_t page = pt[j / P];
      const uint16_t *krow =
          J->k_pool + (((page * J->hkv + g) * P) + (j % P)) * (int64_t)D;
      double acc = 0.0;
      for (int dd = 0; dd < D; ++dd)
        acc += bf16_to_double(qrow[dd]) * bf16_to_double(krow[dd]);
      score[j] = J->scale * acc;
    }
    /* softmax */
    double mx = -INFINITY;
    for (int j = lo; j <= p; ++j)
      if (score[j] > mx) mx = score[j];
    double denom = 0.0;
    for (int j = lo; j <= p; ++j) {
      w[j] = exp(score[j] - mx);
      denom += w[j];
    }
    for (int j = lo; j <= p; ++j) w[j] /= denom;
    if (J->lse) J->lse[t * J->hq + h] = mx + log(denom);
    /* weighted sum of values */
    double *orow = J->out + (t * J->hq + h) * (int64_t)D;
    for (int dd = 0; dd < D; ++dd) orow[dd] = 0.0;
    for (int j = lo; j <= p; ++j) {
      const int64_t page = pt[j / P];
      const uint16_t *vrow =
          J->v_pool + (((page * J->hkv + g) * P) + (j % P)) * (int64_t)D;
      for (int dd = 0; dd < D; ++dd) orow[dd] += w[j] * bf16_to_double(vrow[dd]);
    }
  }
  return 0;
}

static void *worker(void *arg) {
  job_t *J = (job_t *)arg;
  int maxn = 1;
  for (int r = 0; r < J->num_seqs; ++r)
    if (J->context_lens[r] > maxn) maxn = J->context_lens[r];
  double *score = (double *)malloc(sizeof(double) * (size_t)maxn);
  double *w = (double *)malloc(sizeof(double) * (size_t)maxn);
  if (!score || !w) {
    free(score);
    free(w);
    return (void *)1;
  }
  const int64_t items = (int64_t)J->num_seqs * J->hq;
  for (;;) {
    pthread_mutex_lock(&J->lock);
    int64_t it = J->next_item++;
    pthread_mutex_unlock(&J->lock);
    if (it >= items) break;
    run_item(J, (int)(it / J->hq), (int)(it % J->hq), score, w);
  }
  free(score);
  free(w);
  return NULL;
}

/* Validates the logical inputs before anything is computed. */
static int validate(const job_t *J) {
  if (J->num_seqs < 0 || J->hq <= 0 || J->hkv <= 0 || J->d <= 0 ||
      J->page_size <= 0 || J->hq % J->hkv != 0 || J->pt_stride < 0 ||
      J->window < 0)
    return VDO_ERR_ARG;
  if (J->cu_q_lens[0] != 0 || J->cu_q_lens[J->num_seqs] != J->total_q_tokens)
    return VDO_ERR_LENGTHS;
  for (int r = 0; r < J->num_seqs; ++r) {
    const int s = J->cu_q_lens[r + 1] - J->cu_q_lens[r];
    const int n = J->context_lens[r];
    if (s < 1 || s > n) return VDO_ERR_LENGTHS;
    const int npages = (n + J->page_size - 1) / J->page_size;
    if (npages > J->pt_stride) return VDO_ERR_LENGTHS;
    for (int b = 0; b < npages; ++b) {
      const int32_t pg = J->page_table[(int64_t)r * J->pt_stride + b];
      if (pg < 0 || pg >= J->num_pages) return VDO_ERR_PAGE;
    }
  }
  return VDO_OK;
}

/* window: 0 for the full causal prefix, w > 0 for a sliding window of w keys;
 * lse: optional [T, Hq] output of the rows' log-sum-exp (NULL: not written) */
int vdo_paged_attention(int num_seqs, int64_t total_q_tokens, int num_q_heads,
                        int num_kv_heads, int head_dim, int page_size,
                        double scale, int window, const uint16_t *q,
                        const int32_t *cu_q_lens, const int32_t *context_lens,
                        const int32_t *page_table, int pt_stride,
                        const uint16_t *k_pool, const uint16_t *v_pool,
                        int64_t num_pages, const uint8_t *row_select,
                        double *out, double *lse, int num_threads) {
  if (!q || !cu_q_lens || !context_lens || !page_table || !k_pool || !v_pool ||
      !out)
    return VDO_ERR_ARG;
  job_t J;
  memset(&J, 0, sizeof J);
  J.num_seqs = num_seqs;
  J.total_q_tokens = total_q_tokens;
  J.hq = num_q_heads;
  J.hkv = num_kv_heads;
  J.d = head_dim;
  J.page_size = page_size;
  J.scale = scale;
  J.window = window;
  J.q = q;
  J.cu_q_lens = cu_q_lens;
  J.context_lens = context_lens;
  J.page_table = page_table;
  J.pt_stride = pt_stride;
  J.k_pool = k_pool;
  J.v_pool = v_pool;
  J.num_pages = num_pages;
  J.row_select = row_select;
  J.out = out;
  J.lse = lse;
  int rc = validate(&J);
  if (rc != VDO_OK) return rc;

  if (num_threads <= 0) num_threads = (int)sysconf(_SC_NPROCESSORS_ONLN);
  if (num_threads < 1) num_threads = 1;
  pthread_mutex_init(&J.lock, NULL);
  pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)num_threads);
  if (!th) return VDO_ERR_NOMEM;
  int started = 0;
  for (int i = 0; i < num_threads; ++i)
    if (pthread_create(&th[i], NULL, worker, &J) == 0) ++started;
  int failed = started == 0;
  for (int i = 0; i < started; ++i) {
    void *ret = NULL;
    pthread_join(th[i], &ret);
    if (ret) failed = 1;
  }
  free(th);
  pthread_mutex_destroy(&J.lock);
  return failed ? VDO_ERR_NOMEM : VDO_OK;
}

/* The same attention for one request whose keys and values are contiguous,
 * with no page table: q [s][hq][d], k and v [n][hkv][d] (bf16 bits); row i
 * is position p = n - s + i; out [s][hq][d] in double, lse [s][hq] optional
 * (NULL: not written).  Single-threaded; the definition written out again,
 * so that the page-table gather of vdo_paged_attention can be checked
 * against it. */
int vdo_dense_attention(int s, int n, int num_q_heads, int num_kv_heads,
                        int head_dim, double scale, int window,
                        const uint16_t *q, const uint16_t *k, const uint16_t *v,
                        double *out, double *lse) {
  if (!q || !k || !v || !out) return VDO_ERR_ARG;
  if (num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0 ||
      num_q_heads % num_kv_heads != 0 || window < 0)
    return VDO_ERR_ARG;
  if (s < 1 || s > n) return VDO_ERR_LENGTHS;
  const int hq = num_q_heads, hkv = num_kv_heads, D = head_dim;
  double *score = (double *)malloc(sizeof(double) * (size_t)n);
  double *w = (double *)malloc(sizeof(double) * (size_t)n);
  if (!score || !w) {
    free(score);
    free(w);
    return VDO_ERR_NOMEM;
  }
  for (int i = 0; i < s; ++i) {
    const int p = i + (n - s); /* position of row i */
    const int lo = (window > 0 && p - window + 1 > 0) ? p - window + 1 : 0;
    for (int h = 0; h < hq; ++h) {
      const int g = h / (hq / hkv);
      const uint16_t *qrow = q + ((int64_t)i * hq + h) * D;
      for (int j = lo; j <= p; ++j) {
        const uint16_t *krow = k + ((int64_t)j * hkv + g) * D;
        double acc = 0.0;
        for (int dd = 0; dd < D; ++dd)
          acc += bf16_to_double(qrow[dd]) * bf16_to_double(krow[dd]);
        score[j] = scale * acc;
      }
      double mx = -INFINITY;
      for (int j = lo; j <= p; ++j)
        if (score[j] > mx) mx = score[j];
      double denom = 0.0;
      for (int j = lo; j <= p; ++j) {
        w[j] = exp(score[j] - mx);
        denom += w[j];
      }
      for (int j = lo; j <= p; ++j) w[j] = w[j] / denom;
      if (lse) lse[(int64_t)i * hq + h] = mx + log(denom);
      double *orow = out + ((int64_t)i * hq + h) * D;
      for (int dd = 0; dd < D; ++dd) orow[dd] = 0.0;
      for (int j = lo; j <= p; ++j) {
        const uint16_t *vrow = v + ((int64_t)j * hkv + g) * D;
        for (int dd = 0; dd < D; ++dd) orow[dd] += w[j] * bf16_to_double(vrow[dd]);
      }
    }
  }
  free(score);
  free(w);
  return VDO_OK;
}

/* Number of host threads the oracle uses when asked for "all cores". */
int vdo_default_threads(void) { return (int)sysconf(_SC_NPROCESSORS_ONLN); }

/* ------------------------------------------------------------------------ */
/* Linear layer: c[m][n] = sum_k a[m][k] * b[n][k], k ascending, in double.
 * a: M rows of lda bf16 values (the first K used), b: N rows of ldb bf16
 * values (the first K used), c: M rows of N doubles.  Returns 0, or
 * VDO_ERR_ARG for an invalid size or stride. */
typedef struct {
  int64_t M;
  int N, K;
  const uint16_t *a, *b;
  int64_t lda, ldb;
  double *c;
  int64_t next_row;
  pthread_mutex_t lock;
} lin_job_t;

static void *lin_worker(void *arg) {
  lin_job_t *J = (lin_job_t *)arg;
  for (;;) {
    pthread_mutex_lock(&J->lock);
    const int64_t m = J->next_row++;
    pthread_mutex_unlock(&J->lock);
    if (m >= J->M) break;
    const uint16_t *arow = J->a + m * J->lda;
    double *crow = J->c + m * (int64_t)J->N;
    for (int n = 0; n < J->N; ++n) {
      const uint16_t *brow = J->b + (int64_t)n * J->ldb;
      double acc = 0.0;
      for (int k = 0; k < J->K; ++k)
        acc += bf16_to_double(arow[k]) * bf16_to_double(brow[k]);
      crow[n] = acc;
    }
  }
  return NULL;
}

int vdo_linear(int64_t M, int N, int K, const uint16_t *a, int64_t lda,
               const uint16_t *b, int64_t ldb, double *c, int num_threads) {
  if (M < 0 || N < 0 || K < 0 || lda < K || ldb < K) return VDO_ERR_ARG;
  if (M == 0 || N == 0) return VDO_OK;
  if (!a || !b || !c) return VDO_ERR_ARG;
  lin_job_t J;
  memset(&J, 0, sizeof J);
  J.M = M;
  J.N = N;
  J.K = K;
  J.a = a;
  J.b = b;
  J.lda = lda;
  J.ldb = ldb;
  J.c = c;
  if (num_threads <= 0) num_threads = (int)sysconf(_SC_NPROCESSORS_ONLN);
  if (num_threads < 1) num_threads = 1;
  pthread_mutex_init(&J.lock, NULL);
  pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)num_threads);
  if (!th) return VDO_ERR_NOMEM;
  int started = 0;
  for (int i = 0; i < num_threads; ++i)
    if (pthread_create(&th[i], NULL, lin_worker, &J) == 0) ++started;
  for (int i = 0; i < started; ++i) pthread_join(th[i], NULL);
  free(th);
  pthread_mutex_destroy(&J.lock);
  return started ? VDO_OK : VDO_ERR_NOMEM;
}
