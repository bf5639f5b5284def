/*
 * Plain fp64 CPU oracle for causal top-k sparse GQA prefill.
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg load this file's library. The GPU library
 * shares no code, header, table or helper with it.
 *
 * Every function is row-separable: it computes the requested query rows
 * (or selection blocks) only, so any subset of a long sequence can be
 * checked exactly. All arithmetic is double precision, written as the
 * paper's definitions with no blocking, fusion or reordering.
 *
 * Notation (0-based): S tokens, Hq query heads, Hkv KV heads, G = Hq/Hkv,
 * g(h) = floor(h/G), d head dim, d_idx indexer dim, k budget, b selection
 * block size, block r = queries [r*b, min(r*b+b, S)).
 * Layouts: q [S,Hq,d], k and v [S,Hkv,d], q_idx and k_idx [S,d_idx].
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_AGG_MAX 0
#define ORC_AGG_SUM 1

/* Logits of one query row t for one head h against keys 0..t:
 * l[s] = scale * <q[t,h,:], k[s,g(h),:]>  (Section 3, dense GQA attention). */
static void logits_row(int Hq, int Hkv, int d, double scale, const double *q,
                       const double *k, int t, int h, double *l) {
  int G = Hq / Hkv;
  int j = h / G;
  const double *qt = q + ((size_t)t * Hq + h) * d;
  for (int s = 0; s <= t; ++s) {
    const double *ks = k + ((size_t)s * Hkv + j) * d;
    double acc = 0.0;
    for (int c = 0; c < d; ++c) acc += qt[c] * ks[c];
    l[s] = scale * acc;
  }
}

/* Softmax normaliser: log sum_{s<=t} exp(l[s]), computed with the max shift. */
static double log_normaliser(const double *l, int n) {
  double m = -INFINITY;
  for (int s = 0; s < n; ++s) m = l[s] > m ? l[s] : m;
  double z = 0.0;
  for (int s = 0; s < n; ++s) z += exp(l[s] - m);
  return m + log(z);
}

/*
 * Dense causal GQA attention (Section 3, first equation):
 *   A[t,h,s] = softmax_{s'<=t}(<q_{t,h}, k_{s',g(h)}> * scale)_s
 *   o[t,h]   = sum_{s<=t} A[t,h,s] v_{s,g(h)}
 * plus the normaliser lse[t,h] = log sum_{s<=t} exp(l) (Algorithm 1, dense scores and normalisers).
 * rows[i] is a query position; o is [nrows,Hq,d], lse [nrows,Hq] (either may
 * be NULL).
 */
void orc_dense(int S, int Hq, int Hkv, int d, double scale, const double *q,
               const double *k, const double *v, int nrows, const int32_t *rows,
               double *o, double *lse) {
  (void)S;
#pragma omp parallel
  {
    double *l = (double *)malloc(sizeof(double) * (size_t)S);
#pragma omp for schedule(dynamic, 1)
    for (int i = 0; i < nrows; ++i) {
      int t = rows[i];
      for (int h = 0; h < Hq; ++h) {
        int j = h / (Hq / Hkv);
        logits_row(Hq, Hkv, d, scale, q, k, t, h, l);
        double lz = log_normaliser(l, t + 1);
        if (lse) lse[(size_t)i * Hq + h] = lz;
        if (o) {
          double *oi = o + ((size_t)i * Hq + h) * d;
          for (int c = 0; c < d; ++c) oi[c] = 0.0;
          for (int s = 0; s <= t; ++s) {
            double a = exp(l[s] - lz);
            const double *vs = v + ((size_t)s * Hkv + j) * d;
            for (int c = 0; c < d; ++c) oi[c] += a * vs[c];
          }
        }
      }
    }
    free(l);
  }
}

/*
 * Head-averaged attention mass (Section 4.1):
 *   P_t(s) = (1/Hq) sum_h A[t,h,s],  s <= t.
 * Following Algorithm 1, normalisers and head-averaged probabilities: the normaliser of every head is computed
 * first, then the probabilities are reconstructed and averaged over heads.
 * The average runs over the heads [h0, h0 + nh): all Hq heads for the
 * head-averaged token support S_t, or the G heads of KV group r for the
 * per-group support S_{t,r} of the head axis (Section 3, support granularity).
 * P is [nrows,S]; entries s > t are written as 0 and carry no meaning.
 */
void orc_mass_heads(int S, int Hq, int Hkv, int d, double scale, const double *q,
                    const double *k, int h0, int nh, int nrows, const int32_t *rows,
                    double *P) {
#pragma omp parallel
  {
    double *l = (double *)malloc(sizeof(double) * (size_t)S);
#pragma omp for schedule(dynamic, 1)
    for (int i = 0; i < nrows; ++i) {
      int t = rows[i];
      double *Pi = P + (size_t)i * S;
      for (int s = 0; s < S; ++s) Pi[s] = 0.0;
      for (int h = h0; h < h0 + nh; ++h) {
        logits_row(Hq, Hkv, d, scale, q, k, t, h, l);
        double lz = log_normaliser(l, t + 1);
        for (int s = 0; s <= t; ++s) Pi[s] += exp(l[s] - lz);
      }
      for (int s = 0; s <= t; ++s) Pi[s] /= (double)nh;
    }
    free(l);
  }
}

void orc_mass(int S, int Hq, int Hkv, int d, double scale, const double *q,
              const double *k, int nrows, const int32_t *rows, double *P) {
  orc_mass_heads(S, Hq, Hkv, d, scale, q, k, 0, Hq, nrows, rows, P);
}

/*
 * Head-collapsed indexer score (Section 6.3 equation for z):
 *   z[t,s] = ReLU(<q_idx[t], k_idx[s]> * scale_idx),  s <= t
 * with the ReLU skipped when relu == 0. Inputs are the indexer vectors after
 * key normalisation and RoPE. Z is [nrows,S]; entries s > t are 0.
 */
void orc_index_scores(int S, int di, double scale, int relu, const double *qi,
                      const double *ki, int nrows, const int32_t *rows, double *Z) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int i = 0; i < nrows; ++i) {
    int t = rows[i];
    double *Zi = Z + (size_t)i * S;
    const double *qt = qi + (size_t)t * di;
    for (int s = 0; s < S; ++s) {
      if (s > t) { Zi[s] = 0.0; continue; }
      const double *ks = ki + (size_t)s * di;
      double acc = 0.0;
      for (int c = 0; c < di; ++c) acc += qt[c] * ks[c];
      double z = scale * acc;
      if (relu) z = z > 0.0 ? z : 0.0;
      Zi[s] = z;
    }
  }
}

/*
 * Selection-block aggregation (Section 4.2 equation for P_B):
 *   Y[s] = AGG_{i : trows[i] >= s} X[i][s],  s <= max_i trows[i]
 * AGG is max (the paper's rule) or sum. X holds one score row per query of
 * the block ([nt,S]); Y is [S] and is 0 beyond the block's last query.
 */
void orc_block_aggregate(int S, int agg, int nt, const int32_t *trows,
                         const double *X, double *Y) {
  int tmax = -1;
  for (int i = 0; i < nt; ++i) tmax = trows[i] > tmax ? trows[i] : tmax;
  for (int s = 0; s < S; ++s) {
    if (s > tmax) { Y[s] = 0.0; continue; }
    int have = 0;
    double acc = 0.0;
    for (int i = 0; i < nt; ++i) {
      if (trows[i] < s) continue;
      double x = X[(size_t)i * S + s];
      if (!have) { acc = x; have = 1; }
      else if (agg == ORC_AGG_MAX) acc = x > acc ? x : acc;
      else acc += x;
    }
    Y[s] = acc;
  }
}

typedef struct { double y; int32_t s; } cand_t;

/* Order by score descending, then position ascending. */
static int cand_cmp(const void *a, const void *b) {
  const cand_t *x = (const cand_t *)a, *y = (const cand_t *)b;
  if (x->y > y->y) return -1;
  if (x->y < y->y) return 1;
  return (x->s > y->s) - (x->s < y->s);
}

/*
 * Top-k support of one score row (Section 4.1 TopK; Algorithm 1, top-k
 * selection and the sentinel padding of the restricted recomputation). For row i with L = lens[i] valid positions
 * 0..L-1:
 *   - if L <= k every valid position is taken;
 *   - else the Wf = min(W, k) most recent positions are forced, and the
 *     remaining k - Wf are the first of the other positions in the order
 *     (score descending, position ascending).
 * The row of out ([nrows,k]) lists the chosen positions ascending, then -1.
 */
void orc_topk(int nrows, const int32_t *lens, const double *Y, int64_t ldy, int k,
              int W, int32_t *out) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int i = 0; i < nrows; ++i) {
    int L = lens[i];
    const double *y = Y + (size_t)i * ldy;
    int32_t *oi = out + (size_t)i * k;
    for (int c = 0; c < k; ++c) oi[c] = -1;
    if (L <= k) {
      for (int s = 0; s < L; ++s) oi[s] = s;
      continue;
    }
    int Wf = W < k ? W : k;
    int ncand = L - Wf;
    int kp = k - Wf;
    cand_t *c = (cand_t *)malloc(sizeof(cand_t) * (size_t)ncand);
    char *mark = (char *)calloc((size_t)L, 1);
    for (int s = 0; s < ncand; ++s) { c[s].y = y[s]; c[s].s = s; }
    qsort(c, (size_t)ncand, sizeof(cand_t), cand_cmp);
    for (int m = 0; m < kp; ++m) mark[c[m].s] = 1;
    for (int s = ncand; s < L; ++s) mark[s] = 1;
    int n = 0;
    for (int s = 0; s < L; ++s)
      if (mark[s]) oi[n++] = s;
    free(c);
    free(mark);
  }
}

/*
 * Restricted (sparse) attention over a shared support (Section 3, second
 * equation; Section 4.2 per-query causal mask). Query t belongs to block
 * r = t / b and uses U = { s in idx[r,:] : 0 <= s <= t, s < S }:
 *   o[t,h] = sum_{s in U} softmax_U(<q_{t,h}, k_{s,g(h)}> * scale)_s v_{s,g(h)}
 * with o = 0 when U is empty. idx is [R,kk]; the order of a row and any
 * sentinel entries do not matter. o is [nrows,Hq,d]. With per-KV-group
 * supports S_{t,r} (Section 3, head axis), idx is [Hkv,R,kk] and head h
 * reads the table of its group g(h): group_stride = R*kk (0 when shared).
 */
void orc_sparse(int S, int Hq, int Hkv, int d, double scale, const double *q,
                const double *k, const double *v, int b, int kk, const int32_t *idx,
                int64_t group_stride, int nrows, const int32_t *rows, double *o) {
  int G = Hq / Hkv;
#pragma omp parallel
  {
    double *l = (double *)malloc(sizeof(double) * (size_t)(kk > 0 ? kk : 1));
    int32_t *U = (int32_t *)malloc(sizeof(int32_t) * (size_t)(kk > 0 ? kk : 1));
#pragma omp for schedule(dynamic, 1)
    for (int i = 0; i < nrows; ++i) {
      int t = rows[i];
      int r = t / b;
      for (int h = 0; h < Hq; ++h) {
        int j = h / G;
        const int32_t *ir = idx + (size_t)j * group_stride + (size_t)r * kk;
        int n = 0;
        for (int c = 0; c < kk; ++c)
          if (ir[c] >= 0 && ir[c] <= t && ir[c] < S) U[n++] = ir[c];
        double *oi = o + ((size_t)i * Hq + h) * d;
        for (int c = 0; c < d; ++c) oi[c] = 0.0;
        if (n == 0) continue;
        const double *qt = q + ((size_t)t * Hq + h) * d;
        for (int u = 0; u < n; ++u) {
          const double *ks = k + ((size_t)U[u] * Hkv + j) * d;
          double acc = 0.0;
          for (int c = 0; c < d; ++c) acc += qt[c] * ks[c];
          l[u] = scale * acc;
        }
        double lz = log_normaliser(l, n);
        for (int u = 0; u < n; ++u) {
          double a = exp(l[u] - lz);
          const double *vs = v + ((size_t)U[u] * Hkv + j) * d;
          for (int c = 0; c < d; ++c) oi[c] += a * vs[c];
        }
      }
    }
    free(l);
    free(U);
  }
}

/*
 * KL distillation objective (Section 6.2):
 *   L = (1/n) * sum_i KL(P_i || softmax(z_i)),
 *   KL(P || Q) = sum_s P(s) * (log P(s) - log Q(s)),   0 * log 0 = 0,
 * with the softmax over the valid causal keys s <= t_i only:
 *   log Q(s) = z(s) - log sum_{s' <= t_i} exp(z(s')).
 * P is taken as given (a teacher row of the head-averaged mass sums to 1).
 * Gradient of L with respect to z_i(s), s <= t_i:
 *   dL/dz_i(s) = (Q(s) * sum_{s'} P(s') - P(s)) / n,   and 0 for s > t_i.
 * P, z and grad are [n, S]; row i belongs to query t_i = rows[i]. A row with
 * t_i outside [0, S) has KL 0 and gradient 0. kl or grad may be NULL.
 */
void orc_kl(int S, int n, const int32_t *rows, const double *P, const double *z,
            double *kl, double *grad) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int i = 0; i < n; ++i) {
    int t = rows[i];
    const double *Pi = P + (size_t)i * S;
    const double *zi = z + (size_t)i * S;
    double *gi = grad ? grad + (size_t)i * S : NULL;
    if (gi)
      for (int s = 0; s < S; ++s) gi[s] = 0.0;
    if (t < 0 || t >= S) {
      if (kl) kl[i] = 0.0;
      continue;
    }
    double lz = log_normaliser(zi, t + 1);
    double sumP = 0.0, acc = 0.0;
    for (int s = 0; s <= t; ++s) {
      sumP += Pi[s];
      if (Pi[s] > 0.0) acc += Pi[s] * (log(Pi[s]) - (zi[s] - lz));
    }
    if (kl) kl[i] = acc;
    if (gi)
      for (int s = 0; s <= t; ++s) gi[s] = (exp(zi[s] - lz) * sumP - Pi[s]) / n;
  }
}

/*
 * Head-collapsed indexer front end (Section 6.3, first two equations;
 * Algorithm 2, indexer projection and its key normalisation, RoPE and query scale), for token rows t = rows[i] at positions pos0 + t:
 *   q = W_Q x_t,   k = LN(W_K x_t),
 *   LN(a) = (a - mean(a)) / sqrt(var(a) + eps) * gamma + beta   (over d_idx),
 *   q_idx = RoPE(q, pos0 + t),   k_idx = RoPE(k, pos0 + t),
 * where RoPE(a, p) rotates each pair (a[c], a[c + d_idx/2]), c < d_idx/2, by
 * the angle p * theta^(-2c/d_idx):
 *   out[c]           = a[c] cos - a[c + d_idx/2] sin
 *   out[c + d_idx/2] = a[c + d_idx/2] cos + a[c] sin.
 * The 1/sqrt(d_idx) query scale is left to the scorer. x is [S, dm]; wq and
 * wk are [d_idx, dm]; gamma, beta [d_idx]; q_idx, k_idx [nrows, d_idx].
 */
static void rope_row(int di, double p, double theta, const double *a, double *out) {
  int h = di / 2;
  for (int c = 0; c < h; ++c) {
    double ang = p * pow(theta, -2.0 * c / di);
    double cs = cos(ang), sn = sin(ang);
    out[c] = a[c] * cs - a[c + h] * sn;
    out[c + h] = a[c + h] * cs + a[c] * sn;
  }
}

void orc_project(int S, int dm, int di, const double *x, const double *wq, const double *wk,
                 const double *gamma, const double *beta, double eps, double theta, int pos0,
                 int nrows, const int32_t *rows, double *q_idx, double *k_idx) {
#pragma omp parallel
  {
    double *a = (double *)malloc(sizeof(double) * (size_t)di);
    double *b = (double *)malloc(sizeof(double) * (size_t)di);
#pragma omp for schedule(static)
    for (int i = 0; i < nrows; ++i) {
      int t = rows[i];
      const double *xt = x + (size_t)t * dm;
      double p = (double)pos0 + t;
      for (int c = 0; c < di; ++c) {
        double acc = 0.0;
        for (int e = 0; e < dm; ++e) acc += wq[(size_t)c * dm + e] * xt[e];
        a[c] = acc;
      }
      rope_row(di, p, theta, a, q_idx + (size_t)i * di);
      for (int c = 0; c < di; ++c) {
        double acc = 0.0;
        for (int e = 0; e < dm; ++e) acc += wk[(size_t)c * dm + e] * xt[e];
        a[c] = acc;
      }
      double mean = 0.0, var = 0.0;
      for (int c = 0; c < di; ++c) mean += a[c];
      mean /= di;
      for (int c = 0; c < di; ++c) var += (a[c] - mean) * (a[c] - mean);
      var /= di;
      double inv = 1.0 / sqrt(var + eps);
      for (int c = 0; c < di; ++c) b[c] = (a[c] - mean) * inv * gamma[c] + beta[c];
      rope_row(di, p, theta, b, k_idx + (size_t)i * di);
    }
    free(a);
    free(b);
  }
}

/* Threads the parallel loops above run on (reported beside CPU timings). */
int orc_num_threads(void) { return omp_get_max_threads(); }
