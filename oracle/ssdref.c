/*
 * ssdref.c — plain CPU oracle (TEST INFRASTRUCTURE ONLY; see ssdref.h).
 *
 * Written for readability, not speed: fp64 activations, one thread per output
 * element with an ascending-index summation, no blocking or fusion.  The one
 * concession to run time is that the k-loop of a linear layer advances all
 * nodes together (each node keeps its own accumulator), which changes no
 * element's arithmetic.
 */
#include "ssdref.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------ */
/* storage types                                                       */
/* ------------------------------------------------------------------ */

static double bf16_bits_to_double(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Round-to-nearest-even of a double to bfloat16 (8 significant bits, float32
 * exponent range, subnormal quantum 2^-133), done directly from the double so
 * there is no double rounding through float32. */
uint16_t ssdref_round_bf16(double x) {
  if (isnan(x)) return (uint16_t)0x7fc0;
  uint16_t sign = signbit(x) ? (uint16_t)0x8000 : (uint16_t)0;
  double ax = fabs(x);
  if (isinf(ax)) return (uint16_t)(sign | 0x7f80);
  int e;
  frexp(ax, &e); /* ax in [2^(e-1), 2^e) */
  int q_exp = (e - 1) - 7;
  if (q_exp < -133) q_exp = -133;
  double r = nearbyint(ldexp(ax, -q_exp)); /* ties to even under the default mode */
  float f = (float)ldexp(r, q_exp);        /* exact; overflows to inf past the bf16 range */
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  return (uint16_t)(sign | (uint16_t)(u >> 16));
}

static double ld(const void *p, size_t i, int dtype) {
  if (dtype == SSDREF_F32) return (double)((const float *)p)[i];
  return bf16_bits_to_double(((const uint16_t *)p)[i]);
}

static void st_rounded(void *p, size_t i, int dtype, double x) {
  if (dtype == SSDREF_F32)
    ((float *)p)[i] = (float)x;
  else
    ((uint16_t *)p)[i] = ssdref_round_bf16(x);
}

static size_t elem_size(int dtype) { return dtype == SSDREF_F32 ? 4 : 2; }

/* ------------------------------------------------------------------ */
/* tree bookkeeping (Sec. 3.1)                                         */
/* ------------------------------------------------------------------ */

int ssdref_tree_info(const int32_t *parent_idx, int32_t n, int32_t *depth, uint8_t *anc) {
  if (!parent_idx || n <= 0) return SSDREF_E_ARG;
  if (parent_idx[0] != -1) return SSDREF_E_TREE;
  for (int32_t i = 1; i < n; ++i)
    if (parent_idx[i] < 0 || parent_idx[i] >= i) return SSDREF_E_TREE;
  for (int32_t i = 0; i < n; ++i) {
    int32_t dd = 0;
    if (anc) memset(anc + (size_t)i * n, 0, (size_t)n);
    /* walk from i to the root */
    for (int32_t j = i; j != -1; j = parent_idx[j]) {
      if (anc) anc[(size_t)i * n + j] = 1;
      if (j != i) ++dd;
    }
    if (depth) depth[i] = dd;
  }
  return SSDREF_OK;
}

/* root-first list of the nodes on the path root -> i; returns its length */
static int32_t root_path(const int32_t *parent_idx, int32_t i, int32_t *out) {
  int32_t len = 0;
  for (int32_t j = i; j != -1; j = parent_idx[j]) out[len++] = j;
  for (int32_t a = 0, b = len - 1; a < b; ++a, --b) {
    int32_t t = out[a];
    out[a] = out[b];
    out[b] = t;
  }
  return len;
}

/* ------------------------------------------------------------------ */
/* GPT-2 pieces                                                        */
/* ------------------------------------------------------------------ */

/* y = (x - mean) / sqrt(var + eps) * g + b, biased variance, per row */
static void layer_norm(const double *x, int32_t n, int32_t d, const void *g, const void *b, int dt,
                       double eps, double *y) {
  for (int32_t i = 0; i < n; ++i) {
    const double *xi = x + (size_t)i * d;
    double s = 0.0;
    for (int32_t k = 0; k < d; ++k) s += xi[k];
    double mean = s / d;
    double v = 0.0;
    for (int32_t k = 0; k < d; ++k) v += (xi[k] - mean) * (xi[k] - mean);
    double var = v / d;
    double den = sqrt(var + eps);
    for (int32_t k = 0; k < d; ++k)
      y[(size_t)i * d + k] = (xi[k] - mean) / den * ld(g, k, dt) + ld(b, k, dt);
  }
}

/* out[i][o] = (sum_k a[i][k] * W[o][k]) + bias[o]   (bias may be NULL)
 * W is [out_dim][in_dim] in storage type dt, or, when qc is not NULL, the
 * 8-bit weights W[o][k] = qs[o] * qc[o][k] (exact in fp64).  k ascends for
 * every element. */
static void linear(const void *W, const int8_t *qc, const float *qs, const void *bias, int dt, int32_t out_dim,
                   int32_t in_dim, const double *a, int32_t n, double *out, int nt) {
  /* node-minor copy of the input so that one k step touches all nodes */
  double *aT = (double *)malloc(sizeof(double) * (size_t)in_dim * n);
  for (int32_t i = 0; i < n; ++i)
    for (int32_t k = 0; k < in_dim; ++k) aT[(size_t)k * n + i] = a[(size_t)i * in_dim + k];
#pragma omp parallel num_threads(nt)
  {
    double *wrow = (double *)malloc(sizeof(double) * (size_t)in_dim);
    double *acc = (double *)malloc(sizeof(double) * (size_t)n);
#pragma omp for schedule(static)
    for (int32_t o = 0; o < out_dim; ++o) {
      for (int32_t k = 0; k < in_dim; ++k)
        wrow[k] = qc ? (double)qs[o] * (double)qc[(size_t)o * in_dim + k] : ld(W, (size_t)o * in_dim + k, dt);
      for (int32_t i = 0; i < n; ++i) acc[i] = 0.0;
      for (int32_t k = 0; k < in_dim; ++k) {
        const double wk = wrow[k];
        const double *ak = aT + (size_t)k * n;
        for (int32_t i = 0; i < n; ++i) acc[i] += ak[i] * wk;
      }
      double bo = bias ? ld(bias, o, dt) : 0.0;
      for (int32_t i = 0; i < n; ++i) out[(size_t)i * out_dim + o] = bias ? acc[i] + bo : acc[i];
    }
    free(wrow);
    free(acc);
  }
  free(aT);
}

/* GPT-2's tanh approximation of GELU */
static double gelu(double x) {
  const double c = sqrt(2.0 / M_PI);
  return 0.5 * x * (1.0 + tanh(c * (x + 0.044715 * x * x * x)));
}

static int check_cfg(const ssdref_config *c) {
  if (!c) return 0;
  if (c->n_layer <= 0 || c->d_model <= 0 || c->n_head <= 0 || c->d_mlp <= 0 || c->vocab <= 0 || c->n_pos <= 0)
    return 0;
  if (c->d_model % c->n_head) return 0;
  if (c->dtype != SSDREF_F32 && c->dtype != SSDREF_BF16) return 0;
  return 1;
}

/* ------------------------------------------------------------------ */
/* 8-bit weights (Sec. 4, further speed-ups; format in ssdref.h)       */
/* ------------------------------------------------------------------ */

int ssdref_quantize_q8(const uint16_t *w, int32_t rows, int32_t cols, int8_t *codes, float *scales) {
  if (!w || !codes || !scales || rows <= 0 || cols <= 0) return SSDREF_E_ARG;
  for (size_t e = 0; e < (size_t)rows * cols; ++e)
    if (!isfinite(bf16_bits_to_double(w[e]))) return SSDREF_E_ARG;
  for (int32_t o = 0; o < rows; ++o) {
    const uint16_t *row = w + (size_t)o * cols;
    int8_t *out = codes + (size_t)o * cols;
    float a = 0.0f;
    for (int32_t k = 0; k < cols; ++k) {
      const float v = fabsf((float)bf16_bits_to_double(row[k]));
      if (v > a) a = v;
    }
    if (!(a >= 0x1p-100f)) {
      scales[o] = 0.0f;
      memset(out, 0, (size_t)cols);
      continue;
    }
    const float r = 127.0f / a;
    for (int32_t k = 0; k < cols; ++k) {
      const float p = (float)bf16_bits_to_double(row[k]) * r;
      float c = rintf(p);
      if (c > 127.0f) c = 127.0f;
      if (c < -127.0f) c = -127.0f;
      out[k] = (int8_t)c;
    }
    scales[o] = a / 127.0f;
  }
  return SSDREF_OK;
}

/* ------------------------------------------------------------------ */
/* tree verification pass                                              */
/* ------------------------------------------------------------------ */

int ssdref_tree_verify(const ssdref_config *cfg, const ssdref_weights *w, const void *k_cache,
                       const void *v_cache, int32_t max_ctx, int32_t prefix_len, const int32_t *tokens,
                       const int32_t *parent_idx, int32_t n_nodes, void *k_tree, void *v_tree,
                       int32_t max_nodes, float *logits, int32_t n_threads) {
  if (!check_cfg(cfg) || !w || !tokens || !parent_idx || !k_tree || !v_tree || !logits) return SSDREF_E_ARG;
  if (n_nodes <= 0 || prefix_len < 0 || max_ctx < 0 || prefix_len > max_ctx) return SSDREF_E_ARG;
  if (prefix_len > 0 && (!k_cache || !v_cache)) return SSDREF_E_ARG;
  if (n_nodes > max_nodes) return SSDREF_E_CAPACITY;
  const int32_t L = cfg->n_layer, d = cfg->d_model, H = cfg->n_head, dh = d / H, M = cfg->d_mlp;
  const int32_t V = cfg->vocab, n = n_nodes;
  const int dt = cfg->dtype;
  const ssdref_q8 *q8 = w->q8;
  if (q8 && dt != SSDREF_BF16) return SSDREF_E_ARG;
#ifdef _OPENMP
  const int ntu = n_threads > 0 ? n_threads : omp_get_max_threads();
#else
  const int ntu = 1;
#endif
  int32_t *depth = (int32_t *)malloc(sizeof(int32_t) * n);
  int rc = ssdref_tree_info(parent_idx, n, depth, NULL);
  if (rc != SSDREF_OK) {
    free(depth);
    return rc;
  }
  int32_t max_depth = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (tokens[i] < 0 || tokens[i] >= V) {
      free(depth);
      return SSDREF_E_ARG;
    }
    if (depth[i] > max_depth) max_depth = depth[i];
  }
  if (prefix_len + max_depth >= cfg->n_pos) {
    free(depth);
    return SSDREF_E_CAPACITY;
  }

  double *x = (double *)malloc(sizeof(double) * (size_t)n * d);
  double *a = (double *)malloc(sizeof(double) * (size_t)n * d);
  double *qkv = (double *)malloc(sizeof(double) * (size_t)n * 3 * d);
  double *att = (double *)malloc(sizeof(double) * (size_t)n * d);
  double *tmp = (double *)malloc(sizeof(double) * (size_t)n * d);
  double *f = (double *)malloc(sizeof(double) * (size_t)n * M);

  /* embedding: token row plus the row of position prefix_len + depth */
  for (int32_t i = 0; i < n; ++i) {
    const int32_t pos = prefix_len + depth[i];
    for (int32_t k = 0; k < d; ++k)
      x[(size_t)i * d + k] = ld(w->wte, (size_t)tokens[i] * d + k, dt) + ld(w->wpe, (size_t)pos * d + k, dt);
  }

  const double scale = 1.0 / sqrt((double)dh);
  for (int32_t l = 0; l < L; ++l) {
    layer_norm(x, n, d, w->ln1_g[l], w->ln1_b[l], dt, cfg->ln_eps, a);
    linear(w->w_qkv[l], q8 ? q8->qkv_code[l] : NULL, q8 ? q8->qkv_scale[l] : NULL, w->b_qkv[l], dt, 3 * d, d, a,
           n, qkv, ntu);

    /* the batch's own K/V go to the tree scratch, rounded to the storage type */
    for (int32_t i = 0; i < n; ++i)
      for (int32_t h = 0; h < H; ++h)
        for (int32_t j = 0; j < dh; ++j) {
          size_t dst = (((size_t)l * H + h) * max_nodes + i) * dh + j;
          st_rounded(k_tree, dst, dt, qkv[(size_t)i * 3 * d + d + h * dh + j]);
          st_rounded(v_tree, dst, dt, qkv[(size_t)i * 3 * d + 2 * d + h * dh + j]);
        }

    /* attention: the prefix_len cached keys, then the node's root path */
#pragma omp parallel num_threads(ntu)
    {
      double *s = (double *)malloc(sizeof(double) * ((size_t)prefix_len + n));
      int32_t *path = (int32_t *)malloc(sizeof(int32_t) * n);
#pragma omp for schedule(static)
      for (int32_t ih = 0; ih < n * H; ++ih) {
        const int32_t i = ih / H, h = ih % H;
        const double *q = qkv + (size_t)i * 3 * d + h * dh;
        const int32_t plen = root_path(parent_idx, i, path);
        const int32_t nk = prefix_len + plen;
        const size_t cache_base = ((size_t)l * H + h) * max_ctx;
        const size_t tree_base = ((size_t)l * H + h) * max_nodes;
        for (int32_t t = 0; t < nk; ++t) {
          const void *K = t < prefix_len ? k_cache : k_tree;
          const size_t row = t < prefix_len ? cache_base + t : tree_base + path[t - prefix_len];
          double dot = 0.0;
          for (int32_t j = 0; j < dh; ++j) dot += q[j] * ld(K, row * dh + j, dt);
          s[t] = dot * scale;
        }
        double mx = s[0];
        for (int32_t t = 1; t < nk; ++t)
          if (s[t] > mx) mx = s[t];
        double z = 0.0;
        for (int32_t t = 0; t < nk; ++t) {
          s[t] = exp(s[t] - mx);
          z += s[t];
        }
        for (int32_t j = 0; j < dh; ++j) {
          double acc = 0.0;
          for (int32_t t = 0; t < nk; ++t) {
            const void *Vs = t < prefix_len ? v_cache : v_tree;
            const size_t row = t < prefix_len ? cache_base + t : tree_base + path[t - prefix_len];
            acc += s[t] * ld(Vs, row * dh + j, dt);
          }
          att[(size_t)i * d + h * dh + j] = acc / z;
        }
      }
      free(s);
      free(path);
    }

    linear(w->w_o[l], q8 ? q8->o_code[l] : NULL, q8 ? q8->o_scale[l] : NULL, w->b_o[l], dt, d, d, att, n, tmp,
           ntu);
    for (size_t e = 0; e < (size_t)n * d; ++e) x[e] += tmp[e];

    layer_norm(x, n, d, w->ln2_g[l], w->ln2_b[l], dt, cfg->ln_eps, a);
    linear(w->w_fc[l], q8 ? q8->fc_code[l] : NULL, q8 ? q8->fc_scale[l] : NULL, w->b_fc[l], dt, M, d, a, n, f,
           ntu);
    for (size_t e = 0; e < (size_t)n * M; ++e) f[e] = gelu(f[e]);
    linear(w->w_pr[l], q8 ? q8->pr_code[l] : NULL, q8 ? q8->pr_scale[l] : NULL, w->b_pr[l], dt, d, M, f, n, tmp,
           ntu);
    for (size_t e = 0; e < (size_t)n * d; ++e) x[e] += tmp[e];
  }

  layer_norm(x, n, d, w->lnf_g, w->lnf_b, dt, cfg->ln_eps, a);
  /* tied LM head: logits = ln_f(x) . wte^T (or its 8-bit copy), computed in
   * blocks of rows */
  {
    const int32_t blk = 4096;
    double *lg = (double *)malloc(sizeof(double) * (size_t)n * blk);
    for (int32_t v0 = 0; v0 < V; v0 += blk) {
      const int32_t nv = V - v0 < blk ? V - v0 : blk;
      const void *Wv = (const char *)w->wte + (size_t)v0 * d * elem_size(dt);
      linear(Wv, q8 ? q8->head_code + (size_t)v0 * d : NULL, q8 ? q8->head_scale + v0 : NULL, NULL, dt, nv, d, a,
             n, lg, ntu);
      for (int32_t i = 0; i < n; ++i)
        for (int32_t v = 0; v < nv; ++v) logits[(size_t)i * V + v0 + v] = (float)lg[(size_t)i * nv + v];
    }
    free(lg);
  }

  free(x);
  free(a);
  free(qkv);
  free(att);
  free(tmp);
  free(f);
  free(depth);
  return SSDREF_OK;
}

/* ------------------------------------------------------------------ */
/* commit (Sec. 3.1, last step)                                        */
/* ------------------------------------------------------------------ */

int ssdref_kv_commit(const ssdref_config *cfg, void *k_cache, void *v_cache, int32_t max_ctx,
                     int32_t prefix_len, const void *k_tree, const void *v_tree, int32_t max_nodes,
                     const int32_t *path, int32_t path_len) {
  if (!check_cfg(cfg) || !k_cache || !v_cache || !k_tree || !v_tree || !path) return SSDREF_E_ARG;
  if (prefix_len < 0 || path_len < 0) return SSDREF_E_ARG;
  if (prefix_len + path_len > max_ctx) return SSDREF_E_CAPACITY;
  for (int32_t t = 0; t < path_len; ++t)
    if (path[t] < 0 || path[t] >= max_nodes) return SSDREF_E_ARG;
  const int32_t L = cfg->n_layer, H = cfg->n_head, dh = cfg->d_model / cfg->n_head;
  const size_t row_bytes = (size_t)dh * elem_size(cfg->dtype);
  for (int32_t l = 0; l < L; ++l)
    for (int32_t h = 0; h < H; ++h)
      for (int32_t t = 0; t < path_len; ++t) {
        size_t src = (((size_t)l * H + h) * max_nodes + path[t]) * row_bytes;
        size_t dst = (((size_t)l * H + h) * max_ctx + prefix_len + t) * row_bytes;
        memcpy((char *)k_cache + dst, (const char *)k_tree + src, row_bytes);
        memcpy((char *)v_cache + dst, (const char *)v_tree + src, row_bytes);
      }
  return SSDREF_OK;
}

/* ------------------------------------------------------------------ */
/* Philox4x64-10 (Salmon et al., SC'11)                                */
/* ------------------------------------------------------------------ */

void ssdref_philox4x64_10(const uint64_t key[2], const uint64_t ctr[4], uint64_t out[4]) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
  uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint64_t k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += W0;
      k1 += W1;
    }
    unsigned __int128 p0 = (unsigned __int128)M0 * x0;
    unsigned __int128 p1 = (unsigned __int128)M1 * x2;
    uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
    uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    uint64_t y0 = hi1 ^ x1 ^ k0, y1 = lo1, y2 = hi0 ^ x3 ^ k1, y3 = lo0;
    x0 = y0;
    x1 = y1;
    x2 = y2;
    x3 = y3;
  }
  out[0] = x0;
  out[1] = x1;
  out[2] = x2;
  out[3] = x3;
}

double ssdref_uniform(uint64_t seed, uint64_t stream, uint64_t n) {
  uint64_t key[2] = {seed, stream}, ctr[4] = {n, 0, 0, 0}, out[4];
  ssdref_philox4x64_10(key, ctr, out);
  return (double)(out[0] >> 11) * 0x1.0p-53;
}

/* ------------------------------------------------------------------ */
/* accept / reject (Sec. 2.3 and 3.1)                                  */
/* ------------------------------------------------------------------ */

static int32_t argmax_lowest(const float *row, int32_t V) {
  int32_t best = 0;
  for (int32_t v = 1; v < V; ++v)
    if (row[v] > row[best]) best = v;
  return best;
}

/* keep[v] = token v is among the k largest logits of the row, ties at the
 * cut to the lower id (k = 0 or k >= V: every token): the row's ids sorted
 * by (logit descending, id ascending), the first k kept */
static const float *g_sort_row; /* the row qsort compares (calls are not concurrent) */
static int by_logit_then_id(const void *a, const void *b) {
  const int32_t i = *(const int32_t *)a, j = *(const int32_t *)b;
  if (g_sort_row[i] > g_sort_row[j]) return -1;
  if (g_sort_row[i] < g_sort_row[j]) return 1;
  return (i > j) - (i < j);
}

static void top_k_mask(const float *row, int32_t V, int32_t k, uint8_t *keep) {
  if (k <= 0 || k >= V) {
    memset(keep, 1, (size_t)V);
    return;
  }
  int32_t *ids = (int32_t *)malloc(sizeof(int32_t) * V);
  for (int32_t v = 0; v < V; ++v) ids[v] = v;
  g_sort_row = row;
  qsort(ids, (size_t)V, sizeof(int32_t), by_logit_then_id);
  memset(keep, 0, (size_t)V);
  for (int32_t i = 0; i < k; ++i) keep[ids[i]] = 1;
  free(ids);
}

/* p = softmax(logits / T) in fp64, over the top-k tokens only (k = 0: all) */
static void softmax_t(const float *row, int32_t V, double T, int32_t k, double *p) {
  uint8_t *keep = (uint8_t *)malloc((size_t)V);
  top_k_mask(row, V, k, keep);
  double mx = -INFINITY;
  for (int32_t v = 0; v < V; ++v) {
    double z = (double)row[v] / T;
    if (keep[v] && z > mx) mx = z;
  }
  double s = 0.0;
  for (int32_t v = 0; v < V; ++v) {
    p[v] = keep[v] ? exp((double)row[v] / T - mx) : 0.0;
    s += p[v];
  }
  for (int32_t v = 0; v < V; ++v) p[v] /= s;
  free(keep);
}

/* smallest v with r[0] + ... + r[v] > U * Z (ascending fp64 sum); if rounding
 * leaves none, the last v with r[v] > 0 */
static int32_t sample_cdf(const double *r, int32_t V, double Z, double U) {
  const double t = U * Z;
  double c = 0.0;
  int32_t last = 0;
  for (int32_t v = 0; v < V; ++v) {
    c += r[v];
    if (r[v] > 0.0) last = v;
    if (c > t) return v;
  }
  return last;
}

int ssdref_tree_accept(int32_t mode, const int32_t *tokens, const int32_t *parent_idx, int32_t n_nodes,
                       int32_t vocab, const float *draft_probs, const float *logits, double temperature,
                       uint64_t seed, int32_t *path, int32_t *path_len, int32_t *next_token) {
  if (mode == SSDREF_ACCEPT_SAMPLE_DET) return SSDREF_E_ARG;
  return ssdref_tree_accept_k(mode, tokens, parent_idx, n_nodes, vocab, draft_probs, logits, temperature, 0, seed,
                              path, path_len, next_token);
}

int ssdref_tree_accept_k(int32_t mode, const int32_t *tokens, const int32_t *parent_idx, int32_t n_nodes,
                         int32_t vocab, const float *draft_probs, const float *logits, double temperature,
                         int32_t top_k, uint64_t seed, int32_t *path, int32_t *path_len, int32_t *next_token) {
  if (!tokens || !parent_idx || !logits || !path || !path_len || !next_token) return SSDREF_E_ARG;
  if (n_nodes <= 0 || vocab <= 0 || top_k < 0) return SSDREF_E_ARG;
  if (mode != SSDREF_ACCEPT_GREEDY && mode != SSDREF_ACCEPT_SAMPLE_WOR && mode != SSDREF_ACCEPT_SAMPLE_IID &&
      mode != SSDREF_ACCEPT_SAMPLE_DET && mode != SSDREF_ACCEPT_SAMPLE_CDF)
    return SSDREF_E_ARG;
  const int det = mode == SSDREF_ACCEPT_SAMPLE_DET || mode == SSDREF_ACCEPT_SAMPLE_CDF;
  if (mode != SSDREF_ACCEPT_GREEDY && !(temperature > 0.0)) return SSDREF_E_ARG;
  if (mode != SSDREF_ACCEPT_GREEDY && !det && !draft_probs) return SSDREF_E_ARG;
  if (det && draft_probs) return SSDREF_E_ARG;
  const int32_t n = n_nodes, V = vocab;
  int32_t *depth = (int32_t *)malloc(sizeof(int32_t) * n);
  int rc = ssdref_tree_info(parent_idx, n, depth, NULL);
  if (rc != SSDREF_OK) {
    free(depth);
    return rc;
  }
  for (int32_t i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= V) {
      free(depth);
      return SSDREF_E_ARG;
    }

  if (mode == SSDREF_ACCEPT_GREEDY) {
    /* a node is matched when its parent is matched and its token is the
     * parent's argmax; the deepest matched node (lowest index among equals)
     * ends the accepted path and contributes its own argmax */
    int32_t *g = (int32_t *)malloc(sizeof(int32_t) * n);
    uint8_t *m = (uint8_t *)malloc((size_t)n);
    for (int32_t i = 0; i < n; ++i) g[i] = argmax_lowest(logits + (size_t)i * V, V);
    m[0] = 1;
    for (int32_t i = 1; i < n; ++i) m[i] = m[parent_idx[i]] && tokens[i] == g[parent_idx[i]];
    int32_t best = 0;
    for (int32_t i = 1; i < n; ++i)
      if (m[i] && depth[i] > depth[best]) best = i;
    *path_len = root_path(parent_idx, best, path);
    *next_token = g[best];
    free(g);
    free(m);
    free(depth);
    return SSDREF_OK;
  }

  if (mode == SSDREF_ACCEPT_SAMPLE_CDF) {
    /* inverse-CDF coupling: the oracle's token at each node from the node's
     * own uniform, followed down the tree while a child carries it */
    double *pc = (double *)malloc(sizeof(double) * V);
    int32_t u = 0, len = 0, x = 0;
    path[len++] = 0;
    for (;;) {
      softmax_t(logits + (size_t)u * V, V, temperature, top_k, pc);
      x = sample_cdf(pc, V, 1.0, ssdref_uniform(seed, 2, (uint64_t)u));
      int32_t child = -1;
      for (int32_t c = u + 1; c < n && child < 0; ++c)
        if (parent_idx[c] == u && tokens[c] == x) child = c;
      if (child < 0) break;
      path[len++] = child;
      u = child;
    }
    *next_token = x;
    *path_len = len;
    free(pc);
    free(depth);
    return SSDREF_OK;
  }

  /* recursive rejection sampling along the tree */
  double *p = (double *)malloc(sizeof(double) * V);
  double *r = (double *)malloc(sizeof(double) * V);
  double *qq = (double *)malloc(sizeof(double) * V);
  int32_t u = 0, len = 0;
  double Z = 1.0;
  path[len++] = 0;
  for (;;) {
    softmax_t(logits + (size_t)u * V, V, temperature, top_k, p);
    memcpy(r, p, sizeof(double) * V);
    Z = 1.0;
    double Zq = 0.0;
    if (!det) {
      const float *q = draft_probs + (size_t)u * V;
      for (int32_t v = 0; v < V; ++v) {
        qq[v] = (double)q[v];
        Zq += qq[v];
      }
    }
    int32_t accepted = -1;
    for (int32_t c = u + 1; c < n; ++c) {
      if (parent_idx[c] != u) continue;
      const int32_t xt = tokens[c];
      const double U = ssdref_uniform(seed, 0, (uint64_t)c);
      int acc;
      if (det) /* the candidate was proposed with certainty */
        acc = Z > 0.0 && U < r[xt] / Z;
      else if (qq[xt] == 0.0)
        acc = r[xt] > 0.0;
      else
        acc = U < (r[xt] / Z) / (qq[xt] / Zq);
      if (acc) {
        accepted = c;
        break;
      }
      double nz = 0.0;
      if (det) {
        /* rejected: the candidate's token leaves the residual */
        r[xt] = 0.0;
        for (int32_t v = 0; v < V; ++v) nz += r[v];
        Z = nz;
        continue;
      }
      for (int32_t v = 0; v < V; ++v) {
        double t = r[v] / Z - qq[v] / Zq;
        r[v] = t > 0.0 ? t : 0.0;
        nz += r[v];
      }
      Z = nz;
      if (mode == SSDREF_ACCEPT_SAMPLE_WOR) {
        qq[xt] = 0.0;
        double s = 0.0;
        for (int32_t v = 0; v < V; ++v) s += qq[v];
        Zq = s;
      }
    }
    if (accepted < 0) break;
    path[len++] = accepted;
    u = accepted;
  }
  const double U2 = ssdref_uniform(seed, 1, (uint64_t)u);
  if (Z > 0.0)
    *next_token = sample_cdf(r, V, Z, U2);
  else
    *next_token = sample_cdf(p, V, 1.0, U2);
  *path_len = len;
  free(p);
  free(r);
  free(qq);
  free(depth);
  return SSDREF_OK;
}

int32_t ssdref_cdf_pick(const float *row, int32_t vocab, double temperature, double U) {
  if (!row || vocab <= 0 || !(temperature > 0.0) || !(U >= 0.0 && U < 1.0)) return -1;
  double *p = (double *)malloc(sizeof(double) * vocab);
  softmax_t(row, vocab, temperature, 0, p);
  const int32_t x = sample_cdf(p, vocab, 1.0, U);
  free(p);
  return x;
}
