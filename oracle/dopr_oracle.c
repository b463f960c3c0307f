/*
 * dopr_oracle.c -- plain, slow, float64 CPU oracle of the DoPR online scoring
 * step.  TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load it; the product path never does.
 * It shares no code, header, table or helper with the HIP library.
 *
 * What it computes is the plain definition of one decoder layer's online
 * attention with injected prefix states, plus the score head:
 *   - Sec. 3.1 (Eq. 3) and Sec. 3.3: each document d has offline prefix
 *     states C~_d, i.e. per layer the keys and values of L_d = K_infer slots.
 *   - Sec. 3.4: online, C~_d is injected as pre-filled K/V and only the
 *     query tokens plus the score token [q; t_score] are processed.
 *   - Sec. 3.2.2: the query/score tokens see the document only through its
 *     prefix states; among themselves attention is causal.
 *   - Sec. 3.2.3: s(q,d) = MLP(h_score), read here as RMSNorm followed by a
 *     two-row (yes, no) linear head, s = l_yes - l_no.
 * Qwen3 details the paper does not restate (it names only the Qwen3
 * backbone): per-head RMSNorm of q and k before rotate-half RoPE, GQA with
 * contiguous head groups, online positions continuing after the prefix.
 * For the cross-family check (Llama; Appendix, "Generalization Across Model
 * Families") the norm gains may be absent (no QK-norm) and the rotation
 * frequencies may be given by the caller.
 *
 * Inputs are bf16 bit patterns (uint16) converted exactly to double; every
 * intermediate is double; no blocking, fusion or reordering.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_ERR_ARG (-1)
#define ORACLE_ERR_DOC_RANGE (-3)
#define ORACLE_ERR_NOMEM (-7)

/* Exact widening of a bf16 bit pattern: bf16 is the top half of an fp32. */
static double bf16_to_double(uint16_t b) {
  uint32_t u = ((uint32_t)b) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* RMSNorm with weight: y_i = w_i * x_i / sqrt(mean_k x_k^2 + eps). */
static void rms_norm(const double *x, const double *w, int n, double eps,
                     double *y) {
  double ss = 0.0;
  for (int i = 0; i < n; ++i) ss += x[i] * x[i];
  double inv = 1.0 / sqrt(ss / (double)n + eps);
  for (int i = 0; i < n; ++i) y[i] = w[i] * (x[i] * inv);
}

/* Rotate-half rotary embedding at integer position `pos`: for i < D/2 the
 * pair (x_i, x_{i+D/2}) is rotated by angle pos * omega_i, with
 * omega_i = theta^(-2i/D), or inv_freq[i] when the caller gives the
 * frequencies (model families that rescale them, e.g. Llama 3). */
static void rope(double *x, int d, double pos, double theta,
                 const double *inv_freq) {
  int half = d / 2;
  for (int i = 0; i < half; ++i) {
    double freq = inv_freq ? inv_freq[i]
                           : pow(theta, -2.0 * (double)i / (double)d);
    double ang = pos * freq;
    double c = cos(ang), s = sin(ang);
    double a = x[i], b = x[i + half];
    x[i] = a * c - b * s;
    x[i + half] = b * c + a * s;
  }
}

static int doc_is_valid(int32_t doc, int64_t n_docs, const int32_t *doc_len) {
  return doc >= 0 && (int64_t)doc < n_docs && doc_len[doc] >= 0;
}

/*
 * One layer of online prefix attention for a batch of pairs.
 *   doc_ids [P], cu_seqlens [P+1]            pair -> document, token ranges
 *   doc_len [n_docs] (-1 = not resident)     prefix slots per document
 *   doc_off [n_docs]                         element offset of document d's
 *                                            first slot in prefix_k/prefix_v
 *   prefix_k, prefix_v  bf16 [slots, Hkv, D] canonical prefix states
 *   q [Ntok, Hq, D], k/v [Ntok, Hkv, D]      raw online projections (bf16)
 *   q_norm_w, k_norm_w [D]                   RMSNorm weights (bf16)
 *   out [Ntok, Hq, D] double; lse [Ntok, Hq] double (may be NULL)
 *   pair_status [P] (may be NULL): 0, or ORACLE_ERR_DOC_RANGE for a pair
 *   whose document is out of range / not resident (its outputs are 0 and
 *   its lse is -inf).
 * Returns 0, or a negative code for malformed arguments.
 */
/* Element i of an online projection held either as bf16 bit patterns or as
 * doubles (the decoder-layer oracle hands over its own float64 q, k, v). */
static double online_elem(const void *a, int64_t i, int f64) {
  return f64 ? ((const double *)a)[i] : bf16_to_double(((const uint16_t *)a)[i]);
}

/* last_only = 0: every online row, out/lse indexed by token.  last_only = 1:
 * only each pair's last row j = T_p - 1 (its score token), out/lse indexed
 * by pair; the own keys and values of all T_p tokens are still formed.
 * qkv_f64: q, k, v are double arrays instead of bf16. */
static int attention(
    int32_t n_pairs, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    const int32_t *doc_ids, const int32_t *cu_seqlens, int64_t n_docs,
    const int32_t *doc_len, const int64_t *doc_off, const uint16_t *prefix_k,
    const uint16_t *prefix_v, const void *q, const void *k, const void *v,
    const uint16_t *q_norm_w, const uint16_t *k_norm_w, double rms_eps,
    double rope_theta, const double *rope_inv_freq, double softmax_scale,
    double *out, double *lse, int32_t *pair_status, int32_t n_threads,
    int last_only, int qkv_f64) {
  if (n_pairs < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0 ||
      head_dim % 2 || n_q_heads % n_kv_heads)
    return ORACLE_ERR_ARG;
  /* Both gains or neither: without them q and k enter RoPE as given (no
   * per-head RMSNorm, as in attention families without QK-norm). */
  if ((q_norm_w == NULL) != (k_norm_w == NULL)) return ORACLE_ERR_ARG;
  const int qk_norm = q_norm_w != NULL;
  const int D = head_dim, Hq = n_q_heads, Hkv = n_kv_heads;
  const int n_rep = Hq / Hkv;
  for (int32_t p = 0; p < n_pairs; ++p)
    if (cu_seqlens[p + 1] - cu_seqlens[p] < 1) return ORACLE_ERR_ARG;

  double *wq = (double *)malloc(sizeof(double) * D);
  double *wk = (double *)malloc(sizeof(double) * D);
  if (!wq || !wk) { free(wq); free(wk); return ORACLE_ERR_NOMEM; }
  for (int i = 0; i < D; ++i) {
    wq[i] = qk_norm ? bf16_to_double(q_norm_w[i]) : 1.0;
    wk[i] = qk_norm ? bf16_to_double(k_norm_w[i]) : 1.0;
  }

  int failed = 0;
#ifdef _OPENMP
  if (n_threads > 0) omp_set_num_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1) reduction(| : failed)
#endif
  for (int32_t p = 0; p < n_pairs; ++p) {
    const int32_t doc = doc_ids[p];
    const int64_t tok0 = cu_seqlens[p];
    const int T = cu_seqlens[p + 1] - cu_seqlens[p];

    const int j0 = last_only ? T - 1 : 0;

    /* Step 1: retrieve C~_d for the candidate document (Sec. 3.4). */
    if (!doc_is_valid(doc, n_docs, doc_len)) {
      if (pair_status) pair_status[p] = ORACLE_ERR_DOC_RANGE;
      for (int j = j0; j < T; ++j) {
        const int64_t row = last_only ? p : tok0 + j;
        for (int h = 0; h < Hq; ++h) {
          double *o = out + (row * Hq + h) * D;
          for (int i = 0; i < D; ++i) o[i] = 0.0;
          if (lse) lse[row * Hq + h] = -INFINITY;
        }
      }
      continue;
    }
    if (pair_status) pair_status[p] = 0;
    const int L = doc_len[doc];
    const uint16_t *pk = prefix_k + doc_off[doc] * (int64_t)Hkv * D;
    const uint16_t *pv = prefix_v + doc_off[doc] * (int64_t)Hkv * D;

    double *khat = (double *)malloc(sizeof(double) * (size_t)T * Hkv * D);
    double *vown = (double *)malloc(sizeof(double) * (size_t)T * Hkv * D);
    double *x = (double *)malloc(sizeof(double) * D);
    double *qhat = (double *)malloc(sizeof(double) * D);
    double *z = (double *)malloc(sizeof(double) * (size_t)(L + T));
    if (!khat || !vown || !x || !qhat || !z) {
      failed = 1;
      free(khat); free(vown); free(x); free(qhat); free(z);
      continue;
    }

    /* Step 2: own keys k^ = RoPE_{L+j}(RMSNorm(k) * w_k); values as given. */
    for (int j = 0; j < T; ++j)
      for (int g = 0; g < Hkv; ++g) {
        const int64_t ks = ((tok0 + j) * Hkv + g) * D;
        for (int i = 0; i < D; ++i) x[i] = online_elem(k, ks + i, qkv_f64);
        double *dst = khat + ((int64_t)j * Hkv + g) * D;
        if (qk_norm)
          rms_norm(x, wk, D, rms_eps, dst);
        else
          for (int i = 0; i < D; ++i) dst[i] = x[i];
        rope(dst, D, (double)(L + j), rope_theta, rope_inv_freq);
        const int64_t vs = ((tok0 + j) * Hkv + g) * D;
        double *vd = vown + ((int64_t)j * Hkv + g) * D;
        for (int i = 0; i < D; ++i) vd[i] = online_elem(v, vs + i, qkv_f64);
      }

    /* Step 3: every online token j of every q head h attends to all L
     * prefix slots of kv head g = h / n_rep and to its own keys 0..j. */
    for (int jq = j0; jq < T; ++jq)
      for (int h = 0; h < Hq; ++h) {
        const int j = jq;
        const int64_t orow = last_only ? p : tok0 + j;
        const int g = h / n_rep;
        const int64_t qs = ((tok0 + j) * Hq + h) * D;
        for (int i = 0; i < D; ++i) x[i] = online_elem(q, qs + i, qkv_f64);
        if (qk_norm)
          rms_norm(x, wq, D, rms_eps, qhat);
        else
          for (int i = 0; i < D; ++i) qhat[i] = x[i];
        rope(qhat, D, (double)(L + j), rope_theta, rope_inv_freq);

        const int n_keys = L + j + 1;
        for (int t = 0; t < L; ++t) {
          const uint16_t *kt = pk + ((int64_t)t * Hkv + g) * D;
          double dot = 0.0;
          for (int i = 0; i < D; ++i) dot += qhat[i] * bf16_to_double(kt[i]);
          z[t] = softmax_scale * dot;
        }
        for (int t = 0; t <= j; ++t) {
          const double *kt = khat + ((int64_t)t * Hkv + g) * D;
          double dot = 0.0;
          for (int i = 0; i < D; ++i) dot += qhat[i] * kt[i];
          z[L + t] = softmax_scale * dot;
        }
        double zmax = z[0];
        for (int t = 1; t < n_keys; ++t) if (z[t] > zmax) zmax = z[t];
        double denom = 0.0;
        for (int t = 0; t < n_keys; ++t) {
          z[t] = exp(z[t] - zmax);
          denom += z[t];
        }
        double *o = out + (orow * Hq + h) * D;
        for (int i = 0; i < D; ++i) o[i] = 0.0;
        for (int t = 0; t < L; ++t) {
          const uint16_t *vt = pv + ((int64_t)t * Hkv + g) * D;
          const double pt = z[t] / denom;
          for (int i = 0; i < D; ++i) o[i] += pt * bf16_to_double(vt[i]);
        }
        for (int t = 0; t <= j; ++t) {
          const double *vt = vown + ((int64_t)t * Hkv + g) * D;
          const double pt = z[L + t] / denom;
          for (int i = 0; i < D; ++i) o[i] += pt * vt[i];
        }
        if (lse) lse[orow * Hq + h] = zmax + log(denom);
      }
    free(khat); free(vown); free(x); free(qhat); free(z);
  }
  free(wq);
  free(wk);
  return failed ? ORACLE_ERR_NOMEM : ORACLE_OK;
}

int dopr_oracle_prefix_attn(
    int32_t n_pairs, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    const int32_t *doc_ids, const int32_t *cu_seqlens, int64_t n_docs,
    const int32_t *doc_len, const int64_t *doc_off, const uint16_t *prefix_k,
    const uint16_t *prefix_v, const uint16_t *q, const uint16_t *k,
    const uint16_t *v, const uint16_t *q_norm_w, const uint16_t *k_norm_w,
    double rms_eps, double rope_theta, const double *rope_inv_freq,
    double softmax_scale, double *out, double *lse, int32_t *pair_status,
    int32_t n_threads) {
  return attention(n_pairs, n_q_heads, n_kv_heads, head_dim, doc_ids,
                   cu_seqlens, n_docs, doc_len, doc_off, prefix_k, prefix_v,
                   q, k, v, q_norm_w, k_norm_w, rms_eps, rope_theta,
                   rope_inv_freq, softmax_scale, out, lse, pair_status,
                   n_threads, 0, 0);
}

/*
 * The same attention with the online projections q [Ntok, Hq, D] and k, v
 * [Ntok, Hkv, D] given as doubles (the decoder-layer oracle forms them in
 * float64 from its own projections).
 */
int dopr_oracle_prefix_attn_f64(
    int32_t n_pairs, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    const int32_t *doc_ids, const int32_t *cu_seqlens, int64_t n_docs,
    const int32_t *doc_len, const int64_t *doc_off, const uint16_t *prefix_k,
    const uint16_t *prefix_v, const double *q, const double *k,
    const double *v, const uint16_t *q_norm_w, const uint16_t *k_norm_w,
    double rms_eps, double rope_theta, const double *rope_inv_freq,
    double softmax_scale, double *out, double *lse, int32_t *pair_status,
    int32_t n_threads) {
  return attention(n_pairs, n_q_heads, n_kv_heads, head_dim, doc_ids,
                   cu_seqlens, n_docs, doc_len, doc_off, prefix_k, prefix_v,
                   q, k, v, q_norm_w, k_norm_w, rms_eps, rope_theta,
                   rope_inv_freq, softmax_scale, out, lse, pair_status,
                   n_threads, 0, 1);
}

/*
 * Last layer of the online pass: the score head reads only the score
 * token's hidden state (Sec. 3.2.3), so only row j = T_p - 1 of every pair
 * is needed.  Same arguments and the same attention as
 * dopr_oracle_prefix_attn, restricted to that row: out [P, Hq, D] and lse
 * [P, Hq] are indexed by pair.
 */
int dopr_oracle_score_attn(
    int32_t n_pairs, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    const int32_t *doc_ids, const int32_t *cu_seqlens, int64_t n_docs,
    const int32_t *doc_len, const int64_t *doc_off, const uint16_t *prefix_k,
    const uint16_t *prefix_v, const uint16_t *q, const uint16_t *k,
    const uint16_t *v, const uint16_t *q_norm_w, const uint16_t *k_norm_w,
    double rms_eps, double rope_theta, const double *rope_inv_freq,
    double softmax_scale, double *out, double *lse, int32_t *pair_status,
    int32_t n_threads) {
  return attention(n_pairs, n_q_heads, n_kv_heads, head_dim, doc_ids,
                   cu_seqlens, n_docs, doc_len, doc_off, prefix_k, prefix_v,
                   q, k, v, q_norm_w, k_norm_w, rms_eps, rope_theta,
                   rope_inv_freq, softmax_scale, out, lse, pair_status,
                   n_threads, 1, 0);
}

/*
 * Score head on given hidden states (double, [P, W] rows):
 *   h^ = RMSNorm(h) * norm_w; l_yes = w_yes . h^; l_no = w_no . h^;
 *   s = l_yes - l_no.
 * w_head is bf16 [2, W] (row 0 yes, row 1 no).  logits [P,2] may be NULL.
 */
int dopr_oracle_score(int32_t n_pairs, int32_t width, const double *h,
                      const uint16_t *norm_w, const uint16_t *w_head,
                      double rms_eps, double *logits, double *score) {
  if (n_pairs < 0 || width <= 0) return ORACLE_ERR_ARG;
  double *w = (double *)malloc(sizeof(double) * width);
  double *wy = (double *)malloc(sizeof(double) * width);
  double *wn = (double *)malloc(sizeof(double) * width);
  double *hh = (double *)malloc(sizeof(double) * width);
  if (!w || !wy || !wn || !hh) {
    free(w); free(wy); free(wn); free(hh);
    return ORACLE_ERR_NOMEM;
  }
  for (int i = 0; i < width; ++i) {
    w[i] = bf16_to_double(norm_w[i]);
    wy[i] = bf16_to_double(w_head[i]);
    wn[i] = bf16_to_double(w_head[width + i]);
  }
  for (int32_t p = 0; p < n_pairs; ++p) {
    rms_norm(h + (int64_t)p * width, w, width, rms_eps, hh);
    double ly = 0.0, ln = 0.0;
    for (int i = 0; i < width; ++i) {
      ly += wy[i] * hh[i];
      ln += wn[i] * hh[i];
    }
    if (logits) {
      logits[2 * p] = ly;
      logits[2 * p + 1] = ln;
    }
    score[p] = ly - ln;
  }
  free(w); free(wy); free(wn); free(hh);
  return ORACLE_OK;
}

/*
 * Canonical grouping of pairs by document: the valid pairs (document in
 * range and resident) in ascending (doc id, pair index) order, one group per
 * distinct document.  Counting sort over the doc-id space, stable in the
 * pair index.  group_doc/pair_order need n_pairs entries, group_ptr
 * n_pairs + 1.  Writes *n_groups and *n_valid.
 */
int dopr_oracle_group(int32_t n_pairs, const int32_t *doc_ids, int64_t n_docs,
                      const int32_t *doc_len, int32_t *n_groups,
                      int32_t *n_valid, int32_t *group_doc, int32_t *group_ptr,
                      int32_t *pair_order) {
  if (n_pairs < 0 || n_docs < 0) return ORACLE_ERR_ARG;
  int64_t *count = (int64_t *)calloc((size_t)n_docs + 1, sizeof(int64_t));
  if (!count) return ORACLE_ERR_NOMEM;
  for (int32_t p = 0; p < n_pairs; ++p)
    if (doc_is_valid(doc_ids[p], n_docs, doc_len)) count[doc_ids[p] + 1] += 1;
  int32_t g = 0;
  int64_t run = 0;
  for (int64_t d = 0; d < n_docs; ++d) {
    int64_t c = count[d + 1];
    count[d + 1] = run; /* becomes the first output slot of document d */
    if (c > 0) {
      group_doc[g] = (int32_t)d;
      group_ptr[g] = (int32_t)run;
      ++g;
    }
    run += c;
  }
  group_ptr[g] = (int32_t)run;
  for (int32_t p = 0; p < n_pairs; ++p)
    if (doc_is_valid(doc_ids[p], n_docs, doc_len))
      pair_order[count[doc_ids[p] + 1]++] = p;
  *n_groups = g;
  *n_valid = (int32_t)run;
  free(count);
  return ORACLE_OK;
}

/* Document-side prefix memory: sum_d L_d * layers * Hkv * D * 2 (K, V) * 2
 * bytes (bf16), over resident documents. */
int64_t dopr_oracle_store_payload_bytes(int32_t n_layers, int32_t n_kv_heads,
                                        int32_t head_dim, int64_t n_docs,
                                        const int32_t *doc_len) {
  int64_t slots = 0;
  for (int64_t d = 0; d < n_docs; ++d)
    if (doc_len[d] > 0) slots += doc_len[d];
  return slots * (int64_t)n_layers * n_kv_heads * head_dim * 2 * 2;
}

int dopr_oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
