/*
 * fp64 CPU oracle for link-stage attention (Comb / position-independent caching).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the library's product path may link,
 * load or call this file; only the tests, the smoke check and the benchmark's
 * CPU-baseline leg do. It shares no code, header or table with the HIP path.
 *
 * What it computes, for every request r, query row i and query head h:
 *
 *   * The request's linked chunk caches are concatenated in request order
 *     along the document-length axis (Sec. 4.2: the caches of several
 *     documents, each made from position zero, are concatenated along l_doc
 *     in the link stage; Sec. 1 / Fig. 1: the link stage loads and
 *     concatenates the needed KV in any order).
 *   * Every document row is visible to every query row: cross-attention has
 *     no mask (Sec. 4.2, Eq. 7).
 *   * The request's own KV rows follow the documents under the causal mask of
 *     masked self-attention (Sec. 4.1, Eq. 2). Queries are the last L_q of
 *     the L_s own tokens (during decoding new tokens are appended to the
 *     query sequence, Sec. 4), so row i sees own rows 0 .. i + L_s - L_q.
 *   * Optionally, query token t sees only the first q_doc_limits[t] document
 *     rows (the attention side of post-training PIC, Sec. 2 and 6.1:
 *     recomputed tokens attend as in an ordinary prefill of the concatenated
 *     prompt, i.e. causally by their position in it, and every other query
 *     sees all document rows).
 *   * One softmax over the union of visible keys, scaled by tau (Eq. 2 and
 *     Eq. 7 use 1/sqrt(d); here tau is an argument), then H = A V (Eq. 3, 8).
 *   * Multi-head: query head h reads KV head h / (H_q / H_kv) (the paper
 *     presents one head and calls the multi-head extension standard, Sec. 4).
 *   * MLA (absorbed latent form, the DeepSeek-V2-Lite backbone of Sec. 5.1):
 *     one KV head whose value is the first d_v entries of each key row.
 *
 *   out[i,h] = sum_j p_j V_j / sum_j p_j,  p_j = exp(s_j - m),
 *   s_j = tau <Q[i,h], K_j>,  m = max_j s_j,  lse[i,h] = m + log(sum_j p_j).
 *   A row with no visible key gets out = 0 and lse = -inf.
 *
 * Everything is computed in double. bf16 inputs are widened exactly.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_F32 0
#define ORACLE_BF16 1

static double widen(const void *base, int64_t idx, int dtype) {
  if (dtype == ORACLE_BF16) {
    uint32_t u = (uint32_t)((const uint16_t *)base)[idx] << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
  }
  return (double)((const float *)base)[idx];
}

/* Copies rows [0, n) of a token-major [n][heads][width] tensor into dst
 * (same layout, double). For MLA values, `src_width` is the key width and
 * only the first `width` entries of each row are taken. */
static void widen_rows(double *dst, const void *src, int64_t n, int heads, int width,
                       int src_width, int dtype) {
  for (int64_t t = 0; t < n; ++t)
    for (int hh = 0; hh < heads; ++hh)
      for (int e = 0; e < width; ++e)
        dst[(t * heads + hh) * width + e] =
            widen(src, (t * heads + hh) * (int64_t)src_width + e, dtype);
}

/*
 * Arguments (all host memory):
 *   dtype        ORACLE_F32 (float) or ORACLE_BF16 (uint16 bit patterns)
 *   mla          0: separate V tensors; 1: V = first d_v entries of each K row
 *   link_offsets int32 [batch+1]: links of request r are entries
 *                link_offsets[r] .. link_offsets[r+1]-1 of the three arrays below
 *   link_k       per link, token-major K [len][H_kv][d_k]
 *   link_v       per link, token-major V [len][H_kv][d_v] (ignored when mla)
 *   link_len     per link, its token count
 *   q_offsets    int32 [batch+1] query tokens per request (q is [Tq][H_q][d_k])
 *   self_offsets int32 [batch+1] own tokens per request, or NULL (no own KV)
 *   k_self       [Ts][H_kv][d_k];  v_self [Ts][H_kv][d_v] (ignored when mla)
 *   q_doc_limits int32 [Tq]: document rows 0 .. q_doc_limits[t]-1 are visible to
 *                query token t (0 <= limit <= the request's document rows), or
 *                NULL = all
 *   row_select   uint8 [Tq*H_q] (1 = compute this (token, head)), or NULL = all
 *   out          double [Tq][H_q][d_v];  lse double [Tq][H_q]
 * Returns 0, or -1 on inconsistent arguments (nothing written then).
 */
int oracle_link_attn(int dtype, int mla, int batch, int n_q_heads, int n_kv_heads, int d_k,
                     int d_v, const int32_t *link_offsets, const void *const *link_k,
                     const void *const *link_v, const int64_t *link_len,
                     const int32_t *q_offsets, const int32_t *self_offsets, const void *q,
                     const void *k_self, const void *v_self, double tau,
                     const int32_t *q_doc_limits, const uint8_t *row_select, double *out,
                     double *lse) {
  if (batch < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || n_q_heads % n_kv_heads) return -1;
  if (d_k <= 0 || d_v <= 0 || (mla && (n_kv_heads != 1 || d_v > d_k))) return -1;
  const int group = n_q_heads / n_kv_heads;

  for (int r = 0; r < batch; ++r) {
    const int64_t lq = q_offsets[r + 1] - q_offsets[r];
    const int64_t ls = self_offsets ? self_offsets[r + 1] - self_offsets[r] : 0;
    if (lq < 0 || ls < 0 || (self_offsets && lq > ls)) return -1;

    /* Materialise the request's linked document KV, in link order. */
    int64_t ld = 0;
    for (int c = link_offsets[r]; c < link_offsets[r + 1]; ++c) ld += link_len[c];
    if (q_doc_limits)
      for (int64_t i = 0; i < lq; ++i) {
        const int64_t lim = q_doc_limits[q_offsets[r] + i];
        if (lim < 0 || lim > ld) return -1;
      }
    const int64_t nkeys = ld + ls;
    double *kc = malloc(sizeof(double) * (size_t)(nkeys > 0 ? nkeys : 1) * n_kv_heads * d_k);
    double *vc = malloc(sizeof(double) * (size_t)(nkeys > 0 ? nkeys : 1) * n_kv_heads * d_v);
    if (!kc || !vc) { free(kc); free(vc); return -1; }
    int64_t row = 0;
    for (int c = link_offsets[r]; c < link_offsets[r + 1]; ++c) {
      widen_rows(kc + row * n_kv_heads * d_k, link_k[c], link_len[c], n_kv_heads, d_k, d_k, dtype);
      if (mla)
        widen_rows(vc + row * n_kv_heads * d_v, link_k[c], link_len[c], 1, d_v, d_k, dtype);
      else
        widen_rows(vc + row * n_kv_heads * d_v, link_v[c], link_len[c], n_kv_heads, d_v, d_v, dtype);
      row += link_len[c];
    }
    /* The own segment follows the documents. */
    if (ls > 0) {
      const int64_t s0 = self_offsets[r];
      const size_t kstride = (size_t)n_kv_heads * d_k, vstride = (size_t)n_kv_heads * d_v;
      for (int64_t t = 0; t < ls; ++t)
        for (int hh = 0; hh < n_kv_heads; ++hh) {
          for (int e = 0; e < d_k; ++e)
            kc[(ld + t) * kstride + hh * d_k + e] =
                widen(k_self, ((s0 + t) * n_kv_heads + hh) * (int64_t)d_k + e, dtype);
          for (int e = 0; e < d_v; ++e)
            vc[(ld + t) * vstride + hh * d_v + e] =
                mla ? widen(k_self, ((s0 + t) * n_kv_heads + hh) * (int64_t)d_k + e, dtype)
                    : widen(v_self, ((s0 + t) * n_kv_heads + hh) * (int64_t)d_v + e, dtype);
        }
    }

    const int64_t q0 = q_offsets[r];
    const int64_t nrows = lq * n_q_heads;
#pragma omp parallel
    {
      double *s = malloc(sizeof(double) * (size_t)(nkeys > 0 ? nkeys : 1));
      double *qi = malloc(sizeof(double) * (size_t)d_k);
      double *acc = malloc(sizeof(double) * (size_t)d_v);
#pragma omp for schedule(dynamic, 4)
      for (int64_t x = 0; x < nrows; ++x) {
        const int64_t i = x / n_q_heads;
        const int h = (int)(x % n_q_heads);
        const int64_t orow = (q0 + i) * n_q_heads + h;
        if (row_select && !row_select[orow]) continue;
        const int kv = h / group;
        for (int e = 0; e < d_k; ++e) qi[e] = widen(q, orow * d_k + e, dtype);
        /* Visible keys, numbered u = 0 .. nvis-1: document rows 0 .. dvis-1
         * (all of them unless limited), then own rows 0 .. i + ls - lq, which
         * sit at ld .. in kc / vc. */
        const int64_t dvis = q_doc_limits ? q_doc_limits[q0 + i] : ld;
        const int64_t nvis = dvis + (self_offsets ? i + 1 + ls - lq : 0);
        double m = -INFINITY;
        for (int64_t u = 0; u < nvis; ++u) {
          const int64_t j = u < dvis ? u : ld + (u - dvis);
          const double *kj = kc + (j * n_kv_heads + kv) * d_k;
          double dot = 0.0;
          for (int e = 0; e < d_k; ++e) dot += qi[e] * kj[e];
          s[u] = tau * dot;
          if (s[u] > m) m = s[u];
        }
        for (int e = 0; e < d_v; ++e) acc[e] = 0.0;
        double l = 0.0;
        for (int64_t u = 0; u < nvis; ++u) {
          const int64_t j = u < dvis ? u : ld + (u - dvis);
          const double p = exp(s[u] - m);
          const double *vj = vc + (j * n_kv_heads + kv) * d_v;
          l += p;
          for (int e = 0; e < d_v; ++e) acc[e] += p * vj[e];
        }
        double *o = out + orow * d_v;
        if (nvis == 0) {
          for (int e = 0; e < d_v; ++e) o[e] = 0.0;
          lse[orow] = -INFINITY;
        } else {
          for (int e = 0; e < d_v; ++e) o[e] = acc[e] / l;
          lse[orow] = m + log(l);
        }
      }
      free(s);
      free(qi);
      free(acc);
    }
    free(kc);
    free(vc);
  }
  return 0;
}

/* Number of threads an OpenMP region of this library uses. */
int oracle_num_threads(void) {
  int n = 1;
#pragma omp parallel
  {
#pragma omp single
    {
#ifdef _OPENMP
      n = omp_get_num_threads();
#endif
    }
  }
  return n;
}
