/*
 * CPU fp64 oracle for cached-prefix extend attention, full re-prefill and the
 * paged KV append.  TEST INFRASTRUCTURE ONLY: nothing on the product path may
 * link, load or call this file; only the tests, the smoke check and the
 * benchmark's CPU-baseline leg do.  It shares no code with the HIP library.
 *
 * What it computes (the paper's causal attention and KV cache, Sec. II,
 * eq. (causal_attention_1)-(causal_attention_3) and eq. (K_cache)-(V_cache)):
 *
 *   for sequence b, chunk row i (absolute position p = L_b + i), query head h,
 *   kv head g = h / (Hq / Hkv):
 *     keys t = 0 .. p inclusive (a token attends to itself and everything
 *     before it), where key/value t comes from the paged cache for t < L_b and
 *     from the new chunk's own K/V rows for t >= L_b;
 *     s_t = scale * <q, k_t>,  scale = 1/sqrt(d) unless given;
 *     a_t = exp(s_t - max s) / sum_t exp(s_t - max s);
 *     o   = sum_t a_t v_t;   lse = max s + ln sum_t exp(s_t - max s).
 *
 * The cached prefix length L_b is the CSR stable-prefix length (the paper's
 * i* = |X_static| + 1 means tokens 1 .. i*-1 are reused), so L_b = i* - 1.
 * A full re-prefill (the warm-up of asynchronous state reconciliation) is the
 * same computation with L_b = 0.
 *
 * Evaluation is the plain definition in double precision, two passes per row
 * (max, then exponentials and the weighted sum), no blocking, no online
 * rescaling.  bf16 inputs are widened exactly (a bf16 value is the upper 16
 * bits of an IEEE binary32 value).
 *
 * Paged cache layout (the library's contract; one convention for both sides):
 *   pool[num_pages][P][Hkv][d]; logical position t of sequence b lives in
 *   slot = page * P + (t mod P), page = block_table[b * bt_stride + t / P];
 *   a NULL block table means page = b * bt_stride + t / P (each sequence owns
 *   a contiguous run of bt_stride pages).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_F32 = 0, ORACLE_BF16 = 1 };

static double widen(const void* base, int64_t idx, int dtype) {
  if (dtype == ORACLE_BF16) {
    uint32_t bits = (uint32_t)((const uint16_t*)base)[idx] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
  }
  return (double)((const float*)base)[idx];
}

static int64_t cache_slot(const int32_t* block_table, int bt_stride, int P, int b, int64_t t) {
  int64_t page = block_table ? (int64_t)block_table[(int64_t)b * bt_stride + t / P]
                             : (int64_t)b * bt_stride + t / P;
  return page * P + t % P;
}

/* Sequence that owns packed query token `tok` (cu_seqlens is a prefix sum). */
static int owner(const int32_t* cu, int batch, int tok) {
  for (int b = 0; b < batch; ++b)
    if (tok >= cu[b] && tok < cu[b + 1]) return b;
  return -1;
}

/*
 * Attention for the query tokens listed in `rows` (indices into the packed
 * [T_q, Hq, d] query array), all heads.  out: [n_rows, Hq, d], lse: [n_rows, Hq],
 * pairs: [n_rows, Hq] number of (query, key) pairs evaluated.  cache_len may be
 * NULL (every L_b = 0: prefill).  Returns 0, or -1 for a token outside every
 * sequence, or -2 on allocation failure.
 */
int csr_oracle_attention(int dtype, int Hq, int Hkv, int d, int P, double scale, int batch,
                         const void* q, const void* k_new, const void* v_new, const void* k_pool,
                         const void* v_pool, const int32_t* block_table, int bt_stride,
                         const int32_t* cu_seqlens_q, const int32_t* cache_len, int n_rows,
                         const int32_t* rows, double* out, double* lse, int64_t* pairs,
                         int nthreads) {
  const int G = Hq / Hkv;
  if (scale <= 0.0) scale = 1.0 / sqrt((double)d);
  for (int r = 0; r < n_rows; ++r)
    if (owner(cu_seqlens_q, batch, rows[r]) < 0) return -1;
  int status = 0;
  const int64_t ntask = (int64_t)n_rows * Hkv;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int64_t task = 0; task < ntask; ++task) {
    const int r = (int)(task / Hkv), g = (int)(task % Hkv);
    const int tok = rows[r];
    const int b = owner(cu_seqlens_q, batch, tok);
    const int64_t L = cache_len ? cache_len[b] : 0;
    const int64_t i = tok - cu_seqlens_q[b];
    const int64_t nkeys = L + i + 1; /* keys 0 .. L + i inclusive */
    double* s = (double*)malloc(sizeof(double) * (size_t)(G * nkeys));
    double* qv = (double*)malloc(sizeof(double) * (size_t)(G * d));
    double* kv = (double*)malloc(sizeof(double) * (size_t)d);
    double* acc = (double*)calloc((size_t)(G * d), sizeof(double));
    if (!s || !qv || !kv || !acc) {
      free(s); free(qv); free(kv); free(acc);
#ifdef _OPENMP
#pragma omp atomic write
#endif
      status = -2;
      continue;
    }
    for (int j = 0; j < G; ++j)
      for (int c = 0; c < d; ++c)
        qv[j * d + c] = widen(q, ((int64_t)tok * Hq + g * G + j) * d + c, dtype);
    /* pass 1: scores */
    for (int64_t t = 0; t < nkeys; ++t) {
      int64_t base;
      const void* ksrc;
      if (t < L) { base = (cache_slot(block_table, bt_stride, P, b, t) * Hkv + g) * d; ksrc = k_pool; }
      else       { base = ((int64_t)(cu_seqlens_q[b] + (t - L)) * Hkv + g) * d; ksrc = k_new; }
      for (int c = 0; c < d; ++c) kv[c] = widen(ksrc, base + c, dtype);
      for (int j = 0; j < G; ++j) {
        double dot = 0.0;
        for (int c = 0; c < d; ++c) dot += qv[j * d + c] * kv[c];
        s[j * nkeys + t] = scale * dot;
      }
    }
    /* pass 2: softmax weights and the weighted sum of values */
    double m[64], l[64]; /* G <= 64 is checked by the wrapper */
    for (int j = 0; j < G; ++j) {
      m[j] = -INFINITY;
      for (int64_t t = 0; t < nkeys; ++t) if (s[j * nkeys + t] > m[j]) m[j] = s[j * nkeys + t];
      l[j] = 0.0;
      for (int64_t t = 0; t < nkeys; ++t) {
        s[j * nkeys + t] = exp(s[j * nkeys + t] - m[j]);
        l[j] += s[j * nkeys + t];
      }
    }
    for (int64_t t = 0; t < nkeys; ++t) {
      int64_t base;
      const void* vsrc;
      if (t < L) { base = (cache_slot(block_table, bt_stride, P, b, t) * Hkv + g) * d; vsrc = v_pool; }
      else       { base = ((int64_t)(cu_seqlens_q[b] + (t - L)) * Hkv + g) * d; vsrc = v_new; }
      for (int c = 0; c < d; ++c) kv[c] = widen(vsrc, base + c, dtype);
      for (int j = 0; j < G; ++j) {
        const double w = s[j * nkeys + t];
        for (int c = 0; c < d; ++c) acc[j * d + c] += w * kv[c];
      }
    }
    for (int j = 0; j < G; ++j) {
      const int h = g * G + j;
      for (int c = 0; c < d; ++c) out[((int64_t)r * Hq + h) * d + c] = acc[j * d + c] / l[j];
      lse[(int64_t)r * Hq + h] = m[j] + log(l[j]);
      pairs[(int64_t)r * Hq + h] = nkeys;
    }
    free(s); free(qv); free(kv); free(acc);
  }
  return status;
}

/*
 * Append oracle (the paper's append-only growth T_{t+1} = T_t (+) dX_t,
 * Theorem 2): chunk row i of sequence b is copied bit for bit into cache
 * position L_b + i; no other byte of either pool changes.
 */
int csr_oracle_kv_append(int elem_bytes, int Hkv, int d, int P, int batch, const void* k_new,
                         const void* v_new, void* k_pool, void* v_pool,
                         const int32_t* block_table, int bt_stride, const int32_t* cu_seqlens_q,
                         const int32_t* cache_len) {
  const size_t row = (size_t)Hkv * d * elem_bytes; /* one token: all kv heads */
  for (int b = 0; b < batch; ++b) {
    const int64_t L = cache_len ? cache_len[b] : 0;
    for (int64_t i = 0; i < cu_seqlens_q[b + 1] - cu_seqlens_q[b]; ++i) {
      const int64_t slot = cache_slot(block_table, bt_stride, P, b, L + i);
      const int64_t src = cu_seqlens_q[b] + i;
      memcpy((char*)k_pool + slot * row, (const char*)k_new + src * row, row);
      memcpy((char*)v_pool + slot * row, (const char*)v_new + src * row, row);
    }
  }
  return 0;
}
