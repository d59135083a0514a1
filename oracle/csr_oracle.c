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
 * Rotary position embedding (optional; not part of the paper's equations,
 * which take k_n and q_n as the projections of eq. (k) and its query
 * counterpart): RoFormer's rotation (Su et al., 2021) applied to q_n and k_n at
 * their absolute cache position n before they enter the attention and the
 * cache.  The first r dims form r/2 pairs; pair i turns by the angle
 * pos * base^(-2i/r).  Two pairings are in use: "neox" pairs dim i with
 * dim i + r/2, "interleaved" pairs dim 2i with dim 2i + 1.  Dims >= r pass
 * through.  Keys already in the cache were rotated when they were appended, so
 * they are used as stored.
 *
 * FP8 KV cache (optional): keys and values are stored as OCP e4m3 codes (1 sign,
 * 4 exponent bits with bias 7, 3 mantissa bits; no infinities; S.1111.111 is
 * NaN; largest finite 448) with one dequantisation scale per tensor:
 * value = decode(code) * scale.  A value x (its bf16 or fp32 input value, or
 * with RoPE its rotation rounded to fp32) is stored as
 * code = nearest_even_e4m3(clamp(fp32(x * fp32(1 / scale)), -448, 448)).
 * Chunk keys and values enter the attention through that same quantisation,
 * so a key reads back identically whether it comes from the chunk or, on a
 * later call, from the cache.
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
enum { ROPE_NONE = 0, ROPE_NEOX = 1, ROPE_INTERLEAVED = 2 };

/*
 * Rotate one d-vector for absolute position pos (RoFormer's rotary position
 * embedding, see the file comment).  Plain double-precision evaluation of the
 * definition: angle = pos * base^(-2i/r), libm cos/sin.  y may not alias x.
 */
static void rope_row(const double* x, double* y, int d, int r, int style, double base, int64_t pos) {
  for (int c = 0; c < d; ++c) y[c] = x[c];
  if (style == ROPE_NONE) return;
  for (int i = 0; i < r / 2; ++i) {
    const double angle = (double)pos * pow(base, -2.0 * i / r);
    const double cs = cos(angle), sn = sin(angle);
    const int a = style == ROPE_NEOX ? i : 2 * i;
    const int b = style == ROPE_NEOX ? i + r / 2 : 2 * i + 1;
    y[a] = x[a] * cs - x[b] * sn;
    y[b] = x[b] * cs + x[a] * sn;
  }
}

/* Round a double to the nearest bf16 value (ties to even), returned as its
 * 16-bit pattern.  Direct from double: no intermediate rounding to float. */
static uint16_t bf16_from_double(double v) {
  if (isnan(v)) return 0x7fc0;
  const int neg = signbit(v) != 0;
  double a = fabs(v);
  double q;
  if (a == 0.0 || isinf(a)) {
    q = a;
  } else {
    int e;
    (void)frexp(a, &e);               /* a = m * 2^e, m in [0.5, 1) */
    int step = e - 8;                 /* 8 significant bits: spacing 2^(e-8) */
    if (step < -133) step = -133;     /* subnormal spacing */
    q = ldexp(nearbyint(ldexp(a, -step)), step);  /* default rounding: ties to even */
    if (q > 3.3895313892515355e38) q = INFINITY;  /* above the largest bf16 */
  }
  const float f = (float)(neg ? -q : q);  /* exact: q is a bf16 value */
  uint32_t bits;
  memcpy(&bits, &f, sizeof bits);
  return (uint16_t)(bits >> 16);
}

/* OCP e4m3 code of an fp32 value: saturate to +-448, round to nearest even
 * (subnormals in steps of 2^-9), NaN to 0x7f.  Evaluated exactly in double. */
static uint8_t e4m3_encode(float x) {
  if (isnan(x)) return 0x7f;
  const uint8_t sign = signbit(x) ? 0x80 : 0x00;
  double a = fabs((double)x);
  if (a > 448.0) a = 448.0;
  if (a < ldexp(1.0, -6)) return sign | (uint8_t)nearbyint(ldexp(a, 9)); /* 8 is the smallest normal */
  int e;
  (void)frexp(a, &e);              /* a in [2^(e-1), 2^e) */
  int E = e - 1;
  double m = nearbyint(ldexp(a, 3 - E)); /* significand in eighths: 8 .. 16 */
  if (m == 16.0) { m = 8.0; E += 1; }
  return sign | (uint8_t)(((E + 7) << 3) | ((int)m - 8));
}

static double e4m3_decode(uint8_t c) {
  const int e = (c >> 3) & 15, m = c & 7;
  if (e == 15 && m == 7) return NAN;
  const double v = e == 0 ? ldexp((double)m, -9) : ldexp((double)(8 + m), e - 10);
  return (c & 0x80) ? -v : v;
}

/* Stored code of an input value under dequantisation scale `scale`. */
static uint8_t fp8_quantize(double x, float scale) {
  const float inv = 1.0f / scale;
  return e4m3_encode((float)x * inv);
}

int csr_oracle_e4m3_encode(const float* x, uint8_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = e4m3_encode(x[i]);
  return 0;
}

int csr_oracle_e4m3_decode(const uint8_t* c, double* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = e4m3_decode(c[i]);
  return 0;
}

/*
 * Rotate n_rows d-vectors, row k at position pos[k] (fp64 in, fp64 out).
 * Returns -1 for a malformed rotation (odd or out-of-range r, unknown pairing).
 */
int csr_oracle_rope(const double* x, double* y, int64_t n_rows, int d, int r, int style, double base,
                    const int64_t* pos) {
  if (style < ROPE_NONE || style > ROPE_INTERLEAVED || r < 2 || r > d || (r & 1)) return -1;
  for (int64_t k = 0; k < n_rows; ++k) rope_row(x + k * d, y + k * d, d, r, style, base, pos[k]);
  return 0;
}

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
 * NULL (every L_b = 0: prefill).  rope_style != ROPE_NONE rotates each query
 * row and each chunk key (t >= L_b) at its absolute position (rope_dim dims,
 * base rope_theta); cached keys are used as stored.  kv_fp8: the pools hold
 * e4m3 codes (dequantised by k_scale, v_scale) and chunk keys/values enter
 * quantised as they are cached; q_scale > 0 (fp8 cache only) quantises each
 * (rotated) query element the same way under q_scale, the fp8-product mode.
 * Returns 0, or -1 for a token outside every sequence, or -2 on allocation
 * failure.
 */
int csr_oracle_attention(int dtype, int Hq, int Hkv, int d, int P, double scale, int rope_style,
                         int rope_dim, double rope_theta, int kv_fp8, float k_scale, float v_scale,
                         float q_scale, int batch,
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
    double* raw = (double*)malloc(sizeof(double) * (size_t)d);
    double* acc = (double*)calloc((size_t)(G * d), sizeof(double));
    if (!s || !qv || !kv || !raw || !acc) {
      free(s); free(qv); free(kv); free(raw); free(acc);
#ifdef _OPENMP
#pragma omp atomic write
#endif
      status = -2;
      continue;
    }
    for (int j = 0; j < G; ++j) {
      for (int c = 0; c < d; ++c) raw[c] = widen(q, ((int64_t)tok * Hq + g * G + j) * d + c, dtype);
      rope_row(raw, qv + j * d, d, rope_dim, rope_style, rope_theta, L + i);
      if (kv_fp8 && q_scale > 0.f) /* fp8 products: the (rotated) query enters as e4m3 codes too */
        for (int c = 0; c < d; ++c) qv[j * d + c] = e4m3_decode(fp8_quantize(qv[j * d + c], q_scale)) * (double)q_scale;
    }
    /* pass 1: scores */
    for (int64_t t = 0; t < nkeys; ++t) {
      int64_t base;
      const void* ksrc;
      if (t < L) { base = (cache_slot(block_table, bt_stride, P, b, t) * Hkv + g) * d; ksrc = k_pool; }
      else       { base = ((int64_t)(cu_seqlens_q[b] + (t - L)) * Hkv + g) * d; ksrc = k_new; }
      if (t < L && kv_fp8) {
        for (int c = 0; c < d; ++c) kv[c] = e4m3_decode(((const uint8_t*)ksrc)[base + c]) * (double)k_scale;
      } else {
        for (int c = 0; c < d; ++c) raw[c] = widen(ksrc, base + c, dtype);
        if (t < L) memcpy(kv, raw, sizeof(double) * (size_t)d);
        else rope_row(raw, kv, d, rope_dim, rope_style, rope_theta, t);
        if (t >= L && kv_fp8) /* a chunk key enters as it will be cached */
          for (int c = 0; c < d; ++c) kv[c] = e4m3_decode(fp8_quantize(kv[c], k_scale)) * (double)k_scale;
      }
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
      if (t < L && kv_fp8)
        for (int c = 0; c < d; ++c) kv[c] = e4m3_decode(((const uint8_t*)vsrc)[base + c]) * (double)v_scale;
      else if (kv_fp8)
        for (int c = 0; c < d; ++c)
          kv[c] = e4m3_decode(fp8_quantize(widen(vsrc, base + c, dtype), v_scale)) * (double)v_scale;
      else
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
    free(s); free(qv); free(kv); free(raw); free(acc);
  }
  return status;
}

/*
 * Append oracle (the paper's append-only growth T_{t+1} = T_t (+) dX_t,
 * Theorem 2): chunk row i of sequence b goes to cache position L_b + i; no
 * other byte of either pool changes.  Values are copied bit for bit; keys too
 * unless rope_style != ROPE_NONE, in which case each key row is first rotated
 * at its position L_b + i (in double precision) and rounded to the pool's
 * element type (nearest, ties to even).  With kv_fp8 the pools hold e4m3
 * codes: keys (rotated and rounded to fp32 first when RoPE is on) and values
 * are quantised as the file comment defines.
 */
int csr_oracle_kv_append(int dtype, int Hkv, int d, int P, int rope_style, int rope_dim,
                         double rope_theta, int kv_fp8, float k_scale, float v_scale, int batch,
                         const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                         const int32_t* block_table, int bt_stride, const int32_t* cu_seqlens_q,
                         const int32_t* cache_len) {
  const int elem_bytes = dtype == ORACLE_BF16 ? 2 : 4;
  const size_t row = (size_t)Hkv * d * elem_bytes; /* one token: all kv heads */
  double* raw = (double*)malloc(sizeof(double) * (size_t)d);
  double* rot = (double*)malloc(sizeof(double) * (size_t)d);
  if (!raw || !rot) { free(raw); free(rot); return -2; }
  for (int b = 0; b < batch; ++b) {
    const int64_t L = cache_len ? cache_len[b] : 0;
    for (int64_t i = 0; i < cu_seqlens_q[b + 1] - cu_seqlens_q[b]; ++i) {
      const int64_t slot = cache_slot(block_table, bt_stride, P, b, L + i);
      const int64_t src = cu_seqlens_q[b] + i;
      if (kv_fp8) {
        for (int g = 0; g < Hkv; ++g) {
          for (int c = 0; c < d; ++c) raw[c] = widen(k_new, (src * Hkv + g) * d + c, dtype);
          rope_row(raw, rot, d, rope_dim, rope_style, rope_theta, L + i);
          for (int c = 0; c < d; ++c) {
            const int64_t e = (slot * Hkv + g) * d + c;
            ((uint8_t*)k_pool)[e] = fp8_quantize(rot[c], k_scale);
            ((uint8_t*)v_pool)[e] = fp8_quantize(widen(v_new, (src * Hkv + g) * d + c, dtype), v_scale);
          }
        }
        continue;
      }
      memcpy((char*)v_pool + slot * row, (const char*)v_new + src * row, row);
      if (rope_style == ROPE_NONE) {
        memcpy((char*)k_pool + slot * row, (const char*)k_new + src * row, row);
        continue;
      }
      for (int g = 0; g < Hkv; ++g) {
        for (int c = 0; c < d; ++c) raw[c] = widen(k_new, (src * Hkv + g) * d + c, dtype);
        rope_row(raw, rot, d, rope_dim, rope_style, rope_theta, L + i);
        for (int c = 0; c < d; ++c) {
          const int64_t e = (slot * Hkv + g) * d + c;
          if (dtype == ORACLE_BF16) ((uint16_t*)k_pool)[e] = bf16_from_double(rot[c]);
          else ((float*)k_pool)[e] = (float)rot[c];
        }
      }
    }
  }
  free(raw); free(rot);
  return 0;
}
