/*
 * oracle_attn.c -- TEST INFRASTRUCTURE, not part of the product path.
 *
 * Plain, slow, fp64 CPU reference for chunked causal prefill attention.
 * Only tests/, the smoke check and the benchmark's CPU-baseline leg use it.
 * It shares no code with the HIP library.
 *
 * What it computes (plain definition, no tiling, no blocking):
 *   The paper (MOCAP, Section 2.2 "Chunked Pipeline") states that every chunk
 *   attends to the keys and values produced by all chunks before it, and
 *   Eq. (1) in Section 3.2 prices chunk i as c_i (p_i + c_i) with
 *   p_i = sum_{j<i} c_j, i.e. its c_i queries see the p_i prefix keys plus
 *   its own keys.  The paper does not write the attention formula itself;
 *   it is standard scaled dot-product attention with a causal mask:
 *
 *     for chunk-local query row i (absolute position t = P + i), head h,
 *     kv head kvh = floor(h / (Hq / Hkv))            (contiguous GQA groups)
 *       s_j   = scale * <q_i,h , k_j,kvh>            j = 0 .. t (inclusive)
 *       lse   = log( sum_j exp(s_j) )                natural log
 *       o_i,h = sum_j exp(s_j - lse) * v_j,kvh
 *
 *   Keys are read from the logical, contiguous sequence: there is no block
 *   table, no split and no reduced precision here.  Inputs are either fp64
 *   arrays or bf16 bit patterns that are widened exactly to fp64.
 *
 * Layouts (row-major):
 *   q   [L][Hq][d]        the chunk's queries
 *   k,v [>= P+L][Hkv][d]  logical keys/values from position 0
 *   o   [nrows][Hq][d]    fp64 output for the requested rows
 *   lse [Hq][nrows]       fp64, natural log
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double widen(const void* base, int64_t idx, int is_bf16) {
  if (is_bf16) {
    uint32_t bits = ((uint32_t)((const uint16_t*)base)[idx]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
  }
  return ((const double*)base)[idx];
}

/* Returns 0 on success, -1 on bad arguments, -2 on allocation failure. */
int oracle_chunk_attn(const void* q, const void* k, const void* v, int is_bf16,
                      int64_t prefix_len, int64_t chunk_len, int h_q, int h_kv, int d,
                      double scale, const int64_t* rows, int64_t n_rows, double* o,
                      double* lse, int n_threads) {
  if (h_q <= 0 || h_kv <= 0 || d <= 0 || h_q % h_kv != 0 || prefix_len < 0 ||
      chunk_len < 0 || n_rows < 0)
    return -1;
  for (int64_t r = 0; r < n_rows; ++r)
    if (rows[r] < 0 || rows[r] >= chunk_len) return -1;
  const int group = h_q / h_kv;
  const int64_t max_keys = prefix_len + chunk_len;
  int bad_alloc = 0;
#ifdef _OPENMP
  if (n_threads > 0) omp_set_num_threads(n_threads);
#else
  (void)n_threads;
#endif

#pragma omp parallel
  {
    double* s = (double*)malloc(sizeof(double) * (size_t)(max_keys > 0 ? max_keys : 1));
    double* acc = (double*)malloc(sizeof(double) * (size_t)d);
    const int have_buffers = s != NULL && acc != NULL;
    if (!have_buffers) {
#pragma omp atomic write
      bad_alloc = 1;
    }
    /* Every thread of the team reaches the work-sharing loop (OpenMP
       requires it); a thread without buffers takes no task, and the call
       then reports -2. */
    {
#pragma omp for schedule(dynamic, 1)
      for (int64_t task = 0; task < n_rows * h_q; ++task) {
        if (!have_buffers) continue;
        const int64_t r = task / h_q;
        const int h = (int)(task % h_q);
        const int64_t i = rows[r];
        const int64_t t = prefix_len + i; /* absolute position of the query */
        const int kvh = h / group;
        const int64_t q_off = (i * h_q + h) * (int64_t)d;

        /* scores over every visible key j <= t */
        double m = -INFINITY;
        for (int64_t j = 0; j <= t; ++j) {
          const int64_t k_off = (j * h_kv + kvh) * (int64_t)d;
          double dot = 0.0;
          for (int e = 0; e < d; ++e) dot += widen(q, q_off + e, is_bf16) * widen(k, k_off + e, is_bf16);
          s[j] = scale * dot;
          if (s[j] > m) m = s[j];
        }
        double z = 0.0;
        for (int64_t j = 0; j <= t; ++j) z += exp(s[j] - m);
        const double row_lse = m + log(z);

        for (int e = 0; e < d; ++e) acc[e] = 0.0;
        for (int64_t j = 0; j <= t; ++j) {
          const double p = exp(s[j] - row_lse);
          const int64_t v_off = (j * h_kv + kvh) * (int64_t)d;
          for (int e = 0; e < d; ++e) acc[e] += p * widen(v, v_off + e, is_bf16);
        }
        for (int e = 0; e < d; ++e) o[(r * h_q + h) * (int64_t)d + e] = acc[e];
        lse[(int64_t)h * n_rows + r] = row_lse;
      }
    }
    free(s);
    free(acc);
  }
  return bad_alloc ? -2 : 0;
}

/* Number of OpenMP threads a parallel region would use (for reporting). */
int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
