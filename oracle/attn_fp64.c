/*
 * fp64 reference for masked block-sparse attention.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the oracle that the HIP path is
 * checked against; it shares no code with that path and the library never
 * calls it.  Only the tests, the smoke check and the CPU-baseline leg of the
 * benchmark may load it.
 *
 * What it computes (Section 2.1, Eq. 1): for one head, with the effective
 * interaction set E(M) obtained by expanding every active logical block
 * (qb, kb) of the mask M to its token rectangle
 *     [qb*B_Q, (qb+1)*B_Q) x [kb*B_KV, (kb+1)*B_KV),
 *     O = softmax(Q K^T / sqrt(d) + bias_M) V,
 * where bias_M(i, j) = 0 on E(M) and -inf elsewhere.  Row by row:
 *     J_i   = { j : (i, j) in E(M) }
 *     z_ij  = (1/sqrt(d)) * sum_c q_ic k_jc           (j in J_i)
 *     m_i   = max_j z_ij
 *     w_ij  = exp(z_ij - m_i)
 *     L_i   = sum_j w_ij
 *     O_i   = sum_j w_ij v_j / L_i
 *     LSE_i = m_i + ln L_i                             (natural log)
 * Subtracting m_i before exponentiating changes nothing mathematically; it
 * only keeps exp() in range.  A query row with J_i empty has no defined
 * softmax (Eq. 1 gives 0/0); the reading taken here is O_i = 0 and
 * LSE_i = -inf.  Blocks at a ragged sequence end cover only the tokens that
 * exist.
 *
 * Inputs are bfloat16 bit patterns, widened exactly to double; every
 * operation after that is IEEE double.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double bf16_to_double(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/*
 * Strides are in elements and ordered (batch, head, token); the head-dim
 * stride is 1.  The mask of head h in batch b starts at
 * mask + b*mask_stride_b + mask_head_offset[h] and is a row-major
 * [ceil(Nq/bq[h])] x [ceil(Nkv/bkv[h])] byte matrix, nonzero = active.
 *
 * rows: NULL for every (b, h, i) in that nesting order, or an array of
 * nrows triples (b, h, i).  out receives nrows x d doubles, lse nrows doubles
 * (lse may be NULL).  Returns 0, or 1 on an argument error.
 */
int oracle_masked_attention(int32_t B, int32_t H, int32_t Nq, int32_t Nkv, int32_t d,
                            const uint16_t* q, const int64_t* q_stride,
                            const uint16_t* k, const int64_t* k_stride,
                            const uint16_t* v, const int64_t* v_stride,
                            const uint8_t* mask, const int64_t* mask_head_offset, int64_t mask_stride_b,
                            const int32_t* bq, const int32_t* bkv,
                            const int64_t* rows, int64_t nrows,
                            double* out, double* lse) {
  if (B <= 0 || H <= 0 || Nq < 0 || Nkv < 0 || d <= 0) return 1;
  if (!rows) nrows = (int64_t)B * H * Nq;
  for (int32_t h = 0; h < H; ++h)
    if (bq[h] <= 0 || bkv[h] <= 0) return 1;
  if (rows) {
    for (int64_t r = 0; r < nrows; ++r) {
      int64_t b = rows[3 * r], h = rows[3 * r + 1], i = rows[3 * r + 2];
      if (b < 0 || b >= B || h < 0 || h >= H || i < 0 || i >= Nq) return 1;
    }
  }
  const double scale = 1.0 / sqrt((double)d);

#pragma omp parallel
  {
    double* z = (double*)malloc(sizeof(double) * (Nkv > 0 ? (size_t)Nkv : 1));
    int32_t* jj = (int32_t*)malloc(sizeof(int32_t) * (Nkv > 0 ? (size_t)Nkv : 1));
    double* qi = (double*)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(dynamic, 8)
    for (int64_t r = 0; r < nrows; ++r) {
      int64_t b, h, i;
      if (rows) {
        b = rows[3 * r]; h = rows[3 * r + 1]; i = rows[3 * r + 2];
      } else {
        b = r / ((int64_t)H * Nq); h = (r / Nq) % H; i = r % Nq;
      }
      const int64_t nkb = (Nkv + bkv[h] - 1) / bkv[h];
      const uint8_t* mrow = mask + b * mask_stride_b + mask_head_offset[h] + (i / bq[h]) * nkb;
      const uint16_t* qrow = q + b * q_stride[0] + h * q_stride[1] + i * q_stride[2];
      for (int32_t c = 0; c < d; ++c) qi[c] = bf16_to_double(qrow[c]);

      /* J_i and the scaled scores z_ij */
      int64_t n = 0;
      double m = -INFINITY;
      for (int64_t kb = 0; kb < nkb; ++kb) {
        if (!mrow[kb]) continue;
        int64_t j_end = (kb + 1) * bkv[h] < Nkv ? (kb + 1) * bkv[h] : Nkv;
        for (int64_t j = kb * bkv[h]; j < j_end; ++j) {
          const uint16_t* krow = k + b * k_stride[0] + h * k_stride[1] + j * k_stride[2];
          double dot = 0.0;
          for (int32_t c = 0; c < d; ++c) dot += qi[c] * bf16_to_double(krow[c]);
          z[n] = scale * dot;
          jj[n] = (int32_t)j;
          if (z[n] > m) m = z[n];
          ++n;
        }
      }
      double* o = out + r * d;
      for (int32_t c = 0; c < d; ++c) o[c] = 0.0;
      if (n == 0) {
        if (lse) lse[r] = -INFINITY;
        continue;
      }
      double L = 0.0;
      for (int64_t t = 0; t < n; ++t) {
        double w = exp(z[t] - m);
        L += w;
        const uint16_t* vrow = v + b * v_stride[0] + h * v_stride[1] + (int64_t)jj[t] * v_stride[2];
        for (int32_t c = 0; c < d; ++c) o[c] += w * bf16_to_double(vrow[c]);
      }
      for (int32_t c = 0; c < d; ++c) o[c] /= L;
      if (lse) lse[r] = m + log(L);
    }
    free(z);
    free(jj);
    free(qi);
  }
  return 0;
}

/* Number of OpenMP threads a parallel region of this library uses. */
int oracle_num_threads(void) {
  int n = 1;
#pragma omp parallel
  {
#pragma omp single
    {
#ifdef _OPENMP
      extern int omp_get_num_threads(void);
      n = omp_get_num_threads();
#endif
    }
  }
  return n;
}
