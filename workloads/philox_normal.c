/*
 * Counter-based normal variates for the synthetic Q/K/V inputs.
 *
 * Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
 * easy as 1, 2, 3", SC'11) keyed by (config, stream, batch, head) and counted
 * by element index, followed by the Box-Muller transform (Box & Muller, 1958)
 * in double precision, rounded to float32 and then to bfloat16 with
 * round-to-nearest-even.  Every element is a pure function of its key and
 * index, so any slice can be regenerated independently and in parallel.
 *
 * This file draws inputs only; it contains no attention arithmetic.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static void philox4x32_10(uint32_t ctr[4], uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    uint64_t p0 = (uint64_t)PHILOX_M0 * ctr[0];
    uint64_t p1 = (uint64_t)PHILOX_M1 * ctr[2];
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ ctr[1] ^ k0;
    uint32_t n2 = hi0 ^ ctr[3] ^ k1;
    ctr[0] = n0; ctr[1] = lo1; ctr[2] = n2; ctr[3] = lo0;
    k0 += PHILOX_W0; k1 += PHILOX_W1;
  }
}

static uint16_t bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* Four standard normals for one counter value (two Box-Muller pairs). */
static void normals4(uint64_t index, uint32_t k0, uint32_t k1, float out[4]) {
  uint32_t c[4] = {(uint32_t)index, (uint32_t)(index >> 32), 0u, 0u};
  philox4x32_10(c, k0, k1);
  const double two32 = 4294967296.0;
  const double two_pi = 6.283185307179586476925286766559;
  for (int p = 0; p < 2; ++p) {
    double u1 = ((double)c[2 * p] + 1.0) / two32;  /* (0, 1] */
    double u2 = (double)c[2 * p + 1] / two32;      /* [0, 1) */
    double r = sqrt(-2.0 * log(u1));
    out[2 * p] = (float)(r * cos(two_pi * u2));
    out[2 * p + 1] = (float)(r * sin(two_pi * u2));
  }
}

/*
 * Fill a [rows x cols] bfloat16 slice (row stride `ld` elements) with the
 * normals of key (k0, k1).  Element (r, c) takes variate number r*cols + c.
 * cols must be a multiple of 4.
 */
int wl_fill_normal_bf16(uint16_t* out, int64_t rows, int64_t cols, int64_t ld,
                        uint32_t k0, uint32_t k1) {
  if (cols % 4 != 0 || rows < 0) return 1;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    uint16_t* row = out + r * ld;
    for (int64_t c = 0; c < cols; c += 4) {
      float z[4];
      normals4((uint64_t)((r * cols + c) / 4), k0, k1, z);
      for (int e = 0; e < 4; ++e) row[c + e] = bf16_rne(z[e]);
    }
  }
  return 0;
}
