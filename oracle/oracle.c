/*
 * oracle.c -- plain CPU oracle (TEST INFRASTRUCTURE ONLY; see oracle.h).
 *
 * Written from the definitions of the operations, not for speed:
 *   block gather / scatter ............ publish / hydrate of paged KV blocks
 *                                        (paper Sec. 3.2, Table 2)
 *   fragment copy ...................... batched replica moves, prefetch_many
 *                                        (Table 2) and the pipeline's transfer
 *                                        stage (Sec. 5)
 *   block-scaled E4M3 cast ............. a transform_into `spec` rule
 *                                        (Table 2); encoding per the OCP
 *                                        8-bit floating point definition.
 *   inverse cast ....................... E4M3 codes and tile scales back to
 *                                        bf16 (the training-side rule of
 *                                        Sec. 7)
 *   fragment digests ................... the pipeline's verify-integrity
 *                                        stage (Sec. 5): a byte sum and a
 *                                        position-weighted byte sum
 * Build: gcc -O2 -fno-fast-math -fopenmp -shared -fPIC.
 */
#include "oracle.h"

#include <math.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>
#include <xmmintrin.h>

/* Denormals must be honoured: a tile scale can be an fp32 subnormal. */
static void ieee_mode(void) {
  unsigned csr = _mm_getcsr();
  csr &= ~(1u << 15); /* FTZ */
  csr &= ~(1u << 6);  /* DAZ */
  _mm_setcsr(csr);
}

int orc_threads(void) { return omp_get_max_threads(); }
void orc_set_threads(int n) {
  if (n > 0) omp_set_num_threads(n);
}

/* ------------------------------------------------------------------ */
/* Block gather / scatter                                              */
/* ------------------------------------------------------------------ */

int orc_gather_blocks(const uint8_t* const* regions, int32_t num_regions,
                      int64_t num_blocks, int64_t block_bytes,
                      int64_t block_stride, const int32_t* ids, int64_t n,
                      uint8_t* out) {
  for (int64_t i = 0; i < n; i++)
    if (ids[i] < 0 || ids[i] >= num_blocks) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; i++) {
    for (int32_t r = 0; r < num_regions; r++) {
      const uint8_t* from = regions[r] + (int64_t)ids[i] * block_stride;
      uint8_t* to = out + (i * num_regions + r) * block_bytes;
      memcpy(to, from, (size_t)block_bytes);
    }
  }
  return 0;
}

int orc_scatter_blocks(uint8_t* const* regions, int32_t num_regions,
                       int64_t num_blocks, int64_t block_bytes,
                       int64_t block_stride, const int32_t* ids, int64_t n,
                       const uint8_t* in) {
  for (int64_t i = 0; i < n; i++)
    if (ids[i] < 0 || ids[i] >= num_blocks) return -1;
  /* Distinct ids: with a repeat the result would depend on write order. */
  uint8_t* seen = (uint8_t*)calloc((size_t)num_blocks, 1);
  if (!seen) return -3;
  for (int64_t i = 0; i < n; i++) {
    if (seen[ids[i]]) {
      free(seen);
      return -2;
    }
    seen[ids[i]] = 1;
  }
  free(seen);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; i++) {
    for (int32_t r = 0; r < num_regions; r++) {
      uint8_t* to = regions[r] + (int64_t)ids[i] * block_stride;
      const uint8_t* from = in + (i * num_regions + r) * block_bytes;
      memcpy(to, from, (size_t)block_bytes);
    }
  }
  return 0;
}

/* ------------------------------------------------------------------ */
/* Fragment copy                                                       */
/* ------------------------------------------------------------------ */

void orc_copy_fragments(const uint8_t* src, uint8_t* dst, const orc_frag* f,
                        int64_t n) {
#pragma omp parallel for schedule(dynamic, 64)
  for (int64_t d = 0; d < n; d++) {
    if (f[d].len) memcpy(dst + f[d].dst_off, src + f[d].src_off, (size_t)f[d].len);
  }
}

/* ------------------------------------------------------------------ */
/* E4M3 (OCP "fn" flavour)                                             */
/* ------------------------------------------------------------------ */
/* Code layout: S EEEE MMM, exponent bias 7.  Exponent field 0 holds the
 * subnormals m * 2^-9; field e > 0 holds 2^(e-7) * (1 + m/8).  The pattern
 * S.1111.111 is NaN, so the largest finite magnitude is code 0x7E = 448. */

#define E4M3_MAX_CODE 126
static double g_mag[E4M3_MAX_CODE + 1]; /* magnitude of codes 0..126, increasing */

static double e4m3_magnitude(int code) {
  int e = code >> 3, m = code & 7;
  if (e == 0) return ldexp((double)m, -9);
  return ldexp((double)(8 + m), e - 10); /* (1 + m/8) * 2^(e-7) */
}

__attribute__((constructor)) static void e4m3_init(void) {
  for (int c = 0; c <= E4M3_MAX_CODE; c++) g_mag[c] = e4m3_magnitude(c);
}

uint8_t orc_e4m3_encode(float v) {
  if (isnan(v)) return 0x7F;
  uint8_t sign = signbit(v) ? 0x80 : 0x00;
  double a = fabs((double)v); /* exact: every binary32 value is a binary64 value */
  if (a >= g_mag[E4M3_MAX_CODE]) return sign | E4M3_MAX_CODE; /* satfinite */
  /* g_mag[lo] <= a < g_mag[hi] */
  int lo = 0, hi = E4M3_MAX_CODE;
  while (hi - lo > 1) {
    int mid = (lo + hi) / 2;
    if (g_mag[mid] <= a)
      lo = mid;
    else
      hi = mid;
  }
  /* The midpoint of two adjacent E4M3 magnitudes needs at most 5 significant
   * bits, so it is exact in binary64 and the comparisons below are exact. */
  double midpoint = 0.5 * (g_mag[lo] + g_mag[hi]);
  int code;
  if (a < midpoint)
    code = lo;
  else if (a > midpoint)
    code = hi;
  else
    code = (lo & 1) ? hi : lo; /* tie: even mantissa LSB */
  return (uint8_t)(sign | code);
}

float orc_e4m3_decode(uint8_t code) {
  int mag = code & 0x7F;
  if (mag == 0x7F) return NAN;
  float v = (float)e4m3_magnitude(mag);
  return (code & 0x80) ? -v : v;
}

static float bf16_value(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

void orc_cast_fp8_scaled(const uint16_t* x, int64_t n, float scale,
                         uint8_t* q) {
  ieee_mode();
#pragma omp parallel
  {
    ieee_mode();
#pragma omp for schedule(static)
    for (int64_t i = 0; i < n; i++) {
      float quotient = bf16_value(x[i]) / scale; /* binary32, round to nearest even */
      q[i] = orc_e4m3_encode(quotient);
    }
  }
}

void orc_cast_fp8_blockscaled(const uint16_t* x, int64_t rows, int64_t cols,
                              int64_t ld, uint8_t* q, int64_t q_ld,
                              float* scales, int64_t scale_ld) {
  const int64_t T = 128;
  int64_t tile_rows = (rows + T - 1) / T, tile_cols = (cols + T - 1) / T;
  uint32_t nan_bits = 0x7FC00000u;
  float nan_scale;
  memcpy(&nan_scale, &nan_bits, 4);
  ieee_mode();
#pragma omp parallel
  {
    ieee_mode();
#pragma omp for collapse(2) schedule(dynamic, 4)
    for (int64_t ti = 0; ti < tile_rows; ti++) {
      for (int64_t tj = 0; tj < tile_cols; tj++) {
        int64_t r0 = ti * T, r1 = r0 + T < rows ? r0 + T : rows;
        int64_t c0 = tj * T, c1 = c0 + T < cols ? c0 + T : cols;
        float amax = 0.0f;
        int nonfinite = 0;
        for (int64_t r = r0; r < r1; r++)
          for (int64_t c = c0; c < c1; c++) {
            float v = bf16_value(x[r * ld + c]);
            if (!isfinite(v))
              nonfinite = 1;
            else if (fabsf(v) > amax)
              amax = fabsf(v);
          }
        float s;
        if (nonfinite) {
          s = nan_scale;
          for (int64_t r = r0; r < r1; r++)
            for (int64_t c = c0; c < c1; c++) q[r * q_ld + c] = 0x7F;
        } else if (amax == 0.0f) {
          s = 0.0f;
          for (int64_t r = r0; r < r1; r++)
            for (int64_t c = c0; c < c1; c++)
              q[r * q_ld + c] = (x[r * ld + c] & 0x8000u) ? 0x80 : 0x00;
        } else {
          s = amax / 448.0f; /* binary32 quotient, round to nearest even */
          for (int64_t r = r0; r < r1; r++)
            for (int64_t c = c0; c < c1; c++) {
              float quotient = bf16_value(x[r * ld + c]) / s;
              q[r * q_ld + c] = orc_e4m3_encode(quotient);
            }
        }
        scales[ti * scale_ld + tj] = s;
      }
    }
  }
}

/* ------------------------------------------------------------------ */
/* Inverse cast                                                        */
/* ------------------------------------------------------------------ */

/* bf16 keeps the top 16 bits of a binary32 value: round the dropped 16 bits
 * to nearest, ties to the even kept bit. */
uint16_t orc_bf16_round(float v) {
  if (isnan(v)) return 0x7FC0;
  uint32_t u;
  memcpy(&u, &v, 4);
  uint32_t kept = u >> 16, dropped = u & 0xFFFFu;
  if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u))) kept += 1; /* carries into the exponent */
  return (uint16_t)kept;
}

void orc_dequant_fp8_blockscaled(const uint8_t* q, int64_t rows, int64_t cols, int64_t q_ld,
                                 const float* scales, int64_t scale_ld, uint16_t* y,
                                 int64_t y_ld) {
  ieee_mode();
#pragma omp parallel
  {
    ieee_mode();
#pragma omp for schedule(static)
    for (int64_t r = 0; r < rows; r++) {
      for (int64_t c = 0; c < cols; c++) {
        float s = scales[(r / 128) * scale_ld + c / 128];
        float v = orc_e4m3_decode(q[r * q_ld + c]) * s; /* binary32 product, round to nearest even */
        y[r * y_ld + c] = orc_bf16_round(v);
      }
    }
  }
}

/* ------------------------------------------------------------------ */
/* Fragment digests                                                    */
/* ------------------------------------------------------------------ */

void orc_fragment_digests(const uint8_t* base, const orc_frag* f, int64_t n, int use_src,
                          uint64_t* out) {
#pragma omp parallel for schedule(dynamic, 64)
  for (int64_t d = 0; d < n; d++) {
    const uint8_t* p = base + (use_src ? f[d].src_off : f[d].dst_off);
    uint64_t s1 = 0, s2 = 0;
    for (uint64_t i = 0; i < f[d].len; i++) {
      s1 += p[i];
      s2 += (i + 1) * (uint64_t)p[i];
    }
    out[2 * d] = s1;
    out[2 * d + 1] = s2;
  }
}
