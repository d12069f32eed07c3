/*
 * A C program that uses the library through its C ABI alone: device memory
 * from hipMalloc, the calls from tensorcast_hip.h, results checked on the
 * host against expectations this program computes itself.  Exits 0 when
 * every check passes.
 *
 *   1. publish / hydrate: gather 10 blocks of a 2-region pool into a transfer
 *      buffer, scatter them into a second pool (distinct ids);
 *   2. fragments: plan three byte fragments once, copy them twice;
 *   3. digests of the same plan, against sums computed here;
 *   4. the block-scaled fp8 cast of a 256 x 256 bf16 matrix, prepared once
 *      in a workspace with the per-tile table, and its inverse.  Every tile
 *      holds the values {1, 2, 1/2, 448, -7/2} times its own power of two,
 *      so its scale is that power exactly, the E4M3 codes are known
 *      constants and the inverse gives the source back bit for bit.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "tensorcast_hip.h"

#define CHECK_HIP(x)                                                   \
  do {                                                                 \
    hipError_t e_ = (x);                                               \
    if (e_ != hipSuccess) {                                            \
      fprintf(stderr, "HIP error %d at line %d\n", (int)e_, __LINE__); \
      return 1;                                                        \
    }                                                                  \
  } while (0)
#define CHECK_TC(x)                                                                  \
  do {                                                                               \
    tc_status s_ = (x);                                                              \
    if (s_ != TC_OK) {                                                               \
      fprintf(stderr, "%s at line %d: %s\n", #x, __LINE__, tc_status_string(s_));   \
      return 1;                                                                      \
    }                                                                                \
  } while (0)

enum { R = 2, NB = 64, B = 4096, N = 10, POOL = 1 << 20 };
/* the pool (R * NB * B bytes) and the gathered buffer fit in POOL bytes */
typedef char pool_fits[(R * NB * B <= POOL && N * R * B <= POOL) ? 1 : -1];

int main(void) {
  /* 1. gather / scatter */
  /* one host buffer serves as the pool's contents and as the fragment source */
  uint8_t* host = (uint8_t*)malloc(POOL);
  uint8_t* got = (uint8_t*)malloc(POOL);
  if (!host || !got) return 1;
  for (size_t i = 0; i < POOL; ++i) host[i] = (uint8_t)(i * 2654435761u >> 24);
  void *pool_a, *pool_b, *buf, *ids_d;
  CHECK_HIP(hipMalloc(&pool_a, (size_t)R * NB * B));
  CHECK_HIP(hipMalloc(&pool_b, (size_t)R * NB * B));
  CHECK_HIP(hipMalloc(&buf, (size_t)N * R * B));
  CHECK_HIP(hipMalloc(&ids_d, N * sizeof(int32_t)));
  CHECK_HIP(hipMemcpy(pool_a, host, (size_t)R * NB * B, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemset(pool_b, 0, (size_t)R * NB * B));
  const int32_t ids[N] = {5, 63, 0, 17, 42, 8, 33, 1, 60, 21};
  CHECK_HIP(hipMemcpy(ids_d, ids, sizeof(ids), hipMemcpyHostToDevice));
  uint64_t ra[R] = {(uint64_t)(uintptr_t)pool_a, (uint64_t)(uintptr_t)pool_a + (uint64_t)NB * B};
  uint64_t rb[R] = {(uint64_t)(uintptr_t)pool_b, (uint64_t)(uintptr_t)pool_b + (uint64_t)NB * B};
  tc_block_pool pa = {ra, R, NB, B, B}, pb = {rb, R, NB, B, B};
  CHECK_TC(tc_gather_blocks(&pa, (const int32_t*)ids_d, N, buf, 0));
  CHECK_TC(tc_scatter_blocks(&pb, (const int32_t*)ids_d, N, buf, 0));
  CHECK_HIP(hipMemcpy(got, buf, (size_t)N * R * B, hipMemcpyDeviceToHost));
  for (int i = 0; i < N; ++i)
    for (int r = 0; r < R; ++r)
      if (memcmp(got + ((size_t)i * R + r) * B, host + ((size_t)r * NB + ids[i]) * B, B)) {
        fprintf(stderr, "gather: id %d region %d differs\n", ids[i], r);
        return 1;
      }
  CHECK_HIP(hipMemcpy(got, pool_b, (size_t)R * NB * B, hipMemcpyDeviceToHost));
  for (int r = 0; r < R; ++r)
    for (int b = 0; b < NB; ++b) {
      int written = 0;
      for (int i = 0; i < N; ++i) written |= ids[i] == b;
      const uint8_t* g = got + ((size_t)r * NB + b) * B;
      for (int k = 0; k < B; ++k)
        if (g[k] != (written ? host[((size_t)r * NB + b) * B + k] : 0)) {
          fprintf(stderr, "scatter: region %d block %d differs\n", r, b);
          return 1;
        }
    }

  /* 2. planned fragment copy, used twice */
  const tc_fragment fr[3] = {{100, 5000, 3000}, {70000, 100000, 65536}, {9, 900000, 17}};
  void *src, *dst, *fr_d, *ws, *dg;
  CHECK_HIP(hipMalloc(&src, POOL));
  CHECK_HIP(hipMalloc(&dst, POOL));
  CHECK_HIP(hipMalloc(&fr_d, sizeof(fr)));
  CHECK_HIP(hipMemcpy(src, host, POOL, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(fr_d, fr, sizeof(fr), hipMemcpyHostToDevice));
  const size_t ws_bytes = tc_copy_fragments_workspace(3);
  CHECK_HIP(hipMalloc(&ws, ws_bytes));
  CHECK_HIP(hipMalloc(&dg, 6 * sizeof(uint64_t)));
  uint64_t total = 0;
  CHECK_TC(tc_plan_fragments((const tc_fragment*)fr_d, 3, ws, ws_bytes, &total, 0));
  for (int pass = 0; pass < 2; ++pass) {
    CHECK_HIP(hipMemset(dst, 0xEE, POOL));
    CHECK_TC(tc_copy_planned(src, dst, ws, ws_bytes, total, 0));
    CHECK_HIP(hipMemcpy(got, dst, POOL, hipMemcpyDeviceToHost));
    for (int f = 0; f < 3; ++f)
      if (memcmp(got + fr[f].dst_off, host + fr[f].src_off, fr[f].len)) {
        fprintf(stderr, "fragment %d differs (pass %d)\n", f, pass);
        return 1;
      }
    if (got[4999] != 0xEE || got[8000] != 0xEE) {
      fprintf(stderr, "bytes outside the fragments changed\n");
      return 1;
    }
  }

  /* 3. digests of the same plan */
  uint64_t d[6];
  CHECK_TC(tc_digest_planned(src, TC_DIGEST_SRC, ws, ws_bytes, total, 3, (uint64_t*)dg, 0));
  CHECK_HIP(hipMemcpy(d, dg, sizeof(d), hipMemcpyDeviceToHost));
  for (int f = 0; f < 3; ++f) {
    uint64_t s1 = 0, s2 = 0;
    for (uint64_t i = 0; i < fr[f].len; ++i) {
      s1 += host[fr[f].src_off + i];
      s2 += (i + 1) * host[fr[f].src_off + i];
    }
    if (d[2 * f] != s1 || d[2 * f + 1] != s2) {
      fprintf(stderr, "digest of fragment %d differs\n", f);
      return 1;
    }
  }
  /* 4. block-scaled cast and its inverse */
  enum { M = 256, T = 128 };
  static const float base[5] = {1.0f, 2.0f, 0.5f, 448.0f, -3.5f};
  static const uint8_t code[5] = {0x38, 0x40, 0x30, 0x7E, 0xC6}; /* E4M3 of base */
  static const int ex[2][2] = {{-4, -1}, {2, 5}};                  /* tile exponents */
  uint16_t* xb = (uint16_t*)malloc((size_t)M * M * 2);
  uint16_t* yb = (uint16_t*)malloc((size_t)M * M * 2);
  uint8_t* qb = (uint8_t*)malloc((size_t)M * M);
  if (!xb || !yb || !qb) return 1;
  for (int r = 0; r < M; ++r)
    for (int c = 0; c < M; ++c) {
      const float v = ldexpf(base[(r * M + c) % 5], ex[r / T][c / T]);
      uint32_t u;
      memcpy(&u, &v, 4);
      xb[r * M + c] = (uint16_t)(u >> 16); /* exact: at most 3 significant bits */
    }
  void *x_d, *q_d, *s_d, *y_d, *cws, *dws;
  CHECK_HIP(hipMalloc(&x_d, (size_t)M * M * 2));
  CHECK_HIP(hipMalloc(&q_d, (size_t)M * M));
  CHECK_HIP(hipMalloc(&s_d, 4 * sizeof(float)));
  CHECK_HIP(hipMalloc(&y_d, (size_t)M * M * 2));
  CHECK_HIP(hipMemcpy(x_d, xb, (size_t)M * M * 2, hipMemcpyHostToDevice));
  const tc_cast_item item = {0, M, M, M, 0, M, 0, 2};
  const size_t cws_bytes = tc_cast_fp8_workspace_tiles(&item, 1);
  if (cws_bytes < tc_cast_fp8_workspace(1) + 4 * 32) {
    fprintf(stderr, "the tile workspace has no room for the 4 tile entries\n");
    return 1;
  }
  CHECK_HIP(hipMalloc(&cws, cws_bytes));
  tc_tile_plan plan;
  CHECK_TC(tc_cast_fp8_prepare(x_d, q_d, &item, 1, 128, cws, cws_bytes, &plan, 0));
  if (plan.tiled != 1 || plan.full_tiles != 4 || plan.edge_tiles != 0) {
    fprintf(stderr, "cast plan: tiled %u, %llu full and %llu edge tiles\n", plan.tiled,
            (unsigned long long)plan.full_tiles, (unsigned long long)plan.edge_tiles);
    return 1;
  }
  CHECK_TC(tc_cast_fp8_planned(x_d, q_d, (float*)s_d, cws, cws_bytes, &plan, 0));
  float sc[4];
  CHECK_HIP(hipMemcpy(qb, q_d, (size_t)M * M, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(sc, s_d, sizeof(sc), hipMemcpyDeviceToHost));
  for (int t = 0; t < 4; ++t)
    if (sc[t] != ldexpf(1.0f, ex[t / 2][t % 2])) {
      fprintf(stderr, "scale of tile %d: %g\n", t, (double)sc[t]);
      return 1;
    }
  for (int i = 0; i < M * M; ++i)
    if (qb[i] != code[i % 5]) {
      fprintf(stderr, "code %d: 0x%02x, want 0x%02x\n", i, qb[i], code[i % 5]);
      return 1;
    }
  const tc_dequant_item ditem = {0, M, M, M, 0, M, 0, 2};
  const size_t dws_bytes = tc_dequant_fp8_workspace_tiles(&ditem, 1);
  CHECK_HIP(hipMalloc(&dws, dws_bytes));
  tc_tile_plan dplan;
  CHECK_TC(tc_dequant_fp8_prepare(q_d, y_d, &ditem, 1, 128, dws, dws_bytes, &dplan, 0));
  CHECK_TC(tc_dequant_fp8_planned(q_d, (const float*)s_d, y_d, dws, dws_bytes, &dplan, 0));
  CHECK_HIP(hipMemcpy(yb, y_d, (size_t)M * M * 2, hipMemcpyDeviceToHost));
  if (dplan.tiled != 1 || memcmp(yb, xb, (size_t)M * M * 2)) {
    fprintf(stderr, "the inverse cast did not give the source back\n");
    return 1;
  }

  printf("C ABI demo: gather, scatter, planned copies, digests, fp8 cast and inverse correct "
         "(%llu tasks)\n", (unsigned long long)total);
  hipFree(pool_a); hipFree(pool_b); hipFree(buf); hipFree(ids_d);
  hipFree(src); hipFree(dst); hipFree(fr_d); hipFree(ws); hipFree(dg);
  hipFree(x_d); hipFree(q_d); hipFree(s_d); hipFree(y_d); hipFree(cws); hipFree(dws);
  free(host); free(got); free(xb); free(yb); free(qb);
  return 0;
}
