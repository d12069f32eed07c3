/*
 * oracle.h -- plain CPU oracle for the tensor-lifecycle data path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library may include,
 * link or call this code; it exists so that tests, the smoke check and the
 * benchmark's CPU-baseline leg can compare the GPU path against a slow,
 * obviously correct implementation written from the definitions.  It shares
 * no header, type, table or helper with the GPU path.
 *
 * Every routine is a direct transcription of what the operation computes:
 *   - block gather / scatter: the export of a request's paged KV blocks into
 *     one contiguous buffer (publish) and its inverse import (hydrate),
 *     paper Sec. 3.2 "Operation" and Table 2;
 *   - fragment copy: the batched byte moves behind prefetch_many, Table 2,
 *     and the "transfer" stage of the materialization pipeline, Sec. 5;
 *   - bf16 -> fp8 E4M3 cast with one fp32 scale per 128x128 tile: one
 *     concrete `spec` rule for transform_into (Table 2, Sec. 3.2).  The paper
 *     gives no numeric format; the E4M3 encoding follows the OCP 8-bit
 *     floating point definition (bias 7, largest finite 448, NaN S.1111.111,
 *     no infinities), rounding to nearest with ties to even, saturating;
 *   - the inverse cast: codes times the tile's scale, rounded to binary32 and
 *     then to bf16 (the training-side transform_into of Sec. 7);
 *   - fragment digests for the pipeline's verify-integrity stage (Sec. 5):
 *     S1 = sum of the fragment's bytes, S2 = sum of (i + 1) * byte i, both
 *     mod 2^64.
 *
 * Threads: OpenMP over independent units (blocks, fragments, tiles).
 * Floating point: IEEE binary32 division and comparisons; the library is
 * built with -fno-fast-math and clears FTZ/DAZ on every thread it uses.
 */
#ifndef TC_ORACLE_H
#define TC_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  uint64_t src_off; /* byte offset into the source buffer */
  uint64_t dst_off; /* byte offset into the destination buffer */
  uint64_t len;     /* bytes */
} orc_frag;

/* Thread count used by the parallel loops (OpenMP max threads after
 * orc_set_threads). */
int orc_threads(void);
void orc_set_threads(int n);

/* out[(i*R + r)*B + b] = regions[r][ids[i]*stride + b] for i<n, r<R, b<B.
 * Returns 0, or -1 if an id lies outside [0, num_blocks). */
int orc_gather_blocks(const uint8_t* const* regions, int32_t num_regions,
                      int64_t num_blocks, int64_t block_bytes,
                      int64_t block_stride, const int32_t* ids, int64_t n,
                      uint8_t* out);

/* regions[r][ids[i]*stride + b] = in[(i*R + r)*B + b]; ids must be distinct.
 * Returns 0, -1 for an id out of range, -2 for a repeated id. */
int orc_scatter_blocks(uint8_t* const* regions, int32_t num_regions,
                       int64_t num_blocks, int64_t block_bytes,
                       int64_t block_stride, const int32_t* ids, int64_t n,
                       const uint8_t* in);

/* dst[f.dst_off + b] = src[f.src_off + b] for every descriptor f, b < f.len.
 * Destination ranges must be pairwise disjoint. */
void orc_copy_fragments(const uint8_t* src, uint8_t* dst, const orc_frag* f,
                        int64_t n);

/* E4M3 code of an fp32 value: nearest finite magnitude, ties to the code
 * with an even mantissa LSB, |v| beyond 448 and infinities saturate to
 * +-448, NaN -> 0x7F.  Sign is kept for zeros (-0 -> 0x80). */
uint8_t orc_e4m3_encode(float v);
/* Value of an E4M3 code (0x7F / 0xFF decode to NaN). */
float orc_e4m3_decode(uint8_t code);

/* q[i] = enc(RN_f32(bf16(x[i]) / scale)) for i < n. */
void orc_cast_fp8_scaled(const uint16_t* x, int64_t n, float scale,
                         uint8_t* q);

/* One row-major bf16 matrix [rows][cols] (row stride ld elements) cast to
 * E4M3 with one fp32 scale per 128x128 tile (edge tiles partial):
 *   finite tile, amax > 0 : s = RN_f32(amax / 448), q = enc(RN_f32(x / s))
 *   finite tile, amax = 0 : s = 0, q = sign bit only
 *   any Inf/NaN in tile   : s = NaN (0x7FC00000), every q = 0x7F
 * q is [rows][q_ld] bytes, scales is [ceil(rows/128)][scale_ld] floats. */
void orc_cast_fp8_blockscaled(const uint16_t* x, int64_t rows, int64_t cols,
                              int64_t ld, uint8_t* q, int64_t q_ld,
                              float* scales, int64_t scale_ld);

/* Inverse of the block-scaled cast: y = RN_bf16(RN_f32(dec(q) * s)) for
 * every code of a [rows][cols] matrix (row stride q_ld bytes) with the fp32
 * scale of its 128x128 tile (grid row stride scale_ld).  A NaN result (code
 * 0x7F/0xFF, NaN scale, or 0 * Inf) is written as 0x7FC0.  y is [rows][y_ld]
 * raw bf16 patterns. */
void orc_dequant_fp8_blockscaled(const uint8_t* q, int64_t rows, int64_t cols, int64_t q_ld,
                                 const float* scales, int64_t scale_ld, uint16_t* y,
                                 int64_t y_ld);
/* Integrity digest of each fragment (the materialization pipeline's verify
 * stage): with b_i the fragment's i-th byte (i from 0),
 *   S1 = sum_i b_i,   S2 = sum_i (i + 1) * b_i,   both mod 2^64.
 * Read at src_off (use_src != 0) or dst_off of each descriptor; out[2f],
 * out[2f + 1] receive S1, S2 of fragment f. */
void orc_fragment_digests(const uint8_t* base, const orc_frag* f, int64_t n, int use_src,
                          uint64_t* out);

/* RN_bf16 of a binary32 value (ties to even; NaN -> 0x7FC0). */
uint16_t orc_bf16_round(float v);

#ifdef __cplusplus
}
#endif
#endif
