// INT4 variant of the packed expert (the 4-bit, group-64, fp16-scale format;
// the paper reports INT4 as a quality point in Table I and keeps INT8 as its
// format, section IV-B).  Host and device code share these definitions.
//
// Per matrix [rows][K] (gate [R][C], up [R][C], down [C][R]; rows and K
// multiples of 16 and 128) and per row and group of 64 consecutive columns:
//   alpha = max |w| over the group,
//   s     = fp16_rne(fl32(max(alpha, eps) / 7)), 2^-24 if that is zero,
//           65504 if it overflows,
//   q     = clamp(rint_even(fl32(w / s)), -7, 7).
// Layout of a matrix: nibbles, then scales.  Nibbles come in tiles of 16 rows
// x 128 columns (two groups, 1024 bytes; tile-rows in order, column pairs in
// order); the 16-byte run g*16 + i of a tile holds row i, columns
// 16g .. 16g+15 of the first group in bytes 0..7 and of the second group in
// bytes 8..15; in each 8-byte half, byte b carries column 16g + 8*(b/4) + b%4
// in its high nibble and that column + 4 in its low nibble.  So a lane's
// 16-byte load covers two k-steps, and each half becomes the int8 operand of
// one 16x16x64 MFMA (16 consecutive columns, each as 16*q) with two masks and
// a shift.  Scales: fp16 by tile-row, then group, then the tile's 16 rows (32
// bytes per tile-row and group), so the scales of 16 groups of a tile-row are
// one 512-byte run.  The blob holds gate, up and down, zero-padded to 256
// bytes.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace mira {

constexpr int kI4QMax = 7;
constexpr int kI4PairTile = 1024;  // nibble bytes of 16 rows x 128 columns

__host__ __device__ inline size_t i4_nib_bytes(size_t rows, size_t K) { return rows * K / 2; }

__host__ __device__ inline size_t i4_matrix_bytes(size_t rows, size_t K) {
  return rows * K / 2 + rows * (K / 64) * 2;
}

// Offset of the 8 bytes holding row r, columns 16gq .. 16gq+15 of group grp.
__host__ __device__ inline size_t i4_half_run_offset(size_t r, size_t grp, int gq, size_t K) {
  return ((r >> 4) * (K >> 7) + (grp >> 1)) * kI4PairTile + (size_t)(gq * 16 + (int)(r & 15)) * 16 +
         8 * (grp & 1);
}

__host__ __device__ inline size_t i4_scale_offset(size_t r, size_t grp, size_t rows, size_t K) {
  return i4_nib_bytes(rows, K) + ((r >> 4) * (K >> 6) + grp) * 32 + 2 * (r & 15);
}

// fp32 (positive, finite) -> fp16 bits, round to nearest, ties to even, with
// the format's rules: zero becomes the smallest subnormal, overflow the
// largest finite value.
__host__ __device__ inline uint16_t i4_scale_bits(float f) {
  uint32_t u;
  __builtin_memcpy(&u, &f, 4);
  const int e = (int)((u >> 23) & 0xFF);
  const uint32_t m = u & 0x7FFFFFu;
  uint32_t r;
  const int he = e - 127 + 15;
  if (he >= 31) {
    r = 0x7C00u;
  } else if (he <= 0) {
    // subnormal: value / 2^-24 = (m | 2^23) * 2^(e - 126)
    const int shift = 126 - e;  // >= 14
    const uint32_t mm = m | 0x800000u;
    if (shift > 24) {
      r = 0;
    } else {
      r = mm >> shift;
      const uint32_t rem = mm & ((1u << shift) - 1u), half = 1u << (shift - 1);
      if (rem > half || (rem == half && (r & 1u))) ++r;
    }
  } else {
    r = ((uint32_t)he << 10) | (m >> 13);
    const uint32_t rem = m & 0x1FFFu;
    if (rem > 0x1000u || (rem == 0x1000u && (r & 1u))) ++r;
  }
  if (r >= 0x7C00u) r = 0x7BFFu;
  if (r == 0) r = 1;
  return (uint16_t)r;
}

__host__ __device__ inline float i4_scale_value(uint16_t b) {
  const uint32_t e = (b >> 10) & 0x1F, m = b & 0x3FFu;
  float v;
  if (e == 0) {
    v = (float)m * 5.9604644775390625e-8f;  // m * 2^-24, exact
  } else {
    const uint32_t u = ((e - 15 + 127) << 23) | (m << 13);
    __builtin_memcpy(&v, &u, 4);
  }
  return v;
}

}  // namespace mira
