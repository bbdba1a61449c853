// Rotary position embedding at virtual positions, shared by the kernels that
// rotate queries (the attention kernels, at load) and new keys (rope_keys.hip,
// once per step), so that every rotation uses the same table and arithmetic.
//
// The host builds the table once per context: for relative position p (virtual
// position minus pos_offset) and pair j < d/2, tab[(p * d/2 + j) * 2 + {0, 1}] =
// {cos, sin} of p * f_j, times the scaling temperature, computed in double
// precision and rounded to fp32.  Pairs are half-split: (x_j, x_{j + d/2}).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace skv {

typedef unsigned int rope_u32x4 __attribute__((ext_vector_type(4)));

// x_j' = x_j cos - x_{j+d/2} sin
__device__ inline float rope_first(float lo, float hi, float c, float s) { return fmaf(lo, c, -(hi * s)); }
// x_{j+d/2}' = x_{j+d/2} cos + x_j sin
__device__ inline float rope_second(float hi, float lo, float c, float s) { return fmaf(hi, c, lo * s); }

__device__ inline float bf16_lo(unsigned w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(unsigned w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ inline unsigned bf16_pack(float a, float b) {
  return static_cast<unsigned>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(a))) |
         (static_cast<unsigned>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(b))) << 16);
}

// One 16-byte chunk of 8 bf16: `mine` holds dimensions [j0, j0 + 8) of the lower
// half (upper = false) or [d/2 + j0, d/2 + j0 + 8) of the upper half, `other`
// the same dimensions of the other half; tab points at the position's pairs.
__device__ inline rope_u32x4 rope_chunk_bf16(rope_u32x4 mine, rope_u32x4 other, bool upper, int j0,
                                             const float* tab) {
  rope_u32x4 out;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float r[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const float x = e ? bf16_hi(mine[w]) : bf16_lo(mine[w]);
      const float y = e ? bf16_hi(other[w]) : bf16_lo(other[w]);
      const float c = tab[2 * (j0 + 2 * w + e)], s = tab[2 * (j0 + 2 * w + e) + 1];
      r[e] = upper ? rope_second(x, y, c, s) : rope_first(x, y, c, s);
    }
    out[w] = bf16_pack(r[0], r[1]);
  }
  return out;
}

// The same for a chunk of 4 fp32 values (no rounding: the storage type is fp32).
__device__ inline rope_u32x4 rope_chunk_f32(rope_u32x4 mine, rope_u32x4 other, bool upper, int j0,
                                            const float* tab) {
  rope_u32x4 out;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float x = __uint_as_float(mine[e]), y = __uint_as_float(other[e]);
    const float c = tab[2 * (j0 + e)], s = tab[2 * (j0 + e) + 1];
    out[e] = __float_as_uint(upper ? rope_second(x, y, c, s) : rope_first(x, y, c, s));
  }
  return out;
}

}  // namespace skv
