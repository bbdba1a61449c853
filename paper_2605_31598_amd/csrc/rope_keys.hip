// Rotary position embedding of a step's new keys (a frame's T tokens, or the
// decoded tokens), applied once per step before any kernel reads them.
//
// The virtual position of a new key fixes its rotation (the virtual sequence
// length paragraph), so the keys are rotated once here and every later reader
// sees rotated keys: the attention kernels (which rotate only their queries),
// the state update and the decode-cache append (plain copies).  The rotation
// is the one of rope.h, so the result is bit-identical wherever it is used.
#include "internal.h"

namespace skv {

namespace {

// One thread per pair of 16-byte chunks (c, c + half) of one key row: the
// half-split RoPE pairs of those dimensions live in exactly these two chunks.
__global__ __launch_bounds__(256) void rope_keys_kernel(const char* __restrict__ in, char* __restrict__ out,
                                                        int64_t n_pairs, int t, int row_bytes, int elem,
                                                        const float* __restrict__ tab, int pos0) {
  const int chunks = row_bytes >> 4, half = chunks >> 1;
  const int d = row_bytes / elem;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t p = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; p < n_pairs; p += stride) {
    const int64_t row = p / half;
    const int c = static_cast<int>(p - row * half);
    const int r = static_cast<int>(row % t);  // token within its (layer, KV head) block
    const char* src = in + row * row_bytes;
    char* dst = out + row * row_bytes;
    const rope_u32x4 lo = *reinterpret_cast<const rope_u32x4*>(src + c * 16);
    const rope_u32x4 hi = *reinterpret_cast<const rope_u32x4*>(src + (c + half) * 16);
    const float* tb = tab + static_cast<size_t>(pos0 + r) * d;
    const int j0 = c * 16 / elem;
    rope_u32x4 a, b;
    if (elem == 2) {
      a = rope_chunk_bf16(lo, hi, false, j0, tb);
      b = rope_chunk_bf16(hi, lo, true, j0, tb);
    } else {
      a = rope_chunk_f32(lo, hi, false, j0, tb);
      b = rope_chunk_f32(hi, lo, true, j0, tb);
    }
    *reinterpret_cast<rope_u32x4*>(dst + c * 16) = a;
    *reinterpret_cast<rope_u32x4*>(dst + (c + half) * 16) = b;
  }
}

}  // namespace

hipError_t launch_rope_keys(const void* in, void* out, int n_blocks, int t, int row_bytes, int elem,
                            const float* tab, int pos0, hipStream_t s) {
  const int64_t n_pairs = static_cast<int64_t>(n_blocks) * t * (row_bytes >> 5);
  if (n_pairs <= 0) return hipSuccess;
  const int64_t want = (n_pairs + 255) / 256;
  const int grid = static_cast<int>(want < 4096 ? want : 4096);
  hipLaunchKernelGGL(rope_keys_kernel, dim3(grid), dim3(256), 0, s, static_cast<const char*>(in),
                     static_cast<char*>(out), n_pairs, t, row_bytes, elem, tab, pos0);
  return hipGetLastError();
}

}  // namespace skv
