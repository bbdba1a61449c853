// Device implementation of the counter-based input generator of
// workloads/generate.py, for filling benchmark-sized inputs in HBM.
//
// Element i of chunk c is table[mix64(key[c] + (i + 1) * 0x9E3779B97F4A7C15) >> 48],
// where mix64 is the SplitMix64 output function (Steele, Lea & Flood 2014) and
// the 65,536-entry table of rounded normal quantiles is built on the host and
// uploaded, so there is no device floating-point arithmetic and the bytes match
// the host generator exactly.  Holds none of the attention method.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

__device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

template <typename T>
__global__ void fill_kernel(T* out, int64_t per_chunk, int64_t total, const uint64_t* keys, const T* table) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t c = i / per_chunk;
    const uint64_t idx = static_cast<uint64_t>(i - c * per_chunk) + 1ull;
    const uint64_t bits = mix64(keys[c] + idx * 0x9E3779B97F4A7C15ull);
    out[i] = table[bits >> 48];
  }
}

}  // namespace

extern "C" {

// out: device buffer of n_chunks * per_chunk elements; keys: device array of
// n_chunks stream keys; table: device array of 65,536 entries of elem_bytes
// (2 = bf16 bits, 4 = fp32).  Returns 0 on success, -1 on bad arguments, or the
// HIP error code.
int skvgen_fill(void* out, int64_t per_chunk, int32_t n_chunks, const void* keys, const void* table,
                int32_t elem_bytes, void* stream) {
  if (out == nullptr || keys == nullptr || table == nullptr || per_chunk < 1 || n_chunks < 1) return -1;
  const int64_t total = per_chunk * n_chunks;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (elem_bytes == 2) {
    hipLaunchKernelGGL(fill_kernel<uint16_t>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s,
                       static_cast<uint16_t*>(out), per_chunk, total, static_cast<const uint64_t*>(keys),
                       static_cast<const uint16_t*>(table));
  } else if (elem_bytes == 4) {
    hipLaunchKernelGGL(fill_kernel<uint32_t>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s,
                       static_cast<uint32_t*>(out), per_chunk, total, static_cast<const uint64_t*>(keys),
                       static_cast<const uint32_t*>(table));
  } else {
    return -1;
  }
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : static_cast<int>(e);
}

}  // extern "C"
