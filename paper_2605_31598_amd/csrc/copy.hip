// Byte-exact row copies of the frame step: state compaction (admitted frame
// rows into evicted or free slots of the compressed state, Eq. 6) and the
// decode-cache append D_n = D_{n-1} + (K_n, V_n) (Eq. 4).  Both move 16-byte
// chunks with consecutive threads on consecutive chunks.
#include "internal.h"

namespace skv {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void update_kernel(UpdateArgs a) {
  const int lg = blockIdx.x;
  const int chunks = a.row_bytes >> 4;
  const int idx = blockIdx.y * blockDim.x + threadIdx.x;
  const int i = idx / chunks;
  const int c = idx - i * chunks;
  if (i >= a.admit_count[lg]) return;
  const int src = a.admit_src[static_cast<size_t>(lg) * a.T + i];
  const int dst = a.admit_dst[static_cast<size_t>(lg) * a.T + i];
  const size_t s_off = (static_cast<size_t>(lg) * a.T + src) * a.row_bytes + (static_cast<size_t>(c) << 4);
  const size_t d_off = (static_cast<size_t>(lg) * a.B + dst) * a.row_bytes + (static_cast<size_t>(c) << 4);
  const u32x4 kk = *reinterpret_cast<const u32x4*>(static_cast<const char*>(a.kf) + s_off);
  const u32x4 vv = *reinterpret_cast<const u32x4*>(static_cast<const char*>(a.vf) + s_off);
  *reinterpret_cast<u32x4*>(static_cast<char*>(a.ks) + d_off) = kk;
  *reinterpret_cast<u32x4*>(static_cast<char*>(a.vs) + d_off) = vv;
  if (c == 0) {
    a.state_pos[static_cast<size_t>(lg) * a.B + dst] = a.frame_pos0 + src;
    a.state_score[static_cast<size_t>(lg) * a.B + dst] =
        a.pool_score[static_cast<size_t>(lg) * a.pool_stride + a.S + src];
  }
}

__global__ __launch_bounds__(256) void append_kernel(AppendArgs a) {
  const int lg = blockIdx.x;
  const size_t n16 = (static_cast<size_t>(a.T) * a.row_bytes) >> 4;
  const size_t i = static_cast<size_t>(blockIdx.y) * blockDim.x + threadIdx.x;
  if (i >= n16) return;
  const size_t s_off = static_cast<size_t>(lg) * a.T * a.row_bytes + (i << 4);
  const size_t d_off = (static_cast<size_t>(lg) * a.max_tokens + a.first_row) * a.row_bytes + (i << 4);
  const u32x4 kk = *reinterpret_cast<const u32x4*>(static_cast<const char*>(a.kf) + s_off);
  const u32x4 vv = *reinterpret_cast<const u32x4*>(static_cast<const char*>(a.vf) + s_off);
  *reinterpret_cast<u32x4*>(static_cast<char*>(a.ck) + d_off) = kk;
  *reinterpret_cast<u32x4*>(static_cast<char*>(a.cv) + d_off) = vv;
}

hipError_t launch_update(const UpdateArgs& a, hipStream_t s) {
  const int chunks = a.row_bytes >> 4;
  const int total = a.T * chunks;
  dim3 grid(a.n_layers * a.H_kv, (total + 255) / 256);
  hipLaunchKernelGGL(update_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_append(const AppendArgs& a, hipStream_t s) {
  const size_t n16 = (static_cast<size_t>(a.T) * a.row_bytes) >> 4;
  dim3 grid(a.n_layers * a.H_kv, static_cast<unsigned>((n16 + 255) / 256));
  hipLaunchKernelGGL(append_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace skv
