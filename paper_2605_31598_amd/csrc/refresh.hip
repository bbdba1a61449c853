// Frame refresh (Eq. 4 and Eq. 6): one launch, up to three kinds of workgroup.
//
// Selection workgroups, one per (layer, KV head), refresh the compressed state
// (mode 0: attention-driven selection; mode 1, the recency-window baseline: the
// same steps with the position as the selection key): score finalisation, Top-B
// radix select with the lowest-position tie rule, and the state update of the
// admitted rows (select.h).
// Append workgroups, one per (layer, KV head), copy the frame's K/V rows to the
// decode cache D (the detailed state), concurrently with the above.  Streaming
// full attention (no compressed state) launches only these; a launch that
// selects after an earlier append reads the frame's rows back from D.
// Combine workgroups add the output shares of a key-split attention plan.
// A context can also run the stages as three launches (selection with the admit
// lists in global memory, then the state update, then the append), so that each
// can be timed and counted on its own.
#include "select.h"

namespace skv {

namespace {

// State update of one (layer, KV head) as a launch of its own: the admitted frame
// rows the selection launch listed (global admit lists and count) go into their
// slots, with their position and score; the same copies as refresh_state's.
__device__ void update_state(const RefreshArgs& a, int lg) {
  const int tid = threadIdx.x, B = a.B, T = a.T, S = a.S;
  const int count = a.admit_count[lg];
  const int32_t* asrc = a.admit_src + static_cast<size_t>(lg) * T;
  const int32_t* adst = a.admit_dst + static_cast<size_t>(lg) * T;
  const float* pscore = a.pool_score + static_cast<size_t>(lg) * a.pool_stride;
  int32_t* state_pos = a.state_pos + static_cast<size_t>(lg) * B;
  float* sscore = a.state_score + static_cast<size_t>(lg) * B;
  const int chunks = a.row_bytes >> 4;
  const size_t src_base = static_cast<size_t>(lg) * a.kf_rows * a.row_bytes;
  const size_t dst_base = static_cast<size_t>(lg) * B * a.row_bytes;
  for (int idx = tid; idx < count * chunks; idx += blockDim.x) {
    const int i = idx / chunks;
    const int c = idx - i * chunks;
    const int src = asrc[i], dst = adst[i];
    const size_t so = src_base + static_cast<size_t>(src) * a.row_bytes + (static_cast<size_t>(c) << 4);
    const size_t dof = dst_base + static_cast<size_t>(dst) * a.row_bytes + (static_cast<size_t>(c) << 4);
    *reinterpret_cast<u32x4*>(static_cast<char*>(a.ks) + dof) =
        *reinterpret_cast<const u32x4*>(static_cast<const char*>(a.kf) + so);
    *reinterpret_cast<u32x4*>(static_cast<char*>(a.vs) + dof) =
        *reinterpret_cast<const u32x4*>(static_cast<const char*>(a.vf) + so);
    if (c == 0) {
      state_pos[dst] = a.frame_pos0 + src;
      sscore[dst] = pscore[S + src];
    }
  }
}

// Decode-cache append of one (layer, KV head): T contiguous rows of K and V.
// Four 16-byte chunks per thread are loaded before any is stored.
__device__ void append_frame(const RefreshArgs& a, int lg) {
  const int rb = a.row_bytes;
  const int n16 = a.T * (rb >> 4);  // 16-byte chunks of the block
  const size_t src = static_cast<size_t>(lg) * a.kf_rows * rb;
  const size_t dst = (static_cast<size_t>(lg) * a.max_tokens + a.first_row) * rb;
  const char* kf = static_cast<const char*>(a.kf) + src;
  const char* vf = static_cast<const char*>(a.vf) + src;
  char* ck = static_cast<char*>(a.ck) + dst;
  char* cv = static_cast<char*>(a.cv) + dst;
  const int nt = static_cast<int>(blockDim.x);
  constexpr int kU = 4;
  for (int base = threadIdx.x; base < n16; base += kU * nt) {
    u32x4 vv[kU], kv[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const size_t off = static_cast<size_t>(min(base + u * nt, n16 - 1)) << 4;
      vv[u] = *reinterpret_cast<const u32x4*>(vf + off);
      kv[u] = *reinterpret_cast<const u32x4*>(kf + off);
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int i = base + u * nt;
      if (i < n16) {
        const size_t off = static_cast<size_t>(i) << 4;
        *reinterpret_cast<u32x4*>(cv + off) = vv[u];
        *reinterpret_cast<u32x4*>(ck + off) = kv[u];
      }
    }
  }
}

// Output of a key-split attention plan: out = the sum, in split order, of the
// splits' fp32 shares, rounded once to bf16; workgroup c of n_comb takes every
// n_comb-th group of four values.
__device__ void combine_output(const RefreshArgs& a, int c) {
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  const int64_t n4 = a.out_elems / 4;
  const int64_t stride = static_cast<int64_t>(a.n_comb) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(c) * blockDim.x + threadIdx.x; i < n4; i += stride) {
    f32x4 acc = reinterpret_cast<const f32x4*>(a.opart)[i];
    for (int k = 1; k < a.n_ks; ++k) acc += reinterpret_cast<const f32x4*>(a.opart + static_cast<size_t>(k) * n4 * 4)[i];
    unsigned short b[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) b[j] = __builtin_bit_cast(unsigned short, static_cast<__bf16>(acc[j]));
    const uint2 w = {static_cast<unsigned>(b[0]) | (static_cast<unsigned>(b[1]) << 16),
                     static_cast<unsigned>(b[2]) | (static_cast<unsigned>(b[3]) << 16)};
    reinterpret_cast<uint2*>(a.out)[i] = w;
  }
}

}  // namespace

__global__ __launch_bounds__(kSelectThreads) void refresh_kernel(RefreshArgs a) {
  extern __shared__ uint32_t pool_mem[];  // [pool] score bits, then [pool] positions
  __shared__ SelectShared sh;
  const int n_sel = a.select ? a.n_layers * a.H_kv : 0;
  const int n_app = a.append ? a.n_layers * a.H_kv : 0;
  const int b = static_cast<int>(blockIdx.x);
  if (b < n_sel) {
    refresh_state(a, b, sh, pool_mem);
  } else if (b < n_sel + n_app) {
    append_frame(a, b - n_sel);
  } else {
    combine_output(a, b - n_sel - n_app);
  }
}

// The three stages as launches of their own (a context option for measuring each
// stage; the results are the fused launch's, bit for bit).
__global__ __launch_bounds__(kSelectThreads) void refresh_update_kernel(RefreshArgs a) {
  update_state(a, static_cast<int>(blockIdx.x));
}
__global__ __launch_bounds__(kSelectThreads) void refresh_append_kernel(RefreshArgs a) {
  append_frame(a, static_cast<int>(blockIdx.x));
}

hipError_t launch_refresh(const RefreshArgs& a, hipStream_t s) {
  if (a.n_ks > kMaxKeySplits) return hipErrorInvalidValue;  // plans split the keys at most kMaxKeySplits ways
  const size_t lds = a.select ? static_cast<size_t>(a.S + a.T) * 2 * sizeof(uint32_t) : 0;
  const int grid = ((a.select ? 1 : 0) + (a.append ? 1 : 0)) * a.n_layers * a.H_kv + (a.n_ks > 1 ? a.n_comb : 0);
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(refresh_kernel, dim3(grid), dim3(kSelectThreads), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_refresh_update(const RefreshArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(refresh_update_kernel, dim3(a.n_layers * a.H_kv), dim3(kSelectThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_refresh_append(const RefreshArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(refresh_append_kernel, dim3(a.n_layers * a.H_kv), dim3(kSelectThreads), 0, s, a);
  return hipGetLastError();
}

size_t selection_lds_bytes(int P) { return select_lds_bytes(P); }

hipError_t prepare_refresh(int pool_stride) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(refresh_kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize,
                             static_cast<int>(pool_stride * 2 * sizeof(uint32_t)));
}

}  // namespace skv
