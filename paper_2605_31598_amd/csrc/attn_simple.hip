// Scalar attention + importance-score kernel (fp32 arithmetic on VALU).
//
// Runs the fp32 configuration (bf16 contexts use the MFMA kernel).  One wave per
// 64 query rows of one (layer, KV head); rows are
// the G query heads of the group times the T frame tokens.  Two sweeps over the
// candidate keys [state slots; frame tokens] (Eq. 5):
//   sweep 1: row maximum and sum of exp2 -> log2-sum-exp per row;
//   sweep 2: exact normalised P = exp2(x - lse2), O += P V, and per-key column
//            sums of P over the wave's rows, written per row tile (no atomics).
// Mask M_n: candidate j is visible to frame token i iff j < S + i + 1 (state
// keys always, frame key t iff t <= i).
#include "internal.h"

namespace skv {

namespace {

template <typename T>
__device__ inline float load_elem(const T* p);
template <>
__device__ inline float load_elem<float>(const float* p) { return *p; }

template <typename T>
__device__ inline void store_elem(T* p, float x);
template <>
__device__ inline void store_elem<float>(float* p, float x) { *p = x; }

// A value as the storage type holds it (rotated activations are rounded to it).
template <typename T>
__device__ inline float round_storage(float x);
template <>
__device__ inline float round_storage<float>(float x) { return x; }

constexpr int KT = 32;  // keys per LDS tile

}  // namespace

template <typename T, int D>
__global__ __launch_bounds__(64) void attn_simple_kernel(AttnArgs a) {
  __shared__ float ks[KT][D + 1];
  __shared__ float vs[KT][D + 1];
  __shared__ float ps[kSimpleRowsPerTile][KT + 1];

  const int qt = blockIdx.x;
  const int lg = blockIdx.y;
  const int layer = lg / a.H_kv, g = lg % a.H_kv;
  const int tid = threadIdx.x;
  const int GT = a.G * a.T;
  const int r = qt * kSimpleRowsPerTile + tid;
  const bool valid = r < GT;
  const int lim = valid ? a.S + (r % a.T) : -1;  // visible candidates: j <= lim
  const int S = a.S, n_keys = a.S + a.T;

  const T* qrow = static_cast<const T*>(a.q) +
                  (static_cast<size_t>(layer * a.H_q + g * a.G) * a.T + (valid ? r : 0)) * D;
  const T* kst = static_cast<const T*>(a.ks) + static_cast<size_t>(lg) * a.kv_rows * D;
  const T* vst = static_cast<const T*>(a.vs) + static_cast<size_t>(lg) * a.kv_rows * D;
  const T* kfr = static_cast<const T*>(a.kf) + static_cast<size_t>(lg) * a.T * D;
  const T* vfr = static_cast<const T*>(a.vf) + static_cast<size_t>(lg) * a.T * D;
  // no partial buffer: streaming full attention, which computes no scores
  float* part = a.partial ? a.partial + (static_cast<size_t>(lg) * a.tile_stride + qt) * a.pool_stride : nullptr;

  float q[D];
  for (int e = 0; e < D; ++e) q[e] = valid ? load_elem(qrow + e) : 0.f;
  if (a.rope_tab != nullptr && valid) {  // RoPE at the frame token's virtual position
    const float* tb = a.rope_tab + static_cast<size_t>(a.rope_pos0 + r % a.T) * D;
    for (int j = 0; j < D / 2; ++j) {
      const float lo = q[j], hi = q[j + D / 2], c = tb[2 * j], s = tb[2 * j + 1];
      q[j] = round_storage<T>(rope_first(lo, hi, c, s));
      q[j + D / 2] = round_storage<T>(rope_second(hi, lo, c, s));
    }
  }

  auto stage = [&](int t0, bool with_v) {
    for (int idx = tid; idx < KT * D; idx += 64) {
      const int kk = idx / D, e = idx % D;
      const int j = t0 + kk;
      float kx = 0.f, vx = 0.f;
      if (j < S) {
        kx = load_elem(kst + static_cast<size_t>(j) * D + e);
        if (with_v) vx = load_elem(vst + static_cast<size_t>(j) * D + e);
      } else if (j < n_keys) {
        kx = load_elem(kfr + static_cast<size_t>(j - S) * D + e);
        if (with_v) vx = load_elem(vfr + static_cast<size_t>(j - S) * D + e);
      }
      ks[kk][e] = kx;
      if (with_v) vs[kk][e] = vx;
    }
  };

  // Sweep 1: online max / sum in log2 units.
  float m = -1e30f, l = 0.f;
  for (int t0 = 0; t0 < n_keys; t0 += KT) {
    __syncthreads();
    stage(t0, false);
    __syncthreads();
    for (int kk = 0; kk < KT; ++kk) {
      const int j = t0 + kk;
      if (j > lim) break;
      float z = 0.f;
      for (int e = 0; e < D; ++e) z = fmaf(q[e], ks[kk][e], z);
      const float x = z * a.scale_log2;
      const float mn = fmaxf(m, x);
      l = l * exp2f(m - mn) + exp2f(x - mn);
      m = mn;
    }
  }
  const float lse2 = valid ? m + log2f(l) : __builtin_huge_valf();

  // Sweep 2: exact probabilities, output and column sums.
  float o[D];
  for (int e = 0; e < D; ++e) o[e] = 0.f;
  for (int t0 = 0; t0 < n_keys; t0 += KT) {
    __syncthreads();
    stage(t0, true);
    __syncthreads();
    for (int kk = 0; kk < KT; ++kk) {
      const int j = t0 + kk;
      float p = 0.f;
      if (j <= lim) {
        float z = 0.f;
        for (int e = 0; e < D; ++e) z = fmaf(q[e], ks[kk][e], z);
        p = exp2f(z * a.scale_log2 - lse2);
        for (int e = 0; e < D; ++e) o[e] = fmaf(p, vs[kk][e], o[e]);
      }
      ps[tid][kk] = p;
    }
    __syncthreads();
    if (part && tid < KT && t0 + tid < n_keys) {
      float c = 0.f;
      for (int rr = 0; rr < kSimpleRowsPerTile; ++rr) c += ps[rr][tid];
      part[t0 + tid] = c;
    }
  }
  if (valid) {
    T* orow = static_cast<T*>(a.out) + (static_cast<size_t>(layer * a.H_q + g * a.G) * a.T + r) * D;
    for (int e = 0; e < D; ++e) store_elem(orow + e, o[e]);
  }
}

hipError_t launch_attention_simple_f32(const AttnArgs& a, int head_dim, hipStream_t s) {
  dim3 grid((a.G * a.T + kSimpleRowsPerTile - 1) / kSimpleRowsPerTile, a.n_layers * a.H_kv);
  dim3 block(64);
  if (head_dim == 64) hipLaunchKernelGGL((attn_simple_kernel<float, 64>), grid, block, 0, s, a);
  else hipLaunchKernelGGL((attn_simple_kernel<float, 128>), grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace skv
