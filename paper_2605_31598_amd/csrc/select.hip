// Top-B refresh of the compressed state (Eq. 6), one workgroup per (layer, KV head).
//
// 1. Finalise the importance scores of the candidate pool (state slots, then the
//    frame's tokens): s_j = (1/T) * sum over row tiles of the attention kernel's
//    column sums, added in fixed tile order (deterministic, no atomics).
// 2. If the pool exceeds B, find the B-th largest composite key
//    (float bits of s) << 32 | (0xFFFFFFFF - position) with an 8-pass, 8-bit radix
//    select over the pool held in LDS.  Scores are non-negative, so their IEEE
//    bits order like the values; the low word makes the lower position win on
//    equal scores.  Composite keys of distinct positions are distinct, so exactly
//    B keys are >= the threshold.
// 3. Pair evicted state slots (then free slots S, S+1, ...) with admitted frame
//    tokens in ascending order using block-wide scans.  The state update kernel
//    copies the admitted rows; retained slots never move.
#include "internal.h"

namespace skv {

namespace {

__device__ inline uint64_t composite_key(float s, int32_t pos) {
  return (static_cast<uint64_t>(__float_as_uint(s)) << 32) |
         static_cast<uint64_t>(0xFFFFFFFFu - static_cast<uint32_t>(pos));
}

// Exclusive prefix count of `flag` over the workgroup; *total receives the sum.
__device__ inline int block_exclusive_count(bool flag, int* wave_count, int* total) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n_waves = blockDim.x >> 6;
  const uint64_t mask = __ballot(flag);
  const int within = __popcll(mask & ((1ull << lane) - 1ull));
  if (lane == 0) wave_count[wave] = __popcll(mask);
  __syncthreads();
  int before = 0, sum = 0;
  for (int w = 0; w < n_waves; ++w) {
    const int c = wave_count[w];
    before += (w < wave) ? c : 0;
    sum += c;
  }
  __syncthreads();
  *total = sum;
  return before + within;
}

}  // namespace

__global__ __launch_bounds__(kSelectThreads) void select_kernel(SelectArgs a) {
  extern __shared__ uint64_t pool_key[];
  __shared__ uint32_t hist[256];
  __shared__ int wave_count[kSelectThreads / 64];
  __shared__ int sh_digit, sh_remaining;

  const int lg = blockIdx.x;
  const int tid = threadIdx.x;
  const int S = a.S, T = a.T, B = a.B, P = S + T;
  const float* part = a.partial + static_cast<size_t>(lg) * a.n_qtiles * a.pool_stride;
  const int32_t* spos = a.state_pos + static_cast<size_t>(lg) * B;
  float* sscore = a.state_score + static_cast<size_t>(lg) * B;
  float* pscore = a.pool_score + static_cast<size_t>(lg) * a.pool_stride;
  int32_t* ppos = a.pool_pos + static_cast<size_t>(lg) * a.pool_stride;
  int32_t* asrc = a.admit_src + static_cast<size_t>(lg) * T;
  int32_t* adst = a.admit_dst + static_cast<size_t>(lg) * T;

  for (int j = tid; j < P; j += blockDim.x) {
    float acc = 0.f;
    for (int t = 0; t < a.n_qtiles; ++t) acc += part[static_cast<size_t>(t) * a.pool_stride + j];
    const float s = acc * a.inv_T;
    const int32_t pos = j < S ? spos[j] : a.frame_pos0 + (j - S);
    pscore[j] = s;
    ppos[j] = pos;
    pool_key[j] = composite_key(s, pos);
  }
  __syncthreads();

  const bool prune = P > B;
  uint64_t thr = 0;
  if (prune && B > 0) {
    uint64_t prefix = 0;
    int remaining = B;  // rank (from the top) of the wanted key among keys matching `prefix`
    for (int pass = 0; pass < 8; ++pass) {
      const int shift = 56 - 8 * pass;
      for (int i = tid; i < 256; i += blockDim.x) hist[i] = 0u;
      __syncthreads();
      for (int j = tid; j < P; j += blockDim.x) {
        const uint64_t k = pool_key[j];
        const bool match = pass == 0 || ((k ^ prefix) >> (shift + 8)) == 0;
        if (match) atomicAdd(&hist[(k >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (tid < 64) {
        uint32_t c[4];
        for (int b = 0; b < 4; ++b) c[b] = hist[4 * tid + b];
        const uint32_t mine = c[0] + c[1] + c[2] + c[3];
        uint32_t suffix = mine;  // sum over lanes >= tid
        for (int off = 1; off < 64; off <<= 1) {
          const uint32_t o = __shfl_down(suffix, off, 64);
          if (tid + off < 64) suffix += o;
        }
        uint32_t above = suffix - mine;  // keys in higher bins
        for (int b = 3; b >= 0; --b) {
          if (above < static_cast<uint32_t>(remaining) && static_cast<uint32_t>(remaining) <= above + c[b]) {
            sh_digit = 4 * tid + b;
            sh_remaining = remaining - static_cast<int>(above);
          }
          above += c[b];
        }
      }
      __syncthreads();
      prefix |= static_cast<uint64_t>(sh_digit) << shift;
      remaining = sh_remaining;
      __syncthreads();
    }
    thr = prefix;
  }

  // Admitted frame tokens, ascending t.
  int n_adm = 0;
  for (int base = 0; base < T; base += blockDim.x) {
    const int t = base + tid;
    const bool adm = t < T && (!prune || (B > 0 && pool_key[S + t] >= thr));
    int tot;
    const int rank = block_exclusive_count(adm, wave_count, &tot);
    if (adm) asrc[n_adm + rank] = t;
    n_adm += tot;
  }
  // Evicted state slots, ascending slot; retained slots get the new score.
  int n_ev = 0;
  for (int base = 0; base < S; base += blockDim.x) {
    const int j = base + tid;
    const bool ev = j < S && prune && (B == 0 || pool_key[j] < thr);
    if (j < S && !ev) sscore[j] = pscore[j];
    int tot;
    const int rank = block_exclusive_count(ev, wave_count, &tot);
    if (ev) adst[n_ev + rank] = j;
    n_ev += tot;
  }
  // Holes beyond the evicted slots are the free slots S, S+1, ... (state not yet full).
  // Clamping keeps writes inside the B slots even for an invalid forced state
  // with repeated positions.
  const int n_holes = n_ev + (B - S);
  const int count = n_adm < n_holes ? n_adm : n_holes;
  for (int i = n_ev + tid; i < count; i += blockDim.x) adst[i] = S + (i - n_ev);
  if (tid == 0) a.admit_count[lg] = count;
}

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  const size_t lds = static_cast<size_t>(a.S + a.T) * sizeof(uint64_t);
  hipLaunchKernelGGL(select_kernel, dim3(a.n_layers * a.H_kv), dim3(kSelectThreads), lds, s, a);
  return hipGetLastError();
}

hipError_t prepare_select(int pool_stride) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(select_kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize,
                             static_cast<int>(pool_stride * sizeof(uint64_t)));
}

}  // namespace skv
