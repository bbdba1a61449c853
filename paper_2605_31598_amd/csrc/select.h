// Selection and state update of one (layer, KV head) (Eq. 4 and Eq. 6): the
// device code shared by the refresh launch and by the output launch of a
// key-split attention plan, which carries the deferred selection of an earlier
// one-layer call.  Everything here uses blockDim.x, so it runs with any
// workgroup size of up to kSelectThreads threads (a multiple of 64).
//
// 1. Finalise the importance scores of the candidate pool (state slots, then the
//    frame's tokens): s_j = (1/T) * sum over row tiles of the attention kernel's
//    column sums, added in fixed tile order (deterministic, no atomics).
// 2. If the pool exceeds B, find the threshold score s* = the B-th largest score
//    with a radix select over the fp32 bit patterns (non-negative floats order
//    like their bits).  Digits start below the common leading bits of the pool's
//    minimum and maximum, so no pass puts every key into one histogram bin.
// 3. Entries with s > s* are kept; among entries with s == s* (exact ties) the
//    lowest positions fill the remaining places, found by a second radix select
//    over the tied entries' positions (only when the ties straddle the boundary).
// 4. Pair evicted state slots (then free slots S, S+1, ...) with admitted frame
//    tokens in ascending order using block-wide scans, then copy the admitted
//    K/V rows into those slots.  Retained slots never move.
#pragma once
#include "internal.h"

namespace skv {
namespace {

constexpr int kLdsAdmit = 1024;  // frames up to this many tokens keep the admit lists in LDS

struct SelectShared {
  uint32_t hist[2][256];  // radix passes alternate between the two
  uint32_t wave_min[kSelectThreads / 64];
  uint32_t wave_max[kSelectThreads / 64];
  int wave_active[kSelectThreads / 64];
  uint32_t wave_total[kSelectThreads / 64];  // admit/evict scan
  int digit[2], remaining[2];           // one slot per pass parity
  uint32_t count[2];
  uint32_t cand[64];                    // keys of a small final bin, ranked directly
  int n_cand;
  uint32_t res_value;
  int res_need, res_equal;
  int32_t admit_src[kLdsAdmit];  // frame token of the a-th admitted candidate
  int32_t admit_dst[kLdsAdmit];  // state slot it goes to
};

struct RadixResult {
  uint32_t value;  // the rank-th largest key
  int need;        // how many entries equal to `value` fall within the top `rank`
  int equal;       // how many active entries equal `value`
};

// Wave-wide reductions and scans in registers (DPP and lane swaps, no LDS).
template <int CTRL>
__device__ inline uint32_t dpp_u32(uint32_t x) {  // all rows and banks; lanes without a source read 0
  return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), CTRL, 0xF, 0xF, true));
}
// f over all 64 lanes (f associative and commutative), in every lane: partners
// lane ^ 1, lane ^ 2, the mirrored quad, the mirrored half row, then the
// other row of a pair (lanes +-16) and the other half of the wave (lanes +-32).
template <typename F>
__device__ inline uint32_t wave_allreduce(uint32_t x, F f) {
  x = f(x, dpp_u32<0xB1>(x));   // quad_perm [1,0,3,2]
  x = f(x, dpp_u32<0x4E>(x));   // quad_perm [2,3,0,1]
  x = f(x, dpp_u32<0x141>(x));  // row_half_mirror
  x = f(x, dpp_u32<0x140>(x));  // row_mirror
  const auto r16 = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = f(r16[0], r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return f(r32[0], r32[1]);
}
__device__ inline uint32_t wave_min_u32(uint32_t x) {
  return wave_allreduce(x, [](uint32_t a, uint32_t b) { return min(a, b); });
}
__device__ inline uint32_t wave_max_u32(uint32_t x) {
  return wave_allreduce(x, [](uint32_t a, uint32_t b) { return max(a, b); });
}
__device__ inline int wave_sum_i32(int x) {
  return static_cast<int>(wave_allreduce(static_cast<uint32_t>(x), [](uint32_t a, uint32_t b) { return a + b; }));
}
// Inclusive prefix sum over lanes 0..lane: shifts by 1, 2, 4, 8 inside each row of
// 16 lanes, then the totals of rows 0 and 2 into rows 1 and 3 (row_bcast:15) and
// the total of rows 0-1 into rows 2 and 3 (row_bcast:31).
__device__ inline uint32_t wave_inclusive_sum(uint32_t x) {
  x += dpp_u32<0x111>(x);
  x += dpp_u32<0x112>(x);
  x += dpp_u32<0x114>(x);
  x += dpp_u32<0x118>(x);
  x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x142, 0xA, 0xF, false));
  x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x143, 0xC, 0xF, false));
  return x;
}

// Radix select over the active entries j < n: the rank-th largest key
// (1 <= rank <= number of active entries).  Digits of 8 bits start below the
// leading bits that all active keys share.
//
// Two barriers per pass: pass p counts into hist[p % 2] (cleared two passes
// earlier, or at entry) and publishes its digit in slot p % 2, which pass p + 2
// overwrites only after every thread has passed pass p + 1's first barrier.
template <typename KeyFn, typename ActiveFn>
__device__ RadixResult radix_select(int n, int rank, KeyFn key, ActiveFn active, SelectShared& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_waves = blockDim.x >> 6;
  for (int i = tid; i < 2 * 256; i += blockDim.x) sh.hist[i >> 8][i & 255] = 0u;
  if (tid == 0) sh.n_cand = 0;
  uint32_t lo = 0xFFFFFFFFu, hi = 0u;
  int cnt = 0;
  for (int j = tid; j < n; j += blockDim.x) {
    if (active(j)) {
      const uint32_t k = key(j);
      lo = min(lo, k);
      hi = max(hi, k);
      ++cnt;
    }
  }
  lo = wave_min_u32(lo);
  hi = wave_max_u32(hi);
  cnt = wave_sum_i32(cnt);
  if (lane == 0) {
    sh.wave_min[wave] = lo;
    sh.wave_max[wave] = hi;
    sh.wave_active[wave] = cnt;
  }
  __syncthreads();
  // every thread combines the per-wave values itself
  uint32_t l = 0xFFFFFFFFu, h = 0u;
  int n_active = 0;
  for (int w = 0; w < n_waves; ++w) {
    l = min(l, sh.wave_min[w]);
    h = max(h, sh.wave_max[w]);
    n_active += sh.wave_active[w];
  }
  const uint32_t diff = l ^ h;
  if (diff == 0u) {  // all active keys are equal
    __syncthreads();  // the per-wave values are read before a next call writes them
    return {h, rank, n_active};
  }

  const int top_bit = 31 - __clz(static_cast<int>(diff));  // highest bit where active keys differ
  uint32_t prefix = top_bit == 31 ? 0u : (h >> (top_bit + 1)) << (top_bit + 1);
  int remaining = rank;
  int equal = n_active;
  int par = 0;
  for (int shift = top_bit + 1; shift > 0; par ^= 1) {
    const int width = shift >= 8 ? 8 : shift;
    shift -= width;
    const uint32_t dmask = (1u << width) - 1u;
    const uint32_t fixed = ~((dmask << shift) | ((1u << shift) - 1u));  // bits already decided
    uint32_t* hist = sh.hist[par];
    for (int j = tid; j < n; j += blockDim.x) {
      if (!active(j)) continue;
      const uint32_t k = key(j);
      if ((k & fixed) == prefix) atomicAdd(&hist[(k >> shift) & dmask], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane t holds bins 255 - 4t down to 252 - 4t, so a prefix over lanes counts
      // the keys in this lane's bins and every higher one
      uint32_t c[4];
      for (int i = 0; i < 4; ++i) c[i] = hist[255 - 4 * tid - i];
      const uint32_t mine = c[0] + c[1] + c[2] + c[3];
      uint32_t above = wave_inclusive_sum(mine) - mine;  // keys in higher bins
      for (int i = 0; i < 4; ++i) {
        if (above < static_cast<uint32_t>(remaining) && static_cast<uint32_t>(remaining) <= above + c[i]) {
          sh.digit[par] = 255 - 4 * tid - i;
          sh.remaining[par] = remaining - static_cast<int>(above);
          sh.count[par] = c[i];
        }
        above += c[i];
      }
    }
    __syncthreads();
    prefix |= static_cast<uint32_t>(sh.digit[par]) << shift;
    remaining = sh.remaining[par];
    equal = static_cast<int>(sh.count[par]);
    if (shift > 0 && equal <= 64) {
      // Few keys share the prefix: instead of the remaining passes, gather them
      // and let one wave rank them (the same value, count needed and count equal).
      const uint32_t decided = ~((1u << shift) - 1u);
      for (int j = tid; j < n; j += blockDim.x) {
        if (!active(j)) continue;
        const uint32_t k = key(j);
        if ((k & decided) == prefix) sh.cand[atomicAdd(&sh.n_cand, 1)] = k;
      }
      __syncthreads();
      if (wave == 0) {
        const int nc = sh.n_cand;  // = equal
        const uint32_t mine = lane < nc ? sh.cand[lane] : 0u;
        int above = 0, same = 0;
        for (int i = 0; i < nc; ++i) {
          const uint32_t o = sh.cand[i];
          above += o > mine ? 1 : 0;
          same += o == mine ? 1 : 0;
        }
        // the lanes holding the remaining-th largest key (equal keys agree); the lowest writes
        const bool hit = lane < nc && above < remaining && remaining <= above + same;
        const uint64_t hits = __ballot(hit);
        if (hit && lane == __ffsll(static_cast<long long>(hits)) - 1) {
          sh.res_value = mine;
          sh.res_need = remaining - above;
          sh.res_equal = same;
        }
      }
      __syncthreads();
      return {sh.res_value, sh.res_need, sh.res_equal};
    }
    for (int i = tid; i < 256; i += blockDim.x) hist[i] = 0u;  // for pass p + 2
  }
  return {prefix, remaining, equal};
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ void refresh_state(const RefreshArgs& a, int lg, SelectShared& sh, uint32_t* pool_mem) {
  const int tid = threadIdx.x;
  const int S = a.S, T = a.T, B = a.B, P = S + T;
  uint32_t* sbits = pool_mem;
  int32_t* spos = reinterpret_cast<int32_t*>(pool_mem + P);
  const float* part = a.partial + static_cast<size_t>(lg) * a.tile_stride * a.pool_stride;
  const int n_tiles = a.lg_tiles[lg];
  int32_t* state_pos = a.state_pos + static_cast<size_t>(lg) * B;
  float* sscore = a.state_score + static_cast<size_t>(lg) * B;
  float* pscore = a.pool_score + static_cast<size_t>(lg) * a.pool_stride;
  int32_t* ppos = a.pool_pos + static_cast<size_t>(lg) * a.pool_stride;
  // admit lists (at most T entries each): in LDS for frames that fit, else the
  // global per-(layer, KV head) lists; a selection launch that leaves the state
  // update to a launch of its own always writes the global lists
  const bool lds_lists = T <= kLdsAdmit && !a.split_update;
  int32_t* asrc = lds_lists ? sh.admit_src : a.admit_src + static_cast<size_t>(lg) * T;
  int32_t* adst = lds_lists ? sh.admit_dst : a.admit_dst + static_cast<size_t>(lg) * T;

  // Each thread sums up to kJ candidates at a time, loading kTB row tiles of
  // each before adding them, so the loads overlap instead of waiting one by one;
  // the tiles are still added in order 0, 1, ... (padding adds exact zeros).
  constexpr int kJ = 4, kTB = 8;
  for (int j0 = tid; j0 < P; j0 += kJ * static_cast<int>(blockDim.x)) {
    float acc[kJ];
    int32_t pos[kJ];  // loaded with the first batch of tiles
#pragma unroll
    for (int q = 0; q < kJ; ++q) {
      acc[q] = 0.f;
      const int j = j0 + q * static_cast<int>(blockDim.x);
      pos[q] = j < S ? state_pos[j] : a.frame_pos0 + (j - S);
    }
    for (int t0 = 0; t0 < n_tiles; t0 += kTB) {
      float v[kJ][kTB];
#pragma unroll
      for (int q = 0; q < kJ; ++q)
#pragma unroll
        for (int u = 0; u < kTB; ++u) {
          const int j = min(j0 + q * static_cast<int>(blockDim.x), P - 1);
          const int t = min(t0 + u, n_tiles - 1);
          v[q][u] = part[static_cast<size_t>(t) * a.pool_stride + j];
        }
#pragma unroll
      for (int q = 0; q < kJ; ++q)
#pragma unroll
        for (int u = 0; u < kTB; ++u) acc[q] += t0 + u < n_tiles ? v[q][u] : 0.f;
    }
#pragma unroll
    for (int q = 0; q < kJ; ++q) {
      const int j = j0 + q * static_cast<int>(blockDim.x);
      if (j < P) {
        const float s = acc[q] * a.inv_T;
        pscore[j] = s;
        ppos[j] = pos[q];
        sbits[j] = __float_as_uint(s);
        spos[j] = pos[q];
      }
    }
  }
  __syncthreads();

  // selection key: the score bits, or the position for the recency window
  const bool recent = a.mode == 1;
  auto key = [&](int j) -> uint32_t { return recent ? static_cast<uint32_t>(spos[j]) : sbits[j]; };
  const bool prune = P > B;
  uint32_t s_thr = 0u;  // keep key > s_thr, and key == s_thr with position <= p_thr
  int32_t p_thr = 0x7FFFFFFF;
  if (prune && B > 0) {
    const RadixResult r = radix_select(P, B, key, [&](int) { return true; }, sh);
    s_thr = r.value;
    if (r.need < r.equal) {
      // exact ties straddle the boundary: the r.need lowest positions among key == s_thr;
      // a complemented position makes "largest" mean "lowest position"
      const RadixResult q = radix_select(
          P, r.need, [&](int j) { return 0x7FFFFFFFu - static_cast<uint32_t>(spos[j]); },
          [&](int j) { return key(j) == s_thr; }, sh);
      p_thr = static_cast<int32_t>(0x7FFFFFFFu - q.value);
    }
  }
  auto kept = [&](int j) -> bool {
    if (!prune) return true;
    if (B == 0) return false;
    const uint32_t kj = key(j);
    return kj > s_thr || (kj == s_thr && spos[j] <= p_thr);
  };

  // Admitted frame tokens (ascending t) and evicted state slots (ascending
  // slot).  Each thread owns a contiguous chunk of both (at most 32 entries of
  // each: S, T <= 16384 over 512 or more threads); one block-wide scan of its packed
  // counts (admitted in the low 16 bits, evicted in the high 16, totals below
  // 2^16) gives its offsets into both lists.
  const int nt = static_cast<int>(blockDim.x);
  const int lane = tid & 63, wave = tid >> 6, n_waves = nt >> 6;
  const int ca = (T + nt - 1) / nt, ce = (S + nt - 1) / nt;
  const int a0 = tid * ca, e0 = tid * ce;
  uint32_t adm_mask = 0u, ev_mask = 0u;
  for (int i = 0; i < ca; ++i)
    if (a0 + i < T && kept(S + a0 + i)) adm_mask |= 1u << i;
  for (int i = 0; i < ce; ++i)
    if (e0 + i < S && !kept(e0 + i)) ev_mask |= 1u << i;
  const uint32_t mine = static_cast<uint32_t>(__popc(adm_mask)) | (static_cast<uint32_t>(__popc(ev_mask)) << 16);
  const uint32_t incl = wave_inclusive_sum(mine);
  if (lane == 63) sh.wave_total[wave] = incl;
  __syncthreads();
  uint32_t before = incl - mine, total = 0u;
  for (int w = 0; w < n_waves; ++w) {
    const uint32_t c = sh.wave_total[w];
    before += w < wave ? c : 0u;
    total += c;
  }
  const int n_adm = static_cast<int>(total & 0xFFFFu), n_ev = static_cast<int>(total >> 16);
  int ra = static_cast<int>(before & 0xFFFFu), re = static_cast<int>(before >> 16);
  for (int i = 0; i < ca; ++i)
    if (adm_mask >> i & 1u) asrc[ra++] = a0 + i;
  // retained slots get the new score; a valid selection evicts at most as many
  // slots as it admits (<= T), and the bound keeps the list inside its T entries
  for (int i = 0; i < ce; ++i) {
    const int j = e0 + i;
    if (j >= S) break;
    if (ev_mask >> i & 1u) {
      if (re < T) adst[re] = j;
      ++re;
    } else {
      sscore[j] = __uint_as_float(sbits[j]);
    }
  }
  // Holes beyond the evicted slots are the free slots S, S+1, ... (state not yet full).
  // Clamping keeps writes inside the B slots even for an invalid forced state
  // with repeated positions.
  const int n_holes = n_ev + (B - S);
  const int count = n_adm < n_holes ? n_adm : n_holes;
  for (int i = n_ev + tid; i < count; i += blockDim.x) adst[i] = S + (i - n_ev);
  if (a.split_update) {  // the update launch copies the rows
    if (tid == 0) a.admit_count[lg] = count;
    return;
  }
  __syncthreads();  // the admit lists are read back by other threads below

  // State update: admitted frame rows into their slots, 16-byte chunks.
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
      sscore[dst] = __uint_as_float(sbits[S + src]);
    }
  }
}


// LDS bytes refresh_state needs with a pool of P candidates: the shared
// workspace, then the pool's score bits and positions.
constexpr size_t select_lds_bytes(int P) {
  return (sizeof(SelectShared) + 15) / 16 * 16 + static_cast<size_t>(P) * 2 * sizeof(uint32_t);
}

}  // namespace
}  // namespace skv
