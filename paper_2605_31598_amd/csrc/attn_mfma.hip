// bf16 MFMA attention with fused importance scoring, gfx950 (CDNA4).
//
// Computes, for one frame and a range of layers, Eq. 5
//     O = softmax(Q [K_state; K_frame]^T * scale + M_n) [V_state; V_frame]
// and, for every candidate key j, the column sum over the workgroup's query rows
// of the normalised attention A_{i,j}; the selection kernel adds the row tiles and
// divides by T (the importance score of the attention-driven selection).
//
// Work decomposition
//   * A workgroup owns 256 query rows of one (layer, KV head): 8 waves x 32 rows,
//     two waves per SIMD.  Rows are the G query heads sharing the KV head times
//     the T frame tokens (grouped-query packing: every row of the tile reads the
//     same K/V).  Two waves per SIMD let the hardware run one wave's exp/softmax
//     VALU work under the other wave's MFMAs; a single wave does not overlap its
//     own MFMA and VALU streams well on gfx950.
//   * Keys stream through LDS in tiles of 128 (four 32-key blocks), double
//     buffered, K and V both row-major; the next tile's global loads are issued
//     before the current tile's compute.  A block's K (and V) operand reads are
//     all issued before its MFMA chain, and waves raise their priority while
//     issuing MFMAs so the other wave on the SIMD fills the VALU slots.
//   * Two sweeps over the keys.  Sweep 1: S^T = K Q^T -> per-row max and sum of
//     exp2.  Sweep 2: S^T again -> E = exp2(x - row max) -> O += E V (scaled by
//     1/sum at the end) and per-key column sums of P = E / sum.  Exact
//     probabilities are known only after the row statistics, and recomputing
//     K Q^T is cheaper than storing the logits.
//   * Tiles that contain frame keys (the only ones with masked entries) run in a
//     separate loop, keeping mask code off the common path.
//   * The blockIdx -> tile mapping keeps the row tiles of one (layer, KV head)
//     on one XCD so they share K/V in that XCD's L2.
//
// MFMA v_mfma_f32_32x32x16_bf16 (wave64) operand layout, lane l, h = l / 32:
//   A (32x16): A[l % 32][8h .. 8h+7]   B (16x32): B[8h .. 8h+7][l % 32]
//   C (32x32): element v (0..15) of lane l is C[8(v/4) + 4h + v%4][l % 32].
// With S^T = K Q^T (M = keys, N = query rows, K = head dim) lane l holds 16
// keys of query row l % 32, which is the A-operand shape of O = P V once the
// contraction index k = 8h + i of k-step s is taken to mean key
// 16s + 4h + (i < 4 ? i : i + 4).  The matching B operand (V rows of those keys,
// one column per lane) comes from ds_read_b64_tr_b16: inside each group of 16
// lanes, lane j points at V[k0 + j/4][d0 + 4(j%4)] and receives
// V[k0 .. k0+3][d0 + j].
#include "internal.h"

#include <type_traits>

namespace skv {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kWaves = kMfmaWaves;
constexpr int kThreads = kWaves * 64;
constexpr int kRowsWave = kMfmaRowsPerWave;
constexpr int kKT = 128;       // keys per LDS tile (four 32-key blocks)
constexpr int kPadK = 8;       // K row padding (bf16): 16-byte reads conflict-free
constexpr int kPadV = 16;      // V row padding (bf16): transpose reads conflict-free
constexpr int kPadO = 8;       // output staging row padding (bf16)

template <int D>
struct Smem {
  uint16_t k[2][kKT][D + kPadK];
  uint16_t v[2][kKT][D + kPadV];
  float cs[2][kWaves][kKT];     // per-wave column sums of one tile
  float il[kWaves][kRowsWave];  // 1 / row sum, for the output
};

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }  // v_exp_f32

template <int CTRL>
__device__ inline float dpp_f(float x) {
  // DPP lane permutation inside rows of 16 lanes (all rows and banks enabled).
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}

// Sum of cs[16] over the 32 lanes that share h = lane / 32 (the query rows of
// one half-block).  Returns, in every lane, the total of the key
//   key(lane) = 8 * (b3 + 2 * b4) + 4 * h + (b1 + 2 * b2)     (bN = bit N of lane)
// within the 32-key block; lanes differing only in bit 0 return the same key.
// Reduce-scatter: each step halves the values a lane carries while pairing
// lanes that differ in one more row bit.
__device__ inline float column_reduce(const float (&cs)[16], int lane) {
  float c1[8];
#pragma unroll
  for (int v = 0; v < 8; ++v) {  // rows 0<->1 and 2<->3: lanes l and l^16
    const auto pr = __builtin_amdgcn_permlane16_swap(__float_as_uint(cs[v]), __float_as_uint(cs[v + 8]),
                                                     false, false);
    c1[v] = __uint_as_float(pr[0]) + __uint_as_float(pr[1]);
  }
  const bool b3 = lane & 8, b2 = lane & 4, b1 = lane & 2;
  float c2[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {  // lanes i <-> i^8 inside a row
    const float keep = b3 ? c1[v + 4] : c1[v];
    const float send = b3 ? c1[v] : c1[v + 4];
    c2[v] = keep + dpp_f<0x128>(send);
  }
  float c3[2];
#pragma unroll
  for (int v = 0; v < 2; ++v) {  // lanes i <-> 7-i inside each half row (bit 2 differs)
    const float keep = b2 ? c2[v + 2] : c2[v];
    const float send = b2 ? c2[v] : c2[v + 2];
    c3[v] = keep + dpp_f<0x141>(send);
  }
  const float keep = b1 ? c3[1] : c3[0];  // lanes i <-> 3-i inside a quad (bit 1 differs)
  const float send = b1 ? c3[0] : c3[1];
  const float c4 = keep + dpp_f<0x1B>(send);
  return c4 + dpp_f<0xB1>(c4);  // lanes i <-> i^1
}

}  // namespace

// ROPE: rotate Q at the frame tokens' virtual positions (a separate
// instantiation, so the kernel without rotation carries none of its code).  The
// frame's keys arrive rotated (rope_keys.hip), like the state's and the cache's.
template <int D, bool ROPE>
__global__ __launch_bounds__(kThreads, 1) void attn_mfma_kernel(AttnArgs a) {
  constexpr int KS = D / 16;                   // k-steps of K Q^T
  constexpr int DB = D / 32;                   // 32-column blocks of O
  constexpr int KCH = D / 8;                   // 16-byte chunks per K/V row
  constexpr int ITEMS = kKT * KCH / kThreads;  // chunks of one tile staged per thread
  static_assert(ITEMS * kThreads == kKT * KCH, "staging split");

  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  Smem<D>& sm = *reinterpret_cast<Smem<D>*>(smem_raw);

  // The host plan fixes each workgroup's (layer, KV head), row range and
  // row-tile slot; it already places the work of one (layer, KV head) on one XCD.
  const AttnWork wk = a.work[blockIdx.x];
  if (wk.rows <= 0) return;
  const int lg = wk.lg;
  const int layer = lg / a.H_kv, g = lg % a.H_kv;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, h = lane >> 5;
  const int S = a.S, n_keys = a.S + a.T;
  const int n_tiles = (n_keys + kKT - 1) / kKT;
  const int first_masked = S / kKT;  // tiles from here on contain frame keys or the ragged end
  const int row_end = wk.row0 + wk.rows;  // rows of this workgroup: [wk.row0, row_end)
  const int row0 = wk.row0 + wave * kRowsWave;
  const bool active = row0 < row_end;
  const float c = a.scale_log2;

  const uint16_t* qg = static_cast<const uint16_t*>(a.q) + static_cast<size_t>(layer * a.H_q + g * a.G) * a.T * D;
  const uint16_t* kst = static_cast<const uint16_t*>(a.ks) + static_cast<size_t>(lg) * a.B * D;
  const uint16_t* vst = static_cast<const uint16_t*>(a.vs) + static_cast<size_t>(lg) * a.B * D;
  const uint16_t* kfr = static_cast<const uint16_t*>(a.kf) + static_cast<size_t>(lg) * a.T * D;
  const uint16_t* vfr = static_cast<const uint16_t*>(a.vf) + static_cast<size_t>(lg) * a.T * D;
  float* part = a.partial + (static_cast<size_t>(lg) * a.tile_stride + wk.tile) * a.pool_stride;

  // Q^T operand (B of K Q^T) in registers; an invalid row is zero and sees no key.
  const int r_lane = row0 + l32;
  const bool row_valid = r_lane < row_end;
  const int lim = row_valid ? S + (r_lane % a.T) : -1;  // candidate j is visible iff j <= lim
  bf16x8 qreg[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    u32x4 x = {0u, 0u, 0u, 0u};
    if (row_valid) x = *reinterpret_cast<const u32x4*>(qg + static_cast<size_t>(r_lane) * D + ks * 16 + h * 8);
    qreg[ks] = __builtin_bit_cast(bf16x8, x);
  }
  if (ROPE && row_valid) {  // RoPE at the frame token's virtual position
    const float* tb = a.rope_tab + static_cast<size_t>(a.rope_pos0 + r_lane % a.T) * D;
#pragma unroll
    for (int ks = 0; ks < KS / 2; ++ks) {
      const u32x4 lo = __builtin_bit_cast(u32x4, qreg[ks]), hi = __builtin_bit_cast(u32x4, qreg[ks + KS / 2]);
      qreg[ks] = __builtin_bit_cast(bf16x8, rope_chunk_bf16(lo, hi, false, ks * 16 + h * 8, tb));
      qreg[ks + KS / 2] = __builtin_bit_cast(bf16x8, rope_chunk_bf16(hi, lo, true, ks * 16 + h * 8, tb));
    }
  }

  // ---------------- staging (global -> registers -> LDS) ----------------
  u32x4 kpre[ITEMS], vpre[ITEMS];
  // pure: tile t lies wholly inside the state, so no key needs a test; thread
  // tid's item it is row it * (kThreads / KCH) + tid / KCH, chunk tid % KCH.
  const int base_off = (tid / KCH) * D + (tid % KCH) * 8;
  auto load_tile = [&](int t, bool with_v, auto pure) {
    if constexpr (decltype(pure)::value) {
      const uint16_t* kt = kst + static_cast<size_t>(t) * kKT * D + base_off;
      const uint16_t* vt = vst + static_cast<size_t>(t) * kKT * D + base_off;
#pragma unroll
      for (int it = 0; it < ITEMS; ++it) {
        kpre[it] = *reinterpret_cast<const u32x4*>(kt + it * (kThreads / KCH) * D);
        vpre[it] = with_v ? *reinterpret_cast<const u32x4*>(vt + it * (kThreads / KCH) * D) : u32x4{0u, 0u, 0u, 0u};
      }
      return;
    }
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int idx = it * kThreads + tid;
      const int kk = idx / KCH, ch = idx % KCH;
      const int j = t * kKT + kk;
      u32x4 x = {0u, 0u, 0u, 0u}, y = {0u, 0u, 0u, 0u};
      if (j < S) {
        x = *reinterpret_cast<const u32x4*>(kst + static_cast<size_t>(j) * D + ch * 8);
        if (with_v) y = *reinterpret_cast<const u32x4*>(vst + static_cast<size_t>(j) * D + ch * 8);
      } else if (j < n_keys) {
        x = *reinterpret_cast<const u32x4*>(kfr + static_cast<size_t>(j - S) * D + ch * 8);
        if (with_v) y = *reinterpret_cast<const u32x4*>(vfr + static_cast<size_t>(j - S) * D + ch * 8);
      }
      kpre[it] = x;
      vpre[it] = y;
    }
  };
  auto store_tile = [&](int b, bool with_v) {
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int idx = it * kThreads + tid;
      const int kk = idx / KCH, ch = idx % KCH;
      *reinterpret_cast<u32x4*>(&sm.k[b][kk][ch * 8]) = kpre[it];
      if (with_v) *reinterpret_cast<u32x4*>(&sm.v[b][kk][ch * 8]) = vpre[it];
    }
  };

  // S^T block (32 keys x 32 rows) for key block kb of buffer b.
  auto qk = [&](int b, int kb) -> f32x16 {
    __builtin_amdgcn_s_setprio(1);
    u32x4 kop[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kop[ks] = *reinterpret_cast<const u32x4*>(&sm.k[b][kb * 32 + l32][ks * 16 + h * 8]);
    f32x16 acc = {};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kop[ks]), qreg[ks], acc, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < KS; ++i) __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);
#pragma unroll
    for (int i = 0; i < KS; ++i) __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
    __builtin_amdgcn_s_setprio(0);
    return acc;
  };

  // ============================ sweep 1: row statistics ============================
  float m = -1e30f, l = 0.f;
  auto sweep1_tile = [&](int t, auto masked, auto pure_next) {
    const int b = t & 1;
    if (t + 1 < n_tiles) load_tile(t + 1, false, pure_next);
    if (active) {
#pragma unroll
      for (int kb = 0; kb < kKT / 32; ++kb) {
        const f32x16 acc = qk(b, kb);
        float z[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) z[v] = acc[v];
        if constexpr (decltype(masked)::value) {
          const int rel = lim - (t * kKT + kb * 32 + 4 * h);
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (8 * (v >> 2) + (v & 3) > rel) z[v] = -__builtin_huge_valf();
        }
        float mx = z[0];
#pragma unroll
        for (int v = 1; v < 16; ++v) mx = fmaxf(mx, z[v]);
        const float mn = fmaxf(m, mx);
        const float mc = mn * c;
        float sum = 0.f;
#pragma unroll
        for (int v = 0; v < 16; ++v) sum += fast_exp2(fmaf(z[v], c, -mc));
        // Subtract before scaling: equal maxima (including the empty-row sentinel)
        // give exactly exp2(0) = 1.
        l = l * fast_exp2((m - mn) * c) + sum;
        m = mn;
      }
    }
    if (t + 1 < n_tiles) store_tile(b ^ 1, false);
    __syncthreads();
  };
  load_tile(0, false, std::false_type{});
  store_tile(0, false);
  __syncthreads();
  for (int t = 0; t + 1 < first_masked; ++t) sweep1_tile(t, std::false_type{}, std::true_type{});
  if (first_masked > 0) sweep1_tile(first_masked - 1, std::false_type{}, std::false_type{});
  for (int t = first_masked; t < n_tiles; ++t) sweep1_tile(t, std::true_type{}, std::false_type{});

  // Row maximum (log2 units) and 1/sum.  Sweep 2 feeds the PV MFMA with
  // E = exp2(x - max) <= 1, whose largest entry is exactly 1 in bf16, and applies
  // 1/sum in fp32 to the output; the column sums use P = E / sum.
  float mrow, inv_l;
  {
    // the other 16 keys of every 32-key block live in lane ^ 32
    const float mo = __shfl_xor(m, 32, 64);
    const float lo = __shfl_xor(l, 32, 64);
    const float mm = fmaxf(m, mo);
    const float ll = l * fast_exp2((m - mm) * c) + lo * fast_exp2((mo - mm) * c);
    mrow = row_valid ? mm * c : 0.f;
    inv_l = row_valid ? 1.0f / ll : 0.f;
  }

  // ======================== sweep 2: P, O and column sums ========================
  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = f32x16{};

  const int key_lane = 8 * (((lane >> 3) & 1) + 2 * ((lane >> 4) & 1)) + 4 * h + (((lane >> 1) & 1) + 2 * ((lane >> 2) & 1));
  // transpose-read coordinates of this lane inside its 16-lane group
  const int tr_row = 4 * h + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  auto sweep2_tile = [&](int t, auto masked, auto pure_next) {
    const int b = t & 1;
    if (t + 1 < n_tiles) load_tile(t + 1, true, pure_next);
    if (active) {
#pragma unroll
      for (int kb = 0; kb < kKT / 32; ++kb) {
        const f32x16 acc = qk(b, kb);
        const int rel = lim - (t * kKT + kb * 32 + 4 * h);
        bf16x8 pe[2];
        float cs[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float e = fast_exp2(fmaf(acc[v], c, -mrow));
          if constexpr (decltype(masked)::value) {
            if (8 * (v >> 2) + (v & 3) > rel) e = 0.f;
          }
          pe[v >> 3][v & 7] = static_cast<__bf16>(e);
          cs[v] = e * inv_l;
        }
        __builtin_amdgcn_s_setprio(1);
        bf16x8 vop[2][DB];
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const int r = kb * 32 + s * 16 + tr_row;
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(&sm.v[b][r][db * 32 + tr_col]));
            const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(&sm.v[b][r + 8][db * 32 + tr_col]));
            vop[s][db] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
          }
        }
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
          for (int db = 0; db < DB; ++db) o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pe[s], vop[s][db], o[db], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 4 * DB; ++i) __builtin_amdgcn_sched_group_barrier(0x100, 1, 2);
#pragma unroll
        for (int i = 0; i < 2 * DB; ++i) __builtin_amdgcn_sched_group_barrier(0x008, 1, 2);
        __builtin_amdgcn_s_setprio(0);
        const float tot = column_reduce(cs, lane);
        if ((lane & 1) == 0) sm.cs[b][wave][kb * 32 + key_lane] = tot;
      }
    } else {
      for (int i = lane; i < kKT; i += 64) sm.cs[b][wave][i] = 0.f;
    }
    if (t + 1 < n_tiles) store_tile(b ^ 1, true);
    __syncthreads();
    // cross-wave column sums of tile t -> this row tile's partials; buffer b is
    // written again only after the next barrier
    if (tid < kKT) {
      const int j = t * kKT + tid;
      if (j < n_keys) {
        float sum = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) sum += sm.cs[b][w][tid];
        part[j] = sum;
      }
    }
  };
  load_tile(0, true, std::false_type{});
  store_tile(0, true);
  __syncthreads();
  for (int t = 0; t + 1 < first_masked; ++t) sweep2_tile(t, std::false_type{}, std::true_type{});
  if (first_masked > 0) sweep2_tile(first_masked - 1, std::false_type{}, std::false_type{});
  for (int t = first_masked; t < n_tiles; ++t) sweep2_tile(t, std::true_type{}, std::false_type{});

  // ---------------- output: O / sum, staged through LDS for 16-byte stores ----------------
  if (active && h == 0) sm.il[wave][l32] = inv_l;
  __syncthreads();
  uint16_t* ost = reinterpret_cast<uint16_t*>(smem_raw) + static_cast<size_t>(wave) * kRowsWave * (D + kPadO);
  if (active) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int r = 8 * (v >> 2) + 4 * h + (v & 3);
      const float sc = sm.il[wave][r];
#pragma unroll
      for (int db = 0; db < DB; ++db)
        ost[r * (D + kPadO) + db * 32 + l32] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(o[db][v] * sc));
    }
  }
  __syncthreads();
  if (active) {
    uint16_t* og = static_cast<uint16_t*>(a.out) + static_cast<size_t>(layer * a.H_q + g * a.G) * a.T * D;
#pragma unroll
    for (int it = 0; it < kRowsWave * KCH / 64; ++it) {
      const int idx = it * 64 + lane;
      const int r = idx / KCH, ch = idx % KCH;
      if (row0 + r < row_end)
        *reinterpret_cast<u32x4*>(og + static_cast<size_t>(row0 + r) * D + ch * 8) =
            *reinterpret_cast<const u32x4*>(ost + r * (D + kPadO) + ch * 8);
    }
  }
}

hipError_t launch_attention_mfma_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
  const int grid = a.n_work;
  const bool rope = a.rope_tab != nullptr;
  if (head_dim == 128) {
    if (rope)
      hipLaunchKernelGGL((attn_mfma_kernel<128, true>), dim3(grid), dim3(kThreads), sizeof(Smem<128>), s, a);
    else
      hipLaunchKernelGGL((attn_mfma_kernel<128, false>), dim3(grid), dim3(kThreads), sizeof(Smem<128>), s, a);
  } else {
    if (rope)
      hipLaunchKernelGGL((attn_mfma_kernel<64, true>), dim3(grid), dim3(kThreads), sizeof(Smem<64>), s, a);
    else
      hipLaunchKernelGGL((attn_mfma_kernel<64, false>), dim3(grid), dim3(kThreads), sizeof(Smem<64>), s, a);
  }
  return hipGetLastError();
}

hipError_t prepare_attention_mfma() {
  const void* kernels[] = {reinterpret_cast<const void*>(attn_mfma_kernel<128, false>),
                            reinterpret_cast<const void*>(attn_mfma_kernel<128, true>)};
  for (const void* k : kernels) {
    const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, sizeof(Smem<128>));
    if (e != hipSuccess) return e;
  }
  const void* kernels64[] = {reinterpret_cast<const void*>(attn_mfma_kernel<64, false>),
                              reinterpret_cast<const void*>(attn_mfma_kernel<64, true>)};
  for (const void* k : kernels64) {
    const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, sizeof(Smem<64>));
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace skv
