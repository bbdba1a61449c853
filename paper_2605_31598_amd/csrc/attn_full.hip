// Streaming full self-attention of one frame (the Full SA baseline), bf16 MFMA,
// gfx950 (CDNA4).
//
// For one frame n and a range of layers:
//     O = softmax(Q [K_D; K_frame]^T * scale + M_n) [V_D; V_frame]
// where K_D, V_D are the n * T earlier tokens of the layer's decode cache D
// (always visible) and the frame's own keys are causal (Eq. 5 with the whole
// history in place of the compressed state).  No importance scores: a single
// sweep over the keys with an online softmax.
//
// Work decomposition, LDS tiles, K Q^T and the transpose reads of V are those of
// the StateKV attention kernel (256-row workgroups from the host plan, 8 waves
// of 32 query rows, 128-key tiles double-buffered through LDS).  What differs:
//   * The PV product is accumulated transposed, O^T = V^T P^T, with the same
//     registers in swapped operand slots: the V operand read for P V is exactly
//     the A operand of V^T P^T, and P (16 keys of one query row per lane) is
//     exactly its B operand.  The accumulator then holds, in lane l, 64 head
//     dimensions of query row l % 32, so the online-softmax correction of a row
//     is a scalar of the lane that owns the row.
//   * Rescaling follows the row maximum exactly (no slack): when a 32-key block
//     raises the maximum of any row of the wave, every lane multiplies its
//     accumulators by exp2((m_old - m_new) * c), which is 1 for rows whose
//     maximum did not move.  Exponentials are therefore <= 1 and the largest
//     entry of a row is exactly 1 in bf16, as in the StateKV kernel.
#include "internal.h"

#include <type_traits>

namespace skv {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kWaves = kMfmaWaves;
constexpr int kThreads = kWaves * 64;
constexpr int kRowsWave = kMfmaRowsPerWave;
constexpr int kKT = 128;   // keys per LDS tile (four 32-key blocks)
constexpr int kPadK = 8;   // K row padding (bf16): 16-byte reads conflict-free
// V row padding (bf16).  ds_read_b64_tr_b16 serves 32 lanes (four rows x 64 B) per
// LDS pass over 64 four-byte banks; a row stride of 80 (D = 128) or 48 (D = 64)
// dwords, modulo 64, puts those four rows on disjoint banks.  A 16-element pad
// (72 dwords) overlaps them two-way.
constexpr int kPadV = 32;
constexpr int kPadO = 8;   // output staging row padding (bf16)

template <int D>
struct SmemFull {
  uint16_t k[2][kKT][D + kPadK];
  uint16_t v[2][kKT][D + kPadV];
};
static_assert(sizeof(SmemFull<128>) <= 160 * 1024, "gfx950 LDS per workgroup");

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }  // v_exp_f32

__device__ inline unsigned pack_bf16x2(float lo, float hi) {
  return static_cast<unsigned>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(lo))) |
         (static_cast<unsigned>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(hi))) << 16);
}

}  // namespace

// ROPE: rotate Q at the frame tokens' virtual positions (a separate
// instantiation, so the kernel without rotation carries none of its code).  The
// frame's keys arrive rotated (rope_keys.hip), like the state's and the cache's.
template <int D, bool ROPE>
__global__ __launch_bounds__(kThreads, 1) void attn_full_kernel(AttnArgs a) {
  constexpr int KS = D / 16;                   // k-steps of K Q^T
  constexpr int DB = D / 32;                   // 32-dimension blocks of O^T
  constexpr int KCH = D / 8;                   // 16-byte chunks per K/V row
  constexpr int ITEMS = kKT * KCH / kThreads;  // chunks of one tile staged per thread
  static_assert(ITEMS * kThreads == kKT * KCH, "staging split");
  static_assert(kWaves * kRowsWave * (D + kPadO) * 2 <= static_cast<int>(sizeof(SmemFull<D>)), "output staging");

  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  SmemFull<D>& sm = *reinterpret_cast<SmemFull<D>*>(smem_raw);

  const AttnWork wk = a.work[blockIdx.x];
  if (wk.rows <= 0) return;
  const int lg = wk.lg;
  const int layer = lg / a.H_kv, g = lg % a.H_kv;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, h = lane >> 5;
  const int S = a.S, n_keys = a.S + a.T;  // S = cached tokens before this frame
  const int n_tiles = (n_keys + kKT - 1) / kKT;
  const int first_masked = S / kKT;  // tiles from here on contain frame keys or the ragged end
  const int row_end = wk.row0 + wk.rows;
  const int row0 = wk.row0 + wave * kRowsWave;
  const bool active = row0 < row_end;
  const float c = a.scale_log2;

  const uint16_t* qg = static_cast<const uint16_t*>(a.q) + static_cast<size_t>(layer * a.H_q + g * a.G) * a.T * D;
  const uint16_t* kst = static_cast<const uint16_t*>(a.ks) + static_cast<size_t>(lg) * a.kv_rows * D;
  const uint16_t* vst = static_cast<const uint16_t*>(a.vs) + static_cast<size_t>(lg) * a.kv_rows * D;
  const uint16_t* kfr = static_cast<const uint16_t*>(a.kf) + static_cast<size_t>(lg) * a.T * D;
  const uint16_t* vfr = static_cast<const uint16_t*>(a.vf) + static_cast<size_t>(lg) * a.T * D;

  const int r_lane = row0 + l32;
  const bool row_valid = r_lane < row_end;
  const int lim = row_valid ? S + (r_lane % a.T) : -1;  // key j is visible iff j <= lim
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
  // pure: tile t lies wholly among the cached keys, so no key needs a test; thread
  // tid's item it is row it * (kThreads / KCH) + tid / KCH, chunk tid % KCH.
  const int base_off = (tid / KCH) * D + (tid % KCH) * 8;
  auto load_tile = [&](int t, auto pure) {
    if constexpr (decltype(pure)::value) {
      const uint16_t* kt = kst + static_cast<size_t>(t) * kKT * D + base_off;
      const uint16_t* vt = vst + static_cast<size_t>(t) * kKT * D + base_off;
#pragma unroll
      for (int it = 0; it < ITEMS; ++it) {
        kpre[it] = *reinterpret_cast<const u32x4*>(kt + it * (kThreads / KCH) * D);
        vpre[it] = *reinterpret_cast<const u32x4*>(vt + it * (kThreads / KCH) * D);
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
        y = *reinterpret_cast<const u32x4*>(vst + static_cast<size_t>(j) * D + ch * 8);
      } else if (j < n_keys) {
        x = *reinterpret_cast<const u32x4*>(kfr + static_cast<size_t>(j - S) * D + ch * 8);
        y = *reinterpret_cast<const u32x4*>(vfr + static_cast<size_t>(j - S) * D + ch * 8);
      }
      kpre[it] = x;
      vpre[it] = y;
    }
  };
  auto store_tile = [&](int b) {
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int idx = it * kThreads + tid;
      const int kk = idx / KCH, ch = idx % KCH;
      *reinterpret_cast<u32x4*>(&sm.k[b][kk][ch * 8]) = kpre[it];
      *reinterpret_cast<u32x4*>(&sm.v[b][kk][ch * 8]) = vpre[it];
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

  // transpose-read coordinates of this lane inside its 16-lane group
  const int tr_row = 4 * h + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  // ============================ single sweep ============================
  f32x16 ot[DB];  // O^T: lane l holds dims 32 db + 8 (v / 4) + 4 h + v % 4 of row l % 32
#pragma unroll
  for (int db = 0; db < DB; ++db) ot[db] = f32x16{};
  float m = -1e30f;  // running row maximum (logit units), the same in lanes l and l ^ 32
  float l = 0.f;     // this lane's share of the row sum of exp2((x - m) c)

  auto sweep_tile = [&](int t, auto masked, auto pure_next) {
    const int b = t & 1;
    if (t + 1 < n_tiles) load_tile(t + 1, pure_next);
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
        float bm = z[0];
#pragma unroll
        for (int v = 1; v < 16; ++v) bm = fmaxf(bm, z[v]);
        bm = fmaxf(bm, __shfl_xor(bm, 32, 64));  // the block's other 16 keys of this row
        const bool grow = bm > m;
        if (__ballot(grow)) {
          // Subtract before scaling: the first finite maximum replaces the sentinel
          // with a factor of exactly 0, an unchanged maximum gives exactly 1.
          const float f = grow ? fast_exp2((m - bm) * c) : 1.f;
          m = grow ? bm : m;
          l *= f;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) ot[db][v] *= f;
        }
        const float mc = m * c;
        bf16x8 pe[2];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float e = fast_exp2(fmaf(z[v], c, -mc));  // masked: exp2(-inf) = 0
          l += e;
          pe[v >> 3][v & 7] = static_cast<__bf16>(e);
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
          for (int db = 0; db < DB; ++db) ot[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[s][db], pe[s], ot[db], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 4 * DB; ++i) __builtin_amdgcn_sched_group_barrier(0x100, 1, 2);
#pragma unroll
        for (int i = 0; i < 2 * DB; ++i) __builtin_amdgcn_sched_group_barrier(0x008, 1, 2);
        __builtin_amdgcn_s_setprio(0);
      }
    }
    if (t + 1 < n_tiles) store_tile(b ^ 1);
    __syncthreads();
  };
  load_tile(0, std::false_type{});
  store_tile(0);
  __syncthreads();
  for (int t = 0; t + 1 < first_masked; ++t) sweep_tile(t, std::false_type{}, std::true_type{});
  if (first_masked > 0) sweep_tile(first_masked - 1, std::false_type{}, std::false_type{});
  for (int t = first_masked; t < n_tiles; ++t) sweep_tile(t, std::true_type{}, std::false_type{});

  // ---------------- output: O^T / sum, staged through LDS for 16-byte stores ----------------
  const float lt = l + __shfl_xor(l, 32, 64);
  const float inv = row_valid ? 1.0f / lt : 0.f;
  uint16_t* ost = reinterpret_cast<uint16_t*>(smem_raw) + static_cast<size_t>(wave) * kRowsWave * (D + kPadO);
  if (active) {
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d0 = db * 32 + 8 * q4 + 4 * h;
        const u32x2 w = {pack_bf16x2(ot[db][4 * q4] * inv, ot[db][4 * q4 + 1] * inv),
                         pack_bf16x2(ot[db][4 * q4 + 2] * inv, ot[db][4 * q4 + 3] * inv)};
        *reinterpret_cast<u32x2*>(ost + l32 * (D + kPadO) + d0) = w;
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

hipError_t launch_attention_full_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
  const int grid = a.n_work;
  const bool rope = a.rope_tab != nullptr;
  if (head_dim == 128) {
    if (rope)
      hipLaunchKernelGGL((attn_full_kernel<128, true>), dim3(grid), dim3(kThreads), sizeof(SmemFull<128>), s, a);
    else
      hipLaunchKernelGGL((attn_full_kernel<128, false>), dim3(grid), dim3(kThreads), sizeof(SmemFull<128>), s, a);
  } else {
    if (rope)
      hipLaunchKernelGGL((attn_full_kernel<64, true>), dim3(grid), dim3(kThreads), sizeof(SmemFull<64>), s, a);
    else
      hipLaunchKernelGGL((attn_full_kernel<64, false>), dim3(grid), dim3(kThreads), sizeof(SmemFull<64>), s, a);
  }
  return hipGetLastError();
}

hipError_t prepare_attention_full() {
  const void* kernels[] = {reinterpret_cast<const void*>(attn_full_kernel<128, false>),
                            reinterpret_cast<const void*>(attn_full_kernel<128, true>)};
  for (const void* k : kernels) {
    const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, sizeof(SmemFull<128>));
    if (e != hipSuccess) return e;
  }
  const void* kernels64[] = {reinterpret_cast<const void*>(attn_full_kernel<64, false>),
                              reinterpret_cast<const void*>(attn_full_kernel<64, true>)};
  for (const void* k : kernels64) {
    const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, sizeof(SmemFull<64>));
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace skv
