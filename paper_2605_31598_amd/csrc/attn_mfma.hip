// bf16 MFMA attention with fused importance scoring, gfx950 (CDNA4).
//
// Computes, for one frame and a range of layers, Eq. 5
//     O = softmax(Q [K_state; K_frame]^T * scale + M_n) [V_state; V_frame]
// and, for every candidate key j, the column sum over the workgroup's query rows
// of the normalised attention A_{i,j}; the selection kernel adds the row tiles and
// divides by T (the importance score of the attention-driven selection).
//
// Work decomposition
//   * A workgroup owns 256 query rows of one (layer, KV head).  Rows are the G
//     query heads sharing the KV head times the T frame tokens (grouped-query
//     packing: every row of the tile reads the same K/V).  4 waves x 64 rows.
//   * Keys stream through LDS in tiles of 64, double buffered; K row-major,
//     V transposed (V^T) so both MFMA operands are 16-byte LDS reads.
//   * Two sweeps over the keys.  Sweep 1: S^T = K Q^T -> per-row max and sum of
//     exp2.  Sweep 2: S^T again -> E^T = exp2(x - row max) -> O^T += V^T E^T
//     (scaled by 1/sum at the end) and per-key column sums of P = E / sum.
//     Exact probabilities are known only after the row statistics, and
//     recomputing K Q^T is cheaper than storing the logits.
//   * The blockIdx -> tile mapping keeps the row tiles of one (layer, KV head)
//     on one XCD so they share K/V in that XCD's L2.
//
// MFMA v_mfma_f32_32x32x16_bf16 (wave64) operand layout, lane l, h = l / 32:
//   A (32x16): A[l % 32][8h .. 8h+7]   B (16x32): B[8h .. 8h+7][l % 32]
//   C (32x32): element v (0..15) of lane l is C[8(v/4) + 4h + v%4][l % 32].
// With S^T = K Q^T (M = keys, N = query rows, K = head dim) the C registers of
// one lane hold 16 keys of one query row, so P^T can feed the B operand of
// O^T = V^T P^T directly: the 8 values v = 8s..8s+7 of lane l are keys
// 16s + {0..3, 8..11} (h = 0) or 16s + {4..7, 12..15} (h = 1).  V^T is stored
// in LDS with bits 2 and 3 of the key index swapped inside each 16-key group,
// which puts exactly those keys at consecutive addresses.
#include "internal.h"

namespace skv {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kQB = 2;         // 32-row blocks per wave
constexpr int kRowsWave = 64;  // kQB * 32
constexpr int kKT = 64;        // keys per LDS tile (two 32-key blocks)
constexpr int kPad = 8;        // bf16 padding per LDS row (16 bytes)
static_assert(kWaves * kRowsWave == kMfmaRowsPerTile, "tile rows");

template <int D>
struct Smem {
  uint16_t k[2][kKT][D + kPad];     // K rows
  uint16_t vt[2][D][kKT + kPad];    // V^T, key order permuted inside 16-key groups
  float cs[2][kWaves][kKT];         // per-wave column sums of the current tile
};

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }  // v_exp_f32
__device__ inline float fast_log2(float x) { return __builtin_amdgcn_logf(x); }   // v_log_f32

__device__ inline int vt_slot(int kk) {  // swap bits 2 and 3 of the key index
  return (kk & ~12) | ((kk & 4) << 1) | ((kk & 8) >> 1);
}

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

template <int D>
__global__ __launch_bounds__(256, 1) void attn_mfma_kernel(AttnArgs a) {
  constexpr int KS = D / 16;                       // k-steps of K Q^T
  constexpr int DB = D / 32;                       // 32-row blocks of O^T
  constexpr int KCH = D / 8;                       // 16-byte chunks per K/V row
  constexpr int K_ITEMS = kKT * KCH / 256;         // K chunks staged per thread
  constexpr int V_ITEMS = (kKT / 2) * KCH / 256;   // (key pair, chunk) units per thread
  static_assert(K_ITEMS * 256 == kKT * KCH && V_ITEMS * 256 == (kKT / 2) * KCH, "staging split");

  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  Smem<D>& sm = *reinterpret_cast<Smem<D>*>(smem_raw);

  // XCD-aware mapping: consecutive workgroup ids go round-robin over the 8 XCDs;
  // give each XCD a contiguous range of (layer, KV head, row tile) work items.
  const int n_work = a.n_layers * a.H_kv * a.n_qtiles;
  const int per_xcd = gridDim.x >> 3;
  const int wid = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (wid >= n_work) return;
  const int qt = wid % a.n_qtiles;
  const int lg = wid / a.n_qtiles;
  const int layer = lg / a.H_kv, g = lg % a.H_kv;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, h = lane >> 5;
  const int GT = a.G * a.T;
  const int S = a.S, n_keys = a.S + a.T;
  const int n_tiles = (n_keys + kKT - 1) / kKT;
  const int row0 = qt * kMfmaRowsPerTile + wave * kRowsWave;
  const bool wave_active = row0 < GT;
  const float c = a.scale_log2;

  const uint16_t* qg = static_cast<const uint16_t*>(a.q) + static_cast<size_t>(layer * a.H_q + g * a.G) * a.T * D;
  const uint16_t* kst = static_cast<const uint16_t*>(a.ks) + static_cast<size_t>(lg) * a.B * D;
  const uint16_t* vst = static_cast<const uint16_t*>(a.vs) + static_cast<size_t>(lg) * a.B * D;
  const uint16_t* kfr = static_cast<const uint16_t*>(a.kf) + static_cast<size_t>(lg) * a.T * D;
  const uint16_t* vfr = static_cast<const uint16_t*>(a.vf) + static_cast<size_t>(lg) * a.T * D;

  // Q^T operand (B of K Q^T) in registers; invalid rows are zero.
  bf16x8 qreg[kQB][KS];
  int lim[kQB];  // candidate j is visible to the row iff j <= lim (state keys, then causal frame)
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    const int r = row0 + qb * 32 + l32;
    const bool valid = r < GT;
    lim[qb] = valid ? S + (r % a.T) : -1;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (valid) x = *reinterpret_cast<const u32x4*>(qg + static_cast<size_t>(r) * D + ks * 16 + h * 8);
      qreg[qb][ks] = __builtin_bit_cast(bf16x8, x);
    }
  }

  auto row_ptr = [&](const uint16_t* st, const uint16_t* fr, int j) -> const uint16_t* {
    return j < S ? st + static_cast<size_t>(j) * D : fr + static_cast<size_t>(j - S) * D;
  };

  u32x4 kpre[K_ITEMS];
  u32x4 vpre[V_ITEMS][2];
  auto load_k = [&](int t) {
#pragma unroll
    for (int it = 0; it < K_ITEMS; ++it) {
      const int idx = it * 256 + tid;
      const int kk = idx / KCH, ch = idx % KCH;
      const int j = t * kKT + kk;
      u32x4 x = {0u, 0u, 0u, 0u};
      if (j < n_keys) x = *reinterpret_cast<const u32x4*>(row_ptr(kst, kfr, j) + ch * 8);
      kpre[it] = x;
    }
  };
  auto store_k = [&](int b) {
#pragma unroll
    for (int it = 0; it < K_ITEMS; ++it) {
      const int idx = it * 256 + tid;
      const int kk = idx / KCH, ch = idx % KCH;
      *reinterpret_cast<u32x4*>(&sm.k[b][kk][ch * 8]) = kpre[it];
    }
  };
  auto load_v = [&](int t) {
#pragma unroll
    for (int it = 0; it < V_ITEMS; ++it) {
      const int idx = it * 256 + tid;
      const int p = idx % (kKT / 2), ch = idx / (kKT / 2);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int j = t * kKT + 2 * p + e;
        u32x4 x = {0u, 0u, 0u, 0u};
        if (j < n_keys) x = *reinterpret_cast<const u32x4*>(row_ptr(vst, vfr, j) + ch * 8);
        vpre[it][e] = x;
      }
    }
  };
  auto store_v = [&](int b) {
#pragma unroll
    for (int it = 0; it < V_ITEMS; ++it) {
      const int idx = it * 256 + tid;
      const int p = idx % (kKT / 2), ch = idx / (kKT / 2);
      const int col = vt_slot(2 * p);  // even; key 2p+1 lands at col + 1
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const unsigned x0 = vpre[it][0][w], x1 = vpre[it][1][w];
        // element 2w and 2w+1 of the chunk: pair (key 2p, key 2p+1) per d
        const unsigned lo = (x0 & 0xFFFFu) | (x1 << 16);
        const unsigned hi = (x0 >> 16) | (x1 & 0xFFFF0000u);
        *reinterpret_cast<unsigned*>(&sm.vt[b][ch * 8 + 2 * w][col]) = lo;
        *reinterpret_cast<unsigned*>(&sm.vt[b][ch * 8 + 2 * w + 1][col]) = hi;
      }
    }
  };

  // S^T block (32 keys x 32 rows) for key block kb of the tile in buffer b.
  auto qk_block = [&](int b, int kb, f32x16 (&acc)[kQB]) {
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) acc[qb] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const u32x4 x = *reinterpret_cast<const u32x4*>(&sm.k[b][kb * 32 + l32][ks * 16 + h * 8]);
      const bf16x8 av = __builtin_bit_cast(bf16x8, x);
#pragma unroll
      for (int qb = 0; qb < kQB; ++qb)
        acc[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qreg[qb][ks], acc[qb], 0, 0, 0);
    }
  };

  // ---------------- sweep 1: row statistics ----------------
  float m[kQB], l[kQB];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) { m[qb] = -1e30f; l[qb] = 0.f; }

  load_k(0);
  store_k(0);
  __syncthreads();
  for (int t = 0; t < n_tiles; ++t) {
    const int b = t & 1;
    const bool more = t + 1 < n_tiles;
    if (more) load_k(t + 1);
    if (wave_active) {
      const bool masked = t * kKT + kKT > S;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 acc[kQB];
        qk_block(b, kb, acc);
        const int jb = t * kKT + kb * 32 + 4 * h;
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb) {
          float z[16];
#pragma unroll
          for (int v = 0; v < 16; ++v) z[v] = acc[qb][v];
          if (masked) {
            const int rel = lim[qb] - jb;
#pragma unroll
            for (int v = 0; v < 16; ++v)
              if (8 * (v >> 2) + (v & 3) > rel) z[v] = -__builtin_huge_valf();
          }
          float mx = z[0];
#pragma unroll
          for (int v = 1; v < 16; ++v) mx = fmaxf(mx, z[v]);
          const float mn = fmaxf(m[qb], mx);
          const float mc = mn * c;
          float sum = 0.f;
#pragma unroll
          for (int v = 0; v < 16; ++v) sum += fast_exp2(fmaf(z[v], c, -mc));
          // Subtract before scaling: equal maxima (including the empty-row sentinel)
          // give exactly exp2(0) = 1.
          l[qb] = l[qb] * fast_exp2((m[qb] - mn) * c) + sum;
          m[qb] = mn;
        }
      }
    }
    if (more) store_k(b ^ 1);
    __syncthreads();
  }
  // Row maximum (log2 units) and 1/sum.  Sweep 2 feeds the PV MFMA with
  // E = exp2(x - max) <= 1, whose largest entry is exactly 1 in bf16, and applies
  // 1/sum in fp32 to the output; the column sums use P = E / sum in fp32.
  float mrow[kQB], inv_l[kQB];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    // the other 16 keys of every 32-key block live in lane ^ 32
    const float mo = __shfl_xor(m[qb], 32, 64);
    const float lo = __shfl_xor(l[qb], 32, 64);
    const float mm = fmaxf(m[qb], mo);
    const float ll = l[qb] * fast_exp2((m[qb] - mm) * c) + lo * fast_exp2((mo - mm) * c);
    const bool valid = lim[qb] >= 0;
    mrow[qb] = valid ? mm * c : 0.f;
    inv_l[qb] = valid ? 1.0f / ll : 0.f;
  }

  // ---------------- sweep 2: P, O and column sums ----------------
  f32x16 o[kQB][DB];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
    for (int db = 0; db < DB; ++db) o[qb][db] = f32x16{};

  float* part = a.partial + (static_cast<size_t>(lg) * a.n_qtiles + qt) * a.pool_stride;
  const int key_lane = 8 * (((lane >> 3) & 1) + 2 * ((lane >> 4) & 1)) + 4 * h + (((lane >> 1) & 1) + 2 * ((lane >> 2) & 1));

  load_k(0);
  load_v(0);
  store_k(0);
  store_v(0);
  __syncthreads();
  for (int t = 0; t < n_tiles; ++t) {
    const int b = t & 1;
    const bool more = t + 1 < n_tiles;
    if (more) {
      load_k(t + 1);
      load_v(t + 1);
    }
    if (wave_active) {
      const bool masked = t * kKT + kKT > S;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 acc[kQB];
        qk_block(b, kb, acc);
        const int jb = t * kKT + kb * 32 + 4 * h;
        float p[kQB][16];  // E = exp2(x - row max), masked entries 0
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb) {
          const int rel = lim[qb] - jb;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            float x = fast_exp2(fmaf(acc[qb][v], c, -mrow[qb]));
            if (masked && 8 * (v >> 2) + (v & 3) > rel) x = 0.f;
            p[qb][v] = x;
          }
        }
        float cs[16];  // P = E / sum, added over the lane's two rows
#pragma unroll
        for (int v = 0; v < 16; ++v) cs[v] = fmaf(p[0][v], inv_l[0], p[1][v] * inv_l[1]);
        bf16x8 pb[kQB][2];
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
          for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int i = 0; i < 8; ++i) pb[qb][s][i] = static_cast<__bf16>(p[qb][8 * s + i]);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
#pragma unroll
          for (int s = 0; s < 2; ++s) {
            const u32x4 x = *reinterpret_cast<const u32x4*>(&sm.vt[b][db * 32 + l32][kb * 32 + s * 16 + h * 8]);
            const bf16x8 av = __builtin_bit_cast(bf16x8, x);
#pragma unroll
            for (int qb = 0; qb < kQB; ++qb)
              o[qb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb[qb][s], o[qb][db], 0, 0, 0);
          }
        }
        const float tot = column_reduce(cs, lane);
        if ((lane & 1) == 0) sm.cs[b][wave][kb * 32 + key_lane] = tot;
      }
    } else {
      sm.cs[b][wave][lane] = 0.f;
    }
    if (more) {
      store_k(b ^ 1);
      store_v(b ^ 1);
    }
    __syncthreads();
    if (tid < kKT) {
      const int j = t * kKT + tid;
      if (j < n_keys) part[j] = (sm.cs[b][0][tid] + sm.cs[b][1][tid]) + (sm.cs[b][2][tid] + sm.cs[b][3][tid]);
    }
  }

  // ---------------- output ----------------
  if (wave_active) {
    uint16_t* og = static_cast<uint16_t*>(a.out) + static_cast<size_t>(layer * a.H_q + g * a.G) * a.T * D;
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
      const int r = row0 + qb * 32 + l32;
      if (r >= GT) continue;
      uint16_t* orow = og + static_cast<size_t>(r) * D;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) {
          __bf16 w[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) w[u] = static_cast<__bf16>(o[qb][db][vq * 4 + u] * inv_l[qb]);
          uint2 packed;
          packed.x = static_cast<unsigned>(__builtin_bit_cast(uint16_t, w[0])) |
                     (static_cast<unsigned>(__builtin_bit_cast(uint16_t, w[1])) << 16);
          packed.y = static_cast<unsigned>(__builtin_bit_cast(uint16_t, w[2])) |
                     (static_cast<unsigned>(__builtin_bit_cast(uint16_t, w[3])) << 16);
          *reinterpret_cast<uint2*>(orow + db * 32 + vq * 8 + 4 * h) = packed;
        }
      }
    }
  }
}

hipError_t launch_attention_mfma_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
  const int n_work = a.n_layers * a.H_kv * a.n_qtiles;
  const int grid = ((n_work + 7) / 8) * 8;
  if (head_dim == 128) {
    hipLaunchKernelGGL(attn_mfma_kernel<128>, dim3(grid), dim3(256), sizeof(Smem<128>), s, a);
  } else {
    hipLaunchKernelGGL(attn_mfma_kernel<64>, dim3(grid), dim3(256), sizeof(Smem<64>), s, a);
  }
  return hipGetLastError();
}

hipError_t prepare_attention_mfma() {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(attn_mfma_kernel<128>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, sizeof(Smem<128>));
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(attn_mfma_kernel<64>),
                             hipFuncAttributeMaxDynamicSharedMemorySize, sizeof(Smem<64>));
}

}  // namespace skv
