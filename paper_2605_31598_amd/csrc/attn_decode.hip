// Decoding over the detailed cache D (the decoding paragraph of the method: the
// answer is decoded from D, not from the compressed state), bf16 MFMA, gfx950.
//
// t new tokens per call attend to every video token of D, every token decoded
// before, and the new tokens up to themselves (causal).  The cost is one read
// of D per call (5.8 GB for the 7B-shaped stack after 512 frames), so the
// kernel is built to stream HBM: split-key flash decoding.
//   * decode_split_kernel: each wave owns one item = (layer-head, 32-row block
//     of the G t query rows, contiguous key split) and needs nothing from the
//     other waves, so there are no barriers.  K rows go straight from global
//     memory into the A operand of S^T = K Q^T (lane l reads key l % 32), V rows
//     are staged in the wave's own LDS tile for the transpose reads of
//     O^T = V^T P^T (the operand arrangement of the streaming full-attention
//     kernel), and the next block's K/V loads are issued before the current
//     block's MFMAs.  Online softmax per query row (one row per lane pair);
//     the split's unnormalised output, row maximum and row sum go to
//     partial buffers.
//   * decode_combine_kernel: per (layer-head, row block) merges the splits of
//     each row, O = sum_s O_s 2^{(m_s - m) c} / sum_s l_s 2^{(m_s - m) c}.
#include "internal.h"

namespace skv {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kDecWaves = 4;                  // independent waves per workgroup
constexpr int kDecThreads = kDecWaves * 64;
// V row padding (bf16).  ds_read_b64_tr_b16 serves 32 lanes (four rows x 64 B) per
// LDS pass over 64 four-byte banks; a row stride of 80 (D = 128) or 48 (D = 64)
// dwords, modulo 64, puts those four rows on disjoint banks.  A 16-element pad
// (72 dwords) overlaps them two-way.
constexpr int kPadV = 32;

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }  // v_exp_f32

}  // namespace

template <int D>
__global__ __launch_bounds__(kDecThreads, 2) void decode_split_kernel(DecodeArgs a) {
  constexpr int KS = D / 16;   // k-steps of K Q^T
  constexpr int DB = D / 32;   // 32-dimension blocks of O^T
  constexpr int KCH = D / 8;   // 16-byte chunks per row
  constexpr int VIT = 32 * KCH / 64;  // V chunks of one 32-key block per lane
  __shared__ __attribute__((aligned(16))) uint16_t vt[kDecWaves][32][D + kPadV];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l32 = lane & 31, h = lane >> 5;
  const int LH = a.n_layers * a.H_kv;
  const int n_items = LH * a.n_rb * a.n_split;
  const int item = blockIdx.x * kDecWaves + wave;
  if (item >= n_items) return;  // whole wave; the kernel has no barriers
  const int sp = item % a.n_split;
  const int rb = (item / a.n_split) % a.n_rb;
  const int lg = item / (a.n_split * a.n_rb);
  const int layer = lg / a.H_kv, g = lg % a.H_kv;
  const int GT = a.G * a.t;
  const float c = a.scale_log2;

  const int n_keys = a.S + a.n_dec + a.t;
  const int j0 = sp * a.split;
  const int j1 = min(n_keys, j0 + a.split);

  const int r = rb * 32 + l32;  // packed query row (head-in-group major, token minor)
  const bool row_valid = r < GT;
  const int lim = row_valid ? a.S + a.n_dec + (r % a.t) : -1;  // key j is visible iff j <= lim

  const uint16_t* cache_k = static_cast<const uint16_t*>(a.ck) + static_cast<size_t>(lg) * a.max_tokens * D;
  const uint16_t* cache_v = static_cast<const uint16_t*>(a.cv) + static_cast<size_t>(lg) * a.max_tokens * D;
  const uint16_t* new_k = static_cast<const uint16_t*>(a.kn) + static_cast<size_t>(lg) * a.t * D;
  const uint16_t* new_v = static_cast<const uint16_t*>(a.vn) + static_cast<size_t>(lg) * a.t * D;
  // row j of the key sequence: video tokens, earlier decoded tokens, then the new tokens
  auto krow = [&](const uint16_t* cache, const uint16_t* fresh, int j) -> const uint16_t* {
    if (j < a.S) return cache + static_cast<size_t>(j) * D;
    if (j < a.S + a.n_dec) return cache + static_cast<size_t>(a.dec_row0 + (j - a.S)) * D;
    return fresh + static_cast<size_t>(j - a.S - a.n_dec) * D;
  };

  const uint16_t* qg = static_cast<const uint16_t*>(a.q) + static_cast<size_t>(layer * a.H_q + g * a.G) * a.t * D;
  bf16x8 qreg[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    u32x4 x = {0u, 0u, 0u, 0u};
    if (row_valid) x = *reinterpret_cast<const u32x4*>(qg + static_cast<size_t>(r) * D + ks * 16 + h * 8);
    qreg[ks] = __builtin_bit_cast(bf16x8, x);
  }
  if (a.rope_tab != nullptr && row_valid) {  // RoPE at the decoded token's virtual position
    const float* tb = a.rope_tab + static_cast<size_t>(a.rope_pos0 + r % a.t) * D;
#pragma unroll
    for (int ks = 0; ks < KS / 2; ++ks) {
      const u32x4 lo = __builtin_bit_cast(u32x4, qreg[ks]), hi = __builtin_bit_cast(u32x4, qreg[ks + KS / 2]);
      qreg[ks] = __builtin_bit_cast(bf16x8, rope_chunk_bf16(lo, hi, false, ks * 16 + h * 8, tb));
      qreg[ks + KS / 2] = __builtin_bit_cast(bf16x8, rope_chunk_bf16(hi, lo, true, ks * 16 + h * 8, tb));
    }
  }

  // global -> registers for one 32-key block starting at key kb
  u32x4 kreg[KS], vreg[VIT];
  auto load_k = [&](int kb) {
    const int jk = kb + l32;
    const bool kin = jk < j1;
    const uint16_t* kr = kin ? krow(cache_k, new_k, jk) : nullptr;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (kin) x = *reinterpret_cast<const u32x4*>(kr + ks * 16 + h * 8);
      kreg[ks] = x;
    }
  };
  auto load_v = [&](int kb) {
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int idx = it * 64 + lane;
      const int row = idx / KCH, ch = idx % KCH;
      const int jv = kb + row;
      u32x4 y = {0u, 0u, 0u, 0u};
      if (jv < j1) y = *reinterpret_cast<const u32x4*>(krow(cache_v, new_v, jv) + ch * 8);
      vreg[it] = y;
    }
  };

  const int tr_row = 4 * h + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  f32x16 ot[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) ot[db] = f32x16{};
  float m = -1e30f, l = 0.f;

  load_k(j0);
  load_v(j0);
  for (int kb = j0; kb < j1; kb += 32) {
    // V of this block into the wave's LDS tile (this wave's earlier transpose
    // reads of the tile are ahead of these writes in its LDS queue), then the
    // next block's V loads into the freed registers
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int idx = it * 64 + lane;
      const int row = idx / KCH, ch = idx % KCH;
      *reinterpret_cast<u32x4*>(&vt[wave][row][ch * 8]) = vreg[it];
    }
    const bool more = kb + 32 < j1;
    if (more) load_v(kb + 32);
    f32x16 acc = {};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kreg[ks]), qreg[ks], acc, 0, 0, 0);
    if (more) load_k(kb + 32);  // the MFMAs above have read this block's K operands
    float z[16];
    const int rel = lim - (kb + 4 * h);  // key kb + 8(v/4) + 4h + v%4 is visible iff 8(v/4) + v%4 <= rel
    const int end = j1 - (kb + 4 * h);   // ... and exists iff 8(v/4) + v%4 < end
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int o = 8 * (v >> 2) + (v & 3);
      z[v] = (o <= rel && o < end) ? acc[v] : -__builtin_huge_valf();
    }
    float bm = z[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) bm = fmaxf(bm, z[v]);
    bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
    const bool grow = bm > m;
    if (__ballot(grow)) {
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
      const float e = fast_exp2(fmaf(z[v], c, -mc));
      l += e;
      pe[v >> 3][v & 7] = static_cast<__bf16>(e);
    }
    bf16x8 vop[2][DB];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int rr = s * 16 + tr_row;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(&vt[wave][rr][db * 32 + tr_col]));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(&vt[wave][rr + 8][db * 32 + tr_col]));
        vop[s][db] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
    }
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int db = 0; db < DB; ++db) ot[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[s][db], pe[s], ot[db], 0, 0, 0);
  }

  // partials of this split: unnormalised O (row-major [32][D]), row maximum, row sum
  const float lt = l + __shfl_xor(l, 32, 64);
  float* po = a.part_o + static_cast<size_t>(item) * 32 * D + static_cast<size_t>(l32) * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const f32x4 w = {ot[db][4 * q4], ot[db][4 * q4 + 1], ot[db][4 * q4 + 2], ot[db][4 * q4 + 3]};
      *reinterpret_cast<f32x4*>(po + db * 32 + 8 * q4 + 4 * h) = w;
    }
  if (h == 0) {
    a.part_ml[static_cast<size_t>(item) * 64 + l32] = m;
    a.part_ml[static_cast<size_t>(item) * 64 + 32 + l32] = lt;
  }
}

template <int D>
__global__ __launch_bounds__(256) void decode_combine_kernel(DecodeArgs a) {
  constexpr int DPT = D / 8;  // dimensions per thread: 8 threads per row
  const int blk = blockIdx.x;  // (layer-head, row block)
  const int lg = blk / a.n_rb, rb = blk % a.n_rb;
  const int layer = lg / a.H_kv, g = lg % a.H_kv;
  const int row = threadIdx.x >> 3, dq = threadIdx.x & 7;
  const int r = rb * 32 + row;
  if (r >= a.G * a.t) return;  // no barriers below
  const size_t item0 = static_cast<size_t>(blk) * a.n_split;
  const float c = a.scale_log2;
  const float* ml = a.part_ml + item0 * 64 + row;
  float mx = -1e30f;
#pragma unroll 4
  for (int sp = 0; sp < a.n_split; ++sp) mx = fmaxf(mx, ml[static_cast<size_t>(sp) * 64]);
  float acc[DPT];
#pragma unroll
  for (int i = 0; i < DPT; ++i) acc[i] = 0.f;
  float lsum = 0.f;
#pragma unroll 4
  for (int sp = 0; sp < a.n_split; ++sp) {
    const float w = fast_exp2((ml[static_cast<size_t>(sp) * 64] - mx) * c);
    lsum += ml[static_cast<size_t>(sp) * 64 + 32] * w;
    const float* po = a.part_o + (item0 + sp) * 32 * D + static_cast<size_t>(row) * D + dq * DPT;
#pragma unroll
    for (int i = 0; i < DPT; i += 4) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(po + i);
      acc[i] += x[0] * w;
      acc[i + 1] += x[1] * w;
      acc[i + 2] += x[2] * w;
      acc[i + 3] += x[3] * w;
    }
  }
  const float inv = 1.0f / lsum;
  uint16_t* og = static_cast<uint16_t*>(a.out) + (static_cast<size_t>(layer * a.H_q + g * a.G) * a.t + r) * D + dq * DPT;
#pragma unroll
  for (int i = 0; i < DPT; i += 8) {
    u32x4 w;
#pragma unroll
    for (int k = 0; k < 4; ++k)
      w[k] = static_cast<unsigned>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(acc[i + 2 * k] * inv))) |
             (static_cast<unsigned>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(acc[i + 2 * k + 1] * inv))) << 16);
    *reinterpret_cast<u32x4*>(og + i) = w;
  }
}

hipError_t launch_decode_bf16(const DecodeArgs& a, int head_dim, hipStream_t s) {
  const int n_items = a.n_layers * a.H_kv * a.n_rb * a.n_split;
  const int grid = (n_items + kDecWaves - 1) / kDecWaves;
  const int n_blk = a.n_layers * a.H_kv * a.n_rb;
  if (head_dim == 128) {
    hipLaunchKernelGGL(decode_split_kernel<128>, dim3(grid), dim3(kDecThreads), 0, s, a);
    hipLaunchKernelGGL(decode_combine_kernel<128>, dim3(n_blk), dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL(decode_split_kernel<64>, dim3(grid), dim3(kDecThreads), 0, s, a);
    hipLaunchKernelGGL(decode_combine_kernel<64>, dim3(n_blk), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace skv
