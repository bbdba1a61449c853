// bf16 MFMA attention with fused importance scoring, gfx950 (CDNA4).
//
// Computes, for one frame and a range of layers, Eq. 5
//     O = softmax(Q [K_state; K_frame]^T * scale + M_n) [V_state; V_frame]
// and, for every candidate key j, the column sum over the workgroup's query rows
// of the normalised attention A_{i,j}; the selection kernel adds the row tiles and
// divides by T (the importance score of the attention-driven selection).
//
// Work decomposition
//   * A workgroup owns up to 256 query rows of one (layer, KV head): 8 waves x
//     32 rows, two waves per SIMD.  Rows are the G query heads sharing the KV
//     head times the T frame tokens (grouped-query packing: every row of the tile
//     reads the same K/V).  Two waves per SIMD let the hardware run one wave's
//     exp/softmax VALU work under the other wave's MFMAs.
//   * A split workgroup (the short shares the host plan puts in the grid's last
//     round) owns at most 128 rows; waves w and w + 4 take the same 32 rows and
//     the first and the second half of every key tile, combine their row
//     statistics after sweep 1 and their outputs at the end, so the last round
//     also runs two waves per SIMD.
//   * Keys stream through LDS in tiles of 128 (four 32-key blocks), double
//     buffered, K and V both row-major with padded rows.  The load unit copies
//     the next tile global -> LDS (global_load_lds) while the current one is
//     computed, with no registers or LDS store instructions; those copies are
//     issued by the first wave of each SIMD (waves 0-3), whose partner sets the
//     tile's pace, and a range's first tile by all eight.  Operand reads from
//     LDS are issued ahead as inline assembly with explicit waits, and waves
//     raise their priority while issuing MFMAs.
//   * Sweep 2 is software-pipelined over the blocks of a tile: block kb + 1's
//     K Q^T MFMAs are issued interleaved with block kb's exponentials and block
//     kb's PV MFMAs with its column sums (sched_group_barrier), so a wave's VALU
//     work issues between its own dependent MFMAs instead of after them.
//   * Two sweeps over the keys.  Sweep 1: S^T = K Q^T -> per-row max and sum of
//     exp2.  Sweep 2: S^T again -> E = exp2(x - row max) -> O += E V (scaled by
//     1/sum at the end) and per-key column sums of P = E / sum.  Exact
//     probabilities are known only after the row statistics, and recomputing
//     K Q^T is cheaper than storing the logits.
//   * Tiles that contain frame keys (the only ones with masked entries) run in a
//     separate loop, keeping mask code off the common path; there a wave skips the
//     32-key blocks that lie wholly past the causal limit of all its rows.  Tiles
//     wholly inside the state are copied without the per-row clamping to the
//     last key.
//   * The host plan keeps the row tiles of one (layer, KV head) on one XCD so
//     they share K/V in that XCD's L2.
//   * Calls too small to fill the device split the keys into ranges (key-split
//     plans).  The statistics of all ranges of a row range are merged before
//     sweep 2: across two launches (modes 1, 2) or in one (modes 3, 4), whose
//     workgroups publish their ranges' statistics and wait a bounded time for
//     each other's (device-scope stores and flags), computing any range that
//     has not arrived.  Sweep 2 then writes the range's exact column sums and its
//     fp32 share of O; the refresh launch adds the shares.
//   * Instantiations: VAR 0 for everything but key-split output work; VAR 1 for
//     a two-launch output launch and VAR 2 for the one-launch key split, which
//     can also carry an earlier one-layer call's selection and state update
//     (select.h) in extra workgroups after the plan's items.
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
#include "select.h"

#include <type_traits>
#include <utility>

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
// V row padding (bf16).  ds_read_b64_tr_b16 serves 32 lanes (four rows x 64 B) per
// LDS pass over 64 four-byte banks; a row stride of 80 (D = 128) or 48 (D = 64)
// dwords, modulo 64, puts those four rows on disjoint banks.  A 16-element pad
// (72 dwords) overlaps them two-way.
constexpr int kPadV = 32;
constexpr int kPadO = 8;       // output staging row padding (bf16)

template <int D>
struct Smem {
  uint16_t k[2][kKT][D + kPadK];
  uint16_t v[2][kKT][D + kPadV];
  float cs[2][kWaves][kKT];     // per-wave column sums of one tile
  float il[kWaves][kRowsWave];  // 1 / row sum, for the output
};
static_assert(sizeof(Smem<128>) <= 160 * 1024, "gfx950 LDS per workgroup");

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }  // v_exp_f32

template <int CTRL>
__device__ inline float dpp_f(float x) {
  // DPP lane permutation inside rows of 16 lanes (all rows and banks enabled).
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}

template <typename F, int... I>
__device__ inline void static_for_impl(F& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
// f(std::integral_constant<int, i>) for i = 0 .. N-1, unrolled with constant i
template <int N, typename F>
__device__ inline void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// ds_read_b64_tr_b16 at LDS byte address addr + OFF, issued as inline assembly:
// the compiler then does not order it behind the outstanding global -> LDS copies
// of the next tile (it cannot tell the two buffers apart).  The caller waits for
// the result with lgkm_wait before use.
template <int OFF>
__device__ inline s16x4 ds_read_tr(uint32_t addr) {
  s16x4 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}
template <int OFF>
__device__ inline u32x4 ds_read_b128(uint32_t addr) {
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}
// s_waitcnt lgkmcnt(N), ordered before every use of x
template <int N, typename T>
__device__ inline void lgkm_wait(T& x) {
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(x) : "i"(N));
}

// Weighted sum of e[16] over the 32 lanes that share h = lane / 32 (the query
// rows of one half-block), each lane's values scaled by its row's weight.
// Returns, in every lane, the total of the key
//   key(lane) = 8 * (b3 + 2 * b4) + 4 * h + (b1 + 2 * b2)     (bN = bit N of lane)
// within the 32-key block; lanes differing only in bit 0 return the same key.
// Reduce-scatter: each step halves the values a lane carries while pairing
// lanes that differ in one more row bit (partners l ^ 16, l ^ 8, l ^ 4, l ^ 3,
// l ^ 1: the same pairing of rows for every key, so equal columns give equal
// sums).  The first step applies the weights: w0 and w1 are the weights of the
// first and the second value the swap leaves in this lane (own and partner row for
// b4 = 0, partner and own row for b4 = 1).
__device__ inline float column_reduce(const float (&e)[16], int lane, float w0, float w1) {
  float c1[8];
#pragma unroll
  for (int v = 0; v < 8; ++v) {  // rows 0<->1 and 2<->3: lanes l and l^16
    const auto pr = __builtin_amdgcn_permlane16_swap(__float_as_uint(e[v]), __float_as_uint(e[v + 8]),
                                                     false, false);
    c1[v] = fmaf(__uint_as_float(pr[0]), w0, __uint_as_float(pr[1]) * w1);
  }
  // Lanes i <-> i ^ 8, then i <-> i ^ 4, inside each row of 16 lanes.  A lane keeps
  // one of its two values by bit 3 (then bit 2) of its index, and the bank masks of
  // the DPP adds pick the lanes: lanes 0-7 of a row (banks 0, 1) add their partner's
  // first value to their own, lanes 8-15 (banks 2, 3) the second; then banks 0, 2
  // (bit 2 clear) and 1, 3 (bit 2 set).  Two adds per pair, no selects.  The leading
  // s_nop covers the VALU-write to DPP-read hazard on c1; inside the block every
  // DPP source was written at least two instructions earlier.
  const bool b1 = lane & 2;
  float c2[4], c3[2];
  asm("s_nop 1\n"
      "v_add_f32_dpp %0, %6, %6 row_ror:8 row_mask:0xf bank_mask:0x3\n"
      "v_add_f32_dpp %1, %7, %7 row_ror:8 row_mask:0xf bank_mask:0x3\n"
      "v_add_f32_dpp %2, %8, %8 row_ror:8 row_mask:0xf bank_mask:0x3\n"
      "v_add_f32_dpp %3, %9, %9 row_ror:8 row_mask:0xf bank_mask:0x3\n"
      "v_add_f32_dpp %0, %10, %10 row_ror:8 row_mask:0xf bank_mask:0xc\n"
      "v_add_f32_dpp %1, %11, %11 row_ror:8 row_mask:0xf bank_mask:0xc\n"
      "v_add_f32_dpp %2, %12, %12 row_ror:8 row_mask:0xf bank_mask:0xc\n"
      "v_add_f32_dpp %3, %13, %13 row_ror:8 row_mask:0xf bank_mask:0xc\n"
      "v_add_f32_dpp %4, %0, %0 row_shl:4 row_mask:0xf bank_mask:0x5\n"
      "v_add_f32_dpp %5, %1, %1 row_shl:4 row_mask:0xf bank_mask:0x5\n"
      "v_add_f32_dpp %4, %2, %2 row_shr:4 row_mask:0xf bank_mask:0xa\n"
      "v_add_f32_dpp %5, %3, %3 row_shr:4 row_mask:0xf bank_mask:0xa"
      : "=&v"(c2[0]), "=&v"(c2[1]), "=&v"(c2[2]), "=&v"(c2[3]), "=&v"(c3[0]), "=&v"(c3[1])
      : "v"(c1[0]), "v"(c1[1]), "v"(c1[2]), "v"(c1[3]), "v"(c1[4]), "v"(c1[5]), "v"(c1[6]), "v"(c1[7]));
  const float keep = b1 ? c3[1] : c3[0];  // lanes i <-> 3-i inside a quad (bit 1 differs)
  const float send = b1 ? c3[0] : c3[1];
  const float c4 = keep + dpp_f<0x1B>(send);
  return c4 + dpp_f<0xB1>(c4);  // lanes i <-> i^1
}

}  // namespace

// ROPE: rotate Q at the frame tokens' virtual positions (a separate
// instantiation, so the kernel without rotation carries none of its code).  The
// frame's keys arrive rotated (rope_keys.hip), like the state's and the cache's.
template <int D, bool ROPE, int VAR>
__global__ __launch_bounds__(kThreads, 1) void attn_mfma_kernel(AttnArgs a) {
  constexpr int KS = D / 16;                   // k-steps of K Q^T
  constexpr int DB = D / 32;                   // 32-column blocks of O
  constexpr int KCH = D / 8;                   // 16-byte chunks per K/V row

  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  Smem<D>& sm = *reinterpret_cast<Smem<D>*>(smem_raw);

  // Workgroups past the plan's items carry the selection of an earlier
  // one-layer call (instantiations of their own for the launches that can carry
  // one; the host checks that its pool fits this workgroup's LDS).
  if constexpr (VAR != 0) {
    if (static_cast<int>(blockIdx.x) >= a.n_work) {
      refresh_state(a.sel, static_cast<int>(blockIdx.x) - a.n_work, *reinterpret_cast<SelectShared*>(smem_raw),
                    reinterpret_cast<uint32_t*>(smem_raw + select_lds_bytes(0)));
      return;
    }
  }

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
  // key tiles of this work item: all, or its share [kt0, kt1) of a key-split plan
  const int ks = wk.ks;
  auto range_lo = [&](int r) { return static_cast<int>(static_cast<int64_t>(r) * n_tiles / a.n_ks); };
  int kt0 = range_lo(ks), kt1 = range_lo(ks + 1);  // reassigned only by a fused key split's fallback
  const int row_end = wk.row0 + wk.rows;  // rows of this workgroup: [wk.row0, row_end)
  // split workgroup: waves w and w + 4 take the same 32 rows, the first and the
  // second half of every key tile
  const bool split = wk.split != 0;
  const int grp = split ? (wave >> 2) : 0;
  const int rb = split ? (wave & 3) : wave;  // 32-row block of the workgroup
  const int key0 = grp * (kKT / 2);          // first key of this wave's share of a tile
  const int row0 = wk.row0 + rb * kRowsWave;
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
  // The wave's largest limit (a scalar): in tiles with frame keys, the 32-key blocks
  // past it are masked for every row of the wave and are skipped.
  int wlim = lim;
#pragma unroll
  for (int off = 16; off > 0; off >>= 1) wlim = max(wlim, __shfl_xor(wlim, off, 64));
  wlim = __builtin_amdgcn_readfirstlane(wlim);
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

  // ---------------- staging (global -> LDS by the load unit) ----------------
  // global_load_lds_dwordx4: lane i of one instruction writes its 16 bytes at
  // LDS base + 16 i, so one instruction fills 64 consecutive 16-byte slots of the
  // padded tile.  A slot that falls on a row's padding re-loads chunk 0 of its
  // row (padding is never read).  Keys past the end re-load the last key (finite
  // input data; those keys are masked).
  constexpr int KROW = (D + kPadK) / 8, VROW = (D + kPadV) / 8;  // 16-byte slots per padded row
  constexpr int KINS = kKT * KROW / 64, VINS = kKT * VROW / 64;  // instructions per tile
  static_assert(KINS * 64 == kKT * KROW && VINS * 64 == kKT * VROW, "whole instructions per tile");
  // The copies of the next tile, issued while the current one is computed, come
  // from waves 0-3 only: waves w and w + 4 of a workgroup share a SIMD, and the
  // younger one (w + 4) finishes a tile last; copy instructions issued at a
  // tile's start hold a wave until the load unit takes them, so they go to the
  // wave of each pair that would otherwise wait at the tile barrier.  A copy the
  // whole workgroup waits for (a range's first tile) is shared by all eight
  // waves: waves 4-7 take every second instruction of waves 0-3's schedule.
  constexpr int kDW = kWaves / 2;
  constexpr int KIT = (KINS + kDW - 1) / kDW, VIT = (VINS + kDW - 1) / kDW;
  const bool upper = wave >= kDW;
  const int dw = wave & (kDW - 1);  // position in the schedule of waves 0-3
  // element offset of slot q of a tile (rows of D), computed at the copy
  auto slot_off = [&](int q, auto rowc) -> int {
    constexpr int ROW = decltype(rowc)::value;
    const int ch = q % ROW;
    return (q / ROW) * D + (ch < KCH ? ch : 0) * 8;
  };
  auto koff_at = [&](int it) { return slot_off((it * kDW + dw) * 64 + lane, std::integral_constant<int, KROW>{}); };
  auto voff_at = [&](int it) { return slot_off((it * kDW + dw) * 64 + lane, std::integral_constant<int, VROW>{}); };
  auto dma_one = [&](const uint16_t* src, uint16_t* dst_tile, int ins) {
    __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)src,
                                     (void __attribute__((address_space(3)))*)(reinterpret_cast<char*>(dst_tile) + ins * 1024),
                                     16, 0, 0);
  };
  // source of a key row (any key index; clamped to the last key)
  auto key_src = [&](const uint16_t* st, const uint16_t* fr, int j) -> const uint16_t* {
    j = j < n_keys ? j : n_keys - 1;
    return j < S ? st + static_cast<size_t>(j) * D : fr + static_cast<size_t>(j - S) * D;
  };
  // all: every wave takes part (else waves 0-3 issue everything)
  auto dma_tile = [&](int t, int b, bool with_v, auto pure, bool all) __attribute__((always_inline)) {
    if (!all && upper) return;
#pragma unroll
    for (int it = 0; it < KIT; ++it) {
      const int ins = it * kDW + dw;
      if (ins < KINS && (!all || ((it & 1) != 0) == upper)) {
        const uint16_t* src;
        if constexpr (decltype(pure)::value) {
          src = kst + static_cast<size_t>(t) * kKT * D + koff_at(it);
        } else {
          const int ko = koff_at(it), r = ko / D;
          src = key_src(kst, kfr, t * kKT + r) + (ko - r * D);
        }
        dma_one(src, &sm.k[b][0][0], ins);
      }
    }
    if (!with_v) return;
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int ins = it * kDW + dw;
      if (ins < VINS && (!all || ((it & 1) != 0) == upper)) {
        const uint16_t* src;
        if constexpr (decltype(pure)::value) {
          src = vst + static_cast<size_t>(t) * kKT * D + voff_at(it);
        } else {
          const int vo = voff_at(it), r = vo / D;
          src = key_src(vst, vfr, t * kKT + r) + (vo - r * D);
        }
        dma_one(src, &sm.v[b][0][0], ins);
      }
    }
  };
  // the copies of a tile are in LDS once vmcnt drains; the barrier after this
  // publishes them to the workgroup
  auto dma_wait = [] { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };

  // LDS operand reads are issued ahead as inline assembly with explicit waits:
  // the V operand of block kb is read while block kb's exponentials run, the K
  // operand of block kb + 1 during block kb's PV MFMAs and column sums (at most
  // 15 reads are in flight, the reach of lgkmcnt).  A wait for one of these reads
  // counts the reads issued after it; other LDS accesses in flight can only
  // make such a wait longer.
  auto lds_addr = [](const void* p) -> uint32_t {
    return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const char*)p));
  };
  auto issue_k = [&](auto kbc, uint32_t kaddr, u32x4 (&kop)[KS]) {
    constexpr int KB = decltype(kbc)::value;
    static_for<KS>([&](auto ksc) {
      constexpr int ks = decltype(ksc)::value;
      kop[ks] = ds_read_b128<(KB * 32 * (D + kPadK) + ks * 16) * 2>(kaddr);
    });
  };
  // S^T block from the K operand in kop; `later` = reads issued after kop's
  auto qk_mfma = [&](u32x4 (&kop)[KS]) -> f32x16 {
    __builtin_amdgcn_s_setprio(1);
    f32x16 acc = {};
    static_for<KS>([&](auto ksc) {
      constexpr int ks = decltype(ksc)::value;
      lgkm_wait<KS - 1 - ks>(kop[ks]);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kop[ks]), qreg[ks], acc, 0, 0, 0);
    });
    __builtin_amdgcn_s_setprio(0);
    return acc;
  };

  // ============================ sweep 1: row statistics ============================
  float m = -1e30f, l = 0.f;
  // NB = 32-key blocks of a tile this wave takes: 4, or 2 in a split workgroup
  auto sweep1_tile = [&](int t, auto masked, auto pure_next, auto nbc) {
    constexpr int NB = decltype(nbc)::value;
    const int b = t & 1;
    const uint32_t kaddr = lds_addr(&sm.k[b][key0 + l32][h * 8]);
    u32x4 kop[KS];
    if (active) issue_k(std::integral_constant<int, 0>{}, kaddr, kop);
    if (t + 1 < kt1) dma_tile(t + 1, b ^ 1, false, pure_next, false);
    // masked tiles: blocks whose first key is past the wave's limit (a suffix) are skipped
    const int first = t * kKT + key0;
    const int na = !decltype(masked)::value ? NB : wlim < first ? 0 : min(NB, (wlim - first) / 32 + 1);
    if (active) {
      static_for<NB>([&](auto kbc) {
        constexpr int KB = decltype(kbc)::value;
        if constexpr (decltype(masked)::value) {
          if (KB >= na) return;
        }
        const f32x16 acc = qk_mfma(kop);
        if constexpr (KB + 1 < NB) issue_k(std::integral_constant<int, KB + 1>{}, kaddr, kop);
        f32x16 accv = acc;
        asm volatile("" : "+v"(accv));  // keep the exponentials behind the reads just issued
        float z[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) z[v] = accv[v];
        if constexpr (decltype(masked)::value) {
          const int rel = lim - (t * kKT + key0 + KB * 32 + 4 * h);
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
      });
    }
    if (t + 1 < kt1) dma_wait();
    __syncthreads();
  };
  auto sweep1 = [&](auto nbc) {
    const int tm = first_masked < kt1 ? first_masked : kt1;  // unmasked tiles end here
    for (int t = kt0; t + 1 < tm; ++t) sweep1_tile(t, std::false_type{}, std::true_type{}, nbc);
    if (kt0 < tm) sweep1_tile(tm - 1, std::false_type{}, std::false_type{}, nbc);
    for (int t = kt0 > first_masked ? kt0 : first_masked; t < kt1; ++t)
      sweep1_tile(t, std::true_type{}, std::false_type{}, nbc);
  };

  // Row maximum (log2 units) and 1/sum.  Sweep 2 feeds the PV MFMA with
  // E = exp2(x - max) <= 1, whose largest entry is exactly 1 in bf16, and applies
  // 1/sum in fp32 to the output; the column sums use P = E / sum.
  float mrow, inv_l;
  float* stats = a.stats + (static_cast<size_t>(lg) * a.n_ks) * (a.G * a.T) * 2;  // [ks][row] (max, sum)
  if (a.mode == 2) {
    // output launch of a key-split plan: merge the statistics of every key range
    float mm = -1e30f, ll = 0.f;
    if (row_valid) {
      // all loads first, then the merge in split order
      float ms[kMaxKeySplits], lsum[kMaxKeySplits];
#pragma unroll
      for (int s = 0; s < kMaxKeySplits; ++s) {
        ms[s] = -1e30f;
        lsum[s] = 0.f;
        if (s < a.n_ks) {
          const float* st = stats + (static_cast<size_t>(s) * (a.G * a.T) + r_lane) * 2;
          ms[s] = st[0];
          lsum[s] = st[1];
        }
      }
#pragma unroll
      for (int s = 0; s < kMaxKeySplits; ++s) {
        const float mt = fmaxf(mm, ms[s]);
        ll = ll * fast_exp2((mm - mt) * c) + lsum[s] * fast_exp2((ms[s] - mt) * c);
        mm = mt;
      }
    }
    mrow = row_valid ? mm * c : 0.f;
    inv_l = row_valid ? 1.0f / ll : 0.f;
  } else {
    // sweep 1 over key tiles [kt0, kt1): this range's (max, sum) per row, in mm, ll
    float mm, ll;
    auto row_stats = [&]() {
      m = -1e30f;
      l = 0.f;
      if (kt0 < kt1) dma_tile(kt0, kt0 & 1, false, std::false_type{}, true);
      dma_wait();
      __syncthreads();
      if (split)
        sweep1(std::integral_constant<int, kKT / 64>{});
      else
        sweep1(std::integral_constant<int, kKT / 32>{});

      // The other 16 keys of every 32-key block live in lane ^ 32.  Both lanes merge
      // in one operand order (h = 0's statistics first; the merge rounds differently
      // with the operands swapped), so the two lanes of a row hold bit-identical
      // statistics and equal keys get equal column sums wherever they sit in a block.
      const float mo = __shfl_xor(m, 32, 64);
      const float lo = __shfl_xor(l, 32, 64);
      const float ma = h ? mo : m, la = h ? lo : l, mb = h ? m : mo, lb = h ? l : lo;
      mm = fmaxf(ma, mb);
      ll = la * fast_exp2((ma - mm) * c) + lb * fast_exp2((mb - mm) * c);
      if (split) {
        // the other key half of these rows is wave ^ 4's; exchanged through the
        // second column-sum buffer, first written after sweep 2's first barrier;
        // merged with the first half's statistics first in both waves
        float* xm = &sm.cs[1][wave][0];
        if (h == 0) {
          xm[l32] = mm;
          xm[32 + l32] = ll;
        }
        __syncthreads();
        const float* pm = &sm.cs[1][wave ^ 4][0];
        const float mp = pm[l32], lp = pm[32 + l32];
        const float m0 = grp ? mp : mm, l0 = grp ? lp : ll, m1 = grp ? mm : mp, l1 = grp ? ll : lp;
        const float mt = fmaxf(m0, m1);
        ll = l0 * fast_exp2((m0 - mt) * c) + l1 * fast_exp2((m1 - mt) * c);
        mm = mt;
      }
    };
    row_stats();
    if constexpr (VAR == 2) {
      // Fused key split (mode 3): the workgroups of one row range exchange their
      // ranges' statistics through `stats` instead of ending the launch.  Each
      // publishes its own (device-scope stores, then its flag = this launch's
      // epoch), waits for the others' flags for at most wait_ticks of the
      // constant clock, and computes every range still missing itself: sweep 1
      // over that range gives bit for bit what its own workgroup publishes, so
      // the result never depends on who computed what, and every wait ends.
      // Mode 4 waits for nobody (every workgroup computes every range).
      const int GT = a.G * a.T;
      auto publish = [&](int r) {
        if (h == 0 && grp == 0 && row_valid) {
          uint32_t* st = reinterpret_cast<uint32_t*>(stats + (static_cast<size_t>(r) * GT + r_lane) * 2);
          __hip_atomic_store(st, __float_as_uint(mm), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(st + 1, __float_as_uint(ll), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's stores have completed
      };
      publish(ks);
      __syncthreads();  // every wave's stores have completed; the tile buffers are free
      // sweep 2's first tile is copied while the workgroup waits for the others
      if (kt0 < kt1) dma_tile(kt0, kt0 & 1, true, std::false_type{}, true);
      const unsigned all = (1u << a.n_ks) - 1u;
      unsigned* shared_mask = reinterpret_cast<unsigned*>(&sm.il[0][0]);  // free until the epilogue
      if (tid == 0) {
        uint32_t* flags = a.flags + (static_cast<size_t>(lg) * a.tile_stride + wk.tile) * a.n_ks;
        unsigned got = 1u << ks;
        if (a.mode == 3) {
          __hip_atomic_store(&flags[ks], a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          const uint64_t t_end = __builtin_amdgcn_s_memrealtime() + a.wait_ticks;
          for (;;) {
            for (int r = 0; r < a.n_ks; ++r)
              if (!(got >> r & 1u) && __hip_atomic_load(&flags[r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == a.epoch)
                got |= 1u << r;
            if (got == all || __builtin_amdgcn_s_memrealtime() > t_end) break;
            __builtin_amdgcn_s_sleep(2);
          }
        }
        *shared_mask = got;
      }
      __syncthreads();
      unsigned todo = all & ~*shared_mask;
      const bool refill = todo != 0u;
      if (refill) {  // the tile buffers are needed: the copy above lands first
        dma_wait();
        __syncthreads();
      }
      while (todo != 0u) {  // ranges whose statistics did not arrive in time
        const int r = __builtin_ctz(todo);
        todo &= todo - 1u;
        kt0 = range_lo(r);
        kt1 = range_lo(r + 1);
        row_stats();
        publish(r);
      }
      kt0 = range_lo(ks);
      kt1 = range_lo(ks + 1);
      if (refill && kt0 < kt1) dma_tile(kt0, kt0 & 1, true, std::false_type{}, true);
      __syncthreads();  // the ranges computed here are in `stats` before anyone reads them
      // merge every range's statistics in split order (as the output launch of
      // the two-launch scheme does)
      float mg = -1e30f, lg_sum = 0.f;
      if (row_valid) {
        float ms[kMaxKeySplits], lsum[kMaxKeySplits];
#pragma unroll
        for (int r = 0; r < kMaxKeySplits; ++r) {
          ms[r] = -1e30f;
          lsum[r] = 0.f;
          if (r < a.n_ks) {
            const uint32_t* st = reinterpret_cast<const uint32_t*>(stats + (static_cast<size_t>(r) * GT + r_lane) * 2);
            ms[r] = __uint_as_float(__hip_atomic_load(st, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
            lsum[r] = __uint_as_float(__hip_atomic_load(st + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
          }
        }
#pragma unroll
        for (int r = 0; r < kMaxKeySplits; ++r) {
          const float mt = fmaxf(mg, ms[r]);
          lg_sum = lg_sum * fast_exp2((mg - mt) * c) + lsum[r] * fast_exp2((ms[r] - mt) * c);
          mg = mt;
        }
      }
      mm = mg;
      ll = lg_sum;
    }
    if (a.mode == 1) {
      // statistics launch of a key-split plan: this key range's (max, sum) per row
      if (h == 0 && grp == 0 && row_valid) {
        float* st = stats + (static_cast<size_t>(ks) * (a.G * a.T) + r_lane) * 2;
        st[0] = mm;
        st[1] = ll;
      }
      return;
    }
    mrow = row_valid ? mm * c : 0.f;
    inv_l = row_valid ? 1.0f / ll : 0.f;
  }

  // ======================== sweep 2: P, O and column sums ========================
  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = f32x16{};

  const int key_lane = 8 * (((lane >> 3) & 1) + 2 * ((lane >> 4) & 1)) + 4 * h + (((lane >> 1) & 1) + 2 * ((lane >> 2) & 1));
  // column-sum weights (1 / row sum) of the two rows the first reduction step meets
  const float il_partner = __shfl_xor(inv_l, 16, 64);
  const float w0 = (lane & 16) ? il_partner : inv_l, w1 = (lane & 16) ? inv_l : il_partner;
  // transpose-read coordinates of this lane inside its 16-lane group
  const int tr_row = 4 * h + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  // End of a sweep-2 tile: wait for the next tile's copies, then the cross-wave
  // column sums of tile t -> this row tile's partials; buffer b is written again
  // only after the next barrier.  In a split workgroup a key's sums come from the
  // four waves of its half.
  auto finish_tile = [&](int t, int b) {
    if (t + 1 < kt1) dma_wait();
    __syncthreads();
    if (tid < kKT) {
      const int j = t * kKT + tid;
      if (j < n_keys) {
        float sum = 0.f;
        if (split) {
          const int w0 = (tid / (kKT / 2)) * (kWaves / 2);
#pragma unroll
          for (int w = 0; w < kWaves / 2; ++w) sum += sm.cs[b][w0 + w][tid];
        } else {
#pragma unroll
          for (int w = 0; w < kWaves; ++w) sum += sm.cs[b][w][tid];
        }
        part[j] = sum;
      }
    }
  };

  // Tiles with frame keys (masked entries): block by block without the software
  // pipeline, skipping the blocks past the wave's causal limit (a suffix of the
  // tile), whose column sums are 0.
  auto sweep2_masked_tile = [&](int t, auto nbc) {
    constexpr int NB = decltype(nbc)::value;
    const int b = t & 1;
    const uint32_t kaddr = lds_addr(&sm.k[b][key0 + l32][h * 8]);
    const uint32_t vaddr = lds_addr(&sm.v[b][key0 + tr_row][tr_col]);
    const int first = t * kKT + key0;
    const int na = wlim < first ? 0 : min(NB, (wlim - first) / 32 + 1);
    if (t + 1 < kt1) dma_tile(t + 1, b ^ 1, true, std::false_type{}, false);
    if (active) {
      static_for<NB>([&](auto kbc) {
        constexpr int KB = decltype(kbc)::value;
        const int kb = key0 / 32 + KB;  // 32-key block of the tile
        if (KB >= na) {
          sm.cs[b][wave][kb * 32 + key_lane] = 0.f;
          return;
        }
        u32x4 kop[KS];
        issue_k(std::integral_constant<int, KB>{}, kaddr, kop);
        const f32x16 acc = qk_mfma(kop);
        bf16x8 vop[2][DB];
        static_for<2 * DB>([&](auto ic) {
          constexpr int s_ = decltype(ic)::value / DB, db = decltype(ic)::value % DB;
          constexpr int r0 = KB * 32 + s_ * 16;
          const s16x4 lo = ds_read_tr<(r0 * (D + kPadV) + db * 32) * 2>(vaddr);
          const s16x4 hi = ds_read_tr<((r0 + 8) * (D + kPadV) + db * 32) * 2>(vaddr);
          vop[s_][db] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        });
        const int rel = lim - (t * kKT + kb * 32 + 4 * h);
        bf16x8 pe[2];
        float cs[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float e = fast_exp2(fmaf(acc[v], c, -mrow));
          if (8 * (v >> 2) + (v & 3) > rel) e = 0.f;
          pe[v >> 3][v & 7] = static_cast<__bf16>(e);
          cs[v] = e;
        }
        static_for<2 * DB>([&](auto ic) {
          constexpr int i = decltype(ic)::value, s_ = i / DB, db = i % DB;
          lgkm_wait<2 * (2 * DB - 1 - i)>(vop[s_][db]);
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pe[s_], vop[s_][db], o[db], 0, 0, 0);
        });
        sm.cs[b][wave][kb * 32 + key_lane] = column_reduce(cs, lane, w0, w1);
      });
    } else {
      for (int i = lane; i < kKT; i += 64) sm.cs[b][wave][i] = 0.f;
    }
    finish_tile(t, b);
  };

  // Tiles of state keys only (no masked entries), software-pipelined.
  auto sweep2_tile = [&](int t, auto pure_next, auto nbc) {
    constexpr int NB = decltype(nbc)::value;
    const int b = t & 1;
    const uint32_t kaddr = lds_addr(&sm.k[b][key0 + l32][h * 8]);
    // LDS byte address of this lane's transpose-read position in buffer b
    const uint32_t vaddr = lds_addr(&sm.v[b][key0 + tr_row][tr_col]);
    u32x4 kop[KS];
    if (active) issue_k(std::integral_constant<int, 0>{}, kaddr, kop);
    if (t + 1 < kt1) dma_tile(t + 1, b ^ 1, true, pure_next, false);
    if (active) {
      // Software pipeline over the tile's blocks: block kb + 1's K Q^T MFMAs are
      // issued interleaved with block kb's exponentials, block kb's PV MFMAs with
      // its column sums, so the wave's VALU work issues between its own MFMAs.
      f32x16 acc = qk_mfma(kop);
      if constexpr (NB > 1) issue_k(std::integral_constant<int, 1>{}, kaddr, kop);
      static_for<NB>([&](auto kbc) {
        constexpr int KB = decltype(kbc)::value;
        constexpr bool NEXT = KB + 1 < NB;
        const int kb = key0 / 32 + KB;  // 32-key block of the tile
        // wait for the next block's K operand (the latest reads), then read this block's V
        if constexpr (NEXT) {
          static_for<KS>([&](auto ksc) {
            constexpr int ks = decltype(ksc)::value;
            lgkm_wait<KS - 1 - ks>(kop[ks]);
          });
        }
        bf16x8 vop[2][DB];
        static_for<2 * DB>([&](auto ic) {
          constexpr int s_ = decltype(ic)::value / DB, db = decltype(ic)::value % DB;
          constexpr int r0 = KB * 32 + s_ * 16;
          const s16x4 lo = ds_read_tr<(r0 * (D + kPadV) + db * 32) * 2>(vaddr);
          const s16x4 hi = ds_read_tr<((r0 + 8) * (D + kPadV) + db * 32) * 2>(vaddr);
          vop[s_][db] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        });
        f32x16 acc_next = {};
        if constexpr (NEXT) {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            acc_next = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kop[ks]), qreg[ks],
                                                               acc_next, 0, 0, 0);
        }
        bf16x8 pe[2];
        float cs[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float e = fast_exp2(fmaf(acc[v], c, -mrow));
          pe[v >> 3][v & 7] = static_cast<__bf16>(e);
          cs[v] = e;
        }
        if constexpr (NEXT) {
#pragma unroll
          for (int i = 0; i < KS; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x402, 7, 0);
          }
        }
        static_for<2 * DB>([&](auto ic) {
          constexpr int i = decltype(ic)::value, s_ = i / DB, db = i % DB;
          lgkm_wait<2 * (2 * DB - 1 - i)>(vop[s_][db]);
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pe[s_], vop[s_][db], o[db], 0, 0, 0);
        });
        // K operand two blocks ahead (this wave's kop registers are free again)
        if constexpr (KB + 2 < NB) issue_k(std::integral_constant<int, KB + 2>{}, kaddr, kop);
        const float tot = column_reduce(cs, lane, w0, w1);
        sm.cs[b][wave][kb * 32 + key_lane] = tot;  // lanes l and l ^ 1 store the same total
#pragma unroll
        for (int i = 0; i < 2 * DB; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x402, 5, 0);
        }
        acc = acc_next;
      });
    } else {
      for (int i = lane; i < kKT; i += 64) sm.cs[b][wave][i] = 0.f;
    }
    finish_tile(t, b);
  };
  auto sweep2 = [&](auto nbc) {
    const int tm = first_masked < kt1 ? first_masked : kt1;
    for (int t = kt0; t + 1 < tm; ++t) sweep2_tile(t, std::true_type{}, nbc);
    if (kt0 < tm) sweep2_tile(tm - 1, std::false_type{}, nbc);
    for (int t = kt0 > first_masked ? kt0 : first_masked; t < kt1; ++t) sweep2_masked_tile(t, nbc);
  };
  if constexpr (VAR != 2) {  // a fused key split issued this copy before its wait
    if (kt0 < kt1) dma_tile(kt0, kt0 & 1, true, std::false_type{}, true);
  }
  dma_wait();
  __syncthreads();
  if (split)
    sweep2(std::integral_constant<int, kKT / 64>{});
  else
    sweep2(std::integral_constant<int, kKT / 32>{});

  // split workgroup: the second key half's waves hand their unnormalised output
  // to the first half's (LDS holds no tile any more)
  if (split) {
    float* ox = reinterpret_cast<float*>(smem_raw);  // [row block][DB][16][64 lanes]
    static_assert(kWaves / 2 * DB * 16 * 64 * 4 <= 2 * kKT * (D + kPadK) * 2, "exchange fits the K buffers");
    if (grp == 1 && active) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) ox[((rb * DB + db) * 16 + v) * 64 + lane] = o[db][v];
    }
    __syncthreads();
    if (grp == 0 && active) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][v] += ox[((rb * DB + db) * 16 + v) * 64 + lane];
    }
  }
  const bool writer = active && grp == 0;

  // ---------------- output: O / sum, staged through LDS for 16-byte stores ----------------
  if (writer && h == 0) sm.il[wave][l32] = inv_l;
  __syncthreads();
  if (a.mode >= 2) {
    // this key range's share of O (already divided by the merged sum), fp32
    if (writer) {
      float* op = a.opart + static_cast<size_t>(ks) * a.n_layers * a.H_q * a.T * D +
                  static_cast<size_t>(layer * a.H_q + g * a.G) * a.T * D;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = 8 * (v >> 2) + 4 * h + (v & 3);
        const float sc = sm.il[wave][r];
        if (row0 + r < row_end) {
#pragma unroll
          for (int db = 0; db < DB; ++db) op[static_cast<size_t>(row0 + r) * D + db * 32 + l32] = o[db][v] * sc;
        }
      }
    }
    return;
  }
  uint16_t* ost = reinterpret_cast<uint16_t*>(smem_raw) + static_cast<size_t>(wave) * kRowsWave * (D + kPadO);
  if (writer) {
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
  if (writer) {
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

namespace {

template <int D, bool ROPE, int VAR>
void launch_one(const AttnArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL((attn_mfma_kernel<D, ROPE, VAR>), dim3(grid), dim3(kThreads), sizeof(Smem<D>), s, a);
}

template <int D, bool ROPE>
void launch_var(const AttnArgs& a, int grid, int var, hipStream_t s) {
  if (var == 2) launch_one<D, ROPE, 2>(a, grid, s);
  else if (var == 1) launch_one<D, ROPE, 1>(a, grid, s);
  else launch_one<D, ROPE, 0>(a, grid, s);
}

template <int D>
hipError_t prepare_dim() {
  const void* kernels[] = {
      reinterpret_cast<const void*>(attn_mfma_kernel<D, false, 0>), reinterpret_cast<const void*>(attn_mfma_kernel<D, true, 0>),
      reinterpret_cast<const void*>(attn_mfma_kernel<D, false, 1>), reinterpret_cast<const void*>(attn_mfma_kernel<D, true, 1>),
      reinterpret_cast<const void*>(attn_mfma_kernel<D, false, 2>), reinterpret_cast<const void*>(attn_mfma_kernel<D, true, 2>)};
  for (const void* k : kernels) {
    const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, sizeof(Smem<D>));
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

hipError_t launch_attention_mfma_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
  // instantiation: 2 = fused key split (modes 3, 4), 1 = output launch carrying a
  // selection, 0 = everything else; the first two can carry a selection
  const bool fused = a.mode == 3 || a.mode == 4;
  const int var = fused ? 2 : (a.mode == 2 && a.n_sel > 0 ? 1 : 0);
  const int grid = a.n_work + (var != 0 ? a.n_sel : 0);
  if (fused && (a.flags == nullptr || a.n_ks > kMaxKeySplits)) return hipErrorInvalidValue;
  const bool rope = a.rope_tab != nullptr;
  if (head_dim == 128) {
    if (rope) launch_var<128, true>(a, grid, var, s);
    else launch_var<128, false>(a, grid, var, s);
  } else {
    if (rope) launch_var<64, true>(a, grid, var, s);
    else launch_var<64, false>(a, grid, var, s);
  }
  return hipGetLastError();
}

size_t attention_mfma_lds_bytes(int head_dim) { return head_dim == 128 ? sizeof(Smem<128>) : sizeof(Smem<64>); }

hipError_t prepare_attention_mfma() {
  const hipError_t e = prepare_dim<128>();
  return e != hipSuccess ? e : prepare_dim<64>();
}

}  // namespace skv
