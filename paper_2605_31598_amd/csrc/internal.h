// Internal launch interface of the StateKV frame-step kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.h"
#include "rope.h"

namespace skv {

// The refresh launch finishes a frame for `n_layers` layers: score finalisation,
// Top-B selection and state update in one workgroup per (layer, KV head), the
// decode-cache append in a second set of workgroups of the same grid (either
// set can be left out), and the sum of a key-split attention's output shares
// in a third.
struct RefreshArgs {
  const float* partial;      // as in AttnArgs
  const int32_t* lg_tiles;   // [n_layers][H_kv] row tiles the attention launch wrote
  int tile_stride, pool_stride;
  const void* kf;            // [n_layers][H_kv][kf_rows][d]   frame keys: the caller's input
  const void* vf;            //   (kf_rows = T) or the frame's rows of the decode cache (max_tokens)
  int64_t kf_rows;           // row stride of one (layer, KV head) block of kf / vf
  bool select;               // workgroups for the selection and the state update
  bool append;               // workgroups for the decode-cache append
  void* ks;                  // [n_layers][H_kv][B][d]   state slots
  void* vs;
  int32_t* state_pos;        // [n_layers][H_kv][B]
  float* state_score;        // [n_layers][H_kv][B]
  float* pool_score;         // [n_layers][H_kv][pool_stride]
  int32_t* pool_pos;         // [n_layers][H_kv][pool_stride]
  int32_t* admit_src;        // [n_layers][H_kv][T]  frame token of the a-th admitted candidate
  int32_t* admit_dst;        // [n_layers][H_kv][T]  state slot it goes to
  int32_t* admit_count;      // [n_layers][H_kv]     admitted rows (split_update only)
  bool split_update;         // selection only: lists and count to global memory, no row copies
  void* ck;                  // [n_layers][H_kv][max_tokens][d]  decode cache
  void* cv;
  int64_t max_tokens, first_row;  // first_row = frame * T
  int n_layers, H_kv, T, B, S;
  int row_bytes;             // d * element size, a multiple of 16
  int32_t frame_pos0;        // virtual position of frame token 0
  float inv_T;
  int mode;                  // selection rule: 0: Top-B by score, 1: the B most recent
  // key-split attention plans: n_comb more workgroups write the attention
  // output, the sum of the n_ks fp32 shares (AttnArgs::opart), as bf16
  int n_ks;                  // 1: no key split, no combine workgroups
  int n_comb;
  const float* opart;        // [n_ks][out_elems]
  void* out;                 // [out_elems] bf16
  int64_t out_elems;         // a multiple of 4
};

// One attention launch covers `n_layers` consecutive layers of one frame.
// Layer indices inside the struct are relative to the first layer of the call;
// every pointer is already offset to that layer.
struct AttnArgs {
  const void* q;       // [n_layers][H_q][T][d]
  const void* kf;      // [n_layers][H_kv][T][d]   frame keys
  const void* vf;      // [n_layers][H_kv][T][d]   frame values
  const void* ks;      // [n_layers][H_kv][kv_rows][d]  earlier keys, rows 0..S-1 valid: the
  const void* vs;      //   compressed state (kv_rows = B) or the decode cache (kv_rows = max_tokens)
  void* out;           // [n_layers][H_q][T][d]
  float* partial;      // [n_layers][H_kv][tile_stride][pool_stride] column sums of P per row
                       // tile; null for streaming full attention (no scores)
  const AttnWork* work;  // MFMA kernel: one work item per workgroup (n_work of them)
  int n_work;
  int n_layers, H_q, H_kv, G, T, B, S;
  int kv_rows;
  int tile_stride, pool_stride;
  float scale_log2;    // softmax scale * log2(e)
  const float* rope_tab;  // null: no rotation; else rotate Q by {cos, sin} per (relative position,
                          // pair); kf holds the frame's keys already rotated
  int rope_pos0;          // relative position of frame token 0 (n * T)
  // Key-split plans (MFMA kernel): the launch with mode 1 writes each work
  // item's (row max, sum of exp2) over its key range to `stats`, the launch with
  // mode 2 merges them, writes the column sums of its key range and its fp32
  // share of O to `opart`; workgroups of the refresh launch then add the shares.
  // Modes 3 and 4 do both in one launch: the workgroups of one row range
  // exchange their ranges' statistics through `stats` and per-item flags set to
  // `epoch` (mode 3, waiting at most wait_ticks of the constant clock for each
  // other and computing what has not arrived), or each computes every range
  // itself (mode 4).  The output, shares and column sums equal the two launches'.
  int mode;               // 0: whole key range in one launch; 1: statistics; 2: output share; 3, 4: both
  int n_ks;               // key splits of the plan (1: none)
  float* stats;           // [n_layers * H_kv][n_ks][G * T][2]
  float* opart;           // [n_ks][n_layers][H_q][T][d]
  uint32_t* flags;        // modes 3, 4: [n_layers * H_kv][tile_stride][n_ks], zero or an earlier epoch
  uint32_t epoch;         // nonzero, different from every earlier launch's on the same flags
  uint64_t wait_ticks;
  // An output launch (mode 2) can carry the selection of an earlier one-layer
  // call: n_sel more workgroups, one per (layer, KV head) of `sel`, finalise its
  // scores, select and update its state, with the frame's rows read back from
  // the decode cache, where that call appended them.
  int n_sel;
  RefreshArgs sel;
};

// Decode over the detailed cache (split-key flash decoding).  Each wave of the
// split kernel owns one item = (layer-head, 32-row block, key split); the
// combine kernel merges the splits of every row.
struct DecodeArgs {
  const void* q;       // [n_layers][H_q][t][d]   new tokens' queries
  const void* kn;      // [n_layers][H_kv][t][d]  new tokens' keys
  const void* vn;      // [n_layers][H_kv][t][d]  new tokens' values
  const void* ck;      // [n_layers][H_kv][max_tokens][d]  decode cache D
  const void* cv;
  void* out;           // [n_layers][H_q][t][d]
  float* part_o;       // [n_items][32][d]  unnormalised output of each split
  float* part_ml;      // [n_items][2][32]  row maximum (logit units), row sum
  int64_t max_tokens;  // row stride of D
  int64_t dec_row0;    // first decode row of D
  int n_layers, H_q, H_kv, G, t;
  int S;               // video tokens of D (T * frames done)
  int n_dec;           // tokens decoded before this call
  int n_rb;            // 32-row blocks per layer-head: ceil(G t / 32)
  int split;           // keys per split, a multiple of 32
  int n_split;         // ceil((S + n_dec + t) / split)
  float scale_log2;
  const float* rope_tab;  // null: no rotation; else rotate Q (new token i at relative position
  int rope_pos0;          // rope_pos0 + i); kn holds the new keys already rotated
};

constexpr int kDecodeMaxTokens = 64;  // new tokens per decode call
constexpr int kDecodeItems = 2048;    // split items aimed at per call: one wave per SIMD slot of the
                                      // 256-CU device at two waves per SIMD (partials sized for it)

constexpr int kMaxKeySplits = 16;       // key ranges of a key-split attention plan, at most
constexpr int kMfmaRowsPerWave = 32;    // query rows (G*T packed) per attention wave
constexpr int kMfmaWaves = 8;           // waves per attention workgroup (at most)
constexpr int kSimpleRowsPerTile = 64;
constexpr int kSelectThreads = 1024;
constexpr int kMaxPool = 16384;         // B + T limit (selection keeps the pool in LDS)

hipError_t launch_attention_mfma_bf16(const AttnArgs& a, int head_dim, hipStream_t s);
hipError_t launch_attention_full_bf16(const AttnArgs& a, int head_dim, hipStream_t s);
hipError_t launch_attention_simple_f32(const AttnArgs& a, int head_dim, hipStream_t s);
hipError_t launch_decode_bf16(const DecodeArgs& a, int head_dim, hipStream_t s);
hipError_t launch_refresh(const RefreshArgs& a, hipStream_t s);
// The state update and the append as launches of their own (after a launch_refresh
// with select = true, append = false, split_update = true).
hipError_t launch_refresh_update(const RefreshArgs& a, hipStream_t s);
hipError_t launch_refresh_append(const RefreshArgs& a, hipStream_t s);
// Rotates n_blocks * t key rows (t rows per (layer, KV head) block, row r at
// relative position pos0 + r) from `in` to `out`; same layout, either dtype.
hipError_t launch_rope_keys(const void* in, void* out, int n_blocks, int t, int row_bytes, int elem,
                            const float* tab, int pos0, hipStream_t s);
hipError_t prepare_kernels(int head_dim, bool bf16, int pool_stride);
// LDS bytes of an MFMA attention workgroup (what a carried selection may use).
size_t attention_mfma_lds_bytes(int head_dim);
// LDS bytes a selection workgroup needs for a pool of P candidates.
size_t selection_lds_bytes(int P);

}  // namespace skv
