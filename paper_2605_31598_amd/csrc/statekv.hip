// Host runtime of the StateKV frame step: configuration checks, one-time device
// allocation, per-frame launch sequence and the C ABI of include/statekv.h.
//
// Per frame and layer range the stream receives two launches:
//   1. attention + fused column sums of P     (Eq. 5 and the importance score)
//   2. refresh: score finalisation, Top-B selection (Eq. 6, ties to the lowest
//      position) and the state update (admitted rows into evicted or free
//      slots), concurrently with the decode-cache append of the frame's K/V
//      (Eq. 4, detailed state)
// (with skv_config.split_refresh, the refresh runs as three launches instead:
// selection, state update, append, each timed on its own).
// The state size S_n = min(B, n * T) and the frame's virtual positions
// L_n + t are host-side bookkeeping (virtual sequence length paragraph), so the
// step needs no device-to-host synchronisation.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdlib>
#include <algorithm>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/statekv.h"
#include "internal.h"

namespace skv {
hipError_t prepare_refresh(int pool_stride);
hipError_t prepare_attention_mfma();
hipError_t prepare_attention_full();
}  // namespace skv

namespace {

thread_local std::string g_last_error;

skv_status fail(skv_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

skv_status hip_fail(hipError_t e, const char* what) {
  g_last_error = std::string(what) + ": " + hipGetErrorString(e);
  return SKV_ERR_DEVICE;
}

}  // namespace

struct skv_ctx {
  skv_config cfg{};
  hipStream_t stream = nullptr;
  int device = 0;
  int elem = 2;
  int G = 1;
  float scale_log2 = 0.f;
  bool use_mfma = false;
  int tile_stride = 0;  // row-tile slots per (layer, KV head) in `partial`
  int pool_stride = 0;
  size_t row_bytes = 0;
  int64_t max_tokens = 0;

  // device buffers (one allocation each)
  void* state_k = nullptr;   // [L][H_kv][B][d]
  void* state_v = nullptr;
  int32_t* state_pos = nullptr;    // [L][H_kv][B]
  float* state_score = nullptr;
  void* cache_k = nullptr;   // [L][H_kv][max_tokens][d]
  void* cache_v = nullptr;
  float* partial = nullptr;  // [L][H_kv][tile_stride][pool_stride]
  float* pool_score = nullptr;     // [L][H_kv][pool_stride]
  int32_t* pool_pos = nullptr;
  int32_t* admit_src = nullptr;    // [L][H_kv][T]
  int32_t* admit_dst = nullptr;
  int32_t* admit_count = nullptr;  // [L][H_kv] (split refresh launches)
  float* rope_tab = nullptr;       // RoPE {cos, sin} per (relative position, pair), or null
  void* rope_keys = nullptr;       // with RoPE: the step's new keys, rotated: [L][H_kv][new rows][d]
  float* dec_part_o = nullptr;     // decode split partials: [dec_items][32][d]
  float* dec_part_ml = nullptr;    // [dec_items][2][32]
  int dec_items = 0;
  int64_t dec_row0 = 0;            // first decode row of D
  // attention work plans, one per layer_count (index layer_count - 1), in one
  // device allocation; the fp32 path uses fixed 64-row tiles instead
  struct Plan {
    const skv::AttnWork* work = nullptr;
    const int32_t* tiles = nullptr;  // row tiles per (layer, KV head) of the call
    int n_work = 0;
    int n_ks = 1;                    // key splits (calls too small to fill the device)
  };
  std::vector<Plan> plans;
  uint32_t* ks_flags = nullptr;    // fused key-split launches: per-item flags, [L][H_kv][tile_stride][16]
  uint32_t ks_epoch = 0;           // the last such launch's epoch
  uint64_t ks_wait_ticks = 0;      // how long their workgroups wait for each other (constant clock)
  float* split_stats = nullptr;    // key-split plans: per-range row statistics and output shares,
  float* split_out = nullptr;      // sized for the largest such plan (null if none)
  void* scratch = nullptr;         // this device's static scratch (skv_frame_step_noalloc)
  std::vector<void*> allocations;

  // progress of the stream
  bool broken = false;  // a launch failed part-way through a step: steps refuse until reset/seek
  int64_t frame = 0;    // frame being processed
  int next_layer = 0;   // next layer expected within that frame
  int64_t n_decoded = 0;   // tokens decoded after the video (all layers done)
  int dec_next_layer = 0;  // next layer expected within the current decode call
  int dec_pending = 0;     // tokens of the decode call in progress
  std::vector<int32_t> last_pool;  // candidates of each layer's last step
  // A one-layer call's selection and state update, left to the output launch of
  // the next one-layer call on other layers (pend_ra: its refresh arguments,
  // reading the frame's rows back from the decode cache).
  bool pend = false;
  int pend_lb = 0, pend_lc = 0;
  skv::RefreshArgs pend_ra{};

  // timing
  std::vector<hipEvent_t> events;  // (SKV_N_STAGES + 1) per recorded step
  std::vector<uint8_t> recorded;   // per recorded step: bit i set when events[i] was recorded
  int timing_max = 0, timing_n = 0;
  int timing_stride = 1;     // record every timing_stride-th step
  int64_t timing_seen = 0;   // steps since skv_timing_start
};

namespace {

skv_status alloc(skv_ctx* c, size_t bytes, void** out) {
  void* p = nullptr;
  const hipError_t e = hipMalloc(&p, bytes > 0 ? bytes : 16);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(SKV_ERR_OUT_OF_MEMORY, "hipMalloc of " + std::to_string(bytes) + " bytes failed");
  }
  c->allocations.push_back(p);
  *out = p;
  return SKV_OK;
}

void release(skv_ctx* c) {
  for (hipEvent_t e : c->events) (void)hipEventDestroy(e);
  c->events.clear();
  for (void* p : c->allocations) (void)hipFree(p);
  c->allocations.clear();
}

int layer_frames_done(const skv_ctx* c, int layer) {
  return static_cast<int>(c->frame) + (layer < c->next_layer ? 1 : 0);
}

int state_size(const skv_ctx* c, int64_t frames_done) {
  const int64_t seen = frames_done * c->cfg.tokens_per_frame;
  return static_cast<int>(seen < c->cfg.capacity ? seen : c->cfg.capacity);
}

// RoPE table: for relative position p (virtual position pos_offset + p) and pair
// j < d/2, {cos, sin} of (pos_offset + p) * f_j times the YaRN temperature, in
// double precision (exact range reduction of large angles), rounded to fp32.
skv_status build_rope_table(skv_ctx* c) {
  const skv_config& cfg = c->cfg;
  if (cfg.rope == SKV_ROPE_NONE) return SKV_OK;
  const int d = cfg.head_dim, half = d / 2;
  std::vector<double> f(static_cast<size_t>(half));
  double mscale = 1.0;
  for (int j = 0; j < half; ++j) f[j] = std::pow(static_cast<double>(cfg.rope_theta), -2.0 * j / d);
  if (cfg.rope == SKV_ROPE_YARN) {
    const double s = cfg.rope_factor, two_pi = 6.283185307179586476925286766559;
    for (int j = 0; j < half; ++j) {
      const double r = cfg.rope_orig_max * f[j] / two_pi;
      const double g = std::min(1.0, std::max(0.0, (r - 1.0) / (32.0 - 1.0)));
      f[j] = (1.0 - g) * f[j] / s + g * f[j];
    }
    mscale = 0.1 * std::log(s) + 1.0;
  }
  const size_t n_pos = static_cast<size_t>(c->max_tokens);
  std::vector<float> tab(n_pos * d);
  for (size_t p = 0; p < n_pos; ++p) {
    const double pos = static_cast<double>(cfg.pos_offset + static_cast<int64_t>(p));
    for (int j = 0; j < half; ++j) {
      const double ang = pos * f[j];
      tab[p * d + 2 * j] = static_cast<float>(std::cos(ang) * mscale);
      tab[p * d + 2 * j + 1] = static_cast<float>(std::sin(ang) * mscale);
    }
  }
  void* dev = nullptr;
  const skv_status s = alloc(c, tab.size() * sizeof(float), &dev);
  if (s != SKV_OK) return s;
  const hipError_t e = hipMemcpy(dev, tab.data(), tab.size() * sizeof(float), hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy of the RoPE table");
  c->rope_tab = static_cast<float*>(dev);
  return SKV_OK;
}

// Uploads the attention work plan of every layer_count (1 .. n_layers).  The
// plans depend only on the shape and the device's compute-unit count.
skv_status build_plans(skv_ctx* c, int rows) {
  const skv_config& cfg = c->cfg;
  std::vector<skv::AttnPlan> host(static_cast<size_t>(cfg.n_layers));
  if (c->use_mfma) {
    int cu = 0;
    const hipError_t e = hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, c->device);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    const int n_xcd = (cu >= 8 && cu % 8 == 0) ? 8 : 1;  // workgroups go round-robin over the XCDs
    // the full-attention kernel has no split workgroups and no key splits
    const bool split_short = cfg.policy != SKV_POLICY_FULL;
    const int max_ks = split_short ? skv::kMaxKeySplits : 1;
    for (int lc = 1; lc <= cfg.n_layers; ++lc)
      host[static_cast<size_t>(lc - 1)] = skv::plan_attention(lc * cfg.n_kv_heads, rows, skv::kMfmaRowsPerWave,
                                                               skv::kMfmaWaves, n_xcd, cu / n_xcd, split_short,
                                                               max_ks);
  } else {
    // fp32 path: every (layer, KV head) writes ceil(rows / 64) tiles; one
    // table of the largest call serves all calls
    host[static_cast<size_t>(cfg.n_layers - 1)].tiles.assign(static_cast<size_t>(cfg.n_layers) * cfg.n_kv_heads,
                                                              c->tile_stride);
  }
  size_t bytes = 0;
  for (const auto& p : host) bytes += p.items.size() * sizeof(skv::AttnWork) + p.tiles.size() * sizeof(int32_t);
  std::vector<char> blob(bytes);
  void* dev = nullptr;
  skv_status s = alloc(c, bytes, &dev);
  if (s != SKV_OK) return s;
  c->plans.assign(static_cast<size_t>(cfg.n_layers), skv_ctx::Plan{});
  size_t off = 0;
  for (size_t i = 0; i < host.size(); ++i) {
    const auto& p = host[i];
    skv_ctx::Plan& d = c->plans[i];
    d.work = reinterpret_cast<const skv::AttnWork*>(static_cast<char*>(dev) + off);
    d.n_work = static_cast<int>(p.items.size());
    d.n_ks = p.n_ks;
    if (!p.items.empty()) std::memcpy(blob.data() + off, p.items.data(), p.items.size() * sizeof(skv::AttnWork));
    off += p.items.size() * sizeof(skv::AttnWork);
    d.tiles = reinterpret_cast<const int32_t*>(static_cast<char*>(dev) + off);
    if (!p.tiles.empty()) std::memcpy(blob.data() + off, p.tiles.data(), p.tiles.size() * sizeof(int32_t));
    off += p.tiles.size() * sizeof(int32_t);
  }
  if (!c->use_mfma)
    for (auto& d : c->plans) d.tiles = c->plans.back().tiles;
  if (bytes > 0) {
    const hipError_t e = hipMemcpy(dev, blob.data(), bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy of the attention plans");
  }
  // buffers of the key-split plans
  size_t stats_floats = 0, out_floats = 0;
  for (size_t i = 0; i < host.size(); ++i) {
    const size_t lc = i + 1, n_ks = static_cast<size_t>(host[i].n_ks);
    if (n_ks < 2) continue;
    stats_floats = std::max(stats_floats, lc * cfg.n_kv_heads * n_ks * static_cast<size_t>(rows) * 2);
    out_floats = std::max(out_floats, n_ks * lc * cfg.n_q_heads * cfg.tokens_per_frame * cfg.head_dim);
  }
  if (stats_floats > 0) {
    s = alloc(c, stats_floats * sizeof(float), reinterpret_cast<void**>(&c->split_stats));
    if (s != SKV_OK) return s;
    s = alloc(c, out_floats * sizeof(float), reinterpret_cast<void**>(&c->split_out));
    if (s != SKV_OK) return s;
    const size_t flag_bytes = static_cast<size_t>(cfg.n_layers) * cfg.n_kv_heads * c->tile_stride * skv::kMaxKeySplits *
                              sizeof(uint32_t);
    s = alloc(c, flag_bytes, reinterpret_cast<void**>(&c->ks_flags));
    if (s != SKV_OK) return s;
    hipError_t e = hipMemsetAsync(c->ks_flags, 0, flag_bytes, c->stream);
    if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync");
    // the workgroups of a fused key-split launch wait at most 200 us for each other
    int khz = 0;
    e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, c->device);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    c->ks_wait_ticks = static_cast<uint64_t>(khz > 0 ? khz : 100000) * 200 / 1000;
  }
  return SKV_OK;
}

// Scratch of skv_frame_step_noalloc: the per-call buffers of a frame step (column-sum
// partials, key-split row statistics and output shares, admit lists) in one static
// device array, so that the call allocates nothing.  Each device the library runs
// on holds its own copy until the process ends.  In host code `scratch` only names
// the symbol: its device address on the current device comes from
// hipGetSymbolAddress, taken once per device at skv_init and used from then on.
constexpr size_t kScratchBytes = size_t{64} << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_addr[kMaxDevices] = {};

// Device address of `scratch` on `device` (current), resolved on first use.
hipError_t scratch_address(int device, void** out) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_addr[device] == nullptr) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_addr[device] = ptr;
  }
  *out = g_scratch_addr[device];
  return hipSuccess;
}

// Per-call buffers of a frame step.
struct StepScratch {
  bool own_layers;      // partial and admit lists are per layer (their contents outlive the call)
  float* partial;       // [layer_count * H_kv][tile_stride][pool_stride]
  float* split_stats;   // [layer_count * H_kv][n_ks][G * T][2]
  float* split_out;     // [n_ks][layer_count][H_q][T][d]
  int32_t* admit_src;   // [layer_count * H_kv][T]
  int32_t* admit_dst;
  int32_t* admit_count; // [layer_count * H_kv]
};

}  // namespace

extern "C" {

const char* skv_status_string(skv_status s) {
  switch (s) {
    case SKV_OK: return "SKV_OK";
    case SKV_ERR_INVALID_ARG: return "SKV_ERR_INVALID_ARG";
    case SKV_ERR_OUT_OF_MEMORY: return "SKV_ERR_OUT_OF_MEMORY";
    case SKV_ERR_CAPACITY: return "SKV_ERR_CAPACITY";
    case SKV_ERR_ORDER: return "SKV_ERR_ORDER";
    case SKV_ERR_DEVICE: return "SKV_ERR_DEVICE";
    case SKV_ERR_UNSUPPORTED: return "SKV_ERR_UNSUPPORTED";
  }
  return "SKV_STATUS_UNKNOWN";
}

const char* skv_last_error(void) { return g_last_error.c_str(); }

skv_status skv_init(const skv_config* cfg, void* hip_stream, skv_ctx** out) {
  if (out == nullptr) return fail(SKV_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (cfg == nullptr) return fail(SKV_ERR_INVALID_ARG, "cfg is NULL");
  const skv_config& c = *cfg;
  if (c.n_layers < 1 || c.n_q_heads < 1 || c.n_kv_heads < 1 || c.tokens_per_frame < 1 || c.capacity < 0 ||
      c.max_frames < 1)
    return fail(SKV_ERR_INVALID_ARG, "sizes must be positive (capacity >= 0)");
  if (c.n_q_heads % c.n_kv_heads != 0) return fail(SKV_ERR_INVALID_ARG, "n_q_heads must be a multiple of n_kv_heads");
  if (c.head_dim != 64 && c.head_dim != 128) return fail(SKV_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (c.dtype != SKV_BF16 && c.dtype != SKV_F32) return fail(SKV_ERR_INVALID_ARG, "unknown dtype");
  if (!(c.softmax_scale >= 0.f) || !std::isfinite(c.softmax_scale))
    return fail(SKV_ERR_INVALID_ARG, "softmax_scale must be finite and >= 0");
  if (c.pos_offset < 0) return fail(SKV_ERR_INVALID_ARG, "pos_offset must be >= 0");
  if (c.max_decode_tokens < 0) return fail(SKV_ERR_INVALID_ARG, "max_decode_tokens must be >= 0");
  if (c.rope != SKV_ROPE_NONE && c.rope != SKV_ROPE_PLAIN && c.rope != SKV_ROPE_YARN)
    return fail(SKV_ERR_INVALID_ARG, "unknown rope kind");
  if (c.rope != SKV_ROPE_NONE && !(c.rope_theta > 0.f && std::isfinite(c.rope_theta)))
    return fail(SKV_ERR_INVALID_ARG, "rope_theta must be finite and > 0");
  if (c.rope == SKV_ROPE_YARN && (!(c.rope_factor >= 1.f && std::isfinite(c.rope_factor)) || c.rope_orig_max < 1))
    return fail(SKV_ERR_INVALID_ARG, "YaRN needs rope_factor >= 1 and rope_orig_max >= 1");
  const int64_t video_tokens = static_cast<int64_t>(c.max_frames) * c.tokens_per_frame;
  const int64_t max_tokens = video_tokens + c.max_decode_tokens;
  if (c.pos_offset + max_tokens >= (int64_t{1} << 31)) return fail(SKV_ERR_INVALID_ARG, "positions exceed int32");
  if (c.policy != SKV_POLICY_STATEKV && c.policy != SKV_POLICY_RECENT && c.policy != SKV_POLICY_FULL)
    return fail(SKV_ERR_INVALID_ARG, "unknown policy");
  if (c.split_refresh != 0 && c.split_refresh != 1) return fail(SKV_ERR_INVALID_ARG, "split_refresh must be 0 or 1");
  if (c.key_split_mode < 0 || c.key_split_mode > 2) return fail(SKV_ERR_INVALID_ARG, "key_split_mode must be 0, 1 or 2");
  const bool full = c.policy == SKV_POLICY_FULL;
  if (!full && static_cast<int64_t>(c.capacity) + c.tokens_per_frame > skv::kMaxPool)
    return fail(SKV_ERR_UNSUPPORTED, "capacity + tokens_per_frame exceeds 16384");
  const int64_t rows = static_cast<int64_t>(c.n_q_heads / c.n_kv_heads) * c.tokens_per_frame;
  if (rows >= (int64_t{1} << 30)) return fail(SKV_ERR_INVALID_ARG, "too many query rows per KV head");

  skv_ctx* ctx = new skv_ctx();
  ctx->cfg = c;
  if (full) ctx->cfg.capacity = 0;  // no compressed state: the context is the decode cache
  ctx->stream = static_cast<hipStream_t>(hip_stream);
  ctx->elem = c.dtype == SKV_BF16 ? 2 : 4;
  ctx->G = c.n_q_heads / c.n_kv_heads;
  const float scale = c.softmax_scale > 0.f ? c.softmax_scale : 1.0f / std::sqrt(static_cast<float>(c.head_dim));
  ctx->scale_log2 = scale * 1.4426950408889634f;
  ctx->use_mfma = c.dtype == SKV_BF16;
  ctx->tile_stride = ctx->use_mfma ? skv::plan_max_tiles(static_cast<int>(rows), skv::kMfmaRowsPerWave, skv::kMfmaWaves)
                                  : static_cast<int>((rows + skv::kSimpleRowsPerTile - 1) / skv::kSimpleRowsPerTile);
  ctx->pool_stride = ((ctx->cfg.capacity + c.tokens_per_frame + 63) / 64) * 64;
  ctx->row_bytes = static_cast<size_t>(c.head_dim) * ctx->elem;
  ctx->max_tokens = max_tokens;
  ctx->dec_row0 = video_tokens;
  if (c.max_decode_tokens > 0 && c.dtype == SKV_BF16) {
    const int64_t t_max = c.max_decode_tokens < skv::kDecodeMaxTokens ? c.max_decode_tokens : skv::kDecodeMaxTokens;
    const int64_t rb_max = (ctx->G * t_max + 31) / 32;
    const int64_t need = static_cast<int64_t>(c.n_layers) * c.n_kv_heads * rb_max;
    ctx->dec_items = static_cast<int>(need > skv::kDecodeItems ? need : skv::kDecodeItems);
  }
  ctx->last_pool.assign(c.n_layers, 0);

  hipError_t e = hipGetDevice(&ctx->device);
  if (e != hipSuccess) {
    delete ctx;
    return hip_fail(e, "hipGetDevice");
  }
  e = scratch_address(ctx->device, &ctx->scratch);
  if (e != hipSuccess) {
    delete ctx;
    return hip_fail(e, "hipGetSymbolAddress of the static scratch");
  }
  e = skv::prepare_kernels(c.head_dim, c.dtype == SKV_BF16, ctx->pool_stride);
  if (e != hipSuccess) {
    delete ctx;
    return hip_fail(e, "kernel attributes");
  }

  const size_t LH = static_cast<size_t>(c.n_layers) * c.n_kv_heads;
  // rows of new keys per (layer, KV head) in one step: a frame, or one decode call
  const int64_t new_rows =
      std::max<int64_t>(c.tokens_per_frame, std::min<int64_t>(c.max_decode_tokens, skv::kDecodeMaxTokens));
  const size_t B_state = static_cast<size_t>(ctx->cfg.capacity);
  const size_t state_bytes = LH * B_state * ctx->row_bytes;
  const size_t cache_bytes = LH * static_cast<size_t>(max_tokens) * ctx->row_bytes;
  struct Req { void** p; size_t bytes; };
  const Req reqs[] = {
      {&ctx->state_k, state_bytes},
      {&ctx->state_v, state_bytes},
      {reinterpret_cast<void**>(&ctx->state_pos), LH * B_state * sizeof(int32_t)},
      {reinterpret_cast<void**>(&ctx->state_score), LH * B_state * sizeof(float)},
      {&ctx->cache_k, cache_bytes},
      {&ctx->cache_v, cache_bytes},
      {reinterpret_cast<void**>(&ctx->partial), full ? 0 : LH * ctx->tile_stride * ctx->pool_stride * sizeof(float)},
      {reinterpret_cast<void**>(&ctx->pool_score), LH * ctx->pool_stride * sizeof(float)},
      {reinterpret_cast<void**>(&ctx->pool_pos), LH * ctx->pool_stride * sizeof(int32_t)},
      {reinterpret_cast<void**>(&ctx->admit_src), LH * c.tokens_per_frame * sizeof(int32_t)},
      {reinterpret_cast<void**>(&ctx->admit_dst), LH * c.tokens_per_frame * sizeof(int32_t)},
      {reinterpret_cast<void**>(&ctx->admit_count), LH * sizeof(int32_t)},
      {&ctx->rope_keys, c.rope == SKV_ROPE_NONE ? 0 : LH * static_cast<size_t>(new_rows) * ctx->row_bytes},
      {reinterpret_cast<void**>(&ctx->dec_part_o), static_cast<size_t>(ctx->dec_items) * 32 * c.head_dim * sizeof(float)},
      {reinterpret_cast<void**>(&ctx->dec_part_ml), static_cast<size_t>(ctx->dec_items) * 64 * sizeof(float)},
  };
  for (const Req& r : reqs) {
    const skv_status s = alloc(ctx, r.bytes, r.p);
    if (s != SKV_OK) {
      release(ctx);
      delete ctx;
      return s;
    }
    e = hipMemsetAsync(*r.p, 0, r.bytes > 0 ? r.bytes : 16, ctx->stream);
    if (e != hipSuccess) {
      release(ctx);
      delete ctx;
      return hip_fail(e, "hipMemsetAsync");
    }
  }
  skv_status ps = build_plans(ctx, static_cast<int>(rows));
  if (ps == SKV_OK) ps = build_rope_table(ctx);
  if (ps != SKV_OK) {
    release(ctx);
    delete ctx;
    return ps;
  }
  *out = ctx;
  return SKV_OK;
}

}  // extern "C"

namespace {

// Argument, order and capacity checks of a frame step (nothing enqueued).
skv_status check_frame_step(skv_ctx* ctx, int32_t layer_begin, int32_t layer_count, const void* q, const void* k,
                            const void* v, void* out) {
  if (ctx == nullptr) return fail(SKV_ERR_INVALID_ARG, "ctx is NULL");
  if (q == nullptr || k == nullptr || v == nullptr || out == nullptr)
    return fail(SKV_ERR_INVALID_ARG, "q, k, v and out must be device pointers");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
    return fail(SKV_ERR_INVALID_ARG, "q, k, v and out must be 16-byte aligned");
  const skv_config& c = ctx->cfg;
  if (layer_count < 1 || layer_begin < 0 || layer_begin + layer_count > c.n_layers)
    return fail(SKV_ERR_INVALID_ARG, "layer range outside [0, n_layers)");
  if (ctx->broken) return fail(SKV_ERR_DEVICE, "an earlier step failed part-way; call skv_reset or skv_seek");
  if (layer_begin != ctx->next_layer)
    return fail(SKV_ERR_ORDER, "expected layer_begin = " + std::to_string(ctx->next_layer));
  if (ctx->dec_next_layer != 0) return fail(SKV_ERR_ORDER, "a decode call is half done");
  if (ctx->frame >= c.max_frames) return fail(SKV_ERR_CAPACITY, "decode cache is full (max_frames reached)");
  return SKV_OK;
}

// Whether this step records timing events (and takes the next event slots).
bool take_timing(skv_ctx* ctx) {
  if (ctx->timing_n >= ctx->timing_max) return false;
  return ctx->timing_seen++ % ctx->timing_stride == 0;
}

// Enqueues, as a launch of its own, the selection a one-layer call left for a
// later output launch (if any).
hipError_t flush_pending(skv_ctx* ctx) {
  if (!ctx->pend) return hipSuccess;
  ctx->pend = false;
  return skv::launch_refresh(ctx->pend_ra, ctx->stream);
}

// Scratch bytes a frame step of layer_count layers needs (each buffer 256-byte aligned),
// and the buffers carved from `base` when base is not null.
size_t carve_scratch(const skv_ctx* ctx, int32_t layer_count, char* base, StepScratch* sc) {
  const skv_config& c = ctx->cfg;
  const size_t LH = static_cast<size_t>(layer_count) * c.n_kv_heads;
  const size_t rows = static_cast<size_t>(ctx->G) * c.tokens_per_frame;
  const size_t n_ks = static_cast<size_t>(ctx->plans[static_cast<size_t>(layer_count - 1)].n_ks);
  const bool full = c.policy == SKV_POLICY_FULL;
  const size_t sizes[6] = {
      full ? 0 : LH * ctx->tile_stride * ctx->pool_stride * sizeof(float),
      n_ks > 1 ? LH * n_ks * rows * 2 * sizeof(float) : 0,
      n_ks > 1 ? n_ks * layer_count * c.n_q_heads * c.tokens_per_frame * c.head_dim * sizeof(float) : 0,
      LH * c.tokens_per_frame * sizeof(int32_t),
      LH * c.tokens_per_frame * sizeof(int32_t),
      LH * sizeof(int32_t)};
  void* ptrs[6];
  size_t off = 0;
  for (int i = 0; i < 6; ++i) {
    ptrs[i] = sizes[i] > 0 && base != nullptr ? base + off : nullptr;
    off += (sizes[i] + 255) / 256 * 256;
  }
  if (sc != nullptr) {
    sc->own_layers = false;
    sc->partial = static_cast<float*>(ptrs[0]);
    sc->split_stats = static_cast<float*>(ptrs[1]);
    sc->split_out = static_cast<float*>(ptrs[2]);
    sc->admit_src = static_cast<int32_t*>(ptrs[3]);
    sc->admit_dst = static_cast<int32_t*>(ptrs[4]);
    sc->admit_count = static_cast<int32_t*>(ptrs[5]);
  }
  return off;
}

// The launch sequence of a checked frame step, with the per-call buffers in `sc`.
skv_status enqueue_frame_step(skv_ctx* ctx, int32_t layer_begin, int32_t layer_count, const void* q, const void* k,
                              const void* v, void* out, const StepScratch& sc) {
  const skv_config& c = ctx->cfg;
  const int T = c.tokens_per_frame, Hkv = c.n_kv_heads, B = c.capacity, d = c.head_dim;
  const int S = state_size(ctx, ctx->frame);
  const int32_t pos0 = static_cast<int32_t>(c.pos_offset + ctx->frame * T);
  const size_t lh0 = static_cast<size_t>(layer_begin) * Hkv;
  const size_t rb = ctx->row_bytes;

  const bool timing = take_timing(ctx);
  hipEvent_t* ev = timing ? &ctx->events[static_cast<size_t>(ctx->timing_n) * (SKV_N_STAGES + 1)] : nullptr;
  uint8_t* rec = timing ? &ctx->recorded[static_cast<size_t>(ctx->timing_n)] : nullptr;
  if (timing) *rec = 0;
  // event i opens stage i (and closes the stage before it); a stage whose event is not
  // recorded reads 0
  auto mark = [&](int i) -> hipError_t {
    if (!timing) return hipSuccess;
    *rec |= static_cast<uint8_t>(1u << i);
    return hipEventRecord(ev[i], ctx->stream);
  };

  // with RoPE every later reader takes the frame's keys rotated (launched first below)
  const void* k_used = ctx->rope_tab != nullptr ? ctx->rope_keys : k;

  skv::AttnArgs aa{};
  aa.q = q;
  aa.kf = k_used;
  aa.vf = v;
  const bool full = c.policy == SKV_POLICY_FULL;
  if (full) {  // every earlier token, from the decode cache
    aa.ks = static_cast<char*>(ctx->cache_k) + lh0 * ctx->max_tokens * rb;
    aa.vs = static_cast<char*>(ctx->cache_v) + lh0 * ctx->max_tokens * rb;
    aa.kv_rows = static_cast<int>(ctx->max_tokens);
  } else {
    aa.ks = static_cast<char*>(ctx->state_k) + lh0 * B * rb;
    aa.vs = static_cast<char*>(ctx->state_v) + lh0 * B * rb;
    aa.kv_rows = B;
  }
  aa.out = out;
  const skv_ctx::Plan& plan = ctx->plans[static_cast<size_t>(layer_count - 1)];
  aa.partial = full ? nullptr : sc.partial;
  aa.work = plan.work;
  aa.n_work = plan.n_work;
  aa.rope_tab = ctx->rope_tab;
  aa.rope_pos0 = static_cast<int>(ctx->frame * T);
  aa.n_layers = layer_count;
  aa.H_q = c.n_q_heads;
  aa.H_kv = Hkv;
  aa.G = ctx->G;
  aa.T = T;
  aa.B = B;
  aa.S = full ? static_cast<int>(ctx->frame * T) : S;
  aa.tile_stride = ctx->tile_stride;
  aa.pool_stride = ctx->pool_stride;
  aa.scale_log2 = ctx->scale_log2;
  aa.mode = 0;
  aa.n_ks = plan.n_ks;
  aa.stats = sc.split_stats;
  aa.opart = sc.split_out;

  skv::RefreshArgs ra{};
  ra.partial = aa.partial;
  ra.lg_tiles = plan.tiles;
  ra.tile_stride = ctx->tile_stride;
  ra.pool_stride = ctx->pool_stride;
  ra.kf = k_used;
  ra.vf = v;
  ra.kf_rows = T;
  ra.select = !full;
  ra.append = true;
  ra.ks = static_cast<char*>(ctx->state_k) + lh0 * B * rb;
  ra.vs = static_cast<char*>(ctx->state_v) + lh0 * B * rb;
  ra.state_pos = ctx->state_pos + lh0 * B;
  ra.state_score = ctx->state_score + lh0 * B;
  ra.pool_score = ctx->pool_score + lh0 * ctx->pool_stride;
  ra.pool_pos = ctx->pool_pos + lh0 * ctx->pool_stride;
  ra.admit_src = sc.admit_src;
  ra.admit_dst = sc.admit_dst;
  ra.admit_count = sc.admit_count;
  ra.split_update = false;
  ra.ck = static_cast<char*>(ctx->cache_k) + lh0 * ctx->max_tokens * rb;
  ra.cv = static_cast<char*>(ctx->cache_v) + lh0 * ctx->max_tokens * rb;
  ra.max_tokens = ctx->max_tokens;
  ra.first_row = ctx->frame * T;
  ra.n_layers = layer_count;
  ra.H_kv = Hkv;
  ra.T = T;
  ra.B = B;
  ra.S = S;
  ra.row_bytes = static_cast<int>(rb);
  ra.frame_pos0 = pos0;
  ra.inv_T = 1.0f / static_cast<float>(T);
  ra.mode = c.policy == SKV_POLICY_RECENT ? 1 : 0;
  // key-split plans: the refresh launch also adds the attention's output shares
  ra.n_ks = ctx->use_mfma && !full ? plan.n_ks : 1;
  ra.opart = sc.split_out;
  ra.out = out;
  ra.out_elems = static_cast<int64_t>(layer_count) * c.n_q_heads * T * d;
  // one group of four output values per combine thread; beside selection
  // workgroups at most 128 combine workgroups, which leave the memory system to
  // the selections' latency-bound loads
  const int64_t comb_wgs = (ra.out_elems / 4 + skv::kSelectThreads - 1) / skv::kSelectThreads;

  // A key-split call of a multi-layer context (one layer of the real-model calling
  // pattern) leaves its selection and state update to the output launch of the
  // next such call on other layers, where they run beside that call's attention
  // instead of after the output sum; that call carries it (or, when none does,
  // the next use of the state enqueues it on its own).  The frame's rows are
  // then read back from the decode cache, since the caller's k and v may be
  // reused once this call's work is done.
  const bool key_split = ctx->use_mfma && !full && plan.n_ks > 1;
  const bool defer = key_split && sc.own_layers && !c.split_refresh && layer_count < c.n_layers &&
                     skv::selection_lds_bytes(S + T) <= skv::attention_mfma_lds_bytes(d);
  const bool carry = ctx->pend && key_split &&
                     (ctx->pend_lb + ctx->pend_lc <= layer_begin || layer_begin + layer_count <= ctx->pend_lb);
  ra.n_comb = static_cast<int>(std::min<int64_t>(defer ? 1024 : 128, comb_wgs));
  hipError_t e = ctx->pend && !carry ? flush_pending(ctx) : hipSuccess;
  if (e == hipSuccess) e = mark(0);
  if (e == hipSuccess && ctx->rope_tab != nullptr)
    e = skv::launch_rope_keys(k, ctx->rope_keys, layer_count * Hkv, T, static_cast<int>(rb), ctx->elem, ctx->rope_tab,
                              static_cast<int>(ctx->frame * T), ctx->stream);
  if (e == hipSuccess) {
    if (!ctx->use_mfma) {
      e = skv::launch_attention_simple_f32(aa, d, ctx->stream);
    } else if (full) {
      e = skv::launch_attention_full_bf16(aa, d, ctx->stream);
    } else if (plan.n_ks > 1) {  // key-split plan: statistics and output shares (their sum below)
      if (carry) {
        aa.n_sel = ctx->pend_lc * Hkv;
        aa.sel = ctx->pend_ra;
      }
      if (c.key_split_mode == 1) {  // two launches
        aa.mode = 1;
        e = skv::launch_attention_mfma_bf16(aa, d, ctx->stream);
        aa.mode = 2;
        if (e == hipSuccess) e = skv::launch_attention_mfma_bf16(aa, d, ctx->stream);
      } else {  // one launch; its workgroups exchange the statistics (mode 3) or each computes all (4)
        aa.mode = c.key_split_mode == 2 ? 4 : 3;
        aa.flags = ctx->ks_flags;
        aa.epoch = ++ctx->ks_epoch;
        if (aa.epoch == 0u) aa.epoch = ++ctx->ks_epoch;  // 0 is the flags' initial value
        aa.wait_ticks = ctx->ks_wait_ticks;
        e = skv::launch_attention_mfma_bf16(aa, d, ctx->stream);
      }
      if (e == hipSuccess && carry) ctx->pend = false;
    } else {
      e = skv::launch_attention_mfma_bf16(aa, d, ctx->stream);
    }
  }
  if (e == hipSuccess) e = mark(1);
  if (c.split_refresh) {
    // selection (with a key-split plan's output sum), state update, append: three launches
    skv::RefreshArgs rs = ra;
    rs.append = false;
    rs.split_update = true;
    if (e == hipSuccess) e = skv::launch_refresh(rs, ctx->stream);
    if (e == hipSuccess) e = mark(2);
    if (e == hipSuccess && !full) e = skv::launch_refresh_update(ra, ctx->stream);
    if (e == hipSuccess) e = mark(3);
    if (e == hipSuccess) e = skv::launch_refresh_append(ra, ctx->stream);
  } else if (defer) {
    skv::RefreshArgs now = ra;  // the output sum and the append; the selection waits
    now.select = false;
    if (e == hipSuccess) e = skv::launch_refresh(now, ctx->stream);
    if (e == hipSuccess) {
      ctx->pend_ra = ra;
      ctx->pend_ra.append = false;
      ctx->pend_ra.n_ks = 1;
      ctx->pend_ra.kf = static_cast<const char*>(ra.ck) + static_cast<size_t>(ra.first_row) * rb;
      ctx->pend_ra.vf = static_cast<const char*>(ra.cv) + static_cast<size_t>(ra.first_row) * rb;
      ctx->pend_ra.kf_rows = ctx->max_tokens;
      ctx->pend_lb = layer_begin;
      ctx->pend_lc = layer_count;
      ctx->pend = true;
    }
  } else {
    if (e == hipSuccess) e = skv::launch_refresh(ra, ctx->stream);
  }
  if (e == hipSuccess) e = mark(4);
  if (e != hipSuccess) {
    ctx->broken = true;  // earlier launches of this step may be enqueued
    return hip_fail(e, "frame step launch");
  }
  if (timing) ++ctx->timing_n;

  for (int l = layer_begin; l < layer_begin + layer_count; ++l) ctx->last_pool[l] = full ? 0 : S + T;
  ctx->next_layer += layer_count;
  if (ctx->next_layer == c.n_layers) {
    ctx->next_layer = 0;
    ++ctx->frame;
  }
  return SKV_OK;
}

}  // namespace

extern "C" {

skv_status skv_frame_step(skv_ctx* ctx, int32_t layer_begin, int32_t layer_count, const void* q, const void* k,
                          const void* v, void* out) {
  const skv_status s = check_frame_step(ctx, layer_begin, layer_count, q, k, v, out);
  if (s != SKV_OK) return s;
  const skv_config& c = ctx->cfg;
  const size_t lh0 = static_cast<size_t>(layer_begin) * c.n_kv_heads;
  StepScratch sc;
  sc.own_layers = true;
  sc.partial = ctx->partial != nullptr ? ctx->partial + lh0 * ctx->tile_stride * ctx->pool_stride : nullptr;
  sc.split_stats = ctx->split_stats;
  sc.split_out = ctx->split_out;
  sc.admit_src = ctx->admit_src + lh0 * c.tokens_per_frame;
  sc.admit_dst = ctx->admit_dst + lh0 * c.tokens_per_frame;
  sc.admit_count = ctx->admit_count + lh0;
  return enqueue_frame_step(ctx, layer_begin, layer_count, q, k, v, out, sc);
}

skv_status skv_frame_step_noalloc(skv_ctx* ctx, int32_t layer_begin, int32_t layer_count, const void* q,
                                  const void* k, const void* v, void* out) {
  const skv_status s = check_frame_step(ctx, layer_begin, layer_count, q, k, v, out);
  if (s != SKV_OK) return s;
  const size_t need = carve_scratch(ctx, layer_count, nullptr, nullptr);
  if (need > kScratchBytes)
    return fail(SKV_ERR_UNSUPPORTED, "this call needs " + std::to_string(need) + " bytes of scratch, the static " +
                                         "scratch holds " + std::to_string(kScratchBytes) +
                                         "; step fewer layers per call or use skv_frame_step");
  StepScratch sc;
  carve_scratch(ctx, layer_count, static_cast<char*>(ctx->scratch), &sc);
  return enqueue_frame_step(ctx, layer_begin, layer_count, q, k, v, out, sc);
}

skv_status skv_decode_step(skv_ctx* ctx, int32_t layer_begin, int32_t layer_count, int32_t n_tokens,
                           const void* q, const void* k, const void* v, void* out) {
  if (ctx == nullptr) return fail(SKV_ERR_INVALID_ARG, "ctx is NULL");
  if (q == nullptr || k == nullptr || v == nullptr || out == nullptr)
    return fail(SKV_ERR_INVALID_ARG, "q, k, v and out must be device pointers");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
    return fail(SKV_ERR_INVALID_ARG, "q, k, v and out must be 16-byte aligned");
  const skv_config& c = ctx->cfg;
  if (layer_count < 1 || layer_begin < 0 || layer_begin + layer_count > c.n_layers)
    return fail(SKV_ERR_INVALID_ARG, "layer range outside [0, n_layers)");
  if (n_tokens < 1 || n_tokens > skv::kDecodeMaxTokens)
    return fail(SKV_ERR_INVALID_ARG, "n_tokens must be in [1, " + std::to_string(skv::kDecodeMaxTokens) + "]");
  if (c.dtype != SKV_BF16) return fail(SKV_ERR_UNSUPPORTED, "decoding is implemented for bf16 contexts");
  if (ctx->broken) return fail(SKV_ERR_DEVICE, "an earlier step failed part-way; call skv_reset or skv_seek");
  if (ctx->next_layer != 0) return fail(SKV_ERR_ORDER, "a frame is half done");
  if (layer_begin != ctx->dec_next_layer)
    return fail(SKV_ERR_ORDER, "expected layer_begin = " + std::to_string(ctx->dec_next_layer));
  if (ctx->dec_next_layer != 0 && n_tokens != ctx->dec_pending)
    return fail(SKV_ERR_INVALID_ARG, "n_tokens differs from the decode call in progress");
  if (ctx->n_decoded + n_tokens > c.max_decode_tokens)
    return fail(SKV_ERR_CAPACITY, "more tokens than max_decode_tokens");

  const int Hkv = c.n_kv_heads, d = c.head_dim, t = n_tokens;
  const size_t lh0 = static_cast<size_t>(layer_begin) * Hkv;
  const size_t rb = ctx->row_bytes;
  const int S = static_cast<int>(ctx->frame * c.tokens_per_frame);
  const int n_dec = static_cast<int>(ctx->n_decoded);
  const int n_keys = S + n_dec + t;
  const int LH = layer_count * Hkv;
  const int n_rb = (ctx->G * t + 31) / 32;
  const int per = std::max(1, ctx->dec_items / (LH * n_rb));  // splits per (layer-head, row block)
  const int split = std::max(256, ((n_keys + per - 1) / per + 31) / 32 * 32);

  // with RoPE the kernels take the new tokens' keys rotated (launched first below)
  const void* k_used = ctx->rope_tab != nullptr ? ctx->rope_keys : k;

  skv::DecodeArgs da;
  da.q = q;
  da.kn = k_used;
  da.vn = v;
  da.ck = static_cast<char*>(ctx->cache_k) + lh0 * ctx->max_tokens * rb;
  da.cv = static_cast<char*>(ctx->cache_v) + lh0 * ctx->max_tokens * rb;
  da.out = out;
  da.part_o = ctx->dec_part_o;
  da.part_ml = ctx->dec_part_ml;
  da.max_tokens = ctx->max_tokens;
  da.dec_row0 = ctx->dec_row0;
  da.n_layers = layer_count;
  da.H_q = c.n_q_heads;
  da.H_kv = Hkv;
  da.G = ctx->G;
  da.t = t;
  da.S = S;
  da.n_dec = n_dec;
  da.n_rb = n_rb;
  da.split = split;
  da.n_split = (n_keys + split - 1) / split;
  da.scale_log2 = ctx->scale_log2;
  da.rope_tab = ctx->rope_tab;
  da.rope_pos0 = S + n_dec;

  // append of the new tokens' K/V to D's decode rows (the refresh kernel's append-only mode)
  skv::RefreshArgs ra{};
  ra.kf = k_used;
  ra.vf = v;
  ra.ck = static_cast<char*>(ctx->cache_k) + lh0 * ctx->max_tokens * rb;
  ra.cv = static_cast<char*>(ctx->cache_v) + lh0 * ctx->max_tokens * rb;
  ra.max_tokens = ctx->max_tokens;
  ra.first_row = ctx->dec_row0 + n_dec;
  ra.n_layers = layer_count;
  ra.H_kv = Hkv;
  ra.T = t;
  ra.row_bytes = static_cast<int>(rb);
  ra.kf_rows = t;
  ra.select = false;  // append only
  ra.append = true;

  const bool timing = take_timing(ctx);
  hipEvent_t* ev = timing ? &ctx->events[static_cast<size_t>(ctx->timing_n) * (SKV_N_STAGES + 1)] : nullptr;
  uint8_t* rec = timing ? &ctx->recorded[static_cast<size_t>(ctx->timing_n)] : nullptr;
  if (timing) *rec = 0;
  // event i opens stage i (and closes the stage before it); a stage whose event is not
  // recorded reads 0
  auto mark = [&](int i) -> hipError_t {
    if (!timing) return hipSuccess;
    *rec |= static_cast<uint8_t>(1u << i);
    return hipEventRecord(ev[i], ctx->stream);
  };
  hipError_t e = mark(0);
  if (e == hipSuccess && ctx->rope_tab != nullptr)
    e = skv::launch_rope_keys(k, ctx->rope_keys, LH, t, static_cast<int>(rb), ctx->elem, ctx->rope_tab, S + n_dec,
                              ctx->stream);
  if (e == hipSuccess) e = skv::launch_decode_bf16(da, d, ctx->stream);
  if (e == hipSuccess) e = mark(3);
  if (e == hipSuccess) e = skv::launch_refresh(ra, ctx->stream);
  if (e == hipSuccess) e = mark(4);
  if (e != hipSuccess) {
    ctx->broken = true;  // earlier launches of this step may be enqueued
    return hip_fail(e, "decode step launch");
  }
  if (timing) ++ctx->timing_n;

  ctx->dec_pending = t;
  ctx->dec_next_layer += layer_count;
  if (ctx->dec_next_layer == c.n_layers) {
    ctx->dec_next_layer = 0;
    ctx->n_decoded += t;
    ctx->dec_pending = 0;
  }
  return SKV_OK;
}

skv_status skv_state_view(skv_ctx* ctx, int32_t layer, skv_state_view_t* out) {
  if (ctx == nullptr || out == nullptr) return fail(SKV_ERR_INVALID_ARG, "NULL argument");
  const skv_config& c = ctx->cfg;
  if (layer < 0 || layer >= c.n_layers) return fail(SKV_ERR_INVALID_ARG, "layer out of range");
  const size_t lh = static_cast<size_t>(layer) * c.n_kv_heads;
  if (ctx->pend) {  // a deferred selection is enqueued before anyone reads the state
    const hipError_t e = flush_pending(ctx);
    if (e != hipSuccess) {
      ctx->broken = true;
      return hip_fail(e, "deferred selection launch");
    }
  }
  const int done = layer_frames_done(ctx, layer);
  out->k = static_cast<char*>(ctx->state_k) + lh * c.capacity * ctx->row_bytes;
  out->v = static_cast<char*>(ctx->state_v) + lh * c.capacity * ctx->row_bytes;
  out->pos = ctx->state_pos + lh * c.capacity;
  out->score = ctx->state_score + lh * c.capacity;
  out->size = state_size(ctx, done);
  out->capacity = c.capacity;
  out->frame = done;
  out->pool_score = ctx->pool_score + lh * ctx->pool_stride;
  out->pool_pos = ctx->pool_pos + lh * ctx->pool_stride;
  out->pool_size = ctx->last_pool[layer];
  out->pool_stride = ctx->pool_stride;
  return SKV_OK;
}

skv_status skv_decode_cache_view(skv_ctx* ctx, int32_t layer, skv_cache_view_t* out) {
  if (ctx == nullptr || out == nullptr) return fail(SKV_ERR_INVALID_ARG, "NULL argument");
  const skv_config& c = ctx->cfg;
  if (layer < 0 || layer >= c.n_layers) return fail(SKV_ERR_INVALID_ARG, "layer out of range");
  const size_t lh = static_cast<size_t>(layer) * c.n_kv_heads;
  out->k = static_cast<char*>(ctx->cache_k) + lh * ctx->max_tokens * ctx->row_bytes;
  out->v = static_cast<char*>(ctx->cache_v) + lh * ctx->max_tokens * ctx->row_bytes;
  out->n_tokens = static_cast<int64_t>(layer_frames_done(ctx, layer)) * c.tokens_per_frame;
  out->max_tokens = ctx->max_tokens;
  out->n_kv_heads = c.n_kv_heads;
  out->head_dim = c.head_dim;
  out->decode_row0 = ctx->dec_row0;
  out->decode_tokens = ctx->n_decoded + (layer < ctx->dec_next_layer ? ctx->dec_pending : 0);
  return SKV_OK;
}

skv_status skv_reset(skv_ctx* ctx) {
  if (ctx == nullptr) return fail(SKV_ERR_INVALID_ARG, "ctx is NULL");
  ctx->broken = false;
  ctx->pend = false;  // the state starts empty; a deferred selection is void
  ctx->frame = 0;
  ctx->next_layer = 0;
  ctx->n_decoded = 0;
  ctx->dec_next_layer = 0;
  ctx->dec_pending = 0;
  std::fill(ctx->last_pool.begin(), ctx->last_pool.end(), 0);
  return SKV_OK;
}

skv_status skv_seek(skv_ctx* ctx, int64_t frame) {
  if (ctx == nullptr) return fail(SKV_ERR_INVALID_ARG, "ctx is NULL");
  if (frame < 0 || frame >= ctx->cfg.max_frames) return fail(SKV_ERR_INVALID_ARG, "frame out of range");
  ctx->broken = false;
  ctx->pend = false;  // the state is the caller's to set; a deferred selection is void
  ctx->frame = frame;
  ctx->next_layer = 0;
  ctx->n_decoded = 0;
  ctx->dec_next_layer = 0;
  ctx->dec_pending = 0;
  return SKV_OK;
}

skv_status skv_timing_start(skv_ctx* ctx, int32_t max_steps) {
  if (ctx == nullptr || max_steps < 1) return fail(SKV_ERR_INVALID_ARG, "bad timing request");
  for (hipEvent_t e : ctx->events) (void)hipEventDestroy(e);
  ctx->events.assign(static_cast<size_t>(max_steps) * (SKV_N_STAGES + 1), nullptr);
  ctx->recorded.assign(static_cast<size_t>(max_steps), 0);
  for (auto& e : ctx->events) {
    const hipError_t r = hipEventCreate(&e);
    if (r != hipSuccess) {
      ctx->timing_max = 0;
      return hip_fail(r, "hipEventCreate");
    }
  }
  ctx->timing_max = max_steps;
  ctx->timing_n = 0;
  ctx->timing_stride = 1;
  ctx->timing_seen = 0;
  return SKV_OK;
}

skv_status skv_timing_stride(skv_ctx* ctx, int32_t stride) {
  if (ctx == nullptr || stride < 1) return fail(SKV_ERR_INVALID_ARG, "bad timing stride");
  ctx->timing_stride = stride;
  return SKV_OK;
}

skv_status skv_timing_stop(skv_ctx* ctx, int32_t* n_steps, float* ms, int32_t ms_capacity) {
  if (ctx == nullptr || n_steps == nullptr || ms == nullptr) return fail(SKV_ERR_INVALID_ARG, "NULL argument");
  hipError_t e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  const int n = ctx->timing_n < ms_capacity / SKV_N_STAGES ? ctx->timing_n : ms_capacity / SKV_N_STAGES;
  for (int i = 0; i < n; ++i) {
    hipEvent_t* ev = &ctx->events[static_cast<size_t>(i) * (SKV_N_STAGES + 1)];
    const unsigned rec = ctx->recorded[static_cast<size_t>(i)];
    for (int s = 0; s < SKV_N_STAGES; ++s) {
      float t = 0.f;
      int next = s + 1;  // the stage ends at the next recorded event
      while (next <= SKV_N_STAGES && !(rec >> next & 1u)) ++next;
      if ((rec >> s & 1u) && next <= SKV_N_STAGES) {
        e = hipEventElapsedTime(&t, ev[s], ev[next]);
        if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
      }
      ms[i * SKV_N_STAGES + s] = t;
    }
  }
  *n_steps = n;
  for (hipEvent_t ev : ctx->events) (void)hipEventDestroy(ev);
  ctx->events.clear();
  ctx->timing_max = ctx->timing_n = 0;
  return SKV_OK;
}

void skv_destroy(skv_ctx* ctx) {
  if (ctx == nullptr) return;
  release(ctx);
  delete ctx;
}

}  // extern "C"

namespace skv {

hipError_t prepare_kernels(int head_dim, bool bf16, int pool_stride) {
  (void)head_dim;
  hipError_t e = prepare_refresh(pool_stride);
  if (e != hipSuccess) return e;
  if (bf16) e = prepare_attention_mfma();
  if (e != hipSuccess) return e;
  if (bf16) e = prepare_attention_full();
  return e;
}

}  // namespace skv
