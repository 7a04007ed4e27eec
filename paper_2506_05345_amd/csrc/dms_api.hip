// C-ABI entry points of libdms: configuration checks, buffer layout, the host
// context and the per-call argument validation that runs before any HIP call.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "dms_common.h"
#include "dms_fp8.h"
#include "dms_train.h"

namespace dms {

int validate_config(const dms_config& c) {
  if (c.num_layers < 1 || c.max_seqs < 1 || c.max_seqs > kMaxSeqs) return DMS_ERR_INVALID;
  if (c.num_kv_heads < 1 || c.group_size < 1 || c.window < 1) return DMS_ERR_INVALID;
  if (c.group_size > (c.kv_format == DMS_KV_MLA ? kMlaMaxGroup : kMaxGroup)) return DMS_ERR_UNSUPPORTED;
  if (c.head_dim < 1) return DMS_ERR_INVALID;
  if (c.kv_format == DMS_KV_MLA) {
    // latent rows: one KV head, caller decisions, no page retrieval
    if (c.head_dim != kMlaDim) return DMS_ERR_UNSUPPORTED;
    if (c.num_kv_heads != 1 || c.decision_source != DMS_DECIDE_CALLER || c.quest_page_budget != 0)
      return DMS_ERR_UNSUPPORTED;
  } else if (c.head_dim != 64 && c.head_dim != 128) {
    return DMS_ERR_UNSUPPORTED;
  }
  // Split-K partial accumulators (one g x row-width float32 block per
  // partial, kMaxWaves + max_seqs * Hkv partials, kMaxMlaUnits + max_seqs for
  // latent rows) are addressed through a buffer resource with 32-bit byte
  // offsets, so their area must stay below 2 GiB for every page format.
  {
    const bool mla_rows = c.kv_format == DMS_KV_MLA;
    const int64_t row = mla_rows ? kMlaLatent : c.head_dim;
    const int64_t partials = (mla_rows ? kMaxMlaUnits : kMaxWaves) +
                             static_cast<int64_t>(c.max_seqs) * c.num_kv_heads;
    if (partials * c.group_size * row * 4 >= (int64_t(1) << 31)) return DMS_ERR_UNSUPPORTED;
  }
  if (c.page_size != 32 && c.page_size != 64 && c.page_size != 128 && c.page_size != 256)
    return DMS_ERR_INVALID;
  if (c.num_pages < 1 || c.max_pages_per_head < 1 || c.max_chunk_tokens < 0) return DMS_ERR_INVALID;
  if (!(c.softmax_scale <= 0.0f || isfinite(c.softmax_scale))) return DMS_ERR_INVALID;
  if (isnan(c.softmax_scale)) return DMS_ERR_INVALID;
  if (c.eviction != DMS_EVICT_DELAYED && c.eviction != DMS_EVICT_IMMEDIATE) return DMS_ERR_INVALID;
  if (c.decision_source != DMS_DECIDE_CALLER && c.decision_source != DMS_DECIDE_QUERY)
    return DMS_ERR_INVALID;
  if (c.decision_source == DMS_DECIDE_QUERY && !isfinite(c.decision_bias)) return DMS_ERR_INVALID;
  if (c.kv_format != DMS_KV_BF16 && c.kv_format != DMS_KV_FP8 && c.kv_format != DMS_KV_MLA)
    return DMS_ERR_INVALID;
  if (c.quest_page_budget < 0 || c.quest_page_budget > c.max_pages_per_head) return DMS_ERR_INVALID;
  if (c.quest_page_budget > 0 && c.max_pages_per_head > 4096) return DMS_ERR_UNSUPPORTED;
  // slot and page indices are int32 on the device
  if (static_cast<int64_t>(c.max_pages_per_head) * c.page_size >= (int64_t(1) << 31)) return DMS_ERR_INVALID;
  if (static_cast<int64_t>(c.max_seqs) * c.num_kv_heads > (int64_t(1) << 22)) return DMS_ERR_INVALID;
  if (static_cast<int64_t>(c.max_chunk_tokens) * c.num_kv_heads >= (int64_t(1) << 31)) return DMS_ERR_INVALID;
  return DMS_OK;
}

Layout make_layout(const dms_config& c) {
  Layout lo{};
  const size_t S = c.max_seqs, H = c.num_kv_heads, w = c.window;
  const size_t maxp = c.max_pages_per_head, P = c.page_size, D = c.head_dim;
  lo.max_slots = static_cast<int>(maxp * P);
  lo.max_heads = static_cast<int>(S * H);
  const bool mla_rows = c.kv_format == DMS_KV_MLA;
  lo.max_partials = (mla_rows ? kMaxMlaUnits : kMaxWaves) + lo.max_heads;
  lo.ml_stride = mla_rows ? (c.group_size + kMaxGroup - 1) / kMaxGroup * kMaxGroup : kMaxGroup;
  lo.head_groups = mla_rows ? (c.group_size + kMaxGroup - 1) / kMaxGroup : 1;
  // meta
  lo.status = 0;
  lo.layer0 = kAlign;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, kAlign); return o; };
  lo.pos = take(S * 4);
  lo.len = take(S * H * 4);
  lo.ring = take(S * H * w * 4);
  lo.page_table = take(S * H * maxp * 4);
  lo.slot_meta = take(S * H * maxp * P * 4);
  lo.stack = take(static_cast<size_t>(c.num_pages) * 4);
  lo.top = take(4);
  lo.page_bounds = c.quest_page_budget > 0 ? take(static_cast<size_t>(c.num_pages) * 2 * D * 2) : 0;
  lo.layer_stride = off;
  lo.meta_bytes = lo.layer0 + lo.layer_stride * c.num_layers;
  // pool
  lo.page_bytes = c.kv_format == DMS_KV_FP8   ? P / 32 * fp8_tile_bytes(static_cast<int>(D))
                  : c.kv_format == DMS_KV_MLA ? P / 32 * mla_tile_bytes(static_cast<int>(D))
                                              : 2 * P * D * 2;
  lo.pool_bytes = lo.page_bytes * static_cast<size_t>(c.num_pages);
  // workspace
  off = 0;
  const size_t NH = lo.max_heads, NP = lo.max_partials;
  lo.ws_head_desc = take(NH * sizeof(HeadDesc));
  lo.ws_cum_tiles = take((NH + 1) * 4);
  lo.ws_part_ml = take(NP * lo.ml_stride * 8);
  const size_t Dout = c.kv_format == DMS_KV_MLA ? kMlaLatent : D;   // output row width
  lo.ws_part_acc = take(NP * c.group_size * Dout * 4);
  lo.ws_wave_bounds = take((kMaxWaves + 1) * 4);
  lo.ws_wave_desc = take(kMaxWaves * 2 * sizeof(int4));   // per decode wave: first segment
  lo.ws_head_waves = take(NH * sizeof(int4));              // per head: waves holding its tiles
  lo.ws_head_cnt = take(NH * lo.head_groups * 4);
  lo.ws_plan_ctr = take(16);
  lo.ws_ck_need = take(NH * 4);
  lo.ws_ck_fresh = take(NH * 4);
  lo.ws_ck_base = take(NH * 4);
  lo.ws_ck_pos0 = take(S * 4);
  lo.ws_ck_err = take(16);
  lo.ws_ck_slot = take(static_cast<size_t>(c.max_chunk_tokens) * H * 4);
  lo.ws_pf_cum = take((NH + 1) * 4);
  lo.ws_pf_meta = take(static_cast<size_t>(c.max_chunk_tokens) * H * 4);
  // prefill: chunk keys / values (latent rows) and the compacted kept ones,
  // in the pool's tile layout; sequence i of a call starts at tile
  // cu[i] / 32 + i
  lo.pf_tiles_per_head = static_cast<int>((static_cast<size_t>(c.max_chunk_tokens) + 31) / 32 + S + 1);
  lo.ws_pf_tiles = take(2 * H * static_cast<size_t>(lo.pf_tiles_per_head) * D *
                        (c.kv_format == DMS_KV_MLA ? 64 : 128));
  lo.ws_pf_tmeta = take(2 * H * static_cast<size_t>(lo.pf_tiles_per_head) * 32 * 4);   // their key rows
  lo.ws_pf_flags = take(static_cast<size_t>(c.max_chunk_tokens) * H);  // decisions from q
  // kept chunk tokens before every 32-aligned chunk position, per KV head
  // (same indexing as the tiles of one region)
  lo.ws_pf_kb = take(H * static_cast<size_t>(lo.pf_tiles_per_head) * 4);
  lo.ws_pf_order = take(NH * 4);   // attention workgroup rows, heaviest head first
  lo.ws_q_sel = take(NH * static_cast<size_t>(c.quest_page_budget) * 4);
  lo.ws_q_page = take(NH * static_cast<size_t>(c.quest_page_budget) * 4);
  lo.ws_q_len = take(NH * 4);
  lo.workspace_bytes = off;
  return lo;
}

struct Ctx {
  dms_config cfg;
  Layout lo;
  void* meta;
  std::vector<void*> pools;
  void* ws;
  int decode_waves;  // resident decode waves, found on first decode
  // kernel timing session: event pairs and the kind of kernel each timed
  std::vector<hipEvent_t> ev;
  std::vector<int> ev_kind;
  int ev_used = 0;
  bool profiling = false;
};

}  // namespace dms

using dms::Ctx;

struct dms_ctx {
  Ctx c;
};

// Scratch of dms_decode_step_static (see static_scratch below): one copy per
// GPU, held until the process ends.
constexpr size_t kStaticScratchBytes = size_t(32) << 20;
static __device__ __align__(256) char scratch[kStaticScratchBytes];

namespace {

inline hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

inline int hip_rc(hipError_t e) { return e == hipSuccess ? DMS_OK : DMS_ERR_HIP; }

// Latent-attention cache: keys only (the values are part of the key row).
inline bool mla(const dms_ctx* ctx) { return ctx->c.cfg.kv_format == DMS_KV_MLA; }

// Event pair for the next timed launch of a session (or nulls).
void next_events(Ctx& c, int kind, hipEvent_t* a, hipEvent_t* b) {
  *a = nullptr;
  *b = nullptr;
  if (!c.profiling || c.ev_used + 2 > static_cast<int>(c.ev.size())) return;
  *a = c.ev[c.ev_used];
  *b = c.ev[c.ev_used + 1];
  c.ev_kind[c.ev_used / 2] = kind;
  c.ev_used += 2;
}

int check_call(const dms_ctx* ctx, int layer, int n, const void* seq_ids) {
  if (!ctx) return DMS_ERR_INVALID;
  if (layer < 0 || layer >= ctx->c.cfg.num_layers) return DMS_ERR_INVALID;
  if (n < 1 || n > ctx->c.cfg.max_seqs) return DMS_ERR_INVALID;
  if (!seq_ids) return DMS_ERR_INVALID;
  return DMS_OK;
}

int check_chunk(const dms_ctx* ctx, const int32_t* cu, int total, int max_len) {
  if (!cu) return DMS_ERR_INVALID;
  if (total < 0 || total > ctx->c.cfg.max_chunk_tokens) return DMS_ERR_INVALID;
  if (max_len < 0 || max_len > total) return DMS_ERR_INVALID;
  if (total > 0 && max_len == 0) return DMS_ERR_INVALID;
  return DMS_OK;
}

// Page retrieval buffers in the workspace.
const int32_t* quest_lengths(const Ctx& c) {
  return reinterpret_cast<const int32_t*>(static_cast<char*>(c.ws) + c.lo.ws_q_len);
}
const int32_t* quest_pages(const Ctx& c) {
  return reinterpret_cast<const int32_t*>(static_cast<char*>(c.ws) + c.lo.ws_q_sel);
}
const int32_t* quest_phys_pages(const Ctx& c) {
  return reinterpret_cast<const int32_t*>(static_cast<char*>(c.ws) + c.lo.ws_q_page);
}

// ---------------------------------------------------------------------------
// Static scratch of dms_decode_step_static
// ---------------------------------------------------------------------------

// Device memory that dms_decode_step_static works in instead of the caller's
// workspace: planner output (head descriptors, tile prefix sums, per-wave
// ranges, per-head wave spans), split-K partials and arrival counters.  Every
// GPU the library runs on holds its own copy until the process ends.  In host
// code the name is only a stand-in for the symbol; kernels get the device
// address that hipGetSymbolAddress returns for the current device.
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxScratchDevices] = {};

// Device address of the current device's scratch, resolved once per device.
int static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return DMS_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return DMS_ERR_HIP;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return DMS_OK;
}

// Offsets of the decode buffers for a call of `n` sequences over `waves`
// decode waves, packed from offset 0 of the scratch (the meta and pool
// offsets of `lo` are kept).  Returns the bytes used.
size_t static_layout(const dms_config& c, int n, int waves, dms::Layout* lo) {
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = dms::align_up(off + bytes, dms::kAlign); return o; };
  const size_t NH = static_cast<size_t>(n) * c.num_kv_heads, W = static_cast<size_t>(waves);
  lo->ws_head_desc = take(NH * sizeof(dms::HeadDesc));
  lo->ws_cum_tiles = take((NH + 1) * 4);
  // (the entry point takes standard-row formats only: one head group)
  lo->ml_stride = dms::kMaxGroup;
  lo->head_groups = 1;
  lo->ws_part_ml = take((W + NH) * lo->ml_stride * 8);
  lo->ws_part_acc = take((W + NH) * c.group_size * c.head_dim * 4);
  lo->ws_wave_bounds = take((W + 1) * 4);
  lo->ws_wave_desc = take(W * 2 * sizeof(int4));
  lo->ws_head_waves = take(NH * sizeof(int4));
  lo->ws_head_cnt = take(NH * lo->head_groups * 4);
  lo->max_partials = static_cast<int>(W + NH);   // partial index = wave + call head
  return off;
}

int ensure_waves(dms_ctx* ctx) {
  if (ctx->c.decode_waves > 0) return DMS_OK;
  int w = dms::decode_resident_waves(ctx->c.cfg);
  if (w <= 0) return DMS_ERR_HIP;
  ctx->c.decode_waves = w < dms::kMaxWaves ? w : dms::kMaxWaves;
  return DMS_OK;
}

}  // namespace

extern "C" {

int dms_layout(const dms_config* cfg, size_t* meta_bytes, size_t* pool_bytes,
               size_t* workspace_bytes, size_t* page_bytes) {
  if (!cfg) return DMS_ERR_INVALID;
  int rc = dms::validate_config(*cfg);
  if (rc) return rc;
  dms::Layout lo = dms::make_layout(*cfg);
  if (meta_bytes) *meta_bytes = lo.meta_bytes;
  if (pool_bytes) *pool_bytes = lo.pool_bytes;
  if (workspace_bytes) *workspace_bytes = lo.workspace_bytes;
  if (page_bytes) *page_bytes = lo.page_bytes;
  return DMS_OK;
}

int dms_state_layout(const dms_config* cfg, dms_state_offsets* out) {
  if (!cfg || !out) return DMS_ERR_INVALID;
  int rc = dms::validate_config(*cfg);
  if (rc) return rc;
  dms::Layout lo = dms::make_layout(*cfg);
  out->status = lo.status;
  out->layer0 = lo.layer0;
  out->layer_stride = lo.layer_stride;
  out->pos = lo.pos;
  out->len = lo.len;
  out->ring = lo.ring;
  out->page_table = lo.page_table;
  out->slot_meta = lo.slot_meta;
  out->stack = lo.stack;
  out->top = lo.top;
  out->page_bounds = lo.page_bounds;
  return DMS_OK;
}

int dms_create(const dms_config* cfg, void* meta_dev, void* const* pools_dev_host,
               void* workspace_dev, dms_ctx** out) {
  if (!cfg || !meta_dev || !pools_dev_host || !workspace_dev || !out) return DMS_ERR_INVALID;
  int rc = dms::validate_config(*cfg);
  if (rc) return rc;
  for (int l = 0; l < cfg->num_layers; ++l)
    if (!pools_dev_host[l]) return DMS_ERR_INVALID;
  dms_ctx* ctx = new (std::nothrow) dms_ctx;
  if (!ctx) return DMS_ERR_INVALID;
  ctx->c.cfg = *cfg;
  if (!(ctx->c.cfg.softmax_scale > 0.0f))
    ctx->c.cfg.softmax_scale = 1.0f / sqrtf(static_cast<float>(cfg->head_dim));
  ctx->c.lo = dms::make_layout(*cfg);
  ctx->c.meta = meta_dev;
  ctx->c.pools.assign(pools_dev_host, pools_dev_host + cfg->num_layers);
  ctx->c.ws = workspace_dev;
  ctx->c.decode_waves = 0;
  *out = ctx;
  return DMS_OK;
}

int dms_destroy(dms_ctx* ctx) {
  if (!ctx) return DMS_ERR_INVALID;
  for (auto& e : ctx->c.ev) (void)hipEventDestroy(e);
  delete ctx;
  return DMS_OK;
}

int dms_init_state(dms_ctx* ctx, void* stream) {
  if (!ctx) return DMS_ERR_INVALID;
  // set-up of the current device's static scratch (dms_decode_step_static)
  void* sp = nullptr;
  if (int rc = static_scratch(&sp)) return rc;
  return hip_rc(dms::launch_init_state(ctx->c.cfg, ctx->c.lo, ctx->c.meta, ctx->c.ws,
                                       as_stream(stream)));
}

int dms_seq_reset(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev, void* stream) {
  if (!ctx) return DMS_ERR_INVALID;
  if (layer < -1 || layer >= ctx->c.cfg.num_layers) return DMS_ERR_INVALID;
  if (n < 1 || n > ctx->c.cfg.max_seqs || !seq_ids_dev) return DMS_ERR_INVALID;
  return hip_rc(dms::launch_seq_reset(ctx->c.cfg, ctx->c.lo, ctx->c.meta, layer, n, seq_ids_dev,
                                      as_stream(stream)));
}

int dms_append(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev, const void* k_dev,
               const void* v_dev, const uint8_t* flags_dev, void* stream) {
  int rc = check_call(ctx, layer, n, seq_ids_dev);
  if (rc) return rc;
  if (!k_dev || !(v_dev || mla(ctx)) || !flags_dev) return DMS_ERR_INVALID;
  const Ctx& c = ctx->c;
  hipStream_t st = as_stream(stream);
  hipError_t e = dms::launch_plan(c.cfg, c.lo, c.meta, c.ws, layer, n, seq_ids_dev, flags_dev,
                                  nullptr, nullptr, true, 0, nullptr, st);
  if (e == hipSuccess) {
    // with page retrieval the written pages' bounds are recomputed in the
    // same launch as the K / V writes
    e = c.cfg.quest_page_budget > 0
            ? dms::launch_quest_append(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n, k_dev, v_dev, st)
            : dms::launch_scatter(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n, k_dev, v_dev, st);
  }
  return hip_rc(e);
}

int dms_decode(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev, const void* q_dev,
               float* out_dev, void* stream) {
  int rc = check_call(ctx, layer, n, seq_ids_dev);
  if (rc) return rc;
  if (!q_dev || !out_dev) return DMS_ERR_INVALID;
  if ((rc = ensure_waves(ctx))) return rc;
  const Ctx& c = ctx->c;
  hipStream_t st = as_stream(stream);
  const bool quest = c.cfg.quest_page_budget > 0;
  hipError_t e = hipSuccess;
  if (quest) e = dms::launch_quest_select(c.cfg, c.lo, c.meta, c.ws, layer, n, seq_ids_dev, q_dev, st);
  if (e == hipSuccess)
    e = dms::launch_plan(c.cfg, c.lo, c.meta, c.ws, layer, n, seq_ids_dev, nullptr, nullptr, nullptr,
                         false, c.decode_waves, out_dev, st, quest ? quest_lengths(c) : nullptr);
  hipEvent_t e0, e1;
  next_events(ctx->c, DMS_PROFILE_DECODE, &e0, &e1);
  if (e == hipSuccess)
    e = dms::launch_decode(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n, q_dev, nullptr,
                           nullptr, out_dev, c.decode_waves, st, e0, e1, quest ? quest_phys_pages(c) : nullptr);
  return hip_rc(e);
}

namespace {

// Append + decode of one layer; decisions from flags_dev (caller) or from
// q_dev (decisions_out_dev receives them, may be null).
int decode_step(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev, const void* q_dev,
                const void* k_dev, const void* v_dev, const uint8_t* flags_dev,
                uint8_t* decisions_out_dev, float* out_dev, void* stream) {
  const bool from_q = ctx->c.cfg.decision_source == DMS_DECIDE_QUERY;
  const Ctx& c = ctx->c;
  hipStream_t st = as_stream(stream);
  if (c.cfg.quest_page_budget > 0) {
    // page retrieval: plan the append; write K / V, recompute the written
    // pages' bounds and select every head's pages (one launch); then decode
    // over the selection, planning its tiles inside the decode launch (up to
    // 1024 heads) or with the planner
    hipError_t e = dms::launch_plan(c.cfg, c.lo, c.meta, c.ws, layer, n, seq_ids_dev,
                                    from_q ? nullptr : flags_dev, from_q ? q_dev : nullptr,
                                    decisions_out_dev, true, 0, nullptr, st);
    if (e == hipSuccess)
      e = dms::launch_quest_append_select(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n, q_dev, k_dev,
                                          v_dev, st);
    const bool in_launch = n * c.cfg.num_kv_heads <= dms::decode_attended_max_heads();
    if (e == hipSuccess && !in_launch)
      e = dms::launch_plan(c.cfg, c.lo, c.meta, c.ws, layer, n, seq_ids_dev, nullptr, nullptr, nullptr,
                           false, c.decode_waves, out_dev, st, quest_lengths(c));
    hipEvent_t e0, e1;
    next_events(ctx->c, DMS_PROFILE_DECODE, &e0, &e1);
    if (e == hipSuccess)
      e = in_launch ? dms::launch_decode_attended(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n, q_dev,
                                                  out_dev, c.decode_waves, st, e0, e1, quest_phys_pages(c),
                                                  quest_lengths(c))
                    : dms::launch_decode(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n, q_dev, nullptr,
                                         nullptr, out_dev, c.decode_waves, st, e0, e1, quest_phys_pages(c));
    return hip_rc(e);
  }
  if (dms::decode_step_fusable(c.cfg, n)) {
    // one launch: every workgroup plans the append in LDS, the last one to
    // read the state writes it, and the waves decode (writing the new K / V
    // into their slots and merging split heads)
    hipEvent_t e0, e1;
    next_events(ctx->c, DMS_PROFILE_DECODE, &e0, &e1);
    return hip_rc(dms::launch_decode_step(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n,
                                          seq_ids_dev, flags_dev, q_dev, k_dev, v_dev,
                                          decisions_out_dev, out_dev, c.decode_waves, st, e0, e1));
  }
  // planner (slot choice, page pops, state, wave ranges) -> decode, which
  // also writes the new K / V into their slots and merges split heads
  hipError_t e = dms::launch_plan(c.cfg, c.lo, c.meta, c.ws, layer, n, seq_ids_dev,
                                  from_q ? nullptr : flags_dev, from_q ? q_dev : nullptr,
                                  decisions_out_dev, true, c.decode_waves, out_dev, st);
  hipEvent_t e0, e1;
  next_events(ctx->c, DMS_PROFILE_DECODE, &e0, &e1);
  if (e == hipSuccess)
    e = dms::launch_decode(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n, q_dev, k_dev,
                           v_dev, out_dev, c.decode_waves, st, e0, e1);
  return hip_rc(e);
}

// Masked chunk attention then commit; decisions from flags_dev or from q_dev
// (written to decisions_out_dev, or to the workspace when that is null).
int prefill_chunk(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                  const int32_t* cu_seqlens_dev, int total_tokens, int max_seqlen,
                  const void* q_dev, const void* k_dev, const void* v_dev,
                  const uint8_t* flags_dev, uint8_t* decisions_out_dev, float* out_dev,
                  void* stream) {
  const Ctx& c = ctx->c;
  hipStream_t st = as_stream(stream);
  hipError_t e = hipSuccess;
  const uint8_t* flags = flags_dev;
  if (c.cfg.decision_source == DMS_DECIDE_QUERY) {
    uint8_t* buf = decisions_out_dev != nullptr
                       ? decisions_out_dev
                       : reinterpret_cast<uint8_t*>(static_cast<char*>(c.ws) + c.lo.ws_pf_flags);
    e = dms::launch_prefill_decide(c.cfg, q_dev, total_tokens, buf, st);
    flags = buf;
  }
  hipEvent_t e0, e1;
  next_events(ctx->c, DMS_PROFILE_PREFILL, &e0, &e1);
  if (e == hipSuccess)
    e = dms::launch_prefill_attention(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n,
                                      seq_ids_dev, cu_seqlens_dev, total_tokens, max_seqlen, q_dev,
                                      k_dev, v_dev, flags, out_dev, st, e0, e1);
  if (e == hipSuccess)
    e = dms::launch_chunk_commit(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n, seq_ids_dev,
                                 cu_seqlens_dev, total_tokens, max_seqlen, k_dev, v_dev, flags, st);
  if (e == hipSuccess && c.cfg.quest_page_budget > 0)
    e = dms::launch_quest_bounds(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n, true,
                                 seq_ids_dev, st);
  return hip_rc(e);
}

}  // namespace

int dms_decode_step(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev, const void* q_dev,
                    const void* k_dev, const void* v_dev, const uint8_t* flags_dev,
                    float* out_dev, void* stream) {
  int rc = check_call(ctx, layer, n, seq_ids_dev);
  if (rc) return rc;
  if (ctx->c.cfg.decision_source != DMS_DECIDE_CALLER) return DMS_ERR_INVALID;
  if (!q_dev || !k_dev || !(v_dev || mla(ctx)) || !flags_dev || !out_dev) return DMS_ERR_INVALID;
  if ((rc = ensure_waves(ctx))) return rc;
  return decode_step(ctx, layer, n, seq_ids_dev, q_dev, k_dev, v_dev, flags_dev, nullptr, out_dev,
                     stream);
}

int dms_decode_step_static(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                           const void* q_dev, const void* k_dev, const void* v_dev,
                           const uint8_t* flags_dev, float* out_dev, void* stream) {
  int rc = check_call(ctx, layer, n, seq_ids_dev);
  if (rc) return rc;
  const dms_config& cfg = ctx->c.cfg;
  if (cfg.decision_source != DMS_DECIDE_CALLER) return DMS_ERR_INVALID;
  if (cfg.kv_format == DMS_KV_MLA || cfg.quest_page_budget > 0) return DMS_ERR_UNSUPPORTED;
  if (!q_dev || !k_dev || !v_dev || !flags_dev || !out_dev) return DMS_ERR_INVALID;
  if ((rc = ensure_waves(ctx))) return rc;
  const Ctx& c = ctx->c;
  dms::Layout slo = c.lo;
  if (static_layout(cfg, n, c.decode_waves, &slo) > kStaticScratchBytes) return DMS_ERR_SCRATCH;
  void* sp = nullptr;
  if ((rc = static_scratch(&sp))) return rc;
  hipStream_t st = as_stream(stream);
  // the same planner and decode kernels as dms_decode_step; the planner also
  // clears the arrival counters of the call's heads, which an earlier call
  // (of any context) may have left in the scratch
  hipError_t e = dms::launch_plan(cfg, slo, c.meta, sp, layer, n, seq_ids_dev, flags_dev, nullptr,
                                  nullptr, true, c.decode_waves, out_dev, st, nullptr, true);
  hipEvent_t e0, e1;
  next_events(ctx->c, DMS_PROFILE_DECODE, &e0, &e1);
  if (e == hipSuccess)
    e = dms::launch_decode(cfg, slo, c.meta, sp, c.pools[layer], layer, n, q_dev, k_dev, v_dev,
                           out_dev, c.decode_waves, st, e0, e1);
  return hip_rc(e);
}

int dms_decode_step_q(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                      const void* q_dev, const void* k_dev, const void* v_dev,
                      uint8_t* decisions_out_dev, float* out_dev, void* stream) {
  int rc = check_call(ctx, layer, n, seq_ids_dev);
  if (rc) return rc;
  if (ctx->c.cfg.decision_source != DMS_DECIDE_QUERY) return DMS_ERR_INVALID;
  if (!q_dev || !k_dev || !v_dev || !out_dev) return DMS_ERR_INVALID;
  if ((rc = ensure_waves(ctx))) return rc;
  return decode_step(ctx, layer, n, seq_ids_dev, q_dev, k_dev, v_dev, nullptr, decisions_out_dev,
                     out_dev, stream);
}

int dms_append_chunk(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                     const int32_t* cu_seqlens_dev, int total_tokens, int max_seqlen,
                     const void* k_dev, const void* v_dev, const uint8_t* flags_dev,
                     void* stream) {
  int rc = check_call(ctx, layer, n, seq_ids_dev);
  if (rc) return rc;
  if ((rc = check_chunk(ctx, cu_seqlens_dev, total_tokens, max_seqlen))) return rc;
  if (total_tokens == 0) return DMS_OK;
  if (!k_dev || !(v_dev || mla(ctx)) || !flags_dev) return DMS_ERR_INVALID;
  const Ctx& c = ctx->c;
  hipStream_t st = as_stream(stream);
  hipError_t e = dms::launch_chunk_commit(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n,
                                          seq_ids_dev, cu_seqlens_dev, total_tokens, max_seqlen,
                                          k_dev, v_dev, flags_dev, st);
  // page retrieval: a chunk may write into any page of a head (reused slots)
  if (e == hipSuccess && c.cfg.quest_page_budget > 0)
    e = dms::launch_quest_bounds(c.cfg, c.lo, c.meta, c.ws, c.pools[layer], layer, n, true,
                                 seq_ids_dev, st);
  return hip_rc(e);
}

int dms_quest_selection(dms_ctx* ctx, int n, int32_t* pages_out_dev, int32_t* count_out_dev,
                        void* stream) {
  if (!ctx || ctx->c.cfg.quest_page_budget <= 0) return DMS_ERR_INVALID;
  if (n < 1 || n > ctx->c.cfg.max_seqs || !pages_out_dev || !count_out_dev) return DMS_ERR_INVALID;
  const Ctx& c = ctx->c;
  return hip_rc(dms::launch_quest_export(c.cfg, c.lo, c.ws, n, pages_out_dev, count_out_dev,
                                         as_stream(stream)));
}

int dms_prefill_chunk(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                      const int32_t* cu_seqlens_dev, int total_tokens, int max_seqlen,
                      const void* q_dev, const void* k_dev, const void* v_dev,
                      const uint8_t* flags_dev, float* out_dev, void* stream) {
  int rc = check_call(ctx, layer, n, seq_ids_dev);
  if (rc) return rc;
  if (ctx->c.cfg.decision_source != DMS_DECIDE_CALLER) return DMS_ERR_INVALID;
  if ((rc = check_chunk(ctx, cu_seqlens_dev, total_tokens, max_seqlen))) return rc;
  if (total_tokens == 0) return DMS_OK;
  if (!q_dev || !k_dev || !(v_dev || mla(ctx)) || !flags_dev || !out_dev) return DMS_ERR_INVALID;
  return prefill_chunk(ctx, layer, n, seq_ids_dev, cu_seqlens_dev, total_tokens, max_seqlen, q_dev,
                       k_dev, v_dev, flags_dev, nullptr, out_dev, stream);
}

int dms_prefill_chunk_q(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                        const int32_t* cu_seqlens_dev, int total_tokens, int max_seqlen,
                        const void* q_dev, const void* k_dev, const void* v_dev,
                        uint8_t* decisions_out_dev, float* out_dev, void* stream) {
  int rc = check_call(ctx, layer, n, seq_ids_dev);
  if (rc) return rc;
  if (mla(ctx)) return DMS_ERR_UNSUPPORTED;
  if (ctx->c.cfg.decision_source != DMS_DECIDE_QUERY) return DMS_ERR_INVALID;
  if ((rc = check_chunk(ctx, cu_seqlens_dev, total_tokens, max_seqlen))) return rc;
  if (total_tokens == 0) return DMS_OK;
  if (!q_dev || !k_dev || !v_dev || !out_dev) return DMS_ERR_INVALID;
  return prefill_chunk(ctx, layer, n, seq_ids_dev, cu_seqlens_dev, total_tokens, max_seqlen, q_dev,
                       k_dev, v_dev, nullptr, decisions_out_dev, out_dev, stream);
}

int dms_retained_lengths(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                         int32_t* out_dev, void* stream) {
  int rc = check_call(ctx, layer, n, seq_ids_dev);
  if (rc) return rc;
  if (!out_dev) return DMS_ERR_INVALID;
  return hip_rc(dms::launch_retained(ctx->c.cfg, ctx->c.lo, ctx->c.meta, layer, n, seq_ids_dev,
                                     out_dev, as_stream(stream)));
}

int dms_export_state(dms_ctx* ctx, int layer, void* dst_host, size_t bytes, void* stream) {
  if (!ctx || !dst_host) return DMS_ERR_INVALID;
  if (layer < 0 || layer >= ctx->c.cfg.num_layers) return DMS_ERR_INVALID;
  if (bytes < ctx->c.lo.layer_stride) return DMS_ERR_INVALID;
  hipStream_t st = as_stream(stream);
  const char* src = static_cast<const char*>(ctx->c.meta) + ctx->c.lo.layer0 +
                    static_cast<size_t>(layer) * ctx->c.lo.layer_stride;
  hipError_t e = hipStreamSynchronize(st);
  if (e == hipSuccess) e = hipMemcpy(dst_host, src, ctx->c.lo.layer_stride, hipMemcpyDeviceToHost);
  return hip_rc(e);
}

int dms_status(dms_ctx* ctx, void* stream) {
  if (!ctx) return DMS_ERR_INVALID;
  int32_t v = 0;
  hipError_t e = hipStreamSynchronize(as_stream(stream));
  if (e == hipSuccess)
    e = hipMemcpy(&v, static_cast<char*>(ctx->c.meta) + ctx->c.lo.status, sizeof(v),
                  hipMemcpyDeviceToHost);
  if (e != hipSuccess) return DMS_ERR_HIP;
  return v;
}

int dms_clear_status(dms_ctx* ctx, void* stream) {
  if (!ctx) return DMS_ERR_INVALID;
  int32_t* status = reinterpret_cast<int32_t*>(static_cast<char*>(ctx->c.meta) + ctx->c.lo.status);
  return hip_rc(dms::launch_set_status(status, 0, as_stream(stream)));
}

int dms_profile_start(dms_ctx* ctx, int max_launches) {
  if (!ctx || max_launches < 1 || ctx->c.profiling) return DMS_ERR_INVALID;
  Ctx& c = ctx->c;
  c.ev.assign(2 * static_cast<size_t>(max_launches), nullptr);
  c.ev_kind.assign(static_cast<size_t>(max_launches), 0);
  for (auto& e : c.ev) {
    if (hipEventCreate(&e) != hipSuccess) {
      for (auto& x : c.ev)
        if (x) (void)hipEventDestroy(x);
      c.ev.clear();
      return DMS_ERR_HIP;
    }
  }
  c.ev_used = 0;
  c.profiling = true;
  return DMS_OK;
}

int dms_profile_stop(dms_ctx* ctx, float* ms_out, int* launches_out) {
  if (!ctx || !ctx->c.profiling) return DMS_ERR_INVALID;
  Ctx& c = ctx->c;
  float sum[2] = {0.0f, 0.0f};
  int cnt[2] = {0, 0};
  int rc = DMS_OK;
  for (int i = 0; i + 1 < c.ev_used; i += 2) {
    float ms = 0.0f;
    if (hipEventSynchronize(c.ev[i + 1]) != hipSuccess ||
        hipEventElapsedTime(&ms, c.ev[i], c.ev[i + 1]) != hipSuccess) {
      rc = DMS_ERR_HIP;
      break;
    }
    const int k = c.ev_kind[i / 2];
    sum[k] += ms;
    cnt[k] += 1;
  }
  for (int k = 0; k < 2; ++k) {
    if (ms_out) ms_out[k] = sum[k];
    if (launches_out) launches_out[k] = cnt[k];
  }
  for (auto& e : c.ev) (void)hipEventDestroy(e);
  c.ev.clear();
  c.ev_kind.clear();
  c.ev_used = 0;
  c.profiling = false;
  return rc;
}

const char* dms_strerror(int code) {
  switch (code) {
    case DMS_OK: return "ok";
    case DMS_ERR_INVALID: return "invalid configuration or argument";
    case DMS_ERR_UNSUPPORTED: return "unsupported configuration";
    case DMS_ERR_HIP: return "HIP runtime error";
    case DMS_ERR_OUT_OF_PAGES: return "KV page pool exhausted";
    case DMS_ERR_CAPACITY: return "a head exceeds max_pages_per_head";
    case DMS_ERR_BAD_SEQ: return "sequence id out of range or repeated in one call";
    case DMS_ERR_SCRATCH: return "call too large for the library's static scratch";
    default: return "unknown error code";
  }
}

// ---------------------------------------------------------------------------
// Training-time attention
// ---------------------------------------------------------------------------

static int validate_train_config(const dms_train_config* c) {
  if (!c) return DMS_ERR_INVALID;
  if (c->batch < 1 || c->seq_len < 1 || c->num_kv_heads < 1 || c->group_size < 1 || c->window < 1)
    return DMS_ERR_INVALID;
  if (c->group_size > dms::kMaxGroup) return DMS_ERR_UNSUPPORTED;
  if (c->head_dim != dms::kTrainHeadDim) return DMS_ERR_UNSUPPORTED;
  if (isnan(c->softmax_scale) || (c->softmax_scale > 0.0f && !isfinite(c->softmax_scale)))
    return DMS_ERR_INVALID;
  // element offsets of the largest tensors stay below 2^31 rows of head_dim
  const int64_t rows = static_cast<int64_t>(c->batch) * c->seq_len * c->num_kv_heads * c->group_size;
  if (rows >= (int64_t(1) << 31) / 8) return DMS_ERR_INVALID;
  // one grid row per (sequence, KV head)
  if (static_cast<int64_t>(c->batch) * c->num_kv_heads > 65535) return DMS_ERR_INVALID;
  return DMS_OK;
}

int dms_train_workspace(const dms_train_config* cfg, size_t* workspace_bytes) {
  const int rc = validate_train_config(cfg);
  if (rc) return rc;
  if (workspace_bytes) *workspace_bytes = dms::train_workspace_bytes(*cfg);
  return DMS_OK;
}

int dms_train_attention_fwd(const dms_train_config* cfg, const void* q_dev, const void* k_dev,
                            const void* v_dev, const float* alpha_dev, float* out_dev,
                            float* lse_dev, void* workspace_dev, void* stream) {
  const int rc = validate_train_config(cfg);
  if (rc) return rc;
  if (!q_dev || !k_dev || !v_dev || !alpha_dev || !out_dev || !lse_dev || !workspace_dev)
    return DMS_ERR_INVALID;
  return hip_rc(dms::launch_train_fwd(*cfg, q_dev, k_dev, v_dev, alpha_dev, out_dev, lse_dev,
                                      workspace_dev, as_stream(stream)));
}

int dms_train_attention_bwd(const dms_train_config* cfg, const void* q_dev, const void* k_dev,
                            const void* v_dev, const float* alpha_dev, const float* out_dev,
                            const float* lse_dev, const void* dout_dev, float* dq_dev,
                            float* dk_dev, float* dv_dev, float* dalpha_dev,
                            void* workspace_dev, void* stream) {
  const int rc = validate_train_config(cfg);
  if (rc) return rc;
  if (!q_dev || !k_dev || !v_dev || !alpha_dev || !out_dev || !lse_dev || !dout_dev || !dq_dev ||
      !dk_dev || !dv_dev || !dalpha_dev || !workspace_dev)
    return DMS_ERR_INVALID;
  return hip_rc(dms::launch_train_bwd(*cfg, q_dev, k_dev, v_dev, alpha_dev, out_dev, lse_dev,
                                      dout_dev, dq_dev, dk_dev, dv_dev, dalpha_dev, workspace_dev,
                                      as_stream(stream)));
}

int dms_gumbel_sigmoid_fwd(int n, const float* logits_dev, const float* u_dev, float tau,
                           float* alpha_dev, void* stream) {
  if (n < 0 || !(tau > 0.f) || !isfinite(tau)) return DMS_ERR_INVALID;
  if (n == 0) return DMS_OK;
  if (!logits_dev || !u_dev || !alpha_dev) return DMS_ERR_INVALID;
  return hip_rc(dms::launch_gumbel_fwd(n, logits_dev, u_dev, tau, alpha_dev, as_stream(stream)));
}

int dms_gumbel_sigmoid_bwd(int n, const float* alpha_dev, const float* dalpha_dev, float tau,
                           float* dlogits_dev, void* stream) {
  if (n < 0 || !(tau > 0.f) || !isfinite(tau)) return DMS_ERR_INVALID;
  if (n == 0) return DMS_OK;
  if (!alpha_dev || !dalpha_dev || !dlogits_dev) return DMS_ERR_INVALID;
  return hip_rc(dms::launch_gumbel_bwd(n, alpha_dev, dalpha_dev, tau, dlogits_dev, as_stream(stream)));
}

}  // extern "C"
