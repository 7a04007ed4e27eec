// Internal definitions shared by the libdms translation units: buffer layout,
// per-layer state views and small device helpers.  gfx950 (CDNA4) only.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/dms.h"

namespace dms {

constexpr int kTile = 32;            // tokens per decode tile (k of one PV MFMA)
constexpr int kMaxWaves = 8192;      // upper bound on decode waves (workspace sizing)
constexpr int kMaxGroup = 16;        // query heads per KV head (MFMA column count)
constexpr int kMlaDim = 576;         // latent attention row: 512 latent + 64 rotary key dims
constexpr int kMlaLatent = 512;      // of which the latent (the values)
constexpr int kMlaMaxGroup = 128;    // query heads sharing one latent row (groups of kMaxGroup)
constexpr int kMaxMlaUnits = 1024;   // upper bound on latent-attention work units (workspace sizing)
constexpr int kMaxSeqs = 65536;      // sequence-id bitmap of the planning kernel
constexpr uint32_t kFlagBit = 0x80000000u;
constexpr int kAlign = 256;

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Offsets of everything inside the caller's three buffers.
struct Layout {
  // meta
  size_t status, layer0, layer_stride;
  size_t pos, len, ring, page_table, slot_meta, stack, top;
  size_t page_bounds;      // quest: bf16 [num_pages][2][D] per layer (0 when off)
  size_t meta_bytes;
  // pool of one layer
  size_t page_bytes, pool_bytes;
  // workspace
  size_t ws_head_desc, ws_cum_tiles, ws_part_ml, ws_part_acc;
  size_t ws_wave_bounds, ws_wave_desc, ws_head_waves, ws_head_cnt;
  size_t ws_plan_ctr;   // fused decode: workgroups that have read the state this launch
  size_t ws_ck_need, ws_ck_fresh, ws_ck_base, ws_ck_pos0, ws_ck_err, ws_ck_slot;
  size_t ws_pf_cum, ws_pf_meta, ws_pf_tiles, ws_pf_tmeta, ws_pf_flags, ws_pf_kb, ws_pf_order;
  size_t ws_q_sel, ws_q_page, ws_q_len;   // quest: selection [NH][B] (page-table
                                          // indices, physical pages), attended lengths [NH]
  int pf_tiles_per_head;   // tiles of one (region, KV head) in ws_pf_tiles
  size_t workspace_bytes;
  int max_heads, max_partials, max_slots;
  int ml_stride;     // (max, sum) pairs per split-K partial: kMaxGroup, or the latent group rounded up
  int head_groups;   // arrival counters per call head: query-head groups of kMaxGroup (latent rows)
};

// Host-side validation; returns DMS_OK or an error code.
int validate_config(const dms_config& c);
Layout make_layout(const dms_config& c);

// Device view of one layer's state.
struct LayerState {
  int32_t* pos;         // [S]
  int32_t* len;         // [S][Hkv]
  int32_t* ring;        // [S][Hkv][w]
  int32_t* page_table;  // [S][Hkv][max_pages]
  int32_t* slot_meta;   // [S][Hkv][max_slots]
  int32_t* stack;       // [num_pages]
  int32_t* top;         // [1]
  uint16_t* page_bounds;   // quest: [num_pages][2][D] bf16 (null when off)
};

inline LayerState layer_state(const Layout& lo, void* meta, int layer) {
  char* b = static_cast<char*>(meta) + lo.layer0 + static_cast<size_t>(layer) * lo.layer_stride;
  LayerState s;
  s.pos = reinterpret_cast<int32_t*>(b + lo.pos);
  s.len = reinterpret_cast<int32_t*>(b + lo.len);
  s.ring = reinterpret_cast<int32_t*>(b + lo.ring);
  s.page_bounds = lo.page_bounds ? reinterpret_cast<uint16_t*>(b + lo.page_bounds) : nullptr;
  s.page_table = reinterpret_cast<int32_t*>(b + lo.page_table);
  s.slot_meta = reinterpret_cast<int32_t*>(b + lo.slot_meta);
  s.stack = reinterpret_cast<int32_t*>(b + lo.stack);
  s.top = reinterpret_cast<int32_t*>(b + lo.top);
  return s;
}

// Pool page layout.  A page holds P/32 tiles of 32 consecutive slots; each
// tile is 128*D bytes, keys first, then values, both in the order the decode
// MFMAs consume them, as 16-byte pieces of 8 bf16:
//   K part: D/32 x 2 blocks of 1 KB.  Block (s, h) holds dims 32 s .. 32 s + 31
//     of the 16 slots j with (j / 4) % 2 == h, as [G = dims / 8 % 4][r][8 dims]
//     with r = 4 (j / 8) + j % 4 (the rows of the first / second score MFMA);
//   V part: D/16 blocks of 1 KB.  Block b holds dims 16 b .. 16 b + 15 as
//     [G = slots / 8][r = dim % 16][8 slots] (rows of V^T).
// Every load instruction of a decode wave then reads one contiguous 1 KB with
// lane l taking bytes 16 l .. 16 l + 15.
__host__ __device__ inline size_t tile_bytes(int D) { return static_cast<size_t>(D) * 128; }
// Latent-attention pages: a 32-slot tile holds only the key part (the values
// are the first kMlaLatent dims of each row), in the same fragment order.
__host__ __device__ inline size_t mla_tile_bytes(int D) { return static_cast<size_t>(D) * 64; }
__host__ __device__ inline size_t k_elem_off(int j, int e) {
  return (static_cast<size_t>(((e >> 5) * 2 + ((j >> 2) & 1)) * 4 + ((e >> 3) & 3)) * 16 +
          4 * (j >> 3) + (j & 3)) * 16 + (e & 7) * 2;
}
__host__ __device__ inline size_t v_elem_off(int j, int e, int D) {
  return static_cast<size_t>(D) * 64 + (static_cast<size_t>((e >> 4) * 4 + (j >> 3)) * 16 + (e & 15)) * 16 +
         (j & 7) * 2;
}

// Decision of a token appended for call head hh (sequence hh / H, KV head
// hh % H): the caller's flag, or round(sigmoid(x)) = (x > 0) with x = bf16
// element 0 of the first query head of the group plus the offset, in float32
// (Sec. 3.2, App. C).
__device__ inline int token_decision(const uint8_t* flags, const uint16_t* q, int hh, int H, int g,
                                     int D, float bias) {
  if (q == nullptr) return flags[hh] != 0;
  const uint32_t bits = q[static_cast<size_t>(hh) * g * D];   // (i * H + h) * g * D
  return (__uint_as_float(bits << 16) + bias) > 0.f;
}

// Whether the token at position t takes the slot of the token that entered
// w steps ago (ring entry e): delayed eviction -- that token was flagged;
// immediate eviction -- the incoming token's own decision evicts it now.
__device__ inline bool takes_old_slot(int t, int w, int32_t e, int f, int immediate) {
  if (t < w) return false;
  return immediate ? f != 0 : (static_cast<uint32_t>(e) & kFlagBit) != 0;
}

// Per-head descriptor written by the planning kernels, one per (seq in call,
// KV head) in call order: x = retained length L, y = state head index
// (seq * Hkv + head), z = slot written by this call's token (decode), w = 0.
typedef int4 HeadDesc;

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------

// Inclusive prefix sum across one wave64.
__device__ inline int wave_inclusive_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int u = __shfl_up(v, off, 64);
    if (lane >= off) v += u;
  }
  return v;
}

// Exclusive prefix sum across the block (blockDim.x multiple of 64, <= 1024).
// `lds` holds 17 ints.  Returns the exclusive prefix; *total gets the block sum.
__device__ inline int block_exclusive_scan(int v, int* lds, int* total) {
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  int inc = wave_inclusive_scan(v);
  if (lane == 63) lds[wid] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int i = 0; i < nw; ++i) {
      int t = lds[i];
      lds[i] = run;
      run += t;
    }
    lds[16] = run;
  }
  __syncthreads();
  int excl = lds[wid] + inc - v;
  *total = lds[16];
  __syncthreads();
  return excl;
}

// Two exclusive prefix sums across the block in one pass (same contract as
// block_exclusive_scan; `lds` holds 34 ints).
__device__ inline int2 block_exclusive_scan2(int2 v, int* lds, int2* total) {
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const int ix = wave_inclusive_scan(v.x);
  const int iy = wave_inclusive_scan(v.y);
  if (lane == 63) {
    lds[wid] = ix;
    lds[17 + wid] = iy;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int rx = 0, ry = 0;
    for (int i = 0; i < nw; ++i) {
      const int tx = lds[i], ty = lds[17 + i];
      lds[i] = rx;
      lds[17 + i] = ry;
      rx += tx;
      ry += ty;
    }
    lds[16] = rx;
    lds[33] = ry;
  }
  __syncthreads();
  const int2 ex = make_int2(lds[wid] + ix - v.x, lds[17 + wid] + iy - v.y);
  *total = make_int2(lds[16], lds[33]);
  __syncthreads();
  return ex;
}

// Record the first device-side error (vector atomic; never a scalar store).
__device__ inline void set_status(int32_t* status, int code) {
  atomicCAS(reinterpret_cast<int*>(status), 0, code);
}

// ---------------------------------------------------------------------------
// Launchers implemented in the kernel translation units
// ---------------------------------------------------------------------------

struct Ctx;  // host context (dms_api.hip)

hipError_t launch_init_state(const dms_config& c, const Layout& lo, void* meta, void* ws,
                             hipStream_t st);
hipError_t launch_set_status(int32_t* status, int value, hipStream_t st);
hipError_t launch_seq_reset(const dms_config& c, const Layout& lo, void* meta, int layer,
                            int n, const int32_t* seq_ids, hipStream_t st);
// Planning kernel of a decode call: rule R1 for the appended tokens (when
// `append`), per-head descriptors, tile prefix sums and, for `waves` > 0, the
// tile range and first head of every decode wave.  `out` (nullable) gets zeros
// for heads with no retained token.
// `len_override` (nullable, planning without append only): per-head lengths
// to plan instead of the retained lengths (page retrieval).
// `clear_head_counts`: also zero the split-head arrival counters of the
// call's heads (scratch whose earlier contents are unknown).
hipError_t launch_plan(const dms_config& c, const Layout& lo, void* meta, void* ws, int layer,
                       int n, const int32_t* seq_ids, const uint8_t* flags, const void* q,
                       uint8_t* flags_out, bool append, int waves, float* out, hipStream_t st,
                       const int32_t* len_override = nullptr, bool clear_head_counts = false);
// Page retrieval: recompute the bounds of the pages the last planned append
// wrote (all_pages: every page of every head of the call), then select the
// pages of each head for query q.
// Quest: an append's K / V written and the written pages' bounds recomputed.
hipError_t launch_quest_append(const dms_config& c, const Layout& lo, void* meta, void* ws,
                               void* pool, int layer, int n, const void* k, const void* v, hipStream_t st);
// Quest, decode step: the append's K / V and bounds, then every head's selection.
hipError_t launch_quest_append_select(const dms_config& c, const Layout& lo, void* meta, void* ws,
                                      void* pool, int layer, int n, const void* q, const void* k,
                                      const void* v, hipStream_t st);
// Page retrieval, calls of up to decode_attended_max_heads() heads: decode over
// the selected pages, every workgroup planning the tiles over the attended
// lengths (qlen [n * Hkv]) in LDS (no planner launch).
int decode_attended_max_heads();
hipError_t launch_decode_attended(const dms_config& c, const Layout& lo, void* meta, void* ws, void* pool,
                                  int layer, int n, const void* q, float* out, int waves, hipStream_t st,
                                  hipEvent_t ev_start, hipEvent_t ev_stop, const int32_t* qpage,
                                  const int32_t* qlen);
hipError_t launch_quest_bounds(const dms_config& c, const Layout& lo, void* meta, void* ws,
                               void* pool, int layer, int n, bool all_pages, const int32_t* seq_ids,
                               hipStream_t st);
hipError_t launch_quest_select(const dms_config& c, const Layout& lo, void* meta, void* ws,
                               int layer, int n, const int32_t* seq_ids, const void* q,
                               hipStream_t st);
// Copy the last selection (pages, -1 padded) and per-head page counts out.
hipError_t launch_quest_export(const dms_config& c, const Layout& lo, void* ws, int n,
                               int32_t* pages, int32_t* counts, hipStream_t st);
hipError_t launch_scatter(const dms_config& c, const Layout& lo, void* meta, void* ws,
                          void* pool, int layer, int n, const void* k, const void* v,
                          hipStream_t st);
// k / v: the tokens appended by this call's planning kernel (written into the
// pool by the decode kernel itself), or null when nothing was appended.
// qpage (nullable): per head of the call, the physical pages to attend (page
// retrieval), quest_page_budget entries each.
hipError_t launch_decode(const dms_config& c, const Layout& lo, void* meta, void* ws,
                         void* pool, int layer, int n, const void* q, const void* k,
                         const void* v, float* out, int waves, hipStream_t st,
                         hipEvent_t ev_start, hipEvent_t ev_stop, const int32_t* qpage = nullptr);
int decode_resident_waves(const dms_config& c);
// dms_decode_step in one launch (the append planning runs inside the decode
// kernel); for calls where decode_step_fusable holds.
bool decode_step_fusable(const dms_config& c, int n);
hipError_t launch_decode_step(const dms_config& c, const Layout& lo, void* meta, void* ws, void* pool,
                              int layer, int n, const int32_t* seq_ids, const uint8_t* flags,
                              const void* q, const void* k, const void* v, uint8_t* flags_out,
                              float* out, int waves, hipStream_t st, hipEvent_t ev_start,
                              hipEvent_t ev_stop);
// Decode over a latent-attention cache (kv_format DMS_KV_MLA): rows of
// kMlaDim bf16, outputs [n, g, kMlaLatent] float32.
hipError_t launch_decode_mla(const dms_config& c, const Layout& lo, void* meta, void* ws,
                             void* pool, int layer, int n, const void* q, const void* k,
                             float* out, int waves, hipStream_t st, hipEvent_t ev_start,
                             hipEvent_t ev_stop);
int decode_mla_resident_waves(const dms_config& c);
hipError_t launch_retained(const dms_config& c, const Layout& lo, void* meta, int layer, int n,
                           const int32_t* seq_ids, int32_t* out, hipStream_t st);
hipError_t launch_chunk_commit(const dms_config& c, const Layout& lo, void* meta, void* ws,
                               void* pool, int layer, int n, const int32_t* seq_ids,
                               const int32_t* cu, int total_tokens, int max_len, const void* k,
                               const void* v, const uint8_t* flags, hipStream_t st);
hipError_t launch_prefill_decide(const dms_config& c, const void* q, int total_tokens,
                                 uint8_t* flags, hipStream_t st);
hipError_t launch_prefill_attention(const dms_config& c, const Layout& lo, void* meta, void* ws,
                                    void* pool, int layer, int n, const int32_t* seq_ids,
                                    const int32_t* cu, int total_tokens, int max_len,
                                    const void* q, const void* k, const void* v,
                                    const uint8_t* flags, float* out, hipStream_t st,
                                    hipEvent_t ev_start, hipEvent_t ev_stop);

}  // namespace dms
