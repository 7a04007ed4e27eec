// DMS KV-cache management on the device (paper Sec. 3.2, inference): per-head
// paged slots, delayed eviction through the w-entry ring, in-place slot
// recycling, the free-page stack, chunk commits and sequence release.
//
// Every state change of one call is planned before it is applied, so a call
// that would exhaust the page pool (or overflow a head's page table) changes
// nothing and only records the error in the sticky status word.
#include "dms_common.h"
#include "dms_fp8.h"

namespace dms {
namespace {

constexpr int kPlanThreads = 1024;

__device__ inline int load_status(const int32_t* status) {
  return __atomic_load_n(status, __ATOMIC_RELAXED);
}

// ---------------------------------------------------------------------------
// State initialisation and status
// ---------------------------------------------------------------------------

struct InitArgs {
  char* meta;
  int32_t* ck_err;
  int32_t* head_cnt;
  int32_t* plan_ctr;
  int64_t n_heads;
  size_t layer0, layer_stride, pos, len, ring, page_table, stack, top;
  int64_t n_pos, n_len, n_ring, n_pt;
  int num_pages;
};

__global__ void init_state_kernel(InitArgs a) {
  char* b = a.meta + a.layer0 + static_cast<size_t>(blockIdx.y) * a.layer_stride;
  int32_t* pos = reinterpret_cast<int32_t*>(b + a.pos);
  int32_t* len = reinterpret_cast<int32_t*>(b + a.len);
  int32_t* ring = reinterpret_cast<int32_t*>(b + a.ring);
  int32_t* pt = reinterpret_cast<int32_t*>(b + a.page_table);
  int32_t* stack = reinterpret_cast<int32_t*>(b + a.stack);
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  for (int64_t i = t0; i < a.n_pos; i += stride) pos[i] = 0;
  for (int64_t i = t0; i < a.n_len; i += stride) len[i] = 0;
  for (int64_t i = t0; i < a.n_ring; i += stride) ring[i] = 0;
  for (int64_t i = t0; i < a.n_pt; i += stride) pt[i] = -1;
  for (int64_t i = t0; i < a.num_pages; i += stride) stack[i] = a.num_pages - 1 - static_cast<int32_t>(i);
  if (blockIdx.y == 0)
    for (int64_t i = t0; i < a.n_heads; i += stride) a.head_cnt[i] = 0;
  if (t0 == 0) {
    *reinterpret_cast<int32_t*>(b + a.top) = a.num_pages;
    if (blockIdx.y == 0) {
      *reinterpret_cast<int32_t*>(a.meta) = 0;  // status
      a.ck_err[0] = 0;
      a.ck_err[1] = 0;
      a.plan_ctr[0] = 0;
    }
  }
}

__global__ void set_status_kernel(int32_t* status, int value) {
  if (threadIdx.x == 0) atomicExch(reinterpret_cast<int*>(status), value);
}

// ---------------------------------------------------------------------------
// Sequence-id validation shared by the single-block planners
// ---------------------------------------------------------------------------

// Returns true (in every thread) when some id is out of range or repeated.
__device__ bool bad_seq_ids(const int32_t* seq_ids, int n, int max_seqs, uint32_t* seen) {
  for (int i = threadIdx.x; i < (max_seqs + 31) / 32; i += blockDim.x) seen[i] = 0;
  __syncthreads();
  int bad = 0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    int s = seq_ids[i];
    if (s < 0 || s >= max_seqs) {
      bad = 1;
    } else {
      uint32_t bit = 1u << (s & 31);
      uint32_t old = atomicOr(&seen[s >> 5], bit);
      if (old & bit) bad = 1;
    }
  }
  return __syncthreads_or(bad) != 0;
}

// ---------------------------------------------------------------------------
// Sequence release
// ---------------------------------------------------------------------------

struct ResetArgs {
  char* meta;
  size_t layer0, layer_stride;
  size_t pos, len, ring, page_table, stack, top;
  int32_t* status;
  const int32_t* seq_ids;
  int n, H, w, P, maxp, max_seqs, first_layer;
};

__global__ __launch_bounds__(kPlanThreads) void seq_reset_kernel(ResetArgs a) {
  __shared__ uint32_t seen[kMaxSeqs / 32];
  __shared__ int lds[17];
  __shared__ int s_abort;
  if (threadIdx.x == 0) s_abort = load_status(a.status) != 0;
  __syncthreads();
  if (s_abort) return;
  if (bad_seq_ids(a.seq_ids, a.n, a.max_seqs, seen)) {
    if (threadIdx.x == 0) set_status(a.status, DMS_ERR_BAD_SEQ);
    return;
  }
  char* b = a.meta + a.layer0 + static_cast<size_t>(a.first_layer + blockIdx.x) * a.layer_stride;
  int32_t* pos = reinterpret_cast<int32_t*>(b + a.pos);
  int32_t* len = reinterpret_cast<int32_t*>(b + a.len);
  int32_t* ring = reinterpret_cast<int32_t*>(b + a.ring);
  int32_t* pt = reinterpret_cast<int32_t*>(b + a.page_table);
  int32_t* stack = reinterpret_cast<int32_t*>(b + a.stack);
  int32_t* top = reinterpret_cast<int32_t*>(b + a.top);
  const int NH = a.n * a.H;
  const int top0 = *top;
  int run = 0;
  for (int base = 0; base < NH; base += blockDim.x) {
    const int hh = base + threadIdx.x;
    int np = 0, sh = 0;
    if (hh < NH) {
      sh = a.seq_ids[hh / a.H] * a.H + hh % a.H;
      np = (len[sh] + a.P - 1) / a.P;
    }
    int tot;
    int off = block_exclusive_scan(np, lds, &tot);
    if (hh < NH) {
      for (int k = 0; k < np; ++k) {
        stack[top0 + run + off + k] = pt[static_cast<size_t>(sh) * a.maxp + k];
        pt[static_cast<size_t>(sh) * a.maxp + k] = -1;
      }
      len[sh] = 0;
      for (int e = 0; e < a.w; ++e) ring[static_cast<size_t>(sh) * a.w + e] = 0;
    }
    run += tot;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < a.n; i += blockDim.x) pos[a.seq_ids[i]] = 0;
  if (threadIdx.x == 0) *top = top0 + run;
}

// ---------------------------------------------------------------------------
// Decode append planning (rule R1 for one token per sequence) + per-head
// descriptors and tile prefix sums for the decode kernel
// ---------------------------------------------------------------------------

struct PlanArgs {
  LayerState st;
  int32_t* status;
  const int32_t* seq_ids;
  const uint8_t* flags;  // [n, H] caller decisions, or null
  const uint16_t* q;     // [n, Hq, D] bf16: decisions from the borrowed neuron, or null
  uint8_t* flags_out;    // nullable: decisions taken from q
  float bias;            // offset added to the borrowed neuron
  int immediate;         // eviction timing: token t's own decision frees t - w's slot
  int g, D;
  HeadDesc* desc;        // [n*H]
  int32_t* cum_tiles;    // [n*H + 1]
  int32_t* wave_bounds;  // [W + 1] first tile of every decode wave
  int4* wave_desc;       // [2W] first segment of every decode wave (see decode kernel)
  int4* head_waves;      // [n*H] first / last wave holding a tile of the head, live mask
  float* out;            // nullable: zeroed for heads with no retained token
  const int32_t* len_override;   // nullable (no append): lengths to plan, per head of the call
  int32_t* zero_cnt;     // nullable: split-head arrival counters of the call's heads, cleared
  int n, H, w, P, maxp, max_slots, max_seqs, append, W, gD;
};

// Largest index i in [0, NH] with cum[i] <= b (cum non-decreasing).
__device__ inline int upper_index(const int32_t* cum, int NH, int b) {
  int lo = 0, hi = NH;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cum[mid] <= b) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Descriptor of decode wave w's first segment: its tile range [tb, te), the
// head hh holding tile tb with that head's tile range [c0, c1), retained
// length L, state index sh and appended slot z.
__device__ inline void put_wave_desc(int4* wave_desc, int w, int tb, int te, int hh, int c0,
                                     int c1, const int4& d) {
  wave_desc[2 * w] = make_int4(tb, te, hh, c0);
  wave_desc[2 * w + 1] = make_int4(c1, d.x, d.y, d.z);
}

// Waves wf .. wl hold the head's tiles [c0, c1) (c1 > c0); bit i of the mask
// says whether wave wf + i has a non-empty range (waves past 32 are looked up
// by the merge itself).
__device__ inline int4 head_waves_of(const int32_t* bounds, int W, int c0, int c1) {
  int lo = 0, hi = W - 1;            // largest w with bounds[w] <= c0
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (bounds[mid] <= c0) lo = mid; else hi = mid - 1;
  }
  const int wf = lo;
  lo = wf; hi = W - 1;               // smallest w with bounds[w + 1] >= c1
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (bounds[mid + 1] >= c1) hi = mid; else lo = mid + 1;
  }
  const int wl = lo;
  int mask = 0;
  for (int i = 0; i < 32 && wf + i <= wl; ++i)
    if (bounds[wf + i] < bounds[wf + i + 1]) mask |= 1 << i;
  return make_int4(wf, wl, mask, 0);
}

// Tile range of every decode wave: equal contiguous shares of the flat tile
// list (heads that straddle a boundary are merged by the decode kernel),
// each wave's first-segment descriptor, and every head's wave span.
__device__ void wave_ranges(const PlanArgs& a, int NH) {
  const int32_t* cum = a.cum_tiles;
  const int total = cum[NH], W = a.W;
  for (int w = threadIdx.x; w <= W; w += blockDim.x)
    a.wave_bounds[w] = static_cast<int>(static_cast<int64_t>(w) * total / W);
  for (int w = threadIdx.x; w < W; w += blockDim.x) {
    const int tb = static_cast<int>(static_cast<int64_t>(w) * total / W);
    const int te = static_cast<int>(static_cast<int64_t>(w + 1) * total / W);
    if (tb < te) {
      const int hh = min(upper_index(cum, NH, tb), NH - 1);
      put_wave_desc(a.wave_desc, w, tb, te, hh, cum[hh], cum[hh + 1], a.desc[hh]);
    }
  }
  __syncthreads();  // bounds visible to the searches below
  for (int hh = threadIdx.x; hh < NH; hh += blockDim.x)
    if (cum[hh + 1] > cum[hh]) a.head_waves[hh] = head_waves_of(a.wave_bounds, W, cum[hh], cum[hh + 1]);
}

// Decision of the token appended for call head hh: the caller's flag, or
// round(sigmoid(x)) = (x > 0) with x = bf16 element 0 of the first query
// head of the group plus the offset, in float32 (Sec. 3.2, App. C).
__device__ inline int decision(const PlanArgs& a, int hh) {
  return token_decision(a.flags, a.q, hh, a.H, a.g, a.D, a.bias);
}

// Whether the incoming token takes the slot of the token that entered w
// steps ago (ring entry e): delayed eviction -- that token was flagged;
// immediate eviction -- the incoming token's decision evicts it now.
__device__ inline bool takes_slot(const PlanArgs& a, int t, int32_t e, int f) {
  return takes_old_slot(t, a.w, e, f, a.immediate);
}

struct HeadStep {
  int sh, t, slot, reuse, f;
};

__device__ inline HeadStep r1_step(const PlanArgs& a, int hh) {
  HeadStep r;
  const int s = a.seq_ids[hh / a.H];
  r.sh = s * a.H + hh % a.H;
  r.t = a.st.pos[s];
  r.f = decision(a, hh);
  const int32_t e = a.st.ring[static_cast<size_t>(r.sh) * a.w + r.t % a.w];
  r.reuse = takes_slot(a, r.t, e, r.f);
  r.slot = r.reuse ? static_cast<int>(static_cast<uint32_t>(e) & ~kFlagBit) : a.st.len[r.sh];
  return r;
}

// Decode planning when every head of the call has its own thread (n*H <=
// 1024, the usual case).  The dependent global loads are kept to three rounds:
// (status, stack height, sequence ids) -> (pos, L, top of the free stack into
// LDS) -> the ring entry; both prefix sums (page pops, decode tiles) share one
// scan, and each wave's first head is computed arithmetically from the tile
// prefix sums.
__global__ __launch_bounds__(kPlanThreads) void plan_small_kernel(PlanArgs a) {
  __shared__ uint32_t seen[kMaxSeqs / 32];
  __shared__ int lds2[34];
  __shared__ int32_t stack_lds[kPlanThreads];
  __shared__ int s_bad;
  const int tid = threadIdx.x;
  const int NH = a.n * a.H;
  const int status = load_status(a.status);
  const int top0 = *a.st.top;
  const bool act = tid < NH;
  const int s = act ? a.seq_ids[tid / a.H] : 0;
  for (int i = tid; i < (a.max_seqs + 31) / 32; i += blockDim.x) seen[i] = 0;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  if (status != 0) return;
  // one thread per sequence checks its id: in range and not repeated
  if (act && tid % a.H == 0) {
    if (s < 0 || s >= a.max_seqs) {
      s_bad = 1;
    } else {
      const uint32_t bit = 1u << (s & 31);
      if (atomicOr(&seen[s >> 5], bit) & bit) s_bad = 1;
    }
  }
  __syncthreads();
  if (s_bad) {
    if (tid == 0) set_status(a.status, DMS_ERR_BAD_SEQ);
    return;
  }
  const int sh = s * a.H + tid % a.H;
  int t = 0, slot = -1, fresh = 0, need = 0, Lnew = 0, cap = 0, f = 0;
  if (a.append && tid < min(NH, top0)) stack_lds[tid] = a.st.stack[top0 - 1 - tid];
  if (act) {
    const int L = (!a.append && a.len_override != nullptr) ? a.len_override[tid] : a.st.len[sh];
    if (a.append) {
      f = decision(a, tid);
      t = a.st.pos[s];
      const int32_t e = a.st.ring[static_cast<size_t>(sh) * a.w + t % a.w];
      const bool reuse = takes_slot(a, t, e, f);
      slot = reuse ? static_cast<int>(static_cast<uint32_t>(e) & ~kFlagBit) : L;
      fresh = !reuse;
      cap = fresh && slot >= a.max_slots;
      need = fresh && (slot % a.P) == 0;
    }
    Lnew = L + fresh;
  }
  const int tiles = (Lnew + kTile - 1) / kTile;
  int2 tot;
  const int2 ex = block_exclusive_scan2(make_int2(need, tiles), lds2, &tot);  // barriers
  if (a.append) {
    cap = __syncthreads_or(cap);
    if (cap || tot.x > top0) {
      if (tid == 0) set_status(a.status, cap ? DMS_ERR_CAPACITY : DMS_ERR_OUT_OF_PAGES);
      return;
    }
  }
  const int c0 = ex.y, c1 = ex.y + tiles;
  if (act) {
    if (a.append) {
      const uint32_t fb = f ? kFlagBit : 0u;
      if (a.flags_out != nullptr) a.flags_out[tid] = static_cast<uint8_t>(f);
      if (need) a.st.page_table[static_cast<size_t>(sh) * a.maxp + slot / a.P] = stack_lds[ex.x];
      if (fresh) a.st.len[sh] = Lnew;
      a.st.ring[static_cast<size_t>(sh) * a.w + t % a.w] = static_cast<int32_t>(static_cast<uint32_t>(slot) | fb);
      a.st.slot_meta[static_cast<size_t>(sh) * a.max_slots + slot] = static_cast<int32_t>(static_cast<uint32_t>(t) | fb);
      // every head of the sequence read pos before the scan's barriers
      if (tid % a.H == 0) a.st.pos[s] = t + 1;
    }
    a.desc[tid] = make_int4(Lnew, sh, slot, 0);
    a.cum_tiles[tid + 1] = c1;
    if (a.zero_cnt != nullptr) a.zero_cnt[tid] = 0;
    if (a.out != nullptr && Lnew == 0)
      for (int e = 0; e < a.gD; ++e) a.out[static_cast<size_t>(tid) * a.gD + e] = 0.f;
  }
  if (tid == 0) {
    a.cum_tiles[0] = 0;
    if (a.append) *a.st.top = top0 - tot.x;
  }
  if (a.W > 0) {
    // wave w starts at tile floor(w * total / W); the head holding tiles
    // [c0, c1) is where every wave w with ceil(c0 * W / total) <= w <
    // ceil(c1 * W / total) starts, and its tiles lie in waves
    // ceil((c0 + 1) * W / total) - 1 .. ceil(c1 * W / total) - 1
    const int64_t total = tot.y, W = a.W;
    auto bound = [&](int64_t w) { return static_cast<int>(w * total / W); };
    for (int w = tid; w <= a.W; w += blockDim.x) a.wave_bounds[w] = bound(w);
    if (act && c1 > c0) {
      const int w0 = static_cast<int>((c0 * W + total - 1) / total);
      const int w1 = min(a.W, static_cast<int>((c1 * W + total - 1) / total));
      const int4 d = make_int4(Lnew, sh, slot, 0);
      for (int w = w0; w < w1; ++w) put_wave_desc(a.wave_desc, w, bound(w), bound(w + 1), tid, c0, c1, d);
      const int wf = static_cast<int>(((c0 + 1) * W + total - 1) / total) - 1;
      const int wl = min(a.W - 1, w1 - 1);
      int mask = 0;
      for (int i = 0; i < 32 && wf + i <= wl; ++i)
        if (bound(wf + i) < bound(wf + i + 1)) mask |= 1 << i;
      a.head_waves[tid] = make_int4(wf, wl, mask, 0);
    }
  }
}

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(PlanArgs a) {
  __shared__ uint32_t seen[kMaxSeqs / 32];
  __shared__ int lds[17];
  __shared__ int s_abort;
  if (threadIdx.x == 0) s_abort = load_status(a.status) != 0;
  __syncthreads();
  if (s_abort) return;
  if (bad_seq_ids(a.seq_ids, a.n, a.max_seqs, seen)) {
    if (threadIdx.x == 0) set_status(a.status, DMS_ERR_BAD_SEQ);
    return;
  }
  const int NH = a.n * a.H;
  const int top0 = *a.st.top;
  int total_need = 0;
  if (a.append) {
    int cap = 0;
    for (int base = 0; base < NH; base += blockDim.x) {
      const int hh = base + threadIdx.x;
      int need = 0;
      if (hh < NH) {
        HeadStep r = r1_step(a, hh);
        if (!r.reuse) {
          if (r.slot >= a.max_slots) cap = 1;
          need = (r.slot % a.P) == 0;
        }
      }
      int tot;
      block_exclusive_scan(need, lds, &tot);
      total_need += tot;
    }
    cap = __syncthreads_or(cap);
    if (cap || total_need > top0) {
      if (threadIdx.x == 0) set_status(a.status, cap ? DMS_ERR_CAPACITY : DMS_ERR_OUT_OF_PAGES);
      return;
    }
  }
  int run_pop = 0, run_tiles = 0;
  for (int base = 0; base < NH; base += blockDim.x) {
    const int hh = base + threadIdx.x;
    int need = 0, tiles = 0, Lnew = 0, slot = -1, sh = 0, t = 0, fresh = 0, f = 0;
    if (hh < NH) {
      if (a.append) {
        HeadStep r = r1_step(a, hh);
        sh = r.sh;
        t = r.t;
        slot = r.slot;
        f = r.f;
        fresh = !r.reuse;
        need = fresh && (slot % a.P) == 0;
        Lnew = a.st.len[sh] + fresh;
      } else {
        sh = a.seq_ids[hh / a.H] * a.H + hh % a.H;
        Lnew = a.len_override != nullptr ? a.len_override[hh] : a.st.len[sh];
      }
      tiles = (Lnew + kTile - 1) / kTile;
    }
    int totp, tott;
    const int pop = run_pop + block_exclusive_scan(need, lds, &totp);
    const int ct = run_tiles + block_exclusive_scan(tiles, lds, &tott);
    if (hh < NH) {
      if (a.append) {
        const uint32_t fb = f ? kFlagBit : 0u;
        if (a.flags_out != nullptr) a.flags_out[hh] = static_cast<uint8_t>(f);
        if (need) a.st.page_table[static_cast<size_t>(sh) * a.maxp + slot / a.P] = a.st.stack[top0 - 1 - pop];
        if (fresh) a.st.len[sh] = Lnew;
        a.st.ring[static_cast<size_t>(sh) * a.w + t % a.w] = static_cast<int32_t>(static_cast<uint32_t>(slot) | fb);
        a.st.slot_meta[static_cast<size_t>(sh) * a.max_slots + slot] = static_cast<int32_t>(static_cast<uint32_t>(t) | fb);
      }
      a.desc[hh] = make_int4(Lnew, sh, slot, 0);
      a.cum_tiles[hh + 1] = ct + tiles;
      if (a.zero_cnt != nullptr) a.zero_cnt[hh] = 0;
      if (a.out != nullptr && Lnew == 0)
        for (int e = 0; e < a.gD; ++e) a.out[static_cast<size_t>(hh) * a.gD + e] = 0.f;
    }
    run_pop += totp;
    run_tiles += tott;
  }
  if (threadIdx.x == 0) a.cum_tiles[0] = 0;
  __syncthreads();  // every read of pos above happens before these writes
  if (a.append) {
    for (int i = threadIdx.x; i < a.n; i += blockDim.x) a.st.pos[a.seq_ids[i]] += 1;
    if (threadIdx.x == 0) *a.st.top = top0 - total_need;
  }
  if (a.W > 0) wave_ranges(a, NH);
}

// Copy each appended token's K row and V column into its slot.
struct ScatterArgs {
  const int32_t* status;
  const HeadDesc* desc;
  const int32_t* page_table;
  char* pool;
  const uint16_t* k;
  const uint16_t* v;
  size_t page_bytes;
  int D, P, maxp;
  int fp8;   // FP8 pages: rows are quantized on the way in
  int mla;   // latent-attention pages: the key row only
};

__global__ __launch_bounds__(64) void scatter_kernel(ScatterArgs a) {
  if (load_status(a.status) != 0) return;
  const int hh = blockIdx.x;
  const HeadDesc d = a.desc[hh];
  const int slot = d.z;
  const int page = a.page_table[static_cast<size_t>(d.y) * a.maxp + slot / a.P];
  const int row = slot % a.P;
  const int j = row & 31;
  const int lane = threadIdx.x;
  if (a.mla) {
    char* tile = a.pool + static_cast<size_t>(page) * a.page_bytes + (row >> 5) * mla_tile_bytes(a.D);
    for (int part = lane; part < a.D / 8; part += 64)
      *reinterpret_cast<uint4*>(tile + k_elem_off(j, 8 * part)) =
          reinterpret_cast<const uint4*>(a.k + static_cast<size_t>(hh) * a.D)[part];
    return;
  }
  char* tile = a.pool + static_cast<size_t>(page) * a.page_bytes +
               (row >> 5) * (a.fp8 ? fp8_tile_bytes(a.D) : tile_bytes(a.D));
  store_token_kv(tile, j, a.D, lane, a.fp8, a.k + static_cast<size_t>(hh) * a.D, a.v + static_cast<size_t>(hh) * a.D);
}

struct RetainedArgs {
  const int32_t* len;
  const int32_t* seq_ids;
  int32_t* out;
  int n, H;
};

__global__ void retained_kernel(RetainedArgs a) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < a.n * a.H) a.out[i] = a.len[a.seq_ids[i / a.H] * a.H + i % a.H];
}

// ---------------------------------------------------------------------------
// Chunk commit: rule R1 applied to C tokens of each (sequence, head) at once.
//
// For chunk token c at position t = pos0 + c: it reuses the slot of position
// t - w iff t >= w and that token was flagged ("reuse"); otherwise it is
// fresh and takes slot L0 + (number of fresh chunk tokens before c).  A
// reusing token's slot is found by walking back in steps of w until a fresh
// chunk token or a position from before the chunk (read from the ring).
// Only tokens whose slot is not taken over later inside the chunk write K/V.
// ---------------------------------------------------------------------------

struct ChunkArgs {
  LayerState st;
  int32_t* status;
  const int32_t* seq_ids;
  const int32_t* cu;
  const uint8_t* flags;   // [T, H]
  const uint16_t* k;      // [T, H, D]
  const uint16_t* v;
  char* pool;
  size_t page_bytes;
  int32_t* need;          // [n*H] pages to pop per head
  int32_t* fresh;         // [n*H] fresh tokens per head
  int32_t* base;          // [n*H] first pop index per head
  int32_t* pos0;          // [n] position of each sequence before the chunk
  int32_t* err;           // call-local error word, err[1] = stack height before the call
  int32_t* slots;         // [T, H] slot of every chunk token
  int n, H, w, P, D, maxp, max_slots, max_seqs, total, max_len;
  int immediate;          // eviction timing (see chunk_reuse)
  int fp8;                // FP8 pages: rows are quantized on the way in
  int mla;                // latent-attention pages: the key row only
};

__device__ inline int chunk_flag(const ChunkArgs& a, int tok0, int c, int h) {
  return a.flags[static_cast<size_t>(tok0 + c) * a.H + h] != 0;
}

// Does chunk token c (position pos0 + c) reuse the slot of position pos0 + c - w?
// Delayed eviction: iff that token was flagged; immediate: iff token c is.
__device__ inline bool chunk_reuse(const ChunkArgs& a, int sh, int h, int tok0, int pos0, int c) {
  const int t = pos0 + c;
  if (t < a.w) return false;
  if (a.immediate) return chunk_flag(a, tok0, c, h);
  const int j = c - a.w;
  if (j >= 0) return chunk_flag(a, tok0, j, h);
  const int32_t e = a.st.ring[static_cast<size_t>(sh) * a.w + (t - a.w) % a.w];
  return (static_cast<uint32_t>(e) & kFlagBit) != 0;
}

constexpr int kChunkTPT = 16;   // consecutive chunk tokens per thread in the scans

// Pass 1 (one block per head): count fresh tokens and the pages they need,
// and give every fresh token its slot (L0 + its index among the fresh ones;
// the slot array is scratch, so writing it before validation is harmless).
// Each thread takes kChunkTPT consecutive tokens (their flags are loaded
// together), so a 4096-token chunk needs one block scan.
__global__ __launch_bounds__(256) void chunk_count_kernel(ChunkArgs a) {
  __shared__ int lds[17];
  if (load_status(a.status) != 0) return;
  const int hh = blockIdx.x;
  const int i = hh / a.H, h = hh % a.H;
  const int s = a.seq_ids[i];
  const int tok0 = a.cu[i], C = a.cu[i + 1] - a.cu[i];
  bool bad = (s < 0 || s >= a.max_seqs || C < 0 || C > a.max_len || a.cu[0] != 0 ||
              a.cu[a.n] != a.total || tok0 < 0 || tok0 + C > a.total);
  if (bad) {
    if (threadIdx.x == 0) atomicCAS(reinterpret_cast<int*>(a.err), 0, DMS_ERR_INVALID);
    return;
  }
  const int sh = s * a.H + h;
  const int pos0 = a.st.pos[s];
  const int L0 = a.st.len[sh];
  int32_t* slots = a.slots + static_cast<size_t>(tok0) * a.H + h;   // token c at c * H
  int cnt = 0;
  for (int base = 0; base < C; base += blockDim.x * kChunkTPT) {
    const int c0 = base + threadIdx.x * kChunkTPT;
    bool f[kChunkTPT];
    int mine = 0;
#pragma unroll
    for (int u = 0; u < kChunkTPT; ++u) {
      f[u] = c0 + u < C && !chunk_reuse(a, sh, h, tok0, pos0, c0 + u);
      mine += f[u];
    }
    int tot;
    int k = L0 + cnt + block_exclusive_scan(mine, lds, &tot);
#pragma unroll
    for (int u = 0; u < kChunkTPT; ++u)
      if (f[u]) slots[static_cast<size_t>(c0 + u) * a.H] = k++;
    cnt += tot;
  }
  if (threadIdx.x == 0) {
    const int L1 = L0 + cnt;
    if (L1 > a.max_slots) atomicCAS(reinterpret_cast<int*>(a.err), 0, DMS_ERR_CAPACITY);
    a.fresh[hh] = cnt;
    a.need[hh] = (L1 + a.P - 1) / a.P - (L0 + a.P - 1) / a.P;
    if (h == 0) a.pos0[i] = pos0;
  }
}

// Pass 2 (one block): validate ids, order the pops, reserve the pages.
__global__ __launch_bounds__(kPlanThreads) void chunk_pages_kernel(ChunkArgs a) {
  __shared__ uint32_t seen[kMaxSeqs / 32];
  __shared__ int lds[17];
  __shared__ int s_abort;
  if (threadIdx.x == 0) s_abort = load_status(a.status) != 0;
  __syncthreads();
  if (s_abort) return;
  // pass 1 of this call ran iff this pass runs: consume and clear its error word
  const int err = *a.err;
  __syncthreads();
  if (threadIdx.x == 0) a.err[0] = 0;
  if (bad_seq_ids(a.seq_ids, a.n, a.max_seqs, seen)) {
    if (threadIdx.x == 0) set_status(a.status, DMS_ERR_BAD_SEQ);
    return;
  }
  const int NH = a.n * a.H;
  const int top0 = *a.st.top;
  int run = 0;
  for (int base = 0; base < NH; base += blockDim.x) {
    const int hh = base + threadIdx.x;
    const int nd = hh < NH ? a.need[hh] : 0;
    int tot;
    const int off = block_exclusive_scan(nd, lds, &tot);
    if (hh < NH) a.base[hh] = run + off;
    run += tot;
  }
  if (threadIdx.x == 0) {
    if (err != 0) {
      set_status(a.status, err);
    } else if (run > top0) {
      set_status(a.status, DMS_ERR_OUT_OF_PAGES);
    } else {
      *a.st.top = top0 - run;
      a.err[1] = top0;
    }
  }
  __syncthreads();
  // positions advance here: pass 1 has read them, pass 3 uses pos0
  if (err == 0 && run <= top0)
    for (int i = threadIdx.x; i < a.n; i += blockDim.x)
      a.st.pos[a.seq_ids[i]] = a.pos0[i] + (a.cu[i + 1] - a.cu[i]);
}

// Pass 3 (one block per head): reused slots, page table, ring, slot metadata.
__global__ __launch_bounds__(256) void chunk_commit_kernel(ChunkArgs a) {
  if (load_status(a.status) != 0) return;
  const int top_before = a.err[1];
  const int hh = blockIdx.x;
  const int i = hh / a.H, h = hh % a.H;
  const int s = a.seq_ids[i];
  const int sh = s * a.H + h;
  const int tok0 = a.cu[i], C = a.cu[i + 1] - a.cu[i];
  const int pos0 = a.pos0[i];
  const int L0 = a.st.len[sh];
  const size_t pt_base = static_cast<size_t>(sh) * a.maxp;
  int32_t* slots = a.slots + static_cast<size_t>(tok0) * a.H + h;   // token c at c * H
  // new pages, popped in page-index order from this head's reserved range
  const int first_new_page = (L0 + a.P - 1) / a.P;
  for (int k = threadIdx.x; k < a.need[hh]; k += blockDim.x)
    a.st.page_table[pt_base + first_new_page + k] = a.st.stack[top_before - 1 - (a.base[hh] + k)];
  // Reused slots (fresh ones were assigned by pass 1).  A token that reuses
  // takes the slot of the token w before it, so along one residue class
  // c = r, r + w, r + 2w, ... every token holds the slot of the latest fresh
  // token of the class before it, or, for the first ones, the slot the ring
  // gives for position pos0 + r - w.  One forward walk per class, its flags
  // and fresh slots loaded kChunkTPT members at a time.
  for (int r = threadIdx.x; r < min(a.w, C); r += blockDim.x) {
    int carried = -1;
    if (pos0 + r >= a.w) {
      const int32_t e = a.st.ring[static_cast<size_t>(sh) * a.w + (pos0 + r) % a.w];
      carried = static_cast<int>(static_cast<uint32_t>(e) & ~kFlagBit);
    }
    for (int c0 = r; c0 < C; c0 += kChunkTPT * a.w) {
      bool ru[kChunkTPT];
      int sl[kChunkTPT];
#pragma unroll
      for (int u = 0; u < kChunkTPT; ++u) {
        const int c = c0 + u * a.w;
        ru[u] = c < C && chunk_reuse(a, sh, h, tok0, pos0, c);
        sl[u] = (c < C && !ru[u]) ? slots[static_cast<size_t>(c) * a.H] : 0;
      }
#pragma unroll
      for (int u = 0; u < kChunkTPT; ++u) {
        const int c = c0 + u * a.w;
        if (c >= C) break;
        if (ru[u]) slots[static_cast<size_t>(c) * a.H] = carried;
        else carried = sl[u];
      }
    }
  }
  __syncthreads();  // ring reads above complete before the ring is rewritten
  const int ring_from = C > a.w ? C - a.w : 0;
  for (int c = threadIdx.x; c < C; c += blockDim.x) {
    const int fl = chunk_flag(a, tok0, c, h);
    const uint32_t fb = fl ? kFlagBit : 0u;
    const int slot = slots[static_cast<size_t>(c) * a.H];
    if (c >= ring_from)
      a.st.ring[static_cast<size_t>(sh) * a.w + (pos0 + c) % a.w] =
          static_cast<int32_t>(static_cast<uint32_t>(slot) | fb);
    // a token keeps its slot unless the token w later in the chunk takes it
    const bool survives = (c + a.w >= C) || !chunk_reuse(a, sh, h, tok0, pos0, c + a.w);
    if (survives)
      a.st.slot_meta[static_cast<size_t>(sh) * a.max_slots + slot] =
          static_cast<int32_t>(static_cast<uint32_t>(pos0 + c) | fb);
  }
  if (threadIdx.x == 0) a.st.len[sh] = L0 + a.fresh[hh];
}

// Pass 4 (blocks of 256 / (D/8) tokens of one head): K rows and V columns of
// the surviving tokens into their slots, D/8 consecutive lanes per token (an
// aligned lane group: the block size is a multiple of it, so a group is
// entirely inside or outside the chunk and takes every branch together).
// The page table entries of pass 3 are complete: separate launch.
__global__ __launch_bounds__(256) void chunk_copy_kernel(ChunkArgs a) {
  if (load_status(a.status) != 0) return;
  const int hh = blockIdx.y;
  const int i = hh / a.H, h = hh % a.H;
  const int tok0 = a.cu[i], C = a.cu[i + 1] - a.cu[i];
  const int kq = a.D / 8;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= C * kq) return;
  const int c = idx / kq, part = idx % kq;
  const int s = a.seq_ids[i];
  const int sh = s * a.H + h;
  const int pos0 = a.pos0[i];
  if (!((c + a.w >= C) || !chunk_reuse(a, sh, h, tok0, pos0, c + a.w))) return;
  const int slot = a.slots[static_cast<size_t>(tok0 + c) * a.H + h];
  const int page = a.st.page_table[static_cast<size_t>(sh) * a.maxp + slot / a.P];
  const int row = slot % a.P;
  const int j = row & 31;
  const size_t src = (static_cast<size_t>(tok0 + c) * a.H + h) * a.D;
  const uint4 kx = reinterpret_cast<const uint4*>(a.k + src)[part];
  if (a.mla) {
    char* tile = a.pool + static_cast<size_t>(page) * a.page_bytes + (row >> 5) * mla_tile_bytes(a.D);
    *reinterpret_cast<uint4*>(tile + k_elem_off(j, 8 * part)) = kx;
    return;
  }
  const uint4 vx = reinterpret_cast<const uint4*>(a.v + src)[part];
  if (a.fp8) {
    char* tile = a.pool + static_cast<size_t>(page) * a.page_bytes + (row >> 5) * fp8_tile_bytes(a.D);
    fp8_store_token(tile, j, a.D, part, kx, vx);
    return;
  }
  char* tile = a.pool + static_cast<size_t>(page) * a.page_bytes + (row >> 5) * tile_bytes(a.D);
  *reinterpret_cast<uint4*>(tile + k_elem_off(j, 8 * part)) = kx;
  const uint32_t vw[4] = {vx.x, vx.y, vx.z, vx.w};
#pragma unroll
  for (int e = 0; e < 8; ++e)
    *reinterpret_cast<uint16_t*>(tile + v_elem_off(j, part * 8 + e, a.D)) =
        static_cast<uint16_t>(vw[e >> 1] >> (16 * (e & 1)));
}

}  // namespace

hipError_t launch_init_state(const dms_config& c, const Layout& lo, void* meta, void* ws,
                             hipStream_t st) {
  InitArgs a;
  a.meta = static_cast<char*>(meta);
  a.ck_err = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + lo.ws_ck_err);
  a.head_cnt = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + lo.ws_head_cnt);
  a.plan_ctr = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + lo.ws_plan_ctr);
  a.n_heads = static_cast<int64_t>(lo.max_heads) * lo.head_groups;
  a.layer0 = lo.layer0;
  a.layer_stride = lo.layer_stride;
  a.pos = lo.pos;
  a.len = lo.len;
  a.ring = lo.ring;
  a.page_table = lo.page_table;
  a.stack = lo.stack;
  a.top = lo.top;
  a.n_pos = c.max_seqs;
  a.n_len = static_cast<int64_t>(c.max_seqs) * c.num_kv_heads;
  a.n_ring = a.n_len * c.window;
  a.n_pt = a.n_len * c.max_pages_per_head;
  a.num_pages = c.num_pages;
  dim3 grid(256, c.num_layers);
  hipLaunchKernelGGL(init_state_kernel, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_set_status(int32_t* status, int value, hipStream_t st) {
  hipLaunchKernelGGL(set_status_kernel, dim3(1), dim3(64), 0, st, status, value);
  return hipGetLastError();
}

hipError_t launch_seq_reset(const dms_config& c, const Layout& lo, void* meta, int layer, int n,
                            const int32_t* seq_ids, hipStream_t st) {
  ResetArgs a;
  a.meta = static_cast<char*>(meta);
  a.layer0 = lo.layer0;
  a.layer_stride = lo.layer_stride;
  a.pos = lo.pos;
  a.len = lo.len;
  a.ring = lo.ring;
  a.page_table = lo.page_table;
  a.stack = lo.stack;
  a.top = lo.top;
  a.status = reinterpret_cast<int32_t*>(static_cast<char*>(meta) + lo.status);
  a.seq_ids = seq_ids;
  a.n = n;
  a.H = c.num_kv_heads;
  a.w = c.window;
  a.P = c.page_size;
  a.maxp = c.max_pages_per_head;
  a.max_seqs = c.max_seqs;
  a.first_layer = layer < 0 ? 0 : layer;
  const int nl = layer < 0 ? c.num_layers : 1;
  hipLaunchKernelGGL(seq_reset_kernel, dim3(nl), dim3(kPlanThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_plan(const dms_config& c, const Layout& lo, void* meta, void* ws, int layer,
                       int n, const int32_t* seq_ids, const uint8_t* flags, const void* q,
                       uint8_t* flags_out, bool append, int waves, float* out, hipStream_t st,
                       const int32_t* len_override, bool clear_head_counts) {
  PlanArgs a;
  a.len_override = len_override;
  a.zero_cnt = clear_head_counts
                   ? reinterpret_cast<int32_t*>(static_cast<char*>(ws) + lo.ws_head_cnt)
                   : nullptr;
  a.q = static_cast<const uint16_t*>(q);
  a.flags_out = flags_out;
  a.bias = c.decision_bias;
  a.immediate = c.eviction == DMS_EVICT_IMMEDIATE;
  a.g = c.group_size;
  a.D = c.head_dim;
  a.wave_bounds = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + lo.ws_wave_bounds);
  a.wave_desc = reinterpret_cast<int4*>(static_cast<char*>(ws) + lo.ws_wave_desc);
  a.head_waves = reinterpret_cast<int4*>(static_cast<char*>(ws) + lo.ws_head_waves);
  a.out = out;
  a.W = waves;
  // output row of a call head: g query heads of head_dim (of the latent width
  // for a latent-attention cache)
  a.gD = c.group_size * (c.kv_format == DMS_KV_MLA ? kMlaLatent : c.head_dim);
  a.st = layer_state(lo, meta, layer);
  a.status = reinterpret_cast<int32_t*>(static_cast<char*>(meta) + lo.status);
  a.seq_ids = seq_ids;
  a.flags = flags;
  a.desc = reinterpret_cast<HeadDesc*>(static_cast<char*>(ws) + lo.ws_head_desc);
  a.cum_tiles = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + lo.ws_cum_tiles);
  a.n = n;
  a.H = c.num_kv_heads;
  a.w = c.window;
  a.P = c.page_size;
  a.maxp = c.max_pages_per_head;
  a.max_slots = lo.max_slots;
  a.max_seqs = c.max_seqs;
  a.append = append ? 1 : 0;
  if (n * c.num_kv_heads <= kPlanThreads)
    hipLaunchKernelGGL(plan_small_kernel, dim3(1), dim3(kPlanThreads), 0, st, a);
  else
    hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_scatter(const dms_config& c, const Layout& lo, void* meta, void* ws, void* pool,
                          int layer, int n, const void* k, const void* v, hipStream_t st) {
  ScatterArgs a;
  LayerState s = layer_state(lo, meta, layer);
  a.status = reinterpret_cast<const int32_t*>(static_cast<char*>(meta) + lo.status);
  a.desc = reinterpret_cast<const HeadDesc*>(static_cast<char*>(ws) + lo.ws_head_desc);
  a.page_table = s.page_table;
  a.pool = static_cast<char*>(pool);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.page_bytes = lo.page_bytes;
  a.D = c.head_dim;
  a.P = c.page_size;
  a.maxp = c.max_pages_per_head;
  a.fp8 = c.kv_format == DMS_KV_FP8;
  a.mla = c.kv_format == DMS_KV_MLA;
  hipLaunchKernelGGL(scatter_kernel, dim3(n * c.num_kv_heads), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_retained(const dms_config& c, const Layout& lo, void* meta, int layer, int n,
                           const int32_t* seq_ids, int32_t* out, hipStream_t st) {
  RetainedArgs a;
  a.len = layer_state(lo, meta, layer).len;
  a.seq_ids = seq_ids;
  a.out = out;
  a.n = n;
  a.H = c.num_kv_heads;
  const int total = n * c.num_kv_heads;
  hipLaunchKernelGGL(retained_kernel, dim3((total + 255) / 256), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_chunk_commit(const dms_config& c, const Layout& lo, void* meta, void* ws,
                               void* pool, int layer, int n, const int32_t* seq_ids,
                               const int32_t* cu, int total_tokens, int max_len, const void* k,
                               const void* v, const uint8_t* flags, hipStream_t st) {
  ChunkArgs a;
  char* w = static_cast<char*>(ws);
  a.st = layer_state(lo, meta, layer);
  a.status = reinterpret_cast<int32_t*>(static_cast<char*>(meta) + lo.status);
  a.seq_ids = seq_ids;
  a.cu = cu;
  a.flags = flags;
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.pool = static_cast<char*>(pool);
  a.page_bytes = lo.page_bytes;
  a.need = reinterpret_cast<int32_t*>(w + lo.ws_ck_need);
  a.fresh = reinterpret_cast<int32_t*>(w + lo.ws_ck_fresh);
  a.base = reinterpret_cast<int32_t*>(w + lo.ws_ck_base);
  a.pos0 = reinterpret_cast<int32_t*>(w + lo.ws_ck_pos0);
  a.err = reinterpret_cast<int32_t*>(w + lo.ws_ck_err);
  a.slots = reinterpret_cast<int32_t*>(w + lo.ws_ck_slot);
  a.n = n;
  a.H = c.num_kv_heads;
  a.w = c.window;
  a.P = c.page_size;
  a.D = c.head_dim;
  a.maxp = c.max_pages_per_head;
  a.max_slots = lo.max_slots;
  a.max_seqs = c.max_seqs;
  a.total = total_tokens;
  a.max_len = max_len;
  a.immediate = c.eviction == DMS_EVICT_IMMEDIATE;
  a.fp8 = c.kv_format == DMS_KV_FP8;
  a.mla = c.kv_format == DMS_KV_MLA;
  const int NH = n * c.num_kv_heads;
  hipLaunchKernelGGL(chunk_count_kernel, dim3(NH), dim3(256), 0, st, a);
  hipLaunchKernelGGL(chunk_pages_kernel, dim3(1), dim3(kPlanThreads), 0, st, a);
  hipLaunchKernelGGL(chunk_commit_kernel, dim3(NH), dim3(256), 0, st, a);
  if (max_len > 0) {
    const int per_block = 256 / (c.head_dim / 8);   // tokens per copy block
    hipLaunchKernelGGL(chunk_copy_kernel, dim3((max_len + per_block - 1) / per_block, NH), dim3(256), 0,
                       st, a);
  }
  return hipGetLastError();
}

}  // namespace dms
