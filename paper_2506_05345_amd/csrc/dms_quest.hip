// Page retrieval within the DMS retained set (Quest on top of DMS), gfx950.
//
// The paper notes that DMS compresses the KV cache while Quest retrieves
// cache items, so the two can be combined (App. A).  Quest bounds the score
// any key of a page can reach by U = sum_i max(q_i lo_i, q_i hi_i), lo / hi
// the channel-wise min / max of the page's keys, and attends only the pages
// with the largest bounds.  Here the unit is the cache's own page (P slots of
// one KV head holding retained tokens of any positions):
//   * quest_bounds_kernel recomputes lo / hi exactly over a page's live slots
//     whenever an append writes into it (DMS reuses evicted tokens' slots, so
//     bounds can shrink as well as grow);
//   * quest_select_kernel scores every page of a head for its query group
//     (maximum of U over the group's heads, float32 sums in dimension order),
//     keeps the B best (ties to the lower page index) in ascending order and
//     the number of live slots they hold, which the decode planner then
//     splits into tiles like any retained length.
#include "dms_common.h"
#include "dms_fp8.h"

namespace dms {
namespace {

constexpr int kQThreads = 256;
constexpr int kMaxSortPages = 4096;   // max_pages_per_head limit with a budget

struct QuestArgs {
  LayerState st;
  const int32_t* status;
  const HeadDesc* desc;     // after an append: the slot each head wrote (z)
  const int32_t* seq_ids;
  const char* pool;
  const uint16_t* q;        // [n, Hq, D] bf16
  int32_t* sel;             // [NH][B] attended page-table indices, ascending
  int32_t* qlen;            // [NH] live slots in the attended pages
  size_t page_bytes;
  int n, H, g, D, P, maxp, B, fp8, zero_neuron, all_pages;
};

__device__ inline int load_status(const int32_t* status) {
  return __atomic_load_n(status, __ATOMIC_RELAXED);
}

__device__ inline uint16_t f32_to_bf16_exact(float x) {
  // x is a bf16 value (a stored key, or an E4M3 code times a power of two)
  return static_cast<uint16_t>(__float_as_uint(x) >> 16);
}

// Key element (row r of the page, dim d) as stored.
__device__ inline float key_elem(const QuestArgs& a, const char* page, int r, int d) {
  if (a.fp8) {
    const char* tile = page + static_cast<size_t>(r >> 5) * fp8_tile_bytes(a.D);
    const int j = r & 31;
    const uint32_t code = *reinterpret_cast<const uint8_t*>(tile + fp8_k_off(j, d));
    const float scale = *reinterpret_cast<const float*>(tile + fp8_ks_off(j, a.D));
    return __builtin_amdgcn_cvt_pk_f32_fp8(code, false)[0] * scale;   // exact
  }
  const char* tile = page + static_cast<size_t>(r >> 5) * tile_bytes(a.D);
  const uint32_t bits = *reinterpret_cast<const uint16_t*>(tile + k_elem_off(r & 31, d));
  return __uint_as_float(bits << 16);
}

// Grid (pages, heads of the call): page i of head hh -- the page the last
// planned append wrote (all_pages = 0) or every page (all_pages = 1).
__global__ __launch_bounds__(kQThreads) void quest_bounds_kernel(QuestArgs a) {
  __shared__ float red[2][kQThreads];
  if (load_status(a.status) != 0) return;
  const int hh = blockIdx.y;
  const int sh = a.seq_ids[hh / a.H] * a.H + hh % a.H;
  const int L = a.st.len[sh];
  const int i = a.all_pages ? static_cast<int>(blockIdx.x) : a.desc[hh].z / a.P;
  if (i * a.P >= L) return;
  const int valid = min(a.P, L - i * a.P);
  const int pg = a.st.page_table[static_cast<size_t>(sh) * a.maxp + i];
  const char* page = a.pool + static_cast<size_t>(pg) * a.page_bytes;
  const int tid = threadIdx.x;
  const int d = tid % a.D, rg = tid / a.D, nrg = kQThreads / a.D;
  float lo = INFINITY, hi = -INFINITY;
  for (int r = rg; r < valid; r += nrg) {
    const float x = key_elem(a, page, r, d);
    lo = fminf(lo, x);
    hi = fmaxf(hi, x);
  }
  red[0][tid] = lo;
  red[1][tid] = hi;
  __syncthreads();
  if (rg == 0) {
    for (int k = 1; k < nrg; ++k) {
      lo = fminf(lo, red[0][k * a.D + d]);
      hi = fmaxf(hi, red[1][k * a.D + d]);
    }
    uint16_t* b = a.st.page_bounds + static_cast<size_t>(pg) * 2 * a.D;
    b[d] = f32_to_bf16_exact(lo);
    b[a.D + d] = f32_to_bf16_exact(hi);
  }
}

// Sortable bits of a float (larger float -> larger unsigned).
__device__ inline uint32_t orderable(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// One block per head of the call.
__global__ __launch_bounds__(kQThreads) void quest_select_kernel(QuestArgs a) {
  __shared__ float qs[kMaxGroup][128];
  __shared__ unsigned long long keys[kMaxSortPages];
  __shared__ int lds[17];
  if (load_status(a.status) != 0) return;
  const int hh = blockIdx.x;
  const int sh = a.seq_ids[hh / a.H] * a.H + hh % a.H;
  const int L = a.st.len[sh];
  const int npages = (L + a.P - 1) / a.P;
  const int tid = threadIdx.x;
  int32_t* sel = a.sel + static_cast<size_t>(hh) * a.B;
  if (npages <= a.B) {
    for (int i = tid; i < a.B; i += kQThreads) sel[i] = i < npages ? i : -1;
    if (tid == 0) a.qlen[hh] = L;
    return;
  }
  // the group's queries, as float (the borrowed neuron read as 0 in query-decision mode)
  const int h = hh % a.H;
  const uint16_t* qg = a.q + (static_cast<size_t>(hh / a.H) * a.H * a.g + h * a.g) * a.D;
  for (int e = tid; e < a.g * a.D; e += kQThreads) {
    float x = __uint_as_float(static_cast<uint32_t>(qg[e]) << 16);
    if (a.zero_neuron && e == 0) x = 0.f;
    qs[e / a.D][e % a.D] = x;
  }
  int npow = 1;
  while (npow < npages) npow <<= 1;
  for (int p = tid; p < npow; p += kQThreads) keys[p] = 0ull;
  __syncthreads();
  for (int p = tid; p < npages; p += kQThreads) {
    const int pg = a.st.page_table[static_cast<size_t>(sh) * a.maxp + p];
    const uint16_t* b = a.st.page_bounds + static_cast<size_t>(pg) * 2 * a.D;
    float best = -INFINITY;
    for (int hq = 0; hq < a.g; ++hq) {
      float u = 0.f;
      for (int d = 0; d < a.D; ++d) {
        const float lo = __uint_as_float(static_cast<uint32_t>(b[d]) << 16);
        const float hi = __uint_as_float(static_cast<uint32_t>(b[a.D + d]) << 16);
        const float x = qs[hq][d];
        u += fmaxf(x * lo, x * hi);
      }
      best = fmaxf(best, u);
    }
    // larger score first; equal scores: lower page index first
    keys[p] = (static_cast<unsigned long long>(orderable(best)) << 32) | (0xFFFFFFFFu - static_cast<uint32_t>(p));
  }
  __syncthreads();
  // bitonic sort, descending
  for (int k = 2; k <= npow; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int x = tid; x < npow; x += kQThreads) {
        const int y = x ^ j;
        if (y > x) {
          const bool desc = (x & k) == 0;
          const unsigned long long kx = keys[x], ky = keys[y];
          if (desc ? (kx < ky) : (kx > ky)) {
            keys[x] = ky;
            keys[y] = kx;
          }
        }
      }
      __syncthreads();
    }
  }
  // the B best pages, listed in ascending page order
  __shared__ int chosen[kMaxSortPages];
  for (int p = tid; p < npages; p += kQThreads) chosen[p] = 0;
  __syncthreads();
  for (int i = tid; i < a.B; i += kQThreads)
    chosen[0xFFFFFFFFu - static_cast<uint32_t>(keys[i] & 0xFFFFFFFFull)] = 1;
  __syncthreads();
  int run = 0;
  for (int p0 = 0; p0 < npages; p0 += kQThreads) {
    const int p = p0 + tid;
    const int f = p < npages ? chosen[p] : 0;
    int tot;
    const int off = block_exclusive_scan(f, lds, &tot);
    if (f) sel[run + off] = p;
    run += tot;
  }
  if (tid == 0) a.qlen[hh] = a.B * a.P - (chosen[npages - 1] ? npages * a.P - L : 0);
}

// Selection of the last decode call -> caller buffers (one thread per head).
__global__ __launch_bounds__(kQThreads) void quest_export_kernel(const int32_t* sel, int NH, int B,
                                                                 int32_t* pages, int32_t* counts) {
  const int hh = blockIdx.x * kQThreads + threadIdx.x;
  if (hh >= NH) return;
  int cnt = 0;
  for (int i = 0; i < B; ++i) {
    const int p = sel[static_cast<size_t>(hh) * B + i];
    pages[static_cast<size_t>(hh) * B + i] = p;
    cnt += p >= 0;
  }
  counts[hh] = cnt;
}

QuestArgs quest_args(const dms_config& c, const Layout& lo, void* meta, void* ws, int layer, int n) {
  QuestArgs a{};
  char* w = static_cast<char*>(ws);
  a.st = layer_state(lo, meta, layer);
  a.status = reinterpret_cast<const int32_t*>(static_cast<char*>(meta) + lo.status);
  a.desc = reinterpret_cast<const HeadDesc*>(w + lo.ws_head_desc);
  a.sel = reinterpret_cast<int32_t*>(w + lo.ws_q_sel);
  a.qlen = reinterpret_cast<int32_t*>(w + lo.ws_q_len);
  a.page_bytes = lo.page_bytes;
  a.n = n;
  a.H = c.num_kv_heads;
  a.g = c.group_size;
  a.D = c.head_dim;
  a.P = c.page_size;
  a.maxp = c.max_pages_per_head;
  a.B = c.quest_page_budget;
  a.fp8 = c.kv_format == DMS_KV_FP8;
  a.zero_neuron = c.decision_source == DMS_DECIDE_QUERY;
  return a;
}

}  // namespace

hipError_t launch_quest_bounds(const dms_config& c, const Layout& lo, void* meta, void* ws,
                               void* pool, int layer, int n, bool all_pages, const int32_t* seq_ids,
                               hipStream_t st) {
  QuestArgs a = quest_args(c, lo, meta, ws, layer, n);
  a.pool = static_cast<const char*>(pool);
  a.seq_ids = seq_ids;
  a.all_pages = all_pages;
  const dim3 grid(all_pages ? c.max_pages_per_head : 1, n * c.num_kv_heads);
  hipLaunchKernelGGL(quest_bounds_kernel, grid, dim3(kQThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_quest_export(const dms_config& c, const Layout& lo, void* ws, int n,
                               int32_t* pages, int32_t* counts, hipStream_t st) {
  const int NH = n * c.num_kv_heads;
  const int32_t* sel = reinterpret_cast<const int32_t*>(static_cast<char*>(ws) + lo.ws_q_sel);
  hipLaunchKernelGGL(quest_export_kernel, dim3((NH + kQThreads - 1) / kQThreads), dim3(kQThreads), 0,
                     st, sel, NH, c.quest_page_budget, pages, counts);
  return hipGetLastError();
}

hipError_t launch_quest_select(const dms_config& c, const Layout& lo, void* meta, void* ws,
                               int layer, int n, const int32_t* seq_ids, const void* q,
                               hipStream_t st) {
  QuestArgs a = quest_args(c, lo, meta, ws, layer, n);
  a.seq_ids = seq_ids;
  a.q = static_cast<const uint16_t*>(q);
  hipLaunchKernelGGL(quest_select_kernel, dim3(n * c.num_kv_heads), dim3(kQThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace dms
