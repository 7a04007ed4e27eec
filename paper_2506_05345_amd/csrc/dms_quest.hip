// Page retrieval within the DMS retained set (Quest on top of DMS), gfx950.
//
// The paper notes that DMS compresses the KV cache while Quest retrieves
// cache items, so the two can be combined (App. A).  Quest bounds the score
// any key of a page can reach by U = sum_i max(q_i lo_i, q_i hi_i), lo / hi
// the channel-wise min / max of the page's keys, and attends only the pages
// with the largest bounds.  Here the unit is the cache's own page (P slots of
// one KV head holding retained tokens of any positions):
//   * quest_append_kernel writes an appended token's K / V into its slot and
//     recomputes lo / hi exactly over that page's live slots (DMS reuses
//     evicted tokens' slots, so bounds can shrink as well as grow);
//     quest_bounds_kernel does the same for every page after a chunk commit;
//   * quest_select_kernel scores every page of a head for its query group
//     (maximum of U over the group's heads, one wave per page, float32 sums
//     in a fixed order),
//     keeps the B best (ties to the lower page index) in ascending order and
//     the number of live slots they hold, which the decode planner then
//     splits into tiles like any retained length.
#include "dms_common.h"
#include "dms_fp8.h"

namespace dms {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

constexpr int kQThreads = 256;
constexpr int kMaxSortPages = 4096;   // max_pages_per_head limit with a budget
// the select kernel's sort keys and page marks at that limit fit the LDS a
// launch may request
static_assert(kMaxSortPages * (8 + 4) <= 65536, "select LDS");

struct QuestArgs {
  LayerState st;
  const int32_t* status;
  const HeadDesc* desc;     // after an append: the slot each head wrote (z)
  const int32_t* seq_ids;
  const char* pool;
  const uint16_t* q;        // [n, Hq, D] bf16
  const uint16_t* k;        // [n, Hkv, D] bf16: appended keys (quest_append_kernel)
  const uint16_t* v;        // [n, Hkv, D] bf16: appended values
  int32_t* sel;             // [NH][B] attended page-table indices, ascending
  int32_t* qpage;           // [NH][B] their physical pages (what decode reads)
  int32_t* qlen;            // [NH] live slots in the attended pages
  size_t page_bytes;
  int n, H, g, D, P, maxp, B, fp8, zero_neuron, all_pages;
  int sort_pages;           // power of two >= maxp: sort keys in the select kernel's LDS
};

__device__ inline int load_status(const int32_t* status) {
  return __atomic_load_n(status, __ATOMIC_RELAXED);
}

__device__ inline uint16_t f32_to_bf16_exact(float x) {
  // x is a bf16 value (a stored key, or an E4M3 code times a power of two)
  return static_cast<uint16_t>(__float_as_uint(x) >> 16);
}

// Keys of row r, dims e .. e + 7 (e a multiple of 8), as stored.
__device__ inline void key_elems8(const QuestArgs& a, const char* page, int r, int e, float* x) {
  const int j = r & 31;
  if (a.fp8) {
    const char* tile = page + static_cast<size_t>(r >> 5) * fp8_tile_bytes(a.D);
    const uint2 c = *reinterpret_cast<const uint2*>(tile + fp8_k_off(j, e));   // 8 contiguous codes
    const float scale = *reinterpret_cast<const float*>(tile + fp8_ks_off(j, a.D));
    const uint32_t w[2] = {c.x, c.y};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const auto lo = __builtin_amdgcn_cvt_pk_f32_fp8(w[h], false);
      const auto hi = __builtin_amdgcn_cvt_pk_f32_fp8(w[h], true);
      x[4 * h] = lo[0] * scale;       // exact: a code times a power of two
      x[4 * h + 1] = lo[1] * scale;
      x[4 * h + 2] = hi[0] * scale;
      x[4 * h + 3] = hi[1] * scale;
    }
    return;
  }
  const char* tile = page + static_cast<size_t>(r >> 5) * tile_bytes(a.D);
  const uint4 v = *reinterpret_cast<const uint4*>(tile + k_elem_off(j, e));   // 8 contiguous bf16
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}

// lo / hi of page `pg` over its first `valid` rows, written to the page's
// bounds.  Thread t covers dims 8 (t % (D/8)) .. + 7 of rows t / (D/8),
// + rows_per_pass, ...
__device__ void page_bounds(const QuestArgs& a, int pg, int valid) {
  __shared__ float red[2][kQThreads][8];
  const char* page = a.pool + static_cast<size_t>(pg) * a.page_bytes;
  const int tid = threadIdx.x;
  const int per_row = a.D / 8, rows = kQThreads / per_row;
  const int e = 8 * (tid % per_row), r0 = tid / per_row;
  float lo[8], hi[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    lo[k] = INFINITY;
    hi[k] = -INFINITY;
  }
  for (int r = r0; r < valid; r += rows) {
    float x[8];
    key_elems8(a, page, r, e, x);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      lo[k] = fminf(lo[k], x[k]);
      hi[k] = fmaxf(hi[k], x[k]);
    }
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    red[0][tid][k] = lo[k];
    red[1][tid][k] = hi[k];
  }
  __syncthreads();
  if (r0 == 0) {
    for (int g2 = 1; g2 < rows; ++g2) {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        lo[k] = fminf(lo[k], red[0][g2 * per_row + tid][k]);
        hi[k] = fmaxf(hi[k], red[1][g2 * per_row + tid][k]);
      }
    }
    uint16_t* b = a.st.page_bounds + static_cast<size_t>(pg) * 2 * a.D;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      b[e + k] = f32_to_bf16_exact(lo[k]);
      b[a.D + e + k] = f32_to_bf16_exact(hi[k]);
    }
  }
}

// Grid (pages, heads of the call): every page of head hh (after a chunk
// commit), or the page the last planned append wrote (all_pages = 0).
__global__ __launch_bounds__(kQThreads) void quest_bounds_kernel(QuestArgs a) {
  if (load_status(a.status) != 0) return;
  const int hh = blockIdx.y;
  const int sh = a.seq_ids[hh / a.H] * a.H + hh % a.H;
  const int L = a.st.len[sh];
  const int i = a.all_pages ? static_cast<int>(blockIdx.x) : a.desc[hh].z / a.P;
  if (i * a.P >= L) return;
  page_bounds(a, a.st.page_table[static_cast<size_t>(sh) * a.maxp + i], min(a.P, L - i * a.P));
}

// One block per head of the call, after the append's plan: the token's K / V
// into its slot (wave 0), then the bounds of that page over its live slots,
// the new row read back after the barrier (its stores are complete and
// visible to the block's other waves there).
//
// Selection operands of one lane: its query column (head r) split into the
// negative and positive parts, and the bounds of the page it scores first
// (page 16 wave + r), loaded before the append when that page is not the
// one the append rewrites.
struct SelectOps {
  u32x4 qneg[4], qpos[4];
  u32x4 lo[4], hi[4];
  bool have_bounds;
};
__device__ void select_ops(const QuestArgs& a, int hh, int sh, int L, int skip_page, SelectOps& op);
__device__ void select_head(const QuestArgs& a, int hh, int sh, int L, unsigned long long* keys, int* chosen,
                            SelectOps& op);

__device__ inline void append_head(const QuestArgs& a, int hh, const HeadDesc& d) {
  const int i = d.z / a.P, row = d.z % a.P;
  const int pg = a.st.page_table[static_cast<size_t>(d.y) * a.maxp + i];
  if (threadIdx.x < 64) {
    char* tile = const_cast<char*>(a.pool) + static_cast<size_t>(pg) * a.page_bytes +
                 (row >> 5) * (a.fp8 ? fp8_tile_bytes(a.D) : tile_bytes(a.D));
    store_token_kv(tile, row & 31, a.D, threadIdx.x, a.fp8, a.k + static_cast<size_t>(hh) * a.D,
                   a.v + static_cast<size_t>(hh) * a.D);
  }
  __syncthreads();
  page_bounds(a, pg, min(a.P, d.x - i * a.P));
}

__global__ __launch_bounds__(kQThreads) void quest_append_kernel(QuestArgs a) {
  if (load_status(a.status) != 0) return;
  const int hh = blockIdx.x;
  append_head(a, hh, a.desc[hh]);   // desc: (L after the append, state index, slot)
}

// A decode step's append and page selection for one head per block: the
// selection reads every page's bounds, the written page's from this block's
// own stores (visible after the barrier).
__global__ __launch_bounds__(kQThreads) void quest_append_select_kernel(QuestArgs a) {
  extern __shared__ unsigned long long q_dyn[];
  if (load_status(a.status) != 0) return;
  const int hh = blockIdx.x;
  const HeadDesc d = a.desc[hh];
  // the query and every first-round page bound but the appended page's are
  // read before the append, so their loads overlap it
  SelectOps op;
  select_ops(a, hh, d.y, d.x, d.z / a.P, op);
  append_head(a, hh, d);
  __syncthreads();
  select_head(a, hh, d.y, d.x, q_dyn, reinterpret_cast<int*>(q_dyn + a.sort_pages), op);
}

// Sortable bits of a float (larger float -> larger unsigned).
__device__ inline uint32_t orderable(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Scores as one small matrix product: for q_i >= 0 the larger of q_i lo_i,
// q_i hi_i is q_i hi_i, else q_i lo_i, so U = [lo | hi] . [q-; q+] with
// q- = min(q, 0), q+ = max(q, 0) (exact in bf16; the products are exact in
// fp32).  MFMA rows are 16 pages, columns the group's heads, k the 2 D
// entries of a page's bounds (lo then hi).  The borrowed neuron is read as 0
// in query-decision mode.  A operand: lane (page p, G) holds bound entries
// 32 kb + 8 G .. + 7.
__device__ inline void page_bound_ops(const QuestArgs& a, int sh, int p, int npages, u32x4 (&lo)[4], u32x4 (&hi)[4]) {
  const int G = (threadIdx.x & 63) >> 4;
  const uint16_t* b = p < npages
      ? a.st.page_bounds + static_cast<size_t>(a.st.page_table[static_cast<size_t>(sh) * a.maxp + p]) * 2 * a.D
      : nullptr;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    lo[kb] = (b && kb < a.D / 32) ? *reinterpret_cast<const u32x4*>(b + 32 * kb + 8 * G) : u32x4{0u, 0u, 0u, 0u};
    hi[kb] = (b && kb < a.D / 32) ? *reinterpret_cast<const u32x4*>(b + a.D + 32 * kb + 8 * G)
                                  : u32x4{0u, 0u, 0u, 0u};
  }
}

// This lane's query column (head r: dims 32 kb + 8 G .. + 7) and, unless it
// is skip_page, the bounds of its first page.
__device__ void select_ops(const QuestArgs& a, int hh, int sh, int L, int skip_page, SelectOps& op) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, G = lane >> 4;
  const int h = hh % a.H;
  const uint16_t* qg = a.q + (static_cast<size_t>(hh / a.H) * a.H * a.g + h * a.g) * a.D;
  const int npages = (L + a.P - 1) / a.P;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    u32x4 x = {0u, 0u, 0u, 0u};
    if (npages > a.B && r < a.g && kb < a.D / 32) x = *reinterpret_cast<const u32x4*>(qg + r * a.D + 32 * kb + 8 * G);
    if (a.zero_neuron && r == 0 && G == 0 && kb == 0) x[0] &= 0xFFFF0000u;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      // per bf16 half: negative (sign set) -> q-, else q+
      const uint32_t neg = ((x[w] >> 15) & 1u) * 0x0000FFFFu | ((x[w] >> 31) & 1u) * 0xFFFF0000u;
      op.qneg[kb][w] = x[w] & neg;
      op.qpos[kb][w] = x[w] & ~neg;
    }
  }
  const int p = 16 * wave + r;
  op.have_bounds = npages > a.B && p != skip_page;
  if (op.have_bounds) page_bound_ops(a, sh, p, npages, op.lo, op.hi);
}

// Selection of call head hh by one block: keys (sort_pages of them) and
// page marks (maxp) in the caller's LDS; op from select_ops.
__device__ void select_head(const QuestArgs& a, int hh, int sh, int L, unsigned long long* keys, int* chosen,
                            SelectOps& op) {
  __shared__ int lds[17];
  const int npages = (L + a.P - 1) / a.P;
  const int tid = threadIdx.x;
  int32_t* sel = a.sel + static_cast<size_t>(hh) * a.B;
  int32_t* qpage = a.qpage + static_cast<size_t>(hh) * a.B;
  const int32_t* pt = a.st.page_table + static_cast<size_t>(sh) * a.maxp;
  if (npages <= a.B) {
    for (int i = tid; i < a.B; i += kQThreads) {
      sel[i] = i < npages ? i : -1;
      qpage[i] = i < npages ? pt[i] : -1;
    }
    if (tid == 0) a.qlen[hh] = L;
    return;
  }
  const int lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, G = lane >> 4;
  const int kbs = a.D / 32;                  // k-blocks per half (lo or hi)
  int npow = 1;
  while (npow < npages) npow <<= 1;
  for (int p = tid; p < npow; p += kQThreads) keys[p] = 0ull;
  __syncthreads();
  for (int pb = 16 * wave; pb < npages; pb += kQThreads / 4) {
    const int p = pb + r;
    // the first round's bounds came with the operands unless this lane's
    // page is the one the append rewrote
    if (pb != 16 * wave || !op.have_bounds) page_bound_ops(a, sh, p, npages, op.lo, op.hi);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      if (kb < kbs) {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, op.lo[kb]),
                                                      __builtin_bit_cast(bf16x8, op.qneg[kb]), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, op.hi[kb]),
                                                      __builtin_bit_cast(bf16x8, op.qpos[kb]), acc, 0, 0, 0);
      }
    }
    // lane (head r, G) holds pages pb + 4 G + i; maximum over the group's heads
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float u = r < a.g ? acc[i] : -INFINITY;
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) u = fmaxf(u, __shfl_xor(u, off, 16));
      const int pp = pb + 4 * G + i;
      // larger score first; equal scores: lower page index first
      if (r == 0 && pp < npages)
        keys[pp] = (static_cast<unsigned long long>(orderable(u)) << 32) |
                   (0xFFFFFFFFu - static_cast<uint32_t>(pp));
    }
  }
  __syncthreads();
  if (npages <= kQThreads) {
    // rank of each page among all of them (keys are distinct)
    if (tid < npages) {
      const unsigned long long k0 = keys[tid];
      int rank = 0;
      for (int p = 0; p < npages; ++p) rank += keys[p] > k0;
      chosen[tid] = rank < a.B;
    }
    __syncthreads();
  } else {
  // bitonic sort, descending, then the B best marked
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
  for (int p = tid; p < npages; p += kQThreads) chosen[p] = 0;
  __syncthreads();
  for (int i = tid; i < a.B; i += kQThreads)
    chosen[0xFFFFFFFFu - static_cast<uint32_t>(keys[i] & 0xFFFFFFFFull)] = 1;
  __syncthreads();
  }
  // the B best pages, listed in ascending page order
  int run = 0;
  for (int p0 = 0; p0 < npages; p0 += kQThreads) {
    const int p = p0 + tid;
    const int f = p < npages ? chosen[p] : 0;
    int tot;
    const int off = block_exclusive_scan(f, lds, &tot);
    if (f) {
      sel[run + off] = p;
      qpage[run + off] = pt[p];
    }
    run += tot;
  }
  if (tid == 0) a.qlen[hh] = a.B * a.P - (chosen[npages - 1] ? npages * a.P - L : 0);
}

// One block per head of the call.
__global__ __launch_bounds__(kQThreads) void quest_select_kernel(QuestArgs a) {
  // sort keys then page marks, sized at launch so that small page tables
  // leave room for many blocks per CU
  extern __shared__ unsigned long long q_dyn[];
  if (load_status(a.status) != 0) return;
  const int hh = blockIdx.x;
  const int sh = a.seq_ids[hh / a.H] * a.H + hh % a.H;
  SelectOps op;
  select_ops(a, hh, sh, a.st.len[sh], -1, op);
  select_head(a, hh, sh, a.st.len[sh], q_dyn, reinterpret_cast<int*>(q_dyn + a.sort_pages), op);
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
  a.qpage = reinterpret_cast<int32_t*>(w + lo.ws_q_page);
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
  a.sort_pages = 1;
  while (a.sort_pages < c.max_pages_per_head) a.sort_pages <<= 1;
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

hipError_t launch_quest_append(const dms_config& c, const Layout& lo, void* meta, void* ws,
                               void* pool, int layer, int n, const void* k, const void* v, hipStream_t st) {
  QuestArgs a = quest_args(c, lo, meta, ws, layer, n);
  a.pool = static_cast<const char*>(pool);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  hipLaunchKernelGGL(quest_append_kernel, dim3(n * c.num_kv_heads), dim3(kQThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_quest_append_select(const dms_config& c, const Layout& lo, void* meta, void* ws,
                                      void* pool, int layer, int n, const void* q, const void* k,
                                      const void* v, hipStream_t st) {
  QuestArgs a = quest_args(c, lo, meta, ws, layer, n);
  a.pool = static_cast<const char*>(pool);
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  const size_t lds = static_cast<size_t>(a.sort_pages) * 8 + static_cast<size_t>(c.max_pages_per_head) * 4;
  hipLaunchKernelGGL(quest_append_select_kernel, dim3(n * c.num_kv_heads), dim3(kQThreads), lds, st, a);
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
  const size_t lds = static_cast<size_t>(a.sort_pages) * 8 + static_cast<size_t>(c.max_pages_per_head) * 4;
  hipLaunchKernelGGL(quest_select_kernel, dim3(n * c.num_kv_heads), dim3(kQThreads), lds, st, a);
  return hipGetLastError();
}

}  // namespace dms
