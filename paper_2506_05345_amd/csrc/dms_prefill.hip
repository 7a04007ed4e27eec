// DMS-masked chunked prefill attention, gfx950.
//
// Query at position t of a chunk [p0, p0 + C) attends to key j iff j <= t and
// (j > t - w or key j is kept) -- the binary mask of Fig. 1b (Sec. 3.1), passed
// as the per-token decision vector and never materialised (Sec. 3.1
// "Performance Considerations"); the sparsity it creates is used to skip work
// (Sec. 3.2).  Keys come from three places:
//   1. the cache: the L0 live slots of the head before the chunk; all of them
//      are visible except flagged tokens of the last w positions, which expire
//      inside the chunk by the same rule (slot_meta holds owner position and
//      flag);
//   2. kept chunk keys older than the query block's window band -- visible to
//      every query of the block -- gathered from a compacted list built by
//      prefill_list_kernel (flagged keys there are skipped entirely);
//   3. the band [max(p0, t0 - w + 1), t1) of chunk keys, masked per element.
//
// A workgroup (4 waves) owns one (sequence, KV head, block of query
// positions).  Its columns are (position, query head) pairs packed 16 to an
// MFMA column block (16 / g positions x g heads); each wave holds NQ column
// blocks.  Key tiles of 32 are staged into LDS in the pool's tile layout
// (keys [d/32][32][32], values transposed [d][32]), double buffered, and read
// by every wave with 16-byte LDS loads straight into MFMA operand registers;
// scores, masking and the online softmax follow the decode kernel.
#include "dms_common.h"

namespace dms {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

constexpr int kThreads = 256;
constexpr uint32_t kNoKey = 0x7FFFFFFFu;  // key position of padding rows (never visible)
constexpr float kRescale = 8.0f;

__device__ inline int load_status(const int32_t* status) {
  return __atomic_load_n(status, __ATOMIC_RELAXED);
}

__device__ inline f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

struct PrefillArgs {
  const int32_t* status;
  int32_t* status_w;
  const int32_t* seq_ids;
  const int32_t* cu;
  const uint16_t* q;      // [T, Hq, D]
  const uint16_t* k;      // [T, H, D]
  const uint16_t* v;      // [T, H, D]
  const uint8_t* flags;   // [T, H]
  const char* pool;
  const int32_t* page_table;
  const int32_t* slot_meta;
  const int32_t* len;
  const int32_t* pos;
  int32_t* list;          // [H][total]: chunk-local indices of kept tokens
  int32_t* list_cnt;      // [n * H]
  float* out;             // [T, Hq, D]
  size_t page_bytes;
  int n, H, g, w, P, log2P, maxp, max_slots, max_seqs, total, max_len, PB;
  float scale_log2;
};

// Pass 0 (one block per (sequence, head)): validate the chunk boundaries and
// list the kept tokens of the chunk in position order.
__global__ __launch_bounds__(kThreads) void prefill_list_kernel(PrefillArgs a) {
  __shared__ int lds[17];
  if (load_status(a.status) != 0) return;
  const int hh = blockIdx.x;
  const int i = hh / a.H, h = hh % a.H;
  const int s = a.seq_ids[i];
  const int tok0 = a.cu[i], C = a.cu[i + 1] - a.cu[i];
  const bool bad = (s < 0 || s >= a.max_seqs || C < 0 || C > a.max_len || a.cu[0] != 0 ||
                    a.cu[a.n] != a.total || tok0 < 0 || tok0 + C > a.total);
  if (bad) {
    if (threadIdx.x == 0) atomicCAS(reinterpret_cast<int*>(a.status_w), 0, DMS_ERR_INVALID);
    return;
  }
  int run = 0;
  for (int c0 = 0; c0 < C; c0 += blockDim.x) {
    const int c = c0 + threadIdx.x;
    const int kept = (c < C) && a.flags[static_cast<size_t>(tok0 + c) * a.H + h] == 0;
    int tot;
    const int off = block_exclusive_scan(kept, lds, &tot);
    if (kept) a.list[static_cast<size_t>(h) * a.total + tok0 + run + off] = c;
    run += tot;
  }
  if (threadIdx.x == 0) a.list_cnt[hh] = run;
}

template <int D>
struct Frag {
  u32x4 ka[D / 32];
  u32x4 kb[D / 32];
  u32x4 vt[D / 16];
};

// Staging of one 32-key tile: each thread moves 16-byte pieces; pool tiles
// are copied as they are, chunk keys are transposed on the way in.
template <int D>
struct Stage {
  static constexpr int kPieces = (D * 128) / 16 / kThreads;  // 16-byte pieces per thread
  u32x4 kx[kPieces / 2];   // key pieces (chunk source) or first half (pool source)
  u32x4 vx[kPieces / 2];   // value pieces
  uint32_t meta;           // this thread's key row (threads 0..31): position | flag << 31
};

template <int D, int NQ>
__global__ __launch_bounds__(kThreads, 2) void prefill_kernel(PrefillArgs a) {
  __shared__ __attribute__((aligned(16))) char tile_lds[2][D * 128];
  __shared__ uint32_t meta_lds[2][32];
  if (load_status(a.status) != 0) return;
  const int hh = blockIdx.y;
  const int i = hh / a.H, h = hh % a.H;
  const int tok0 = a.cu[i], C = a.cu[i + 1] - a.cu[i];
  const int pb0 = blockIdx.x * a.PB;
  if (pb0 >= C) return;
  const int s = a.seq_ids[i];
  const int sh = s * a.H + h;
  const int p0 = a.pos[s];
  const int L0 = a.len[sh];
  const int t0 = p0 + pb0;
  const int t1 = p0 + min(C, pb0 + a.PB);
  const int band_lo = max(p0, t0 - a.w + 1);
  // kept chunk keys strictly before the band: prefix of the sorted list
  const int32_t* lst = a.list + static_cast<size_t>(h) * a.total + tok0;
  int lo_i = 0, hi_i = a.list_cnt[hh];
  while (lo_i < hi_i) {
    const int mid = (lo_i + hi_i) >> 1;
    if (lst[mid] < band_lo - p0) lo_i = mid + 1; else hi_i = mid;
  }
  const int n_pre = lo_i;
  const int nc = (L0 + 31) >> 5;
  const int np = (n_pre + 31) >> 5;
  const int nb = (t1 - band_lo + 31) >> 5;
  const int ntiles = nc + np + nb;
  const int32_t* pt = a.page_table + static_cast<size_t>(sh) * a.maxp;
  const int32_t* smeta = a.slot_meta + static_cast<size_t>(sh) * a.max_slots;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, G = lane >> 4;
  const int Hq = a.H * a.g;
  const int pcb = 16 / a.g;  // positions per column block

  // ---- columns of this lane: (position, query head) in each column block
  int tcol[NQ];
  u32x4 qf[NQ][D / 32];
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
    const int cb = wave * NQ + qb;
    const int pl = r / a.g, qh = r % a.g;
    const int t = t0 + cb * pcb + pl;
    const bool ok = (pl < pcb) && (t < t1);
    tcol[qb] = ok ? t : -1;
    const u32x4 z = {0u, 0u, 0u, 0u};
    const char* qrow = reinterpret_cast<const char*>(
        a.q + (static_cast<size_t>(tok0 + (t - p0)) * Hq + h * a.g + qh) * D);
#pragma unroll
    for (int s2 = 0; s2 < D / 32; ++s2)
      qf[qb][s2] = ok ? *reinterpret_cast<const u32x4*>(qrow + (32 * s2 + 8 * G) * 2) : z;
  }

  // ---- staging: global -> registers (A), registers -> LDS (B)
  Stage<D> stg;
  constexpr int KP = Stage<D>::kPieces / 2;
  auto stage_load = [&](int k) {
    if (k < nc) {
      const int sb = k * 32;
      const char* tile = a.pool + static_cast<size_t>(pt[sb >> a.log2P]) * a.page_bytes +
                         static_cast<size_t>((sb & (a.P - 1)) >> 5) * (D * 128);
#pragma unroll
      for (int m = 0; m < KP; ++m) {
        stg.kx[m] = *reinterpret_cast<const u32x4*>(tile + (tid + m * kThreads) * 16);
        stg.vx[m] = *reinterpret_cast<const u32x4*>(tile + D * 64 + (tid + m * kThreads) * 16);
      }
      if (tid < 32) {
        stg.meta = sb + tid < L0 ? static_cast<uint32_t>(smeta[sb + tid]) : kNoKey;
      }
    } else {
      // chunk keys: row j of the tile, 16-byte piece e8 of the row
      const bool pre = k < nc + np;
      const int base = pre ? (k - nc) * 32 : band_lo - p0 + (k - nc - np) * 32;
      const int lim = pre ? n_pre : t1 - p0;   // exclusive bound (list index / chunk index)
#pragma unroll
      for (int m = 0; m < KP; ++m) {
        const int pc = tid + m * kThreads;
        const int j = pc / (D / 8), e8 = pc % (D / 8);
        const int idx = base + j;
        const u32x4 z = {0u, 0u, 0u, 0u};
        if (idx < lim) {
          const int c = pre ? lst[idx] : idx;
          const size_t row = (static_cast<size_t>(tok0 + c) * a.H + h) * D + 8 * e8;
          stg.kx[m] = *reinterpret_cast<const u32x4*>(a.k + row);
          stg.vx[m] = *reinterpret_cast<const u32x4*>(a.v + row);
        } else {
          stg.kx[m] = z;
          stg.vx[m] = z;
        }
      }
      if (tid < 32) {
        const int idx = base + tid;
        if (idx < lim) {
          const int c = pre ? lst[idx] : idx;
          const uint32_t f = pre ? 0u : (a.flags[static_cast<size_t>(tok0 + c) * a.H + h] ? kFlagBit : 0u);
          stg.meta = static_cast<uint32_t>(p0 + c) | f;
        } else {
          stg.meta = kNoKey;
        }
      }
    }
  };
  auto stage_store = [&](int k, int buf) {
    char* dst = tile_lds[buf];
    if (k < nc) {
      const int valid = min(32, L0 - k * 32);
#pragma unroll
      for (int m = 0; m < KP; ++m) {
        const int off = (tid + m * kThreads) * 16;
        *reinterpret_cast<u32x4*>(dst + off) = stg.kx[m];
        u32x4 x = stg.vx[m];
        // value elements of rows >= valid are zeroed (pool slots past L hold
        // stale data); element i of the piece is row (off % 64) / 2 + i
        const int j0 = (off & 63) >> 1;
        if (j0 + 8 > valid) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (j0 + e >= valid) x[e >> 1] &= (e & 1) ? 0x0000FFFFu : 0xFFFF0000u;
        }
        *reinterpret_cast<u32x4*>(dst + D * 64 + off) = x;
      }
    } else {
#pragma unroll
      for (int m = 0; m < KP; ++m) {
        const int pc = tid + m * kThreads;
        const int j = pc / (D / 8), e8 = pc % (D / 8);
        const int e0 = 8 * e8;
        *reinterpret_cast<u32x4*>(dst + (e0 >> 5) * 2048 + j * 64 + (e0 & 31) * 2) = stg.kx[m];
        const u32x4 x = stg.vx[m];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint16_t val = static_cast<uint16_t>((e & 1) ? (x[e >> 1] >> 16) : (x[e >> 1] & 0xFFFFu));
          *reinterpret_cast<uint16_t*>(dst + D * 64 + (e0 + e) * 64 + j * 2) = val;
        }
      }
    }
    if (tid < 32) meta_lds[buf][tid] = stg.meta;
  };

  // ---- accumulators
  f32x4 o[NQ][D / 16];
  float m_ref[NQ], l_run[NQ];
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
#pragma unroll
    for (int b = 0; b < D / 16; ++b) o[qb][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_ref[qb] = -INFINITY;
    l_run[qb] = 0.f;
  }
  const uint32_t lo_k = static_cast<uint32_t>((8 * (r >> 2) + (r & 3)) * 64 + 16 * G);
  const uint32_t lo_v = static_cast<uint32_t>(D * 64 + r * 64 + 16 * G);

  if (ntiles > 0) {
    stage_load(0);
    stage_store(0, 0);
  }
  __syncthreads();
  for (int k = 0; k < ntiles; ++k) {
    const int buf = k & 1;
    if (k + 1 < ntiles) stage_load(k + 1);
    // operands of this tile from LDS
    const char* tl = tile_lds[buf];
    Frag<D> f;
#pragma unroll
    for (int s2 = 0; s2 < D / 32; ++s2) {
      f.ka[s2] = *reinterpret_cast<const u32x4*>(tl + lo_k + s2 * 2048);
      f.kb[s2] = *reinterpret_cast<const u32x4*>(tl + lo_k + 256 + s2 * 2048);
    }
#pragma unroll
    for (int b = 0; b < D / 16; ++b) f.vt[b] = *reinterpret_cast<const u32x4*>(tl + lo_v + b * 1024);
    uint32_t km[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) km[j] = meta_lds[buf][8 * G + j];
#pragma unroll
    for (int qb = 0; qb < NQ; ++qb) {
      f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s2 = 0; s2 < D / 32; ++s2) {
        s0 = mfma_bf16(f.ka[s2], qf[qb][s2], s0);
        s1 = mfma_bf16(f.kb[s2], qf[qb][s2], s1);
      }
      const int t = tcol[qb];
      float sc[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float raw = j < 4 ? s0[j] : s1[j - 4];
        const int kp = static_cast<int>(km[j] & ~kFlagBit);
        const bool kflag = (km[j] & kFlagBit) != 0;
        const bool vis = (t >= 0) && (km[j] != kNoKey) && kp <= t && (kp > t - a.w || !kflag);
        sc[j] = vis ? raw * a.scale_log2 : -INFINITY;
      }
      float mx = fmaxf(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3])),
                       fmaxf(fmaxf(sc[4], sc[5]), fmaxf(sc[6], sc[7])));
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const bool raise = mx > m_ref[qb] + kRescale;   // false while mx is -inf
      if (__builtin_amdgcn_ballot_w64(raise)) {
        const float m_new = raise ? mx : m_ref[qb];
        const float alpha = m_ref[qb] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_ref[qb] - m_new);
        l_run[qb] *= alpha;
#pragma unroll
        for (int b = 0; b < D / 16; ++b) o[qb][b] *= alpha;
        m_ref[qb] = m_new;
      }
      bf16x8 p;
      float psum = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float e = sc[j] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sc[j] - m_ref[qb]);
        const __bf16 pb = static_cast<__bf16>(e);
        p[j] = pb;
        psum += static_cast<float>(pb);
      }
      l_run[qb] += psum;
      const u32x4 pu = __builtin_bit_cast(u32x4, p);
#pragma unroll
      for (int b = 0; b < D / 16; ++b) o[qb][b] = mfma_bf16(f.vt[b], pu, o[qb][b]);
    }
    if (k + 1 < ntiles) stage_store(k + 1, buf ^ 1);
    __syncthreads();
  }

  // ---- outputs
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
    float l = l_run[qb];
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    const int t = tcol[qb];
    if (t >= 0) {
      const int qh = r % a.g;
      const float inv = 1.0f / l;
      float* dst = a.out + (static_cast<size_t>(tok0 + (t - p0)) * Hq + h * a.g + qh) * D + 4 * G;
#pragma unroll
      for (int b = 0; b < D / 16; ++b) *reinterpret_cast<f32x4*>(dst + 16 * b) = o[qb][b] * inv;
    }
  }
}

constexpr int kNQ = 2;

template <int D>
hipError_t launch_prefill_d(const dms_config& c, const Layout& lo, void* meta, void* ws, void* pool,
                            int layer, int n, const int32_t* seq_ids, const int32_t* cu,
                            int total_tokens, int max_len, const void* q, const void* k,
                            const void* v, const uint8_t* flags, float* out, hipStream_t st,
                            hipEvent_t ev_start, hipEvent_t ev_stop) {
  char* w = static_cast<char*>(ws);
  LayerState ls = layer_state(lo, meta, layer);
  PrefillArgs a;
  a.status = reinterpret_cast<const int32_t*>(static_cast<char*>(meta) + lo.status);
  a.status_w = reinterpret_cast<int32_t*>(static_cast<char*>(meta) + lo.status);
  a.seq_ids = seq_ids;
  a.cu = cu;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.flags = flags;
  a.pool = static_cast<const char*>(pool);
  a.page_table = ls.page_table;
  a.slot_meta = ls.slot_meta;
  a.len = ls.len;
  a.pos = ls.pos;
  a.list = reinterpret_cast<int32_t*>(w + lo.ws_pf_meta);
  a.list_cnt = reinterpret_cast<int32_t*>(w + lo.ws_pf_cum);
  a.out = out;
  a.page_bytes = lo.page_bytes;
  a.n = n;
  a.H = c.num_kv_heads;
  a.g = c.group_size;
  a.w = c.window;
  a.P = c.page_size;
  a.log2P = __builtin_ctz(static_cast<unsigned>(c.page_size));
  a.maxp = c.max_pages_per_head;
  a.max_slots = lo.max_slots;
  a.max_seqs = c.max_seqs;
  a.total = total_tokens;
  a.max_len = max_len;
  a.PB = 4 * kNQ * (16 / c.group_size);
  a.scale_log2 = c.softmax_scale * 1.4426950408889634f;
  const int NH = n * c.num_kv_heads;
  hipLaunchKernelGGL(prefill_list_kernel, dim3(NH), dim3(kThreads), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 grid((max_len + a.PB - 1) / a.PB, NH);
  if (ev_start) (void)hipEventRecord(ev_start, st);
  hipLaunchKernelGGL((prefill_kernel<D, kNQ>), grid, dim3(kThreads), 0, st, a);
  e = hipGetLastError();
  if (ev_stop) (void)hipEventRecord(ev_stop, st);
  return e;
}

}  // namespace

hipError_t launch_prefill_attention(const dms_config& c, const Layout& lo, void* meta, void* ws,
                                    void* pool, int layer, int n, const int32_t* seq_ids,
                                    const int32_t* cu, int total_tokens, int max_len,
                                    const void* q, const void* k, const void* v,
                                    const uint8_t* flags, float* out, hipStream_t st,
                                    hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (c.head_dim == 128)
    return launch_prefill_d<128>(c, lo, meta, ws, pool, layer, n, seq_ids, cu, total_tokens,
                                 max_len, q, k, v, flags, out, st, ev_start, ev_stop);
  return launch_prefill_d<64>(c, lo, meta, ws, pool, layer, n, seq_ids, cu, total_tokens, max_len,
                              q, k, v, flags, out, st, ev_start, ev_stop);
}

}  // namespace dms
