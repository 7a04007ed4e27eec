// DMS-masked chunked prefill attention, gfx950.
//
// Query at position t of a chunk [p0, p0 + C) attends to key j iff j <= t and
// (j > t - w or key j is kept) -- the binary mask of Fig. 1b (Sec. 3.1), passed
// as the per-token decision vector and never materialised (Sec. 3.1
// "Performance Considerations"); the sparsity it creates is used to skip work
// (Sec. 3.2).  For a block of queries [t0, t1) keys come from three places:
//   1. the cache: the L0 live slots of the head before the chunk; all of them
//      are visible except flagged tokens of the last w positions, which expire
//      inside the chunk by the same rule (slot_meta holds owner position and
//      flag);
//   2. kept chunk keys before the band -- visible to every query of the
//      block; flagged ones there are hidden from all of them and skipped;
//   3. the band: the chunk tiles from the one holding max(p0, t0 - w + 1) to
//      t1, masked per element.
//
// Pass 0 lists the kept chunk tokens; pass 1 copies the chunk's keys and
// values, in chunk order and in kept order, into workspace tiles in the
// pool's tile layout (16-byte pieces in the decode MFMAs' fragment order:
// keys by (k-step, half, lane), values transposed), so the attention pass
// stages every source the same way.
//
// Attention pass: a workgroup (4 waves) owns one (sequence, KV head, block of
// query positions).  Its columns are (position, query head) pairs, the g
// heads of a position consecutive, packed 16 to an MFMA column block (a
// position's heads may straddle two blocks); each wave holds NQ column
// blocks.  Key tiles of 32 are staged into LDS in the order the MFMA
// operand loads consume them (no bank conflicts) -- by hardware copies into
// four buffers for bf16 pages under delayed eviction, through registers into
// two otherwise -- and read by every wave with 16-byte LDS loads straight
// into operand registers.  A tile is masked per element only when some query
// of the block does not see one of its keys; the online softmax works in the
// exp2 domain with a lazy rescale.  Pass 0 also counts the kept chunk tokens
// before every 32-aligned position and a one-block pass ranks the call's
// (sequence, head) rows by work; the attention launch keeps as many
// workgroups as fit on the chip, each taking (row, query block) items in
// that order.
#include <type_traits>

#include "dms_common.h"
#include "dms_fp8.h"

namespace dms {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

constexpr int kThreads = 256;
// Attention pass workgroup: eight waves for FP8 pages at d = 128 (one
// workgroup per CU, two waves per SIMD), else four.  Each of a chunk's query
// blocks stages every cached tile of its head, so more waves per workgroup
// means fewer stagings per query: with FP8 pages a staging dequantizes the
// tile, and eight waves ran 3229 vs 3747 us per call at the 32B-shaped stress
// step; with bf16 pages eight waves ran slower (2585 vs 2480 us: more waves
// at every barrier).
template <int D, bool FP8>
constexpr int attn_threads() { return FP8 && D == 128 ? 512 : 256; }
constexpr uint32_t kNoKey = 0x7FFFFFFFu;  // key position of padding rows (never visible)
constexpr float kRescale = 8.0f;          // lazy rescale threshold, log2 units
constexpr float kMInit = -1.0e30f;        // running max before the first visible key

typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

// LDS tile layout.  A wave's MFMA operand load -- lane (r, G) = (lane % 16,
// lane / 16) takes 16 bytes -- is free of bank conflicts when the 64 lanes
// read one contiguous 1 KB block in lane order (measured on gfx950; rows of
// 64 bytes read column-wise are not).  The pool's tile layout is already in
// that order (dms_common.h): keys as 1 KB blocks per (32-dim slice, score
// MFMA row set), values (V^T) as 1 KB blocks per 16 dims, lane-ordered pieces
// inside each.  So staging copies a tile's 16-byte piece P to LDS slot P.

// max over the four lanes r, r + 16, r + 32, r + 48 (the key rows of one column)
__device__ inline float col_max(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const uint32_t v = __float_as_uint(y);
  const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

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
  int32_t* kept_before;   // [H][tph]: kept chunk tokens before chunk position 32 j (tile indexing)
  int32_t* order;         // [n * H]: (sequence, head) of attention grid row y, or null (row y itself)
  int32_t* work_ctr;      // attention work items taken so far (zeroed by pass 0)
  int nx, items;          // query blocks per grid row; rows x nx
  char* tiles;            // [2][H][tph] tiles: chunk tokens, then compacted kept tokens
  uint32_t* tmeta;        // [2][H][tph][32]: key rows of those tiles (position | flag << 31)
  float* out;             // [T, Hq, D]
  size_t page_bytes;
  int n, H, g, w, P, log2P, maxp, max_slots, max_seqs, total, max_len, PB, tph;
  int immediate;    // eviction timing: key j is hidden by the decision of j + w
  int zero_neuron;  // element 0 of each group's first query head is read as 0
  float scale_log2;
};

// Decision that hides chunk key c (chunk-local) once it leaves the window:
// its own (delayed eviction) or that of chunk token c + w (immediate
// eviction; none yet if c + w is past the chunk).
__device__ inline bool key_flag(const PrefillArgs& a, int tok0, int C, int c, int h) {
  const int x = a.immediate ? c + a.w : c;
  return x < C && a.flags[static_cast<size_t>(tok0 + x) * a.H + h] != 0;
}
__device__ inline bool key_kept(const PrefillArgs& a, int tok0, int C, int c, int h) {
  return !key_flag(a, tok0, C, c, h);
}

// Decisions from the borrowed query neuron (Sec. 3.2 rounding, App. C):
// flags[t][h] = (bf16 q[t][h * g][0] + bias > 0) in float32.
__global__ __launch_bounds__(kThreads) void prefill_decide_kernel(const uint16_t* q, uint8_t* flags,
                                                                  int total, int H, int g, int D,
                                                                  float bias) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(total) * H) return;
  const uint32_t bits = q[static_cast<size_t>(idx) * g * D];
  flags[idx] = (__uint_as_float(bits << 16) + bias) > 0.f;
}

__device__ inline size_t ws_tile(const PrefillArgs& a, int region, int h, int i, int k) {
  return ((static_cast<size_t>(region) * a.H + h) * a.tph + a.cu[i] / 32 + i + k);
}
// kept_before entry of chunk position 32 j of sequence i, head h
__device__ inline size_t ws_kb(const PrefillArgs& a, int h, int i, int j) {
  return static_cast<size_t>(h) * a.tph + a.cu[i] / 32 + i + j;
}

// Pass 0 (one block per (sequence, head)): validate the chunk boundaries,
// list the kept tokens of the chunk in position order and count them before
// every 32-aligned position.
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
  if (hh == 0 && threadIdx.x == 0 && a.work_ctr) *a.work_ctr = 0;
  int run = 0;
  for (int c0 = 0; c0 < C; c0 += blockDim.x) {
    const int c = c0 + threadIdx.x;
    const int kept = (c < C) && key_kept(a, tok0, C, c, h);
    int tot;
    const int off = block_exclusive_scan(kept, lds, &tot);
    if (kept) a.list[static_cast<size_t>(h) * a.total + tok0 + run + off] = c;
    if (c < C && (c & 31) == 0) a.kept_before[ws_kb(a, h, i, c >> 5)] = run + off;
    run += tot;
  }
  if (threadIdx.x == 0) a.list_cnt[hh] = run;
}


// Attention grid rows by decreasing work (rows are dispatched in order, so
// the longest heads start first and the short ones fill the tail): one
// workgroup ranks the n * H (sequence, head) rows by their live length plus
// half their kept chunk tokens (the cached keys every block of the row
// attends to, and the mean of its kept-prefix keys); ties keep row order.
constexpr int kOrderMax = 512;
__global__ __launch_bounds__(kThreads) void prefill_order_kernel(PrefillArgs a) {
  __shared__ int work[kOrderMax];
  if (load_status(a.status) != 0) return;
  const int NH = a.n * a.H;
  for (int x = threadIdx.x; x < NH; x += kThreads) {
    const int i = x / a.H, h = x % a.H;
    work[x] = a.len[a.seq_ids[i] * a.H + h] + a.list_cnt[x] / 2;
  }
  __syncthreads();
  for (int x = threadIdx.x; x < NH; x += kThreads) {
    const int wx = work[x];
    int rank = 0;
    for (int y = 0; y < NH; ++y) rank += work[y] > wx || (work[y] == wx && y < x);
    a.order[rank] = x;
  }
}

// Pass 1 (one block per (32-token tile, sequence x head, region)): copy the
// chunk's keys and values -- region 0: in chunk order; region 1: the kept
// tokens in list order -- into workspace tiles in the pool's tile layout
// (fragment order, values transposed); rows past the end are 0.
template <int D, bool FP8>
__global__ __launch_bounds__(kThreads) void prefill_tile_kernel(PrefillArgs a) {
  __shared__ uint16_t vrows[32][D + 2];
  if (load_status(a.status) != 0) return;
  const int k = blockIdx.x, hh = blockIdx.y, region = blockIdx.z;
  const int i = hh / a.H, h = hh % a.H;
  const int tok0 = a.cu[i], C = a.cu[i + 1] - a.cu[i];
  const int cnt = region ? a.list_cnt[hh] : C;
  if (k * 32 >= cnt) return;
  const int32_t* lst = a.list + static_cast<size_t>(h) * a.total + tok0;
  const int tid = threadIdx.x;
  constexpr int kPieces = 32 * D / 8;   // 16-byte pieces of 32 rows
  if (tid < 32) {
    // the tile's key rows as the pool's slot metadata has them: position |
    // flag << 31 (kept-list rows carry no flag); rows past the end: no key
    const int idx = 32 * k + tid;
    const int p0 = a.pos[a.seq_ids[i]];
    uint32_t mt = kNoKey;
    if (idx < cnt)
      mt = region ? static_cast<uint32_t>(p0 + lst[idx])
                  : (static_cast<uint32_t>(p0 + idx) | (key_flag(a, tok0, C, idx, h) ? kFlagBit : 0u));
    a.tmeta[ws_tile(a, region, h, i, k) * 32 + tid] = mt;
  }
  if constexpr (FP8) {
    // FP8 pages: the chunk's rows are quantized exactly as the commit will
    // store them (D/8 consecutive threads per row; rows past the end get
    // zero codes)
    char* tile = a.tiles + ws_tile(a, region, h, i, k) * fp8_tile_bytes(D);
    for (int pc = tid; pc < kPieces; pc += kThreads) {
      const int j = pc / (D / 8), part = pc % (D / 8);
      const int idx = 32 * k + j;
      uint4 kx = make_uint4(0u, 0u, 0u, 0u), vx = make_uint4(0u, 0u, 0u, 0u);
      if (idx < cnt) {
        const int c = region ? lst[idx] : idx;
        const size_t row = (static_cast<size_t>(tok0 + c) * a.H + h) * D + 8 * part;
        kx = *reinterpret_cast<const uint4*>(a.k + row);
        vx = *reinterpret_cast<const uint4*>(a.v + row);
      }
      fp8_store_token(tile, j, D, part, kx, vx);
    }
    return;
  }
  char* tile = a.tiles + ws_tile(a, region, h, i, k) * (D * 128);
  for (int pc = tid; pc < kPieces; pc += kThreads) {
    const int j = pc / (D / 8), e0 = 8 * (pc % (D / 8));
    const int idx = 32 * k + j;
    u32x4 kx = {0u, 0u, 0u, 0u}, vx = {0u, 0u, 0u, 0u};
    if (idx < cnt) {
      const int c = region ? lst[idx] : idx;
      const size_t row = (static_cast<size_t>(tok0 + c) * a.H + h) * D + e0;
      kx = *reinterpret_cast<const u32x4*>(a.k + row);
      vx = *reinterpret_cast<const u32x4*>(a.v + row);
    }
    *reinterpret_cast<u32x4*>(tile + k_elem_off(j, e0)) = kx;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      vrows[j][e0 + 2 * e] = static_cast<uint16_t>(vx[e] & 0xFFFFu);
      vrows[j][e0 + 2 * e + 1] = static_cast<uint16_t>(vx[e] >> 16);
    }
  }
  __syncthreads();
  // value piece q: dim q / 4, keys 8 (q % 4) .. + 7 (contiguous in the tile)
  for (int q = tid; q < kPieces; q += kThreads) {
    const int e = q >> 2, j0 = 8 * (q & 3);
    u32x4 x;
#pragma unroll
    for (int t = 0; t < 4; ++t)
      x[t] = static_cast<uint32_t>(vrows[j0 + 2 * t][e]) | (static_cast<uint32_t>(vrows[j0 + 2 * t + 1][e]) << 16);
    *reinterpret_cast<u32x4*>(tile + v_elem_off(j0, e, D)) = x;
  }
}

template <int D>
struct Frag {
  u32x4 ka[D / 32];
  u32x4 kb[D / 32];
  u32x4 vt[D / 16];
};

// Staging of one 32-key tile: each thread moves 16-byte pieces of a tile in
// the pool layout (a pool page or a workspace tile) through registers.
template <int D>
struct Stage {
  static constexpr int kPieces = (D * 128) / 16 / attn_threads<D, false>();  // 16-byte pieces per thread
  u32x4 kx[kPieces / 2];   // key pieces
  u32x4 vx[kPieces / 2];   // value pieces
  uint32_t meta;           // this thread's key row (threads 0..31): position | flag << 31
};

// FP8 staging: each thread moves 16-byte pieces of the code part (keys then
// values) and threads 0..15 one 16-byte piece of the scales.
template <int D>
struct StageF8 {
  static constexpr int kPieces = (D * 64) / 16;              // code pieces per tile
  static constexpr int kPer = (kPieces + attn_threads<D, true>() - 1) / attn_threads<D, true>();
  u32x4 cx[kPer];
  float ks[kPer];          // key scale of the token a key piece belongs to
  u32x4 sx;                // scales: [G][key scales (8) | value scales (8)]
  uint32_t meta;
};

// Online-softmax weights of one key tile for one column block: s0 / s1 are
// the scores of key rows 8 G .. 8 G + 3 and 8 G + 4 .. 8 G + 7 of the lane's
// column t.  kp / kx (read only when masked): position and expiry (first
// query that no longer sees it) of those rows; vsc (FP8): their value scales.
// Rescales o and l_run when the column's max rises past the threshold;
// returns the weights rounded to bf16 for the PV MFMAs.
template <int D, bool FP8>
__device__ __forceinline__ u32x4 col_weights(f32x4 s0, f32x4 s1, const float (&vsc)[8], bool masked,
                                             const int (&kp)[8], const int (&kx)[8], int t,
                                             f32x4 (&o)[D / 16], float& m_ref, float& l_run, float thr,
                                             float scale_log2) {
  float sc[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    sc[j] = s0[j];
    sc[j + 4] = s1[j];
  }
  if (masked) {
#pragma unroll
    for (int j = 0; j < 8; ++j) sc[j] = (kp[j] <= t && t < kx[j]) ? sc[j] : -INFINITY;
  }
  float mx = fmaxf(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3])),
                   fmaxf(fmaxf(sc[4], sc[5]), fmaxf(sc[6], sc[7])));
  mx = col_max(mx);
  const bool raise = mx > m_ref + thr;   // false while the column has seen no key
  if (__builtin_amdgcn_ballot_w64(raise)) {
    const float m_new = raise ? mx : m_ref;
    const float alpha = __builtin_amdgcn_exp2f((m_ref - m_new) * scale_log2);
    l_run *= alpha;
#pragma unroll
    for (int b = 0; b < D / 16; ++b) o[b] *= alpha;
    m_ref = m_new;
  }
  // p = 2^((s - m) * scale); hidden keys give exactly 0
  const float mb = m_ref * scale_log2;
  float e[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) e[j] = __builtin_amdgcn_exp2f(fmaf(sc[j], scale_log2, -mb));
  // P is rounded to bf16 for the MFMA; the denominator adds the same
  // rounded values (dot with (1, 1)), so a single dominant key returns its
  // value row exactly
  u32x4 pu;
  const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const f32x2 pr = {e[2 * j], e[2 * j + 1]};
    const bf16x2 pb = __builtin_convertvector(pr, bf16x2);
    pu[j] = __builtin_bit_cast(uint32_t, pb);
    l_run = __builtin_amdgcn_fdot2_f32_bf16(pb, ones, l_run, false);
    if constexpr (FP8) {
      // PV weights carry the value scale: rounding commutes with a
      // power-of-two factor, so these are the rounded weights times it
      const f32x2 pv = {e[2 * j] * vsc[2 * j], e[2 * j + 1] * vsc[2 * j + 1]};
      pu[j] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pv, bf16x2));
    }
  }
  return pu;
}

// Scores, online softmax and PV of one key tile for the NQ column blocks of a
// wave.
template <int D, int NQ, bool FP8>
__device__ __forceinline__ void attend_tile(const Frag<D>& f, const float (&vsc)[8], bool masked,
                                            const int (&kp)[8], const int (&kx)[8],
                                            const int (&tcol)[NQ], const u32x4 (&qf)[NQ][D / 32],
                                            f32x4 (&o)[NQ][D / 16], float (&m_ref)[NQ],
                                            float (&l_run)[NQ], float thr, float scale_log2) {
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s2 = 0; s2 < D / 32; ++s2) {
      s0 = mfma_bf16(f.ka[s2], qf[qb][s2], s0);
      s1 = mfma_bf16(f.kb[s2], qf[qb][s2], s1);
    }
    const u32x4 pu = col_weights<D, FP8>(s0, s1, vsc, masked, kp, kx, tcol[qb], o[qb], m_ref[qb], l_run[qb],
                                         thr, scale_log2);
#pragma unroll
    for (int b = 0; b < D / 16; ++b) o[qb][b] = mfma_bf16(f.vt[b], pu, o[qb][b]);
  }
}

template <int D, int NQ, bool FP8>
__global__ __launch_bounds__((attn_threads<D, FP8>()), (512 / attn_threads<D, FP8>())) void prefill_kernel(PrefillArgs a) {
  constexpr int kThreads = attn_threads<D, FP8>();
  __shared__ __attribute__((aligned(16))) char tile_lds[2][D * 128];
  __shared__ __attribute__((aligned(16))) float scale_lds[2][64];   // FP8: tile scales
  __shared__ uint32_t meta_lds[2][32];
  __shared__ int masked_lds[2];   // tile has a key hidden from some query of the block
  __shared__ int item_lds[2];
  if (load_status(a.status) != 0) return;
  // attention of work item `item` = (grid row item / nx, query block item % nx)
  auto attend = [&](int item) {
  const int row = item / a.nx;
  const int hh = a.order ? a.order[row] : row;
  const int i = hh / a.H, h = hh % a.H;
  const int tok0 = a.cu[i], C = a.cu[i + 1] - a.cu[i];
  const int pb0 = (item - row * a.nx) * a.PB;
  if (pb0 >= C) return;
  const int s = a.seq_ids[i];
  const int sh = s * a.H + h;
  const int p0 = a.pos[s];
  const int L0 = a.len[sh];
  const int t0 = p0 + pb0;
  const int t1 = p0 + min(C, pb0 + a.PB);
  // band: chunk tiles from the one holding max(p0, t0 - w + 1) up to t1
  const int band_c0 = (max(0, pb0 - a.w + 1) >> 5) << 5;   // chunk-local, < C
  // kept chunk keys strictly before the band (a prefix of the sorted list),
  // counted by pass 0
  const int32_t* lst = a.list + static_cast<size_t>(h) * a.total + tok0;
  const int n_pre = a.kept_before[ws_kb(a, h, i, band_c0 >> 5)];
  const int nc = (L0 + 31) >> 5;
  const int np = (n_pre + 31) >> 5;
  const int nb = (t1 - p0 - band_c0 + 31) >> 5;
  constexpr size_t kTB = FP8 ? static_cast<size_t>(D) * 64 + 256 : static_cast<size_t>(D) * 128;
  const char* pre_tiles = a.tiles + ws_tile(a, 1, h, i, 0) * kTB;
  const char* band_tiles = a.tiles + ws_tile(a, 0, h, i, band_c0 >> 5) * kTB;
  const int ntiles = nc + np + nb;
  const int32_t* pt = a.page_table + static_cast<size_t>(sh) * a.maxp;
  const int32_t* smeta = a.slot_meta + static_cast<size_t>(sh) * a.max_slots;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, G = lane >> 4;
  const int Hq = a.H * a.g;

  // ---- columns of this lane: column c of the workgroup's (wave, block,
  // lane r) is query head c % g at position t0 + c / g (a position's heads
  // may straddle two column blocks)
  int tcol[NQ];
  u32x4 qf[NQ][D / 32];
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
    const int col = (wave * NQ + qb) * 16 + r;
    const int pl = col / a.g, qh = col % a.g;
    const int t = t0 + pl;
    const bool ok = (pl < a.PB) && (t < t1);
    tcol[qb] = ok ? t : -1;
    const u32x4 z = {0u, 0u, 0u, 0u};
    const char* qrow = reinterpret_cast<const char*>(
        a.q + (static_cast<size_t>(tok0 + (t - p0)) * Hq + h * a.g + qh) * D);
#pragma unroll
    for (int s2 = 0; s2 < D / 32; ++s2)
      qf[qb][s2] = ok ? *reinterpret_cast<const u32x4*>(qrow + (32 * s2 + 8 * G) * 2) : z;
    // the borrowed decision neuron takes no part in attention (App. C)
    if (a.zero_neuron && qh == 0 && G == 0) qf[qb][0][0] &= 0xFFFF0000u;
  }

  // ---- staging: global -> registers (A), registers -> LDS (B)
  using StageT = typename std::conditional<FP8, StageF8<D>, Stage<D>>::type;
  StageT stg;
  auto stage_load = [&](int k) {
    const char* tile;
    if (k < nc) {
      const int sb = k * 32;
      tile = a.pool + static_cast<size_t>(pt[sb >> a.log2P]) * a.page_bytes +
             static_cast<size_t>((sb & (a.P - 1)) >> 5) * kTB;
      if (tid < 32) {
        uint32_t mt = sb + tid < L0 ? static_cast<uint32_t>(smeta[sb + tid]) : kNoKey;
        if (a.immediate && mt != kNoKey) {
          // a cached key j is hidden by the decision of position j + w, which
          // (for a live key) lies in this chunk or later
          const int kp = static_cast<int>(mt & ~kFlagBit);
          const int x = kp + a.w - p0;
          mt = static_cast<uint32_t>(kp) |
               ((x >= 0 && x < C && a.flags[static_cast<size_t>(tok0 + x) * a.H + h]) ? kFlagBit : 0u);
        }
        stg.meta = mt;
      }
    } else if (k < nc + np) {
      const int kk = k - nc;
      tile = pre_tiles + static_cast<size_t>(kk) * kTB;
      if (tid < 32) {
        const int idx = kk * 32 + tid;
        stg.meta = idx < n_pre ? static_cast<uint32_t>(p0 + lst[idx]) : kNoKey;
      }
    } else {
      const int kb = k - nc - np;
      tile = band_tiles + static_cast<size_t>(kb) * kTB;
      if (tid < 32) {
        const int c = band_c0 + kb * 32 + tid;
        stg.meta = c < t1 - p0 ? (static_cast<uint32_t>(p0 + c) |
                                  (key_flag(a, tok0, C, c, h) ? kFlagBit : 0u))
                               : kNoKey;
      }
    }
    if constexpr (FP8) {
#pragma unroll
      for (int m = 0; m < StageF8<D>::kPer; ++m) {
        const int Q = tid + m * kThreads;
        if (Q < StageF8<D>::kPieces) stg.cx[m] = *reinterpret_cast<const u32x4*>(tile + Q * 16);
        if (Q < 2 * D) {
          // key piece (p, h, lane L): all 16 codes belong to slot 8 (r/4) + r%4 + 4 h
          const int r = Q & 15, j = 8 * (r >> 2) + (r & 3) + 4 * ((Q >> 6) & 1);
          stg.ks[m] = *reinterpret_cast<const float*>(tile + D * 64 + (j >> 3) * 64 + (j & 7) * 4);
        }
      }
      if (tid < 16) stg.sx = *reinterpret_cast<const u32x4*>(tile + D * 64 + tid * 16);
    } else {
      constexpr int KP = Stage<D>::kPieces / 2;
#pragma unroll
      for (int m = 0; m < KP; ++m) {
        stg.kx[m] = *reinterpret_cast<const u32x4*>(tile + (tid + m * kThreads) * 16);
        stg.vx[m] = *reinterpret_cast<const u32x4*>(tile + D * 64 + (tid + m * kThreads) * 16);
      }
    }
  };
  auto stage_store = [&](int k, int buf) {
    char* dst = tile_lds[buf];
    // pool slots past L hold stale data: their value elements are zeroed
    // (workspace tiles are zero past their last row)
    const int valid = k < nc ? min(32, L0 - k * 32) : 32;
    if constexpr (FP8) {
      // a 16-byte code piece becomes two bf16 LDS slots (exact conversion);
      // the FP8 tile order matches the LDS fragment order (dms_fp8.h)
#pragma unroll
      for (int m = 0; m < StageF8<D>::kPer; ++m) {
        const int Q = tid + m * kThreads;
        if (Q < StageF8<D>::kPieces) {
          u32x4 x = stg.cx[m];
          int P0, step;
          float scale = 1.0f;
          if (Q < 2 * D) {            // keys: piece (p, h, lane L), dequantized exactly
            P0 = 256 * (Q >> 7) + (Q & 127);
            step = 128;
            scale = stg.ks[m];
          } else {                    // values: piece (p, lane L), slots 8G .. 8G+7
            const int Qv = Q - 2 * D;
            P0 = D * 4 + 128 * (Qv >> 6) + (Qv & 63);
            step = 64;
            const int nv = valid - 8 * ((Qv >> 4) & 3);
            if (nv < 8) {
              const uint64_t keep8 = nv <= 0 ? 0ull : (~0ull >> (8 * (8 - nv)));
              const uint32_t klo = static_cast<uint32_t>(keep8), khi = static_cast<uint32_t>(keep8 >> 32);
              x[0] &= klo;
              x[1] &= khi;
              x[2] &= klo;
              x[3] &= khi;
            }
          }
          u32x4 lo, hi;
#pragma unroll
          for (int w2 = 0; w2 < 2; ++w2) {
            lo[2 * w2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x[w2], scale, false));
            lo[2 * w2 + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x[w2], scale, true));
            hi[2 * w2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x[2 + w2], scale, false));
            hi[2 * w2 + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x[2 + w2], scale, true));
          }
          *reinterpret_cast<u32x4*>(dst + P0 * 16) = lo;
          *reinterpret_cast<u32x4*>(dst + (P0 + step) * 16) = hi;
        }
      }
      if (tid < 16) {
        // scale piece tid: group G = tid / 4, key (tid % 4 < 2) or value scales of
        // slots 8 G + 4 (tid % 2) .. + 3; missing slots get 0
        u32x4 x = stg.sx;
        const int j0 = 8 * (tid >> 2) + 4 * (tid & 1);
#pragma unroll
        for (int c = 0; c < 4; ++c)
          if (j0 + c >= valid) x[c] = 0u;
        *reinterpret_cast<u32x4*>(&scale_lds[buf][4 * tid]) = x;
      }
    } else {
      constexpr int KP = Stage<D>::kPieces / 2;
#pragma unroll
      for (int m = 0; m < KP; ++m) {
        const int P = tid + m * kThreads;
        *reinterpret_cast<u32x4*>(dst + P * 16) = stg.kx[m];
        u32x4 x = stg.vx[m];
        // element i of the value piece is key row 8 G + i
        const int j0 = 8 * ((P >> 4) & 3);
        if (j0 + 8 > valid) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (j0 + e >= valid) x[e >> 1] &= (e & 1) ? 0x0000FFFFu : 0xFFFF0000u;
        }
        *reinterpret_cast<u32x4*>(dst + D * 64 + P * 16) = x;
      }
    }
    if (tid < 64) {
      // a key row needs the per-element mask iff some query t in [t0, t1)
      // does not see it: padding, causal (position > t0) or flagged and
      // expiring by t1 - 1
      bool need = false;
      if (tid < 32) {
        const uint32_t mt = stg.meta;
        const int kp = static_cast<int>(mt & ~kFlagBit);
        need = mt == kNoKey || kp > t0 || ((mt & kFlagBit) && kp + a.w <= t1 - 1);
        meta_lds[buf][tid] = mt;
      }
      const uint64_t any = __builtin_amdgcn_ballot_w64(need);
      if (tid == 0) masked_lds[buf] = any != 0;
    }
  };

  // ---- accumulators
  f32x4 o[NQ][D / 16];
  float m_ref[NQ], l_run[NQ];
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
#pragma unroll
    for (int b = 0; b < D / 16; ++b) o[qb][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_ref[qb] = kMInit;
    l_run[qb] = 0.f;
  }
  const uint32_t lo_k = static_cast<uint32_t>(lane * 16);
  const uint32_t lo_v = static_cast<uint32_t>(D * 64 + lane * 16);
  const float thr = kRescale / a.scale_log2;   // rescale threshold in score units

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
      f.kb[s2] = *reinterpret_cast<const u32x4*>(tl + lo_k + 1024 + s2 * 2048);
    }
#pragma unroll
    for (int b = 0; b < D / 16; ++b) f.vt[b] = *reinterpret_cast<const u32x4*>(tl + lo_v + b * 1024);
    float vsc[8];   // FP8: value scales of rows 8G .. 8G+7 (keys are staged dequantized)
    if constexpr (FP8) {
      const f32x4 v0 = *reinterpret_cast<const f32x4*>(&scale_lds[buf][16 * G + 8]);
      const f32x4 v1 = *reinterpret_cast<const f32x4*>(&scale_lds[buf][16 * G + 12]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        vsc[j] = v0[j];
        vsc[j + 4] = v1[j];
      }
    }
    const bool masked = __builtin_amdgcn_readfirstlane(masked_lds[buf]) != 0;
    int kp[8], kx[8];   // key position and expiry (first query that no longer sees it)
    if (masked) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t km = meta_lds[buf][8 * G + j];
        kp[j] = static_cast<int>(km & ~kFlagBit);
        kx[j] = (km & kFlagBit) ? kp[j] + a.w : 0x7FFFFFFF;
      }
    }
    attend_tile<D, NQ, FP8>(f, vsc, masked, kp, kx, tcol, qf, o, m_ref, l_run, thr, a.scale_log2);
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
      const int qh = ((wave * NQ + qb) * 16 + r) % a.g;
      const float inv = 1.0f / l;
      float* dst = a.out + (static_cast<size_t>(tok0 + (t - p0)) * Hq + h * a.g + qh) * D + 4 * G;
#pragma unroll
      for (int b = 0; b < D / 16; ++b) *reinterpret_cast<f32x4*>(dst + 16 * b) = o[qb][b] * inv;
    }
  }
};

  // items as in the bf16 pass: grid position first, then the counter
  int item = blockIdx.x, buf = 0;
  if (threadIdx.x == 0) item_lds[0] = gridDim.x + atomicAdd(a.work_ctr, 1);
  while (item < a.items) {
    attend(item);
    __syncthreads();   // the fetched index is visible; every wave is done with the LDS buffers
    const int next = item_lds[buf];
    if (threadIdx.x == 0) item_lds[buf ^ 1] = gridDim.x + atomicAdd(a.work_ctr, 1);
    buf ^= 1;
    item = next;
  }
}

// ---- bf16 pages under delayed eviction: tiles copied by the hardware.
// Every key source is a plain copy -- pool tiles with their slot metadata,
// workspace tiles with the metadata pass 1 wrote -- so global -> LDS loads
// (global_load_lds) move tiles and key rows into four LDS buffers, each tile
// by one wave (the address work is done once per tile) two tiles ahead of
// the one being attended, with no staging registers or LDS stores.  Rows
// past a source's end are fixed up when read: pool slots past the live
// length hold stale data (values zeroed in registers, keys hidden),
// kept-list rows from the band on are hidden.
//
// The LDS destination of a copy goes in M0, written by the same inline
// assembly statement as the load; nothing else in this kernel reads M0.  The
// compiler does not count these loads, so the kernel waits for them itself
// (vmcnt) before the barrier that publishes a tile.
#define DMS_LDS __attribute__((address_space(3)))
#define DMS_CONST __attribute__((address_space(4)))

constexpr int wait_vm(int n) { return 0x0F70 | (n & 15) | ((n >> 4) << 14); }

__device__ inline uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((DMS_LDS const char*)p));
}

// 64 lanes x 16 bytes from g (per lane) to LDS m0 + 16 lane
__device__ inline void lds_copy16(const char* g, uint32_t m0) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" : : "s"(m0), "v"(g) : "memory", "m0");
}
// 64 lanes x 4 bytes from g (per lane) to LDS m0 + 4 lane
__device__ inline void lds_copy4(const char* g, uint32_t m0) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off" : : "s"(m0), "v"(g) : "memory", "m0");
}

// ---- attention pass, the two column blocks of a wave half a tile apart.
// With every step of a tile in one order (scores, weights, PV) the weights'
// VALU work (maxima, exponentials, bf16 rounding, denominators) waits for the
// score MFMAs and the PV MFMAs wait for it.  Here a tile k is attended in two
// halves, each pairing one block's weights with MFMAs of the other block:
//   A(k): weights of block 0 on tile k   | scores of block 1 on tile k, then
//                                        | PV of block 1 on tile k - 1
//   B(k): weights of block 1 on tile k   | scores of block 0 on tile k + 1,
//                                        | then PV of block 0 on tile k
// A half starts with its block's mask, column maxima and (rare, wave-uniform)
// rescale; the rest is one straight stretch in which scheduling groups
// alternate single MFMAs with a share of the VALU work and of the LDS operand
// reads.  Tile k + 1's keys and key rows are read during A(k) (after the
// score MFMAs of tile k have taken theirs), tile k's values at its end, so
// one register set holds each operand.  Four LDS buffers: at the start of
// A(k) one barrier publishes tile k + 1 and frees the buffer of tile k - 1,
// into which tile k + 3 is copied.
template <int M, int V, int R, int I = 0>
__device__ __forceinline__ void interleave() {
  if constexpr (I < M) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
    constexpr int nr = R / M + (I < R % M ? 1 : 0);
    if constexpr (nr > 0) __builtin_amdgcn_sched_group_barrier(0x100, nr, 0);   // LDS reads
    constexpr int nv = V / M + (I < V % M ? 1 : 0);
    if constexpr (nv > 0) __builtin_amdgcn_sched_group_barrier(0x002, nv, 0);   // VALU
    interleave<M, V, R, I + 1>();
  }
}

template <int D>
__global__ __launch_bounds__(256, 2) void prefill_pipe_kernel(PrefillArgs a) {
  constexpr int NQ = 2;
  constexpr int kBuf = 4;
  constexpr int kTB = D * 128;
  constexpr int kLoads = D / 32;   // 1 KB copies per wave and tile (four waves)
  constexpr int KS = D / 32;       // k-steps of a score MFMA chain
  constexpr int OB = D / 16;       // 16-dim output blocks
  __shared__ __attribute__((aligned(16))) char tile_lds[kBuf][kTB];
  __shared__ __attribute__((aligned(16))) uint32_t meta_lds[kBuf][64];   // rows 0..31, twice
  __shared__ int item_lds[2];
  if (load_status(a.status) != 0) return;
  // attention of work item `item` = (grid row item / nx, query block item % nx)
  auto attend = [&](int item) {
  const int row = item / a.nx;
  const int hh = a.order ? a.order[row] : row;
  const int i = hh / a.H, h = hh % a.H;
  const int tok0 = a.cu[i], C = a.cu[i + 1] - a.cu[i];
  const int pb0 = (item - row * a.nx) * a.PB;
  if (pb0 >= C) return;
  const int s = a.seq_ids[i];
  const int sh = s * a.H + h;
  const int p0 = a.pos[s];
  const int L0 = a.len[sh];
  const int t0 = p0 + pb0;
  const int t1 = p0 + min(C, pb0 + a.PB);
  const int band_c0 = (max(0, pb0 - a.w + 1) >> 5) << 5;   // chunk-local, < C
  // kept chunk keys strictly before the band, counted by pass 0
  const int n_pre = a.kept_before[ws_kb(a, h, i, band_c0 >> 5)];
  const int nc = (L0 + 31) >> 5;
  const int np = (n_pre + 31) >> 5;
  const int nb = (t1 - p0 - band_c0 + 31) >> 5;
  const int ntiles = nc + np + nb;
  const char* pre_tiles = a.tiles + ws_tile(a, 1, h, i, 0) * kTB;
  const char* band_tiles = a.tiles + ws_tile(a, 0, h, i, band_c0 >> 5) * kTB;
  const uint32_t* pre_meta = a.tmeta + ws_tile(a, 1, h, i, 0) * 32;
  const uint32_t* band_meta = a.tmeta + ws_tile(a, 0, h, i, band_c0 >> 5) * 32;
  const DMS_CONST int32_t* pt = (const DMS_CONST int32_t*)(a.page_table + static_cast<size_t>(sh) * a.maxp);
  const uint32_t* smeta = reinterpret_cast<const uint32_t*>(a.slot_meta + static_cast<size_t>(sh) * a.max_slots);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, G = lane >> 4;
  const int Hq = a.H * a.g;

  // column c of the workgroup's 128 (wave, block, lane r) is query head c % g
  // at position t0 + c / g; a position's g heads may straddle two column
  // blocks, so only the last 128 mod g columns go unused
  int tcol[NQ];
  u32x4 qf[NQ][KS];
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
    const int col = (wave * NQ + qb) * 16 + r;
    const int pl = col / a.g, qh = col % a.g;
    const int t = t0 + pl;
    const bool ok = (pl < a.PB) && (t < t1);
    tcol[qb] = ok ? t : -1;
    const u32x4 z = {0u, 0u, 0u, 0u};
    const char* qrow = reinterpret_cast<const char*>(
        a.q + (static_cast<size_t>(tok0 + (t - p0)) * Hq + h * a.g + qh) * D);
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2)
      qf[qb][s2] = ok ? *reinterpret_cast<const u32x4*>(qrow + (32 * s2 + 8 * G) * 2) : z;
    if (a.zero_neuron && qh == 0 && G == 0) qf[qb][0][0] &= 0xFFFF0000u;
  }

  // pool page of tile k (only read for k < nc)
  auto page_of = [&](int k) { return k < nc ? pt[(32 * k) >> a.log2P] : 0; };
  // tile k is copied by wave k % 4 alone (the address work is done once per
  // tile), 1 KB per instruction
  auto issue = [&](int k, int page) {
    if (wave != (k & 3)) return;
    const char* tile;
    const uint32_t* mt;
    if (k < nc) {
      const int sb = 32 * k;
      tile = a.pool + static_cast<size_t>(page) * a.page_bytes + static_cast<size_t>((sb & (a.P - 1)) >> 5) * kTB;
      mt = smeta + sb;
    } else if (k < nc + np) {
      tile = pre_tiles + static_cast<size_t>(k - nc) * kTB;
      mt = pre_meta + (k - nc) * 32;
    } else {
      tile = band_tiles + static_cast<size_t>(k - nc - np) * kTB;
      mt = band_meta + (k - nc - np) * 32;
    }
    const int b = k % kBuf;
    const uint32_t dst = lds_addr(tile_lds[b]);
#pragma unroll
    for (int m = 0; m < 4 * kLoads; ++m) lds_copy16(tile + m * 1024 + lane * 16, dst + m * 1024);
    lds_copy4(reinterpret_cast<const char*>(mt + (lane & 31)), lds_addr(meta_lds[b]));
  };
  // tile k has landed once the wave that copied it has no copy in flight
  // (its next copy is issued after tile k is published)
  auto wait_tile = [&](int k) {
    if (wave == (k & 3)) __builtin_amdgcn_s_waitcnt(wait_vm(0));
  };

  f32x4 o[NQ][OB];
  float m_ref[NQ], l_run[NQ];
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
#pragma unroll
    for (int b = 0; b < OB; ++b) o[qb][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_ref[qb] = kMInit;
    l_run[qb] = 0.f;
  }
  const uint32_t lo_k = static_cast<uint32_t>(lane * 16);
  const uint32_t lo_v = static_cast<uint32_t>(D * 64 + lane * 16);
  const float thr = kRescale / a.scale_log2;
  const float sl2 = a.scale_log2;

  // operand registers: keys (and key rows) of one tile, values of one tile
  u32x4 ka[KS], kb[KS], vt[OB];
  uint32_t nrow = 0;
  u32x4 nm0, nm1;
  auto read_k = [&](int k) {
    const char* tl = tile_lds[k % kBuf];
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) {
      ka[s2] = *reinterpret_cast<const u32x4*>(tl + lo_k + s2 * 2048);
      kb[s2] = *reinterpret_cast<const u32x4*>(tl + lo_k + 1024 + s2 * 2048);
    }
    nrow = meta_lds[k % kBuf][lane];
    nm0 = *reinterpret_cast<const u32x4*>(&meta_lds[k % kBuf][8 * G]);
    nm1 = *reinterpret_cast<const u32x4*>(&meta_lds[k % kBuf][8 * G + 4]);
  };
  auto read_v = [&](int k) {
    const char* tl = tile_lds[k % kBuf];
#pragma unroll
    for (int b = 0; b < OB; ++b) vt[b] = *reinterpret_cast<const u32x4*>(tl + lo_v + b * 1024);
  };
  auto scores = [&](int qb, float (&sc)[8]) {
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) {
      s0 = mfma_bf16(ka[s2], qf[qb][s2], s0);
      s1 = mfma_bf16(kb[s2], qf[qb][s2], s1);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      sc[j] = s0[j];
      sc[j + 4] = s1[j];
    }
  };
  auto pv = [&](int qb, u32x4 pu) {
#pragma unroll
    for (int b = 0; b < OB; ++b) o[qb][b] = mfma_bf16(vt[b], pu, o[qb][b]);
  };
  // mask, column max and lazy rescale of one block's scores
  auto head = [&](int qb, float (&sc)[8], bool masked, const int (&kp)[8], const int (&kx)[8]) {
    if (masked) {
      const int t = tcol[qb];
#pragma unroll
      for (int j = 0; j < 8; ++j) sc[j] = (kp[j] <= t && t < kx[j]) ? sc[j] : -INFINITY;
    }
    float mx = fmaxf(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3])),
                     fmaxf(fmaxf(sc[4], sc[5]), fmaxf(sc[6], sc[7])));
    mx = col_max(mx);
    const bool raise = mx > m_ref[qb] + thr;
    if (__builtin_amdgcn_ballot_w64(raise)) {
      const float m_new = raise ? mx : m_ref[qb];
      const float alpha = __builtin_amdgcn_exp2f((m_ref[qb] - m_new) * sl2);
      l_run[qb] *= alpha;
#pragma unroll
      for (int b = 0; b < OB; ++b) o[qb][b] *= alpha;
      m_ref[qb] = m_new;
    }
  };
  // weights p = 2^((s - m) scale) rounded to bf16, in two parts: the first
  // forms half of the exponentials, the second the rest, the rounding and
  // the denominator (which adds the rounded values, dot with (1, 1))
  auto weights1 = [&](int qb, const float (&sc)[8], float (&e)[8]) {
    const float mb = m_ref[qb] * sl2;
#pragma unroll
    for (int j = 0; j < 8; ++j) e[j] = fmaf(sc[j], sl2, -mb);
#pragma unroll
    for (int j = 0; j < 4; ++j) e[j] = __builtin_amdgcn_exp2f(e[j]);
  };
  auto weights2 = [&](int qb, float (&e)[8]) {
#pragma unroll
    for (int j = 4; j < 8; ++j) e[j] = __builtin_amdgcn_exp2f(e[j]);
    u32x4 pu;
    const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x2 pr = {e[2 * j], e[2 * j + 1]};
      const bf16x2 pb = __builtin_convertvector(pr, bf16x2);
      pu[j] = __builtin_bit_cast(uint32_t, pb);
      l_run[qb] = __builtin_amdgcn_fdot2_f32_bf16(pb, ones, l_run[qb], false);
    }
    return pu;
  };

  for (int j = 0; j < min(kBuf - 1, ntiles); ++j) issue(j, page_of(j));
  int page = page_of(kBuf - 1);   // page of the next tile to copy
  // the query loads and this wave's first copy are in flight together; both
  // complete here, so that no wait the compiler places for the query loads
  // can fall inside the loop
  __builtin_amdgcn_s_waitcnt(wait_vm(0));
  float sc0[8], sc1[8];
  u32x4 pu1 = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int b = 0; b < OB; ++b) vt[b] = u32x4{0u, 0u, 0u, 0u};
  if (ntiles > 0) {
    wait_tile(0);
    __syncthreads();
    read_k(0);
    scores(0, sc0);
  }
  for (int k = 0; k < ntiles; ++k) {
    // ---- A(k) head: publish tile k + 1, copy tile k + 3 into tile k - 1's buffer
    if (k + 1 < ntiles) wait_tile(k + 1);
    __syncthreads();
    if (k + 3 < ntiles) issue(k + 3, page);
    // key rows of tile k; rows past the source's end hold no key
    const int rows = k < nc ? L0 - 32 * k : (k < nc + np ? n_pre - 32 * (k - nc) : 32);
    uint32_t mrow = nrow;
    u32x4 m0 = nm0, m1 = nm1;
    if (rows < 32) {
      if ((lane & 31) >= rows) mrow = kNoKey;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (8 * G + j >= rows) m0[j] = kNoKey;
        if (8 * G + 4 + j >= rows) m1[j] = kNoKey;
      }
    }
    // a key row needs the per-element mask iff some query t in [t0, t1)
    // does not see it: no key, causal (position > t0) or flagged and
    // expiring by t1 - 1
    const int kpr = static_cast<int>(mrow & ~kFlagBit);
    const bool need = mrow == kNoKey || kpr > t0 || ((mrow & kFlagBit) && kpr + a.w <= t1 - 1);
    const bool masked = __builtin_amdgcn_ballot_w64(need) != 0;
    int kp[8], kx[8];
    if (masked) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t km = j < 4 ? m0[j] : m1[j - 4];
        kp[j] = static_cast<int>(km & ~kFlagBit);
        kx[j] = (km & kFlagBit) ? kp[j] + a.w : 0x7FFFFFFF;
      }
    }
    head(0, sc0, masked, kp, kx);
    // ---- A(k) stretch
    float e[8];
    __builtin_amdgcn_sched_barrier(0);
    scores(1, sc1);
    weights1(0, sc0, e);
    interleave<2 * KS, 12, 0>();
    __builtin_amdgcn_sched_barrier(0);
    pv(1, pu1);
    read_k(k + 1);
    const u32x4 pu0 = weights2(0, e);
    interleave<OB, 12, 2 * KS + 3>();
    __builtin_amdgcn_sched_barrier(0);
    // the weights are formed here, beside the MFMAs above, not next to their
    // first use in B(k)
    asm volatile("" : : "v"(pu0), "v"(l_run[0]));
    read_v(k);
    __builtin_amdgcn_sched_barrier(0);
    // ---- B(k) head
    if (rows < 32) {
      // stale pool slots: value elements of rows 8 G + e >= rows are zeroed
      u32x4 keep;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        keep[q] = (8 * G + 2 * q < rows ? 0x0000FFFFu : 0u) | (8 * G + 2 * q + 1 < rows ? 0xFFFF0000u : 0u);
#pragma unroll
      for (int b = 0; b < OB; ++b) vt[b] &= keep;
    }
    head(1, sc1, masked, kp, kx);
    // ---- B(k) stretch
    __builtin_amdgcn_sched_barrier(0);
    scores(0, sc0);
    weights1(1, sc1, e);
    interleave<2 * KS, 12, 0>();
    __builtin_amdgcn_sched_barrier(0);
    pv(0, pu0);
    pu1 = weights2(1, e);
    interleave<OB, 12, 0>();
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" : : "v"(pu1), "v"(l_run[1]));
    // after this iteration's last LDS operand use: a scalar load in flight
    // would turn every LDS wait before it into a full one
    if (k + 4 < nc) page = pt[(32 * (k + 4)) >> a.log2P];
  }
  if (ntiles > 0) pv(1, pu1);

  // ---- outputs
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
    float l = l_run[qb];
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    const int t = tcol[qb];
    if (t >= 0) {
      const int qh = ((wave * NQ + qb) * 16 + r) % a.g;
      const float inv = 1.0f / l;
      float* dst = a.out + (static_cast<size_t>(tok0 + (t - p0)) * Hq + h * a.g + qh) * D + 4 * G;
#pragma unroll
      for (int b = 0; b < OB; ++b) *reinterpret_cast<f32x4*>(dst + 16 * b) = o[qb][b] * inv;
    }
  }
};

  // Items one after another: the first from the workgroup's grid position, the
  // rest in order from a counter that pass 0 zeroed, each fetched one item
  // ahead.  Rows come heaviest first, so the last items to start are short
  // and the workgroups finish together (the launch has as many workgroups as
  // fit on the chip at once).
  int item = blockIdx.x, buf = 0;
  if (threadIdx.x == 0) item_lds[0] = gridDim.x + atomicAdd(a.work_ctr, 1);
  while (item < a.items) {
    attend(item);
    __syncthreads();   // the fetched index is visible; every wave is done with the LDS buffers
    const int next = item_lds[buf];
    if (threadIdx.x == 0) item_lds[buf ^ 1] = gridDim.x + atomicAdd(a.work_ctr, 1);
    buf ^= 1;
    item = next;
  }
}

constexpr int kNQ = 2;

// compute units of the current device (queried once)
int cu_count() {
  static int n = 0;
  if (n == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
      n = v;
    else
      return 256;
  }
  return n;
}

template <int D, bool FP8>
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
  a.tiles = w + lo.ws_pf_tiles;
  a.tmeta = reinterpret_cast<uint32_t*>(w + lo.ws_pf_tmeta);
  a.kept_before = reinterpret_cast<int32_t*>(w + lo.ws_pf_kb);
  a.order = nullptr;
  a.work_ctr = a.list_cnt + lo.max_heads;   // the word after the per-head counts
  a.nx = a.items = 0;
  a.tph = lo.pf_tiles_per_head;
  a.immediate = c.eviction == DMS_EVICT_IMMEDIATE;
  a.zero_neuron = c.decision_source == DMS_DECIDE_QUERY;
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
  const bool pipe = !FP8 && !a.immediate;
  // positions per attention workgroup: its (position, head) columns fill 16
  // per column block, kNQ blocks per wave
  a.PB = (pipe ? 256 : attn_threads<D, FP8>()) / 64 * kNQ * 16 / c.group_size;
  a.scale_log2 = c.softmax_scale * 1.4426950408889634f;
  const int NH = n * c.num_kv_heads;
  // the timing events bracket every pass
  if (ev_start) (void)hipEventRecord(ev_start, st);
  hipLaunchKernelGGL(prefill_list_kernel, dim3(NH), dim3(kThreads), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (NH > 1 && NH <= kOrderMax) {
    a.order = reinterpret_cast<int32_t*>(w + lo.ws_pf_order);
    hipLaunchKernelGGL(prefill_order_kernel, dim3(1), dim3(kThreads), 0, st, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((prefill_tile_kernel<D, FP8>), dim3((max_len + 31) / 32, NH, 2), dim3(kThreads), 0,
                     st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 grid((max_len + a.PB - 1) / a.PB, NH);
  // as many workgroups as fit on the chip at once, each taking work items
  // until none is left
  a.nx = static_cast<int>(grid.x);
  a.items = a.nx * NH;
  if (pipe)
    hipLaunchKernelGGL((prefill_pipe_kernel<D>), dim3(min(a.items, 2 * cu_count())), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((prefill_kernel<D, kNQ, FP8>),
                       dim3(min(a.items, 512 / attn_threads<D, FP8>() * cu_count())),
                       dim3(attn_threads<D, FP8>()), 0, st, a);
  e = hipGetLastError();
  if (ev_stop) (void)hipEventRecord(ev_stop, st);
  return e;
}


// ---------------------------------------------------------------------------
// Chunked prefill over a latent-attention (MLA) cache: one KV head of
// 576-dim rows shared by the g query heads, in the absorbed form of the
// latent decode: column (position t, query head h) scores row j by q . row
// over all 576 dims and sums the rows' first 512 (latent) dims.  The mask and
// the three key sources are the standard prefill's.  Columns are packed 16
// per MFMA block -- 16 / g positions x g heads for g <= 16, else one position
// x 16 of its heads -- and each of a workgroup's four waves takes one column
// block (its 16 x 512 float32 accumulators fill most of a wave's registers).
// Per 32-row tile staged in LDS a wave runs 36 score MFMAs, reading the rows
// in their stored fragment order, and 32 PV MFMAs whose V^T operand (8 rows
// of one latent dim per lane) comes from the LDS transpose read.
// ---------------------------------------------------------------------------
typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;
typedef short v4i16 __attribute__((ext_vector_type(4)));

constexpr int kMlaThreads = 256;
constexpr int kMlaKSteps = kMlaDim / 32;                         // 18
constexpr int kMlaTileBytes = kMlaDim * 64;                      // 32 rows of 576 bf16
constexpr int kMlaPieces = kMlaTileBytes / 16 / kMlaThreads;     // staged 16-byte pieces per thread (9)
constexpr int kMlaOBlocks = kMlaLatent / 16;                     // 16-dim row blocks of O^T (32)
constexpr int kMlaScoreBatch = 3;                                // score k-steps whose operands are read together
static_assert(kMlaTileBytes % (16 * kMlaThreads) == 0, "tile staged evenly");

__device__ inline u32x2 tr_read16(const char* p) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                       (__attribute__((address_space(3))) v4i16*)(p)));
}

// Pass 1 for latent rows (one block per (32-token tile, sequence, region)):
// the chunk's rows in chunk order (region 0) and the kept ones in list order
// (region 1) into workspace tiles in the pool's layout; rows past the end
// are 0.
__global__ __launch_bounds__(kThreads) void prefill_tile_mla_kernel(PrefillArgs a) {
  if (load_status(a.status) != 0) return;
  const int k = blockIdx.x, i = blockIdx.y, region = blockIdx.z;
  const int tok0 = a.cu[i], C = a.cu[i + 1] - a.cu[i];
  const int cnt = region ? a.list_cnt[i] : C;
  if (k * 32 >= cnt) return;
  const int32_t* lst = a.list + tok0;
  char* tile = a.tiles + ws_tile(a, region, 0, i, k) * kMlaTileBytes;
  constexpr int kRow = kMlaDim / 8;   // 16-byte pieces per row
  for (int pc = threadIdx.x; pc < 32 * kRow; pc += kThreads) {
    const int j = pc / kRow, e0 = 8 * (pc % kRow);
    const int idx = 32 * k + j;
    u32x4 x = {0u, 0u, 0u, 0u};
    if (idx < cnt) {
      const int c = region ? lst[idx] : idx;
      x = *reinterpret_cast<const u32x4*>(a.k + static_cast<size_t>(tok0 + c) * kMlaDim + e0);
    }
    *reinterpret_cast<u32x4*>(tile + k_elem_off(j, e0)) = x;
  }
}

__global__ __launch_bounds__(kMlaThreads, 1) void prefill_mla_kernel(PrefillArgs a) {
  __shared__ __attribute__((aligned(16))) char tile_lds[2][kMlaTileBytes];
  __shared__ uint32_t meta_lds[2][32];
  __shared__ int masked_lds[2];
  if (load_status(a.status) != 0) return;
  const int i = blockIdx.y;   // sequence of the call (one KV head)
  const int tok0 = a.cu[i], C = a.cu[i + 1] - a.cu[i];
  const int g = a.g;
  const int pcb = g <= kMaxGroup ? kMaxGroup / g : 1;     // positions per column block
  const int cgs = (g + kMaxGroup - 1) / kMaxGroup;        // column blocks per position set
  const int ncb = (C + pcb - 1) / pcb * cgs;
  const int cb0 = blockIdx.x * (kMlaThreads / 64);
  if (cb0 >= ncb) return;
  const int cb1 = min(cb0 + kMlaThreads / 64, ncb) - 1;
  const int s = a.seq_ids[i];
  const int sh = s;
  const int p0 = a.pos[s];
  const int L0 = a.len[sh];
  // the block's positions [t0, t1)
  const int t0 = p0 + (cb0 / cgs) * pcb;
  const int t1 = p0 + min(C, (cb1 / cgs + 1) * pcb);
  // band: chunk tiles from the one holding max(p0, t0 - w + 1) up to t1
  const int band_c0 = (max(0, t0 - a.w + 1 - p0) >> 5) << 5;   // chunk-local, < C
  // kept chunk keys strictly before the band (a prefix of the sorted list),
  // counted by pass 0
  const int32_t* lst = a.list + tok0;
  const int n_pre = a.kept_before[ws_kb(a, 0, i, band_c0 >> 5)];
  const int nc = (L0 + 31) >> 5;
  const int np = (n_pre + 31) >> 5;
  const int nb = (t1 - p0 - band_c0 + 31) >> 5;
  const char* pre_tiles = a.tiles + ws_tile(a, 1, 0, i, 0) * kMlaTileBytes;
  const char* band_tiles = a.tiles + ws_tile(a, 0, 0, i, band_c0 >> 5) * kMlaTileBytes;
  const int ntiles = nc + np + nb;
  const int32_t* pt = a.page_table + static_cast<size_t>(sh) * a.maxp;
  const int32_t* smeta = a.slot_meta + static_cast<size_t>(sh) * a.max_slots;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, G = lane >> 4;
  // ---- this wave's column block and this lane's column (position, head)
  const int cb = cb0 + wave;
  const bool active = cb < ncb;
  const int pbk = cb / cgs, hg = cb % cgs;
  int pl, qh;
  bool ok;
  if (g <= kMaxGroup) {
    pl = r / g;
    qh = r % g;
    ok = pl < pcb;
  } else {
    pl = 0;
    qh = kMaxGroup * hg + r;
    ok = qh < g;
  }
  const int cpos = pbk * pcb + pl;   // chunk-local position
  ok = ok && active && cpos < C;
  const int tcol = ok ? p0 + cpos : -1;
  u32x4 qf[kMlaKSteps];
  {
    const char* qrow = reinterpret_cast<const char*>(
        a.q + (static_cast<size_t>(tok0 + (ok ? cpos : 0)) * g + (ok ? qh : 0)) * kMlaDim);
#pragma unroll
    for (int s2 = 0; s2 < kMlaKSteps; ++s2)
      qf[s2] = ok ? *reinterpret_cast<const u32x4*>(qrow + (32 * s2 + 8 * G) * 2) : u32x4{0u, 0u, 0u, 0u};
  }

  // ---- staging: global -> registers, registers -> LDS (the tile as stored)
  u32x4 kx[kMlaPieces];
  uint32_t smt = kNoKey;
  auto stage_load = [&](int k) {
    const char* tile;
    if (k < nc) {
      const int sb = k * 32;
      tile = a.pool + static_cast<size_t>(pt[sb >> a.log2P]) * a.page_bytes +
             static_cast<size_t>((sb & (a.P - 1)) >> 5) * kMlaTileBytes;
      if (tid < 32) {
        uint32_t mt = sb + tid < L0 ? static_cast<uint32_t>(smeta[sb + tid]) : kNoKey;
        if (a.immediate && mt != kNoKey) {
          const int kp = static_cast<int>(mt & ~kFlagBit);
          const int x = kp + a.w - p0;
          mt = static_cast<uint32_t>(kp) |
               ((x >= 0 && x < C && a.flags[static_cast<size_t>(tok0 + x)]) ? kFlagBit : 0u);
        }
        smt = mt;
      }
    } else if (k < nc + np) {
      const int kk = k - nc;
      tile = pre_tiles + static_cast<size_t>(kk) * kMlaTileBytes;
      if (tid < 32) {
        const int idx = kk * 32 + tid;
        smt = idx < n_pre ? static_cast<uint32_t>(p0 + lst[idx]) : kNoKey;
      }
    } else {
      const int kb = k - nc - np;
      tile = band_tiles + static_cast<size_t>(kb) * kMlaTileBytes;
      if (tid < 32) {
        const int c = band_c0 + kb * 32 + tid;
        smt = c < t1 - p0 ? (static_cast<uint32_t>(p0 + c) | (key_flag(a, tok0, C, c, 0) ? kFlagBit : 0u))
                          : kNoKey;
      }
    }
#pragma unroll
    for (int m = 0; m < kMlaPieces; ++m) kx[m] = *reinterpret_cast<const u32x4*>(tile + (tid + m * kMlaThreads) * 16);
  };
  auto stage_store = [&](int k, int buf) {
    char* dst = tile_lds[buf];
    // pool slots past L hold stale bits (a freed page may hold NaNs): their
    // rows are zeroed, which zeroes them in the V^T operand too
    const int valid = k < nc ? min(32, L0 - k * 32) : 32;
#pragma unroll
    for (int m = 0; m < kMlaPieces; ++m) {
      const int P = tid + m * kMlaThreads;
      // piece P: 1 KB block P / 64 of half (P / 64) % 2, lane row P % 16
      const int pr = P & 15, row = 8 * (pr >> 2) + (pr & 3) + 4 * ((P >> 6) & 1);
      const u32x4 x = row < valid ? kx[m] : u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4*>(dst + P * 16) = x;
    }
    if (tid < 64) {
      // a key row needs the per-element mask iff some query of the block does
      // not see it: padding, causal (position > t0) or flagged and expiring
      // by t1 - 1
      bool need = false;
      if (tid < 32) {
        const uint32_t mt = smt;
        const int kp = static_cast<int>(mt & ~kFlagBit);
        need = mt == kNoKey || kp > t0 || ((mt & kFlagBit) && kp + a.w <= t1 - 1);
        meta_lds[buf][tid] = mt;
      }
      const uint64_t any = __builtin_amdgcn_ballot_w64(need);
      if (tid == 0) masked_lds[buf] = any != 0;
    }
  };

  // ---- accumulators: O^T rows 16 b + 4G .. + 3 of column r
  f32x4 o[kMlaOBlocks];
#pragma unroll
  for (int b = 0; b < kMlaOBlocks; ++b) o[b] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_ref = kMInit, l_run = 0.f;
  const float thr = kRescale / a.scale_log2;   // rescale threshold in score units
  // transpose-read address of this lane in a tile (row block 0, rows 0-3 of
  // each 8): lane 16 G' + 4 j + q reads dims 4q .. 4q + 3 of row 8 G' + j
  const int tr_j = (lane & 15) >> 2, tr_q = lane & 3;
  const int tr_off = (tr_q >> 1) * 256 + (4 * G + tr_j) * 16 + 8 * (tr_q & 1);

  if (ntiles > 0) {
    stage_load(0);
    stage_store(0, 0);
  }
  __syncthreads();
  for (int k = 0; k < ntiles; ++k) {
    const int buf = k & 1;
    if (k + 1 < ntiles) stage_load(k + 1);
    const char* tl = tile_lds[buf];
    if (active) {
      // scores: the 36 A pieces (piece 2s + h: half h, k-step s) read in
      // batches, the next batch in flight while one is multiplied
      f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
      u32x4 kp2[2][2 * kMlaScoreBatch];
      const char* kl = tl + lane * 16;
#pragma unroll
      for (int e = 0; e < 2 * kMlaScoreBatch; ++e) kp2[0][e] = *reinterpret_cast<const u32x4*>(kl + e * 1024);
#pragma unroll
      for (int bt = 0; bt < kMlaKSteps / kMlaScoreBatch; ++bt) {
        if (bt + 1 < kMlaKSteps / kMlaScoreBatch) {
#pragma unroll
          for (int e = 0; e < 2 * kMlaScoreBatch; ++e)
            kp2[(bt + 1) & 1][e] = *reinterpret_cast<const u32x4*>(kl + (2 * kMlaScoreBatch * (bt + 1) + e) * 1024);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int e = 0; e < kMlaScoreBatch; ++e) {
          s0 = mfma_bf16(kp2[bt & 1][2 * e], qf[kMlaScoreBatch * bt + e], s0);
          s1 = mfma_bf16(kp2[bt & 1][2 * e + 1], qf[kMlaScoreBatch * bt + e], s1);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      // lane (r, G): keys 8G .. 8G+3 (s0) and 8G+4 .. 8G+7 (s1) of column r
      float sc[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sc[j] = s0[j];
        sc[j + 4] = s1[j];
      }
      if (__builtin_amdgcn_readfirstlane(masked_lds[buf]) != 0) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const uint32_t km = meta_lds[buf][8 * G + j];
          const int kpos = static_cast<int>(km & ~kFlagBit);
          const int kexp = (km & kFlagBit) ? kpos + a.w : 0x7FFFFFFF;
          sc[j] = (kpos <= tcol && tcol < kexp) ? sc[j] : -INFINITY;
        }
      }
      float mx = fmaxf(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3])),
                       fmaxf(fmaxf(sc[4], sc[5]), fmaxf(sc[6], sc[7])));
      mx = col_max(mx);
      const bool raise = mx > m_ref + thr;   // false while the column has seen no key
      if (__builtin_amdgcn_ballot_w64(raise)) {
        const float m_new = raise ? mx : m_ref;
        const float alpha = __builtin_amdgcn_exp2f((m_ref - m_new) * a.scale_log2);
        l_run *= alpha;
#pragma unroll
        for (int b = 0; b < kMlaOBlocks; ++b) o[b] *= alpha;
        m_ref = m_new;
      }
      const float mb = m_ref * a.scale_log2;
      u32x4 pu;
      const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x2 pr = {__builtin_amdgcn_exp2f(fmaf(sc[2 * j], a.scale_log2, -mb)),
                          __builtin_amdgcn_exp2f(fmaf(sc[2 * j + 1], a.scale_log2, -mb))};
        const bf16x2 pb = __builtin_convertvector(pr, bf16x2);
        pu[j] = __builtin_bit_cast(uint32_t, pb);
        l_run = __builtin_amdgcn_fdot2_f32_bf16(pb, ones, l_run, false);
      }
      // PV: V^T of latent row block b (dims 16 b ..), rows 8G .. 8G+7, from
      // the transpose read; four blocks' reads ahead of their products
#pragma unroll
      for (int b0 = 0; b0 < kMlaOBlocks; b0 += 4) {
        u32x4 vt[4];
#pragma unroll
        for (int i2 = 0; i2 < 4; ++i2) {
          const int b = b0 + i2;
          const char* base = tl + (b >> 1) * 2048 + (b & 1) * 512 + tr_off;
          const u32x2 lo = tr_read16(base), hi = tr_read16(base + 1024);
          vt[i2] = u32x4{lo[0], lo[1], hi[0], hi[1]};
        }
#pragma unroll
        for (int i2 = 0; i2 < 4; ++i2) o[b0 + i2] = mfma_bf16(vt[i2], pu, o[b0 + i2]);
      }
    }
    if (k + 1 < ntiles) stage_store(k + 1, buf ^ 1);
    __syncthreads();
  }

  // ---- outputs
  float l = l_run;
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (tcol >= 0) {
    const float inv = 1.0f / l;
    float* dst = a.out + (static_cast<size_t>(tok0 + cpos) * g + qh) * kMlaLatent + 4 * G;
#pragma unroll
    for (int b = 0; b < kMlaOBlocks; ++b) *reinterpret_cast<f32x4*>(dst + 16 * b) = o[b] * inv;
  }
}

hipError_t launch_prefill_mla(const dms_config& c, const Layout& lo, void* meta, void* ws, void* pool,
                              int layer, int n, const int32_t* seq_ids, const int32_t* cu,
                              int total_tokens, int max_len, const void* q, const void* k,
                              const uint8_t* flags, float* out, hipStream_t st, hipEvent_t ev_start,
                              hipEvent_t ev_stop) {
  char* w = static_cast<char*>(ws);
  LayerState ls = layer_state(lo, meta, layer);
  PrefillArgs a;
  a.status = reinterpret_cast<const int32_t*>(static_cast<char*>(meta) + lo.status);
  a.status_w = reinterpret_cast<int32_t*>(static_cast<char*>(meta) + lo.status);
  a.seq_ids = seq_ids;
  a.cu = cu;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = nullptr;
  a.flags = flags;
  a.pool = static_cast<const char*>(pool);
  a.page_table = ls.page_table;
  a.slot_meta = ls.slot_meta;
  a.len = ls.len;
  a.pos = ls.pos;
  a.list = reinterpret_cast<int32_t*>(w + lo.ws_pf_meta);
  a.list_cnt = reinterpret_cast<int32_t*>(w + lo.ws_pf_cum);
  a.tiles = w + lo.ws_pf_tiles;
  a.tmeta = reinterpret_cast<uint32_t*>(w + lo.ws_pf_tmeta);
  a.kept_before = reinterpret_cast<int32_t*>(w + lo.ws_pf_kb);
  a.order = nullptr;
  a.work_ctr = nullptr;
  a.nx = a.items = 0;
  a.tph = lo.pf_tiles_per_head;
  a.immediate = c.eviction == DMS_EVICT_IMMEDIATE;
  a.zero_neuron = 0;
  a.out = out;
  a.page_bytes = lo.page_bytes;
  a.n = n;
  a.H = 1;
  a.g = c.group_size;
  a.w = c.window;
  a.P = c.page_size;
  a.log2P = __builtin_ctz(static_cast<unsigned>(c.page_size));
  a.maxp = c.max_pages_per_head;
  a.max_slots = lo.max_slots;
  a.max_seqs = c.max_seqs;
  a.total = total_tokens;
  a.max_len = max_len;
  a.PB = 0;
  a.scale_log2 = c.softmax_scale * 1.4426950408889634f;
  // the timing events bracket every pass
  if (ev_start) (void)hipEventRecord(ev_start, st);
  hipLaunchKernelGGL(prefill_list_kernel, dim3(n), dim3(kThreads), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(prefill_tile_mla_kernel, dim3((max_len + 31) / 32, n, 2), dim3(kThreads), 0, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int g = c.group_size;
  const int pcb = g <= kMaxGroup ? kMaxGroup / g : 1;
  const int cgs = (g + kMaxGroup - 1) / kMaxGroup;
  const int ncb = (max_len + pcb - 1) / pcb * cgs;
  const int per_block = kMlaThreads / 64;
  hipLaunchKernelGGL(prefill_mla_kernel, dim3((ncb + per_block - 1) / per_block, n), dim3(kMlaThreads), 0, st, a);
  e = hipGetLastError();
  if (ev_stop) (void)hipEventRecord(ev_stop, st);
  return e;
}

}  // namespace

hipError_t launch_prefill_decide(const dms_config& c, const void* q, int total_tokens,
                                 uint8_t* flags, hipStream_t st) {
  const int64_t n = static_cast<int64_t>(total_tokens) * c.num_kv_heads;
  const int blocks = static_cast<int>((n + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(prefill_decide_kernel, dim3(blocks), dim3(kThreads), 0, st,
                     static_cast<const uint16_t*>(q), flags, total_tokens, c.num_kv_heads,
                     c.group_size, c.head_dim, c.decision_bias);
  return hipGetLastError();
}

hipError_t launch_prefill_attention(const dms_config& c, const Layout& lo, void* meta, void* ws,
                                    void* pool, int layer, int n, const int32_t* seq_ids,
                                    const int32_t* cu, int total_tokens, int max_len,
                                    const void* q, const void* k, const void* v,
                                    const uint8_t* flags, float* out, hipStream_t st,
                                    hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (c.kv_format == DMS_KV_MLA)
    return launch_prefill_mla(c, lo, meta, ws, pool, layer, n, seq_ids, cu, total_tokens, max_len, q, k, flags,
                              out, st, ev_start, ev_stop);
  const bool fp8 = c.kv_format == DMS_KV_FP8;
  if (c.head_dim == 128)
    return fp8 ? launch_prefill_d<128, true>(c, lo, meta, ws, pool, layer, n, seq_ids, cu, total_tokens,
                                             max_len, q, k, v, flags, out, st, ev_start, ev_stop)
               : launch_prefill_d<128, false>(c, lo, meta, ws, pool, layer, n, seq_ids, cu, total_tokens,
                                              max_len, q, k, v, flags, out, st, ev_start, ev_stop);
  return fp8 ? launch_prefill_d<64, true>(c, lo, meta, ws, pool, layer, n, seq_ids, cu, total_tokens,
                                          max_len, q, k, v, flags, out, st, ev_start, ev_stop)
             : launch_prefill_d<64, false>(c, lo, meta, ws, pool, layer, n, seq_ids, cu, total_tokens,
                                           max_len, q, k, v, flags, out, st, ev_start, ev_stop);
}

}  // namespace dms
