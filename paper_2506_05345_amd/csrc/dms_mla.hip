// DMS decode over a multi-head latent attention (MLA) cache, gfx950.
//
// The paper names MLA (DeepSeek-V2) as a direction for DMS (Sec. 6) without
// a scheme.  Reading taken here: an MLA layer caches, per token, one row
// shared by all query heads -- the compressed latent c_t (512 dims) followed
// by the decoupled rotary key (64 dims) -- so it is one KV head with
// g = all query heads.  DMS gives that row one decision per token and evicts
// it by the same delayed rule (Sec. 3.1), so the bookkeeping (planner, slots,
// pages, chunk commit) is the standard path's with Hkv = 1.  Decode works in
// the absorbed form: with the query already multiplied into the latent space
// (q~ = W_UK^T q_nope, 512 dims) and its rotary part (64 dims), a head scores
// a row by q . row over all 576 dims and its output is the softmax-weighted
// sum of the rows' first 512 dims (the latent; W_UV is applied by the caller).
//
// Work split: the planner's units are tile ranges (one per CU), each an
// equal contiguous share of the call's 32-row tiles.  A block of eight waves
// takes one unit and up to 64 query heads (four groups of 16; DeepSeek-V2's
// 128 heads are two blocks per unit, dispatched to one XCD together so that
// the second reads the unit's rows mostly from that XCD's L2).  Per tile:
//  * the block copies the tile (36 KB, 36 one-KB wave loads) straight into
//    one of four LDS buffers with global->LDS loads, three tiles ahead of the
//    one being computed;
//  * wave i < groups scores the tile for its 16 heads: the rows are stored in
//    the fragment order of the 16x16x32 score MFMA (A operand: 16 rows, 32
//    dims; two halves of 16 rows), so its A operands are 1 KB contiguous LDS
//    reads; it keeps the group's running maximum and sum and leaves the
//    tile's probabilities (bf16) and the rescale factor in LDS;
//  * every wave then multiplies the probabilities of all the block's groups
//    into its own 64 latent dims (O^T = V^T P, 16 output dims x 16 heads per
//    MFMA).  The V^T operand (8 consecutive rows of one dim per lane) is the
//    transpose of how rows are stored; the LDS transpose read of gfx950
//    (ds_read_b64_tr_b16) forms it straight from the tile, reading 512
//    contiguous bytes per instruction.
// At a segment end (the unit's part of one head) each wave writes its 64
// dims of every head of the block: the head's output when the unit covered
// the whole head, else one partial per (unit, head); the block that
// completes a split head's tile count merges its partials in unit order.
#include "dms_common.h"

namespace dms {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;
typedef short v4i16 __attribute__((ext_vector_type(4)));
#define DMS_LDS __attribute__((address_space(3)))

constexpr int kWaves = 8;                    // waves per block
constexpr int kScorers = 4;                  // waves 0-3 score (one group each), 4-7 multiply by V
constexpr int kBlockGroups = kScorers;       // query-head groups of kMaxGroup per block
constexpr int kBlockHeads = kBlockGroups * kMaxGroup;
constexpr int kPvWaves = kWaves - kScorers;
constexpr int kNBuf = 4;                     // LDS tile buffers
constexpr int kD = kMlaDim;                  // row: latent + rotary key
constexpr int kDv = kMlaLatent;              // latent (value) dims
constexpr int kKBlocks = kD / 32;            // 32-dim k-steps of the score MFMA (18)
constexpr int kTileBytes = kD * 64;          // 32 rows of 576 bf16
constexpr int kTileLoads = kTileBytes / 1024;            // 1-KB wave loads per tile (36)
constexpr int kLoadsPerWave = kTileLoads / kPvWaves;     // issued by each V wave (9)
constexpr int kPvBlocks = kDv / 16 / kPvWaves;           // 16-dim row blocks per V wave (8)
constexpr float kRescale = 8.0f;             // lazy rescale threshold, log2 units
constexpr int kMergeBatch = 2;               // partials a merge loads together
constexpr int kScoreBatch = 3;               // k-steps of score operands read from LDS together
// Workgroups per dispatch batch: a multiple of the eight XCDs, so that the
// blocks of one unit (one per 64 query heads) share an XCD (workgroup i runs
// on XCD i % 8) and read the unit's tiles close together in time.
constexpr int kUnitBatch = 32;

static_assert(kTileLoads % kPvWaves == 0, "tile loads split evenly over the V waves");
static_assert(kDv % (16 * kPvWaves) == 0, "latent dims split evenly over the V waves");
static_assert(kKBlocks % kScoreBatch == 0, "score k-steps split evenly into batches");
static_assert(2 * kLoadsPerWave < 64, "s_waitcnt vmcnt range");

__device__ inline int load_status(const int32_t* status) {
  return __atomic_load_n(status, __ATOMIC_RELAXED);
}
__device__ inline int ldc(const int32_t* p, size_t i) {
  typedef const int32_t __attribute__((address_space(4))) CT;
  return ((CT*)p)[i];
}
__device__ inline int4 ldc(const int4* p, size_t i) {
  typedef int __attribute__((ext_vector_type(4))) i32x4;
  typedef const i32x4 __attribute__((address_space(4))) CT;
  const i32x4 v = ((CT*)p)[i];
  return make_int4(v[0], v[1], v[2], v[3]);
}
// A wave-uniform pointer taken into scalar registers: a table read through it
// is a scalar load.
template <typename T>
__device__ inline const T* uniform_ptr(const T* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
  return reinterpret_cast<const T*>((static_cast<uint64_t>(hi) << 32) | lo);
}
__device__ inline f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ inline void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline float load_coherent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// s_waitcnt immediates (expcnt and lgkmcnt left free)
constexpr int wait_vm(int n) { return 0x0F70 | (n & 15) | ((n >> 4) << 14); }
constexpr int kBufferDword3 = 0x00020000;
constexpr int kCachePolicySc1 = 0x10;     // coherent at the device level (past the die's L2)

struct MlaParams {
  size_t page_bytes;
  int part_acc_bytes;   // size of the partial accumulator area (< 2 GiB)
  int g, maxp, log2P;
  int W;                // the planner's units (tile ranges)
  int nblk;             // blocks per unit: ceil(g / 64)
  int head_groups;      // arrival counters per call head
  int ml_stride;        // (max, sum) pairs per partial
  float scale_log2;
};

struct MlaPtrs {
  const int32_t* status;
  const HeadDesc* desc;
  const int32_t* cum_tiles;
  const int32_t* wave_bounds;
  const int4* wave_desc;
  const int4* head_waves;
  int32_t* head_cnt;
  const int32_t* page_table;
  char* pool;
  const uint16_t* q;
  const uint16_t* k_in;
  float2* part_ml;
  float* part_acc;
  float* out;
};

struct Smem {
  char tile[kNBuf][kTileBytes];             // tiles as stored (score fragment order)
  u32x4 p[kBlockGroups][64];                // bf16 probabilities, PV B operand order
  float alpha[kBlockGroups][kMaxGroup];     // rescale of a group's accumulators
  float2 ml[kBlockGroups][kMaxGroup];       // (max, sum) at a segment end
  int4 raise4;                              // per group: its maximum rose (rescale)
  int last;
};

// A V wave's share of one tile copy: wave loads v, v + 4, ... of 1 KB, each
// lane's 16 bytes landing at the same offset in LDS (M0 = the LDS address of
// the wave's KB).  Written as assembly so that the compiler does not order
// every later LDS read behind these loads (its wait inserter cannot tell the
// four buffers apart and would drain the copies of the tiles ahead); the
// kernel waits for them itself (wait_tile + barrier).  Nothing else in this
// kernel uses M0.
__device__ inline void tile_to_lds(const char* src, char* dst, int v, int lane, bool stream) {
  const uint32_t lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((DMS_LDS char*)dst));
  const char* g = src + lane * 16;
#pragma unroll
  for (int k = 0; k < kLoadsPerWave; ++k) {
    const int p = v + kPvWaves * k;
    const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds + p * 1024);
    if (stream)
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off nt" : : "s"(m0), "v"(g + p * 1024) : "memory", "m0");
    else
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" : : "s"(m0), "v"(g + p * 1024) : "memory", "m0");
  }
}

// Wait until this V wave's loads of the tile about to be computed have
// landed, `ahead` later tiles (0 .. 2) still in flight behind them.
__device__ inline void wait_tile(int ahead) {
  if (ahead >= 2) __builtin_amdgcn_s_waitcnt(wait_vm(2 * kLoadsPerWave));
  else if (ahead == 1) __builtin_amdgcn_s_waitcnt(wait_vm(kLoadsPerWave));
  else __builtin_amdgcn_s_waitcnt(wait_vm(0));
}

__device__ inline u32x2 tr_read(const char* p) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((DMS_LDS v4i16*)(p)));
}

// One role of the block's waves over the unit's segments (the part of one
// head in the unit's tile range).  Both roles pass the same barriers in the
// same order; their register sets (query fragments and score operands of a
// scorer, accumulators of a V wave) are live in different code.
template <bool kScore>
__device__ __forceinline__ void run_role(Smem& S, const MlaPtrs& P, const MlaParams& a, int unit, int blk,
                                         int wid, int lane) {
  const int h0 = blk * kBlockHeads;                              // first query head of the block
  const int nh = min(kBlockHeads, a.g - h0);                     // its query heads
  const int ngrp = (nh + kMaxGroup - 1) / kMaxGroup;             // its groups of 16
  const int r = lane & 15, G = lane >> 4;
  const int4 wd0 = ldc(P.wave_desc, 2 * unit), wd1 = ldc(P.wave_desc, 2 * unit + 1);
  int tb = ldc(P.wave_bounds, unit);
  const int te = ldc(P.wave_bounds, unit + 1);
  const int tpp_log2 = a.log2P - 5;
  const int tpp_mask = (1 << tpp_log2) - 1;
  // scorer: its group; V wave: its index (latent dims 128 v ..)
  const int sg = wid;
  const bool active = kScore && sg < ngrp;
  const int gq = active ? min(kMaxGroup, nh - kMaxGroup * sg) : 1;
  const int qr = min(r, gq - 1);
  const int v = wid - kScorers;
  // transpose-read address of this lane in a tile (row block 0, rows 0-3 of
  // each 8): lane 16 G' + 4 j + q reads dims 4q .. 4q + 3 of row 8 G' + j
  const int tr_j = (lane & 15) >> 2, tr_q = lane & 3;
  const int tr_off = (tr_q >> 1) * 256 + (4 * G + tr_j) * 16 + 8 * (tr_q & 1);
  const __amdgpu_buffer_rsrc_t acc_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      P.part_acc, static_cast<short>(0), a.part_acc_bytes, kBufferDword3);
  int hh = wd0.z;
  bool first = true;
  while (tb < te) {
    int c0, c1;
    HeadDesc d;
    if (first) {
      c0 = wd0.w;
      c1 = wd1.x;
      d = make_int4(wd1.y, wd1.z, wd1.w, 0);
      first = false;
    } else {
      while (ldc(P.cum_tiles, hh + 1) <= tb) ++hh;
      c0 = ldc(P.cum_tiles, hh);
      c1 = ldc(P.cum_tiles, hh + 1);
      d = ldc(P.desc, hh);
    }
    const int seg_end = min(te, c1);
    const int L = d.x;
    const int32_t* pt = P.page_table + static_cast<size_t>(d.y) * a.maxp;
    auto tile_of = [&](int t) -> const char* {
      return P.pool + static_cast<size_t>(ldc(uniform_ptr(pt), t >> tpp_log2)) * a.page_bytes +
             static_cast<size_t>(t & tpp_mask) * kTileBytes;
    };
    const int t_lo = tb - c0;
    const int n = seg_end - tb;       // the segment's tiles
    const bool whole = tb == c0 && seg_end == c1;
    const size_t pid = static_cast<size_t>(unit) + hh;
    // the token this call appends (slot d.z), if it falls in the segment:
    // the first V wave holds its row (72 pieces of 16 bytes) and patches the
    // tile in LDS
    const int tz = d.z >> 5;
    const bool has_tok = P.k_in != nullptr && tz >= t_lo && tz < t_lo + n;
    const bool tok_wave = !kScore && v == 0;
    uint4 tok0 = make_uint4(0u, 0u, 0u, 0u), tok1 = make_uint4(0u, 0u, 0u, 0u);
    // scorer: query fragments of its group (B operand: column r = head r)
    u32x4 qf[kScore ? kKBlocks : 1];
    float m = -INFINITY, l = 0.f;     // scorer: the group's running max / sum (per lane)
    // V wave: O^T accumulators of its 128 dims for every group of the block
    f32x4 acc[kScore ? 1 : kBlockGroups][kScore ? 1 : kPvBlocks];
    if constexpr (kScore) {
      if (active) {
        const char* qrow = reinterpret_cast<const char*>(
            P.q + (static_cast<size_t>(hh) * a.g + h0 + kMaxGroup * sg + qr) * kD);
#pragma unroll
        for (int s = 0; s < kKBlocks; ++s) {
          const u32x4 x = *reinterpret_cast<const u32x4*>(qrow + (32 * s + 8 * G) * 2);
          qf[s] = r < gq ? x : u32x4{0u, 0u, 0u, 0u};
        }
      }
    } else {
      if (has_tok && tok_wave) {
        const uint4* src = reinterpret_cast<const uint4*>(P.k_in + static_cast<size_t>(hh) * kD);
        tok0 = src[lane];
        if (lane < kD / 8 - 64) tok1 = src[64 + lane];
      }
      // the first tiles of the segment in flight
      for (int i = 0; i < min(kNBuf - 1, n); ++i) tile_to_lds(tile_of(t_lo + i), S.tile[i], v, lane, blk == a.nblk - 1);
#pragma unroll
      for (int gi = 0; gi < kBlockGroups; ++gi)
#pragma unroll
        for (int b = 0; b < kPvBlocks; ++b) acc[gi][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    for (int i = 0; i < n; ++i) {
      const int t = t_lo + i;
      const char* tl = S.tile[i & (kNBuf - 1)];
      // i == 0: the token row was loaded before the tiles
      if constexpr (!kScore) wait_tile(i == 0 ? 0 : min(kNBuf - 2, n - 1 - i));
      __syncthreads();   // tile i is in LDS; every wave is done with tile i - 1
      if constexpr (!kScore) {
        if (i + kNBuf - 1 < n)
          tile_to_lds(tile_of(t + kNBuf - 1), S.tile[(i + kNBuf - 1) & (kNBuf - 1)], v, lane, blk == a.nblk - 1);
      }
      if (has_tok && t == tz) {
        if (tok_wave) {
          char* tw = S.tile[i & (kNBuf - 1)];
          const int j = d.z & 31;
          *reinterpret_cast<uint4*>(tw + k_elem_off(j, 8 * lane)) = tok0;
          if (lane < kD / 8 - 64) *reinterpret_cast<uint4*>(tw + k_elem_off(j, 8 * (64 + lane))) = tok1;
        }
        __syncthreads();
      }
      // rows at or past L are stale in the head's last tile
      const int valid = (i == n - 1 && seg_end == c1) ? L - t * kTile : kTile;
      if constexpr (kScore) {
        if (active) {
          // the tile's 36 A pieces (1 KB each, piece 2s + h: half h, k-step
          // s) read from LDS in batches of kScoreBatch k-steps, the next
          // batch's reads in flight while the current one is multiplied
          f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
          u32x4 kp[2][2 * kScoreBatch];
          const char* kl = tl + lane * 16;
#pragma unroll
          for (int e = 0; e < 2 * kScoreBatch; ++e) kp[0][e] = *reinterpret_cast<const u32x4*>(kl + e * 1024);
#pragma unroll
          for (int bt = 0; bt < kKBlocks / kScoreBatch; ++bt) {
            if (bt + 1 < kKBlocks / kScoreBatch) {
#pragma unroll
              for (int e = 0; e < 2 * kScoreBatch; ++e)
                kp[(bt + 1) & 1][e] = *reinterpret_cast<const u32x4*>(kl + (2 * kScoreBatch * (bt + 1) + e) * 1024);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int e = 0; e < kScoreBatch; ++e) {
              sa = mfma_bf16(kp[bt & 1][2 * e], qf[kScoreBatch * bt + e], sa);
              sb = mfma_bf16(kp[bt & 1][2 * e + 1], qf[kScoreBatch * bt + e], sb);
            }
            __builtin_amdgcn_sched_barrier(0);
          }
          // lane (r, G): scores of rows 8G .. 8G+3 (sa) and 8G+4 .. 8G+7 (sb), head r
          float sc[8];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            sc[e] = sa[e] * a.scale_log2;
            sc[4 + e] = sb[e] * a.scale_log2;
          }
          const int nv = valid - 8 * G;
#pragma unroll
          for (int e = 0; e < 8; ++e) sc[e] = e < nv ? sc[e] : -INFINITY;
          float mx = fmaxf(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3])),
                           fmaxf(fmaxf(sc[4], sc[5]), fmaxf(sc[6], sc[7])));
          mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
          mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
          const bool up = mx > m + kRescale;
          const bool any = __builtin_amdgcn_ballot_w64(up) != 0;
          float alpha = 1.0f;
          if (any) {
            const float m_new = up ? mx : m;
            alpha = __builtin_amdgcn_exp2f(m - m_new);   // 0 from m = -inf
            l *= alpha;
            m = m_new;
          }
          bf16x8 pr;
          float psum = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const __bf16 pb = static_cast<__bf16>(__builtin_amdgcn_exp2f(sc[e] - m));
            pr[e] = pb;
            psum += static_cast<float>(pb);
          }
          l += psum;
          S.p[sg][lane] = __builtin_bit_cast(u32x4, pr);
          if (G == 0) S.alpha[sg][r] = alpha;
          if (lane == 0) reinterpret_cast<int*>(&S.raise4)[sg] = any;
        }
      }
      __syncthreads();   // probabilities and rescale factors of every group
      if constexpr (!kScore) {
        // V^T operands of this wave's row blocks (latent dims 128 v + 16 b ..),
        // rows 8G .. 8G+7 per lane, straight from the tile
        u32x4 vt[kPvBlocks];
#pragma unroll
        for (int b = 0; b < kPvBlocks; ++b) {
          const int rb = kPvBlocks * v + b;
          const char* base = tl + (rb >> 1) * 2048 + (rb & 1) * 512 + tr_off;
          const u32x2 lo = tr_read(base), hi = tr_read(base + 1024);
          vt[b] = u32x4{lo[0], lo[1], hi[0], hi[1]};
        }
        // every group's probabilities, rescale flag and factor
        const int4 up4 = S.raise4;
        const int upg[kBlockGroups] = {up4.x, up4.y, up4.z, up4.w};
        u32x4 pb[kBlockGroups];
        float al[kBlockGroups];
#pragma unroll
        for (int gi = 0; gi < kBlockGroups; ++gi) {
          pb[gi] = S.p[gi][lane];
          al[gi] = S.alpha[gi][r];
        }
        if (valid < kTile) {
          // stale rows of a freed page may hold any bits: zero them in V
          const int nv = valid - 8 * G;
#pragma unroll
          for (int b = 0; b < kPvBlocks; ++b)
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              const uint32_t keep = (2 * w < nv ? 0x0000FFFFu : 0u) | (2 * w + 1 < nv ? 0xFFFF0000u : 0u);
              vt[b][w] &= keep;
            }
        }
#pragma unroll
        for (int gi = 0; gi < kBlockGroups; ++gi) {
          if (gi < ngrp) {
            if (upg[gi]) {
#pragma unroll
              for (int b = 0; b < kPvBlocks; ++b) acc[gi][b] *= al[gi];
            }
#pragma unroll
            for (int b = 0; b < kPvBlocks; ++b) acc[gi][b] = mfma_bf16(vt[b], pb[gi], acc[gi][b]);
          }
        }
      }
    }
    // segment end: the scorers' (max, sum) for the V waves
    if constexpr (kScore) {
      if (active) {
        l += __shfl_xor(l, 16, 64);
        l += __shfl_xor(l, 32, 64);
        if (G == 0) S.ml[sg][r] = make_float2(m, l);
      }
    }
    __syncthreads();
    if constexpr (!kScore) {
      if (has_tok && tok_wave && blk == 0) {
        // the appended token's row into the pool (the tile in LDS was patched)
        char* tile = const_cast<char*>(tile_of(tz));
        const int j = d.z & 31;
        *reinterpret_cast<uint4*>(tile + k_elem_off(j, 8 * lane)) = tok0;
        if (lane < kD / 8 - 64) *reinterpret_cast<uint4*>(tile + k_elem_off(j, 8 * (64 + lane))) = tok1;
      }
#pragma unroll
      for (int gi = 0; gi < kBlockGroups; ++gi) {
        const int head = kMaxGroup * gi + r;     // within the block
        if (gi < ngrp && head < nh) {
          const float2 ml = S.ml[gi][r];
          if (whole) {
            const float inv = 1.0f / ml.y;
            float* o = P.out + (static_cast<size_t>(hh) * a.g + h0 + head) * kDv + 128 * v + 4 * G;
#pragma unroll
            for (int b = 0; b < kPvBlocks; ++b) *reinterpret_cast<f32x4*>(o + 16 * b) = acc[gi][b] * inv;
          } else {
            // the unit's partial, with stores that are complete at the
            // device's coherence point once this wave's vmcnt drains
            if (v == 0 && G == 0) {
              float* pm = reinterpret_cast<float*>(P.part_ml + pid * a.ml_stride + h0 + head);
              store_coherent(pm, ml.x);
              store_coherent(pm + 1, ml.y);
            }
            const uint32_t o = static_cast<uint32_t>(((pid * a.g + h0 + head) * kDv + 128 * v + 4 * G) * 4);
#pragma unroll
            for (int b = 0; b < kPvBlocks; ++b)
              __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[gi][b]), acc_rsrc, o + 64 * b, 0,
                                                     kCachePolicySc1);
          }
        }
      }
      __builtin_amdgcn_s_waitcnt(wait_vm(0));
    }
    if (!whole) {
      // Split head: once the V waves' partials are stored, add the unit's
      // tiles to the head's arrival counter (one per block of 64 heads); the
      // block that completes the count merges the head's partials, each V
      // wave its 128 dims of every head of the block, and resets the counter.
      __syncthreads();
      if (wid == 0 && lane == 0) {
        const int prev = atomicAdd(&P.head_cnt[hh * a.head_groups + blk], seg_end - tb);
        S.last = prev + (seg_end - tb) == c1 - c0;
      }
      __syncthreads();
      if (S.last) {
        if constexpr (!kScore) {
          const int4 hw = ldc(P.head_waves, hh);
          for (int gi = 0; gi < ngrp; ++gi) {
            const int head = kMaxGroup * gi + min(r, nh - kMaxGroup * gi - 1);
            float Mh = -INFINITY, dh = 0.f;
            f32x4 nacc[kPvBlocks];
#pragma unroll
            for (int b = 0; b < kPvBlocks; ++b) nacc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
            for (int u0 = hw.x; u0 <= hw.y; u0 += kMergeBatch) {
              bool lv[kMergeBatch];
              float mv[kMergeBatch], sv[kMergeBatch];
              u32x4 x[kMergeBatch][kPvBlocks];
#pragma unroll
              for (int j = 0; j < kMergeBatch; ++j) {
                const int u = u0 + j;
                lv[j] = u <= hw.y && ldc(P.wave_bounds, u) < ldc(P.wave_bounds, u + 1);
                const size_t pj = static_cast<size_t>(lv[j] ? u : hw.x) + hh;
                const float* pm = reinterpret_cast<const float*>(P.part_ml + pj * a.ml_stride + h0 + head);
                mv[j] = lv[j] ? load_coherent(pm) : -INFINITY;
                sv[j] = lv[j] ? load_coherent(pm + 1) : 0.f;
                const uint32_t o = static_cast<uint32_t>(((pj * a.g + h0 + head) * kDv + 128 * v + 4 * G) * 4);
#pragma unroll
                for (int b = 0; b < kPvBlocks; ++b)
                  x[j][b] = lv[j] ? __builtin_amdgcn_raw_buffer_load_b128(acc_rsrc, o + 64 * b, 0, kCachePolicySc1)
                                  : u32x4{0u, 0u, 0u, 0u};
              }
              float bm = mv[0];
#pragma unroll
              for (int j = 1; j < kMergeBatch; ++j) bm = fmaxf(bm, mv[j]);
              if (bm > Mh) {   // the first batch always raises Mh from -inf (its sums are 0)
                const float sc = __builtin_amdgcn_exp2f(Mh - bm);
                dh *= sc;
#pragma unroll
                for (int b = 0; b < kPvBlocks; ++b) nacc[b] *= sc;
                Mh = bm;
              }
#pragma unroll
              for (int j = 0; j < kMergeBatch; ++j) {
                const float wt = lv[j] ? __builtin_amdgcn_exp2f(mv[j] - Mh) : 0.f;
                dh += wt * sv[j];
#pragma unroll
                for (int b = 0; b < kPvBlocks; ++b) nacc[b] += wt * __builtin_bit_cast(f32x4, x[j][b]);
              }
            }
            if (kMaxGroup * gi + r < nh) {
              const float inv = 1.0f / dh;
              float* o = P.out + (static_cast<size_t>(hh) * a.g + h0 + kMaxGroup * gi + r) * kDv + 128 * v + 4 * G;
#pragma unroll
              for (int b = 0; b < kPvBlocks; ++b) *reinterpret_cast<f32x4*>(o + 16 * b) = nacc[b] * inv;
            }
          }
        } else if (wid == 0 && lane == 0) {
          __hip_atomic_store(&P.head_cnt[hh * a.head_groups + blk], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    }
    __syncthreads();   // LDS (max, sum) and buffers are free for the next segment
    tb = seg_end;
    ++hh;
  }
}

__global__ __launch_bounds__(kWaves * 64, 1) void decode_mla_kernel(MlaPtrs P, MlaParams a) {
  __shared__ __attribute__((aligned(16))) Smem S;
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // the planner's unit (this block's tile range) and the block's 64 heads
  const int per = kUnitBatch * a.nblk;
  const int unit = static_cast<int>(blockIdx.x) / per * kUnitBatch + static_cast<int>(blockIdx.x) % kUnitBatch;
  const int blk = static_cast<int>(blockIdx.x) % per / kUnitBatch;
  if (unit >= a.W) return;
  if (load_status(P.status) != 0) return;
  if (ldc(P.wave_bounds, unit) >= ldc(P.wave_bounds, unit + 1)) return;
  if (wid < kScorers) run_role<true>(S, P, a, unit, blk, wid, lane);
  else run_role<false>(S, P, a, unit, blk, wid, lane);
}

}  // namespace

hipError_t launch_decode_mla(const dms_config& c, const Layout& lo, void* meta, void* ws,
                             void* pool, int layer, int n, const void* q, const void* k,
                             float* out, int waves, hipStream_t st, hipEvent_t ev_start,
                             hipEvent_t ev_stop) {
  (void)n;   // the call's heads are those the planner laid out for the units
  char* w = static_cast<char*>(ws);
  MlaParams a;
  a.page_bytes = lo.page_bytes;
  a.part_acc_bytes = static_cast<int>(static_cast<size_t>(lo.max_partials) * c.group_size * kDv * 4);
  a.g = c.group_size;
  a.maxp = c.max_pages_per_head;
  a.log2P = __builtin_ctz(static_cast<unsigned>(c.page_size));
  a.W = waves;
  a.nblk = (c.group_size + kBlockHeads - 1) / kBlockHeads;
  a.head_groups = lo.head_groups;
  a.ml_stride = lo.ml_stride;
  a.scale_log2 = c.softmax_scale * 1.4426950408889634f;
  if (a.nblk > a.head_groups) return hipErrorInvalidValue;
  const int blocks = (waves + kUnitBatch - 1) / kUnitBatch * kUnitBatch * a.nblk;
  if (ev_start) (void)hipEventRecord(ev_start, st);
  MlaPtrs P;
  P.status = reinterpret_cast<const int32_t*>(static_cast<char*>(meta) + lo.status);
  P.desc = reinterpret_cast<const HeadDesc*>(w + lo.ws_head_desc);
  P.cum_tiles = reinterpret_cast<const int32_t*>(w + lo.ws_cum_tiles);
  P.wave_bounds = reinterpret_cast<const int32_t*>(w + lo.ws_wave_bounds);
  P.wave_desc = reinterpret_cast<const int4*>(w + lo.ws_wave_desc);
  P.head_waves = reinterpret_cast<const int4*>(w + lo.ws_head_waves);
  P.head_cnt = reinterpret_cast<int32_t*>(w + lo.ws_head_cnt);
  P.page_table = layer_state(lo, meta, layer).page_table;
  P.pool = static_cast<char*>(pool);
  P.q = static_cast<const uint16_t*>(q);
  P.k_in = static_cast<const uint16_t*>(k);
  P.part_ml = reinterpret_cast<float2*>(w + lo.ws_part_ml);
  P.part_acc = reinterpret_cast<float*>(w + lo.ws_part_acc);
  P.out = out;
  hipLaunchKernelGGL(decode_mla_kernel, dim3(blocks), dim3(kWaves * 64), 0, st, P, a);
  hipError_t e = hipGetLastError();
  if (ev_stop) (void)hipEventRecord(ev_stop, st);
  return e;
}

int decode_mla_resident_waves(const dms_config& c) {
  int dev = 0, cus = 0, blocks = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, decode_mla_kernel, kWaves * 64, 0) != hipSuccess ||
      blocks < 1)
    return -1;
  // the planner's units: tile ranges taken by one block per 64 query heads,
  // as many as fit on the CUs at once (one block per CU).  Fewer, longer
  // units for wide groups split fewer heads: each split costs a partial of
  // g x 512 float32 written and read back (256 KB at 128 heads).
  const int nblk = (c.group_size + kBlockHeads - 1) / kBlockHeads;
  const int units = (cus < kMaxMlaUnits ? cus : kMaxMlaUnits) / nblk;
  return units > 0 ? units : 1;
}

}  // namespace dms
