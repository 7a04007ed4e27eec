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
// Work split: the planner's units are tile ranges (one per CU), each taking
// an equal contiguous share of the call's tiles.  A query group wider than 16
// heads (DeepSeek-V2: 128) is attended as groups of 16, one block per (unit,
// head group): every group's block reads the unit's tiles, and the blocks of
// one unit are dispatched to the same XCD close together so that the later
// readers mostly hit that XCD's L2.  A block deals each segment's
// tiles (the part of one head in its share) to its four waves in turn, and at
// the segment's end the four fold their partials through LDS -- into the
// head's output when the block covered the whole head, else into one partial
// per (block, head), a few per head.  The block that completes a split
// head's tile count merges its partials (each wave folding a quarter of the
// dims, partials loaded in batches), as the standard kernel's last arriving
// wave does; with one partial per wave (16 heads x 512 float32 each, 16x the
// standard kernel's) that lone merge was a latency-bound tail, and a separate
// combine launch cost more than folding in LDS first.  Per 32-slot tile:
//  * keys: the row is stored in the fragment order of the 16x16x32 score
//    MFMA (A operand: tile rows, k = 32 dims); the tile is read in two halves
//    of 16 rows, half h holding slots 8(r/4) + r%4 + 4h, with the next half's
//    loads always in flight while the current one is computed;
//  * values: the 16x16x32 PV MFMA needs, per lane, 8 consecutive slots of one
//    latent dim -- the transpose of how the rows arrive.  Each wave writes the
//    latent part of its tile to its own LDS area as [dim][slot] (2-byte
//    stores) and reads the V^T operands back as 16-byte pieces;
//  * the two score halves of a lane hold slots 8G .. 8G+3 and 8G+4 .. 8G+7,
//    exactly the k slice of the PV B operand, so probabilities stay in
//    registers (as in the standard kernel).
#include "dms_common.h"

namespace dms {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;

constexpr int kWavesPerBlock = 4;
constexpr int kD = kMlaDim;             // row: latent + rotary key
constexpr int kDv = kMlaLatent;         // latent (value) dims
constexpr int kKBlocks = kD / 32;       // 32-dim k-steps of the score MFMA (18)
constexpr int kLBlocks = kDv / 32;      // of them latent (16)
constexpr int kOBlocks = kDv / 16;      // 16-dim row blocks of O^T (32)
constexpr int kVtStride = 72;           // LDS bytes per latent dim: 32 slots + pad
constexpr float kRescale = 8.0f;        // lazy rescale threshold, log2 units
constexpr int kMergeBatch = 4;             // partials a merge loads together
constexpr int kPvGroup = 4;             // PV blocks whose V^T reads are in flight together

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
// is a scalar load, which the vector loads in flight do not wait behind.
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
__device__ inline u32x4 ldkv(const char* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ inline void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline float load_coherent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
constexpr int kWaitVmcnt0 = 0x0F70;       // s_waitcnt vmcnt(0)
constexpr int kBufferDword3 = 0x00020000;
constexpr int kCachePolicySc1 = 0x10;     // coherent at the device level (past the die's L2)

struct MlaParams {
  size_t page_bytes;
  int part_acc_bytes;   // size of the partial accumulator area (< 2 GiB)
  int g, maxp, log2P;
  int W;                // the planner's units (tile ranges)
  int ngroups;          // query-head groups of kMaxGroup (one workgroup per unit and group)
  int ml_stride;        // (max, sum) pairs per partial
  float scale_log2;
};

// Workgroups per dispatch batch: a multiple of the eight XCDs, so that the
// workgroups of every head group of one unit share an XCD (workgroup i runs
// on XCD i % 8) and read that unit's tiles close together in time -- the
// later groups' reads then mostly hit that XCD's L2.
constexpr int kUnitBatch = 32;

// Latent piece s of this lane's row (dims 32s + 8G .. +7 of slot `slot`)
// into the wave's [dim][slot] LDS area; a slot at or past the valid rows is
// written as zeros (a freed page may hold any bytes).
__device__ inline void piece_to_lds(u32x4 x, char* vt, int s, int slot, bool live, int G) {
  if (!live) x = u32x4{0u, 0u, 0u, 0u};
  char* base = vt + (32 * s + 8 * G) * kVtStride + slot * 2;
#pragma unroll
  for (int e = 0; e < 8; ++e)
    *reinterpret_cast<uint16_t*>(base + e * kVtStride) = static_cast<uint16_t>(x[e >> 1] >> (16 * (e & 1)));
}

// The wave's LDS area passes between its lanes (written by the lanes that
// loaded a slot, read by the lanes that multiply a latent dim): the wave's
// LDS operations complete in order, and these fences keep the compiler from
// moving accesses across the hand-over.
__device__ inline void lds_handoff() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

struct Acc {
  f32x4 o[kOBlocks];   // O^T rows 16b + 4G .. +3 of column r (query head r)
  float m, l;
};

// Softmax of one tile (scores of slots 8G .. 8G+3 in sa, 8G+4 .. 8G+7 in sb)
// and its PV products with the transposed latent in LDS.
__device__ inline void finish_tile(Acc& acc, f32x4 sa, f32x4 sb, const char* vt, float scale,
                                   int valid, int r, int G) {
  float sc[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sc[i] = sa[i] * scale;
    sc[4 + i] = sb[i] * scale;
  }
  const int nv = valid - 8 * G;
#pragma unroll
  for (int j = 0; j < 8; ++j) sc[j] = j < nv ? sc[j] : -INFINITY;
  float mx = fmaxf(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3])),
                   fmaxf(fmaxf(sc[4], sc[5]), fmaxf(sc[6], sc[7])));
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const bool raise = mx > acc.m + kRescale;
  if (__builtin_amdgcn_ballot_w64(raise)) {
    const float m_new = raise ? mx : acc.m;
    const float alpha = __builtin_amdgcn_exp2f(acc.m - m_new);
    acc.l *= alpha;
#pragma unroll
    for (int b = 0; b < kOBlocks; ++b) acc.o[b] *= alpha;
    acc.m = m_new;
  }
  bf16x8 p;
  float psum = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const __bf16 pb = static_cast<__bf16>(__builtin_amdgcn_exp2f(sc[j] - acc.m));
    p[j] = pb;
    psum += static_cast<float>(pb);
  }
  acc.l += psum;
  const u32x4 pu = __builtin_bit_cast(u32x4, p);
  // V^T operand of row block b: latent dim 16b + r, slots 8G .. 8G+7; read
  // kPvGroup blocks ahead of the products that use them (reading all 32
  // first would not fit in registers)
  const char* vrow = vt + r * kVtStride + 16 * G;
  auto read_v = [&](int b) {
    const u32x2 lo = *reinterpret_cast<const u32x2*>(vrow + 16 * b * kVtStride);
    const u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + 16 * b * kVtStride + 8);
    return u32x4{lo[0], lo[1], hi[0], hi[1]};
  };
  u32x4 v[2][kPvGroup];
#pragma unroll
  for (int i = 0; i < kPvGroup; ++i) v[0][i] = read_v(i);
#pragma unroll
  for (int b0 = 0; b0 < kOBlocks; b0 += kPvGroup) {
    const int cur = (b0 / kPvGroup) & 1;
    if (b0 + kPvGroup < kOBlocks) {
#pragma unroll
      for (int i = 0; i < kPvGroup; ++i) v[cur ^ 1][i] = read_v(b0 + kPvGroup + i);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < kPvGroup; ++i) acc.o[b0 + i] = mfma_bf16(v[cur][i], pu, acc.o[b0 + i]);
  }
}

__global__ __launch_bounds__(256, 1) void decode_mla_kernel(
    const int32_t* __restrict__ status, const HeadDesc* __restrict__ desc,
    const int32_t* __restrict__ cum_tiles, const int32_t* __restrict__ wave_bounds,
    const int4* __restrict__ wave_desc, const int4* __restrict__ head_waves,
    int32_t* __restrict__ head_cnt, const int32_t* __restrict__ page_table,
    char* __restrict__ pool, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_in,
    float2* __restrict__ part_ml, float* __restrict__ part_acc, float* __restrict__ out,
    MlaParams a) {
  __shared__ __attribute__((aligned(16))) char vt_lds[kWavesPerBlock][kDv * kVtStride];
  __shared__ float2 ml_lds[kWavesPerBlock][kMaxGroup];
  __shared__ int s_last;
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // the planner's unit (this block's tile range) and the group of kMaxGroup
  // query heads this block attends for
  const int per = kUnitBatch * a.ngroups;
  const int unit = static_cast<int>(blockIdx.x) / per * kUnitBatch + static_cast<int>(blockIdx.x) % kUnitBatch;
  const int grp = static_cast<int>(blockIdx.x) % per / kUnitBatch;
  if (unit >= a.W) return;
  const int h0 = grp * kMaxGroup;                    // first query head of the group
  const int gq = min(kMaxGroup, a.g - h0);           // query heads in the group
  const int r = lane & 15, G = lane >> 4;
  char* vt = vt_lds[wid];
  const int4 wd0 = ldc(wave_desc, 2 * unit), wd1 = ldc(wave_desc, 2 * unit + 1);
  int tb = ldc(wave_bounds, unit);
  const int te = ldc(wave_bounds, unit + 1);
  if (load_status(status) != 0) return;
  if (tb >= te) return;
  const int tpp_log2 = a.log2P - 5;
  const int tpp_mask = (1 << tpp_log2) - 1;
  constexpr size_t kTileBytes = static_cast<size_t>(kD) * 64;
  int hh = wd0.z;
  bool first = true;
  const int qr = min(r, gq - 1);
  const __amdgpu_buffer_rsrc_t acc_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      part_acc, static_cast<short>(0), a.part_acc_bytes, kBufferDword3);
  while (tb < te) {
    int c0, c1;
    HeadDesc d;
    if (first) {
      c0 = wd0.w;
      c1 = wd1.x;
      d = make_int4(wd1.y, wd1.z, wd1.w, 0);
      first = false;
    } else {
      while (ldc(cum_tiles, hh + 1) <= tb) ++hh;
      c0 = ldc(cum_tiles, hh);
      c1 = ldc(cum_tiles, hh + 1);
      d = ldc(desc, hh);
    }
    const int seg_end = min(te, c1);
    const int L = d.x;
    const int32_t* pt = page_table + static_cast<size_t>(d.y) * a.maxp;
    auto tile_of = [&](int t) -> const char* {
      return pool + static_cast<size_t>(ldc(uniform_ptr(pt), t >> tpp_log2)) * a.page_bytes +
             static_cast<size_t>(t & tpp_mask) * kTileBytes;
    };
    const int t_lo = tb - c0;
    const int t_hi = seg_end - c0;
    // the segment's tiles are dealt to the block's waves in turn: this wave
    // takes t_lo + wid, t_lo + wid + 4, ...
    const int t_first = t_lo + wid;
    Acc acc;
#pragma unroll
    for (int b = 0; b < kOBlocks; ++b) acc.o[b] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc.m = -INFINITY;
    acc.l = 0.f;
    if (t_first < t_hi) {
      // query fragments (B operand of the score MFMA): column r = query head r
      u32x4 qf[kKBlocks];
      const char* qrow = reinterpret_cast<const char*>(q + (static_cast<size_t>(hh) * a.g + h0 + qr) * kD);
#pragma unroll
      for (int s = 0; s < kKBlocks; ++s) {
        const u32x4 x = *reinterpret_cast<const u32x4*>(qrow + (32 * s + 8 * G) * 2);
        qf[s] = r < gq ? x : u32x4{0u, 0u, 0u, 0u};
      }
      // the token appended by this call (slot d.z) is written into its tile
      // by the wave that reads that tile, before its loads (by that wave of
      // every head group's block: the same bytes, each block's own store
      // ordered before its own loads)
      const int tz = d.z >> 5;
      if (k_in != nullptr && tz >= t_first && tz < t_hi && ((tz - t_first) & 3) == 0) {
        char* tile = const_cast<char*>(tile_of(tz));
        const int j = d.z & 31;
        const uint4* src = reinterpret_cast<const uint4*>(k_in + static_cast<size_t>(hh) * kD);
        // 72 pieces: one per lane, then 8 more (no lane loop, whose divergent
        // exit would push the uniform values used after it into VGPRs)
        *reinterpret_cast<uint4*>(tile + k_elem_off(j, 8 * lane)) = src[lane];
        if (lane < kD / 8 - 64)
          *reinterpret_cast<uint4*>(tile + k_elem_off(j, 8 * (64 + lane))) = src[64 + lane];
      }
      // slot of this lane's row in half h: 8 (r / 4) + r % 4 + 4 h
      const int row0 = 8 * (r >> 2) + (r & 3);
      // The tile's 36 pieces (half h, k-step s: 1 KB at h * 1024 + s * 2048)
      // stream through 18 registers sets: piece s of a half is consumed
      // (score MFMA, latent to LDS) and its register set refilled with the
      // piece 18 positions later -- the other half, or the wave's next tile
      // -- so 17 to 18 pieces (18 KB) stay in flight with 72 registers.
      u32x4 kr[kKBlocks];
      const char* cur = tile_of(t_first) + lane * 16;
      // issued in piece order (the waits below count on it)
#pragma unroll
      for (int s = 0; s < kKBlocks; ++s) {
        kr[s] = ldkv(cur + s * 2048);
        __builtin_amdgcn_sched_barrier(0);
      }
      int t = t_first;
      for (; t + kWavesPerBlock < t_hi; t += kWavesPerBlock) {
        const char* nxt = tile_of(t + kWavesPerBlock) + lane * 16;
        f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < kKBlocks; ++s) {
          sa = mfma_bf16(kr[s], qf[s], sa);
          if (s < kLBlocks) piece_to_lds(kr[s], vt, s, row0, true, G);
          kr[s] = ldkv(cur + 1024 + s * 2048);
          if (s % 3 == 2) __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int s = 0; s < kKBlocks; ++s) {
          sb = mfma_bf16(kr[s], qf[s], sb);
          if (s < kLBlocks) piece_to_lds(kr[s], vt, s, row0 + 4, true, G);
          kr[s] = ldkv(nxt + s * 2048);
          if (s % 3 == 2) __builtin_amdgcn_sched_barrier(0);
        }
        lds_handoff();
        finish_tile(acc, sa, sb, vt, a.scale_log2, kTile, r, G);
        lds_handoff();
        cur = nxt;
      }
      {
        // the wave's last tile: rows at or past L are stale in the head's last tile
        const int valid = (t == t_hi - 1 && seg_end == c1) ? L - t * kTile : kTile;
        f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < kKBlocks; ++s) {
          sa = mfma_bf16(kr[s], qf[s], sa);
          if (s < kLBlocks) piece_to_lds(kr[s], vt, s, row0, row0 < valid, G);
          kr[s] = ldkv(cur + 1024 + s * 2048);
          if (s % 3 == 2) __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int s = 0; s < kKBlocks; ++s) {
          sb = mfma_bf16(kr[s], qf[s], sb);
          if (s < kLBlocks) piece_to_lds(kr[s], vt, s, row0 + 4, row0 + 4 < valid, G);
        }
        lds_handoff();
        finish_tile(acc, sa, sb, vt, a.scale_log2, valid, r, G);
        lds_handoff();
      }
    }
    // Block combine of the four waves' partials of this head, through LDS:
    // each wave stages (m, l) and its accumulators in its own area, then
    // folds the four for 8 of the 32 row blocks.  The result is the head's
    // output when the block covered all its tiles, else the block's partial
    // of a split head.
    float l = acc.l;
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
#pragma unroll
    for (int b = 0; b < kOBlocks; ++b)
      *reinterpret_cast<f32x4*>(vt + (b * 64 + lane) * 16) = acc.o[b];
    if (G == 0) ml_lds[wid][r] = make_float2(acc.m, l);
    __syncthreads();
    float mj[kWavesPerBlock], M = -INFINITY;
#pragma unroll
    for (int j = 0; j < kWavesPerBlock; ++j) {
      mj[j] = ml_lds[j][r].x;
      M = fmaxf(M, mj[j]);
    }
    float den = 0.f, wj[kWavesPerBlock];
#pragma unroll
    for (int j = 0; j < kWavesPerBlock; ++j) {
      wj[j] = __builtin_amdgcn_exp2f(mj[j] - M);   // 0 for a wave without tiles (m = -inf)
      den += wj[j] * ml_lds[j][r].y;
    }
    constexpr int kBlocksPerWave = kOBlocks / kWavesPerBlock;
    f32x4 num[kBlocksPerWave];
#pragma unroll
    for (int i = 0; i < kBlocksPerWave; ++i) {
      const int b = wid * kBlocksPerWave + i;
      num[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < kWavesPerBlock; ++j)
        num[i] += wj[j] * *reinterpret_cast<const f32x4*>(vt_lds[j] + (b * 64 + lane) * 16);
    }
    if (r < gq) {
      if (tb == c0 && seg_end == c1) {
        const float inv = 1.0f / den;
        float* o = out + (static_cast<size_t>(hh) * a.g + h0 + r) * kDv + 4 * G;
#pragma unroll
        for (int i = 0; i < kBlocksPerWave; ++i)
          *reinterpret_cast<f32x4*>(o + 16 * (wid * kBlocksPerWave + i)) = num[i] * inv;
      } else {
        // the block's partial, with stores that are complete at the device's
        // coherence point once this wave's vmcnt drains
        const size_t pid = static_cast<size_t>(unit) + hh;
        if (wid == 0 && G == 0) {
          float* ml = reinterpret_cast<float*>(part_ml + pid * a.ml_stride + h0 + r);
          store_coherent(ml, M);
          store_coherent(ml + 1, den);
        }
        const uint32_t o = static_cast<uint32_t>(((pid * a.g + h0 + r) * kDv + 4 * G) * 4);
#pragma unroll
        for (int i = 0; i < kBlocksPerWave; ++i)
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, num[i]), acc_rsrc,
                                                 o + 64 * (wid * kBlocksPerWave + i), 0, kCachePolicySc1);
      }
    }
    if (!(tb == c0 && seg_end == c1)) {
      // Split head: once the block's partial is stored, add its tiles to the
      // head's arrival counter; the block that completes the count merges
      // the head's partials (one per block, a few per head), each wave
      // folding its 8 row blocks, and resets the counter.
      __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
      __syncthreads();
      if (threadIdx.x == 0) {
        const int prev = atomicAdd(&head_cnt[hh * a.ngroups + grp], seg_end - tb);
        s_last = prev + (seg_end - tb) == c1 - c0;
      }
      __syncthreads();
      if (s_last) {
        // batches of kMergeBatch partials: their (m, l) and rows are loaded
        // together (one round trip) and folded into a running maximum
        const int4 hw = ldc(head_waves, hh);
        float Mh = -INFINITY, dh = 0.f;
        f32x4 nh[kBlocksPerWave];
#pragma unroll
        for (int i = 0; i < kBlocksPerWave; ++i) nh[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int u0 = hw.x; u0 <= hw.y; u0 += kMergeBatch) {
          bool lv[kMergeBatch];
          float mv[kMergeBatch], lv_l[kMergeBatch];
          u32x4 x[kMergeBatch][kBlocksPerWave];
#pragma unroll
          for (int j = 0; j < kMergeBatch; ++j) {
            const int u = u0 + j;
            lv[j] = u <= hw.y && ldc(wave_bounds, u) < ldc(wave_bounds, u + 1);
            const size_t pid = static_cast<size_t>(lv[j] ? u : hw.x) + hh;
            const float* ml = reinterpret_cast<const float*>(part_ml + pid * a.ml_stride + h0 + r);
            mv[j] = lv[j] ? load_coherent(ml) : -INFINITY;
            lv_l[j] = lv[j] ? load_coherent(ml + 1) : 0.f;
            const uint32_t o = static_cast<uint32_t>(((pid * a.g + h0 + (r < gq ? r : 0)) * kDv + 4 * G) * 4);
#pragma unroll
            for (int i = 0; i < kBlocksPerWave; ++i)
              x[j][i] = lv[j] ? __builtin_amdgcn_raw_buffer_load_b128(acc_rsrc, o + 64 * (wid * kBlocksPerWave + i), 0,
                                                                       kCachePolicySc1)
                              : u32x4{0u, 0u, 0u, 0u};
          }
          float bm = mv[0];
#pragma unroll
          for (int j = 1; j < kMergeBatch; ++j) bm = fmaxf(bm, mv[j]);
          if (bm > Mh) {   // the first batch always raises Mh from -inf (its sums are 0)
            const float sc = __builtin_amdgcn_exp2f(Mh - bm);
            dh *= sc;
#pragma unroll
            for (int i = 0; i < kBlocksPerWave; ++i) nh[i] *= sc;
            Mh = bm;
          }
#pragma unroll
          for (int j = 0; j < kMergeBatch; ++j) {
            const float wt = lv[j] ? __builtin_amdgcn_exp2f(mv[j] - Mh) : 0.f;
            dh += wt * lv_l[j];
#pragma unroll
            for (int i = 0; i < kBlocksPerWave; ++i) nh[i] += wt * __builtin_bit_cast(f32x4, x[j][i]);
          }
        }
        if (r < gq) {
          const float inv = 1.0f / dh;
          float* o = out + (static_cast<size_t>(hh) * a.g + h0 + r) * kDv + 4 * G;
#pragma unroll
          for (int i = 0; i < kBlocksPerWave; ++i)
            *reinterpret_cast<f32x4*>(o + 16 * (wid * kBlocksPerWave + i)) = nh[i] * inv;
        }
        if (threadIdx.x == 0)
          __hip_atomic_store(&head_cnt[hh * a.ngroups + grp], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    __syncthreads();   // the staged partials are read before the next segment's tiles reuse the areas
    tb = seg_end;
    ++hh;
  }
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
  a.ngroups = lo.head_groups;
  a.ml_stride = lo.ml_stride;
  a.scale_log2 = c.softmax_scale * 1.4426950408889634f;
  const int blocks = (waves + kUnitBatch - 1) / kUnitBatch * kUnitBatch * a.ngroups;
  if (ev_start) (void)hipEventRecord(ev_start, st);
  hipLaunchKernelGGL(decode_mla_kernel, dim3(blocks), dim3(256), 0, st,
                     reinterpret_cast<const int32_t*>(static_cast<char*>(meta) + lo.status),
                     reinterpret_cast<const HeadDesc*>(w + lo.ws_head_desc),
                     reinterpret_cast<const int32_t*>(w + lo.ws_cum_tiles),
                     reinterpret_cast<const int32_t*>(w + lo.ws_wave_bounds),
                     reinterpret_cast<const int4*>(w + lo.ws_wave_desc),
                     reinterpret_cast<const int4*>(w + lo.ws_head_waves),
                     reinterpret_cast<int32_t*>(w + lo.ws_head_cnt),
                     layer_state(lo, meta, layer).page_table, static_cast<char*>(pool),
                     static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                     reinterpret_cast<float2*>(w + lo.ws_part_ml),
                     reinterpret_cast<float*>(w + lo.ws_part_acc), out, a);
  hipError_t e = hipGetLastError();
  if (ev_stop) (void)hipEventRecord(ev_stop, st);
  return e;
}

int decode_mla_resident_waves() {
  int dev = 0, cus = 0, blocks = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, decode_mla_kernel, 256, 0) != hipSuccess ||
      blocks < 1)
    return -1;
  // the planner's units are blocks (one per CU): each block's four waves
  // share its tile range (one block per unit and query-head group)
  return cus < kMaxMlaUnits ? cus : kMaxMlaUnits;
}

}  // namespace dms
