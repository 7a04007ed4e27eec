// GQA split-K flash-decode over the retained DMS slots, gfx950.
//
// After the append of step t, the live slots of a head are exactly the keys
// visible to query t (paper Sec. 3.1-3.2: a flagged key leaves the cache when
// it leaves the window), so decode attention needs no mask: every query head
// of a group attends to slots 0 .. L-1 of its KV head.  The cost is the KV
// bytes read (Sec. 1; Appendix I), so the kernel is built around streaming
// those bytes once:
//
//  * Work split: the retained tokens of all (sequence, KV head) pairs of the
//    call are cut into 32-token tiles, and the flat tile list is divided into
//    equal contiguous ranges, one per wave, one wave per SIMD ("stream-K"):
//    ragged per-head lengths (Sec. 3.1: heads compress at different rates) do
//    not unbalance the chip.  A wave covering a whole head writes the final
//    output; a head split over several waves gets partials (running max, sum,
//    accumulator).  At the end of its range a wave adds its tile counts to
//    the heads it shares, and the wave that completes a head's count merges
//    its partials with log-sum-exp weights (device-coherent accesses, no L2
//    flush), so no wait interrupts the tile stream.
//  * Pages are stored tile-major: the 32 tokens of a tile are one contiguous
//    block, in the order the MFMAs consume it (keys as the A operand of
//    S^T = K Q^T, transposed values as the A operand of O^T = V^T P^T; layout
//    in dms_common.h).  Per tile each lane issues 16-byte loads straight into
//    operand registers, and every load instruction of a wave reads one
//    contiguous 1 KB.  No LDS round trip is needed.
//    The group's g query heads fill g of the 16 MFMA columns.
//  * The 16x16 accumulator layout puts rows 4*(lane/16) .. +3 of column
//    lane%16 in each lane.  Tile rows of the first / second score MFMA are
//    assigned tokens 8*(r/4) + r%4 and 8*(r/4) + 4 + r%4, so after both MFMAs
//    lane group G holds the scores of tokens 8G .. 8G+7 -- exactly the k
//    slice the PV MFMA's B operand wants in that lane.  Scores never leave
//    registers.
//  * Online softmax in the exp2 domain: per-lane max over its 8 scores, then
//    two cross-row shuffles; the running sum stays per lane until the end.
#include "dms_common.h"
#include "dms_fp8.h"

namespace dms {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

constexpr int kWavesPerBlock = 4;

__device__ inline int load_status(const int32_t* status) {
  return __atomic_load_n(status, __ATOMIC_RELAXED);
}

__device__ inline f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ inline u32x4 ldg16(const char* p) { return *reinterpret_cast<const u32x4*>(p); }
// Reads of tables that no kernel running with this one writes (planner
// output, page tables): through the constant address space, so that a
// wave-uniform index becomes a scalar load even inside loops that store to
// the pool (a vector load there would need vmcnt(0) before its value is used
// and drain the wave's tile pipeline).
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
// Cache-tile reads: every byte is read once per step, so the loads are
// non-temporal (measured on MI355X: a shuffled 32 KB-page stream reaches
// 7.1 TB/s this way against 6.3 TB/s with ordinary loads).
__device__ inline u32x4 ldkv(const char* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// Device-coherent (sc1) float store / load: agent-scope relaxed atomics, which
// on gfx950 write through / read around the per-XCD L2.
__device__ inline void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline float load_coherent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// s_waitcnt vmcnt(0): all of this wave's vector memory operations complete.
constexpr int kWaitVmcnt0 = 0x0F70;
// Raw buffer resource word 3 (32-bit data format, no swizzle) and the sc1
// cache-policy bit of buffer loads / stores (agent-coherent access).
constexpr int kBufferDword3 = 0x00020000;
constexpr int kCachePolicySc1 = 0x10;

struct DecodeParams {
  size_t page_bytes;
  int part_acc_bytes;   // size of the split-K accumulator area (< 2 GiB: validate_config)
  int NH, g, maxp, P, log2P, W;
  int zero_neuron;   // element 0 of the group's first query head is read as 0
  int qB;            // page retrieval: pages attended per head (selection stride)
  float scale_log2;  // softmax scale * log2(e)
  int defer_merge;   // split heads are merged by merge_kernel after the launch
};

// Scores are exponentiated against a per-lane reference max that is only
// raised when a tile's max exceeds it by more than this (log2 units), so the
// accumulator is rescaled rarely; probabilities stay below 2^kRescale.
constexpr float kRescale = 8.0f;

template <int D>
struct Frag {
  u32x4 ka[D / 32];  // K rows of score MFMA 0 (tokens 8*(r/4) + r%4)
  u32x4 kb[D / 32];  // K rows of score MFMA 1 (tokens 8*(r/4) + 4 + r%4)
  u32x4 vt[D / 16];  // V^T rows d = 16b + r, tokens 8G .. 8G+7
};

// Load one full 32-slot tile (wave-uniform address).  The tile is stored in
// fragment order (see dms_common.h), so load instruction i of the wave reads
// the contiguous 1 KB block i and lane l takes bytes 16 l .. 16 l + 15.
template <int D>
__device__ inline void load_tile(Frag<D>& f, const char* tile, int lane) {
  const char* p = tile + lane * 16;
#pragma unroll
  for (int s = 0; s < D / 32; ++s) {
    f.ka[s] = ldkv(p + s * 2048);
    f.kb[s] = ldkv(p + s * 2048 + 1024);
  }
#pragma unroll
  for (int b = 0; b < D / 16; ++b) f.vt[b] = ldkv(p + D * 64 + b * 1024);
}

// Last, partial tile of a head: rows at or past L are not read and the value
// elements of those tokens are zero.
template <int D>
__device__ inline void load_tail(Frag<D>& f, const char* tile, int lane, int valid, int r, int G) {
  const int ta = 8 * (r >> 2) + (r & 3);
  const u32x4 z = {0u, 0u, 0u, 0u};
  const char* p = tile + lane * 16;
#pragma unroll
  for (int s = 0; s < D / 32; ++s) {
    f.ka[s] = ta < valid ? ldkv(p + s * 2048) : z;
    f.kb[s] = ta + 4 < valid ? ldkv(p + s * 2048 + 1024) : z;
  }
  const int nv = valid - 8 * G;  // tokens of this lane's 8 that exist
#pragma unroll
  for (int b = 0; b < D / 16; ++b) {
    u32x4 x = nv > 0 ? ldkv(p + D * 64 + b * 1024) : z;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j >= nv) {  // element j holds token 8G + j
        const unsigned int keep = (j & 1) ? 0x0000FFFFu : 0xFFFF0000u;
        x[j >> 1] &= keep;
      }
    }
    f.vt[b] = x;
  }
}

template <int D>
struct Acc {
  f32x4 o[D / 16];
  float m, l;  // reference max (log2 units) and this lane's partial sum
};

// Scores, online softmax and PV accumulation for one tile; `valid` live tokens.
template <int D>
__device__ inline void compute_tile(Acc<D>& acc, const Frag<D>& f, const u32x4* qf, float scale,
                                    int valid, int G) {
  f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < D / 32; ++s) {
    s0 = mfma_bf16(f.ka[s], qf[s], s0);
    s1 = mfma_bf16(f.kb[s], qf[s], s1);
  }
  float sc[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sc[i] = s0[i] * scale;
    sc[4 + i] = s1[i] * scale;
  }
  if (valid < kTile) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (8 * G + j >= valid) sc[j] = -INFINITY;
  }
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
    for (int b = 0; b < D / 16; ++b) acc.o[b] *= alpha;
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
#pragma unroll
  for (int b = 0; b < D / 16; ++b) acc.o[b] = mfma_bf16(f.vt[b], pu, acc.o[b]);
}

// ---------------------------------------------------------------------------
// FP8 pages (layout in dms_fp8.h).  Per tile each lane loads D/64 x 2 key
// chunks, D/32 value chunks and its 8 slots' key / value scales (16 bytes
// each); chunks are converted to the same bf16 MFMA operands as above in
// registers (one conversion per two codes, exact).  Keys: the fp32 scores are
// multiplied by the key scale; values: the bf16 weights by the value scale
// (powers of two, so both are exact and the denominator keeps the unscaled
// weights).
// ---------------------------------------------------------------------------
template <int D>
struct FragF8 {
  u32x4 k[D / 64][2];  // key chunks of score MFMA rows blocks 0 / 1
  u32x4 v[D / 32];     // value chunks (two V^T rows each)
  u32x4 s[4];          // key scales (s[0], s[1]) and value scales (s[2], s[3]) of slots 8G ..
};

template <int D>
__device__ inline void load_tile_f8(FragF8<D>& f, const char* tile, int lane, int G) {
#pragma unroll
  for (int p = 0; p < D / 64; ++p) {
    f.k[p][0] = ldkv(tile + p * 2048 + lane * 16);
    f.k[p][1] = ldkv(tile + p * 2048 + 1024 + lane * 16);
  }
#pragma unroll
  for (int p = 0; p < D / 32; ++p) f.v[p] = ldkv(tile + D * 32 + p * 1024 + lane * 16);
#pragma unroll
  for (int i = 0; i < 4; ++i) f.s[i] = ldkv(tile + D * 64 + G * 64 + i * 16);
}

// Last, partial tile: key rows of missing slots are not read, value codes and
// scales of missing slots are zeroed (a freed page may hold any bytes).
template <int D>
__device__ inline void load_tail_f8(FragF8<D>& f, const char* tile, int lane, int valid, int r, int G) {
  const int ta = 8 * (r >> 2) + (r & 3);
  const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int p = 0; p < D / 64; ++p) {
    f.k[p][0] = ta < valid ? ldkv(tile + p * 2048 + lane * 16) : z;
    f.k[p][1] = ta + 4 < valid ? ldkv(tile + p * 2048 + 1024 + lane * 16) : z;
  }
  const int nv = valid - 8 * G;   // slots of this lane's 8 that exist
  // byte i of each 8-byte half is slot 8G + i
  const uint64_t keep8 = nv >= 8 ? ~0ull : (nv <= 0 ? 0ull : (~0ull >> (8 * (8 - nv))));
  const uint32_t klo = static_cast<uint32_t>(keep8), khi = static_cast<uint32_t>(keep8 >> 32);
#pragma unroll
  for (int p = 0; p < D / 32; ++p) {
    u32x4 x = nv > 0 ? ldkv(tile + D * 32 + p * 1024 + lane * 16) : z;
    x[0] &= klo;
    x[1] &= khi;
    x[2] &= klo;
    x[3] &= khi;
    f.v[p] = x;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    u32x4 x = nv > 0 ? ldkv(tile + D * 64 + G * 64 + i * 16) : z;
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if ((i & 1) * 4 + c >= nv) x[c] = 0u;
    f.s[i] = x;
  }
}

// 8 E4M3 codes (two words) -> 8 bf16 (exact)
__device__ inline u32x4 f8_to_bf16x8(uint32_t w0, uint32_t w1) {
  u32x4 a;
  a[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, false));
  a[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, true));
  a[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w1, 1.0f, false));
  a[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w1, 1.0f, true));
  return a;
}

template <int D>
__device__ inline void compute_tile_f8(Acc<D>& acc, const FragF8<D>& f, const u32x4* qf, float scale,
                                       int valid, int G) {
  f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int p = 0; p < D / 64; ++p) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      s0 = mfma_bf16(f8_to_bf16x8(f.k[p][0][2 * j], f.k[p][0][2 * j + 1]), qf[2 * p + j], s0);
      s1 = mfma_bf16(f8_to_bf16x8(f.k[p][1][2 * j], f.k[p][1][2 * j + 1]), qf[2 * p + j], s1);
    }
  }
  float sc[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sc[i] = s0[i] * (scale * __uint_as_float(f.s[0][i]));
    sc[4 + i] = s1[i] * (scale * __uint_as_float(f.s[1][i]));
  }
  if (valid < kTile) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (8 * G + j >= valid) sc[j] = -INFINITY;
  }
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
    for (int b = 0; b < D / 16; ++b) acc.o[b] *= alpha;
    acc.m = m_new;
  }
  bf16x8 p;
  float psum = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const __bf16 pb = static_cast<__bf16>(__builtin_amdgcn_exp2f(sc[j] - acc.m));
    const float pf = static_cast<float>(pb);
    psum += pf;
    // the value scale of slot 8G + j (zero for a missing slot)
    p[j] = static_cast<__bf16>(pf * __uint_as_float(f.s[2 + (j >> 2)][j & 3]));
  }
  acc.l += psum;
  const u32x4 pu = __builtin_bit_cast(u32x4, p);
#pragma unroll
  for (int b = 0; b < D / 16; b += 2) {
    const u32x4 x = f.v[b / 2];
    acc.o[b] = mfma_bf16(f8_to_bf16x8(x[0], x[1]), pu, acc.o[b]);
    acc.o[b + 1] = mfma_bf16(f8_to_bf16x8(x[2], x[3]), pu, acc.o[b + 1]);
  }
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// First tile of wave w when `total` tiles are split over W waves in equal
// contiguous shares (w = W gives `total`); the planner and the fused decode
// launch split a call this way.
__device__ inline int wave_start(int64_t w, int total, int W) {
  return static_cast<int>(w * total / W);
}

// Waves wf .. wl hold tiles [c0, c1) of a head (c1 > c0): wave_start(wf) <= c0 <
// wave_start(wf + 1) and wave_start(wl) < c1 <= wave_start(wl + 1); bit i of the
// mask says whether wave wf + i has a non-empty range (i < 32).
__device__ inline int4 head_span(int c0, int c1, int total, int W) {
  const int64_t T = total, Wl = W;
  const int wf = static_cast<int>(((c0 + 1) * Wl + T - 1) / T) - 1;
  const int wl = min(W - 1, static_cast<int>((c1 * Wl + T - 1) / T) - 1);
  // wave_start(w) = floor(w T / W), stepped through the span: each step adds
  // T / W and carries the remainder
  const int q = total / W, rstep = total % W;
  int rem = static_cast<int>(static_cast<int64_t>(wf) * T % Wl);
  int mask = 0;
  for (int i = 0; i < 32 && wf + i <= wl; ++i) {
    rem += rstep;
    const int grow = q + (rem >= W ? 1 : 0);   // tiles of wave wf + i
    if (rem >= W) rem -= W;
    if (grow > 0) mask |= 1 << i;
  }
  return make_int4(wf, wl, mask, 0);
}

constexpr int kMergeBatch = 64;   // partials whose (max, sum) one round of loads fetches (one per lane)
constexpr int kMergeLoads = 32;   // 16-byte accumulator loads in flight per lane in the merge

// Log-sum-exp merge of the partials a head got from waves wf .. wl (index
// w + hh; waves with an empty range wrote none).  Every access is
// agent-coherent, and the merge is bound by the round trips of one wave, so
// as many loads as possible are in flight together: lane i fetches partial
// b0 + i's (max, sum) for every row, the head's g x D outputs are spread
// over the lanes as PPL 16-byte pieces each, and the pieces of U partials
// (U * PPL <= kMergeLoads) are all requested before any is used -- the first
// U together with the (max, sum) loads.  Loads of partials that turn out
// dead (no tiles) or that lie past the span read in-range stale bytes and
// are discarded by a select, never multiplied.
template <int D, int PPL>
__device__ __forceinline__ void merge_head(const float2* part_ml, __amdgpu_buffer_rsrc_t acc_rsrc,
                           int total, int W, float* out, int wf, int wl, int hh, int g,
                           int lane, float (*wts)[kMaxGroup]) {
  constexpr int U = kMergeLoads / PPL > 0 ? kMergeLoads / PPL : 1;
  const int pieces = g * D / 4;
  const int nparts = wl - wf + 1;
  int row[PPL];
#pragma unroll
  for (int j = 0; j < PPL; ++j) row[j] = min(4 * (lane + 64 * j) / D, kMaxGroup - 1);
  auto acc_load = [&](int u, int j) -> u32x4 {
    // partial wf + min(u, nparts - 1): always inside the written span's slots
    const size_t p2 = static_cast<size_t>(wf + min(u, nparts - 1)) + hh;
    const int f = min(lane + 64 * j, pieces - 1);
    return __builtin_amdgcn_raw_buffer_load_b128(
        acc_rsrc, static_cast<uint32_t>((p2 * g * D + 4 * f) * 4), 0, kCachePolicySc1);
  };
  f32x4 num[PPL];
#pragma unroll
  for (int j = 0; j < PPL; ++j) num[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float den[kMaxGroup];
#pragma unroll
  for (int r = 0; r < kMaxGroup; ++r) den[r] = 0.f;
  // pass 1: row maxima; the lane's (max, sum) of the last batch stay in registers
  float M[kMaxGroup], ml_m[kMaxGroup], ml_l[kMaxGroup];
#pragma unroll
  for (int r = 0; r < kMaxGroup; ++r) M[r] = -INFINITY;
  u32x4 x[U][PPL];    // accumulator pieces in flight; the first batch goes out with the (max, sum) loads
  bool live = false;
  for (int b0 = 0; b0 < nparts; b0 += kMergeBatch) {
    const int w2 = wf + b0 + lane;
    live = b0 + lane < nparts && wave_start(w2, total, W) < wave_start(w2 + 1, total, W);
    const float* ml = reinterpret_cast<const float*>(part_ml + (static_cast<size_t>(live ? w2 : wf) + hh) * kMaxGroup);
#pragma unroll
    for (int r = 0; r < kMaxGroup; ++r) {
      ml_m[r] = (live && r < g) ? load_coherent(ml + 2 * r) : -INFINITY;
      ml_l[r] = (live && r < g) ? load_coherent(ml + 2 * r + 1) : 0.f;
    }
    if (b0 == 0) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < PPL; ++j) x[u][j] = acc_load(u, j);
    }
#pragma unroll
    for (int r = 0; r < kMaxGroup; ++r) M[r] = fmaxf(M[r], ml_m[r]);
  }
#pragma unroll
  for (int r = 0; r < kMaxGroup; ++r)
    if (r < g) M[r] = wave_max(M[r]);
  // pass 2: weights through LDS, then the accumulators U partials at a time
  for (int b0 = 0; b0 < nparts; b0 += kMergeBatch) {
    if (nparts > kMergeBatch) {   // only the last batch's (max, sum) were kept
      const int w2 = wf + b0 + lane;
      live = b0 + lane < nparts && wave_start(w2, total, W) < wave_start(w2 + 1, total, W);
      const float* ml = reinterpret_cast<const float*>(part_ml + (static_cast<size_t>(live ? w2 : wf) + hh) * kMaxGroup);
#pragma unroll
      for (int r = 0; r < kMaxGroup; ++r) {
        ml_m[r] = (live && r < g) ? load_coherent(ml + 2 * r) : -INFINITY;
        ml_l[r] = (live && r < g) ? load_coherent(ml + 2 * r + 1) : 0.f;
      }
    }
#pragma unroll
    for (int r = 0; r < kMaxGroup; ++r) {
      if (r < g) {
        const float sc = live ? __builtin_amdgcn_exp2f(ml_m[r] - M[r]) : 0.f;
        wts[lane][r] = sc;
        den[r] += sc * ml_l[r];
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int nb = min(kMergeBatch, nparts - b0);
    for (int i0 = 0; i0 < nb; i0 += U) {
      if (b0 != 0 || i0 != 0) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int j = 0; j < PPL; ++j) x[u][j] = acc_load(b0 + i0 + u, j);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int j = 0; j < PPL; ++j) {
          // a zero weight marks a partial past the span or of a wave without
          // tiles (stale bytes), or one that underflowed: it adds nothing
          const float wu = i0 + u < nb ? wts[i0 + u][row[j]] : 0.f;
          const f32x4 v = __builtin_bit_cast(f32x4, x[u][j]);
          num[j] += wu != 0.f ? wu * v : f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
    }
    __builtin_amdgcn_wave_barrier();   // weights of this batch read before the next overwrites them
  }
#pragma unroll
  for (int r = 0; r < kMaxGroup; ++r)
    if (r < g) den[r] = wave_sum(den[r]);
  float* o = out + static_cast<size_t>(hh) * g * D;
#pragma unroll
  for (int j = 0; j < PPL; ++j) {
    const int f = lane + 64 * j;
    if (f < pieces) {
      float d = den[0];
#pragma unroll
      for (int r = 1; r < kMaxGroup; ++r) if (r == row[j]) d = den[r];
      *reinterpret_cast<f32x4*>(o + 4 * f) = num[j] * (1.0f / d);
    }
  }
}

// merge_head with the piece count per lane, PPL = ceil(g * D / 256), fixed at
// compile time (the in-flight load batch is sized by it).
template <int D>
__device__ __forceinline__ void merge_head_any(const float2* part_ml, __amdgpu_buffer_rsrc_t acc_rsrc,
                               int total, int W, float* out, int wf, int wl, int hh,
                               int g, int lane, float (*wts)[kMaxGroup]) {
  switch ((g * D / 4 + 63) / 64) {
    case 1: merge_head<D, 1>(part_ml, acc_rsrc, total, W, out, wf, wl, hh, g, lane, wts); break;
    case 2: merge_head<D, 2>(part_ml, acc_rsrc, total, W, out, wf, wl, hh, g, lane, wts); break;
    case 3: merge_head<D, 3>(part_ml, acc_rsrc, total, W, out, wf, wl, hh, g, lane, wts); break;
    case 4: merge_head<D, 4>(part_ml, acc_rsrc, total, W, out, wf, wl, hh, g, lane, wts); break;
    default:
      if constexpr (D > 64) {
        if ((g * D / 4 + 63) / 64 <= 6)
          merge_head<D, 6>(part_ml, acc_rsrc, total, W, out, wf, wl, hh, g, lane, wts);
        else
          merge_head<D, 8>(part_ml, acc_rsrc, total, W, out, wf, wl, hh, g, lane, wts);
      }
      break;
  }
}

// Merge of at most 4 partials (the usual case): every load -- each lane's
// partial (max, sum) and all 16-byte accumulator pieces of all partials --
// is issued in one round; weights are passed between lanes by shuffles.
template <int D>
__device__ __forceinline__ void merge_head_small(const float2* part_ml, __amdgpu_buffer_rsrc_t acc_rsrc,
                                 int live_mask, float* out, int wf, int np, int hh,
                                 int g, int lane) {
  constexpr int kMaxPieces = kMaxGroup * D / 4 / 64;
  constexpr int kMaxParts = 4;
  const int pieces = g * D / 4;
  const bool live = lane < np && ((live_mask >> lane) & 1);
  const float* ml = reinterpret_cast<const float*>(
      part_ml + (static_cast<size_t>(wf + (lane < np ? lane : 0)) + hh) * kMaxGroup);
  float m[kMaxGroup], l[kMaxGroup];
#pragma unroll
  for (int r = 0; r < kMaxGroup; ++r) {
    m[r] = (live && r < g) ? load_coherent(ml + 2 * r) : -INFINITY;
    l[r] = (live && r < g) ? load_coherent(ml + 2 * r + 1) : 0.f;
  }
  // partials of waves that got no tiles were never written (stale bytes):
  // neither loaded nor added
  u32x4 x[kMaxPieces][kMaxParts];
#pragma unroll
  for (int j = 0; j < kMaxPieces; ++j) {
    const int f = lane + 64 * j;
#pragma unroll
    for (int u = 0; u < kMaxParts; ++u) {
      const size_t p2 = static_cast<size_t>(wf + u) + hh;
      x[j][u] = (f < pieces && u < np && ((live_mask >> u) & 1))
                    ? __builtin_amdgcn_raw_buffer_load_b128(
                          acc_rsrc, static_cast<uint32_t>((p2 * g * D + 4 * f) * 4), 0, kCachePolicySc1)
                    : u32x4{0u, 0u, 0u, 0u};
    }
  }
  float wgt[kMaxGroup], den[kMaxGroup];
#pragma unroll
  for (int r = 0; r < kMaxGroup; ++r) {
    if (r < g) {
      const float M = wave_max(m[r]);
      wgt[r] = live ? __builtin_amdgcn_exp2f(m[r] - M) : 0.f;
      den[r] = wave_sum(wgt[r] * l[r]);
    }
  }
  float* o = out + static_cast<size_t>(hh) * g * D;
#pragma unroll
  for (int j = 0; j < kMaxPieces; ++j) {
    const int f = lane + 64 * j;
    const int row = min(4 * f / D, kMaxGroup - 1);
    f32x4 num = {0.f, 0.f, 0.f, 0.f};
    float d = 1.f;
#pragma unroll
    for (int r = 0; r < kMaxGroup; ++r) {
      if (r < g) {
        // every lane takes part in the shuffles; only rows it owns are kept
#pragma unroll
        for (int u = 0; u < kMaxParts; ++u) {
          const float wu = __shfl(wgt[r], u, 64);
          if (r == row && u < np && ((live_mask >> u) & 1)) num += wu * __builtin_bit_cast(f32x4, x[j][u]);
        }
        if (r == row) d = den[r];
      }
    }
    if (f < pieces) *reinterpret_cast<f32x4*>(o + 4 * f) = num * (1.0f / d);
  }
}

// Where a decode launch finds the call's work split: the planning kernel's
// output in the workspace (GlobalPlan) or the plan every workgroup of a fused
// launch builds in LDS (LdsPlan).  Both give, for call head hh, its tile range
// [cum(hh), cum(hh + 1)) in the flat tile list and its descriptor (retained
// length, state head, slot appended by this call, and the page popped for
// that slot when the page table may not hold it yet, else -1); every value is
// uniform across the wave.
struct GlobalPlan {
  const HeadDesc* desc;
  const int32_t* cum;
  const int32_t* wave_bounds;
  const int4* wave_desc;
  const int4* head_waves;   // per head: first / last wave holding its tiles, live mask
  int total;
  // the planner's descriptor of wave w's first segment comes with its range,
  // so a wave starts after one round of scalar loads
  __device__ __forceinline__ bool first(int w, int& tb, int& te, int& hh, int& c0, int& c1, HeadDesc& d) const {
    const int4 wd0 = ldc(wave_desc, 2 * w), wd1 = ldc(wave_desc, 2 * w + 1);
    tb = ldc(wave_bounds, w);
    te = ldc(wave_bounds, w + 1);
    hh = wd0.z;
    c0 = wd0.w;
    c1 = wd1.x;
    d = make_int4(wd1.y, wd1.z, wd1.w, -1);
    return tb < te;
  }
  __device__ __forceinline__ void next(int& hh, int tb, int& c0, int& c1, HeadDesc& d) const {
    while (ldc(cum, hh + 1) <= tb) ++hh;
    c0 = ldc(cum, hh);
    c1 = ldc(cum, hh + 1);
    d = ldc(desc, hh);
    d.w = -1;   // the planner has written the page table
  }
  __device__ __forceinline__ int4 span(int hh, int) const { return ldc(head_waves, hh); }
};

struct LdsPlan {
  const int* cum;      // [NH + 1]
  const int4* desc;    // [NH]
  int total, W, NH;
  __device__ __forceinline__ int cum_at(int i) const { return __builtin_amdgcn_readfirstlane(cum[i]); }
  __device__ __forceinline__ HeadDesc head(int hh) const {
    const int4 v = desc[hh];
    return make_int4(__builtin_amdgcn_readfirstlane(v.x), __builtin_amdgcn_readfirstlane(v.y),
                     __builtin_amdgcn_readfirstlane(v.z), __builtin_amdgcn_readfirstlane(v.w));
  }
  __device__ __forceinline__ bool first(int w, int& tb, int& te, int& hh, int& c0, int& c1, HeadDesc& d) const {
    tb = wave_start(w, total, W);
    te = wave_start(w + 1, total, W);
    if (tb >= te) return false;
    int lo = 0, hi = NH - 1;   // the head holding tile tb: largest hh with cum[hh] <= tb
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (cum_at(mid) <= tb) lo = mid; else hi = mid - 1;
    }
    hh = lo;
    c0 = cum_at(hh);
    c1 = cum_at(hh + 1);
    d = head(hh);
    return true;
  }
  __device__ __forceinline__ void next(int& hh, int tb, int& c0, int& c1, HeadDesc& d) const {
    while (cum_at(hh + 1) <= tb) ++hh;
    c0 = cum_at(hh);
    c1 = cum_at(hh + 1);
    d = head(hh);
  }
  __device__ __forceinline__ int4 span(int hh, int W_) const {
    return head_span(cum_at(hh), cum_at(hh + 1), total, W_);
  }
};

// Tiles [t_lo, t_hi) of call head hh (descriptor d; `head_end`: the range
// ends with the head's last tile) streamed into acc: query fragments, the
// appended token written into its tile by the wave whose range covers it
// (before the range's loads: same-wave stores and loads to one address stay
// in order), then the tiles, two register sets in flight.
template <int D, bool FP8>
__device__ __forceinline__ void stream_segment(
  Acc<D>& acc, int hh, const HeadDesc& d, int t_lo, int t_hi, bool head_end,
  const int32_t* __restrict__ page_table, const int32_t* __restrict__ qpage, char* __restrict__ pool,
  const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_in, const uint16_t* __restrict__ v_in,
  const DecodeParams& a) {
  const int lane = threadIdx.x & 63;
  const int r = lane & 15, G = lane >> 4;
  const int tiles_per_page_log2 = a.log2P - 5;
  const int L = d.x;
  const int32_t* pt = page_table + static_cast<size_t>(d.y) * a.maxp;
  // page retrieval: the head's tiles run over the physical pages of its
  // selection only
  const int32_t* pages = qpage != nullptr ? qpage + static_cast<size_t>(hh) * a.qB : pt;
  // query fragments (B operand): column r = query head r of the group
  u32x4 qf[D / 32];
  const u32x4 z = {0u, 0u, 0u, 0u};
  const char* qrow = reinterpret_cast<const char*>(q + (static_cast<size_t>(hh) * a.g + r) * D);
#pragma unroll
  for (int s = 0; s < D / 32; ++s) qf[s] = r < a.g ? ldg16(qrow + (32 * s + 8 * G) * 2) : z;
  // the borrowed decision neuron takes no part in attention (App. C)
  if (a.zero_neuron && r == 0 && G == 0) qf[0][0] &= 0xFFFF0000u;
#pragma unroll
  for (int b = 0; b < D / 16; ++b) acc.o[b] = f32x4{0.f, 0.f, 0.f, 0.f};
  acc.m = -INFINITY;
  acc.l = 0.f;
  const int full_hi = (head_end && (L & (kTile - 1))) ? t_hi - 1 : t_hi;
  // tile t of the head: page from a scalar load (the whole wave works on
  // one head), then the tile's 16 KB block inside the page
  constexpr size_t kTileBytes = FP8 ? static_cast<size_t>(D) * 64 + 256 : static_cast<size_t>(D) * 128;
  // a page this call popped (fused launch) is taken from the plan: its
  // page-table entry may not be written yet
  const int new_pi = d.w >= 0 ? (d.z >> 5) >> tiles_per_page_log2 : -1;
  auto tile_in = [&](const int32_t* pl, int t) -> char* {
    const int pi = t >> tiles_per_page_log2;
    const int pg = pi == new_pi ? d.w : ldc(pl, pi);
    return pool + static_cast<size_t>(pg) * a.page_bytes +
           static_cast<size_t>(t & ((1 << tiles_per_page_log2) - 1)) * kTileBytes;
  };
  auto tile_of = [&](int t) -> char* { return tile_in(pages, t); };
  // The token appended by this call (slot d.z) is written into its tile by
  // the one wave whose segment covers that tile, before the segment's
  // loads: same-wave stores and loads to one address stay in order.
  if (k_in != nullptr && d.z >= t_lo * kTile && d.z < t_hi * kTile) {
    char* tile = tile_in(pt, d.z >> 5);
    const int j = d.z & 31;
    if constexpr (FP8) {
      if (lane < D / 8)
        fp8_store_token(tile, j, D, lane, reinterpret_cast<const uint4*>(k_in + static_cast<size_t>(hh) * D)[lane],
                        reinterpret_cast<const uint4*>(v_in + static_cast<size_t>(hh) * D)[lane]);
    } else {
      if (lane < D / 8)
        *reinterpret_cast<u32x4*>(tile + k_elem_off(j, 8 * lane)) =
            reinterpret_cast<const u32x4*>(k_in + static_cast<size_t>(hh) * D)[lane];
#pragma unroll
      for (int e = lane; e < D; e += 64)
        *reinterpret_cast<uint16_t*>(tile + v_elem_off(j, e, D)) = v_in[static_cast<size_t>(hh) * D + e];
    }
  }
  if constexpr (FP8) {
    if (t_lo < full_hi) {
      // two register sets, as for bf16 (a third set, keeping two FP8 tiles
      // in flight, measured slower)
      FragF8<D> fa, fb;
      // the next tile's address is formed a tile ahead and a scheduling
      // barrier keeps its loads ahead of this tile's waits (1.5% faster
      // than leaving the order to the compiler, which waited for part of
      // the current tile first)
      int t = t_lo;
      const int last = full_hi - 1;
      load_tile_f8<D>(fa, tile_of(t), lane, G);
      __builtin_amdgcn_sched_barrier(0);
      const char* pb = tile_of(min(t + 1, last));
      for (; t + 2 < full_hi; t += 2) {
        load_tile_f8<D>(fb, pb, lane, G);
        __builtin_amdgcn_sched_barrier(0);
        const char* pa = tile_of(t + 2);
        compute_tile_f8<D>(acc, fa, qf, a.scale_log2, kTile, G);
        load_tile_f8<D>(fa, pa, lane, G);
        __builtin_amdgcn_sched_barrier(0);
        pb = tile_of(min(t + 3, last));
        compute_tile_f8<D>(acc, fb, qf, a.scale_log2, kTile, G);
      }
      if (t + 1 < full_hi) {
        load_tile_f8<D>(fb, pb, lane, G);
        __builtin_amdgcn_sched_barrier(0);
        compute_tile_f8<D>(acc, fa, qf, a.scale_log2, kTile, G);
        compute_tile_f8<D>(acc, fb, qf, a.scale_log2, kTile, G);
      } else {
        compute_tile_f8<D>(acc, fa, qf, a.scale_log2, kTile, G);
      }
    }
    if (full_hi < t_hi) {
      FragF8<D> ft;
      load_tail_f8<D>(ft, tile_of(full_hi), lane, L - full_hi * kTile, r, G);
      compute_tile_f8<D>(acc, ft, qf, a.scale_log2, L - full_hi * kTile, G);
    }
  } else {
  if (t_lo < full_hi) {
    // Two register sets; the next tile's loads are always in flight while
    // the current one is computed (the prefetch is unconditional inside the
    // loop so the compiler's wait counts only cover the older tile).
    Frag<D> fa, fb;
    int t = t_lo;
    load_tile<D>(fa, tile_of(t), lane);
    for (; t + 2 < full_hi; t += 2) {
      load_tile<D>(fb, tile_of(t + 1), lane);
      compute_tile<D>(acc, fa, qf, a.scale_log2, kTile, G);
      load_tile<D>(fa, tile_of(t + 2), lane);
      compute_tile<D>(acc, fb, qf, a.scale_log2, kTile, G);
    }
    if (t + 1 < full_hi) {
      load_tile<D>(fb, tile_of(t + 1), lane);
      compute_tile<D>(acc, fa, qf, a.scale_log2, kTile, G);
      compute_tile<D>(acc, fb, qf, a.scale_log2, kTile, G);
    } else {
      compute_tile<D>(acc, fa, qf, a.scale_log2, kTile, G);
    }
  }
  if (full_hi < t_hi) {
    Frag<D> ft;
    load_tail<D>(ft, tile_of(full_hi), lane, L - full_hi * kTile, r, G);
    compute_tile<D>(acc, ft, qf, a.scale_log2, L - full_hi * kTile, G);
  }
  }
}

// One decode wave's work: stream its tile range (split-K over the retained
// slots of the heads it covers), write whole heads' outputs, publish partials
// of heads it shares, and merge the heads whose tile count it completes.
template <int D, bool FP8, class Plan>
__device__ __forceinline__ void decode_wave(
    const Plan& plan, int wave, int W, int32_t* __restrict__ head_cnt,
    const int32_t* __restrict__ page_table, const int32_t* __restrict__ qpage,
    char* __restrict__ pool, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_in,
    const uint16_t* __restrict__ v_in, float2* __restrict__ part_ml, float* __restrict__ part_acc,
    float* __restrict__ out, const DecodeParams& a, float (*merge_wts)[kMaxGroup]) {
  const int lane = threadIdx.x & 63;
  const int r = lane & 15, G = lane >> 4;
  int tb, te, hh, c0, c1;
  HeadDesc d;
  if (!plan.first(wave, tb, te, hh, c0, c1, d)) return;
  bool first = true;
  // heads shared with other waves (at most the first and the last segment),
  // published at the end: head, tiles of this wave, tiles of the head
  int p_hh0 = 0, p_cnt0 = 0, p_tot0 = 0, p_hh1 = 0, p_cnt1 = 0, p_tot1 = 0;
  int npend = 0;
  while (tb < te) {
    if (!first) plan.next(hh, tb, c0, c1, d);
    first = false;
    const int seg_end = min(te, c1);
    Acc<D> acc;
    stream_segment<D, FP8>(acc, hh, d, tb - c0, seg_end - c0, seg_end == c1, page_table, qpage, pool, q, k_in,
                           v_in, a);
    float l = acc.l;
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    if (tb == c0 && seg_end == c1) {
      if (r < a.g) {
        const float inv = 1.0f / l;
        float* o = out + (static_cast<size_t>(hh) * a.g + r) * D + 4 * G;
#pragma unroll
        for (int b = 0; b < D / 16; ++b) *reinterpret_cast<f32x4*>(o + 16 * b) = acc.o[b] * inv;
      }
    } else {
      // Split head: publish this wave's partial; the wave that completes the
      // head's tile count merges all partials by log-sum-exp and writes the
      // output.  Partials of head hh come from consecutive waves w, stored at
      // index w + hh.
      // Partials are written and read with agent-coherent (sc1) accesses, so
      // no L2 write-back / invalidate is needed: the stores are complete at
      // the coherence point once vmcnt drains, before the counter is bumped.
      const size_t pid = static_cast<size_t>(wave) + hh;
      const __amdgpu_buffer_rsrc_t acc_rsrc = __builtin_amdgcn_make_buffer_rsrc(
          part_acc, static_cast<short>(0), a.part_acc_bytes, kBufferDword3);
      if (r < a.g) {
        float* ml = reinterpret_cast<float*>(part_ml + pid * kMaxGroup + r);
        if (G == 0) {
          store_coherent(ml, acc.m);
          store_coherent(ml + 1, l);
        }
        const uint32_t o = static_cast<uint32_t>(((pid * a.g + r) * D + 4 * G) * 4);
#pragma unroll
        for (int b = 0; b < D / 16; ++b)
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc.o[b]), acc_rsrc,
                                                 o + 64 * b, 0, kCachePolicySc1);
      }
      if (npend == 0) {
        p_hh0 = hh;
        p_cnt0 = seg_end - tb;
        p_tot0 = c1 - c0;
      } else {
        p_hh1 = hh;
        p_cnt1 = seg_end - tb;
        p_tot1 = c1 - c0;
      }
      ++npend;
    }
    tb = seg_end;
    ++hh;
  }
  // Heads shared with other waves (at most the first and the last segment):
  // once this wave's partial stores are complete, add its tile counts to
  // the heads' arrival counters; the wave that completes a head's count
  // merges all its partials by log-sum-exp and writes the output.  Deferring
  // this to the end of the range keeps the tile stream free of waits.  In
  // a planned launch (defer_merge) the merges run after it instead.
  if (npend > 0 && !a.defer_merge) {
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    int prev = 0;
    if (lane < npend) prev = atomicAdd(&head_cnt[lane == 0 ? p_hh0 : p_hh1], lane == 0 ? p_cnt0 : p_cnt1);
    const int prev0 = __shfl(prev, 0, 64), prev1 = __shfl(prev, 1, 64);
    const __amdgpu_buffer_rsrc_t acc_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        part_acc, static_cast<short>(0), a.part_acc_bytes, kBufferDword3);
    for (int i = 0; i < npend; ++i) {
      if (i == 0 ? prev0 + p_cnt0 != p_tot0 : prev1 + p_cnt1 != p_tot1) continue;
      const int mh = i == 0 ? p_hh0 : p_hh1;
      const int4 hw = plan.span(mh, W);   // waves wf .. wl hold the head's tiles
      const int wf = hw.x, wl = hw.y;
      if (wl - wf < 4)
        merge_head_small<D>(part_ml, acc_rsrc, hw.z, out, wf, wl - wf + 1, mh, a.g, lane);
      else
        merge_head_any<D>(part_ml, acc_rsrc, plan.total, W, out, wf, wl, mh, a.g, lane, merge_wts);
      if (lane == 0) __hip_atomic_store(&head_cnt[mh], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Decode launch after the planning kernel (workspace plan).
template <int D, bool FP8>
__global__ __launch_bounds__(256, 1) void decode_kernel(
    const int32_t* __restrict__ status, const HeadDesc* __restrict__ desc,
    const int32_t* __restrict__ cum_tiles, const int32_t* __restrict__ wave_bounds,
    const int4* __restrict__ wave_desc, const int4* __restrict__ head_waves,
    int32_t* __restrict__ head_cnt,
    const int32_t* __restrict__ page_table, const int32_t* __restrict__ qpage,
    char* __restrict__ pool, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_in,
    const uint16_t* __restrict__ v_in, float2* __restrict__ part_ml, float* __restrict__ part_acc,
    float* __restrict__ out, DecodeParams a) {
  __shared__ float merge_wts[kWavesPerBlock][kMergeBatch][kMaxGroup];
  if (load_status(status) != 0) return;
  // wave index is uniform across the wave; say so, so that everything derived
  // from it (head, tile, page) lives in scalar registers
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const GlobalPlan plan{desc, cum_tiles, wave_bounds, wave_desc, head_waves, ldc(cum_tiles, a.NH)};
  decode_wave<D, FP8>(plan, blockIdx.x * kWavesPerBlock + wid, a.W, head_cnt, page_table, qpage,
                      pool, q, k_in, v_in, part_ml, part_acc, out, a, merge_wts[wid]);
}

// ---------------------------------------------------------------------------
// Fused decode step: append planning inside the decode launch
// ---------------------------------------------------------------------------

constexpr int kFuseMaxHeads = 1024;   // call heads a fused launch plans in LDS
constexpr int kFuseHeadsPerThread = kFuseMaxHeads / 256;

struct FusedArgs {
  LayerState st;
  int32_t* status;
  const int32_t* seq_ids;
  const uint8_t* flags;    // [n, H] caller decisions, or null (decisions from q)
  const uint16_t* q_dec;   // queries for the borrowed-neuron decisions, or null
  uint8_t* flags_out;      // nullable: decisions taken from q
  int32_t* plan_ctr;       // workgroups of this launch that have read the state
  float bias;
  int immediate, n, H, w, P, maxp, max_slots, max_seqs, g, D;
};

// Rule R1 for one appended token per (sequence, KV head) of the call, done by
// every workgroup of the launch into its LDS: each head's slot (the slot of
// the token w positions back when that one leaves the cache, else the next
// fresh one), the pages popped in call order, the retained lengths and the
// tile prefix sums of the work split.  The loads form three dependent rounds
// (sequence ids and decisions; positions and lengths, issued for clamped ids
// before the ids are validated; ring entries and stack).  Nothing is written
// to the state here: once a workgroup has read it, its first thread adds one
// to a launch counter in the workspace without waiting for the result, and
// the workgroup whose add completes the count writes the new state after its
// decode work (write_state), when every other workgroup has finished reading.
// Returns false in every thread when the call does nothing (a sticky error was
// set before, or this call sets one; all workgroups take the same decision
// from the same data).  *total gets the call's tile count, *new_top the stack
// height after the call's pops; *ticket, in thread 0, the counter value before
// its add.
__device__ __forceinline__ bool fused_plan(const FusedArgs& f, int* s_cum, int4* s_desc, int2* s_aux,
                                           uint32_t* s_seen, int32_t* s_stack, int* s_scan,
                                           int* total, int* ticket, int* new_top) {
  const int tid = threadIdx.x;
  const int NH = f.n * f.H;
  // round 1: status and stack height (one thread reads them for the whole
  // workgroup: another workgroup may set the status meanwhile, and every
  // thread must take the same exit), sequence ids, decisions
  if (tid == 0) {
    s_scan[0] = load_status(f.status);
    s_scan[1] = *f.st.top;
  }
  for (int i = tid; i < ((f.max_seqs + 31) >> 5); i += blockDim.x) s_seen[i] = 0;
  int seq[kFuseHeadsPerThread], dec[kFuseHeadsPerThread], pos[kFuseHeadsPerThread];
  int L[kFuseHeadsPerThread];
#pragma unroll
  for (int k = 0; k < kFuseHeadsPerThread; ++k) {
    const int hh = kFuseHeadsPerThread * tid + k;
    seq[k] = hh < NH ? f.seq_ids[hh / f.H] : 0;
    dec[k] = hh < NH ? token_decision(f.flags, f.q_dec, hh, f.H, f.g, f.D, f.bias) : 0;
  }
  // round 2, issued before the ids are validated (clamped into range; the
  // values are only used once the ids are known to be valid)
#pragma unroll
  for (int k = 0; k < kFuseHeadsPerThread; ++k) {
    const int hh = kFuseHeadsPerThread * tid + k;
    const int s = min(max(seq[k], 0), f.max_seqs - 1);
    pos[k] = hh < NH ? f.st.pos[s] : 0;
    L[k] = hh < NH ? f.st.len[s * f.H + hh % f.H] : 0;
  }
  __syncthreads();
  const int status = s_scan[0];
  const int top0 = s_scan[1];
  // sequence ids in range and not repeated
  int bad = 0;
  if (status == 0) {
#pragma unroll
    for (int k = 0; k < kFuseHeadsPerThread; ++k) {
      const int hh = kFuseHeadsPerThread * tid + k;
      if (hh < NH && hh % f.H == 0) {
        const int s = seq[k];
        if (s < 0 || s >= f.max_seqs) {
          bad = 1;
        } else {
          const uint32_t bit = 1u << (s & 31);
          if (atomicOr(&s_seen[s >> 5], bit) & bit) bad = 1;
        }
      }
    }
  }
  bad = __syncthreads_or(bad);   // also orders s_scan's reads above before its reuse
  if (status != 0) return false;
  if (bad) {
    if (tid == 0) set_status(f.status, DMS_ERR_BAD_SEQ);
    return false;
  }
  // round 3: ring entries, and the pages this call may pop in pop order
  for (int i = tid; i < min(NH, top0); i += blockDim.x) s_stack[i] = f.st.stack[top0 - 1 - i];
  int sh[kFuseHeadsPerThread], slot[kFuseHeadsPerThread], fresh[kFuseHeadsPerThread];
  int need[kFuseHeadsPerThread];
  int cap = 0, my_need = 0, my_tiles = 0;
#pragma unroll
  for (int k = 0; k < kFuseHeadsPerThread; ++k) {
    const int hh = kFuseHeadsPerThread * tid + k;
    sh[k] = slot[k] = fresh[k] = need[k] = 0;
    if (hh < NH) {
      sh[k] = seq[k] * f.H + hh % f.H;
      const int32_t e = f.st.ring[static_cast<size_t>(sh[k]) * f.w + pos[k] % f.w];
      const bool reuse = takes_old_slot(pos[k], f.w, e, dec[k], f.immediate);
      slot[k] = reuse ? static_cast<int>(static_cast<uint32_t>(e) & ~kFlagBit) : L[k];
      fresh[k] = !reuse;
      cap |= fresh[k] && slot[k] >= f.max_slots;
      need[k] = fresh[k] && (slot[k] % f.P) == 0;
      L[k] += fresh[k];
    }
    my_need += need[k];
    my_tiles += (L[k] + kTile - 1) / kTile;
  }
  int2 tot;
  const int2 ex = block_exclusive_scan2(make_int2(my_need, my_tiles), s_scan, &tot);
  cap = __syncthreads_or(cap);
  if (cap || tot.x > top0) {
    if (tid == 0) set_status(f.status, cap ? DMS_ERR_CAPACITY : DMS_ERR_OUT_OF_PAGES);
    return false;
  }
  int pop = ex.x, ct = ex.y;
#pragma unroll
  for (int k = 0; k < kFuseHeadsPerThread; ++k) {
    const int hh = kFuseHeadsPerThread * tid + k;
    if (hh < NH) {
      const int pg = need[k] ? s_stack[pop] : -1;
      pop += need[k];
      ct += (L[k] + kTile - 1) / kTile;
      s_desc[hh] = make_int4(L[k], sh[k], slot[k], pg);
      s_aux[hh] = make_int2(pos[k], dec[k] | (fresh[k] << 1));
      s_cum[hh + 1] = ct;
    }
  }
  if (tid == 0) s_cum[0] = 0;
  *total = tot.y;
  *new_top = top0 - tot.x;
  // every load of the state above has returned (its values are in LDS or
  // registers): count this workgroup as done reading; the last to count
  // writes the new state
  __syncthreads();
  if (tid == 0) *ticket = atomicAdd(f.plan_ctr, 1);
  return true;
}

// The new state of the call's heads (one wave of the workgroup that read the
// state last): rings, slot owners, lengths, new page-table entries, positions,
// stack height, decisions taken; then the launch counter is reset.
__device__ __forceinline__ void write_state(const FusedArgs& f, const int4* s_desc, const int2* s_aux,
                                            int top0_minus_pops, int lane) {
  const int NH = f.n * f.H;
  for (int hh = lane; hh < NH; hh += 64) {
    const int4 d = s_desc[hh];       // Lnew, state head, slot, page popped (-1: none)
    const int2 x = s_aux[hh];        // position, decision | fresh << 1
    const int dec = x.y & 1;
    const uint32_t fb = dec ? kFlagBit : 0u;
    if (f.flags_out != nullptr) f.flags_out[hh] = static_cast<uint8_t>(dec);
    if (d.w >= 0) f.st.page_table[static_cast<size_t>(d.y) * f.maxp + d.z / f.P] = d.w;
    if (x.y & 2) f.st.len[d.y] = d.x;
    f.st.ring[static_cast<size_t>(d.y) * f.w + x.x % f.w] = static_cast<int32_t>(static_cast<uint32_t>(d.z) | fb);
    f.st.slot_meta[static_cast<size_t>(d.y) * f.max_slots + d.z] = static_cast<int32_t>(static_cast<uint32_t>(x.x) | fb);
    if (hh % f.H == 0) f.st.pos[f.seq_ids[hh / f.H]] = x.x + 1;
  }
  if (lane == 0) {
    *f.st.top = top0_minus_pops;
    __hip_atomic_store(f.plan_ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Calls whose every head has at most kHeadBlockTiles tiles run S workgroups
// per head (S = 1 .. kHeadBlockParts, as many as the launch has workgroups
// for): workgroup s takes the s-th of S contiguous parts of the head's
// tiles, its four waves quarters of that part, and the waves fold their
// results through LDS.  With S = 1 the fold writes the output: no split-K
// partial goes through memory and no arrival counter is taken.  Measured at
// a 1.5B-shaped step (64 heads of ~40 tiles spread over ~320 waves) the
// per-wave global merges -- partial stores, the arrival atomic, then the
// merging wave's coherent loads -- held the launch for up to 18 us of its
// 36.  With S > 1 each workgroup publishes one folded partial and the last
// of the S merges them (at most four partials, one coherent round trip).
constexpr int kHeadBlockTiles = 64;
constexpr int kHeadBlockParts = 4;

template <int D, bool FP8>
__device__ __forceinline__ void decode_head_block(const LdsPlan& plan, int hh, int S, int s,
                                                  const int32_t* __restrict__ page_table,
                                                  char* __restrict__ pool, const uint16_t* __restrict__ q,
                                                  const uint16_t* __restrict__ k_in, const uint16_t* __restrict__ v_in,
                                                  int32_t* __restrict__ head_cnt, float2* __restrict__ part_ml,
                                                  float* __restrict__ part_acc, float* __restrict__ out,
                                                  const DecodeParams& a, f32x4 (*fold)[D / 16][64],
                                                  float2 (*fold_ml)[kMaxGroup]) {
  const int lane = threadIdx.x & 63;
  const int r = lane & 15, G = lane >> 4;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c0 = plan.cum_at(hh), c1 = plan.cum_at(hh + 1);
  const int n = c1 - c0;
  const HeadDesc d = plan.head(hh);
  // this workgroup's part of the head's tiles, then this wave's quarter of it
  const int p_lo = s * n / S, p_hi = (s + 1) * n / S;
  const int t_lo = p_lo + wid * (p_hi - p_lo) / kWavesPerBlock;
  const int t_hi = p_lo + (wid + 1) * (p_hi - p_lo) / kWavesPerBlock;
  Acc<D> acc;
  if (t_lo < t_hi) {
    stream_segment<D, FP8>(acc, hh, d, t_lo, t_hi, t_hi == n, page_table, nullptr, pool, q, k_in, v_in, a);
  } else {
#pragma unroll
    for (int b = 0; b < D / 16; ++b) acc.o[b] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc.m = -INFINITY;
    acc.l = 0.f;
  }
  float l = acc.l;
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
#pragma unroll
  for (int b = 0; b < D / 16; ++b) fold[wid][b][lane] = acc.o[b];
  if (G == 0) fold_ml[wid][r] = make_float2(acc.m, l);
  __syncthreads();
  // wave wid folds row blocks wid * D/64 .. of the four waves' results
  float mj[kWavesPerBlock], M = -INFINITY;
#pragma unroll
  for (int j = 0; j < kWavesPerBlock; ++j) {
    mj[j] = fold_ml[j][r].x;
    M = fmaxf(M, mj[j]);
  }
  float den = 0.f, wj[kWavesPerBlock];
#pragma unroll
  for (int j = 0; j < kWavesPerBlock; ++j) {
    // 0 for a wave without tiles (m = -inf); a part without tiles (S > 1,
    // fewer tiles than parts) folds to m = -inf, l = 0, accumulators 0
    wj[j] = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mj[j] - M);
    den += wj[j] * fold_ml[j][r].y;
  }
  constexpr int kBlocks = D / 16 / kWavesPerBlock;
  if (S == 1) {
    if (r < a.g) {
      const float inv = 1.0f / den;
      float* o = out + (static_cast<size_t>(hh) * a.g + r) * D + 4 * G;
#pragma unroll
      for (int i = 0; i < kBlocks; ++i) {
        const int b = wid * kBlocks + i;
        f32x4 num = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < kWavesPerBlock; ++j) num += wj[j] * fold[j][b][lane];
        *reinterpret_cast<f32x4*>(o + 16 * b) = num * inv;
      }
    }
    return;
  }
  // Part s of S: publish the folded partial (max, denominator, unnormalized
  // accumulators) at index hh * S + s with agent-coherent stores; once every
  // wave's stores are complete, count the part in; the workgroup that
  // completes the count merges the S partials.
  const size_t pid = static_cast<size_t>(hh) * S + s;
  const __amdgpu_buffer_rsrc_t acc_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      part_acc, static_cast<short>(0), a.part_acc_bytes, kBufferDword3);
  if (r < a.g) {
    if (wid == 0 && G == 0) {
      float* ml = reinterpret_cast<float*>(part_ml + pid * kMaxGroup + r);
      store_coherent(ml, M);
      store_coherent(ml + 1, den);
    }
    const uint32_t o = static_cast<uint32_t>(((pid * a.g + r) * D + 4 * G) * 4);
#pragma unroll
    for (int i = 0; i < kBlocks; ++i) {
      const int b = wid * kBlocks + i;
      f32x4 num = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < kWavesPerBlock; ++j) num += wj[j] * fold[j][b][lane];
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, num), acc_rsrc, o + 64 * b, 0,
                                             kCachePolicySc1);
    }
  }
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  __syncthreads();
  if (wid == 0) {
    int prev = 0;
    if (lane == 0) prev = atomicAdd(&head_cnt[hh], 1);
    prev = __shfl(prev, 0, 64);
    if (prev == S - 1) {
      // partial u of the head sits at index (wf + u) + hh = hh * S + u
      merge_head_small<D>(part_ml, acc_rsrc, (1 << S) - 1, out, hh * S - hh, S, hh, a.g, lane);
      if (lane == 0) __hip_atomic_store(&head_cnt[hh], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Decode waves of a fused launch: at least kFuseMinTiles tiles per wave and at
// least one wave per workgroup (so every compute unit streams), at most all
// resident waves.  Fewer, longer waves split small calls into fewer parts.
constexpr int kFuseMinTiles = 8;

// dms_decode_step in one launch (calls of up to kFuseMaxHeads heads without
// page retrieval): fused planning, then the decode waves.  With fewer active
// waves than resident ones, logical wave lw runs as wave lw / B of workgroup
// lw % B (B workgroups), spreading the active waves over all compute units.
template <int D, bool FP8>
__global__ __launch_bounds__(256, 1) void decode_step_kernel(
    FusedArgs f, int32_t* __restrict__ head_cnt, char* __restrict__ pool,
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_in,
    const uint16_t* __restrict__ v_in, float2* __restrict__ part_ml, float* __restrict__ part_acc,
    float* __restrict__ out, DecodeParams a) {
  __shared__ float merge_wts[kWavesPerBlock][kMergeBatch][kMaxGroup];
  __shared__ int s_cum[kFuseMaxHeads + 1];
  __shared__ int4 s_desc[kFuseMaxHeads];
  __shared__ int2 s_aux[kFuseMaxHeads];
  __shared__ uint32_t s_seen[kMaxSeqs / 32];
  __shared__ int32_t s_stack[kFuseMaxHeads];
  __shared__ int s_scan[34];
  __shared__ f32x4 s_fold[kWavesPerBlock][D / 16][64];
  __shared__ float2 s_fold_ml[kWavesPerBlock][kMaxGroup];
  int total = 0, ticket = 0, new_top = 0;
  if (!fused_plan(f, s_cum, s_desc, s_aux, s_seen, s_stack, s_scan, &total, &ticket, &new_top)) return;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nb = gridDim.x;
  const int T = __builtin_amdgcn_readfirstlane(total);
  // every workgroup takes the same decision from the same plan
  int wide = 0;
  for (int hh = threadIdx.x; hh < a.NH; hh += blockDim.x) wide |= s_cum[hh + 1] - s_cum[hh] > kHeadBlockTiles;
  wide = __syncthreads_or(wide);
  if (!wide && a.NH <= nb) {
    const int S = min(kHeadBlockParts, nb / a.NH);
    if (static_cast<int>(blockIdx.x) < a.NH * S)
      decode_head_block<D, FP8>(LdsPlan{s_cum, s_desc, T, 1, a.NH}, blockIdx.x / S, S, blockIdx.x % S,
                                f.st.page_table, pool, q, k_in, v_in, head_cnt, part_ml, part_acc, out, a, s_fold,
                                s_fold_ml);
  } else {
    const int W = min(a.W, max(nb, (T + kFuseMinTiles - 1) / kFuseMinTiles));
    const int lw = W == a.W ? blockIdx.x * kWavesPerBlock + wid : wid * nb + blockIdx.x;
    const LdsPlan plan{s_cum, s_desc, T, W, a.NH};
    if (lw < W)
      decode_wave<D, FP8>(plan, lw, W, head_cnt, f.st.page_table, nullptr, pool, q, k_in, v_in,
                          part_ml, part_acc, out, a, merge_wts[wid]);
  }
  // the workgroup whose count completed the launch's writes the new state
  if (wid == 0 && __shfl(ticket, 0, 64) == nb - 1) write_state(f, s_desc, s_aux, new_top, threadIdx.x & 63);
}

// Split heads of a planned decode launch, merged after it: one wave per call
// head whose tiles span several waves; its partials are complete and visible
// at the launch boundary.  Merging inside the decode launch put the merges'
// coherent loads behind the stream's requests in the memory queues: at the
// 32B-shaped stress step a merge after its arrival count took 7-25 us while
// the count itself took ~1 us.
template <int D>
__global__ __launch_bounds__(256) void merge_kernel(const int32_t* __restrict__ status,
                                                    const int32_t* __restrict__ cum_tiles,
                                                    const int4* __restrict__ head_waves,
                                                    const float2* __restrict__ part_ml, float* __restrict__ part_acc,
                                                    float* __restrict__ out, DecodeParams a) {
  __shared__ float merge_wts[kWavesPerBlock][kMergeBatch][kMaxGroup];
  if (load_status(status) != 0) return;
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int hh = blockIdx.x * kWavesPerBlock + wid;
  if (hh >= a.NH) return;
  if (ldc(cum_tiles, hh + 1) <= ldc(cum_tiles, hh)) return;   // no tiles (the planner zeroed its output)
  const int4 hw = ldc(head_waves, hh);
  const int wf = hw.x, wl = hw.y;
  if (wf == wl) return;   // one wave held the whole head and wrote its output
  const __amdgpu_buffer_rsrc_t acc_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      part_acc, static_cast<short>(0), a.part_acc_bytes, kBufferDword3);
  if (wl - wf < 4)
    merge_head_small<D>(part_ml, acc_rsrc, hw.z, out, wf, wl - wf + 1, hh, a.g, lane);
  else
    merge_head_any<D>(part_ml, acc_rsrc, ldc(cum_tiles, a.NH), a.W, out, wf, wl, hh, a.g, lane, merge_wts[wid]);
}

// Decode over Quest's selection (page retrieval) with the work split planned
// in every workgroup: the tile prefix sums over the call's attended lengths
// (qlen) and the head descriptors go to LDS, then the waves decode as with
// the planner's split.  Replaces the planner launch between the selection and
// the decode for calls of up to kFuseMaxHeads heads.
template <int D, bool FP8>
__global__ __launch_bounds__(256, 1) void decode_attended_kernel(
    const int32_t* __restrict__ status, const HeadDesc* __restrict__ desc, const int32_t* __restrict__ qlen,
    int32_t* __restrict__ head_cnt, const int32_t* __restrict__ page_table, const int32_t* __restrict__ qpage,
    char* __restrict__ pool, const uint16_t* __restrict__ q, float2* __restrict__ part_ml,
    float* __restrict__ part_acc, float* __restrict__ out, DecodeParams a) {
  __shared__ float merge_wts[kWavesPerBlock][kMergeBatch][kMaxGroup];
  __shared__ int s_cum[kFuseMaxHeads + 1];
  __shared__ int4 s_desc[kFuseMaxHeads];
  __shared__ int s_scan[17];
  if (load_status(status) != 0) return;
  constexpr int kPer = kFuseMaxHeads / 256;   // heads per thread
  const int tid = threadIdx.x;
  const int NH = a.NH;
  int len[kPer], sh[kPer], mine = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int hh = kPer * tid + k;
    len[k] = hh < NH ? qlen[hh] : 0;
    sh[k] = hh < NH ? desc[hh].y : 0;   // state head (the append plan's descriptor)
  }
#pragma unroll
  for (int k = 0; k < kPer; ++k) mine += (len[k] + kTile - 1) / kTile;
  int total = 0;
  int c = block_exclusive_scan(mine, s_scan, &total);
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int hh = kPer * tid + k;
    if (hh < NH) {
      c += (len[k] + kTile - 1) / kTile;
      s_cum[hh + 1] = c;
      s_desc[hh] = make_int4(len[k], sh[k], -1, -1);   // no appended slot, no pending page
      // a head that attends nothing (never after an append) gets zero rows
      if (len[k] == 0 && blockIdx.x == 0)
        for (int e = 0; e < a.g * D; ++e) out[static_cast<size_t>(hh) * a.g * D + e] = 0.f;
    }
  }
  if (tid == 0) s_cum[0] = 0;
  __syncthreads();
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const LdsPlan plan{s_cum, s_desc, __builtin_amdgcn_readfirstlane(total), a.W, NH};
  decode_wave<D, FP8>(plan, blockIdx.x * kWavesPerBlock + wid, a.W, head_cnt, page_table, qpage, pool, q,
                      nullptr, nullptr, part_ml, part_acc, out, a, merge_wts[wid]);
}

DecodeParams decode_params(const dms_config& c, const Layout& lo, int D, int n, int waves) {
  DecodeParams a;
  a.page_bytes = lo.page_bytes;
  a.part_acc_bytes = static_cast<int>(static_cast<size_t>(lo.max_partials) * c.group_size * D * 4);
  a.NH = n * c.num_kv_heads;
  a.g = c.group_size;
  a.maxp = c.max_pages_per_head;
  a.P = c.page_size;
  a.log2P = __builtin_ctz(static_cast<unsigned>(c.page_size));
  a.W = waves;
  a.zero_neuron = c.decision_source == DMS_DECIDE_QUERY;
  a.qB = c.quest_page_budget;
  a.scale_log2 = c.softmax_scale * 1.4426950408889634f;
  a.defer_merge = 0;
  return a;
}

template <int D, bool FP8>
hipError_t launch_decode_step_d(const dms_config& c, const Layout& lo, void* meta, void* ws,
                                void* pool, int layer, int n, const int32_t* seq_ids,
                                const uint8_t* flags, const void* q, const void* k, const void* v,
                                uint8_t* flags_out, float* out, int waves, hipStream_t st,
                                hipEvent_t ev_start, hipEvent_t ev_stop) {
  char* w = static_cast<char*>(ws);
  FusedArgs f;
  f.st = layer_state(lo, meta, layer);
  f.status = reinterpret_cast<int32_t*>(static_cast<char*>(meta) + lo.status);
  f.seq_ids = seq_ids;
  const bool from_q = c.decision_source == DMS_DECIDE_QUERY;
  f.flags = from_q ? nullptr : flags;
  f.q_dec = from_q ? static_cast<const uint16_t*>(q) : nullptr;
  f.flags_out = flags_out;
  f.plan_ctr = reinterpret_cast<int32_t*>(w + lo.ws_plan_ctr);
  f.bias = c.decision_bias;
  f.immediate = c.eviction == DMS_EVICT_IMMEDIATE;
  f.n = n;
  f.H = c.num_kv_heads;
  f.w = c.window;
  f.P = c.page_size;
  f.maxp = c.max_pages_per_head;
  f.max_slots = lo.max_slots;
  f.max_seqs = c.max_seqs;
  f.g = c.group_size;
  f.D = D;
  const DecodeParams a = decode_params(c, lo, D, n, waves);
  if (ev_start) (void)hipEventRecord(ev_start, st);
  hipLaunchKernelGGL((decode_step_kernel<D, FP8>), dim3(waves / kWavesPerBlock), dim3(256), 0, st, f,
                     reinterpret_cast<int32_t*>(w + lo.ws_head_cnt), static_cast<char*>(pool),
                     static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                     static_cast<const uint16_t*>(v), reinterpret_cast<float2*>(w + lo.ws_part_ml),
                     reinterpret_cast<float*>(w + lo.ws_part_acc), out, a);
  hipError_t e = hipGetLastError();
  if (ev_stop) (void)hipEventRecord(ev_stop, st);
  return e;
}

template <int D, bool FP8>
hipError_t launch_decode_d(const dms_config& c, const Layout& lo, void* meta, void* ws, void* pool,
                           int layer, int n, const void* q, const void* k, const void* v, float* out,
                           int waves, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop,
                           const int32_t* qpage) {
  char* w = static_cast<char*>(ws);
  const int32_t* status = reinterpret_cast<const int32_t*>(static_cast<char*>(meta) + lo.status);
  const int32_t* cum = reinterpret_cast<const int32_t*>(w + lo.ws_cum_tiles);
  float2* part_ml = reinterpret_cast<float2*>(w + lo.ws_part_ml);
  float* part_acc = reinterpret_cast<float*>(w + lo.ws_part_acc);
  DecodeParams a = decode_params(c, lo, D, n, waves);
  a.defer_merge = 1;
  if (ev_start) (void)hipEventRecord(ev_start, st);
  hipLaunchKernelGGL((decode_kernel<D, FP8>), dim3(waves / kWavesPerBlock), dim3(256), 0, st, status,
                     reinterpret_cast<const HeadDesc*>(w + lo.ws_head_desc), cum,
                     reinterpret_cast<const int32_t*>(w + lo.ws_wave_bounds),
                     reinterpret_cast<const int4*>(w + lo.ws_wave_desc),
                     reinterpret_cast<const int4*>(w + lo.ws_head_waves),
                     reinterpret_cast<int32_t*>(w + lo.ws_head_cnt),
                     layer_state(lo, meta, layer).page_table, qpage, static_cast<char*>(pool),
                     static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                     static_cast<const uint16_t*>(v), part_ml, part_acc, out, a);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) {
    hipLaunchKernelGGL((merge_kernel<D>), dim3((a.NH + kWavesPerBlock - 1) / kWavesPerBlock), dim3(256), 0, st,
                       status, cum, reinterpret_cast<const int4*>(w + lo.ws_head_waves), part_ml, part_acc, out, a);
    e = hipGetLastError();
  }
  if (ev_stop) (void)hipEventRecord(ev_stop, st);
  return e;
}

}  // namespace

hipError_t launch_decode(const dms_config& c, const Layout& lo, void* meta, void* ws, void* pool,
                         int layer, int n, const void* q, const void* k, const void* v, float* out,
                         int waves, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop,
                         const int32_t* qpage) {
  if (c.kv_format == DMS_KV_MLA)
    return launch_decode_mla(c, lo, meta, ws, pool, layer, n, q, k, out, waves, st, ev_start, ev_stop);
  const bool fp8 = c.kv_format == DMS_KV_FP8;
  if (c.head_dim == 128)
    return fp8 ? launch_decode_d<128, true>(c, lo, meta, ws, pool, layer, n, q, k, v, out, waves, st,
                                            ev_start, ev_stop, qpage)
               : launch_decode_d<128, false>(c, lo, meta, ws, pool, layer, n, q, k, v, out, waves, st,
                                             ev_start, ev_stop, qpage);
  return fp8 ? launch_decode_d<64, true>(c, lo, meta, ws, pool, layer, n, q, k, v, out, waves, st,
                                         ev_start, ev_stop, qpage)
             : launch_decode_d<64, false>(c, lo, meta, ws, pool, layer, n, q, k, v, out, waves, st,
                                          ev_start, ev_stop, qpage);
}

template <int D, bool FP8>
hipError_t launch_decode_attended_d(const dms_config& c, const Layout& lo, void* meta, void* ws, void* pool,
                                    int layer, int n, const void* q, float* out, int waves, hipStream_t st,
                                    hipEvent_t ev_start, hipEvent_t ev_stop, const int32_t* qpage,
                                    const int32_t* qlen) {
  char* w = static_cast<char*>(ws);
  const DecodeParams a = decode_params(c, lo, D, n, waves);
  if (ev_start) (void)hipEventRecord(ev_start, st);
  hipLaunchKernelGGL((decode_attended_kernel<D, FP8>), dim3(waves / kWavesPerBlock), dim3(256), 0, st,
                     reinterpret_cast<const int32_t*>(static_cast<char*>(meta) + lo.status),
                     reinterpret_cast<const HeadDesc*>(w + lo.ws_head_desc), qlen,
                     reinterpret_cast<int32_t*>(w + lo.ws_head_cnt), layer_state(lo, meta, layer).page_table, qpage,
                     static_cast<char*>(pool), static_cast<const uint16_t*>(q),
                     reinterpret_cast<float2*>(w + lo.ws_part_ml), reinterpret_cast<float*>(w + lo.ws_part_acc),
                     out, a);
  hipError_t e = hipGetLastError();
  if (ev_stop) (void)hipEventRecord(ev_stop, st);
  return e;
}

int decode_attended_max_heads() { return kFuseMaxHeads; }

hipError_t launch_decode_attended(const dms_config& c, const Layout& lo, void* meta, void* ws, void* pool,
                                  int layer, int n, const void* q, float* out, int waves, hipStream_t st,
                                  hipEvent_t ev_start, hipEvent_t ev_stop, const int32_t* qpage,
                                  const int32_t* qlen) {
  const bool fp8 = c.kv_format == DMS_KV_FP8;
  if (c.head_dim == 128)
    return fp8 ? launch_decode_attended_d<128, true>(c, lo, meta, ws, pool, layer, n, q, out, waves, st, ev_start,
                                                     ev_stop, qpage, qlen)
               : launch_decode_attended_d<128, false>(c, lo, meta, ws, pool, layer, n, q, out, waves, st, ev_start,
                                                      ev_stop, qpage, qlen);
  return fp8 ? launch_decode_attended_d<64, true>(c, lo, meta, ws, pool, layer, n, q, out, waves, st, ev_start,
                                                  ev_stop, qpage, qlen)
             : launch_decode_attended_d<64, false>(c, lo, meta, ws, pool, layer, n, q, out, waves, st, ev_start,
                                                   ev_stop, qpage, qlen);
}

// Calls of at most this many KV heads take the fused launch.  Measured on
// MI355X (step time, fused / planner + decode): 1.5B-shaped 32 x 2 heads 1.00
// / 1.15 ms (the fused launch also splits the call over fewer, longer waves,
// so heads are merged from ~6 partials instead of ~16-33); 7B-shaped 64 x 4
// heads 3.75 / 3.71 ms; 32B-shaped 128 x 8 heads 24.36 / 24.37 ms.  The
// in-kernel planning costs about what the planning kernel does (three
// dependent rounds of loads of cold state, ~8-10 us), so it only pays where
// the smaller split does.
constexpr int kFuseCallHeads = 128;

bool decode_step_fusable(const dms_config& c, int n) {
  static_assert(kFuseCallHeads <= kFuseMaxHeads, "fused calls are planned in LDS");
  return c.kv_format != DMS_KV_MLA && c.quest_page_budget == 0 &&
         static_cast<int64_t>(n) * c.num_kv_heads <= kFuseCallHeads;
}

hipError_t launch_decode_step(const dms_config& c, const Layout& lo, void* meta, void* ws, void* pool,
                              int layer, int n, const int32_t* seq_ids, const uint8_t* flags,
                              const void* q, const void* k, const void* v, uint8_t* flags_out,
                              float* out, int waves, hipStream_t st, hipEvent_t ev_start,
                              hipEvent_t ev_stop) {
  const bool fp8 = c.kv_format == DMS_KV_FP8;
  if (c.head_dim == 128)
    return fp8 ? launch_decode_step_d<128, true>(c, lo, meta, ws, pool, layer, n, seq_ids, flags, q, k, v,
                                                 flags_out, out, waves, st, ev_start, ev_stop)
               : launch_decode_step_d<128, false>(c, lo, meta, ws, pool, layer, n, seq_ids, flags, q, k, v,
                                                  flags_out, out, waves, st, ev_start, ev_stop);
  return fp8 ? launch_decode_step_d<64, true>(c, lo, meta, ws, pool, layer, n, seq_ids, flags, q, k, v,
                                              flags_out, out, waves, st, ev_start, ev_stop)
             : launch_decode_step_d<64, false>(c, lo, meta, ws, pool, layer, n, seq_ids, flags, q, k, v,
                                               flags_out, out, waves, st, ev_start, ev_stop);
}

// One decode wave per SIMD (a block of 4 waves per CU).  Measured on MI355X
// at the Qwen-R1-32B-shaped workload this beats two per SIMD (fewer split
// heads to merge, same bandwidth); the launch must fit entirely, so the
// occupancy of the kernel is checked.
int decode_resident_waves(const dms_config& c) {
  if (c.kv_format == DMS_KV_MLA) return decode_mla_resident_waves(c);
  int dev = 0, cus = 0, blocks = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
  const bool fp8 = c.kv_format == DMS_KV_FP8;
  hipError_t e = c.head_dim == 128
      ? (fp8 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, decode_kernel<128, true>, 256, 0)
             : hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, decode_kernel<128, false>, 256, 0))
      : (fp8 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, decode_kernel<64, true>, 256, 0)
             : hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, decode_kernel<64, false>, 256, 0));
  if (e != hipSuccess || blocks < 1) return -1;
  int fblocks = 0;
  e = c.head_dim == 128
      ? (fp8 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&fblocks, decode_step_kernel<128, true>, 256, 0)
             : hipOccupancyMaxActiveBlocksPerMultiprocessor(&fblocks, decode_step_kernel<128, false>, 256, 0))
      : (fp8 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&fblocks, decode_step_kernel<64, true>, 256, 0)
             : hipOccupancyMaxActiveBlocksPerMultiprocessor(&fblocks, decode_step_kernel<64, false>, 256, 0));
  if (e != hipSuccess || fblocks < 1) return -1;
  int waves = cus * kWavesPerBlock;
  if (waves > kMaxWaves) waves = kMaxWaves / kWavesPerBlock * kWavesPerBlock;
  return waves;
}

}  // namespace dms
