// Training-time DMS attention with continuous decisions, gfx950.
//
// Sec. 3.1 (Eq. 1, Fig. 1b): each key j of a KV head carries alpha_j in
// [0, 1]; the scaled scores of every query head reading that KV head get the
// additive mask M_alpha: -inf for j > t, 0 for the w most recent positions
// (j > t - w, delayed eviction), log(1 - alpha_j) for older keys.  The mask
// is never materialised: the key's bias travels with its tile, and tiles are
// classified per block of queries as entirely old (bias per key), entirely
// inside the window (no bias) or mixed (per-element select).
//
// Passes (all MFMA v_mfma_f32_16x16x32_bf16, fp32 accumulation):
//   tile   -- every input tensor [B, T, H, d] becomes 32-token tiles holding
//             a row part (keys-as-rows MFMA operand order) and a transposed
//             part (dims-as-rows order), so every kernel stages tiles with
//             contiguous 16-byte copies and reads operands conflict-free;
//   fwd    -- query-major online softmax, as in the masked prefill: out, lse;
//   rowsum -- D_t = sum_d dout * out per query row;
//   dq     -- query-major: recompute P, dP = dO V^T, dS = P (dP - D),
//             dQ = scale dS K;
//   dkv    -- key-major: each wave keeps 16 keys' K and V operands in
//             registers and walks the query tiles of every query head of the
//             group: dV = P^T dO, dK = scale dS^T Q and
//             dalpha_j = -sum_t exp(s_tj - lse_t) (dP_tj - D_t) over t >= j + w
//             (the probability without the (1 - alpha_j) factor, so the
//             gradient stays finite where alpha_j = 1).
#include <cmath>

#include "dms_common.h"
#include "dms_train.h"

namespace dms {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

constexpr int kThreads = 256;
constexpr int kTrainD = kTrainHeadDim;
constexpr float kRescale = 8.0f;      // lazy rescale threshold, log2 units
constexpr float kMInit = -1.0e30f;    // running max before the first visible key
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ inline f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ inline u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ inline void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// max / sum over the four lanes r, r + 16, r + 32, r + 48
__device__ inline float col_max(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const uint32_t v = __float_as_uint(y);
  const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ inline float col_sum(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const uint32_t v = __float_as_uint(y);
  const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// The dispatcher deals workgroups to the 8 XCDs round-robin by linear id, and
// each XCD has its own L2.  Map the linear id so that the workgroups one XCD
// receives, in dispatch order, are a contiguous range of logical ids
// (x fastest): the blocks of one (sequence, head) then share an L2 and start
// together.
constexpr int kXcds = 8;
__device__ inline int2 xcd_order() {
  const int nx = gridDim.x;
  const int N = nx * gridDim.y;
  const int id = blockIdx.x + nx * blockIdx.y;
  const int x = id % kXcds, k = id / kXcds;
  const int L = x * (N / kXcds) + min(x, N % kXcds) + k;
  return int2{L % nx, L / nx};
}

// 8 fp32 values -> 4 packed bf16 pairs (round to nearest even)
__device__ inline u32x4 pack_bf16(const float* e) {
  u32x4 u;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const f32x2 pr = {e[2 * j], e[2 * j + 1]};
    u[j] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pr, bf16x2));
  }
  return u;
}

// ---------------------------------------------------------------------------
// Tile layout (one 32-token tile of one head: D * 128 bytes)
//   row part, bytes [0, D*64): 16-byte slot P holds dims 32 (P / 128) +
//     8 ((P / 16) % 4) .. + 7 of tile row (r % 4) + 8 (r / 4) + 4 ((P / 64) % 2),
//     r = P % 16 -- the order in which MFMA A-operand loads of "rows" (two
//     16-row blocks whose rows are tokens 8 (r / 4) + r % 4 and that + 4)
//     read it: lane L of the load for dims [32 s, 32 s + 32) reads slot
//     128 s + L (first block) or 128 s + 64 + L (second block);
//   transposed part, bytes [D*64, D*128): slot P holds tokens 8 ((P / 16) % 4)
//     .. + 7 of dim 16 (P / 64) + P % 16 -- the A operand of a product over
//     the tile's tokens, dims 16 b .. + 15 at slots 64 b + L.
// ---------------------------------------------------------------------------
struct TileArgs {
  const uint16_t* x;   // [B, T, H, D]
  char* tiles;         // [B, H, nt] tiles
  int T, H, nt;
};

template <int D>
__global__ __launch_bounds__(kThreads) void train_tile_kernel(TileArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t rows[32][D + 8];
  const int k = blockIdx.x, bh = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x;
  for (int q = tid; q < 32 * D / 8; q += kThreads) {
    const int row = q / (D / 8), e0 = 8 * (q % (D / 8));
    const int t = 32 * k + row;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (t < a.T) v = ld16(a.x + ((static_cast<size_t>(b) * a.T + t) * a.H + h) * D + e0);
    st16(&rows[row][e0], v);
  }
  __syncthreads();
  char* tile = a.tiles + (static_cast<size_t>(bh) * a.nt + k) * (D * 128);
  for (int P = tid; P < D * 4; P += kThreads) {
    const int r = P & 15, c = (P >> 4) & 3, hh = (P >> 6) & 1, s = P >> 7;
    const int j = (r & 3) + 8 * (r >> 2) + 4 * hh;
    st16(tile + P * 16, ld16(&rows[j][32 * s + 8 * c]));
    const int G = c, e = 16 * (P >> 6) + r;
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      v[i] = static_cast<uint32_t>(rows[8 * G + 2 * i][e]) |
             (static_cast<uint32_t>(rows[8 * G + 2 * i + 1][e]) << 16);
    st16(tile + D * 64 + P * 16, v);
  }
}

// ---------------------------------------------------------------------------
// Shared arguments of the attention passes
// ---------------------------------------------------------------------------
struct TrainArgs {
  const uint16_t* q;       // [B, T, Hq, D]
  const uint16_t* k;       // [B, T, H, D]
  const uint16_t* v;
  const uint16_t* dout;    // [B, T, Hq, D]
  const float* alpha;      // [B, T, H]
  const float* out;        // [B, T, Hq, D]
  const float* lse;        // [B, Hq, T]
  const float* dsum;       // [B, Hq, T]
  const char* ktiles;      // [B, H, nt]
  const char* vtiles;
  const char* qtiles;      // [B, Hq, nt]
  const char* dotiles;
  float* o_out;
  float* lse_out;
  float* dsum_out;
  float* dq;
  float* dk;
  float* dv;
  float* dalpha;
  int B, T, H, g, w, nt, PB;
  float scale_log2;        // softmax scale * log2(e)
};

// Mask class of keys [j0, j1) for queries [q0, q1): 0 = every key older
// than every query's window (bias log(1 - alpha)), 1 = every key inside every
// query's window and not after any query (no bias), 2 = per element.
__device__ inline int mask_class(int j0, int j1, int q0, int q1, int w, int T) {
  if (j1 - 1 <= q0 - w) return 0;
  if (j0 > q1 - 1 - w && j1 - 1 <= q0 && q1 <= T) return 1;
  return 2;
}

// Key bias log2(1 - alpha) / (scale * log2 e): in raw score units, so that
// adding it to q.k and scaling gives log2 of the weight (-inf at alpha = 1).
__device__ inline float key_bias_raw(const TrainArgs& a, int b, int h, int j) {
  if (j >= a.T) return 0.f;
  const float al = a.alpha[(static_cast<size_t>(b) * a.T + j) * a.H + h];
  return __log2f(1.0f - al) / a.scale_log2;
}

// ---------------------------------------------------------------------------
// Forward.  Workgroup = (sequence b, KV head h, block of PB query positions);
// columns are (position, query head) pairs, the g heads of a position
// consecutive, 16 per MFMA column block (a position's heads may straddle two
// blocks), NQ blocks per wave.  Key tiles 0 .. ceil(t1 / 32) - 1
// (causal) are staged through LDS: K row part, V transposed part.
// ---------------------------------------------------------------------------
template <int D, int NQ>
__global__ __launch_bounds__(kThreads, 2) void train_fwd_kernel(TrainArgs a) {
  __shared__ __attribute__((aligned(16))) char tile_lds[2][D * 128];
  __shared__ float bias_lds[2][32];
  const int2 wg = xcd_order();               // latest (longest) query blocks first
  const int bh = wg.y;
  const int b = bh / a.H, h = bh % a.H;
  const int t0 = (gridDim.x - 1 - wg.x) * a.PB;
  if (t0 >= a.T) return;
  const int t1 = min(a.T, t0 + a.PB);
  const int ntiles = (t1 + 31) >> 5;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, G = lane >> 4;
  const int Hq = a.H * a.g;

  int tcol[NQ];
  u32x4 qf[NQ][D / 32];
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
    const int col = (wave * NQ + qb) * 16 + r;
    const int pl = col / a.g, qh = col % a.g;
    const int t = t0 + pl;
    const bool ok = (pl < a.PB) && (t < t1);
    tcol[qb] = ok ? t : -1;
    const uint16_t* qrow = a.q + ((static_cast<size_t>(b) * a.T + (ok ? t : 0)) * Hq + h * a.g + qh) * D;
#pragma unroll
    for (int s2 = 0; s2 < D / 32; ++s2)
      qf[qb][s2] = ok ? ld16(qrow + 32 * s2 + 8 * G) : u32x4{0u, 0u, 0u, 0u};
  }

  constexpr int KP = D * 4 / kThreads;   // 16-byte slots per thread per part
  const char* kt = a.ktiles + static_cast<size_t>(bh) * a.nt * (D * 128);
  const char* vt = a.vtiles + static_cast<size_t>(bh) * a.nt * (D * 128) + D * 64;
  u32x4 sk[KP], sv[KP];
  float sb = 0.f;
  auto stage_load = [&](int k) {
#pragma unroll
    for (int m = 0; m < KP; ++m) {
      const int P = tid + m * kThreads;
      sk[m] = ld16(kt + static_cast<size_t>(k) * (D * 128) + P * 16);
      sv[m] = ld16(vt + static_cast<size_t>(k) * (D * 128) + P * 16);
    }
    if (tid < 32) sb = key_bias_raw(a, b, h, 32 * k + tid);
  };
  auto stage_store = [&](int buf) {
#pragma unroll
    for (int m = 0; m < KP; ++m) {
      const int P = tid + m * kThreads;
      st16(tile_lds[buf] + P * 16, sk[m]);
      st16(tile_lds[buf] + D * 64 + P * 16, sv[m]);
    }
    if (tid < 32) bias_lds[buf][tid] = sb;
  };

  f32x4 o[NQ][D / 16];
  float m_ref[NQ], l_run[NQ];
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
#pragma unroll
    for (int bb = 0; bb < D / 16; ++bb) o[qb][bb] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_ref[qb] = kMInit;
    l_run[qb] = 0.f;
  }
  const float thr = kRescale / a.scale_log2;
  const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);

  stage_load(0);
  stage_store(0);
  __syncthreads();
  for (int k = 0; k < ntiles; ++k) {
    const int buf = k & 1;
    if (k + 1 < ntiles) stage_load(k + 1);
    const char* tl = tile_lds[buf];
    u32x4 ka[D / 32], kb[D / 32], vt2[D / 16];
#pragma unroll
    for (int s2 = 0; s2 < D / 32; ++s2) {
      ka[s2] = ld16(tl + s2 * 2048 + lane * 16);
      kb[s2] = ld16(tl + s2 * 2048 + 1024 + lane * 16);
    }
#pragma unroll
    for (int bb = 0; bb < D / 16; ++bb) vt2[bb] = ld16(tl + D * 64 + bb * 1024 + lane * 16);
    const int jt = 32 * k;
    const int cls = mask_class(jt, jt + 32, t0, t1, a.w, a.T);
    float kbias[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) kbias[j] = bias_lds[buf][8 * G + j];
#pragma unroll
    for (int qb = 0; qb < NQ; ++qb) {
      f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s2 = 0; s2 < D / 32; ++s2) {
        s0 = mfma_bf16(ka[s2], qf[qb][s2], s0);
        s1 = mfma_bf16(kb[s2], qf[qb][s2], s1);
      }
      float sc[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sc[j] = s0[j];
        sc[j + 4] = s1[j];
      }
      if (cls == 0) {
#pragma unroll
        for (int j = 0; j < 8; ++j) sc[j] += kbias[j];
      } else if (cls == 2) {
        const int t = tcol[qb];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int key = jt + 8 * G + j;
          sc[j] = key > t ? -INFINITY : (key > t - a.w ? sc[j] : sc[j] + kbias[j]);
        }
      }
      float mx = fmaxf(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3])),
                       fmaxf(fmaxf(sc[4], sc[5]), fmaxf(sc[6], sc[7])));
      mx = col_max(mx);
      const bool raise = mx > m_ref[qb] + thr;
      if (__builtin_amdgcn_ballot_w64(raise)) {
        const float m_new = raise ? mx : m_ref[qb];
        const float alpha_s = __builtin_amdgcn_exp2f((m_ref[qb] - m_new) * a.scale_log2);
        l_run[qb] *= alpha_s;
#pragma unroll
        for (int bb = 0; bb < D / 16; ++bb) o[qb][bb] *= alpha_s;
        m_ref[qb] = m_new;
      }
      const float mb = m_ref[qb] * a.scale_log2;
      float e[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) e[j] = __builtin_amdgcn_exp2f(fmaf(sc[j], a.scale_log2, -mb));
      // the denominator adds the bf16-rounded weights the MFMA uses (dot
      // with (1, 1) on each packed pair as it is made)
      u32x4 pu;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x2 pr = {e[2 * j], e[2 * j + 1]};
        const bf16x2 pb = __builtin_convertvector(pr, bf16x2);
        pu[j] = __builtin_bit_cast(uint32_t, pb);
        l_run[qb] = __builtin_amdgcn_fdot2_f32_bf16(pb, ones, l_run[qb], false);
      }
#pragma unroll
      for (int bb = 0; bb < D / 16; ++bb) o[qb][bb] = mfma_bf16(vt2[bb], pu, o[qb][bb]);
    }
    if (k + 1 < ntiles) stage_store(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
    const float l = col_sum(l_run[qb]);
    const int t = tcol[qb];
    if (t >= 0) {
      const int qh = ((wave * NQ + qb) * 16 + r) % a.g;
      float* dst = a.o_out + ((static_cast<size_t>(b) * a.T + t) * Hq + h * a.g + qh) * D + 4 * G;
      const float inv = 1.0f / l;
#pragma unroll
      for (int bb = 0; bb < D / 16; ++bb) *reinterpret_cast<f32x4*>(dst + 16 * bb) = o[qb][bb] * inv;
      if (G == 0)
        a.lse_out[(static_cast<size_t>(b) * Hq + h * a.g + qh) * a.T + t] =
            (m_ref[qb] * a.scale_log2 + __log2f(l)) * kLn2;
    }
  }
}

// D = sum_d dout * out for every (b, query head, t); 16 lanes per row.
__global__ __launch_bounds__(kThreads) void train_rowsum_kernel(TrainArgs a, int D) {
  const int Hq = a.H * a.g;
  const int64_t rows = static_cast<int64_t>(a.B) * a.T * Hq;
  const int64_t row = (static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x) >> 4;
  const int sub = threadIdx.x & 15;
  float s = 0.f;
  if (row < rows) {
    for (int e = sub * 8; e < D; e += 128) {
      const u32x4 d8 = ld16(a.dout + row * D + e);
      const f32x4 o0 = *reinterpret_cast<const f32x4*>(a.out + row * D + e);
      const f32x4 o1 = *reinterpret_cast<const f32x4*>(a.out + row * D + e + 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float lo = __uint_as_float(d8[i] << 16), hi = __uint_as_float(d8[i] & 0xFFFF0000u);
        s += lo * (i < 2 ? o0[2 * i] : o1[2 * i - 4]) + hi * (i < 2 ? o0[2 * i + 1] : o1[2 * i - 3]);
      }
    }
  }
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) s += __shfl_xor(s, off, 16);
  if (row < rows && sub == 0) {
    // row = (b * T + t) * Hq + qh  ->  dsum[(b * Hq + qh) * T + t]
    const int qh = static_cast<int>(row % Hq);
    const int64_t bt = row / Hq;
    const int t = static_cast<int>(bt % a.T), bb = static_cast<int>(bt / a.T);
    a.dsum_out[(static_cast<size_t>(bb) * Hq + qh) * a.T + t] = s;
  }
}

// ---------------------------------------------------------------------------
// dQ pass.  Same workgroups and columns as the forward.  Per key tile: K row
// part (S^T = K Q^T), V row part (dP^T = V dO^T), K transposed part
// (dQ^T += K^T dS^T).
// ---------------------------------------------------------------------------
template <int D, int NQ>
__global__ __launch_bounds__(kThreads, 1) void train_dq_kernel(TrainArgs a) {
  __shared__ __attribute__((aligned(16))) char tile_lds[2][D * 192];
  __shared__ float bias_lds[2][32];
  const int2 wg = xcd_order();
  const int bh = wg.y;
  const int b = bh / a.H, h = bh % a.H;
  const int t0 = (gridDim.x - 1 - wg.x) * a.PB;
  if (t0 >= a.T) return;
  const int t1 = min(a.T, t0 + a.PB);
  const int ntiles = (t1 + 31) >> 5;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, G = lane >> 4;
  const int Hq = a.H * a.g;

  int tcol[NQ];
  u32x4 qf[NQ][D / 32], df[NQ][D / 32];
  float lse2[NQ], dcol[NQ];
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
    const int col = (wave * NQ + qb) * 16 + r;
    const int pl = col / a.g, qh = col % a.g;
    const int t = t0 + pl;
    const bool ok = (pl < a.PB) && (t < t1);
    tcol[qb] = ok ? t : -1;
    const size_t row = (static_cast<size_t>(b) * a.T + (ok ? t : 0)) * Hq + h * a.g + qh;
#pragma unroll
    for (int s2 = 0; s2 < D / 32; ++s2) {
      qf[qb][s2] = ok ? ld16(a.q + row * D + 32 * s2 + 8 * G) : u32x4{0u, 0u, 0u, 0u};
      df[qb][s2] = ok ? ld16(a.dout + row * D + 32 * s2 + 8 * G) : u32x4{0u, 0u, 0u, 0u};
    }
    const size_t li = (static_cast<size_t>(b) * Hq + h * a.g + qh) * a.T + (ok ? t : 0);
    lse2[qb] = ok ? a.lse[li] * kLog2e : 0.f;
    dcol[qb] = ok ? a.dsum[li] : 0.f;
  }

  constexpr int KP = D * 4 / kThreads;
  const char* kt = a.ktiles + static_cast<size_t>(bh) * a.nt * (D * 128);
  const char* vt = a.vtiles + static_cast<size_t>(bh) * a.nt * (D * 128);
  u32x4 sk[KP], sv[KP], skt[KP];
  float sb = 0.f;
  auto stage_load = [&](int k) {
    const size_t off = static_cast<size_t>(k) * (D * 128);
#pragma unroll
    for (int m = 0; m < KP; ++m) {
      const int P = tid + m * kThreads;
      sk[m] = ld16(kt + off + P * 16);
      sv[m] = ld16(vt + off + P * 16);
      skt[m] = ld16(kt + off + D * 64 + P * 16);
    }
    if (tid < 32) sb = key_bias_raw(a, b, h, 32 * k + tid);
  };
  auto stage_store = [&](int buf) {
#pragma unroll
    for (int m = 0; m < KP; ++m) {
      const int P = tid + m * kThreads;
      st16(tile_lds[buf] + P * 16, sk[m]);
      st16(tile_lds[buf] + D * 64 + P * 16, sv[m]);
      st16(tile_lds[buf] + D * 128 + P * 16, skt[m]);
    }
    if (tid < 32) bias_lds[buf][tid] = sb;
  };

  f32x4 dqa[NQ][D / 16];
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb)
#pragma unroll
    for (int bb = 0; bb < D / 16; ++bb) dqa[qb][bb] = f32x4{0.f, 0.f, 0.f, 0.f};

  stage_load(0);
  stage_store(0);
  __syncthreads();
  for (int k = 0; k < ntiles; ++k) {
    const int buf = k & 1;
    if (k + 1 < ntiles) stage_load(k + 1);
    const char* tl = tile_lds[buf];
    u32x4 ka[D / 32], kb[D / 32], va[D / 32], vb[D / 32], ktr[D / 16];
#pragma unroll
    for (int s2 = 0; s2 < D / 32; ++s2) {
      ka[s2] = ld16(tl + s2 * 2048 + lane * 16);
      kb[s2] = ld16(tl + s2 * 2048 + 1024 + lane * 16);
      va[s2] = ld16(tl + D * 64 + s2 * 2048 + lane * 16);
      vb[s2] = ld16(tl + D * 64 + s2 * 2048 + 1024 + lane * 16);
    }
#pragma unroll
    for (int bb = 0; bb < D / 16; ++bb) ktr[bb] = ld16(tl + D * 128 + bb * 1024 + lane * 16);
    const int jt = 32 * k;
    const int cls = mask_class(jt, jt + 32, t0, t1, a.w, a.T);
    float kbias[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) kbias[j] = bias_lds[buf][8 * G + j];
#pragma unroll
    for (int qb = 0; qb < NQ; ++qb) {
      f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = s0, p0 = s0, p1 = s0;
#pragma unroll
      for (int s2 = 0; s2 < D / 32; ++s2) {
        s0 = mfma_bf16(ka[s2], qf[qb][s2], s0);
        s1 = mfma_bf16(kb[s2], qf[qb][s2], s1);
        p0 = mfma_bf16(va[s2], df[qb][s2], p0);
        p1 = mfma_bf16(vb[s2], df[qb][s2], p1);
      }
      float sc[8], dp[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sc[j] = s0[j];
        sc[j + 4] = s1[j];
        dp[j] = p0[j];
        dp[j + 4] = p1[j];
      }
      if (cls == 0) {
#pragma unroll
        for (int j = 0; j < 8; ++j) sc[j] += kbias[j];
      } else if (cls == 2) {
        const int t = tcol[qb];   // -1 for unused columns: every key is masked
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int key = jt + 8 * G + j;
          sc[j] = key > t ? -INFINITY : (key > t - a.w ? sc[j] : sc[j] + kbias[j]);
        }
      }
      float ds[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sc[j], a.scale_log2, -lse2[qb]));
        ds[j] = p * (dp[j] - dcol[qb]);
      }
      const u32x4 du = pack_bf16(ds);
#pragma unroll
      for (int bb = 0; bb < D / 16; ++bb) dqa[qb][bb] = mfma_bf16(ktr[bb], du, dqa[qb][bb]);
    }
    if (k + 1 < ntiles) stage_store(buf ^ 1);
    __syncthreads();
  }

  const float scale = a.scale_log2 / kLog2e;
#pragma unroll
  for (int qb = 0; qb < NQ; ++qb) {
    const int t = tcol[qb];
    if (t >= 0) {
      const int qh = ((wave * NQ + qb) * 16 + r) % a.g;
      float* dst = a.dq + ((static_cast<size_t>(b) * a.T + t) * Hq + h * a.g + qh) * D + 4 * G;
#pragma unroll
      for (int bb = 0; bb < D / 16; ++bb) *reinterpret_cast<f32x4*>(dst + 16 * bb) = dqa[qb][bb] * scale;
    }
  }
}

// ---------------------------------------------------------------------------
// dK / dV / dalpha pass.  Workgroup = (b, KV head h, 64 keys); wave w owns
// keys j0 + 16 w .. + 15 as the 16 columns of its MFMAs, with those keys' K
// and V (B operands) in registers.  It walks every query head of the group
// and every 32-position query tile from the block's first key on (the last
// tile first); per tile the Q and dO tiles (row and transposed parts), lse and
// D are staged.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kThreads, 2) void train_dkv_kernel(TrainArgs a) {
  __shared__ __attribute__((aligned(16))) char tile_lds[2][D * 256];
  __shared__ __attribute__((aligned(16))) float row_lds[2][2][32];   // lse (log2 units), D per row
  const int2 wg = xcd_order();               // earliest (longest) key blocks first
  const int bh = wg.y;
  const int b = bh / a.H, h = bh % a.H;
  const int j0 = wg.x * 64;
  if (j0 >= a.T) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, G = lane >> 4;
  const int Hq = a.H * a.g;
  const int j = j0 + 16 * wave + r;          // this lane's key
  const bool jok = j < a.T;

  u32x4 kf[D / 32], vf[D / 32];
  {
    const size_t row = (static_cast<size_t>(b) * a.T + (jok ? j : 0)) * a.H + h;
#pragma unroll
    for (int s2 = 0; s2 < D / 32; ++s2) {
      kf[s2] = jok ? ld16(a.k + row * D + 32 * s2 + 8 * G) : u32x4{0u, 0u, 0u, 0u};
      vf[s2] = jok ? ld16(a.v + row * D + 32 * s2 + 8 * G) : u32x4{0u, 0u, 0u, 0u};
    }
  }
  const float al = jok ? a.alpha[(static_cast<size_t>(b) * a.T + j) * a.H + h] : 0.f;
  const float keep = 1.0f - al;              // weight of the key outside the window
  f32x4 dka[D / 16], dva[D / 16];
#pragma unroll
  for (int bb = 0; bb < D / 16; ++bb) {
    dka[bb] = f32x4{0.f, 0.f, 0.f, 0.f};
    dva[bb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  float dal = 0.f;

  const int pt0 = j0 >> 5;
  const int nsteps = a.g * (a.nt - pt0);     // (query tile, query head) pairs
  constexpr int KP = D * 4 / kThreads;
  // Two register sets: the tiles of step s + 2 are loaded while step s is
  // computed, and step s + 1's are written to LDS at its end.
  u32x4 ra[4][KP], rb[4][KP];
  float rowa = 0.f, rowb = 0.f;
  // steps walk the query tiles from the last one down, every query head of
  // the group per tile: the blocks of one (sequence, head) that run together
  // read the same tile at about the same time
  int ld_qh = 0, ld_pt = a.nt - 1;           // next step to load
  auto stage_load = [&](u32x4 (&rg)[4][KP], float& row) {
    const size_t tix = (static_cast<size_t>(b) * Hq + h * a.g + ld_qh) * a.nt + ld_pt;
    const char* qt = a.qtiles + tix * (D * 128);
    const char* dt = a.dotiles + tix * (D * 128);
#pragma unroll
    for (int m = 0; m < KP; ++m) {
      const int P = tid + m * kThreads;
      rg[0][m] = ld16(qt + P * 16);
      rg[1][m] = ld16(qt + D * 64 + P * 16);
      rg[2][m] = ld16(dt + P * 16);
      rg[3][m] = ld16(dt + D * 64 + P * 16);
    }
    if (tid < 64) {
      const int t = 32 * ld_pt + (tid & 31);
      const size_t li = (static_cast<size_t>(b) * Hq + h * a.g + ld_qh) * a.T + t;
      row = t < a.T ? (tid < 32 ? a.lse[li] * kLog2e : a.dsum[li]) : 0.f;
    }
    if (++ld_qh == a.g) {
      ld_qh = 0;
      --ld_pt;
    }
  };
  auto stage_store = [&](int buf, const u32x4 (&rg)[4][KP], float row) {
#pragma unroll
    for (int m = 0; m < KP; ++m) {
      const int P = tid + m * kThreads;
#pragma unroll
      for (int part = 0; part < 4; ++part) st16(tile_lds[buf] + part * (D * 64) + P * 16, rg[part][m]);
    }
    if (tid < 64) row_lds[buf][tid >> 5][tid & 31] = row;
  };

  int step_qh = 0, tq = 32 * (a.nt - 1);     // step being computed
  auto compute = [&](int buf) {
    const char* tl = tile_lds[buf];
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = s0, p0 = s0, p1 = s0;
#pragma unroll
    for (int s2 = 0; s2 < D / 32; ++s2) {
      const u32x4 qa = ld16(tl + s2 * 2048 + lane * 16);
      const u32x4 qb = ld16(tl + s2 * 2048 + 1024 + lane * 16);
      const u32x4 da = ld16(tl + D * 128 + s2 * 2048 + lane * 16);
      const u32x4 db = ld16(tl + D * 128 + s2 * 2048 + 1024 + lane * 16);
      s0 = mfma_bf16(qa, kf[s2], s0);
      s1 = mfma_bf16(qb, kf[s2], s1);
      p0 = mfma_bf16(da, vf[s2], p0);
      p1 = mfma_bf16(db, vf[s2], p1);
    }
    // lane (key r, G) now holds rows (queries) tq + 8 G + i, i = 0..7
    const f32x4 l2a = *reinterpret_cast<const f32x4*>(&row_lds[buf][0][8 * G]);
    const f32x4 l2b = *reinterpret_cast<const f32x4*>(&row_lds[buf][0][8 * G + 4]);
    const f32x4 dda = *reinterpret_cast<const f32x4*>(&row_lds[buf][1][8 * G]);
    const f32x4 ddb = *reinterpret_cast<const f32x4*>(&row_lds[buf][1][8 * G + 4]);
    const int cls = mask_class(j0, j0 + 64, tq, tq + 32, a.w, a.T);
    float pr[8], ds[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float raw = i < 4 ? s0[i] : s1[i - 4];
      const float dpd = (i < 4 ? p0[i] : p1[i - 4]) - (i < 4 ? dda[i] : ddb[i - 4]);
      const float l2 = i < 4 ? l2a[i] : l2b[i - 4];
      const float pu = __builtin_amdgcn_exp2f(fmaf(raw, a.scale_log2, -l2));   // exp(s - lse) w/o bias
      float p;
      bool old;
      if (cls == 0) {
        p = pu * keep;
        old = true;
      } else if (cls == 1) {
        p = pu;
        old = false;
      } else {
        const int t = tq + 8 * G + i;
        const bool vis = j <= t && t < a.T && jok;
        old = vis && j <= t - a.w;
        p = vis ? (old ? pu * keep : pu) : 0.f;
      }
      pr[i] = p;
      ds[i] = p * dpd;
      if (old) dal = fmaf(pu, dpd, dal);
    }
    const u32x4 pu8 = pack_bf16(pr);
    const u32x4 du8 = pack_bf16(ds);
#pragma unroll
    for (int bb = 0; bb < D / 16; ++bb) {
      dva[bb] = mfma_bf16(ld16(tl + D * 192 + bb * 1024 + lane * 16), pu8, dva[bb]);
      dka[bb] = mfma_bf16(ld16(tl + D * 64 + bb * 1024 + lane * 16), du8, dka[bb]);
    }
    if (++step_qh == a.g) {
      step_qh = 0;
      tq -= 32;
    }
  };

  stage_load(ra, rowa);
  if (nsteps > 1) stage_load(rb, rowb);
  stage_store(0, ra, rowa);
  __syncthreads();
  for (int step = 0; step < nsteps; step += 2) {
    if (step + 2 < nsteps) stage_load(ra, rowa);
    compute(0);
    if (step + 1 < nsteps) stage_store(1, rb, rowb);
    __syncthreads();
    if (step + 1 >= nsteps) break;
    if (step + 3 < nsteps) stage_load(rb, rowb);
    compute(1);
    if (step + 2 < nsteps) stage_store(0, ra, rowa);
    __syncthreads();
  }

  dal = col_sum(dal);
  if (jok) {
    const float scale = a.scale_log2 / kLog2e;
    const size_t row = (static_cast<size_t>(b) * a.T + j) * a.H + h;
    float* dkd = a.dk + row * D + 4 * G;
    float* dvd = a.dv + row * D + 4 * G;
#pragma unroll
    for (int bb = 0; bb < D / 16; ++bb) {
      *reinterpret_cast<f32x4*>(dkd + 16 * bb) = dka[bb] * scale;
      *reinterpret_cast<f32x4*>(dvd + 16 * bb) = dva[bb];
    }
    if (G == 0) a.dalpha[row] = -dal;
  }
}

__global__ __launch_bounds__(kThreads) void gumbel_fwd_kernel(int n, const float* x, const float* u,
                                                              float inv_tau, float* alpha) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= n) return;
  const float uu = u[i];
  const float z = (x[i] + (__logf(uu) - __logf(1.0f - uu))) * inv_tau;
  alpha[i] = 1.0f / (1.0f + __expf(-z));
}

__global__ __launch_bounds__(kThreads) void gumbel_bwd_kernel(int n, const float* alpha, const float* da,
                                                              float inv_tau, float* dx) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= n) return;
  const float al = alpha[i];
  dx[i] = da[i] * al * (1.0f - al) * inv_tau;
}

constexpr int kNQ = 2;

struct TrainLayout {
  size_t ktiles, vtiles, qtiles, dotiles, dsum, bytes;
  int nt;
};

TrainLayout train_layout(const dms_train_config& c) {
  TrainLayout l{};
  const size_t B = c.batch, T = c.seq_len, H = c.num_kv_heads, Hq = H * c.group_size;
  const size_t D = c.head_dim;
  l.nt = static_cast<int>((T + 31) / 32);
  const size_t tile = D * 128;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, kAlign); return o; };
  l.ktiles = take(B * H * l.nt * tile);
  l.vtiles = take(B * H * l.nt * tile);
  l.qtiles = take(B * Hq * l.nt * tile);
  l.dotiles = take(B * Hq * l.nt * tile);
  l.dsum = take(B * Hq * T * 4);
  l.bytes = off;
  return l;
}

TrainArgs train_args(const dms_train_config& c, const TrainLayout& l, void* ws) {
  TrainArgs a{};
  char* w = static_cast<char*>(ws);
  a.ktiles = w + l.ktiles;
  a.vtiles = w + l.vtiles;
  a.qtiles = w + l.qtiles;
  a.dotiles = w + l.dotiles;
  a.dsum = reinterpret_cast<const float*>(w + l.dsum);
  a.dsum_out = reinterpret_cast<float*>(w + l.dsum);
  a.B = c.batch;
  a.T = c.seq_len;
  a.H = c.num_kv_heads;
  a.g = c.group_size;
  a.w = c.window;
  a.nt = l.nt;
  a.PB = 4 * kNQ * 16 / c.group_size;   // (position, head) columns packed across column blocks
  const float scale = c.softmax_scale > 0.f ? c.softmax_scale : 1.0f / sqrtf(static_cast<float>(c.head_dim));
  a.scale_log2 = scale * kLog2e;
  return a;
}

hipError_t tile(const void* x, int B, int T, int H, int nt, char* tiles, hipStream_t st) {
  TileArgs t{static_cast<const uint16_t*>(x), tiles, T, H, nt};
  hipLaunchKernelGGL(train_tile_kernel<kTrainD>, dim3(nt, B * H), dim3(kThreads), 0, st, t);
  return hipGetLastError();
}

}  // namespace

size_t train_workspace_bytes(const dms_train_config& c) { return train_layout(c).bytes; }

hipError_t launch_train_fwd(const dms_train_config& c, const void* q, const void* k, const void* v,
                            const float* alpha, float* out, float* lse, void* ws, hipStream_t st) {
  const TrainLayout l = train_layout(c);
  TrainArgs a = train_args(c, l, ws);
  char* w = static_cast<char*>(ws);
  hipError_t e = tile(k, c.batch, c.seq_len, c.num_kv_heads, l.nt, w + l.ktiles, st);
  if (e == hipSuccess) e = tile(v, c.batch, c.seq_len, c.num_kv_heads, l.nt, w + l.vtiles, st);
  if (e != hipSuccess) return e;
  a.q = static_cast<const uint16_t*>(q);
  a.alpha = alpha;
  a.o_out = out;
  a.lse_out = lse;
  dim3 grid((c.seq_len + a.PB - 1) / a.PB, c.batch * c.num_kv_heads);
  hipLaunchKernelGGL((train_fwd_kernel<kTrainD, kNQ>), grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_train_bwd(const dms_train_config& c, const void* q, const void* k, const void* v,
                            const float* alpha, const float* out, const float* lse,
                            const void* dout, float* dq, float* dk, float* dv, float* dalpha,
                            void* ws, hipStream_t st) {
  const TrainLayout l = train_layout(c);
  TrainArgs a = train_args(c, l, ws);
  char* w = static_cast<char*>(ws);
  const int Hq = c.num_kv_heads * c.group_size;
  hipError_t e = tile(k, c.batch, c.seq_len, c.num_kv_heads, l.nt, w + l.ktiles, st);
  if (e == hipSuccess) e = tile(v, c.batch, c.seq_len, c.num_kv_heads, l.nt, w + l.vtiles, st);
  if (e == hipSuccess) e = tile(q, c.batch, c.seq_len, Hq, l.nt, w + l.qtiles, st);
  if (e == hipSuccess) e = tile(dout, c.batch, c.seq_len, Hq, l.nt, w + l.dotiles, st);
  if (e != hipSuccess) return e;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.dout = static_cast<const uint16_t*>(dout);
  a.alpha = alpha;
  a.out = out;
  a.lse = lse;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.dalpha = dalpha;
  const int64_t rows = static_cast<int64_t>(c.batch) * c.seq_len * Hq;
  hipLaunchKernelGGL(train_rowsum_kernel, dim3(static_cast<unsigned>((rows * 16 + kThreads - 1) / kThreads)),
                     dim3(kThreads), 0, st, a, c.head_dim);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(train_dkv_kernel<kTrainD>, dim3((c.seq_len + 63) / 64, c.batch * c.num_kv_heads),
                     dim3(kThreads), 0, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 grid((c.seq_len + a.PB - 1) / a.PB, c.batch * c.num_kv_heads);
  hipLaunchKernelGGL((train_dq_kernel<kTrainD, kNQ>), grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gumbel_fwd(int n, const float* x, const float* u, float tau, float* alpha,
                             hipStream_t st) {
  hipLaunchKernelGGL(gumbel_fwd_kernel, dim3((n + kThreads - 1) / kThreads), dim3(kThreads), 0, st, n,
                     x, u, 1.0f / tau, alpha);
  return hipGetLastError();
}

hipError_t launch_gumbel_bwd(int n, const float* alpha, const float* da, float tau, float* dx,
                             hipStream_t st) {
  hipLaunchKernelGGL(gumbel_bwd_kernel, dim3((n + kThreads - 1) / kThreads), dim3(kThreads), 0, st, n,
                     alpha, da, 1.0f / tau, dx);
  return hipGetLastError();
}

}  // namespace dms
