// FP8 (OCP E4M3) KV pages: tile layout and the row quantizer shared by every
// kernel that writes a token into the pool.
//
// KV quantization is one of the methods the paper names as orthogonal to DMS
// (App. B).  Each retained K row and V row of a (token, KV head) is stored as
// E4M3 codes with one power-of-two scale 2^e per row: e is the smallest
// integer with max|x| * 2^-e <= 448, the codes are the round-to-nearest-even
// E4M3 values of x * 2^-e (gfx950's conversion instructions implement OCP
// E4M3 with that rounding), and the stored value is code * 2^e.  Because the
// scale is a power of two, applying it is exact: decode multiplies fp32
// scores by the key scale and bf16 softmax weights by the value scale without
// rounding.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dms {

// FP8 tile of 32 slots, 64*D + 256 bytes, in the order the decode MFMAs
// consume it (lane L = 16 G + r, r = L % 16, G = L / 16):
//   keys   [D/64][2][64 lanes][16 B]: block h, lane L hold slot
//          8 (r/4) + r%4 + 4 h; byte 8 j + i is dim 64 p + 32 j + 8 G + i
//   values [D/32][64 lanes][16 B] at 32*D: byte 8 j + i of lane L is
//          dim 32 p + 16 j + r of slot 8 G + i
//   scales at 64*D: [4 G][key scales of slots 8G .. 8G+7 (8 f32) |
//          value scales of the same slots (8 f32)]
__host__ __device__ inline size_t fp8_tile_bytes(int D) { return static_cast<size_t>(D) * 64 + 256; }
__host__ __device__ inline size_t fp8_k_off(int j, int e) {
  const int h = (j >> 2) & 1, r = 4 * (j >> 3) + (j & 3);
  return static_cast<size_t>(e >> 6) * 2048 + h * 1024 + (16 * ((e >> 3) & 3) + r) * 16 +
         8 * ((e >> 5) & 1) + (e & 7);
}
__host__ __device__ inline size_t fp8_v_off(int j, int e, int D) {
  return static_cast<size_t>(D) * 32 + (e >> 5) * 1024 + (16 * (j >> 3) + (e & 15)) * 16 +
         8 * ((e >> 4) & 1) + (j & 7);
}
__host__ __device__ inline size_t fp8_ks_off(int j, int D) {
  return static_cast<size_t>(D) * 64 + (j >> 3) * 64 + (j & 7) * 4;
}
__host__ __device__ inline size_t fp8_vs_off(int j, int D) { return fp8_ks_off(j, D) + 32; }

// Row exponent: the smallest e with amax * 2^-e <= 448 = 0.875 * 2^9
// (0 for an all-zero row).
__device__ inline int fp8_row_exponent(float amax) {
  if (!(amax > 0.f)) return 0;
  int E;
  const float m = frexpf(amax, &E);   // amax = m 2^E, m in [0.5, 1)
  return m <= 0.875f ? E - 9 : E - 8;
}

// Quantize dims 8 i .. 8 i + 7 of one bf16 row held by lane i of an aligned
// group of `group` = D/8 lanes (all of them active): returns the 8 E4M3 codes
// (dim order, low byte first) and sets *e to the row exponent.
__device__ inline uint2 fp8_quantize8(uint4 x8, int group, int* e) {
  const uint32_t wd[4] = {x8.x, x8.y, x8.z, x8.w};
  float x[8];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    x[2 * w] = __uint_as_float(wd[w] << 16);
    x[2 * w + 1] = __uint_as_float(wd[w] & 0xFFFF0000u);
  }
  float amax = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(x[i]));
  for (int off = 1; off < group; off <<= 1) amax = fmaxf(amax, __shfl_xor(amax, off, 64));
  const int ex = fp8_row_exponent(amax);
  *e = ex;
  uint32_t w[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    int v = __builtin_amdgcn_cvt_pk_fp8_f32(ldexpf(x[4 * h], -ex), ldexpf(x[4 * h + 1], -ex), 0, false);
    v = __builtin_amdgcn_cvt_pk_fp8_f32(ldexpf(x[4 * h + 2], -ex), ldexpf(x[4 * h + 3], -ex), v, true);
    w[h] = static_cast<uint32_t>(v);
  }
  return make_uint2(w[0], w[1]);
}

// Write one token's quantized K and V rows into slot j of an FP8 tile.  Lane
// i < D/8 of the calling group holds dims 8 i .. 8 i + 7 of both rows.
__device__ inline void fp8_store_token(char* tile, int j, int D, int i, uint4 k8, uint4 v8) {
  int ek, ev;
  const uint2 kc = fp8_quantize8(k8, D / 8, &ek);
  const uint2 vc = fp8_quantize8(v8, D / 8, &ev);
  // the 8 key codes are 8 contiguous bytes of the key part
  *reinterpret_cast<uint2*>(tile + fp8_k_off(j, 8 * i)) = kc;
  // value codes go to 8 different 16-byte lane slots
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const uint32_t wv = b < 4 ? vc.x : vc.y;
    *reinterpret_cast<uint8_t*>(tile + fp8_v_off(j, 8 * i + b, D)) =
        static_cast<uint8_t>(wv >> (8 * (b & 3)));
  }
  if (i == 0) {
    *reinterpret_cast<float*>(tile + fp8_ks_off(j, D)) = ldexpf(1.0f, ek);
    *reinterpret_cast<float*>(tile + fp8_vs_off(j, D)) = ldexpf(1.0f, ev);
  }
}

// Write one token's K row and V column into slot j of its tile, bf16 or FP8
// pages (`tile`: the 32-slot tile holding the slot).  Called by the 64 lanes
// of one wave; lane i < D/8 holds dims 8 i .. 8 i + 7 of both rows.
__device__ inline void store_token_kv(char* tile, int j, int D, int lane, bool fp8, const uint16_t* k,
                                      const uint16_t* v) {
  if (fp8) {
    if (lane < D / 8)
      fp8_store_token(tile, j, D, lane, reinterpret_cast<const uint4*>(k)[lane],
                      reinterpret_cast<const uint4*>(v)[lane]);
    return;
  }
  if (lane < D / 8) *reinterpret_cast<uint4*>(tile + k_elem_off(j, 8 * lane)) = reinterpret_cast<const uint4*>(k)[lane];
  for (int e = lane; e < D; e += 64) *reinterpret_cast<uint16_t*>(tile + v_elem_off(j, e, D)) = v[e];
}

}  // namespace dms
