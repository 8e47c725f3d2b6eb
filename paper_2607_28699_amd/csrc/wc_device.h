// Device-side building blocks shared by the WitCert kernels (gfx950, wave64).
//
//  * Philox4x32-10 (Salmon et al., SC'11), the counter-based dither source of
//    the paper's write and read kernels (Sec. 6.2).
//  * Round-up fp16 conversion for stored scales and witnesses, nearest-even
//    bf16, and the OCP fp8 E4M3 raw cast (nearest-even, saturating).
//  * The band map of the residual witness (Sec. 4.1, Lemma RoPE band unitarity).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wc {

constexpr int kBlockTokens = 16;

// ---- Philox4x32-10 --------------------------------------------------------
// Round: (hi0, lo0) = M0*x0, (hi1, lo1) = M1*x2 (64-bit products);
// x <- (hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0); key += (W0, W1) between rounds.
struct U4 {
  uint32_t x, y, z, w;
};

__device__ __forceinline__ U4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                            uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    // three-input exclusive or in one instruction (bitop3 truth table 0x96)
    const uint32_t n0 = __builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), c1, k0, 0x96);
    const uint32_t n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), c3, k1, 0x96);
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
  }
  return U4{c0, c1, c2, c3};
}

// Dither of channels 16*group .. 16*group+15 of one slot: counter
// (group, slot low word, slot high word, layer<<16 | kv_head), key = seed.
// Byte i of the 16 output bytes (little-endian within words) is channel 16*group+i.
__device__ __forceinline__ U4 dither_block(int group, int64_t slot, uint32_t layer_head,
                                           uint32_t key0, uint32_t key1) {
  return philox4x32_10((uint32_t)group, (uint32_t)(uint64_t)slot,
                       (uint32_t)((uint64_t)slot >> 32), layer_head, key0, key1);
}

// xi = (u - 127.5) / 256 = u/256 - 127.5/256: exact in fp32 (one fma).
__device__ __forceinline__ float dither_value(uint32_t u) {
  return fmaf((float)u, 0.00390625f, -0.498046875f);
}

// ---- format conversions -----------------------------------------------------
__device__ __forceinline__ uint16_t f16_bits(_Float16 h) {
  return __builtin_bit_cast(uint16_t, h);
}
__device__ __forceinline__ float f16_to_f32(uint16_t b) {
  return (float)__builtin_bit_cast(_Float16, b);
}

// Smallest fp16 >= f for finite f >= 0 (inf above 65504).
__device__ __forceinline__ uint16_t f16_round_up(float f) {
  const _Float16 h = (_Float16)f;  // nearest-even (default rounding mode)
  uint16_t b = f16_bits(h);
  if ((float)h < f) b += 1;
  return b;
}

// Smallest fp16 value >= d (d finite, >= 0).  Rounding up is monotone and every
// fp16 value is an fp32 value, so it is the fp16 round-up of the fp32 round-up of
// d: nearest fp32, one fp32 step up if that fell below d, then f16_round_up.
__device__ __forceinline__ uint16_t f16_round_up_f64(double d) {
  float f = (float)d;
  if ((double)f < d) f = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, f) + 1u);
  return f16_round_up(f);
}

// Largest fp16 value <= d (d finite, >= 0; 65504 above the range), the same way
// down: nearest fp32, one step down if above d, nearest fp16, one step down if
// above.
__device__ __forceinline__ uint16_t f16_round_down_f64(double d) {
  float f = (float)d;
  if ((double)f > d) f = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, f) - 1u);
  const _Float16 h = (_Float16)f;
  uint16_t b = f16_bits(h);
  if ((float)h > f) b -= 1;
  return b;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __builtin_bit_cast(float, (uint32_t)b << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// OCP E4M3 ("fn"): bias 7, 3 mantissa bits, max 448, subnormal quantum 2^-9.
__device__ __forceinline__ uint8_t f32_to_e4m3_sat(float x) {
  const uint32_t sign = (__builtin_bit_cast(uint32_t, x) >> 24) & 0x80u;
  const float a = fabsf(x);
  if (!(a < 448.0f)) return (uint8_t)(sign | 0x7Eu);
  if (a < 0.015625f) {                     // below 2^-6: quantum 2^-9
    const float m = rintf(a * 512.0f);     // 0..8; 8 is the smallest normal (code 0x08)
    return (uint8_t)(sign | (uint32_t)m);
  }
  const int e = (int)((__builtin_bit_cast(uint32_t, a) >> 23) & 0xFFu) - 127;  // -6..8
  const float q = __builtin_bit_cast(float, (uint32_t)(e - 3 + 127) << 23);     // 2^(e-3)
  const float r = rintf(a / q) * q;        // exact power-of-two scaling, nearest-even
  const uint32_t ru = __builtin_bit_cast(uint32_t, r);
  const uint32_t er = ((ru >> 23) & 0xFFu) - 127u + 7u;
  const uint32_t mr = (ru >> 20) & 7u;
  return (uint8_t)(sign | (er << 3) | mr);
}

__device__ __forceinline__ float e4m3_to_f32(uint32_t b) {
  const uint32_t e = (b >> 3) & 15u, m = b & 7u;
  float v = e ? __builtin_bit_cast(float, ((e + 120u) << 23) | (m << 20))
              : (float)m * 0.001953125f;
  return (b & 0x80u) ? -v : v;
}

// ---- page layout of the key and value arrays --------------------------------
// A page (16 tokens of one KV head) is stored as 16-byte pieces, ordered so that
// every 16-byte load instruction of the matrix-core decode covers whole cache
// lines: piece (i, g, r) lies at byte ((i*4 + g)*16 + r)*16, i < CL = D*E/64
// (E bytes per element).  Keys: piece (i, g, r) holds bytes (g*CL + i)*16 ..
// +15 of token r's row (D elements, channel order).  Values: token quad q's
// row holds D channels x 4 tokens (token t of the quad, channel c at element
// 4c + t), and piece (i, q, r) holds its bytes (r*CL + i)*16 .. +15.
// Offsets in bytes within the page.
__host__ __device__ inline int kpage_off(int t, int c, int D, int E) {
  const int CL = D * E / 64, b = c * E, p = b >> 4;
  return (((p % CL) * 4 + p / CL) * 16 + t) * 16 + (b & 15);
}
__host__ __device__ inline int vpage_off(int t, int c, int D, int E) {
  const int CL = D * E / 64, b = (4 * c + (t & 3)) * E, p = b >> 4;
  return (((p % CL) * 4 + (t >> 2)) * 16 + p / CL) * 16 + (b & 15);
}

// ---- band map -----------------------------------------------------------------
// Band of channel c: pairs are (j, j + D/2) (rotate-half) or (2j, 2j+1)
// (interleaved); band b holds pairs b*P .. b*P+P-1 with P = D / (2B).
__device__ __forceinline__ int band_of(int c, int D, int B, int interleaved) {
  const int P = D / (2 * B);
  const int pair = interleaved ? (c >> 1) : (c < D / 2 ? c : c - D / 2);
  return pair / P;
}

// The c-th channel (0 .. 2P-1) of band b.
__device__ __forceinline__ int band_channel(int b, int k, int D, int B, int interleaved) {
  const int P = D / (2 * B);
  if (interleaved) return 2 * b * P + k;
  return k < P ? b * P + k : D / 2 + b * P + (k - P);
}

// ---- wave reductions (wave64) ---------------------------------------------------
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace wc
