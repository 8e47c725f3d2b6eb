// Metered decode attention on the matrix cores (head_dim 128, bf16 queries).
//
// Same computation as the vector path (read path of the meter loop, Sec. 6;
// Theorem black-box logit bound; Theorem sound replacement; split-KV merge of
// Sec. 6.2), laid out for CDNA4 wave64 MFMA.  One wave owns one split of one
// (sequence, KV head) and walks it in 16-token pages:
//
//   QK^T  S = K Q^T with v_mfma_f32_16x16x32_f16: A = 16 tokens x 32 channels of
//         int8 codes (exact in fp16), B = the G (<= 16) queries in fp16.  The
//         dither enters as a second product with D = 2u - 255 = 512 xi (an odd
//         integer, exact in fp16): q . khat = s (q . code - q . D / 512).
//   bound c_t = sm_scale sum_b ||q_b|| w_{t,b}: one more MFMA, witness (fp16,
//         exact) times band norms split into fp16 hi + lo parts.
//   softmax online over the page; the running max is only raised when a page
//         exceeds it by more than kSlack (then the accumulators are rescaled),
//         so the common case needs no cross-lane exchange.
//   PV    O^T = V^T W with v_mfma_f32_16x16x16_f16: A = value codes of 16 channels
//         x 4 tokens per lane group (the value pages are stored token-quad
//         interleaved so this is one 32-byte load), B = p_t s^v_t in fp16, and a
//         second product with the dither, transposed through LDS.
//
// Lane l: r = l % 16 (token in the QK operands, head in B and in the results,
// channel row in the PV operands), g = l / 16 (k-group).  The channel order of
// the QK contraction is permuted so that lane group g owns channels 32g..32g+31,
// i.e. exactly the two Philox calls (16 channels each) it regenerates.
#include <float.h>

#include "wc_device.h"
#include "wc_launch.h"

namespace wc {

namespace {

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h4_t __attribute__((ext_vector_type(4)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef short s8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));

constexpr int kD = 128;
constexpr int kWaves = 4;
constexpr int kRow = 272;  // LDS bytes per token row of the dither transpose (256 + pad)
// The running max is raised only when a page exceeds it by more than kSlack, so
// softmax weights stay below e^2.  Weights enter the fp16 PV operand multiplied
// by kWScale = 2^8 (undone at the end), which keeps small weights out of the fp16
// subnormal range; the product stays below 65504 for value scales up to 34.
constexpr float kSlack = 2.0f;
constexpr float kWScale = 256.0f;

__device__ __forceinline__ uint32_t as_u32(h2_t v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ h2_t as_h2(uint32_t v) { return __builtin_bit_cast(h2_t, v); }

// Two signed int8 (bytes 0 and 1 of x, pre-biased by 0x80) -> fp16 pair, exact:
// fp16 bits 0x6400 | u = 1024 + u, minus 1152.
__device__ __forceinline__ h2_t i8pair_lo(uint32_t xb) {
  const uint32_t v = (xb & 0xFFu) | ((xb & 0xFF00u) << 8) | 0x64006400u;
  return as_h2(v) - h2_t{(_Float16)1152.0f, (_Float16)1152.0f};
}
__device__ __forceinline__ h2_t i8pair_hi(uint32_t xb) {
  const uint32_t v = ((xb >> 16) & 0xFFu) | ((xb >> 8) & 0xFF0000u) | 0x64006400u;
  return as_h2(v) - h2_t{(_Float16)1152.0f, (_Float16)1152.0f};
}
// Two dither bytes u -> fp16 pair 2u - 255, exact in two steps: (1024 + u) - 1024
// = u, then 2u - 255.  (A single 2 * (1024 + u) - 2303 is not exact: 2303 is odd
// and above 2048, where fp16 values are spaced by 2.)
__device__ __forceinline__ h2_t dpair_lo(uint32_t u) {
  const uint32_t v = (u & 0xFFu) | ((u & 0xFF00u) << 8) | 0x64006400u;
  const h2_t b = as_h2(v) - h2_t{(_Float16)1024.0f, (_Float16)1024.0f};
  return b * h2_t{(_Float16)2.0f, (_Float16)2.0f} - h2_t{(_Float16)255.0f, (_Float16)255.0f};
}
__device__ __forceinline__ h2_t dpair_hi(uint32_t u) {
  const uint32_t v = ((u >> 16) & 0xFFu) | ((u >> 8) & 0xFF0000u) | 0x64006400u;
  const h2_t b = as_h2(v) - h2_t{(_Float16)1024.0f, (_Float16)1024.0f};
  return b * h2_t{(_Float16)2.0f, (_Float16)2.0f} - h2_t{(_Float16)255.0f, (_Float16)255.0f};
}
// Two E4M3 bytes -> fp16 pair holding value / 256 (exact; the 256 is folded
// into the scale): sign to bit 15, exponent/mantissa bits shifted by 7.
__device__ __forceinline__ uint32_t e4m3pair(uint32_t b0, uint32_t b1) {
  const uint32_t lo = ((b0 & 0x7Fu) << 7) | ((b0 & 0x80u) << 8);
  const uint32_t hi = ((b1 & 0x7Fu) << 7) | ((b1 & 0x80u) << 8);
  return lo | (hi << 16);
}
// Two bf16 -> fp16 pair (exact for |x| in the fp16 normal range).
__device__ __forceinline__ uint32_t bf16pair_to_f16(uint32_t w) {
  const float a = bf16_to_f32((uint16_t)(w & 0xFFFFu));
  const float b = bf16_to_f32((uint16_t)(w >> 16));
  return as_u32(h2_t{(_Float16)a, (_Float16)b});
}

__device__ __forceinline__ h8_t pack8(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  const uint4 v = make_uint4(a, b, c, d);
  return __builtin_bit_cast(h8_t, v);
}
__device__ __forceinline__ h4_t pack4(uint32_t a, uint32_t b) {
  const uint2 v = make_uint2(a, b);
  return __builtin_bit_cast(h4_t, v);
}

__device__ __forceinline__ float xor_max(float v, int m) { return fmaxf(v, __shfl_xor(v, m, 64)); }

// e^c - 1 for 0 <= c <= 1 by its Taylor series to c^10/10! (relative error < 3e-7).
__device__ __forceinline__ float expm1_small(float c) {
  float s = 1.0f / 3628800.0f;
  s = fmaf(s, c, 1.0f / 362880.0f);
  s = fmaf(s, c, 1.0f / 40320.0f);
  s = fmaf(s, c, 1.0f / 5040.0f);
  s = fmaf(s, c, 1.0f / 720.0f);
  s = fmaf(s, c, 1.0f / 120.0f);
  s = fmaf(s, c, 1.0f / 24.0f);
  s = fmaf(s, c, 1.0f / 6.0f);
  s = fmaf(s, c, 0.5f);
  s = fmaf(s, c, 1.0f);
  return s * c;
}

template <int KIND, bool METER>
__global__ __launch_bounds__(256, 2) void decode_mfma_kernel(DecodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t dsh[kWaves][16 * kRow];
  __shared__ float qn_s[kWaves][16][16];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const int unit = blockIdx.y;
  const int b = unit / a.n_kv, kv = unit % a.n_kv;
  if (a.mask_kv != nullptr && a.mask_kv[unit] == 0) return;
  const int split = blockIdx.x * kWaves + wave;
  const int G = a.group;
  const int B = a.n_bands;
  const int L = a.seq_lens[b];
  const int t_begin = split * a.split_tokens;
  if (split >= a.n_splits || t_begin >= L) return;  // whole waves leave; no block barrier below
  const int t_end = min(min(L, t_begin + a.split_tokens), a.max_blocks * kBlockTokens);

  // ---- queries of head r (zero for padding heads), channels 32g .. 32g+31 ----
  const bool hv = r < G;
  const uint16_t* qp = reinterpret_cast<const uint16_t*>(a.q) +
                       ((int64_t)b * a.n_q + (int64_t)kv * G + (hv ? r : 0)) * kD + 32 * g;
  uint32_t qraw[16];
  {
    const uint4* q4 = reinterpret_cast<const uint4*>(qp);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint4 v = hv ? q4[i] : make_uint4(0, 0, 0, 0);
      qraw[4 * i] = v.x; qraw[4 * i + 1] = v.y; qraw[4 * i + 2] = v.z; qraw[4 * i + 3] = v.w;
    }
  }
  // B operands of QK: kt-th MFMA uses channels 32g + 8kt .. 32g + 8kt + 7.
  // The matrix cores align the products of one instruction to the largest and
  // drop bits below its 24-bit window, so a massive-activation channel would cost
  // the other channels their precision.  Each query is therefore split into
  // q_hi = round(q / delta) * delta (at most 11 bits on a per-head power-of-two
  // grid delta, so q_hi * code products are exact multiples of delta and sum
  // exactly) and the remainder q_lo = q - q_hi (|q_lo| <= delta/2), each with
  // its own accumulator.
  h8_t qhi[4], qlo[4];
  s8_t qbf[4];
  if constexpr (KIND == WC_KIND_BF16) {
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const uint4 v = make_uint4(qraw[4 * kt], qraw[4 * kt + 1], qraw[4 * kt + 2], qraw[4 * kt + 3]);
      qbf[kt] = __builtin_bit_cast(s8_t, v);
    }
  } else {
    float qmax = 0.0f;
#pragma unroll
    for (int i = 0; i < 32; ++i)
      qmax = fmaxf(qmax, fabsf(bf16_to_f32((uint16_t)((qraw[i >> 1] >> (16 * (i & 1))) & 0xFFFFu))));
    qmax = xor_max(xor_max(qmax, 16), 32);
    int ex = 0;
    (void)frexpf(qmax, &ex);                          // qmax < 2^ex
    const float delta = qmax > 0.0f ? ldexpf(1.0f, ex - 11) : 1.0f;
    const float inv_delta = qmax > 0.0f ? ldexpf(1.0f, 11 - ex) : 1.0f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      uint32_t hw[4], lw[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t w = qraw[4 * kt + j];
        const float x0 = bf16_to_f32((uint16_t)(w & 0xFFFFu)), x1 = bf16_to_f32((uint16_t)(w >> 16));
        const float h0 = rintf(x0 * inv_delta) * delta, h1 = rintf(x1 * inv_delta) * delta;
        hw[j] = as_u32(h2_t{(_Float16)h0, (_Float16)h1});
        lw[j] = as_u32(h2_t{(_Float16)(x0 - h0), (_Float16)(x1 - h1)});
      }
      qhi[kt] = pack8(hw[0], hw[1], hw[2], hw[3]);
      qlo[kt] = pack8(lw[0], lw[1], lw[2], lw[3]);
    }
  }
  // band norms ||q_b|| * sm_scale -> witness-MFMA B operand (hi parts for g < 2, lo for g >= 2)
  h8_t qnop = pack8(0, 0, 0, 0);
  if constexpr (METER) {
    for (int i = lane; i < 256; i += 64) (&qn_s[wave][0][0])[i] = 0.0f;
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const float x = bf16_to_f32((uint16_t)((qraw[i >> 1] >> (16 * (i & 1))) & 0xFFFFu));
      atomicAdd(&qn_s[wave][r][band_of(32 * g + i, kD, B, a.interleaved)], x * x);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
    uint32_t hw[4];
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      _Float16 hv2[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int band = 8 * (g & 1) + 2 * e2 + j;
        const float x = band < B ? sqrtf(qn_s[wave][r][band]) * a.sm_scale : 0.0f;
        const _Float16 hi = (_Float16)x;
        hv2[j] = (g < 2) ? hi : (_Float16)(x - (float)hi);
      }
      hw[e2] = as_u32(h2_t{hv2[0], hv2[1]});
    }
    qnop = pack8(hw[0], hw[1], hw[2], hw[3]);
  }

  f4_t o1[8], o2[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    o1[j] = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
    o2[j] = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
  }
  float m_run = -INFINITY, l_run = 0.0f, n_run = 0.0f;
  const uint32_t layer_head = ((uint32_t)a.layer << 16) | (uint32_t)kv;
  uint8_t* my_dsh = dsh[wave];
  const int32_t* trow = a.table + (int64_t)b * a.max_blocks;

  for (int t0 = t_begin; t0 < t_end; t0 += kBlockTokens) {
    const int64_t blk = trow[t0 / kBlockTokens];
    const int64_t page = blk * a.n_kv + kv;

    // ---------------- loads ----------------
    uint32_t kw[16];   // key bytes of token r, channels 32g.. (64 B for bf16)
    constexpr int KB = KIND == WC_KIND_BF16 ? 64 : 32;
    {
      const uint4* kp = reinterpret_cast<const uint4*>(reinterpret_cast<const uint8_t*>(a.k_data) +
                                                       (page * kBlockTokens + r) * (kD * (KB / 32)) + KB * g);
#pragma unroll
      for (int i = 0; i < KB / 16; ++i) {
        const uint4 v = kp[i];
        kw[4 * i] = v.x; kw[4 * i + 1] = v.y; kw[4 * i + 2] = v.z; kw[4 * i + 3] = v.w;
      }
    }
    uint32_t vw[16];   // value bytes: channels 8r .. 8r+7 of token quad g (4 tokens each)
    {
      const uint4* vp = reinterpret_cast<const uint4*>(
          reinterpret_cast<const uint8_t*>(a.v_data) +
          page * (kBlockTokens * kD * (KB / 32)) + (g * kD + 8 * r) * 4 * (KB / 32));
#pragma unroll
      for (int i = 0; i < KB / 16; ++i) {
        const uint4 v = vp[i];
        vw[4 * i] = v.x; vw[4 * i + 1] = v.y; vw[4 * i + 2] = v.z; vw[4 * i + 3] = v.w;
      }
    }
    float sk[4], sv[4];
    if constexpr (KIND == WC_KIND_INT8_DITHER) {
      const uint2 ks = *reinterpret_cast<const uint2*>(a.k_scale + page * kBlockTokens + 4 * g);
      const uint2 vs = *reinterpret_cast<const uint2*>(a.v_scale + page * kBlockTokens + 4 * g);
      sk[0] = f16_to_f32((uint16_t)(ks.x & 0xFFFFu)); sk[1] = f16_to_f32((uint16_t)(ks.x >> 16));
      sk[2] = f16_to_f32((uint16_t)(ks.y & 0xFFFFu)); sk[3] = f16_to_f32((uint16_t)(ks.y >> 16));
      sv[0] = f16_to_f32((uint16_t)(vs.x & 0xFFFFu)); sv[1] = f16_to_f32((uint16_t)(vs.x >> 16));
      sv[2] = f16_to_f32((uint16_t)(vs.y & 0xFFFFu)); sv[3] = f16_to_f32((uint16_t)(vs.y >> 16));
#pragma unroll
      for (int e = 0; e < 4; ++e) sv[e] *= kWScale;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sk[e] = KIND == WC_KIND_FP8_RAW ? 256.0f : 1.0f;
        sv[e] = kWScale;
      }
    }
    uint4 wit = make_uint4(0, 0, 0, 0);   // bands 8(g%2) .. 8(g%2)+7 of token r (B is 8 or 16)
    if constexpr (METER) {
      if (8 * (g & 1) < B)
        wit = *reinterpret_cast<const uint4*>(a.k_witness + (page * kBlockTokens + r) * B + 8 * (g & 1));
    }

    // ---------------- QK^T and the bound ----------------
    const f4_t z4 = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
    f4_t s1 = z4, s1l = z4, s2 = z4, s2l = z4;   // code and dither products, q_hi and q_lo parts
    uint32_t dq[16];   // dither 2u-255 of token r, channels 32g.., fp16 pairs
    if constexpr (KIND == WC_KIND_INT8_DITHER) {
      const int64_t slot = blk * kBlockTokens + r;
      const U4 r0 = dither_block(2 * g, slot, layer_head, a.key0, a.key1);
      const U4 r1 = dither_block(2 * g + 1, slot, layer_head, a.key0, a.key1);
      const uint32_t u[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        dq[2 * i] = as_u32(dpair_lo(u[i]));
        dq[2 * i + 1] = as_u32(dpair_hi(u[i]));
      }
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        uint32_t c[4];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const uint32_t x = kw[2 * kt + j] ^ 0x80808080u;
          c[2 * j] = as_u32(i8pair_lo(x));
          c[2 * j + 1] = as_u32(i8pair_hi(x));
        }
        const h8_t ka = pack8(c[0], c[1], c[2], c[3]);
        const h8_t da = pack8(dq[4 * kt], dq[4 * kt + 1], dq[4 * kt + 2], dq[4 * kt + 3]);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka, qhi[kt], s1, 0, 0, 0);
        s1l = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka, qlo[kt], s1l, 0, 0, 0);
        s2 = __builtin_amdgcn_mfma_f32_16x16x32_f16(da, qhi[kt], s2, 0, 0, 0);
        s2l = __builtin_amdgcn_mfma_f32_16x16x32_f16(da, qlo[kt], s2l, 0, 0, 0);
      }
      // dither of this page to LDS (row = token r, channels 32g..32g+31)
      uint4* dst = reinterpret_cast<uint4*>(my_dsh + r * kRow + 64 * g);
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[i] = make_uint4(dq[4 * i], dq[4 * i + 1], dq[4 * i + 2], dq[4 * i + 3]);
    } else if constexpr (KIND == WC_KIND_FP8_RAW) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        uint32_t c[4];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const uint32_t x = kw[2 * kt + j];
          c[2 * j] = e4m3pair(x & 0xFFu, (x >> 8) & 0xFFu);
          c[2 * j + 1] = e4m3pair((x >> 16) & 0xFFu, x >> 24);
        }
        const h8_t ka = pack8(c[0], c[1], c[2], c[3]);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka, qhi[kt], s1, 0, 0, 0);
        s1l = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka, qlo[kt], s1l, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const uint4 v = make_uint4(kw[4 * kt], kw[4 * kt + 1], kw[4 * kt + 2], kw[4 * kt + 3]);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(s8_t, v), qbf[kt], s1, 0, 0, 0);
      }
    }
    f4_t cb = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
    if constexpr (METER) {
      cb = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8_t, wit), qnop, cb, 0, 0, 0);
    }

    // ---------------- online softmax and meter numerator ----------------
    // this lane: head r, tokens t0 + 4g + e
    float lg[4];
    float loc = -INFINITY;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool valid = t0 + 4 * g + e < t_end;
      float s = s1[e] + s1l[e];
      if constexpr (KIND == WC_KIND_INT8_DITHER) s = fmaf(s2[e] + s2l[e], -0.001953125f, s);
      lg[e] = valid ? s * (sk[e] * a.sm_scale) : -INFINITY;
      loc = fmaxf(loc, lg[e]);
    }
    if (__ballot(loc > m_run + kSlack) != 0) {
      const float full = xor_max(xor_max(loc, 16), 32);
      const float m_new = fmaxf(m_run, full);
      const float alpha = __expf(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
      n_run *= alpha;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        o1[j] *= alpha;
        o2[j] *= alpha;
      }
    }
    float wgt[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool valid = t0 + 4 * g + e < t_end;
      const float p = valid ? __expf(lg[e] - m_run) : 0.0f;
      l_run += p;
      if constexpr (METER) {
        const float c = cb[e];
        const float term = c > 1.0f ? __expf(lg[e] - m_run + c) - p : p * expm1_small(c);
        n_run += valid ? term : 0.0f;
      }
      wgt[e] = valid ? p * sv[e] : 0.0f;
    }
    const h4_t wop = h4_t{(_Float16)wgt[0], (_Float16)wgt[1], (_Float16)wgt[2], (_Float16)wgt[3]};

    // ---------------- P V ----------------
    if constexpr (KIND == WC_KIND_INT8_DITHER) {
      __builtin_amdgcn_s_waitcnt(0xc07f);   // LDS writes of this page done
      __builtin_amdgcn_wave_barrier();
      uint4 rows[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        rows[e] = *reinterpret_cast<const uint4*>(my_dsh + (4 * g + e) * kRow + 16 * r);
#pragma unroll
      for (int jt = 0; jt < 8; ++jt) {
        const uint32_t x = vw[jt] ^ 0x80808080u;     // codes of channel 8r+jt, tokens 4g..4g+3
        const h4_t vc = pack4(as_u32(i8pair_lo(x)), as_u32(i8pair_hi(x)));
        o1[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(vc, wop, o1[jt], 0, 0, 0);
        const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&rows[0]);
        const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&rows[1]);
        const uint32_t* r2 = reinterpret_cast<const uint32_t*>(&rows[2]);
        const uint32_t* r3 = reinterpret_cast<const uint32_t*>(&rows[3]);
        const int sh = 16 * (jt & 1);
        const uint32_t d01 = ((r0[jt >> 1] >> sh) & 0xFFFFu) | (((r1[jt >> 1] >> sh) & 0xFFFFu) << 16);
        const uint32_t d23 = ((r2[jt >> 1] >> sh) & 0xFFFFu) | (((r3[jt >> 1] >> sh) & 0xFFFFu) << 16);
        o2[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(d01, d23), wop, o2[jt], 0, 0, 0);
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);   // LDS reads done before the next page overwrites
      __builtin_amdgcn_wave_barrier();
    } else if constexpr (KIND == WC_KIND_FP8_RAW) {
#pragma unroll
      for (int jt = 0; jt < 8; ++jt) {
        const uint32_t x = vw[jt];
        uint32_t lo = e4m3pair(x & 0xFFu, (x >> 8) & 0xFFu);
        uint32_t hi = e4m3pair((x >> 16) & 0xFFu, x >> 24);
        // tokens past the end may hold any byte pattern (the 0x7F NaN code): zero them
        if (t0 + 4 * g + 0 >= t_end) lo &= 0xFFFF0000u;
        if (t0 + 4 * g + 1 >= t_end) lo &= 0x0000FFFFu;
        if (t0 + 4 * g + 2 >= t_end) hi &= 0xFFFF0000u;
        if (t0 + 4 * g + 3 >= t_end) hi &= 0x0000FFFFu;
        o1[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(lo, hi), wop, o1[jt], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int jt = 0; jt < 8; ++jt) {
        // bf16 values of channel 8r+jt, tokens 4g..4g+3: 8 bytes at offset 8*jt
        uint32_t lo = bf16pair_to_f16(vw[2 * jt]);
        uint32_t hi = bf16pair_to_f16(vw[2 * jt + 1]);
        if (t0 + 4 * g + 0 >= t_end) lo &= 0xFFFF0000u;
        if (t0 + 4 * g + 1 >= t_end) lo &= 0x0000FFFFu;
        if (t0 + 4 * g + 2 >= t_end) hi &= 0xFFFF0000u;
        if (t0 + 4 * g + 3 >= t_end) hi &= 0x0000FFFFu;
        o1[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(lo, hi), wop, o1[jt], 0, 0, 0);
      }
    }
  }

  // ---- partial record of this split: running max, sums over all lane groups, output ----
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  if constexpr (METER) {
    n_run += __shfl_xor(n_run, 16, 64);
    n_run += __shfl_xor(n_run, 32, 64);
    if (isnan(n_run)) n_run = INFINITY;
  }
  if (!hv) return;
  const int64_t R = (int64_t)partial_record_floats(kD);
  float* rec = a.part + (((int64_t)b * a.n_q + (int64_t)kv * G + r) * a.n_splits + split) * R;
  // rows 4g+e of tile jt hold channel 8(4g+e)+jt = 32g + 8e + jt
  // fp8 operands hold value/256, so the weight scale already cancels there
  constexpr float unscale = KIND == WC_KIND_FP8_RAW ? 1.0f : 1.0f / kWScale;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float v[8];
#pragma unroll
    for (int jt = 0; jt < 8; ++jt) {
      v[jt] = o1[jt][e];
      if constexpr (KIND == WC_KIND_INT8_DITHER) v[jt] = fmaf(o2[jt][e], -0.001953125f, v[jt]);
      v[jt] *= unscale;
    }
    float4* dst = reinterpret_cast<float4*>(rec + 32 * g + 8 * e);
    dst[0] = make_float4(v[0], v[1], v[2], v[3]);
    dst[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
  if (g == 0) {
    rec[kD] = m_run;
    rec[kD + 1] = l_run;
    rec[kD + 2] = n_run;
  }
}

}  // namespace

bool mfma_decode_supported(const DecodeArgs& a) {
  return a.head_dim == kD && a.q_dtype == WC_BF16 && a.group <= 16 &&
         (a.kind == WC_KIND_BF16 || a.n_bands == 8 || a.n_bands == 16);
}

hipError_t launch_decode_mfma(const DecodeArgs& a, bool metered, hipStream_t st) {
  const dim3 grid((a.n_splits + kWaves - 1) / kWaves, a.batch * a.n_kv);
  if (!metered)
    hipLaunchKernelGGL((decode_mfma_kernel<WC_KIND_BF16, false>), grid, dim3(64 * kWaves), 0, st, a);
  else if (a.kind == WC_KIND_INT8_DITHER)
    hipLaunchKernelGGL((decode_mfma_kernel<WC_KIND_INT8_DITHER, true>), grid, dim3(64 * kWaves), 0, st, a);
  else
    hipLaunchKernelGGL((decode_mfma_kernel<WC_KIND_FP8_RAW, true>), grid, dim3(64 * kWaves), 0, st, a);
  return hipGetLastError();
}

}  // namespace wc
