// Metered decode attention on the matrix cores (head_dim 128, bf16 queries).
//
// Same computation as the vector path (read path of the meter loop, Sec. 6;
// Theorem black-box logit bound; Theorem sound replacement; split-KV merge of
// Sec. 6.2), laid out for CDNA4 wave64 MFMA.  A workgroup of four waves owns one
// split of one (sequence, KV head); each wave walks a contiguous quarter of it in
// 16-token pages, and the four partial states are merged in LDS before one
// partial record is written.
//
//   QK^T  S = K Q^T with v_mfma_f32_16x16x32_f16: A = 16 tokens x 32 channels of
//         int8 codes (exact in fp16), B = the G (<= 16) queries in fp16.  The
//         dither enters as a second product with D = 2048 + 2u (exact in fp16,
//         built from the Philox byte u by a byte permute); since 512 xi = 2u - 255,
//         q . khat = s (q . code - (q . D - 2303 sum(q)) / 512).
//   bound c_t = sm_scale sum_b ||q_b|| w_{t,b}: one more MFMA, witness (fp16,
//         exact) times band norms split into fp16 hi + lo parts.
//   softmax online over the page; the running max is only raised when a page
//         exceeds it by more than kSlack (then the accumulators are rescaled),
//         so the common case needs no cross-lane exchange.
//   PV    O^T = V^T W with v_mfma_f32_16x16x16_f16: A = value codes of 16 channels
//         x 4 tokens per lane group (the value pages are stored token-quad
//         interleaved, so this is one 32-byte load), B = p_t s^v_t in fp16, and a
//         second product with D, transposed through LDS; the 2303 offset is
//         removed with the running sum of the fp16 weights.
//
// Lane l: r = l % 16 (token in the QK operands, head in B and in the results,
// channel row in the PV operands), g = l / 16 (k-group).  The channel order of
// the QK contraction is permuted so that lane group g owns channels 32g..32g+31,
// i.e. exactly the two Philox calls (16 channels each) it regenerates.  Pages are
// double-buffered in registers: the next page's loads are in flight while the
// current page is computed.
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
constexpr float kDOff = 2303.0f;   // 2048 + 255: D = 2u + 2048 = 512 xi + 2303

__device__ __forceinline__ uint32_t as_u32(h2_t v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ h2_t as_h2(uint32_t v) { return __builtin_bit_cast(h2_t, v); }

// Byte permutes: result byte i is byte sel_i of {hi:lo} (0..3 = lo, 4..7 = hi).
__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}
constexpr uint32_t kSelLo = 0x04010400u;   // bytes 0, 1 of lo, each under byte 0 of hi
constexpr uint32_t kSelHi = 0x04030402u;   // bytes 2, 3 of lo
constexpr uint32_t kSelH0 = 0x05040100u;   // low halves of lo and hi
constexpr uint32_t kSelH1 = 0x07060302u;   // high halves of lo and hi

// Two int8 codes (already xor 0x80: u = code + 128) -> fp16 (1024 + u) - 1152, exact.
__device__ __forceinline__ uint32_t codes2(uint32_t xb, uint32_t sel) {
  return as_u32(as_h2(perm(0x64646464u, xb, sel)) - h2_t{(_Float16)1152.0f, (_Float16)1152.0f});
}
// Two dither bytes u -> fp16 2048 + 2u (bits 0x6800 | u), exact, one permute.
__device__ __forceinline__ uint32_t dith2(uint32_t u, uint32_t sel) {
  return perm(0x68686868u, u, sel);
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
  return __builtin_bit_cast(h8_t, make_uint4(a, b, c, d));
}
__device__ __forceinline__ h4_t pack4(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(h4_t, make_uint2(a, b));
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

// Loaded bytes of one 16-token page for one lane.
template <int KIND>
struct PageRegs {
  static constexpr int NW = KIND == WC_KIND_BF16 ? 16 : 8;
  uint32_t kw[NW];   // keys of token r, channels 32g..32g+31
  uint32_t vw[NW];   // values of channels 8r..8r+7 for token quad g
  uint2 ks, vs;      // fp16 scales of tokens 4g..4g+3
  uint4 wit;         // witness bands 8(g%2).. of token r
  int64_t blk;
};

template <int KIND, bool METER>
__device__ __forceinline__ void load_page(const DecodeArgs& a, const int32_t* trow, int t0, int kv,
                                          int r, int g, PageRegs<KIND>& p) {
  constexpr int KB = KIND == WC_KIND_BF16 ? 64 : 32;   // bytes per lane and tensor
  p.blk = trow[t0 / kBlockTokens];
  const int64_t page = p.blk * a.n_kv + kv;
  const uint4* kp = reinterpret_cast<const uint4*>(reinterpret_cast<const uint8_t*>(a.k_data) +
                                                   (page * kBlockTokens + r) * (kD * (KB / 32)) + KB * g);
  const uint4* vp = reinterpret_cast<const uint4*>(reinterpret_cast<const uint8_t*>(a.v_data) +
                                                   page * (kBlockTokens * kD * (KB / 32)) +
                                                   (g * kD + 8 * r) * 4 * (KB / 32));
#pragma unroll
  for (int i = 0; i < KB / 16; ++i) {
    const uint4 k4 = kp[i], v4 = vp[i];
    p.kw[4 * i] = k4.x; p.kw[4 * i + 1] = k4.y; p.kw[4 * i + 2] = k4.z; p.kw[4 * i + 3] = k4.w;
    p.vw[4 * i] = v4.x; p.vw[4 * i + 1] = v4.y; p.vw[4 * i + 2] = v4.z; p.vw[4 * i + 3] = v4.w;
  }
  if constexpr (KIND == WC_KIND_INT8_DITHER) {
    p.ks = *reinterpret_cast<const uint2*>(a.k_scale + page * kBlockTokens + 4 * g);
    p.vs = *reinterpret_cast<const uint2*>(a.v_scale + page * kBlockTokens + 4 * g);
  }
  if constexpr (METER) {
    p.wit = make_uint4(0, 0, 0, 0);
    if (8 * (g & 1) < a.n_bands)
      p.wit = *reinterpret_cast<const uint4*>(a.k_witness + (page * kBlockTokens + r) * a.n_bands + 8 * (g & 1));
  }
}

// Running state of one wave.
struct WaveState {
  f4_t o1[8], o2[8];
  float m, l, n, wsum;
};

template <int KIND, bool METER>
__device__ __forceinline__ void process_page(const DecodeArgs& a, const PageRegs<KIND>& cur, int t0,
                                             int t_end, int r, int g, uint32_t layer_head,
                                             const h8_t (&qop)[4], const s8_t (&qbf)[4],
                                             const h8_t& qnop, float qsum, uint8_t* my_dsh,
                                             WaveState& st) {
  float sk[4], sv[4];
  if constexpr (KIND == WC_KIND_INT8_DITHER) {
    sk[0] = f16_to_f32((uint16_t)(cur.ks.x & 0xFFFFu)); sk[1] = f16_to_f32((uint16_t)(cur.ks.x >> 16));
    sk[2] = f16_to_f32((uint16_t)(cur.ks.y & 0xFFFFu)); sk[3] = f16_to_f32((uint16_t)(cur.ks.y >> 16));
    sv[0] = f16_to_f32((uint16_t)(cur.vs.x & 0xFFFFu)); sv[1] = f16_to_f32((uint16_t)(cur.vs.x >> 16));
    sv[2] = f16_to_f32((uint16_t)(cur.vs.y & 0xFFFFu)); sv[3] = f16_to_f32((uint16_t)(cur.vs.y >> 16));
#pragma unroll
    for (int e = 0; e < 4; ++e) sv[e] *= kWScale;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      sk[e] = KIND == WC_KIND_FP8_RAW ? 256.0f : 1.0f;
      sv[e] = kWScale;
    }
  }

  // ---------------- QK^T and the bound ----------------
  const f4_t z4 = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
  f4_t s1 = z4, s2 = z4;   // code products, dither products
  if constexpr (KIND == WC_KIND_INT8_DITHER) {
    const int64_t slot = cur.blk * kBlockTokens + r;
    const U4 r0 = dither_block(2 * g, slot, layer_head, a.key0, a.key1);
    const U4 r1 = dither_block(2 * g + 1, slot, layer_head, a.key0, a.key1);
    const uint32_t u[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
    uint32_t dq[16];   // 2048 + 2u of token r, channels 32g + 2i, 32g + 2i + 1
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      dq[2 * i] = dith2(u[i], kSelLo);
      dq[2 * i + 1] = dith2(u[i], kSelHi);
    }
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const uint32_t x0 = cur.kw[2 * kt] ^ 0x80808080u, x1 = cur.kw[2 * kt + 1] ^ 0x80808080u;
      const h8_t ka = pack8(codes2(x0, kSelLo), codes2(x0, kSelHi), codes2(x1, kSelLo), codes2(x1, kSelHi));
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka, qop[kt], s1, 0, 0, 0);
      s2 = __builtin_amdgcn_mfma_f32_16x16x32_f16(
          pack8(dq[4 * kt], dq[4 * kt + 1], dq[4 * kt + 2], dq[4 * kt + 3]), qop[kt], s2, 0, 0, 0);
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
        const uint32_t x = cur.kw[2 * kt + j];
        c[2 * j] = e4m3pair(x & 0xFFu, (x >> 8) & 0xFFu);
        c[2 * j + 1] = e4m3pair((x >> 16) & 0xFFu, x >> 24);
      }
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(pack8(c[0], c[1], c[2], c[3]), qop[kt], s1, 0, 0, 0);
    }
  } else {
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const uint4 v = make_uint4(cur.kw[4 * kt], cur.kw[4 * kt + 1], cur.kw[4 * kt + 2], cur.kw[4 * kt + 3]);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(s8_t, v), qbf[kt], s1, 0, 0, 0);
    }
  }
  f4_t cb = z4;
  if constexpr (METER) {
    cb = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8_t, cur.wit), qnop, cb, 0, 0, 0);
  }

  // ---------------- online softmax and meter numerator ----------------
  // this lane: head r, tokens t0 + 4g + e
  float lg[4];
  float loc = -INFINITY;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bool valid = t0 + 4 * g + e < t_end;
    float sc = s1[e];
    if constexpr (KIND == WC_KIND_INT8_DITHER) sc = fmaf(s2[e] - kDOff * qsum, -0.001953125f, sc);
    lg[e] = valid ? sc * (sk[e] * a.sm_scale) : -INFINITY;
    loc = fmaxf(loc, lg[e]);
  }
  if (__ballot(loc > st.m + kSlack) != 0) {
    const float full = xor_max(xor_max(loc, 16), 32);
    const float m_new = fmaxf(st.m, full);
    const float alpha = __expf(st.m - m_new);
    st.m = m_new;
    st.l *= alpha;
    st.n *= alpha;
    st.wsum *= alpha;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      st.o1[j] *= alpha;
      st.o2[j] *= alpha;
    }
  }
  float wgt[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bool valid = t0 + 4 * g + e < t_end;
    const float x = lg[e] - st.m;
    const float p = valid ? __expf(x) : 0.0f;
    st.l += p;
    if constexpr (METER) {
      // p (e^c - 1): Taylor series below 1; above, e^(x + c) - p in the log domain
      // so that a token whose weight underflows still counts with its bound
      const float c = cb[e];
      const float small = p * expm1_small(fminf(c, 1.0f));
      const float big = __expf(x + c) - p;
      st.n += valid ? (c > 1.0f ? big : small) : 0.0f;
    }
    wgt[e] = valid ? p * sv[e] : 0.0f;
  }
  const h4_t wop = h4_t{(_Float16)wgt[0], (_Float16)wgt[1], (_Float16)wgt[2], (_Float16)wgt[3]};
  if constexpr (KIND == WC_KIND_INT8_DITHER)
    st.wsum += ((float)wop[0] + (float)wop[1]) + ((float)wop[2] + (float)wop[3]);

  // ---------------- P V ----------------
  if constexpr (KIND == WC_KIND_INT8_DITHER) {
    __builtin_amdgcn_s_waitcnt(0xc07f);   // LDS writes of this page done
    __builtin_amdgcn_wave_barrier();
    uint4 rows[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      rows[e] = *reinterpret_cast<const uint4*>(my_dsh + (4 * g + e) * kRow + 16 * r);
    const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&rows[0]);
    const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&rows[1]);
    const uint32_t* r2 = reinterpret_cast<const uint32_t*>(&rows[2]);
    const uint32_t* r3 = reinterpret_cast<const uint32_t*>(&rows[3]);
#pragma unroll
    for (int jt = 0; jt < 8; ++jt) {
      const uint32_t x = cur.vw[jt] ^ 0x80808080u;     // codes of channel 8r+jt, tokens 4g..4g+3
      st.o1[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(codes2(x, kSelLo), codes2(x, kSelHi)), wop,
                                                        st.o1[jt], 0, 0, 0);
      const uint32_t sel = (jt & 1) ? kSelH1 : kSelH0;
      const uint32_t d01 = perm(r1[jt >> 1], r0[jt >> 1], sel);
      const uint32_t d23 = perm(r3[jt >> 1], r2[jt >> 1], sel);
      st.o2[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(d01, d23), wop, st.o2[jt], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);   // LDS reads done before the next page overwrites
    __builtin_amdgcn_wave_barrier();
  } else if constexpr (KIND == WC_KIND_FP8_RAW) {
#pragma unroll
    for (int jt = 0; jt < 8; ++jt) {
      const uint32_t x = cur.vw[jt];
      uint32_t lo = e4m3pair(x & 0xFFu, (x >> 8) & 0xFFu);
      uint32_t hi = e4m3pair((x >> 16) & 0xFFu, x >> 24);
      // tokens past the end may hold any byte pattern (the 0x7F NaN code): zero them
      if (t0 + 4 * g + 0 >= t_end) lo &= 0xFFFF0000u;
      if (t0 + 4 * g + 1 >= t_end) lo &= 0x0000FFFFu;
      if (t0 + 4 * g + 2 >= t_end) hi &= 0xFFFF0000u;
      if (t0 + 4 * g + 3 >= t_end) hi &= 0x0000FFFFu;
      st.o1[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(lo, hi), wop, st.o1[jt], 0, 0, 0);
    }
  } else {
#pragma unroll
    for (int jt = 0; jt < 8; ++jt) {
      // bf16 values of channel 8r+jt, tokens 4g..4g+3: 8 bytes at offset 8*jt
      uint32_t lo = bf16pair_to_f16(cur.vw[2 * jt]);
      uint32_t hi = bf16pair_to_f16(cur.vw[2 * jt + 1]);
      if (t0 + 4 * g + 0 >= t_end) lo &= 0xFFFF0000u;
      if (t0 + 4 * g + 1 >= t_end) lo &= 0x0000FFFFu;
      if (t0 + 4 * g + 2 >= t_end) hi &= 0xFFFF0000u;
      if (t0 + 4 * g + 3 >= t_end) hi &= 0x0000FFFFu;
      st.o1[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(lo, hi), wop, st.o1[jt], 0, 0, 0);
    }
  }
}

template <int KIND, bool METER>
__global__ __launch_bounds__(256, 2) void decode_mfma_kernel(DecodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t dsh[KIND == WC_KIND_INT8_DITHER ? kWaves : 1][16 * kRow];
  __shared__ float qn_s[kWaves][16][16];
  __shared__ __attribute__((aligned(16))) float acc_s[kWaves][16][kD];
  __shared__ float ml_s[kWaves][16][3];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const int unit = blockIdx.y;
  const int b = unit / a.n_kv, kv = unit % a.n_kv;
  if (a.mask_kv != nullptr && a.mask_kv[unit] == 0) return;   // whole workgroup
  const int G = a.group;
  const int B = a.n_bands;
  const int L = a.seq_lens[b];
  const int wg_begin = blockIdx.x * a.split_tokens;
  if (blockIdx.x >= a.n_splits || wg_begin >= L) return;      // whole workgroup
  const int wg_end = min(min(L, wg_begin + a.split_tokens), a.max_blocks * kBlockTokens);
  // this wave's share: a contiguous run of pages of the workgroup's split
  const int n_pages = (wg_end - wg_begin + kBlockTokens - 1) / kBlockTokens;
  const int ppw = (n_pages + kWaves - 1) / kWaves;
  const int t_begin = wg_begin + wave * ppw * kBlockTokens;
  const int t_end = min(wg_end, t_begin + ppw * kBlockTokens);

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
  // B operands of QK: the kt-th MFMA uses channels 32g + 8kt .. 32g + 8kt + 7.
  h8_t qop[4];
  s8_t qbf[4];
  float qsum = 0.0f;   // sum of the fp16 queries of head r over all channels
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    if constexpr (KIND == WC_KIND_BF16) {
      qbf[kt] = __builtin_bit_cast(s8_t, make_uint4(qraw[4 * kt], qraw[4 * kt + 1], qraw[4 * kt + 2],
                                                    qraw[4 * kt + 3]));
    } else {
      uint32_t w[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        w[j] = bf16pair_to_f16(qraw[4 * kt + j]);
        const h2_t h = as_h2(w[j]);
        qsum += (float)h[0] + (float)h[1];
      }
      qop[kt] = pack8(w[0], w[1], w[2], w[3]);
    }
  }
  qsum += __shfl_xor(qsum, 16, 64);
  qsum += __shfl_xor(qsum, 32, 64);
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

  WaveState st;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    st.o1[j] = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
    st.o2[j] = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
  }
  st.m = -INFINITY;
  st.l = st.n = st.wsum = 0.0f;
  const uint32_t layer_head = ((uint32_t)a.layer << 16) | (uint32_t)kv;
  uint8_t* my_dsh = dsh[KIND == WC_KIND_INT8_DITHER ? wave : 0];
  const int32_t* trow = a.table + (int64_t)b * a.max_blocks;

  // two page buffers used alternately: loads of one are in flight while the other is computed
  PageRegs<KIND> pa, pb;
  if (t_begin < t_end) load_page<KIND, METER>(a, trow, t_begin, kv, r, g, pa);
  for (int t0 = t_begin; t0 < t_end; t0 += 2 * kBlockTokens) {
    const int t1 = t0 + kBlockTokens;
    if (t1 < t_end) load_page<KIND, METER>(a, trow, t1, kv, r, g, pb);
    process_page<KIND, METER>(a, pa, t0, t_end, r, g, layer_head, qop, qbf, qnop, qsum, my_dsh, st);
    if (t1 >= t_end) break;
    if (t1 + kBlockTokens < t_end) load_page<KIND, METER>(a, trow, t1 + kBlockTokens, kv, r, g, pa);
    process_page<KIND, METER>(a, pb, t1, t_end, r, g, layer_head, qop, qbf, qnop, qsum, my_dsh, st);
  }

  // ---- merge the four waves of the workgroup, write one partial record ----
  st.l += __shfl_xor(st.l, 16, 64);
  st.l += __shfl_xor(st.l, 32, 64);
  if constexpr (METER) {
    st.n += __shfl_xor(st.n, 16, 64);
    st.n += __shfl_xor(st.n, 32, 64);
  }
  if constexpr (KIND == WC_KIND_INT8_DITHER) {
    st.wsum += __shfl_xor(st.wsum, 16, 64);
    st.wsum += __shfl_xor(st.wsum, 32, 64);
  }
  // fp8 operands hold value/256, so the weight scale already cancels there
  constexpr float unscale = KIND == WC_KIND_FP8_RAW ? 1.0f : 1.0f / kWScale;
  // rows 4g+e of tile jt hold channel 8(4g+e)+jt = 32g + 8e + jt
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float v[8];
#pragma unroll
    for (int jt = 0; jt < 8; ++jt) {
      v[jt] = st.o1[jt][e];
      if constexpr (KIND == WC_KIND_INT8_DITHER)
        v[jt] = fmaf(st.o2[jt][e] - kDOff * st.wsum, -0.001953125f, v[jt]);
      v[jt] *= unscale;
    }
    float4* dst = reinterpret_cast<float4*>(&acc_s[wave][r][32 * g + 8 * e]);
    dst[0] = make_float4(v[0], v[1], v[2], v[3]);
    dst[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
  if (g == 0) {
    ml_s[wave][r][0] = st.m;     // -inf for a wave without tokens
    ml_s[wave][r][1] = st.l;
    ml_s[wave][r][2] = st.n;
  }
  __syncthreads();
  const int64_t R = (int64_t)partial_record_floats(kD);
  if (wave == 0 && hv) {   // one partial record per (query head, split)
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, ml_s[w][r][0]);
    float f[kWaves], lsum = 0.0f, nsum = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float mw = ml_s[w][r][0];
      f[w] = mw == -INFINITY ? 0.0f : __expf(mw - M);
      lsum = fmaf(f[w], ml_s[w][r][1], lsum);
      if constexpr (METER) nsum = fmaf(f[w], ml_s[w][r][2], nsum);
    }
    if (isnan(nsum)) nsum = INFINITY;
    float* rec = a.part + (((int64_t)b * a.n_q + (int64_t)kv * G + r) * a.n_splits + blockIdx.x) * R;
#pragma unroll
    for (int i = 0; i < 32; i += 4) {
      float4 sum = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float4 x = *reinterpret_cast<const float4*>(&acc_s[w][r][32 * g + i]);
        sum.x = fmaf(f[w], x.x, sum.x);
        sum.y = fmaf(f[w], x.y, sum.y);
        sum.z = fmaf(f[w], x.z, sum.z);
        sum.w = fmaf(f[w], x.w, sum.w);
      }
      *reinterpret_cast<float4*>(rec + 32 * g + i) = sum;
    }
    if (g == 0) {
      rec[kD] = M;
      rec[kD + 1] = lsum;
      rec[kD + 2] = nsum;
    }
  }

}

}  // namespace

bool mfma_decode_supported(const DecodeArgs& a) {
  return a.head_dim == kD && a.q_dtype == WC_BF16 && a.group <= 16 &&
         (a.kind == WC_KIND_BF16 || a.n_bands == 8 || a.n_bands == 16);
}

hipError_t launch_decode_mfma(const DecodeArgs& a, bool metered, hipStream_t st) {
  const dim3 grid(a.n_splits, a.batch * a.n_kv);
  if (!metered)
    hipLaunchKernelGGL((decode_mfma_kernel<WC_KIND_BF16, false>), grid, dim3(64 * kWaves), 0, st, a);
  else if (a.kind == WC_KIND_INT8_DITHER)
    hipLaunchKernelGGL((decode_mfma_kernel<WC_KIND_INT8_DITHER, true>), grid, dim3(64 * kWaves), 0, st, a);
  else
    hipLaunchKernelGGL((decode_mfma_kernel<WC_KIND_FP8_RAW, true>), grid, dim3(64 * kWaves), 0, st, a);
  return hipGetLastError();
}

}  // namespace wc
