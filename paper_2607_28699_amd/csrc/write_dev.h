// Device side of the write path, shared by the write kernel and the decode
// kernel that writes a step's new tokens before it reads them (Sec. 4.2
// subtractive dither; Sec. 6.2 research kernels and storage side; Sec. 4.1 Eq.
// witness).
//
// One token-head (one token of one KV head, K and V together) is handled by
// D/16 lanes, lane g owning channels 16g .. 16g+15 -- exactly one Philox call
// of dither, shared by K and V.  The squared key residuals stay in registers: a
// band is one run of consecutive channels (interleaved pairs) or two runs half a
// head apart (rotate-half pairs), so each lane sums its runs and the partner
// lanes' runs arrive by shuffles; each band norm is then rounded up to fp16.  The
// residuals are exact in float64 (a dequantized value needs 28 bits), and
// squares, sums and square roots are taken in float64 too, so the stored witness
// is the fp16 round-up of the float64 band norm.
#pragma once

#include "wc_device.h"
#include "wc_launch.h"

namespace wc {

template <int D, typename TIn>
__device__ __forceinline__ void load16(const TIn* src, float (&x)[16]) {
  if constexpr (sizeof(TIn) == 4) {
    const float4* p = reinterpret_cast<const float4*>(src);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float4 v = p[i];
      x[4 * i] = v.x; x[4 * i + 1] = v.y; x[4 * i + 2] = v.z; x[4 * i + 3] = v.w;
    }
  } else {
    const uint4* p = reinterpret_cast<const uint4*>(src);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      uint4 v = p[i];
      uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[8 * i + 2 * j] = bf16_to_f32((uint16_t)(w[j] & 0xFFFFu));
        x[8 * i + 2 * j + 1] = bf16_to_f32((uint16_t)(w[j] >> 16));
      }
    }
  }
}

// Per-token, per-head fp16 scale s = round_up(fl32(amax / 126.5)) and fl32(1/s).
__device__ __forceinline__ void int8_scale(float amax, uint16_t& s_bits, float& s, float& inv) {
  s_bits = f16_round_up(__fdiv_rn(amax, 126.5f));
  s = f16_to_f32(s_bits);
  inv = s > 0.0f ? __fdiv_rn(1.0f, s) : 0.0f;
}

// Dithered code round(x * inv + xi) (Sec. 4.2): the product is rounded to fp32
// before the dither is added, never fused with the add into one fma, so that a
// code next to a half-integer is decided as the quantizer defines it.
__device__ __forceinline__ float dither_code(float x, float inv, float xi) {
#pragma clang fp contract(off)
  return rintf(x * inv + xi);
}

// Value rows of a token, staged in LDS by the write kernel: the codes (or bf16
// values of an exact copy) in channel order, stored afterwards by token quads as
// whole 16-byte pieces of the page (null pointers: stored here, element by element).
struct VStage {
  uint32_t* codes;   // [D / 4] words: the token's D value codes
  uint32_t* exact;   // [D / 2] words: the token's D bf16 values of the exact copy
};

// bf16 copy of one token-head's 16 channels (this lane's share) into an exact cache
// (values to vst.exact when staged).
template <int D>
__device__ __forceinline__ void store_exact(void* k_data, void* v_data, int64_t bh, int off, int g,
                                            const float (&k)[16], const float (&v)[16], bool active,
                                            uint32_t* vst) {
  uint32_t kw[8], vw[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    kw[i] = (uint32_t)f32_to_bf16_rne(k[2 * i]) | ((uint32_t)f32_to_bf16_rne(k[2 * i + 1]) << 16);
    vw[i] = (uint32_t)f32_to_bf16_rne(v[2 * i]) | ((uint32_t)f32_to_bf16_rne(v[2 * i + 1]) << 16);
  }
  if (vst != nullptr) {
    reinterpret_cast<uint4*>(vst + 8 * g)[0] = make_uint4(vw[0], vw[1], vw[2], vw[3]);
    reinterpret_cast<uint4*>(vst + 8 * g)[1] = make_uint4(vw[4], vw[5], vw[6], vw[7]);
  }
  if (!active) return;
  uint8_t* kpg = reinterpret_cast<uint8_t*>(k_data) + bh * (kBlockTokens * D * 2);
  *reinterpret_cast<uint4*>(kpg + kpage_off(off, 16 * g, D, 2)) = make_uint4(kw[0], kw[1], kw[2], kw[3]);
  *reinterpret_cast<uint4*>(kpg + kpage_off(off, 16 * g + 8, D, 2)) = make_uint4(kw[4], kw[5], kw[6], kw[7]);
  if (vst != nullptr) return;
  uint8_t* vpg = reinterpret_cast<uint8_t*>(v_data) + bh * (kBlockTokens * D * 2);
#pragma unroll
  for (int i = 0; i < 16; ++i)
    *reinterpret_cast<uint16_t*>(vpg + vpage_off(off, 16 * g + i, D, 2)) =
        (uint16_t)(vw[i >> 1] >> (16 * (i & 1)));
}

// Value codes of one lane's 16 channels: to the token's staged row, or byte by
// byte into the token-quad interleaved page.
template <int D>
__device__ __forceinline__ void store_vcodes(const WriteArgs& a, int64_t bh, int off, int g, const uint32_t (&vc)[4],
                                             bool active, uint32_t* vst) {
  if (vst != nullptr) {
    reinterpret_cast<uint4*>(vst)[g] = make_uint4(vc[0], vc[1], vc[2], vc[3]);
    return;
  }
  if (!active) return;
#pragma unroll
  for (int i = 0; i < 16; ++i)
    reinterpret_cast<uint8_t*>(a.v_data)[bh * (kBlockTokens * D) + vpage_off(off, 16 * g + i, D, 1)] =
        (uint8_t)(vc[i >> 2] >> (8 * (i & 3)));
}

// Key witness of one token-head (Sec. 4.1, Eq. witness) from this lane's squared
// residuals q2 of channels 16g .. 16g+15: band b holds the channels of RoPE pairs
// bP .. bP+P-1, P = D / (2B), i.e. one run of R = D/B channels (interleaved) or
// two runs of R = D/(2B) channels D/2 apart (rotate-half).  R is a power of two:
// a lane holds 16/R runs (R <= 16) or a share of one (then the run's lanes add by
// shuffles); a rotate-half band adds the run of lane g + D/32.  The lanes holding
// a band's first run store its fp16 round-up, their bands in one store.
template <int D>
__device__ __forceinline__ void store_witness(const WriteArgs& a, const double (&q2)[16], int64_t bh, int off,
                                              int g, bool active) {
  constexpr int LPT = D / 16;
  const int B = a.n_bands;
  const int R = a.interleaved ? D / B : D / (2 * B);
  double s2[8], s4[4], s8[2];
#pragma unroll
  for (int i = 0; i < 8; ++i) s2[i] = q2[2 * i] + q2[2 * i + 1];
#pragma unroll
  for (int i = 0; i < 4; ++i) s4[i] = s2[2 * i] + s2[2 * i + 1];
  s8[0] = s4[0] + s4[1];
  s8[1] = s4[2] + s4[3];
  double run[8];
  int nrun;
  if (R == 2) {
    nrun = 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) run[i] = s2[i];
  } else if (R == 4) {
    nrun = 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) run[i] = s4[i];
  } else if (R == 8) {
    nrun = 2;
    run[0] = s8[0];
    run[1] = s8[1];
  } else {
    nrun = 1;
    run[0] = s8[0] + s8[1];
    for (int o = 1; o < R / 16; o <<= 1) run[0] += __shfl_xor(run[0], o, LPT);
  }
  if (!a.interleaved) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (j < nrun) run[j] += __shfl_xor(run[j], LPT / 2, LPT);
  }
  const bool owner = (a.interleaved || g < LPT / 2) && (R <= 16 || g % (R / 16) == 0);
  if (!owner || !active) return;
  uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
  for (int j = 0; j < 8; ++j)
    if (j < nrun) w[j >> 1] |= (uint32_t)f16_round_up_f64(sqrt(run[j])) << (16 * (j & 1));
  // bands b0 .. b0+nrun-1 of the token's row (B fp16 values; aligned to 2 nrun bytes)
  uint8_t* dst = reinterpret_cast<uint8_t*>(a.k_witness) + ((bh * kBlockTokens + off) * B + (16 * g) / R) * 2;
  if (nrun == 8) *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
  else if (nrun == 4) *reinterpret_cast<uint2*>(dst) = make_uint2(w[0], w[1]);
  else if (nrun == 2) *reinterpret_cast<uint32_t*>(dst) = w[0];
  else *reinterpret_cast<uint16_t*>(dst) = (uint16_t)w[0];
}

// One token-head of the write (token tok, KV head h; in_range false: nothing to
// do), by the D/16 lanes that own it, lane g holding channels 16g .. 16g+15
// (lanes g of one token-head are consecutive and aligned: the reductions are
// shuffles of width D/16).  Quantizes K and V, stores codes, scales, bypassed
// values, the value side, the exact copy and the key witness.  Returns the slot
// written, or -1 when the token is skipped.  With vst the value rows go to LDS
// (VStage) for the caller to store.  BYP: the cache may bypass outlier pairs
// (a.n_pairs > 0); without it the per-channel bypass selects are compiled out.
template <int D, int KIND, typename TIn, bool BYP>
__device__ __forceinline__ int64_t write_token_head(const WriteArgs& a, int64_t tok, int h, bool in_range, int g,
                                                    VStage vst = VStage{nullptr, nullptr}) {
  constexpr int LPT = D / 16;                 // lanes per token-head
  const int64_t slot = in_range ? a.slots[tok] : -1;
  const bool active = in_range && slot >= 0 && slot < a.n_slots;   // others are skipped

  // (the inputs are requested with the slot, not after it: a skipped token's values
  // are computed on but never stored)
  float k[16], v[16];
  if (in_range) {
    const TIn* kp = reinterpret_cast<const TIn*>(a.k) + (tok * a.n_kv + h) * D + 16 * g;
    const TIn* vp = reinterpret_cast<const TIn*>(a.v) + (tok * a.n_kv + h) * D + 16 * g;
    load16<D>(kp, k);
    load16<D>(vp, v);
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) k[i] = v[i] = 0.0f;
  }
  const int64_t blk = active ? slot / kBlockTokens : 0;
  const int off = active ? (int)(slot % kBlockTokens) : 0;
  const int64_t bh = blk * a.n_kv + h;        // (block, head) page index
  const int64_t slot_out = active ? slot : -1;   // the witness pass skips what this one skipped

  double vr2 = 0.0, vn2 = 0.0;   // value side: ||vhat - v||^2 and ||v||^2 of this lane's channels
  const bool vside = a.v_resid != nullptr;
  double q2[16];                 // squared key residuals of this lane's channels
  if constexpr (KIND == WC_KIND_INT8_DITHER) {
    // Bypassed key channels of this lane (outlier RoPE pairs, Sec. 6.2): out of the
    // amax, code 0, value kept in fp16 (bit i: channel 16g + i).
    uint32_t bmask = 0;
    const int32_t* plist = a.pairs + (int64_t)h * a.n_pairs;
    if constexpr (BYP) {
      for (int i = 0; i < a.n_pairs; ++i) {
        const int j = plist[i];
#pragma unroll
        for (int sec = 0; sec < 2; ++sec) {
          const int c = pair_channel(j, sec, D, a.interleaved) - 16 * g;
          if (c >= 0 && c < 16) bmask |= 1u << c;
        }
      }
    }
    float ak = 0.0f, av = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (!BYP || ((bmask >> i) & 1u) == 0) ak = fmaxf(ak, fabsf(k[i]));
      av = fmaxf(av, fabsf(v[i]));
    }
    // group scales (Sec. 6.2 storage side, Table 4): the 32-channel group of this
    // lane is lanes g, g^1, and its fp16 scale is formed from the group's amax as the
    // token scale is from the token's
    const bool grouped = a.group_scales != 0;
    if (grouped) {
      ak = fmaxf(ak, __shfl_xor(ak, 1, LPT));
      av = fmaxf(av, __shfl_xor(av, 1, LPT));
    } else {
#pragma unroll
      for (int o = 1; o < LPT; o <<= 1) {
        ak = fmaxf(ak, __shfl_xor(ak, o, LPT));
        av = fmaxf(av, __shfl_xor(av, o, LPT));
      }
    }
    uint16_t skb, svb;
    float sk, ikk, sv, ivv;
    int8_scale(ak, skb, sk, ikk);
    int8_scale(av, svb, sv, ivv);
    const double stk = (double)sk, stv = (double)sv;

    const U4 rnd = dither_block(g, slot, ((uint32_t)a.layer << 16) | (uint32_t)h, a.key0, a.key1);
    const uint32_t words[4] = {rnd.x, rnd.y, rnd.z, rnd.w};
    uint32_t kc[4] = {0, 0, 0, 0}, vc[4] = {0, 0, 0, 0};
    float dv[16];   // cv - xi of the value channels (the value side's residuals)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const bool byp = BYP && ((bmask >> i) & 1u);
      const float xi = dither_value((words[i >> 2] >> (8 * (i & 3))) & 0xFFu);
      // a bypassed channel quantizes 0 (|xi| < 1/2, so its code is 0)
      const float ck = dither_code(byp ? 0.0f : k[i], ikk, xi);
      const float cv = dither_code(v[i], ivv, xi);
      double rk = stk * (double)(ck - xi) - (double)k[i];                      // khat - k (step of the group)
      if constexpr (BYP)
        if (byp) rk = (double)(float)(_Float16)k[i] - (double)k[i];           // fp16(k) - k
      q2[i] = rk * rk;
      dv[i] = cv - xi;
      // codes are stored excess-128: byte = code + 128 (an exact integer in 1 .. 255,
      // converted and placed into its byte by one instruction)
      kc[i >> 2] = __builtin_amdgcn_cvt_pk_u8_f32(ck + 128.0f, i & 3, kc[i >> 2]);
      vc[i >> 2] = __builtin_amdgcn_cvt_pk_u8_f32(cv + 128.0f, i & 3, vc[i >> 2]);
    }
    if (vside) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const double rv = stv * (double)dv[i] - (double)v[i];                  // vhat - v
        vr2 = fma(rv, rv, vr2);
        vn2 = fma((double)v[i], (double)v[i], vn2);
      }
    }
    store_vcodes<D>(a, bh, off, g, vc, active, vst.codes);
    if (active) {
      *reinterpret_cast<uint4*>(reinterpret_cast<uint8_t*>(a.k_data) + bh * (kBlockTokens * D) +
                                kpage_off(off, 16 * g, D, 1)) = make_uint4(kc[0], kc[1], kc[2], kc[3]);
      if (grouped) {   // the first lane of each group stores the group's scales
        if ((g & 1) == 0) {
          a.k_scale[(bh * kBlockTokens + off) * (D / 32) + (g >> 1)] = skb;
          a.v_scale[(bh * kBlockTokens + off) * (D / 32) + (g >> 1)] = svb;
        }
      } else if (g == 0) {
        a.k_scale[bh * kBlockTokens + off] = skb;
        a.v_scale[bh * kBlockTokens + off] = svb;
      }
      if (BYP && bmask != 0) {
        // fp16 (nearest-even) values of the bypassed channels, in pair order
        const TIn* kp = reinterpret_cast<const TIn*>(a.k) + (tok * a.n_kv + h) * D;
        uint16_t* orow = a.k_outlier + (bh * kBlockTokens + off) * (int64_t)(2 * a.n_pairs);
        for (int i = 0; i < a.n_pairs; ++i) {
          const int j = plist[i];
#pragma unroll
          for (int sec = 0; sec < 2; ++sec) {
            const int c = pair_channel(j, sec, D, a.interleaved);
            if (c >= 16 * g && c < 16 * g + 16) {
              const float x = sizeof(TIn) == 4 ? (float)reinterpret_cast<const float*>(kp)[c]
                                               : bf16_to_f32(reinterpret_cast<const uint16_t*>(kp)[c]);
              orow[2 * i + sec] = f16_bits((_Float16)x);
            }
          }
        }
      }
    }
  } else if constexpr (KIND == WC_KIND_FP8_RAW) {
    uint32_t kc[4] = {0, 0, 0, 0}, vc[4] = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t bk = f32_to_e4m3_sat(k[i]);
      const uint32_t bv = f32_to_e4m3_sat(v[i]);
      const double rk = (double)e4m3_to_f32(bk) - (double)k[i];
      q2[i] = rk * rk;
      if (vside) {
        const double rv = (double)e4m3_to_f32(bv) - (double)v[i];
        vr2 = fma(rv, rv, vr2);
        vn2 = fma((double)v[i], (double)v[i], vn2);
      }
      kc[i >> 2] |= bk << (8 * (i & 3));
      vc[i >> 2] |= bv << (8 * (i & 3));
    }
    store_vcodes<D>(a, bh, off, g, vc, active, vst.codes);
    if (active) {
      *reinterpret_cast<uint4*>(reinterpret_cast<uint8_t*>(a.k_data) + bh * (kBlockTokens * D) +
                                kpage_off(off, 16 * g, D, 1)) = make_uint4(kc[0], kc[1], kc[2], kc[3]);
    }
  } else {  // WC_KIND_BF16: exact cache, no witness
    store_exact<D>(a.k_data, a.v_data, bh, off, g, k, v, active, vst.exact);
    return slot_out;
  }
  if (a.x_k_data != nullptr) store_exact<D>(a.x_k_data, a.x_v_data, bh, off, g, k, v, active, vst.exact);
  store_witness<D>(a, q2, bh, off, g, active);
  if (vside) {   // value side (Sec. 3 output bound): residual norm up, value norm down
#pragma unroll
    for (int o = 1; o < LPT; o <<= 1) {
      vr2 += __shfl_xor(vr2, o, LPT);
      vn2 += __shfl_xor(vn2, o, LPT);
    }
    if (active && g == 0) {
      a.v_resid[bh * kBlockTokens + off] = f16_round_up_f64(sqrt(vr2));
      a.v_norm[bh * kBlockTokens + off] = f16_round_down_f64(sqrt(vn2));
    }
  }
  return slot_out;
}

}  // namespace wc
