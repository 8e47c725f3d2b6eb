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
//         dither enters as a second product into the same accumulator with
//         E = -(4 + u/256) (exact in fp16: bits 0xC400 | u, one byte permute from
//         the Philox byte u); since xi = (u - 127.5)/256 = -E - 4 - 127.5/256,
//         q . khat = s (q . code + q . E + (4 + 127.5/256) sum(q)).
//   bound c_t = sm_scale sum_b ||q_b|| w_{t,b}: one more MFMA, witness (fp16,
//         exact) times band norms split into fp16 hi + lo parts.
//   softmax online over the page; the running max is only raised when a page
//         exceeds it by more than kSlack (then the accumulators are rescaled),
//         so the common case needs no cross-lane exchange.
//   PV    O^T = V^T W with v_mfma_f32_16x16x16_f16: A = value codes + 1152 (the
//         stored byte as fp16 1024 + u, one permute) of 16 channels x 4 tokens per
//         lane group (the value pages are stored token-quad interleaved, so this is
//         one 32-byte load), B = p_t s^v_t in fp16, and a second product with E,
//         transposed through LDS, into the same accumulators; the offset
//         1152 - 4 - 127.5/256 is removed at the end with the running sum of the
//         fp16 weights.
//
// Lane l: r = l % 16 (token in the QK operands, head in B and in the results,
// channel row in the PV operands), g = l / 16 (k-group).  The channel order of
// the QK contraction is permuted so that lane group g owns channels 32g..32g+31,
// i.e. exactly the two Philox calls (16 channels each) it regenerates.  Pages
// stream through a ring of register buffers: the next pages' loads are in flight
// while the current page is computed.
//
// Group scales (GS; Sec. 6.2 storage side, Table 4: one fp16 scale per token and
// 32-channel group): every QK product must then cover one group, so that its sum
// can be weighted by the token's group scale.  The lane's 32 key channels (one
// group) are exchanged among the four lane groups, 8 channels at a time, with two
// rounds of gfx950 lane swaps (a 4 x 4 block transpose: permlane32, then
// permlane16): after it, chunk G of lane (r, g) holds channels 32G + 8g .. of
// token r, and product G of the codes and of the dither gives group G's exact
// partial q . (code - xi), weighted in fp32 by s_{t,G}.  The keys' logits stay
// exact.  In PV the rows of lane (r, g) are channels 8r .. 8r + 7, all in group
// r / 4, so the value scale enters the fp16 value operand: s_{t,G} 2^-ve (code + E)
// with two fp16 roundings (the per-token path rounds its weight p s_t to fp16
// instead, an error of the same order), and the dither offset is removed with
// one more product of the scales and the weights.
#pragma once

#include <float.h>

#include <type_traits>

#include "merge_dev.h"
#include "wc_device.h"
#include "wc_launch.h"
#include "write_dev.h"

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
// by 2^8 (cancelled by the same factor in the weight sum), which keeps small
// weights out of the fp16 subnormal range.  The INT8 operand p s^v 2^8 also
// carries 2^-ve, ve a running value exponent (0 at the start, raised to cover a
// page's largest value scale, with the accumulators rescaled by the exact power
// of two), so it stays below e^2 2^8 < 65504 for any fp16 value scale.
constexpr float kSlack = 2.0f;
constexpr float kQOff = 4.498046875f;    // 4 + 127.5/256: code - xi = code + E + kQOff
constexpr float kVOff = 1147.501953125f; // 1152 - kQOff: (code + 1152) + E = code - xi + kVOff

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

// Two codes stored excess-128 (byte u = code + 128) -> fp16 (1024 + u) - 1152 = code, exact.
__device__ __forceinline__ uint32_t codes2(uint32_t xb, uint32_t sel) {
  return as_u32(as_h2(perm(0x64646464u, xb, sel)) - h2_t{(_Float16)1152.0f, (_Float16)1152.0f});
}
// Two stored bytes u -> fp16 1024 + u = code + 1152 (exact): the value operand of
// PV, whose offset is removed once at the end with the weight sum.
__device__ __forceinline__ uint32_t ucodes2(uint32_t xb, uint32_t sel) {
  return perm(0x64646464u, xb, sel);
}
// Two dither bytes u -> fp16 E = -(4 + u/256) (bits 0xC400 | u), exact, one permute.
__device__ __forceinline__ uint32_t ndith2(uint32_t u, uint32_t sel) {
  return perm(0xC4C4C4C4u, u, sel);
}
// Two E4M3 bytes (bytes 0, 1 of w, or 2, 3 with HI) -> fp16 pair, one gfx950
// conversion instruction at scale 1: every E4M3 value, subnormals included, is
// a normal fp16 number (|x| in [2^-9, 448]), so the conversion is exact.
template <bool HI>
__device__ __forceinline__ uint32_t e4m3x2(uint32_t w) {
  return as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, HI));
}
// Two bf16 -> fp16 pair (exact for |x| in the fp16 normal range).
__device__ __forceinline__ uint32_t bf16pair_to_f16(uint32_t w) {
  const float a = bf16_to_f32((uint16_t)(w & 0xFFFFu));
  const float b = bf16_to_f32((uint16_t)(w >> 16));
  return as_u32(h2_t{(_Float16)a, (_Float16)b});
}

// The same times 2^k (k <= 0, a power of two in f32): exact unless the result
// leaves the fp16 normal range.
__device__ __forceinline__ uint32_t bf16pair_to_f16_scaled(uint32_t w, float two_k) {
  const float a = bf16_to_f32((uint16_t)(w & 0xFFFFu)) * two_k;
  const float b = bf16_to_f32((uint16_t)(w >> 16)) * two_k;
  return as_u32(h2_t{(_Float16)a, (_Float16)b});
}


__device__ __forceinline__ h8_t pack8(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  return __builtin_bit_cast(h8_t, make_uint4(a, b, c, d));
}
__device__ __forceinline__ h4_t pack4(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(h4_t, make_uint2(a, b));
}

// (butterfly steps without LDS: merge_dev.h)
template <int M>
__device__ __forceinline__ float xor_max(float v) { return bfly_max<M>(v); }

// Loaded bytes of one 16-token page for one lane.
template <int KIND>
struct PageRegs {
  static constexpr int NW = KIND == WC_KIND_BF16 ? 16 : 8;
  uint32_t kw[NW];   // keys of token r, channels 32g..32g+31
  uint32_t vw[NW];   // values of channels 8r..8r+7 for token quad g
  uint2 ks, vs;      // fp16 scales of tokens 4g..4g+3 (group scales: vs holds those of group r/4)
  uint32_t kg;       // group scales: dword r % 8 of the key scales of tokens 4g..4g+3 ([token][group] fp16)
  uint4 wit;         // witness bands 8(g%2).. of token r (zeros where 8(g%2) >= n_bands)
  uint4 ov;          // fp16 keys of bypassed pairs: values 8g .. 8g+7 of token r (when 8g < 2m)
  uint2 vr, vn;      // value side: stored ||vhat - v|| and ||v|| of tokens 4g..4g+3
  int blk;           // cache block of the page (wave-uniform)
};

// Buffer resource over one page of one tensor.  A page past the end of the
// wave's range gets an empty resource: its loads return zeros without touching
// memory, so every load is issued unconditionally and the in-order load counter
// stays exact (a conditional load makes the compiler wait for all of them).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t page_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}
// Page data is read once per call: the loads carry the nontemporal hint (cache
// policy bit 1, "nt" on gfx950), which lets a streaming read reach 7.1-7.3 TB/s
// on the part against 6.3 TB/s with ordinary loads (measured with plain read
// kernels over 4 GiB).
constexpr int kPageAux = 2;
__device__ __forceinline__ uint4 bload16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kPageAux));
}
__device__ __forceinline__ uint2 bload8(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kPageAux));
}
__device__ __forceinline__ uint32_t bload2x2(__amdgpu_buffer_rsrc_t r, int off0, int off1) {
  const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(r, off0, 0, kPageAux);
  const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(r, off1, 0, kPageAux);
  return lo | (hi << 16);
}

template <int KIND, bool METER, bool TB, bool BYP, bool VM, bool GS>
__device__ __forceinline__ void load_page(const DecodeArgs& a, int blk, bool valid, int kv, int r,
                                          int g, int wit_off, PageRegs<KIND>& p) {
  constexpr int KB = KIND == WC_KIND_BF16 ? 64 : 32;   // bytes per lane and tensor
  constexpr int PB = kBlockTokens * kD * (KB / 32);    // bytes per page and tensor
  p.blk = blk;
  // an entry outside the cache reads zeros: its resources start at the cache's first
  // page and cover nothing, so no address outside the cache is ever formed
  valid = valid && (int64_t)(uint32_t)blk < a.num_blocks;
  const int64_t page = valid ? (int64_t)blk * a.n_kv + kv : 0;
  const auto kr = page_rsrc(reinterpret_cast<const uint8_t*>(a.k_data) + page * PB, valid ? PB : 0);
  const auto vr = page_rsrc(reinterpret_cast<const uint8_t*>(a.v_data) + page * PB, valid ? PB : 0);
  // piece (i, g, r) of the page layout (kpage_off / vpage_off): keys of token r,
  // channels 32g + 32i/CL ..; values of quad g, channels 8r ..; one 16-byte piece
  // per lane and instruction, so each instruction covers whole cache lines
  const int lane = 16 * g + r;
#pragma unroll
  for (int i = 0; i < KB / 16; ++i) {
    const uint4 k4 = bload16(kr, (64 * i + lane) * 16), v4 = bload16(vr, (64 * i + lane) * 16);
    p.kw[4 * i] = k4.x; p.kw[4 * i + 1] = k4.y; p.kw[4 * i + 2] = k4.z; p.kw[4 * i + 3] = k4.w;
    p.vw[4 * i] = v4.x; p.vw[4 * i + 1] = v4.y; p.vw[4 * i + 2] = v4.z; p.vw[4 * i + 3] = v4.w;
  }
  if constexpr (KIND == WC_KIND_INT8_DITHER && GS) {
    // [16 tokens][4 groups] fp16 per page and tensor: token t, group G at byte 8t + 2G
    constexpr int kGS = kD / 32;
    const int sb = valid ? 2 * kBlockTokens * kGS : 0;
    // (every lane of a row needs the same 32 bytes: one dword per lane, shared by
    // row broadcasts in process_page)
    const auto kr = page_rsrc(a.k_scale + page * kBlockTokens * kGS, sb);
    p.kg = __builtin_amdgcn_raw_buffer_load_b32(kr, 32 * g + 4 * (r & 7), 0, kPageAux);
    // the value scales of the lane's PV rows (group r/4) for tokens 4g .. 4g+3
    const auto vr = page_rsrc(a.v_scale + page * kBlockTokens * kGS, sb);
    const int vo = 32 * g + 2 * (r >> 2);
    p.vs = make_uint2(bload2x2(vr, vo, vo + 8), bload2x2(vr, vo + 16, vo + 24));
  } else if constexpr (KIND == WC_KIND_INT8_DITHER) {
    const int sb = valid ? 2 * kBlockTokens : 0;
    p.ks = bload8(page_rsrc(a.k_scale + page * kBlockTokens, sb), 8 * g);
    p.vs = bload8(page_rsrc(a.v_scale + page * kBlockTokens, sb), 8 * g);
  }
  if constexpr (METER && !TB) {   // Tier B reads no witness
    const int wb = valid ? 2 * kBlockTokens * a.n_bands : 0;
    p.wit = bload16(page_rsrc(a.k_witness + page * kBlockTokens * a.n_bands, wb), wit_off);
  }
  if constexpr (BYP) {
    // rows of 4m bytes; a lane past its row's values reads the next row (or, at the
    // page end, zeros from the resource bound) and masks them in process_page
    const int ob = 4 * a.n_pairs * kBlockTokens;
    p.ov = bload16(page_rsrc(a.k_outlier + page * (2 * a.n_pairs * kBlockTokens), valid ? ob : 0),
                   r * 4 * a.n_pairs + 16 * g);
  }
  if constexpr (VM) {
    const int sb = valid ? 2 * kBlockTokens : 0;
    p.vr = bload8(page_rsrc(a.v_resid + page * kBlockTokens, sb), 8 * g);
    p.vn = bload8(page_rsrc(a.v_norm + page * kBlockTokens, sb), 8 * g);
  }
}

// A page marked as repaired (persistent repair, Sec. 6 gate): its bf16 keys and
// values from the exact store, in the bf16 page layout, with the stored value
// norm (value side) and no witness, scale or value residual, so that the page
// enters with bound 0.
template <bool VM>
__device__ __forceinline__ void load_exact_page(const DecodeArgs& a, int blk, bool valid, int kv, int r, int g,
                                                PageRegs<WC_KIND_BF16>& p) {
  constexpr int PB = kBlockTokens * kD * 2;   // bytes per bf16 page and tensor
  p.blk = blk;
  valid = valid && (int64_t)(uint32_t)blk < a.num_blocks;
  const int64_t page = valid ? (int64_t)blk * a.n_kv + kv : 0;
  const auto kr = page_rsrc(reinterpret_cast<const uint8_t*>(a.x_k_data) + page * PB, valid ? PB : 0);
  const auto vr = page_rsrc(reinterpret_cast<const uint8_t*>(a.x_v_data) + page * PB, valid ? PB : 0);
  const int lane = 16 * g + r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint4 k4 = bload16(kr, (64 * i + lane) * 16), v4 = bload16(vr, (64 * i + lane) * 16);
    p.kw[4 * i] = k4.x; p.kw[4 * i + 1] = k4.y; p.kw[4 * i + 2] = k4.z; p.kw[4 * i + 3] = k4.w;
    p.vw[4 * i] = v4.x; p.vw[4 * i + 1] = v4.y; p.vw[4 * i + 2] = v4.z; p.vw[4 * i + 3] = v4.w;
  }
  p.ks = p.vs = p.vr = make_uint2(0, 0);
  p.wit = p.ov = make_uint4(0, 0, 0, 0);
  p.vn = VM ? bload8(page_rsrc(a.v_norm + page * kBlockTokens, valid ? 2 * kBlockTokens : 0), 8 * g)
            : make_uint2(0, 0);
}

// Running state of one wave.  Logits are kept in log2 units; every weight carries
// an extra factor 2^8 (the exponent is raised by 8), which keeps the fp16 PV
// operand out of the subnormal range and cancels in out / l and n / l.
struct WaveState {
  f4_t o1[8];            // PV accumulators (INT8: code and dither products together)
  float m, l, n, wsum;   // running max (log2 units), sum of weights, meter numerator, sum of fp16 weights
  float nb;              // meter numerator of the current block segment (block repair's shares)
  int ve;                // INT8 value exponent (wave-uniform, scalar): PV weights carry 2^-ve, and 2^ve
                         // bounds the value scales seen so far
  float ev, vmax;        // value side: sum of weights x stored ||vhat - v||, largest stored ||v||
  f4_t ws4;              // group scales: sum_t w_t s_{t,g} 2^-ve of the lane's output group (rows 4g..4g+3)
};

// Per-wave constants of the page loop.
struct WaveConst {
  h8_t qop[4];     // fp16 queries, B operands of QK (channels 32g + 8kt ..)
  s8_t qbf[4];     // bf16 queries (bf16 cache)
  h8_t qnop;       // band norms * sm_scale * log2(e), hi (g < 2) / lo (g >= 2) parts
  float s1_init;   // (4 + 127.5/256) sum(q): the dither offset, preloaded into the code accumulator
  float lmul;      // logit multiplier: sm_scale * log2(e)
  float ab2;       // Tier B: (alpha_h + beta_h) * log2(e)
  h8_t qo;         // bypassed pairs: fp16 queries at the stored values 8g .. 8g+7
  h8_t qa;         // their magnitudes (Tier B rounding term)
  float gmul;      // Tier B: sm_scale * 2^-11 * log2(e)
  float gc;        // Tier B: sm_scale * 2^-25 * log2(e) * sum |q_c| over the bypassed channels
  uint32_t layer_head;
  bool ov_lo, ov_hi;   // this lane's stored values 8g..8g+3, 8g+4..8g+7 exist (< 2m)
  // group scales: qop[G] holds channels 32G + 8g .. of head r (the group-ordered
  // products); (4 + 127.5/256) times the group's query sum; Tier B's radius
  // coefficients log2(e)^2 sm^2 rt^2 ||q_G||^2 and log2(e) sm ||q_G||_1 / 256
  float qoff[4], ta2[4], tb1[4];
};

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kWExp = 8.0f;                 // weights carry 2^kWExp
constexpr float kSlack2 = kSlack * kLog2e;    // kSlack in log2 units
constexpr float kTaylorMax = 0.5f * kLog2e;   // c <= 0.5 in log2 units

// 2^x - 1 for 0 <= x <= log2(e)/2 (that is e^c - 1, c = x ln 2 <= 1/2) by the
// Taylor series of e^c to c^7/7! (relative error below 2e-7).
__device__ __forceinline__ float exp2m1_small(float x) {
  float s = 1.5252733804059840e-05f;
  s = fmaf(s, x, 1.5403530393381609e-04f);
  s = fmaf(s, x, 1.3333558146428443e-03f);
  s = fmaf(s, x, 9.6181291076284772e-03f);
  s = fmaf(s, x, 5.5504108664821580e-02f);
  s = fmaf(s, x, 2.4022650695910071e-01f);
  s = fmaf(s, x, 6.9314718055994531e-01f);
  return s * x;
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// DPP row shifts within each 16-lane row: lanes 8..15 take `from` of lane - 8
// (lanes 0..7 keep `keep`); lanes 0..7 take `v` of lane + 8 (lanes 8..15 get 0).
__device__ __forceinline__ float dpp_from_lower8(float keep, float from) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, keep),
                                                               __builtin_bit_cast(int, from),
                                                               0x118 /* row_shr:8 */, 0xF, 0xC, false));
}
__device__ __forceinline__ uint32_t dpp_from_upper8(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x108 /* row_shl:8 */, 0xF, 0x3, false);
}

// 4 x 4 block transpose of 2-dword chunks across the four lane groups (16 lanes
// each): afterwards chunk c of lane group g holds what chunk g of lane group c
// held.  Two butterfly rounds of gfx950 lane swaps: permlane32 exchanges the upper
// lane groups of chunks 0, 1 with the lower lane groups of chunks 2, 3 (bit 1 of
// lane group and chunk), permlane16 the odd lane groups of chunks 0, 2 with the
// even lane groups of chunks 1, 3 (bit 0).
__device__ __forceinline__ void transpose_chunks(uint32_t (&w)[8]) {
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      const auto x = __builtin_amdgcn_permlane32_swap(w[2 * c + d], w[2 * c + 4 + d], false, false);
      w[2 * c + d] = x[0];
      w[2 * c + 4 + d] = x[1];
    }
#pragma unroll
  for (int c = 0; c < 4; c += 2)
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      const auto x = __builtin_amdgcn_permlane16_swap(w[2 * c + d], w[2 * c + 2 + d], false, false);
      w[2 * c + d] = x[0];
      w[2 * c + 2 + d] = x[1];
    }
}

// Dword k of each 16-lane row, to every lane of the row (DPP row_newbcast:k).
template <int k>
__device__ __forceinline__ uint32_t row_bcast(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x150 + k, 0xF, 0xF, true);
}
// The key group scales of tokens 4g..4g+3 as 8 dwords (token e: dwords 2e, 2e+1
// hold groups 0, 1 and 2, 3), gathered from the row's lanes 0..7.
__device__ __forceinline__ void key_group_scales(uint32_t kg, uint32_t (&w)[8]) {
  w[0] = row_bcast<0>(kg); w[1] = row_bcast<1>(kg); w[2] = row_bcast<2>(kg); w[3] = row_bcast<3>(kg);
  w[4] = row_bcast<4>(kg); w[5] = row_bcast<5>(kg); w[6] = row_bcast<6>(kg); w[7] = row_bcast<7>(kg);
}

// One 16-token page.  FULL: every token of the page is below t_end (no masking).
template <int KIND, bool METER, bool FULL, bool HALF, bool TB, bool BYP, bool VM, bool GS>
__device__ __forceinline__ void process_page(const DecodeArgs& a, const PageRegs<KIND>& cur, int t0,
                                             int t_end, int r, int g, const WaveConst& wc,
                                             uint8_t* my_dsh, WaveState& st) {
  // ---------------- QK^T and the bound ----------------
  const f4_t z4 = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
  f4_t s1 = z4;   // code and dither products
  uint32_t kgw[8];   // group scales: key scales of tokens 4g..4g+3
  if constexpr (KIND == WC_KIND_INT8_DITHER && GS) {
    const int64_t slot = (int64_t)cur.blk * kBlockTokens + r;
    const U4 r0 = dither_block(2 * g, slot, wc.layer_head, a.key0, a.key1);
    const U4 r1 = dither_block(2 * g + 1, slot, wc.layer_head, a.key0, a.key1);
    uint32_t u[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
    uint32_t kw[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) kw[i] = cur.kw[i];
    // chunk G: channels 32G + 8g .. 32G + 8g + 7 of token r
    transpose_chunks(u);
    transpose_chunks(kw);
    uint32_t dq[16];   // E of token r, chunk G = dq[4G .. 4G+3]
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      dq[2 * i] = ndith2(u[i], kSelLo);
      dq[2 * i + 1] = ndith2(u[i], kSelHi);
    }
    f4_t acc[4];
#pragma unroll
    for (int G = 0; G < 4; ++G) {
      const uint32_t x0 = kw[2 * G], x1 = kw[2 * G + 1];
      const h8_t ka = pack8(codes2(x0, kSelLo), codes2(x0, kSelHi), codes2(x1, kSelLo), codes2(x1, kSelHi));
      acc[G] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka, wc.qop[G], z4, 0, 0, 0);
      const h8_t kd = pack8(dq[4 * G], dq[4 * G + 1], dq[4 * G + 2], dq[4 * G + 3]);
      acc[G] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kd, wc.qop[G], acc[G], 0, 0, 0);
    }
    // dither of this page to LDS (row = token r; chunk G at channels 32G + 8g ..)
#pragma unroll
    for (int G = 0; G < 4; ++G)
      *reinterpret_cast<uint4*>(my_dsh + r * kRow + 64 * G + 16 * g) =
          make_uint4(dq[4 * G], dq[4 * G + 1], dq[4 * G + 2], dq[4 * G + 3]);
    // q . (code - xi) of group G is acc + (4 + 127.5/256) sum_G(q); weighted by s_{t,G}
    key_group_scales(cur.kg, kgw);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const h2_t s01 = as_h2(kgw[2 * e]), s23 = as_h2(kgw[2 * e + 1]);
      float v = (float)s01[0] * (acc[0][e] + wc.qoff[0]);
      v = fmaf((float)s01[1], acc[1][e] + wc.qoff[1], v);
      v = fmaf((float)s23[0], acc[2][e] + wc.qoff[2], v);
      v = fmaf((float)s23[1], acc[3][e] + wc.qoff[3], v);
      s1[e] = v;
    }
  } else if constexpr (KIND == WC_KIND_INT8_DITHER) {
    s1 = f4_t{wc.s1_init, wc.s1_init, wc.s1_init, wc.s1_init};
    const int64_t slot = (int64_t)cur.blk * kBlockTokens + r;
    const U4 r0 = dither_block(2 * g, slot, wc.layer_head, a.key0, a.key1);
    const U4 r1 = dither_block(2 * g + 1, slot, wc.layer_head, a.key0, a.key1);
    const uint32_t u[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
    uint32_t dq[16];   // E of token r, channels 32g + 2i, 32g + 2i + 1
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      dq[2 * i] = ndith2(u[i], kSelLo);
      dq[2 * i + 1] = ndith2(u[i], kSelHi);
    }
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const uint32_t x0 = cur.kw[2 * kt], x1 = cur.kw[2 * kt + 1];   // excess-128 codes
      const h8_t ka = pack8(codes2(x0, kSelLo), codes2(x0, kSelHi), codes2(x1, kSelLo), codes2(x1, kSelHi));
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka, wc.qop[kt], s1, 0, 0, 0);
      const h8_t kd = pack8(dq[4 * kt], dq[4 * kt + 1], dq[4 * kt + 2], dq[4 * kt + 3]);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(kd, wc.qop[kt], s1, 0, 0, 0);
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
        c[2 * j] = e4m3x2<false>(x);
        c[2 * j + 1] = e4m3x2<true>(x);
      }
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(pack8(c[0], c[1], c[2], c[3]), wc.qop[kt], s1, 0, 0, 0);
    }
  } else {
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const uint4 v = make_uint4(cur.kw[4 * kt], cur.kw[4 * kt + 1], cur.kw[4 * kt + 2], cur.kw[4 * kt + 3]);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(s8_t, v), wc.qbf[kt], s1, 0, 0, 0);
    }
  }
  f4_t cb = z4;
  if constexpr (METER && !TB) {
    const uint4 w = cur.wit;
    cb = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8_t, w),
                                                wc.qnop, cb, 0, 0, 0);
  }
  // bypassed pairs (Sec. 6.2): q . khat over their channels from the stored fp16
  // values (the query operand of the code products is zero there), and for Tier B
  // sum |q_c| |khat_c| for the fp16 rounding bound
  f4_t so = z4, go = z4;
  if constexpr (BYP) {
    const uint32_t o0 = wc.ov_lo ? cur.ov.x : 0u, o1 = wc.ov_lo ? cur.ov.y : 0u;
    const uint32_t o2 = wc.ov_hi ? cur.ov.z : 0u, o3 = wc.ov_hi ? cur.ov.w : 0u;
    so = __builtin_amdgcn_mfma_f32_16x16x32_f16(pack8(o0, o1, o2, o3),
                                                wc.qo, so, 0, 0, 0);
    if constexpr (TB) {
      constexpr uint32_t kAbs = 0x7FFF7FFFu;
      go = __builtin_amdgcn_mfma_f32_16x16x32_f16(pack8(o0 & kAbs, o1 & kAbs, o2 & kAbs, o3 & kAbs),
                                                  wc.qa, go, 0, 0, 0);
    }
  }

  // ---------------- online softmax and meter numerator ----------------
  // Lane (r, g) holds head r, tokens t0 + 4g + e.  HALF (at most 8 heads per KV
  // head): the lanes of heads 8..15 are padding, so tokens 4g+2, 4g+3 of head r
  // move to lane r + 8 (one DPP row shift per value) and every lane does the
  // softmax and meter work of two tokens.  Logits are in log2 units.
  constexpr int NT = HALF ? 2 : 4;
  const bool upper = HALF && r >= 8;
  const int tok0 = 4 * g + (upper ? 2 : 0);            // first token of this lane
  float scv[4], cbv[4], sov[4], gov[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    scv[e] = s1[e];   // INT8: q . (code - xi)
    cbv[e] = cb[e];
    sov[e] = so[e];
    gov[e] = go[e];
  }
  uint32_t ksw0 = cur.ks.x, ksw1 = cur.ks.y, vsw0 = cur.vs.x, vsw1 = cur.vs.y;
  if constexpr (HALF) {
    scv[0] = dpp_from_lower8(scv[0], scv[2]);
    scv[1] = dpp_from_lower8(scv[1], scv[3]);
    if constexpr (METER && !TB) {
      cbv[0] = dpp_from_lower8(cbv[0], cbv[2]);
      cbv[1] = dpp_from_lower8(cbv[1], cbv[3]);
    }
    if constexpr (BYP) {
      sov[0] = dpp_from_lower8(sov[0], sov[2]);
      sov[1] = dpp_from_lower8(sov[1], sov[3]);
      if constexpr (TB) {
        gov[0] = dpp_from_lower8(gov[0], gov[2]);
        gov[1] = dpp_from_lower8(gov[1], gov[3]);
      }
    }
    if constexpr (KIND == WC_KIND_INT8_DITHER) {
      ksw0 = upper ? cur.ks.y : cur.ks.x;
      vsw0 = upper ? cur.vs.y : cur.vs.x;
    }
  }
  const h2_t ksh[2] = {as_h2(ksw0), as_h2(ksw1)};
  const h2_t vsh[2] = {as_h2(vsw0), as_h2(vsw1)};
  // value side: this lane's tokens' stored residual and value norms
  const h2_t vrh[2] = {as_h2(HALF && upper ? cur.vr.y : cur.vr.x), as_h2(cur.vr.y)};
  const h2_t vnh[2] = {as_h2(HALF && upper ? cur.vn.y : cur.vn.x), as_h2(cur.vn.y)};
  if constexpr (TB && GS) {
    // Tier B over group steps (Sec. 4.2 with the group scales): in log2 units
    // u_t = sqrt(sum_G s_{t,G}^2 ta2_G) + sum_G s_{t,G} tb1_G for head r, tokens
    // 4g..4g+3 (HALF: tokens 4g+2, 4g+3 then move to lane r + 8, like the logits)
    float rad[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const h2_t a01 = as_h2(kgw[2 * e]), a23 = as_h2(kgw[2 * e + 1]);
      const float s0 = (float)a01[0], s1g = (float)a01[1], s2 = (float)a23[0], s3 = (float)a23[1];
      float v2 = s0 * s0 * wc.ta2[0];
      v2 = fmaf(s1g * s1g, wc.ta2[1], v2);
      v2 = fmaf(s2 * s2, wc.ta2[2], v2);
      v2 = fmaf(s3 * s3, wc.ta2[3], v2);
      float lin = s0 * wc.tb1[0];
      lin = fmaf(s1g, wc.tb1[1], lin);
      lin = fmaf(s2, wc.tb1[2], lin);
      lin = fmaf(s3, wc.tb1[3], lin);
      rad[e] = __builtin_amdgcn_sqrtf(v2) + lin;
    }
    if constexpr (HALF) {
      rad[0] = dpp_from_lower8(rad[0], rad[2]);
      rad[1] = dpp_from_lower8(rad[1], rad[3]);
    }
#pragma unroll
    for (int e = 0; e < NT; ++e) {
      const float extra = BYP ? fmaf(gov[e], wc.gmul, wc.gc) : 0.0f;
      cbv[e] = rad[e] + extra;
    }
  } else if constexpr (TB) {
    // Tier B (Sec. 4.2): the radius u_t = (alpha_h + beta_h) s_t from the stored
    // key scale of each of this lane's tokens, in log2 units
#pragma unroll
    for (int e = 0; e < NT; ++e) {
      const float extra = BYP ? fmaf(gov[e], wc.gmul, wc.gc) : 0.0f;
      cbv[e] = fmaf((float)ksh[e >> 1][e & 1], wc.ab2, extra);
    }
  }
  bool valid[NT];
  float lg[NT];
  float loc = -INFINITY;
#pragma unroll
  for (int e = 0; e < NT; ++e) {
    valid[e] = FULL || t0 + tok0 + e < t_end;
    float sc = scv[e];
    if constexpr (KIND == WC_KIND_INT8_DITHER && GS) {
      sc = (BYP ? sc + sov[e] : sc) * wc.lmul;   // (the group scales are in scv already)
    } else if constexpr (KIND == WC_KIND_INT8_DITHER) {
      // (fma with a +0 addend keeps the fp16 operand inside one mixed-precision fma)
      sc = fmaf((float)ksh[e >> 1][e & 1], sc, BYP ? sov[e] : 0.0f) * wc.lmul;
    } else {
      sc = sc * wc.lmul;
    }
    lg[e] = valid[e] ? sc : -INFINITY;
    loc = fmaxf(loc, lg[e]);
  }
  if (__ballot(loc > st.m + kSlack2) != 0) {
    float full = HALF ? xor_max<8>(loc) : loc;     // lanes r and r + 8 share head r's max
    full = xor_max<32>(xor_max<16>(full));
    const float m_new = fmaxf(st.m, full);
    const float alpha = exp2_fast(st.m - m_new);
    st.m = m_new;
    st.l *= alpha;
    st.n *= alpha;
    st.nb *= alpha;
    st.wsum *= alpha;
    st.ws4 *= alpha;
    if constexpr (VM) st.ev *= alpha;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      st.o1[j] *= alpha;
    }
  }
  // (group scales: those of the lane's PV rows, group r/4)
  uint32_t vsx = cur.vs.x, vsy = cur.vs.y;
  if constexpr (KIND == WC_KIND_INT8_DITHER) {
    // a value scale above 2^ve raises ve to cover the page (rare: value scales of a
    // sequence vary little); the accumulated weights are rescaled by 2^(ve - ve')
    // (tokens past the end may hold any stale scale: left out)
    if constexpr (!FULL) {
      const int tq = t_end - (t0 + 4 * g);   // valid tokens among 4g .. 4g+3
      vsx &= tq >= 2 ? 0xFFFFFFFFu : (tq == 1 ? 0x0000FFFFu : 0u);
      vsy &= tq >= 4 ? 0xFFFFFFFFu : (tq == 3 ? 0x0000FFFFu : 0u);
    }
    // (scales are non-negative fp16: their bit patterns order like their values;
    // 2^ve has the bits (15 + ve) << 10, +inf for ve = 16, above every fp16 scale)
    typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
    const u16x2 pm2 = __builtin_elementwise_max(__builtin_bit_cast(u16x2, vsx), __builtin_bit_cast(u16x2, vsy));
    const uint32_t pbits = max((uint32_t)pm2[0], (uint32_t)pm2[1]);
    if (__ballot(pbits > (uint32_t)(15 + st.ve) << 10) != 0) {
      const float pmax = (float)__builtin_bit_cast(_Float16, (uint16_t)pbits);
      const float wmax = xor_max<32>(xor_max<16>(xor_max<8>(xor_max<4>(xor_max<2>(xor_max<1>(pmax))))));
      int e2;
      (void)frexpf(wmax, &e2);                    // wmax < 2^e2 (e2 <= 16 for fp16 scales)
      const int ve_new = __builtin_amdgcn_readfirstlane(max(st.ve, e2));
      const float alpha = __builtin_bit_cast(float, (uint32_t)(127 + st.ve - ve_new) << 23);   // 2^(ve - ve')
      st.ve = ve_new;
      st.wsum *= alpha;
      st.ws4 *= alpha;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        st.o1[j] *= alpha;
      }
    }
  }
  // 2^-ve as fp16 bits in both halves (normal up to ve = 14, subnormal above; exact)
  const uint32_t vmul_h = st.ve <= 14 ? (uint32_t)(15 - st.ve) << 10 : 1u << (24 - st.ve);
  const h2_t vmul = as_h2(vmul_h * 0x00010001u);
  const float mo = st.m - kWExp;
  _Float16 wh[NT];
#pragma unroll
  for (int e = 0; e < NT; ++e) {
    const float x = lg[e] - mo;
    const float p = exp2_fast(x);                    // 2^8 softmax weight; 0 for masked tokens
    st.l += p;
    if constexpr (VM) {
      // (a masked token's stored bytes may be anything: leave them out)
      st.ev += valid[e] ? p * (float)vrh[e >> 1][e & 1] : 0.0f;
      st.vmax = fmaxf(st.vmax, valid[e] ? (float)vnh[e >> 1][e & 1] : 0.0f);
    }
    if constexpr (METER) {
      // p (e^c - 1): Taylor series for c <= 1/2; above, 2^(x + c) - p, which
      // also counts a token whose weight underflows with its bound
      const float c = cbv[e];
      const float small = p * exp2m1_small(__builtin_amdgcn_fmed3f(c, 0.0f, kTaylorMax));
      const float big = exp2_fast(x + c) - p;
      const float term = valid[e] ? (c > kTaylorMax ? big : small) : 0.0f;
      st.n += term;
      st.nb += term;
    }
    float w = p;   // (group scales: the value scale is in the value operand)
    if constexpr (KIND == WC_KIND_INT8_DITHER && !GS) w = fmaf((float)(vsh[e >> 1] * vmul)[e & 1], p, 0.0f);
    wh[e] = valid[e] ? (_Float16)w : (_Float16)0.0f;
  }
  const h2_t one = h2_t{(_Float16)1.0f, (_Float16)1.0f};
  h4_t wop;
  if constexpr (HALF) {
    // the PV operand of head r takes tokens 4g+2, 4g+3 back from lane r + 8
    const uint32_t w01 = as_u32(h2_t{wh[0], wh[1]});
    wop = pack4(w01, dpp_from_upper8(w01));
    if constexpr (KIND == WC_KIND_INT8_DITHER && !GS)
      st.wsum = __builtin_amdgcn_fdot2(as_h2(w01), one, st.wsum, false);
  } else {
    const h2_t w01 = h2_t{wh[0], wh[1]}, w23 = h2_t{wh[NT - 2], wh[NT - 1]};
    wop = h4_t{wh[0], wh[1], wh[NT - 2], wh[NT - 1]};
    if constexpr (KIND == WC_KIND_INT8_DITHER && !GS)
      st.wsum = __builtin_amdgcn_fdot2(w23, one, __builtin_amdgcn_fdot2(w01, one, st.wsum, false), false);
  }
  // validity of tokens 4g .. 4g+3 (the k index of the PV operands)
  bool vtok[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) vtok[e] = FULL || t0 + 4 * g + e < t_end;

  // ---------------- P V ----------------
  if constexpr (KIND == WC_KIND_INT8_DITHER && GS) {
    // value operand s_{t,r/4} 2^-ve (code + E) of channel 8r+jt, tokens 4g..4g+3
    // (scales of tokens past the end are zero: vsx, vsy above)
    const h2_t s01 = as_h2(vsx) * vmul, s23 = as_h2(vsy) * vmul;
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
      const uint32_t x = cur.vw[jt];     // codes (excess-128) of channel 8r+jt, tokens 4g..4g+3
      const uint32_t sel = (jt & 1) ? kSelH1 : kSelH0;
      const h2_t d01 = as_h2(perm(r1[jt >> 1], r0[jt >> 1], sel));
      const h2_t d23 = as_h2(perm(r3[jt >> 1], r2[jt >> 1], sel));
      const h2_t a01 = __builtin_elementwise_fma(d01, s01, as_h2(codes2(x, kSelLo)) * s01);
      const h2_t a23 = __builtin_elementwise_fma(d23, s23, as_h2(codes2(x, kSelHi)) * s23);
      st.o1[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(as_u32(a01), as_u32(a23)), wop, st.o1[jt], 0, 0, 0);
    }
    // sum_t w_t s_{t,G} 2^-ve: rows 4G..4G+3 of lane group G's scales (row r of this
    // lane is group r/4), so lane (r, g) of the result holds group g, head r
    st.ws4 = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(as_u32(s01), as_u32(s23)), wop, st.ws4, 0, 0, 0);
    __builtin_amdgcn_s_waitcnt(0xc07f);   // LDS reads done before the next page overwrites
    __builtin_amdgcn_wave_barrier();
  } else if constexpr (KIND == WC_KIND_INT8_DITHER) {
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
      const uint32_t x = cur.vw[jt];     // codes (excess-128) of channel 8r+jt, tokens 4g..4g+3
      st.o1[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(ucodes2(x, kSelLo), ucodes2(x, kSelHi)), wop,
                                                        st.o1[jt], 0, 0, 0);
    }
    // (the dither products go to the same accumulators after all eight code products)
#pragma unroll
    for (int jt = 0; jt < 8; ++jt) {
      const uint32_t sel = (jt & 1) ? kSelH1 : kSelH0;
      const uint32_t d01 = perm(r1[jt >> 1], r0[jt >> 1], sel);
      const uint32_t d23 = perm(r3[jt >> 1], r2[jt >> 1], sel);
      st.o1[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(d01, d23), wop, st.o1[jt], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);   // LDS reads done before the next page overwrites
    __builtin_amdgcn_wave_barrier();
  } else if constexpr (KIND == WC_KIND_FP8_RAW) {
#pragma unroll
    for (int jt = 0; jt < 8; ++jt) {
      const uint32_t x = cur.vw[jt];
      uint32_t lo = e4m3x2<false>(x);
      uint32_t hi = e4m3x2<true>(x);
      if constexpr (!FULL) {
        // tokens past the end may hold any byte pattern (the 0x7F NaN code): zero them
        if (!vtok[0]) lo &= 0xFFFF0000u;
        if (!vtok[1]) lo &= 0x0000FFFFu;
        if (!vtok[2]) hi &= 0xFFFF0000u;
        if (!vtok[3]) hi &= 0x0000FFFFu;
      }
      st.o1[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(lo, hi), wop, st.o1[jt], 0, 0, 0);
    }
  } else {
    // bf16 values enter PV as fp16 times 2^-ve: a value above 2^(15 + ve) raises ve
    // (rare), with the output accumulators rescaled by the exact power of two
    // (tokens past the end may hold any bytes: they are zeroed first)
    uint32_t vw[16];
    {
      const int tq = FULL ? 4 : t_end - (t0 + 4 * g);   // valid tokens among 4g .. 4g+3
      const uint32_t m01 = tq >= 2 ? 0xFFFFFFFFu : (tq == 1 ? 0x0000FFFFu : 0u);
      const uint32_t m23 = tq >= 4 ? 0xFFFFFFFFu : (tq == 3 ? 0x0000FFFFu : 0u);
#pragma unroll
      for (int i = 0; i < 16; ++i) vw[i] = cur.vw[i] & ((i & 1) ? m23 : m01);
    }
    typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
    u16x2 am = u16x2{0, 0};
#pragma unroll
    for (int i = 0; i < 16; ++i)
      am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, vw[i] & 0x7FFF7FFFu));
    const float pmax = __builtin_bit_cast(float, (uint32_t)max(am[0], am[1]) << 16);
    if (__ballot(pmax > __builtin_bit_cast(float, (uint32_t)(142 + st.ve) << 23)) != 0) {
      const float wmax = xor_max<32>(xor_max<16>(xor_max<8>(xor_max<4>(xor_max<2>(xor_max<1>(pmax))))));
      int e2;
      (void)frexpf(wmax, &e2);                    // wmax < 2^e2
      const int ve_new = __builtin_amdgcn_readfirstlane(max(st.ve, e2 - 15));
      const float alpha = __builtin_bit_cast(float, (uint32_t)(127 + st.ve - ve_new) << 23);
      st.ve = ve_new;
      st.wsum *= alpha;   // (the INT8 weights of a mixed cache carry 2^-ve too)
      st.ws4 *= alpha;
#pragma unroll
      for (int j = 0; j < 8; ++j) st.o1[j] *= alpha;
    }
    const float vsc = __builtin_bit_cast(float, (uint32_t)(127 - st.ve) << 23);   // 2^-ve
#pragma unroll
    for (int jt = 0; jt < 8; ++jt) {
      // bf16 values of channel 8r+jt, tokens 4g..4g+3: 8 bytes at offset 8*jt
      uint32_t lo, hi;
      if (st.ve == 0) {
        lo = bf16pair_to_f16(vw[2 * jt]);
        hi = bf16pair_to_f16(vw[2 * jt + 1]);
      } else {
        lo = bf16pair_to_f16_scaled(vw[2 * jt], vsc);
        hi = bf16pair_to_f16_scaled(vw[2 * jt + 1], vsc);
      }
      st.o1[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(pack4(lo, hi), wop, st.o1[jt], 0, 0, 0);
    }
  }
}

// Block segments (block repair's shares, Sec. 6.3): the wave's pages split at the
// 256-token repair blocks.  A segment's numerator (summed over the lanes of each
// head) goes with its frame, first page and length into the next of the wave's
// share slots; every slot the wave owns is written (unused ones with 0 pages).
struct Segment {
  int first;   // first page of the open segment
  int slot;    // next share slot of this wave
};
template <bool HALF>
__device__ __forceinline__ void flush_segment(const DecodeArgs& a, WaveState& st, Segment& sg, int last_page,
                                              float4* my_slots, int r, int g) {
  float t = st.nb;
  if constexpr (HALF) t = bfly_add<8>(t);   // lanes r and r + 8 hold tokens of head r
  t = bfly_add<16>(t);
  t = bfly_add<32>(t);
  if (g == 0 && r < a.group && sg.slot < a.share_slots / kWaves)
    my_slots[sg.slot] = make_float4(t, (st.m - kWExp) * kLn2, __builtin_bit_cast(float, sg.first),
                                    __builtin_bit_cast(float, last_page - sg.first));
  ++sg.slot;
  sg.first = last_page;
  st.nb = 0.0f;
}

// The new token of sequence b, KV head kv (the step's token of that sequence, by
// the workgroup that reads it): lanes 0 .. kD/16 - 1 of wave 0 quantize and store
// it as the write kernel does (write_dev.h, witness included); the barrier after
// the stores comes before any wave of the workgroup requests a page.
template <int KIND>
__device__ __forceinline__ void step_write(const DecodeArgs& a, int b, int kv, int wave, int lane) {
  constexpr int LPT = kD / 16;
  if (wave == 0 && lane < LPT) {
    (void)write_token_head<kD, KIND, uint16_t, false>(a.sw, b, kv, true, lane);   // (no bypassed pairs)
    // the stores are complete (acknowledged) before the barrier, not only ordered
    // by it: no wave can then read the page before the new token is in it
    __builtin_amdgcn_s_waitcnt(0);
  }
  __syncthreads();
}

// REP: the cache carries repair marks (a.repaired set; a quantized kind), a
// separate instantiation so that caches without marks run the loop unchanged.
// The workgroup's LDS.  Per wave, one region that holds in turn its query band
// norms (prologue), a page's dither rows (INT8 caches, page loop) and its output
// rows for the in-workgroup merge (epilogue): only that wave touches it, in that
// order.  Then the waves' scalars for the merge, the queries (bf16 rows of 256
// bytes, +16 pad) and the certified step's gate flag.
struct DecodeWaveLds {
  union {
    struct {
      __attribute__((aligned(16))) uint8_t dsh[16 * kRow];
      float qn[16][16];
    } loop;
    __attribute__((aligned(16))) float acc[16][kD];
  };
};
template <int KIND>
struct DecodeLds {
  DecodeWaveLds w[kWaves];
  float ml_s[kWaves][16][6];
  uint4 q_lds[16][17];
  int gate_flag_s;
};

// One workgroup of the decode: linear workgroup index lin (decode_position_at).
template <int KIND, bool METER, bool HALF, bool TB, bool BYP, bool VM, bool REP, bool GS>
__device__ __forceinline__ void decode_block(const DecodeArgs& a, uint32_t lin, DecodeLds<KIND>& lds) {
  auto& ml_s = lds.ml_s;
  auto& q_lds = lds.q_lds;
  int& gate_flag_s = lds.gate_flag_s;
  // a decode step's new token is written by the plain Tier A variants (the ones the
  // step call fuses; the others keep their registers) and, in the speculative
  // certified step, into the exact cache by the exact fallback
  constexpr bool kStep = (METER && !TB && !BYP && !VM && !GS) || (KIND == WC_KIND_BF16 && !REP);

  // the wave index is uniform: page addresses then live in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const DecodePos pos = decode_position_at(lin, a.batch, a.n_kv, a.n_splits);
  const int unit = __builtin_amdgcn_readfirstlane(pos.unit), split = __builtin_amdgcn_readfirstlane(pos.split);
  const int b = unit / a.n_kv, kv = unit % a.n_kv;
  gate_clear(a, unit, split);
  const int G = a.group;
  const int B = a.n_bands;
  const int wg_begin = split * a.split_tokens;
  const int32_t* trow = a.table + (int64_t)b * a.max_blocks;
  // The workgroup's queries (G x 256 bytes) are requested first, once per
  // workgroup (thread = 16 bytes of one head), and shared through LDS below: every
  // workgroup of a (sequence, KV head) reads the same bytes, and loading them per
  // wave made one L2 channel a hot spot at kernel start that held back the first
  // page requests.
  uint4 qv = make_uint4(0, 0, 0, 0);
  if (threadIdx.x < a.group * 16)
    qv = reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(a.q) +
                                        ((int64_t)b * a.n_q + (int64_t)kv * a.group) * kD)[threadIdx.x];
  const int L = a.seq_lens[b];

  // Requests that need no sequence length go out with it: this wave's block
  // numbers as if its split were full (it is, except for a sequence's last
  // split) and the queries, so that their latency overlaps that of the length.
  const int ppw_full = a.split_tokens / (kBlockTokens * kWaves);
  const int pg_spec = wg_begin / kBlockTokens + wave * ppw_full;
  const int nc_spec = max(0, min(min(64, ppw_full), a.max_blocks - pg_spec));
  const int tv_spec = lane < nc_spec ? trow[pg_spec + lane] : 0;
  const bool hv = r < G;

  // certified step: the exact fallback decides its unit's gate from the metered
  // records first (split 0 always, for the masks; splits past the end skip it)
  bool ungated = false;
  if (KIND == WC_KIND_BF16 && a.gate_part != nullptr && (split == 0 || wg_begin < L))
    ungated = !unit_gate(a, b, kv, split, wave, lane, &gate_flag_s);
  // whole workgroup: a KV head not routed here, or a split past the sequence end
  // (evaluated together, so that the length load is not held back behind the mask)
  const bool unrouted = ungated || (a.mask_kv != nullptr && a.mask_kv[unit] == 0);
  if (unrouted | (split >= a.n_splits) | (wg_begin >= L)) return;
  if constexpr (kStep) {
    if (a.step_write && split == (L - 1) / a.split_tokens) step_write<KIND>(a, b, kv, wave, lane);
  }
  const int wg_end = min(min(L, wg_begin + a.split_tokens), a.max_blocks * kBlockTokens);
  // this wave's share: a quarter of the workgroup's pages (rounded up; a full
  // split gives split_tokens / 4 tokens); a sequence's last split is divided the
  // same way, so that all four waves share a short sequence
  const int ppw = ((wg_end - wg_begin + kBlockTokens - 1) / kBlockTokens + kWaves - 1) / kWaves;
  const int t_begin = min(wg_begin + wave * ppw * kBlockTokens, wg_end);
  const int t_end = min(wg_end, t_begin + ppw * kBlockTokens);

  // Pages stream through a ring of three register buffers, so two pages are in
  // flight while one is computed.  Block numbers come 64 pages at a time from one
  // vector load of the table and are read out with readlane (wave-uniform).  The
  // first two pages are requested before the queries are prepared.
  // full pages go through the ring; a last page that reaches past t_end is done after it
  const int np = t_end > t_begin ? (t_end - t_begin) / kBlockTokens : 0;
  const int pg0 = t_begin / kBlockTokens;
  // (a lane without bands -- 8 (g % 2) >= B -- reads past the page's witness
  // bytes, which the buffer range check turns into zeros)
  const int wit_off = 8 * (g & 1) < B ? 2 * (r * B + 8 * (g & 1)) : 1 << 30;
  PageRegs<KIND> p0, p1, p2;
  int nc = 0, tv = 0;
  // persistent repair: the chunk's repair marks (lane j: page j), requested with
  // the first two pages and read before the third is requested; a marked page is
  // not read here (its loads get empty resources) and is served from the exact
  // store after the loop
  constexpr bool has_rep = REP && KIND != WC_KIND_BF16;   // (the exact cache has no marks)
  int fl = 0;
  uint64_t emask = 0;
  auto blk_at = [&](int j) { return __builtin_amdgcn_readlane(tv, min(j, nc - 1)); };
  auto marked = [&](int j) { return j < 64 && ((emask >> j) & 1u) != 0; };
  // (scheduling barriers keep each page's loads together, so that waiting for
  // one page never waits for a later one)
  auto start_chunk = [&](int c0) {
    nc = min(64, np - c0);
    if (c0 == 0 && pg0 == pg_spec && nc <= nc_spec) tv = tv_spec;   // the early request holds them
    else tv = lane < nc ? trow[pg0 + c0 + lane] : 0;
    if (has_rep)
      fl = lane < nc && (int64_t)(uint32_t)tv < a.num_blocks ? a.repaired[(int64_t)tv * a.n_kv + kv] : 0;
    load_page<KIND, METER, TB, BYP, VM, GS>(a, blk_at(0), true, kv, r, g, wit_off, p0);
    __builtin_amdgcn_sched_barrier(0);
    load_page<KIND, METER, TB, BYP, VM, GS>(a, blk_at(1), 1 < nc, kv, r, g, wit_off, p1);
    __builtin_amdgcn_sched_barrier(0);
  };
  if (np > 0) start_chunk(0);

  // ---- queries of head r, channels 32g .. 32g+31, from LDS ----
  // Padding heads (r >= G) get zeros: their scores and weights land in result
  // columns that are never written out.
  uint32_t qraw[16];
  {
    if (threadIdx.x < G * 16) q_lds[threadIdx.x >> 4][threadIdx.x & 15] = qv;
    // a barrier fenced for LDS only: a full workgroup fence would also wait for
    // the page loads just issued
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint4 v = hv ? q_lds[r][4 * g + i] : make_uint4(0, 0, 0, 0);
      qraw[4 * i] = v.x; qraw[4 * i + 1] = v.y; qraw[4 * i + 2] = v.z; qraw[4 * i + 3] = v.w;
    }
  }

  WaveConst wc;
  // Bypassed pairs (Sec. 6.2 fixed-channel bypass): the query channels of this
  // lane that are bypassed leave the code products (qk); their keys come from the
  // stored fp16 values through wc.qo.  Tier A's band norms keep the whole query.
  uint32_t qk[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) qk[i] = qraw[i];
  wc.gmul = wc.gc = 0.0f;
  wc.ov_lo = wc.ov_hi = false;
  if constexpr (BYP) {
    const int m = a.n_pairs;
    const int32_t* pl = a.pairs + (int64_t)kv * m;
    uint32_t mw = 0;   // bypassed channels among 32g .. 32g+31
    for (int i = 0; i < m; ++i) {
      const int j = pl[i];
#pragma unroll
      for (int sec = 0; sec < 2; ++sec) {
        const int c = pair_channel(j, sec, kD, a.interleaved) - 32 * g;
        if ((unsigned)c < 32u) mw |= 1u << c;
      }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i)
      qk[i] &= (((mw >> (2 * i)) & 1u) ? 0u : 0xFFFFu) | (((mw >> (2 * i + 1)) & 1u) ? 0u : 0xFFFF0000u);
    const uint16_t* qrow = reinterpret_cast<const uint16_t*>(a.q) +
                           ((int64_t)b * a.n_q + (int64_t)kv * G + (hv ? r : 0)) * kD;
    uint32_t qw[4], qaw[4];
    float asum = 0.0f;
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      uint32_t w = 0;
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int pos = 8 * g + 2 * e2 + h2;   // stored value pos: pair pos/2, channel pos%2
        if (pos < 2 * m) {
          const _Float16 hx = (_Float16)bf16_to_f32(qrow[pair_channel(pl[pos >> 1], pos & 1, kD, a.interleaved)]);
          w |= (uint32_t)f16_bits(hx) << (16 * h2);
          asum += fabsf((float)hx);
        }
      }
      qw[e2] = w;
      qaw[e2] = w & 0x7FFF7FFFu;
    }
    wc.qo = pack8(qw[0], qw[1], qw[2], qw[3]);
    wc.qa = pack8(qaw[0], qaw[1], qaw[2], qaw[3]);
    wc.ov_lo = 8 * g < 2 * m;
    wc.ov_hi = 8 * g + 4 < 2 * m;
    if constexpr (TB) {
      asum = bfly_add<16>(asum);
      asum = bfly_add<32>(asum);
      wc.gmul = a.sm_scale * 0x1p-11f * kLog2e;
      wc.gc = a.sm_scale * 0x1p-25f * kLog2e * asum;
      if constexpr (HALF) wc.gc = dpp_from_lower8(wc.gc, wc.gc);
    }
  }
  wc.layer_head = ((uint32_t)a.layer << 16) | (uint32_t)kv;
  wc.lmul = a.sm_scale * kLog2e;
  // B operands of QK: the kt-th MFMA uses channels 32g + 8kt .. 32g + 8kt + 7.
  float qsum = 0.0f;   // sum of the fp16 queries of head r over all channels
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    if constexpr (KIND == WC_KIND_BF16) {
      wc.qbf[kt] = __builtin_bit_cast(s8_t, make_uint4(qraw[4 * kt], qraw[4 * kt + 1], qraw[4 * kt + 2],
                                                       qraw[4 * kt + 3]));
    } else {
      uint32_t w[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        w[j] = bf16pair_to_f16(qk[4 * kt + j]);
        qsum = __builtin_amdgcn_fdot2(as_h2(w[j]), h2_t{(_Float16)1.0f, (_Float16)1.0f}, qsum, false);
      }
      wc.qop[kt] = pack8(w[0], w[1], w[2], w[3]);
    }
  }
  qsum = bfly_add<16>(qsum);
  qsum = bfly_add<32>(qsum);
  wc.s1_init = kQOff * qsum;
#pragma unroll
  for (int G = 0; G < 4; ++G) wc.qoff[G] = wc.ta2[G] = wc.tb1[G] = 0.0f;
  if constexpr (GS) {
    // group-ordered B operands: chunk G = channels 32G + 8g .. 32G + 8g + 7 of head
    // r (bypassed channels zeroed: bit 8G + j of mg for channel 32G + 8g + j)
    uint32_t mg = 0;
    if constexpr (BYP) {
      const int32_t* pl = a.pairs + (int64_t)kv * a.n_pairs;
      for (int i = 0; i < a.n_pairs; ++i)
#pragma unroll
        for (int sec = 0; sec < 2; ++sec) {
          const int c = pair_channel(pl[i], sec, kD, a.interleaved);
          const int o = (c & 31) - 8 * g;
          if ((unsigned)o < 8u) mg |= 1u << (8 * (c >> 5) + o);
        }
    }
    float n2[4], l1[4];
#pragma unroll
    for (int G = 0; G < 4; ++G) {
      const uint4 v = hv ? q_lds[r][4 * G + g] : make_uint4(0, 0, 0, 0);
      uint32_t w[4] = {v.x, v.y, v.z, v.w};
      float qs = 0.0f;
      n2[G] = l1[G] = 0.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int bit = 8 * G + 2 * i;
        w[i] &= (((mg >> bit) & 1u) ? 0u : 0xFFFFu) | (((mg >> (bit + 1)) & 1u) ? 0u : 0xFFFF0000u);
        const uint32_t h = bf16pair_to_f16(w[i]);
        qs = __builtin_amdgcn_fdot2(as_h2(h), h2_t{(_Float16)1.0f, (_Float16)1.0f}, qs, false);
        if constexpr (TB) {
          const float x0 = bf16_to_f32((uint16_t)(w[i] & 0xFFFFu)), x1 = bf16_to_f32((uint16_t)(w[i] >> 16));
          n2[G] = fmaf(x1, x1, fmaf(x0, x0, n2[G]));
          l1[G] += fabsf(x0) + fabsf(x1);
        }
        w[i] = h;
      }
      wc.qop[G] = pack8(w[0], w[1], w[2], w[3]);
      qs = bfly_add<16>(qs);
      qs = bfly_add<32>(qs);
      wc.qoff[G] = kQOff * qs;
    }
    if constexpr (TB) {
      // u_t = sm (rt sqrt(sum_G s_G^2 ||q_G||^2) + sum_G s_G ||q_G||_1 / 256), in log2 units
      const float rt = sqrtf(2.0f * logf(2.0f * (float)L / a.tierb_delta) / 12.0f);
      const float c = a.sm_scale * kLog2e;
#pragma unroll
      for (int G = 0; G < 4; ++G) {
        float x = n2[G], y = l1[G];
        x = bfly_add<16>(x);
        x = bfly_add<32>(x);
        y = bfly_add<16>(y);
        y = bfly_add<32>(y);
        wc.ta2[G] = (c * rt) * (c * rt) * x;   // (head r: the radii are formed before the HALF shift)
        wc.tb1[G] = c * y * (1.0f / 256.0f);
      }
    }
  }
  // band norms ||q_b|| * sm_scale * log2(e) -> witness-MFMA B operand (hi parts
  // for g < 2, lo for g >= 2); the bound then comes out in log2 units
  wc.qnop = pack8(0, 0, 0, 0);
  wc.ab2 = 0.0f;
  if constexpr (TB && GS) {
    // (the group radius coefficients are set above)
  } else if constexpr (TB) {
    float sq = 0.0f, l1 = 0.0f;   // ||q||^2 and ||q||_1 of head r (channels not bypassed)
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const float x = bf16_to_f32((uint16_t)((qk[i >> 1] >> (16 * (i & 1))) & 0xFFFFu));
      sq = fmaf(x, x, sq);
      l1 += fabsf(x);
    }
    sq = bfly_add<16>(sq);
    sq = bfly_add<32>(sq);
    l1 = bfly_add<16>(l1);
    l1 = bfly_add<32>(l1);
    wc.ab2 = tierb_factor(sq, l1, L, a.tierb_delta, a.sm_scale) * kLog2e;
    // with two tokens per lane, lanes r + 8 hold tokens of head r
    if constexpr (HALF) wc.ab2 = dpp_from_lower8(wc.ab2, wc.ab2);
  } else if constexpr (METER) {
    // Squares of this lane's 32 channels summed in runs of 4.  The band of
    // channel 32g + i is base + i / S with S = 64 / B (rotate-half pairs (j, j + 64))
    // or 128 / B (adjacent pairs), so runs of 4 coarsen exactly into the lane's bands.
    float p4[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      float acc = 0.0f;
#pragma unroll
      for (int i = 4 * k; i < 4 * k + 4; ++i) {
        const float x = bf16_to_f32((uint16_t)((qraw[i >> 1] >> (16 * (i & 1))) & 0xFFFFu));
        acc = fmaf(x, x, acc);
      }
      p4[k] = acc;
    }
    const int S = (a.interleaved ? 2 * kD : kD) / (2 * B);   // 4, 8 or 16
    const int nl = 32 / S;                                     // bands touched by this lane
    const int base = 32 * (a.interleaved ? g : (g & 1)) / S;
    float pb[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      if (S == 4) pb[k] = p4[k];
      else if (S == 8) pb[k] = k < 4 ? p4[2 * k] + p4[2 * k + 1] : 0.0f;
      else pb[k] = k < 2 ? (p4[4 * k] + p4[4 * k + 1]) + (p4[4 * k + 2] + p4[4 * k + 3]) : 0.0f;
    }
    // rotate-half: lanes g and g ^ 2 hold the two halves of the same pairs
    if (!a.interleaved) {
#pragma unroll
      for (int k = 0; k < 8; ++k) pb[k] = bfly_add<32>(pb[k]);
    }
    if (a.interleaved || g < 2) {
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (k < nl) lds.w[wave].loop.qn[r][base + k] = pb[k];
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
    const float nmul = a.sm_scale * kLog2e;
    uint32_t hw[4];
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      _Float16 hv2[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int band = 8 * (g & 1) + 2 * e2 + j;
        const float x = band < B ? __builtin_amdgcn_sqrtf(lds.w[wave].loop.qn[r][band]) * nmul : 0.0f;
        const _Float16 hi = (_Float16)x;
        hv2[j] = (g < 2) ? hi : (_Float16)(x - (float)hi);
      }
      hw[e2] = as_u32(h2_t{hv2[0], hv2[1]});
    }
    wc.qnop = pack8(hw[0], hw[1], hw[2], hw[3]);
  }

  WaveState st;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    st.o1[j] = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
  }
  st.m = -INFINITY;
  st.l = st.n = st.wsum = st.nb = 0.0f;
  st.ws4 = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
  // group scales: the value scales enter the fp16 value operand as s 2^-ve <= 1;
  // starting at 2^-14 keeps every fp16 scale's operand a normal number
  st.ve = GS ? -14 : 0;
  st.ev = st.vmax = 0.0f;
  uint8_t* my_dsh = lds.w[wave].loop.dsh;

  // Two workgroups share each SIMD, and instruction issue favours the older
  // wave, so the later workgroup would finish long after the earlier one, alone
  // on its SIMD.  A wave's issue priority therefore falls with its progress: the
  // wave that is behind gets the issue slots, and the pair finishes together.
  auto set_priority = [&](int done) {
    const int left4 = 4 * (np - done);
    if (left4 > 3 * np) __builtin_amdgcn_s_setprio(3);
    else if (left4 > 2 * np) __builtin_amdgcn_s_setprio(2);
    else if (left4 > np) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(0);
  };
  // block segments: a page that starts a 256-token repair block closes the open
  // segment (wave-uniform test)
  const bool rec_shares = METER && a.shares != nullptr;
  Segment sg{t_begin / kBlockTokens, 0};
  float4* my_slots = rec_shares ? a.shares + (((int64_t)b * a.n_q + (int64_t)kv * G + (hv ? r : 0)) * a.n_splits +
                                              split) * a.share_slots + wave * (a.share_slots / kWaves)
                                : nullptr;
  auto seg_check = [&](int t0) {
    if (rec_shares && (t0 & (kRepairBlockTokens - 1)) == 0 && t0 / kBlockTokens > sg.first)
      flush_segment<HALF>(a, st, sg, t0 / kBlockTokens, my_slots, r, g);
  };
  bool any_marked = false;
  for (int c0 = 0; c0 < np;) {
    const int tb = t_begin + c0 * kBlockTokens;
    emask = has_rep ? (uint64_t)__ballot(fl != 0) : 0;
    any_marked |= emask != 0;
    // No early exit from this loop: a break lets the compiler's load counting
    // assume the ring order may differ on the back edge and wait for every page.
    for (int j = 0; j < nc; j += 3) {
      set_priority(c0 + j);
      load_page<KIND, METER, TB, BYP, VM, GS>(a, blk_at(j + 2), j + 2 < nc && !marked(j + 2), kv, r, g, wit_off, p2);
      __builtin_amdgcn_sched_barrier(0);
      seg_check(tb + j * kBlockTokens);
      if (!marked(j))
        process_page<KIND, METER, true, HALF, TB, BYP, VM, GS>(a, p0, tb + j * kBlockTokens, t_end, r, g, wc, my_dsh, st);
      load_page<KIND, METER, TB, BYP, VM, GS>(a, blk_at(j + 3), j + 3 < nc && !marked(j + 3), kv, r, g, wit_off, p0);
      __builtin_amdgcn_sched_barrier(0);
      if (j + 1 < nc) {
        seg_check(tb + (j + 1) * kBlockTokens);
        if (!marked(j + 1))
          process_page<KIND, METER, true, HALF, TB, BYP, VM, GS>(a, p1, tb + (j + 1) * kBlockTokens, t_end, r, g, wc, my_dsh, st);
      }
      load_page<KIND, METER, TB, BYP, VM, GS>(a, blk_at(j + 4), j + 4 < nc && !marked(j + 4), kv, r, g, wit_off, p1);
      __builtin_amdgcn_sched_barrier(0);
      if (j + 2 < nc) {
        seg_check(tb + (j + 2) * kBlockTokens);
        if (!marked(j + 2))
          process_page<KIND, METER, true, HALF, TB, BYP, VM, GS>(a, p2, tb + (j + 2) * kBlockTokens, t_end, r, g, wc, my_dsh, st);
      }
    }
    c0 += 64;
    if (c0 < np) start_chunk(c0);
  }
  __builtin_amdgcn_s_setprio(0);
  const int t_last = t_begin + np * kBlockTokens;
  if (t_last < t_end) {   // a partial last page: tokens from t_end on are masked
    const int blk = trow[t_last / kBlockTokens];
    const bool last_marked =
        has_rep && (int64_t)(uint32_t)blk < a.num_blocks && a.repaired[(int64_t)blk * a.n_kv + kv] != 0;
    any_marked |= last_marked;
    seg_check(t_last);
    if (!last_marked) {
      load_page<KIND, METER, TB, BYP, VM, GS>(a, blk, true, kv, r, g, wit_off, p0);
      process_page<KIND, METER, false, HALF, TB, BYP, VM, GS>(a, p0, t_last, t_end, r, g, wc, my_dsh, st);
    }
  }
  if (rec_shares) {
    // the last segment, then the wave's unused slots (0 pages)
    if (t_end > t_begin) flush_segment<HALF>(a, st, sg, (t_end + kBlockTokens - 1) / kBlockTokens, my_slots, r, g);
    for (int sl = sg.slot; sl < a.share_slots / kWaves; ++sl)
      if (g == 0 && r < G) my_slots[sl] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  }

  // ---- pages served from the exact store (persistent repair), two in flight:
  // exact logits against the whole bf16 query, exact values, bound 0 ----
  if (has_rep && any_marked) {
    WaveConst wx = wc;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint4 v = hv ? q_lds[r][4 * g + i] : make_uint4(0, 0, 0, 0);
      wx.qbf[i] = __builtin_bit_cast(s8_t, v);
    }
    const int np_all = np + (t_last < t_end ? 1 : 0);
    auto process_exact = [&](const PageRegs<WC_KIND_BF16>& p, int jj) {
      const int t0 = t_begin + jj * kBlockTokens;
      if (t0 + kBlockTokens <= t_end)
        process_page<WC_KIND_BF16, METER, true, HALF, false, false, VM, false>(a, p, t0, t_end, r, g, wx, my_dsh, st);
      else
        process_page<WC_KIND_BF16, METER, false, HALF, false, false, VM, false>(a, p, t0, t_end, r, g, wx, my_dsh, st);
    };
    for (int c0 = 0; c0 < np_all; c0 += 64) {
      const int nc2 = min(64, np_all - c0);
      const int tv2 = lane < nc2 ? trow[pg0 + c0 + lane] : 0;
      const int fl2 = lane < nc2 && (int64_t)(uint32_t)tv2 < a.num_blocks ? a.repaired[(int64_t)tv2 * a.n_kv + kv] : 0;
      uint64_t em = (uint64_t)__ballot(fl2 != 0);
      auto next = [&]() {
        if (em == 0) return -1;
        const int j = __builtin_ctzll(em);
        em &= em - 1;
        return j;
      };
      PageRegs<WC_KIND_BF16> pa, pb;
      int ja = next();
      load_exact_page<VM>(a, __builtin_amdgcn_readlane(tv2, max(ja, 0)), ja >= 0, kv, r, g, pa);
      while (ja >= 0) {
        const int jb = next();
        load_exact_page<VM>(a, __builtin_amdgcn_readlane(tv2, max(jb, 0)), jb >= 0, kv, r, g, pb);
        process_exact(pa, c0 + ja);
        if (jb < 0) break;
        ja = next();
        load_exact_page<VM>(a, __builtin_amdgcn_readlane(tv2, max(ja, 0)), ja >= 0, kv, r, g, pa);
        process_exact(pb, c0 + jb);
      }
    }
  }

  // ---- merge the four waves of the workgroup, write one partial record ----
  if constexpr (HALF) {   // lanes r and r + 8 hold different tokens of head r
    st.l = bfly_add<8>(st.l);
    if constexpr (METER) st.n = bfly_add<8>(st.n);
    if constexpr (KIND == WC_KIND_INT8_DITHER) st.wsum = bfly_add<8>(st.wsum);
    if constexpr (VM) {
      st.ev = bfly_add<8>(st.ev);
      st.vmax = bfly_max<8>(st.vmax);
    }
  }
  if constexpr (VM) {
    st.ev = bfly_add<16>(st.ev);
    st.ev = bfly_add<32>(st.ev);
    st.vmax = bfly_max<16>(st.vmax);
    st.vmax = bfly_max<32>(st.vmax);
  }
  st.l = bfly_add<16>(st.l);
  st.l = bfly_add<32>(st.l);
  if constexpr (METER) {
    st.n = bfly_add<16>(st.n);
    st.n = bfly_add<32>(st.n);
  }
  if constexpr (KIND == WC_KIND_INT8_DITHER) {
    st.wsum = bfly_add<16>(st.wsum);
    st.wsum = bfly_add<32>(st.wsum);
  }
  const float wsum = st.wsum;
  // rows 4g+e of tile jt hold channel 8(4g+e)+jt = 32g + 8e + jt
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float v[8];
#pragma unroll
    for (int jt = 0; jt < 8; ++jt) {
      v[jt] = st.o1[jt][e];
      if constexpr (KIND == WC_KIND_INT8_DITHER && GS)
        v[jt] = fmaf(kQOff, st.ws4[e], v[jt]);   // channel 32g + 8e + jt is in group g
      else if constexpr (KIND == WC_KIND_INT8_DITHER)
        v[jt] = fmaf(-kVOff, wsum, v[jt]);
    }
    float4* dst = reinterpret_cast<float4*>(&lds.w[wave].acc[r][32 * g + 8 * e]);
    dst[0] = make_float4(v[0], v[1], v[2], v[3]);
    dst[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
  if (g == 0) {
    ml_s[wave][r][0] = st.m;     // -inf for a wave without tokens
    ml_s[wave][r][1] = st.l;
    ml_s[wave][r][2] = st.n;
    ml_s[wave][r][3] = st.ev;
    ml_s[wave][r][4] = st.vmax;
    ml_s[wave][r][5] = (float)st.ve;
  }
  __syncthreads();
  const int64_t R = (int64_t)partial_record_floats(kD);
  if (wave == 0 && hv) {   // one partial record per (query head, split)
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, ml_s[w][r][0]);
    // (weights carry 2^kWExp: the record is written without it, in the same units
    // as the vector path's records)
    float f[kWaves], lsum = 0.0f, nsum = 0.0f, esum = 0.0f, vmax = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float mw = ml_s[w][r][0];
      f[w] = mw == -INFINITY ? 0.0f : exp2_fast(mw - M - kWExp);
      lsum = fmaf(f[w], ml_s[w][r][1], lsum);
      if constexpr (METER) nsum = fmaf(f[w], ml_s[w][r][2], nsum);
      if constexpr (VM) {
        esum = fmaf(f[w], ml_s[w][r][3], esum);
        vmax = fmaxf(vmax, ml_s[w][r][4]);
      }
    }
    if (isnan(nsum)) nsum = INFINITY;
    // the output accumulators also carry each wave's 2^-ve (INT8 and bf16 values; 0 for fp8
    // values unless the wave read exact pages)
    float fo[kWaves];
#pragma unroll
    for (int w = 0; w < kWaves; ++w) fo[w] = f[w] * exp2_fast(ml_s[w][r][5]);
    float* rec = a.part + (((int64_t)b * a.n_q + (int64_t)kv * G + r) * a.n_splits + split) * R;
#pragma unroll
    for (int i = 0; i < 32; i += 4) {
      float4 sum = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float4 x = *reinterpret_cast<const float4*>(&lds.w[w].acc[r][32 * g + i]);
        sum.x = fmaf(fo[w], x.x, sum.x);
        sum.y = fmaf(fo[w], x.y, sum.y);
        sum.z = fmaf(fo[w], x.z, sum.z);
        sum.w = fmaf(fo[w], x.w, sum.w);
      }
      *reinterpret_cast<float4*>(rec + 32 * g + i) = sum;
    }
    if (g == 0) {
      rec[kD] = M * kLn2;   // records hold the max in natural-log units
      rec[kD + 1] = lsum;
      rec[kD + 2] = nsum;
      rec[kD + 3] = esum;
      rec[kD + 4] = vmax;

    }
  }

}

template <int KIND, bool METER, bool HALF, bool TB, bool BYP, bool VM, bool REP, bool GS>
__global__ __launch_bounds__(256, 2) void decode_mfma_kernel(DecodeArgs a) {
  __shared__ DecodeLds<KIND> lds;
  decode_block<KIND, METER, HALF, TB, BYP, VM, REP, GS>(a, blockIdx.x + gridDim.x * blockIdx.y, lds);
}

// Speculative certified step: the metered decode (KIND_M, Tier A) and the exact
// fallback of every unit in one launch of 2 nb workgroups (nb = n_splits x batch x
// n_kv each).  Linear index j: groups of eight alternate between the two decodes
// (group 2i to the metered one, 2i + 1 to the exact one), each keeping its own
// linear order within every XCD (j mod 8); the last partial group of each follows.
// Every compute unit then holds both kinds, the metered decode's vector and matrix
// work beside the exact fallback's memory streaming.
template <int KIND_M, bool HALF>
__global__ __launch_bounds__(256, 2) void decode_spec_kernel(DecodeArgs am, DecodeArgs ax, uint32_t nb) {
  __shared__ DecodeLds<WC_KIND_INT8_DITHER> lds;   // (the largest layout)
  const uint32_t j = blockIdx.x, full = nb / 8u * 8u;
  bool metered;
  uint32_t lin;
  if (j < 2u * full) {
    metered = ((j >> 3) & 1u) == 0;
    lin = (j >> 4) * 8u + (j & 7u);
  } else {
    const uint32_t rest = nb - full, k = j - 2u * full;
    metered = k < rest;
    lin = full + (metered ? k : k - rest);
  }
  if (metered)
    decode_block<KIND_M, true, HALF, false, false, false, false, false>(
        am, lin, reinterpret_cast<DecodeLds<KIND_M>&>(lds));
  else
    decode_block<WC_KIND_BF16, false, HALF, false, false, false, false, false>(
        ax, lin, reinterpret_cast<DecodeLds<WC_KIND_BF16>&>(lds));
}

}  // namespace

// The INT8 variants (Tier B, bypassed pairs) of one (HALF, VM, REP, GS).
template <bool HALF, bool VM, bool REP, bool GS>
void launch_decode_mfma_int8(const DecodeArgs& a, bool tb, bool byp, const dim3& grid, const dim3& block,
                             hipStream_t st) {
  constexpr int K = WC_KIND_INT8_DITHER;
  if (tb && byp) hipLaunchKernelGGL((decode_mfma_kernel<K, true, HALF, true, true, VM, REP, GS>), grid, block, 0, st, a);
  else if (tb) hipLaunchKernelGGL((decode_mfma_kernel<K, true, HALF, true, false, VM, REP, GS>), grid, block, 0, st, a);
  else if (byp) hipLaunchKernelGGL((decode_mfma_kernel<K, true, HALF, false, true, VM, REP, GS>), grid, block, 0, st, a);
  else hipLaunchKernelGGL((decode_mfma_kernel<K, true, HALF, false, false, VM, REP, GS>), grid, block, 0, st, a);
}

// Metered decode over a group-scaled INT8 cache (its instantiations have a
// translation unit of their own, decode_mfma_gs.hip).
void launch_decode_mfma_gs(const DecodeArgs& a, bool tb, bool byp, bool vm, const dim3& grid, const dim3& block,
                           hipStream_t st);

}  // namespace wc
