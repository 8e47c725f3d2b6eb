// Metered decode attention, vector-ALU path (fp32 arithmetic throughout).
//
// Read path of the meter loop (Sec. 6): over a split of the KV axis one
// workgroup regenerates the Philox dither of every cached token, dequantizes,
// forms the compressed logits of the G query heads of one KV head, keeps an
// online softmax, accumulates the meter numerator sum_t e^{l_t - m} (e^{c_t} - 1)
// with c_t = sm_scale * sum_b ||q_b|| w_{t,b} (Theorem black-box logit bound),
// and the unnormalized output.  A second kernel merges the split partials under
// the LSE weights; A merges exactly like the output because it is a softmax-
// weighted average (Sec. 6.2, SGLang decode kernel).  The same kernels, without
// the meter and restricted to routed KV heads, serve the exact bf16 fallback.
//
// Tile of 64 tokens, 256 threads, three phases separated by barriers:
//   1  thread (token i, quarter of the channels): dither + dequant + partial
//      dot products with all G queries, reduced over the 4 quarter-lanes;
//      per-token bound c_t from the stored witness.
//   2  wave w, heads w, w+4, ...: lane = token; running max / sum / meter
//      numerator, weights p_t * s^v_t to LDS.
//   3  thread (channel, head subset): rescale and accumulate p_t * (code - xi).
#include <float.h>

#include "wc_device.h"
#include "merge_dev.h"
#include "wc_launch.h"

namespace wc {

namespace {

constexpr int kT = 64;        // tokens per tile
constexpr int kGMax = 16;     // query heads per KV head
constexpr int kThreads = 256;

template <int D, int KIND, int QT, bool METER>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(DecodeArgs a) {
  constexpr int CH = D / 4;            // phase-1 channels per thread
  constexpr int NG = CH / 16;          // Philox groups per thread
  constexpr int NHS = kThreads / D;    // phase-3 head subsets
  constexpr int HPT = kGMax / NHS;     // phase-3 heads per thread (max)

  __shared__ float q_s[kGMax][D];
  __shared__ float qbn_s[kGMax][16];
  __shared__ float ab_s[kGMax];       // Tier-B factor per head
  __shared__ float qo_s[kGMax][32];   // bypassed pairs: q at the stored values' channels
  __shared__ float logit_s[kGMax][kT];
  __shared__ float cb_s[kGMax][kT];
  __shared__ float pw_s[kGMax][kT];
  __shared__ uint32_t xi_s[kT][D / 4];
  __shared__ float vs_s[kT];
  __shared__ float vr_s[kT], vn_s[kT];   // value side: stored ||vhat - v|| and ||v|| of the tile
  __shared__ float vg_s[kT][D / 32];      // group scales: the tile's value group scales
  __shared__ float qg_s[kGMax][8];        // group scales, Tier B: ||q_g||^2 (0..3), ||q_g||_1 (4..7)
  __shared__ float alpha_s[kGMax];
  __shared__ int64_t slot_s[kT];
  __shared__ uint8_t ex_s[kT];            // persistent repair: the token's page is served exactly

  const DecodePos pos = decode_position(a.batch, a.n_kv, a.n_splits);
  const int split = pos.split, unit = pos.unit;
  const int b = unit / a.n_kv, kv = unit % a.n_kv;
  gate_clear(a, unit, split);
  const int L = a.seq_lens[b];
  const int t_begin = split * a.split_tokens;
  // certified step: the exact fallback decides its unit's gate from the metered
  // records first (split 0 always, for the masks; splits past the end skip it)
  if (KIND == WC_KIND_BF16 && a.gate_part != nullptr && (split == 0 || t_begin < L)) {
    __shared__ int gate_flag_s;
    if (!unit_gate(a, b, kv, split, __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), threadIdx.x & 63,
                   &gate_flag_s))
      return;
  }
  if (a.mask_kv != nullptr && a.mask_kv[unit] == 0) return;
  if (t_begin >= L) return;
  // clamp to what the block table can address (guards a seq_lens above max_seq_len)
  const int t_end = min(min(L, t_begin + a.split_tokens), a.max_blocks * kBlockTokens);
  const int G = a.group;
  const int B = a.n_bands;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;

  for (int i = tid; i < G * D; i += kThreads) {
    const int h = i / D, c = i % D;
    const int64_t qi = ((int64_t)b * a.n_q + (int64_t)kv * G + h) * D + c;
    q_s[h][c] = QT == WC_F32 ? reinterpret_cast<const float*>(a.q)[qi]
                             : bf16_to_f32(reinterpret_cast<const uint16_t*>(a.q)[qi]);
  }
  __syncthreads();
  // Bypassed pairs (Sec. 6.2 fixed-channel bypass): q at the channels of the
  // stored fp16 values goes to qo_s and leaves q_s, so the code products skip
  // those channels; Tier A's band norms are taken from the whole query first.
  const int m2 = 2 * a.n_pairs;
  const int32_t* plist = a.pairs + (int64_t)kv * a.n_pairs;
  if constexpr (METER) {
    for (int i = tid; i < G * B; i += kThreads) {
      const int h = i / B, bb = i % B;
      float acc = 0.0f;
      for (int k = 0; k < D / B; ++k) {
        const float x = q_s[h][band_channel(bb, k, D, B, a.interleaved)];
        acc = fmaf(x, x, acc);
      }
      qbn_s[h][bb] = sqrtf(acc) * a.sm_scale;
    }
  }
  if (m2 > 0) {
    for (int i = tid; i < G * m2; i += kThreads) {
      const int h = i / m2, pos = i % m2;
      qo_s[h][pos] = q_s[h][pair_channel(plist[pos >> 1], pos & 1, D, a.interleaved)];
    }
    __syncthreads();
    for (int i = tid; i < G * m2; i += kThreads) {
      const int h = i / m2, pos = i % m2;
      q_s[h][pair_channel(plist[pos >> 1], pos & 1, D, a.interleaved)] = 0.0f;
    }
    __syncthreads();
  }
  const bool grouped = KIND == WC_KIND_INT8_DITHER && a.group_scales != 0;
  if constexpr (METER) {
    if (a.tierb_delta > 0.0f) {
      for (int h = tid; h < G; h += kThreads) {
        float sq = 0.0f, l1 = 0.0f;
        for (int c = 0; c < D; ++c) {
          sq = fmaf(q_s[h][c], q_s[h][c], sq);
          l1 += fabsf(q_s[h][c]);
        }
        ab_s[h] = tierb_factor(sq, l1, L, a.tierb_delta, a.sm_scale);
      }
      if (grouped) {   // per-group norms of the quantized channels
        for (int i = tid; i < G * (D / 32); i += kThreads) {
          const int h = i / (D / 32), gg = i % (D / 32);
          float sq = 0.0f, l1 = 0.0f;
          for (int c = 32 * gg; c < 32 * gg + 32; ++c) {
            sq = fmaf(q_s[h][c], q_s[h][c], sq);
            l1 += fabsf(q_s[h][c]);
          }
          qg_s[h][gg] = sq;
          qg_s[h][4 + gg] = l1;
        }
      }
    }
  }
  // Tier B over group steps: u_t = sm (rt sqrt(sum_g s_g^2 ||q_g||^2) + sum_g s_g ||q_g||_1 / 256)
  const float rt = METER && grouped && a.tierb_delta > 0.0f
                       ? sqrtf(2.0f * logf(2.0f * (float)L / a.tierb_delta) / 12.0f) : 0.0f;

  const bool vm = METER && a.meter_v != nullptr;   // value side
  float m_run[4], l_run[4], n_run[4], e_run[4], vmax_run = 0.0f;
  float nb_run[4];   // meter numerator of the open block segment, per head slot
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    m_run[k] = -INFINITY;
    l_run[k] = 0.0f;
    n_run[k] = 0.0f;
    e_run[k] = 0.0f;
    nb_run[k] = 0.0f;
  }
  // Block segments (block repair's shares, Sec. 6.3): the split's tiles (64
  // tokens, each inside one 256-token repair block) grouped by repair block; a
  // segment's numerator, frame, first page and length go to the split's next
  // share slot, and every slot of the split is written (unused ones with 0 pages).
  const bool rec_shares = METER && a.shares != nullptr;
  int seg_first = t_begin / kBlockTokens, seg_slot = 0;
  auto flush_segment = [&](int last_page) {
    if (lane == 0) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int h = wave + 4 * k;
        if (h < G && seg_slot < a.share_slots)
          a.shares[(((int64_t)b * a.n_q + (int64_t)kv * G + h) * a.n_splits + split) * a.share_slots + seg_slot] =
              make_float4(nb_run[k], m_run[k], __builtin_bit_cast(float, seg_first),
                          __builtin_bit_cast(float, last_page - seg_first));
      }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) nb_run[k] = 0.0f;
    ++seg_slot;
    seg_first = last_page;
  };
  const int c3 = tid % D, hs = tid / D;
  float acc[HPT];
#pragma unroll
  for (int k = 0; k < HPT; ++k) acc[k] = 0.0f;
  const uint32_t layer_head = ((uint32_t)a.layer << 16) | (uint32_t)kv;

  for (int t0 = t_begin; t0 < t_end; t0 += kT) {
    if (rec_shares && (t0 & (kRepairBlockTokens - 1)) == 0 && t0 / kBlockTokens > seg_first)
      flush_segment(t0 / kBlockTokens);
    __syncthreads();
    // ---------------- phase 1: logits and per-token bounds ----------------
    {
      const int i = tid >> 2, part = tid & 3;
      const int t = t0 + i;
      // a table entry outside the cache leaves the token out (no access outside it)
      const int32_t e = t < t_end ? a.table[(int64_t)b * a.max_blocks + t / kBlockTokens] : -1;
      const bool valid = t < t_end && (int64_t)(uint32_t)e < a.num_blocks;
      int64_t slot = -1;
      if (valid) slot = (int64_t)e * kBlockTokens + t % kBlockTokens;
      if (part == 0) slot_s[i] = slot;
      const int c0 = part * CH;
      const int64_t page = valid ? (slot / kBlockTokens) * a.n_kv + kv : 0;
      const int off = valid ? (int)(slot % kBlockTokens) : 0;
      // a page marked as repaired is read from the exact store with bound 0
      const bool ex = KIND != WC_KIND_BF16 && valid && a.repaired != nullptr && a.repaired[page] != 0;
      if (part == 0) ex_s[i] = ex ? 1 : 0;
      float kval[CH];
#pragma unroll
      for (int c = 0; c < CH; ++c) kval[c] = 0.0f;
      if (ex) {
        const uint8_t* kpg = reinterpret_cast<const uint8_t*>(a.x_k_data) + page * (kBlockTokens * D * 2);
#pragma unroll
        for (int v4 = 0; v4 < CH / 8; ++v4) {
          const uint4 cw = *reinterpret_cast<const uint4*>(kpg + kpage_off(off, c0 + 8 * v4, D, 2));
          const uint32_t wds[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
          for (int w4 = 0; w4 < 4; ++w4) {
            kval[8 * v4 + 2 * w4] = bf16_to_f32((uint16_t)(wds[w4] & 0xFFFFu));
            kval[8 * v4 + 2 * w4 + 1] = bf16_to_f32((uint16_t)(wds[w4] >> 16));
          }
        }
        if (part == 0) vs_s[i] = 1.0f;
        if (grouped)
          for (int gg = part; gg < D / 32; gg += 4) vg_s[i][gg] = 1.0f;
      } else if (valid) {
        if constexpr (KIND == WC_KIND_INT8_DITHER) {
          const uint8_t* kpg = reinterpret_cast<const uint8_t*>(a.k_data) + page * (kBlockTokens * D);
          const int64_t srow = page * kBlockTokens + off;
#pragma unroll
          for (int gi = 0; gi < NG; ++gi) {
            const uint4 cw = *reinterpret_cast<const uint4*>(kpg + kpage_off(off, c0 + 16 * gi, D, 1));
            const U4 r = dither_block(c0 / 16 + gi, slot, layer_head, a.key0, a.key1);
            const uint32_t codes[4] = {cw.x, cw.y, cw.z, cw.w};
            const uint32_t rw[4] = {r.x, r.y, r.z, r.w};
            const float sg = scale_of(a.k_scale, srow, c0 + 16 * gi, D, grouped);   // the channels' step
#pragma unroll
            for (int w4 = 0; w4 < 4; ++w4) {
              xi_s[i][(c0 + 16 * gi) / 4 + w4] = rw[w4];
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                const float code = (float)((int32_t)((codes[w4] >> (8 * j)) & 0xFFu) - 128);   // excess-128
                const float xi = dither_value((rw[w4] >> (8 * j)) & 0xFFu);
                kval[16 * gi + 4 * w4 + j] = sg * (code - xi);
              }
            }
          }
          if (part == 0) vs_s[i] = grouped ? 1.0f : f16_to_f32(a.v_scale[srow]);   // (groups: per channel below)
          if (grouped)
            for (int gg = part; gg < D / 32; gg += 4) vg_s[i][gg] = f16_to_f32(a.v_scale[srow * (D / 32) + gg]);
        } else if constexpr (KIND == WC_KIND_FP8_RAW) {
          const uint8_t* kpg = reinterpret_cast<const uint8_t*>(a.k_data) + page * (kBlockTokens * D);
#pragma unroll
          for (int gi = 0; gi < NG; ++gi) {
            const uint4 cw = *reinterpret_cast<const uint4*>(kpg + kpage_off(off, c0 + 16 * gi, D, 1));
            const uint32_t codes[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
            for (int w4 = 0; w4 < 4; ++w4)
#pragma unroll
              for (int j = 0; j < 4; ++j)
                kval[16 * gi + 4 * w4 + j] = e4m3_to_f32((codes[w4] >> (8 * j)) & 0xFFu);
          }
          if (part == 0) vs_s[i] = 1.0f;
        } else {
          const uint8_t* kpg = reinterpret_cast<const uint8_t*>(a.k_data) + page * (kBlockTokens * D * 2);
#pragma unroll
          for (int v4 = 0; v4 < CH / 8; ++v4) {
            const uint4 cw = *reinterpret_cast<const uint4*>(kpg + kpage_off(off, c0 + 8 * v4, D, 2));
            const uint32_t wds[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
            for (int w4 = 0; w4 < 4; ++w4) {
              kval[8 * v4 + 2 * w4] = bf16_to_f32((uint16_t)(wds[w4] & 0xFFFFu));
              kval[8 * v4 + 2 * w4 + 1] = bf16_to_f32((uint16_t)(wds[w4] >> 16));
            }
          }
          if (part == 0) vs_s[i] = 1.0f;
        }
      } else if (part == 0) {
        vs_s[i] = 0.0f;
        if (grouped)
          for (int gg = 0; gg < D / 32; ++gg) vg_s[i][gg] = 0.0f;
      }
      if (vm && part == 0) {
        vr_s[i] = valid && !ex ? f16_to_f32(a.v_resid[page * kBlockTokens + off]) : 0.0f;
        vn_s[i] = valid ? f16_to_f32(a.v_norm[page * kBlockTokens + off]) : 0.0f;
      }
      // stored fp16 values of the bypassed pairs: positions part, part + 4, ...
      // (an exact token: its bf16 keys at those channels)
      float kov[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int pos = part + 4 * k;
        if (ex && pos < m2) {
          const int ch = pair_channel(plist[pos >> 1], pos & 1, D, a.interleaved);
          kov[k] = bf16_to_f32(*reinterpret_cast<const uint16_t*>(
              reinterpret_cast<const uint8_t*>(a.x_k_data) + page * (kBlockTokens * D * 2) + kpage_off(off, ch, D, 2)));
        } else {
          kov[k] = (valid && pos < m2) ? f16_to_f32(a.k_outlier[(page * kBlockTokens + off) * m2 + pos]) : 0.0f;
        }
      }
      for (int h = 0; h < G; ++h) {
        float d = 0.0f;
#pragma unroll
        for (int c = 0; c < CH; ++c) d = fmaf(q_s[h][c0 + c], kval[c], d);
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (part + 4 * k < m2) d = fmaf(qo_s[h][part + 4 * k], kov[k], d);
        d += __shfl_xor(d, 1, 4);
        d += __shfl_xor(d, 2, 4);
        if (part == 0) logit_s[h][i] = valid ? d * a.sm_scale : -INFINITY;
      }
      if (METER && a.tierb_delta > 0.0f) {   // Tier B: u_t = (alpha_h + beta_h) s_t, no witness
        const float s = valid && !ex && !grouped ? f16_to_f32(a.k_scale[page * kBlockTokens + off]) : 0.0f;
        for (int h = 0; h < G; ++h) {
          // fp16 rounding bound of the bypassed channels: sm sum |q_c| (2^-11 |khat_c| + 2^-25)
          float gb = 0.0f;
#pragma unroll
          for (int k = 0; k < 8; ++k)
            if (part + 4 * k < m2)
              gb = fmaf(fabsf(qo_s[h][part + 4 * k]), fmaf(fabsf(kov[k]), 0x1p-11f, 0x1p-25f), gb);
          gb += __shfl_xor(gb, 1, 4);
          gb += __shfl_xor(gb, 2, 4);
          if (ex) gb = 0.0f;   // (exact keys: no rounding term)
          if (part == 0) {
            if (grouped) {
              float s2 = 0.0f, s1 = 0.0f;
              for (int gg = 0; gg < D / 32; ++gg) {
                const float sg = valid && !ex ? scale_of(a.k_scale, page * kBlockTokens + off, 32 * gg, D, true) : 0.0f;
                s2 = fmaf(sg * sg, qg_s[h][gg], s2);
                s1 = fmaf(sg, qg_s[h][4 + gg], s1);
              }
              cb_s[h][i] = a.sm_scale * (fmaf(rt, sqrtf(s2), s1 * (1.0f / 256.0f)) + gb);
            } else {
              cb_s[h][i] = fmaf(ab_s[h], s, gb * a.sm_scale);
            }
          }
        }
      } else if constexpr (METER) {
        float wv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        if (valid && !ex) {
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int bb = part + 4 * k;
            if (bb < B) wv[k] = f16_to_f32(a.k_witness[(page * kBlockTokens + off) * B + bb]);
          }
        }
        for (int h = 0; h < G; ++h) {
          float cp = 0.0f;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int bb = part + 4 * k;
            if (bb < B) cp = fmaf(qbn_s[h][bb], wv[k], cp);
          }
          cp += __shfl_xor(cp, 1, 4);
          cp += __shfl_xor(cp, 2, 4);
          if (part == 0) cb_s[h][i] = cp;
        }
      }
    }
    __syncthreads();
    // ---------------- phase 2: online softmax and meter numerator ----------------
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int h = wave + 4 * k;
      if (h < G) {
        const float l = logit_s[h][lane];
        const float m_new = fmaxf(m_run[k], wave_max(l));
        const float alpha = expf(m_run[k] - m_new);
        const float p = expf(l - m_new);
        float term = 0.0f;
        if constexpr (METER) {
          const float c = cb_s[h][lane];
          // p (e^c - 1); for large c in the log domain so that a token whose
          // weight underflows still counts with its bound (never truncate c)
          term = c > 1.0f ? expf(l - m_new + c) - p : p * expm1f(c);
        }
        const float lsum = wave_sum(p);
        l_run[k] = fmaf(alpha, l_run[k], lsum);
        if constexpr (METER) {
          const float nn = fmaf(alpha, n_run[k], wave_sum(term));
          n_run[k] = isnan(nn) ? INFINITY : nn;
          const float nbq = fmaf(alpha, nb_run[k], wave_sum(term));
          nb_run[k] = isnan(nbq) ? INFINITY : nbq;
        }
        if (vm) {
          e_run[k] = fmaf(alpha, e_run[k], wave_sum(p * vr_s[lane]));
          vmax_run = fmaxf(vmax_run, wave_max(vn_s[lane]));
        }
        m_run[k] = m_new;
        pw_s[h][lane] = p * vs_s[lane];
        if (lane == 0) alpha_s[h] = alpha;
      }
    }
    __syncthreads();
    // ---------------- phase 3: P V ----------------
    {
#pragma unroll
      for (int k = 0; k < HPT; ++k) {
        const int h = hs + k * NHS;
        if (h < G) acc[k] *= alpha_s[h];
      }
      for (int qd = 0; qd < kT / 4; ++qd) {
        const int i0 = 4 * qd;
        const int64_t slot = slot_s[i0];
        if (slot < 0) continue;   // past the end, or a table entry outside the cache
        const int64_t page = (slot / kBlockTokens) * a.n_kv + kv;
        const int off = (int)(slot % kBlockTokens);   // multiple of 4
        float vv[4];
        if (KIND == WC_KIND_BF16 || ex_s[i0]) {   // (a quad lies in one page: one mark)
          const void* vd = KIND == WC_KIND_BF16 ? a.v_data : a.x_v_data;
          const uint2 w = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint8_t*>(vd) +
                                                          page * (kBlockTokens * D * 2) + vpage_off(off, c3, D, 2));
          vv[0] = bf16_to_f32((uint16_t)(w.x & 0xFFFFu));
          vv[1] = bf16_to_f32((uint16_t)(w.x >> 16));
          vv[2] = bf16_to_f32((uint16_t)(w.y & 0xFFFFu));
          vv[3] = bf16_to_f32((uint16_t)(w.y >> 16));
        } else {
          const uint32_t w = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint8_t*>(a.v_data) +
                                                              page * (kBlockTokens * D) + vpage_off(off, c3, D, 1));
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const uint32_t byte = (w >> (8 * j)) & 0xFFu;
            if constexpr (KIND == WC_KIND_INT8_DITHER) {
              const uint32_t u = (xi_s[i0 + j][c3 >> 2] >> (8 * (c3 & 3))) & 0xFFu;
              vv[j] = (float)((int32_t)byte - 128) - dither_value(u);   // excess-128 code
              if (grouped) vv[j] *= vg_s[i0 + j][c3 >> 5];
            } else {
              vv[j] = e4m3_to_f32(byte);
            }
          }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (t0 + i0 + j >= t_end) vv[j] = 0.0f;
#pragma unroll
        for (int k = 0; k < HPT; ++k) {
          const int h = hs + k * NHS;
          if (h < G) {
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[k] = fmaf(pw_s[h][i0 + j], vv[j], acc[k]);
          }
        }
      }
    }
  }

  if (rec_shares) {
    flush_segment((t_end + kBlockTokens - 1) / kBlockTokens);
    if (lane == 0) {
      for (int sl = seg_slot; sl < a.share_slots; ++sl)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int h = wave + 4 * k;
          if (h < G)
            a.shares[(((int64_t)b * a.n_q + (int64_t)kv * G + h) * a.n_splits + split) * a.share_slots + sl] =
                make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        }
    }
  }
  const int64_t R = (int64_t)partial_record_floats(D);
  const int64_t rec_base = ((int64_t)b * a.n_q + (int64_t)kv * G) * a.n_splits + split;
#pragma unroll
  for (int k = 0; k < HPT; ++k) {
    const int h = hs + k * NHS;
    if (h < G) a.part[(rec_base + (int64_t)h * a.n_splits) * R + c3] = acc[k];
  }
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int h = wave + 4 * k;
      if (h < G) {
        float* rec = a.part + (rec_base + (int64_t)h * a.n_splits) * R;
        rec[D] = m_run[k];
        rec[D + 1] = l_run[k];
        rec[D + 2] = n_run[k];
        rec[D + 3] = e_run[k];
        rec[D + 4] = vmax_run;

      }
    }
  }
}

// Merge of the split records of one (sequence, query head) under the LSE
// weights: out = sum_j e^{m_j - M} acc_j / L, A - 1 = sum_j e^{m_j - M} N_j / L with
// L = sum_j e^{m_j - M} l_j; raw = (A-1)(A+1)/2 (+inf on overflow), meter = min(1, raw)
// (Sec. 6.2: A merges exactly like the output).  The statistics (M, L, the
// numerators) come from split_stats (merge_dev.h), in the same bits wherever they
// are formed.
constexpr int kMergeWaves = 4;   // waves per merge workgroup when a head has more than 32 splits

// The statistics a merge needs: of the output rows (so; the exact records of a
// routed head in a certified step's final merge) and of the metered records for
// the meter (sm).  Up to 64 splits both records' scalars are read in one round trip.
template <bool METER, bool VM>
__device__ __forceinline__ void merge_stats(const float* rec0, const float* src0, bool routed, int64_t R, int ns,
                                            int n_avail, int lane, SplitStats& so, SplitStats& sm) {
  const int D = (int)R - 8;
  if (n_avail <= 64 && routed) {
    const int jr = min(lane, n_avail - 1);
    const float4 tx = *reinterpret_cast<const float4*>(src0 + (int64_t)jr * R + D);
    const float4 tm = *reinterpret_cast<const float4*>(rec0 + (int64_t)jr * R + D);
    const float tv = VM ? rec0[(int64_t)jr * R + D + 4] : 0.0f;
    so = stats_of_lanes<false, false>(tx, 0.0f, ns, lane);
    sm = stats_of_lanes<METER, VM>(tm, tv, ns, lane);
    return;
  }
  if (routed) {
    so = split_stats<false, false>(src0, R, D, ns, n_avail, lane);
    sm = split_stats<METER, VM>(rec0, R, D, ns, n_avail, lane);
  } else {
    so = sm = split_stats<METER, VM>(rec0, R, D, ns, n_avail, lane);
  }
}

// Split-KV merge (Sec. 6.2): one workgroup per (sequence, query head).  The
// output rows go 32 splits at a time to the waves in turn: lane j % 32 weighs split
// j, every lane holds its channels of all 32 partial outputs (all of a chunk's
// loads are issued together, before the statistics), and the weights reach the
// channel lanes through readlane.  The waves' sums are added in LDS in wave order.
// Final merge of a certified step (a.x_part set): the heads of a routed KV head
// (gate_mask_kv, stored by the exact fallback's prologue) take their output from
// the exact records, the others from the metered ones; meter and raw always from
// the metered records.  Speculative certified step (a.merge_gate): the exact
// records cover every unit and each wave decides its unit's gate itself from the
// metered records, with the statistics the exact fallback's prologue uses (every
// wave of the unit's workgroups stores the same masks).
template <int D, bool METER, bool VM, int NW>
__global__ __launch_bounds__(64 * NW) void merge_kernel(DecodeArgs a) {
  constexpr int C = D / 64;   // channels per lane
  __shared__ float acc_s[NW][D];
  const int bh = blockIdx.x;
  const int b = bh / a.n_q, h = bh % a.n_q;
  const int unit = b * a.n_kv + h / a.group;
  if (a.mask_kv != nullptr && a.mask_kv[unit] == 0) return;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int64_t R = (int64_t)partial_record_floats(D);
  const bool fin = a.x_part != nullptr;
  bool routed = fin && !a.merge_gate && a.gate_mask_kv[unit] != 0;
  const float* rec0 = a.part + (int64_t)bh * a.n_splits * R;
  const float* xrec0 = fin ? a.x_part + (int64_t)bh * a.n_splits * R : rec0;
  const int jl = lane & 31;
  const int L = a.seq_lens[b];
  // The rows of a chunk (32 splits from j0; rows past the last split repeat it) and
  // lane jl's split max; the rows are requested before the sequence length is
  // known, and rows past the last active split are read (they exist in the
  // workspace) but not used.
  auto load_chunk = [&](const float* s0, int j0, float (&ov)[32][C]) {
    const int nr = min(32, a.n_splits - j0);
    const float mj = s0[(int64_t)(j0 + min(jl, nr - 1)) * R + D];
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const float* src = s0 + (int64_t)(j0 + min(j, nr - 1)) * R + C * lane;
      if constexpr (C == 2) {
        const float2 v = *reinterpret_cast<const float2*>(src);
        ov[j][0] = v.x;
        ov[j][1] = v.y;
      } else {
        ov[j][0] = src[0];
      }
    }
    return mj;
  };
  // Speculative certified step: the exact rows of this wave's first chunk are
  // requested before the unit's gate is decided, so that the gate's loads go out
  // with them (the guess is the step's premise, a routed unit; a unit that is not
  // reads its metered rows afterwards).
  // Its own head's statistics come with the gate (the metered records' -- the same
  // bits as merge_stats -- and, up to 64 splits, the exact records' from scalars
  // fetched with the rows), so no further round trip precedes the merge.
  float ovp[32][C];
  float mjp = 0.0f;
  bool pre = false, gstats = false;
  float4 txp = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  SplitStats gsm{};
  if (fin && a.merge_gate) {
    if (32 * wave < a.n_splits) {
      mjp = load_chunk(xrec0, 32 * wave, ovp);
      pre = true;
    }
    gstats = !VM && a.n_splits <= 64;
    if (gstats) txp = *reinterpret_cast<const float4*>(xrec0 + (int64_t)min(lane, a.n_splits - 1) * R + D);
    routed = unit_gate_wave(a, b, h / a.group, lane, h % a.group, &gsm);
    pre = pre && routed;
  }
  const float* src0 = routed ? xrec0 : rec0;   // output rows
  auto stats = [&](int ns_, SplitStats& so_, SplitStats& sm_) {
    if (gstats) {
      sm_ = gsm;
      so_ = routed ? stats_of_lanes<false, false>(txp, 0.0f, ns_, lane) : gsm;
    } else {
      merge_stats<METER, VM>(rec0, src0, routed, R, ns_, a.n_splits, lane, so_, sm_);
    }
  };

  float acc[C];
#pragma unroll
  for (int c = 0; c < C; ++c) acc[c] = 0.0f;
  SplitStats so{}, sm{};   // the output rows' statistics; the meter's (the metered records)
  bool have = false;
  int ns = 0;
  for (int j0 = 32 * wave; j0 < a.n_splits; j0 += 32 * NW) {
    float ov[32][C];
    float mj_raw;
    if (pre && j0 == 32 * wave) {
#pragma unroll
      for (int j = 0; j < 32; ++j)
#pragma unroll
        for (int c = 0; c < C; ++c) ov[j][c] = ovp[j][c];
      mj_raw = mjp;
    } else {
      mj_raw = load_chunk(src0, j0, ov);
    }
    ns = active_splits(L, a.split_tokens, a.n_splits);
    if (j0 >= ns) break;
    const int nj = min(32, ns - j0);
    if (!have) {   // the statistics (the first chunk's loads are in flight)
      stats(ns, so, sm);
      have = true;
    }
    const float mj = jl < nj ? mj_raw : -INFINITY;
    const float ej = mj == -INFINITY ? 0.0f : __expf(mj - so.M);
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      if (j < nj) {
        const float e = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ej), j));
#pragma unroll
        for (int c = 0; c < C; ++c) acc[c] = fmaf(e, ov[j][c], acc[c]);
      }
    }
  }
  ns = active_splits(L, a.split_tokens, a.n_splits);
  if (!have && wave == 0) stats(ns, so, sm);
#pragma unroll
  for (int c = 0; c < C; ++c) acc_s[wave][C * lane + c] = acc[c];
  if constexpr (NW > 1) __syncthreads();
  if (wave != 0) return;
  // The meter and the gate first: the gate's counter atomic is then in flight
  // while the output row is formed and stored, and its result is used after.
  int gate_unit = -1, gate_old = -1;
  if constexpr (METER) {
    if (lane == 0) {
      const float raw = raw_of(sm, ns);
      a.meter[bh] = fminf(1.0f, raw);
      if (a.raw != nullptr) a.raw[bh] = raw;
      const float mv = VM ? meter_v_of(sm, ns) : 0.0f;
      if constexpr (VM) a.meter_v[bh] = mv;
      if (fin) {
        // (the gate was decided and stored by the exact fallback's prologue): counts
        // of gated query heads and, by each KV head's first query head, routed KV heads
        if (a.gate_count != nullptr) {
          // (the speculative merge's own head: the gate unit_gate_wave stored)
          const bool own = a.merge_gate ? gated_of(raw, 0.0f, a.gate_tau, false, 0.0f) : a.gate_mask_q[bh] != 0;
          if (own) atomicAdd(a.gate_count, 1);
          if (h % a.group == 0 && routed) atomicAdd(a.gate_count + 1, 1);
        }
      } else if (a.gate_mask_q != nullptr) {
        // the gate of this query head (the joint one: pass_K and pass_V); its KV
        // head is counted by the first gated head
        const bool gated = gated_of(raw, mv, a.gate_tau, VM, a.gate_tau_v);
        a.gate_mask_q[bh] = gated ? 1 : 0;
        if (gated) {
          gate_unit = unit;
          a.gate_mask_kv[gate_unit] = 1;
          gate_old = atomicAdd(a.gate_unit + gate_unit, 1);
        }
      }
    }
  }
#pragma unroll
  for (int c = 0; c < C; ++c) {
    float o = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) o += acc_s[w][C * lane + c];
    o = ns > 0 ? o / so.l : 0.0f;
    const int64_t oi = (int64_t)bh * D + C * lane + c;
    if (a.out_dtype == WC_F32)
      reinterpret_cast<float*>(a.out)[oi] = o;
    else
      reinterpret_cast<uint16_t*>(a.out)[oi] = f32_to_bf16_rne(o);
  }
  if (METER && gate_unit >= 0 && a.gate_count != nullptr) {   // (lane 0 of a gated head)
    asm volatile("" : "+v"(gate_old));   // (keeps the wait for the counter here)
    atomicAdd(a.gate_count, 1);
    if (gate_old == 0) atomicAdd(a.gate_count + 1, 1);
  }
}

template <int D, int KIND, int QT, bool METER>
hipError_t launch_dq(const DecodeArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((decode_split_kernel<D, KIND, QT, METER>), dim3(a.n_splits, a.batch * a.n_kv),
                     dim3(kThreads), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.no_merge) return e;
  return launch_merge(a, METER, st);
}

template <int D, int KIND, bool METER>
hipError_t launch_dk(const DecodeArgs& a, hipStream_t st) {
  return a.q_dtype == WC_F32 ? launch_dq<D, KIND, WC_F32, METER>(a, st)
                             : launch_dq<D, KIND, WC_BF16, METER>(a, st);
}

template <int D>
hipError_t launch_d(const DecodeArgs& a, bool metered, hipStream_t st) {
  if (!metered) return launch_dk<D, WC_KIND_BF16, false>(a, st);
  return a.kind == WC_KIND_INT8_DITHER ? launch_dk<D, WC_KIND_INT8_DITHER, true>(a, st)
                                       : launch_dk<D, WC_KIND_FP8_RAW, true>(a, st);
}

}  // namespace

int choose_split_tokens_total(int n_kv, int64_t max_seq_len, int64_t total_tokens, int64_t target) {
  // about `target` workgroups over all (sequence, KV head) token ranges: a long
  // sequence gets many splits, a short one one
  int64_t st = (total_tokens * n_kv + target - 1) / target;
  st = (st + 63) / 64 * 64;
  if (st < 256) st = 256;
  const int64_t cap = (max_seq_len + 63) / 64 * 64;
  if (st > cap && cap >= 256) st = cap;
  return (int)st;
}

int choose_split_tokens(int batch, int n_kv, int64_t max_seq_len, int requested, int64_t target) {
  if (requested > 0) return (requested + 63) / 64 * 64;
  // about `target` workgroups over the longest sequence
  const int64_t units = (int64_t)batch * n_kv;
  int64_t splits = target / (units > 0 ? units : 1);
  if (splits < 1) splits = 1;
  int64_t st = (max_seq_len + splits - 1) / splits;
  st = (st + 63) / 64 * 64;
  if (st < 256) st = 256;
  return (int)st;
}

template <int D, int NW>
void launch_merge_w(const DecodeArgs& a, bool metered, hipStream_t st) {
  const dim3 grid(a.batch * a.n_q), block(64 * NW);
  if (!metered) hipLaunchKernelGGL((merge_kernel<D, false, false, NW>), grid, block, 0, st, a);
  else if (a.meter_v != nullptr) hipLaunchKernelGGL((merge_kernel<D, true, true, NW>), grid, block, 0, st, a);
  else hipLaunchKernelGGL((merge_kernel<D, true, false, NW>), grid, block, 0, st, a);
}

// One wave per head takes up to 32 records in one round trip; more splits get four.
template <int D>
void launch_merge_d(const DecodeArgs& a, bool metered, hipStream_t st) {
  if (a.n_splits <= 32) launch_merge_w<D, 1>(a, metered, st);
  else launch_merge_w<D, kMergeWaves>(a, metered, st);
}

hipError_t launch_merge(const DecodeArgs& a, bool metered, hipStream_t st) {
  if (a.head_dim == 64) launch_merge_d<64>(a, metered, st);
  else launch_merge_d<128>(a, metered, st);
  return hipGetLastError();
}

hipError_t launch_decode(const DecodeArgs& a, bool metered, hipStream_t st) {
  if (a.batch == 0 || a.n_q == 0) return hipSuccess;
  if (a.use_mfma && mfma_decode_supported(a)) {
    hipError_t e = launch_decode_mfma(a, metered, st);
    return e != hipSuccess || a.no_merge ? e : launch_merge(a, metered, st);
  }
  return a.head_dim == 64 ? launch_d<64>(a, metered, st) : launch_d<128>(a, metered, st);
}

}  // namespace wc
