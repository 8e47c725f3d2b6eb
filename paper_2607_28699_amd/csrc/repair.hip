// Block-granular repair of routed KV heads (Sec. 6.3, block-level paging).
//
// The certificate is block decomposable: A - 1 = sum_t ptilde_t (e^{c_t} - 1) splits
// into per-block shares, and a block taken from the exact store contributes exact
// logits and values with bound 0.  One workgroup per routed (sequence, KV head):
//   1  rebuild each query head's merged state (max M, weight sum L, meter
//      numerator N, unnormalized output O) in float64 from the split records of
//      the metered decode that routed it, and the share of every block (a quarter
//      of a split: the records carry the four blocks' numerators);
//   2  order the blocks by the sum of their shares over the G query heads (ties
//      to the lower block), up to the repair budget;
//   3  take the blocks in that order; for each, recompute its tokens' compressed
//      logits, bounds and values and their exact logits and values (the exact
//      bf16 cache), and move L, N and O from the compressed to the exact terms:
//        L += sum (e^{l_t - M} - e^{lt_t - M}),  N -= sum e^{lt_t - M} (e^{c_t} - 1),
//        O += sum (e^{l_t - M} v_t - e^{lt_t - M} vhat_t);
//      after each block A = 1 + N / L per head; stop when every head passes tau.
// A repaired KV head gets its new outputs, meter and raw, and leaves the route
// mask; a KV head the budget cannot repair keeps its mask (whole-head fallback).
// Arithmetic of the state and the corrections is float64; logits and bounds are
// formed in fp32 as in the vector decode path.
#include <float.h>

#include "wc_device.h"
#include "wc_launch.h"

namespace wc {

namespace {

constexpr int kRThreads = 256;
constexpr int kRTile = 64;       // tokens per tile (4 threads per token in phase 1)
constexpr int kRGMax = 16;
constexpr int kRMaxBlocks = 4096;

template <int D, int QT>
__global__ __launch_bounds__(kRThreads) void repair_kernel(RepairArgs ra) {
  const DecodeArgs& a = ra.d;
  constexpr int CH = D / 4;
  constexpr int NG = CH / 16;
  constexpr int NHS = kRThreads / D;

  __shared__ float q_s[kRGMax][D];
  __shared__ float qk_s[kRGMax][D];      // q with bypassed channels zeroed (Tier B terms)
  __shared__ float qbn_s[kRGMax][16];
  __shared__ float ab_s[kRGMax];
  __shared__ int8_t opos_s[D];           // stored-value position of a bypassed channel, else -1
  __shared__ double M_s[kRGMax], L_s[kRGMax], N_s[kRGMax];
  __shared__ double O_s[kRGMax][D];
  __shared__ float T_s[kRMaxBlocks];     // block totals over the heads (-1: taken)
  __shared__ int order_s[64];
  __shared__ float lq_s[kRGMax][kRTile], lx_s[kRGMax][kRTile], cb_s[kRGMax][kRTile];
  __shared__ double wq_s[kRGMax][kRTile], wx_s[kRGMax][kRTile];
  __shared__ uint32_t xi_s[kRTile][D / 4];
  __shared__ float vs_s[kRTile];
  __shared__ int64_t slot_s[kRTile];
  __shared__ float red_v[kRThreads];
  __shared__ int red_i[kRThreads];
  __shared__ int stop_s;

  const int unit = blockIdx.x;
  const int b = unit / a.n_kv, kv = unit % a.n_kv;
  const int tid = threadIdx.x;
  if (ra.n_rep != nullptr && tid == 0) ra.n_rep[unit] = 0;
  if (a.mask_kv == nullptr || a.mask_kv[unit] == 0) return;   // nothing routed here
  const int L = a.seq_lens[b];
  const int G = a.group;
  const int B = a.n_bands;
  const int bs = a.split_tokens / 4;                          // tokens per block
  const int Lc = min(L, a.max_blocks * kBlockTokens);
  const int ns = min((Lc + a.split_tokens - 1) / a.split_tokens, a.n_splits);
  const int nb = min((Lc + bs - 1) / bs, 4 * ns);
  if (nb <= 0) return;
  const int64_t R = (int64_t)partial_record_floats(D);
  const float* recs = a.part + ((int64_t)b * a.n_q + (int64_t)kv * G) * a.n_splits * R;
  const bool tierb = a.tierb_delta > 0.0f;
  const int m2 = 2 * a.n_pairs;
  const uint32_t layer_head = ((uint32_t)a.layer << 16) | (uint32_t)kv;

  // ---- queries, band norms, Tier-B factors, bypassed channels ----
  for (int i = tid; i < G * D; i += kRThreads) {
    const int h = i / D, c = i % D;
    const int64_t qi = ((int64_t)b * a.n_q + (int64_t)kv * G + h) * D + c;
    const float x = QT == WC_F32 ? reinterpret_cast<const float*>(a.q)[qi]
                                 : bf16_to_f32(reinterpret_cast<const uint16_t*>(a.q)[qi]);
    q_s[h][c] = x;
    qk_s[h][c] = x;
  }
  for (int c = tid; c < D; c += kRThreads) opos_s[c] = -1;
  __syncthreads();
  if (m2 > 0) {
    const int32_t* pl = a.pairs + (int64_t)kv * a.n_pairs;
    if (tid < m2) opos_s[pair_channel(pl[tid >> 1], tid & 1, D, a.interleaved)] = (int8_t)tid;
    __syncthreads();
    for (int i = tid; i < G * D; i += kRThreads)
      if (opos_s[i % D] >= 0) qk_s[i / D][i % D] = 0.0f;
  }
  for (int i = tid; i < G * B; i += kRThreads) {
    const int h = i / B, bb = i % B;
    float acc = 0.0f;
    for (int k = 0; k < D / B; ++k) {
      const float x = q_s[h][band_channel(bb, k, D, B, a.interleaved)];
      acc = fmaf(x, x, acc);
    }
    qbn_s[h][bb] = sqrtf(acc) * a.sm_scale;
  }
  __syncthreads();
  if (tierb && tid < G) {
    float sq = 0.0f, l1 = 0.0f;
    for (int c = 0; c < D; ++c) {
      sq = fmaf(qk_s[tid][c], qk_s[tid][c], sq);
      l1 += fabsf(qk_s[tid][c]);
    }
    ab_s[tid] = tierb_factor(sq, l1, L, a.tierb_delta, a.sm_scale);
  }

  // ---- merged state of each query head from the split records ----
  if (tid < G) {
    double M = -INFINITY;
    for (int j = 0; j < ns; ++j) M = fmax(M, (double)recs[((int64_t)tid * a.n_splits + j) * R + D]);
    double Ls = 0.0, Ns = 0.0;
    for (int j = 0; j < ns; ++j) {
      const float* rc = recs + ((int64_t)tid * a.n_splits + j) * R;
      const double w = exp((double)rc[D] - M);
      Ls += w * rc[D + 1];
      Ns += w * rc[D + 2];
    }
    M_s[tid] = M;
    L_s[tid] = Ls;
    N_s[tid] = Ns;
  }
  __syncthreads();
  for (int i = tid; i < G * D; i += kRThreads) {
    const int h = i / D, c = i % D;
    double o = 0.0;
    for (int j = 0; j < ns; ++j) {
      const float* rc = recs + ((int64_t)h * a.n_splits + j) * R;
      o += exp((double)rc[D] - M_s[h]) * rc[c];
    }
    O_s[h][c] = o;
  }
  // block totals: sum over the heads of e^{m_j - M} n_{j,w} / L
  for (int i = tid; i < nb; i += kRThreads) {
    const int j = i >> 2, w = i & 3;
    double t = 0.0;
    for (int h = 0; h < G; ++h) {
      const float* rc = recs + ((int64_t)h * a.n_splits + j) * R;
      t += exp((double)rc[D] - M_s[h]) * rc[D + 8 + w] / L_s[h];
    }
    T_s[i] = (float)t;
  }
  __syncthreads();

  // ---- repair order: the budget's largest blocks, ties to the lower index ----
  const int K = min(ra.max_rep, nb);
  for (int k = 0; k < K; ++k) {
    float bv = -2.0f;
    int bi = 0x7fffffff;
    for (int i = tid; i < nb; i += kRThreads)
      if (T_s[i] > bv) {
        bv = T_s[i];
        bi = i;
      }
    red_v[tid] = bv;
    red_i[tid] = bi;
    __syncthreads();
    for (int o = kRThreads / 2; o > 0; o >>= 1) {
      if (tid < o) {
        const float ov = red_v[tid + o];
        const int oi = red_i[tid + o];
        if (ov > red_v[tid] || (ov == red_v[tid] && oi < red_i[tid])) {
          red_v[tid] = ov;
          red_i[tid] = oi;
        }
      }
      __syncthreads();
    }
    if (tid == 0) {
      order_s[k] = red_i[0];
      T_s[red_i[0]] = -1.0f;
    }
    __syncthreads();
  }

  // ---- take the blocks in order until every head passes ----
  int done = -1;
  for (int k = 0; k < K && done < 0; ++k) {
    const int blk = order_s[k];
    const int b0 = blk * bs, b1 = min(b0 + bs, Lc);
    for (int tt = b0; tt < b1; tt += kRTile) {
      // phase 1: compressed and exact logits, bounds (thread: token i, channel quarter)
      {
        const int i = tid >> 2, part = tid & 3;
        const int t = tt + i;
        const bool valid = t < b1;
        int64_t slot = -1;
        if (valid) slot = (int64_t)a.table[(int64_t)b * a.max_blocks + t / kBlockTokens] * kBlockTokens +
                          t % kBlockTokens;
        if (part == 0) slot_s[i] = slot;
        const int c0 = part * CH;
        const int64_t page = valid ? (slot / kBlockTokens) * a.n_kv + kv : 0;
        const int off = valid ? (int)(slot % kBlockTokens) : 0;
        float kq[CH], kx[CH];
        float s = 0.0f;
#pragma unroll
        for (int c = 0; c < CH; ++c) kq[c] = kx[c] = 0.0f;
        if (valid) {
          if (a.kind == WC_KIND_INT8_DITHER) {
            const uint8_t* kp = reinterpret_cast<const uint8_t*>(a.k_data) + (page * kBlockTokens + off) * D + c0;
            s = f16_to_f32(a.k_scale[page * kBlockTokens + off]);
#pragma unroll
            for (int gi = 0; gi < NG; ++gi) {
              const U4 r = dither_block(c0 / 16 + gi, slot, layer_head, a.key0, a.key1);
              const uint32_t rw[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
              for (int w4 = 0; w4 < 4; ++w4) {
                xi_s[i][(c0 + 16 * gi) / 4 + w4] = rw[w4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                  const int c = 16 * gi + 4 * w4 + j;
                  const float code = (float)((int32_t)kp[c] - 128);
                  kq[c] = s * (code - dither_value((rw[w4] >> (8 * j)) & 0xFFu));
                }
              }
            }
            if (m2 > 0) {
#pragma unroll
              for (int c = 0; c < CH; ++c) {
                const int op = opos_s[c0 + c];
                if (op >= 0) kq[c] = f16_to_f32(a.k_outlier[(page * kBlockTokens + off) * m2 + op]);
              }
            }
            if (part == 0) vs_s[i] = f16_to_f32(a.v_scale[page * kBlockTokens + off]);
          } else {   // FP8_RAW
            const uint8_t* kp = reinterpret_cast<const uint8_t*>(a.k_data) + (page * kBlockTokens + off) * D + c0;
#pragma unroll
            for (int c = 0; c < CH; ++c) kq[c] = e4m3_to_f32(kp[c]);
            if (part == 0) vs_s[i] = 1.0f;
          }
          const uint16_t* xp = reinterpret_cast<const uint16_t*>(ra.x_k_data) + (page * kBlockTokens + off) * D + c0;
#pragma unroll
          for (int c = 0; c < CH; ++c) kx[c] = bf16_to_f32(xp[c]);
        } else if (part == 0) {
          vs_s[i] = 0.0f;
        }
        // Tier A: witness bound; Tier B: radius from the key scale (+ rounding of bypassed values)
        float wv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        if (valid && !tierb) {
#pragma unroll
          for (int k4 = 0; k4 < 4; ++k4) {
            const int bb = part + 4 * k4;
            if (bb < B) wv[k4] = f16_to_f32(a.k_witness[(page * kBlockTokens + off) * B + bb]);
          }
        }
        for (int h = 0; h < G; ++h) {
          float dq = 0.0f, dx = 0.0f, cp = 0.0f;
#pragma unroll
          for (int c = 0; c < CH; ++c) {
            dq = fmaf(q_s[h][c0 + c], kq[c], dq);
            dx = fmaf(q_s[h][c0 + c], kx[c], dx);
          }
          if (!tierb) {
#pragma unroll
            for (int k4 = 0; k4 < 4; ++k4) {
              const int bb = part + 4 * k4;
              if (bb < B) cp = fmaf(qbn_s[h][bb], wv[k4], cp);
            }
          } else if (m2 > 0) {
#pragma unroll
            for (int c = 0; c < CH; ++c)
              if (opos_s[c0 + c] >= 0) cp = fmaf(fabsf(q_s[h][c0 + c]), fmaf(fabsf(kq[c]), 0x1p-11f, 0x1p-25f), cp);
            cp *= a.sm_scale;
          }
          dq += __shfl_xor(dq, 1, 4);
          dq += __shfl_xor(dq, 2, 4);
          dx += __shfl_xor(dx, 1, 4);
          dx += __shfl_xor(dx, 2, 4);
          cp += __shfl_xor(cp, 1, 4);
          cp += __shfl_xor(cp, 2, 4);
          if (part == 0) {
            lq_s[h][i] = dq * a.sm_scale;
            lx_s[h][i] = dx * a.sm_scale;
            cb_s[h][i] = tierb ? fmaf(ab_s[h], s, cp) : cp;
          }
        }
      }
      __syncthreads();
      // phase 2: weights and the L, N corrections (thread: head tid / 16, tokens tid % 16 + 16 k)
      {
        const int h = tid >> 4, l16 = tid & 15;
        double dl = 0.0, dn = 0.0;
        if (h < G) {
          for (int k4 = 0; k4 < kRTile / 16; ++k4) {
            const int i = l16 + 16 * k4;
            double wq = 0.0, wx = 0.0;
            if (tt + i < b1) {
              wq = exp((double)lq_s[h][i] - M_s[h]);
              wx = exp((double)lx_s[h][i] - M_s[h]);
              dl += wx - wq;
              dn -= wq * expm1((double)cb_s[h][i]);
            }
            wq_s[h][i] = wq;
            wx_s[h][i] = wx;
          }
        }
        for (int o = 8; o > 0; o >>= 1) {
          dl += __shfl_xor(dl, o, 16);
          dn += __shfl_xor(dn, o, 16);
        }
        if (h < G && l16 == 0) {
          L_s[h] += dl;
          N_s[h] += dn;
        }
      }
      __syncthreads();
      // phase 3: the output correction (thread: channel, head subset)
      {
        const int c3 = tid % D, hs = tid / D;
        for (int i = 0; i < kRTile && tt + i < b1; ++i) {
          const int64_t slot = slot_s[i];
          const int64_t page = (slot / kBlockTokens) * a.n_kv + kv;
          const int off = (int)(slot % kBlockTokens);
          const int64_t vi = page * (kBlockTokens * D) + ((off >> 2) * D + c3) * 4 + (off & 3);
          const uint8_t byte = reinterpret_cast<const uint8_t*>(a.v_data)[vi];
          float vq;
          if (a.kind == WC_KIND_INT8_DITHER) {
            const uint32_t u = (xi_s[i][c3 >> 2] >> (8 * (c3 & 3))) & 0xFFu;
            vq = vs_s[i] * ((float)((int32_t)byte - 128) - dither_value(u));
          } else {
            vq = e4m3_to_f32(byte);
          }
          const float vx = bf16_to_f32(reinterpret_cast<const uint16_t*>(ra.x_v_data)[vi]);
          for (int h = hs; h < G; h += NHS) O_s[h][c3] += wx_s[h][i] * (double)vx - wq_s[h][i] * (double)vq;
        }
      }
      __syncthreads();
    }
    // after the block: does every head pass?
    if (tid == 0) {
      bool pass = true;
      for (int h = 0; h < G; ++h) {
        if (!(L_s[h] > 0.0)) {
          pass = false;
          break;
        }
        const double am1 = N_s[h] / L_s[h];
        const double raw = 0.5 * am1 * (2.0 + am1);
        pass = pass && ((ra.tau >= 1.0f ? raw : fmin(1.0, raw)) <= (double)ra.tau);
      }
      stop_s = pass ? k : -1;
    }
    __syncthreads();
    done = stop_s;
  }

  if (ra.rep_list != nullptr)
    for (int k = tid; k < ra.max_rep; k += kRThreads)
      ra.rep_list[(int64_t)unit * ra.max_rep + k] = k < K ? order_s[k] : -1;
  if (done < 0) {
    if (tid == 0 && ra.n_rep != nullptr) ra.n_rep[unit] = -1;   // left to the whole-head fallback
    return;
  }
  // repaired: new outputs, meter and raw; the KV head leaves the route mask
  for (int i = tid; i < G * D; i += kRThreads) {
    const int h = i / D, c = i % D;
    const float o = (float)(O_s[h][c] / L_s[h]);
    const int64_t oi = ((int64_t)b * a.n_q + (int64_t)kv * G + h) * D + c;
    if (a.out_dtype == WC_F32) reinterpret_cast<float*>(a.out)[oi] = o;
    else reinterpret_cast<uint16_t*>(a.out)[oi] = f32_to_bf16_rne(o);
  }
  if (tid < G) {
    const double am1 = N_s[tid] / L_s[tid];
    const float raw = (float)(0.5 * am1 * (2.0 + am1));
    const int64_t hi = (int64_t)b * a.n_q + (int64_t)kv * G + tid;
    a.meter[hi] = fminf(1.0f, raw);
    if (a.raw != nullptr) a.raw[hi] = raw;
  }
  if (tid == 0) {
    ra.mask_kv_out[unit] = 0;
    if (ra.n_rep != nullptr) ra.n_rep[unit] = done + 1;
  }
}

}  // namespace

hipError_t launch_repair(const RepairArgs& a, hipStream_t st) {
  const dim3 grid(a.d.batch * a.d.n_kv), block(kRThreads);
  if (a.d.head_dim == 64) {
    if (a.d.q_dtype == WC_F32) hipLaunchKernelGGL((repair_kernel<64, WC_F32>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((repair_kernel<64, WC_BF16>), grid, block, 0, st, a);
  } else {
    if (a.d.q_dtype == WC_F32) hipLaunchKernelGGL((repair_kernel<128, WC_F32>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((repair_kernel<128, WC_BF16>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

int repair_max_blocks() { return kRMaxBlocks; }

}  // namespace wc
