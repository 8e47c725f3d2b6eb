// Block-granular repair of routed KV heads (Sec. 6.3, block-level paging).
//
// The certificate is block decomposable: A - 1 = sum_t ptilde_t (e^{c_t} - 1) splits
// into per-block shares, and a block taken from the exact store contributes exact
// logits and values with bound 0.  Blocks are taken in decreasing order of their
// shares until every query head of the KV head passes tau.  The walk is
// sequential only in its stop rule; the block corrections are independent, so
// the work runs in three kinds of launches:
//   rank   one workgroup per (sequence, KV head): the merged state of each query
//          head (max M, weight sum L, meter numerator N) in float64 from the split
//          records of the metered decode that routed it; the block totals (sum over
//          the G heads of the block's share; a block is a fixed run of 256 tokens,
//          its share the sum of the block segments the decode recorded); the repair
//          order (largest first, ties to the lower block) up to the budget; and a
//          predicted block count, the
//          first prefix after which every head passes when only N moves (the
//          exact logits usually move L very little);
//   block  one workgroup per (candidate, 64-token tile, routed KV head) of a round:
//          compressed and exact logits, bounds and values of the tile, and the
//          corrections that move L, N and the unnormalized output O from the
//          compressed to the exact terms,
//            dL = sum (e^{l_t - M} - e^{lt_t - M}),  dN = -sum e^{lt_t - M} (e^{c_t} - 1),
//            dO = sum (e^{l_t - M} v_t - e^{lt_t - M} vhat_t)   (float64);
//   scan   one workgroup per KV head: adds the round's corrections in order, stops
//          at the first block after which every head passes, and for a repaired
//          head writes its meter and raw and clears its route mask;
//   final  one workgroup per (repaired KV head, query head): the output, the
//          records' merged output plus the taken blocks' corrections (fixed
//          summation order) over the repaired weight sum.
// Round 0 covers the predicted count plus one block, round 1 the rest of the
// budget (its launches exit at once where round 0 finished).  A KV head the
// budget cannot repair keeps its mask (whole-head fallback).  Logits and bounds
// are formed in fp32 as in the vector decode path.
#include <float.h>

#include "wc_device.h"
#include "wc_launch.h"

namespace wc {

namespace {

constexpr int kRThreads = 256;
constexpr int kRTile = 64;        // tokens per block-kernel workgroup
constexpr int kRGMax = 16;
constexpr int kRMaxBlocks = 4096;
constexpr int kRMaxRep = 64;

enum : int32_t { kIdle = 0, kActive = 1, kRepaired = 2, kExhausted = 3 };

// Per-(sequence, KV head) header at the start of its workspace slice.
struct RepHeader {
  int32_t status, K, round0_end, n_taken, n_cand;
  int32_t order[kRMaxRep];
  double M[kRGMax], L[kRGMax], N[kRGMax];
};
static_assert(sizeof(RepHeader) <= kRepHeaderBytes, "repair header");

__device__ __forceinline__ RepHeader* header_of(const RepairArgs& ra, int unit) {
  return reinterpret_cast<RepHeader*>(static_cast<char*>(ra.rws) + (size_t)unit * ra.unit_bytes);
}
// Corrections of candidate j, tile k: G records of D + 2 doubles (dO[D], dL, dN).
__device__ __forceinline__ double* corr_of(const RepairArgs& ra, int unit, int j, int k) {
  const size_t rec = (size_t)ra.d.group * (ra.d.head_dim + 2);
  return reinterpret_cast<double*>(static_cast<char*>(ra.rws) + (size_t)unit * ra.unit_bytes +
                                   kRepHeaderBytes) + ((size_t)j * ra.tiles + k) * rec;
}

__device__ __forceinline__ bool head_passes(double L, double N, float tau) {
  if (!(L > 0.0)) return false;
  const double am1 = N / L;
  const double raw = 0.5 * am1 * (2.0 + am1);
  return (tau >= 1.0f ? raw : fmin(1.0, raw)) <= (double)tau;
}

struct UnitGeom {
  int b, kv, L, Lc, ns, nb;
};
__device__ __forceinline__ UnitGeom unit_geom(const DecodeArgs& a, int unit) {
  UnitGeom u;
  u.b = unit / a.n_kv;
  u.kv = unit % a.n_kv;
  u.L = a.seq_lens[u.b];
  u.Lc = min(u.L, a.max_blocks * kBlockTokens);
  u.ns = min((u.Lc + a.split_tokens - 1) / a.split_tokens, a.n_splits);
  u.nb = (u.Lc + kRepairBlockTokens - 1) / kRepairBlockTokens;
  return u;
}

// Tokens [b0, b1) of block i: the fixed 256-token run (Sec. 6.3).
__device__ __forceinline__ void block_range(int i, int Lc, int& b0, int& b1) {
  b0 = min(i * kRepairBlockTokens, Lc);
  b1 = min(b0 + kRepairBlockTokens, Lc);
}

// Share of block i for query head h (rows of G heads): the sum of the block's
// segments e^{m - M_h} n over the splits that overlap it, in split and slot order.
__device__ __forceinline__ double block_share(const DecodeArgs& a, const float4* sh_unit, int i, int h,
                                              int ns, double M) {
  const int j0 = i * kRepairBlockTokens / a.split_tokens;
  const int j1 = min((i * kRepairBlockTokens + kRepairBlockTokens - 1) / a.split_tokens, ns - 1);
  double t = 0.0;
  for (int j = j0; j <= j1; ++j) {
    const float4* e = sh_unit + ((int64_t)h * a.n_splits + j) * a.share_slots;
    for (int sl = 0; sl < a.share_slots; ++sl) {
      const float4 x = e[sl];
      const int first = __builtin_bit_cast(int, x.z), pages = __builtin_bit_cast(int, x.w);
      if (pages > 0 && first * kBlockTokens / kRepairBlockTokens == i) t += exp((double)x.y - M) * (double)x.x;
    }
  }
  return t;
}

// ---------------------------------------------------------------------------
// rank: merged state, block order, predicted count
template <int D>
__global__ __launch_bounds__(kRThreads) void repair_rank_kernel(RepairArgs ra) {
  const DecodeArgs& a = ra.d;
  __shared__ double T_s[kRMaxBlocks];
  __shared__ float sh_s[kRGMax][kRMaxRep];
  __shared__ uint64_t pass_s[kRGMax];
  __shared__ int order_s[kRMaxRep];
  __shared__ double M_s[kRGMax], L_s[kRGMax];
  __shared__ int n_cand_s;

  const int unit = blockIdx.x;
  const int tid = threadIdx.x;
  RepHeader* hd = header_of(ra, unit);
  if (tid == 0) {
    hd->status = kIdle;
    if (ra.n_rep != nullptr) ra.n_rep[unit] = 0;
  }
  if (a.mask_kv[unit] == 0) return;   // nothing routed here
  const UnitGeom u = unit_geom(a, unit);
  if (u.nb <= 0) return;
  const int G = a.group;
  const int64_t R = (int64_t)partial_record_floats(D);
  const float* recs = a.part + ((int64_t)u.b * a.n_q + (int64_t)u.kv * G) * a.n_splits * R;

  // merged state of each query head: one wave per head, lanes over the splits
  const int wave = tid >> 6, lane = tid & 63;
  for (int h = wave; h < G; h += kRThreads / 64) {
    const float* rh = recs + (int64_t)h * a.n_splits * R;
    double M = -INFINITY;
    for (int j = lane; j < u.ns; j += 64) M = fmax(M, (double)rh[j * R + D]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) M = fmax(M, __shfl_xor(M, o, 64));
    double Ls = 0.0, Ns = 0.0;
    for (int j = lane; j < u.ns; j += 64) {
      const double w = exp((double)rh[j * R + D] - M);
      Ls += w * rh[j * R + D + 1];
      Ns += w * rh[j * R + D + 2];
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      Ls += __shfl_xor(Ls, o, 64);
      Ns += __shfl_xor(Ns, o, 64);
    }
    if (lane == 0) {
      M_s[h] = M;
      L_s[h] = Ls;
      hd->M[h] = M;
      hd->L[h] = Ls;
      hd->N[h] = Ns;
    }
  }
  __syncthreads();
  // block totals: sum over the heads of the block's share / L; a block whose
  // positions all lie in pages marked as repaired is no candidate (total -1)
  const float4* sh_unit = a.shares + ((int64_t)u.b * a.n_q + (int64_t)u.kv * G) * a.n_splits * a.share_slots;
  if (tid == 0) n_cand_s = 0;
  __syncthreads();
  for (int i = tid; i < u.nb; i += kRThreads) {
    bool done = a.repaired != nullptr;
    if (done) {
      int b0, b1;
      block_range(i, u.Lc, b0, b1);
      for (int pg = b0 / kBlockTokens; done && pg <= (b1 - 1) / kBlockTokens; ++pg) {
        const int32_t e = a.table[(int64_t)u.b * a.max_blocks + pg];
        done = (int64_t)(uint32_t)e < a.num_blocks && a.repaired[(int64_t)e * a.n_kv + u.kv] != 0;
      }
    }
    double t = -1.0;
    if (!done) {
      t = 0.0;
      for (int h = 0; h < G; ++h) t += block_share(a, sh_unit, i, h, u.ns, M_s[h]) / L_s[h];
      atomicAdd(&n_cand_s, 1);
    }
    T_s[i] = t;
  }
  __syncthreads();
  const int n_cand = n_cand_s;
  // repair order: the budget's largest blocks, ties to the lower index.  Up to
  // 1024 blocks every block counts the blocks ahead of it; beyond, one wave takes
  // an arg-max per step.
  const int K = min(ra.max_rep, n_cand);
  if (u.nb <= 1024) {
    for (int i = tid; i < u.nb; i += kRThreads) {
      const double ti = T_s[i];
      int rank = 0;
      for (int j = 0; j < u.nb; ++j) {
        const double tj = T_s[j];
        rank += (tj > ti || (tj == ti && j < i)) ? 1 : 0;
      }
      if (rank < K) order_s[rank] = i;
    }
  } else if (tid < 64) {
    for (int k = 0; k < K; ++k) {
      double bv = -2.0;
      int bi = 0x7fffffff;
      for (int i = tid; i < u.nb; i += 64)
        if (T_s[i] > bv) {
          bv = T_s[i];
          bi = i;
        }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const double ov = __shfl_xor(bv, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (ov > bv || (ov == bv && oi < bi)) {
          bv = ov;
          bi = oi;
        }
      }
      if (tid == 0) {
        order_s[k] = bi;
        T_s[bi] = -1.0;
      }
      __builtin_amdgcn_wave_barrier();   // (one wave: LDS accesses stay in program order)
    }
  }
  __syncthreads();
  // predicted count: per head, N minus the taken shares (L held fixed)
  for (int i = tid; i < G * K; i += kRThreads) {
    const int h = i / K, k = i % K;
    sh_s[h][k] = (float)block_share(a, sh_unit, order_s[k], h, u.ns, M_s[h]);
  }
  __syncthreads();
  if (tid < G) {
    double N = hd->N[tid];
    uint64_t bits = 0;
    for (int k = 0; k < K; ++k) {
      N -= sh_s[tid][k];
      if (head_passes(L_s[tid], N, ra.tau)) bits |= 1ull << k;
    }
    pass_s[tid] = bits;
  }
  __syncthreads();
  if (tid == 0) {
    uint64_t all = K == 64 ? ~0ull : ((1ull << K) - 1);
    for (int h = 0; h < G; ++h) all &= pass_s[h];
    const int pred = all ? __builtin_ctzll(all) + 1 : K;
    hd->K = K;
    hd->n_cand = n_cand;
    hd->n_taken = 0;
    hd->round0_end = min(K, ra.round0_cap > 0 ? ra.round0_cap : pred + 1);
    hd->status = kActive;
  }
  for (int k = tid; k < kRMaxRep; k += kRThreads) hd->order[k] = k < K ? order_s[k] : -1;
  if (ra.rep_list != nullptr)
    for (int k = tid; k < ra.max_rep; k += kRThreads)
      ra.rep_list[(int64_t)unit * ra.max_rep + k] = k < K ? order_s[k] : -1;
}

// ---------------------------------------------------------------------------
// block: corrections of one 64-token tile of one candidate block
template <int D, int QT, int GM>
__global__ __launch_bounds__(kRThreads, 4) void repair_block_kernel(RepairArgs ra, int round) {
  const DecodeArgs& a = ra.d;
  constexpr int CH = D / 4;
  constexpr int NG = CH / 16;
  constexpr int NSUB = kRThreads / D;   // channel-thread subsets in the output pass

  __shared__ float q_s[GM][D];
  __shared__ float qbn_s[GM][16];
  __shared__ float ab_s[GM];
  __shared__ int8_t opos_s[D];           // stored-value position of a bypassed channel, else -1
  __shared__ double wq_s[GM][kRTile], wx_s[GM][kRTile];
  __shared__ uint32_t xi_s[kRTile][D / 16 * 4];
  __shared__ float vs_s[kRTile][4];      // value scale of each token and 32-channel group
  __shared__ int64_t slot_s[kRTile];
  __shared__ double dl_s[GM], dn_s[GM];
  __shared__ uint16_t ko_s[kRTile][32];  // stored fp16 values of the bypassed pairs (2m <= 32)
  __shared__ float qg_s[GM][8];          // group scales, Tier B: ||q_g||^2 (0..3), ||q_g||_1 (4..7)
  // logits and bounds of phases 1-2, then the output reduction of phase 3
  constexpr int kLogitBytes = 3 * GM * kRTile * 4;
  constexpr int kRedBytes = (NSUB > 1 ? NSUB - 1 : 1) * GM * D * 8;
  __shared__ __align__(16) char un_s[kLogitBytes > kRedBytes ? kLogitBytes : kRedBytes];
  float (*lq_s)[kRTile] = reinterpret_cast<float (*)[kRTile]>(un_s);
  float (*lx_s)[kRTile] = reinterpret_cast<float (*)[kRTile]>(un_s + GM * kRTile * 4);
  float (*cb_s)[kRTile] = reinterpret_cast<float (*)[kRTile]>(un_s + 2 * GM * kRTile * 4);
  double (*red_s)[GM][D] = reinterpret_cast<double (*)[GM][D]>(un_s);

  const int unit = blockIdx.y;
  const RepHeader* hd = header_of(ra, unit);
  if (hd->status != kActive) return;
  const int j = blockIdx.x / ra.tiles, tile = blockIdx.x % ra.tiles;
  const int j_lo = round == 0 ? 0 : hd->round0_end;
  const int j_hi = round == 0 ? hd->round0_end : hd->K;
  if (j < j_lo || j >= j_hi) return;
  const UnitGeom u = unit_geom(a, unit);
  const int b = u.b, kv = u.kv;
  const int tid = threadIdx.x;
  const int G = a.group;
  const int B = a.n_bands;
  const int blk = hd->order[j];
  int b0, b1;
  block_range(blk, u.Lc, b0, b1);
  const int t_lo = b0 + tile * kRTile;
  const int t_hi = min(t_lo + kRTile, b1);
  const int nv = max(t_hi - t_lo, 0);     // tokens of this tile
  const bool tierb = a.tierb_delta > 0.0f;
  const int m2 = 2 * a.n_pairs;
  const uint32_t layer_head = ((uint32_t)a.layer << 16) | (uint32_t)kv;
  double* out_rec = corr_of(ra, unit, j, tile);
  const int rec = D + 2;
  if (nv == 0) {
    for (int i = tid; i < G * rec; i += kRThreads) out_rec[i] = 0.0;
    return;
  }

  // ---- queries (bypassed channels zeroed for the compressed key), band norms,
  // Tier-B factors ----
  for (int c = tid; c < D; c += kRThreads) opos_s[c] = -1;
  for (int i = tid; i < G * D; i += kRThreads) {
    const int h = i / D, c = i % D;
    const int64_t qi = ((int64_t)b * a.n_q + (int64_t)kv * G + h) * D + c;
    q_s[h][c] = QT == WC_F32 ? reinterpret_cast<const float*>(a.q)[qi]
                             : bf16_to_f32(reinterpret_cast<const uint16_t*>(a.q)[qi]);
  }
  __syncthreads();
  if (m2 > 0 && tid < m2) {
    const int32_t* pl = a.pairs + (int64_t)kv * a.n_pairs;
    opos_s[pair_channel(pl[tid >> 1], tid & 1, D, a.interleaved)] = (int8_t)tid;
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
  const bool grouped = a.group_scales != 0;
  if (tierb && tid < G) {
    float sq = 0.0f, l1 = 0.0f;
    for (int c = 0; c < D; ++c) {
      const float x = opos_s[c] >= 0 ? 0.0f : q_s[tid][c];
      sq = fmaf(x, x, sq);
      l1 += fabsf(x);
      if (grouped && (c & 31) == 31) {   // per-group norms of the quantized channels
        qg_s[tid][c >> 5] = sq;
        qg_s[tid][4 + (c >> 5)] = l1;
        sq = l1 = 0.0f;
      }
    }
    if (!grouped) ab_s[tid] = tierb_factor(sq, l1, u.L, a.tierb_delta, a.sm_scale);
  }
  const float rt = tierb && grouped ? sqrtf(2.0f * logf(2.0f * (float)u.L / a.tierb_delta) / 12.0f) : 0.0f;
  __syncthreads();

  // ---- phase 1: compressed and exact logits, bounds (thread: token i, channel quarter) ----
  {
    const int i = tid >> 2, part = tid & 3;
    const int t = t_lo + i;
    // a table entry outside the caches leaves the token out (no access outside them)
    // (a token of a page marked as repaired is exact in the decode's records already:
    // no correction)
    const int32_t e = i < nv ? a.table[(int64_t)b * a.max_blocks + t / kBlockTokens] : -1;
    const bool valid = i < nv && (int64_t)(uint32_t)e < a.num_blocks &&
                       !(a.repaired != nullptr && a.repaired[(int64_t)e * a.n_kv + kv] != 0);
    int64_t slot = -1;
    if (valid) slot = (int64_t)e * kBlockTokens + t % kBlockTokens;
    if (part == 0) slot_s[i] = slot;
    const int c0 = part * CH;
    const int64_t row = valid ? ((slot / kBlockTokens) * a.n_kv + kv) * kBlockTokens + slot % kBlockTokens : 0;
    if (m2 > 0) {   // the token's bypassed values to LDS (quarter of the row per thread)
      for (int e = part; e < m2; e += 4) ko_s[i][e] = valid ? a.k_outlier[row * m2 + e] : (uint16_t)0;
      __syncthreads();
    }
    // per head: q . khat, q . k and the Tier-B rounding term, channel by channel
    float dq[GM], dx[GM], cq[GM];
#pragma unroll
    for (int h = 0; h < GM; ++h) dq[h] = dx[h] = cq[h] = 0.0f;
    float ksg[4] = {0.0f, 0.0f, 0.0f, 0.0f};   // key step of each 32-channel group of the token
    if (valid) {
      uint32_t kb[CH / 4];
      const int64_t kpage = row / kBlockTokens;   // (block, KV head) page
      const int koff = (int)(row % kBlockTokens);
      const uint8_t* kpg = reinterpret_cast<const uint8_t*>(a.k_data) + kpage * (kBlockTokens * D);
#pragma unroll
      for (int w = 0; w < CH / 16; ++w) {
        const uint4 x = *reinterpret_cast<const uint4*>(kpg + kpage_off(koff, c0 + 16 * w, D, 1));
        kb[4 * w] = x.x; kb[4 * w + 1] = x.y; kb[4 * w + 2] = x.z; kb[4 * w + 3] = x.w;
      }
      uint32_t xb[CH / 2];
      const uint8_t* xpg = reinterpret_cast<const uint8_t*>(ra.x_k_data) + kpage * (kBlockTokens * D * 2);
#pragma unroll
      for (int w = 0; w < CH / 8; ++w) {
        const uint4 x = *reinterpret_cast<const uint4*>(xpg + kpage_off(koff, c0 + 8 * w, D, 2));
        xb[4 * w] = x.x; xb[4 * w + 1] = x.y; xb[4 * w + 2] = x.z; xb[4 * w + 3] = x.w;
      }
      const bool int8 = a.kind == WC_KIND_INT8_DITHER;
      if (int8)
        for (int gg = 0; gg < D / 32; ++gg) ksg[gg] = scale_of(a.k_scale, row, 32 * gg, D, grouped);
      if (part == 0)
        for (int gg = 0; gg < D / 32; ++gg) vs_s[i][gg] = int8 ? scale_of(a.v_scale, row, 32 * gg, D, grouped) : 1.0f;
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
        uint32_t rw[4] = {0, 0, 0, 0};
        if (int8) {
          const U4 r = dither_block(c0 / 16 + gi, slot, layer_head, a.key0, a.key1);
          rw[0] = r.x; rw[1] = r.y; rw[2] = r.z; rw[3] = r.w;
#pragma unroll
          for (int w4 = 0; w4 < 4; ++w4) xi_s[i][(c0 + 16 * gi) / 4 + w4] = rw[w4];
        }
#pragma unroll
        for (int w4 = 0; w4 < 4; ++w4) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int c = 16 * gi + 4 * w4 + e;
            const uint32_t byte = (kb[c >> 2] >> (8 * (c & 3))) & 0xFFu;
            const float sg = ksg[(c0 + c) >> 5];
            float kq = int8 ? sg * ((float)((int32_t)byte - 128) - dither_value((rw[w4] >> (8 * e)) & 0xFFu))
                            : e4m3_to_f32(byte);
            const int op = m2 > 0 ? opos_s[c0 + c] : -1;
            if (op >= 0) kq = f16_to_f32(ko_s[i][op]);   // bypassed pair: stored fp16
            const float kx = bf16_to_f32((uint16_t)(xb[c >> 1] >> (16 * (c & 1))));
#pragma unroll
            for (int h = 0; h < GM; ++h) {
              if (h < G) {
                const float qc = q_s[h][c0 + c];
                dq[h] = fmaf(qc, kq, dq[h]);
                dx[h] = fmaf(qc, kx, dx[h]);
                if (tierb && op >= 0) cq[h] = fmaf(fabsf(qc), fmaf(fabsf(kq), 0x1p-11f, 0x1p-25f), cq[h]);
              }
            }
          }
        }
      }
    } else if (part == 0) {
      for (int gg = 0; gg < 4; ++gg) vs_s[i][gg] = 0.0f;
    }
    // Tier A: witness bound; Tier B: radius from the key scale (+ rounding of bypassed values)
    float wv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (valid && !tierb) {
#pragma unroll
      for (int k4 = 0; k4 < 4; ++k4) {
        const int bb = part + 4 * k4;
        if (bb < B) wv[k4] = f16_to_f32(a.k_witness[row * B + bb]);
      }
    }
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      if (h >= G) continue;
      float cp = 0.0f;
      if (!tierb) {
#pragma unroll
        for (int k4 = 0; k4 < 4; ++k4) {
          const int bb = part + 4 * k4;
          if (bb < B) cp = fmaf(qbn_s[h][bb], wv[k4], cp);
        }
      } else if (m2 > 0) {
        cp = cq[h] * a.sm_scale;
      }
      float vq = dq[h], vx = dx[h];
      vq += __shfl_xor(vq, 1, 4);
      vq += __shfl_xor(vq, 2, 4);
      vx += __shfl_xor(vx, 1, 4);
      vx += __shfl_xor(vx, 2, 4);
      cp += __shfl_xor(cp, 1, 4);
      cp += __shfl_xor(cp, 2, 4);
      if (part == 0) {
        lq_s[h][i] = vq * a.sm_scale;
        lx_s[h][i] = vx * a.sm_scale;
        if (tierb && grouped) {
          float s2 = 0.0f, s1 = 0.0f;
          for (int gg = 0; gg < D / 32; ++gg) {
            const float sg = ksg[gg];
            s2 = fmaf(sg * sg, qg_s[h][gg], s2);
            s1 = fmaf(sg, qg_s[h][4 + gg], s1);
          }
          cb_s[h][i] = a.sm_scale * (fmaf(rt, sqrtf(s2), s1 * (1.0f / 256.0f))) + cp;
        } else {
          cb_s[h][i] = tierb ? fmaf(ab_s[h], ksg[0], cp) : cp;
        }
      }
    }
  }
  __syncthreads();

  // ---- phase 2: weights and the L, N corrections (thread: head tid / 16, tokens tid % 16 + 16 k) ----
  {
    const int h = tid >> 4, l16 = tid & 15;
    double dl = 0.0, dn = 0.0;
    if (h < G) {
      const double M = hd->M[h];
#pragma unroll
      for (int k4 = 0; k4 < kRTile / 16; ++k4) {
        const int i = l16 + 16 * k4;
        double wq = 0.0, wx = 0.0;
        if (i < nv) {
          wq = exp((double)lq_s[h][i] - M);
          wx = exp((double)lx_s[h][i] - M);
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
      dl_s[h] = dl;
      dn_s[h] = dn;
    }
  }
  __syncthreads();

  // ---- phase 3: the output correction (thread: channel c, token quads sub, sub + NSUB, ..) ----
  {
    const int c = tid % D, sub = tid / D;
    double acc[GM];
#pragma unroll
    for (int h = 0; h < GM; ++h) acc[h] = 0.0;
    constexpr int NQ = kRTile / 4 / NSUB;   // quads per thread
    uint32_t vb[NQ];
    uint2 xb[NQ];
#pragma unroll
    for (int qq = 0; qq < NQ; ++qq) {
      const int i0 = 4 * (sub + NSUB * qq);
      vb[qq] = 0;
      xb[qq] = make_uint2(0, 0);
      const int64_t slot = i0 < nv ? slot_s[i0] : -1;
      if (slot >= 0) {   // (a table entry outside the caches left the quad out)
        const int64_t page = (slot / kBlockTokens) * a.n_kv + kv;
        const int t = (int)(slot % kBlockTokens);   // first token of the quad
        vb[qq] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint8_t*>(a.v_data) +
                                                    page * (kBlockTokens * D) + vpage_off(t, c, D, 1));
        xb[qq] = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint8_t*>(ra.x_v_data) +
                                                 page * (kBlockTokens * D * 2) + vpage_off(t, c, D, 2));
      }
    }
#pragma unroll
    for (int qq = 0; qq < NQ; ++qq) {
      const int i0 = 4 * (sub + NSUB * qq);
      if (i0 >= nv) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = i0 + e;
        if (i >= nv) break;
        const uint32_t byte = (vb[qq] >> (8 * e)) & 0xFFu;
        float vq;
        if (a.kind == WC_KIND_INT8_DITHER) {
          const uint32_t xw = xi_s[i][c >> 2];
          vq = vs_s[i][c >> 5] * ((float)((int32_t)byte - 128) - dither_value((xw >> (8 * (c & 3))) & 0xFFu));
        } else {
          vq = e4m3_to_f32(byte);
        }
        const uint32_t xw2 = e < 2 ? xb[qq].x : xb[qq].y;
        const float vx = bf16_to_f32((uint16_t)(xw2 >> (16 * (e & 1))));
#pragma unroll
        for (int h = 0; h < GM; ++h)
          if (h < G) acc[h] += wx_s[h][i] * (double)vx - wq_s[h][i] * (double)vq;
      }
    }
    __syncthreads();   // the logit arrays are dead: their LDS takes the reduction
    if (sub > 0) {
#pragma unroll
      for (int h = 0; h < GM; ++h)
        if (h < G) red_s[sub - 1][h][c] = acc[h];
    }
    __syncthreads();
    if (sub == 0) {
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        if (h < G) {
          double o = acc[h];
          for (int s2 = 1; s2 < NSUB; ++s2) o += red_s[s2 - 1][h][c];
          out_rec[h * rec + c] = o;
        }
      }
    }
  }
  if (tid < G) {
    out_rec[tid * rec + D] = dl_s[tid];
    out_rec[tid * rec + D + 1] = dn_s[tid];
  }
}

// ---------------------------------------------------------------------------
// scan: add the round's corrections in order, stop at the first passing prefix
template <int D>
__global__ __launch_bounds__(kRThreads) void repair_scan_kernel(RepairArgs ra, int round) {
  const DecodeArgs& a = ra.d;
  __shared__ double dL_s[kRMaxRep][kRGMax], dN_s[kRMaxRep][kRGMax];
  __shared__ uint64_t pass_s[kRGMax];
  __shared__ int done_s;

  const int unit = blockIdx.x;
  const int tid = threadIdx.x;
  RepHeader* hd = header_of(ra, unit);
  if (hd->status != kActive) return;
  const int G = a.group;
  const int j_lo = round == 0 ? 0 : hd->round0_end;
  const int j_hi = round == 0 ? hd->round0_end : hd->K;
  const bool last = round == 1;
  const int n = j_hi - j_lo;
  const int rec = D + 2;

  // per (candidate, head): the tiles' dL, dN added in tile order
  for (int i = tid; i < n * G; i += kRThreads) {
    const int jj = i / G, h = i % G;
    double dl = 0.0, dn = 0.0;
    for (int k0 = 0; k0 < ra.tiles; k0 += 4) {
      double l4[4], n4[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double* cr = corr_of(ra, unit, j_lo + jj, min(k0 + e, ra.tiles - 1)) + h * rec;
        l4[e] = k0 + e < ra.tiles ? cr[D] : 0.0;
        n4[e] = k0 + e < ra.tiles ? cr[D + 1] : 0.0;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        dl += l4[e];
        dn += n4[e];
      }
    }
    dL_s[jj][h] = dl;
    dN_s[jj][h] = dn;
  }
  __syncthreads();
  // once every candidate block is taken no compressed token is left: the
  // numerator is 0 by definition (the corrections would leave the rounding of
  // the records' fp32 sums)
  const int nb_all = hd->n_cand;
  if (tid < G) {
    double L = hd->L[tid], N = hd->N[tid];
    uint64_t bits = 0;
    for (int jj = 0; jj < n; ++jj) {
      L += dL_s[jj][tid];
      N += dN_s[jj][tid];
      if (head_passes(L, j_lo + jj + 1 >= nb_all ? 0.0 : N, ra.tau)) bits |= 1ull << jj;
    }
    pass_s[tid] = bits;
  }
  __syncthreads();
  if (tid == 0) {
    uint64_t all = n >= 64 ? ~0ull : ((1ull << n) - 1);
    for (int h = 0; h < G; ++h) all &= pass_s[h];
    done_s = all ? j_lo + __builtin_ctzll(all) : -1;   // last candidate taken
  }
  __syncthreads();
  const int done = done_s;
  if (done < 0) {
    if (tid < G) {   // carry the state into the next round
      double L = hd->L[tid], N = hd->N[tid];
      for (int jj = 0; jj < n; ++jj) {
        L += dL_s[jj][tid];
        N += dN_s[jj][tid];
      }
      hd->L[tid] = L;
      hd->N[tid] = N;
    }
    __syncthreads();
    if (tid == 0 && last) {
      hd->status = kExhausted;
      if (ra.n_rep != nullptr) ra.n_rep[unit] = -1;   // left to the whole-head fallback
    }
    return;
  }

  // repaired after candidate `done`: state, meter and raw; the outputs follow in
  // the final kernel
  if (tid < G) {
    double L = hd->L[tid], N = hd->N[tid];
    for (int jj = 0; jj <= done - j_lo; ++jj) {
      L += dL_s[jj][tid];
      N += dN_s[jj][tid];
    }
    if (done + 1 >= nb_all) N = 0.0;
    hd->L[tid] = L;
    hd->N[tid] = N;
    const double am1 = N / L;
    const float raw = (float)(0.5 * am1 * (2.0 + am1));
    const UnitGeom u = unit_geom(a, unit);
    const int64_t hi = (int64_t)u.b * a.n_q + (int64_t)u.kv * G + tid;
    a.meter[hi] = fminf(1.0f, raw);
    if (a.raw != nullptr) a.raw[hi] = raw;
  }
  __syncthreads();
  if (tid == 0) {
    hd->n_taken = done + 1;
    hd->status = kRepaired;
    ra.mask_kv_out[unit] = 0;
    if (ra.n_rep != nullptr) ra.n_rep[unit] = done + 1;
  }
}

// ---------------------------------------------------------------------------
// final: outputs of a repaired KV head, one workgroup per (KV head, query head):
// the merged unnormalized output from the split records plus the corrections of
// the taken blocks, summed in a fixed order, over the repaired weight sum
template <int D>
__global__ __launch_bounds__(kRThreads) void repair_final_kernel(RepairArgs ra) {
  const DecodeArgs& a = ra.d;
  constexpr int CW = 32;                  // channels per workgroup
  constexpr int NSUB = kRThreads / CW;    // threads per channel
  __shared__ double red_s[NSUB][CW];
  __shared__ double w_s[kRThreads];
  const int unit = blockIdx.x, h = blockIdx.y;
  const RepHeader* hd = header_of(ra, unit);
  if (hd->status != kRepaired || h >= a.group) return;
  const int G = a.group;
  const int tid = threadIdx.x;
  const int cl = tid % CW, sub = tid / CW;
  const int c = blockIdx.z * CW + cl;
  const int rec = D + 2;
  const UnitGeom u = unit_geom(a, unit);
  const int P = hd->n_taken * ra.tiles;      // (candidate, tile) records, candidate-major
  const double* base = corr_of(ra, unit, 0, 0) + h * rec + c;
  const size_t stride = (size_t)G * rec;
  double o = 0.0;
  constexpr int U = 8;
  for (int p0 = sub * U; p0 < P; p0 += NSUB * U) {
    double v[U];
#pragma unroll
    for (int e = 0; e < U; ++e) v[e] = p0 + e < P ? base[(size_t)(p0 + e) * stride] : 0.0;
#pragma unroll
    for (int e = 0; e < U; ++e) o += v[e];
  }
  // the merged output of the split records: split weights once per workgroup
  // (chunks of kRThreads splits), each thread's share of the splits
  const int64_t R = (int64_t)partial_record_floats(D);
  const float* recs = a.part + (((int64_t)u.b * a.n_q + (int64_t)u.kv * G + h) * a.n_splits) * R;
  const double M = hd->M[h];
  for (int j0 = 0; j0 < u.ns; j0 += kRThreads) {
    __syncthreads();
    if (j0 + tid < u.ns) w_s[tid] = exp((double)recs[(j0 + tid) * R + D] - M);
    __syncthreads();
    const int nj = min(kRThreads, u.ns - j0);
    for (int jb = sub * U; jb < nj; jb += NSUB * U) {
      float v[U];
#pragma unroll
      for (int e = 0; e < U; ++e) v[e] = jb + e < nj ? recs[(j0 + jb + e) * R + c] : 0.0f;
#pragma unroll
      for (int e = 0; e < U; ++e)
        if (jb + e < nj) o += w_s[jb + e] * (double)v[e];
    }
  }
  red_s[sub][cl] = o;
  __syncthreads();
  if (sub == 0) {
    double t = red_s[0][cl];
    for (int s2 = 1; s2 < NSUB; ++s2) t += red_s[s2][cl];
    const float of = (float)(t / hd->L[h]);
    const int64_t oi = ((int64_t)u.b * a.n_q + (int64_t)u.kv * G + h) * D + c;
    if (a.out_dtype == WC_F32) reinterpret_cast<float*>(a.out)[oi] = of;
    else reinterpret_cast<uint16_t*>(a.out)[oi] = f32_to_bf16_rne(of);
  }
}

// ---------------------------------------------------------------------------
// write-back (persistent repair): one workgroup per (sequence, KV head); thread
// (page, token) of the pages to mark zeroes the token's witness, token 0 marks
// the page
__global__ __launch_bounds__(kRThreads) void repair_write_back_kernel(WriteBackArgs w) {
  const int unit = blockIdx.x;
  const int b = unit / w.n_kv, kv = unit % w.n_kv;
  const bool whole = w.whole_kv != nullptr && w.whole_kv[unit] != 0;
  const int n = w.n_rep != nullptr ? min(w.n_rep[unit], w.max_rep) : 0;
  if (!whole && n <= 0) return;
  const int Lc = min(w.seq_lens[b], w.max_blocks * kBlockTokens);
  const int npages = (Lc + kBlockTokens - 1) / kBlockTokens;
  constexpr int kPPB = kRepairBlockTokens / kBlockTokens;   // pages per repair block
  const int total = whole ? npages : n * kPPB;
  for (int idx = threadIdx.x; idx < total * kBlockTokens; idx += kRThreads) {
    const int pk = idx / kBlockTokens, tok = idx % kBlockTokens;
    int pg = pk;
    if (!whole) {
      const int blk = w.list[(int64_t)unit * w.max_rep + pk / kPPB];
      if (blk < 0 || blk >= kRMaxBlocks) continue;
      pg = blk * kPPB + pk % kPPB;
    }
    if (pg >= npages) continue;
    const int32_t e = w.table[(int64_t)b * w.max_blocks + pg];
    if ((int64_t)(uint32_t)e >= w.num_blocks) continue;
    const int64_t page = (int64_t)e * w.n_kv + kv;
    if (w.k_witness != nullptr)
      for (int bb = 0; bb < w.n_bands; ++bb) w.k_witness[(page * kBlockTokens + tok) * w.n_bands + bb] = 0;
    if (tok == 0) w.repaired[page] = 1;
  }
}

template <int D, int QT>
void launch_repair_d(const RepairArgs& a, hipStream_t st) {
  const int units = a.d.batch * a.d.n_kv;
  const dim3 block(kRThreads);
  hipLaunchKernelGGL((repair_rank_kernel<D>), dim3(units), block, 0, st, a);
  const dim3 bgrid(a.max_rep * a.tiles, units);
  for (int round = 0; round < 2; ++round) {
    if (a.d.group <= 8) hipLaunchKernelGGL((repair_block_kernel<D, QT, 8>), bgrid, block, 0, st, a, round);
    else hipLaunchKernelGGL((repair_block_kernel<D, QT, kRGMax>), bgrid, block, 0, st, a, round);
    hipLaunchKernelGGL((repair_scan_kernel<D>), dim3(units), block, 0, st, a, round);
  }
  hipLaunchKernelGGL((repair_final_kernel<D>), dim3(units, a.d.group, D / 32), block, 0, st, a);
}

}  // namespace

hipError_t launch_repair(const RepairArgs& a, hipStream_t st) {
  if (a.d.head_dim == 64) {
    if (a.d.q_dtype == WC_F32) launch_repair_d<64, WC_F32>(a, st);
    else launch_repair_d<64, WC_BF16>(a, st);
  } else {
    if (a.d.q_dtype == WC_F32) launch_repair_d<128, WC_F32>(a, st);
    else launch_repair_d<128, WC_BF16>(a, st);
  }
  return hipGetLastError();
}

int repair_max_blocks() { return kRMaxBlocks; }

hipError_t launch_write_back(const WriteBackArgs& w, hipStream_t st) {
  if (w.batch * w.n_kv == 0) return hipSuccess;
  hipLaunchKernelGGL(repair_write_back_kernel, dim3(w.batch * w.n_kv), dim3(kRThreads), 0, st, w);
  return hipGetLastError();
}

size_t repair_unit_bytes(int group, int head_dim, int max_rep, int tiles) {
  const size_t b = kRepHeaderBytes + (size_t)max_rep * tiles * group * (head_dim + 2) * sizeof(double);
  return (b + 255) / 256 * 256;
}

}  // namespace wc
