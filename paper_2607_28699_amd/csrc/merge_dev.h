// Split-KV merge statistics and the gate (Sec. 6.2: the meter's numerator
// merges across splits exactly like the output; Sec. 6 meter loop: the gate at
// tau, any of a KV head's query heads).  One wave computes the statistics of one
// (sequence, query head) from its split records in a fixed order -- split j at
// lane j % 64, the largest split max first, then the LSE-weighted sums by one
// shuffle tree per 64 splits -- so every kernel that forms them (the split merge,
// the gate in the exact fallback's prologue, the final merge of a certified step)
// gets the same bits, and the gate a kernel decides is the one the merged meter
// shows.
#pragma once

#include <float.h>

#include "wc_launch.h"

namespace wc {

struct SplitStats {
  float M;      // largest split max (natural-log units); -inf without splits
  float l, n;   // sum_j e^{m_j - M} l_j, and the meter numerators likewise
  float e, v;   // value side: weighted residual sum, largest stored value norm
};

// One butterfly step over the wave: op(x, the value of lane i ^ O), in every lane.
// O = 1, 2: quad permutes; O = 4: two row shifts by 4, one for each half of every
// 8-lane group; O = 8: a row rotation by 8 (DPP); O = 16, 32: gfx950's lane-group
// swaps, which leave a lane's own value and its partner's in the two results (in
// that order in the lower lane group of each pair, reversed in the upper one: op
// is commutative).  No step goes through LDS.
template <int O, typename Op>
__device__ __forceinline__ float butterfly(float x, Op op) {
  const int v = __builtin_bit_cast(int, x);
  if constexpr (O == 16 || O == 32) {
    const auto p = O == 16 ? __builtin_amdgcn_permlane16_swap(v, v, false, false)
                           : __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return op(__builtin_bit_cast(float, (int)p[0]), __builtin_bit_cast(float, (int)p[1]));
  } else {
    int r;
    if constexpr (O == 1) {
      r = __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);
    } else if constexpr (O == 2) {
      r = __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);
    } else if constexpr (O == 4) {
      r = __builtin_amdgcn_update_dpp(v, v, 0x104, 0xF, 0x5, false);   // banks 0, 2: lane + 4
      r = __builtin_amdgcn_update_dpp(r, v, 0x114, 0xF, 0xA, false);   // banks 1, 3: lane - 4
    } else {
      static_assert(O == 8, "butterfly steps 1 .. 32");
      r = __builtin_amdgcn_mov_dpp(v, 0x128, 0xF, 0xF, false);
    }
    return op(x, __builtin_bit_cast(float, r));
  }
}

struct AddOp {
  __device__ float operator()(float a, float b) const { return a + b; }
};
struct MaxOp {
  __device__ float operator()(float a, float b) const { return fmaxf(a, b); }
};

// x plus, or the max of x and, the value of lane i ^ O.
template <int O>
__device__ __forceinline__ float bfly_add(float x) {
  return butterfly<O>(x, AddOp{});
}
template <int O>
__device__ __forceinline__ float bfly_max(float x) {
  return butterfly<O>(x, MaxOp{});
}

// One butterfly step of the weighted scalars' sums (and the value norms' max).
template <bool METER, bool VM, int O>
__device__ __forceinline__ void reduce_step(float& dl, float& dn, float& de, float& dv) {
  dl = butterfly<O>(dl, AddOp{});
  if constexpr (METER) dn = butterfly<O>(dn, AddOp{});
  if constexpr (VM) {
    de = butterfly<O>(de, AddOp{});
    dv = butterfly<O>(dv, MaxOp{});
  }
}

// Max over the wave by the same butterfly.
__device__ __forceinline__ float butterfly_max(float m) {
  m = butterfly<1>(m, MaxOp{});
  m = butterfly<2>(m, MaxOp{});
  m = butterfly<4>(m, MaxOp{});
  m = butterfly<8>(m, MaxOp{});
  m = butterfly<16>(m, MaxOp{});
  return butterfly<32>(m, MaxOp{});
}

// Adds the weighted scalars of one record per lane (one butterfly over the wave).
// The products are rounded before the butterfly: fused into its first add, lane i
// would form fma(w_i, y_i, w_j y_j) and lane j fma(w_j, y_j, w_i y_i), and the two
// halves of each pair would then hold sums one ulp apart.
template <bool METER, bool VM>
__device__ __forceinline__ void reduce_stats(SplitStats& s, float w, const float4& t, float tv) {
#pragma clang fp contract(off)
  float dl = w * t.y, dn = METER ? w * t.z : 0.0f, de = VM ? w * t.w : 0.0f, dv = tv;
  reduce_step<METER, VM, 1>(dl, dn, de, dv);
  reduce_step<METER, VM, 2>(dl, dn, de, dv);
  reduce_step<METER, VM, 4>(dl, dn, de, dv);
  reduce_step<METER, VM, 8>(dl, dn, de, dv);
  reduce_step<METER, VM, 16>(dl, dn, de, dv);
  reduce_step<METER, VM, 32>(dl, dn, de, dv);
  s.l += dl;
  if constexpr (METER) s.n += dn;
  if constexpr (VM) {
    s.e += de;
    s.v = fmaxf(s.v, dv);
  }
}

// Statistics of at most 64 splits whose scalars (t: max, weight sum, meter
// numerator, value residual sum; tv: value norm) lane j holds for split j (lanes
// at or past ns are left out).
template <bool METER, bool VM>
__device__ __forceinline__ SplitStats stats_of_lanes(float4 t, float tv, int ns, int lane) {
  SplitStats s{-INFINITY, 0.0f, 0.0f, 0.0f, 0.0f};
  if (lane >= ns) {
    t = make_float4(-INFINITY, 0.0f, 0.0f, 0.0f);
    tv = 0.0f;
  }
  s.M = butterfly_max(t.x);
  const float w = t.x == -INFINITY ? 0.0f : __expf(t.x - s.M);
  reduce_stats<METER, VM>(s, w, t, tv);
  return s;
}

// stats_of_lanes for up to 32 splits in each half of the wave (split j at lane j
// of the half): the butterfly stops at step 16, so each half holds its own
// records' statistics.  They are the bits stats_of_lanes gives for the same
// records (its step 32 would only add the other half's zeros and -inf maxima).
__device__ __forceinline__ SplitStats stats_of_half_lanes(float4 t, int ns, int hl) {
#pragma clang fp contract(off)
  SplitStats s{-INFINITY, 0.0f, 0.0f, 0.0f, 0.0f};
  if (hl >= ns) t = make_float4(-INFINITY, 0.0f, 0.0f, 0.0f);
  float m = t.x;
  m = butterfly<1>(m, MaxOp{});
  m = butterfly<2>(m, MaxOp{});
  m = butterfly<4>(m, MaxOp{});
  m = butterfly<8>(m, MaxOp{});
  s.M = butterfly<16>(m, MaxOp{});
  const float w = t.x == -INFINITY ? 0.0f : __expf(t.x - s.M);
  float dl = w * t.y, dn = w * t.z, de = 0.0f, dv = 0.0f;
  reduce_step<true, false, 1>(dl, dn, de, dv);
  reduce_step<true, false, 2>(dl, dn, de, dv);
  reduce_step<true, false, 4>(dl, dn, de, dv);
  reduce_step<true, false, 8>(dl, dn, de, dv);
  reduce_step<true, false, 16>(dl, dn, de, dv);
  s.l += dl;
  s.n += dn;
  return s;
}

// Statistics of the first ns records at rec0 (record stride R floats, the
// scalars at offset D: max, weight sum, meter numerator, value residual sum,
// value norm) of the n_avail >= ns records the workspace holds.  Whole wave;
// every lane returns the same values.  Up to 64 records are read in one round
// trip (records past ns are read -- they exist -- but not used).
template <bool METER, bool VM>
__device__ __forceinline__ SplitStats split_stats(const float* rec0, int64_t R, int D, int ns, int n_avail,
                                                  int lane) {
  if (n_avail <= 64) {
    const int jr = min(lane, n_avail - 1);
    const float4 t = *reinterpret_cast<const float4*>(rec0 + (int64_t)jr * R + D);
    const float tv = VM ? rec0[(int64_t)jr * R + D + 4] : 0.0f;
    return stats_of_lanes<METER, VM>(t, tv, ns, lane);
  }
  SplitStats s{-INFINITY, 0.0f, 0.0f, 0.0f, 0.0f};
  for (int j0 = 0; j0 < ns; j0 += 64) {
    const int j = j0 + lane;
    const float m = j < ns ? rec0[(int64_t)j * R + D] : -INFINITY;
    s.M = fmaxf(s.M, m);
  }
  s.M = butterfly_max(s.M);
  for (int j0 = 0; j0 < ns; j0 += 64) {
    const int j = j0 + lane;
    const bool ok = j < ns;
    const float4 t = ok ? *reinterpret_cast<const float4*>(rec0 + (int64_t)j * R + D)
                        : make_float4(-INFINITY, 0.0f, 0.0f, 0.0f);
    const float w = t.x == -INFINITY ? 0.0f : __expf(t.x - s.M);
    reduce_stats<METER, VM>(s, w, t, VM && ok ? rec0[(int64_t)j * R + D + 4] : 0.0f);
  }
  return s;
}

// raw = (A-1)(A+1)/2 with A - 1 = n / l (+inf on overflow or a NaN numerator),
// 0 without splits.
__device__ __forceinline__ float raw_of(const SplitStats& s, int ns) {
  if (ns <= 0) return 0.0f;
  const float nt = isnan(s.n) ? INFINITY : s.n;
  const float am1 = nt / s.l;
  float raw = 0.5f * am1 * (2.0f + am1);
  if (!(raw <= FLT_MAX)) raw = INFINITY;
  return raw;
}

// Value meter: sum_t ptilde_t rho_t over the largest stored value norm (0/0 = 0).
__device__ __forceinline__ float meter_v_of(const SplitStats& s, int ns) {
  const float ev = ns > 0 ? s.e / s.l : 0.0f;
  float mv = s.v > 0.0f ? ev / s.v : (ev > 0.0f ? INFINITY : 0.0f);
  if (isnan(mv)) mv = INFINITY;
  return mv;
}

// The gate of one query head: meter (raw for tau >= 1) above tau, or (joint
// gate) the value meter above tau_v.
__device__ __forceinline__ bool gated_of(float raw, float mv, float tau, bool vm, float tau_v) {
  const float meter = fminf(1.0f, raw);
  return (tau >= 1.0f ? raw : meter) > tau || (vm && mv > tau_v);
}

// Active splits of a sequence of length L.
__device__ __forceinline__ int active_splits(int L, int split_tokens, int n_splits) {
  return min((L + split_tokens - 1) / split_tokens, n_splits);
}

// Gate of one (sequence b, KV head kv) from the metered decode's records
// (a.gate_part, the same split layout), evaluated by a 4-wave workgroup of the
// exact fallback before it reads anything: each wave takes query heads wave,
// wave + 4, ...; the workgroup of split 0 stores mask_q of the unit's heads and
// mask_kv of the unit.  Returns whether the unit is routed (uniform over the
// workgroup; contains a barrier).
__device__ __forceinline__ bool unit_gate(const DecodeArgs& a, int b, int kv, int split, int wave, int lane,
                                          int* flag_s) {
  if (threadIdx.x == 0) *flag_s = 0;
  __syncthreads();
  const int64_t R = (int64_t)partial_record_floats(a.head_dim);
  const float* base = a.gate_part + (int64_t)(b * a.n_q + kv * a.group) * a.n_splits * R;
  bool any = false;
  auto decide = [&](const SplitStats& s, int hh, int ns) {
    const bool g = gated_of(raw_of(s, ns), 0.0f, a.gate_tau, false, 0.0f);
    any |= g;
    if (lane == 0 && split == 0) a.gate_mask_q[b * a.n_q + kv * a.group + hh] = g ? 1 : 0;
  };
  if (a.n_splits <= 64) {
    // every head of this wave in one round trip (up to 4: G <= 16), the length too;
    // the loads are unconditional (past the last head: its record again), so that
    // none waits for another
    const int jr = min(lane, a.n_splits - 1);
    float4 t[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int hc = min(wave + 4 * i, a.group - 1);
      t[i] = *reinterpret_cast<const float4*>(base + ((int64_t)hc * a.n_splits + jr) * R + a.head_dim);
    }
    const int ns = active_splits(a.seq_lens[b], a.split_tokens, a.n_splits);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (wave + 4 * i < a.group) decide(stats_of_lanes<true, false>(t[i], 0.0f, ns, lane), wave + 4 * i, ns);
  } else {
    const int ns = active_splits(a.seq_lens[b], a.split_tokens, a.n_splits);
    for (int hh = wave; hh < a.group; hh += 4)
      decide(split_stats<true, false>(base + (int64_t)hh * a.n_splits * R, R, a.head_dim, ns, a.n_splits, lane), hh,
             ns);
  }
  if (any && lane == 0) atomicOr(flag_s, 1);
  __syncthreads();
  const bool routed = *flag_s != 0;
  if (split == 0 && threadIdx.x == 0) a.gate_mask_kv[b * a.n_kv + kv] = routed ? 1 : 0;
  return routed;
}

// The same gate as unit_gate, decided by one wave without barriers (the final
// merge of a speculative certified step): every query head of the unit from the
// metered records a.gate_part, up to 64 splits of all heads in one load round
// trip (more splits: split_stats per head); lane 0 stores mask_q of the unit's
// heads and mask_kv (every wave that calls it stores the same values).  Returns
// whether the unit is routed (uniform over the wave); own_stats receives head
// own's statistics.
__device__ __forceinline__ bool unit_gate_wave(const DecodeArgs& a, int b, int kv, int lane, int own,
                                               SplitStats* own_stats) {
  const int64_t R = (int64_t)partial_record_floats(a.head_dim);
  const float* base = a.gate_part + (int64_t)(b * a.n_q + kv * a.group) * a.n_splits * R;
  const int ns = active_splits(a.seq_lens[b], a.split_tokens, a.n_splits);
  bool any = false;
  auto decide = [&](const SplitStats& s, int hh) {
    const bool g = gated_of(raw_of(s, ns), 0.0f, a.gate_tau, false, 0.0f);
    any |= g;
    if (hh == own) *own_stats = s;
    if (lane == 0) a.gate_mask_q[b * a.n_q + kv * a.group + hh] = g ? 1 : 0;
  };
  if (a.n_splits <= 32) {
    // two heads at a time, head 2p in lanes 0 .. 31 and head 2p + 1 in lanes 32 .. 63
    // (split j at lane j of the half); each head's statistics are then read from the
    // first lane of its half
    const int hl = lane & 31, jr = min(hl, a.n_splits - 1);
    float4 t[8];   // (G <= 16; unconditional loads, past the last head its record again)
#pragma unroll
    for (int p2 = 0; p2 < 8; ++p2) {
      const int hc = min(2 * p2 + (lane >> 5), a.group - 1);
      t[p2] = *reinterpret_cast<const float4*>(base + ((int64_t)hc * a.n_splits + jr) * R + a.head_dim);
    }
    auto from_lane = [](const SplitStats& s, int src) {
      const auto rl = [src](float x) {
        return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), src));
      };
      return SplitStats{rl(s.M), rl(s.l), rl(s.n), 0.0f, 0.0f};
    };
#pragma unroll
    for (int p2 = 0; p2 < 8; ++p2) {
      if (2 * p2 < a.group) {
        const SplitStats s = stats_of_half_lanes(t[p2], ns, hl);
        decide(from_lane(s, 0), 2 * p2);
        if (2 * p2 + 1 < a.group) decide(from_lane(s, 32), 2 * p2 + 1);
      }
    }
  } else if (a.n_splits <= 64) {
    const int jr = min(lane, a.n_splits - 1);
    float4 t[16];   // (G <= 16; unconditional loads, past the last head its record again)
#pragma unroll
    for (int hh = 0; hh < 16; ++hh) {
      const int hc = min(hh, a.group - 1);
      t[hh] = *reinterpret_cast<const float4*>(base + ((int64_t)hc * a.n_splits + jr) * R + a.head_dim);
    }
#pragma unroll
    for (int hh = 0; hh < 16; ++hh)
      if (hh < a.group) decide(stats_of_lanes<true, false>(t[hh], 0.0f, ns, lane), hh);
  } else {
    for (int hh = 0; hh < a.group; ++hh)
      decide(split_stats<true, false>(base + (int64_t)hh * a.n_splits * R, R, a.head_dim, ns, a.n_splits, lane), hh);
  }
  if (lane == 0) a.gate_mask_kv[b * a.n_kv + kv] = any ? 1 : 0;
  return any;
}

}  // namespace wc
