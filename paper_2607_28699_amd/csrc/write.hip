// Write path of the certified cache: dithered INT8 quantizer, raw fp8 cast, bf16
// copy, and the residual witness (Sec. 4.2 subtractive dither; Sec. 6.2 research
// kernels and storage side; Sec. 4.1 Eq. witness).  The per-token-head work is in
// write_dev.h; here are the write kernel (D/16 lanes per token-head, the witness
// after a workgroup barrier), the black-box witness and the pair selection.
#include "wc_device.h"
#include "wc_launch.h"
#include "write_dev.h"

namespace wc {

namespace {

constexpr int kWriteThreads = 256;

// Byte transpose of four words (rows t = tokens, bytes c = channels): word c of
// the result holds byte c of w0, w1, w2, w3 -- one channel's codes of a token quad.
__device__ __forceinline__ uint4 transpose_bytes(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3) {
  const uint32_t lo01 = __builtin_amdgcn_perm(w1, w0, 0x05010400u);   // w0.b0 w1.b0 w0.b1 w1.b1
  const uint32_t hi01 = __builtin_amdgcn_perm(w1, w0, 0x07030602u);   // w0.b2 w1.b2 w0.b3 w1.b3
  const uint32_t lo23 = __builtin_amdgcn_perm(w3, w2, 0x05010400u);
  const uint32_t hi23 = __builtin_amdgcn_perm(w3, w2, 0x07030602u);
  return make_uint4(__builtin_amdgcn_perm(lo23, lo01, 0x05040100u), __builtin_amdgcn_perm(lo23, lo01, 0x07060302u),
                    __builtin_amdgcn_perm(hi23, hi01, 0x05040100u), __builtin_amdgcn_perm(hi23, hi01, 0x07060302u));
}

// Workgroup: TH consecutive tokens of one KV head (grid: token blocks x KV heads),
// D/16 lanes per token (codes, scales, witness and the exact copy's keys are
// stored by the token's lanes).  Each token's value row (codes, and the exact
// copy's bf16 values) is staged in LDS; after the barrier, a token quad of the
// workgroup that fills one quad of a page (slots 4s .. 4s+3 in order, the common
// case of a prefill) is stored as whole 16-byte pieces of the page's interleaved
// quad row, any other token element by element.
template <int D, int KIND, typename TIn, bool BYP>
__global__ __launch_bounds__(kWriteThreads) void quantize_write_kernel(WriteArgs a) {
  constexpr int LPT = D / 16;                 // lanes per token
  constexpr int TH = kWriteThreads / LPT;     // tokens per workgroup
  constexpr int NQ = TH / 4;                  // token quads per workgroup
  constexpr bool kCodes = KIND != WC_KIND_BF16;
  __shared__ uint32_t vq_s[kCodes ? TH : 1][D / 4];   // value codes
  __shared__ uint32_t vx_s[TH][D / 2];        // bf16 values of the exact copy (or of a bf16 cache)
  __shared__ int64_t slot_s[TH];

  const int tid = threadIdx.x;
  const int lth = tid / LPT;
  const int g = tid % LPT;
  const int h = blockIdx.y;
  const int64_t tok = (int64_t)blockIdx.x * TH + lth;
  const bool in_range = tok < a.n_tok;
  const bool exact_copy = KIND == WC_KIND_BF16 || a.x_k_data != nullptr;
  const VStage vst{kCodes ? vq_s[lth] : nullptr, exact_copy ? vx_s[lth] : nullptr};
  const int64_t slot = write_token_head<D, KIND, TIn, BYP>(a, in_range ? tok : 0, h, in_range, g, vst);
  if (g == 0) slot_s[lth] = slot;
  __syncthreads();

  // ---- value rows by token quads ----
  {
    // thread (quad q, piece p); a code quad row is D x 4 bytes (D/4 pieces), a bf16 one
    // twice that
    constexpr int PC = D / 4;                 // 16-byte pieces of a code quad row
    static_assert(NQ * PC == kWriteThreads, "one code piece per thread");
    const int q = tid / PC, p = tid % PC;
    const int64_t s0 = slot_s[4 * q];
    bool whole = s0 >= 0 && (s0 & 3) == 0;
#pragma unroll
    for (int t = 1; t < 4; ++t) whole = whole && slot_s[4 * q + t] == s0 + t;
    const int64_t bh0 = whole ? (s0 / kBlockTokens) * a.n_kv + h : 0;
    const int off0 = whole ? (int)(s0 % kBlockTokens) : 0;
    if constexpr (kCodes) {
      // piece p: channels 4p .. 4p+3 of the quad's four tokens
      uint8_t* vpg = reinterpret_cast<uint8_t*>(a.v_data);
      if (whole) {
        const uint4 o = transpose_bytes(vq_s[4 * q][p], vq_s[4 * q + 1][p], vq_s[4 * q + 2][p], vq_s[4 * q + 3][p]);
        *reinterpret_cast<uint4*>(vpg + bh0 * (kBlockTokens * D) + vpage_off(off0, 4 * p, D, 1)) = o;
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int64_t st = slot_s[4 * q + t];
          if (st < 0) continue;
          const int64_t bh = (st / kBlockTokens) * a.n_kv + h;
          const uint32_t w = vq_s[4 * q + t][p];
#pragma unroll
          for (int c = 0; c < 4; ++c)
            vpg[bh * (kBlockTokens * D) + vpage_off((int)(st % kBlockTokens), 4 * p + c, D, 1)] = (uint8_t)(w >> (8 * c));
        }
      }
    }
    if (exact_copy) {
      // pieces p and p + D/4 of the bf16 quad row: channels 2p', 2p'+1 of the four tokens
      uint8_t* xpg = reinterpret_cast<uint8_t*>(KIND == WC_KIND_BF16 ? a.v_data : a.x_v_data);
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int pp = p + half * PC;   // 0 .. D/2 - 1
        if (whole) {
          const uint32_t w0 = vx_s[4 * q][pp], w1 = vx_s[4 * q + 1][pp], w2 = vx_s[4 * q + 2][pp],
                         w3 = vx_s[4 * q + 3][pp];
          const uint4 o = make_uint4(__builtin_amdgcn_perm(w1, w0, 0x05040100u), __builtin_amdgcn_perm(w3, w2, 0x05040100u),
                                     __builtin_amdgcn_perm(w1, w0, 0x07060302u), __builtin_amdgcn_perm(w3, w2, 0x07060302u));
          *reinterpret_cast<uint4*>(xpg + bh0 * (kBlockTokens * D * 2) + vpage_off(off0, 2 * pp, D, 2)) = o;
        } else {
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const int64_t st = slot_s[4 * q + t];
            if (st < 0) continue;
            const int64_t bh = (st / kBlockTokens) * a.n_kv + h;
            const uint32_t w = vx_s[4 * q + t][pp];
#pragma unroll
            for (int c = 0; c < 2; ++c)
              *reinterpret_cast<uint16_t*>(xpg + bh * (kBlockTokens * D * 2) +
                                           vpage_off((int)(st % kBlockTokens), 2 * pp + c, D, 2)) =
                  (uint16_t)(w >> (16 * c));
          }
        }
      }
    }
  }
}

template <typename T>
__device__ __forceinline__ float load_any(const void* p, int64_t i, int dt) {
  if (dt == WC_F32) return reinterpret_cast<const float*>(p)[i];
  if (dt == WC_BF16) return bf16_to_f32(reinterpret_cast<const uint16_t*>(p)[i]);
  return f16_to_f32(reinterpret_cast<const uint16_t*>(p)[i]);
}

__global__ __launch_bounds__(256) void witness_kernel(WitnessArgs a) {
  const int64_t item = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (item >= a.n_vec * a.n_bands) return;
  const int64_t vec = item / a.n_bands;
  const int b = (int)(item % a.n_bands);
  const int per_band = a.head_dim / a.n_bands;
  double acc = 0.0;   // float64: the inputs' difference is exact, the round-up is taken once
  for (int kk = 0; kk < per_band; ++kk) {
    const int c = band_channel(b, kk, a.head_dim, a.n_bands, a.interleaved);
    const double r = (double)load_any<float>(a.xhat, vec * a.head_dim + c, a.xhat_dtype) -
                     (double)load_any<float>(a.x, vec * a.head_dim + c, a.x_dtype);
    acc += r * r;
  }
  a.w_out[item] = f16_round_up_f64(sqrt(acc));
}

template <int D, int KIND, bool BYP>
hipError_t launch_write_dtb(const WriteArgs& a, hipStream_t st) {
  constexpr int TH = kWriteThreads / (D / 16);
  const dim3 grid((unsigned)((a.n_tok + TH - 1) / TH), (unsigned)a.n_kv);
  if (a.in_dtype == WC_F32)
    hipLaunchKernelGGL((quantize_write_kernel<D, KIND, float, BYP>), grid, dim3(kWriteThreads), 0, st, a);
  else
    hipLaunchKernelGGL((quantize_write_kernel<D, KIND, uint16_t, BYP>), grid, dim3(kWriteThreads), 0, st, a);
  return hipGetLastError();
}

template <int D, int KIND>
hipError_t launch_write_dt(const WriteArgs& a, hipStream_t st) {
  // (bypassed pairs: INT8 keys only)
  if constexpr (KIND == WC_KIND_INT8_DITHER)
    if (a.n_pairs > 0) return launch_write_dtb<D, KIND, true>(a, st);
  return launch_write_dtb<D, KIND, false>(a, st);
}

template <int D>
hipError_t launch_write_d(const WriteArgs& a, hipStream_t st) {
  switch (a.kind) {
    case WC_KIND_INT8_DITHER: return launch_write_dt<D, WC_KIND_INT8_DITHER>(a, st);
    case WC_KIND_FP8_RAW: return launch_write_dt<D, WC_KIND_FP8_RAW>(a, st);
    default: return launch_write_dt<D, WC_KIND_BF16>(a, st);
  }
}

}  // namespace

hipError_t launch_quantize_write(const WriteArgs& a, hipStream_t st) {
  if (a.n_tok == 0) return hipSuccess;
  return a.head_dim == 64 ? launch_write_d<64>(a, st) : launch_write_d<128>(a, st);
}

// Fixed outlier pairs of each KV head (Sec. 6.2 fixed-channel bypass), in two
// passes so that the sum over many rows uses the whole GPU and stays
// deterministic: (1) workgroup (chunk c, head h) sums the float64 energies
// ||(k_t)_pair j||^2 of all D/2 pairs over its rows into part[h][c][j] (thread =
// pair x row stream, streams added in a fixed order); (2) one wave per head adds
// the chunks in order and takes the m largest (ties to the lower index), written
// in ascending order.
constexpr int kEnThreads = 256;

template <int D, typename TIn>
__global__ __launch_bounds__(kEnThreads) void pair_energy_kernel(SelectArgs a) {
  constexpr int NP = D / 2;
  constexpr int TS = kEnThreads / NP;
  __shared__ double e_s[TS][NP];
  const int c = blockIdx.x, h = blockIdx.y;
  const int tid = threadIdx.x;
  const int j = tid % NP, ts = tid / NP;
  const int c0 = pair_channel(j, 0, D, a.interleaved), c1 = pair_channel(j, 1, D, a.interleaved);
  const int64_t rows = (a.n_tok + a.n_chunks - 1) / a.n_chunks;
  const int64_t r0 = (int64_t)c * rows, r1 = min(a.n_tok, r0 + rows);
  const TIn* base = reinterpret_cast<const TIn*>(a.k) + (int64_t)h * D;
  const int64_t stride = (int64_t)a.n_kv * D;
  auto val = [&](int64_t t, int ch) -> double {
    const TIn* row = base + t * stride;
    if constexpr (sizeof(TIn) == 4) return (double)reinterpret_cast<const float*>(row)[ch];
    else return (double)bf16_to_f32(reinterpret_cast<const uint16_t*>(row)[ch]);
  };
  double acc = 0.0;
  int64_t t = r0 + ts;
  for (; t + 3 * TS < r1; t += 4 * TS) {   // four rows in flight
    double x[8];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      x[2 * u] = val(t + u * TS, c0);
      x[2 * u + 1] = val(t + u * TS, c1);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) acc = fma(x[u], x[u], acc);
  }
  for (; t < r1; t += TS) {
    const double x0 = val(t, c0), x1 = val(t, c1);
    acc = fma(x1, x1, fma(x0, x0, acc));
  }
  e_s[ts][j] = acc;
  __syncthreads();
  if (tid < NP) {
    double e = 0.0;
    for (int s2 = 0; s2 < TS; ++s2) e += e_s[s2][tid];
    a.part[((int64_t)h * a.n_chunks + c) * NP + tid] = e;
  }
}

__global__ __launch_bounds__(64) void select_pairs_kernel(SelectArgs a) {
  const int NP = a.head_dim / 2;
  const int h = blockIdx.x, lane = threadIdx.x;
  double e = -1.0;   // lanes past the last pair never win (energies are >= 0)
  if (lane < NP) {
    e = 0.0;
    for (int c = 0; c < a.n_chunks; ++c) e += a.part[((int64_t)h * a.n_chunks + c) * NP + lane];
  }
  uint64_t chosen = 0;
  for (int i = 0; i < a.m; ++i) {
    double be = e;
    int bj = lane;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const double oe = __shfl_xor(be, o, 64);
      const int oj = __shfl_xor(bj, o, 64);
      if (oe > be || (oe == be && oj < bj)) {
        be = oe;
        bj = oj;
      }
    }
    chosen |= 1ull << bj;
    if (lane == bj) e = -2.0;
  }
  if ((chosen >> lane) & 1ull)
    a.pairs_out[(int64_t)h * a.m + __popcll(chosen & ((1ull << lane) - 1ull))] = lane;
}

int select_chunks(int64_t n_tok) {
  const int64_t c = (n_tok + 2047) / 2048;
  return (int)(c < 1 ? 1 : (c > 64 ? 64 : c));
}

hipError_t launch_select_pairs(const SelectArgs& a, hipStream_t st) {
  const dim3 grid(a.n_chunks, a.n_kv), block(kEnThreads);
  if (a.head_dim == 128) {
    if (a.in_dtype == WC_F32) hipLaunchKernelGGL((pair_energy_kernel<128, float>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((pair_energy_kernel<128, uint16_t>), grid, block, 0, st, a);
  } else {
    if (a.in_dtype == WC_F32) hipLaunchKernelGGL((pair_energy_kernel<64, float>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((pair_energy_kernel<64, uint16_t>), grid, block, 0, st, a);
  }
  hipLaunchKernelGGL(select_pairs_kernel, dim3(a.n_kv), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_witness(const WitnessArgs& a, hipStream_t st) {
  const int64_t items = a.n_vec * a.n_bands;
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(witness_kernel, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace wc
