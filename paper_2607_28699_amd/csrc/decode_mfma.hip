// Metered decode attention on the matrix cores: the per-token-scale and bf16
// variants and the dispatch (the kernel itself is in decode_mfma.h).
#include "decode_mfma.h"

namespace wc {

bool step_write_fusable(const DecodeArgs& a) {
  // the kernel variants that carry the step write: Tier A over a cache without
  // bypassed pairs or group scales
  return a.use_mfma && mfma_decode_supported(a) && a.tierb_delta <= 0.0f && a.meter_v == nullptr &&
         a.n_pairs == 0 && a.group_scales == 0;
}

bool mfma_decode_supported(const DecodeArgs& a) {
  return a.head_dim == kD && a.q_dtype == WC_BF16 && a.group <= 16 &&
         (a.kind == WC_KIND_BF16 || a.n_bands == 8 || a.n_bands == 16) &&
         (a.group_scales == 0 || a.kind == WC_KIND_INT8_DITHER);
}

template <bool HALF, bool VM, bool REP>
void launch_decode_mfma_g(const DecodeArgs& a, bool metered, bool tb, bool byp, const dim3& grid,
                          const dim3& block, hipStream_t st) {
  if (!metered) {
    if constexpr (!VM && !REP)
      hipLaunchKernelGGL((decode_mfma_kernel<WC_KIND_BF16, false, HALF, false, false, false, false, false>), grid, block, 0,
                         st, a);
  } else if (a.kind == WC_KIND_FP8_RAW) {
    hipLaunchKernelGGL((decode_mfma_kernel<WC_KIND_FP8_RAW, true, HALF, false, false, VM, REP, false>), grid, block, 0, st,
                       a);
  } else {
    launch_decode_mfma_int8<HALF, VM, REP, false>(a, tb, byp, grid, block, st);
  }
}

template <bool HALF, bool VM>
void launch_decode_mfma_r(const DecodeArgs& a, bool metered, bool tb, bool byp, const dim3& grid,
                          const dim3& block, hipStream_t st) {
  // repair marks apply to the quantized caches of the metered decodes
  if (metered && a.repaired != nullptr) launch_decode_mfma_g<HALF, VM, true>(a, metered, tb, byp, grid, block, st);
  else launch_decode_mfma_g<HALF, VM, false>(a, metered, tb, byp, grid, block, st);
}

bool spec_decode_fusable(const DecodeArgs& am, const DecodeArgs& ax) {
  return am.use_mfma && ax.use_mfma && mfma_decode_supported(am) && mfma_decode_supported(ax) &&
         (am.kind == WC_KIND_INT8_DITHER || am.kind == WC_KIND_FP8_RAW) && ax.kind == WC_KIND_BF16 &&
         am.tierb_delta <= 0.0f && am.meter_v == nullptr && am.n_pairs == 0 && am.group_scales == 0 &&
         am.repaired == nullptr && am.group == ax.group && am.n_splits == ax.n_splits;
}

hipError_t launch_decode_spec(const DecodeArgs& am, const DecodeArgs& ax, hipStream_t st) {
  const uint32_t nb = (uint32_t)am.n_splits * (uint32_t)am.batch * (uint32_t)am.n_kv;
  const dim3 grid(2 * nb), block(64 * kWaves);
  const bool fp8 = am.kind == WC_KIND_FP8_RAW;
  if (am.group <= 8) {
    if (fp8) hipLaunchKernelGGL((decode_spec_kernel<WC_KIND_FP8_RAW, true>), grid, block, 0, st, am, ax, nb);
    else hipLaunchKernelGGL((decode_spec_kernel<WC_KIND_INT8_DITHER, true>), grid, block, 0, st, am, ax, nb);
  } else {
    if (fp8) hipLaunchKernelGGL((decode_spec_kernel<WC_KIND_FP8_RAW, false>), grid, block, 0, st, am, ax, nb);
    else hipLaunchKernelGGL((decode_spec_kernel<WC_KIND_INT8_DITHER, false>), grid, block, 0, st, am, ax, nb);
  }
  return hipGetLastError();
}

hipError_t launch_decode_mfma(const DecodeArgs& a, bool metered, hipStream_t st) {
  const dim3 grid(a.n_splits, a.batch * a.n_kv);   // workgroup order: decode_position()
  const dim3 block(64 * kWaves);
  const bool tb = metered && a.tierb_delta > 0.0f;   // Tier B: INT8 dithered cache only
  const bool byp = metered && a.n_pairs > 0;        // bypassed pairs: INT8 keys only
  const bool vm = metered && a.meter_v != nullptr;    // value side
  if (metered && a.group_scales != 0) {
    launch_decode_mfma_gs(a, tb, byp, vm, grid, block, st);
  } else if (a.group <= 8) {
    if (vm) launch_decode_mfma_r<true, true>(a, metered, tb, byp, grid, block, st);
    else launch_decode_mfma_r<true, false>(a, metered, tb, byp, grid, block, st);
  } else {
    if (vm) launch_decode_mfma_r<false, true>(a, metered, tb, byp, grid, block, st);
    else launch_decode_mfma_r<false, false>(a, metered, tb, byp, grid, block, st);
  }
  return hipGetLastError();
}

}  // namespace wc
