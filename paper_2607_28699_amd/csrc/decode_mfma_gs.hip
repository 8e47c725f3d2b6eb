// Metered decode on the matrix cores over a group-scaled INT8 cache (Sec. 6.2
// storage side, Table 4): the GS instantiations of the kernel in decode_mfma.h.
#include "decode_mfma.h"

namespace wc {

namespace {

template <bool HALF, bool VM>
void launch_gs(const DecodeArgs& a, bool tb, bool byp, const dim3& grid, const dim3& block, hipStream_t st) {
  // repair marks: a separate instantiation, as for the per-token caches
  if (a.repaired != nullptr) launch_decode_mfma_int8<HALF, VM, true, true>(a, tb, byp, grid, block, st);
  else launch_decode_mfma_int8<HALF, VM, false, true>(a, tb, byp, grid, block, st);
}

}  // namespace

void launch_decode_mfma_gs(const DecodeArgs& a, bool tb, bool byp, bool vm, const dim3& grid, const dim3& block,
                           hipStream_t st) {
  if (a.group <= 8) {
    if (vm) launch_gs<true, true>(a, tb, byp, grid, block, st);
    else launch_gs<true, false>(a, tb, byp, grid, block, st);
  } else {
    if (vm) launch_gs<false, true>(a, tb, byp, grid, block, st);
    else launch_gs<false, false>(a, tb, byp, grid, block, st);
  }
}

}  // namespace wc
