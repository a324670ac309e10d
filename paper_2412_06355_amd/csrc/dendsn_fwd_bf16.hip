// Forward-kernel instantiations and dispatch for bf16 storage.
// V: bit 0 = Mexican-hat activation, bit 1 = residual dendrite.
#include "dendsn_kernels.h"

namespace dendsn {

template <int BL, int L>
static hipError_t launch_fwd_v(const dim3& grid, const FwdArgs& fa, int v, size_t lds, hipStream_t stream) {
  switch (v) {
    case 0: dendsn_fwd_kernel<bf16_t, BL, L, 0><<<grid, dim3(kThreads), lds, stream>>>(fa); break;
    case 1: dendsn_fwd_kernel<bf16_t, BL, L, 1><<<grid, dim3(kThreads), lds, stream>>>(fa); break;
    case 2: dendsn_fwd_kernel<bf16_t, BL, L, 2><<<grid, dim3(kThreads), lds, stream>>>(fa); break;
    case 3: dendsn_fwd_kernel<bf16_t, BL, L, 3><<<grid, dim3(kThreads), lds, stream>>>(fa); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_fwd_bf16(const Plan& pl, const FwdArgs& fa, int v, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(pl.ntiles * pl.G));
#define DENDSN_CASE(BL_, L_) \
  if (pl.BL == BL_ && pl.L == L_) return launch_fwd_v<BL_, L_>(grid, fa, v, size_t(pl.lds), stream);
  DENDSN_FAST_BF16(DENDSN_CASE)
  DENDSN_GENERIC(DENDSN_CASE)
#undef DENDSN_CASE
  return hipErrorInvalidValue;
}

}  // namespace dendsn
