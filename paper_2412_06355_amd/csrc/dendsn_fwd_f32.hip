// Forward-kernel instantiations and dispatch for f32 storage.
// V: bit 0 = Mexican-hat activation, bit 1 = residual dendrite.
// Bit 6 of V = Stateless Dendrite (the runtime v passed in: psi | residual << 1 |
// stateless << 2, mapped by variant_bits).
#include "dendsn_kernels.h"

namespace dendsn {

template <int BL, int L>
static hipError_t launch_fwd_v(const dim3& grid, const FwdArgs& fa, int v, size_t lds, hipStream_t stream) {
  switch (v & 7) {
#define DENDSN_V(n) \
    case n: dendsn_fwd_kernel<float, BL, L, variant_bits(n)><<<grid, dim3(kThreads), lds, stream>>>(fa); break;
    DENDSN_EACH_VARIANT(DENDSN_V)
#undef DENDSN_V
  }
  return hipGetLastError();
}

hipError_t launch_fwd_f32(const Plan& pl, const FwdArgs& fa, int v, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(pl.ntiles * pl.G));
#define DENDSN_CASE(BL_, L_) \
  if (pl.BL == BL_ && pl.L == L_) return launch_fwd_v<BL_, L_>(grid, fa, v, size_t(pl.lds), stream);
  DENDSN_FAST_F32_FWD(DENDSN_CASE)
  DENDSN_GENERIC(DENDSN_CASE)
#undef DENDSN_CASE
  return hipErrorInvalidValue;
}

}  // namespace dendsn
