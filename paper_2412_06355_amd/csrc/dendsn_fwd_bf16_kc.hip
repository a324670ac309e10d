// Forward-kernel instantiations and dispatch for bf16 storage with KC = 2 or 4
// compartments per branch.  V: bit 0 = Mexican-hat activation, bit 1 = residual
// dendrite, bits 2-3 = log2(KC).
// Bit 6 of V = Stateless Dendrite (the runtime v passed in: psi | residual << 1 |
// stateless << 2, mapped by variant_bits).
#include "dendsn_kernels.h"

namespace dendsn {

template <int BL, int L, int KC>
static hipError_t launch_fwd_kc_v(const dim3& grid, const FwdArgs& fa, int v, size_t lds, hipStream_t stream) {
  constexpr int VK = (KC == 2 ? 1 : 2) << 2;
  switch (v & 7) {
#define DENDSN_V(n) \
    case n: dendsn_fwd_kernel<bf16_t, BL, L, VK | variant_bits(n)><<<grid, dim3(kThreads), lds, stream>>>(fa); break;
    DENDSN_EACH_VARIANT(DENDSN_V)
#undef DENDSN_V
  }
  return hipGetLastError();
}

hipError_t launch_fwd_bf16_kc(const Plan& pl, const FwdArgs& fa, int v, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(pl.ntiles * pl.G));
#define DENDSN_FAST_CASE(BL_, L_, KC_) \
  if (pl.fast && pl.BL == BL_ && pl.L == L_ && pl.KC == KC_) return launch_fwd_kc_v<BL_, L_, KC_>(grid, fa, v, size_t(pl.lds), stream);
#define DENDSN_GENERIC_CASE(BL_, L_, KC_) \
  if (!pl.fast && pl.BL == BL_ && pl.L == L_ && pl.KC == KC_) return launch_fwd_kc_v<BL_, L_, KC_>(grid, fa, v, size_t(pl.lds), stream);
  DENDSN_KC_FAST_BF16(DENDSN_FAST_CASE)
  DENDSN_KC_GENERIC(DENDSN_GENERIC_CASE)
#undef DENDSN_FAST_CASE
#undef DENDSN_GENERIC_CASE
  return hipErrorInvalidValue;
}

}  // namespace dendsn
