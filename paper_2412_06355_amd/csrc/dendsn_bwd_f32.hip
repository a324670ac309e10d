// Backward-kernel instantiations and dispatch for f32 storage.
// V: bit 0 = Mexican-hat activation, bit 1 = residual dendrite,
// bit 5 = sigmoid surrogate (DENDSN_SG); KS: stash steps.
// Bit 6 of V = Stateless Dendrite (the runtime v passed in: psi | residual << 1 |
// stateless << 2, mapped by variant_bits).
#include "dendsn_kernels.h"

#ifndef DENDSN_SG
#error "compile once per surrogate: -DDENDSN_SG=0 (atan) or 1 (sigmoid)"
#endif

namespace dendsn {

constexpr int kVS = DENDSN_SG << 5;  // surrogate bit of the variant

template <int BL, int L, int KS>
static hipError_t launch_bwd_v(const dim3& grid, const BwdArgs& ba, int v, size_t lds, hipStream_t stream) {
  switch (v & 7) {
#define DENDSN_V(n) \
    case n: dendsn_bwd_kernel<float, BL, L, kVS | variant_bits(n), KS><<<grid, dim3(kThreads), lds, stream>>>(ba); break;
    DENDSN_EACH_VARIANT(DENDSN_V)
#undef DENDSN_V
  }
  return hipGetLastError();
}

hipError_t DENDSN_SG_NAME(launch_bwd_f32)(const Plan& pl, const BwdArgs& ba, int v, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(pl.ntiles * pl.G));
#define DENDSN_FAST_CASE(BL_, L_)                                                   \
  if (pl.BL == BL_ && pl.L == L_ && pl.fast) {                                      \
    if (pl.KS == 4) return launch_bwd_v<BL_, L_, 4>(grid, ba, v, size_t(pl.lds), stream);           \
    if constexpr (BL_ <= 4)                                                         \
      if (pl.KS == 8) return launch_bwd_v<BL_, L_, 8>(grid, ba, v, size_t(pl.lds), stream);         \
    return hipErrorInvalidValue;                                                    \
  }
#define DENDSN_GENERIC_CASE(BL_, L_)                                                \
  if (pl.BL == BL_ && pl.L == L_ && !pl.fast && pl.KS == DENDSN_GENERIC_KS)         \
    return launch_bwd_v<BL_, L_, DENDSN_GENERIC_KS>(grid, ba, v, size_t(pl.lds), stream);
  DENDSN_FAST_F32(DENDSN_FAST_CASE)
  DENDSN_GENERIC(DENDSN_GENERIC_CASE)
#undef DENDSN_FAST_CASE
#undef DENDSN_GENERIC_CASE
  return hipErrorInvalidValue;
}

}  // namespace dendsn
