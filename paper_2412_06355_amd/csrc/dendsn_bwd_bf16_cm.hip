// Backward-kernel instantiations and dispatch for bf16 storage in the
// channel-major layout (X / grad_x [T, batch, C, P, S], stash capacity 4).
// V: bit 0 = Mexican-hat activation, bit 1 = residual dendrite, bits 2-3 =
// log2(KC), bit 4 = channel-major, bit 5 = sigmoid
// surrogate (DENDSN_SG).
// Bit 6 of V = Stateless Dendrite (the runtime v passed in: psi | residual << 1 |
// stateless << 2, mapped by variant_bits).
#include "dendsn_kernels.h"

#ifndef DENDSN_SG
#error "compile once per surrogate: -DDENDSN_SG=0 (atan) or 1 (sigmoid)"
#endif

namespace dendsn {

constexpr int kVS = DENDSN_SG << 5;  // surrogate bit of the variant

template <int BL, int L, int KC>
static hipError_t launch_bwd_cm_v(const dim3& grid, const BwdArgs& ba, int v, size_t lds, hipStream_t stream) {
  constexpr int VK = 16 | ((KC == 1 ? 0 : (KC == 2 ? 1 : 2)) << 2);
  switch (v & 7) {
#define DENDSN_V(n) \
    case n: dendsn_bwd_kernel<bf16_t, BL, L, kVS | VK | variant_bits(n), 4><<<grid, dim3(kThreads), lds, stream>>>(ba); break;
    DENDSN_EACH_VARIANT(DENDSN_V)
#undef DENDSN_V
  }
  return hipGetLastError();
}

hipError_t DENDSN_SG_NAME(launch_bwd_bf16_cm)(const Plan& pl, const BwdArgs& ba, int v, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(pl.ntiles * pl.G));
  if (!pl.cm || pl.KS != 4) return hipErrorInvalidValue;
#define DENDSN_CASE(BL_, L_, KC_) \
  if (pl.BL == BL_ && pl.L == L_ && pl.KC == KC_) return launch_bwd_cm_v<BL_, L_, KC_>(grid, ba, v, size_t(pl.lds), stream);
  DENDSN_CM(DENDSN_CASE)
#undef DENDSN_CASE
  return hipErrorInvalidValue;
}

}  // namespace dendsn
